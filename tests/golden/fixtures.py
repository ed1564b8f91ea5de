"""Reader for the small text fixtures in this folder."""

import os

HERE = os.path.dirname(os.path.abspath(__file__))


def _value(tok):
    if tok.startswith("0x"):
        return int(tok, 16)
    if any(c in tok for c in ".eE"):
        return float(tok)
    return int(tok)


def load(name):
    """Parse a fixture file into {case: {key: [values]}}."""
    cases = {}
    cur = None
    with open(os.path.join(HERE, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            if line.startswith("[") and line.endswith("]"):
                cur = cases.setdefault(line[1:-1], {})
                continue
            key, vals = line.split("=", 1)
            cur[key.strip()] = [_value(t) for t in vals.split()]
    return cases
