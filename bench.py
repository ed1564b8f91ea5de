#!/usr/bin/env python3
"""W4A4 linear benchmark on one MI355X: effective TOPS on the FLUX-12B MLP linears.

One step = the whole hot path (per-token int4 quantisation of the activations,
int4 x int4 contraction with exact accumulation, fused dequantising epilogue)
for both FLUX-12B MLP linears back-to-back:
  up:   X [4608, 3072] -> N = 12288, with bias
  down: X [9216, 12288] -> N = 3072 (two images)
Weights are packed once before timing (offline, as at model load).  Inputs are
seeded synthetic tensors already resident in HBM.

The library computes the layer on two engines with bit-identical results:
  * bf6:  codes carried as BF6 on gfx950's 6-bit MFMA (fp32 accumulation,
          exact for integer codes), the faster one, timed as `value`;
  * int8: packed int4 codes widened to int8 for the int8 MFMA (int32
          accumulation), reported beside it under `engines`.

Timing protocol.  The first tens of steps of a process run up to 30% slower
than the rest, so every timed configuration is first warmed up for at least
--warmup steps, at least MIN_WARM_STEPS steps and at least MIN_WARM_SECONDS of
GPU work, whichever is longest (the count used is reported).  The timed region
is exactly --steps steps between two HIP events on the stream the library
launches on, with a synchronisation on both sides; value = sum(2 M N K) / (its
time / steps).  Per-step events inside it give the median, p10 and p90, and a
sampler thread reads the GFX clock and the socket power (amdsmi) meanwhile.
A "cold" variant writes a 512 MiB buffer between steps, which flushes the
256 MB last-level cache (MALL), and times each step alone.

The line also carries the roofline of the dominant kernel (the down-projection
GEMM of the bf6 engine, against the 6-bit MFMA peak), timed per launch with
HIP events on the stream the library launches on; the quantisers' bandwidth
next to a plain device copy timed in the same run; and the CPU oracle timed on
the whole step on the host cores (repeated until about ten seconds have
passed, its outputs compared with the GPU's), single-threaded on the tiny and
the attention-projection workloads, and as a Python-integer brute force on the
tiny one.

`secondary` reports, from the same run, the same measurement for other
layers: the FLUX MLP step with ternary weights (W1.58A4, on both engines) and
group-wise (group64, on both engines, with the bound its fp32 group fold puts
on the VALU), the FLUX MLP-down linear alone for one image (M = 4608), the 8B
diffusion-LLM block linears (W4A4, W1.58A4 and group128, each on both
engines, with per-linear times) and the DiT attention projection and fused QKV
linears.
"""

import argparse
import json
import os
import sys
import threading
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_INT8_TOPS = 5000.0     # MI355X dense int8 MFMA, published
PEAK_FP6_TOPS = 10100.0     # MI355X dense fp6 / fp4 MFMA, published
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E, published
# Non-packed fp32 VALU: 256 CUs x 4 SIMDs x 16 lanes per clock x 2.4 GHz (a
# wave64 instruction takes four clocks), in lane-operations per second.
PEAK_VALU_LANE_OPS = 256 * 4 * 16 * 2.4e9
# VALU instructions per output and K-group of the group-wise fold: convert,
# two multiplies and an add after the operand shift on the int8 engine; the
# two multiplies and the add on the bf6 engine (the matrix core returns fp32).
GROUP_FOLD_VALU = {"int8": 5, "bf6": 3}

MIN_WARM_STEPS = 200
MIN_WARM_SECONDS = 0.2
FLUSH_BYTES = 512 << 20


def parse_args():
    p = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20,
                   help=f"minimum warm-up steps (at least {MIN_WARM_STEPS} steps and "
                        f"{MIN_WARM_SECONDS} s are run whatever this says)")
    p.add_argument("--cold-steps", type=int, default=30, help="steps of the MALL-flushed variant")
    p.add_argument("--no-cpu-baseline", action="store_true", help="skip the oracle CPU baseline leg")
    p.add_argument("--cpu-seconds", type=float, default=10.0, help="minimum CPU time of the oracle baseline")
    p.add_argument("--no-secondary", action="store_true", help="skip the secondary workloads")
    p.add_argument("--copy-calib", action="store_true",
                   help="also run a plain 256 MiB device copy (calibrates HBM byte counters under rocprofv3)")
    p.add_argument("--secondary-filter", default="",
                   help="run only the secondary cases whose workload or layer name contains this text")
    p.add_argument("--operand-study", action="store_true",
                   help="also time the dominant GEMM on all-zero, constant, workload and random codes")
    p.add_argument("--full-rounds", action="store_true",
                   help="also time both engines' GEMMs on 8192x12288 -> 4096, whose tiles fill whole rounds")
    p.add_argument("--overlap-study", action="store_true",
                   help="also time the step with the down-projection's quantiser on a second stream")
    p.add_argument("--min-warm-steps", type=int, default=MIN_WARM_STEPS,
                   help="warm-up floor in steps (lower it only for counter-collection runs, which "
                        "serialise every launch)")
    p.add_argument("--min-warm-seconds", type=float, default=MIN_WARM_SECONDS, help="warm-up floor in seconds")
    return p.parse_args()


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_flux_mlp.json")
GEMM_SOURCE = os.path.join(ROOT, "paper_2609_33601_amd", "csrc", "f6.hip")


def recorded_traffic(kernel_linear):
    """HBM bytes per launch of the dominant kernel from the committed counter
    runs, or None if there are none or the kernel source changed since."""
    import hashlib

    try:
        rec = json.load(open(TRAFFIC_FILE))
        sha = hashlib.sha256(open(GEMM_SOURCE, "rb").read()).hexdigest()
    except (OSError, ValueError):
        return None
    if rec.get("gemm_source_sha256") != sha:
        return None
    k = rec.get("kernels", {}).get(kernel_linear)
    if not k:
        return None
    return k["fetch_bytes"] + k["write_bytes"]


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def percentiles(xs):
    s = sorted(xs)
    if not s:
        return {}

    def q(p):
        # linear interpolation between order statistics
        i = p * (len(s) - 1)
        lo = int(i)
        hi = min(lo + 1, len(s) - 1)
        return s[lo] + (s[hi] - s[lo]) * (i - lo)

    return {"median": q(0.5), "p10": q(0.1), "p90": q(0.9), "min": s[0], "max": s[-1]}


class ClockMonitor:
    """Samples the GFX clock (MHz) and the socket power (W) with amdsmi in a
    background thread; summary(t0, t1) reduces the samples taken between two
    perf_counter() times."""

    def __init__(self, period_s=0.001):
        self.period = period_s
        self.samples = []
        self.error = None
        self._stop = threading.Event()
        self._thread = None
        self._h = None
        try:
            import amdsmi

            amdsmi.amdsmi_init()
            self._amdsmi = amdsmi
            self._h = amdsmi.amdsmi_get_processor_handles()[0]
        except Exception as e:  # noqa: BLE001
            self.error = f"amdsmi unavailable: {e!r}"[:200]

    def read(self):
        # amdsmi_get_clock_info reads the current GFX clock; the gpu-metrics
        # table was seen to return stale values at this sampling rate
        if self._h is None:
            return None

        def num(v):
            return v if isinstance(v, (int, float)) and v > 0 else None

        rec = {"t": time.perf_counter(), "gfx_mhz": None, "power_w": None}
        try:
            rec["gfx_mhz"] = num(self._amdsmi.amdsmi_get_clock_info(self._h, self._amdsmi.AmdSmiClkType.GFX)
                                 .get("clk"))
        except Exception as e:  # noqa: BLE001
            self.error = f"clock info: {e!r}"[:200]
        try:
            p = self._amdsmi.amdsmi_get_power_info(self._h)
            rec["power_w"] = num(p.get("current_socket_power")) or num(p.get("average_socket_power"))
        except Exception:  # noqa: BLE001
            pass
        return rec if rec["gfx_mhz"] is not None else None

    def _run(self):
        while not self._stop.is_set():
            r = self.read()
            if r is not None:
                self.samples.append(r)
            time.sleep(self.period)

    def start(self):
        if self._h is not None:
            self._thread = threading.Thread(target=self._run, daemon=True)
            self._thread.start()
        return self

    def stop(self):
        self._stop.set()
        if self._thread is not None:
            self._thread.join(timeout=2)

    def summary(self, t0, t1):
        if self._h is None:
            return {"error": self.error}
        inside = [s for s in self.samples if t0 <= s["t"] <= t1]
        before = [s for s in self.samples if s["t"] < t0]
        after = [s for s in self.samples if s["t"] > t1]
        out = {"samples_in_region": len(inside), "period_ms": self.period * 1e3}

        def stats(key, ss):
            v = [s[key] for s in ss if s.get(key) is not None]
            return None if not v else {"mean": sum(v) / len(v), "min": min(v), "max": max(v)}

        out["gfx_mhz"] = stats("gfx_mhz", inside)
        out["power_w"] = stats("power_w", inside)
        out["gfx_mhz_before"] = before[-1]["gfx_mhz"] if before else None
        out["gfx_mhz_after"] = after[0]["gfx_mhz"] if after else None
        if self.error:
            out["error"] = self.error
        return out


_X_CACHE = {}


def _x_key(lin):
    return (lin.M, lin.K, lin.x_dist, lin.x_seed, lin.outlier_frac, lin.outlier_factor)


def _make_x(lin):
    key = _x_key(lin)
    if key not in _X_CACHE:
        _X_CACHE[key] = lin.make_x()
    return _X_CACHE[key]


def check_shared_inputs(linears):
    """A linear marked as sharing its input with the one before it must draw
    exactly the same activations (same shape, distribution, seed and
    outliers), since it reuses that linear's quantised activations."""
    for prev, lin in zip(linears, linears[1:]):
        if lin.shares_input and _x_key(prev) != _x_key(lin):
            raise ValueError(f"{lin.name} is marked as sharing the input of {prev.name}, "
                             f"but their activations differ: {_x_key(prev)} vs {_x_key(lin)}")
    if linears and linears[0].shares_input:
        raise ValueError(f"{linears[0].name} is marked as sharing an input but has no predecessor")


class Prepared:
    """Device-resident inputs, packed weight and output/workspace buffers of one linear.

    fmt "int4" packs the weight for the W4A4 layer (int8 engine), "bf6" for
    the same layer on the bf6 engine, "ternary" for W1.58A4 (int8 engine),
    "ternary_bf6" for W1.58A4 on the bf6 engine, "group64" /
    "group128" for group-wise W4A4 with that group size (int8 engine), and
    "group64_bf6" / "group128_bf6" for the same on the bf6 engine.
    """

    def __init__(self, lin, torch, jq, fmt="int4"):
        self.lin = lin
        self.fmt = fmt
        self.engine = "bf6" if fmt.endswith("bf6") else "int8"
        self.x_bits = _make_x(lin)
        self.w_bits = lin.make_w()
        self.b_bits = lin.make_bias()
        self.x = jq.bf16_tensor(self.x_bits, "cuda")
        w = jq.bf16_tensor(self.w_bits, "cuda")
        ws_bytes = jq.jq_w4a4_workspace_bytes(lin.M, lin.K)
        self.G = None
        if fmt.startswith("group") and fmt.endswith("_bf6"):
            G = self.G = int(fmt[5:-4])
            wq4, self.sw = jq.jq_pack_weight_int4_group(w, G)
            self.wq = jq.jq_int4_to_f6_weight(wq4)
            del wq4
            self.linear = lambda x, wq, sw, b, y, workspace: jq.jq_w4a4g_f6_linear(x, wq, sw, G, b, y=y,
                                                                                  workspace=workspace)
            ws_bytes = jq.jq_w4a4g_f6_workspace_bytes(lin.M, lin.K, G)
        elif fmt.startswith("group"):
            G = self.G = int(fmt[5:])
            self.wq, self.sw = jq.jq_pack_weight_int4_group(w, G)
            self.linear = lambda x, wq, sw, b, y, workspace: jq.jq_w4a4g_linear(x, wq, sw, G, b, y=y,
                                                                               workspace=workspace)
            ws_bytes = jq.jq_w4a4g_workspace_bytes(lin.M, lin.K, G)
        elif fmt == "bf6":
            self.wq4, self.sw = jq.jq_pack_weight_int4(w)
            self.wq = jq.jq_int4_to_f6_weight(self.wq4)
            self.linear = jq.jq_w4a4_f6_linear
            ws_bytes = jq.jq_w4a4_f6_workspace_bytes(lin.M, lin.K)
        elif fmt == "ternary_bf6":
            wt, self.sw = jq.jq_pack_weight_ternary(w)
            self.wq = jq.jq_ternary_to_f6_weight(wt)
            del wt
            self.linear = jq.jq_w4a4_f6_linear
            ws_bytes = jq.jq_w4a4_f6_workspace_bytes(lin.M, lin.K)
        else:
            pack = jq.jq_pack_weight_ternary if fmt == "ternary" else jq.jq_pack_weight_int4
            self.linear = jq.jq_w158a4_linear if fmt == "ternary" else jq.jq_w4a4_linear
            self.wq, self.sw = pack(w)
        del w
        self.b = None if self.b_bits is None else jq.bf16_tensor(self.b_bits, "cuda")
        self.y = torch.empty((lin.M, lin.N), dtype=torch.bfloat16, device="cuda")
        self.ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
        self.q = torch.empty((lin.M, lin.K // 2), dtype=torch.uint8, device="cuda")
        self.s = torch.empty((lin.M,), dtype=torch.float32, device="cuda")
        if fmt in ("bf6", "ternary_bf6"):
            self.q = torch.empty((jq.jq_f6_operand_bytes(lin.M, lin.K),), dtype=torch.uint8, device="cuda")
        # The layer split in two, for linears that share their input (the
        # dLLM block's gate and up): quantise once, then one GEMM per linear.
        K, q, s, b, y, wq, sw = lin.K, self.q, self.s, self.b, self.y, self.wq, self.sw
        if fmt.startswith("group"):
            G = self.G
            self.s = s = torch.empty((lin.M, lin.K // G), dtype=torch.float32, device="cuda")
            if fmt.endswith("_bf6"):
                self.q = q = torch.empty((jq.jq_f6_operand_bytes(lin.M, lin.K),), dtype=torch.uint8, device="cuda")
                self.quantize = lambda: jq.jq_quantize_act_group_f6(self.x, G, xf6=q, scale=s)
                self.gemm = lambda qq, ss: jq.jq_w4a4g_f6_gemm(qq, ss, wq, sw, G, b, y=y)
            else:
                self.quantize = lambda: jq.jq_quantize_act_group(self.x, G, q=q, scale=s)
                self.gemm = lambda qq, ss: jq.jq_w4a4g_gemm(qq, ss, wq, sw, G, b, y=y)
        elif fmt in ("bf6", "ternary_bf6"):
            self.quantize = lambda: jq.jq_quantize_act_f6(self.x, xf6=q, scale=s)
            self.gemm = lambda qq, ss: jq.jq_w4a4_f6_gemm(qq, ss, K, wq, sw, b, y=y)
        else:
            g = jq.jq_w158a4_gemm if fmt == "ternary" else jq.jq_w4a4_gemm
            self.quantize = lambda: jq.jq_quantize_act(self.x, q=q, scale=s)
            self.gemm = lambda qq, ss: g(qq, ss, wq, sw, b, y=y)
        self.shares_input = lin.shares_input

    def run(self):
        """The whole layer through its linear entry point."""
        self.linear(self.x, self.wq, self.sw, self.b, y=self.y, workspace=self.ws)


def make_step(preps):
    """One pass over the linears: each a whole quantise + GEMM layer; a linear
    that shares the previous one's input reuses its quantised activations."""
    check_shared_inputs([p.lin for p in preps])
    split = any(p.shares_input for p in preps)

    def step():
        qs = None
        for p in preps:
            if p.shares_input and qs is not None:
                p.gemm(*qs)
            elif split:
                qs = p.quantize()
                p.gemm(*qs)
            else:
                p.run()

    return step


def warm_up(torch, step, min_steps):
    """Run the step until at least min_steps steps and MIN_WARM_SECONDS have passed; returns the count."""
    n = 0
    t0 = time.perf_counter()
    while n < min_steps or time.perf_counter() - t0 < MIN_WARM_SECONDS:
        for _ in range(10):
            step()
        n += 10
        torch.cuda.synchronize()
    return n


def time_steps(torch, step, steps, warmup, clock=None):
    """Warm up, then time exactly `steps` steps on the current stream: the mean
    from the bracketing events, the distribution from per-step events."""
    stream = torch.cuda.current_stream()
    warm = warm_up(torch, step, max(warmup, MIN_WARM_STEPS))
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev[0].record(stream)
    for i in range(steps):
        step()
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    per = [ev[i].elapsed_time(ev[i + 1]) * 1e3 for i in range(steps)]
    out = {"us_per_step": ev[0].elapsed_time(ev[steps]) / steps * 1e3, "warmup_steps": warm,
           "wall_us_per_step": (t1 - t0) / steps * 1e6, "per_step_us": percentiles(per)}
    if clock is not None:
        out["clock"] = clock.summary(t0, t1)
    return out


def time_cold(torch, step, steps):
    """Each step timed alone after a 512 MiB write that flushes the MALL."""
    stream = torch.cuda.current_stream()
    flush = torch.empty(FLUSH_BYTES // 4, dtype=torch.float32, device="cuda")
    per = []
    for i in range(steps):
        flush.fill_(float(i))
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        step()
        e1.record(stream)
        torch.cuda.synchronize()
        per.append(e0.elapsed_time(e1) * 1e3)
    del flush
    return {"steps": steps, "flush_bytes": FLUSH_BYTES, "per_step_us": percentiles(per),
            "mean_us": sum(per) / len(per)}


def time_copy(torch, nbytes=256 << 20, reps=50):
    """A plain device-to-device copy: bytes read + written per second."""
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(10):
        dst.copy_(src)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) / reps * 1e3
    del src, dst
    return {"bytes_copied": nbytes, "us": us, "GBs_read_plus_write": 2 * nbytes / us / 1e3}


def per_linear_times(torch, preps, n_launch):
    """The quantiser and the GEMM of each linear, each launch bracketed by
    events on the stream it runs on; averages in us."""
    stream = torch.cuda.current_stream()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(len(preps) * n_launch)]
    for it in range(n_launch):
        qs = None
        for j, p in enumerate(preps):
            e = evs[it * len(preps) + j]
            e[0].record(stream)
            if not (p.shares_input and qs is not None):
                qs = p.quantize()
            e[1].record(stream)
            p.gemm(*qs)
            e[2].record(stream)
    torch.cuda.synchronize()
    out = []
    for j, p in enumerate(preps):
        tq = [evs[it * len(preps) + j][0].elapsed_time(evs[it * len(preps) + j][1]) * 1e3 for it in range(n_launch)]
        tg = [evs[it * len(preps) + j][1].elapsed_time(evs[it * len(preps) + j][2]) * 1e3 for it in range(n_launch)]
        out.append((sum(tq) / n_launch, sum(tg) / n_launch, percentiles(tg)))
    return out


def cpu_baseline(preps, target_s):
    """The oracle as it stands: on every row of the timed workload, repeated
    until target_s seconds have passed (all BLAS threads); single-threaded on
    the tiny and the attention-projection workloads; and the Python-integer
    brute force of the tiny workload's contraction."""
    import numpy as np
    import oracle
    from paper_2609_33601_amd import jq, workloads

    try:
        from threadpoolctl import threadpool_info, threadpool_limits

        blas = [i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"]
        cores = max(blas) if blas else 1
    except Exception:  # noqa: BLE001
        threadpool_limits = None
        cores = 1
    packed = [oracle.pack_weight_int4(p.w_bits) for p in preps]  # offline step, untimed

    def run():
        return [oracle.w4a4_linear(p.x_bits, rq, rs, p.b_bits) for p, (rq, rs) in zip(preps, packed)]

    ops_once = sum(2 * p.lin.M * p.lin.N * p.lin.K for p in preps)
    c0 = os.times()
    t0 = time.perf_counter()
    outs = run()
    reps = 1
    while time.perf_counter() - t0 < target_s:
        run()
        reps += 1
    t = time.perf_counter() - t0
    c1 = os.times()
    cpu_s = (c1.user - c0.user) + (c1.system - c0.system)
    # the oracle's outputs double as a parity check of every GPU output of the step
    mism = sum(int(np.sum(jq.bf16_bits(p.y) != ref)) for p, ref in zip(preps, outs))
    res = {
        "value": reps * ops_once / t / 1e12,
        "unit": "TOPS",
        "cores": int(cores),
        "kind": "oracle",
        "sample": f"the whole step (every row of the {len(preps)} linears, {ops_once / 1e9:.0f} G int ops) "
                  f"run {reps} times in {t:.1f} s; weights packed beforehand",
        "seconds": t,
        "cores_note": "cores = BLAS threads of the float64 code product; "
                      "effective_parallelism = process CPU time / wall time",
        "effective_parallelism": cpu_s / t,
        "host_cpus": os.cpu_count(),
        "affinity_cpus": len(os.sched_getaffinity(0)),
        "gpu_outputs_differing_from_oracle": mism,
    }
    # single-threaded oracle on the tiny and the attention-projection linears
    single = {}
    for name in ("tiny", "attn_proj"):
        lin = workloads.WORKLOADS[name].linears[0]
        xb, wb, bb = lin.make_x(), lin.make_w(), lin.make_bias()
        rq, rs = oracle.pack_weight_int4(wb)
        ctx = threadpool_limits(1, "blas") if threadpool_limits else None
        if ctx is not None:
            ctx.__enter__()
        try:
            n, t0 = 0, time.perf_counter()
            while n == 0 or time.perf_counter() - t0 < 0.5:
                oracle.w4a4_linear(xb, rq, rs, bb)
                n += 1
            ts = (time.perf_counter() - t0) / n
        finally:
            if ctx is not None:
                ctx.__exit__(None, None, None)
        single[name] = {"M": lin.M, "K": lin.K, "N": lin.N, "seconds": ts, "TOPS": lin.ops / ts / 1e12, "runs": n}
    res["single_thread"] = single
    # Python-integer brute force of the tiny workload's contraction
    lin = workloads.WORKLOADS["tiny"].linears[0]
    qx, _ = oracle.quantize_act(lin.make_x())
    qw, _ = oracle.pack_weight_int4(lin.make_w())
    ux, uw = oracle.unpack_int4(qx), oracle.unpack_int4(qw)
    t0 = time.perf_counter()
    bf = oracle.brute_force_gemm(ux, uw)
    tb = time.perf_counter() - t0
    res["brute_force_tiny"] = {"M": lin.M, "K": lin.K, "N": lin.N, "seconds": tb,
                               "TOPS": lin.ops / tb / 1e12,
                               "equals_code_gemm": bool(np.array_equal(bf, oracle.code_gemm(ux, uw)))}
    return res


def operand_study(torch, jq, lin, prep, clock, launches=200):
    """The bf6 GEMM of one linear (the MLP-down one: the dominant kernel) on
    operands of different switching activity: all-zero codes, every code 1,
    the workload's codes and uniformly random int4 codes (weights and
    activations alike; random codes are re-encoded by the library's
    converters).  A GEMM whose time does not depend on the data is bound by
    its own structure, not by the chip's power limit."""
    M, K, N = lin.M, lin.K, lin.N
    g = torch.Generator(device="cuda")
    g.manual_seed(5)
    rnd_x = torch.randint(0, 256, (M, K // 2), dtype=torch.uint8, device="cuda", generator=g)
    rnd_w = torch.randint(0, 256, (N, K // 2), dtype=torch.uint8, device="cuda", generator=g)
    one_x = torch.full((M, K // 2), 0x11, dtype=torch.uint8, device="cuda")
    one_w = torch.full((N, K // 2), 0x11, dtype=torch.uint8, device="cuda")
    xq, xs = prep.quantize()
    cases = {
        "zero": (torch.zeros_like(xq), torch.zeros_like(prep.wq)),
        "ones": (jq.jq_int4_to_f6(one_x), jq.jq_int4_to_f6_weight(one_w)),
        "workload": (xq, prep.wq),
        "random": (jq.jq_int4_to_f6(rnd_x), jq.jq_int4_to_f6_weight(rnd_w)),
    }
    del rnd_x, rnd_w, one_x, one_w
    y = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    stream = torch.cuda.current_stream()
    out = {}
    for name, (xa, wa) in cases.items():
        for _ in range(MIN_WARM_STEPS):
            jq.jq_w4a4_f6_gemm(xa, xs, K, wa, prep.sw, None, y=y)
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        e0.record(stream)
        for _ in range(launches):
            jq.jq_w4a4_f6_gemm(xa, xs, K, wa, prep.sw, None, y=y)
        e1.record(stream)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        us = e0.elapsed_time(e1) / launches * 1e3
        out[name] = {"avg_us": us, "TOPS": lin.ops / us / 1e6, "clock": clock.summary(t0, t1)}
        log(f"operand study {lin.name} {name}: {us:.1f} us, {lin.ops / us / 1e6:.0f} TOPS")
    return {"linear": lin.name, "M": M, "K": K, "N": N, "launches": launches, "cases": out}


def full_rounds(torch, jq, workloads, launches=100):
    """Both engines' GEMMs on a shape whose output tiles fill whole rounds of
    the chip's block slots (8192 x 12288 -> 4096: 512 tiles of 256 x 256 for
    the bf6 engine's 256 one-block CUs, 1024 tiles of 128 x 256 for the int8
    engine's 512 two-block slots), next to the FLUX MLP-down shape
    (9216 x 12288 -> 3072), whose tiles leave the last round part-empty.
    Inputs have the MLP-down statistics."""
    base = workloads.FLUX_MLP.linears[1]
    full = workloads.Linear("full_rounds_8192x12288x4096", M=8192, K=12288, N=4096, x_dist=base.x_dist,
                            x_seed=base.x_seed, outlier_frac=base.outlier_frac,
                            outlier_factor=base.outlier_factor, w_std=base.w_std, w_seed=base.w_seed)
    stream = torch.cuda.current_stream()
    out = []
    for lin in (base, full):
        p6 = Prepared(lin, torch, jq, "bf6")
        p4 = Prepared(lin, torch, jq, "int4")
        for eng, p in (("bf6", p6), ("int8", p4)):
            qs = p.quantize()
            for _ in range(MIN_WARM_STEPS):
                p.gemm(*qs)
            torch.cuda.synchronize()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(launches):
                p.gemm(*qs)
            e1.record(stream)
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) / launches * 1e3
            tops = lin.ops / us / 1e6
            peak = PEAK_FP6_TOPS if eng == "bf6" else PEAK_INT8_TOPS
            out.append({"linear": lin.name, "M": lin.M, "K": lin.K, "N": lin.N, "engine": eng, "avg_us": us,
                        "TOPS": tops, "frac_mfma_peak": tops / peak, "pct_int8_peak": 100 * tops / PEAK_INT8_TOPS})
            log(f"full rounds {lin.name} {eng}: {us:.1f} us, {tops:.0f} TOPS ({100 * tops / peak:.1f}% of its peak)")
        del p6, p4
        torch.cuda.empty_cache()
    return out


def workloads_mod():
    from paper_2609_33601_amd import workloads

    return workloads


def overlap_study(torch, jq, preps, steps=200):
    """The bf6 step with the down-projection's quantiser moved to a second
    stream (equal priority), so that it can run beside the up-projection's
    quantiser and GEMM, against the same step on one stream.  The inputs of
    the two linears are independent, so the order is free."""
    up, dn = preps
    main = torch.cuda.current_stream()
    side = torch.cuda.Stream()

    def serial():
        for p in preps:
            p.gemm(*p.quantize())

    def side_first():
        e = torch.cuda.Event()
        e.record(main)
        side.wait_event(e)  # the previous step is done with the down operand
        with torch.cuda.stream(side):
            qd = dn.quantize()
        up.gemm(*up.quantize())
        e2 = torch.cuda.Event()
        e2.record(side)
        main.wait_event(e2)
        dn.gemm(*qd)

    def both_quantisers_first():
        e = torch.cuda.Event()
        e.record(main)
        side.wait_event(e)
        with torch.cuda.stream(side):
            qd = dn.quantize()
        qu = up.quantize()
        e2 = torch.cuda.Event()
        e2.record(side)
        main.wait_event(e2)
        up.gemm(*qu)
        dn.gemm(*qd)

    def batched():
        # both inputs quantised in one launch (jq_quantize_act_f6_batch), then the GEMMs
        (qu, qd), (su, sd) = jq.jq_quantize_act_f6_batch([up.x, dn.x], [up.q, dn.q], [up.s, dn.s])
        up.gemm(qu, su)
        dn.gemm(qd, sd)

    # small inputs, where a launch's latency outweighs its bytes: the three
    # distinct inputs of the 8B dLLM block (gate/up, o-proj, down) for 64
    # tokens, quantised by three launches or by one
    small = [lin for lin in workloads_mod().WORKLOADS["dllm_block"].linears if not lin.shares_input]
    sx = [jq.bf16_tensor(lin.make_x()[:64], "cuda") for lin in small]
    sq = [torch.empty((jq.jq_f6_operand_bytes(*x.shape),), dtype=torch.uint8, device="cuda") for x in sx]
    ss = [torch.empty((x.shape[0],), dtype=torch.float32, device="cuda") for x in sx]

    def small_separate():
        for x, q, s_ in zip(sx, sq, ss):
            jq.jq_quantize_act_f6(x, q, s_)

    def small_batched():
        jq.jq_quantize_act_f6_batch(sx, sq, ss)

    out = {}
    for name, fn in (("small inputs (3 x 64 tokens of the dLLM block): three launches", small_separate),
                     ("small inputs (3 x 64 tokens of the dLLM block): one batched launch", small_batched)):
        r = time_steps(torch, fn, steps, 20)
        out[name] = {"us_per_step": r["us_per_step"], "per_step_us": r["per_step_us"]}
        log(f"overlap study: {name}: {r['us_per_step']:.1f} us")
    for name, fn in (("one stream", serial), ("down quantiser on a second stream, beside the up linear", side_first),
                     ("both quantisers side by side, then the GEMMs", both_quantisers_first),
                     ("both inputs quantised in one launch, then the GEMMs", batched)):
        r = time_steps(torch, fn, steps, 20)
        out[name] = {"us_per_step": r["us_per_step"], "per_step_us": r["per_step_us"]}
        log(f"overlap study: {name}: {r['us_per_step']:.1f} us/step")
    return out


def secondary(torch, jq, workloads, steps, warmup, n_launch, only=""):
    cases = [(workloads.FLUX_MLP, "ternary_bf6"), (workloads.FLUX_MLP, "ternary"),
             (workloads.WORKLOADS["mlp_down_1img"], "bf6"), (workloads.WORKLOADS["mlp_down_1img"], "int4"),
             (workloads.WORKLOADS["dllm_block"], "bf6"), (workloads.WORKLOADS["dllm_block"], "int4"),
             (workloads.WORKLOADS["dllm_block"], "ternary_bf6"), (workloads.WORKLOADS["dllm_block"], "ternary"),
             (workloads.WORKLOADS["attn_proj"], "bf6"), (workloads.WORKLOADS["attn_proj"], "int4"),
             (workloads.WORKLOADS["qkv"], "bf6"), (workloads.WORKLOADS["qkv"], "int4"),
             (workloads.FLUX_MLP, "group64_bf6"), (workloads.FLUX_MLP, "group64"),
             (workloads.WORKLOADS["dllm_block"], "group128_bf6"), (workloads.WORKLOADS["dllm_block"], "group128")]
    layer_names = {"ternary": "W1.58A4 (int8 engine)", "ternary_bf6": "W1.58A4 (bf6 engine)",
                   "int4": "W4A4 (int8 engine)", "bf6": "W4A4 (bf6 engine)",
                   "group64": "W4A4 group64 (int8 engine)", "group128": "W4A4 group128 (int8 engine)",
                   "group64_bf6": "W4A4 group64 (bf6 engine)", "group128_bf6": "W4A4 group128 (bf6 engine)"}
    cases = [(wl, fmt) for wl, fmt in cases if not only or only in wl.name or only in layer_names[fmt]]
    out = []
    for wl, fmt in cases:
        check_shared_inputs(list(wl.linears))
        preps = [Prepared(lin, torch, jq, fmt) for lin in wl.linears]
        r = time_steps(torch, make_step(preps), steps, warmup)
        us = r["us_per_step"]
        tops = wl.ops / (us * 1e-6) / 1e12
        layer = layer_names[fmt]
        per = per_linear_times(torch, preps, n_launch)
        rec = {"workload": wl.description, "layer": layer, "us_per_step": us, "effective_TOPS": tops,
               "pct_int8_peak": 100.0 * tops / PEAK_INT8_TOPS, "warmup_steps": r["warmup_steps"],
               "per_step_us": r["per_step_us"],
               "linears": [{"name": p.lin.name, "M": p.lin.M, "K": p.lin.K, "N": p.lin.N,
                            "quantize_us": tq if not (p.shares_input and j > 0) else 0.0, "gemm_us": tg,
                            "gemm_TOPS": p.lin.ops / tg / 1e6}
                           for j, (p, (tq, tg, _)) in enumerate(zip(preps, per))]}
        if preps[0].G is not None:
            # the fp32 group fold on the VALU: GROUP_FOLD_VALU instructions per output and group
            lane_ops = GROUP_FOLD_VALU[preps[0].engine] * sum(p.lin.M * p.lin.N * (p.lin.K // p.G) for p in preps)
            bound_us = lane_ops / PEAK_VALU_LANE_OPS * 1e6
            rec["valu_fold_bound"] = {"valu_per_output_group": GROUP_FOLD_VALU[preps[0].engine],
                                      "lane_ops": lane_ops, "peak_lane_ops_per_s": PEAK_VALU_LANE_OPS,
                                      "bound_us": bound_us, "frac": bound_us / us}
        log(f"secondary {wl.name} {layer}: {us:.1f} us/step, {tops:.0f} effective TOPS "
            f"(median {r['per_step_us']['median']:.1f}, warm-up {r['warmup_steps']} steps)")
        out.append(rec)
        del preps
        torch.cuda.empty_cache()
    return out


def main():
    global MIN_WARM_STEPS, MIN_WARM_SECONDS
    args = parse_args()
    MIN_WARM_STEPS, MIN_WARM_SECONDS = args.min_warm_steps, args.min_warm_seconds
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the W4A4 linear "
              "shards without communication over tokens (M) and is measured at N=1.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_33601_amd import jq, workloads

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    jq.lib()
    clock = ClockMonitor().start()
    wl = workloads.FLUX_MLP
    log("preparing", wl.description)
    preps = [Prepared(lin, torch, jq, "bf6") for lin in wl.linears]
    preps4 = [Prepared(lin, torch, jq, "int4") for lin in wl.linears]
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    step = make_step(preps)

    head = time_steps(torch, step, args.steps, args.warmup, clock)
    ms_per_step = head["us_per_step"] / 1e3
    value = wl.ops / (ms_per_step * 1e-3) / 1e12
    log(f"bf6 engine: warm-up {head['warmup_steps']} steps, timed {args.steps} steps: "
        f"{head['us_per_step']:.1f} us/step (median {head['per_step_us']['median']:.1f}, "
        f"p10 {head['per_step_us']['p10']:.1f}, p90 {head['per_step_us']['p90']:.1f}); clock {head.get('clock')}")

    # The same step on the int8 engine (same layer, bit-identical outputs).
    r8 = time_steps(torch, make_step(preps4), args.steps, args.warmup, clock)
    us_int8 = r8["us_per_step"]
    log(f"int8 engine: {us_int8:.1f} us/step, {wl.ops / (us_int8 * 1e-6) / 1e12:.0f} effective TOPS")

    cold = time_cold(torch, step, args.cold_steps)
    log(f"cold (MALL flushed before each step): median {cold['per_step_us']['median']:.1f} us")
    copy = time_copy(torch)
    log(f"device copy: {copy['GBs_read_plus_write']:.0f} GB/s read + write")

    # Per-kernel durations: the two kernels each linear launches, bracketed by
    # events on the stream they run on, for both engines.
    n_launch = max(args.steps, 20)
    kernels = []
    for engine, pp in (("bf6", preps), ("int8", preps4)):
        warm_up(torch, make_step(pp), MIN_WARM_STEPS)
        for p, (tq_us, tg_us, tg_dist) in zip(pp, per_linear_times(torch, pp, n_launch)):
            lin = p.lin
            code_bytes = jq.jq_f6_operand_bytes(lin.M, lin.K) if engine == "bf6" else lin.M * lin.K // 2
            q_bytes = 2 * lin.M * lin.K + code_bytes + 4 * lin.M
            g_ops = 2 * lin.M * lin.N * lin.K
            peak = PEAK_FP6_TOPS if engine == "bf6" else PEAK_INT8_TOPS
            q_gbs = q_bytes / tq_us / 1e3
            kernels.append({"engine": engine, "linear": lin.name, "kernel": "quantize_rows", "avg_us": tq_us,
                            "algorithmic_bytes": q_bytes, "achieved_GBs": q_gbs,
                            "frac_hbm_peak": q_gbs / PEAK_HBM_GBS,
                            "frac_of_device_copy": q_gbs / copy["GBs_read_plus_write"]})
            kernels.append({"engine": engine, "linear": lin.name, "kernel": "w4a4_gemm", "avg_us": tg_us,
                            "per_launch_us": tg_dist,
                            "ops": g_ops, "achieved_TOPS": g_ops / tg_us / 1e6, "peak_TOPS": peak,
                            "frac_mfma_peak": g_ops / tg_us / 1e6 / peak,
                            "pct_int8_peak": 100.0 * g_ops / tg_us / 1e6 / PEAK_INT8_TOPS})
            log(f"{engine} {lin.name}: quantize {tq_us:.1f} us ({q_gbs:.0f} GB/s), "
                f"gemm {tg_us:.1f} us ({g_ops / tg_us / 1e6:.0f} TOPS)")
    dom = max((k for k in kernels if k["kernel"] == "w4a4_gemm" and k["engine"] == "bf6"), key=lambda k: k["ops"])
    roofline = {"bound": "mfma", "achieved": dom["achieved_TOPS"], "peak": PEAK_FP6_TOPS, "unit": "TOP/s",
                "frac": dom["achieved_TOPS"] / PEAK_FP6_TOPS, "traffic": recorded_traffic(dom["linear"]),
                "kernel": f"w4a4_f6_gemm ({dom['linear']}, bf6 operands, fp32 accumulation)",
                "avg_launch_us": dom["avg_us"],
                "peak_note": "MI355X dense fp6 MFMA; the same kernel is at "
                             f"{100.0 * dom['achieved_TOPS'] / PEAK_INT8_TOPS:.0f}% of the dense int8 peak"}

    if args.copy_calib:
        # Reference for FETCH_SIZE / WRITE_SIZE: a plain device copy of 256 MiB.
        src = torch.empty(256 << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # Re-run the timed configuration once so that y holds the step's outputs for the oracle comparison.
    step()
    torch.cuda.synchronize()
    for p4 in preps4:
        p4.run()
    torch.cuda.synchronize()
    engines_equal = all(torch.equal(a.y.view(torch.int16), b.y.view(torch.int16)) for a, b in zip(preps, preps4))
    del preps4
    torch.cuda.empty_cache()
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(preps, args.cpu_seconds)
        log(f"cpu oracle: {cpu['value']:.4f} TOPS on {cpu['cores']} threads; {cpu['sample']}; "
            f"gpu/oracle differing outputs: {cpu['gpu_outputs_differing_from_oracle']}")

    study = None
    if args.operand_study:
        study = operand_study(torch, jq, wl.linears[1], preps[1], clock)
    ovl = overlap_study(torch, jq, preps) if args.overlap_study else None
    fr = full_rounds(torch, jq, workloads) if args.full_rounds else None

    sec = None
    if not args.no_secondary:
        sec = secondary(torch, jq, workloads, max(10, min(args.steps, 50)), args.warmup, 20,
                        args.secondary_filter)
    clock.stop()

    props = torch.cuda.get_device_properties(0)
    out = {
        "metric": "W4A4 linear effective TOPS + % int8 MFMA peak at FLUX-12B MLP shape",
        "value": value,
        "unit": "TOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "warmup_steps_run": head["warmup_steps"],
        "warmup_floor": {"steps": MIN_WARM_STEPS, "seconds": MIN_WARM_SECONDS},
        "ms_per_step": ms_per_step,
        "per_step_us": head["per_step_us"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf6 codes, fp32 accumulation (exact for int4 codes)",
        "data": "synthetic (seeded; FLUX-12B MLP activation/weight statistics)",
        "pct_int8_peak": 100.0 * value / PEAK_INT8_TOPS,
        "config": {
            "workload": wl.description,
            "linears": [{"name": l.name, "M": l.M, "K": l.K, "N": l.N, "bias": l.bias_std is not None}
                        for l in wl.linears],
            "ops_per_step": wl.ops,
            "engine": "bf6",
            "parallelism": "none (1 GPU)",
            "device": f"{props.name} {getattr(props, 'gcnArchName', '')} CUs={props.multi_processor_count}",
        },
        "clock": head.get("clock"),
        "clock_note": "amdsmi readings (refreshed by the driver far less often than the sampling period; "
                      "the effective clock of a kernel is in profiles/counters_flux_mlp.md)",
        "cold": {**cold, "effective_TOPS_median": wl.ops / (cold["per_step_us"]["median"] * 1e-6) / 1e12},
        "engines": {
            "bf6": {"us_per_step": head["us_per_step"], "effective_TOPS": value,
                    "pct_int8_peak": 100.0 * value / PEAK_INT8_TOPS, "per_step_us": head["per_step_us"],
                    "warmup_steps": head["warmup_steps"],
                    "gemm_plan": {l.name: dict(zip(("waves", "tile_rows"), jq.jq_f6_gemm_plan(
                        l.M, l.N, l.K, props.multi_processor_count))) for l in wl.linears}},
            "int8": {"us_per_step": us_int8, "effective_TOPS": wl.ops / (us_int8 * 1e-6) / 1e12,
                     "pct_int8_peak": 100.0 * wl.ops / (us_int8 * 1e-6) / 1e12 / PEAK_INT8_TOPS,
                     "per_step_us": r8["per_step_us"], "warmup_steps": r8["warmup_steps"],
                     "clock": r8.get("clock"),
                     "gemm_plan": {l.name: {"tile_rows": jq.jq_gemm_plan(l.M, l.N, l.K, props.multi_processor_count)}
                                   for l in wl.linears},
                     "dtype": "int8 (widened int4 codes), int32 accumulation"},
            "outputs_bit_identical": bool(engines_equal),
        },
        "device_copy": copy,
        "roofline": roofline,
        "cpu_baseline": cpu,
        "kernels": kernels,
        "secondary": sec,
    }
    if study is not None:
        out["operand_study"] = study
    if ovl is not None:
        out["overlap_study"] = ovl
    if fr is not None:
        out["full_rounds"] = fr
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
