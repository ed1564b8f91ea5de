"""Host-side checks of bench.py: the one-GPU contract, the workload it times and
the committed traffic record it reports (no GPU needed)."""

import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2609_33601_amd import workloads  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_headline_workload_is_the_flux_mlp_pair():
    up, down = workloads.FLUX_MLP.linears
    assert (up.M, up.K, up.N) == (4608, 3072, 12288) and up.bias_std is not None
    assert (down.M, down.K, down.N) == (9216, 12288, 3072) and down.bias_std is None
    assert workloads.FLUX_MLP.ops == 2 * (4608 * 3072 * 12288 + 9216 * 12288 * 3072)


@pytest.mark.parametrize("linear", ["mlp_down", "mlp_up"])
def test_traffic_record_is_well_formed(linear):
    rec = json.load(open(bench.TRAFFIC_FILE))
    k = rec["kernels"][linear]
    assert len(rec["gemm_source_sha256"]) == 64
    # measured HBM bytes can only exceed what the kernel must move
    assert k["fetch_bytes"] + k["write_bytes"] >= k["algorithmic_bytes"] > 0
    # the scales come from a plain device copy of known size
    assert 0.5 < rec["fetch_scale"] < 4 and 0.5 < rec["write_scale"] < 4


def test_shared_input_linears_draw_identical_activations():
    # every workload linear marked as sharing its predecessor's input draws the same activations
    for wl in list(workloads.WORKLOADS.values()) + [workloads.FLUX_MLP]:
        bench.check_shared_inputs(list(wl.linears))
    gate, up = workloads.WORKLOADS["dllm_block"].linears[:2]
    assert up.shares_input and bench._x_key(gate) == bench._x_key(up)


def test_shared_input_mismatch_is_refused():
    import dataclasses

    gate, up = workloads.WORKLOADS["dllm_block"].linears[:2]
    with pytest.raises(ValueError):
        bench.check_shared_inputs([gate, dataclasses.replace(up, x_seed=up.x_seed + 1)])
    with pytest.raises(ValueError):
        bench.check_shared_inputs([dataclasses.replace(gate, K=2 * gate.K), up])
    with pytest.raises(ValueError):
        bench.check_shared_inputs([up])


def test_percentiles_interpolate_order_statistics():
    p = bench.percentiles([float(v) for v in range(11)])
    assert (p["median"], p["p10"], p["p90"], p["min"], p["max"]) == (5.0, 1.0, 9.0, 0.0, 10.0)


def test_group_fold_bound_uses_the_valu_peak():
    # 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz of non-packed fp32 VALU
    assert bench.PEAK_VALU_LANE_OPS == 256 * 4 * 16 * 2.4e9
    assert bench.GROUP_FOLD_VALU == {"int8": 5, "bf6": 3}
