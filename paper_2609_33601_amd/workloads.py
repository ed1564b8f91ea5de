"""Seeded synthetic inputs for the W4A4 linear.

This module only draws random numbers and shapes them into the workloads the
paper's deployed models run (FLUX-12B-class DiT block linears and 8B
diffusion-LLM block linears, Sec. 4 experimental matrix).  It holds none of the
layer's arithmetic: no quantisation, packing, contraction or epilogue.  Both the
CPU oracle and the GPU path take their inputs from here.

Everything is returned as numpy arrays of bf16 bit patterns (uint16).  The fp32
-> bf16 conversion of the drawn values is torch's CPU cast (round-to-nearest-
even), a library routine.

Recipe (per linear):
  * activations X [M,K]: standard normal, Student-t(3)/sqrt(3) (unit variance,
    heavy tails) or GELU(standard normal) (exact erf GELU); then
    round(frac*K) distinct whole columns ("outlier channels", chosen by their
    own generator) are multiplied by a factor;
  * weights W [N,K]: N(0, std^2);
  * bias [N] (where the workload has one): N(0, 0.01^2).
Generators are numpy PCG64 seeded per tensor: X = base, W = base+1,
bias = base+2, outlier columns = base+3; a workload with several linears uses
base = 10*j for its j-th distinct input or weight.
"""

from dataclasses import dataclass, field
from typing import Optional, Tuple

import numpy as np


def _to_bf16_bits(x_f32: np.ndarray) -> np.ndarray:
    import torch

    t = torch.from_numpy(np.ascontiguousarray(x_f32, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def activations(M: int, K: int, dist: str, seed: int,
                outlier_frac: float = 0.0, outlier_factor: float = 1.0) -> np.ndarray:
    """Synthetic activations X [M,K] as bf16 bits."""
    g = _rng(seed)
    if dist == "normal":
        x = g.standard_normal((M, K), dtype=np.float32)
    elif dist == "student_t3":
        x = (g.standard_t(3.0, size=(M, K)) / np.sqrt(3.0)).astype(np.float32)
    elif dist == "gelu_normal":
        import torch

        z = torch.from_numpy(g.standard_normal((M, K), dtype=np.float32))
        x = torch.nn.functional.gelu(z, approximate="none").numpy()
    else:
        raise ValueError(f"unknown activation distribution {dist!r}")
    n_out = int(round(outlier_frac * K))
    if n_out > 0:
        cols = _rng(seed + 3).choice(K, size=n_out, replace=False)
        x[:, cols] *= np.float32(outlier_factor)
    return _to_bf16_bits(x)


def weights(N: int, K: int, std: float, seed: int) -> np.ndarray:
    """Synthetic weight W [N,K] ~ N(0, std^2) as bf16 bits."""
    w = _rng(seed).standard_normal((N, K), dtype=np.float32) * np.float32(std)
    return _to_bf16_bits(w)


def bias(N: int, std: float, seed: int) -> np.ndarray:
    """Synthetic bias [N] ~ N(0, std^2) as bf16 bits."""
    b = _rng(seed).standard_normal((N,), dtype=np.float32) * np.float32(std)
    return _to_bf16_bits(b)


@dataclass(frozen=True)
class Linear:
    """One linear y = x W^T + b of a workload."""

    name: str
    M: int
    K: int
    N: int
    x_dist: str
    x_seed: int
    outlier_frac: float
    outlier_factor: float
    w_std: float
    w_seed: int
    bias_std: Optional[float] = None
    bias_seed: int = 2
    # the input is the previous linear's (one quantisation serves both)
    shares_input: bool = False

    @property
    def ops(self) -> int:
        return 2 * self.M * self.N * self.K

    def make_x(self) -> np.ndarray:
        return activations(self.M, self.K, self.x_dist, self.x_seed,
                           self.outlier_frac, self.outlier_factor)

    def make_w(self) -> np.ndarray:
        return weights(self.N, self.K, self.w_std, self.w_seed)

    def make_bias(self) -> Optional[np.ndarray]:
        if self.bias_std is None:
            return None
        return bias(self.N, self.bias_std, self.bias_seed)


@dataclass(frozen=True)
class Workload:
    name: str
    description: str
    linears: Tuple[Linear, ...] = field(default_factory=tuple)

    @property
    def ops(self) -> int:
        return sum(l.ops for l in self.linears)


def _dit_act(M, K, seed=0, frac=0.005, factor=50.0):
    return dict(M=M, K=K, x_dist="student_t3", x_seed=seed,
                outlier_frac=frac, outlier_factor=factor)


WORKLOADS = {
    "tiny": Workload(
        "tiny", "W4A4 linear 64x256 -> 256, normal activations with 1% outlier channels x20",
        (Linear("tiny", M=64, K=256, N=256, x_dist="normal", x_seed=0,
                outlier_frac=0.01, outlier_factor=20.0, w_std=0.02, w_seed=1),),
    ),
    "attn_proj": Workload(
        "attn_proj", "DiT attention projection 4608x3072 -> 3072",
        (Linear("attn_proj", N=3072, w_std=0.02, w_seed=1, **_dit_act(4608, 3072)),),
    ),
    "qkv": Workload(
        "qkv", "DiT fused QKV 4608x3072 -> 9216 with bias",
        (Linear("qkv", N=9216, w_std=0.02, w_seed=1, bias_std=0.01, bias_seed=2,
                **_dit_act(4608, 3072)),),
    ),
    "mlp_up": Workload(
        "mlp_up", "FLUX-12B MLP-up 4608x3072 -> 12288 with bias",
        (Linear("mlp_up", N=12288, w_std=0.02, w_seed=1, bias_std=0.01, bias_seed=2,
                **_dit_act(4608, 3072)),),
    ),
    "mlp_down": Workload(
        "mlp_down", "FLUX-12B MLP-down, two images: 9216x12288 -> 3072, GELU activations",
        (Linear("mlp_down", M=9216, K=12288, N=3072, x_dist="gelu_normal", x_seed=0,
                outlier_frac=0.005, outlier_factor=30.0, w_std=0.01, w_seed=1),),
    ),
    "mlp_down_1img": Workload(
        "mlp_down_1img", "FLUX-12B MLP-down, one image: 4608x12288 -> 3072",
        (Linear("mlp_down_1img", M=4608, K=12288, N=3072, x_dist="gelu_normal", x_seed=0,
                outlier_frac=0.005, outlier_factor=30.0, w_std=0.01, w_seed=1),),
    ),
    "dllm_block": Workload(
        "dllm_block",
        "8B diffusion-LLM block: gate, up (4096x4096 -> 12288, shared input), "
        "o-proj 4096x4096 -> 4096, down 4096x12288 -> 4096",
        (
            Linear("dllm_gate", N=12288, w_std=0.02, w_seed=1, **_dit_act(4096, 4096, seed=0)),
            Linear("dllm_up", N=12288, w_std=0.02, w_seed=11, shares_input=True, **_dit_act(4096, 4096, seed=0)),
            Linear("dllm_o", N=4096, w_std=0.02, w_seed=21, **_dit_act(4096, 4096, seed=0)),
            Linear("dllm_down", N=4096, w_std=0.02, w_seed=31, **_dit_act(4096, 12288, seed=10)),
        ),
    ),
}

# The headline step: the two FLUX-12B MLP linears run back-to-back.
FLUX_MLP = Workload(
    "flux_mlp",
    "FLUX-12B MLP linears back-to-back: up 4608x3072 -> 12288 (+bias), "
    "down 9216x12288 -> 3072 (two images)",
    (WORKLOADS["mlp_up"].linears[0], WORKLOADS["mlp_down"].linears[0]),
)
