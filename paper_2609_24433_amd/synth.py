"""Seeded synthetic inputs for the quantized projection.

This module only draws random numbers.  It holds none of the projection's
arithmetic (no transform, no quantizer, no GEMM): activations are returned as
raw bf16 rows, weights as raw fp32 matrices, and integer codes as plain random
integers.  Both the GPU path and the CPU oracle consume what it returns, so
nothing here may depend on either of them.

Distributions follow the workloads the paper motivates (Sec. III-A: per-token
activation spread with a few huge channels at the worst language layer):
token rows are N(0, 1) or Student-t(3), with a seeded set of outlier channels
multiplied by a constant factor across all tokens; weights are N(0, 0.02).
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import numpy as np
import torch


def outlier_channels(K: int, frac: float, seed: int) -> np.ndarray:
    """Sorted indices of round(frac*K) distinct channels, drawn with `seed`."""
    n = int(round(frac * K))
    if n <= 0:
        return np.zeros(0, dtype=np.int64)
    rng = np.random.default_rng(seed)
    return np.sort(rng.choice(K, size=n, replace=False)).astype(np.int64)


def activations(M: int, K: int, *, seed: int, outlier_frac: float = 0.0,
                outlier_scale: float = 1.0, outlier_seed: Optional[int] = None,
                dist: str = "normal") -> torch.Tensor:
    """bf16 [M, K] token rows (CPU tensor).

    dist: "normal" -> N(0,1); "student_t3" -> Student-t with 3 degrees of freedom.
    Outlier channels (drawn with `outlier_seed`, default seed+1) are scaled by
    `outlier_scale` in every token.  fp32 -> bf16 uses torch's round-to-nearest-even.
    """
    rng = np.random.default_rng(seed)
    if dist == "normal":
        x = rng.standard_normal((M, K), dtype=np.float32)
    elif dist == "student_t3":
        x = rng.standard_t(3.0, size=(M, K)).astype(np.float32)
    else:
        raise ValueError(f"unknown distribution {dist!r}")
    if outlier_frac > 0.0:
        idx = outlier_channels(K, outlier_frac, seed + 1 if outlier_seed is None else outlier_seed)
        x[:, idx] *= np.float32(outlier_scale)
    return torch.from_numpy(x).to(torch.bfloat16)


def weights(N: int, K: int, *, seed: int, std: float = 0.02) -> np.ndarray:
    """fp32 [N, K] weight matrix ~ N(0, std^2) (row j = output channel j)."""
    rng = np.random.default_rng(seed)
    w = rng.standard_normal((N, K), dtype=np.float32)
    w *= np.float32(std)
    return w


def channel_vector(K: int, *, seed: int, low: float, high: float) -> np.ndarray:
    """fp32 [K] vector ~ U(low, high): a positive per-channel gain or smoothing scale."""
    rng = np.random.default_rng(seed)
    return rng.uniform(low, high, size=K).astype(np.float32)


def random_codes(M: int, K: int, bits: int, *, seed: int) -> np.ndarray:
    """int8 [M, K] integers uniform in [-(2^(bits-1)-1), 2^(bits-1)-1]."""
    q = (1 << (bits - 1)) - 1
    rng = np.random.default_rng(seed)
    return rng.integers(-q, q + 1, size=(M, K), dtype=np.int8)


def permutation(K: int, *, seed: int) -> np.ndarray:
    """int32 [K]: a uniformly random permutation of 0..K-1."""
    return np.random.default_rng(seed).permutation(K).astype(np.int32)


def orthogonal_blocks(nb: int, b: int, *, seed: int) -> np.ndarray:
    """fp32 [nb, b, b]: nb random orthogonal b x b matrices (Q factors of Gaussian draws), the
    shape of a stored per-block rotation whose entries are dense and of mixed sign."""
    rng = np.random.default_rng(seed)
    return np.stack([np.linalg.qr(rng.standard_normal((b, b)))[0] for _ in range(nb)]).astype(np.float32)


def random_scales(n: int, *, seed: int, low: float = 1e-3, high: float = 1e-1) -> np.ndarray:
    """fp32 [n] positive scales ~ U(low, high)."""
    rng = np.random.default_rng(seed)
    return rng.uniform(low, high, size=n).astype(np.float32)


# ---------------------------------------------------------------------------
# Named workloads.  Shapes are those of a VLA language backbone / action expert;
# each projection lists (name, site, K, N, bits).  A site is one shared activation
# that several projections consume (Sec. III-B).
# ---------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class Projection:
    name: str
    site: str
    K: int
    N: int
    bits: int
    weight_seed: int


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    M: int
    b: int
    projections: List[Projection]
    outlier_frac: float
    outlier_scale: float
    dist: str
    seed_base: int

    def sites(self) -> Dict[str, int]:
        """site -> K, in first-use order."""
        out: Dict[str, int] = {}
        for p in self.projections:
            out.setdefault(p.site, p.K)
        return out

    def site_activation(self, site: str, step: int, M: Optional[int] = None) -> torch.Tensor:
        """bf16 [M, K] activation of `site` at denoising/forward step `step`."""
        names = list(self.sites().keys())
        s = names.index(site)
        K = self.sites()[site]
        return activations(self.M if M is None else M, K,
                           seed=self.seed_base + 100 + 10 * s + step,
                           outlier_frac=self.outlier_frac, outlier_scale=self.outlier_scale,
                           outlier_seed=self.seed_base + 50 + s, dist=self.dist)

    def projection_weight(self, p: Projection) -> np.ndarray:
        return weights(p.N, p.K, seed=p.weight_seed)

    def ops_per_step(self, M: Optional[int] = None) -> int:
        m = self.M if M is None else M
        return sum(2 * m * p.N * p.K for p in self.projections)


def _layer(name: str, M: int, width: int, kv: int, ffn: int, seed_base: int,
           o_bits: int = 4, down_bits: int = 4) -> Workload:
    spec = [("q", "A", width, width, 4), ("k", "A", width, kv, 4), ("v", "A", width, kv, 4),
            ("o", "O", width, width, o_bits), ("gate", "B", width, ffn, 4),
            ("up", "B", width, ffn, 4), ("down", "D", ffn, width, down_bits)]
    projs = [Projection(n, s, K, N, bits, seed_base + i) for i, (n, s, K, N, bits) in enumerate(spec)]
    return Workload(name, M, 128, projs, 0.005, 50.0, "normal", seed_base)


def action_expert_layer() -> Workload:
    """Action-expert layer at width 1024: M=50 action tokens per denoising step,
    q/k/v/o 1024->1024 (k/v 1024->256), gate/up 1024->4096, down 4096->1024,
    all W4A4, Hadamard block 128, 0.5% outlier channels x50."""
    return _layer("action_expert_w1024_m50", 50, 1024, 256, 4096, 2000)


def backbone_layer() -> Workload:
    """Language-backbone layer at width 2048: M=816 prefix tokens, q/o 2048->2048,
    k/v 2048->256, gate/up 2048->16384, down 16384->2048, all W4A4, block 128."""
    return _layer("backbone_w2048_m816", 816, 2048, 256, 16384, 3000)


def backbone_layer_mixed(layer: int = 0) -> Workload:
    """Backbone layer with o_proj and down_proj in W8A8 (selective INT8, Sec. III-G)."""
    return _layer(f"backbone_mixed_l{layer}", 816, 2048, 256, 16384, 4000 + 10 * layer,
                  o_bits=8, down_bits=8)


def single_linear() -> Workload:
    """Single W4A4 linear: M=64, K=N=1024, block 64, N(0,1) rows with 1% outliers x30."""
    return Workload("single_m64_k1024_n1024", 64, 64,
                    [Projection("linear", "X", 1024, 1024, 4, 1)], 0.01, 30.0, "normal", 0)


def down_proj_sweep_point(M: int, b: int, bits: int) -> Workload:
    """Down-projection stress point: K=16384 -> N=2048, Student-t(3) rows with
    0.5% outlier channels x100."""
    seed = 5000 + 100 * bits + 10 * [1, 16, 50, 256, 816, 4096].index(M) + [32, 64, 128, 256].index(b) \
        if M in (1, 16, 50, 256, 816, 4096) and b in (32, 64, 128, 256) else 5999
    return Workload(f"down_k16384_n2048_m{M}_b{b}_w{bits}a{bits}", M, b,
                    [Projection("down", "D", 16384, 2048, bits, seed + 7)], 0.005, 100.0,
                    "student_t3", seed)
