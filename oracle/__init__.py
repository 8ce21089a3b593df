"""CPU oracle for the FoldQuantVLA runtime quantized projection.

TEST INFRASTRUCTURE.  Only tests/, the smoke check and the benchmark's
cpu_baseline leg may import this package.  It shares no code with the GPU
library and never imports it; it takes plain numpy arrays / CPU tensors.

Parts:
  * fq_oracle.c (via ctypes): the fp32 contract of the runtime prologue
    (blockwise FWHT butterfly, per-token absmax, quantize; Sec. III-C, eq. (5)),
    canonical INT4 packing, the brute-force int64 contraction and the double
    rescale (eq. (8)).
  * definitions.py: float64 definitions written out with explicit matrices
    (Sylvester H_b, block rotation R, eq. (2) fold, eq. (5), eq. (8)).
  * exact.py: exact rational arithmetic of eq. (5) for tiny inputs.
  * GPTQ in the transformed coordinates (eq. (7)): the second moment and the damped
    inverse factor with numpy (float64 matmul, inverse, Cholesky), the column sweep in
    fq_oracle.c.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import numpy as np

from . import build as _build

_LIB = None


def _lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(_build.LIB) or os.path.getmtime(_build.LIB) < os.path.getmtime(_build.SRC):
            _build.build()
        lib = ctypes.CDLL(_build.LIB)
        i64, i32, f32 = ctypes.c_int64, ctypes.c_int, ctypes.c_float
        vp = ctypes.c_void_p
        lib.fqo_fwht_quant_bf16.argtypes = [vp, i64, vp, vp, i64, i64, i64, i32, f32, vp, vp, vp]
        lib.fqo_fwht_quant_f32.argtypes = [vp, i64, vp, vp, i64, i64, i64, i32, f32, vp, vp, vp]
        lib.fqo_pack_int4.argtypes = [vp, i64, i64, vp]
        lib.fqo_transform.argtypes = [vp, i32, i64, vp, vp, i64, i64, i64, vp]
        lib.fqo_gptq_sweep.argtypes = [vp, i64, vp, i64, i64, i32, i64, f32, vp, vp, vp]
        lib.fqo_gemm_i64.argtypes = [vp, vp, i64, i64, i64, vp]
        lib.fqo_dequant.argtypes = [vp, vp, vp, vp, i64, i64, vp]
        lib.fqo_w4a16.argtypes = [vp, i64, vp, vp, vp, i64, i64, i64, vp, vp]
        lib.fqo_rotate_quant_bf16.argtypes = [vp, i64, vp, vp, vp, vp, i64, i64, i64, i32, f32, vp, vp, vp]
        lib.fqo_rotate_quant_f32.argtypes = [vp, i64, vp, vp, vp, vp, i64, i64, i64, i32, f32, vp, vp, vp]
        lib.fqo_fwht_block_f32.argtypes = [vp, i64]
        lib.fqo_fwht_block_f32.restype = None
        lib.fqo_inv_sqrt_b.argtypes = [i64]
        lib.fqo_inv_sqrt_b.restype = f32
        lib.fqo_max_threads.restype = i32
        lib.fqo_set_threads.argtypes = [i32]
        lib.fqo_set_threads.restype = None
        for name in ("fqo_fwht_quant_bf16", "fqo_fwht_quant_f32", "fqo_pack_int4", "fqo_gemm_i64",
                     "fqo_dequant", "fqo_w4a16", "fqo_rotate_quant_bf16", "fqo_rotate_quant_f32"):
            getattr(lib, name).restype = i32
        _LIB = lib
    return _LIB


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _check(rc: int, what: str):
    if rc != 0:
        raise ValueError(f"oracle {what}: bad arguments")


def max_threads() -> int:
    return int(_lib().fqo_max_threads())


def set_threads(n: int) -> None:
    _lib().fqo_set_threads(int(n))


def inv_sqrt_b(b: int) -> np.float32:
    """c_b, the float nearest to 1/sqrt(b)."""
    return np.float32(_lib().fqo_inv_sqrt_b(int(b)))


def fwht_block(v: np.ndarray) -> np.ndarray:
    """fp32 butterfly FWHT of one block (length = power of two), unnormalized."""
    out = np.ascontiguousarray(v, dtype=np.float32).copy()
    _lib().fqo_fwht_block_f32(_ptr(out), out.size)
    return out


def bf16_bits(x) -> np.ndarray:
    """uint16 bit patterns of a bf16 torch tensor (no conversion)."""
    import torch
    assert x.dtype == torch.bfloat16
    return x.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def fwht_quant(x, b: int, bits: int, clip_ratio: float = 1.0,
               chan_mult: Optional[np.ndarray] = None,
               post_mult: Optional[np.ndarray] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Runtime prologue on tokens (Alg. 1 runtime; eq. (5)).

    x: bf16 torch tensor [M, K] or uint16 bit array, or float32 array [M, K].
    chan_mult: optional fp32 [K] multiplier applied before the rotation (fold-before S^-1).
    post_mult: optional fp32 [K] multiplier applied after it (fold-after P^-1, Sec. III-C).
    Returns (codes int8 [M, K] unpacked, delta float32 [M]).
    """
    lib = _lib()
    if not isinstance(x, np.ndarray):
        x = bf16_bits(x)
    M, K = x.shape
    codes = np.zeros((M, K), dtype=np.int8)
    delta = np.zeros(M, dtype=np.float32)
    scratch = np.zeros(max(1, max_threads()) * max(K, 1), dtype=np.float32)
    cm = None if chan_mult is None else np.ascontiguousarray(chan_mult, dtype=np.float32)
    pm = None if post_mult is None else np.ascontiguousarray(post_mult, dtype=np.float32)
    if x.dtype == np.uint16:
        xx = np.ascontiguousarray(x)
        rc = lib.fqo_fwht_quant_bf16(_ptr(xx), K, _ptr(cm), _ptr(pm), M, K, b, bits, clip_ratio,
                                     _ptr(codes), _ptr(delta), _ptr(scratch))
    elif x.dtype == np.float32:
        xx = np.ascontiguousarray(x)
        rc = lib.fqo_fwht_quant_f32(_ptr(xx), K, _ptr(cm), _ptr(pm), M, K, b, bits, clip_ratio,
                                    _ptr(codes), _ptr(delta), _ptr(scratch))
    else:
        raise TypeError(f"unsupported dtype {x.dtype}")
    _check(rc, "fwht_quant")
    return codes, delta


def quantize_weights(w: np.ndarray, b: int, bits: int, col_scale: Optional[np.ndarray] = None,
                     post_scale: Optional[np.ndarray] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Offline fold + round-to-nearest (Alg. 1 offline; eq. (2) with T = P^-1 R S^-1).

    Row j of the folded weight W S R^T P is p . R (s . w_j) (fold-before S, fold-after P,
    Sec. III-C); it is rounded with the same per-row rule as a token at r = 1.
    Returns (codes int8 [N, K], s_w float32 [N]).
    """
    return fwht_quant(np.ascontiguousarray(w, dtype=np.float32), b, bits, 1.0, col_scale, post_scale)


def rotate_quant(x, perm: Optional[np.ndarray], blocks: np.ndarray, b: int, bits: int,
                 clip_ratio: float = 1.0, chan_mult: Optional[np.ndarray] = None,
                 post_mult: Optional[np.ndarray] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Prologue with the stored composite rotation of Sec. III-C in place of the block
    Hadamard: gather by `perm` (int32 [K], output position c takes input channel perm[c];
    None = identity), per-block orthogonal matrices `blocks` fp32 [K/b, b, b] applied as an
    fma chain in ascending j, then eq. (5) with nothing deferred to delta.
    x: bf16 torch tensor / uint16 bits, or float32 rows (the weight side).
    Returns (codes int8 [M, K], delta float32 [M])."""
    lib = _lib()
    if not isinstance(x, np.ndarray):
        x = bf16_bits(x)
    M, K = x.shape
    codes = np.zeros((M, K), dtype=np.int8)
    delta = np.zeros(M, dtype=np.float32)
    scratch = np.zeros(max(1, max_threads()) * 3 * max(K, 1), dtype=np.float32)
    pm_ = None if perm is None else np.ascontiguousarray(perm, dtype=np.int32)
    bl = np.ascontiguousarray(blocks, dtype=np.float32)
    assert bl.shape == (K // b, b, b)
    cm = None if chan_mult is None else np.ascontiguousarray(chan_mult, dtype=np.float32)
    po = None if post_mult is None else np.ascontiguousarray(post_mult, dtype=np.float32)
    xx = np.ascontiguousarray(x)
    fn = lib.fqo_rotate_quant_bf16 if xx.dtype == np.uint16 else lib.fqo_rotate_quant_f32
    if xx.dtype not in (np.uint16, np.float32):
        raise TypeError(f"unsupported dtype {xx.dtype}")
    rc = fn(_ptr(xx), K, _ptr(pm_), _ptr(bl), _ptr(cm), _ptr(po), M, K, b, bits, clip_ratio,
            _ptr(codes), _ptr(delta), _ptr(scratch))
    _check(rc, "rotate_quant")
    return codes, delta


def quantize_weights_rotated(w: np.ndarray, perm: Optional[np.ndarray], blocks: np.ndarray, b: int,
                             bits: int, col_scale: Optional[np.ndarray] = None,
                             post_scale: Optional[np.ndarray] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Offline fold + RTN for the composite rotation R = B P: row j of W S R^T P_out is
    p . R (s . w_j), rounded with the token rule at r = 1."""
    return rotate_quant(np.ascontiguousarray(w, dtype=np.float32), perm, blocks, b, bits, 1.0,
                        col_scale, post_scale)


def pack_int4(codes: np.ndarray) -> np.ndarray:
    """Canonical nibble packing: channel 2i -> low nibble of byte i."""
    codes = np.ascontiguousarray(codes, dtype=np.int8)
    M, K = codes.shape
    out = np.zeros((M, K // 2), dtype=np.uint8)
    _check(_lib().fqo_pack_int4(_ptr(codes), M, K, _ptr(out)), "pack_int4")
    return out


def gemm(qa: np.ndarray, qw: np.ndarray) -> np.ndarray:
    """acc[t, j] = sum_c qa[t, c] qw[j, c] in int64 (eq. (8) accumulator)."""
    qa = np.ascontiguousarray(qa, dtype=np.int8)
    qw = np.ascontiguousarray(qw, dtype=np.int8)
    M, K = qa.shape
    N, K2 = qw.shape
    assert K == K2
    acc = np.zeros((M, N), dtype=np.int64)
    _check(_lib().fqo_gemm_i64(_ptr(qa), _ptr(qw), M, N, K, _ptr(acc)), "gemm")
    return acc


def dequant(acc: np.ndarray, delta: np.ndarray, s_w: np.ndarray,
            bias: Optional[np.ndarray] = None) -> np.ndarray:
    """y[t, j] = s_w[j] delta[t] acc[t, j] + bias[j] in double (eq. (8))."""
    acc = np.ascontiguousarray(acc, dtype=np.int64)
    M, N = acc.shape
    y = np.zeros((M, N), dtype=np.float64)
    d = np.ascontiguousarray(delta, dtype=np.float32)
    s = np.ascontiguousarray(s_w, dtype=np.float32)
    bb = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
    _check(_lib().fqo_dequant(_ptr(acc), _ptr(d), _ptr(s), _ptr(bb), M, N, _ptr(y)), "dequant")
    return y


def w4a16(x, w_codes: np.ndarray, s_w: np.ndarray,
          bias: Optional[np.ndarray] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Weight-only INT4 projection (Sec. III-A, the adaptive layer-norm modulation path):
    bf16 tokens x [M, K] (torch tensor or uint16 bits) times INT4 weight codes [N, K] with
    per-output-channel scales.  Returns (acc, y) in float64: acc = x q^T, y = s_w acc + bias."""
    lib = _lib()
    if not isinstance(x, np.ndarray):
        x = bf16_bits(x)
    xx = np.ascontiguousarray(x, dtype=np.uint16)
    M, K = xx.shape
    qw = np.ascontiguousarray(w_codes, dtype=np.int8)
    N, K2 = qw.shape
    assert K == K2
    acc = np.zeros((M, N), dtype=np.float64)
    y = np.zeros((M, N), dtype=np.float64)
    s = np.ascontiguousarray(s_w, dtype=np.float32)
    bb = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
    _check(lib.fqo_w4a16(_ptr(xx), K, _ptr(qw), _ptr(s), _ptr(bb), M, N, K, _ptr(acc), _ptr(y)), "w4a16")
    return acc, y


def linear(x, w_codes: np.ndarray, s_w: np.ndarray, b: int, bits: int,
           clip_ratio: float = 1.0, smooth_inv: Optional[np.ndarray] = None,
           bias: Optional[np.ndarray] = None, post_inv: Optional[np.ndarray] = None):
    """Whole runtime path of Alg. 1 for one consumer: returns (codes, delta, acc, y)."""
    codes, delta = fwht_quant(x, b, bits, clip_ratio, smooth_inv, post_inv)
    acc = gemm(codes, w_codes)
    y = dequant(acc, delta, s_w, bias)
    return codes, delta, acc, y


def transform(x, b: int, chan_mult: Optional[np.ndarray] = None,
              post_mult: Optional[np.ndarray] = None) -> np.ndarray:
    """The prologue's transform alone (optional fold-before multiplier, unnormalized
    blockwise butterfly, optional fold-after multiplier), fp32 [M, K]: the coordinates of
    eq. (7).  x: bf16 torch tensor / uint16 bits, or float32 rows (weights)."""
    if not isinstance(x, np.ndarray):
        x = bf16_bits(x)
    xx = np.ascontiguousarray(x)
    if xx.dtype not in (np.uint16, np.float32):
        raise TypeError(f"unsupported dtype {xx.dtype}")
    M, K = xx.shape
    z = np.zeros((M, K), dtype=np.float32)
    cm = None if chan_mult is None else np.ascontiguousarray(chan_mult, dtype=np.float32)
    po = None if post_mult is None else np.ascontiguousarray(post_mult, dtype=np.float32)
    _check(_lib().fqo_transform(_ptr(xx), int(xx.dtype == np.uint16), K, _ptr(cm), _ptr(po), M, K, b,
                                _ptr(z)), "transform")
    return z


def gptq_hessian(z: np.ndarray) -> np.ndarray:
    """G = Z Z^T of eq. (7) in float64 (z: calibration tokens as rows [T, K], so G = z^T z)."""
    z64 = np.asarray(z, dtype=np.float64)
    return z64.T @ z64


def gptq_damped(G: np.ndarray, damp: float = 0.01) -> np.ndarray:
    """H = G + lambda I with lambda = damp * mean(diag G) (the GPTQ method's diagonal damping
    named in Sec. III-F); a second moment that is all zero (no calibration signal) gives I."""
    G = np.asarray(G, dtype=np.float64)
    lam = damp * float(np.mean(np.diag(G)))
    if lam == 0.0:
        return np.eye(G.shape[0])
    return G + lam * np.eye(G.shape[0])


def gptq_factor(G: np.ndarray, damp: float = 0.01) -> np.ndarray:
    """U: upper triangular with H^-1 = U^T U, H the damped second moment (float64)."""
    H = gptq_damped(G, damp)
    return np.ascontiguousarray(np.linalg.cholesky(np.linalg.inv(H)).T)


def gptq_sweep(w_t: np.ndarray, U: np.ndarray, bits: int, blk: int = 128,
               scale_mult: float = 1.0) -> Tuple[np.ndarray, np.ndarray]:
    """The GPTQ column sweep on folded rows w_t fp32 [N, K] with factor U fp64 [K, K].
    Returns (codes int8 [N, K], scales fp32 [N]); scales = fl32(max|row| * scale_mult / q)."""
    w_t = np.ascontiguousarray(w_t, dtype=np.float32)
    U = np.ascontiguousarray(U, dtype=np.float64)
    N, K = w_t.shape
    assert U.shape == (K, K)
    codes = np.zeros((N, K), dtype=np.int8)
    scales = np.zeros(N, dtype=np.float32)
    scratch = np.zeros(max(1, max_threads()) * (K + blk), dtype=np.float64)
    _check(_lib().fqo_gptq_sweep(_ptr(w_t), K, _ptr(U), N, K, bits, blk, float(scale_mult), _ptr(codes),
                                 _ptr(scales), _ptr(scratch)), "gptq_sweep")
    return codes, scales


def gptq_quantize_weights(w: np.ndarray, calib, b: int, bits: int, col_scale: Optional[np.ndarray] = None,
                          post_scale: Optional[np.ndarray] = None, smooth_inv: Optional[np.ndarray] = None,
                          post_inv: Optional[np.ndarray] = None, damp: float = 0.01,
                          blk: int = 128) -> Tuple[np.ndarray, np.ndarray]:
    """Eq. (7) end to end: calibration tokens (bf16 [T, K]) through the prologue's transform
    (with the tokens' multipliers), G = Z Z^T, the damped factor, and the sweep over the
    folded weight rows (row j = p . H_b (s . w_j), unnormalized; scale carries c_b)."""
    z = transform(calib, b, smooth_inv, post_inv)
    U = gptq_factor(gptq_hessian(z), damp)
    w_t = transform(np.ascontiguousarray(w, dtype=np.float32), b, col_scale, post_scale)
    return gptq_sweep(w_t, U, bits, blk, float(inv_sqrt_b(b)))
