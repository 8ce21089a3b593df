"""Python binding of libfq (the C ABI in include/fq.h), over torch device tensors.

Argument marshalling only: tensors are used for their device pointers and torch's
current HIP stream; every step of the projection runs in the library's kernels.
If libfq.so is missing the import fails loudly; there is no CPU fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfq.so")

FQ_OK = 0
_STATUS = {1: "FQ_ERR_NULL", 2: "FQ_ERR_SHAPE", 3: "FQ_ERR_UNSUPPORTED", 4: "FQ_ERR_ALIGN",
           5: "FQ_ERR_WORKSPACE", 6: "FQ_ERR_HIP", 7: "FQ_ERR_ALIAS"}

EXPORTED = ["fq_fwht_quant", "fq_quantize_weights", "fq_packed_weight_bytes", "fq_pack_weights",
            "fq_unpack_weights", "fq_gemm_workspace_bytes", "fq_gemm_w4a4", "fq_gemm_w8a8",
            "fq_linear_workspace_bytes", "fq_linear", "fq_gemm_w4a16_workspace_bytes", "fq_gemm_w4a16",
            "fq_rotate_quant_workspace_bytes", "fq_rotate_quant", "fq_quantize_weights_rotated",
            "fq_transform", "fq_gptq_hessian", "fq_gptq_factor_workspace_bytes", "fq_gptq_factor",
            "fq_gptq_sweep_workspace_bytes", "fq_gptq_sweep",
            "fq_linear_static_max_workspace_bytes", "fq_linear_static",
            "fq_status_string", "fq_last_error"]


class FQError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{_STATUS.get(status, status)}: {message}")
        self.status = status


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                          "(python -m paper_2609_24433_amd.build)")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i64, i32, f32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
    sig = {
        "fq_fwht_quant": [vp, i64, vp, vp, i64, i64, i32, i32, f32, vp, vp, vp],
        "fq_quantize_weights": [vp, i64, vp, vp, i64, i64, i32, i32, vp, vp, vp],
        "fq_pack_weights": [vp, i64, i64, i32, vp, vp],
        "fq_unpack_weights": [vp, i64, i64, i32, vp, vp],
        "fq_gemm_w4a4": [vp, vp, vp, vp, vp, vp, i64, vp, i64, i64, i64, vp, sz, vp],
        "fq_gemm_w8a8": [vp, vp, vp, vp, vp, vp, i64, vp, i64, i64, i64, vp, sz, vp],
        "fq_linear": [vp, i64, vp, vp, i64, i64, i64, i32, i32, f32, vp, vp, vp, vp, i64, vp, sz, vp],
        "fq_gemm_w4a16": [vp, i64, vp, vp, vp, vp, i64, vp, i64, i64, i64, vp, sz, vp],
        "fq_rotate_quant": [vp, i64, vp, vp, vp, vp, i64, i64, i32, i32, f32, vp, vp, vp, sz, vp],
        "fq_quantize_weights_rotated": [vp, i64, vp, vp, vp, vp, i64, i64, i32, i32, vp, vp, vp, sz, vp],
        "fq_transform": [vp, i32, i64, vp, vp, i64, i64, i32, vp, vp],
        "fq_gptq_hessian": [vp, i64, i64, i64, vp, i32, vp],
        "fq_gptq_factor": [vp, i64, ctypes.c_double, vp, vp, sz, vp],
        "fq_gptq_sweep": [vp, i64, vp, i64, i64, i32, i32, vp, vp, vp, sz, vp],
        "fq_linear_static": [vp, i64, vp, vp, i64, i64, i64, i32, i32, f32, vp, vp, vp, vp, i64, vp],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    for name, args in {"fq_packed_weight_bytes": [i64, i64, i32],
                       "fq_gemm_workspace_bytes": [i64, i64, i64, i32],
                       "fq_linear_workspace_bytes": [i64, i64, i64, i32],
                       "fq_gemm_w4a16_workspace_bytes": [i64, i64, i64],
                       "fq_rotate_quant_workspace_bytes": [i64, i64],
                       "fq_gptq_factor_workspace_bytes": [i64],
                       "fq_gptq_sweep_workspace_bytes": [i64, i64],
                       "fq_linear_static_max_workspace_bytes": []}.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = sz
    lib.fq_status_string.argtypes = [ctypes.c_int]
    lib.fq_status_string.restype = ctypes.c_char_p
    lib.fq_last_error.argtypes = []
    lib.fq_last_error.restype = ctypes.c_char_p
    return lib


LIB = _load()


def _check(rc: int) -> None:
    if rc != FQ_OK:
        raise FQError(rc, LIB.fq_last_error().decode())


def _p(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream: Optional[torch.cuda.Stream] = None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


# ---------------------------------------------------------------- raw C-ABI calls (pointers)

def fwht_quant_raw(x_ptr, ldx, smooth_ptr, M, K, b, bits, clip_ratio, codes_ptr, delta_ptr, stream_ptr,
                   post_ptr=None):
    _check(LIB.fq_fwht_quant(x_ptr, ldx, smooth_ptr, post_ptr, M, K, b, bits, clip_ratio, codes_ptr, delta_ptr,
                             stream_ptr))


# ---------------------------------------------------------------- tensor API

def code_bytes(K: int, bits: int) -> int:
    return K * bits // 8


def _require(cond: bool, msg: str) -> None:
    if not cond:
        raise ValueError(msg)


def _check_out(out: Optional[torch.Tensor], M: int, N: int) -> None:
    """A caller-supplied output must be what the library writes: bf16 [M, N] rows with unit
    column stride (the row stride is passed on as ldy)."""
    if out is not None:
        _require(out.dtype == torch.bfloat16 and tuple(out.shape) == (M, N) and (M == 0 or out.stride(1) == 1),
                 "out: bf16 [M, N] with unit column stride")


def fwht_quant(x: torch.Tensor, b: int, bits: int, clip_ratio: float = 1.0,
               smooth_inv: Optional[torch.Tensor] = None, out_codes: Optional[torch.Tensor] = None,
               out_delta: Optional[torch.Tensor] = None,
               post_inv: Optional[torch.Tensor] = None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Prologue: x bf16 [M, K] (row stride x.stride(0)) -> (codes uint8 [M, K*bits/8], delta fp32 [M]).
    smooth_inv: fold-before S^-1 (before the rotation); post_inv: fold-after P^-1 (after it)."""
    M, K = x.shape
    assert x.dtype == torch.bfloat16 and (M == 0 or x.stride(1) == 1)
    if out_codes is not None:
        _require(out_codes.dtype in (torch.uint8, torch.int8) and out_codes.is_contiguous()
                 and tuple(out_codes.shape) == (M, code_bytes(K, bits)), "out_codes: contiguous [M, K*bits/8] bytes")
    if out_delta is not None:
        _require(out_delta.dtype == torch.float32 and out_delta.is_contiguous() and out_delta.numel() == M,
                 "out_delta: contiguous fp32 [M]")
    codes = out_codes if out_codes is not None else torch.empty((M, code_bytes(K, bits)), dtype=torch.uint8, device=x.device)
    delta = out_delta if out_delta is not None else torch.empty((M,), dtype=torch.float32, device=x.device)
    _check(LIB.fq_fwht_quant(_p(x), x.stride(0) if M else K, _p(smooth_inv), _p(post_inv), M, K, b, bits,
                             clip_ratio, _p(codes), _p(delta), _stream()))
    return codes, delta


def quantize_weights(w: torch.Tensor, b: int, bits: int, col_scale: Optional[torch.Tensor] = None,
                     post_scale: Optional[torch.Tensor] = None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Offline fold + RTN: w fp32 [N, K] -> (codes int8 [N, K], scales fp32 [N]).
    col_scale: fold-before S (before the rotation); post_scale: fold-after P (after it)."""
    N, K = w.shape
    assert w.dtype == torch.float32 and w.stride(1) == 1
    codes = torch.empty((N, K), dtype=torch.int8, device=w.device)
    scale = torch.empty((N,), dtype=torch.float32, device=w.device)
    _check(LIB.fq_quantize_weights(_p(w), w.stride(0), _p(col_scale), _p(post_scale), N, K, b, bits, _p(codes),
                                   _p(scale), _stream()))
    return codes, scale


def packed_weight_bytes(N: int, K: int, bits: int) -> int:
    return int(LIB.fq_packed_weight_bytes(N, K, bits))


def pack_weights(codes: torch.Tensor, bits: int) -> torch.Tensor:
    N, K = codes.shape
    assert codes.dtype == torch.int8 and codes.is_contiguous()
    out = torch.empty((packed_weight_bytes(N, K, bits),), dtype=torch.uint8, device=codes.device)
    _check(LIB.fq_pack_weights(_p(codes), N, K, bits, _p(out), _stream()))
    return out


def unpack_weights(packed: torch.Tensor, N: int, K: int, bits: int) -> torch.Tensor:
    out = torch.empty((N, K), dtype=torch.int8, device=packed.device)
    _check(LIB.fq_unpack_weights(_p(packed), N, K, bits, _p(out), _stream()))
    return out


def gemm_workspace_bytes(M: int, N: int, K: int, bits: int) -> int:
    return int(LIB.fq_gemm_workspace_bytes(M, N, K, bits))


def linear_workspace_bytes(M: int, N: int, K: int, bits: int) -> int:
    return int(LIB.fq_linear_workspace_bytes(M, N, K, bits))


def workspace(nbytes: int, device) -> torch.Tensor:
    """Scratch for the GEMM / fused-linear entry points (no initialization needed)."""
    return torch.empty((max(nbytes, 256),), dtype=torch.uint8, device=device)


def gemm(a_codes: torch.Tensor, delta: torch.Tensor, w_packed: torch.Tensor, w_scale: torch.Tensor,
         N: int, K: int, bits: int, bias: Optional[torch.Tensor] = None, want_acc: bool = False,
         ws: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None):
    """Integer GEMM + eq. (8) epilogue.  Returns y bf16 [M, N] (and int32 acc if want_acc)."""
    M = a_codes.shape[0]
    _require(a_codes.dtype in (torch.uint8, torch.int8) and tuple(a_codes.shape) == (M, code_bytes(K, bits))
             and a_codes.is_contiguous(), "a_codes: canonical contiguous [M, K*bits/8] bytes")
    _check_out(out, M, N)
    y = out if out is not None else torch.empty((M, N), dtype=torch.bfloat16, device=a_codes.device)
    acc = torch.empty((M, N), dtype=torch.int32, device=a_codes.device) if want_acc else None
    if ws is None:
        ws = workspace(gemm_workspace_bytes(M, N, K, bits), a_codes.device)
    fn = LIB.fq_gemm_w4a4 if bits == 4 else LIB.fq_gemm_w8a8
    _check(fn(_p(a_codes), _p(delta), _p(w_packed), _p(w_scale), _p(bias), _p(y), y.stride(0) if M else N, _p(acc),
              M, N, K, _p(ws), ws.numel(), _stream()))
    return (y, acc) if want_acc else y


def linear(x: torch.Tensor, w_packed: torch.Tensor, w_scale: torch.Tensor, N: int, b: int, bits: int,
           clip_ratio: float = 1.0, smooth_inv: Optional[torch.Tensor] = None,
           bias: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
           out: Optional[torch.Tensor] = None, post_inv: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Fused projection: bf16 x [M, K] -> bf16 y [M, N]."""
    M, K = x.shape
    assert x.dtype == torch.bfloat16 and (M == 0 or x.stride(1) == 1)
    _check_out(out, M, N)
    y = out if out is not None else torch.empty((M, N), dtype=torch.bfloat16, device=x.device)
    if ws is None:
        ws = workspace(linear_workspace_bytes(M, N, K, bits), x.device)
    _check(LIB.fq_linear(_p(x), x.stride(0) if M else K, _p(smooth_inv), _p(post_inv), M, K, N, b, bits, clip_ratio,
                         _p(w_packed), _p(w_scale), _p(bias), _p(y), y.stride(0) if M else N, _p(ws), ws.numel(),
                         _stream()))
    return y


def linear_static(x: torch.Tensor, w_packed: torch.Tensor, w_scale: torch.Tensor, N: int, b: int, bits: int,
                  clip_ratio: float = 1.0, smooth_inv: Optional[torch.Tensor] = None,
                  bias: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None,
                  post_inv: Optional[torch.Tensor] = None) -> torch.Tensor:
    """fq_linear without a workspace argument: the library's own device scratch (calls that
    overlap on one device race)."""
    M, K = x.shape
    _require(x.dtype == torch.bfloat16 and (M == 0 or x.stride(1) == 1), "x: bf16 [M, K] with unit column stride")
    _check_out(out, M, N)
    y = out if out is not None else torch.empty((M, N), dtype=torch.bfloat16, device=x.device)
    _check(LIB.fq_linear_static(_p(x), x.stride(0) if M else K, _p(smooth_inv), _p(post_inv), M, K, N, b, bits,
                                clip_ratio, _p(w_packed), _p(w_scale), _p(bias), _p(y), y.stride(0) if M else N,
                                _stream()))
    return y


def rotate_quant(x: torch.Tensor, perm: Optional[torch.Tensor], blocks: torch.Tensor, b: int, bits: int,
                 clip_ratio: float = 1.0, smooth_inv: Optional[torch.Tensor] = None,
                 post_inv: Optional[torch.Tensor] = None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Prologue with the stored composite rotation (permutation int32 [K] or None, blocks fp32
    [K/b, b, b]): x bf16 [M, K] -> (codes [M, K*bits/8], delta fp32 [M])."""
    M, K = x.shape
    assert x.dtype == torch.bfloat16 and (M == 0 or x.stride(1) == 1)
    codes = torch.empty((M, code_bytes(K, bits)), dtype=torch.uint8, device=x.device)
    delta = torch.empty((M,), dtype=torch.float32, device=x.device)
    ws = workspace(int(LIB.fq_rotate_quant_workspace_bytes(M, K)), x.device)
    _check(LIB.fq_rotate_quant(_p(x), x.stride(0) if M else K, _p(perm), _p(blocks), _p(smooth_inv), _p(post_inv),
                               M, K, b, bits, clip_ratio, _p(codes), _p(delta), _p(ws), ws.numel(), _stream()))
    return codes, delta


def quantize_weights_rotated(w: torch.Tensor, perm: Optional[torch.Tensor], blocks: torch.Tensor, b: int,
                             bits: int, col_scale: Optional[torch.Tensor] = None,
                             post_scale: Optional[torch.Tensor] = None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Offline fold + RTN for the composite rotation: w fp32 [N, K] -> (codes int8 [N, K], scales fp32 [N])."""
    N, K = w.shape
    assert w.dtype == torch.float32 and w.stride(1) == 1
    codes = torch.empty((N, K), dtype=torch.int8, device=w.device)
    scale = torch.empty((N,), dtype=torch.float32, device=w.device)
    ws = workspace(int(LIB.fq_rotate_quant_workspace_bytes(N, K)), w.device)
    _check(LIB.fq_quantize_weights_rotated(_p(w), w.stride(0), _p(perm), _p(blocks), _p(col_scale),
                                           _p(post_scale), N, K, b, bits, _p(codes), _p(scale), _p(ws),
                                           ws.numel(), _stream()))
    return codes, scale


def transform(x: torch.Tensor, b: int, pre_mult: Optional[torch.Tensor] = None,
              post_mult: Optional[torch.Tensor] = None) -> torch.Tensor:
    """The prologue's transform without quantization: bf16 or fp32 rows [M, K] -> fp32 [M, K]
    (unnormalized blockwise butterfly between the optional multipliers)."""
    M, K = x.shape
    assert x.dtype in (torch.bfloat16, torch.float32) and (M == 0 or x.stride(1) == 1)
    z = torch.empty((M, K), dtype=torch.float32, device=x.device)
    _check(LIB.fq_transform(_p(x), int(x.dtype == torch.float32), x.stride(0) if M else K, _p(pre_mult),
                            _p(post_mult), M, K, b, _p(z), _stream()))
    return z


def gptq_hessian(z: torch.Tensor, G: Optional[torch.Tensor] = None, accumulate: bool = False) -> torch.Tensor:
    """G (+)= z^T z in fp64 for transformed tokens z fp32 [T, K]."""
    T, K = z.shape
    assert z.dtype == torch.float32 and (T == 0 or z.stride(1) == 1)
    if G is None:
        G = torch.empty((K, K), dtype=torch.float64, device=z.device)
    _check(LIB.fq_gptq_hessian(_p(z), z.stride(0) if T else K, T, K, _p(G), int(accumulate), _stream()))
    return G


def gptq_factor(G: torch.Tensor, damp: float = 0.01) -> torch.Tensor:
    """U fp64 [K, K] upper triangular with (G + damp * mean(diag G) I)^-1 = U^T U."""
    K = G.shape[0]
    assert G.dtype == torch.float64 and G.is_contiguous()
    U = torch.empty((K, K), dtype=torch.float64, device=G.device)
    ws = workspace(int(LIB.fq_gptq_factor_workspace_bytes(K)), G.device)
    _check(LIB.fq_gptq_factor(_p(G), K, damp, _p(U), _p(ws), ws.numel(), _stream()))
    return U


def gptq_sweep(w_t: torch.Tensor, U: torch.Tensor, b: int, bits: int) -> Tuple[torch.Tensor, torch.Tensor]:
    """GPTQ column sweep on weight rows w_t fp32 [N, K] transformed with block size b ->
    (codes int8 [N, K], scales fp32 [N])."""
    N, K = w_t.shape
    assert w_t.dtype == torch.float32 and w_t.stride(1) == 1 and U.dtype == torch.float64 and U.is_contiguous()
    codes = torch.empty((N, K), dtype=torch.int8, device=w_t.device)
    scales = torch.empty((N,), dtype=torch.float32, device=w_t.device)
    ws = workspace(int(LIB.fq_gptq_sweep_workspace_bytes(N, K)), w_t.device)
    _check(LIB.fq_gptq_sweep(_p(w_t), w_t.stride(0), _p(U), N, K, b, bits, _p(codes), _p(scales), _p(ws),
                             ws.numel(), _stream()))
    return codes, scales


def gptq_quantize_weights(w: torch.Tensor, calib: torch.Tensor, b: int, bits: int,
                          col_scale: Optional[torch.Tensor] = None, post_scale: Optional[torch.Tensor] = None,
                          smooth_inv: Optional[torch.Tensor] = None, post_inv: Optional[torch.Tensor] = None,
                          damp: float = 0.01) -> Tuple[torch.Tensor, torch.Tensor]:
    """Eq. (7) on the GPU: calibration tokens (bf16 [T, K]) through the runtime transform,
    G = Z Z^T, the damped factor, and the sweep over the folded weight rows (fp32 [N, K]).
    Returns (codes int8 [N, K], scales fp32 [N]) in the layout of quantize_weights."""
    z = transform(calib, b, smooth_inv, post_inv)
    U = gptq_factor(gptq_hessian(z), damp)
    w_t = transform(w, b, col_scale, post_scale)
    return gptq_sweep(w_t, U, b, bits)


def w4a16_workspace_bytes(M: int, N: int, K: int) -> int:
    return int(LIB.fq_gemm_w4a16_workspace_bytes(M, N, K))


def gemm_w4a16(x: torch.Tensor, w_packed: torch.Tensor, w_scale: torch.Tensor, N: int,
               bias: Optional[torch.Tensor] = None, want_acc: bool = False, ws: Optional[torch.Tensor] = None,
               out: Optional[torch.Tensor] = None):
    """Weight-only INT4 projection: bf16 x [M, K] times packed INT4 weights -> bf16 y [M, N]
    (and the fp32 sums if want_acc)."""
    M, K = x.shape
    assert x.dtype == torch.bfloat16 and (M == 0 or x.stride(1) == 1)
    _check_out(out, M, N)
    y = out if out is not None else torch.empty((M, N), dtype=torch.bfloat16, device=x.device)
    acc = torch.empty((M, N), dtype=torch.float32, device=x.device) if want_acc else None
    if ws is None:
        ws = workspace(w4a16_workspace_bytes(M, N, K), x.device)
    _check(LIB.fq_gemm_w4a16(_p(x), x.stride(0) if M else K, _p(w_packed), _p(w_scale), _p(bias), _p(y),
                             y.stride(0) if M else N, _p(acc), M, N, K, _p(ws), ws.numel(), _stream()))
    return (y, acc) if want_acc else y


class QuantLinear:
    """One consumer projection: folded, rounded and packed weights kept resident on the device."""

    def __init__(self, w: torch.Tensor, b: int, bits: int, col_scale: Optional[torch.Tensor] = None,
                 bias: Optional[torch.Tensor] = None, post_scale: Optional[torch.Tensor] = None):
        self.N, self.K = w.shape
        self.b, self.bits = b, bits
        codes, self.w_scale = quantize_weights(w, b, bits, col_scale, post_scale)
        self.w_packed = pack_weights(codes, bits)
        self.bias = bias

    def __call__(self, x: torch.Tensor, clip_ratio: float = 1.0, smooth_inv: Optional[torch.Tensor] = None,
                 ws: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None,
                 post_inv: Optional[torch.Tensor] = None) -> torch.Tensor:
        return linear(x, self.w_packed, self.w_scale, self.N, self.b, self.bits, clip_ratio, smooth_inv,
                      self.bias, ws, out, post_inv)
