"""Property tests of the projection on the GPU.  The first draws shapes (M 0..300, K a
multiple of 128 and of b, N a multiple of 16), block sizes 1..256, both bit widths and
special rows (zeros, one nonzero, equal magnitudes, a power-of-two copy of another row, a
huge outlier), with a fixed derandomized sequence of examples.  Each example through the
C ABI against the oracle: codes and delta bit-exact, INT32 accumulators bit-exact, bf16
within 1e-2 of the row absmax.  The second draws fused projections with fold presets,
clip ratios and bias (see its docstring)."""
import math

import numpy as np
import pytest
import torch
from hypothesis import HealthCheck, given, settings, strategies as st

import oracle
from paper_2609_24433_amd import synth
from tests.gpu_util import DEV, assert_bf16_close, canonical_codes, flush

pytestmark = pytest.mark.gpu


def fq():
    from paper_2609_24433_amd import fq as _fq
    return _fq


def _tokens(M, K, seed, special):
    x = synth.activations(M, K, seed=seed, outlier_frac=0.01, outlier_scale=30.0).float()
    if M >= 3:
        if special == "zeros":
            x[1] = 0.0
        elif special == "single":
            x[1] = 0.0
            x[1, K // 3] = -5.0
        elif special == "equal":
            x[1] = torch.where(torch.arange(K) % 3 == 0, 1.5, -1.5)
        elif special == "pow2":
            x[1] = x[2] * 2.0 ** -9
        elif special == "outlier":
            x[1, K - 1] = 3.0e4
    return x.to(torch.bfloat16)


@settings(max_examples=30, derandomize=True, deadline=None, suppress_health_check=list(HealthCheck))
@given(st.data())
def test_projection_property(data):
    bits = data.draw(st.sampled_from([4, 8]), label="bits")
    b = 2 ** data.draw(st.integers(0, 8), label="log2 b")
    unit = 128 * b // math.gcd(128, b)
    K = unit * data.draw(st.integers(1, max(1, 2048 // unit)), label="K units")
    M = data.draw(st.integers(0, 300), label="M")
    N = 16 * data.draw(st.integers(1, 24), label="N / 16")
    special = data.draw(st.sampled_from(["none", "zeros", "single", "equal", "pow2", "outlier"]), label="rows")
    seed = data.draw(st.integers(0, 1 << 16), label="seed")
    flush(f"fuzz M={M} K={K} N={N} b={b} bits={bits} rows={special} seed={seed}")
    f = fq()
    x = _tokens(M, K, seed, special)
    w = synth.weights(N, K, seed=seed + 1)
    codes_d, delta_d = f.fwht_quant(x.to(DEV), b, bits)
    wc_d, sw_d = f.quantize_weights(torch.from_numpy(w).to(DEV), b, bits)
    packed = f.pack_weights(wc_d, bits)
    y, acc = f.gemm(codes_d, delta_d, packed, sw_d, N, K, bits, want_acc=True)
    torch.cuda.synchronize()
    codes, delta = oracle.fwht_quant(x, b, bits)
    wc, s_w = oracle.quantize_weights(w, b, bits)
    np.testing.assert_array_equal(delta_d.cpu().numpy(), delta)
    np.testing.assert_array_equal(codes_d.cpu().numpy(), canonical_codes(codes, bits))
    np.testing.assert_array_equal(wc_d.cpu().numpy(), wc)
    np.testing.assert_array_equal(sw_d.cpu().numpy(), s_w)
    acc_ref = oracle.gemm(codes, wc)
    np.testing.assert_array_equal(acc.cpu().numpy().astype(np.int64), acc_ref)
    assert_bf16_close(y, oracle.dequant(acc_ref, delta, s_w))


@settings(max_examples=30, derandomize=True, deadline=None, suppress_health_check=list(HealthCheck))
@given(st.data())
def test_linear_property(data):
    """The fused projection (one kernel per workgroup row block for M <= 64 and K <= 2048
    (1024 for INT8), prologue + GEMM above that) under drawn fold presets (none, fold-before,
    fold-after, both), clip ratios and bias: codes and delta of the prologue bit-exact, the
    fused output identical bit for bit to the two separate entry points on the same codes,
    and within 1e-2 of the row absmax of the oracle's eq. (8) output."""
    bits = data.draw(st.sampled_from([4, 8]), label="bits")
    b = 2 ** data.draw(st.integers(0, 8), label="log2 b")
    unit = 128 * b // math.gcd(128, b)
    K = unit * data.draw(st.integers(1, max(1, 2048 // unit)), label="K units")
    M = data.draw(st.one_of(st.integers(0, 64), st.integers(65, 160)), label="M")
    N = 16 * data.draw(st.integers(1, 24), label="N / 16")
    r = data.draw(st.sampled_from([1.0, 0.9, 0.75]), label="clip ratio")
    fold = data.draw(st.sampled_from(["none", "before", "after", "both"]), label="fold")
    with_bias = data.draw(st.booleans(), label="bias")
    seed = data.draw(st.integers(0, 1 << 16), label="seed")
    flush(f"fuzz linear M={M} K={K} N={N} b={b} bits={bits} r={r} fold={fold} bias={with_bias} seed={seed}")
    f = fq()
    x = _tokens(M, K, seed, "none")
    w = synth.weights(N, K, seed=seed + 1)
    s = synth.channel_vector(K, seed=seed + 2, low=0.5, high=2.0) if fold in ("before", "both") else None
    pv = synth.channel_vector(K, seed=seed + 3, low=0.5, high=2.0) if fold in ("after", "both") else None
    s_inv = None if s is None else (1.0 / s).astype(np.float32)
    p_inv = None if pv is None else (1.0 / pv).astype(np.float32)
    bias = synth.random_scales(N, seed=seed + 4, low=-0.1, high=0.1) if with_bias else None
    dev = lambda a: None if a is None else torch.from_numpy(a).to(DEV)
    lin = f.QuantLinear(torch.from_numpy(w).to(DEV), b, bits, col_scale=dev(s), bias=dev(bias), post_scale=dev(pv))
    xd = x.to(DEV)
    y = lin(xd, clip_ratio=r, smooth_inv=dev(s_inv), post_inv=dev(p_inv))
    codes, delta = f.fwht_quant(xd, b, bits, r, smooth_inv=dev(s_inv), post_inv=dev(p_inv))
    y2 = f.gemm(codes, delta, lin.w_packed, lin.w_scale, N, K, bits, bias=lin.bias)
    torch.cuda.synchronize()
    assert torch.equal(y, y2)
    wc, s_w = oracle.quantize_weights(w, b, bits, s, pv)
    np.testing.assert_array_equal(lin.w_scale.cpu().numpy(), s_w)
    np.testing.assert_array_equal(f.unpack_weights(lin.w_packed, N, K, bits).cpu().numpy(), wc)
    c_ref, d_ref, acc_ref, y_ref = oracle.linear(x, wc, s_w, b, bits, clip_ratio=r, smooth_inv=s_inv, bias=bias,
                                                 post_inv=p_inv)
    np.testing.assert_array_equal(codes.cpu().numpy(), canonical_codes(c_ref, bits))
    np.testing.assert_array_equal(delta.cpu().numpy(), d_ref)
    assert_bf16_close(y, y_ref)
