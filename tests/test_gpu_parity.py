"""GPU parity: the HIP path through the C ABI against the CPU oracle on the same seeded inputs.

Bar: activation/weight codes and scales bit-exact; INT32 accumulators bit-exact given
identical codes; bf16 outputs within 1e-2 of each row's absmax.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_24433_amd import synth
from tests.gpu_util import DEV, assert_bf16_close, canonical_codes, flush

pytestmark = pytest.mark.gpu


def fq():
    from paper_2609_24433_amd import fq as _fq
    return _fq


# ------------------------------------------------------------------ prologue (eq. (5))

QUANT_CASES = [
    # (M, K, b, bits, r)
    (37, 1024, 1, 4, 1.0), (37, 1024, 2, 8, 1.0), (37, 1024, 4, 4, 1.0), (37, 1024, 8, 8, 1.0),
    (37, 1024, 16, 4, 1.0), (37, 1024, 32, 4, 1.0), (37, 1024, 64, 4, 1.0), (37, 1024, 128, 8, 1.0),
    (37, 1024, 256, 4, 1.0), (70, 384, 128, 4, 0.85), (3, 4096, 128, 4, 1.0), (5, 16384, 256, 8, 1.0),
    (5, 16384, 32, 4, 1.0), (9, 2048, 64, 8, 0.7), (1, 128, 128, 4, 1.0), (300, 1152, 128, 4, 1.0),
    (2, 32768, 128, 4, 1.0), (2, 32768, 8, 8, 1.0), (4, 8192, 256, 4, 1.0), (130, 640, 128, 8, 1.0),
    # rows of 2 chunks per thread with the last chunks of the row past K
    (3, 12288, 128, 4, 1.0), (17, 6144, 256, 4, 0.9), (6, 24576, 64, 8, 0.8), (5, 24576, 128, 4, 1.0),
]


@pytest.mark.parametrize("M,K,b,bits,r", QUANT_CASES)
def test_fwht_quant_bit_exact(M, K, b, bits, r):
    flush(f"fwht_quant M={M} K={K} b={b} bits={bits} r={r}")
    x = synth.activations(M, K, seed=M * 7 + K + b, outlier_frac=0.005, outlier_scale=50.0)
    codes, delta = fq().fwht_quant(x.to(DEV), b, bits, r)
    torch.cuda.synchronize()
    c_ref, d_ref = oracle.fwht_quant(x, b, bits, r)
    np.testing.assert_array_equal(codes.cpu().numpy(), canonical_codes(c_ref, bits))
    np.testing.assert_array_equal(delta.cpu().numpy(), d_ref)


@pytest.mark.parametrize("bits", [4, 8])
def test_fwht_quant_special_rows_and_stride(bits):
    flush(f"fwht_quant special rows bits={bits}")
    M, K, b = 12, 1024, 64
    full = synth.activations(M, K + 64, seed=3, dist="student_t3")  # ldx = K + 64
    full[2].zero_()                                    # zero token
    full[4] = 0
    full[4, 100] = 3.0                                 # single nonzero
    full[5] = 1.0                                      # all equal
    full[6] = (full[6].float() * 2.0 ** -100).bfloat16()  # tiny magnitudes
    full[7] = (full[7].float() * 2.0 ** 100).bfloat16()   # huge magnitudes
    full[8, :8] = torch.tensor([14, 5, 3, 1, -5, -3, -1, 9], dtype=torch.bfloat16)
    full[8, 8:] = 0                                     # exact ties at b = 1 ... (b = 64 mixes them)
    xd = full.to(DEV)[:, :K]
    assert xd.stride(0) == K + 64
    codes, delta = fq().fwht_quant(xd, b, bits)
    torch.cuda.synchronize()
    c_ref, d_ref = oracle.fwht_quant(full[:, :K].contiguous(), b, bits)
    np.testing.assert_array_equal(codes.cpu().numpy(), canonical_codes(c_ref, bits))
    np.testing.assert_array_equal(delta.cpu().numpy(), d_ref)
    assert d_ref[2] == 0


def test_fwht_quant_exact_ties_b1():
    flush("fwht_quant ties")
    x = torch.zeros(4, 128, dtype=torch.bfloat16)
    x[:, :8] = torch.tensor([14, 5, 3, 1, -5, -3, -1, 9], dtype=torch.bfloat16)
    codes, delta = fq().fwht_quant(x.to(DEV), 1, 4)
    torch.cuda.synchronize()
    c_ref, d_ref = oracle.fwht_quant(x, 1, 4)
    assert c_ref[0, :8].tolist() == [7, 2, 2, 0, -2, -2, 0, 4]
    np.testing.assert_array_equal(codes.cpu().numpy(), canonical_codes(c_ref, 4))


@pytest.mark.parametrize("b,bits", [(64, 4), (128, 8), (16, 4)])
def test_fwht_quant_fold_before_multiplier(b, bits):
    flush(f"fwht_quant smooth b={b} bits={bits}")
    M, K = 33, 2048
    x = synth.activations(M, K, seed=77, outlier_frac=0.01, outlier_scale=30.0)
    s_inv = synth.channel_vector(K, seed=78, low=0.2, high=3.0)
    codes, delta = fq().fwht_quant(x.to(DEV), b, bits, 1.0, torch.from_numpy(s_inv).to(DEV))
    torch.cuda.synchronize()
    c_ref, d_ref = oracle.fwht_quant(x, b, bits, 1.0, s_inv)
    np.testing.assert_array_equal(codes.cpu().numpy(), canonical_codes(c_ref, bits))
    np.testing.assert_array_equal(delta.cpu().numpy(), d_ref)


@pytest.mark.parametrize("b,bits,M,K", [(64, 4, 33, 2048), (128, 8, 33, 2048), (256, 4, 5, 16384),
                                         (128, 4, 50, 4096), (16, 8, 70, 384)])
def test_fwht_quant_fold_after_multiplier(b, bits, M, K):
    # Sec. III-C fold-after: P^-1 after the rotation, bit-exact (alone and with S^-1 before it)
    flush(f"fwht_quant post b={b} bits={bits} M={M} K={K}")
    x = synth.activations(M, K, seed=79, outlier_frac=0.01, outlier_scale=30.0)
    p_inv = synth.channel_vector(K, seed=80, low=0.2, high=3.0)
    s_inv = synth.channel_vector(K, seed=81, low=0.5, high=2.0)
    pd, sd = torch.from_numpy(p_inv).to(DEV), torch.from_numpy(s_inv).to(DEV)
    codes, delta = fq().fwht_quant(x.to(DEV), b, bits, 1.0, post_inv=pd)
    codes2, delta2 = fq().fwht_quant(x.to(DEV), b, bits, 0.9, sd, post_inv=pd)
    torch.cuda.synchronize()
    c_ref, d_ref = oracle.fwht_quant(x, b, bits, 1.0, None, p_inv)
    np.testing.assert_array_equal(codes.cpu().numpy(), canonical_codes(c_ref, bits))
    np.testing.assert_array_equal(delta.cpu().numpy(), d_ref)
    c_ref2, d_ref2 = oracle.fwht_quant(x, b, bits, 0.9, s_inv, p_inv)
    np.testing.assert_array_equal(codes2.cpu().numpy(), canonical_codes(c_ref2, bits))
    np.testing.assert_array_equal(delta2.cpu().numpy(), d_ref2)


# ------------------------------------------------------------------ offline weights

@pytest.mark.parametrize("N,K,b,bits,scaled", [(64, 1024, 64, 4, False), (48, 2048, 128, 8, True),
                                                (256, 4096, 128, 4, True), (32, 16384, 256, 4, False),
                                                (16, 128, 1, 8, False)])
def test_quantize_weights_bit_exact(N, K, b, bits, scaled):
    flush(f"quantize_weights N={N} K={K} b={b} bits={bits}")
    w = synth.weights(N, K, seed=N + K)
    w[3] = 0.0
    cs = synth.channel_vector(K, seed=5, low=0.5, high=1.5) if scaled else None
    codes, scale = fq().quantize_weights(torch.from_numpy(w).to(DEV), b, bits,
                                         None if cs is None else torch.from_numpy(cs).to(DEV))
    torch.cuda.synchronize()
    c_ref, s_ref = oracle.quantize_weights(w, b, bits, cs)
    np.testing.assert_array_equal(codes.cpu().numpy(), c_ref)
    np.testing.assert_array_equal(scale.cpu().numpy(), s_ref)


@pytest.mark.parametrize("N,K,b,bits", [(64, 1024, 64, 4), (48, 2048, 128, 8), (32, 16384, 256, 4)])
def test_quantize_weights_fold_after_bit_exact(N, K, b, bits):
    flush(f"quantize_weights post N={N} K={K} b={b} bits={bits}")
    w = synth.weights(N, K, seed=N + K + 1)
    w[2] = 0.0
    pv = synth.channel_vector(K, seed=6, low=0.5, high=1.5)
    codes, scale = fq().quantize_weights(torch.from_numpy(w).to(DEV), b, bits, None, torch.from_numpy(pv).to(DEV))
    torch.cuda.synchronize()
    c_ref, s_ref = oracle.quantize_weights(w, b, bits, None, pv)
    np.testing.assert_array_equal(codes.cpu().numpy(), c_ref)
    np.testing.assert_array_equal(scale.cpu().numpy(), s_ref)


@pytest.mark.parametrize("bits", [4, 8])
@pytest.mark.parametrize("N,K", [(16, 128), (48, 1024), (272, 2176)])
def test_pack_unpack_round_trip(bits, N, K):
    flush(f"pack N={N} K={K} bits={bits}")
    c = torch.from_numpy(synth.random_codes(N, K, bits, seed=N * K)).to(DEV)
    packed = fq().pack_weights(c, bits)
    assert packed.numel() == N * K * bits // 8
    back = fq().unpack_weights(packed, N, K, bits)
    torch.cuda.synchronize()
    assert torch.equal(back, c)


# ------------------------------------------------------------------ GEMM + epilogue (eq. (8))

GEMM_CASES = [
    # (M, N, K) -- streaming kernel for M <= 64, tiled kernel above (64 x 128 tiles on
    # these small grids; 128 x 128 in the full-size tests), split-K where the plan asks
    (1, 16, 128), (16, 48, 1024), (17, 256, 1024), (50, 2048, 4096), (64, 272, 2048),
    (65, 256, 1024), (130, 400, 1024), (300, 272, 2048), (50, 1024, 16384), (200, 128, 8192),
    # long K: 16-row blocks over 128-step slices (one or two K slices), one K range per
    # wave, 16 output channels per workgroup up to 32 rows, 32 from 33 rows on
    (33, 64, 32768), (64, 96, 16384), (1, 2048, 16384), (16, 1040, 16384), (20, 2048, 32768),
    # a second K slice with one step, and one whose later waves hold no step at all
    (40, 272, 16512), (1, 2048, 18432),
    # 4096 <= K < 16384 (four wave groups sharing one slice; K split in two)
    (50, 1024, 4096), (33, 512, 8192), (1, 4096, 4224), (17, 1024, 12288),
    # k-group GEMM (INT4; 128 x 64 tiles, K over the workgroup's four waves): ragged rows
    # and a ragged last column tile; 65 k steps, so one wave takes a step more than the rest
    (700, 2000, 8192), (816, 2048, 8320),
]


@pytest.mark.parametrize("bits", [4, 8])
@pytest.mark.parametrize("M,N,K", GEMM_CASES)
def test_gemm_acc_bit_exact_and_output(bits, M, N, K):
    flush(f"gemm w{bits}a{bits} M={M} N={N} K={K}")
    qa = synth.random_codes(M, K, bits, seed=M + N)
    qw = synth.random_codes(N, K, bits, seed=K + 1)
    delta = synth.random_scales(M, seed=M)
    s_w = synth.random_scales(N, seed=N)
    bias = synth.random_scales(N, seed=N + 1, low=-0.5, high=0.5)
    qa[M // 2] = 0
    delta[M // 2] = 0.0
    f = fq()
    a_dev = torch.from_numpy(canonical_codes(qa, bits)).to(DEV)
    w_pk = f.pack_weights(torch.from_numpy(qw).to(DEV), bits)
    y, acc = f.gemm(a_dev, torch.from_numpy(delta).to(DEV), w_pk, torch.from_numpy(s_w).to(DEV), N, K,
                    bits, bias=torch.from_numpy(bias).to(DEV), want_acc=True)
    torch.cuda.synchronize()
    acc_ref = oracle.gemm(qa, qw)
    np.testing.assert_array_equal(acc.cpu().numpy().astype(np.int64), acc_ref)
    y_ref = oracle.dequant(acc_ref, delta, s_w, bias)
    assert_bf16_close(y, y_ref)
    # the zero token gives y = bias exactly
    assert torch.equal(y[M // 2].cpu(), torch.from_numpy(bias).to(torch.bfloat16))


def test_gemm_workspace_reuse_and_no_bias():
    flush("gemm workspace reuse")
    f = fq()
    M, N, K, bits = 40, 512, 8192, 4
    ws = f.workspace(max(f.gemm_workspace_bytes(M, N, K, bits), f.gemm_workspace_bytes(20, N, K, bits)), DEV)
    qw = synth.random_codes(N, K, bits, seed=9)
    w_pk = f.pack_weights(torch.from_numpy(qw).to(DEV), bits)
    s_w = synth.random_scales(N, seed=10)
    for rep, m in enumerate((M, 20, M)):
        qa = synth.random_codes(m, K, bits, seed=100 + rep)
        delta = synth.random_scales(m, seed=200 + rep)
        y, acc = f.gemm(torch.from_numpy(canonical_codes(qa, bits)).to(DEV), torch.from_numpy(delta).to(DEV),
                        w_pk, torch.from_numpy(s_w).to(DEV), N, K, bits, want_acc=True, ws=ws)
        torch.cuda.synchronize()
        acc_ref = oracle.gemm(qa, qw)
        np.testing.assert_array_equal(acc.cpu().numpy().astype(np.int64), acc_ref)
        assert_bf16_close(y, oracle.dequant(acc_ref, delta, s_w))


# ------------------------------------------------------------------ the fused projection

LINEAR_CASES = [
    # (M, K, N, b, bits)
    (64, 1024, 1024, 64, 4),     # single W4A4 linear (configuration 1)
    (50, 1024, 256, 128, 4), (50, 4096, 1024, 128, 4), (50, 1024, 4096, 128, 4),
    (16, 16384, 2048, 32, 8), (1, 16384, 2048, 256, 4), (77, 2048, 256, 128, 8),
    (130, 2048, 2048, 128, 4), (33, 512, 48, 16, 4), (0, 1024, 256, 64, 4),
    (200, 16384, 256, 128, 4),   # tiled GEMM with K split in 4 (split-K epilogue)
    (700, 8192, 2000, 128, 4),   # k-group GEMM fed k-step-major codes by the prologue
]


@pytest.mark.parametrize("M,K,N,b,bits", LINEAR_CASES)
def test_linear_matches_oracle(M, K, N, b, bits):
    flush(f"linear M={M} K={K} N={N} b={b} bits={bits}")
    f = fq()
    x = synth.activations(M, K, seed=M + K + N, outlier_frac=0.005, outlier_scale=50.0)
    w = synth.weights(N, K, seed=N + 3)
    bias = synth.random_scales(N, seed=4, low=-0.1, high=0.1)
    lin = f.QuantLinear(torch.from_numpy(w).to(DEV), b, bits, bias=torch.from_numpy(bias).to(DEV))
    xd = x.to(DEV)
    y = lin(xd)
    # same codes through the separate entry points: the fused output must be identical bit for bit
    codes, delta = f.fwht_quant(xd, b, bits)
    y2 = f.gemm(codes, delta, lin.w_packed, lin.w_scale, N, K, bits, bias=lin.bias)
    torch.cuda.synchronize()
    assert torch.equal(y, y2)
    wc, s_w = oracle.quantize_weights(w, b, bits)
    np.testing.assert_array_equal(lin.w_scale.cpu().numpy(), s_w)
    c_ref, d_ref, acc_ref, y_ref = oracle.linear(x, wc, s_w, b, bits, bias=bias)
    np.testing.assert_array_equal(codes.cpu().numpy(), canonical_codes(c_ref, bits))
    np.testing.assert_array_equal(delta.cpu().numpy(), d_ref)
    assert_bf16_close(y, y_ref)


def test_linear_clip_and_smoothing():
    flush("linear clip + smoothing")
    f = fq()
    M, K, N, b, bits = 24, 2048, 512, 64, 4
    x = synth.activations(M, K, seed=8, outlier_frac=0.01, outlier_scale=30.0)
    w = synth.weights(N, K, seed=9)
    s = synth.channel_vector(K, seed=10, low=0.5, high=2.0)
    s_inv = (1.0 / s).astype(np.float32)
    lin = f.QuantLinear(torch.from_numpy(w).to(DEV), b, bits, col_scale=torch.from_numpy(s).to(DEV))
    y = lin(x.to(DEV), clip_ratio=0.9, smooth_inv=torch.from_numpy(s_inv).to(DEV))
    torch.cuda.synchronize()
    wc, s_w = oracle.quantize_weights(w, b, bits, s)
    _, _, _, y_ref = oracle.linear(x, wc, s_w, b, bits, clip_ratio=0.9, smooth_inv=s_inv)
    assert_bf16_close(y, y_ref)


@pytest.mark.parametrize("M,K,N,bits", [(50, 1024, 1536, 4), (24, 2048, 512, 8), (200, 2048, 384, 4)])
def test_linear_fold_after(M, K, N, bits):
    """Fold-after preset end to end: weights W R^T P rounded on the GPU, tokens P^-1 R x."""
    flush(f"linear fold-after M={M} K={K} N={N} bits={bits}")
    f = fq()
    b = 128
    x = synth.activations(M, K, seed=12, outlier_frac=0.01, outlier_scale=30.0)
    w = synth.weights(N, K, seed=13)
    pv = synth.channel_vector(K, seed=14, low=0.5, high=2.0)
    p_inv = (1.0 / pv).astype(np.float32)
    lin = f.QuantLinear(torch.from_numpy(w).to(DEV), b, bits, post_scale=torch.from_numpy(pv).to(DEV))
    ws = f.workspace(f.linear_workspace_bytes(M, N, K, bits), DEV)
    y = lin(x.to(DEV), ws=ws, post_inv=torch.from_numpy(p_inv).to(DEV))
    torch.cuda.synchronize()
    wc, s_w = oracle.quantize_weights(w, b, bits, None, pv)
    np.testing.assert_array_equal(lin.w_scale.cpu().numpy(), s_w)
    np.testing.assert_array_equal(f.unpack_weights(lin.w_packed, N, K, bits).cpu().numpy(), wc)
    _, _, _, y_ref = oracle.linear(x, wc, s_w, b, bits, post_inv=p_inv)
    assert_bf16_close(y, y_ref)
