"""GPU parity of the one-kernel projection for few tokens (M <= 64, K <= 2048; 1024 for W8A8).

fq_linear runs it whenever fq_linear_workspace_bytes is 0.  Each workgroup recomputes the
prologue of its own rows, so every output must equal, bit for bit, the two-kernel path
through the public entry points (fq_fwht_quant, then fq_gemm_w4a4 / fq_gemm_w8a8) on the
same inputs; a subset is also checked against the oracle (codes and scales through the
prologue entry point, bf16 outputs within 1e-2 of the row absmax, a zero token giving
the bias exactly).  Shapes cover the row block sizes the planner picks (1 to 8 rows, one
wave per row), ragged last row blocks and channel groups, rows of one and two 1024-channel
chunks per lane, every block size from 1 to 256, both widths, the fold multipliers,
r < 1 and strided inputs and outputs.
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


CASES = [
    # (M, K, N, b, bits)
    (50, 1024, 1536, 128, 4), (50, 1024, 1024, 128, 4), (50, 1024, 8192, 128, 4), (64, 1024, 1024, 64, 4),
    (1, 1024, 256, 128, 4), (2, 2048, 2048, 256, 4), (3, 128, 16, 128, 4), (7, 384, 48, 32, 4),
    (8, 1152, 1040, 64, 4), (9, 2048, 4096, 16, 4), (16, 1920, 80, 8, 4), (17, 640, 1536, 1, 4),
    (33, 2048, 256, 2, 4), (63, 256, 4096, 256, 4), (49, 1024, 8192, 4, 4), (64, 2048, 8192, 128, 4),
    (50, 1024, 1536, 128, 8), (64, 1024, 1024, 256, 8), (5, 128, 48, 1, 8), (31, 896, 4096, 128, 8),
    (12, 768, 1040, 32, 8), (1, 1024, 16, 64, 8),
]


def _tensors(M, K, N, b, bits, seed):
    f = fq()
    x = synth.activations(M, K, seed=seed, outlier_frac=0.01, outlier_scale=40.0)
    w = synth.weights(N, K, seed=seed + 1)
    bias = synth.random_scales(N, seed=seed + 2, low=-0.2, high=0.2)
    lin = f.QuantLinear(torch.from_numpy(w).to(DEV), b, bits, bias=torch.from_numpy(bias).to(DEV))
    return x, w, bias, lin


@pytest.mark.parametrize("M,K,N,b,bits", CASES)
def test_one_kernel_equals_two_kernel_path(M, K, N, b, bits):
    flush(f"fused small M={M} K={K} N={N} b={b} bits={bits}")
    f = fq()
    assert f.linear_workspace_bytes(M, N, K, bits) == 0, "shape expected on the one-kernel path"
    x, w, bias, lin = _tensors(M, K, N, b, bits, seed=M * 7 + K + N + b)
    xd = x.to(DEV)
    y = lin(xd)
    codes, delta = f.fwht_quant(xd, b, bits)
    y2 = f.gemm(codes, delta, lin.w_packed, lin.w_scale, N, K, bits, bias=lin.bias)
    torch.cuda.synchronize()
    assert torch.equal(y, y2)


@pytest.mark.parametrize("M,K,N,b,bits", [(50, 1024, 1536, 128, 4), (50, 2048, 1024, 128, 4), (3, 128, 16, 128, 4),
                                          (33, 2048, 256, 2, 4), (50, 1024, 1536, 128, 8), (5, 128, 48, 1, 8)])
def test_one_kernel_matches_oracle(M, K, N, b, bits):
    flush(f"fused small vs oracle M={M} K={K} N={N} b={b} bits={bits}")
    f = fq()
    x, w, bias, lin = _tensors(M, K, N, b, bits, seed=M + 3 * K + N)
    xn = x.clone()
    xn[min(1, M - 1)] = 0  # a zero token gives the bias exactly
    y = lin(xn.to(DEV))
    torch.cuda.synchronize()
    wc, s_w = oracle.quantize_weights(w, b, bits)
    np.testing.assert_array_equal(lin.w_scale.cpu().numpy(), s_w)
    np.testing.assert_array_equal(f.unpack_weights(lin.w_packed, N, K, bits).cpu().numpy(), wc)
    _, _, _, y_ref = oracle.linear(xn, wc, s_w, b, bits, bias=bias)
    assert_bf16_close(y, y_ref)
    z = min(1, M - 1)
    assert torch.equal(y[z].cpu(), torch.from_numpy(bias).to(torch.bfloat16))


@pytest.mark.parametrize("bits", [4, 8])
def test_one_kernel_multipliers_clip_and_strides(bits):
    """Fold-before and fold-after multipliers, r < 1, a strided input and a strided output,
    against the two-kernel path on the same arguments."""
    flush(f"fused small multipliers bits={bits}")
    f = fq()
    M, K, N, b = 21, 1024, 272, 64
    ldx, ldy = K + 64, N + 24
    x_full = synth.activations(M, ldx, seed=31, outlier_frac=0.01, outlier_scale=30.0).to(DEV)
    x = x_full[:, :K]
    w = synth.weights(N, K, seed=32)
    s = torch.from_numpy(synth.channel_vector(K, seed=33, low=0.5, high=2.0)).to(DEV)
    p = torch.from_numpy(synth.channel_vector(K, seed=34, low=0.5, high=2.0)).to(DEV)
    s_inv, p_inv = (1.0 / s).contiguous(), (1.0 / p).contiguous()
    lin = f.QuantLinear(torch.from_numpy(w).to(DEV), b, bits, col_scale=s, post_scale=p)
    assert f.linear_workspace_bytes(M, N, K, bits) == 0
    y_full = torch.zeros((M, ldy), dtype=torch.bfloat16, device=DEV)
    y = y_full[:, :N]
    f.linear(x, lin.w_packed, lin.w_scale, N, b, bits, clip_ratio=0.8, smooth_inv=s_inv, post_inv=p_inv, out=y)
    codes, delta = f.fwht_quant(x, b, bits, clip_ratio=0.8, smooth_inv=s_inv, post_inv=p_inv)
    y2 = f.gemm(codes, delta, lin.w_packed, lin.w_scale, N, K, bits)
    torch.cuda.synchronize()
    assert torch.equal(y, y2)
    assert torch.count_nonzero(y_full[:, N:]) == 0  # nothing written past N
    c_ref, d_ref = oracle.fwht_quant(x.cpu().contiguous(), b, bits, clip_ratio=0.8, chan_mult=s_inv.cpu().numpy(),
                                     post_mult=p_inv.cpu().numpy())
    np.testing.assert_array_equal(codes.cpu().numpy(), canonical_codes(c_ref, bits))
    np.testing.assert_array_equal(delta.cpu().numpy(), d_ref)


def test_one_kernel_graph_replays():
    """The one-kernel projection captured in a HIP graph: every replay, with fresh inputs
    and eager work between replays, equals an eager call bit for bit."""
    flush("fused small graph replays")
    f = fq()
    M, K, N, b, bits = 50, 1024, 1536, 128, 4
    _, _, _, lin = _tensors(M, K, N, b, bits, seed=77)
    xs = [synth.activations(M, K, seed=80 + i, outlier_frac=0.005, outlier_scale=50.0).to(DEV) for i in range(3)]
    x = xs[0].clone()
    y = torch.empty((M, N), dtype=torch.bfloat16, device=DEV)
    g = torch.cuda.CUDAGraph()
    st = torch.cuda.Stream()
    st.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(st):
        lin(x, out=y)
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=st):
            lin(x, out=y)
    torch.cuda.current_stream().wait_stream(st)
    for i in range(6):
        x.copy_(xs[i % 3])
        g.replay()
        torch.cuda.synchronize()
        ref = lin(xs[i % 3])
        torch.cuda.synchronize()
        assert torch.equal(y, ref), f"replay {i}"
