"""GPU parity of the weight-only INT4 projection (W4A16, Sec. III-A adaptive layer-norm
modulation path) through the C ABI against the oracle on the same seeded inputs.

Bar: the weights' codes and scales bit-exact (per-output-channel rounding at b = 1); the
fp32 sums within the rigorous floating-point summation bound (K - 1) 2^-24 sum |x q| of
the exact (float64) sums, whatever order the matrix cores add in; bf16 outputs within
1e-2 of each row's absmax; a zero token gives the bias exactly.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_24433_amd import synth
from tests.gpu_util import DEV, assert_bf16_close, flush

pytestmark = pytest.mark.gpu


def fq():
    from paper_2609_24433_amd import fq as _fq
    return _fq


CASES = [
    # (M, K, N, ldx_pad, bias): one K slice, split K, row blocks, strided input, tiny and ragged M
    (1, 1024, 6144, 0, False), (3, 1024, 256, 8, True), (16, 2048, 512, 0, False), (17, 2048, 256, 0, True),
    (50, 4096, 1024, 0, False), (1, 16384, 2048, 0, True), (16, 16384, 512, 16, False), (64, 128, 16, 0, False),
    (70, 1024, 256, 0, True), (130, 2048, 128, 8, False), (2, 32768, 64, 0, False),
    # a single token past 16 k steps stages only its own row: ragged wave groups, one
    # slice of up to 64 k steps (K = 8064: 63), split K beyond (K = 12160: 3 slices, ragged)
    (1, 2176, 128, 0, True), (1, 4096, 256, 8, False), (1, 8064, 48, 8, True), (1, 12160, 48, 8, True),
    (1, 32768, 64, 0, False),
]


@pytest.mark.parametrize("M,K,N,pad,with_bias", CASES)
def test_w4a16_parity(M, K, N, pad, with_bias):
    flush(f"w4a16 M={M} K={K} N={N} pad={pad} bias={with_bias}")
    f = fq()
    full = synth.activations(M, K + pad, seed=M + K + N, outlier_frac=0.01, outlier_scale=30.0)
    x = full[:, :K]
    if M > 2:
        full[1].zero_()  # a zero token
    w = synth.weights(N, K, seed=K + N)
    bias = synth.channel_vector(N, seed=N + 3, low=-0.5, high=0.5) if with_bias else None
    codes, s_w = f.quantize_weights(torch.from_numpy(w).to(DEV), 1, 4)
    packed = f.pack_weights(codes, 4)
    xd = full.to(DEV)[:, :K]
    bd = None if bias is None else torch.from_numpy(bias).to(DEV)
    y, acc = f.gemm_w4a16(xd, packed, s_w, N, bias=bd, want_acc=True)
    torch.cuda.synchronize()

    q_ref, s_ref = oracle.quantize_weights(w, 1, 4)
    np.testing.assert_array_equal(codes.cpu().numpy(), q_ref)
    np.testing.assert_array_equal(s_w.cpu().numpy(), s_ref)
    acc_ref, y_ref = oracle.w4a16(x.contiguous(), q_ref, s_ref, bias)

    absx = np.abs(x.float().numpy().astype(np.float64))
    bound = (K - 1) * 2.0 ** -24 * (absx @ np.abs(q_ref.astype(np.float64)).T) + 1e-30
    err = np.abs(acc.cpu().numpy().astype(np.float64) - acc_ref)
    assert np.all(err <= bound), float((err / bound).max())
    assert_bf16_close(y, y_ref)
    if M > 2:
        want = torch.zeros(N, dtype=torch.float32) if bias is None else torch.from_numpy(bias)
        assert torch.equal(y[1].cpu(), want.to(torch.bfloat16))


def test_w4a16_split_workspace_reuse():
    """Split K: the workspace (fp32 partial sums) needs no initialization (here: random
    bytes) and one workspace serves calls of different shapes one after the other."""
    flush("w4a16 split-K workspace reuse")
    f = fq()
    shapes = [(1, 16384, 512), (16, 16384, 256), (1, 32768, 128), (3, 8192, 512), (1, 16384, 512)]
    need = max(f.w4a16_workspace_bytes(M, N, K) for M, K, N in shapes)
    assert need > 0
    ws = torch.randint(0, 256, (need,), dtype=torch.uint8, device=DEV)
    for i, (M, K, N) in enumerate(shapes):
        x = synth.activations(M, K, seed=40 + i, outlier_frac=0.01, outlier_scale=30.0)
        w = synth.weights(N, K, seed=50 + i)
        codes, s_w = f.quantize_weights(torch.from_numpy(w).to(DEV), 1, 4)
        packed = f.pack_weights(codes, 4)
        y, acc = f.gemm_w4a16(x.to(DEV), packed, s_w, N, ws=ws, want_acc=True)
        torch.cuda.synchronize()
        q_ref, s_ref = oracle.quantize_weights(w, 1, 4)
        acc_ref, y_ref = oracle.w4a16(x.contiguous(), q_ref, s_ref, None)
        absx = np.abs(x.float().numpy().astype(np.float64))
        bound = (K - 1) * 2.0 ** -24 * (absx @ np.abs(q_ref.astype(np.float64)).T) + 1e-30
        err = np.abs(acc.cpu().numpy().astype(np.float64) - acc_ref)
        assert np.all(err <= bound), (M, K, N, float((err / bound).max()))
        assert_bf16_close(y, y_ref)
