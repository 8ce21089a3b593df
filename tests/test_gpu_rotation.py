"""GPU parity of the stored composite rotation (Sec. III-C: channel permutation followed by
per-block matrices, in place of the block Hadamard) through the C ABI against the oracle
on the same seeded inputs.

Bar: codes and scales bit-exact.  Both sides run the same fp32 fused multiply-add chain in
ascending j per output channel, so every rounding is shared; the integer GEMM over the
rotated codes is then bit-exact too, and bf16 outputs sit within 1e-2 of each row's absmax.
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


def _dev(a):
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


CASES = [
    # (M, K, b, bits, perm, pre, post, ldx_pad): every block size, ragged M against the
    # transform's rows per workgroup, strided rows, the largest K
    (1, 128, 1, 4, True, False, False, 0), (17, 256, 2, 8, True, True, False, 8), (33, 1024, 8, 4, False, False, True, 0),
    (16, 1024, 16, 4, True, False, False, 0), (50, 2048, 32, 8, True, True, True, 16), (50, 1024, 64, 4, True, False, False, 0),
    (130, 2048, 128, 4, True, True, True, 0), (3, 2048, 128, 8, False, False, False, 8), (2, 32768, 64, 4, True, True, False, 0),
    (257, 512, 4, 4, True, False, False, 0),
    # the language prologue's shape (M = 816, K 2048) and larger grids at b = 16 and 32
    (816, 2048, 128, 4, True, True, True, 0), (300, 8192, 32, 8, True, False, False, 0),
    (100, 4096, 16, 4, False, True, False, 8),
]


@pytest.mark.parametrize("M,K,b,bits,use_perm,pre,post,pad", CASES)
def test_rotate_quant_bit_exact(M, K, b, bits, use_perm, pre, post, pad):
    flush(f"rotate_quant M={M} K={K} b={b} bits={bits} perm={use_perm} pre={pre} post={post} pad={pad}")
    f = fq()
    full = synth.activations(M, K + pad, seed=M * 7 + K + b, outlier_frac=0.01, outlier_scale=30.0)
    if M > 2:
        full[1].zero_()  # a zero token: codes 0, delta 0
    x = full[:, :K].contiguous()
    perm = synth.permutation(K, seed=K + b) if use_perm else None
    blocks = synth.orthogonal_blocks(K // b, b, seed=b + 5)
    s_inv = synth.channel_vector(K, seed=K + 1, low=0.25, high=4.0) if pre else None
    p_inv = synth.channel_vector(K, seed=K + 2, low=0.5, high=2.0) if post else None
    codes, delta = f.rotate_quant(full.to(DEV)[:, :K], _dev(perm), _dev(blocks), b, bits, 1.0, _dev(s_inv), _dev(p_inv))
    torch.cuda.synchronize()
    c_ref, d_ref = oracle.rotate_quant(x, perm, blocks, b, bits, 1.0, s_inv, p_inv)
    np.testing.assert_array_equal(delta.cpu().numpy(), d_ref)
    np.testing.assert_array_equal(codes.cpu().numpy(), canonical_codes(c_ref, bits))
    if M > 2:
        assert d_ref[1] == 0.0 and not c_ref[1].any()


@pytest.mark.parametrize("bits,clip", [(4, 0.9), (8, 0.75)])
def test_rotate_quant_clip_ratio(bits, clip):
    flush(f"rotate_quant clip={clip} bits={bits}")
    f = fq()
    M, K, b = 20, 1024, 64
    x = synth.activations(M, K, seed=41, dist="student_t3")
    perm = synth.permutation(K, seed=42)
    blocks = synth.orthogonal_blocks(K // b, b, seed=43)
    codes, delta = f.rotate_quant(x.to(DEV), _dev(perm), _dev(blocks), b, bits, clip)
    torch.cuda.synchronize()
    c_ref, d_ref = oracle.rotate_quant(x, perm, blocks, b, bits, clip)
    np.testing.assert_array_equal(delta.cpu().numpy(), d_ref)
    np.testing.assert_array_equal(codes.cpu().numpy(), canonical_codes(c_ref, bits))


@pytest.mark.parametrize("N,K,b,bits,scales", [(48, 1024, 64, 4, True), (32, 2048, 128, 8, False), (16, 256, 8, 4, True)])
def test_quantize_weights_rotated_bit_exact(N, K, b, bits, scales):
    flush(f"quantize_weights_rotated N={N} K={K} b={b} bits={bits} scales={scales}")
    f = fq()
    w = synth.weights(N, K, seed=N + K)
    perm = synth.permutation(K, seed=K + 9)
    blocks = synth.orthogonal_blocks(K // b, b, seed=b + 11)
    cs = synth.channel_vector(K, seed=3, low=0.25, high=4.0) if scales else None
    ps = synth.channel_vector(K, seed=4, low=0.5, high=2.0) if scales else None
    codes, s_w = f.quantize_weights_rotated(_dev(w), _dev(perm), _dev(blocks), b, bits, _dev(cs), _dev(ps))
    torch.cuda.synchronize()
    c_ref, s_ref = oracle.quantize_weights_rotated(w, perm, blocks, b, bits, cs, ps)
    np.testing.assert_array_equal(s_w.cpu().numpy(), s_ref)
    np.testing.assert_array_equal(codes.cpu().numpy(), c_ref)


@pytest.mark.parametrize("M,K,N,bits", [(50, 2048, 256, 4), (17, 1024, 128, 8)])
def test_rotated_projection_end_to_end(M, K, N, bits):
    """Rotated weights and tokens through the integer GEMM: the rotation cancels in the product
    (Sec. III-C), the accumulators match the oracle's exactly."""
    flush(f"rotated projection M={M} K={K} N={N} bits={bits}")
    f = fq()
    b = 64
    x = synth.activations(M, K, seed=61, outlier_frac=0.01, outlier_scale=30.0)
    w = synth.weights(N, K, seed=62)
    perm = synth.permutation(K, seed=63)
    blocks = synth.orthogonal_blocks(K // b, b, seed=64)
    bias = synth.channel_vector(N, seed=65, low=-0.5, high=0.5)
    wc, s_w = f.quantize_weights_rotated(_dev(w), _dev(perm), _dev(blocks), b, bits)
    packed = f.pack_weights(wc, bits)
    codes, delta = f.rotate_quant(x.to(DEV), _dev(perm), _dev(blocks), b, bits)
    y, acc = f.gemm(codes, delta, packed, s_w, N, K, bits, bias=_dev(bias), want_acc=True)
    torch.cuda.synchronize()
    wc_ref, sw_ref = oracle.quantize_weights_rotated(w, perm, blocks, b, bits)
    ca_ref, d_ref = oracle.rotate_quant(x, perm, blocks, b, bits)
    acc_ref = oracle.gemm(ca_ref, wc_ref)
    np.testing.assert_array_equal(acc.cpu().numpy().astype(np.int64), acc_ref)
    assert_bf16_close(y, oracle.dequant(acc_ref, d_ref, sw_ref, bias))
