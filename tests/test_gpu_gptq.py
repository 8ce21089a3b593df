"""GPU parity of GPTQ in the transformed coordinates (eq. (7), Sec. III-F) through the C ABI
against the oracle on the same seeded inputs.

Bar: the transform bit-exact (the prologue's fp32 butterfly and multiplies); the second
moment within the fp64 summation bound (T + 1) 2^-53 sum_t |z_ti z_tj| (any order); the
factor within 1e-9 of its largest entry (fp64 Cholesky and inverse in a different
blocking than LAPACK's, on damped, well-conditioned second moments), the identity exactly
for an empty second moment; the sweep bit-exact given the same factor (its fp64 contract
fixes every operation and order); end to end, scales bit-exact, codes equal but for the
rare decisions a last-bit difference of the factor moves, and the eq. (7) objective
within 1% of the oracle's.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import definitions as D
from paper_2609_24433_amd import synth
from tests.gpu_util import DEV, flush

pytestmark = pytest.mark.gpu


def fq():
    from paper_2609_24433_amd import fq as _fq
    return _fq


def _dev(a):
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


@pytest.mark.parametrize("M,K,b,pre,post,weights", [
    (7, 128, 1, False, False, False), (33, 1024, 16, True, False, False), (50, 2048, 64, True, True, False),
    (3, 4096, 256, False, True, False), (20, 1024, 128, True, True, True), (17, 512, 64, False, False, True),
])
def test_transform_bit_exact(M, K, b, pre, post, weights):
    flush(f"transform M={M} K={K} b={b} pre={pre} post={post} weights={weights}")
    f = fq()
    if weights:
        x = synth.weights(M, K, seed=K + b)
        xd = _dev(x)
    else:
        x = synth.activations(M, K, seed=K + b, outlier_frac=0.01, outlier_scale=30.0)
        xd = x.to(DEV)
    pm = synth.channel_vector(K, seed=3, low=0.25, high=4.0) if pre else None
    qm = synth.channel_vector(K, seed=4, low=0.5, high=2.0) if post else None
    z = f.transform(xd, b, _dev(pm), _dev(qm))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(z.cpu().numpy(), oracle.transform(x, b, pm, qm))


def _calib(T, K, b, seed):
    x = synth.activations(T, K, seed=seed, outlier_frac=0.02, outlier_scale=20.0, dist="student_t3")
    return oracle.transform(x, b)


@pytest.mark.parametrize("T,K", [(300, 256), (1000, 1024), (70, 128)])
def test_hessian_within_summation_bound(T, K):
    flush(f"gptq_hessian T={T} K={K}")
    f = fq()
    z = _calib(T, K, 64, seed=T + K)
    G = f.gptq_hessian(_dev(z))
    torch.cuda.synchronize()
    ref = oracle.gptq_hessian(z)
    za = np.abs(z.astype(np.float64))
    bound = (T + 1) * 2.0 ** -53 * (za.T @ za) + 1e-300
    err = np.abs(G.cpu().numpy() - ref)
    assert np.all(err <= bound), float((err / bound).max())
    # streamed in two batches: the same sums up to rounding
    G2 = f.gptq_hessian(_dev(z[: T // 2]))
    f.gptq_hessian(_dev(z[T // 2:]), G2, accumulate=True)
    torch.cuda.synchronize()
    assert np.all(np.abs(G2.cpu().numpy() - ref) <= 2 * bound)
    # no tokens and no accumulation: zero
    G0 = f.gptq_hessian(_dev(z[:0]), G2)
    torch.cuda.synchronize()
    assert not G0.cpu().numpy().any()


@pytest.mark.parametrize("K", [128, 256, 384, 640, 1024])
def test_factor_matches_oracle(K):
    flush(f"gptq_factor K={K}")
    f = fq()
    z = _calib(3 * K, K, 64, seed=K)
    G = oracle.gptq_hessian(z)
    U = f.gptq_factor(_dev(G), 0.01)
    torch.cuda.synchronize()
    Ug = U.cpu().numpy()
    Ur = oracle.gptq_factor(G, 0.01)
    assert np.all(np.tril(Ug, -1) == 0) and np.all(np.diag(Ug) > 0)
    assert np.abs(Ug - Ur).max() <= 1e-9 * np.abs(Ur).max()
    H = oracle.gptq_damped(G, 0.01)
    np.testing.assert_allclose(Ug.T @ Ug @ H, np.eye(K), atol=1e-8)
    # an empty second moment gives the identity exactly
    Ui = f.gptq_factor(torch.zeros((K, K), dtype=torch.float64, device=DEV), 0.01)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(Ui.cpu().numpy(), np.eye(K))


@pytest.mark.parametrize("N,K,bits", [(48, 128, 4), (17, 384, 4), (40, 1024, 4), (33, 512, 8)])
def test_sweep_bit_exact_given_the_factor(N, K, bits):
    flush(f"gptq_sweep N={N} K={K} bits={bits}")
    f = fq()
    b = 64
    w = synth.weights(N, K, seed=N + K)
    w[min(5, N - 1)] = 0.0  # a zero row
    w_t = oracle.transform(w, b)
    U = oracle.gptq_factor(oracle.gptq_hessian(_calib(2 * K, K, b, seed=K + 1)), 0.01)
    cb = float(oracle.inv_sqrt_b(b))
    codes, scales = f.gptq_sweep(_dev(w_t), _dev(U), b, bits)
    torch.cuda.synchronize()
    c_ref, s_ref = oracle.gptq_sweep(w_t, U, bits, 128, cb)
    np.testing.assert_array_equal(scales.cpu().numpy(), s_ref)
    np.testing.assert_array_equal(codes.cpu().numpy(), c_ref)
    rtn, _, _ = D.quantize_eq5(w_t, bits)
    assert (c_ref != rtn).mean() > 0.02  # the error feedback is exercised


@pytest.mark.parametrize("N,K,b", [(64, 256, 64), (96, 1024, 128)])
def test_gptq_end_to_end(N, K, b):
    flush(f"gptq end to end N={N} K={K} b={b}")
    f = fq()
    calib = synth.activations(2 * K, K, seed=K + 7, outlier_frac=0.02, outlier_scale=20.0, dist="student_t3")
    w = synth.weights(N, K, seed=N + 11)
    s = synth.channel_vector(K, seed=12, low=0.5, high=2.0)
    s_inv = (1.0 / s).astype(np.float32)
    codes, scales = f.gptq_quantize_weights(_dev(w), calib.to(DEV), b, 4, col_scale=_dev(s), smooth_inv=_dev(s_inv))
    torch.cuda.synchronize()
    c_ref, s_ref = oracle.gptq_quantize_weights(w, calib, b, 4, col_scale=s, smooth_inv=s_inv)
    np.testing.assert_array_equal(scales.cpu().numpy(), s_ref)
    cg = codes.cpu().numpy()
    assert (cg != c_ref).mean() < 0.01
    z = oracle.transform(calib, b, s_inv).astype(np.float64)
    w_t = oracle.transform(w, b, s).astype(np.float64)
    step = (s_ref / oracle.inv_sqrt_b(b)).astype(np.float64)[:, None]
    e_gpu = D.gptq_objective(w_t, cg * step, z)
    e_ref = D.gptq_objective(w_t, c_ref * step, z)
    assert abs(e_gpu - e_ref) <= 0.01 * e_ref
    rtn, _ = oracle.quantize_weights(w, b, 4, s)
    assert e_gpu < D.gptq_objective(w_t, rtn * step, z)
