"""fq_linear_static (the fused projection for callers that cannot allocate: its scratch is
a device array inside the library) against fq_linear with a caller workspace, through the
C ABI: bit for bit, on consecutive calls that reuse the scratch, the later ones smaller,
on the two-kernel path (prologue codes and split-K partials in the scratch) and the
one-kernel path (no scratch), both widths; and the rejection of a shape that needs more
scratch than the library holds."""
import numpy as np
import pytest
import torch

from paper_2609_24433_amd import synth
from tests.gpu_util import DEV, flush

pytestmark = pytest.mark.gpu


def fq():
    from paper_2609_24433_amd import fq as _fq
    return _fq


def _case(M, K, N, b, bits, seed):
    f = fq()
    x = synth.activations(M, K, seed=seed, outlier_frac=0.005, outlier_scale=50.0).to(DEV)
    w = torch.from_numpy(synth.weights(N, K, seed=seed + 1)).to(DEV)
    bias = torch.from_numpy(synth.random_scales(N, seed=seed + 2, low=-0.1, high=0.1)).to(DEV)
    lin = f.QuantLinear(w, b, bits, bias=bias)
    return x, lin


@pytest.mark.parametrize("bits", [4, 8])
def test_static_scratch_equals_caller_workspace(bits):
    f = fq()
    # largest first, then smaller calls reusing the scratch (its contents from the last call)
    shapes = [(816, 16384, 2048, 128), (50, 16384, 2048, 128), (16, 4096, 1024, 64), (50, 1024, 1536, 128),
              (130, 2048, 512, 32)]
    for i, (M, K, N, b) in enumerate(shapes):
        flush(f"linear_static M={M} K={K} N={N} b={b} bits={bits}")
        need = f.linear_workspace_bytes(M, N, K, bits)
        assert need <= f.LIB.fq_linear_static_max_workspace_bytes()
        x, lin = _case(M, K, N, b, bits, seed=100 * i + bits)
        y_static = f.linear_static(x, lin.w_packed, lin.w_scale, N, b, bits, bias=lin.bias)
        ws = f.workspace(need, DEV)
        y_ref = f.linear(x, lin.w_packed, lin.w_scale, N, b, bits, bias=lin.bias, ws=ws)
        torch.cuda.synchronize()
        assert torch.equal(y_static, y_ref), (M, K, N, b, bits)
        # a second call in a row on the same scratch, fresh tokens of fewer rows
        x2 = synth.activations(max(1, M // 3), K, seed=7 + i, outlier_frac=0.01, outlier_scale=30.0).to(DEV)
        y2 = f.linear_static(x2, lin.w_packed, lin.w_scale, N, b, bits, bias=lin.bias)
        y2_ref = f.linear(x2, lin.w_packed, lin.w_scale, N, b, bits, bias=lin.bias,
                          ws=f.workspace(f.linear_workspace_bytes(x2.shape[0], N, K, bits), DEV))
        torch.cuda.synchronize()
        assert torch.equal(y2, y2_ref), (x2.shape[0], K, N, b, bits)


def test_static_scratch_rejects_oversized_shape():
    f = fq()
    M, K, N, bits = 4096, 32768, 2048, 8  # 128 MiB of intermediate codes
    assert f.linear_workspace_bytes(M, N, K, bits) > f.LIB.fq_linear_static_max_workspace_bytes()
    x = torch.zeros((16, 16), dtype=torch.bfloat16, device=DEV)  # never read: rejected first
    rc = f.LIB.fq_linear_static(f._p(x), K, None, None, M, K, N, 128, bits, 1.0, f._p(x), f._p(x), None, f._p(x),
                                N, f._stream())
    assert rc == 5 and b"fq_linear_static holds" in f.LIB.fq_last_error()
