"""The projection under HIP graph capture (how the benchmark times it): each replay, with
fresh inputs copied into the captured buffers and eager work between replays, equals an
eager call on the same inputs bit for bit (every kernel is deterministic; split-K partials
are added in a fixed order)."""
import numpy as np
import pytest
import torch

from paper_2609_24433_amd import synth
from tests.gpu_util import DEV, flush

pytestmark = pytest.mark.gpu


def fq():
    from paper_2609_24433_amd import fq as _fq
    return _fq


def _replays_match(make_call, x_buf, inputs, out):
    """Capture make_call() (writing `out` from `x_buf`), then for each input: copy it into
    x_buf, replay, and compare with an eager call on a separate output."""
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        make_call()
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=s):
            make_call()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for xin in inputs:
        x_buf.copy_(xin)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = out.clone()
        ref_out = out.clone().zero_()  # eager work between replays, and the eager reference
        make_call(ref_out)
        torch.cuda.synchronize()
        assert torch.equal(got, ref_out)


@pytest.mark.parametrize("M,K,N,bits", [(50, 4096, 1024, 4), (816, 16384, 2048, 4), (50, 16384, 2048, 8),
                                        (33, 32768, 256, 4)])
def test_linear_graph_replays(M, K, N, bits):
    flush(f"graph linear M={M} K={K} N={N} bits={bits}")
    f = fq()
    b = 128
    w = torch.from_numpy(synth.weights(N, K, seed=K + N)).to(DEV)
    lin = f.QuantLinear(w, b, bits)
    x_buf = synth.activations(M, K, seed=1).to(DEV)
    y = torch.empty((M, N), dtype=torch.bfloat16, device=DEV)
    ws = f.workspace(f.linear_workspace_bytes(M, N, K, bits), DEV)

    def call(out=None):
        f.linear(x_buf, lin.w_packed, lin.w_scale, N, b, bits, ws=ws, out=y if out is None else out)

    inputs = [synth.activations(M, K, seed=s, outlier_frac=0.005, outlier_scale=50.0).to(DEV) for s in (2, 3, 4)]
    _replays_match(call, x_buf, inputs, y)


def test_w4a16_and_rotation_graph_replays():
    flush("graph w4a16 + composite rotation")
    f = fq()
    M, K, N, b = 16, 16384, 512, 128
    codes, s_w = f.quantize_weights(torch.from_numpy(synth.weights(N, K, seed=5)).to(DEV), 1, 4)
    packed = f.pack_weights(codes, 4)
    x_buf = synth.activations(M, K, seed=6).to(DEV)
    y = torch.empty((M, N), dtype=torch.bfloat16, device=DEV)
    ws = f.workspace(f.w4a16_workspace_bytes(M, N, K), DEV)

    def call_w16(out=None):
        f.gemm_w4a16(x_buf, packed, s_w, N, ws=ws, out=y if out is None else out)

    _replays_match(call_w16, x_buf, [synth.activations(M, K, seed=s).to(DEV) for s in (7, 8)], y)

    # a single token: only its row staged, K in 4 slices and the split-K epilogue
    x1 = synth.activations(1, K, seed=14).to(DEV)
    y1 = torch.empty((1, N), dtype=torch.bfloat16, device=DEV)
    ws1 = f.workspace(f.w4a16_workspace_bytes(1, N, K), DEV)

    def call_w16_one(out=None):
        f.gemm_w4a16(x1, packed, s_w, N, ws=ws1, out=y1 if out is None else out)

    _replays_match(call_w16_one, x1, [synth.activations(1, K, seed=s).to(DEV) for s in (15, 16)], y1)

    Kr = 2048
    perm = torch.from_numpy(synth.permutation(Kr, seed=9)).to(DEV)
    blocks = torch.from_numpy(synth.orthogonal_blocks(Kr // b, b, seed=10)).to(DEV)
    xr = synth.activations(40, Kr, seed=11).to(DEV)
    codes_out = torch.empty((40, Kr // 2), dtype=torch.uint8, device=DEV)
    delta_out = torch.empty((40,), dtype=torch.float32, device=DEV)
    wsr = f.workspace(int(f.LIB.fq_rotate_quant_workspace_bytes(40, Kr)), DEV)

    def call_rot(out=None):
        c = codes_out if out is None else out
        f._check(f.LIB.fq_rotate_quant(f._p(xr), Kr, f._p(perm), f._p(blocks), None, None, 40, Kr, b, 4, 1.0,
                                       f._p(c), f._p(delta_out), f._p(wsr), wsr.numel(), f._stream()))

    _replays_match(call_rot, xr, [synth.activations(40, Kr, seed=s).to(DEV) for s in (12, 13)], codes_out)
