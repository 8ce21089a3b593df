"""Teacher-forced parity of the 18-layer selective-INT8 backbone chain that the benchmark
times (bench.MixedChain: M = 816 tokens, width 2048, q|k|v and gate|up W4A4, o and down
W8A8, block 128, RMSNorm gains folded into q|k|v and gate|up by eq. (4)).

The chain runs on the device layer by layer on the seeded backbone-layer weights.  At every
layer, each projection's recorded bf16 input and output are checked against the oracle on
rows that straddle the GEMM's row tiles (0/63/64, 127/128, 255/256, 511/512, 767/768, the
ragged last rows) plus seeded random rows:
  * the folded, rounded weights (codes and scales of all N rows) bit for bit;
  * the prologue's codes and scales on the sampled rows bit for bit (eq. (5));
  * the bf16 outputs on the sampled rows within 1e-2 of each row's absmax (eq. (8)).
Each projection is checked on the input the chain actually gave it (teacher forcing), so
an error at layer l cannot hide behind the drift of earlier layers.  The 18 layers are
split over three tests that continue one chain; a test run alone first advances the chain
to its first layer unchecked.
"""
import numpy as np
import pytest
import torch

import bench
import oracle
from paper_2609_24433_amd import synth
from tests.gpu_util import DEV, assert_bf16_close, canonical_codes, flush

pytestmark = pytest.mark.gpu

LAYERS = 18
M = bench.MixedChain.M
ROWS = np.unique(np.concatenate([
    [0, 1, 63, 64, 127, 128, 255, 256, 511, 512, 767, 768, 799, 800, 814, 815],
    np.random.default_rng(2609).choice(M, 8, replace=False)]))


class _State:
    chain = None
    next_layer = 0


def _fq():
    from paper_2609_24433_amd import fq
    return fq


def _advance(to_layer, check):
    """Run the chain up to (not including) `to_layer`, checking each layer when `check`."""
    fq = _fq()
    if _State.chain is None:
        _State.chain = bench.MixedChain(torch, fq, synth, DEV, b=128)
        _State.next_layer = 0
    ch = _State.chain
    while _State.next_layer < to_layer:
        l = _State.next_layer
        w, gain = bench.MixedChain.layer_weights(synth, l)
        ch.add_layer(w, gain)
        rec = ch.layer(l, record=check)
        if check:
            torch.cuda.synchronize()
            _check_layer(fq, ch, l, w, gain, rec)
        _State.next_layer += 1


def _check_layer(fq, ch, l, w, gain, rec):
    b = ch.b
    for site, (n, k, bits) in bench.MixedChain.SHAPES.items():
        flush(f"chain layer {l} site {site} (N={n} K={k} W{bits}A{bits}) rows {len(ROWS)}")
        lin = ch.lins[l][site]
        x_in, y_out = rec[site]
        assert x_in.shape == (M, k) and y_out.shape == (M, n)
        wc, s_w = oracle.quantize_weights(w[site], b, bits, col_scale=gain.get(site))
        np.testing.assert_array_equal(lin.w_scale.cpu().numpy(), s_w, err_msg=f"layer {l} site {site} weight scales")
        np.testing.assert_array_equal(fq.unpack_weights(lin.w_packed, n, k, bits).cpu().numpy(), wc,
                                      err_msg=f"layer {l} site {site} weight codes")
        rows = torch.from_numpy(ROWS).to(DEV)
        xs = x_in.index_select(0, rows).cpu()
        codes, delta = fq.fwht_quant(x_in, b, bits)
        c_ref, d_ref, _, y_ref = oracle.linear(xs, wc, s_w, b, bits)
        np.testing.assert_array_equal(codes.index_select(0, rows).cpu().numpy(), canonical_codes(c_ref, bits),
                                      err_msg=f"layer {l} site {site} activation codes")
        np.testing.assert_array_equal(delta.index_select(0, rows).cpu().numpy(), d_ref,
                                      err_msg=f"layer {l} site {site} activation scales")
        assert_bf16_close(y_out.index_select(0, rows), y_ref)


@pytest.mark.parametrize("first,last", [(0, 6), (6, 12), (12, 18)])
def test_chain_layers(first, last):
    flush(f"chain layers {first}..{last - 1}")
    if _State.chain is not None and _State.next_layer > first:
        _State.chain, _State.next_layer = None, 0
        torch.cuda.empty_cache()
    _advance(first, check=False)
    _advance(last, check=True)
    h = _State.chain.h
    assert torch.isfinite(h).all()
    if last == LAYERS:
        _State.chain = None
        torch.cuda.empty_cache()
