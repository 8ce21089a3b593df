"""GPU parity at the workloads' full sizes, through the same fused entry point and launch
plan that the benchmark times (fq_linear via QuantLinear, workspace supplied).

* prologue codes and per-token scales: every row, bit-exact against the oracle;
* weight codes and per-channel scales: bit-exact;
* INT32 accumulators: bit-exact on sampled rows (the oracle's brute-force GEMM on those
  rows; a token's codes depend on its own row only, so the sample is exact);
* bf16 outputs: within 1e-2 of each row's absmax on the same rows.
Rows are sampled on both sides of every 128-row tile boundary and at the batch ends.
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


def sample_rows(M: int, extra: int = 4, seed: int = 0) -> np.ndarray:
    rows = {0, M - 1}
    for t in range(128, M, 128):
        rows.update((t - 1, t))
    rng = np.random.default_rng(seed)
    rows.update(rng.integers(0, M, size=extra).tolist())
    return np.array(sorted(r for r in rows if 0 <= r < M), dtype=np.int64)


def site_groups(wl):
    """Consumers of one activation site with one bit width share a fused projection."""
    groups = []
    for p in wl.projections:
        if groups and groups[-1][0] == p.site and groups[-1][1] == p.bits:
            groups[-1][2].append(p)
        else:
            groups.append((p.site, p.bits, [p]))
    return groups


def run_and_check(x: torch.Tensor, w: np.ndarray, b: int, bits: int, rows=None, col_scale=None,
                  bias=None):
    """One fused projection on the GPU, checked against the oracle; returns the GPU output."""
    f = fq()
    M, K = x.shape
    N = w.shape[0]
    cs = None if col_scale is None else torch.from_numpy(col_scale).to(DEV)
    bd = None if bias is None else torch.from_numpy(bias).to(DEV)
    lin = f.QuantLinear(torch.from_numpy(w).to(DEV), b, bits, bias=bd, col_scale=cs)
    xd = x.to(DEV)
    ws = f.workspace(f.linear_workspace_bytes(M, N, K, bits), DEV)
    y = lin(xd, ws=ws)
    codes, delta = f.fwht_quant(xd, b, bits)
    torch.cuda.synchronize()

    wc, s_w = oracle.quantize_weights(w, b, bits, col_scale)
    np.testing.assert_array_equal(lin.w_scale.cpu().numpy(), s_w)
    np.testing.assert_array_equal(f.unpack_weights(lin.w_packed, N, K, bits).cpu().numpy(), wc)

    c_ref, d_ref = oracle.fwht_quant(x, b, bits)
    np.testing.assert_array_equal(codes.cpu().numpy(), canonical_codes(c_ref, bits))
    np.testing.assert_array_equal(delta.cpu().numpy(), d_ref)

    rows = np.arange(M) if rows is None else rows
    acc_ref = oracle.gemm(c_ref[rows], wc)
    y_ref = oracle.dequant(acc_ref, d_ref[rows], s_w, bias)
    assert_bf16_close(y[torch.from_numpy(rows).to(DEV)], y_ref)
    # the accumulators behind those outputs, through the GEMM entry point on the same codes
    _, acc = f.gemm(codes, delta, lin.w_packed, lin.w_scale, N, K, bits, bias=lin.bias, want_acc=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(acc.cpu().numpy()[rows].astype(np.int64), acc_ref)
    return y


# ------------------------------------------------------------------ single linear (M=64)

def test_single_linear_full():
    wl = synth.single_linear()
    p = wl.projections[0]
    flush(f"full size: {wl.name}")
    x = synth.activations(wl.M, p.K, seed=0, outlier_frac=wl.outlier_frac, outlier_scale=wl.outlier_scale)
    run_and_check(x, wl.projection_weight(p), wl.b, p.bits)


# ------------------------------------------------------------------ action-expert layer (M=50)

@pytest.mark.parametrize("step", [0, 9])
def test_action_expert_layer_full(step):
    wl = synth.action_expert_layer()
    for site, bits, ps in site_groups(wl):
        w = np.concatenate([wl.projection_weight(p) for p in ps], axis=0)
        flush(f"full size: {wl.name} step {step} site {site} N={w.shape[0]} K={w.shape[1]}")
        run_and_check(wl.site_activation(site, step), w, wl.b, bits)


# ------------------------------------------------------------------ backbone layer (M=816)

@pytest.mark.parametrize("site", ["A", "O", "B", "D"])
def test_backbone_layer_sampled(site):
    wl = synth.backbone_layer()
    for s, bits, ps in site_groups(wl):
        if s != site:
            continue
        w = np.concatenate([wl.projection_weight(p) for p in ps], axis=0)
        flush(f"full size: {wl.name} site {site} N={w.shape[0]} K={w.shape[1]}")
        run_and_check(wl.site_activation(site, 0), w, wl.b, bits, rows=sample_rows(wl.M, seed=ord(site)))


# ------------------------------------------------------------------ selective-INT8 chain

def _rmsnorm_bf16(y: torch.Tensor) -> torch.Tensor:
    """RMSNorm without its gain (the gain is folded into the next weights), bf16 out."""
    v = y.float().cpu().numpy().astype(np.float32)
    r = v / np.sqrt(np.mean(v * v, axis=1, keepdims=True) + np.float32(1e-6))
    return torch.from_numpy(r.astype(np.float32)).to(torch.bfloat16)


def test_backbone_mixed_chain_two_layers():
    """Layer 0's down-projection output feeds layer 1 through RMSNorm; the norm's random
    per-channel gain is folded into layer 1's weights.  o_proj and down_proj are W8A8."""
    x = None
    for layer in (0, 1):
        wl = synth.backbone_layer_mixed(layer)
        gain = synth.channel_vector(2048, seed=7000 + layer, low=0.5, high=1.5)
        rows = sample_rows(wl.M, extra=2, seed=layer)
        y_site = {}
        for site, bits, ps in site_groups(wl):
            w = np.concatenate([wl.projection_weight(p) for p in ps], axis=0)
            if site == "A" and x is not None:
                xin, cs = x, gain
            else:
                xin, cs = wl.site_activation(site, 0), None
            flush(f"full size: {wl.name} site {site} w{bits}a{bits} N={w.shape[0]} K={w.shape[1]}")
            y_site[site] = run_and_check(xin, w, wl.b, bits, rows=rows, col_scale=cs)
        assert {p.bits for p in wl.projections if p.name in ("o", "down")} == {8}
        x = _rmsnorm_bf16(y_site["D"])


# ------------------------------------------------------------------ down-projection sweep

SWEEP = [
    # (M, b, bits): every M, every b and both widths appear
    (1, 32, 4), (16, 64, 4), (50, 128, 4), (256, 256, 4), (816, 32, 4), (4096, 128, 4),
    (1, 256, 8), (16, 128, 8), (50, 64, 8), (256, 32, 8), (816, 128, 8), (4096, 256, 8),
    (50, 256, 4), (816, 64, 8),
]


@pytest.mark.parametrize("M,b,bits", SWEEP)
def test_down_proj_sweep(M, b, bits):
    wl = synth.down_proj_sweep_point(M, b, bits)
    p = wl.projections[0]
    flush(f"full size: {wl.name}")
    x = wl.site_activation("D", 0)
    run_and_check(x, wl.projection_weight(p), b, bits, rows=sample_rows(M, seed=M + b))


# ------------------------------------------------------------------ k-group plan, fused path

@pytest.mark.parametrize("M,N", [(1700, 2000), (3072, 2048)])
def test_fused_kgroup_wide_plan_sampled(M, N):
    """A fused projection whose prologue writes the codes k-step major takes the k-group
    GEMM on grids of up to 1023 tiles of 128 x 64 at K = 16384, where the GEMM entry point
    (canonical codes) keeps the LDS-ring kernel: ragged rows and columns against the oracle
    on sampled rows, and the two outputs identical bit for bit everywhere."""
    flush(f"full size: fused k-group plan M={M} K=16384 N={N}")
    f = fq()
    K, b, bits = 16384, 128, 4
    x = synth.activations(M, K, seed=M, outlier_frac=0.005, outlier_scale=50.0)
    w = synth.weights(N, K, seed=N + 7)
    y = run_and_check(x, w, b, bits, rows=sample_rows(M, seed=M))
    lin = f.QuantLinear(torch.from_numpy(w).to(DEV), b, bits)
    codes, delta = f.fwht_quant(x.to(DEV), b, bits)
    y2 = f.gemm(codes, delta, lin.w_packed, lin.w_scale, N, K, bits)
    torch.cuda.synchronize()
    assert torch.equal(y, y2)
