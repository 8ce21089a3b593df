"""Benchmark of the W4A4 runtime quantized projection on one MI355X.

Default workload: the action-expert layer at width 1024 (M = 50 action tokens per
denoising step; q/k/v/o 1024->1024 with k/v 1024->256, gate/up 1024->4096, down
4096->1024; all W4A4 with Hadamard block 128; 10 denoising steps with fresh seeded
activations and shared weights).  One step = one denoising step of the whole hot path
as Alg. 1 runs it at runtime: each of the 4 activation sites is transformed and
quantized once and its consumers (q|k|v, o, gate|up, down) run their integer GEMMs
with the rescale epilogue -- one fused projection (fq_linear) per site, the consumers of
a site packed as one weight matrix.  Weights are folded, rounded and packed on the
device before timing; inputs are resident in HBM when the timed region starts.

The 10-step denoising loop is captured into one HIP graph (each step also into a graph
of its own, for a remainder of K) and the timed region runs exactly K steps.  Prints ONE JSON line, which also carries `points`: the graded single projections
(down-projection K 16384 -> N 2048 at M = 50 / 816 / 4096 and gate-projection M = 816,
cold weights), the rest of the down-projection sweep (M = 1, 16, 256, 4096 in W4A4 and
W8A8; the prologue at b = 32, 64, 128, 256), the 18-layer selective-INT8 backbone chain
(time per layer and end to end, cosine against the fp32 chain), the weight-only INT4
projection, the
prologue alone with the composite rotation beside the block Hadamard, and the offline
GPTQ stages.

  python bench.py [--steps K] [--warmup W] [--no-cpu-baseline] [--no-points] [--only-points]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0      # MI355X HBM3E, GB/s
INT8_PEAK_TOPS = 5000.0    # MI355X dense INT8 MFMA, TOPS (no INT4 MFMA on gfx950)
BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA, TFLOP/s (the W4A16 path)
FP32_VALU_PEAK_TFLOPS = 157.3  # MI355X fp32 vector ALU, TFLOP/s (the composite rotation's fma chains)
FP64_PEAK_TFLOPS = 78.6        # MI355X fp64 vector ALU, TFLOP/s (the GPTQ stages)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-points", action="store_true")
    ap.add_argument("--only-points", action="store_true",
                    help="measure only the graded single projections (profiling aid)")
    ap.add_argument("--quiet", action="store_true")
    ap.add_argument("--traffic-site", default=None,
                    help="run only this site's fused projection 100 times (for HBM counter runs)")
    ap.add_argument("--gemm-counters", action="store_true",
                    help="run the tiled-GEMM points (K 16384 -> N 2048, M 816 and 4096) 10 times each, eagerly, "
                         "for rocprofv3 --pmc runs")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run a plain 256 MiB copy-like kernel 20 times (counter calibration)")
    return ap.parse_args()


def log(args, msg):
    if not args.quiet:
        print(msg, file=sys.stderr, flush=True)


# --------------------------------------------------------------------------- algorithmic bytes

def gemm_bytes(M, N, K, bits, bias=False):
    """x codes + packed W + s_w + delta + y (bf16) (+ bias)."""
    return M * K * bits // 8 + N * K * bits // 8 + 4 * N + 4 * M + 2 * M * N + (4 * N if bias else 0)


def quant_bytes(M, K, bits):
    """bf16 x in, codes + delta out."""
    return 2 * M * K + M * K * bits // 8 + 4 * M


def linear_bytes(M, N, K, bits, bias=False):
    """bf16 x + packed W + s_w + bf16 y (+ bias); intermediate codes excluded."""
    return 2 * M * K + N * K * bits // 8 + 4 * N + 2 * M * N + (4 * N if bias else 0)


# --------------------------------------------------------------------------- HBM traffic

TRAFFIC_FILE = os.path.join(ROOT, "profiles", "site_traffic.json")
CSRC = os.path.join(ROOT, "paper_2609_24433_amd", "csrc")


TRAFFIC_SOURCES = ("fq_api.cpp", "fq_codes.hpp", "fq_device.hpp", "fq_gemm.hip", "fq_quant.hip")  # what a site's projection runs


def sources_digest():
    """SHA-256 over the sources of the kernels a fused projection runs (and the entry point
    that plans them): counter readings are void once any of them changes."""
    import hashlib
    h = hashlib.sha256()
    for name in TRAFFIC_SOURCES:
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()


def measured_traffic(site, part="linear"):
    """HBM bytes per call of `site` from the committed rocprofv3 counter runs (FETCH_SIZE
    and WRITE_SIZE, each scaled by the same counter on a copy of known size): the whole
    fused projection (part "linear") or its GEMM kernel alone (part "gemm"); None when
    there is no reading for these sources and this site."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    r = t.get("sites", {}).get(site)
    if t.get("sources_sha256") != sources_digest() or r is None:
        return None
    pre = "" if part == "linear" else "gemm_"
    if pre + "fetch_kib_per_call" not in r:
        return None
    fetch = r[pre + "fetch_kib_per_call"] * 1024 * t["copy_bytes_read"] / (t["copy_fetch_kib"] * 1024)
    write = r[pre + "write_kib_per_call"] * 1024 * t["copy_bytes_written"] / (t["copy_write_kib"] * 1024)
    return int(round(fetch + write))


def traffic_run(torch, fq, synth, dev, site):
    st = ExpertStep(torch, fq, synth, dev)
    for i in range(100):
        st.run_site(site, i % st.n_steps)
    torch.cuda.synchronize()
    print(json.dumps({"traffic_site": site, "calls": 100}), flush=True)


def copy_calibration(torch, dev):
    n = 64 << 20  # float32 elements: 256 MiB read and 256 MiB written per launch
    a = torch.ones(n, dtype=torch.float32, device=dev)
    b = torch.empty_like(a)
    for _ in range(20):
        torch.add(a, 0.0, out=b)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": 4 * n, "copy_bytes_written": 4 * n, "launches": 20}), flush=True)


# --------------------------------------------------------------------------- workload

class ExpertStep:
    """Device state of the action-expert layer.  Consumers of one activation site share
    that site's transform and quantization (Alg. 1 runtime; Sec. III-B shared sites), so
    their folded weights are packed as one matrix (q|k|v, gate|up): per-output-channel
    scales make this exactly the same as separate consumers.  One fused projection
    (fq_linear) runs per site."""

    def __init__(self, torch, fq, synth, dev, n_steps=10):
        self.torch, self.fq = torch, fq
        self.wl = synth.action_expert_layer()
        wl = self.wl
        self.b = wl.b
        self.sites = wl.sites()
        self.site_projs = {s: [p for p in wl.projections if p.site == s] for s in self.sites}
        self.site_N = {s: sum(p.N for p in ps) for s, ps in self.site_projs.items()}
        self.w_host = {s: np.concatenate([wl.projection_weight(p) for p in ps], axis=0)
                       for s, ps in self.site_projs.items()}
        self.lin = {}
        for s in self.sites:
            w = torch.from_numpy(self.w_host[s]).to(dev)
            self.lin[s] = fq.QuantLinear(w, wl.b, 4)
            del w
        self.x = {s: [wl.site_activation(s, t).to(dev) for t in range(n_steps)] for s in self.sites}
        M = wl.M
        self.y = {s: torch.empty((M, N), dtype=torch.bfloat16, device=dev) for s, N in self.site_N.items()}
        self.ws = {s: fq.workspace(fq.linear_workspace_bytes(M, self.site_N[s], K, 4), dev)
                   for s, K in self.sites.items()}
        self.n_steps = n_steps

    def run_site(self, s, t):
        self.lin[s](self.x[s][t], ws=self.ws[s], out=self.y[s])

    def gemm_call(self, s, t=0):
        """The site's GEMM alone, on the codes and scales of step t's prologue: a
        callable that launches it (for timing the GEMM kernel by itself)."""
        fq, wl = self.fq, self.wl
        K, N = self.sites[s], self.site_N[s]
        codes, delta = fq.fwht_quant(self.x[s][t], self.b, 4)
        ws = fq.workspace(fq.gemm_workspace_bytes(wl.M, N, K, 4), codes.device)
        lin, y = self.lin[s], self.y[s]
        return lambda i: fq.gemm(codes, delta, lin.w_packed, lin.w_scale, N, K, 4, ws=ws, out=y)

    def run(self, t):
        """Enqueue one denoising step: the 4 sites in order."""
        for s in self.sites:
            self.run_site(s, t)


def check_step(st, oracle, torch):
    """Every site of step 0 against the oracle (bf16 within 1e-2 of the row absmax)."""
    st.run(0)
    torch.cuda.synchronize()
    for s in st.sites:
        wc, s_w = oracle.quantize_weights(st.w_host[s], st.b, 4)
        _, _, _, y_ref = oracle.linear(st.x[s][0].cpu(), wc, s_w, st.b, 4)
        yg = st.y[s].float().cpu().numpy().astype(np.float64)
        tol = 1e-2 * np.abs(y_ref).max(axis=1, keepdims=True)
        if not np.all(np.abs(yg - y_ref) <= tol):
            raise SystemExit(f"bench parity check failed at site {s}: GPU output differs from the oracle")


def cpu_baseline(st, oracle, torch, budget_s=15.0):
    """The oracle on the host cores: whole denoising steps (4 site prologues + the 7
    consumers' contractions and rescales) until about budget_s seconds are spent."""
    wq = {s: oracle.quantize_weights(st.w_host[s], st.b, 4) for s in st.sites}
    xs = {s: [a.cpu() for a in st.x[s]] for s in st.sites}
    steps, t0 = 0, time.perf_counter()
    while True:
        t = steps % st.n_steps
        for s in st.sites:
            codes, delta = oracle.fwht_quant(xs[s][t], st.b, 4)
            wc, s_w = wq[s]
            oracle.dequant(oracle.gemm(codes, wc), delta, s_w)
        steps += 1
        el = time.perf_counter() - t0
        if el >= budget_s or steps >= 1000:
            break
    ops = st.wl.ops_per_step() * steps
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            model = next((l.split(":", 1)[1].strip() for l in f if l.startswith("model name")), model)
    except OSError:
        pass
    return {"value": ops / el / 1e12, "unit": "TOPS", "cores": oracle.max_threads(), "kind": "oracle",
            "sample": f"{steps} denoising steps of the action-expert layer (M=50, 7 projections), "
                      f"{el:.1f} s", "cpu_model": model, "nproc": os.cpu_count()}


def graph_of(torch, fn, reps):
    """Capture `reps` back-to-back calls of fn(i) into one HIP graph."""
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        fn(0)
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=s):
            for i in range(reps):
                fn(i)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    return g


def time_graph(torch, g, replays):
    """Average seconds per replay of g, HIP events on the replay stream."""
    g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(replays):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / 1e3 / replays


def replay_spread(torch, g, replays):
    """Seconds of each of `replays` replays of g, timed one by one with HIP events (for the
    p10 / median / p90 of the per-call time)."""
    g.replay()
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(replays + 1)]
    ev[0].record()
    for r in range(replays):
        g.replay()
        ev[r + 1].record()
    torch.cuda.synchronize()
    return [ev[r].elapsed_time(ev[r + 1]) / 1e3 for r in range(replays)]


def time_graph_steps(torch, graphs, K, W, loop=None):
    """Seconds for exactly K denoising steps after W untimed ones.  graphs[t] is step t of
    the loop; `loop`, if given, is one graph of the whole loop (len(graphs) steps), which
    runs the whole loops and the step graphs the remainder."""
    n = len(graphs)

    def run(count):
        if loop is not None:
            for _ in range(count // n):
                loop.replay()
            for t in range(count % n):
                graphs[t].replay()
        else:
            for i in range(count):
                graphs[i % n].replay()

    run(W)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    run(K)
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / 1e3  # seconds


def gemm_counter_run(torch, fq, synth, dev):
    """The tiled GEMM on the down-projection K 16384 -> N 2048 at M = 816 and 4096 (W4A4),
    10 eager calls each, for counter collection."""
    for M in (816, 4096):
        K, N, b, bits = 16384, 2048, 128, 4
        lin = fq.QuantLinear(torch.from_numpy(synth.weights(N, K, seed=K + N + bits)).to(dev), b, bits)
        x = synth.activations(M, K, seed=M + K, outlier_frac=0.005, outlier_scale=50.0).to(dev)
        codes, delta = fq.fwht_quant(x, b, bits)
        ws = fq.workspace(fq.gemm_workspace_bytes(M, N, K, bits), dev)
        y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
        for _ in range(10):
            fq.gemm(codes, delta, lin.w_packed, lin.w_scale, N, K, bits, ws=ws, out=y)
        torch.cuda.synchronize()
        print(json.dumps({"gemm_counters": {"M": M, "K": K, "N": N, "calls": 10}}), flush=True)


def measure_points(torch, fq, synth, dev, log_fn):
    """Graded single-projection points, cold: weights rotate through >= 1 GiB of copies so
    they come from HBM; each point is a graph of back-to-back calls, warmed up with >= 20
    calls, then replayed >= 21 times with HIP events around every replay; `us` is the
    median per-call time (p10 / p90 and the mean beside it)."""
    out = []

    def run_point(name, M, K, N, b, bits, kind, warm=False):
        wl = synth.down_proj_sweep_point(M, b, bits) if K == 16384 else None
        w = torch.from_numpy(synth.weights(N, K, seed=K + N + bits)).to(dev)
        lin = fq.QuantLinear(w, b, bits)
        del w
        wbytes = lin.w_packed.numel()
        # cold: weights rotate through >= 1 GiB of copies; warm: one copy, resident in the caches
        copies = 1 if warm else max(2, min(64, (1 << 30) // wbytes + 1))
        wp = [lin.w_packed.clone() for _ in range(copies)]
        x = (wl.site_activation("D", 0) if wl is not None else
             synth.activations(M, K, seed=M + K, outlier_frac=0.005, outlier_scale=50.0)).to(dev)
        y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
        codes, delta = fq.fwht_quant(x, b, bits)
        if kind == "linear":
            ws = fq.workspace(fq.linear_workspace_bytes(M, N, K, bits), dev)
            call = lambda i: fq.linear(x, wp[i % copies], lin.w_scale, N, b, bits, ws=ws, out=y)
            nbytes = linear_bytes(M, N, K, bits)
        elif kind == "w4a16":
            ws = fq.workspace(fq.w4a16_workspace_bytes(M, N, K), dev)
            call = lambda i: fq.gemm_w4a16(x, wp[i % copies], lin.w_scale, N, ws=ws, out=y)
            nbytes = linear_bytes(M, N, K, 4)
        else:
            ws = fq.workspace(fq.gemm_workspace_bytes(M, N, K, bits), dev)
            call = lambda i: fq.gemm(codes, delta, wp[i % copies], lin.w_scale, N, K, bits, ws=ws, out=y)
            nbytes = gemm_bytes(M, N, K, bits)
        # a graph of back-to-back calls; >= 20 warm-up calls, then 21 replays timed one by one
        # (>= 100 calls in all): the median per-call time is the point's figure, p10 / p90 and
        # the mean beside it
        calls = 50 if warm else copies
        g = graph_of(torch, call, calls)
        for _ in range(max(1, -(-20 // calls))):
            g.replay()
        reps = max(21, -(-100 // calls) | 1)
        spread = sorted(t / calls * 1e6 for t in replay_spread(torch, g, reps))
        us = spread[reps // 2]
        us_mean = sum(spread) / reps
        ops = 2.0 * M * N * K
        t_hbm = nbytes / HBM_PEAK_GBS / 1e3
        t_mfma = ops / (BF16_PEAK_TFLOPS if kind == "w4a16" else INT8_PEAK_TOPS) / 1e6
        rec = {"name": name, "kind": kind, "M": M, "K": K, "N": N, "b": b, "bits": bits, "weights": "warm" if warm else "cold",
               "us": round(us, 3), "us_p10_p90": [round(spread[reps // 10], 3), round(spread[reps - 1 - reps // 10], 3)],
               "us_mean": round(us_mean, 3),
               "TOPS": round(ops / us / 1e6, 2), "GBps": round(nbytes / us / 1e3, 1),
               "bound": "hbm" if t_hbm >= t_mfma else "mfma",
               "roofline_frac": round(max(t_hbm, t_mfma) / us, 4)}
        log_fn(json.dumps(rec))
        out.append(rec)
        del wp, lin, ws, g
        torch.cuda.empty_cache()

    run_point("down_w4a4_m50_linear", 50, 16384, 2048, 128, 4, "linear")
    run_point("down_w4a4_m50_gemm", 50, 16384, 2048, 128, 4, "gemm")
    run_point("down_w8a8_m50_linear", 50, 16384, 2048, 128, 8, "linear")
    run_point("gate_w4a4_m816_linear", 816, 2048, 16384, 128, 4, "linear")
    run_point("down_w4a4_m816_linear", 816, 16384, 2048, 128, 4, "linear")
    run_point("down_w4a4_m816_gemm", 816, 16384, 2048, 128, 4, "gemm")
    run_point("down_w8a8_m816_linear", 816, 16384, 2048, 128, 8, "linear")
    run_point("down_w4a4_m4096_gemm", 4096, 16384, 2048, 128, 4, "gemm")
    # the rest of the down-projection sweep's token counts (K 16384 -> N 2048, b = 128)
    for bits_ in (4, 8):
        for M_ in (1, 16, 256, 4096):
            run_point(f"down_w{bits_}a{bits_}_m{M_}_linear", M_, 16384, 2048, 128, bits_, "linear")
    # warm: the same weights every call (resident in the 256 MB MALL), as shared weights are
    # across denoising steps
    run_point("down_w4a4_m50_linear_warm", 50, 16384, 2048, 128, 4, "linear", warm=True)
    run_point("down_w4a4_m816_linear_warm", 816, 16384, 2048, 128, 4, "linear", warm=True)
    # weight-only INT4 (adaptive layer-norm modulation path): b = 1, no rotation
    run_point("adaln_w4a16_m1", 1, 1024, 6144, 1, 4, "w4a16")
    run_point("down_w4a16_m1", 1, 16384, 2048, 1, 4, "w4a16")
    run_point("down_w4a16_m16", 16, 16384, 2048, 1, 4, "w4a16")
    out += measure_bf16_context(torch, synth, dev, log_fn, out)
    out += measure_prologue_points(torch, fq, synth, dev, log_fn)
    out += measure_mixed_chain(torch, fq, synth, dev, log_fn)
    out += measure_gptq_points(torch, fq, synth, dev, log_fn)
    return out


def measure_bf16_context(torch, synth, dev, log_fn, pts):
    """Context only (the analog of the paper's floating-point engine control): the same
    down-projection shapes as a plain bf16 matrix product (torch.matmul, the vendor GEMM
    library), weights rotating through >= 1 GiB of copies like the W4A4 points.  Each record
    carries the fused W4A4 projection's speed-up over it."""
    out = []
    lin_us = {(p["M"], p["K"], p["N"]): p["us"] for p in pts
              if p["kind"] == "linear" and p["bits"] == 4 and p.get("weights") == "cold"}
    for (M, K, N) in ((50, 16384, 2048), (816, 16384, 2048), (816, 2048, 16384)):
        wt = torch.from_numpy(synth.weights(N, K, seed=K + N).T.copy()).to(dev).to(torch.bfloat16)  # [K, N]
        copies = max(2, min(64, (1 << 30) // (wt.numel() * 2) + 1))
        ws = [wt.clone() for _ in range(copies)]
        del wt
        x = synth.activations(M, K, seed=M + K, outlier_frac=0.005, outlier_scale=50.0).to(dev)
        y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
        g = graph_of(torch, lambda i: torch.matmul(x, ws[i % copies], out=y), copies)
        us = time_graph(torch, g, max(1, 200 // copies)) / copies * 1e6
        rec = {"name": f"context_bf16_matmul_m{M}_k{K}_n{N}", "kind": "bf16_matmul", "M": M, "K": K, "N": N,
               "us": round(us, 3), "TFLOPS": round(2.0 * M * N * K / us / 1e6, 2),
               "w4a4_linear_speedup": round(us / lin_us[(M, K, N)], 2) if (M, K, N) in lin_us else None}
        log_fn(json.dumps(rec))
        out.append(rec)
        del ws, x, y, g
        torch.cuda.empty_cache()
    return out


def measure_gptq_points(torch, fq, synth, dev, log_fn):
    """GPTQ in the transformed coordinates (offline): each stage timed with events over one
    call after a warm-up call.  Algorithmic fp64 flops: second moment T K (K + 1) (the
    distinct entries), factor 2 K^3 / 3 (Cholesky and triangular inverse), sweep N K^2."""
    out = []
    for (name, N, K, T) in (("ae_qkv_gptq", 1536, 1024, 2048), ("ae_down_gptq", 1024, 4096, 2048)):
        b = 128
        calib = synth.activations(T, K, seed=K + 5, outlier_frac=0.005, outlier_scale=50.0).to(dev)
        w = torch.from_numpy(synth.weights(N, K, seed=K + N)).to(dev)
        z = fq.transform(calib, b)
        w_t = fq.transform(w, b)
        G = fq.gptq_hessian(z)
        U = fq.gptq_factor(G)
        stages = (("hessian", lambda: fq.gptq_hessian(z, G), T * K * (K + 1)),
                  ("factor", lambda: fq.gptq_factor(G), 2 * K ** 3 / 3),
                  ("sweep", lambda: fq.gptq_sweep(w_t, U, b, 4), N * K ** 2))
        rec = {"name": name, "kind": "gptq", "N": N, "K": K, "T": T, "b": b, "bits": 4}
        total = 0.0
        for sname, fn, flops in stages:
            fn()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) * 1e3
            total += us
            rec[f"{sname}_us"] = round(us, 1)
            rec[f"{sname}_fp64_frac"] = round(flops / (us * 1e-6) / (FP64_PEAK_TFLOPS * 1e12), 4)
        rec["total_us"] = round(total, 1)
        log_fn(json.dumps(rec))
        out.append(rec)
        del calib, w, z, w_t, G, U
        torch.cuda.empty_cache()
    return out


def measure_prologue_points(torch, fq, synth, dev, log_fn):
    """The activation prologue alone, block Hadamard butterfly against the stored composite
    rotation (permutation + dense per-block matrices) on the same tokens.  Algorithmic bytes:
    x, codes and scales, plus the permutation and the blocks for the composite one; its
    2 M K b flops (fp32 fma chains) give the ALU side of its roofline."""
    out = []
    for (name, M, K, b) in (("ae_prologue_m50_k1024", 50, 1024, 128), ("ae_prologue_m50_k4096", 50, 4096, 128),
                            ("lang_prologue_m816_k2048", 816, 2048, 128)):
        x = synth.activations(M, K, seed=M + K + 7, outlier_frac=0.005, outlier_scale=50.0).to(dev)
        perm = torch.from_numpy(synth.permutation(K, seed=K)).to(dev)
        blocks = torch.from_numpy(synth.orthogonal_blocks(K // b, b, seed=b)).to(dev)
        codes = torch.empty((M, K // 2), dtype=torch.uint8, device=dev)
        delta = torch.empty((M,), dtype=torch.float32, device=dev)
        ws = fq.workspace(int(fq.LIB.fq_rotate_quant_workspace_bytes(M, K)), dev)
        reps = 50
        base = M * (2 * K + K // 2 + 4)
        for kind in ("fwht", "rotate"):
            if kind == "fwht":
                call = lambda i: fq._check(fq.LIB.fq_fwht_quant(fq._p(x), K, None, None, M, K, b, 4, 1.0, fq._p(codes),
                                                                 fq._p(delta), fq._stream()))
                nbytes, flops = base, 0
            else:
                call = lambda i: fq._check(fq.LIB.fq_rotate_quant(fq._p(x), K, fq._p(perm), fq._p(blocks), None, None,
                                                                   M, K, b, 4, 1.0, fq._p(codes), fq._p(delta),
                                                                   fq._p(ws), ws.numel(), fq._stream()))
                nbytes, flops = base + 4 * K + 4 * K * b, 2.0 * M * K * b
            g = graph_of(torch, call, reps)
            us = time_graph(torch, g, 4) / reps * 1e6
            t_hbm = nbytes / HBM_PEAK_GBS / 1e3
            t_alu = flops / FP32_VALU_PEAK_TFLOPS / 1e6
            rec = {"name": f"{name}_{kind}", "kind": f"prologue_{kind}", "M": M, "K": K, "b": b, "bits": 4,
                   "us": round(us, 3), "GBps": round(nbytes / us / 1e3, 1),
                   "bound": "hbm" if t_hbm >= t_alu else "alu", "roofline_frac": round(max(t_hbm, t_alu) / us, 4)}
            log_fn(json.dumps(rec))
            out.append(rec)
            del g
        del x, perm, blocks, codes, delta, ws
        torch.cuda.empty_cache()
    # the butterfly prologue at every block size of the down-projection sweep (M = 816,
    # K = 16384, Student-t rows): log2 b stages, the last log2(b / 16) across lanes
    M, K = 816, 16384
    for b in (32, 64, 128, 256):
        x = synth.down_proj_sweep_point(M, b, 4).site_activation("D", 0).to(dev)
        codes = torch.empty((M, K // 2), dtype=torch.uint8, device=dev)
        delta = torch.empty((M,), dtype=torch.float32, device=dev)
        call = lambda i: fq._check(fq.LIB.fq_fwht_quant(fq._p(x), K, None, None, M, K, b, 4, 1.0, fq._p(codes),
                                                         fq._p(delta), fq._stream()))
        reps = 20
        g = graph_of(torch, call, reps)
        us = time_graph(torch, g, 4) / reps * 1e6
        nbytes = M * (2 * K + K // 2 + 4)
        rec = {"name": f"sweep_prologue_m816_b{b}_fwht", "kind": "prologue_fwht", "M": M, "K": K, "b": b, "bits": 4,
               "us": round(us, 3), "GBps": round(nbytes / us / 1e3, 1), "bound": "hbm",
               "roofline_frac": round(nbytes / HBM_PEAK_GBS / 1e3 / us, 4)}
        log_fn(json.dumps(rec))
        out.append(rec)
        del g, x, codes, delta
        torch.cuda.empty_cache()
    return out


def measure_mixed_chain(torch, fq, synth, dev, log_fn, layers=18):
    """Selective-INT8 language backbone: `layers` layers of the width-2048 shapes at
    M = 816 (q|k|v 2048 -> 2560 and gate|up 2048 -> 32768 W4A4; o 2048 -> 2048 and down
    16384 -> 2048 W8A8; b = 128).  Per layer: a = RMSNorm(h) (eps 1e-6), q|k|v = Lin_A(a)
    with the norm's gain folded into the weights; o = Lin_O(q), q standing in for the
    attention output; h1 = h + o; g|u = Lin_B(RMSNorm(h1)), gain folded; d =
    Lin_D(silu(g) * u); h = h1 + d.  Norms, SwiGLU and residuals run in fp32 torch (outside
    the projection).  Weights N(0, 0.02) drawn on the device (torch generator seeded
    4000 + layer), gains U(0.5, 1.5); h0 = the backbone's seeded activations.  Times the
    whole quantized chain and its 4 fused projections per layer (HIP graphs) and reports
    the cosine of the final hidden state against the same chain in fp32 with the
    unquantized weights and explicit gains."""
    M, D, KV, F, b = 816, 2048, 256, 16384, 128
    shapes = {"A": (D + 2 * KV, D, 4), "O": (D, D, 8), "B": (2 * F, D, 4), "D": (D, F, 8)}

    def layer_weights(l):
        g = torch.Generator(device=dev)
        g.manual_seed(4000 + l)
        w = {s_: torch.randn((n, k), generator=g, device=dev, dtype=torch.float32) * 0.02
             for s_, (n, k, _) in shapes.items()}
        gain = {s_: torch.rand((D,), generator=g, device=dev, dtype=torch.float32) + 0.5 for s_ in ("A", "B")}
        return w, gain

    def rms(h):
        return h * torch.rsqrt(torch.mean(h * h, dim=1, keepdim=True) + 1e-6)

    lins, ws_bytes = [], 0
    for l in range(layers):
        w, gain = layer_weights(l)
        lins.append({s_: fq.QuantLinear(w[s_], b, bits, col_scale=gain.get(s_))
                     for s_, (_, _, bits) in shapes.items()})
        ws_bytes = max([ws_bytes] + [fq.linear_workspace_bytes(M, n, k, bits) for n, k, bits in shapes.values()])
        del w, gain
    ws = fq.workspace(ws_bytes, dev)
    h0 = synth.backbone_layer_mixed(0).site_activation("A", 0).to(dev).float()
    h = torch.empty_like(h0)
    a_in = torch.empty((M, D), dtype=torch.bfloat16, device=dev)
    qkv = torch.empty((M, D + 2 * KV), dtype=torch.bfloat16, device=dev)
    o = torch.empty((M, D), dtype=torch.bfloat16, device=dev)
    b_in = torch.empty((M, D), dtype=torch.bfloat16, device=dev)
    gu = torch.empty((M, 2 * F), dtype=torch.bfloat16, device=dev)
    m_in = torch.empty((M, F), dtype=torch.bfloat16, device=dev)
    dn = torch.empty((M, D), dtype=torch.bfloat16, device=dev)

    def forward(i):
        h.copy_(h0)
        for L in lins:
            a_in.copy_(rms(h))
            L["A"](a_in, ws=ws, out=qkv)
            L["O"](qkv[:, :D], ws=ws, out=o)
            h.add_(o.float())
            b_in.copy_(rms(h))
            L["B"](b_in, ws=ws, out=gu)
            m_in.copy_(torch.nn.functional.silu(gu[:, :F].float()) * gu[:, F:].float())
            L["D"](m_in, ws=ws, out=dn)
            h.add_(dn.float())

    def projections(i):
        for L in lins:
            L["A"](a_in, ws=ws, out=qkv)
            L["O"](qkv[:, :D], ws=ws, out=o)
            L["B"](b_in, ws=ws, out=gu)
            L["D"](m_in, ws=ws, out=dn)

    g_chain = graph_of(torch, forward, 1)
    us_chain = time_graph(torch, g_chain, 5) * 1e6
    g_chain.replay()
    torch.cuda.synchronize()
    h_q = h.clone()
    g_proj = graph_of(torch, projections, 1)
    us_proj = time_graph(torch, g_proj, 5) * 1e6
    del g_chain, g_proj

    # fp32 reference chain (unquantized weights, gains applied to the activations)
    hr = h0.clone()
    for l in range(layers):
        w, gain = layer_weights(l)
        qkv_r = (gain["A"] * rms(hr)) @ w["A"].t()
        hr = hr + qkv_r[:, :D] @ w["O"].t()
        gu_r = (gain["B"] * rms(hr)) @ w["B"].t()
        hr = hr + (torch.nn.functional.silu(gu_r[:, :F]) * gu_r[:, F:]) @ w["D"].t()
        del w, gain
    cos = torch.nn.functional.cosine_similarity(h_q.flatten(), hr.flatten(), dim=0).item()
    ops = layers * 2.0 * M * sum(n * k for n, k, _ in shapes.values())
    rec = {"name": f"mixed_chain_{layers}l_m{M}", "kind": "chain", "layers": layers, "M": M, "b": b,
           "us_total": round(us_chain, 1), "us_per_layer": round(us_chain / layers, 2),
           "projections_us_per_layer": round(us_proj / layers, 2),
           "projection_TOPS": round(ops / us_proj / 1e6, 1), "cosine_vs_fp32": round(cos, 6)}
    log_fn(json.dumps(rec))
    del lins, ws
    torch.cuda.empty_cache()
    return [rec]


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the projection's multi-GPU sharding is a design note, not a measured path).",
              file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2609_24433_amd import fq, synth
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    K_steps, W = args.steps, args.warmup

    if args.copy_calibration:
        copy_calibration(torch, dev)
        return
    if args.gemm_counters:
        gemm_counter_run(torch, fq, synth, dev)
        return
    if args.traffic_site:
        traffic_run(torch, fq, synth, dev, args.traffic_site)
        return
    if args.only_points:
        print(json.dumps({"points": measure_points(torch, fq, synth, dev, lambda m: log(args, m))}), flush=True)
        return
    st = ExpertStep(torch, fq, synth, dev)
    import oracle  # the parity check and the CPU baseline only
    check_step(st, oracle, torch)
    log(args, "parity check ok")

    # the denoising loop (10 steps) captured as one graph, as a serving loop runs it;
    # one graph per step covers a remainder of K, and is also timed on its own
    graphs = [graph_of(torch, lambda i, t=t: st.run(t), 1) for t in range(st.n_steps)]
    loop = graph_of(torch, lambda i: st.run(i), st.n_steps)
    elapsed = time_graph_steps(torch, graphs, K_steps, W, loop=loop)
    ops_step = st.wl.ops_per_step()
    value = ops_step * K_steps / elapsed / 1e12
    ms_step = elapsed * 1e3 / K_steps
    per_step_graphs = time_graph_steps(torch, graphs, K_steps, W) * 1e6 / K_steps
    log(args, f"loop graph replay: {ms_step * 1e3:.2f} us/step, {value:.3f} TOPS; "
              f"one graph per step: {per_step_graphs:.2f} us/step")

    # per-site fused projection duration: a graph of 50 back-to-back calls per site
    # (weights resident, as across the denoising steps), HIP events around the replays
    M = st.wl.M
    per_site = {}
    for s_, K in st.sites.items():
        g = graph_of(torch, lambda i, s_=s_: st.run_site(s_, i % st.n_steps), 50)
        per_site[s_] = time_graph(torch, g, 4) / 50 * 1e6
    log(args, "per-site fused projection us: " + ", ".join(f"{k}={v:.2f}" for k, v in per_site.items()))
    # the dominant kernel: the longest single launch of the step, a site's GEMM (each
    # site's GEMM timed alone as a graph of 50 back-to-back launches, weights resident)
    gemm_site = {}
    for s_ in st.sites:
        g = graph_of(torch, st.gemm_call(s_), 50)
        gemm_site[s_] = time_graph(torch, g, 4) / 50 * 1e6
    dom = max(gemm_site, key=lambda k: gemm_site[k])
    Kd, Nd = st.sites[dom], st.site_N[dom]
    dom_bytes = gemm_bytes(M, Nd, Kd, 4)
    ach = dom_bytes / gemm_site[dom] / 1e3  # GB/s
    lin_bytes = linear_bytes(M, Nd, Kd, 4)
    log(args, "per-site GEMM kernel us: " + ", ".join(f"{k}={v:.2f}" for k, v in gemm_site.items()))

    rec = {
        "metric": "W4A4 fused-linear TOPS and us/projection at M=50 and M=816; % of roofline",
        "value": round(value, 4), "unit": "TOPS", "n_gpus": 1, "steps": K_steps, "warmup": W,
        "ms_per_step": round(ms_step, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "int4 (int8 MFMA, int32 acc) / fp32 prologue / bf16 io",
        "data": "synthetic (seeded N(0,1) tokens with 0.5% outlier channels x50; N(0,0.02) weights)",
        "config": {"workload": "action-expert layer, width 1024, M=50 tokens per denoising step, "
                               "q/k/v/o/gate/up/down W4A4, block 128, 10 steps of fresh activations; "
                               "one fused projection per activation site (q|k|v and gate|up grouped)",
                   "M": M, "b": st.wl.b, "projections": 7, "sites": 4,
                   "graph": f"the {st.n_steps}-step denoising loop as one HIP graph",
                   "us_per_step_one_graph_per_step": round(per_step_graphs, 3),
                   "us_per_projection": round(ms_step * 1e3 / 7, 3),
                   "us_per_site": {k: round(v, 3) for k, v in per_site.items()},
                   "gemm_us_per_site": {k: round(v, 3) for k, v in gemm_site.items()}},
        "roofline": {"bound": "hbm", "kernel": f"gemm_stream_kernel, site {dom} GEMM, M={M} K={Kd} N={Nd} "
                                               f"(the step's longest launch)",
                     "achieved": round(ach, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBS, 4),
                     "traffic": measured_traffic(dom, "gemm"),
                     "kernel_us": round(gemm_site[dom], 3), "algorithmic_bytes": dom_bytes,
                     "fused_projection": {"site": dom, "us": round(per_site[dom], 3),
                                          "algorithmic_bytes": lin_bytes,
                                          "achieved": round(lin_bytes / per_site[dom] / 1e3, 1),
                                          "frac": round(lin_bytes / per_site[dom] / 1e3 / HBM_PEAK_GBS, 4),
                                          "traffic": measured_traffic(dom, "linear")}},
    }
    if not args.no_points:
        rec["points"] = measure_points(torch, fq, synth, dev, lambda m: log(args, m))
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(st, oracle, torch)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
