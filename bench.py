"""Benchmark of the W4A4 runtime quantized projection on one MI355X.

Workload of the headline line: the action-expert layer at width 1024 (M = 50 action
tokens per denoising step; q/k/v/o 1024->1024 with k/v 1024->256, gate/up 1024->4096,
down 4096->1024; all W4A4 with Hadamard block 128; 10 denoising steps with fresh seeded
activations and shared weights).  One step = one denoising step of the whole hot path as
Alg. 1 runs it at runtime: each of the 4 activation sites is transformed and quantized
once and its consumers (q|k|v, o, gate|up, down) run their integer GEMMs with the rescale
epilogue -- one fused projection (fq_linear) per site, the consumers of a site packed as
one weight matrix.  Weights are folded, rounded and packed on the device before timing;
inputs are resident in HBM when the timed region starts.  The 10-step denoising loop is
captured into one HIP graph (each step also into a graph of its own, for a remainder of K)
and the timed region runs exactly K steps.

The JSON line also carries
  roofline   the step's longest launch, timed with cold weights (rotating copies of >= 1 GiB
             so that they come from HBM), resident weights beside it;
  graded     the graded single projections: the down-projection K 16384 -> N 2048 at
             M = 50, 816 and 4096, W4A4 and W8A8, the fused projection and its GEMM alone,
             and the backbone's gate (2048 -> 16384) and down projections at M = 816, cold;
  points     every other configuration: the single linear (M 64, 1024 -> 1024, b 64), the
             action-expert sites with cold and resident weights, every projection of the
             backbone layer at M = 816, the whole down-projection sweep (48 points: M in
             {1, 16, 50, 256, 816, 4096} x b in {32, 64, 128, 256} x W4A4 / W8A8), the
             prologue alone (block Hadamard against the composite rotation), weight-only
             INT4, the offline GPTQ stages, the 18-layer selective-INT8 backbone chain at
             b = 128 and b = 1, and bf16 torch.matmul context points;
  cpu_baseline  the CPU oracle on the host cores (all threads, and one thread).
Each graded and point record carries `rocprof_us`, the per-call kernel time of the same
point in the committed rocprofv3 summary (profiles/points_kernels_by_grid.json, written by
--summarize-trace from a `--rocprof-points` trace) while its source digest matches.

  python bench.py [--steps K] [--warmup W] [--no-cpu-baseline] [--no-points] [--points GROUPS]
  python bench.py --rocprof-points           (under rocprofv3 --kernel-trace --stats)
  python bench.py --summarize-trace CSV --manifest STDOUT_OF_THAT_RUN
  python bench.py --traffic-site S | --counter-point P | --copy-calibration   (under rocprofv3 --pmc)
  python bench.py --summarize-traffic DIR | --summarize-counters DIR --counter-points P,...
  python bench.py --summarize-stats CSV --bench-json STDOUT_OF_A_TRACED_DEFAULT_RUN
"""
from __future__ import annotations

import argparse
import hashlib
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
COLD_BYTES = 1 << 30       # weights rotate through >= 1 GiB of copies (4x the 256 MB MALL)

CSRC = os.path.join(ROOT, "paper_2609_24433_amd", "csrc")
PROFILES = os.path.join(ROOT, "profiles")
TRAFFIC_FILE = os.path.join(PROFILES, "site_traffic.json")
POINTS_TRACE_FILE = os.path.join(PROFILES, "points_kernels_by_grid.json")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-points", action="store_true")
    ap.add_argument("--quiet", action="store_true")
    ap.add_argument("--traffic-site", default=None,
                    help="run only this site's fused projection 100 times (for HBM counter runs)")
    ap.add_argument("--counter-point", default=None,
                    help="run one named point's calls eagerly (for rocprofv3 --pmc runs)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run a plain 256 MiB copy-like kernel 20 times (counter calibration)")
    ap.add_argument("--rocprof-points", action="store_true",
                    help="run every timed point eagerly, one idle-separated segment each (for a kernel trace)")
    ap.add_argument("--summarize-trace", default=None, metavar="CSV",
                    help="summarize a --rocprof-points kernel trace into profiles/ and exit")
    ap.add_argument("--manifest", default=None, help="stdout of the --rocprof-points run (its point list)")
    ap.add_argument("--summarize-traffic", default=None, metavar="DIR",
                    help="summarize --traffic-site / --copy-calibration counter runs under DIR into profiles/ and exit")
    ap.add_argument("--summarize-counters", default=None, metavar="DIR",
                    help="summarize --counter-point counter runs under DIR into profiles/ and exit")
    ap.add_argument("--counter-points", default=None, help="comma-separated points for --summarize-counters")
    ap.add_argument("--summarize-stats", default=None, metavar="CSV",
                    help="write profiles/bench_kernel_stats.md from a --stats kernel summary of the default run and exit")
    ap.add_argument("--bench-json", default=None, help="stdout of the traced run, for --summarize-stats")
    ap.add_argument("--points", default=None, help="comma-separated point groups to run (default: all)")
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


def roofline(nbytes, ops, us, peak_ops=INT8_PEAK_TOPS):
    """Bound, achieved and fraction of the roofline for one call of `us` microseconds."""
    t_hbm = nbytes / HBM_PEAK_GBS / 1e3
    t_mfma = ops / peak_ops / 1e6
    if t_hbm >= t_mfma:
        return {"bound": "hbm", "achieved": round(nbytes / us / 1e3, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(t_hbm / us, 4)}
    return {"bound": "mfma", "achieved": round(ops / us / 1e6, 1), "peak": peak_ops, "unit": "TOPS",
            "frac": round(t_mfma / us, 4)}


# --------------------------------------------------------------------------- source digest

def sources_digest():
    """SHA-256 over the library sources: a profile reading is void once any of them changes."""
    h = hashlib.sha256()
    for name in sorted(os.listdir(CSRC)):
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()


def measured_traffic(site, part="linear"):
    """HBM bytes per call of `site` from the committed rocprofv3 counter runs (FETCH_SIZE
    and WRITE_SIZE, each scaled by the same counter on a copy of known size); None when
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


def rocprof_points():
    """name -> committed rocprof summary record of a point (kernel time per call, kernels
    by grid), or {} when the summary does not match these sources."""
    try:
        with open(POINTS_TRACE_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return {}
    if t.get("sources_sha256") != sources_digest():
        return {}
    return t.get("points", {})


# --------------------------------------------------------------------------- timing

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
    """Seconds of each of `replays` replays of g, timed one by one with HIP events."""
    g.replay()
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(replays + 1)]
    ev[0].record()
    for r in range(replays):
        g.replay()
        ev[r + 1].record()
    torch.cuda.synchronize()
    return [ev[r].elapsed_time(ev[r + 1]) / 1e3 for r in range(replays)]


def time_calls(torch, call, calls):
    """Per-call microseconds of call(i): a graph of `calls` back-to-back calls, warmed up
    with >= 20 calls, then >= 21 replays timed one by one; (median, p10, p90, mean)."""
    g = graph_of(torch, call, calls)
    for _ in range(max(1, -(-20 // calls))):
        g.replay()
    reps = max(21, -(-100 // calls) | 1)
    spread = sorted(t / calls * 1e6 for t in replay_spread(torch, g, reps))
    del g
    return spread[reps // 2], spread[reps // 10], spread[reps - 1 - reps // 10], sum(spread) / reps


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


# --------------------------------------------------------------------------- the denoising step

class ExpertStep:
    """Device state of the action-expert layer.  Consumers of one activation site share
    that site's transform and quantization (Alg. 1 runtime; Sec. III-B shared sites), so
    their folded weights are packed as one matrix (q|k|v, gate|up): per-output-channel
    scales make this exactly the same as separate consumers.  One fused projection
    (fq_linear) runs per site.  copies > 1 keeps that many copies of the packed weights,
    call c using copy c % copies (cold weights)."""

    def __init__(self, torch, fq, synth, dev, n_steps=10, copies=1):
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
        self.copies = copies
        self.wp = {s: [self.lin[s].w_packed] + [self.lin[s].w_packed.clone() for _ in range(copies - 1)]
                   for s in self.sites}
        self.x = {s: [wl.site_activation(s, t).to(dev) for t in range(n_steps)] for s in self.sites}
        M = wl.M
        self.y = {s: torch.empty((M, N), dtype=torch.bfloat16, device=dev) for s, N in self.site_N.items()}
        self.ws = {s: fq.workspace(fq.linear_workspace_bytes(M, self.site_N[s], K, 4), dev)
                   for s, K in self.sites.items()}
        self.n_steps = n_steps

    def run_site(self, s, t, c=0):
        lin = self.lin[s]
        self.fq.linear(self.x[s][t % self.n_steps], self.wp[s][c % self.copies], lin.w_scale, self.site_N[s], self.b,
                       4, ws=self.ws[s], out=self.y[s])

    def run(self, t, c=0):
        """Enqueue one denoising step: the 4 sites in order."""
        for s in self.sites:
            self.run_site(s, t, c)

    def weight_bytes(self):
        return sum(w.numel() for w in (self.lin[s].w_packed for s in self.sites))


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


# --------------------------------------------------------------------------- single-projection points

def cold_copies(nbytes):
    return max(2, min(64, COLD_BYTES // max(1, nbytes) + 1))


def point_specs(groups=None):
    """Every timed single-projection point: (group, name, M, K, N, b, bits, kind, weights).
    kind: linear (fq_linear, the fused projection), gemm (the GEMM alone, on the prologue's
    codes), w4a16 (weight-only INT4); weights: cold or warm."""
    specs = []

    def add(g, n, M, K, N, b, bits, kind, w="cold"):
        specs.append((g, n, M, K, N, b, bits, kind, w))

    # graded: the down-projection K 16384 -> N 2048 (down-projection sweep data, b = 128) and the
    # backbone's gate and down projections at M = 816
    for M in (50, 816, 4096):
        for bits in (4, 8):
            for kind in ("linear", "gemm"):
                add("graded", f"down_m{M}_w{bits}a{bits}_{kind}", M, 16384, 2048, 128, bits, kind)
    for kind in ("linear", "gemm"):
        add("graded", f"backbone_gate_m816_w4a4_{kind}", 816, 2048, 16384, 128, 4, kind)
        add("graded", f"backbone_down_m816_w4a4_{kind}", 816, 16384, 2048, 128, 4, kind)
    # the single linear (M = 64, K = N = 1024, b = 64)
    for w in ("cold", "warm"):
        add("single", f"single_m64_k1024_n1024_{w}", 64, 1024, 1024, 64, 4, "linear", w)
    # action-expert sites, cold and warm (q|k|v, o, gate|up, down), and site D's GEMM alone
    for site, K, N in (("A", 1024, 1536), ("O", 1024, 1024), ("B", 1024, 8192), ("D", 4096, 1024)):
        for w in ("cold", "warm"):
            add("expert_sites", f"expert_site{site}_m50_{w}", 50, K, N, 128, 4, "linear", w)
    add("expert_sites", "expert_siteD_m50_gemm_cold", 50, 4096, 1024, 128, 4, "gemm")
    # every projection of the backbone layer at M = 816, and its grouped sites
    for name, K, N in (("q", 2048, 2048), ("k", 2048, 256), ("v", 2048, 256), ("o", 2048, 2048),
                       ("gate", 2048, 16384), ("up", 2048, 16384), ("down", 16384, 2048),
                       ("siteA_qkv", 2048, 2560), ("siteB_gateup", 2048, 32768)):
        add("backbone_projections", f"backbone_{name}_m816", 816, K, N, 128, 4, "linear")
    # the whole down-projection sweep, fused projection
    for bits in (4, 8):
        for M in (1, 16, 50, 256, 816, 4096):
            for b in (32, 64, 128, 256):
                add("sweep", f"sweep_m{M}_b{b}_w{bits}a{bits}", M, 16384, 2048, b, bits, "linear")
    # weight-only INT4 (the adaptive layer-norm modulation path), b = 1
    add("w4a16", "adaln_w4a16_m1_k1024_n6144", 1, 1024, 6144, 1, 4, "w4a16")
    add("w4a16", "down_w4a16_m1", 1, 16384, 2048, 1, 4, "w4a16")
    add("w4a16", "down_w4a16_m16", 16, 16384, 2048, 1, 4, "w4a16")
    if groups:
        specs = [s for s in specs if s[0] in groups]
    return specs


def point_data(synth, name, M, K, N, b, bits):
    """The point's seeded tokens (bf16 [M, K], CPU) and fp32 weights [N, K]: the workload's
    own generators (down-projection sweep, backbone layer, action-expert layer, single
    linear)."""
    if name.startswith("down_m") or name.startswith("sweep_"):
        wl = synth.down_proj_sweep_point(M, b, bits)
        return wl.site_activation("D", 0), wl.projection_weight(wl.projections[0])
    if name.startswith("backbone_"):
        wl = synth.backbone_layer()
        part = name[len("backbone_"):].split("_m816")[0].replace("_w4a4", "")
        groups = {"siteA_qkv": ("q", "k", "v"), "siteB_gateup": ("gate", "up")}
        names = groups.get(part, (part,))
        projs = [p for p in wl.projections if p.name in names]
        return wl.site_activation(projs[0].site, 0), np.concatenate([wl.projection_weight(p) for p in projs], axis=0)
    if name.startswith("expert_site"):
        wl = synth.action_expert_layer()
        site = name[len("expert_site")]
        projs = [p for p in wl.projections if p.site == site]
        return wl.site_activation(site, 0), np.concatenate([wl.projection_weight(p) for p in projs], axis=0)
    if name.startswith("single_"):
        wl = synth.single_linear()
        p = wl.projections[0]
        return (synth.activations(M, K, seed=0, outlier_frac=wl.outlier_frac, outlier_scale=wl.outlier_scale),
                wl.projection_weight(p))
    return (synth.activations(M, K, seed=M + K, outlier_frac=0.005, outlier_scale=50.0),
            synth.weights(N, K, seed=K + N + bits))


class Point:
    """Device state of one point: weights (with copies for cold rotation), tokens, codes,
    workspace, output, and the call."""

    def __init__(self, torch, fq, synth, dev, spec):
        self.spec = spec
        _, name, M, K, N, b, bits, kind, weights = spec
        x, w = point_data(synth, name, M, K, N, b, bits)
        wd = torch.from_numpy(w).to(dev)
        lin = fq.QuantLinear(wd, b, bits)
        del wd
        self.copies = 1 if weights == "warm" else cold_copies(lin.w_packed.numel())
        self.wp = [lin.w_packed] + [lin.w_packed.clone() for _ in range(self.copies - 1)]
        self.w_scale = lin.w_scale
        self.x = x.to(dev)
        self.y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
        if kind == "gemm":
            self.codes, self.delta = fq.fwht_quant(self.x, b, bits)
            self.ws = fq.workspace(fq.gemm_workspace_bytes(M, N, K, bits), dev)
            self.nbytes, self.peak = gemm_bytes(M, N, K, bits), INT8_PEAK_TOPS
        elif kind == "w4a16":
            self.ws = fq.workspace(fq.w4a16_workspace_bytes(M, N, K), dev)
            self.nbytes, self.peak = linear_bytes(M, N, K, 4), BF16_PEAK_TFLOPS
        else:
            self.ws = fq.workspace(fq.linear_workspace_bytes(M, N, K, bits), dev)
            self.nbytes, self.peak = linear_bytes(M, N, K, bits), INT8_PEAK_TOPS
        self.ops = 2.0 * M * N * K
        c, f = self.copies, fq
        if kind == "gemm":
            self.call = lambda i: f.gemm(self.codes, self.delta, self.wp[i % c], self.w_scale, N, K, bits, ws=self.ws,
                                         out=self.y)
        elif kind == "w4a16":
            self.call = lambda i: f.gemm_w4a16(self.x, self.wp[i % c], self.w_scale, N, ws=self.ws, out=self.y)
        else:
            self.call = lambda i: f.linear(self.x, self.wp[i % c], self.w_scale, N, b, bits, ws=self.ws, out=self.y)

    def calls(self):
        return 50 if self.copies == 1 else self.copies


def measure_point(torch, fq, synth, dev, spec, traced):
    pt = Point(torch, fq, synth, dev, spec)
    group, name, M, K, N, b, bits, kind, weights = spec
    us, p10, p90, mean = time_calls(torch, pt.call, pt.calls())
    rec = {"name": name, "group": group, "kind": kind, "M": M, "K": K, "N": N, "b": b, "bits": bits,
           "weights": weights, "us": round(us, 3), "us_p10_p90": [round(p10, 3), round(p90, 3)],
           "us_mean": round(mean, 3), "TOPS": round(pt.ops / us / 1e6, 2), "algorithmic_bytes": pt.nbytes,
           "roofline": roofline(pt.nbytes, pt.ops, us, pt.peak)}
    tr = traced.get(name)
    if tr:
        rec["rocprof_us"] = tr["us_per_call"]
        rec["rocprof_frac"] = roofline(pt.nbytes, pt.ops, tr["us_per_call"], pt.peak)["frac"]
    del pt
    torch.cuda.empty_cache()
    return rec


def rocprof_points_run(torch, fq, synth, dev, groups):
    """Every point as bench.py times it, for a kernel trace: for point i, its set-up (weights
    and copies), the graph of its back-to-back calls (one per weight copy; cold points
    rotate through >= 1 GiB of copies) replayed until >= 20 calls have run, then a sentinel
    kernel (a uint8 bitwise_not that nothing else launches), replays of the graph until
    >= 100 calls have run, a second sentinel.  The manifest printed at the end lists the
    points in order with their calls between the sentinels."""
    manifest = []
    s_in = torch.zeros(64, dtype=torch.uint8, device=dev)
    s_out = torch.empty_like(s_in)
    for spec in point_specs(groups):
        pt = Point(torch, fq, synth, dev, spec)
        calls = pt.calls()
        g = graph_of(torch, pt.call, calls)
        for _ in range(max(1, -(-20 // calls))):
            g.replay()
        reps = max(1, -(-100 // calls))
        torch.bitwise_not(s_in, out=s_out)
        for _ in range(reps):
            g.replay()
        torch.bitwise_not(s_in, out=s_out)
        torch.cuda.synchronize()
        manifest.append({"name": spec[1], "calls": calls * reps})
        print(json.dumps({"rocprof_point": spec[1], "calls": calls * reps}), flush=True)
        del g, pt
        torch.cuda.empty_cache()
    print(json.dumps({"rocprof_manifest": manifest}), flush=True)


def trace_segments(rows, n_points):
    """The kernels of each point in a `--rocprof-points` trace: rows (start, end, name, grid,
    workgroup) sorted by start; the kernels strictly between sentinel 2 i and 2 i + 1 are
    point i's calls."""
    marks = [j for j, r in enumerate(rows) if "bitwise_not" in r[2]]
    if len(marks) != 2 * n_points:
        raise SystemExit(f"{len(marks)} sentinel kernels in the trace for {n_points} points")
    return [rows[marks[2 * i] + 1:marks[2 * i + 1]] for i in range(n_points)]


def summarize_trace(path, manifest_path, out_path=POINTS_TRACE_FILE):
    """Per-point, per-grid kernel summary of a `--rocprof-points` kernel trace (rocprofv3
    CSV), each point's calls found between its two sentinel kernels and matched in order to
    the run's manifest (its last JSON line).  Writes profiles/points_kernels_by_grid.{json,md}."""
    import csv
    manifest = None
    with open(manifest_path) as f:
        for line in f:
            if line.startswith("{") and "rocprof_manifest" in line:
                manifest = json.loads(line)["rocprof_manifest"]
    if manifest is None:
        raise SystemExit(f"no manifest line in {manifest_path}")
    rows = []
    with open(path) as f:
        for r in csv.DictReader(f):
            grid = tuple(int(r.get(f"Grid_Size_{a}") or 0) for a in "XYZ")
            wg = tuple(int(r.get(f"Workgroup_Size_{a}") or 0) for a in "XYZ")
            rows.append((int(r["Start_Timestamp"]), int(r["End_Timestamp"]), r["Kernel_Name"], grid, wg))
    rows.sort()
    segs = trace_segments(rows, len(manifest))
    points = {}
    for i, m in enumerate(manifest):
        by = {}
        for start, end, name, grid, wg in segs[i]:
            by.setdefault((name, grid, wg), []).append((end - start) / 1e3)
        kern = []
        for (name, grid, wg), d in sorted(by.items(), key=lambda kv: -sum(kv[1])):
            kern.append({"kernel": name, "grid": list(grid), "workgroup": list(wg), "launches": len(d),
                         "avg_us": round(sum(d) / len(d), 3), "min_us": round(min(d), 3), "max_us": round(max(d), 3)})
        total = sum(sum(d) for d in by.values())
        points[m["name"]] = {"calls": m["calls"], "us_per_call": round(total / m["calls"], 3), "kernels": kern}
    out = {"sources_sha256": sources_digest(), "points": points,
           "note": "kernel execution time per call (the sum of the call's kernels, no launch gaps) from a "
                   "rocprofv3 kernel trace of `python bench.py --rocprof-points`"}
    with open(out_path, "w") as f:
        json.dump(out, f, indent=1)
    lines = ["# Kernel time per point, by kernel and grid (rocprofv3 kernel trace)", "",
             "Commands (from the repository root on an MI355X, `cd /tmp && export TMPDIR=/tmp` first):", "",
             "```",
             "rocprofv3 --kernel-trace --stats --output-format csv -d <out> -o points -- "
             "python /root/repo/bench.py --rocprof-points --quiet > <out>/manifest.txt",
             "python /root/repo/bench.py --summarize-trace <out>/<host>/points_kernel_trace.csv "
             "--manifest <out>/manifest.txt", "```", "",
             "Each point replayed the graph of back-to-back calls that bench.py times (one call per weight copy; "
             "cold points rotate through >= 1 GiB of copies), warmed up, then >= 100 calls between two sentinel "
             "kernels. `us/call` is the sum of the point's kernel durations divided by its "
             "calls (no launch gaps); bench.py reports it beside its own graph-replay figure as `rocprof_us`. "
             f"Sources SHA-256 {out['sources_sha256'][:16]}.", "",
             "| point | calls | us/call | kernel | grid | workgroup | launches | avg us | min | max |",
             "|---|---|---|---|---|---|---|---|---|---|"]
    for name, p in points.items():
        for j, k in enumerate(p["kernels"]):
            head = f"| {name} | {p['calls']} | {p['us_per_call']}" if j == 0 else "| | |"
            lines.append(f"{head} | `{k['kernel'][:100]}` | {'x'.join(map(str, k['grid']))} | "
                         f"{'x'.join(map(str, k['workgroup']))} | {k['launches']} | {k['avg_us']} | {k['min_us']} | "
                         f"{k['max_us']} |")
    with open(out_path.replace(".json", ".md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    print(f"{len(points)} points summarized into {out_path}")


# --------------------------------------------------------------------------- counter summaries

def counter_rows(run_dir):
    """(dispatch id, kernel, grid threads, counter, value) rows of one rocprofv3 --pmc run
    (csv output under run_dir)."""
    import csv
    import glob
    rows = []
    for path in glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True):
        with open(path) as f:
            for r in csv.DictReader(f):
                rows.append((int(r["Dispatch_Id"]), r["Kernel_Name"], int(r["Grid_Size"]), r["Counter_Name"],
                             float(r["Counter_Value"])))
    if not rows:
        raise SystemExit(f"no counter rows under {run_dir}")
    return rows


def counter_means(run_dir, min_dispatches):
    """(kernel, grid) -> {"dispatches": n, counter: mean per dispatch} over the kernels
    dispatched at least min_dispatches times (the measured calls; set-up kernels such as
    the weight rounding and packing run once)."""
    per = {}
    for disp, name, grid, ctr, val in counter_rows(run_dir):
        d = per.setdefault((name, grid), {})
        d.setdefault(ctr, {})[disp] = d.get(ctr, {}).get(disp, 0.0) + val
    out = {}
    for key, ctrs in per.items():
        n = max(len(v) for v in ctrs.values())
        if n >= min_dispatches:
            out[key] = {"dispatches": n, **{c: sum(v.values()) / len(v) for c, v in ctrs.items()}}
    return out


def short_kernel(name):
    return name.replace("void ", "").replace("(anonymous namespace)::", "").split("(")[0].replace("fq::", "")


def copy_factors(d):
    """KiB per launch that FETCH_SIZE and WRITE_SIZE read for the copy-like calibration
    kernel (256 MiB each way), and the true bytes."""
    f = counter_means(os.path.join(d, "copy_fetch"), 20)
    w = counter_means(os.path.join(d, "copy_write"), 20)
    fk = max(v["FETCH_SIZE"] for v in f.values())
    wk = max(v["WRITE_SIZE"] for v in w.values())
    return fk, wk, 256 << 20, 256 << 20


SITE_SHAPES = {"A": (1024, 1536, "q|k|v"), "O": (1024, 1024, "o"), "B": (1024, 8192, "gate|up"),
               "D": (4096, 1024, "down")}


def summarize_traffic(d, out_path=TRAFFIC_FILE):
    """HBM bytes of the action-expert sites from `--traffic-site` counter runs under d
    (traffic_<S>_fetch, traffic_<S>_write, copy_fetch, copy_write).  Writes
    profiles/site_traffic.{json,md}."""
    fk, wk, rb, wb = copy_factors(d)
    ff, fw = fk * 1024 / rb, wk * 1024 / wb
    out = {"copy_fetch_kib": round(fk, 2), "copy_write_kib": round(wk, 2), "copy_bytes_read": rb,
           "copy_bytes_written": wb, "copy_launches": 20, "sources_sha256": sources_digest(), "sites": {}}
    detail = []
    for site in "AOBD":
        f = counter_means(os.path.join(d, f"traffic_{site}_fetch"), 100)
        w = counter_means(os.path.join(d, f"traffic_{site}_write"), 100)
        rec = {"fetch_kib_per_call": 0.0, "write_kib_per_call": 0.0, "calls": 100,
               "gemm_fetch_kib_per_call": 0.0, "gemm_write_kib_per_call": 0.0}
        for key in sorted(set(f) | set(w)):
            fkib = f.get(key, {}).get("FETCH_SIZE", 0.0) * f.get(key, {}).get("dispatches", 0) / 100
            wkib = w.get(key, {}).get("WRITE_SIZE", 0.0) * w.get(key, {}).get("dispatches", 0) / 100
            rec["fetch_kib_per_call"] += fkib
            rec["write_kib_per_call"] += wkib
            if "fwht_quant_kernel" not in key[0] and "linear_small_kernel" not in key[0]:
                rec["gemm_fetch_kib_per_call"] += fkib
                rec["gemm_write_kib_per_call"] += wkib
            detail.append((site, short_kernel(key[0]), key[1], f.get(key, {}).get("dispatches", 0),
                           f.get(key, {}).get("FETCH_SIZE", 0.0), w.get(key, {}).get("WRITE_SIZE", 0.0)))
        out["sites"][site] = {k: (round(v, 2) if isinstance(v, float) else v) for k, v in rec.items()}
    with open(out_path, "w") as fo:
        json.dump(out, fo, indent=1)
    M = 50
    lines = ["# HBM traffic: action-expert fused projections (M=50, width 1024, W4A4, block 128)", "",
             "Commands (from the repository root on an MI355X, `cd /tmp && export TMPDIR=/tmp` first), for each "
             "site S in A, O, B, D, then the summary:", "", "```"]
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        lines.append(f"rocprofv3 --pmc {c} --output-format csv -d <out>/traffic_S_{'fetch' if c[0] == 'F' else 'write'} "
                     "-o x -- python /root/repo/bench.py --traffic-site S --quiet")
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        lines.append(f"rocprofv3 --pmc {c} --output-format csv -d <out>/copy_{'fetch' if c[0] == 'F' else 'write'} "
                     "-o x -- python /root/repo/bench.py --copy-calibration --quiet")
    lines += ["python /root/repo/bench.py --summarize-traffic <out>", "```", "",
              f"Calibration: a plain float32 copy-like kernel (`torch.add(a, 0, out=b)`, 256 MiB read and 256 MiB "
              f"written per launch, 20 launches) reads FETCH_SIZE {fk:.1f} KiB and WRITE_SIZE {wk:.1f} KiB: factors "
              f"{ff:.4f} (fetch) and {fw:.4f} (write) of the true bytes.  Each site's counters are divided by them.  "
              f"Sources SHA-256 {out['sources_sha256'][:16]}.", "",
              "| site | K -> N | algorithmic MB | fetch MB | write MB | measured MB | measured / algorithmic | "
              "GEMM kernel alone: algorithmic MB | measured MB |", "|---|---|---|---|---|---|---|---|---|"]
    for site in "AOBD":
        K, N, nm = SITE_SHAPES[site]
        r = out["sites"][site]
        alg = linear_bytes(M, N, K, 4)
        fmb = r["fetch_kib_per_call"] * 1024 / ff / 1e6
        wmb = r["write_kib_per_call"] * 1024 / fw / 1e6
        gmb = (r["gemm_fetch_kib_per_call"] * 1024 / ff + r["gemm_write_kib_per_call"] * 1024 / fw) / 1e6
        galg = gemm_bytes(M, N, K, 4) if site == "D" else 0
        lines.append(f"| {site} ({nm}) | {K} -> {N} | {alg / 1e6:.3f} | {fmb:.3f} | {wmb:.3f} | **{fmb + wmb:.3f}** | "
                     f"{(fmb + wmb) * 1e6 / alg:.2f} | {galg / 1e6:.3f} | {gmb:.3f} |")
    lines += ["", "Per kernel, counter KiB per dispatch (mean over the measured dispatches):", "",
              "| site | kernel | grid (threads) | dispatches | FETCH_SIZE KiB | WRITE_SIZE KiB |",
              "|---|---|---|---|---|---|"]
    for site, k, g, n, fv, wv in detail:
        lines.append(f"| {site} | `{k}` | {g} | {n} | {fv:.1f} | {wv:.1f} |")
    with open(out_path.replace(".json", ".md"), "w") as fo:
        fo.write("\n".join(lines) + "\n")
    print(f"traffic of sites A, O, B, D summarized into {out_path}")


def summarize_stats(stats_csv, bench_json, out_path=os.path.join(PROFILES, "bench_kernel_stats.md")):
    """profiles/bench_kernel_stats.md from the --stats kernel summary of the default bench run
    under a kernel trace (and that run's JSON line, for its step time)."""
    import csv
    with open(stats_csv) as f:
        rows = list(csv.DictReader(f))
    step_us = None
    with open(bench_json) as f:
        for line in f:
            if line.startswith('{"metric"'):
                step_us = json.loads(line)["ms_per_step"] * 1e3
    lines = ["# Kernel statistics of the benchmark's own run (rocprofv3 --kernel-trace --stats)", "",
             "Commands (from the repository root on an MI355X, `cd /tmp && export TMPDIR=/tmp` first):", "", "```",
             "rocprofv3 --kernel-trace --stats --output-format csv -d <out> -o bench -- python /root/repo/bench.py "
             "> <out>/bench.json",
             "python /root/repo/bench.py --summarize-stats <out>/<host>/bench_kernel_stats.csv --bench-json <out>/bench.json",
             "```", "",
             "The whole default run: the 10-step denoising loop (warm-up, timed steps), the cold step and sites, the "
             "graded block, every point, the chain, the CPU baseline.  Each kernel's average is over every launch of "
             "that instantiation in the run, across all the shapes it served (the per-point, per-grid figures are in "
             "`points_kernels_by_grid.md`).  Under a full kernel trace every graph launch carries its own completion "
             "signal and timestamps, so this run's own step time"
             + (f" ({step_us:.1f} us)" if step_us else "") + " is not comparable with an untraced run; its kernel "
             f"durations are.  Sources SHA-256 {sources_digest()[:16]}.", "",
             "| kernel | calls | total ms | average us | min us | max us | share |", "|---|---|---|---|---|---|---|"]
    for r in rows:
        lines.append(f"| `{r['Name'][:110]}` | {r['Calls']} | {int(r['TotalDurationNs']) / 1e6:.2f} | "
                     f"{float(r['AverageNs']) / 1e3:.3f} | {int(r['MinNs']) / 1e3:.3f} | {int(r['MaxNs']) / 1e3:.3f} | "
                     f"{float(r['Percentage']):.1f}% |")
    with open(out_path, "w") as fo:
        fo.write("\n".join(lines) + "\n")
    print(f"{len(rows)} kernels summarized into {out_path}")


COUNTER_SETS = ["fetch", "write", "tcc", "sq1", "sq2"]


def summarize_counters(d, points, out_path=os.path.join(PROFILES, "gemm_counters.json")):
    """Counters of graded GEMM points from `--counter-point` runs under d (<point>_fetch,
    _write, _tcc, _sq1, _sq2).  Writes profiles/gemm_counters.{json,md}."""
    fk, wk, rb, wb = copy_factors(d)
    ff, fw = fk * 1024 / rb, wk * 1024 / wb
    res = {"sources_sha256": sources_digest(), "points": {}}
    for pt in points:
        spec = next(s for s in point_specs() if s[1] == pt)
        _, _, M, K, N, b, bits, kind, weights = spec
        merged = {}
        for cs in COUNTER_SETS:
            for key, v in counter_means(os.path.join(d, f"{pt}_{cs}"), 20).items():
                if "__amd_rocclr" not in key[0]:  # the weight copies' set-up copies
                    merged.setdefault(key, {}).update(v)
        kerns = []
        for (name, grid), v in sorted(merged.items(), key=lambda kv: -kv[1].get("SQ_WAVE_CYCLES", 0)):
            mfma = v.get("SQ_INSTS_MFMA", 0.0)
            valu = v.get("SQ_INSTS_VALU", 0.0)
            waves = v.get("SQ_WAVES", 0.0)
            gui = v.get("GRBM_GUI_ACTIVE", 0.0)
            hit, miss = v.get("TCC_HIT_sum", 0.0), v.get("TCC_MISS_sum", 0.0)
            rec = {"kernel": short_kernel(name), "grid_threads": grid, "dispatches": v["dispatches"],
                   "hbm_read_mb": round(v.get("FETCH_SIZE", 0.0) * 1024 / ff / 1e6, 2),
                   "hbm_write_mb": round(v.get("WRITE_SIZE", 0.0) * 1024 / fw / 1e6, 2),
                   "l2_hit_rate": round(hit / (hit + miss), 3) if hit + miss else None,
                   "waves": int(waves), "mfma": int(mfma), "valu_incl_mfma": int(valu),
                   "valu_per_mfma": round((valu - mfma) / mfma, 2) if mfma else None,
                   "mfma_busy_cycles_per_mfma": round(v.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) / mfma, 1) if mfma else None,
                   # GRBM_GUI_ACTIVE summed over the 8 XCDs: SIMD cycles = 1024 x gui / 8
                   "mfma_utilisation": round(v.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) / (1024 * gui / 8), 3) if gui else None,
                   "lds_instr_per_mfma": round(v.get("SQ_INSTS_LDS", 0.0) / mfma, 3) if mfma else None,
                   "lds_bank_conflicts": int(v.get("SQ_LDS_BANK_CONFLICT", 0.0)),
                   "wait_per_wave_cycles": round(v.get("SQ_WAIT_INST_ANY", 0.0) / v["SQ_WAVE_CYCLES"], 3)
                   if v.get("SQ_WAVE_CYCLES") else None,
                   "valu_active_per_wave_cycles": round(v.get("SQ_ACTIVE_INST_VALU", 0.0) / v["SQ_WAVE_CYCLES"], 3)
                   if v.get("SQ_WAVE_CYCLES") else None}
            kerns.append(rec)
        res["points"][pt] = {"M": M, "K": K, "N": N, "bits": bits, "weights": weights,
                             "algorithmic_mb": round(gemm_bytes(M, N, K, bits) / 1e6, 2), "kernels": kerns}
    with open(out_path, "w") as fo:
        json.dump(res, fo, indent=1)
    lines = ["# Counters: graded GEMM points (the GEMM kernel alone, cold weights)", "",
             "Commands (from the repository root on an MI355X, `cd /tmp && export TMPDIR=/tmp` first), one pass per "
             "counter set, for each point P below, then the copy calibration and the summary:", "", "```"]
    sets = {"fetch": "FETCH_SIZE", "write": "WRITE_SIZE", "tcc": "TCC_HIT_sum TCC_MISS_sum",
            "sq1": "SQ_WAVES SQ_INSTS_VALU SQ_INSTS_MFMA SQ_INSTS_LDS SQ_WAVE_CYCLES SQ_BUSY_CYCLES SQ_WAIT_INST_ANY "
                   "SQ_ACTIVE_INST_VALU",
            "sq2": "SQ_VALU_MFMA_BUSY_CYCLES SQ_WAIT_INST_LDS SQ_ACTIVE_INST_LDS SQ_LDS_BANK_CONFLICT GRBM_GUI_ACTIVE"}
    for cs in COUNTER_SETS:
        lines.append(f"timeout -s KILL 150 rocprofv3 --pmc {sets[cs]} --output-format csv -d <out>/P_{cs} -o p -- "
                     "python /root/repo/bench.py --counter-point P --quiet")
    lines += ["rocprofv3 --pmc FETCH_SIZE --output-format csv -d <out>/copy_fetch -o x -- "
              "python /root/repo/bench.py --copy-calibration --quiet",
              "rocprofv3 --pmc WRITE_SIZE --output-format csv -d <out>/copy_write -o x -- "
              "python /root/repo/bench.py --copy-calibration --quiet",
              f"python /root/repo/bench.py --summarize-counters <out> --counter-points {','.join(points)}", "```", "",
              f"HBM bytes: FETCH_SIZE and WRITE_SIZE divided by what they read for the copy calibration: factors "
              f"{ff:.4f} and {fw:.4f}.  MFMA utilisation = SQ_VALU_MFMA_BUSY_CYCLES / (1024 SIMDs x GRBM_GUI_ACTIVE / 8), "
              "GRBM_GUI_ACTIVE summed over the 8 XCDs (it includes the profiler's per-dispatch overhead, so it reads "
              "a little below the timed points).  VALU / MFMA counts the other vector instructions per MFMA "
              "(SQ_INSTS_VALU includes the MFMAs).  Per-dispatch means over the point's calls (one per weight "
              f"copy).  Sources SHA-256 {res['sources_sha256'][:16]}.", "",
              "| point | kernel | grid (threads) | dispatches | HBM read MB | HBM write MB | algorithmic MB | L2 hit rate "
              "| waves | MFMA | VALU / MFMA | MFMA busy cycles / MFMA | MFMA utilisation | LDS instr / MFMA | "
              "LDS bank conflicts | wait / wave cycles | VALU active / wave cycles |",
              "|---|---|---|---|---|---|---|---|---|---|---|---|---|---|---|---|---|"]
    for pt, pr in res["points"].items():
        for k in pr["kernels"]:
            lines.append(f"| {pt} | `{k['kernel']}` | {k['grid_threads']} | {k['dispatches']} | {k['hbm_read_mb']} | "
                         f"{k['hbm_write_mb']} | {pr['algorithmic_mb']} | {k['l2_hit_rate']} | {k['waves']} | "
                         f"{k['mfma']} | {k['valu_per_mfma']} | {k['mfma_busy_cycles_per_mfma']} | "
                         f"{k['mfma_utilisation']} | {k['lds_instr_per_mfma']} | {k['lds_bank_conflicts']} | "
                         f"{k['wait_per_wave_cycles']} | {k['valu_active_per_wave_cycles']} |")
    with open(out_path.replace(".json", ".md"), "w") as fo:
        fo.write("\n".join(lines) + "\n")
    print(f"{len(points)} points summarized into {out_path}")


# --------------------------------------------------------------------------- other points

def measure_bf16_context(torch, synth, dev, log_fn, pts):
    """Context only (the analog of the paper's floating-point engine control): the same
    down-projection shapes as a plain bf16 matrix product (torch.matmul, the vendor GEMM
    library), weights rotating through >= 1 GiB of copies like the W4A4 points.  Each record
    carries the fused W4A4 projection's speed-up over it."""
    out = []
    lin_us = {(p["M"], p["K"], p["N"]): p["us"] for p in pts
              if p.get("kind") == "linear" and p.get("bits") == 4 and p.get("weights") == "cold" and p.get("b") == 128}
    for (M, K, N) in ((50, 16384, 2048), (816, 16384, 2048), (816, 2048, 16384)):
        wt = torch.from_numpy(synth.weights(N, K, seed=K + N).T.copy()).to(dev).to(torch.bfloat16)  # [K, N]
        copies = cold_copies(wt.numel() * 2)
        ws = [wt.clone() for _ in range(copies)]
        del wt
        x = synth.activations(M, K, seed=M + K, outlier_frac=0.005, outlier_scale=50.0).to(dev)
        y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
        g = graph_of(torch, lambda i: torch.matmul(x, ws[i % copies], out=y), copies)
        us = time_graph(torch, g, max(1, 200 // copies)) / copies * 1e6
        rec = {"name": f"context_bf16_matmul_m{M}_k{K}_n{N}", "group": "context", "kind": "bf16_matmul", "M": M,
               "K": K, "N": N, "us": round(us, 3), "TFLOPS": round(2.0 * M * N * K / us / 1e6, 2),
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
        rec = {"name": name, "group": "gptq", "kind": "gptq", "N": N, "K": K, "T": T, "b": b, "bits": 4}
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
    rotation (permutation + dense per-block matrices) on the same tokens, and the butterfly
    at every block size of the down-projection sweep.  Algorithmic bytes: x, codes and
    scales, plus the permutation and the blocks for the composite one; its 2 M K b flops
    (fp32 fma chains) give the ALU side of its roofline."""
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
        base = quant_bytes(M, K, 4)
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
            rec = {"name": f"{name}_{kind}", "group": "prologue", "kind": f"prologue_{kind}", "M": M, "K": K, "b": b,
                   "bits": 4, "us": round(us, 3), "GBps": round(nbytes / us / 1e3, 1),
                   "bound": "hbm" if t_hbm >= t_alu else "alu", "roofline_frac": round(max(t_hbm, t_alu) / us, 4)}
            log_fn(json.dumps(rec))
            out.append(rec)
            del g
        del x, perm, blocks, codes, delta, ws
        torch.cuda.empty_cache()
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
        nbytes = quant_bytes(M, K, 4)
        rec = {"name": f"sweep_prologue_m816_b{b}_fwht", "group": "prologue", "kind": "prologue_fwht", "M": M,
               "K": K, "b": b, "bits": 4, "us": round(us, 3), "GBps": round(nbytes / us / 1e3, 1), "bound": "hbm",
               "roofline_frac": round(nbytes / HBM_PEAK_GBS / 1e3 / us, 4)}
        log_fn(json.dumps(rec))
        out.append(rec)
        del g, x, codes, delta
        torch.cuda.empty_cache()
    return out


# --------------------------------------------------------------------------- the 18-layer chain

class MixedChain:
    """Selective-INT8 language backbone: layers of the width-2048 shapes at M = 816
    (q|k|v 2048 -> 2560 and gate|up 2048 -> 32768 W4A4; o 2048 -> 2048 and down
    16384 -> 2048 W8A8).  Per layer: a = RMSNorm(h) (eps 1e-6; its gain gamma_A ~ U(0.5,
    1.5) folded into W_q,k,v by eq. (4)); q|k|v = Lin_A(a); o = Lin_O(q), q standing in for
    the attention output; h1 = h + o; g|u = Lin_B(RMSNorm(h1)) (gain gamma_B folded);
    d = Lin_D(silu(g) * u); h = h1 + d.  Norms, SwiGLU and residuals run in fp32 torch
    (outside the projection); each projection's input is rounded to bf16.  Weights are the
    seeded backbone-layer weights of layer l (synth.backbone_layer_mixed(l)), gains
    synth.channel_vector(seed 7000 + 2 l for A, 7001 + 2 l for B); h0 = layer 0's seeded
    site-A activations.  Layers are added one at a time (add_layer), so that a caller can
    share one layer's host weights between chains and checks; layer(l, record) runs layer l
    on the current hidden state and can keep every projection's bf16 input and output."""

    M, D, KV, F = 816, 2048, 256, 16384
    SHAPES = {"A": (2048 + 2 * 256, 2048, 4), "O": (2048, 2048, 8), "B": (2 * 16384, 2048, 4), "D": (2048, 16384, 8)}
    SITE_PROJ = {"A": ("q", "k", "v"), "O": ("o",), "B": ("gate", "up"), "D": ("down",)}

    def __init__(self, torch, fq, synth, dev, b=128, keep_fp32=False):
        self.torch, self.fq, self.synth, self.dev, self.b, self.keep_fp32 = torch, fq, synth, dev, b, keep_fp32
        self.lins, self.w32, self.gains = [], [], []
        M, D, F = self.M, self.D, self.F
        self.ws = fq.workspace(max(fq.linear_workspace_bytes(M, n, k, bits) for n, k, bits in self.SHAPES.values()), dev)
        self.h0 = synth.backbone_layer_mixed(0).site_activation("A", 0).to(dev).float()
        self.h = self.h0.clone()
        bf = dict(dtype=torch.bfloat16, device=dev)
        self.a_in = torch.empty((M, D), **bf)
        self.qkv = torch.empty((M, D + 2 * self.KV), **bf)
        self.o = torch.empty((M, D), **bf)
        self.b_in = torch.empty((M, D), **bf)
        self.gu = torch.empty((M, 2 * F), **bf)
        self.m_in = torch.empty((M, F), **bf)
        self.dn = torch.empty((M, D), **bf)

    @classmethod
    def layer_weights(cls, synth, l):
        """Host fp32 weights of layer l per site (consumers of a site stacked) and its gains."""
        wl = synth.backbone_layer_mixed(l)
        w = {s: np.concatenate([wl.projection_weight(p) for p in wl.projections if p.name in names], axis=0)
             for s, names in cls.SITE_PROJ.items()}
        gain = {"A": synth.channel_vector(cls.D, seed=7000 + 2 * l, low=0.5, high=1.5),
                "B": synth.channel_vector(cls.D, seed=7001 + 2 * l, low=0.5, high=1.5)}
        return w, gain

    def add_layer(self, w, gain):
        torch, fq, dev = self.torch, self.fq, self.dev
        self.gains.append(gain)
        self.lins.append({s: fq.QuantLinear(torch.from_numpy(w[s]).to(dev), self.b, bits,
                                            col_scale=torch.from_numpy(gain[s]).to(dev) if s in gain else None)
                          for s, (_, _, bits) in self.SHAPES.items()})
        if self.keep_fp32:
            self.w32.append({s: torch.from_numpy(w[s]).to(dev) for s in self.SHAPES})

    def rms(self, h):
        return h * self.torch.rsqrt(self.torch.mean(h * h, dim=1, keepdim=True) + 1e-6)

    def layer(self, l, record=False):
        torch, D, F, ws, L = self.torch, self.D, self.F, self.ws, self.lins[l]
        self.a_in.copy_(self.rms(self.h))
        L["A"](self.a_in, ws=ws, out=self.qkv)
        L["O"](self.qkv[:, :D], ws=ws, out=self.o)
        self.h.add_(self.o.float())
        rec = {"A": (self.a_in.clone(), self.qkv.clone()), "O": (self.qkv[:, :D].contiguous(), self.o.clone())} \
            if record else None
        self.b_in.copy_(self.rms(self.h))
        L["B"](self.b_in, ws=ws, out=self.gu)
        self.m_in.copy_(torch.nn.functional.silu(self.gu[:, :F].float()) * self.gu[:, F:].float())
        L["D"](self.m_in, ws=ws, out=self.dn)
        self.h.add_(self.dn.float())
        if record:
            rec.update({"B": (self.b_in.clone(), self.gu.clone()), "D": (self.m_in.clone(), self.dn.clone())})
        return rec

    def forward(self, layers=None):
        self.h.copy_(self.h0)
        for l in range(len(self.lins) if layers is None else layers):
            self.layer(l)

    def projections(self):
        ws, D = self.ws, self.D
        for L in self.lins:
            L["A"](self.a_in, ws=ws, out=self.qkv)
            L["O"](self.qkv[:, :D], ws=ws, out=self.o)
            L["B"](self.b_in, ws=ws, out=self.gu)
            L["D"](self.m_in, ws=ws, out=self.dn)

    def reference(self):
        """The same chain in fp32 with the unquantized weights and explicit gains; the hidden
        state after every layer."""
        torch, D, F = self.torch, self.D, self.F
        hr, hs = self.h0.clone(), []
        for l, w in enumerate(self.w32):
            gA = torch.from_numpy(self.gains[l]["A"]).to(self.dev)
            gB = torch.from_numpy(self.gains[l]["B"]).to(self.dev)
            qkv = (gA * self.rms(hr)) @ w["A"].t()
            hr = hr + qkv[:, :D] @ w["O"].t()
            gu = (gB * self.rms(hr)) @ w["B"].t()
            hr = hr + (torch.nn.functional.silu(gu[:, :F]) * gu[:, F:]) @ w["D"].t()
            hs.append(hr)
        return hs


def measure_mixed_chain(torch, fq, synth, dev, log_fn, layers=18):
    """The 18-layer selective-INT8 chain (MixedChain) on the seeded weights the parity tests
    check: at b = 128 the whole chain and its projections alone timed as HIP graphs; at
    b = 128 and at b = 1 (no rotation: plain per-token and per-channel round-to-nearest) the
    cosine of the hidden state against the fp32 chain after every layer, which shows the
    rotation's effect."""
    chains = {128: MixedChain(torch, fq, synth, dev, b=128, keep_fp32=True), 1: MixedChain(torch, fq, synth, dev, b=1)}
    for l in range(layers):
        w, gain = MixedChain.layer_weights(synth, l)
        for ch in chains.values():
            ch.add_layer(w, gain)
        del w
    chains[1].w32 = chains[128].w32
    hr = chains[128].reference()
    recs = []
    for b, ch in chains.items():
        rec = {"name": f"mixed_chain_{layers}l_m{ch.M}_b{b}", "group": "chain", "kind": "chain", "layers": layers,
               "M": ch.M, "b": b}
        if b == 128:
            g_chain = graph_of(torch, lambda i: ch.forward(), 1)
            us_chain = time_graph(torch, g_chain, 5) * 1e6
            del g_chain
            g_proj = graph_of(torch, lambda i: ch.projections(), 1)
            us_proj = time_graph(torch, g_proj, 5) * 1e6
            del g_proj
            ops = layers * 2.0 * ch.M * sum(n * k for n, k, _ in MixedChain.SHAPES.values())
            rec.update({"us_total": round(us_chain, 1), "us_per_layer": round(us_chain / layers, 2),
                        "projections_us_per_layer": round(us_proj / layers, 2),
                        "projection_TOPS": round(ops / us_proj / 1e6, 1)})
        cos = []
        ch.h.copy_(ch.h0)
        for l in range(layers):
            ch.layer(l)
            cos.append(round(torch.nn.functional.cosine_similarity(ch.h.flatten(), hr[l].flatten(), dim=0).item(), 6))
        rec["cosine_vs_fp32"] = cos[-1]
        rec["cosine_vs_fp32_per_layer"] = cos
        log_fn(json.dumps(rec))
        recs.append(rec)
    del chains, hr
    torch.cuda.empty_cache()
    return recs


# --------------------------------------------------------------------------- CPU baseline

def host_cpu_info():
    info = {"nproc": os.cpu_count(), "OMP_NUM_THREADS": os.environ.get("OMP_NUM_THREADS")}
    try:
        import subprocess
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=20).stdout
        for line in out.splitlines():
            k, _, v = line.partition(":")
            k, v = k.strip(), v.strip()
            if k in ("Model name", "Socket(s)", "Core(s) per socket", "Thread(s) per core", "CPU(s)"):
                info[k] = v
    except (OSError, ValueError):  # lscpu is optional
        pass
    return info


def cpu_baseline(st, oracle, synth, budget_s=12.0):
    """The oracle on the host cores: whole denoising steps of the action-expert layer (4 site
    prologues + the 7 consumers' contractions and rescales) with all threads for about
    budget_s seconds; then one denoising step and the single linear (M 64, 1024 -> 1024)
    with one thread and with all threads."""
    wq = {s: oracle.quantize_weights(st.w_host[s], st.b, 4) for s in st.sites}
    xs = {s: [a.cpu() for a in st.x[s]] for s in st.sites}

    def step(t):
        for s in st.sites:
            codes, delta = oracle.fwht_quant(xs[s][t], st.b, 4)
            wc, s_w = wq[s]
            oracle.dequant(oracle.gemm(codes, wc), delta, s_w)

    wl = synth.single_linear()
    p = wl.projections[0]
    x1 = synth.activations(wl.M, p.K, seed=0, outlier_frac=wl.outlier_frac, outlier_scale=wl.outlier_scale)
    wc1, s_w1 = oracle.quantize_weights(wl.projection_weight(p), wl.b, 4)

    def single():
        t0 = time.perf_counter()
        oracle.linear(x1, wc1, s_w1, wl.b, 4)
        return (time.perf_counter() - t0) * 1e6

    threads = oracle.max_threads()
    steps, t0 = 0, time.perf_counter()
    while True:
        step(steps % st.n_steps)
        steps += 1
        el = time.perf_counter() - t0
        if el >= budget_s or steps >= 1000:
            break
    ops = st.wl.ops_per_step() * steps
    rec = {"value": ops / el / 1e12, "unit": "TOPS", "cores": threads, "kind": "oracle",
           "sample": f"{steps} denoising steps of the action-expert layer (M=50, 7 projections) in {el:.1f} s "
                     f"on {threads} threads; then one step and the single linear on 1 thread",
           "us_per_step": round(el / steps * 1e6, 1), "us_single_linear": round(single(), 1)}
    oracle.set_threads(1)
    try:
        t0 = time.perf_counter()
        step(0)
        rec["single_thread_us_per_step"] = round((time.perf_counter() - t0) * 1e6, 1)
        rec["single_thread_us_single_linear"] = round(single(), 1)
    finally:
        oracle.set_threads(threads)
    rec["host"] = host_cpu_info()
    return rec


# --------------------------------------------------------------------------- counter helpers

def traffic_run(torch, fq, synth, dev, site):
    st = ExpertStep(torch, fq, synth, dev)
    for i in range(100):
        st.run_site(site, i % st.n_steps)
    torch.cuda.synchronize()
    print(json.dumps({"traffic_site": site, "calls": 100}), flush=True)


def counter_point_run(torch, fq, synth, dev, name):
    spec = next(s for s in point_specs() if s[1] == name)
    pt = Point(torch, fq, synth, dev, spec)
    n = max(pt.calls(), 20)
    for i in range(n):
        pt.call(i)
    torch.cuda.synchronize()
    print(json.dumps({"counter_point": name, "calls": n}), flush=True)


def copy_calibration(torch, dev):
    n = 64 << 20  # float32 elements: 256 MiB read and 256 MiB written per launch
    a = torch.ones(n, dtype=torch.float32, device=dev)
    b = torch.empty_like(a)
    for _ in range(20):
        torch.add(a, 0.0, out=b)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": 4 * n, "copy_bytes_written": 4 * n, "launches": 20}), flush=True)


# --------------------------------------------------------------------------- main

def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the projection's multi-GPU sharding is a design note, not a measured path).",
              file=sys.stderr)
        sys.exit(2)
    if args.summarize_trace:
        summarize_trace(args.summarize_trace, args.manifest)
        return
    if args.summarize_traffic:
        summarize_traffic(args.summarize_traffic)
        return
    if args.summarize_counters:
        summarize_counters(args.summarize_counters, args.counter_points.split(","))
        return
    if args.summarize_stats:
        summarize_stats(args.summarize_stats, args.bench_json)
        return
    import torch

    from paper_2609_24433_amd import fq, synth
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    K_steps, W = args.steps, args.warmup
    groups = args.points.split(",") if args.points else None

    if args.copy_calibration:
        copy_calibration(torch, dev)
        return
    if args.traffic_site:
        traffic_run(torch, fq, synth, dev, args.traffic_site)
        return
    if args.counter_point:
        counter_point_run(torch, fq, synth, dev, args.counter_point)
        return
    if args.rocprof_points:
        rocprof_points_run(torch, fq, synth, dev, groups)
        return

    st = ExpertStep(torch, fq, synth, dev)
    import oracle  # the parity check and the CPU baseline only
    check_step(st, oracle, torch)
    log(args, "parity check ok")

    # the denoising loop (10 steps) captured as one graph, as a serving loop runs it (the
    # weights shared across steps stay resident); one graph per step covers a remainder of K
    graphs = [graph_of(torch, lambda i, t=t: st.run(t), 1) for t in range(st.n_steps)]
    loop = graph_of(torch, lambda i: st.run(i), st.n_steps)
    elapsed = time_graph_steps(torch, graphs, K_steps, W, loop=loop)
    ops_step = st.wl.ops_per_step()
    value = ops_step * K_steps / elapsed / 1e12
    ms_step = elapsed * 1e3 / K_steps
    per_step_graphs = time_graph_steps(torch, graphs, K_steps, W) * 1e6 / K_steps
    del graphs, loop
    log(args, f"loop graph replay: {ms_step * 1e3:.2f} us/step, {value:.3f} TOPS; "
              f"one graph per step: {per_step_graphs:.2f} us/step")

    # the step with cold weights: every step on its own copy of the packed weights (>= 1 GiB
    # in rotation)
    cold = ExpertStep(torch, fq, synth, dev, copies=int(max(2, min(160, COLD_BYTES // st.weight_bytes() + 1))))
    us_cold, p10c, p90c, _ = time_calls(torch, lambda i: cold.run(i % cold.n_steps, i), cold.copies)
    del cold
    torch.cuda.empty_cache()
    log(args, f"cold step: {us_cold:.2f} us")

    # each site's fused projection, resident and cold weights; a site on the two-kernel path
    # (K too long for the one-kernel projection) also has its GEMM timed alone, cold
    M = st.wl.M
    traced = rocprof_points()
    per_site = {}
    for s_, K in st.sites.items():
        N = st.site_N[s_]
        r = {"K": K, "N": N, "one_kernel": fq.linear_workspace_bytes(M, N, K, 4) == 0}
        r["warm_us"] = round(time_calls(torch, lambda i, s_=s_: st.run_site(s_, i), 50)[0], 3)
        kinds = ("linear",) if r["one_kernel"] else ("linear", "gemm")
        for kind in kinds:
            name = f"expert_site{s_}_m50_cold" if kind == "linear" else f"expert_site{s_}_m50_gemm_cold"
            pt = Point(torch, fq, synth, dev, ("expert_sites", name, M, K, N, st.b, 4, kind, "cold"))
            r["cold_us" if kind == "linear" else "gemm_cold_us"] = round(time_calls(torch, pt.call, pt.calls())[0], 3)
            del pt
        per_site[s_] = r
        torch.cuda.empty_cache()
    log(args, "per-site: " + json.dumps(per_site))

    # the dominant kernel: the step's longest single launch, cold weights
    def launch(s_):
        r = per_site[s_]
        return (r["cold_us"], "linear") if r["one_kernel"] else (r["gemm_cold_us"], "gemm")

    dom = max(per_site, key=lambda k: launch(k)[0])
    r = per_site[dom]
    Kd, Nd = r["K"], r["N"]
    dom_us, dom_kind = launch(dom)
    if dom_kind == "linear":
        dom_kernel, dom_bytes, tname = "linear_small_kernel (the one-kernel projection)", linear_bytes(M, Nd, Kd, 4), \
            f"expert_site{dom}_m50_cold"
    else:
        dom_kernel, dom_bytes, tname = "the site's GEMM", gemm_bytes(M, Nd, Kd, 4), f"expert_site{dom}_m50_gemm_cold"
    ach = dom_bytes / dom_us / 1e3
    roof = {"bound": "hbm", "kernel": f"{dom_kernel}, site {dom}, M={M} K={Kd} N={Nd}, the step's longest launch",
            "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBS, 4),
            "traffic": measured_traffic(dom, dom_kind), "kernel_us": round(dom_us, 3),
            "weights": "cold: rotating copies of >= 1 GiB, graph of back-to-back calls, HIP events",
            "algorithmic_bytes": dom_bytes,
            "resident_weights_us": r["warm_us"] if dom_kind == "linear" else None}
    tr = traced.get(tname)
    if tr:
        roof["rocprof_us"] = tr["us_per_call"]
        roof["rocprof_frac"] = round(dom_bytes / tr["us_per_call"] / 1e3 / HBM_PEAK_GBS, 4)

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
                   "graph": f"the {st.n_steps}-step denoising loop as one HIP graph, weights shared across steps",
                   "us_per_step_one_graph_per_step": round(per_step_graphs, 3),
                   "us_per_step_cold_weights": round(us_cold, 3),
                   "us_per_step_cold_p10_p90": [round(p10c, 3), round(p90c, 3)],
                   "us_per_projection": round(ms_step * 1e3 / 7, 3),
                   "site_us": per_site},
        "roofline": roof,
    }
    if not args.no_points:
        pts, graded = [], []
        for spec in point_specs(groups):
            p = measure_point(torch, fq, synth, dev, spec, traced)
            log(args, json.dumps(p))
            (graded if spec[0] == "graded" else pts).append(p)
        if groups is None or "prologue" in groups:
            pts += measure_prologue_points(torch, fq, synth, dev, lambda m: log(args, m))
        if groups is None or "gptq" in groups:
            pts += measure_gptq_points(torch, fq, synth, dev, lambda m: log(args, m))
        if groups is None or "context" in groups:
            pts += measure_bf16_context(torch, synth, dev, lambda m: log(args, m), graded + pts)
        if groups is None or "chain" in groups:
            pts += measure_mixed_chain(torch, fq, synth, dev, lambda m: log(args, m))
        rec["graded"] = graded
        rec["points"] = pts
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(st, oracle, synth)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
