"""Host-side logic of bench.py (CPU): the timed region runs exactly K denoising steps,
whether whole loops are replayed as one graph or step by step; the algorithmic byte
counts the roofline divides by; `--gpus` above 1 is refused."""
import subprocess
import sys
import types

import pytest

import bench


class _Graph:
    def __init__(self, log, name, steps):
        self.log, self.name, self.steps = log, name, steps

    def replay(self):
        self.log.append((self.name, self.steps))


class _Event:
    def __init__(self, enable_timing=False):
        self.t = 0.0

    def record(self):
        pass

    def elapsed_time(self, other):
        return 1.0


def _fake_torch():
    cuda = types.SimpleNamespace(Event=_Event, synchronize=lambda: None)
    return types.SimpleNamespace(cuda=cuda)


@pytest.mark.parametrize("K,W", [(200, 20), (7, 3), (23, 10), (10, 0), (0, 5)])
@pytest.mark.parametrize("use_loop", [False, True])
def test_exactly_k_steps(K, W, use_loop):
    n = 10
    log = []
    steps = [_Graph(log, f"step{t}", 1) for t in range(n)]
    loop = _Graph(log, "loop", n) if use_loop else None
    bench.time_graph_steps(_fake_torch(), steps, K, W, loop=loop)
    total = sum(s for _, s in log)
    assert total == K + W
    if use_loop:
        # whole loops first, then the remainder's steps in order
        assert [name for name, _ in log].count("loop") == W // n + K // n


def test_byte_counts():
    M, N, K = 50, 8192, 1024
    assert bench.gemm_bytes(M, N, K, 4) == M * K // 2 + N * K // 2 + 4 * N + 4 * M + 2 * M * N
    assert bench.linear_bytes(M, N, K, 4) == 2 * M * K + N * K // 2 + 4 * N + 2 * M * N
    assert bench.gemm_bytes(M, N, K, 8) == M * K + N * K + 4 * N + 4 * M + 2 * M * N


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, bench.__file__, "--gpus", "2"], capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr)


def test_trace_summary_splits_points_at_sentinels(tmp_path):
    """A synthetic rocprofv3 kernel trace: set-up kernels outside the sentinel pairs are left
    out, each point's kernels are grouped by name and grid, and us/call divides by the
    manifest's call count."""
    import json
    hdr = ("Kind,Agent_Id,Queue_Id,Kernel_Id,Kernel_Name,Correlation_Id,Start_Timestamp,End_Timestamp,"
           "Workgroup_Size_X,Workgroup_Size_Y,Workgroup_Size_Z,Grid_Size_X,Grid_Size_Y,Grid_Size_Z")
    sent = "void at::native::vectorized_elementwise_kernel<4, at::native::bitwise_not_kernel_cuda>"
    t = [0]

    def row(name, dur_ns, grid=(256, 1, 1), wg=(256, 1, 1)):
        t[0] += 1000
        s = t[0]
        t[0] += dur_ns
        return f'KERNEL_DISPATCH,1,1,1,"{name}",1,{s},{t[0]},{wg[0]},{wg[1]},{wg[2]},{grid[0]},{grid[1]},{grid[2]}'

    lines = [hdr, row("setup_a", 50_000), row(sent, 100)]
    lines += [row("gemm", 4000, (512, 2, 1)) for _ in range(3)] + [row("prologue", 1000) for _ in range(3)]
    lines += [row(sent, 100), row("setup_b", 70_000), row(sent, 100)]
    lines += [row("gemm", 6000, (512, 1, 4)), row("gemm", 8000, (512, 1, 4))]
    lines += [row(sent, 100)]
    csv_path = tmp_path / "k_kernel_trace.csv"
    csv_path.write_text("\n".join(lines) + "\n")
    man = tmp_path / "manifest.txt"
    man.write_text(json.dumps({"rocprof_manifest": [{"name": "p0", "calls": 3}, {"name": "p1", "calls": 2}]}) + "\n")
    out = tmp_path / "summary.json"
    bench.summarize_trace(str(csv_path), str(man), str(out))
    pts = json.loads(out.read_text())["points"]
    assert pts["p0"]["us_per_call"] == 5.0
    assert {k["kernel"]: k["launches"] for k in pts["p0"]["kernels"]} == {"gemm": 3, "prologue": 3}
    assert pts["p1"]["us_per_call"] == 7.0
    assert pts["p1"]["kernels"][0]["grid"] == [512, 1, 4] and pts["p1"]["kernels"][0]["min_us"] == 6.0
    assert (tmp_path / "summary.md").exists()
    man.write_text(json.dumps({"rocprof_manifest": [{"name": "p0", "calls": 3}]}) + "\n")
    with pytest.raises(SystemExit):
        bench.summarize_trace(str(csv_path), str(man), str(out))
