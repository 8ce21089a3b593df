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
