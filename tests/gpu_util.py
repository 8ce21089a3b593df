"""Shared helpers of the GPU parity tests (comparison rules, device transfer)."""
import numpy as np
import torch

DEV = torch.device("cuda:0") if torch.cuda.is_available() else None


def canonical_codes(codes_i8: np.ndarray, bits: int) -> np.ndarray:
    """Oracle codes in the library's canonical byte layout (through the oracle's own packer)."""
    import oracle
    if bits == 4:
        return oracle.pack_int4(codes_i8)
    return codes_i8.view(np.uint8)


def assert_bf16_close(y_gpu: torch.Tensor, y_ref: np.ndarray, rel: float = 1e-2):
    """Per row t: max_j |y_gpu - y_ref| <= rel * max_j |y_ref| (zero rows must match exactly)."""
    yg = y_gpu.float().cpu().numpy().astype(np.float64)
    assert yg.shape == y_ref.shape
    amax = np.abs(y_ref).max(axis=1, keepdims=True) if y_ref.size else y_ref
    err = np.abs(yg - y_ref)
    bad = err > rel * amax
    if bad.any():
        t, j = np.argwhere(bad)[0]
        raise AssertionError(f"row {t} col {j}: gpu {yg[t, j]} ref {y_ref[t, j]} (row absmax {amax[t, 0]})")


def flush(msg: str):
    print(msg, flush=True)
