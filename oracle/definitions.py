"""Float64 definitions written out with explicit matrices (test infrastructure).

Each function is the paper's formula evaluated directly, with no fast transform
and no reordering, so it can be checked against the paper by eye:
  * sylvester(b): H_b[i, j] = (-1)^popcount(i & j), the Sylvester +-1 matrix in
    natural order (Sec. III-C).
  * block_rotation(K, b): R = I_{K/b} (x) H_b / sqrt(b) (Sec. III-C).
  * fold_weight(W, b, s, p): W~ = W S R^T P, the consumer weight of the fold presets
    (Sec. III-C: fold-before (S^-1, I) gives W S R^T, fold-after (I, P^-1) gives
    W R^T P; eq. (2)).
  * transform_tokens(X, b, s_inv, p_inv): z_t = P^-1 R S^-1 x_t.
  * composite_rotation(perm, blocks): R = B P, the stored composite rotation of
    Sec. III-C (channel permutation P, block-diagonal B of per-block matrices).
  * quantize_eq5(Z, bits, r): eq. (5) in float64 with the zero-token rule.
  * integer_output(qw, s_w, qa, delta, bias): eq. (8).
"""
from __future__ import annotations

from typing import Optional, Tuple

import numpy as np


def sylvester(b: int) -> np.ndarray:
    """H_b with entries (-1)^popcount(i & j); b a power of two."""
    assert b >= 1 and b & (b - 1) == 0
    i = np.arange(b)[:, None]
    j = np.arange(b)[None, :]
    bits_and = i & j
    parity = np.zeros_like(bits_and)
    v = bits_and.copy()
    while v.any():
        parity ^= v & 1
        v >>= 1
    return np.where(parity == 1, -1.0, 1.0)


def block_rotation(K: int, b: int) -> np.ndarray:
    """R = I_{K/b} (x) H_b / sqrt(b), float64 [K, K]."""
    assert K % b == 0
    return np.kron(np.eye(K // b), sylvester(b) / np.sqrt(b))


def transform_tokens(X: np.ndarray, b: int, s_inv: Optional[np.ndarray] = None,
                     p_inv: Optional[np.ndarray] = None) -> np.ndarray:
    """z_t = P^-1 R S^-1 x_t for every row x_t of X (float64 [M, K])."""
    X = np.asarray(X, dtype=np.float64)
    if s_inv is not None:
        X = X * np.asarray(s_inv, dtype=np.float64)[None, :]
    R = block_rotation(X.shape[1], b)
    Z = X @ R.T
    if p_inv is not None:
        Z = Z * np.asarray(p_inv, dtype=np.float64)[None, :]
    return Z


def fold_weight(W: np.ndarray, b: int, s: Optional[np.ndarray] = None,
                p: Optional[np.ndarray] = None) -> np.ndarray:
    """W~ = W S R^T P (float64 [N, K])."""
    W = np.asarray(W, dtype=np.float64)
    if s is not None:
        W = W * np.asarray(s, dtype=np.float64)[None, :]
    R = block_rotation(W.shape[1], b)
    Wt = W @ R.T
    if p is not None:
        Wt = Wt * np.asarray(p, dtype=np.float64)[None, :]
    return Wt


def composite_rotation(perm: Optional[np.ndarray], blocks: np.ndarray) -> np.ndarray:
    """R = B P (float64 [K, K]): (P v)_c = v_perm[c], B = diag(Q_0, Q_1, ...)."""
    nb, b, _ = blocks.shape
    K = nb * b
    P = np.eye(K)[np.arange(K) if perm is None else np.asarray(perm)]
    B = np.zeros((K, K))
    for k in range(nb):
        B[k * b:(k + 1) * b, k * b:(k + 1) * b] = blocks[k]
    return B @ P


def quantize_eq5(Z: np.ndarray, bits: int, r: float = 1.0) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Eq. (5) per row: delta = r ||z||_inf / q, codes = clip(round(z / delta), -q, q).

    Returns (codes int64 [M, K], delta float64 [M], ratio float64 [M, K] = z / delta)
    so callers can see how close each element sits to a rounding tie.
    A zero row gives codes 0 and delta 0.
    """
    Z = np.asarray(Z, dtype=np.float64)
    q = 2 ** (bits - 1) - 1
    amax = np.abs(Z).max(axis=1) if Z.shape[1] else np.zeros(Z.shape[0])
    delta = r * amax / q
    safe = np.where(delta > 0, delta, 1.0)
    ratio = np.where(delta[:, None] > 0, Z / safe[:, None], 0.0)
    codes = np.clip(np.rint(ratio), -q, q).astype(np.int64)
    return codes, delta, ratio


def integer_output(qw: np.ndarray, s_w: np.ndarray, qa: np.ndarray, delta: np.ndarray,
                   bias: Optional[np.ndarray] = None) -> np.ndarray:
    """Eq. (8): y[t, j] = s_w[j] delta[t] sum_c qw[j, c] qa[t, c] + b_j (float64 [M, N])."""
    acc = np.asarray(qa, dtype=np.int64) @ np.asarray(qw, dtype=np.int64).T
    y = acc.astype(np.float64) * np.asarray(s_w, np.float64)[None, :] * np.asarray(delta, np.float64)[:, None]
    if bias is not None:
        y = y + np.asarray(bias, np.float64)[None, :]
    return y


def obs_round_rows(Wt: np.ndarray, H: np.ndarray, bits: int) -> Tuple[np.ndarray, np.ndarray]:
    """The rounding eq. (7) asks of GPTQ, written as its defining sequence of optimal-brain-
    surgeon steps in float64 with explicit linear solves (no Cholesky factor): the columns
    of each row are rounded in order; before column c is rounded, every column not yet
    rounded holds the value that minimizes (w - w0) H (w - w0)^T given the rounded ones.
    Rounding uses the row's fixed step max|w0| / q.  Returns (codes int64 [N, K], the
    smallest distance of any rounding argument from a half-integer, for tie screening)."""
    Wt = np.asarray(Wt, dtype=np.float64)
    H = np.asarray(H, dtype=np.float64)
    N, K = Wt.shape
    q = 2 ** (bits - 1) - 1
    codes = np.zeros((N, K), dtype=np.int64)
    margin = np.inf
    for j in range(N):
        w0 = Wt[j]
        A = np.abs(w0).max()
        if A == 0.0:
            continue
        step = A / q
        w = w0.copy()
        for c in range(K):
            t = w[c] / step
            margin = min(margin, abs(abs(t - np.floor(t)) - 0.5))
            codes[j, c] = int(np.clip(np.rint(t), -q, q))
            fixed = np.arange(c + 1)
            free = np.arange(c + 1, K)
            if free.size:
                d = codes[j, fixed] * step - w0[fixed]
                w[free] = w0[free] - np.linalg.solve(H[np.ix_(free, free)], H[np.ix_(free, fixed)] @ d)
    return codes, margin


def gptq_objective(Wt: np.ndarray, Q: np.ndarray, Z: np.ndarray) -> float:
    """||(W~ - Q) Z||_F^2 of eq. (7) in float64 (Z: calibration tokens as rows [T, K])."""
    D = np.asarray(Wt, np.float64) - np.asarray(Q, np.float64)
    return float(np.sum((D @ np.asarray(Z, np.float64).T) ** 2))
