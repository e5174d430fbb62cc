"""Brute-force checkers for the affine recurrence (float64, tiny sizes only).

TEST INFRASTRUCTURE ONLY (same rules as ``oracle.deer_oracle``).

* ``block_bidiagonal_solve``: the recurrence y_t = J_t y_{t-1} + b_t, y_0 = 0,
  written as one dense linear system whose matrix has identity blocks on the
  diagonal and -J_t below it (eq. blockdiag_jacobian), solved by LAPACK.
* ``compose`` / ``all_bracketings``: the affine-pair composition
  (A2, b2) o (A1, b1) = (A2 A1, A2 b1 + b2) (scheduled-sampling appendix,
  incompatibility with parallel scan) folded in every binary-tree order.
* ``chunked_scan``: the recurrence evaluated the way a chunked parallel scan
  does it (chunk aggregates, carry across chunks, fix-up from the carry), to
  pin the decomposition itself for every chunk size.
"""
from __future__ import annotations

import numpy as np


def block_bidiagonal_solve(J: np.ndarray, b: np.ndarray) -> np.ndarray:
    """J [T, M, M] (J[k] = J_{k+1}), b [T, M] -> y [T, M]."""
    T, M = b.shape
    R = np.eye(T * M)
    for t in range(1, T):
        R[t * M:(t + 1) * M, (t - 1) * M:t * M] = -J[t]
    return np.linalg.solve(R, b.reshape(-1)).reshape(T, M)


def block_bidiagonal_adjoint_solve(J: np.ndarray, g: np.ndarray) -> np.ndarray:
    """Solve V^T R = g^T for the same block matrix R (eq. adjoint_eq with the sign
    convention lam = -v): returns lam with R^T lam = g."""
    T, M = g.shape
    R = np.eye(T * M)
    for t in range(1, T):
        R[t * M:(t + 1) * M, (t - 1) * M:t * M] = -J[t]
    return np.linalg.solve(R.T, g.reshape(-1)).reshape(T, M)


def compose(e2, e1):
    """(A2, b2) o (A1, b1) = (A2 A1, A2 b1 + b2)."""
    A2, b2 = e2
    A1, b1 = e1
    return A2 @ A1, A2 @ b1 + b2


def all_bracketings(elems):
    """Every full binary bracketing of e_n o ... o e_1 (elems listed e_1 first)."""
    n = len(elems)
    if n == 1:
        return [elems[0]]
    out = []
    for split in range(1, n):
        for left in all_bracketings(elems[:split]):
            for right in all_bracketings(elems[split:]):
                out.append(compose(right, left))
    return out


def chunked_scan(J: np.ndarray, b: np.ndarray, chunk: int) -> np.ndarray:
    """y_t = J_t y_{t-1} + b_t via chunks of length `chunk`:
    (1) per chunk, P_c = J_e ... J_s and v_c = local result from a zero carry;
    (2) carries y_end(c) = P_c y_end(c-1) + v_c;
    (3) each chunk re-run from its carry."""
    T, M = b.shape
    starts = list(range(0, T, chunk))
    aggs = []
    for s in starts:
        P = np.eye(M)
        v = np.zeros(M)
        for k in range(s, min(s + chunk, T)):
            P = J[k] @ P
            v = J[k] @ v + b[k]
        aggs.append((P, v))
    carries = []
    c = np.zeros(M)
    for P, v in aggs:
        carries.append(c)
        c = P @ c + v
    y = np.empty_like(b)
    for s, cin in zip(starts, carries):
        prev = cin
        for k in range(s, min(s + chunk, T)):
            prev = J[k] @ prev + b[k]
            y[k] = prev
    return y
