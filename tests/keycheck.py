"""Validity of int8 retrieval keys computed by another summation order.

The key of a state h is code_j = round-half-even(v_j * 127 / max_i |v_i|)
with v = R h (Section 4, "Memory and retrieval"). The projection is a sum of
H products; any fp64 evaluation order of it lies within gamma_H * sum_k
|R_jk h_k| of the exact value (gamma_n = n u / (1 - n u), u = 2^-53, fused or
separate multiply-adds alike). Two evaluations therefore round a scaled value
x_j differently only where x_j lies within their joint error of a
half-integer. check_codes() requires equality everywhere else and one of the
two neighbouring integers there, and reports how many codes fell into that
band.
"""
import numpy as np

U = 2.0 ** -53


def scaled_bounds(R: np.ndarray, h: np.ndarray, v: np.ndarray):
    """x = v * 127 / max|v| per row and a bound on |x' - x| for x' from any
    other fp64 evaluation order of the same projection."""
    R = np.asarray(R, np.float64)
    h = np.atleast_2d(np.asarray(h, np.float64))
    v = np.atleast_2d(v)
    H = R.shape[1]
    gamma = H * U / (1.0 - H * U)
    s = np.abs(h) @ np.abs(R).T                   # [n][kd]: sum_k |R_jk h_k|
    e = 2.0 * gamma * s * (1.0 + 1e-6)            # two evaluations
    m = np.abs(v).max(axis=1, keepdims=True)
    E = e.max(axis=1, keepdims=True)
    with np.errstate(divide="ignore", invalid="ignore"):
        x = np.where(m > 0, v * 127.0 / m, 0.0)
        d = np.where(m > E, 127.0 * (e + np.abs(v) * E / m) / (m - E), np.inf)
    d = d + 8.0 * U * 127.0
    return x, d


def check_codes(codes: np.ndarray, R: np.ndarray, h: np.ndarray, v: np.ndarray) -> int:
    """Assert that `codes` are valid keys of h given the oracle's projection
    v = oracle.key_project(R, h); return the number of codes within the
    rounding band of a half-integer (where either neighbour is valid)."""
    codes = np.atleast_2d(codes).astype(np.int64)
    x, d = scaled_bounds(R, h, v)
    near = np.abs(np.abs(x - np.floor(x)) - 0.5) <= d
    want = np.clip(np.rint(x), -127, 127).astype(np.int64)
    lo = np.clip(np.floor(x), -127, 127).astype(np.int64)
    hi = np.clip(np.ceil(x), -127, 127).astype(np.int64)
    ok = (codes == want) | (near & ((codes == lo) | (codes == hi)))
    zero_rows = (np.abs(v).max(axis=1) == 0)
    ok[zero_rows] = codes[zero_rows] == 0
    bad = np.argwhere(~ok)
    assert len(bad) == 0, (f"{len(bad)} invalid codes, first {bad[:6].tolist()}: "
                           f"got {codes[tuple(bad[0])]}, scaled {x[tuple(bad[0])]!r}")
    return int(near.sum())
