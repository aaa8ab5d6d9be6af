"""CPU oracle for two-sided adaptive rounding (GPTQ-2D, arXiv 2607.27042).

TEST INFRASTRUCTURE ONLY. Only the test suite, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` may import this package. The product
library never links, loads or calls it, and it shares no code with the GPU path.

This module is argument marshalling around ``oracle.c`` (plain C, fp64):

* ``gram_left`` / ``gram_right``  -- G = A^T A, H = B B^T (Sec. 3.2, Eq. GH)
* ``feedback``                    -- unit-lower LDL factor of an inverse Gram,
                                     by explicit inverse then LDL (Sec. 3.1)
* ``factors``                     -- per-axis L, U of the two-sided problem
                                     (Sec. 4.1)
* ``round_1d``                    -- Algorithm 1
* ``round_quartic``               -- Algorithm 1 on vec(X) under an explicit
                                     Kronecker Gram H (x) G (Eq. kron-objective)
* ``round_kron``                  -- Algorithm 1 on vec(X) with F = U^T (x) L
                                     (Eq. vectorized-feedback)
* ``round_nested``                -- Algorithm 5, the cubic oracle (Appendix A)
* ``round_nested_corner``         -- Algorithm 5 on a leading block
* ``round_gptq2d``                -- Algorithm 3 (Sec. 4.2)
* ``round_implicit``              -- Algorithm 6 (Appendix B)
* ``objective``                   -- ||A (Z - X) B||_F^2 by definition
* ``trajectory_values``           -- the value every entry had when it was
                                     rounded, given all rounding errors E:
                                     Y = X + L E U - E (Eq. Y-LEU)
* ``trajectory_check``            -- judges a whole (Z, Y) against that
                                     definition and the window rule
* ``round_reverse``               -- the same rounding in reverse order (from the
                                     last row and column, the direction of YAQA,
                                     Sec. 2): Algorithm 5 on the index-reversed
                                     problem (P X P, A P, P B), reversed back

Every sweep returns ``(Z, Ypre, counts, hard)``: the rounded matrix (int32),
the value each entry had when it was rounded, the synchronised-replay counters
``{"window", "hard", "range"}`` and the flat indices of the first hard
mismatches.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

_lib = None


def build(force: bool = False) -> str:
    """Compile ``oracle.c`` into ``liboracle.so`` with gcc and OpenMP."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O3", "-fopenmp", "-fPIC", "-shared", "-Wall", "-o", tmp, _SRC, "-lm"]
        subprocess.check_call(cmd)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(_LIB)
        dp = ctypes.POINTER(ctypes.c_double)
        ip = ctypes.POINTER(ctypes.c_int32)
        lp = ctypes.POINTER(ctypes.c_int64)
        i = ctypes.c_int
        lib.orc_gram_left.argtypes = [i, dp, dp]
        lib.orc_gram_right.argtypes = [i, dp, dp]
        lib.orc_inverse.argtypes = [i, dp, dp]
        lib.orc_inverse.restype = i
        lib.orc_ldl.argtypes = [i, dp, dp, dp]
        lib.orc_ldl.restype = i
        lib.orc_feedback.argtypes = [i, dp, dp, dp]
        lib.orc_feedback.restype = i
        lib.orc_factors.argtypes = [i, i, dp, dp, dp, dp, dp, dp]
        lib.orc_factors.restype = i
        lib.orc_round_1d.argtypes = [i, dp, dp, ip, ctypes.c_double, ip, dp, lp, lp, i]
        lib.orc_round_1d.restype = i
        lib.orc_round_quartic.argtypes = [i, i, dp, dp, dp, ip, ctypes.c_double, ip, dp, lp, lp, i]
        lib.orc_round_quartic.restype = i
        for name in ("orc_round_kron", "orc_round_nested", "orc_round_gptq2d", "orc_round_implicit"):
            f = getattr(lib, name)
            f.argtypes = [i, i, dp, dp, dp, ip, ctypes.c_double, ip, dp, lp, lp, i]
            f.restype = i
        lib.orc_round_nested_corner.argtypes = [i, i, i, i, dp, dp, dp, ip, ctypes.c_double, ip, dp,
                                                lp, lp, i]
        lib.orc_round_nested_corner.restype = i
        lib.orc_round_nested_cols.argtypes = [i, i, i, dp, dp, dp, ip, ctypes.c_double, ip, dp, lp, lp, i]
        lib.orc_round_nested_cols.restype = i
        lib.orc_objective.argtypes = [i, i, dp, ip, dp, dp]
        lib.orc_objective.restype = ctypes.c_double
        lib.orc_num_threads.argtypes = []
        lib.orc_num_threads.restype = i
        _lib = lib
    return _lib


class OracleError(RuntimeError):
    pass


_STATUS = {0: "ok", -2: "singular or not positive definite", -4: "out of memory",
           -7: "rounded value outside int32"}


def _check(st: int, what: str):
    if st != 0:
        raise OracleError(f"{what}: {_STATUS.get(st, st)}")


def _d(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def _dp(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _ip(a):
    if a is None:
        return ctypes.cast(None, ctypes.POINTER(ctypes.c_int32))
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def _lp(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int64))


def num_threads() -> int:
    return int(_load().orc_num_threads())


def gram_left(A) -> np.ndarray:
    A = _d(A)
    m = A.shape[0]
    G = np.empty((m, m))
    _load().orc_gram_left(m, _dp(A), _dp(G))
    return G


def gram_right(B) -> np.ndarray:
    B = _d(B)
    n = B.shape[0]
    H = np.empty((n, n))
    _load().orc_gram_right(n, _dp(B), _dp(H))
    return H


def inverse(M) -> np.ndarray:
    M = _d(M)
    d = M.shape[0]
    out = np.empty((d, d))
    _check(_load().orc_inverse(d, _dp(M), _dp(out)), "inverse")
    return out


def ldl(S):
    S = _d(S)
    d = S.shape[0]
    F = np.empty((d, d))
    D = np.empty(d)
    _check(_load().orc_ldl(d, _dp(S), _dp(F), _dp(D)), "ldl")
    return F, D


def feedback(Q):
    """Unit-lower F and diagonal lam with Q^{-1} = F diag(lam) F^T."""
    Q = _d(Q)
    d = Q.shape[0]
    F = np.empty((d, d))
    lam = np.empty(d)
    _check(_load().orc_feedback(d, _dp(Q), _dp(F), _dp(lam)), "feedback")
    return F, lam


def factors(A, B):
    """(L, lamL, U, lamU) for the bases A (m x m) and B (n x n)."""
    A = _d(A)
    B = _d(B)
    m, n = A.shape[0], B.shape[0]
    L = np.empty((m, m))
    U = np.empty((n, n))
    lamL = np.empty(m)
    lamU = np.empty(n)
    _check(_load().orc_factors(m, n, _dp(A), _dp(B), _dp(L), _dp(lamL), _dp(U), _dp(lamU)),
           "factors")
    return L, lamL, U, lamU


def _replay_args(hint, shape, tau, hard_cap):
    h = None if hint is None else np.ascontiguousarray(hint, dtype=np.int32)
    if h is not None and h.shape != shape:
        raise ValueError("hint shape mismatch")
    counts = np.zeros(3, dtype=np.int64)
    hard = np.zeros(max(hard_cap, 1), dtype=np.int64)
    return h, counts, hard


def _result(Z, Y, counts, hard, hard_cap):
    c = {"window": int(counts[0]), "hard": int(counts[1]), "range": int(counts[2])}
    return Z, Y, c, hard[: min(c["hard"], hard_cap)].copy()


def round_1d(x, F, hint=None, tau=0.0, hard_cap=64):
    x = _d(x)
    F = _d(F)
    d = x.shape[0]
    h, counts, hard = _replay_args(hint, (d,), tau, hard_cap)
    z = np.empty(d, dtype=np.int32)
    y = np.empty(d)
    _check(_load().orc_round_1d(d, _dp(x), _dp(F), _ip(h), float(tau), _ip(z), _dp(y), _lp(counts),
                                _lp(hard), hard_cap), "round_1d")
    return _result(z, y, counts, hard, hard_cap)


def round_quartic(X, A, B, hint=None, tau=0.0, hard_cap=64):
    X = _d(X)
    A = _d(A)
    B = _d(B)
    m, n = X.shape
    h, counts, hard = _replay_args(hint, (m, n), tau, hard_cap)
    Z = np.empty((m, n), dtype=np.int32)
    Y = np.empty((m, n))
    _check(_load().orc_round_quartic(m, n, _dp(X), _dp(A), _dp(B), _ip(h), float(tau), _ip(Z),
                                     _dp(Y), _lp(counts), _lp(hard), hard_cap), "round_quartic")
    return _result(Z, Y, counts, hard, hard_cap)


def _sweep(name, X, L, U, hint, tau, hard_cap):
    X = _d(X)
    L = _d(L)
    U = _d(U)
    m, n = X.shape
    if L.shape != (m, m) or U.shape != (n, n):
        raise ValueError("factor shape mismatch")
    h, counts, hard = _replay_args(hint, (m, n), tau, hard_cap)
    Z = np.empty((m, n), dtype=np.int32)
    Y = np.empty((m, n))
    f = getattr(_load(), name)
    _check(f(m, n, _dp(X), _dp(L), _dp(U), _ip(h), float(tau), _ip(Z), _dp(Y), _lp(counts),
             _lp(hard), hard_cap), name)
    return _result(Z, Y, counts, hard, hard_cap)


def round_kron(X, L, U, hint=None, tau=0.0, hard_cap=64):
    return _sweep("orc_round_kron", X, L, U, hint, tau, hard_cap)


def round_nested(X, L, U, hint=None, tau=0.0, hard_cap=64):
    return _sweep("orc_round_nested", X, L, U, hint, tau, hard_cap)


def round_gptq2d(X, L, U, hint=None, tau=0.0, hard_cap=64):
    return _sweep("orc_round_gptq2d", X, L, U, hint, tau, hard_cap)


def round_implicit(X, L, U, hint=None, tau=0.0, hard_cap=64):
    return _sweep("orc_round_implicit", X, L, U, hint, tau, hard_cap)


def round_nested_columns(X, L, U, ncols):
    """Algorithm 5 on the first ncols columns of the problem only: Z and the
    corrected values of those columns (an error at (i, j) reaches only columns
    >= j, Eq. rank-one-update, so they are the whole sweep's). Bounds the CPU
    work of a large problem when the sweep is timed."""
    X = _d(X)
    L = _d(L)
    U = _d(U)
    m, n = X.shape
    if L.shape != (m, m) or U.shape != (n, n):
        raise ValueError("factor shape mismatch")
    if not (0 <= ncols <= n):
        raise ValueError("ncols out of range")
    h, counts, hard = _replay_args(None, (m, n), 0.0, 64)
    Z = np.zeros((m, n), dtype=np.int32)
    Y = np.zeros((m, n))
    _check(_load().orc_round_nested_cols(m, n, int(ncols), _dp(X), _dp(L), _dp(U), _ip(h), 0.0, _ip(Z),
                                         _dp(Y), _lp(counts), _lp(hard), 64), "round_nested_cols")
    return Z[:, :ncols].copy(), Y[:, :ncols].copy()


def round_nested_corner(X, L, U, m1, n1, hint=None, tau=0.0, hard_cap=64):
    """Algorithm 5 on the leading m1 x n1 block of the full problem."""
    X = _d(X)
    L = _d(L)
    U = _d(U)
    m, n = X.shape
    if not (0 < m1 <= m and 0 < n1 <= n):
        raise ValueError("corner out of range")
    h, counts, hard = _replay_args(hint, (m1, n1), tau, hard_cap)
    Z = np.empty((m1, n1), dtype=np.int32)
    Y = np.empty((m1, n1))
    _check(_load().orc_round_nested_corner(m, n, m1, n1, _dp(X), _dp(L), _dp(U), _ip(h), float(tau),
                                           _ip(Z), _dp(Y), _lp(counts), _lp(hard), hard_cap),
           "round_nested_corner")
    return _result(Z, Y, counts, hard, hard_cap)


def objective(X, Z, A, B) -> float:
    X = _d(X)
    Z = np.ascontiguousarray(Z, dtype=np.int32)
    A = _d(A)
    B = _d(B)
    m, n = X.shape
    return float(_load().orc_objective(m, n, _dp(X), _ip(Z), _dp(A), _dp(B)))


def trajectory_values(X, L, U, E) -> np.ndarray:
    """Corrected values of the sweep whose rounding errors are E.

    After the whole sweep Z - X = L E U (Eq. Y-LEU; proof of Theorem 2). The
    value an entry (i, j) had when it was rounded is X_ij plus the pushes of
    every entry rounded before it, and those are exactly the entries
    (i', j') != (i, j) with i' <= i and j' <= j (Eq. rank-one-update). That is
    (L E U)_ij without its own term L_ii E_ij U_jj = E_ij, so
    Y = X + L E U - E. Two dense fp64 products (a library matmul as a step),
    which makes this the oracle's check at sizes its sweeps cannot replay."""
    X, L, U, E = _d(X), _d(L), _d(U), _d(E)
    m, n = X.shape
    if L.shape != (m, m) or U.shape != (n, n) or E.shape != (m, n):
        raise ValueError("shape mismatch")
    return X + (L @ E) @ U - E


def trajectory_check(X, L, U, Z, Y, tau):
    """Judges a complete result (Z, Y) of a sweep under factors L, U against
    the definition above: with E = Z - Y the errors the sweep made, the values
    Y' = X + L E U - E are what the greedy trajectory rounds from, and each
    entry must be the nearest integer to its Y' (ties to even). An entry
    where it is not counts as a "window" entry when Y' lies within tau of the
    half-integer between the two candidates, otherwise as a "hard" mismatch
    (the rule of the synchronised replay). Returns (max |Y' - Y|, counts,
    flat indices of the first hard mismatches)."""
    Z = np.asarray(Z)
    Y = _d(Y)
    Yp = trajectory_values(X, L, U, Z.astype(np.float64) - Y)
    dev = float(np.abs(Yp - Y).max()) if Yp.size else 0.0
    Zr = np.rint(Yp)
    off = np.flatnonzero(Zr.ravel() != Z.ravel())
    zo = Z.ravel()[off].astype(np.float64)
    yo = Yp.ravel()[off]
    near = (np.abs(zo - Zr.ravel()[off]) == 1.0) & (np.abs(yo - 0.5 * (zo + Zr.ravel()[off])) <= tau)
    counts = {"window": int(near.sum()), "hard": int((~near).sum())}
    return dev, counts, off[~near][:64]


def reverse_problem(X, A, B):
    """The index-reversed problem (P X P, A P, P B), P the reversal
    permutation: ||A (Z - X) B|| = ||(A P)(P Z P - P X P)(P B)||, so rounding it
    forward rounds the original from its last row and column."""
    X = _d(X)
    A = _d(A)
    B = _d(B)
    return (np.ascontiguousarray(X[::-1, ::-1]), np.ascontiguousarray(A[:, ::-1]),
            np.ascontiguousarray(B[::-1, :]))


def round_reverse(X, A, B, hint=None, tau=0.0, hard_cap=64):
    """Two-sided rounding in reverse order (Sec. 2: YAQA's direction): the
    factors and Algorithm 5 of the index-reversed problem, Z and the values
    rounded from reversed back. A hint is given in the original order."""
    Xr, Ar, Br = reverse_problem(X, A, B)
    L, lamL, U, lamU = factors(Ar, Br)
    h = None if hint is None else np.ascontiguousarray(np.asarray(hint)[::-1, ::-1])
    Z, Y, c, hard = round_nested(Xr, L, U, hint=h, tau=tau, hard_cap=hard_cap)
    m, n = Z.shape
    # flat indices of hard mismatches in the original order
    hard = np.array([(m - 1 - k // n) * n + (n - 1 - k % n) for k in hard], dtype=np.int64)
    return np.ascontiguousarray(Z[::-1, ::-1]), np.ascontiguousarray(Y[::-1, ::-1]), c, hard
