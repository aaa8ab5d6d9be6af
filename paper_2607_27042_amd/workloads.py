"""Seeded synthetic workloads for two-sided rounding ``||A (Z - X) B||_F^2``.

This module only draws inputs. It holds none of the rounding method's
arithmetic, and it is the one piece shared by the GPU tests, the benchmark and
the oracle tests (each imports it on its own; the GPU binding does not).

The paper (arXiv 2607.27042) has no experiments, so every workload is a
synthetic stand-in with the shapes and spectra of layer-wise quantisation
problems:

====  ==============  ==========================================================
name  shape / dtype   construction
====  ==============  ==========================================================
c1    64 x 64, f64    X = 4 N(0,1). W is 256 x 64 N(0,1), G = W^T W / 256 + 0.01 I,
                      A = chol(G)^T (upper). B likewise from its own stream.
c2    512 x 384, f32  X = 3 N(0,1). W is 2048 x d N(0,1) with column k scaled by
                      exp(U[ln 0.1, ln 10]); G = W^T W / 2048 + 0.01 I; A = chol(G)^T.
c3    4096^2, f32     X = N(0, 0.02^2) / (0.02 / 3) (LLM-like weights in units of a
                      per-tensor step). T is 8192 x d iid Student-t(4);
                      G = T^T T / 8192; G += 0.01 mean(diag G) I; A = chol(G)^T.
c4    4096 x 11008,   X = 3 N(0,1). 16384 activation rows g + sqrt(50) V h with
      f32             g ~ N(0, I_d), h ~ N(0, I_32), V a d x 32 orthonormal basis
                      (QR of a Gaussian); G = W^T W / 16384 + 0.01 mean(diag G) I.
c5    8192^2, f32     X ~ U[-7.5, 7.5]. A = strict_upper(N(0,1)) / sqrt(8192) +
      and f64         diag(exp(U[ln 0.5, ln 2])); B likewise.
====  ==============  ==========================================================

Readings: "Cholesky-transpose of G" is ``A = chol_lower(G)^T`` (upper), so
``A^T A = G``; "B built the same way" applies the same recipe to B, so B is
upper triangular and ``B B^T`` has the spectrum of its Gram. Each role draws
from ``numpy.random.default_rng([config, role])`` with role 0 = X, 1 = A side,
2 = B side. Everything is built in float64 and cast once to the run dtype; the
oracle widens the cast values back to float64 exactly.
"""
from __future__ import annotations

import dataclasses
import hashlib
import os

import numpy as np

__all__ = ["Problem", "CONFIGS", "make_config", "random_problem", "config_names"]


@dataclasses.dataclass
class Problem:
    name: str
    X: np.ndarray  # m x n, run dtype
    A: np.ndarray  # m x m, run dtype
    B: np.ndarray  # n x n, run dtype
    dtype: str     # "f32" or "f64"

    @property
    def m(self) -> int:
        return self.X.shape[0]

    @property
    def n(self) -> int:
        return self.X.shape[1]

    def widened(self):
        """X, A, B as float64 (exact widening of the run-dtype values)."""
        return (self.X.astype(np.float64), self.A.astype(np.float64),
                self.B.astype(np.float64))


# (config id) -> (m, n, dtypes)
CONFIGS = {
    1: (64, 64, ("f64",)),
    2: (512, 384, ("f32",)),
    3: (4096, 4096, ("f32",)),
    4: (4096, 11008, ("f32",)),
    5: (8192, 8192, ("f32", "f64")),
}


def config_names():
    out = []
    for k, (m, n, dts) in CONFIGS.items():
        for dt in dts:
            out.append((k, dt))
    return out


def _np_dtype(dt: str):
    return {"f32": np.float32, "f64": np.float64}[dt]


def _chol_t(G: np.ndarray) -> np.ndarray:
    """Upper triangular A with A^T A = G (transpose of the lower Cholesky factor)."""
    return np.ascontiguousarray(np.linalg.cholesky(G).T)


def _basis_c1(d, rng):
    W = rng.standard_normal((256, d))
    G = W.T @ W / 256.0 + 0.01 * np.eye(d)
    return _chol_t(G)


def _basis_c2(d, rng):
    W = rng.standard_normal((2048, d))
    W *= np.exp(rng.uniform(np.log(0.1), np.log(10.0), size=d))[None, :]
    G = W.T @ W / 2048.0 + 1e-2 * np.eye(d)
    return _chol_t(G)


def _damped(G):
    G[np.diag_indices_from(G)] += 0.01 * float(np.mean(np.diag(G)))
    return G


def _basis_c3(d, rng):
    T = rng.standard_t(4.0, size=(8192, d))
    G = T.T @ T / 8192.0
    return _chol_t(_damped(G))


def _basis_c4(d, rng, rows=16384, rank=32, strength=50.0):
    V, _ = np.linalg.qr(rng.standard_normal((d, rank)))
    G = np.zeros((d, d))
    chunk = 4096
    for r0 in range(0, rows, chunk):
        r = min(chunk, rows - r0)
        W = rng.standard_normal((r, d)) + np.sqrt(strength) * (rng.standard_normal((r, rank)) @ V.T)
        G += W.T @ W
    G /= rows
    return _chol_t(_damped(G))


def _basis_c5(d, rng):
    A = np.triu(rng.standard_normal((d, d)), 1) / np.sqrt(d)
    A[np.diag_indices(d)] = np.exp(rng.uniform(np.log(0.5), np.log(2.0), size=d))
    return A


_BASIS = {1: _basis_c1, 2: _basis_c2, 3: _basis_c3, 4: _basis_c4, 5: _basis_c5}


def _seed(k, role, layer):
    return [k, role] if layer == 0 else [k, role, layer]


def _x(k, m, n, layer=0):
    rng = np.random.default_rng(_seed(k, 0, layer))
    if k == 1:
        return 4.0 * rng.standard_normal((m, n))
    if k == 2:
        return 3.0 * rng.standard_normal((m, n))
    if k == 3:
        return rng.normal(0.0, 0.02, size=(m, n)) / (0.02 / 3.0)
    if k == 4:
        return 3.0 * rng.standard_normal((m, n))
    if k == 5:
        return rng.uniform(-7.5, 7.5, size=(m, n))
    raise KeyError(k)


def _cache_path(tag: str):
    root = os.environ.get("GPTQ2D_INPUT_CACHE")
    if not root:
        return None
    os.makedirs(root, exist_ok=True)
    return os.path.join(root, tag + ".npy")


def _cached(tag, fn):
    p = _cache_path(tag)
    if p and os.path.exists(p):
        return np.load(p, allow_pickle=False)
    v = fn()
    if p:
        np.save(p, v, allow_pickle=False)
    return v


def make_config(k: int, dtype: str | None = None, layer: int = 0) -> Problem:
    """The synthetic problem of config ``k`` (1..5) in run dtype ``dtype``.
    ``layer`` > 0 draws another problem from the same recipe (its own X and
    bases, as the layers of one model), for batched runs."""
    m, n, dts = CONFIGS[k]
    dt = dtype or dts[0]
    if dt not in dts:
        raise ValueError(f"config {k} is defined for {dts}, not {dt}")
    npdt = _np_dtype(dt)
    sfx = "" if layer == 0 else f"_l{layer}"
    X = _cached(f"c{k}_X{sfx}", lambda: _x(k, m, n, layer))
    A = _cached(f"c{k}_A{sfx}", lambda: _BASIS[k](m, np.random.default_rng(_seed(k, 1, layer))))
    B = _cached(f"c{k}_B{sfx}", lambda: _BASIS[k](n, np.random.default_rng(_seed(k, 2, layer))))
    name = f"c{k}_{m}x{n}_{dt}{sfx}"
    return Problem(name, np.ascontiguousarray(X.astype(npdt)),
                   np.ascontiguousarray(A.astype(npdt)), np.ascontiguousarray(B.astype(npdt)), dt)


def random_problem(m: int, n: int, seed: int, dtype: str = "f64", kind: str = "wishart",
                   xscale: float = 3.0) -> Problem:
    """A small random problem for shape sweeps.

    kind: "wishart" (A = chol(W^T W / r + 0.05 I)^T, the default), "general"
    (dense non-triangular, diagonally shifted Gaussian bases), "diag"
    (diagonal bases), "lower" (lower-triangular A, upper-triangular B),
    "identity_right" (B = I) or "identity_left" (A = I).
    """
    rng = np.random.default_rng([1000 + seed, m, n])

    def wishart(d):
        r = max(2 * d, 8)
        W = rng.standard_normal((r, d))
        return _chol_t(W.T @ W / r + 0.05 * np.eye(d))

    def general(d):
        return rng.standard_normal((d, d)) / np.sqrt(d) + 2.0 * np.eye(d)

    def diag(d):
        return np.diag(np.exp(rng.uniform(-1.0, 1.0, size=d)))

    def tri(d, lower):
        T = rng.standard_normal((d, d)) / np.sqrt(d)
        T = np.tril(T, -1) if lower else np.triu(T, 1)
        T[np.diag_indices(d)] = np.exp(rng.uniform(np.log(0.5), np.log(2.0), size=d))
        return T

    X = xscale * rng.standard_normal((m, n))
    if kind == "wishart":
        A, B = wishart(m), wishart(n)
    elif kind == "general":
        A, B = general(m), general(n)
    elif kind == "diag":
        A, B = diag(m), diag(n)
    elif kind == "lower":
        A, B = tri(m, True), tri(n, False)
    elif kind == "identity_right":
        A, B = wishart(m), np.eye(n)
    elif kind == "identity_left":
        A, B = np.eye(m), wishart(n)
    else:
        raise ValueError(kind)
    npdt = _np_dtype(dtype)
    name = f"rand_{kind}_{m}x{n}_s{seed}_{dtype}"
    return Problem(name, np.ascontiguousarray(X.astype(npdt)), np.ascontiguousarray(A.astype(npdt)),
                   np.ascontiguousarray(B.astype(npdt)), dtype)


def digest(a: np.ndarray) -> str:
    """Short content hash of an array (used to label fixtures)."""
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()[:16]
