"""The array-framework realisation of the paper's blocked sweep
(Algorithm 4, the comparison point timed by bench.py --array-baseline),
checked on the CPU against the oracle's Algorithm 5 sweep: the same Z under
the replay rule, the same corrected values, and Z - X = L E U. Block widths
from 1 (every push through a flush) to one block over the whole matrix
(Algorithm 3 alone)."""
import numpy as np
import pytest
import torch

import array_baseline as ab
import oracle
from paper_2607_27042_amd import workloads as wl


@pytest.mark.parametrize("m,n,w,kind", [(1, 1, 4, "wishart"), (5, 7, 1, "wishart"), (7, 5, 3, "general"),
                                        (33, 20, 8, "wishart"), (64, 70, 16, "general"),
                                        (40, 30, 200, "wishart"), (100, 90, 5, "diag")])
def test_blocked_sweep_matches_oracle(m, n, w, kind):
    p = wl.random_problem(m, n, 3, "f64", kind)
    X, A, B = p.widened()
    L, lamL, U, lamU = oracle.factors(A, B)
    Z, Y, E = ab.blocked_sweep(torch.from_numpy(X), torch.from_numpy(L), torch.from_numpy(U), w=w)
    Z, Y, E = Z.numpy(), Y.numpy(), E.numpy()
    Zo, Yo, c, hard = oracle.round_nested(X, L, U, hint=Z.astype(np.int32), tau=1e-12)
    assert c["hard"] == 0 and c["window"] == 0 and c["range"] == 0, c
    assert np.abs(Y - Yo).max() <= 1e-12 * max(1.0, np.abs(Yo).max())
    assert np.abs(E).max() <= 0.5
    assert np.abs((Z - X) - L @ E @ U).max() <= 1e-11 * max(1.0, np.abs(X).max())


# ---- the padded skew layout (Sec. 5, Fig. 2)

def test_skew_layout_construction():
    """Fig. 2's 3 x 4 example: row stride r = 2m + n - 2 = 8, entry (i, j) in
    row s = i + j at position m - 1 + j; an anti-diagonal is a contiguous row
    piece in column order, a matrix column a stride-r line, a matrix row a
    stride-(r + 1) line; (m + n - 1)(2m + n - 2) cells hold the m n entries."""
    m, n = 3, 4
    r = ab.skew_stride(m, n)
    assert r == 8
    flat = torch.full(((m + n - 1) * r,), -1.0, dtype=torch.float64)
    M = torch.arange(1, m * n + 1, dtype=torch.float64).reshape(m, n)
    ab.skew_matrix(flat, m, n).copy_(M)
    for i in range(m):
        for j in range(n):
            assert flat[(i + j) * r + m - 1 + j] == M[i, j]
    for s in range(m + n - 1):
        jlo, jhi = max(0, s - m + 1), min(s, n - 1)
        piece = flat[s * r + m - 1 + jlo: s * r + m + jhi]
        assert torch.equal(piece, torch.stack([M[s - j, j] for j in range(jlo, jhi + 1)]))
    for j in range(n):
        assert torch.equal(flat[j * r + m - 1 + j:: r][:m], M[:, j])
    for i in range(m):
        assert torch.equal(flat[i * r + m - 1:: r + 1][:n], M[i, :])
    assert int((flat != -1.0).sum()) == m * n
    assert flat.numel() == (m + n - 1) * (2 * m + n - 2)


@pytest.mark.parametrize("m,n,w,kind", [(1, 1, 4, "wishart"), (5, 7, 1, "wishart"), (7, 5, 3, "general"),
                                        (33, 20, 8, "wishart"), (64, 70, 16, "general"),
                                        (40, 30, 200, "wishart"), (3, 40, 8, "general"), (40, 3, 8, "general"),
                                        (1, 30, 4, "general")])
def test_skew_sweep_matches(m, n, w, kind):
    """Algorithm 4 on the skew layout: the same Z, Y, E as the natural-layout
    form, bit for bit, the oracle's replay, and padding cells that stay zero
    (every update outside the matrix is skipped)."""
    p = wl.random_problem(m, n, 3, "f64", kind)
    X, A, B = p.widened()
    L, lamL, U, lamU = oracle.factors(A, B)
    args = (torch.from_numpy(X), torch.from_numpy(L), torch.from_numpy(U))
    arrays = {}
    Zs, Ys, Es = ab.blocked_sweep_skew(*args, w=w, arrays=arrays)
    Zn, Yn, En = ab.blocked_sweep(*args, w=w)
    assert torch.equal(Zs, Zn) and torch.equal(Ys, Yn) and torch.equal(Es, En)
    Zo, Yo, c, hard = oracle.round_nested(X, L, U, hint=Zs.numpy().astype(np.int32), tau=1e-12)
    assert c["hard"] == 0 and c["window"] == 0 and c["range"] == 0, c
    r = ab.skew_stride(m, n)
    data = torch.zeros_like(arrays["E"], dtype=torch.bool)
    ab.skew_matrix(data, m, n).fill_(True)
    for key in ("E", "C", "Z"):
        assert not bool(arrays[key][~data].ne(0).any()), key
    assert data[:(m + n - 1) * r].sum() == m * n


@pytest.mark.parametrize("m,n,w", [(40, 9, 8), (9, 40, 8), (33, 20, 4), (1, 25, 3), (25, 1, 3), (30, 30, 7)])
def test_orientation_choice(m, n, w):
    """Sec. 5's orientation choice: the transposed problem (X^T under B^T,
    A^T, factors U^T and L^T, i.e. the mirror buffer D = E U) rounds to the
    transpose of the same Z (Theorem 1; the oracle's replay passes in both
    orientations), and "auto" picks the one with fewer skew cells."""
    p = wl.random_problem(m, n, 4, "f64", "general")
    X, A, B = p.widened()
    L, lamL, U, lamU = oracle.factors(A, B)
    # the transposed problem's factors are the transposed factors
    Lt, _, Ut, _ = oracle.factors(B.T.copy(), A.T.copy())
    assert np.abs(Lt - U.T).max() <= 1e-10 * max(1.0, np.abs(U).max())
    assert np.abs(Ut - L.T).max() <= 1e-10 * max(1.0, np.abs(L).max())
    args = (torch.from_numpy(X), torch.from_numpy(L), torch.from_numpy(U))
    Zr, Yr, Er = ab.blocked_sweep_oriented(*args, w=w, orient="rows")
    Zc, Yc, Ec = ab.blocked_sweep_oriented(*args, w=w, orient="columns")
    for Z in (Zr, Zc):
        Zo, Yo, c, hard = oracle.round_nested(X, L, U, hint=Z.numpy().astype(np.int32), tau=1e-12)
        assert c["hard"] == 0 and c["range"] == 0 and c["window"] <= 1, c
    assert int((Zr != Zc).sum()) <= 1
    assert float((Yr - Yc).abs().max()) <= 1e-9 * max(1.0, float(Yr.abs().max()))
    Za, _, _ = ab.blocked_sweep_oriented(*args, w=w, orient="auto")
    assert torch.equal(Za, Zc if m > n else Zr)
    assert ab.skew_cells(min(m, n), max(m, n)) <= ab.skew_cells(m, n)


# ---- the implicit-Y form (Appendix B, Algorithm 6) with tensor operations

@pytest.mark.parametrize("m,n,kind,rows", [(1, 1, "wishart", None), (5, 7, "wishart", None), (33, 20, "general", 4),
                                           (64, 70, "wishart", None), (100, 3, "general", 2), (3, 60, "diag", None)])
def test_implicit_sweep_matches_oracle(m, n, kind, rows):
    """Only C = L E is kept and Y_ij = X_ij + C_i,1:j U_1:j,j is read on demand:
    the same Z under the oracle's replay, Y to 1e-12, Z - X = L E U, and the
    same Z as the oracle's own Algorithm 6 and the blocked form; anti-diagonals
    split into pieces of `rows` entries give the same result."""
    p = wl.random_problem(m, n, 5, "f64", kind)
    X, A, B = p.widened()
    L, lamL, U, lamU = oracle.factors(A, B)
    Zt, Yt, Et = ab.implicit_sweep(torch.from_numpy(X), torch.from_numpy(L), torch.from_numpy(U), rows=rows)
    Z, Y, E = Zt.numpy(), Yt.numpy(), Et.numpy()
    Zo, Yo, c, hard = oracle.round_nested(X, L, U, hint=Z.astype(np.int32), tau=1e-12)
    assert c["hard"] == 0 and c["window"] == 0 and c["range"] == 0, c
    assert np.abs(Y - Yo).max() <= 1e-12 * max(1.0, np.abs(Yo).max())
    assert np.abs((Z - X) - L @ E @ U).max() <= 1e-11 * max(1.0, np.abs(X).max())
    Zi, _, _, _ = oracle.round_implicit(X, L, U)
    assert np.array_equal(Zi, Z.astype(np.int32))
    Zb, _, _ = ab.blocked_sweep(torch.from_numpy(X), torch.from_numpy(L), torch.from_numpy(U), w=8)
    assert torch.equal(Zb, Zt)
