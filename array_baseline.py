"""The paper's own array-framework realisation of the sweep, as a comparison
point for the HIP path (it is not part of that path and nothing in the
library calls it).

Blocked GPTQ-2D (Sec. 4.3, Algorithm 4) written with PyTorch tensor
operations, on any device: blocks of w consecutive anti-diagonals; inside a
block every anti-diagonal is rounded in parallel with the fold and both
pushes clipped at the block's last anti-diagonal (Algorithm 3 restricted to
the block); after the block, the down flush (the band of E through L, which
also completes C = L E below the block) and the right flush (the band of C
through U) reach every later entry as batched matrix-vector products over
windows of w columns of L and w rows of U that shift with the receiving
column or row. Indices are 0-based: anti-diagonal s holds the entries
i + j = s, s = 0 .. m + n - 2.

blocked_sweep keeps the natural layout and addresses anti-diagonals by index
tensors; blocked_sweep_skew keeps the working matrices in the padded skew
layout of Sec. 5, where every access is a fixed-stride slice;
blocked_sweep_oriented adds Sec. 5's orientation choice (the transposed
problem, whose buffer is the mirror D = E U of Appendix B); implicit_sweep
is the implicit-Y form of Appendix B (Algorithm 6), which keeps only C = L E.

Ties of the rounding go to even (torch.round), as in the library and the
oracle. The factors are inputs: L unit lower (m x m) and U unit upper
(n x n) of the inverse Grams, with L_ii = U_jj = 1.
"""
from __future__ import annotations

import torch


def _diag_rows(m: int, n: int, s: int, device):
    lo, hi = max(0, s - n + 1), min(s, m - 1)
    return torch.arange(lo, hi + 1, device=device)


def blocked_sweep(X: torch.Tensor, L: torch.Tensor, U: torch.Tensor, w: int = 16,
                  col_chunk: int | None = None):
    """Z (rounded values, X's dtype), Y (corrected values) and E = Z - Y of
    Algorithm 4 with block width w. col_chunk bounds the columns (rows) whose
    flush windows are gathered at once (memory: col_chunk * max(m, n) * w
    values)."""
    m, n = X.shape
    dev, dt = X.device, X.dtype
    Y = X.clone()
    C = torch.zeros_like(X)
    E = torch.zeros_like(X)
    Z = torch.zeros_like(X)
    S = m + n - 1
    chunk = col_chunk or max(1, (1 << 25) // (max(m, n) * w))
    ar_w = torch.arange(w, device=dev)
    # zero-padded factors so that every window of w columns (rows) exists
    Lp = torch.zeros((m, m + 2 * w), dtype=dt, device=dev)
    Lp[:, w:w + m] = L
    Up = torch.zeros((n + 2 * w, n), dtype=dt, device=dev)
    Up[w:w + n, :] = U
    Ep = torch.zeros((m + 2 * w, n), dtype=dt, device=dev)  # E with w zero rows above and below
    Cp = torch.zeros((m, n + 2 * w), dtype=dt, device=dev)  # C with w zero columns left and right
    ii = torch.arange(m, device=dev)[:, None]
    jj = torch.arange(n, device=dev)[None, :]
    for s0 in range(0, S, w):
        s1 = min(s0 + w - 1, S - 1)
        # ---- inside the block: Algorithm 3 with the fold and pushes clipped at s1
        for s in range(s0, s1 + 1):
            I = _diag_rows(m, n, s, dev)
            J = s - I
            y = Y[I, J]
            z = torch.round(y)
            e = z - y
            Z[I, J] = z
            E[I, J] = e
            D = s1 - s  # rows i .. i + D (columns j .. j + D) stay inside the block
            R = I[:, None] + torch.arange(D + 1, device=dev)[None, :]
            ok = R < m
            Rc = torch.where(ok, R, torch.zeros_like(R))
            M = torch.where(ok, L[Rc, I[:, None]] * e[:, None], torch.zeros((), dtype=dt, device=dev))
            Jb = J[:, None].expand_as(R)
            C.index_put_((Rc[ok], Jb[ok]), M[ok], accumulate=True)  # fold (L_ii = 1: C_ij gets E_ij)
            if D > 0:
                ok1 = ok[:, 1:]
                Y.index_put_((Rc[:, 1:][ok1], Jb[:, 1:][ok1]), M[:, 1:][ok1], accumulate=True)  # push down
                Q = J[:, None] + 1 + torch.arange(D, device=dev)[None, :]
                okq = Q < n
                Qc = torch.where(okq, Q, torch.zeros_like(Q))
                cij = C[I, J]
                V = cij[:, None] * U[J[:, None], Qc]
                Ib = I[:, None].expand_as(Q)
                Y.index_put_((Ib[okq], Qc[okq]), V[okq], accumulate=True)  # push right
        if s1 == S - 1:
            break
        later = (ii + jj) > s1
        # ---- down flush: M_ij = sum over the block rows r = s0-j .. s1-j of L_ir E_rj
        Ep[w:w + m, :] = torch.where((ii + jj >= s0) & (ii + jj <= s1), E, torch.zeros((), dtype=dt, device=dev))
        M = torch.empty_like(X)
        for c0 in range(0, n, chunk):
            js = torch.arange(c0, min(n, c0 + chunk), device=dev)
            r0 = s0 - js  # first block row of column j (may be negative)
            # rows outside the matrix land in the zero padding (clamped there)
            cols = (r0[:, None] + ar_w[None, :] + w).clamp(0, m + 2 * w - 1)
            Lw = Lp[:, cols]                              # m x nj x w: the shifting windows of L
            Ew = Ep[cols, js[:, None]]                    # nj x w
            M[:, js] = torch.bmm(Lw.permute(1, 0, 2).contiguous(), Ew[:, :, None].contiguous())[:, :, 0].T
        M = torch.where(later, M, torch.zeros((), dtype=dt, device=dev))
        C += M
        Y += M
        # ---- right flush: Y_ij += sum over the block columns t = s0-i .. s1-i of C_it U_tj
        Cp[:, w:w + n] = torch.where((ii + jj >= s0) & (ii + jj <= s1), C, torch.zeros((), dtype=dt, device=dev))
        for r0_ in range(0, m, chunk):
            is_ = torch.arange(r0_, min(m, r0_ + chunk), device=dev)
            t0 = s0 - is_
            rows = (t0[:, None] + ar_w[None, :] + w).clamp(0, n + 2 * w - 1)
            Uw = Up[rows, :]                              # ni x w x n: the shifting windows of U
            Cw = Cp[is_[:, None], rows]                   # ni x w
            V = torch.bmm(Cw[:, None, :].contiguous(), Uw.contiguous())[:, 0, :]
            Y[is_, :] += torch.where(later[is_, :], V, torch.zeros((), dtype=dt, device=dev))
    return Z, Y, E


def skew_stride(m: int, n: int) -> int:
    """Row stride r = 2m + n - 2 of the padded skew array (Sec. 5): m - 1
    positions on either side of the n-wide band, where a matrix row line
    (stride r + 1) overhangs at its ends."""
    return 2 * m + n - 2


def skew_matrix(flat: torch.Tensor, m: int, n: int) -> torch.Tensor:
    """The m x n matrix held in a padded skew array, as a strided view: entry
    (i, j) sits in row s = i + j at position m - 1 + j, i.e. at
    i r + (m - 1) + j (r + 1) (Sec. 5, the construction)."""
    r = skew_stride(m, n)
    return flat.as_strided((m, n), (r, r + 1), m - 1)


def blocked_sweep_skew(X: torch.Tensor, L: torch.Tensor, U: torch.Tensor, w: int = 16,
                       col_chunk: int | None = None, arrays: dict | None = None):
    """Algorithm 4 with Y, Z, C and E in the padded skew layout of Sec. 5.

    Every access of the sweep is a slice with fixed strides: anti-diagonal s
    is a contiguous piece of row s; the fold and the push down go to the
    rows below it at the same positions (strides r, 1) and the push right
    one position further per row (strides r + 1, 1); the down flush reads
    each matrix column's window of w anti-diagonals of E as a stride-r line
    and the right flush each matrix row's window of C as a stride-(r + 1)
    line. Index ranges outside the matrix are skipped (their updates are
    zero), so the padding cells stay zero and the flush windows read zeros
    there. Returns Z, Y, E as m x n matrices; the same values as
    blocked_sweep, which keeps the natural layout and addresses
    anti-diagonals by index tensors. If arrays is a dict, it receives the
    flat skew arrays ("Y", "Z", "C", "E")."""
    m, n = X.shape
    dev, dt = X.device, X.dtype
    r = skew_stride(m, n)
    S = m + n - 1
    # rows beyond the last anti-diagonal absorb the zero updates of pushes
    # that leave the matrix past its last rows or columns
    size = (S + w + 1) * r
    Yf = torch.zeros(size, dtype=dt, device=dev)
    Cf = torch.zeros_like(Yf)
    Ef = torch.zeros_like(Yf)
    Zf = torch.zeros_like(Yf)
    Yd, Cd, Ed, Zd = (skew_matrix(t, m, n) for t in (Yf, Cf, Ef, Zf))
    Yd.copy_(X)
    chunk = col_chunk or max(1, (1 << 25) // (max(m, n) * w))
    ar_w = torch.arange(w, device=dev)
    Lp = torch.zeros((m, m + 2 * w), dtype=dt, device=dev)
    Lp[:, w:w + m] = L
    Up = torch.zeros((n + 2 * w, n), dtype=dt, device=dev)
    Up[w:w + n, :] = U
    ii = torch.arange(m, device=dev)[:, None]
    jj = torch.arange(n, device=dev)[None, :]
    zero = torch.zeros((), dtype=dt, device=dev)
    for s0 in range(0, S, w):
        s1 = min(s0 + w - 1, S - 1)
        for s in range(s0, s1 + 1):
            jlo, jhi = max(0, s - m + 1), min(s, n - 1)
            nt = jhi - jlo + 1
            base = s * r + m - 1 + jlo  # anti-diagonal s: Yf[base : base + nt], column j = jlo + t
            J = torch.arange(jlo, jhi + 1, device=dev)
            I = s - J
            y = Yf[base:base + nt]
            z = torch.round(y)
            e = z - y
            Zf[base:base + nt] = z
            Ef[base:base + nt] = e
            D = s1 - s
            d = torch.arange(D + 1, device=dev)[:, None]
            R = I[None, :] + d  # target rows i + d (rows of the view)
            ok = R < m
            M = torch.where(ok, L[torch.where(ok, R, 0), I[None, :]] * e[None, :], zero)
            # fold (d = 0: C_ij gets E_ij, L_ii = 1) and push down: the rows below, same positions
            Cf.as_strided((D + 1, nt), (r, 1), base).add_(M)
            if D > 0:
                Yf.as_strided((D, nt), (r, 1), base + r).add_(M[1:])
                Q = J[None, :] + d[1:]  # target columns j + d
                okq = Q < n
                V = torch.where(okq, Cf[base:base + nt][None, :] * U[J[None, :], torch.where(okq, Q, 0)], zero)
                # push right: one position further per row below
                Yf.as_strided((D, nt), (r + 1, 1), base + r + 1).add_(V)
        if s1 == S - 1:
            break
        wb = s1 - s0 + 1
        later = (ii + jj) > s1
        # ---- down flush: column j's window of the block, E(s0 + d - j, j), d < wb
        E2 = Ef.as_strided((n, wb), (1, r), s0 * r + m - 1)
        M = torch.empty((m, n), dtype=dt, device=dev)
        for c0 in range(0, n, chunk):
            js = torch.arange(c0, min(n, c0 + chunk), device=dev)
            # rows outside the matrix land in the zero padding (clamped there)
            cols = ((s0 - js)[:, None] + ar_w[None, :wb] + w).clamp(0, m + 2 * w - 1)
            Lw = Lp[:, cols]  # m x nj x wb: the shifting windows of L
            M[:, js] = torch.bmm(Lw.permute(1, 0, 2).contiguous(), E2[js][:, :, None].contiguous())[:, :, 0].T
        M = torch.where(later, M, zero)
        Cd.add_(M)
        Yd.add_(M)
        # ---- right flush: row i's window of the block, C(i, s0 - i + d), read
        # as the stride-(r + 1) lines in reverse row order and flipped back
        Cw = Cf.as_strided((m, wb), (1, r + 1), s0 * (r + 1)).flip(0)
        for r0_ in range(0, m, chunk):
            is_ = torch.arange(r0_, min(m, r0_ + chunk), device=dev)
            rows = ((s0 - is_)[:, None] + ar_w[None, :wb] + w).clamp(0, n + 2 * w - 1)
            Uw = Up[rows, :]  # ni x wb x n: the shifting windows of U
            V = torch.bmm(Cw[is_][:, None, :].contiguous(), Uw.contiguous())[:, 0, :]
            Yd[is_, :] += torch.where(later[is_, :], V, zero)
    if arrays is not None:
        arrays.update(Y=Yf, Z=Zf, C=Cf, E=Ef)
    return Zd.clone(), Yd.clone(), Ed.clone()


def skew_cells(m: int, n: int) -> int:
    """Cells of one padded skew array: (m + n - 1)(2m + n - 2) for m n entries."""
    return (m + n - 1) * skew_stride(m, n)


def blocked_sweep_oriented(X: torch.Tensor, L: torch.Tensor, U: torch.Tensor, w: int = 16,
                           orient: str = "auto", col_chunk: int | None = None):
    """Algorithm 4 on the skew layout in the orientation Sec. 5 suggests:
    rounding X^T under the swapped bases (B^T, A^T) is the same problem, with
    feedback factors U^T (rows) and L^T (columns), and its skew arrays need
    (m + n - 1)(2n + m - 2) cells instead of (m + n - 1)(2m + n - 2), fewer when
    m > n. orient "auto" takes the orientation with the smaller first
    dimension, "rows" keeps X, "columns" transposes. In the transposed sweep
    the buffer is U^T E^T = (E U)^T: the right-hand buffer D = E U of
    Appendix B, kept by rows instead of C = L E by columns. Returns Z, Y, E of
    X (transposed back)."""
    m, n = X.shape
    if orient not in ("auto", "rows", "columns"):
        raise ValueError(f"orient must be auto, rows or columns, not {orient!r}")
    flip = orient == "columns" or (orient == "auto" and m > n)
    if not flip:
        return blocked_sweep_skew(X, L, U, w=w, col_chunk=col_chunk)
    Zt, Yt, Et = blocked_sweep_skew(X.T.contiguous(), U.T.contiguous(), L.T.contiguous(), w=w,
                                    col_chunk=col_chunk)
    return Zt.T.contiguous(), Yt.T.contiguous(), Et.T.contiguous()


def implicit_sweep(X: torch.Tensor, L: torch.Tensor, U: torch.Tensor, rows: int | None = None):
    """The implicit-Y form of Appendix B (Algorithm 6) with tensor operations:
    only the buffer C = L E is kept. For every entry (i, j) of anti-diagonal
    s at once, Y_ij = X_ij + C_i,1:j U_1:j,j, a row of C against a column of
    U (U is unit upper, so the full row product is that prefix sum), then the
    rounding; then each rounded entry adds L_i:m,i E_ij to column j of C (L is
    unit lower: the full column is that suffix). Two batched products per
    anti-diagonal, O(mn max(m, n)) in all. rows bounds the entries of an
    anti-diagonal handled at once (memory: rows * max(m, n) values). Returns
    Z, Y, E."""
    m, n = X.shape
    dev, dt = X.device, X.dtype
    C = torch.zeros_like(X)
    Z = torch.zeros_like(X)
    Y = torch.zeros_like(X)
    E = torch.zeros_like(X)
    step = rows or max(1, (1 << 24) // max(m, n))
    for s in range(m + n - 1):
        jlo, jhi = max(0, s - m + 1), min(s, n - 1)
        for a in range(jlo, jhi + 1, step):
            J = torch.arange(a, min(jhi, a + step - 1) + 1, device=dev)
            I = s - J
            y = X[I, J] + (C[I, :] * U[:, J].T).sum(dim=1)
            z = torch.round(y)
            Z[I, J] = z
            Y[I, J] = y
            E[I, J] = z - y
        # the column updates after the whole anti-diagonal is rounded (the
        # entries of one anti-diagonal read none of each other's updates)
        J = torch.arange(jlo, jhi + 1, device=dev)
        I = s - J
        C[:, J] += L[:, I] * E[I, J][None, :]
    return Z, Y, E
