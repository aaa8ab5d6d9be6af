"""Plain-numpy model of the GPU decomposition of the sweep (test helper).

It mirrors what the HIP kernels do -- 64 x 64 tiles swept one tile
anti-diagonal per launch, Algorithm 3 inside each tile, the two immediate
predecessors pulled by the sweeping tile, and every older contribution
delivered by the library's own task plan (``gptq2d_schedule_tasks``) -- so
that the blocking and the delivery plan can be checked against the oracle on
the CPU. It is NOT the oracle and is never used as one.
"""
import numpy as np

from paper_2607_27042_amd import binding

T = 64


def _pad(M, rows, cols, identity=False):
    out = np.eye(rows, cols) if identity else np.zeros((rows, cols))
    out[: M.shape[0], : M.shape[1]] = M
    return out


def tile_model_round(X, L, U, g=4):
    m, n = X.shape
    mp, np_ = -(-m // T) * T, -(-n // T) * T
    MT, NT = mp // T, np_ // T
    Xp, Lp, Up = _pad(X, mp, np_), _pad(L, mp, mp, True), _pad(U, np_, np_, True)
    P = np.zeros((mp, np_))
    R = np.zeros((mp, np_))
    E = np.zeros((mp, np_))
    C = np.zeros((mp, np_))
    Yo = np.zeros((mp, np_))
    tasks, offs = binding.gptq2d_schedule_tasks(m, n, g)

    def blk(i):
        return slice(i * T, (i + 1) * T)

    for k in range(MT + NT - 1):
        for x, ti, tj, w in tasks[offs[k]:offs[k + 1]]:
            d, ow = x & 1, (x >> 1) & 1
            nr, nc = ((x >> 2) & 1) + 1, ((x >> 3) & 1) + 1
            src = slice((w & 0xFFFF) * T, (w >> 16) * T)
            rows = slice(ti * T, (ti + nr) * T)
            cols = slice(tj * T, (tj + nc) * T)
            if d == 0:
                v = Lp[rows, src] @ E[src, cols]
                P[rows, cols] = v if ow else P[rows, cols] + v
            else:
                v = C[rows, src] @ Up[src, cols]
                R[rows, cols] = v if ow else R[rows, cols] + v
        for I in range(max(0, k - NT + 1), min(k, MT - 1) + 1):
            J = k - I
            Dn = np.zeros((T, T))
            Rt = Xp[blk(I), blk(J)].copy()
            if I >= 1:
                Dn += Lp[blk(I), blk(I - 1)] @ E[blk(I - 1), blk(J)]
            if I >= 2:
                Dn += P[blk(I), blk(J)]
            if J >= 1:
                Rt += C[blk(I), blk(J - 1)] @ Up[blk(J - 1), blk(J)]
            if J >= 2:
                Rt += R[blk(I), blk(J)]
            Lt, Ut = Lp[blk(I), blk(I)], Up[blk(J), blk(J)]
            yt, ct, et = np.zeros((T, T)), np.zeros((T, T)), np.zeros((T, T))
            for s in range(2 * T - 1):
                act = [(i, s - i) for i in range(max(0, s - T + 1), min(s, T - 1) + 1)]
                for i, j in act:
                    y = Rt[i, j] + Dn[i, j]
                    z = np.rint(y)
                    e = z - y
                    yt[i, j], et[i, j], ct[i, j] = y, e, Dn[i, j] + e
                for i, j in act:
                    Dn[i + 1:, j] += Lt[i + 1:, i] * et[i, j]
                    Rt[i, j + 1:] += ct[i, j] * Ut[j, j + 1:]
            E[blk(I), blk(J)] = et
            C[blk(I), blk(J)] = ct
            Yo[blk(I), blk(J)] = yt
    Y = Yo[:m, :n]
    return np.rint(Y).astype(np.int32), Y
