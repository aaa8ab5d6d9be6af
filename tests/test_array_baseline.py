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
