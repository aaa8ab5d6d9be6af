"""The paper's array-framework realisation of the sweep (Sec. 4.3, Algorithm 4;
array_baseline.py, the comparison point timed by bench.py --array-baseline),
in the natural layout and in the padded skew layout of Sec. 5, and the
implicit-Y form of Appendix B (Algorithm 6), run on the GPU: its Z passes the oracle's replay (Algorithm 5) and equals the HIP
library's Z on the same problem and the same factors. The two share no code:
one is batched PyTorch tensor operations, the other the library's kernels
through the C ABI."""
import numpy as np
import pytest
import torch

import array_baseline as ab
import oracle
from paper_2607_27042_amd import workloads as wl

import parity as pr

pytestmark = pytest.mark.gpu


# block widths from 1 to wider than the matrix; ragged shapes
@pytest.mark.parametrize("m,n,w,kind", [(64, 64, 16, "wishart"), (100, 90, 8, "general"),
                                        (130, 70, 32, "wishart"), (37, 150, 1, "general"),
                                        (70, 60, 200, "wishart")])
@pytest.mark.parametrize("layout", ["natural", "skew", "implicit"])
def test_array_baseline_on_device(m, n, w, kind, layout):
    p = wl.random_problem(m, n, 11, "f64", kind)
    X, A, B = p.widened()
    L, lamL, U, lamU = oracle.factors(A, B)
    dev = torch.device("cuda")
    args = (torch.from_numpy(X).to(dev), torch.from_numpy(L).to(dev), torch.from_numpy(U).to(dev))
    if layout == "implicit":  # Algorithm 6 (Appendix B): no blocks, only C = L E kept
        Zt, Yt, Et = ab.implicit_sweep(*args)
    else:
        sweep = ab.blocked_sweep if layout == "natural" else ab.blocked_sweep_skew
        Zt, Yt, Et = sweep(*args, w=w)
    torch.cuda.synchronize()
    Z = Zt.cpu().numpy()
    Y = Yt.cpu().numpy()
    E = Et.cpu().numpy()
    print(f"[array baseline on the device] {m} x {n}, w = {w}, {kind}, {layout} layout", flush=True)
    Zo, Yo, c, hard = oracle.round_nested(X, L, U, hint=Z.astype(np.int32), tau=1e-12)
    assert c["hard"] == 0 and c["window"] == 0 and c["range"] == 0, c
    assert np.abs(Y - Yo).max() <= 1e-12 * max(1.0, np.abs(Yo).max())
    assert np.abs(E).max() <= 0.5
    # the library on the oracle's factors: the same rounding, entry by entry
    res = pr.gpu_run(p, factors=(L, lamL, U, lamU))
    assert np.array_equal(res["Z"], Z.astype(np.int32))
    assert np.abs(res["Y"] - Y).max() <= 1e-12 * max(1.0, np.abs(Y).max())
