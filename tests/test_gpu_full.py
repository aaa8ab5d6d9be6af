"""GPU parity at the full sizes of the five synthetic workloads.

At these sizes the oracle cannot replay a whole sweep in test time, so each
run is judged on what the oracle can compute exactly and on properties that
hold at any size:

- the leading 1280 x 1280 block of the sweep is self-contained (an entry only
  depends on entries above and to the left of it), so the oracle replays that
  corner with the GPU's own factors and the GPU's Z as hints, under the same
  window rule as the small cases;
- every rounding error satisfies |E| <= 1/2 and Z - X = L E U (Eq. Y-LEU),
  probed with random vectors over the whole matrix;
- the factors satisfy L^T G L = Lambda_L^{-1} and U H U^T = Lambda_U^{-1}
  (the LDL factorisations of the inverse Grams, Sec. 3.1), probed with random
  vectors through A and B, never forming G or H;
- the objective reported by the GPU equals ||A (Z - X) B||_F^2 evaluated by
  its definition in fp64 (Eq. objective), to 1e-5 (fp32) / 1e-10 (fp64).
"""
import numpy as np
import pytest

from paper_2607_27042_amd import workloads as wl

import parity as pr

pytestmark = pytest.mark.gpu

CORNER = 1280


def _factor_residual(M, F, lam, left, nprobe=3, seed=1):
    """max relative residual of F^T (M^T M) F = diag(1/lam) (left) or
    F (M M^T) F^T = diag(1/lam) (right), probed with random vectors."""
    rng = np.random.default_rng(seed)
    worst = 0.0
    for _ in range(nprobe):
        v = rng.standard_normal(F.shape[0])
        if left:
            r = F.T @ (M.T @ (M @ (F @ v)))
        else:
            r = F @ (M @ (M.T @ (F.T @ v)))
        ref = v / lam
        worst = max(worst, np.linalg.norm(r - ref) / np.linalg.norm(ref))
    return worst


@pytest.mark.parametrize("k,dtype", [(3, "f32"), (4, "f32"), (5, "f32"), (5, "f64")],
                         ids=["c3_f32", "c4_f32", "c5_f32", "c5_f64"])
def test_full_size_config(k, dtype):
    p = wl.make_config(k, dtype)
    print(f"[full] {p.name}: GPU factor + sweep", flush=True)
    res = pr.gpu_run(p)
    X, A, B = p.widened()

    # P2 on the self-contained leading corner
    m1, n1 = min(CORNER, p.m), min(CORNER, p.n)
    Zo, Yo, c, hard = pr.replay(p, res["L"], res["U"], res["Z"], corner=(m1, n1))
    pr.assert_replay_pass(p, c, hard, m1 * n1)

    # properties over the whole matrix
    pr.property_checks(p, res)

    # factors: LDL of the inverse Grams
    assert _factor_residual(A, res["L"], res["lamL"], left=True) <= 1e-9
    assert _factor_residual(B, res["U"], res["lamU"], left=False) <= 1e-9

    # objective by its definition
    D = res["Z"].astype(np.float64) - X
    obj_def = float(np.linalg.norm((A @ D) @ B) ** 2)
    pr.assert_objective(p, res["obj"], obj_def)
