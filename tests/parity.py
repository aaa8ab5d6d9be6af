"""Helpers of the GPU parity tests: run the library through its C ABI and
judge the result against the oracle with the synchronised-replay rule.

Rule (for every run): the oracle replays the sweep with the GPU's Z as hints.
An entry where the oracle would round the other way counts as a "window"
entry if the oracle's value lies within tau of the half-integer between the
two candidates (tau = 1e-6 for fp32 inputs, 1e-12 for fp64), otherwise as a
hard mismatch. Pass: no hard mismatch and at most 1e-4 of all entries in the
window. The objective agrees to 1e-5 (fp32) or 1e-10 (fp64) relative.
"""
import numpy as np
import torch

import oracle
from paper_2607_27042_amd import binding

TAU = {"f32": 1e-6, "f64": 1e-12}
OBJ_RTOL = {"f32": 1e-5, "f64": 1e-10}
TORCH_DT = {"f32": torch.float32, "f64": torch.float64}


def to_dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def gpu_run(prob, factors=None, want_y=True, reverse=False):
    """Factor (or import ``factors`` = (L, lamL, U, lamU) numpy fp64) and
    round on the GPU, in reverse order if ``reverse`` (the factors are then
    those of the index-reversed problem). Returns a dict of numpy results."""
    X = to_dev(prob.X)
    if factors is None:
        f = binding.Factors.from_bases(to_dev(prob.A), to_dev(prob.B), reverse=reverse)
    else:
        L, lamL, U, lamU = factors
        f = binding.Factors(prob.m, prob.n, reverse=reverse)
        f.load(to_dev(L), to_dev(U), to_dev(lamL), to_dev(lamU))
    Z, Y, obj = binding.round_matrix(f, X, want_y=want_y)
    L, U, lamL, lamU = f.export()
    torch.cuda.synchronize()
    out = {
        "Z": Z.cpu().numpy(),
        "Y": None if Y is None else Y.cpu().numpy().astype(np.float64),
        "obj": float(obj.cpu()[0]),
        "L": L.cpu().numpy(), "U": U.cpu().numpy(),
        "lamL": lamL.cpu().numpy(), "lamU": lamU.cpu().numpy(),
    }
    f.close()
    return out


def replay(prob, L, U, Zg, corner=None):
    """Oracle replay (Algorithm 5) of the GPU's Z under factors L, U."""
    X = prob.X.astype(np.float64)
    tau = TAU[prob.dtype]
    if corner is None:
        Zo, Yo, c, hard = oracle.round_nested(X, L, U, hint=Zg, tau=tau)
    else:
        m1, n1 = corner
        Zo, Yo, c, hard = oracle.round_nested_corner(X, L, U, m1, n1,
                                                     hint=np.ascontiguousarray(Zg[:m1, :n1]), tau=tau)
    return Zo, Yo, c, hard


def assert_replay_pass(prob, c, hard, entries):
    assert c["range"] == 0
    assert c["hard"] == 0, f"{prob.name}: {c['hard']} hard mismatches, first at {hard[:8]}"
    assert c["window"] <= 1e-4 * entries, f"{prob.name}: {c['window']} window entries"


def assert_objective(prob, obj_gpu, obj_ref):
    rel = abs(obj_gpu - obj_ref) / max(abs(obj_ref), 1e-300)
    assert rel <= OBJ_RTOL[prob.dtype], f"{prob.name}: objective rel err {rel:.3e}"


def property_checks(prob, res, nprobe=2, seed=0):
    """Properties that hold at any size: |E| <= 1/2, Z = rint(Y) for the
    fp64 values, and Z - X = L E U with E = Z - Y (Eq. Y-LEU), probed with
    random vectors. For fp32 runs Y comes back rounded to fp32, so the bounds
    carry that rounding."""
    Z = res["Z"].astype(np.float64)
    Y = res["Y"]
    E = Z - Y
    assert np.abs(E).max() <= 0.5 + (0 if prob.dtype == "f64" else 1e-5)
    X = prob.X.astype(np.float64)
    L, U = res["L"], res["U"]
    rng = np.random.default_rng(seed)
    for _ in range(nprobe):
        v = rng.standard_normal(prob.n)
        lhs = (Z - X) @ v
        rhs = L @ (E @ (U @ v))
        scale = np.abs(L).max() * np.abs(U).max() * np.sqrt(prob.m * prob.n) * np.abs(v).max()
        tol = 1e-9 if prob.dtype == "f64" else 1e-5
        assert np.abs(lhs - rhs).max() <= tol * scale


def widened_run(prob, reverse=False):
    """The F64 entry points on the exactly widened inputs of an fp32 problem:
    the library computes in fp64 either way, so Z and the factors must be the
    fp32 run's bit for bit, and Y comes back unrounded."""
    X, A, B = prob.widened()
    import paper_2607_27042_amd.workloads as wl
    return gpu_run(wl.Problem(prob.name + "_w64", X, A, B, "f64"), reverse=reverse)


def assert_same_run(res32, res64):
    """An fp32 run and the F64 run on its widened inputs agree bit for bit
    (Y up to the fp32 rounding of the returned values)."""
    assert np.array_equal(res32["Z"], res64["Z"]), "Z differs between the F32 and the widened F64 run"
    for k in ("L", "U", "lamL", "lamU"):
        assert np.array_equal(res32[k], res64[k]), f"{k} differs between the F32 and F64 runs"
    assert np.array_equal(res32["Y"].astype(np.float32), res64["Y"].astype(np.float32))
    assert res32["obj"] == res64["obj"]


def assert_trajectory(prob, res, dev_tol=1e-9):
    """Every entry of a full result against the oracle's definition of the
    trajectory (Eq. Y-LEU): with E = Z - Y, the value each entry is rounded
    from is Y' = X + L E U - E, Y must equal Y' to dev_tol, and Z = rint(Y')
    everywhere except window entries (within tau of a tie), at most 1e-4 of
    all entries. res["Y"] must be the unrounded fp64 values."""
    X = prob.X.astype(np.float64)
    dev, c, hard = oracle.trajectory_check(X, res["L"], res["U"], res["Z"], res["Y"], TAU[prob.dtype])
    print(f"[trajectory] {prob.name}: max |Y' - Y| = {dev:.3e}, window {c['window']}, hard {c['hard']}",
          flush=True)
    assert dev <= dev_tol, f"{prob.name}: |Y' - Y| = {dev:.3e}"
    assert c["hard"] == 0, f"{prob.name}: {c['hard']} hard mismatches, first at {hard[:8]}"
    assert c["window"] <= 1e-4 * X.size, f"{prob.name}: {c['window']} window entries"
