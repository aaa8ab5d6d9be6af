"""GPU parity: the HIP path through the C ABI against the oracle.

P1 -- the GPU factors against the oracle's (explicit inverse + LDL).
P2 -- the GPU sweep, replayed by the oracle with the GPU's exported factors
      (bit-identical factor data, no shared code).
P3 -- end to end: the oracle's own factors.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_27042_amd import binding, workloads as wl

import parity as pr

pytestmark = pytest.mark.gpu

SHAPES = [(1, 1), (1, 100), (100, 1), (5, 7), (63, 65), (64, 64), (65, 64), (130, 200),
          (200, 130), (256, 320)]


def _factor_close(got, ref, tol):
    err = np.abs(got - ref).max() / max(1.0, np.abs(ref).max())
    assert err <= tol, err


# (384, 128) and (640, 384): Gram tiles split between two work groups, ranges
# across the two sides; (320, 512): only the second side on 128-wide tiles
@pytest.mark.parametrize("m,n", [(1, 1), (5, 7), (63, 65), (130, 200), (256, 320), (384, 128), (600, 520),
                                 (640, 384), (320, 512)])
@pytest.mark.parametrize("dtype", ["f64", "f32"])
def test_factors_match_oracle(m, n, dtype):
    p = wl.random_problem(m, n, 1, dtype, "wishart")
    res = pr.gpu_run(p)
    X, A, B = p.widened()
    L, lamL, U, lamU = oracle.factors(A, B)
    _factor_close(res["L"], L, 1e-10)
    _factor_close(res["U"], U, 1e-10)
    np.testing.assert_allclose(res["lamL"], lamL, rtol=1e-10)
    np.testing.assert_allclose(res["lamU"], lamU, rtol=1e-10)
    assert np.array_equal(np.triu(res["L"], 1), np.zeros((m, m)))
    assert np.array_equal(np.diag(res["L"]), np.ones(m))
    assert np.array_equal(np.tril(res["U"], -1), np.zeros((n, n)))


@pytest.mark.parametrize("m,n,decades", [(200, 150, 6), (130, 70, 9)])
def test_ill_conditioned_bases(m, n, decades):
    """Gram matrices whose eigenvalues spread over 10^decades (Eq. GH with
    A^T A = Q diag(ev) Q^T, Q orthogonal). The feedback factors of the inverse
    Grams (Sec. 3.1) are then ill-determined in any fp64 route, so the
    library is held to the spread between fp64 routes: its factors may differ
    from the oracle's (explicit inverse, then LDL) by at most ten times what a
    third route differs by (numpy's Cholesky of the index-reversed Gram and
    its inverse, R = J chol(J Q J) J, F = R^{-T} diag(R)). Several 64 x 64
    diagonal blocks and a ragged last one; the sweep under the library's
    factors then passes the oracle's replay. The library's factors agree with
    the third route to a few units of cond * eps."""
    rng = np.random.default_rng([51, m, n, decades])

    def basis(d):
        Qm, _ = np.linalg.qr(rng.standard_normal((d, d)))
        G = (Qm * np.logspace(-decades, 0, d)) @ Qm.T
        return np.ascontiguousarray(np.linalg.cholesky((G + G.T) / 2).T)

    def third_route(Q):
        d = Q.shape[0]
        Jr = np.eye(d)[::-1]
        R = Jr @ np.linalg.cholesky(Jr @ Q @ Jr) @ Jr
        return np.linalg.inv(R).T @ np.diag(np.diag(R)), np.diag(R) ** -2.0

    A, B = basis(m), basis(n).T.copy()
    X = 3.0 * rng.standard_normal((m, n))
    p = wl.Problem(f"illcond_{m}x{n}_1e{decades}", X, A, B, "f64")
    print(f"[ill-conditioned] {m}x{n}, cond 1e{decades}", flush=True)
    res = pr.gpu_run(p)
    L, lamL, U, lamU = oracle.factors(A, B)
    L3, lamL3 = third_route(A.T @ A)
    F3, lamU3 = third_route(B @ B.T)
    U3 = F3.T
    floor = 100.0 * 10.0 ** decades * np.finfo(np.float64).eps

    def rel(x, ref):
        return np.abs(x - ref).max() / max(1.0, np.abs(ref).max())

    for got, ref, alt in ((res["L"], L, L3), (res["U"], U, U3)):
        assert rel(got, ref) <= 10.0 * max(rel(alt, ref), floor), (rel(got, ref), rel(alt, ref))
        # the two Cholesky routes agree far more closely than either with the
        # explicit inverse (measured 1e-11 at cond 1e6 and 1.4e-8 at 1e9,
        # against 3e-8 and 1.8e-2 from the oracle)
        assert rel(got, alt) <= floor, rel(got, alt)
    for got, ref, alt in ((res["lamL"], lamL, lamL3), (res["lamU"], lamU, lamU3)):
        r_got = np.abs(got / ref - 1.0).max()
        assert r_got <= 10.0 * max(np.abs(alt / ref - 1.0).max(), floor), r_got
    Zo, Yo, c, hard = pr.replay(p, res["L"], res["U"], res["Z"])
    pr.assert_replay_pass(p, c, hard, m * n)


def test_factors_lower_triangular_closed_form():
    """A lower => L = A^{-1} diag(A); B upper => U = diag(B) B^{-1}."""
    import scipy.linalg as sla
    p = wl.random_problem(150, 90, 2, "f64", "lower")
    res = pr.gpu_run(p)
    A, B = p.A, p.B
    _factor_close(res["L"], sla.solve_triangular(A, np.diag(np.diag(A)), lower=True), 1e-11)
    _factor_close(res["U"], np.diag(np.diag(B)) @ sla.solve_triangular(B, np.eye(90)), 1e-11)


def _envelope_bases(kind, m, n, seed):
    """Bases whose Gram panels have the structures the Gram's envelope meets:
    block-diagonal A (128-blocks: every Gram tile off the block diagonal is
    exactly zero) with banded upper B; lower-triangular A with upper B
    (envelopes from opposite ends); dense A and B (the whole range)."""
    rng = np.random.default_rng([77, seed, m, n])

    def chol_block(d):
        W = rng.standard_normal((2 * d, d))
        return np.linalg.cholesky(W.T @ W / (2 * d) + 0.05 * np.eye(d)).T

    def banded(d, bw):
        T = np.triu(rng.standard_normal((d, d)) / np.sqrt(bw))
        T = np.tril(T, bw)
        T[np.diag_indices(d)] = np.exp(rng.uniform(np.log(0.5), np.log(2.0), size=d))
        return T

    if kind == "blockdiag":
        A = np.zeros((m, m))
        for b in range(0, m, 128):
            A[b:b + 128, b:b + 128] = chol_block(128)
        B = banded(n, 100)
    elif kind == "lower":
        A = chol_block(m).T
        B = chol_block(n)
    else:
        A = rng.standard_normal((m, m)) / np.sqrt(m) + 2.0 * np.eye(m)
        B = rng.standard_normal((n, n)) / np.sqrt(n) + 2.0 * np.eye(n)
    X = 3.0 * rng.standard_normal((m, n))
    return wl.Problem(f"envelope-{kind}-{m}x{n}", X, A, B, "f64")


@pytest.mark.parametrize("kind", ["blockdiag", "lower", "general"])
@pytest.mark.parametrize("m,n", [(384, 256), (256, 640)])
def test_gram_envelope_structures(kind, m, n):
    """Fast-path Grams (dimensions multiples of 128) on bases whose panels
    have zero blocks: the factors against the oracle's, the sweep replayed
    under the GPU's factors and the objective against the definition. The
    handle first factors a dense problem, so its Gram buffer holds nonzero
    values; the block-diagonal basis must then give a block-diagonal L (the
    Gram tiles with an empty envelope are written as zeros)."""
    p = _envelope_bases(kind, m, n, 1)
    X, A, B = p.widened()
    dense = _envelope_bases("general", m, n, 2)
    f = binding.Factors(m, n)
    f.compute(pr.to_dev(dense.A), pr.to_dev(dense.B))
    binding.gptq2d_factor_check(f.handle)
    f.compute(pr.to_dev(p.A), pr.to_dev(p.B))
    binding.gptq2d_factor_check(f.handle)
    Z, Y, obj = binding.round_matrix(f, pr.to_dev(p.X))
    Lg, Ug, lamLg, lamUg = (t.cpu().numpy() for t in f.export())
    Zg, Yg, objg = Z.cpu().numpy(), Y.cpu().numpy(), float(obj.cpu()[0])
    f.close()
    L, lamL, U, lamU = oracle.factors(A, B)
    _factor_close(Lg, L, 1e-10)
    _factor_close(Ug, U, 1e-10)
    np.testing.assert_allclose(lamLg, lamL, rtol=1e-10)
    np.testing.assert_allclose(lamUg, lamU, rtol=1e-10)
    if kind == "blockdiag":
        blk = np.arange(m) // 128
        assert np.all(Lg[blk[:, None] != blk[None, :]] == 0.0)
    Zo, Yo, c, hard = pr.replay(p, Lg, Ug, Zg)
    pr.assert_replay_pass(p, c, hard, m * n)
    assert np.abs(Yg - Yo).max() <= 1e-9
    pr.assert_objective(p, objg, oracle.objective(X, Zo, A, B))


@pytest.mark.parametrize("m,n", SHAPES)
@pytest.mark.parametrize("dtype", ["f64", "f32"])
def test_sweep_with_imported_factors(m, n, dtype):
    """The sweep alone: oracle factors imported, replay with the same data."""
    p = wl.random_problem(m, n, 4, dtype, "wishart")
    X, A, B = p.widened()
    fac = oracle.factors(A, B)
    res = pr.gpu_run(p, factors=fac)
    L, lamL, U, lamU = fac
    Zo, Yo, c, hard = pr.replay(p, L, U, res["Z"])
    pr.assert_replay_pass(p, c, hard, m * n)
    tol = 1e-9 if dtype == "f64" else 2e-6 * max(1.0, np.abs(Yo).max())
    assert np.abs(res["Y"] - Yo).max() <= tol
    pr.assert_objective(p, res["obj"], oracle.objective(X, Zo, A, B))


@pytest.mark.parametrize("m,n", SHAPES)
@pytest.mark.parametrize("kind", ["wishart", "general"])
def test_end_to_end(m, n, kind):
    p = wl.random_problem(m, n, 5, "f64", kind)
    X, A, B = p.widened()
    res = pr.gpu_run(p)
    # P2: replay under the GPU's own factors
    Zo, Yo, c, hard = pr.replay(p, res["L"], res["U"], res["Z"])
    pr.assert_replay_pass(p, c, hard, m * n)
    assert np.abs(res["Y"] - Yo).max() <= 1e-9
    # P3: the oracle's own factors
    L, lamL, U, lamU = oracle.factors(A, B)
    Zo3, Yo3, c3, hard3 = pr.replay(p, L, U, res["Z"])
    pr.assert_replay_pass(p, c3, hard3, m * n)
    pr.assert_objective(p, res["obj"], oracle.objective(X, Zo3, A, B))
    pr.property_checks(p, res)


@pytest.mark.parametrize("m,n,dtype", [(1000, 700, "f32"), (700, 1000, "f64"), (2085, 1547, "f32")])
def test_mid_size_full_replay(m, n, dtype):
    """Ragged mid-size problems (16 x 11, 11 x 16 and 33 x 25 tiles: far batches onto
    2 x 2 super-tiles, near deliveries of every shape, edge tiles): the whole
    sweep replayed by the oracle with the GPU's factors, then the oracle's own
    factors and the objective."""
    p = wl.random_problem(m, n, 11, dtype, "wishart")
    X, A, B = p.widened()
    print(f"[mid] {m}x{n} {dtype}: GPU factor + sweep", flush=True)
    res = pr.gpu_run(p)
    Zo, Yo, c, hard = pr.replay(p, res["L"], res["U"], res["Z"])
    pr.assert_replay_pass(p, c, hard, m * n)
    tol = 1e-9 if dtype == "f64" else 2e-6 * max(1.0, np.abs(Yo).max())
    assert np.abs(res["Y"] - Yo).max() <= tol
    L, lamL, U, lamU = oracle.factors(A, B)
    Zo3, Yo3, c3, hard3 = pr.replay(p, L, U, res["Z"])
    pr.assert_replay_pass(p, c3, hard3, m * n)
    pr.assert_objective(p, res["obj"], oracle.objective(X, Zo3, A, B))
    pr.property_checks(p, res)


# (256, 384), (384, 128): both sides' Grams on the 128-wide path (the
# reversal skipped in the panel transpose); the others take the 64-wide path
@pytest.mark.parametrize("m,n,dtype", [(1, 1, "f64"), (5, 7, "f64"), (63, 65, "f32"), (130, 200, "f64"),
                                       (256, 384, "f32"), (384, 128, "f64"), (700, 1000, "f32")])
def test_reverse_order(m, n, dtype):
    """Rounding from the last row and column on (Sec. 2, the direction of
    YAQA): the factors are those of the index-reversed problem (A P, P B), and
    the oracle's reverse-order rounding replays the GPU's Z in X's indexing,
    under the oracle's own factors and under the GPU's."""
    p = wl.random_problem(m, n, 13, dtype, "wishart")
    X, A, B = p.widened()
    Xr, Ar, Br = oracle.reverse_problem(X, A, B)
    print(f"[reverse] {m}x{n} {dtype}", flush=True)
    res = pr.gpu_run(p, reverse=True)
    L, lamL, U, lamU = oracle.factors(Ar, Br)
    _factor_close(res["L"], L, 1e-10)
    _factor_close(res["U"], U, 1e-10)
    np.testing.assert_allclose(res["lamL"], lamL, rtol=1e-10)
    np.testing.assert_allclose(res["lamU"], lamU, rtol=1e-10)
    tau = pr.TAU[dtype]
    Zo, Yo, c, hard = oracle.round_reverse(X, A, B, hint=res["Z"], tau=tau)
    pr.assert_replay_pass(p, c, hard, m * n)
    tol = 1e-9 if dtype == "f64" else 2e-6 * max(1.0, np.abs(Yo).max())
    assert np.abs(res["Y"] - Yo).max() <= tol
    pr.assert_objective(p, res["obj"], oracle.objective(X, Zo, A, B))
    # the same replay under the GPU's factors, on the reversed problem
    Zg, Yg, cg, hardg = oracle.round_nested(Xr, res["L"], res["U"],
                                            hint=np.ascontiguousarray(res["Z"][::-1, ::-1]), tau=tau)
    pr.assert_replay_pass(p, cg, hardg, m * n)
    # the sweep alone, with the oracle's factors imported into a reverse-order handle
    res2 = pr.gpu_run(p, factors=(L, lamL, U, lamU), reverse=True)
    Zo2, Yo2, c2, hard2 = oracle.round_reverse(X, A, B, hint=res2["Z"], tau=tau)
    pr.assert_replay_pass(p, c2, hard2, m * n)
    if m * n >= 4096:
        # the two orders are different trajectories
        fwd = pr.gpu_run(p)
        assert not np.array_equal(fwd["Z"], res["Z"])


@pytest.mark.parametrize("m,n,dtype", [(130, 200, "f64"), (384, 256, "f32"), (700, 1000, "f32")])
def test_transposed_problem_same_z(m, n, dtype):
    """||A (Z - X) B|| = ||B^T (Z^T - X^T) A^T||, and the column-major sweep of
    the transposed problem is the row-major order of the original, another
    admissible order: by Theorem 1 the GPU's Z of (X^T, B^T, A^T) is the
    transpose of its Z of (X, A, B), and the objectives agree."""
    p = wl.random_problem(m, n, 17, dtype, "general")
    print(f"[transpose] {m}x{n} {dtype}", flush=True)
    res = pr.gpu_run(p)
    pt = wl.Problem(p.name + "_T", np.ascontiguousarray(p.X.T), np.ascontiguousarray(p.B.T),
                    np.ascontiguousarray(p.A.T), p.dtype)
    rt = pr.gpu_run(pt)
    mism = int((res["Z"] != rt["Z"].T).sum())
    assert mism <= 1e-4 * m * n, mism
    rel = abs(res["obj"] - rt["obj"]) / res["obj"]
    assert rel <= pr.OBJ_RTOL[dtype], rel
    # and the oracle agrees with the transposed run too
    Xt, At, Bt = pt.widened()
    L, lamL, U, lamU = oracle.factors(At, Bt)
    Zo, Yo, c, hard = oracle.round_nested(Xt, L, U, hint=rt["Z"], tau=pr.TAU[dtype])
    pr.assert_replay_pass(pt, c, hard, m * n)


@pytest.mark.parametrize("kind", ["diag", "identity_right", "identity_left", "lower"])
def test_special_bases(kind):
    p = wl.random_problem(97, 131, 6, "f64", kind)
    X, A, B = p.widened()
    res = pr.gpu_run(p)
    L, lamL, U, lamU = oracle.factors(A, B)
    Zo, Yo, c, hard = pr.replay(p, L, U, res["Z"])
    pr.assert_replay_pass(p, c, hard, p.m * p.n)
    if kind == "diag":
        assert np.array_equal(res["Z"], np.rint(X).astype(np.int32))


@pytest.mark.parametrize("k,dtype", [(1, "f64"), (2, "f32")])
def test_small_configs(k, dtype):
    p = wl.make_config(k, dtype)
    X, A, B = p.widened()
    res = pr.gpu_run(p)
    Zo, Yo, c, hard = pr.replay(p, res["L"], res["U"], res["Z"])
    pr.assert_replay_pass(p, c, hard, p.m * p.n)
    L, lamL, U, lamU = oracle.factors(A, B)
    Zo3, Yo3, c3, hard3 = pr.replay(p, L, U, res["Z"])
    pr.assert_replay_pass(p, c3, hard3, p.m * p.n)
    pr.assert_objective(p, res["obj"], oracle.objective(X, Zo3, A, B))


def test_deterministic():
    p = wl.random_problem(300, 260, 7, "f64", "wishart")
    a = pr.gpu_run(p)
    b = pr.gpu_run(p)
    assert np.array_equal(a["Z"], b["Z"])
    assert np.array_equal(a["Y"].view(np.int64), b["Y"].view(np.int64))
    assert a["obj"] == b["obj"]


def test_singular_basis_is_reported():
    A = torch.zeros((70, 70), dtype=torch.float64, device="cuda")
    B = torch.eye(40, dtype=torch.float64, device="cuda")
    with pytest.raises(binding.Gptq2dError) as ei:
        binding.Factors.from_bases(A, B)
    assert ei.value.status == -2


def test_nonfinite_input_is_reported():
    p = wl.random_problem(80, 90, 8, "f64", "wishart")
    f = binding.Factors.from_bases(pr.to_dev(p.A), pr.to_dev(p.B))
    X = pr.to_dev(p.X)
    X[10, 20] = float("nan")
    with pytest.raises(binding.Gptq2dError) as ei:
        binding.round_matrix(f, X)
    assert ei.value.status == -3


def _with_x(p, X):
    return wl.Problem(p.name + "_x", np.ascontiguousarray(X.astype(p.X.dtype)), p.A, p.B, p.dtype)


@pytest.mark.parametrize("kind", ["diag", "general"])
def test_overflow_is_reported(kind):
    """A rounded value outside int32 is an error on both sides: one entry of
    3e9 gives GPTQ2D_ERR_OVERFLOW on the GPU and a range error in the oracle."""
    p = wl.random_problem(70, 130, 3, "f64", kind)
    X = p.X.copy()
    X[37, 101] = 3e9
    q = _with_x(p, X)
    print(f"[overflow] {kind}", flush=True)
    with pytest.raises(binding.Gptq2dError) as ei:
        pr.gpu_run(q)
    assert ei.value.status == -7
    Xw, A, B = q.widened()
    L, lamL, U, lamU = oracle.factors(A, B)
    with pytest.raises(oracle.OracleError, match="int32"):
        oracle.round_nested(Xw, L, U)


def test_int32_ends_are_accepted():
    """-2^31 and 2^31 - 1 are valid results (diagonal bases: Y = X exactly)."""
    p = wl.random_problem(65, 70, 4, "f64", "diag")
    X = p.X.copy()
    X[0, 0] = -2147483648.0
    X[64, 69] = 2147483647.4
    X[10, 3] = -2147483648.4
    res = pr.gpu_run(_with_x(p, X))
    assert res["Z"][0, 0] == -2147483648 and res["Z"][64, 69] == 2147483647
    assert res["Z"][10, 3] == -2147483648
    assert np.array_equal(res["Z"], np.rint(X).astype(np.int32))


@pytest.mark.parametrize("dtype", ["f64", "f32"])
def test_exact_ties(dtype):
    """Exact half-integer ties (Theorem 1 only asks for a deterministic rule;
    both sides break them to even). With diagonal bases Y = X exactly, so
    every entry of an X on the half-integer grid is a tie and Z is the
    half-even rounding of X. Under a general basis X on a grid of halves puts
    a tie at least at the first entry, and the oracle replays the sweep."""
    rng = np.random.default_rng(99)
    m, n = 131, 150
    p = wl.random_problem(m, n, 12, dtype, "diag")
    X = rng.integers(-40, 40, size=(m, n)) + 0.5
    res = pr.gpu_run(_with_x(p, X))
    assert np.array_equal(res["Z"], np.rint(X).astype(np.int32))
    assert np.array_equal(res["Y"], X)
    g = wl.random_problem(m, n, 13, dtype, "general")
    Xg = rng.integers(-80, 80, size=(m, n)) / 2.0
    Xg[0, 0] = 2.5
    q = _with_x(g, Xg)
    res = pr.gpu_run(q)
    assert res["Z"][0, 0] == 2
    Zo, Yo, c, hard = pr.replay(q, res["L"], res["U"], res["Z"])
    pr.assert_replay_pass(q, c, hard, m * n)
    L, lamL, U, lamU = oracle.factors(*q.widened()[1:])
    Zo3, Yo3, c3, hard3 = pr.replay(q, L, U, res["Z"])
    pr.assert_replay_pass(q, c3, hard3, m * n)


def test_argument_errors():
    p = wl.random_problem(70, 50, 9, "f64", "wishart")
    f = binding.Factors.from_bases(pr.to_dev(p.A), pr.to_dev(p.B))
    X = pr.to_dev(p.X)
    Z = torch.empty((70, 50), dtype=torch.int32, device="cuda")
    small = torch.empty(128, dtype=torch.uint8, device="cuda")
    with pytest.raises(binding.Gptq2dError) as ei:
        binding.gptq2d_round(f.handle, X, Z, None, None, small)
    assert ei.value.status == -6
    with pytest.raises(ValueError):
        binding.gptq2d_round(f.handle, X[:, :40], Z, None, None, f.workspace())


def test_stage_timing_is_transparent():
    """Timing the stage launches with events changes no result, and the
    record counts one pair per stage launch (MT + NT - 1 per round)."""
    p = wl.random_problem(200, 330, 10, "f32", "wishart")
    f = binding.Factors.from_bases(pr.to_dev(p.A), pr.to_dev(p.B))
    X = pr.to_dev(p.X)
    Z0, Y0, o0 = binding.round_matrix(f, X)
    binding.gptq2d_stage_timing(f.handle, True)
    Z1, Y1, o1 = binding.round_matrix(f, X)
    Z2, Y2, o2 = binding.round_matrix(f, X)
    ms, cnt = binding.gptq2d_stage_time(f.handle)
    assert cnt == 2 * ((200 + 63) // 64 + (330 + 63) // 64 - 1)
    assert ms > 0.0
    assert binding.gptq2d_stage_time(f.handle) == (0.0, 0)
    binding.gptq2d_stage_timing(f.handle, False)
    binding.round_matrix(f, X)
    assert binding.gptq2d_stage_time(f.handle)[1] == 0
    for Z, Y, o in ((Z1, Y1, o1), (Z2, Y2, o2)):
        assert torch.equal(Z, Z0) and torch.equal(Y, Y0) and float(o[0]) == float(o0[0])
    f.close()


def test_concurrent_host_threads():
    """Two host threads, each with its own handle, stream and workspace, round
    at the same time: each gets the result of running alone."""
    import threading
    probs = [wl.random_problem(300, 260, 60 + i, "f64", "wishart") for i in range(2)]
    ref = [pr.gpu_run(p) for p in probs]
    out = [None, None]
    err = []

    def work(i):
        try:
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                p = probs[i]
                f = binding.Factors.from_bases(pr.to_dev(p.A), pr.to_dev(p.B), stream=s)
                for _ in range(3):
                    Z, Y, obj = binding.round_matrix(f, pr.to_dev(p.X), stream=s)
                s.synchronize()
                out[i] = (Z.cpu().numpy(), float(obj.cpu()[0]))
                f.close()
        except Exception as e:  # reported below
            err.append(e)

    ts = [threading.Thread(target=work, args=(i,)) for i in range(2)]
    for t in ts:
        t.start()
    for t in ts:
        t.join()
    assert not err, err
    for i in range(2):
        assert np.array_equal(out[i][0], ref[i]["Z"])
        assert out[i][1] == ref[i]["obj"]


@pytest.mark.parametrize("reverse", [False, True])
def test_graph_capture_replays(reverse):
    """A whole step (factorisation, with its second stream forked and joined
    by events, then the sweep's stage launches) captured in a HIP graph:
    every replay, with eager work and synchronisations between the replays,
    gives the eager result."""
    p = wl.random_problem(520, 390, 31, "f32", "wishart")
    A, B, X = pr.to_dev(p.A), pr.to_dev(p.B), pr.to_dev(p.X)
    f = binding.Factors(p.m, p.n, reverse=reverse)
    ws = f.workspace()
    Z = torch.empty((p.m, p.n), dtype=torch.int32, device="cuda")
    Y = torch.empty_like(X)
    obj = torch.empty(1, dtype=torch.float64, device="cuda")
    s = torch.cuda.Stream()

    def step():
        binding.gptq2d_factor_compute(f.handle, A, B, s)
        binding.gptq2d_round(f.handle, X, Z, Y, obj, ws, s)

    with torch.cuda.stream(s):
        step()
    torch.cuda.synchronize()
    Zref, Yref, oref = Z.clone(), Y.clone(), float(obj[0])
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        step()
    torch.cuda.synchronize()
    for _ in range(3):
        Z.fill_(-1)
        Y.fill_(0.0)
        obj.fill_(0.0)
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(Z, Zref) and torch.equal(Y, Yref) and float(obj[0]) == oref
        with torch.cuda.stream(s):
            step()
        torch.cuda.synchronize()
    binding.gptq2d_round_check(f.handle, ws, s)
    del g
    f.close()
