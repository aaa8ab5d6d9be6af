"""CPU checks of the C ABI library: it loads, exports every declared entry
point, validates arguments without touching a device, and its host-side
delivery plan is a partition of the deferred feedback."""
import ctypes
import itertools

import numpy as np
import pytest

from paper_2607_27042_amd import binding, build


@pytest.fixture(scope="module")
def lib():
    if build.is_stale():
        build.build()
    return binding.load()


def test_exports_every_declared_symbol(lib):
    names = binding.declared_functions()
    assert len(names) >= 15
    for name in names:
        assert hasattr(lib, name), name


def test_status_strings_and_version(lib):
    assert binding.gptq2d_version() == 100
    for code in binding.STATUS:
        s = binding.gptq2d_status_string(code)
        assert s and s != "unknown status"
    assert binding.gptq2d_status_string(12345) == "unknown status"


def test_null_handle_is_rejected(lib):
    null = ctypes.c_void_p(0)
    assert lib.gptq2d_factors_shape(null, None, None) == -1
    assert "NULL" in binding.gptq2d_last_error()
    assert lib.gptq2d_round(null, 0, null, 4, null, 4, null, 4, null, null, 0, null) == -1
    assert lib.gptq2d_factor_compute(null, 0, null, 4, null, 4, null) == -1
    assert lib.gptq2d_round_workspace_size(null) == 0
    assert lib.gptq2d_stage_timing(null, 1) == -1
    assert lib.gptq2d_stage_time(null, None, None) == -1
    assert lib.gptq2d_factors_set_order(null, 1) == -1
    assert lib.gptq2d_round_batched_workspace_size(0, None) == 0
    assert lib.gptq2d_round_batched_workspace_size(2, None) == 0
    nulls = (ctypes.c_void_p * 2)(None, None)
    assert lib.gptq2d_round_batched_workspace_size(2, nulls) == 0
    assert lib.gptq2d_round_batched(0, None, 0, None, None, None, None, None, None, None, None, 0, None) == -1
    assert lib.gptq2d_round_batched(2, nulls, 0, nulls, None, nulls, None, None, None, None, None, 0,
                                    None) == -1
    assert lib.gptq2d_round_batched_check(None, None) == -1
    assert lib.gptq2d_factor_batched_workspace_size(0) == 0
    assert lib.gptq2d_factor_batched_workspace_size(3) >= 256
    assert lib.gptq2d_factor_batched(0, None, 0, None, None, None, None, None, 0, None) == -1
    assert lib.gptq2d_factor_batched(2, nulls, 0, nulls, None, nulls, None, None, 0, None) == -1
    assert lib.gptq2d_factor_batched_check(0, None, None) == -1
    out = ctypes.c_void_p()
    assert lib.gptq2d_factors_create(0, 5, ctypes.byref(out)) == -1
    assert lib.gptq2d_factors_create(5, 70000, ctypes.byref(out)) == -1
    lib.gptq2d_factors_destroy(null)


def _task_fields(x):
    return x & 1, (x >> 1) & 1, ((x >> 2) & 1) + 1, ((x >> 3) & 1) + 1


def _check_plan(m, n, g):
    tasks, offs = binding.gptq2d_schedule_tasks(m, n, g)
    MT, NT = (m + 63) // 64, (n + 63) // 64
    S = MT + NT - 1
    assert len(offs) == S + 1 and offs[0] == 0 and offs[-1] == len(tasks)
    assert (np.diff(offs) >= 0).all()
    got = {}
    for k in range(S):
        seen = set()
        for x, ti, tj, w in tasks[offs[k]:offs[k + 1]]:
            d, ow, nr, nc = _task_fields(x)
            s0, s1 = w & 0xFFFF, w >> 16
            assert 0 <= ti and ti + nr <= MT and 0 <= tj and tj + nc <= NT and s0 < s1
            for r in range(nr):
                for c in range(nc):
                    I, J = ti + r, tj + c
                    assert I + J >= k + 1, "delivered after the target was swept"
                    key = (d, I, J)
                    assert key not in seen, "two tasks of one launch write the same buffer"
                    seen.add(key)
                    # the sources of this target: tiles (s, J) or (I, s)
                    fixed = J if d == 0 else I
                    assert (s1 - 1) + fixed <= k - 1, "a source is not finished before the launch"
                    got.setdefault(key, []).append((k, s0, s1, ow))
    # every target receives every source except its immediate predecessor,
    # exactly once, and the first delivery overwrites
    for ti, tj in itertools.product(range(MT), range(NT)):
        for d in (0, 1):
            lim = (ti if d == 0 else tj) - 2
            lst = got.get((d, ti, tj), [])
            if lim < 0:
                assert not lst
                continue
            lst.sort()
            pos = 0
            for _, s0, s1, _ in sorted(lst, key=lambda e: e[1]):
                assert s0 == pos
                pos = s1
            assert pos == lim + 1
            assert [ow for *_, ow in lst] == [1] + [0] * (len(lst) - 1)
            assert max(r - l for _, l, r, _ in lst) <= max(g, 2)


@pytest.mark.parametrize("m,n", [(1, 1), (64, 64), (65, 200), (512, 384), (700, 130), (2048, 64)])
@pytest.mark.parametrize("g", [1, 2, 4, 7])
def test_delivery_plan_is_exact(lib, m, n, g):
    _check_plan(m, n, g)


def _read_fig1():
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "fig1_dependency_3x4.txt")
    out = {}
    for line in open(path):
        if line.startswith("#") or not line.strip():
            continue
        key, *rest = line.split()
        out[key] = rest
    return out


def test_fig1_wavefronts(lib):
    """The library's launch plan against Fig. 1 (tests/golden), read at tile
    level on a grid of 3 x 4 tiles: as many launches as the figure has
    wavefronts, every tile swept once, every arrow of the figure ((i, j) ->
    (i, j+1) and (i, j) -> (i+1, j)) from an earlier launch to a later one,
    and the red anti-diagonal I_4 swept together in one launch."""
    g = _read_fig1()
    m, n = int(g["shape"][0]), int(g["shape"][1])
    rows = binding.gptq2d_schedule_sweeps(m * 64, n * 64)
    assert len(rows) == int(g["wavefronts"][0])
    launch = {}
    for k, (lo, hi) in enumerate(rows):
        for i in range(lo, hi + 1):
            t = (i + 1, k - i + 1)  # 1-based, as in the figure
            assert 1 <= t[1] <= n and t not in launch
            launch[t] = k
    assert len(launch) == m * n
    for (i, j), k in launch.items():
        for t in ((i, j + 1), (i + 1, j)):
            if t in launch:
                assert launch[t] > k, (i, j, t)
    red = [tuple(int(v) for v in e.split(",")) for e in g["red_set"][1:]]
    ks = {launch[t] for t in red}
    assert len(ks) == 1
    assert sorted(t for t, k in launch.items() if k in ks) == sorted(red)
    # the same structure at a ragged size: tile rows never go out of range
    rows = binding.gptq2d_schedule_sweeps(700, 130)
    assert len(rows) == 11 + 3 - 1 and (rows[:, 0] <= rows[:, 1]).all()


def test_missing_library_fails_loudly(monkeypatch):
    """Without the built HIP library the binding raises; there is no fallback."""
    monkeypatch.setattr(binding, "_lib", None)
    monkeypatch.setattr(binding, "LIB_PATH", "/nonexistent/libgptq2d.so")
    with pytest.raises(RuntimeError, match="not built"):
        binding.load()


def test_bench_refuses_several_gpus():
    """bench.py measures one GPU; --gpus N > 1 exits with a message before
    touching any device."""
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "exactly one GPU" in r.stderr


def test_binding_refuses_aliased_or_short_views():
    """The binding hands the library a pointer and a row stride; a view whose
    rows alias each other (expanded, overlapping as_strided) or whose last
    row runs past its storage is refused before any call."""
    import torch
    base = torch.zeros((6, 8), dtype=torch.float32)
    assert binding._layout(base, 6, 8, "X") == 8
    assert binding._layout(base[:, 2:7], 6, 5, "X") == 8
    assert binding._layout(base[2:3], 1, 8, "X") == 8
    with pytest.raises(ValueError, match="row stride"):
        binding._layout(torch.zeros(8).expand(6, 8), 6, 8, "X")
    with pytest.raises(ValueError, match="row stride"):
        binding._layout(torch.zeros(20).as_strided((6, 8), (2, 1)), 6, 8, "Z")
    short = torch.zeros(48)
    view = short.view(6, 8)
    short.untyped_storage().resize_(40 * 4)  # the storage shrinks under the view
    with pytest.raises(ValueError, match="storage"):
        binding._layout(view, 6, 8, "Y")
    with pytest.raises(ValueError, match="unit column stride"):
        binding._layout(base.t(), 8, 6, "X")
