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


def test_fig1_wavefronts(lib):
    """The 3 x 4 example of Fig. 1 has 6 anti-diagonal wavefronts, and the
    4th set (s = 4, 1-based) is {(1,3), (2,2), (3,1)}; at tile level a
    3 x 4 grid of tiles has the same structure (6 launches)."""
    tasks, offs = binding.gptq2d_schedule_tasks(3 * 64, 4 * 64, 1)
    assert len(offs) - 1 == 6
    waves = [[(i + 1, s - i + 1) for i in range(3) if 0 <= s - i < 4] for s in range(6)]
    assert waves[2] == [(1, 3), (2, 2), (3, 1)]


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
