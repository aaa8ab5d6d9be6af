"""The entry point that allocates nothing (gptq2d_round_noalloc) against
gptq2d_round through the C ABI: the same kernels on the same data, so Z, Y
and the objective must be bit-identical. Two calls in a row, the second on a
smaller problem, show that what the first call leaves in the library's
fixed workspace does not leak into the next one."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2607_27042_amd import binding, workloads as wl

pytestmark = pytest.mark.gpu


def _to_dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _noalloc(f, X, want_y=True):
    lib = binding.load()
    m, n = f.m, f.n
    Z = torch.full((m, n), -7, dtype=torch.int32, device="cuda")
    Y = torch.full((m, n), float("nan"), dtype=X.dtype, device="cuda") if want_y else None
    obj = torch.full((1,), float("nan"), dtype=torch.float64, device="cuda")
    word = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    st = lib.gptq2d_round_noalloc(ctypes.c_void_p(f.handle), binding._dt(X), ctypes.c_void_p(X.data_ptr()),
                                  X.stride(0), ctypes.c_void_p(Z.data_ptr()), Z.stride(0),
                                  ctypes.c_void_p(0 if Y is None else Y.data_ptr()),
                                  n if Y is None else Y.stride(0), ctypes.c_void_p(obj.data_ptr()),
                                  ctypes.c_void_p(word.data_ptr()), stream)
    assert st == 0, binding.gptq2d_last_error()
    assert lib.gptq2d_round_check(ctypes.c_void_p(f.handle), ctypes.c_void_p(word.data_ptr()), stream) == 0
    assert int(word.cpu()[0]) == 0
    return Z, Y, obj


@pytest.mark.parametrize("dtype", ["f32", "f64"])
def test_noalloc_matches_round(dtype):
    # 1000 x 700 needs 22.9 MB of workspace, 300 x 260 2.7 MB: both fit
    for m, n, seed in ((1000, 700, 1), (300, 260, 2)):
        p = wl.random_problem(m, n, seed, dtype, "wishart")
        print(f"[noalloc] {m}x{n} {dtype}", flush=True)
        f = binding.Factors.from_bases(_to_dev(p.A), _to_dev(p.B))
        X = _to_dev(p.X)
        Z1, Y1, o1 = binding.round_matrix(f, X)
        Z2, Y2, o2 = _noalloc(f, X)
        torch.cuda.synchronize()
        assert torch.equal(Z1, Z2)
        assert torch.equal(Y1, Y2)
        assert float(o1[0]) == float(o2[0])
        # without Y, and once more on the same handle
        Z3, _, o3 = _noalloc(f, X, want_y=False)
        assert torch.equal(Z1, Z3) and float(o1[0]) == float(o3[0])
        f.close()


def test_noalloc_errors():
    """Too large for the fixed workspace: WORKSPACE with the sizes in the
    message; a missing status word: INVALID_ARG. Nothing is launched."""
    lib = binding.load()
    f = binding.Factors(2048, 1536)
    X = torch.zeros((2048, 1536), dtype=torch.float32, device="cuda")
    Z = torch.empty((2048, 1536), dtype=torch.int32, device="cuda")
    word = torch.zeros(1, dtype=torch.int32, device="cuda")
    args = [ctypes.c_void_p(f.handle), 0, ctypes.c_void_p(X.data_ptr()), 1536, ctypes.c_void_p(Z.data_ptr()),
            1536, ctypes.c_void_p(0), 1536, ctypes.c_void_p(0)]
    st = lib.gptq2d_round_noalloc(*args, ctypes.c_void_p(word.data_ptr()), ctypes.c_void_p(0))
    assert st == -6
    assert "64 MiB" in binding.gptq2d_last_error()
    f.close()
    g = binding.Factors(64, 64)
    X = torch.zeros((64, 64), dtype=torch.float32, device="cuda")
    Z = torch.empty((64, 64), dtype=torch.int32, device="cuda")
    st = lib.gptq2d_round_noalloc(ctypes.c_void_p(g.handle), 0, ctypes.c_void_p(X.data_ptr()), 64,
                                  ctypes.c_void_p(Z.data_ptr()), 64, ctypes.c_void_p(0), 64, ctypes.c_void_p(0),
                                  ctypes.c_void_p(0), ctypes.c_void_p(0))
    assert st == -1
    g.close()
