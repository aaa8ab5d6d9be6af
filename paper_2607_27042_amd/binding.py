"""Thin Python binding of ``libgptq2d.so`` (the C ABI in ``include/gptq2d.h``).

Argument marshalling only: every step of the factorisation and of the sweep
runs in the library's HIP kernels. PyTorch supplies device memory and the
current stream. The library must be built (``__graft_entry__.build()``); a
missing library is an error, never a fallback.

The functions named like the C entry points take and return the same things,
with torch tensors in place of device pointers and Python ints in place of
handles. ``Factors`` and ``round_matrix`` are conveniences built from them.
"""
from __future__ import annotations

import ctypes
import os
import re

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "lib", "libgptq2d.so")
HEADER = os.path.join(os.path.dirname(_HERE), "include", "gptq2d.h")

F32, F64 = 0, 1
STATUS = {0: "OK", -1: "ERR_INVALID_ARG", -2: "ERR_SINGULAR", -3: "ERR_NONFINITE", -4: "ERR_OOM",
          -5: "ERR_HIP", -6: "ERR_WORKSPACE", -7: "ERR_OVERFLOW", -8: "ERR_TIMEOUT"}

_lib = None


class Gptq2dError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        self.status = status
        super().__init__(f"{where}: {STATUS.get(status, status)}: {detail}")


def declared_functions() -> list[str]:
    """Names of the functions declared in include/gptq2d.h."""
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gptq2d_[a-z_]+)\s*\(", text)))


def load():
    """Load the built library (raises if it is not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build() first")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_size_t
    ip32 = ctypes.POINTER(ctypes.c_int32)
    sigs = {
        "gptq2d_factors_create": (i32, [i32, i32, ctypes.POINTER(vp)]),
        "gptq2d_factors_destroy": (None, [vp]),
        "gptq2d_factors_shape": (i32, [vp, ctypes.POINTER(i32), ctypes.POINTER(i32)]),
        "gptq2d_factors_set_order": (i32, [vp, i32]),
        "gptq2d_factor_compute": (i32, [vp, i32, vp, i64, vp, i64, vp]),
        "gptq2d_factor_check": (i32, [vp, vp]),
        "gptq2d_factor": (i32, [i32, i32, i32, vp, i64, vp, i64, vp, ctypes.POINTER(vp)]),
        "gptq2d_factor_batched_workspace_size": (sz, [i32]),
        "gptq2d_factor_batched": (i32, [i32, vp, i32, vp, vp, vp, vp, vp, sz, vp]),
        "gptq2d_factor_batched_check": (i32, [i32, vp, vp]),
        "gptq2d_factors_export": (i32, [vp, vp, i64, vp, i64, vp, vp, vp]),
        "gptq2d_factors_import": (i32, [vp, vp, i64, vp, i64, vp, vp, vp]),
        "gptq2d_round_workspace_size": (sz, [vp]),
        "gptq2d_round": (i32, [vp, i32, vp, i64, vp, i64, vp, i64, vp, vp, sz, vp]),
        "gptq2d_round_check": (i32, [vp, vp, vp]),
        "gptq2d_round_noalloc": (i32, [vp, i32, vp, i64, vp, i64, vp, i64, vp, vp, vp]),
        "gptq2d_round_batched_workspace_size": (sz, [i32, vp]),
        "gptq2d_round_batched": (i32, [i32, vp, i32, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
        "gptq2d_round_batched_check": (i32, [vp, vp]),
        "gptq2d_status_string": (ctypes.c_char_p, [i32]),
        "gptq2d_last_error": (ctypes.c_char_p, []),
        "gptq2d_version": (i32, []),
        "gptq2d_schedule_tasks": (i64, [i32, i32, i32, ip32, i64, ip32]),
        "gptq2d_schedule_sweeps": (i64, [i32, i32, ip32, i64]),
        "gptq2d_stage_timing": (i32, [vp, i32]),
        "gptq2d_stage_time": (i32, [vp, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(i64)]),
    }
    for name, (res, args) in sigs.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


def _check(st: int, where: str):
    if st != 0:
        raise Gptq2dError(st, where, load().gptq2d_last_error().decode())


def _stream(stream=None):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.float64:
        return F64
    raise TypeError(f"unsupported dtype {t.dtype}")


def _layout(t: torch.Tensor, rows: int, cols: int, what: str) -> int:
    """Leading dimension of a rows x cols row-major view, after checking that
    the library may read (or write) every row of it without touching memory
    outside the tensor or another row."""
    if t.dim() != 2 or tuple(t.shape) != (rows, cols):
        raise ValueError(f"{what} must be {rows} x {cols}, got {tuple(t.shape)}")
    if t.stride(1) != 1 and cols > 1:
        raise ValueError(f"{what} must be row-major with unit column stride")
    ld = t.stride(0) if rows > 1 else cols
    if rows > 1 and ld < cols:
        # an expanded or overlapping view: rows would alias each other
        raise ValueError(f"{what} has row stride {ld} < {cols} columns (expanded or overlapping view)")
    # the last element the library touches must lie inside the storage
    need = (t.storage_offset() + (rows - 1) * ld + cols) * t.element_size()
    if need > t.untyped_storage().nbytes():
        raise ValueError(f"{what}: rows x ld exceed the tensor's storage")
    return int(ld)


def _mat(t: torch.Tensor, rows: int, cols: int, what: str):
    if not t.is_cuda:
        raise ValueError(f"{what} must be a device tensor")
    ld = _layout(t, rows, cols, what)
    return ctypes.c_void_p(t.data_ptr()), ld


def _ptr(t):
    return ctypes.c_void_p(0 if t is None else t.data_ptr())


# ---------------------------------------------------------------------------
# C entry points
# ---------------------------------------------------------------------------

def gptq2d_version() -> int:
    return int(load().gptq2d_version())


def gptq2d_status_string(st: int) -> str:
    return load().gptq2d_status_string(st).decode()


def gptq2d_last_error() -> str:
    return load().gptq2d_last_error().decode()


def gptq2d_factors_create(m: int, n: int) -> int:
    h = ctypes.c_void_p()
    _check(load().gptq2d_factors_create(m, n, ctypes.byref(h)), "gptq2d_factors_create")
    return h.value


def gptq2d_factors_destroy(h: int) -> None:
    load().gptq2d_factors_destroy(ctypes.c_void_p(h))


def gptq2d_factors_shape(h: int):
    m, n = ctypes.c_int(), ctypes.c_int()
    _check(load().gptq2d_factors_shape(ctypes.c_void_p(h), ctypes.byref(m), ctypes.byref(n)),
           "gptq2d_factors_shape")
    return m.value, n.value


def gptq2d_factors_set_order(h: int, reverse: bool) -> None:
    _check(load().gptq2d_factors_set_order(ctypes.c_void_p(h), int(bool(reverse))),
           "gptq2d_factors_set_order")


def gptq2d_factor_compute(h: int, A: torch.Tensor, B: torch.Tensor, stream=None) -> None:
    m, n = gptq2d_factors_shape(h)
    if A.dtype != B.dtype:
        raise TypeError("A and B must share a dtype")
    pa, lda = _mat(A, m, m, "A")
    pb, ldb = _mat(B, n, n, "B")
    _check(load().gptq2d_factor_compute(ctypes.c_void_p(h), _dt(A), pa, lda, pb, ldb, _stream(stream)),
           "gptq2d_factor_compute")


def gptq2d_factor_check(h: int, stream=None) -> None:
    _check(load().gptq2d_factor_check(ctypes.c_void_p(h), _stream(stream)), "gptq2d_factor_check")


def gptq2d_factor_batched_workspace_size(count: int) -> int:
    return int(load().gptq2d_factor_batched_workspace_size(count))


def gptq2d_factor_batched(handles, As, Bs, workspace: torch.Tensor, stream=None, shapes=None,
                          prepare=False):
    """Factorisations of len(handles) problems (distinct handles) in common
    launches per shape. prepare=True: as for gptq2d_round_batched."""
    count = len(handles)
    if count == 0 or len(As) != count or len(Bs) != count:
        raise ValueError("one A and one B per handle")
    dt = _dt(As[0])
    ap, al, bp, bl = [], [], [], []
    for p, h in enumerate(handles):
        m, n = shapes[p] if shapes is not None else gptq2d_factors_shape(h)
        if _dt(As[p]) != dt or _dt(Bs[p]) != dt:
            raise TypeError("every A and B of a batch must have the same dtype")
        a, la = _mat(As[p], m, m, f"A[{p}]")
        b, lb = _mat(Bs[p], n, n, f"B[{p}]")
        ap.append(a.value); al.append(la); bp.append(b.value); bl.append(lb)
    VP, I64 = ctypes.c_void_p * count, ctypes.c_int64 * count
    args = (count, _handles(handles), dt, VP(*ap), I64(*al), VP(*bp), I64(*bl), _ptr(workspace),
            workspace.numel() * workspace.element_size(), _stream(stream))
    fn = load().gptq2d_factor_batched

    def call():
        _check(fn(*args), "gptq2d_factor_batched")
    if prepare:
        return call
    call()


def gptq2d_factor_batched_check(handles, stream=None) -> None:
    _check(load().gptq2d_factor_batched_check(len(handles), _handles(handles), _stream(stream)),
           "gptq2d_factor_batched_check")


def gptq2d_factor(A: torch.Tensor, B: torch.Tensor, stream=None) -> int:
    if A.dtype != B.dtype:
        raise TypeError("A and B must share a dtype")
    m, n = A.shape[0], B.shape[0]
    pa, lda = _mat(A, m, m, "A")
    pb, ldb = _mat(B, n, n, "B")
    h = ctypes.c_void_p()
    _check(load().gptq2d_factor(m, n, _dt(A), pa, lda, pb, ldb, _stream(stream), ctypes.byref(h)),
           "gptq2d_factor")
    return h.value


def gptq2d_factors_export(h: int, stream=None):
    m, n = gptq2d_factors_shape(h)
    dev = torch.cuda.current_device()
    L = torch.empty((m, m), dtype=torch.float64, device=dev)
    U = torch.empty((n, n), dtype=torch.float64, device=dev)
    lamL = torch.empty(m, dtype=torch.float64, device=dev)
    lamU = torch.empty(n, dtype=torch.float64, device=dev)
    _check(load().gptq2d_factors_export(ctypes.c_void_p(h), _ptr(L), m, _ptr(U), n, _ptr(lamL),
                                        _ptr(lamU), _stream(stream)), "gptq2d_factors_export")
    return L, U, lamL, lamU


def gptq2d_factors_import(h: int, L, U, lamL, lamU, stream=None) -> None:
    m, n = gptq2d_factors_shape(h)
    for t in (L, U, lamL, lamU):
        if t.dtype != torch.float64 or not t.is_cuda:
            raise TypeError("factors must be float64 device tensors")
    pl, ldl = _mat(L, m, m, "L")
    pu, ldu = _mat(U, n, n, "U")
    if lamL.numel() != m or lamU.numel() != n or not lamL.is_contiguous() or not lamU.is_contiguous():
        raise ValueError("lamL / lamU have the wrong size or layout")
    _check(load().gptq2d_factors_import(ctypes.c_void_p(h), pl, ldl, pu, ldu, _ptr(lamL), _ptr(lamU),
                                        _stream(stream)), "gptq2d_factors_import")


def gptq2d_round_workspace_size(h: int) -> int:
    return int(load().gptq2d_round_workspace_size(ctypes.c_void_p(h)))


def gptq2d_round(h: int, X: torch.Tensor, Z: torch.Tensor, Y, objective, workspace: torch.Tensor,
                 stream=None) -> None:
    m, n = gptq2d_factors_shape(h)
    px, ldx = _mat(X, m, n, "X")
    if Z.dtype != torch.int32:
        raise TypeError("Z must be int32")
    pz, ldz = _mat(Z, m, n, "Z")
    if Y is not None:
        if Y.dtype != X.dtype:
            raise TypeError("Y must have X's dtype")
        py, ldy = _mat(Y, m, n, "Y")
    else:
        py, ldy = ctypes.c_void_p(0), n
    if objective is not None and (objective.dtype != torch.float64 or not objective.is_cuda):
        raise TypeError("objective must be a float64 device tensor")
    _check(load().gptq2d_round(ctypes.c_void_p(h), _dt(X), px, ldx, pz, ldz, py, ldy, _ptr(objective),
                               _ptr(workspace), workspace.numel() * workspace.element_size(),
                               _stream(stream)), "gptq2d_round")


def gptq2d_round_noalloc(h: int, X: torch.Tensor, Z: torch.Tensor, Y, objective, status_word: torch.Tensor,
                         stream=None) -> None:
    """gptq2d_round with the library's own fixed workspace; status_word is a
    one-element int32 device tensor (check it with gptq2d_round_check)."""
    m, n = gptq2d_factors_shape(h)
    px, ldx = _mat(X, m, n, "X")
    if Z.dtype != torch.int32:
        raise TypeError("Z must be int32")
    pz, ldz = _mat(Z, m, n, "Z")
    if Y is not None:
        if Y.dtype != X.dtype:
            raise TypeError("Y must have X's dtype")
        py, ldy = _mat(Y, m, n, "Y")
    else:
        py, ldy = ctypes.c_void_p(0), n
    if objective is not None and (objective.dtype != torch.float64 or not objective.is_cuda):
        raise TypeError("objective must be a float64 device tensor")
    if status_word.dtype != torch.int32 or not status_word.is_cuda or status_word.numel() < 1:
        raise TypeError("status_word must be an int32 device tensor")
    _check(load().gptq2d_round_noalloc(ctypes.c_void_p(h), _dt(X), px, ldx, pz, ldz, py, ldy,
                                       _ptr(objective), _ptr(status_word), _stream(stream)),
           "gptq2d_round_noalloc")


def gptq2d_round_check(h: int, workspace: torch.Tensor, stream=None) -> None:
    _check(load().gptq2d_round_check(ctypes.c_void_p(h), _ptr(workspace), _stream(stream)),
           "gptq2d_round_check")


def _handles(handles):
    arr = (ctypes.c_void_p * len(handles))(*[int(h) for h in handles])
    return arr


def gptq2d_round_batched_workspace_size(handles) -> int:
    return int(load().gptq2d_round_batched_workspace_size(len(handles), _handles(handles)))


def gptq2d_round_batched(handles, Xs, Zs, Ys, objective, workspace: torch.Tensor, stream=None,
                         shapes=None, prepare=False):
    """Problems p = 0 .. len(handles)-1 in common launches; Ys may be None (or
    hold None entries); objective None or a float64 device tensor of
    len(handles) entries. With prepare=True nothing is enqueued: the argument
    arrays are built once and a function of no arguments is returned that
    enqueues the call (for loops over the same tensors)."""
    count = len(handles)
    if not (len(Xs) == len(Zs) == count) or (Ys is not None and len(Ys) != count):
        raise ValueError("one X, Z (and Y) per handle")
    if count == 0:
        raise ValueError("empty batch")
    dt = _dt(Xs[0])
    xp, xl, zp, zl, yp, yl = [], [], [], [], [], []
    for p, h in enumerate(handles):
        m, n = shapes[p] if shapes is not None else gptq2d_factors_shape(h)
        if _dt(Xs[p]) != dt:
            raise TypeError("every X of a batch must have the same dtype")
        a, la = _mat(Xs[p], m, n, f"X[{p}]")
        if Zs[p].dtype != torch.int32:
            raise TypeError("Z must be int32")
        b, lb = _mat(Zs[p], m, n, f"Z[{p}]")
        xp.append(a.value); xl.append(la); zp.append(b.value); zl.append(lb)
        if Ys is not None:
            if Ys[p] is None:
                yp.append(None); yl.append(n)
            else:
                if Ys[p].dtype != Xs[p].dtype:
                    raise TypeError("Y must have X's dtype")
                c, lc = _mat(Ys[p], m, n, f"Y[{p}]")
                yp.append(c.value); yl.append(lc)
    if objective is not None and (objective.dtype != torch.float64 or not objective.is_cuda
                                  or objective.numel() < count or not objective.is_contiguous()):
        raise TypeError("objective must be a contiguous float64 device tensor of count entries")
    VP, I64 = ctypes.c_void_p * count, ctypes.c_int64 * count
    X_a, ldx_a, Z_a, ldz_a = VP(*xp), I64(*xl), VP(*zp), I64(*zl)
    Y_a = VP(*yp) if Ys is not None else None
    ldy_a = I64(*yl) if Ys is not None else None
    args = (count, _handles(handles), dt, X_a, ldx_a, Z_a, ldz_a, Y_a, ldy_a, _ptr(objective),
            _ptr(workspace), workspace.numel() * workspace.element_size(), _stream(stream))
    fn = load().gptq2d_round_batched

    def call():
        _check(fn(*args), "gptq2d_round_batched")
    if prepare:
        return call
    call()


def gptq2d_round_batched_check(workspace: torch.Tensor, stream=None) -> None:
    _check(load().gptq2d_round_batched_check(_ptr(workspace), _stream(stream)),
           "gptq2d_round_batched_check")


def gptq2d_stage_timing(h: int, enable: bool) -> None:
    _check(load().gptq2d_stage_timing(ctypes.c_void_p(h), int(bool(enable))), "gptq2d_stage_timing")


def gptq2d_stage_time(h: int):
    """(summed stage-kernel launch time in ms, launches) since the last read."""
    ms, cnt = ctypes.c_double(0.0), ctypes.c_int64(0)
    _check(load().gptq2d_stage_time(ctypes.c_void_p(h), ctypes.byref(ms), ctypes.byref(cnt)),
           "gptq2d_stage_time")
    return float(ms.value), int(cnt.value)


def gptq2d_schedule_tasks(m: int, n: int, g: int):
    """Host-only delivery plan: (tasks int32[T, 4], offsets int32[MT+NT])."""
    import numpy as np
    lib = load()
    total = lib.gptq2d_schedule_tasks(m, n, g, None, 0, None)
    if total < 0:
        raise ValueError(gptq2d_last_error())
    mt, nt = (m + 63) // 64, (n + 63) // 64
    offs = np.zeros(mt + nt, dtype=np.int32)
    tasks = np.zeros((max(total, 1), 4), dtype=np.int32)
    lib.gptq2d_schedule_tasks(m, n, g, tasks.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), total,
                              offs.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)))
    return tasks[:total], offs


def gptq2d_schedule_sweeps(m: int, n: int):
    """Host-only list of the tiles each sweep launch rounds: int32[S, 2] of
    (first, last) tile row; row I of launch k is tile (I, k - I)."""
    import numpy as np
    lib = load()
    total = lib.gptq2d_schedule_sweeps(m, n, None, 0)
    if total < 0:
        raise ValueError(gptq2d_last_error())
    rows = np.zeros((total, 2), dtype=np.int32)
    lib.gptq2d_schedule_sweeps(m, n, rows.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), total)
    return rows


# ---------------------------------------------------------------------------
# Conveniences
# ---------------------------------------------------------------------------

class Factors:
    """Owning wrapper of a factor handle."""

    def __init__(self, m: int, n: int, reverse: bool = False):
        """reverse: round from the last row and column on (the factors are then
        those of the index-reversed problem)."""
        self.m, self.n = m, n
        self.handle = gptq2d_factors_create(m, n)
        self.reverse = bool(reverse)
        if self.reverse:
            gptq2d_factors_set_order(self.handle, True)

    @classmethod
    def from_bases(cls, A: torch.Tensor, B: torch.Tensor, check: bool = True, stream=None,
                   reverse: bool = False):
        f = cls(A.shape[0], B.shape[0], reverse)
        f.compute(A, B, stream)
        if check:
            gptq2d_factor_check(f.handle, stream)
        return f

    def compute(self, A, B, stream=None):
        gptq2d_factor_compute(self.handle, A, B, stream)

    def export(self, stream=None):
        return gptq2d_factors_export(self.handle, stream)

    def load(self, L, U, lamL, lamU, stream=None):
        gptq2d_factors_import(self.handle, L, U, lamL, lamU, stream)

    def workspace(self) -> torch.Tensor:
        return torch.empty(gptq2d_round_workspace_size(self.handle), dtype=torch.uint8,
                           device=torch.cuda.current_device())

    def close(self):
        if getattr(self, "handle", None):
            gptq2d_factors_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def round_matrix(f: Factors, X: torch.Tensor, want_y: bool = True, workspace=None, check=True,
                 stream=None):
    """Z (int32), Y (X's dtype or None) and the objective (float64 device scalar)."""
    m, n = f.m, f.n
    Z = torch.empty((m, n), dtype=torch.int32, device=X.device)
    Y = torch.empty((m, n), dtype=X.dtype, device=X.device) if want_y else None
    obj = torch.empty(1, dtype=torch.float64, device=X.device)
    ws = workspace if workspace is not None else f.workspace()
    gptq2d_round(f.handle, X, Z, Y, obj, ws, stream)
    if check:
        gptq2d_round_check(f.handle, ws, stream)
    return Z, Y, obj


def round_batched(factors, Xs, want_y: bool = True, workspace=None, check=True, stream=None):
    """Round problem p = X[p] with factors[p] (a Factors may repeat), all in
    common launches. Returns lists of Z, Y (or None) and the objectives as one
    float64 device tensor."""
    handles = [f.handle for f in factors]
    dev = Xs[0].device
    Zs = [torch.empty((f.m, f.n), dtype=torch.int32, device=dev) for f in factors]
    Ys = [torch.empty((f.m, f.n), dtype=X.dtype, device=dev) for f, X in zip(factors, Xs)] if want_y else None
    obj = torch.empty(len(factors), dtype=torch.float64, device=dev)
    ws = workspace if workspace is not None else torch.empty(
        gptq2d_round_batched_workspace_size(handles), dtype=torch.uint8, device=dev)
    gptq2d_round_batched(handles, Xs, Zs, Ys, obj, ws, stream, shapes=[(f.m, f.n) for f in factors])
    if check:
        gptq2d_round_batched_check(ws, stream)
    return Zs, Ys, obj


def factor_batched(factors, As, Bs, check=True, stream=None, workspace=None):
    """Compute the factors of every Factors in ``factors`` (distinct) from its
    bases As[p], Bs[p], in common launches per shape."""
    handles = [f.handle for f in factors]
    ws = workspace if workspace is not None else torch.empty(
        gptq2d_factor_batched_workspace_size(len(handles)), dtype=torch.uint8, device=As[0].device)
    gptq2d_factor_batched(handles, As, Bs, ws, stream, shapes=[(f.m, f.n) for f in factors])
    if check:
        gptq2d_factor_batched_check(handles, stream)
