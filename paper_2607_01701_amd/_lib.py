"""ctypes binding to libt2vattn: argument marshalling only.

Every step of the computation runs in the HIP library; this module only turns
torch tensors and numpy arrays into pointers and sizes, and raises on a non-OK
status. There is no fallback: if the library is missing, calls raise.
"""
from __future__ import annotations

import contextlib
import ctypes
import os
import threading

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libt2vattn.so")
HOST_LIB_PATH = os.path.join(_PKG, "libt2vattn_host.so")
# The same calls with bounds checks (debugging; see "Checked library" in include/t2vattn.h).
CHECKED_LIB_PATH = os.path.join(_PKG, "libt2vattn_checked.so")

T2V_OK = 0
T2V_ERR_INVALID_ARG = 1
T2V_ERR_UNSUPPORTED = 2
T2V_ERR_HIP = 3
T2V_ERR_OOM = 4
T2V_ERR_BOUNDS = 5
STATUS_NAMES = {0: "T2V_OK", 1: "T2V_ERR_INVALID_ARG", 2: "T2V_ERR_UNSUPPORTED", 3: "T2V_ERR_HIP",
                4: "T2V_ERR_OOM", 5: "T2V_ERR_BOUNDS"}

ORDER_NATURAL = 0
ORDER_LONGEST_FIRST = 1

# Symbols declared in include/t2vattn.h.
EXPORTS = ("t2v_attn_fwd", "t2v_attn_bwd", "t2v_attn_fwd_qk", "t2v_attn_bwd_qk", "t2v_last_error",
           "t2v_release_cache", "t2v_build_worklist", "t2v_plan_makespan", "t2v_timing_enable", "t2v_kernel_times",
           "t2v_version", "t2v_list_schedule", "t2v_plan_cascades", "t2v_probe_mfma_peak", "t2v_trace_set",
           "t2v_trace_count", "t2v_attn_bwd_noalloc")
KERNEL_SLOTS = ("fwd", "bwd_pre", "bwd_dkdv", "bwd_dq")
HOST_EXPORTS = ("t2v_last_error", "t2v_build_worklist", "t2v_plan_makespan", "t2v_version", "t2v_list_schedule",
                "t2v_plan_cascades")

_vp = ctypes.c_void_p
_i32p = ctypes.POINTER(ctypes.c_int32)
_f32p = ctypes.c_void_p  # device float* passed as an address


class T2VError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


def _declare(lib, full: bool):
    lib.t2v_last_error.restype = ctypes.c_char_p
    lib.t2v_last_error.argtypes = []
    lib.t2v_version.restype = ctypes.c_char_p
    lib.t2v_version.argtypes = []
    lib.t2v_build_worklist.restype = ctypes.c_int
    lib.t2v_build_worklist.argtypes = [_i32p, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, _i32p,
                                       ctypes.c_int, ctypes.POINTER(ctypes.c_int)]
    lib.t2v_plan_makespan.restype = ctypes.c_int
    lib.t2v_plan_makespan.argtypes = [_i32p, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                      ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]
    _dp = ctypes.POINTER(ctypes.c_double)
    lib.t2v_list_schedule.restype = ctypes.c_int
    lib.t2v_list_schedule.argtypes = [ctypes.c_int, _i32p, _i32p, _i32p, _dp, ctypes.c_int, _dp, _dp]
    lib.t2v_plan_cascades.restype = ctypes.c_int
    lib.t2v_plan_cascades.argtypes = [ctypes.c_int, _i32p, _i32p, ctypes.c_int, _i32p, _dp, _dp, ctypes.c_double,
                                      ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_double, ctypes.c_int,
                                      ctypes.c_uint64, _i32p, _dp, _dp]
    if full:
        lib.t2v_attn_fwd.restype = ctypes.c_int
        lib.t2v_attn_fwd.argtypes = [_vp, _vp, _vp, _i32p, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                     ctypes.c_float, _vp, _f32p, _vp]
        lib.t2v_attn_bwd.restype = ctypes.c_int
        lib.t2v_attn_bwd.argtypes = [_vp, _vp, _vp, _vp, _f32p, _i32p, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                     ctypes.c_float, _vp, _vp, _vp, _vp, _f32p, _vp]
        lib.t2v_attn_bwd_noalloc.restype = ctypes.c_int
        lib.t2v_attn_bwd_noalloc.argtypes = [_vp, _vp, _vp, _vp, _f32p, _i32p, ctypes.c_int, ctypes.c_int,
                                             ctypes.c_int, ctypes.c_float, _vp, _vp, _vp, _vp, _vp]
        lib.t2v_attn_fwd_qk.restype = ctypes.c_int
        lib.t2v_attn_fwd_qk.argtypes = [_vp, _vp, _vp, _i32p, _i32p, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                        ctypes.c_float, _vp, _f32p, _vp]
        lib.t2v_attn_bwd_qk.restype = ctypes.c_int
        lib.t2v_attn_bwd_qk.argtypes = [_vp, _vp, _vp, _vp, _f32p, _i32p, _i32p, ctypes.c_int, ctypes.c_int,
                                        ctypes.c_int, ctypes.c_float, _vp, _vp, _vp, _vp, _f32p, _vp]
        lib.t2v_release_cache.restype = None
        lib.t2v_release_cache.argtypes = []
        lib.t2v_timing_enable.restype = ctypes.c_int
        lib.t2v_timing_enable.argtypes = [ctypes.c_int]
        lib.t2v_kernel_times.restype = ctypes.c_int
        lib.t2v_kernel_times.argtypes = [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int)]
        lib.t2v_probe_mfma_peak.restype = ctypes.c_int
        lib.t2v_trace_set.restype = ctypes.c_int
        lib.t2v_trace_set.argtypes = [_vp, ctypes.c_int64]
        lib.t2v_trace_count.restype = ctypes.c_int
        lib.t2v_trace_count.argtypes = [ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_int)]
        lib.t2v_probe_mfma_peak.argtypes = [_vp, ctypes.c_int, ctypes.c_int, _vp, _dp, _dp, _dp]
    return lib


_lib = None
_host_lib = None
_checked_lib = None
_route = threading.local()  # .checked: this thread's calls go to the checked library


def lib():
    """The HIP library (loaded once), or the checked library inside use_checked_library() or
    when the environment sets T2V_CHECKED=1 (to run a whole program against it). Raises if
    it has not been built."""
    global _lib
    if getattr(_route, "checked", False) or os.environ.get("T2V_CHECKED") == "1":
        return checked_lib()
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2607_01701_amd.build`")
        _lib = _declare(ctypes.CDLL(LIB_PATH), full=True)
    return _lib


def checked_lib():
    """The checked library (same calls, bounds-checked; loaded once). Raises if not built."""
    global _checked_lib
    if _checked_lib is None:
        if not os.path.exists(CHECKED_LIB_PATH):
            raise ImportError(f"{CHECKED_LIB_PATH} is missing: build it with `python -m paper_2607_01701_amd.build`")
        _checked_lib = _declare(ctypes.CDLL(CHECKED_LIB_PATH), full=True)
    return _checked_lib


@contextlib.contextmanager
def use_checked_library():
    """Inside the block, this thread's calls through this module go to the checked library."""
    prev = getattr(_route, "checked", False)
    _route.checked = True
    try:
        yield checked_lib()
    finally:
        _route.checked = prev


def host_lib():
    """The host-only scheduler library (g++ build, no HIP)."""
    global _host_lib
    if _host_lib is None:
        if not os.path.exists(HOST_LIB_PATH):
            raise ImportError(f"{HOST_LIB_PATH} is missing: build it with `python -m paper_2607_01701_amd.build`")
        _host_lib = _declare(ctypes.CDLL(HOST_LIB_PATH), full=False)
    return _host_lib


def _cu_array(cu_seqlens) -> np.ndarray:
    a = np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int32))
    if a.ndim != 1 or a.shape[0] < 1:
        raise ValueError("cu_seqlens must be a 1-D array with nseq + 1 entries")
    return a


def _check(L, status: int):
    if status != T2V_OK:
        raise T2VError(status, L.t2v_last_error().decode())


# ----------------------------------------------------------------- raw C-ABI names

def t2v_attn_fwd(q, k, v, cu_seqlens, nseq, heads, head_dim, scale, out, lse, stream):
    """Direct call of t2v_attn_fwd with integer addresses; returns the status."""
    cu = _cu_array(cu_seqlens)
    return lib().t2v_attn_fwd(q, k, v, cu.ctypes.data_as(_i32p), nseq, heads, head_dim, scale, out, lse, stream)


def t2v_attn_bwd(q, k, v, out, lse, cu_seqlens, nseq, heads, head_dim, scale, dout, dq, dk, dv, delta_ws,
                 stream):
    """Direct call of t2v_attn_bwd with integer addresses; returns the status."""
    cu = _cu_array(cu_seqlens)
    return lib().t2v_attn_bwd(q, k, v, out, lse, cu.ctypes.data_as(_i32p), nseq, heads, head_dim, scale, dout,
                              dq, dk, dv, delta_ws, stream)


def t2v_attn_bwd_noalloc(q, k, v, out, lse, cu_seqlens, nseq, heads, head_dim, scale, dout, dq, dk, dv, stream):
    """Direct call of t2v_attn_bwd_noalloc with integer addresses; returns the status."""
    cu = _cu_array(cu_seqlens)
    return lib().t2v_attn_bwd_noalloc(q, k, v, out, lse, cu.ctypes.data_as(_i32p), nseq, heads, head_dim, scale,
                                      dout, dq, dk, dv, stream)


def t2v_attn_fwd_qk(q, k, v, cu_seqlens_q, cu_seqlens_k, nseq, heads, head_dim, scale, out, lse, stream):
    """Direct call of t2v_attn_fwd_qk with integer addresses; returns the status."""
    cq, ck = _cu_array(cu_seqlens_q), _cu_array(cu_seqlens_k)
    return lib().t2v_attn_fwd_qk(q, k, v, cq.ctypes.data_as(_i32p), ck.ctypes.data_as(_i32p), nseq, heads, head_dim,
                                 scale, out, lse, stream)


def t2v_attn_bwd_qk(q, k, v, out, lse, cu_seqlens_q, cu_seqlens_k, nseq, heads, head_dim, scale, dout, dq, dk, dv,
                    delta_ws, stream):
    """Direct call of t2v_attn_bwd_qk with integer addresses; returns the status."""
    cq, ck = _cu_array(cu_seqlens_q), _cu_array(cu_seqlens_k)
    return lib().t2v_attn_bwd_qk(q, k, v, out, lse, cq.ctypes.data_as(_i32p), ck.ctypes.data_as(_i32p), nseq, heads,
                                 head_dim, scale, dout, dq, dk, dv, delta_ws, stream)


def t2v_last_error(L=None) -> str:
    return (L or lib()).t2v_last_error().decode()


def t2v_release_cache() -> None:
    lib().t2v_release_cache()


def t2v_timing_enable(on: bool) -> None:
    _check(lib(), lib().t2v_timing_enable(1 if on else 0))


def t2v_kernel_times() -> dict:
    """{kernel: (summed ms, launches)} since the previous read."""
    ms = (ctypes.c_double * 4)()
    n = (ctypes.c_int * 4)()
    _check(lib(), lib().t2v_kernel_times(ms, n))
    return {name: (ms[i], n[i]) for i, name in enumerate(KERNEL_SLOTS)}


def t2v_probe_mfma_peak(rec, blocks: int, iters: int, stream) -> dict:
    """MFMA throughput probe (measurement context); rec: device address of 3 * blocks uint64."""
    ms, tf, ghz = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
    _check(lib(), lib().t2v_probe_mfma_peak(rec, int(blocks), int(iters), stream, ctypes.byref(ms),
                                            ctypes.byref(tf), ctypes.byref(ghz)))
    return {"ms": ms.value, "tflops": tf.value, "ghz": ghz.value}


def t2v_trace_set(dev_records, capacity: int) -> None:
    """Arms (device address of 4 * capacity uint64) or disarms (None, 0) the workgroup trace."""
    _check(lib(), lib().t2v_trace_set(dev_records, int(capacity)))


def t2v_trace_count() -> tuple:
    """(records taken since the trace was armed, launches that did not fit)."""
    n, o = ctypes.c_int64(), ctypes.c_int()
    _check(lib(), lib().t2v_trace_count(ctypes.byref(n), ctypes.byref(o)))
    return n.value, o.value


def t2v_version(L=None) -> str:
    return (L or lib()).t2v_version().decode()


def t2v_build_worklist(cu_seqlens, heads: int, block: int, order: int = ORDER_LONGEST_FIRST, L=None) -> np.ndarray:
    """The scheduler's work list as an int32 array [n_items, 4] = (row0, len, tile0, head)."""
    L = L or host_lib()
    cu = _cu_array(cu_seqlens)
    nseq = cu.shape[0] - 1
    n = ctypes.c_int(0)
    _check(L, L.t2v_build_worklist(cu.ctypes.data_as(_i32p), nseq, heads, block, order, None, 0, ctypes.byref(n)))
    items = np.zeros((n.value, 4), dtype=np.int32)
    _check(L, L.t2v_build_worklist(cu.ctypes.data_as(_i32p), nseq, heads, block, order,
                                   items.ctypes.data_as(_i32p), n.value, ctypes.byref(n)))
    return items


def t2v_plan_makespan(items: np.ndarray, block: int, slots: int, L=None):
    """(greedy list-scheduling makespan, lower bound) of a work list, in rows x keys."""
    L = L or host_lib()
    it = np.ascontiguousarray(items, dtype=np.int32)
    ms, lb = ctypes.c_double(0), ctypes.c_double(0)
    _check(L, L.t2v_plan_makespan(it.ctypes.data_as(_i32p), it.shape[0], block, slots, ctypes.byref(ms),
                                  ctypes.byref(lb)))
    return ms.value, lb.value


# ----------------------------------------------------------------- torch convenience

def _stream_handle(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _check_tensor(t, name, shape, dtype=None):
    """Shape, dtype, layout and device of a tensor passed to the library, checked in that order
    (the library sees only pointers, so a wrong size would be read or written past its end)."""
    import torch
    dtype = torch.bfloat16 if dtype is None else dtype
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if t.dtype != dtype:
        raise ValueError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _check_on_device(named):
    """Last of the checks: every tensor is on a GPU (the same one as the first)."""
    first = None
    for name, t in named:
        if not t.is_cuda:
            raise ValueError(f"{name} must be a CUDA tensor")
        if first is None:
            first = t.device
        elif t.device != first:
            raise ValueError(f"{name} is on {t.device}, the other tensors on {first}")


def _check_offsets(cu: np.ndarray, rows: int, name: str):
    """The last offset must equal the packed tensor's row count (T = cu_seqlens[nseq])."""
    if int(cu[-1]) != int(rows):
        raise ValueError(f"{name}[-1] = {int(cu[-1])} does not match the {int(rows)} rows of the packed tensors")


def attn_fwd(q, k, v, cu_seqlens, scale: float, out=None, lse=None, stream=None, cu_seqlens_k=None):
    """Forward pass on torch tensors q [Tq, H, D], k, v [Tk, H, D] (bf16, on the GPU).

    cu_seqlens holds the query offsets; cu_seqlens_k the key offsets (None: self-attention,
    Tk = Tq, t2v_attn_fwd; otherwise t2v_attn_fwd_qk). Returns (out [Tq, H, D] bf16, lse [H, Tq] fp32).
    """
    import torch
    T, H, D = q.shape
    Tk = T if cu_seqlens_k is None else k.shape[0]
    _check_tensor(q, "q", (T, H, D))
    for name, t in (("k", k), ("v", v)):
        _check_tensor(t, name, (Tk, H, D))
    cu = _cu_array(cu_seqlens)
    _check_offsets(cu, T, "cu_seqlens")
    if cu_seqlens_k is not None:
        _check_offsets(_cu_array(cu_seqlens_k), Tk, "cu_seqlens_k")
    if out is None:
        out = torch.empty_like(q)
    if lse is None:
        lse = torch.empty((H, T), dtype=torch.float32, device=q.device)
    _check_tensor(out, "out", (T, H, D))
    _check_tensor(lse, "lse", (H, T), torch.float32)
    _check_on_device((("q", q), ("k", k), ("v", v), ("out", out), ("lse", lse)))
    L = lib()
    if cu_seqlens_k is None:
        st = L.t2v_attn_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), cu.ctypes.data_as(_i32p), cu.shape[0] - 1, H,
                            D, float(scale), out.data_ptr(), lse.data_ptr(), _stream_handle(stream))
    else:
        ck = _cu_array(cu_seqlens_k)
        st = L.t2v_attn_fwd_qk(q.data_ptr(), k.data_ptr(), v.data_ptr(), cu.ctypes.data_as(_i32p),
                               ck.ctypes.data_as(_i32p), cu.shape[0] - 1, H, D, float(scale), out.data_ptr(),
                               lse.data_ptr(), _stream_handle(stream))
    _check(L, st)
    return out, lse


def attn_bwd(q, k, v, out, lse, dout, cu_seqlens, scale: float, dq=None, dk=None, dv=None, delta_ws=None,
             stream=None, cu_seqlens_k=None):
    """Backward pass; returns (dq [Tq, H, D], dk, dv [Tk, H, D]) in bf16 (see attn_fwd for cu_seqlens_k)."""
    import torch
    T, H, D = q.shape
    Tk = T if cu_seqlens_k is None else k.shape[0]
    for name, t in (("q", q), ("out", out), ("dout", dout)):
        _check_tensor(t, name, (T, H, D))
    for name, t in (("k", k), ("v", v)):
        _check_tensor(t, name, (Tk, H, D))
    _check_tensor(lse, "lse", (H, T), torch.float32)
    cu = _cu_array(cu_seqlens)
    _check_offsets(cu, T, "cu_seqlens")
    if cu_seqlens_k is not None:
        _check_offsets(_cu_array(cu_seqlens_k), Tk, "cu_seqlens_k")
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(k) if dk is None else dk
    dv = torch.empty_like(k) if dv is None else dv
    if delta_ws is None:
        delta_ws = torch.empty((2, H, T), dtype=torch.float32, device=q.device)
    _check_tensor(dq, "dq", (T, H, D))
    _check_tensor(dk, "dk", (Tk, H, D))
    _check_tensor(dv, "dv", (Tk, H, D))
    _check_tensor(delta_ws, "delta_ws", (2, H, T), torch.float32)
    _check_on_device((("q", q), ("k", k), ("v", v), ("out", out), ("lse", lse), ("dout", dout), ("dq", dq),
                      ("dk", dk), ("dv", dv), ("delta_ws", delta_ws)))
    L = lib()
    if cu_seqlens_k is None:
        st = L.t2v_attn_bwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), lse.data_ptr(),
                            cu.ctypes.data_as(_i32p), cu.shape[0] - 1, H, D, float(scale), dout.data_ptr(),
                            dq.data_ptr(), dk.data_ptr(), dv.data_ptr(), delta_ws.data_ptr(), _stream_handle(stream))
    else:
        ck = _cu_array(cu_seqlens_k)
        st = L.t2v_attn_bwd_qk(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), lse.data_ptr(),
                               cu.ctypes.data_as(_i32p), ck.ctypes.data_as(_i32p), cu.shape[0] - 1, H, D, float(scale),
                               dout.data_ptr(), dq.data_ptr(), dk.data_ptr(), dv.data_ptr(), delta_ws.data_ptr(),
                               _stream_handle(stream))
    _check(L, st)
    return dq, dk, dv
