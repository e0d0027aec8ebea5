"""C ABI on the CPU: the libraries load, export every declared symbol, and reject bad
arguments before anything is launched. No compute call is made here (no GPU); tensor
pointers are fake addresses that validation never dereferences."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2607_01701_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "t2vattn.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(t2v_\w+)\s*\(", src)))


def test_header_declares_the_abi():
    names = declared_functions()
    for n in ("t2v_attn_fwd", "t2v_attn_bwd", "t2v_last_error", "t2v_release_cache", "t2v_build_worklist"):
        assert n in names
    assert set(names) == set(_lib.EXPORTS)


def test_hip_library_exports_every_symbol():
    L = _lib.lib()
    for n in declared_functions():
        assert hasattr(L, n), n
    assert "gfx950" in _lib.t2v_version(L)


def test_checked_library_exports_every_symbol():
    L = _lib.checked_lib()
    for n in declared_functions():
        assert hasattr(L, n), n
    assert "gfx950" in _lib.t2v_version(L)


def test_host_library_exports():
    L = _lib.host_lib()
    for n in _lib.HOST_EXPORTS:
        assert hasattr(L, n), n


A = 0x100000  # fake, 16-byte aligned, never dereferenced
MB = 1 << 20


def fwd(cu, nseq=None, heads=2, head_dim=128, scale=0.125, q=A, k=A + 64 * MB, v=A + 128 * MB,
        out=A + 192 * MB, lse=A + 256 * MB):
    cu = np.asarray(cu, dtype=np.int32)
    nseq = cu.shape[0] - 1 if nseq is None else nseq
    L = _lib.lib()
    st = L.t2v_attn_fwd(q, k, v, cu.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), nseq, heads, head_dim, scale,
                        out, lse, None)
    return st, _lib.t2v_last_error(L)


def bwd(cu, **kw):
    cu = np.asarray(cu, dtype=np.int32)
    p = dict(q=A, k=A + 64 * MB, v=A + 128 * MB, out=A + 192 * MB, lse=A + 256 * MB, dout=A + 320 * MB,
             dq=A + 384 * MB, dk=A + 448 * MB, dv=A + 512 * MB, delta=A + 576 * MB, heads=2, head_dim=128,
             scale=0.125)
    p.update(kw)
    L = _lib.lib()
    st = L.t2v_attn_bwd(p["q"], p["k"], p["v"], p["out"], p["lse"],
                        cu.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), cu.shape[0] - 1, p["heads"],
                        p["head_dim"], p["scale"], p["dout"], p["dq"], p["dk"], p["dv"], p["delta"], None)
    return st, _lib.t2v_last_error(L)


INV, UNS = _lib.T2V_ERR_INVALID_ARG, _lib.T2V_ERR_UNSUPPORTED


@pytest.mark.parametrize("cu,kw,status,msg", [
    ([1, 5], {}, INV, "cu_seqlens[0]"),
    ([0, 5, 3], {}, INV, "non-decreasing"),
    ([0, 5], {"nseq": -1}, INV, "nseq"),
    ([0, 5], {"heads": 0}, INV, "heads"),
    ([0, 5], {"head_dim": 96}, UNS, "head_dim"),
    ([0, 5], {"head_dim": 256}, UNS, "head_dim"),
    ([0, 5], {"scale": float("nan")}, INV, "scale"),
    ([0, 5], {"scale": float("inf")}, INV, "scale"),
    ([0, 5], {"q": 0}, INV, "q is NULL"),
    ([0, 5], {"lse": 0}, INV, "lse is NULL"),
    ([0, 5], {"k": A + 64 * MB + 8}, INV, "aligned"),
    ([0, 5], {"out": A}, INV, "overlaps"),
    ([0, 5], {"lse": A + 128 * MB + 16}, INV, "overlaps"),
    ([0, 5], {"heads": 1 << 21}, INV, "too large"),
    ([0, 5], {"heads": (1 << 15) + 1}, INV, "too large"),  # H * D just above 2^22 at D = 128
])
def test_fwd_validation(cu, kw, status, msg):
    st, err = fwd(cu, **kw)
    assert st == status, err
    assert msg in err


def test_fwd_cu_null():
    L = _lib.lib()
    st = L.t2v_attn_fwd(A, A + MB, A + 2 * MB, None, 1, 2, 128, 0.1, A + 3 * MB, A + 4 * MB, None)
    assert st == INV


def test_fwd_empty_is_ok_without_launch():
    # T = 0: nothing to do, no HIP call is needed, pointers may even be NULL.
    st, _ = fwd([0, 0, 0], q=0, k=0, v=0, out=0, lse=0)
    assert st == _lib.T2V_OK
    st, _ = fwd([0], q=0, k=0, v=0, out=0, lse=0)
    assert st == _lib.T2V_OK


@pytest.mark.parametrize("kw,msg", [
    ({"dq": A + 448 * MB}, "overlaps"),        # dq aliases dk
    ({"dv": A}, "overlaps"),                   # dv aliases q
    ({"delta": A + 256 * MB}, "overlaps"),     # delta aliases lse
    ({"delta": A + 320 * MB - 8 * 20}, "overlaps"),  # second half of delta_ws reaches dout
    ({"dout": 0}, "dout is NULL"),
    ({"delta": 0}, "delta_ws is NULL"),
    ({"dk": A + 448 * MB + 2}, "aligned"),
    ({"head_dim": 32}, "head_dim"),
])
def test_bwd_validation(kw, msg):
    st, err = bwd([0, 7, 20], **kw)
    assert st in (INV, UNS), err
    assert msg in err


def test_bwd_empty_is_ok():
    st, _ = bwd([0, 0], q=0, k=0, v=0, out=0, lse=0, dout=0, dq=0, dk=0, dv=0, delta=0)
    assert st == _lib.T2V_OK


def test_checked_library_validates_before_any_device_call():
    """The checked library refuses bad arguments like the product library, and returns T2V_OK
    for an empty pack, without a device call: its checks start at a call's first launch."""
    with _lib.use_checked_library():
        st, err = fwd([0, 5], heads=(1 << 15) + 1)
        assert st == INV and "too large" in err
        st, _ = fwd([0, 0, 0], q=0, k=0, v=0, out=0, lse=0)
        assert st == _lib.T2V_OK
        st, err = bwd([0, 7, 20], dout=0)
        assert st == INV and "dout is NULL" in err
        assert _lib.lib() is _lib.checked_lib()
    assert _lib.lib() is not _lib.checked_lib()


def test_checked_routing_is_per_thread_and_by_environment(monkeypatch):
    """use_checked_library() routes only the calling thread; T2V_CHECKED=1 routes every call."""
    import threading
    seen = {}
    with _lib.use_checked_library():
        t = threading.Thread(target=lambda: seen.setdefault("other", _lib.lib()))
        t.start()
        t.join()
        assert _lib.lib() is _lib.checked_lib()
    assert seen["other"] is not _lib.checked_lib()
    monkeypatch.setenv("T2V_CHECKED", "1")
    assert _lib.lib() is _lib.checked_lib()
    monkeypatch.delenv("T2V_CHECKED")
    assert _lib.lib() is not _lib.checked_lib()


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(_lib, "_lib", None)
    monkeypatch.setattr(_lib, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(ImportError):
        _lib.lib()


def fwd_qk(cuq, cuk, heads=2, head_dim=128, scale=0.125, q=A, k=A + 64 * MB, v=A + 128 * MB, out=A + 192 * MB,
           lse=A + 256 * MB, nseq=None):
    P = ctypes.POINTER(ctypes.c_int32)
    cq = None if cuq is None else np.asarray(cuq, dtype=np.int32)
    ck = None if cuk is None else np.asarray(cuk, dtype=np.int32)
    n = (cq if cq is not None else ck).shape[0] - 1 if nseq is None else nseq
    L = _lib.lib()
    st = L.t2v_attn_fwd_qk(q, k, v, None if cq is None else cq.ctypes.data_as(P),
                           None if ck is None else ck.ctypes.data_as(P), n, heads, head_dim, scale, out, lse, None)
    return st, _lib.t2v_last_error(L)


@pytest.mark.parametrize("cuq,cuk,kw,msg", [
    ([0, 5, 9], [0, 0, 3], {}, "has queries but no keys"),
    ([0, 0, 9], [0, 4, 7], {}, "has keys but no queries"),
    ([0, 5, 9], [0, 3, 1], {}, "cu_seqlens_k"),
    ([0, 5, 9], [1, 3, 4], {}, "cu_seqlens_k"),
    ([0, 5, 9], None, {}, "NULL"),
    (None, [0, 5, 9], {}, "NULL"),
    ([0, 5, 9], [0, 2, 3], {"head_dim": 96}, "head_dim"),
    # out spans Tq = 9 rows of 2 x 128 bf16 (4,608 bytes): it reaches v placed right after it
    ([0, 5, 9], [0, 2, 3], {"out": A + 192 * MB, "v": A + 192 * MB + 4096}, "overlaps"),
    # lse spans H * Tq floats = 72 bytes
    ([0, 5, 9], [0, 2, 3], {"lse": A + 256 * MB, "k": A + 256 * MB + 64}, "overlaps"),
])
def test_fwd_qk_validation(cuq, cuk, kw, msg):
    st, err = fwd_qk(cuq, cuk, **kw)
    assert st in (INV, UNS), err
    assert msg in err


def test_fwd_qk_sizes_follow_each_stream():
    """k and v are sized by Tk, not Tq. With Tq = 9 and Tk = 3 (k spans 1,536 bytes), out placed
    2 KB after k overlaps nothing; lse is then made to overlap out, so validation still stops the
    call, and the message shows which check fired."""
    st, err = fwd_qk([0, 5, 9], [0, 2, 3], k=A + 64 * MB, out=A + 64 * MB + 2048, lse=A + 64 * MB + 2048 + 256)
    assert st == INV
    assert "input k" not in err and "overlaps output" in err


def test_fwd_qk_empty_is_ok():
    st, _ = fwd_qk([0, 0, 0], [0, 0, 0], q=0, k=0, v=0, out=0, lse=0)
    assert st == _lib.T2V_OK


def test_bwd_qk_validation():
    P = ctypes.POINTER(ctypes.c_int32)
    cq = np.asarray([0, 4, 10], dtype=np.int32)
    ck = np.asarray([0, 0, 6], dtype=np.int32)
    L = _lib.lib()
    st = L.t2v_attn_bwd_qk(A, A + 64 * MB, A + 128 * MB, A + 192 * MB, A + 256 * MB, cq.ctypes.data_as(P),
                           ck.ctypes.data_as(P), 2, 2, 128, 0.125, A + 320 * MB, A + 384 * MB, A + 448 * MB,
                           A + 512 * MB, A + 576 * MB, None)
    assert st == INV and "no keys" in _lib.t2v_last_error(L)
    ck = np.asarray([0, 3, 6], dtype=np.int32)
    # dk (Tk = 6 rows, 3 KB) aliasing dv
    st = L.t2v_attn_bwd_qk(A, A + 64 * MB, A + 128 * MB, A + 192 * MB, A + 256 * MB, cq.ctypes.data_as(P),
                           ck.ctypes.data_as(P), 2, 2, 128, 0.125, A + 320 * MB, A + 384 * MB, A + 448 * MB,
                           A + 448 * MB + 1024, A + 576 * MB, None)
    assert st == INV and "overlaps" in _lib.t2v_last_error(L)


def test_mfma_probe_validation():
    """The MFMA probe rejects NULL buffers and out-of-range sizes before touching the GPU."""
    L = _lib.lib()
    d = ctypes.c_double()
    ref = ctypes.byref(d)
    assert L.t2v_probe_mfma_peak(None, 4, 10, None, ref, ref, ref) == _lib.T2V_ERR_INVALID_ARG
    assert "NULL" in _lib.t2v_last_error(L)
    fake = ctypes.c_void_p(4096)  # never dereferenced: the sizes are rejected first
    for blocks, iters in ((0, 10), (4, 0), (1 << 21, 10), (4, 1 << 25)):
        assert L.t2v_probe_mfma_peak(fake, blocks, iters, None, ref, ref, ref) == _lib.T2V_ERR_INVALID_ARG
        assert "blocks must be" in _lib.t2v_last_error(L)
    assert L.t2v_probe_mfma_peak(fake, 4, 10, None, None, ref, ref) == _lib.T2V_ERR_INVALID_ARG


def test_trace_set_validation():
    """The workgroup trace rejects a negative capacity, a capacity without a buffer and a
    misaligned buffer; disarming (NULL, 0) is always accepted."""
    L = _lib.lib()
    assert L.t2v_trace_set(None, -1) == _lib.T2V_ERR_INVALID_ARG
    assert L.t2v_trace_set(None, 5) == _lib.T2V_ERR_INVALID_ARG
    assert L.t2v_trace_set(ctypes.c_void_p(4100), 5) == _lib.T2V_ERR_INVALID_ARG  # not 8-byte aligned
    assert "aligned" in _lib.t2v_last_error(L)
    assert L.t2v_trace_set(None, 0) == _lib.T2V_OK
    assert _lib.t2v_trace_count() == (0, 0)


C_CONSUMER = r"""
#include <stdio.h>
#include "t2vattn.h"

int main(void) {
  const int32_t cu[4] = {0, 300, 300, 700};  /* the middle clip is empty */
  int32_t items[4 * 16];
  int n = -1;
  double ms = 0.0, lb = 0.0;
  if (t2v_build_worklist(cu, 3, 2, 256, T2V_ORDER_LONGEST_FIRST, NULL, 0, &n) != T2V_OK || n != 8) return 1;
  if (t2v_build_worklist(cu, 3, 2, 256, T2V_ORDER_LONGEST_FIRST, items, 16, &n) != T2V_OK) return 2;
  if (t2v_plan_makespan(items, n, 256, 4, &ms, &lb) != T2V_OK || ms < lb || lb <= 0.0) return 3;
#ifdef WITH_GPU_LIBRARY
  /* validation happens before any device work: a NULL tensor is refused */
  if (t2v_attn_fwd(NULL, NULL, NULL, cu, 3, 2, 128, 0.1f, NULL, NULL, NULL) != T2V_ERR_INVALID_ARG) return 4;
#else
  if (t2v_build_worklist(NULL, 3, 2, 256, T2V_ORDER_LONGEST_FIRST, NULL, 0, &n) != T2V_ERR_INVALID_ARG) return 4;
#endif
  printf("%s | %s\n", t2v_version(), t2v_last_error());
  return 0;
}
"""


@pytest.mark.parametrize("lib", ["t2vattn_host", "t2vattn", "t2vattn_checked"])
def test_header_is_plain_c_and_links(tmp_path, lib):
    """A C99 program that includes only the public header, built with -pedantic -Werror,
    links against the host-only and the GPU library and runs (no device work)."""
    import shutil
    import subprocess
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    src = tmp_path / "consumer.c"
    src.write_text(C_CONSUMER)
    exe = str(tmp_path / "consumer")
    libdir = os.path.dirname(_lib.LIB_PATH)
    gpu = ["-DWITH_GPU_LIBRARY"] if lib != "t2vattn_host" else []
    r = subprocess.run(["gcc", "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror", *gpu, "-I",
                        os.path.join(ROOT, "include"), str(src), "-o", exe, f"-L{libdir}", f"-l{lib}",
                        f"-Wl,-rpath,{libdir}"], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, (r.returncode, r.stdout, r.stderr)
    assert "libt2vattn" in r.stdout
    assert ("NULL" if lib != "t2vattn_host" else "cu_seqlens") in r.stdout  # the refused call's message


# ----------------------------------------------------------------- torch binding checks
#
# The C ABI sees only pointers, so the torch wrappers check every tensor's shape, dtype and
# layout, and that cu_seqlens ends at the packed row count, before anything is launched.
# These run on CPU tensors: the shape, dtype and layout checks come before the device check.

def _cpu(shape, dtype=None):
    import torch
    return torch.zeros(shape, dtype=torch.bfloat16 if dtype is None else dtype)


@pytest.mark.parametrize("case,msg", [
    ("cu_short", "does not match the 10 rows"),
    ("cu_long", "does not match the 10 rows"),
    ("out_shape", "out has shape"),
    ("lse_dtype", "lse has dtype"),
    ("lse_shape", "lse has shape"),
    ("q_noncontig", "q must be contiguous"),
    ("cpu_tensor", "must be a CUDA tensor"),
])
def test_attn_fwd_wrapper_rejects_before_launch(case, msg):
    import torch
    from paper_2607_01701_amd import attn_fwd
    T, H, D = 10, 2, 64
    q, k, v = _cpu((T, H, D)), _cpu((T, H, D)), _cpu((T, H, D))
    cu, kw = [0, 4, 10], {}
    if case == "cu_short":
        cu = [0, 4, 9]
    elif case == "cu_long":
        cu = [0, 4, 11]
    elif case == "out_shape":
        kw["out"] = _cpu((T + 1, H, D))
    elif case == "lse_dtype":
        kw["lse"] = _cpu((H, T), torch.bfloat16)
    elif case == "lse_shape":
        kw["lse"] = _cpu((T, H), torch.float32)
    elif case == "q_noncontig":
        q = _cpu((T, D, H)).transpose(1, 2)
    with pytest.raises(ValueError, match=msg):
        attn_fwd(q, k, v, cu, 0.125, **kw)


@pytest.mark.parametrize("case,msg", [
    ("cu_short", "does not match the 10 rows"),
    ("cu_k_short", "cu_seqlens_k.* does not match the 6 rows"),
    ("dq_shape", "dq has shape"),
    ("dk_shape", "dk has shape"),
    ("dv_dtype", "dv has dtype"),
    ("ws_shape", "delta_ws has shape"),
    ("ws_dtype", "delta_ws has dtype"),
    ("lse_shape", "lse has shape"),
])
def test_attn_bwd_wrapper_rejects_before_launch(case, msg):
    import torch
    from paper_2607_01701_amd import attn_bwd
    T, Tk, H, D = 10, 6, 2, 64
    cross = case == "cu_k_short"
    nk = Tk if cross else T
    q, out, g = _cpu((T, H, D)), _cpu((T, H, D)), _cpu((T, H, D))
    k, v = _cpu((nk, H, D)), _cpu((nk, H, D))
    lse = _cpu((H, T), torch.float32)
    cu, kw = [0, 4, 10], {}
    if cross:
        kw["cu_seqlens_k"] = [0, 2, 5]
    if case == "cu_short":
        cu = [0, 4, 8]
    elif case == "dq_shape":
        kw["dq"] = _cpu((T, H, D + 1))
    elif case == "dk_shape":
        kw["dk"] = _cpu((T - 1, H, D))
    elif case == "dv_dtype":
        kw["dv"] = _cpu((T, H, D), torch.float16)
    elif case == "ws_shape":
        kw["delta_ws"] = _cpu((H, T), torch.float32)  # [H, T]: half of what the library writes
    elif case == "ws_dtype":
        kw["delta_ws"] = _cpu((2, H, T), torch.bfloat16)
    elif case == "lse_shape":
        lse = _cpu((H, T + 1), torch.float32)
    with pytest.raises(ValueError, match=msg):
        attn_bwd(q, k, v, out, lse, g, cu, 0.125, **kw)


def test_noalloc_refuses_a_pack_beyond_its_scratch_before_any_device_call():
    """t2v_attn_bwd_noalloc keeps Delta / lse (8 * heads * T bytes) and the work lists in a
    64 MiB static array; a larger call is refused during validation (fake pointers: nothing
    is dereferenced or launched)."""
    L = _lib.lib()
    H, D = 64, 64
    T = (64 << 20) // (8 * H) + 64
    cu = np.array([0, T], dtype=np.int32)
    p = [A + i * 4096 * MB for i in range(9)]
    st = L.t2v_attn_bwd_noalloc(p[0], p[1], p[2], p[3], p[4], cu.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), 1,
                                H, D, 0.125, p[5], p[6], p[7], p[8], None)
    msg = _lib.t2v_last_error(L)
    assert st == INV and "bytes of scratch" in msg and "67108864" in msg, (st, msg)
