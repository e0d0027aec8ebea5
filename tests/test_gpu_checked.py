"""The checked library on the GPU (libt2vattn_checked.so: the same sources with every work
list checked on the host against cu_seqlens and every row the kernels copy into LDS checked
on the device against its clip). On packs that reach every kernel form (edge lengths, several
tiles, empty clips, head_dim 64 and 128, narrow and wide tiles, cross-attention with the
dK/dV loop split, the persistent grid, the no-allocation backward) every call returns T2V_OK,
so no work item and no copied row leaves its clip, and every output equals the product
library's bitwise. With the canary (bounds taken one row short) the kernels' checks report,
and the next call without it is clean again."""
import pytest

from paper_2607_01701_amd import _lib
from paper_2607_01701_amd.workload import make_pack, make_pack_qk

from gpu_util import dev_inputs, log, run_hip

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


PACKS = [
    ("edge_lengths_d128", lambda: make_pack([1, 2, 63, 64, 65, 127, 128, 129, 1000], 2, 128, seed=61)),
    ("edge_lengths_d64", lambda: make_pack([1, 2, 63, 64, 65, 127, 128, 129, 1000], 2, 64, seed=62)),
    ("zero_length_clips", lambda: make_pack([0, 37, 0, 300, 0], 2, 128, seed=63)),
    ("multi_tile_d128", lambda: make_pack([2000, 513, 257, 4100], 3, 128, seed=64)),
    ("cross_d128", lambda: make_pack_qk([1000, 5, 2000, 129], [256, 3, 77, 600], 2, 128, seed=65)),
    # short key segments against long query segments: the dK/dV loops are split into pieces
    ("cross_split_d128", lambda: make_pack_qk([9000, 300, 4500, 0, 2600], [100, 50, 256, 0, 1], 2, 128, seed=66)),
    ("cross_split_d64", lambda: make_pack_qk([7000, 2100, 65], [33, 500, 129], 3, 64, seed=67)),
]
MODES = [("default", {}), ("narrow", {"T2V_QTILE": "narrow"}), ("wide", {"T2V_QTILE": "wide"}),
         ("persistent", {"T2V_PERSISTENT": "1"})]


@pytest.mark.parametrize("mode,env", MODES, ids=[m[0] for m in MODES])
def test_checked_library_finds_nothing_and_matches(mode, env, monkeypatch):
    import torch
    for k, v in env.items():
        monkeypatch.setenv(k, v)
    for name, make in PACKS:
        pack = make()
        d = dev_inputs(pack)
        log(f"case checked library {mode}: {name}")
        want = run_hip(pack, d)
        with _lib.use_checked_library():
            got = run_hip(pack, d)  # raises T2VError (T2V_ERR_BOUNDS) on any violation
        for k in want:
            assert torch.equal(got[k], want[k]), f"{name} {mode}: {k} differs from the product library"


def test_checked_no_allocation_backward():
    import torch
    pack = make_pack([1, 65, 300, 2049], 2, 128, seed=68)
    d = dev_inputs(pack)
    log("case checked library: no-allocation backward")
    want = run_hip(pack, d)
    H, D, T = pack.heads, pack.head_dim, pack.total_tokens
    nseq = len(pack.cu_seqlens) - 1
    outs = {n: torch.empty_like(d["q"]) for n in ("dq", "dk", "dv")}
    with _lib.use_checked_library():
        st = _lib.t2v_attn_bwd_noalloc(d["q"].data_ptr(), d["k"].data_ptr(), d["v"].data_ptr(),
                                       want["out"].data_ptr(), want["lse"].data_ptr(), pack.cu_seqlens, nseq, H, D,
                                       pack.scale, d["dout"].data_ptr(), outs["dq"].data_ptr(),
                                       outs["dk"].data_ptr(), outs["dv"].data_ptr(),
                                       torch.cuda.current_stream().cuda_stream)
        assert st == _lib.T2V_OK, _lib.t2v_last_error()
    torch.cuda.synchronize()
    for k in outs:
        assert torch.equal(outs[k], want[k]), k


def test_canary_makes_the_kernel_checks_report(monkeypatch):
    """T2V_CHECK_CANARY=1 takes one row off every bound the kernels check, so the last row
    of every clip is reported (the copies themselves are unchanged); without it the same
    calls are clean."""
    from paper_2607_01701_amd import attn_bwd, attn_fwd
    pack = make_pack([70, 300], 2, 128, seed=69)
    d = dev_inputs(pack)
    log("case checked library: canary")
    with _lib.use_checked_library():
        monkeypatch.setenv("T2V_CHECK_CANARY", "1")
        with pytest.raises(_lib.T2VError) as e:
            attn_fwd(d["q"], d["k"], d["v"], pack.cu_seqlens, pack.scale)
        assert e.value.status == _lib.T2V_ERR_BOUNDS
        assert "forward kernel" in str(e.value) and "-row segment" in str(e.value), str(e.value)
        monkeypatch.delenv("T2V_CHECK_CANARY")
        out, lse = attn_fwd(d["q"], d["k"], d["v"], pack.cu_seqlens, pack.scale)
        monkeypatch.setenv("T2V_CHECK_CANARY", "1")
        with pytest.raises(_lib.T2VError) as e:
            attn_bwd(d["q"], d["k"], d["v"], out, lse, d["dout"], pack.cu_seqlens, pack.scale)
        assert e.value.status == _lib.T2V_ERR_BOUNDS
        assert "dK/dV kernel" in str(e.value) or "dQ kernel" in str(e.value), str(e.value)
        monkeypatch.delenv("T2V_CHECK_CANARY")
        attn_bwd(d["q"], d["k"], d["v"], out, lse, d["dout"], pack.cu_seqlens, pack.scale)
