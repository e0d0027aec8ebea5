"""The per-workgroup trace on the GPU: tracing leaves every output bitwise unchanged, each
traced launch takes exactly one record per work item in work-list order, the records are
well formed, and launches that do not fit are run untraced and counted."""
import numpy as np
import pytest

from paper_2607_01701_amd import _lib
from paper_2607_01701_amd.workload import make_pack

from gpu_util import dev_inputs, log, run_hip

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def n_items(pack, rows):
    return _lib.t2v_build_worklist(pack.cu_seqlens, pack.heads, rows).shape[0]


def test_trace_records_and_results(monkeypatch):
    import torch
    monkeypatch.setenv("T2V_QTILE", "wide")  # 256-row forward and dQ tiles
    pack = make_pack([2000, 513, 257, 1], 3, 128, seed=70)
    dev = dev_inputs(pack)
    plain = {k: v.clone() for k, v in run_hip(pack, dev).items()}
    nf, nkv, nq = n_items(pack, 256), n_items(pack, 128), n_items(pack, 256)
    cap = nf + nkv + nq
    rec = torch.zeros(4 * cap, dtype=torch.int64, device="cuda")
    log(f"case traced step: {nf} + {nkv} + {nq} workgroups")
    _lib.t2v_trace_set(rec.data_ptr(), cap)
    try:
        traced = run_hip(pack, dev)
        n, over = _lib.t2v_trace_count()
    finally:
        _lib.t2v_trace_set(None, 0)
    for k in plain:
        assert torch.equal(plain[k], traced[k]), f"{k} changed under tracing"
    assert (n, over) == (cap, 0)
    r = rec.view(cap, 4).cpu().numpy().astype(np.uint64)
    slots = r[:, 3]
    assert np.array_equal(slots, np.repeat(np.array([0, 2, 3], dtype=np.uint64), [nf, nkv, nq]))
    t0, t1 = r[:, 1].astype(np.int64), r[:, 2].astype(np.int64)
    assert np.all(t0 > 0) and np.all(t1 >= t0)
    # the three launches run in stream order
    assert t0[nf:nf + nkv].min() >= t1[:nf].max() and t0[nf + nkv:].min() >= t1[nf:nf + nkv].max()
    cus = np.unique(r[:, 0])
    ncu = torch.cuda.get_device_properties(0).multi_processor_count
    assert 1 < len(cus) <= ncu and np.all((r[:, 0] >> np.uint64(16)) < 16)


def test_trace_overflow_runs_untraced(monkeypatch):
    import torch
    monkeypatch.setenv("T2V_QTILE", "wide")  # 256-row forward tiles
    pack = make_pack([300, 40], 2, 64, seed=71)
    dev = dev_inputs(pack)
    nf = n_items(pack, 256)
    rec = torch.zeros(4 * nf, dtype=torch.int64, device="cuda")
    _lib.t2v_trace_set(rec.data_ptr(), nf)  # room for the forward only
    try:
        run_hip(pack, dev)
        n, over = _lib.t2v_trace_count()
    finally:
        _lib.t2v_trace_set(None, 0)
    assert (n, over) == (nf, 2)
