"""T2V_PERSISTENT=1 (forward and dK/dV kernels on a persistent grid, each workgroup striding
over the work list) gives results bitwise equal to the default one-workgroup-per-item launch,
on self and cross packs, both head dims, a pack whose dK/dV loop is split, and with the
workgroup trace armed (one record per item either way)."""
import numpy as np
import pytest

from paper_2607_01701_amd.workload import make_pack, make_pack_qk

from gpu_util import dev_inputs, log, run_hip

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


PACKS = [
    ("self D=128", lambda: make_pack([3000, 1, 700, 129, 2048, 64], 3, 128, seed=71)),
    ("self D=64", lambda: make_pack([1500, 513, 257, 2], 2, 64, seed=72)),
    ("cross", lambda: make_pack_qk([2000, 63, 1000], [256, 1, 77], 2, 128, seed=73)),
    ("split loop", lambda: make_pack_qk([9000, 4500], [100, 256], 1, 128, seed=74)),
]


@pytest.mark.parametrize("name", [p[0] for p in PACKS])
def test_persistent_grid_is_bitwise_equal(name, monkeypatch):
    import torch
    pack = dict(PACKS)[name]()
    log(f"case persistent vs default: {name}")
    d = dev_inputs(pack)
    monkeypatch.setenv("T2V_PERSISTENT", "0")
    ref = {k: v.clone() for k, v in run_hip(pack, d).items()}
    monkeypatch.setenv("T2V_PERSISTENT", "1")
    got = run_hip(pack, d)
    for k in ref:
        assert torch.equal(ref[k], got[k]), f"{k} differs on the persistent grid"


def test_persistent_grid_trace_has_one_record_per_item(monkeypatch):
    import torch
    from paper_2607_01701_amd import _lib
    pack = make_pack([4000, 300], 2, 128, seed=75)
    d = dev_inputs(pack)
    monkeypatch.setenv("T2V_PERSISTENT", "1")
    run_hip(pack, d)  # build and cache the work lists
    cap = 1 << 16
    rec = torch.zeros(4 * cap, dtype=torch.int64, device="cuda")
    _lib.t2v_trace_set(rec.data_ptr(), cap)
    run_hip(pack, d)
    n, over = _lib.t2v_trace_count()
    _lib.t2v_trace_set(None, 0)
    r = rec[: 4 * n].view(n, 4).cpu().numpy()
    log(f"persistent trace: {n} records, {over} overflowed")
    assert over == 0 and n > 0
    assert np.all(r[:, 2] >= r[:, 1]) and np.all(r[:, 1] > 0), "every item's record is written"
    assert set(np.unique(r[:, 3]).tolist()) <= {0, 2, 3}
