"""The device work-list cache under pressure: more distinct packs than it holds (the least
recently used lists are released while results stay bitwise the same), and several host
threads calling on their own streams at once (each result bitwise equal to the same call
made alone)."""
import threading

import numpy as np
import pytest

from paper_2607_01701_amd.workload import make_pack

from gpu_util import dev_inputs, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def run_on(pack, dev, stream):
    import torch
    from paper_2607_01701_amd import attn_bwd, attn_fwd
    with torch.cuda.stream(stream):
        out, lse = attn_fwd(dev["q"], dev["k"], dev["v"], pack.cu_seqlens, pack.scale)
        dq, dk, dv = attn_bwd(dev["q"], dev["k"], dev["v"], out, lse, dev["dout"], pack.cu_seqlens, pack.scale)
    stream.synchronize()
    return {"out": out, "lse": lse, "dq": dq, "dk": dk, "dv": dv}


def same(a, b):
    import torch
    return all(torch.equal(a[k], b[k]) for k in a)


def test_eviction_keeps_results():
    import torch
    s = torch.cuda.current_stream()
    first = make_pack([100, 37], 2, 64, seed=60)
    d0 = dev_inputs(first)
    ref = {k: v.clone() for k, v in run_on(first, d0, s).items()}
    log("case 70 distinct packs through the cache (it holds 64)")
    for i in range(70):
        p = make_pack([40 + i, 3 + (i % 5)], 2, 64, seed=61 + i)
        run_on(p, dev_inputs(p), s)
    again = run_on(first, d0, s)
    assert same(ref, again)


def test_threads_on_their_own_streams():
    import torch
    packs = [make_pack([300 + 50 * i, 129, 7 * (i + 1)], 2, 128, seed=80 + i) for i in range(4)]
    devs = [dev_inputs(p) for p in packs]
    alone = []
    for p, d in zip(packs, devs):
        alone.append({k: v.clone() for k, v in run_on(p, d, torch.cuda.current_stream()).items()})
    log("case 4 threads x 5 calls on separate streams")
    results, errors = [None] * 4, []

    def worker(i):
        try:
            st = torch.cuda.Stream()
            for _ in range(5):
                r = run_on(packs[i], devs[i], st)
            results[i] = {k: v.clone() for k, v in r.items()}
        except Exception as e:  # reported below
            errors.append(repr(e))

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(4)]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads), "a worker thread did not finish"
    assert not errors, errors
    torch.cuda.synchronize()
    for i in range(4):
        assert same(alone[i], results[i]), f"thread {i} differs from the single-threaded result"


def test_log_prints_the_plan_summary(monkeypatch, capfd):
    import torch
    from paper_2607_01701_amd import attn_fwd
    monkeypatch.setenv("T2V_LOG", "1")
    monkeypatch.setenv("T2V_QTILE", "wide")  # 256-row forward tiles
    pack = make_pack([777, 41], 2, 64, seed=90)  # lengths no other test uses: a new work list
    d = dev_inputs(pack)
    attn_fwd(d["q"], d["k"], d["v"], pack.cu_seqlens, pack.scale)
    torch.cuda.synchronize()
    err = capfd.readouterr().err
    assert "t2v: work list: 2 sequences, 2 heads, 256-row tiles, longest-first order: 10 items" in err, err
    assert "predicted makespan" in err and "lower bound" in err


def test_forced_allocation_failure_is_reported_and_recovers(monkeypatch):
    import torch
    from paper_2607_01701_amd import _lib, attn_fwd
    pack = make_pack([611, 29], 2, 128, seed=91)  # a new work list
    d = dev_inputs(pack)
    out = torch.full_like(d["q"], 7.0)
    monkeypatch.setenv("T2V_TEST_FAIL_ALLOC", "1")
    with pytest.raises(_lib.T2VError) as ei:
        attn_fwd(d["q"], d["k"], d["v"], pack.cu_seqlens, pack.scale, out=out)
    assert ei.value.status == _lib.T2V_ERR_OOM and "forced" in str(ei.value)
    torch.cuda.synchronize()
    assert bool((out == 7.0).all()), "a failed call wrote its output"
    monkeypatch.delenv("T2V_TEST_FAIL_ALLOC")
    o1, _ = attn_fwd(d["q"], d["k"], d["v"], pack.cu_seqlens, pack.scale)
    o2, _ = attn_fwd(d["q"], d["k"], d["v"], pack.cu_seqlens, pack.scale)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2)
