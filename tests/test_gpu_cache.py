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


def test_fresh_packs_on_concurrent_streams_reuse_list_memory():
    """Work-list memory is recycled while kernels on other streams still run: four threads,
    each on its own stream, call fwd + bwd on 30 packs no other call uses (360 work lists
    through a cache of 64, so lists are released and their memory handed to new ones while
    launches are in flight). Every result must equal the same call made alone. All buffers
    are sized for the largest pack, so even a list overwritten too early would stay inside
    them (and show up as a wrong result, not a fault)."""
    import ctypes
    import torch
    from paper_2607_01701_amd import _lib
    rng = np.random.default_rng(123)
    n_threads, per = 4, 30
    H, D = 2, 128
    packs = [[int(x) for x in rng.integers(1, 700, size=int(rng.integers(1, 5)))] for _ in range(n_threads * per)]
    tmax = max(sum(p) for p in packs)
    gen = torch.Generator(device="cuda").manual_seed(5)
    q, k, v, g = (torch.randn((tmax, H, D), generator=gen, device="cuda").to(torch.bfloat16) for _ in range(4))
    L = _lib.lib()
    sc = 1.0 / D ** 0.5

    def call(lengths, bufs, stream):
        cu = np.ascontiguousarray(np.concatenate([[0], np.cumsum(lengths)]), dtype=np.int32)
        cp = cu.ctypes.data_as(_lib._i32p)
        n = len(lengths)
        s = stream.cuda_stream
        st = L.t2v_attn_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), cp, n, H, D, sc, bufs["out"].data_ptr(),
                            bufs["lse"].data_ptr(), s)
        assert st == 0, _lib.t2v_last_error(L)
        st = L.t2v_attn_bwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), bufs["out"].data_ptr(), bufs["lse"].data_ptr(),
                            cp, n, H, D, sc, g.data_ptr(), bufs["dq"].data_ptr(), bufs["dk"].data_ptr(),
                            bufs["dv"].data_ptr(), bufs["ws"].data_ptr(), s)
        assert st == 0, _lib.t2v_last_error(L)
        T = int(cu[-1])
        # lse is [H, T] for this call's T: its first H * T floats (not a [:, :T] slice).
        return {"out": bufs["out"][:T].clone(), "dq": bufs["dq"][:T].clone(), "dk": bufs["dk"][:T].clone(),
                "dv": bufs["dv"][:T].clone(), "lse": bufs["lse"].view(-1)[:H * T].view(H, T).clone()}

    def buffers():
        b = {n: torch.zeros((tmax, H, D), dtype=torch.bfloat16, device="cuda") for n in ("out", "dq", "dk", "dv")}
        b["lse"] = torch.zeros((H, tmax), dtype=torch.float32, device="cuda")
        b["ws"] = torch.zeros((2, H, tmax), dtype=torch.float32, device="cuda")
        return b

    log(f"case {n_threads} threads x {per} fresh packs (alone first)")
    main = torch.cuda.current_stream()
    b0 = buffers()
    alone = []
    for p in packs:
        alone.append(call(p, b0, main))
    torch.cuda.synchronize()
    _lib.t2v_release_cache()  # the threaded calls all miss the cache
    results, errors = [None] * len(packs), []

    def worker(t):
        try:
            st = torch.cuda.Stream()
            with torch.cuda.stream(st):  # buffers filled on the same stream as the calls that write them
                bufs = buffers()
                for j in range(per):
                    i = t * per + j
                    results[i] = call(packs[i], bufs, st)
            st.synchronize()
        except Exception as e:  # reported below
            errors.append(repr(e))

    threads = [threading.Thread(target=worker, args=(t,)) for t in range(n_threads)]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=300)
    assert not any(t.is_alive() for t in threads), "a worker thread did not finish"
    assert not errors, errors
    torch.cuda.synchronize()
    bad = [i for i in range(len(packs)) if not same(alone[i], results[i])]
    assert not bad, f"{len(bad)} packs differ from their single-stream result, first {packs[bad[0]]}"
