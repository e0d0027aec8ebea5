"""Host tile scheduler (CPU, host-only library): coverage, order, balance, makespan bound."""
import numpy as np
import pytest

from paper_2607_01701_amd._lib import (ORDER_LONGEST_FIRST, ORDER_NATURAL, T2VError, t2v_build_worklist,
                                       t2v_plan_makespan)
from paper_2607_01701_amd.workload import WORKLOADS, cu_from_lengths, make_workload

NXCD = 8


def expected_items(cu, H, block):
    out = set()
    for s in range(len(cu) - 1):
        L = cu[s + 1] - cu[s]
        for h in range(H):
            for t in range(0, L, block):
                out.add((int(cu[s]), int(L), t, h))
    return out


CASES = [
    ([256, 384], 2, 128),
    ([0, 5, 0, 129, 1, 0], 3, 128),
    ([4096] * 8, 24, 256),
    ([1280, 6912, 20280, 1280, 6912], 24, 128),
    ([100800] + [1024] * 64, 40, 128),
    ([], 4, 128),
    ([0, 0], 2, 64),
]


@pytest.mark.parametrize("order", [ORDER_NATURAL, ORDER_LONGEST_FIRST])
@pytest.mark.parametrize("lens,H,block", CASES)
def test_every_tile_exactly_once(lens, H, block, order):
    cu = cu_from_lengths(lens)
    items = t2v_build_worklist(cu, H, block, order)
    got = [tuple(int(x) for x in r) for r in items]
    assert len(got) == len(set(got))
    assert set(got) == expected_items(cu, H, block)


def test_natural_order_is_pack_order():
    cu = cu_from_lengths([5, 300, 0, 70])
    items = t2v_build_worklist(cu, 2, 128, ORDER_NATURAL)
    keys = [(r[0], r[3], r[2]) for r in items]  # (clip start, head, tile)
    assert keys == sorted(keys)


@pytest.mark.parametrize("lens,H,block", CASES)
def test_longest_first_per_xcd(lens, H, block):
    """Within each XCD's share (workgroups b = x mod 8) clips run longest first and one
    (clip, head)'s tiles are contiguous."""
    cu = cu_from_lengths(lens)
    items = t2v_build_worklist(cu, H, block, ORDER_LONGEST_FIRST)
    for x in range(NXCD):
        q = items[x::NXCD]
        assert np.all(np.diff(q[:, 1]) <= 0), "clip lengths must not increase"
        seen_done = set()
        prev = None
        for r in q:
            g = (int(r[0]), int(r[3]))
            if g != prev:
                assert g not in seen_done, "a (clip, head) group was interrupted"
                if prev is not None:
                    seen_done.add(prev)
                prev = g


def _xcd_costs(items, block):
    rows = np.minimum(block, items[:, 1] - items[:, 2]).astype(np.float64)
    cost = rows * items[:, 1]
    return np.array([cost[x::NXCD].sum() for x in range(NXCD)]), cost


@pytest.mark.parametrize("name", ["hetero", "skew", "uniform", "long"])
def test_xcd_cost_balance(name):
    p = make_workload(name, tensors=False)
    block = 256
    items = t2v_build_worklist(p.cu_seqlens, p.heads, block, ORDER_LONGEST_FIRST)
    per, cost = _xcd_costs(items, block)
    # Whole groups are dealt, so an XCD can exceed the mean by at most about one group.
    groups = {}
    for r, c in zip(items, cost):
        groups[(r[0], r[3])] = groups.get((r[0], r[3]), 0.0) + c
    assert per.max() - per.mean() <= max(groups.values()) + cost.max()
    assert per.max() <= 1.10 * per.mean()


@pytest.mark.parametrize("name,heads", [("skew", 5), ("hetero", 3), ("long", 3), ("uniform", 3)])
def test_xcd_cost_balance_with_few_heavy_groups(name, heads):
    """One GPU's share under head sharding (a workload at H / 8 heads): few (clip, head)
    groups, each heavier than an even XCD share. Equal item counts per XCD must not pin whole
    heavy groups to some XCDs (before groups were split by cost: max / mean 1.59 for the
    skewed pack at 5 heads, 1.40 for the heterogeneous mix at 3)."""
    p = make_workload(name, tensors=False)
    for block in (256, 128):
        items = t2v_build_worklist(p.cu_seqlens, heads, block, ORDER_LONGEST_FIRST)
        per, _ = _xcd_costs(items, block)
        assert per.max() <= 1.02 * per.mean(), (block, per / per.mean())
        mk, lb = t2v_plan_makespan(items, block, 256)
        if block == 128:
            assert mk <= 1.06 * lb, (mk, lb)


@pytest.mark.parametrize("name", WORKLOADS)
def test_workload_item_counts(name):
    """Item counts of the workloads at 128-row tiles of the query offsets (hetero and cross at seed 0;
    cross tiles its 16 video clips over 12 heads)."""
    expect = {"tiny": 10, "uniform": 6144, "hetero": 21960, "long": 14184, "skew": 52000, "cross": 10980}
    p = make_workload(name, tensors=False)
    items = t2v_build_worklist(p.cu_seqlens, p.heads, 128, ORDER_LONGEST_FIRST)
    assert items.shape[0] == expect[name]


def test_hetero_seed0_lengths():
    p = make_workload("hetero", tensors=False)
    assert p.lengths.tolist() == [6912, 20280, 6912, 6912, 1280, 1280, 1280, 1280, 1280, 20280, 1280, 6912, 6912,
                                  20280, 6912, 6912]
    assert p.total_tokens == 116904 and p.sum_sq_len == 1578095808


def test_makespan_bounds_and_longest_first_helps():
    p = make_workload("skew", tensors=False)
    block, slots = 256, 256
    nat = t2v_build_worklist(p.cu_seqlens, p.heads, block, ORDER_NATURAL)
    lpt = t2v_build_worklist(p.cu_seqlens, p.heads, block, ORDER_LONGEST_FIRST)
    ms_n, lb_n = t2v_plan_makespan(nat, block, slots)
    ms_l, lb_l = t2v_plan_makespan(lpt, block, slots)
    assert lb_n == lb_l
    assert ms_l >= lb_l and ms_n >= lb_n
    # Greedy list scheduling in any order is within total/m + max item (Graham).
    total = float(np.sum(np.minimum(block, lpt[:, 1] - lpt[:, 2]).astype(np.float64) * lpt[:, 1]))
    largest = float(np.max(np.minimum(block, lpt[:, 1] - lpt[:, 2]).astype(np.float64) * lpt[:, 1]))
    assert ms_l <= total / slots + largest * 1.0001 + 1e-6 * total
    assert ms_l <= ms_n * 1.0001


def test_makespan_simple_case():
    # 4 equal items on 2 workers (not a multiple of 8 workers: one list): makespan = 2 items.
    cu = cu_from_lengths([256])
    items = t2v_build_worklist(cu, 2, 128, ORDER_NATURAL)  # 2 tiles x 2 heads
    ms, lb = t2v_plan_makespan(items, 128, 2)
    assert ms == 2 * 128 * 256 and lb == 2 * 128 * 256


def test_worklist_errors():
    with pytest.raises(T2VError):
        t2v_build_worklist(np.array([1, 5], dtype=np.int32), 2, 128)
    with pytest.raises(T2VError):
        t2v_build_worklist(np.array([0, 5, 3], dtype=np.int32), 2, 128)
    with pytest.raises(T2VError):
        t2v_build_worklist(np.array([0, 5], dtype=np.int32), 0, 128)
    with pytest.raises(T2VError):
        t2v_build_worklist(np.array([0, 5], dtype=np.int32), 2, 128, order=7)
