"""Cascade scheduling (paper Section IV-A, Eqs. (1)-(7); Alg. 1) on the CPU.

The brute-force oracle (oracle/cascade_milp.py) is pinned first against hand-solved
instances, closed forms and lower bounds; then the native list scheduler and genetic
algorithm (csrc/t2v_plan.cpp, through the host-only library) are checked against it:
every schedule they return satisfies the constraints, and on tiny random DAGs the GA reaches
the exact optimum.
"""
import types

import numpy as np
import pytest

import oracle.cascade_milp as milp
from paper_2607_01701_amd import _lib, planner


# ---------------------------------------------------------------- oracle pins

def check_chain_is_sum_of_fastest(mod):
    """A chain runs one cascade at a time: the optimum is the sum of each one's fastest degree."""
    preds = [[], [0], [1]]
    K = [1, 2, 4]
    lat = [[6, 3.5, 2.5], [4, 2.2, 1.9], [9, 5, 2.6]]
    mem = [[0, 0, 0]] * 3
    T, deg, _ = mod.solve_exact(preds, K, lat, mem, 1.0, 4)
    return abs(T - (2.5 + 1.9 + 2.6)) < 1e-12 and deg == [4, 4, 4]


def check_single_gpu_is_sum(mod):
    """Independent cascades on one GPU (K = {1}) run back to back: T = sum of latencies."""
    preds = [[], [], [], []]
    lat = [[3.0], [1.5], [2.0], [0.25]]
    T, _, _ = mod.solve_exact(preds, [1], lat, [[0]] * 4, 1.0, 1)
    return abs(T - 6.75) < 1e-12


def check_wide_cluster_is_max(mod):
    """With GPUs for everyone and no precedence, the optimum is the slowest cascade's fastest degree."""
    preds = [[], [], []]
    K = [1, 2]
    lat = [[4, 2.5], [7, 3], [1, 0.9]]
    T, _, _ = mod.solve_exact(preds, K, lat, [[0, 0]] * 3, 1.0, 6)
    return abs(T - 3.0) < 1e-12


def check_hand_solved(mod):
    """Three equal cascades, K = {1, 2}, N = 2, L = 4 at k = 1 and 2.5 at k = 2. All at k = 1
    takes 8 (two waves), all at k = 2 takes 7.5; two at k = 1 side by side then one at k = 2
    takes 4 + 2.5 = 6.5, which is optimal: any schedule's GPU-time is at least 13 when one
    cascade runs at k = 2 (6.5 on two GPUs), and with all at k = 1 three jobs of 4 need 8."""
    preds = [[], [], []]
    T, deg, _ = mod.solve_exact(preds, [1, 2], [[4, 2.5]] * 3, [[0, 0]] * 3, 1.0, 2)
    return abs(T - 6.5) < 1e-12 and sorted(deg) == [1, 1, 2]


def check_memory_forces_degree(mod):
    """Eq. (6): a cascade that does not fit one GPU at k = 1 must take k = 2. On N = 2 it then
    holds both GPUs for 3, and the other cascade (1 at k = 1) runs before or after it: T = 4."""
    preds = [[], []]
    lat = [[1.0, 3.0], [1.0, 3.0]]
    mem = [[10.0, 5.0], [1.0, 0.5]]
    T, deg, _ = mod.solve_exact(preds, [1, 2], lat, mem, 8.0, 2)
    return deg == [2, 1] and abs(T - 4.0) < 1e-12


def check_precedence_and_resources_bind(mod):
    """A diamond 0 -> {1, 2} -> 3 on N = 2 with K = {1, 2}: cascades 1 and 2 share the two GPUs
    at k = 1 (2 + 2) or run one after the other at k = 2 (1.5 + 1.5); optimum 1 + 2 + 1 = 4."""
    preds = [[], [0], [0], [1, 2]]
    lat = [[2, 1], [2, 1.5], [2, 1.5], [2, 1]]
    T, _, _ = mod.solve_exact(preds, [1, 2], lat, [[0, 0]] * 4, 1.0, 2)
    return abs(T - 4.0) < 1e-12


PINS = {
    "chain": check_chain_is_sum_of_fastest,
    "single_gpu": check_single_gpu_is_sum,
    "wide_cluster": check_wide_cluster_is_max,
    "hand_solved": check_hand_solved,
    "memory": check_memory_forces_degree,
    "diamond": check_precedence_and_resources_bind,
}


@pytest.mark.parametrize("name", sorted(PINS))
def test_oracle_pin(name):
    assert PINS[name](milp), name


def random_instance(rng, n, K, n_gpus, p_edge=0.35, mem_cap=None):
    preds = [[p for p in range(c) if rng.random() < p_edge] for c in range(n)]
    base = rng.uniform(1.0, 10.0, size=n)
    lat = [[float(base[c] / k ** rng.uniform(0.5, 0.95)) for k in K] for c in range(n)]
    mem = [[float(rng.uniform(0.0, 2.0) / k) for k in K] for c in range(n)]
    return preds, lat, mem, (1.0 if mem_cap is None else mem_cap)


def lower_bound(preds, K, lat, mem, cap, N):
    n = len(preds)
    feas = [[j for j, k in enumerate(K) if mem[c][j] <= cap and k <= N] for c in range(n)]
    fastest = [min(lat[c][j] for j in feas[c]) for c in range(n)]
    area = sum(min(K[j] * lat[c][j] for j in feas[c]) for c in range(n)) / N
    longest = [0.0] * n
    for c in range(n):  # predecessors have smaller indices
        longest[c] = fastest[c] + max((longest[p] for p in preds[c]), default=0.0)
    return max(area, max(longest))


def test_oracle_respects_lower_bounds_and_constraints():
    rng = np.random.default_rng(0)
    for _ in range(25):
        n = int(rng.integers(2, 6))
        K = [1, 2, 4]
        N = int(rng.choice([2, 4]))
        preds, lat, mem, cap = random_instance(rng, n, K, N)
        T, deg, st = milp.solve_exact(preds, K, lat, mem, cap, N)
        ok, T2, msg = milp.check_schedule(preds, K, lat, mem, cap, N, deg, st)
        assert ok, msg
        assert abs(T2 - T) < 1e-9
        assert T >= lower_bound(preds, K, lat, mem, cap, N) - 1e-9


MUTANTS = {
    "no_resource_check": ("        if ok:\n            return t\n", "        return t\n"),
    "no_precedence": ("        release = max((end[p] for p in preds[c]), default=0.0)", "        release = 0.0"),
    "no_memory_check": ("if mem[c][j] <= mem_cap and k <= n_gpus]", "if k <= n_gpus]"),
    "end_uses_start": ("        start[c], end[c] = t, t + lat[c]", "        start[c], end[c] = t, lat[c]"),
}


def _mutant(old, new):
    src = open(milp.__file__).read()
    assert src.count(old) >= 1, old
    mod = types.ModuleType("milp_mutant")
    exec(compile(src.replace(old, new), "milp_mutant", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_oracle_mutants_are_caught(name):
    mod = _mutant(*MUTANTS[name])
    failing = [p for p, fn in PINS.items() if not fn(mod)]
    assert failing, f"mutant {name} passed every pin"


# ---------------------------------------------------------------- checker pins
#
# The checker decides whether a schedule satisfies Eqs. (2)-(7); the planner's validity claims
# rest on it. Each negative case below breaks exactly one constraint of a schedule the checker
# must accept, so a checker that skips that constraint (or accepts everything) fails a pin.
# Instance: 0 -> 2 (precedence), three cascades, K = {1, 3}, N = 3, W = 1.
CHK = dict(preds=[[], [], [0]], degrees=[1, 3], latency=[[2.0, 1.5], [3.0, 2.0], [1.0, 0.75]],
           mem=[[0.5, 0.25], [2.0, 0.9], [0.5, 0.25]], mem_cap=1.0, n_gpus=3)
# Valid: 0 at k = 1 on [0, 2), 1 at k = 3 on [2, 4) (it does not fit one GPU: Mem = 2 > W),
# 2 at k = 1 on [4, 5): makespan 5. Touching intervals (an end equal to a start) are legal.
CHK_VALID = ([1, 3, 1], [0.0, 2.0, 4.0], 5.0)
CHK_BAD = {
    # Eq. (4): cascade 2 runs on [1, 2), before its predecessor 0 ends at 2 (two GPUs busy).
    "precedence": ([1, 3, 1], [0.0, 2.0, 1.0], "predecessor"),
    # Eq. (5): degree 2 is not in K = {1, 3}, although two GPUs are free for it.
    "degree_not_in_K": ([1, 3, 2], [0.0, 2.0, 4.0], "not in K"),
    # Eq. (6): cascade 1 at k = 1 needs Mem = 2 > W = 1; it runs alone on [2, 5).
    "memory": ([1, 1, 1], [0.0, 2.0, 5.0], "memory"),
    # Eq. (7): 0 (k = 1) on [0, 2) and 1 (k = 3) on [1, 3) overlap: four GPUs in use > N = 3.
    "capacity": ([1, 3, 1], [0.0, 1.0, 3.0], "GPUs in use"),
    # Eq. (7) with usage rising at a start inside an interval that began earlier: 1 (k = 3) on
    # [0, 2), then 0 (k = 1) from 1.5; 2 after 0.
    "capacity_late_start": ([1, 3, 1], [1.5, 0.0, 3.5], "GPUs in use"),
}


def test_checker_accepts_the_valid_schedule():
    deg, st, T = CHK_VALID
    ok, T2, msg = milp.check_schedule(CHK["preds"], CHK["degrees"], CHK["latency"], CHK["mem"], CHK["mem_cap"],
                                      CHK["n_gpus"], deg, st)
    assert ok, msg
    assert T2 == T


@pytest.mark.parametrize("name", sorted(CHK_BAD))
def test_checker_rejects_one_broken_constraint(name):
    deg, st, why = CHK_BAD[name]
    ok, _, msg = milp.check_schedule(CHK["preds"], CHK["degrees"], CHK["latency"], CHK["mem"], CHK["mem_cap"],
                                     CHK["n_gpus"], deg, st)
    assert not ok and why in msg, (name, msg)


def test_checker_pins_are_one_constraint_each():
    """Each negative case differs from a legal schedule by one constraint only: with that one
    constraint relaxed (N = 3 for capacity, W = 2 for memory, K widened, the edge dropped) the
    same schedule is accepted."""
    relax = {"precedence": dict(preds=[[], [], []]), "degree_not_in_K": dict(degrees=[1, 3, 2]),
             "memory": dict(mem_cap=2.0), "capacity": dict(n_gpus=4), "capacity_late_start": dict(n_gpus=4)}
    for name, (deg, st, _) in CHK_BAD.items():
        args = dict(CHK)
        args.update(relax[name])
        lat, mem = args["latency"], args["mem"]
        if len(args["degrees"]) == 3:  # K widened: latency / memory columns for k = 3
            lat = [row + [row[-1]] for row in lat]
            mem = [row + [row[-1]] for row in mem]
        ok, _, msg = milp.check_schedule(args["preds"], args["degrees"], lat, mem, args["mem_cap"], args["n_gpus"],
                                         deg, st)
        assert ok, (name, msg)


def _checker_pins_hold(mod):
    args = (CHK["preds"], CHK["degrees"], CHK["latency"], CHK["mem"], CHK["mem_cap"], CHK["n_gpus"])
    deg, st, T = CHK_VALID
    ok, T2, _ = mod.check_schedule(*args, deg, st)
    if not ok or T2 != T:
        return False
    return all(not mod.check_schedule(*args, d, s)[0] for d, s, _ in CHK_BAD.values())


CHECKER_MUTANTS = {
    "accept_everything": ("    n = len(preds)\n    if len(deg) != n", "    return True, 0.0, 'ok'\n    n = len(preds)\n    if len(deg) != n"),
    "no_precedence": ("            if starts[c] < end[p] - tol:", "            if False:"),
    # an unknown degree read as the largest one in K
    "no_degree_set": ("        if deg[c] not in degrees:\n            return False, None, f\"cascade {c}: degree {deg[c]} not in K\"  # Eq. (5)\n        j = degrees.index(deg[c])",
                      "        j = degrees.index(deg[c]) if deg[c] in degrees else len(degrees) - 1"),
    "no_memory": ("        if mem[c][j] > mem_cap:", "        if False:"),
    "no_capacity": ("        if used > n_gpus:", "        if False:"),
    "capacity_at_time_zero_only": ("    for t in sorted(set(starts)):", "    for t in [0.0]:"),
    "end_is_latency": ("    end = [starts[c] + lat[c] for c in range(n)]", "    end = [lat[c] for c in range(n)]"),
}


def test_checker_pins_hold_for_the_checker():
    assert _checker_pins_hold(milp)


@pytest.mark.parametrize("name", sorted(CHECKER_MUTANTS))
def test_checker_mutants_are_caught(name):
    mod = _mutant(*CHECKER_MUTANTS[name])
    assert not _checker_pins_hold(mod), f"checker mutant {name} passed every pin"


# ---------------------------------------------------------------- native planner

def test_library_exports_planner():
    for L in (_lib.host_lib(), _lib.lib()):
        assert hasattr(L, "t2v_list_schedule") and hasattr(L, "t2v_plan_cascades")


def test_list_schedule_is_valid_and_matches_a_serial_schedule():
    """The native list schedule satisfies Eqs. (2)-(7), and equals the oracle's serial scheme run
    on the same order (highest bottom level first among ready cascades)."""
    rng = np.random.default_rng(1)
    for _ in range(30):
        n = int(rng.integers(1, 9))
        K = [1, 2, 4]
        N = int(rng.choice([1, 2, 4, 8]))
        preds, lat, mem, cap = random_instance(rng, n, K, N)
        js = [int(rng.integers(0, 3)) for _ in range(n)]
        deg = [min(K[j], N) for j in js]
        lt = [lat[c][K.index(deg[c])] for c in range(n)]
        starts, T = planner.list_schedule(preds, deg, lt, N)
        ok, T2, msg = milp.check_schedule(preds, K, lat, [[0] * 3] * n, 1.0, N, deg, list(starts))
        assert ok, msg
        assert abs(T2 - T) < 1e-9
        # the same order through the oracle's serial scheme
        succs = [[c for c in range(n) if p in preds[c]] for p in range(n)]
        bottom = [0.0] * n
        for c in reversed(range(n)):
            bottom[c] = lt[c] + max((bottom[s] for s in succs[c]), default=0.0)
        done, order = set(), []
        while len(order) < n:
            ready = [c for c in range(n) if c not in done and all(p in done for p in preds[c])]
            c = max(ready, key=lambda x: (bottom[x], -x))
            order.append(c)
            done.add(c)
        st2, T3 = milp.serial_schedule(order, preds, deg, lt, N)
        assert np.allclose(st2, starts) and abs(T3 - T) < 1e-9


def test_ga_reaches_the_exact_optimum_on_tiny_dags():
    """Alg. 1 on tiny DAGs (2-6 cascades, K = {1, 2, 4}, N = 2 or 4) against brute force."""
    rng = np.random.default_rng(2)
    gaps = []
    for _ in range(40):
        n = int(rng.integers(2, 7))
        K = [1, 2, 4]
        N = int(rng.choice([2, 4]))
        preds, lat, mem, cap = random_instance(rng, n, K, N, mem_cap=1.2)
        T_opt, _, _ = milp.solve_exact(preds, K, lat, mem, cap, N)
        if not np.isfinite(T_opt):
            continue
        deg, st, T = planner.plan(preds, K, lat, mem, cap, N, population=32, generations=60, seed=7)
        ok, T2, msg = milp.check_schedule(preds, K, lat, mem, cap, N, list(deg), list(st))
        assert ok, msg
        assert abs(T2 - T) < 1e-9
        assert T >= T_opt - 1e-9
        gaps.append(T / T_opt - 1.0)
    gaps = np.asarray(gaps)
    assert gaps.size >= 30
    # The GA searches degrees only and the list scheduler fixes the order by critical-path
    # priority, so an instance whose optimum needs another order keeps a gap (measured: 36 of
    # 40 exact, worst 12%).
    assert np.mean(gaps < 1e-9) >= 0.85, gaps
    assert gaps.max() < 0.15, gaps


def test_ga_is_deterministic_and_beats_static_degrees():
    rng = np.random.default_rng(3)
    n, K, N = 24, [1, 2, 4, 8], 8
    preds, lat, mem, cap = random_instance(rng, n, K, N, p_edge=0.1, mem_cap=0.6)
    a = planner.plan(preds, K, lat, mem, cap, N, seed=11)
    b = planner.plan(preds, K, lat, mem, cap, N, seed=11)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1]) and a[2] == b[2]
    # every uniform feasible degree ("static parallelism") is no better than the GA
    for k in K:
        j = K.index(k)
        if all(mem[c][j] <= cap for c in range(n)) and k <= N:
            _, Tk = planner.list_schedule(preds, [k] * n, [lat[c][j] for c in range(n)], N)
            assert a[2] <= Tk + 1e-9


@pytest.mark.parametrize("kw,msg", [
    ({"preds": [[1], [0]]}, "cycle"),
    ({"preds": [[0], []]}, "bad predecessor"),
    ({"preds": [[5], []]}, "bad predecessor"),
    ({"mem_cap": 0.0}, "no feasible degree"),
    ({"population": 1}, "hyper-parameters"),
    ({"elite": 9}, "hyper-parameters"),
    ({"mutation": 1.5}, "hyper-parameters"),
    ({"n_gpus": 0}, "n_gpus"),
])
def test_plan_validation(kw, msg):
    args = dict(preds=[[], [0]], degrees=[1, 2], latency=[[2, 1], [3, 2]], mem=[[1, 0.5], [1, 0.5]], mem_cap=2.0,
                n_gpus=2, population=8, generations=2, mutation=0.1, elite=2, seed=0)
    args.update(kw)
    with pytest.raises(_lib.T2VError) as e:
        planner.plan(**args)
    assert msg in str(e.value)


def test_empty_problem():
    deg, st, T = planner.plan([], [1, 2], [], [], 1.0, 2)
    assert T == 0.0 and deg.size == 0
