"""Exact (brute-force) cascade scheduling for tiny instances, and a constraint checker.

TEST INFRASTRUCTURE ONLY. Nothing on the product path may import, call or run this
module; only ``tests/`` and ``bench.py`` use it. It shares no code with the native
planner (csrc/t2v_plan.cpp) and imports nothing from the package.

The problem (paper Section IV-A, Eqs. (1)-(7)): cascades c with direct predecessors P_c;
choose for each cascade one parallel degree k from K (Eq. (5)), memory-feasible
(Mem_{c,k} <= W, Eq. (6)), and a launch time s_c, so that every cascade starts after its
predecessors end (Eq. (4)), the GPUs in use at any time t, summed over the active cascades
A_t = {c : s_c <= t < e_c}, never exceed N (Eq. (7)), with e_c = s_c + L_{c,k} (Eq. (2)),
minimising the makespan T = max_c e_c (Eqs. (1), (3)).

Exactness. For a fixed degree assignment this is a resource-constrained project scheduling
problem with one renewable resource (N GPUs) and a regular objective (makespan). Some
optimal schedule is then "active" (no cascade can start earlier without delaying another),
and the serial schedule-generation scheme — take the cascades in a precedence-feasible
order, start each at the earliest time at which its predecessors have ended and its k GPUs
are free for its whole duration — produces every active schedule when run over every
precedence-feasible order. Enumerating all degree assignments and all such orders therefore
reaches the MILP optimum. Exponential: only for a handful of cascades.
"""
from __future__ import annotations

import itertools


def _earliest_start(release: float, dur: float, need: int, placed, n_gpus: int) -> float:
    """Earliest t >= release with need + (GPUs used by `placed` over [t, t + dur)) <= n_gpus.

    placed: list of (start, end, k). Usage only changes at starts and ends, so the
    earliest feasible start is the release time or one of the placed end times.
    """
    if need > n_gpus:
        return float("inf")
    cands = sorted({release} | {e for _, e, _ in placed if e > release})
    for t in cands:
        points = [t] + [s for s, _, _ in placed if t < s < t + dur]
        ok = True
        for p in points:
            used = sum(k for s, e, k in placed if s <= p < e)
            if used + need > n_gpus:
                ok = False
                break
        if ok:
            return t
    return float("inf")  # unreachable: after the last end everything is free


def serial_schedule(order, preds, deg, lat, n_gpus):
    """Serial schedule-generation scheme for one precedence-feasible order.

    order: cascade indices; preds[c]: list of predecessors; deg[c], lat[c]: chosen degree and
    its latency. Returns (starts, makespan).
    """
    n = len(deg)
    start = [0.0] * n
    end = [0.0] * n
    placed = []
    for c in order:
        release = max((end[p] for p in preds[c]), default=0.0)
        t = _earliest_start(release, lat[c], deg[c], placed, n_gpus)
        start[c], end[c] = t, t + lat[c]
        placed.append((t, t + lat[c], deg[c]))
    return start, max(end, default=0.0)


def _topological_orders(preds):
    n = len(preds)
    succs = [[] for _ in range(n)]
    for c in range(n):
        for p in preds[c]:
            succs[p].append(c)

    def rec(done, indeg, prefix):
        if len(prefix) == n:
            yield list(prefix)
            return
        for c in range(n):
            if not done[c] and indeg[c] == 0:
                done[c] = True
                for s in succs[c]:
                    indeg[s] -= 1
                prefix.append(c)
                yield from rec(done, indeg, prefix)
                prefix.pop()
                for s in succs[c]:
                    indeg[s] += 1
                done[c] = False

    yield from rec([False] * n, [len(p) for p in preds], [])


def solve_exact(preds, degrees, latency, mem, mem_cap, n_gpus):
    """Optimal makespan, degrees and starts of the cascade scheduling problem.

    preds: list of predecessor lists; degrees: K (list of ints); latency[c][j], mem[c][j]:
    L_{c,K[j]}, Mem_{c,K[j]}. Returns (T, degree per cascade, starts), or (inf, None, None)
    when no assignment is feasible.
    """
    n = len(preds)
    choices = []
    for c in range(n):
        ok = [j for j, k in enumerate(degrees) if mem[c][j] <= mem_cap and k <= n_gpus]
        if not ok:
            return float("inf"), None, None
        choices.append(ok)
    orders = list(_topological_orders(preds))
    best = (float("inf"), None, None)
    for js in itertools.product(*choices):
        deg = [degrees[j] for j in js]
        lat = [latency[c][j] for c, j in enumerate(js)]
        for order in orders:
            starts, T = serial_schedule(order, preds, deg, lat, n_gpus)
            if T < best[0]:
                best = (T, deg, starts)
    return best


def check_schedule(preds, degrees, latency, mem, mem_cap, n_gpus, deg, starts, tol=1e-9):
    """Checks a schedule against Eqs. (2)-(7); returns (ok, makespan, message)."""
    n = len(preds)
    if len(deg) != n or len(starts) != n:
        return False, None, "wrong lengths"
    lat = []
    for c in range(n):
        if deg[c] not in degrees:
            return False, None, f"cascade {c}: degree {deg[c]} not in K"  # Eq. (5)
        j = degrees.index(deg[c])
        if mem[c][j] > mem_cap:
            return False, None, f"cascade {c}: memory {mem[c][j]} > W"  # Eq. (6)
        if starts[c] < -tol:
            return False, None, f"cascade {c}: negative start"
        lat.append(latency[c][j])
    end = [starts[c] + lat[c] for c in range(n)]  # Eq. (2)
    for c in range(n):
        for p in preds[c]:
            if starts[c] < end[p] - tol:
                return False, None, f"cascade {c} starts before predecessor {p} ends"  # Eq. (4)
    for t in sorted(set(starts)):  # usage only rises at starts
        used = sum(deg[c] for c in range(n) if starts[c] <= t + tol and t < end[c] - tol)
        if used > n_gpus:
            return False, None, f"{used} GPUs in use at t={t} > N"  # Eq. (7)
    return True, max(end, default=0.0), "ok"  # Eq. (3)
