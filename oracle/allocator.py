"""Oracle for the layer allocator of section IV (test infrastructure).

Only tests/ (and nothing in the product path) import this module.  It
restates, in plain Python and in the paper's order and notation, the
two-stage heuristic of section IV-D (Algorithm 1: coarse allocation by
memory; Algorithm 2: workload fine-tuning) over the partition index pi
(device i holds layers pi[i] .. pi[i+1]-1), and computes the exact optimum
of the allocation problem of section IV-C for a fixed device order by
dynamic programming (with a brute-force enumeration for tiny cases).

Readings where the paper is silent or ambiguous:
  * initial partition: "each device has the same number of layers";
    with L not a multiple of D, pi[i] = floor(i L / D) (later devices get
    the extra layers);
  * workload: section IV-D charges dt[i] lf[j] + ct[i] per layer (ct per
    layer), the program of section IV-C charges ct[i] once per device; both
    are provided (per_layer_ct=True is section IV-D's);
  * Algorithm 2 evaluates "this device" and "next device" workloads on the
    partition as already changed earlier in the same sweep, against the
    target fixed at the start of the sweep;
  * "is memory satisfied after change": after moving one layer, the
    receiving device's block fits its memory (<=);
  * Algorithm 1 stops with an error when a sweep changes nothing; a search
    that keeps changing for L*D sweeps is reported the same way;
  * the optimum keeps the device order (contiguous blocks in device order,
    each device at least one layer), the order the heuristic keeps.
"""
from __future__ import annotations

import itertools


def equal_partition(L, D):
    return [(i * L) // D for i in range(D + 1)]


def num_layers(pi, i):
    return pi[i + 1] - pi[i]


def allocated_memory(lm, pi, i):
    return sum(lm[j] for j in range(pi[i], pi[i + 1]))


def device_workload(dt, ct, lf, pi, i, per_layer_ct=True):
    """Section IV-D: sum over the device's layers of dt[i]*lf[j] + ct[i];
    section IV-C (per_layer_ct=False): dt[i]*sum lf[j] + ct[i]."""
    if per_layer_ct:
        return sum(dt[i] * lf[j] + ct[i] for j in range(pi[i], pi[i + 1]))
    return dt[i] * sum(lf[j] for j in range(pi[i], pi[i + 1])) + ct[i]


def memory_satisfied(lm, dm, pi):
    return all(allocated_memory(lm, pi, i) <= dm[i] for i in range(len(dm)))


def coarse_allocation(lm, dm):
    """Algorithm 1.  Returns (pi, sweeps, ok)."""
    L, D = len(lm), len(dm)
    pi = equal_partition(L, D)
    am = [allocated_memory(lm, pi, i) for i in range(D)]
    sweeps = 0
    while True:
        if all(am[i] <= dm[i] for i in range(D)):
            return pi, sweeps, True
        if sweeps > L * D:
            return pi, sweeps, False
        before = list(pi)
        for i in range(D - 1):
            while am[i] > dm[i] and num_layers(pi, i) > 1:
                pi[i + 1] -= 1
                am = [allocated_memory(lm, pi, k) for k in range(D)]
            while dm[i] > am[i] + lm[pi[i + 1]] and num_layers(pi, i + 1) > 1:
                pi[i + 1] += 1
                am = [allocated_memory(lm, pi, k) for k in range(D)]
        sweeps += 1
        if pi == before:
            return pi, sweeps, False


def fine_allocation(dt, dm, ct, lf, lm, pi, max_iter):
    """Algorithm 2 from partition pi.  Returns (pi, rounds)."""
    D = len(dt)
    pi = list(pi)
    counter = 0
    while counter < max_iter:
        target = sum(device_workload(dt, ct, lf, pi, i) for i in range(D)) / D
        before = list(pi)
        for i in range(D - 1):
            this_w = device_workload(dt, ct, lf, pi, i)
            first_of_next = pi[i + 1]
            if (this_w < target and num_layers(pi, i + 1) > 1
                    and allocated_memory(lm, pi, i) + lm[first_of_next] <= dm[i]):
                pi[i + 1] += 1
            else:
                next_w = device_workload(dt, ct, lf, pi, i + 1)
                last_of_this = pi[i + 1] - 1
                last_w = dt[i] * lf[last_of_this] + ct[i]
                if (next_w < target and this_w - last_w > target and num_layers(pi, i) > 1
                        and allocated_memory(lm, pi, i + 1) + lm[last_of_this] <= dm[i + 1]):
                    pi[i + 1] -= 1
        counter += 1
        if pi == before:
            break
    return pi, counter


def optimal_partition(dt, dm, ct, lf, lm, per_layer_ct=True):
    """Exact min over contiguous device-ordered partitions (every device at
    least one layer, every block within its device's memory) of the largest
    device workload, by dynamic programming over (device, layers placed).
    Returns (best, pi) or (inf, None) when no partition fits."""
    L, D = len(lf), len(dt)
    INF = float("inf")
    # best[i][k]: min over placements of the first k layers on devices < i of the max workload
    best = [[INF] * (L + 1) for _ in range(D + 1)]
    arg = [[-1] * (L + 1) for _ in range(D + 1)]
    best[0][0] = 0.0
    for i in range(D):
        for k in range(L + 1):
            if best[i][k] == INF:
                continue
            for e in range(k + 1, L + 1):
                blk = [k, e]
                if allocated_memory(lm, blk, 0) > dm[i]:
                    break  # memory only grows with the block
                w = device_workload([dt[i]], [ct[i]], lf, blk, 0, per_layer_ct)
                cand = max(best[i][k], w)
                if cand < best[i + 1][e]:
                    best[i + 1][e] = cand
                    arg[i + 1][e] = k
    if best[D][L] == INF:
        return INF, None
    pi = [0] * (D + 1)
    pi[D] = L
    for i in range(D, 0, -1):
        pi[i - 1] = arg[i][pi[i]]
    return best[D][L], pi


def brute_force_partition(dt, dm, ct, lf, lm, per_layer_ct=True):
    """Same optimum by enumerating every composition (tiny cases only)."""
    L, D = len(lf), len(dt)
    best, best_pi = float("inf"), None
    for cuts in itertools.combinations(range(1, L), D - 1):
        pi = [0] + list(cuts) + [L]
        if not memory_satisfied(lm, dm, pi):
            continue
        w = max(device_workload(dt, ct, lf, pi, i, per_layer_ct) for i in range(D))
        if w < best:
            best, best_pi = w, pi
    return best, best_pi
