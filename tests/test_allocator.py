"""Layer allocator of section IV (host code, no GPU).

The oracle (oracle/allocator.py) is pinned first: its exact optimum against
brute-force enumeration and closed forms, and its two heuristic stages
(Algorithm 1 and Algorithm 2) against traces worked out by hand from the
algorithms' text.  The C ABI (alloc_coarse, alloc_fine, alloc_workloads)
must then give the oracle's partition indices and sweep/round counts
exactly, and its workloads bit for bit (same summation order)."""
import math
import random

import pytest

from oracle import allocator as A


def random_instance(rng, L, D, tight=False):
    dt = [float(rng.randint(1, 7)) for _ in range(D)]  # slow-down factors 1..7
    ct = [rng.choice([0.0, 0.01, 0.5]) * rng.random() for _ in range(D)]
    lf = [rng.choice([0.05, 1.0, 3.0, 4.0]) * (0.5 + rng.random()) for _ in range(L)]
    lm = [0.5 + rng.random() for _ in range(L)]
    total = sum(lm)
    if tight:
        dm = [total / D * (0.6 + 1.2 * rng.random()) for _ in range(D)]
    else:
        dm = [total for _ in range(D)]
    return dt, dm, ct, lf, lm


# ---------------------------------------------------------------- oracle pins
def test_optimum_matches_brute_force():
    rng = random.Random(1)
    for trial in range(300):
        L = rng.randint(1, 8)
        D = rng.randint(1, min(4, L))
        dt, dm, ct, lf, lm = random_instance(rng, L, D, tight=trial % 2 == 1)
        for per_layer in (True, False):
            a, pa = A.optimal_partition(dt, dm, ct, lf, lm, per_layer)
            b, pb = A.brute_force_partition(dt, dm, ct, lf, lm, per_layer)
            assert a == b, (trial, a, b)
            if a < math.inf:
                w = max(A.device_workload(dt, ct, lf, pa, i, per_layer) for i in range(D))
                assert w == a and A.memory_satisfied(lm, dm, pa)


def test_optimum_closed_forms():
    # one device holds everything
    best, pi = A.optimal_partition([2.0], [100.0], [0.5], [1.0, 2.0, 3.0], [1.0] * 3, False)
    assert pi == [0, 3] and best == 2.0 * 6.0 + 0.5
    # identical devices and layers, L a multiple of D: the equal split, L/D layers each
    best, pi = A.optimal_partition([1.5] * 4, [1e9] * 4, [0.0] * 4, [2.0] * 12, [1.0] * 12)
    assert best == 3 * 3.0 and pi == [0, 3, 6, 9, 12]
    # a device twice as slow gets half the layers: 10 unit layers on dt = 2, 1, 1 split
    # 2 / 4 / 4, every workload 4
    best, _ = A.optimal_partition([2.0, 1.0, 1.0], [1e9] * 3, [0.0] * 3, [1.0] * 10, [1.0] * 10)
    assert best == 4.0
    # infeasible memory
    best, pi = A.optimal_partition([1.0, 1.0], [1.0, 1.0], [0.0, 0.0], [1.0] * 3, [1.0] * 3)
    assert best == math.inf and pi is None


def test_coarse_allocation_hand_trace():
    # 6 layers of 2 units on devices with 3, 20, 20: the equal split
    # [0,2,4,6] overloads device 0 (4 > 3); the sweep gives its last layer
    # to device 1 (pi[1] = 1), device 0 cannot take it back (3 > 2 + 2 is
    # false), device 1 then takes device 2's first layer while it fits and
    # device 2 keeps one (pi[2] = 5); the next check finds every device fits.
    pi, sweeps, ok = A.coarse_allocation([2.0] * 6, [3.0, 20.0, 20.0])
    assert ok and pi == [0, 1, 5, 6] and sweeps == 1
    # already fitting: no sweep
    pi, sweeps, ok = A.coarse_allocation([1.0] * 10, [4.0, 4.0, 4.0])
    assert ok and pi == [0, 3, 6, 10] and sweeps == 0
    # every layer is larger than every device: the first sweep changes nothing
    pi, sweeps, ok = A.coarse_allocation([5.0] * 3, [4.0] * 3)
    assert not ok and pi == [0, 1, 2, 3] and sweeps == 1


def test_fine_allocation_hand_trace():
    # speeds dt = 1, 2, 1 on 10 unit layers from [0,3,6,10] (workloads 3,6,4,
    # target 13/3).  Round 1: device 0 (3) takes layer 3 -> 4; device 1 (now
    # 4, below target) takes layer 6 -> [0,4,7,10] = 4,6,3.  Round 2 (target
    # 13/3 again): device 0 (4) takes -> 5; device 1 (4) takes -> [0,5,8,10] =
    # 5,6,2.  Round 3: device 0 is above target and device 1 is not below;
    # device 1 is above but 6 - 2 = 4 is not above 13/3: nothing changes.
    pi, rounds = A.fine_allocation([1.0, 2.0, 1.0], [10.0] * 3, [0.0] * 3, [1.0] * 10,
                                   [1.0] * 10, [0, 3, 6, 10], 50)
    assert pi == [0, 5, 8, 10] and rounds == 3
    # max_iter bounds the rounds
    pi, rounds = A.fine_allocation([1.0, 2.0, 1.0], [10.0] * 3, [0.0] * 3, [1.0] * 10,
                                   [1.0] * 10, [0, 3, 6, 10], 1)
    assert pi == [0, 4, 7, 10] and rounds == 1
    # memory blocks the first move: device 0 may hold only 3 layers
    pi, rounds = A.fine_allocation([1.0, 2.0, 1.0], [3.0, 10.0, 10.0], [0.0] * 3, [1.0] * 10,
                                   [1.0] * 10, [0, 3, 6, 10], 50)
    assert pi[1] == 3


def test_fine_allocation_homogeneous_fixed_point():
    # equal devices, equal layers, L a multiple of D: every device is at the
    # target, nothing moves, and the result is the optimum
    dt, ct, lf, lm = [2.0] * 4, [0.1] * 4, [1.0] * 16, [1.0] * 16
    pi, rounds = A.fine_allocation(dt, [1e9] * 4, ct, lf, lm, A.equal_partition(16, 4), 20)
    assert pi == [0, 4, 8, 12, 16] and rounds == 1
    best, _ = A.optimal_partition(dt, [1e9] * 4, ct, lf, lm)
    assert max(A.device_workload(dt, ct, lf, pi, i) for i in range(4)) == best


def test_heuristic_is_valid_and_bounded_by_the_optimum():
    rng = random.Random(2)
    for trial in range(200):
        L = rng.randint(2, 40)
        D = rng.randint(1, min(8, L))
        dt, dm, ct, lf, lm = random_instance(rng, L, D, tight=trial % 3 == 0)
        pi, _, ok = A.coarse_allocation(lm, dm)
        if not ok:
            continue
        assert A.memory_satisfied(lm, dm, pi)
        pi, _ = A.fine_allocation(dt, dm, ct, lf, lm, pi, 100)
        assert pi[0] == 0 and pi[-1] == L and all(b > a for a, b in zip(pi, pi[1:]))
        assert A.memory_satisfied(lm, dm, pi)
        h = max(A.device_workload(dt, ct, lf, pi, i) for i in range(D))
        best, _ = A.optimal_partition(dt, dm, ct, lf, lm)
        assert best <= h * (1 + 1e-12)


# ------------------------------------------------------------ C ABI parity
def _lib():
    try:
        import paper_2202_11836_amd as P
        P.load_library()
        return P
    except RuntimeError as e:  # library not built
        pytest.skip(str(e))


def test_c_abi_matches_oracle():
    P = _lib()
    rng = random.Random(3)
    for trial in range(400):
        L = rng.randint(1, 60)
        D = rng.randint(1, min(8, L))
        dt, dm, ct, lf, lm = random_instance(rng, L, D, tight=trial % 2 == 0)
        opi, osweeps, ok = A.coarse_allocation(lm, dm)
        if ok:
            pi, sweeps = P.alloc_coarse(lm, dm)
            assert (pi, sweeps) == (opi, osweeps), trial
        else:
            with pytest.raises(P.AllocError) as e:
                P.alloc_coarse(lm, dm)
            assert e.value.status == P.ALLOC_ENOFIT and e.value.pi == opi
            opi = A.equal_partition(L, D)
            dm = [1e9] * D
        max_iter = rng.choice([0, 1, 3, 100])
        fpi, frounds = A.fine_allocation(dt, dm, ct, lf, lm, opi, max_iter)
        pi, rounds = P.alloc_fine(dt, dm, ct, lf, lm, opi, max_iter)
        assert (pi, rounds) == (fpi, frounds), trial
        for mode, per_layer in ((P.ALLOC_CT_PER_LAYER, True), (P.ALLOC_CT_PER_DEVICE, False)):
            w = P.alloc_workloads(dt, ct, lf, fpi, mode)
            assert w == [A.device_workload(dt, ct, lf, fpi, i, per_layer) for i in range(D)]


def test_c_abi_rejects_bad_input():
    P = _lib()
    bad = [
        lambda: P.alloc_coarse([1.0], [1.0, 1.0]),               # L < D
        lambda: P.alloc_coarse([], []),                          # D < 1
        lambda: P.alloc_coarse([1.0, -1.0], [5.0]),              # negative
        lambda: P.alloc_coarse([1.0, float("nan")], [5.0]),      # non-finite
        lambda: P.alloc_fine([1.0, 1.0], [9.0, 9.0], [0.0, 0.0], [1.0] * 4, [1.0] * 4,
                             [0, 0, 4], 5),                      # empty block
        lambda: P.alloc_fine([1.0, 1.0], [9.0, 9.0], [0.0, 0.0], [1.0] * 4, [1.0] * 4,
                             [0, 1, 3], 5),                      # pi[D] != L
        lambda: P.alloc_fine([1.0, 1.0], [9.0, 9.0], [0.0, 0.0], [1.0] * 4, [1.0] * 4,
                             [0, 2, 4], -1),                     # max_iter < 0
        lambda: P.alloc_workloads([1.0], [0.0], [1.0, 1.0], [0, 2], 7),  # mode
    ]
    for f in bad:
        with pytest.raises(P.AllocError) as e:
            f()
        assert e.value.status == P.ALLOC_EINVAL
