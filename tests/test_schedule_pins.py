"""Pins of the kernel-to-bubble packing oracle (§4.2, ScheduleKernels).

Earliest-fit in chain order is the componentwise-earliest feasible
assignment: for every feasible order-keeping assignment b, the packer's
interval a_i <= b_i for every kernel i (exchange argument: whatever b puts
into an interval at or after the packer's previous interval also fits there
for the packer).  So exhaustive enumeration pins it: the packer succeeds
exactly when some feasible assignment exists, and then each kernel sits in
the earliest interval any feasible assignment uses for it.
"""

import random

import pytest

from oracle import schedule as S


def _random_case(rng, n_max=5, m_max=5):
    n = rng.randint(1, n_max)
    m = rng.randint(1, m_max)
    kus = [rng.randint(0, 4) for _ in range(n)]
    comm = [rng.random() < 0.25 for _ in range(n)]
    ius = [rng.randint(0, 6) for _ in range(m)]
    bub = [rng.random() < 0.7 for _ in range(m)]
    return kus, comm, ius, bub


def _check_against_brute_force(pack, kus, comm, ius, bub):
    where, off = pack(kus, comm, ius, bub)
    all_ok = S.brute_force_assignments(kus, comm, ius, bub)
    if all_ok:
        assert -1 not in where
        assert S.feasible(where, kus, comm, ius, bub)
        assert where == [min(b[i] for b in all_ok) for i in range(len(kus))]
        for i in range(len(kus)):  # offsets: the earlier kernels of the same interval
            assert off[i] == sum(float(kus[j]) for j in range(i) if where[j] == where[i])
    else:
        assert -1 in where
        k = where.index(-1)
        assert all(w == -1 for w in where[k:])
        # the placed prefix is itself the earliest feasible placement of the prefix,
        # and the prefix one kernel longer has no feasible placement at all
        pre = S.brute_force_assignments(kus[:k], comm[:k], ius, bub) if k else [[]]
        assert pre and where[:k] == [min(b[i] for b in pre) for i in range(k)]
        assert not S.brute_force_assignments(kus[:k + 1], comm[:k + 1], ius, bub)


def test_matches_exhaustive_enumeration():
    rng = random.Random(1234)
    for _ in range(3000):
        _check_against_brute_force(S.schedule_kernels, *_random_case(rng))


def test_closed_cases():
    # everything fits into the first bubble, back to back
    assert S.schedule_kernels([1, 2, 3], [0, 0, 0], [6, 9], [1, 1]) == ([0, 0, 0], [0.0, 1.0, 3.0])
    # a kernel longer than every bubble blocks itself and every later kernel
    assert S.schedule_kernels([1, 9, 1], [0, 0, 0], [5, 5, 5], [1, 1, 1]) == ([0, -1, -1], [0.0, -1.0, -1.0])
    # the chain order is kept even when a later bubble would take a kernel earlier
    assert S.schedule_kernels([3, 1], [0, 0], [2, 3, 9], [1, 1, 1])[0] == [1, 2]
    # communication kernels go to LLM computation, never into bubbles
    assert S.schedule_kernels([1, 1, 1], [0, 1, 0], [5, 5, 5], [1, 0, 1]) == ([0, 1, 2], [0.0, 0.0, 0.0])
    assert S.schedule_kernels([1], [1], [5, 5], [1, 1])[0] == [-1]
    # an exact fit is a fit; zero-length kernels fit anywhere of their kind
    assert S.schedule_kernels([2, 3, 0], [0, 0, 0], [5, 0], [1, 1])[0] == [0, 0, 0]
    # no kernels / no intervals
    assert S.schedule_kernels([], [], [3], [1]) == ([], [])
    assert S.schedule_kernels([1], [0], [], []) == ([-1], [-1.0])


# ---- plausible mistakes planted in copies of the oracle must fail the pins

def _mutant(kind):
    def pack(kus, comm, ius, bub):
        n, m = len(kus), len(ius)
        where, off = [-1] * n, [-1.0] * n
        cur, used = 0, 0.0
        for i in range(n):
            d = float(kus[i])
            ok = False
            for j in range(0 if kind == "revisit" else cur, m):
                if kind != "ignore_kind" and bool(bub[j]) == bool(comm[i]):
                    continue
                start = used if (j == cur and kind != "reset_used") else 0.0
                fits = start + d < ius[j] if kind == "strict" else start + d <= ius[j]
                if fits:
                    where[i], off[i] = j, start
                    cur, used = j, start + d
                    ok = True
                    break
            if not ok:
                break
        return where, off
    return pack


@pytest.mark.parametrize("kind", ["revisit", "ignore_kind", "reset_used", "strict"])
def test_planted_mistakes_fail_the_pin(kind):
    rng = random.Random(99)
    caught = False
    for _ in range(3000):
        try:
            _check_against_brute_force(_mutant(kind), *_random_case(rng))
        except AssertionError:
            caught = True
            break
    assert caught, kind
