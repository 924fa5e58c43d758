"""The static part of the decode's row schedule, restated on the CPU.

The decode kernel cuts the static units of all slabs (in slab order) into G
contiguous ranges [w*Ru/G, (w+1)*Ru/G), one per workgroup, and numbers the
visits of each slab: with Ru >= G by the workgroup's rank from the first
workgroup whose range meets the slab (ceil((Ps+1)*G/Ru) - 1), with Ru < G by
the unit's index in the slab (ranges then hold at most one unit; empty
ranges take no slot).  These closed forms must give every unit to exactly
one workgroup and each slab the slots 0..count-1, with count at most
min(G, units + 1) -- the bound the workspace is sized by.  Brute force over
random length mixes checks that.
"""
import random

import pytest


def ceil_div(a, b):
    return -(-a // b)


def visits_and_slots(units, G):
    """Brute force: (workgroup, slab, units covered, slot) for every visit."""
    P = [0]
    for u in units:
        P.append(P[-1] + u)
    Ru = P[-1]
    out = []
    for w in range(G):
        lo, hi = w * Ru // G, (w + 1) * Ru // G
        u = lo
        while u < hi:
            s = next(i for i in range(len(units)) if P[i] <= u < P[i] + units[i])
            e = min(hi, P[s] + units[s])
            slot = w - (ceil_div((P[s] + 1) * G, Ru) - 1) if Ru >= G else u - P[s]
            out.append((w, s, range(u, e), slot))
            u = e
    return P, Ru, out


def static_visits(Ps, st, Ru, G):
    if st <= 0:
        return 0
    if Ru < G:
        return st
    return (ceil_div((Ps + st) * G, Ru) - 1) - (ceil_div((Ps + 1) * G, Ru) - 1) + 1


@pytest.mark.parametrize("seed", range(6))
def test_static_ranges_cover_once_and_slots_are_dense(seed):
    rng = random.Random(seed)
    for _ in range(400):
        S = rng.randint(1, 40)
        G = rng.choice([1, 2, 3, 7, 64, 88, 256, 512])
        units = [rng.choice([0, 0, 1, 2, 3, rng.randint(0, 300)]) for _ in range(S)]
        if sum(units) == 0:
            continue
        P, Ru, visits = visits_and_slots(units, G)
        cover = [0] * Ru
        slots = {}
        for w, s, rows, slot in visits:
            for x in rows:
                cover[x] += 1
            slots.setdefault(s, []).append(slot)
        assert all(c == 1 for c in cover)
        for s, st in enumerate(units):
            count = static_visits(P[s], st, Ru, G)
            assert sorted(slots.get(s, [])) == list(range(count))
            assert count <= min(G, st + 1)


def test_one_slab_holding_everything_uses_every_workgroup():
    # the worst case the static slot count is sized for: one slab, G slots
    P, Ru, visits = visits_and_slots([10_000], 256)
    assert sorted(v[3] for v in visits) == list(range(256))


@pytest.mark.parametrize("seed", range(3))
def test_range_walks_slab_to_slab(seed):
    """Whole-slab ranges: a visit that is not the last of its workgroup's
    range ends at its slab's end, and the next visit starts at the first unit
    of the next slab that has units, so the kernel can step to it without a
    search (every slab of one sequence holds the same number of units)."""
    rng = random.Random(100 + seed)
    for _ in range(200):
        per_b = rng.choice([1, 2, 8, 32])
        B = rng.randint(1, 12)
        G = rng.choice([1, 3, 64, 256])
        seq_units = [rng.choice([0, 1, 2, 5, rng.randint(0, 40)]) for _ in range(B)]
        units = [u for u in seq_units for _ in range(per_b)]
        if sum(units) == 0:
            continue
        P, Ru, visits = visits_and_slots(units, G)
        for (w0, s0, r0, _), (w1, s1, r1, _) in zip(visits, visits[1:]):
            if w0 != w1:
                continue
            assert r0.stop == P[s0] + units[s0]
            assert s1 == next(i for i in range(s0 + 1, len(units)) if units[i] > 0)
            assert r1.start == P[s1]
            if (s0 + 1) % per_b != 0:
                assert s1 == s0 + 1 and units[s1] == units[s0]
