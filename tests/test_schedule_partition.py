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
