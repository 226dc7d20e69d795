"""Pins for the oracle's integer bookkeeping (CPU only): exhaustive brute
force over every id vector of a tiny alphabet."""
import itertools

import numpy as np

from oracle import plan


def _brute_groups(vid):
    # stable sort of (slot, index) pairs, by a different route than the oracle
    pairs = sorted((int(a), t) for t, a in enumerate(vid) if a >= 0)
    table = []
    for s in sorted({a for a, _ in pairs}):
        rows = [t for a, t in pairs if a == s]
        start = [i for i, (a, _) in enumerate(pairs) if a == s][0]
        table.append((s, start, len(rows)))
    return table, [t for _, t in pairs]


def test_groups_exhaustive():
    for L in range(0, 6):
        for ids in itertools.product([-1, 0, 1, 2], repeat=L):
            table, perm = plan.groups(ids)
            bt, bp = _brute_groups(ids)
            assert table == bt
            assert list(perm) == bp
            assert sum(c for _, _, c in table) == sum(1 for a in ids if a >= 0)


def test_validate():
    loaded = [True, False, True]
    vid, err = plan.validate([0, 1, 2, 3, -1, -5, 2], loaded)
    assert list(vid) == [0, -1, 2, -1, -1, -1, 2]
    assert err
    vid, err = plan.validate([0, -1, 2], loaded)
    assert list(vid) == [0, -1, 2] and not err
    vid, err = plan.validate([], loaded)
    assert len(vid) == 0 and not err


def test_segments_exhaustive():
    for L in range(0, 7):
        for ids in itertools.product([-1, 0, 1], repeat=L):
            segs = plan.segments(ids)
            rebuilt = [a for s, n, a in segs for _ in range(n)]
            assert rebuilt == list(ids)
            for (s0, n0, a0), (s1, n1, a1) in zip(segs, segs[1:]):
                assert s0 + n0 == s1 and a0 != a1
            assert all(n > 0 for _, n, _ in segs)


def test_group_rows_includes_none():
    g = plan.group_rows(np.array([2, -1, 2, 0]))
    assert [s for s, _ in g] == [-1, 0, 2]
    assert list(g[2][1]) == [0, 2]
