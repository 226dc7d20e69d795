"""Token-to-adapter bookkeeping -- TEST INFRASTRUCTURE ONLY (see package doc).

Serving unmerged adapters batches requests that use different adapters
(Sec. 1; Sec. 2 on S-LoRA's heterogeneous batching).  Every token carries an
adapter id; -1 means "no adapter".  This module states, in the plainest
form, the integer results the GPU path must reproduce exactly:

* ``validate``: an id that is out of range or names a slot that holds no
  adapter is treated as -1, and an error is reported;
* ``groups``: tokens grouped by adapter slot, slots ascending, tokens in each
  group ascending (a stable sort by slot);
* ``segments``: maximal runs of equal id in the given token order.

Pins (tests/test_oracle_plan.py): brute force on every id vector over a tiny
alphabet, and invariants (groups partition the valid tokens, counts add up).
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

import numpy as np


def validate(ids: Sequence[int], loaded: Sequence[bool]) -> Tuple[np.ndarray, bool]:
    """Return ``(vid, error)``: ``vid[t] = ids[t]`` when it names a loaded
    slot, -1 otherwise; ``error`` is true when some id other than -1 was
    replaced."""
    n = len(loaded)
    vid = np.full(len(ids), -1, dtype=np.int32)
    error = False
    for t, a in enumerate(ids):
        a = int(a)
        if a == -1:
            continue
        if 0 <= a < n and bool(loaded[a]):
            vid[t] = a
        else:
            error = True
    return vid, error


def group_rows(ids: Sequence[int]) -> List[Tuple[int, np.ndarray]]:
    """``[(slot, rows)]`` for every distinct id (ascending, including -1),
    rows ascending."""
    ids = np.asarray(ids, dtype=np.int64)
    out = []
    for s in sorted(set(int(v) for v in ids)):
        out.append((s, np.nonzero(ids == s)[0]))
    return out


def groups(vid: Sequence[int]):
    """Adapter groups over validated ids: returns ``(slot, start, count)``
    per group (slots ascending, -1 excluded) and ``perm``, the valid tokens
    listed group after group, ascending inside each group."""
    table = []
    perm = []
    for s, rows in group_rows(vid):
        if s < 0:
            continue
        table.append((s, len(perm), len(rows)))
        perm.extend(int(r) for r in rows)
    return table, np.asarray(perm, dtype=np.int32)


def segments(ids: Sequence[int]) -> List[Tuple[int, int, int]]:
    """Maximal runs of equal id in the given order: ``(start, length, id)``."""
    out = []
    t = 0
    ids = [int(v) for v in ids]
    while t < len(ids):
        u = t
        while u < len(ids) and ids[u] == ids[t]:
            u += 1
        out.append((t, u - t, ids[t]))
        t = u
    return out
