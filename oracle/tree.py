"""Rows of one iteration as a forest: parent, position and visibility (oracle).

Sec. 3.2 ("Rejection Recycling"): candidate n-grams are verified in parallel
next to the draft; App. A Alg. 1 (input assembly): the real-active draft is
followed by every pseudo-active block (its accepted tokens, then its draft),
each conditioned on everything before it.  One forward pass covers them all
when the rows form a forest:

* a segment is a run of rows ``first .. first+n_rows-1`` forming a chain;
  its first row hangs under ``attach`` (-1: a root, predicted by the last
  committed row), every later row under the row before it;
* the prediction a row is checked against is the argmax of its parent;
* ``pos[r] = C + depth(r)``: a row sits one position after its parent;
* row r sees the committed prefix, its ancestors and itself.

A linear Jacobi draft of n rows is one segment with ``attach = -1``, which
gives the causal triangle of Eq. 3.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

ROLE_RA, ROLE_CAND, ROLE_PSEUDO = 0, 1, 2


@dataclass(frozen=True)
class Segment:
    first: int          # first row
    n_rows: int         # rows in the chain (>= 1)
    attach: int         # parent row of the first row; -1 = root
    role: int           # ROLE_RA, ROLE_CAND or ROLE_PSEUDO
    verify_from: int    # rows [first, first + verify_from) are context only


def check_segments(segs, R):
    """The segments must tile rows 0..R-1 in order and attach backwards."""
    if not segs:
        raise ValueError("no segments")
    nxt = 0
    for i, s in enumerate(segs):
        if s.first != nxt or s.n_rows < 1:
            raise ValueError(f"segment {i} does not continue the row order")
        if not (-1 <= s.attach < s.first):
            raise ValueError(f"segment {i} attaches forward")
        if not (0 <= s.verify_from <= s.n_rows):
            raise ValueError(f"segment {i} verify_from out of range")
        nxt += s.n_rows
    if nxt != R:
        raise ValueError("segments do not cover all rows")
    if segs[0].attach != -1:
        raise ValueError("first segment must be a root chain")


def build(segs, R, C):
    """parent [R] (-1 = root), pos [R] = C + depth, vis [R, R] bool."""
    check_segments(segs, R)
    parent = np.full(R, -1, dtype=np.int64)
    for s in segs:
        parent[s.first] = s.attach
        for i in range(1, s.n_rows):
            parent[s.first + i] = s.first + i - 1
    depth = np.zeros(R, dtype=np.int64)
    vis = np.zeros((R, R), dtype=bool)
    for r in range(R):           # parents precede children, so one pass suffices
        p = parent[r]
        if p >= 0:
            depth[r] = depth[p] + 1
            vis[r] = vis[p]
        vis[r, r] = True
    return parent, C + depth, vis


def match(tokens, g, parent, r):
    """Row r reached its fixed point: its token is its parent's prediction."""
    return parent[r] >= 0 and int(tokens[r]) == int(g[parent[r]])


def verify(tokens, g, parent, segs):
    """Per segment: longest run of matching rows from first + verify_from."""
    out = []
    for s in segs:
        m = 0
        for i in range(s.verify_from, s.n_rows):
            if match(tokens, g, parent, s.first + i):
                m += 1
            else:
                break
        out.append(m)
    return out


def winner_path(segs, m, parent):
    """Real-active winner among the Jacobi draft (segment 0) and candidates.

    The winner has the most newly accepted tokens; ties go to segment 0, then
    to the lowest candidate index.  Returns (segment index, committed rows):
    the chain of rows from the root down to the winner's last accepted row.
    """
    best, best_m = 0, m[0]
    for i, s in enumerate(segs):
        if s.role == ROLE_CAND and m[i] > best_m:
            best, best_m = i, m[i]
    s = segs[best]
    k = s.verify_from + best_m          # rows of the segment on the path
    last = s.first + k - 1 if k > 0 else s.attach
    rows = []
    while last >= 0:
        rows.append(int(last))
        last = parent[last]
    return best, rows[::-1]
