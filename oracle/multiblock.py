"""Multi-block decoding with rejection recycling (oracle), App. A Alg. 1.

Sec. 3.2: up to K blocks are refined at once.  The block at the KV boundary
is real-active (RA): only its tokens are accepted and committed.  The others
are pseudo-active: their tokens are only pseudo-accepted, conditioned on the
blocks before them, and are verified again once promoted to RA.  Rejection
recycling keeps a fixed-size pool of n-grams taken from unconverged drafts; an
n-gram whose first token equals the current pending token becomes a candidate
that is verified next to the RA draft, and the branch with most accepted
tokens wins.  Both are lossless: only greedily verified RA tokens commit.

The paper leaves several choices open; this module takes these readings
(listed in the design doc with the reasons):

1. RA draft: block mode of Eq. 3/4 (shrinks to n - |a_RA|); row 0 is the
   pending token p.
2. Assemble (Alg. 1): RA draft, then every pseudo block b as a_b || q_b (n
   rows, chained after the previous block; a_b rows are context only), then
   up to ``n_cand`` candidates.
3. Candidates: pool entries e with e[0] = p, most recent first; rows e[1:L]
   with L = min(len(e), cand_len, |q_RA|), attached under RA row 0; skipped
   when empty, equal to the RA draft's prefix, or a duplicate.
4. Winner: most accepted tokens; ties to the RA draft, then the lowest
   candidate.  Commit its path; p' = argmax of the path's last row.
5. Pool: after each iteration the RA draft's rejected suffix d[a_RA:] (its own
   count, whoever won) is pushed if it has >= 2 tokens; FIFO of ``pool_cap``.
6. RA tail: [g of the winner branch from its last accepted row on], padded
   with pad ids and truncated to n - |a_RA|.
7. Pseudo block tail: a_b grows by the matched prefix of q_b; every other
   q_b token becomes its parent row's prediction (Jacobi update).
8. Spawn (after the update): if some block has |a_b| >= s = ceil(r n) and
   fewer than K blocks exist, append a block whose draft is q_RA right-padded
   with pad ids to n.
9. Promote: when |a_RA| = n, the next block in position order becomes RA
   with draft (a_b || q_b) and row 0 replaced by p'; without one, a fresh
   [p', pad ...] block.
10. Stop when max_new tokens are committed.
"""
from __future__ import annotations

import math

from . import tree
from .jacobi import pad_id


class Block:
    def __init__(self, start, acc, draft):
        self.start = start      # absolute position of the block's first token
        self.acc = list(acc)    # accepted (RA: committed) or pseudo-accepted
        self.draft = list(draft)


def generate_multiblock(backend, prompt, n: int, K: int, r: float, max_new: int,
                        n_cand: int = 8, cand_len: int = 16, pool_cap: int = 64,
                        pad_seed: int = 2):
    """Returns (tokens, trace); trace holds one dict per iteration."""
    V = backend.vocab
    s_thr = math.ceil(r * n)
    p = backend.prefill(prompt)
    C = backend.length
    ra = Block(C, [], [p] + [pad_id(pad_seed, C + i, V) for i in range(1, n)])
    pseudo = []
    pool = []
    out, trace = [], []
    while len(out) < max_new:
        C = backend.length
        # ---- assemble -------------------------------------------------
        tokens = list(ra.draft)
        segs = [tree.Segment(0, len(ra.draft), -1, tree.ROLE_RA, 1)]
        last = len(tokens) - 1
        for b in pseudo:
            rows = b.acc + b.draft
            segs.append(tree.Segment(len(tokens), len(rows), last, tree.ROLE_PSEUDO, len(b.acc)))
            tokens += rows
            last = len(tokens) - 1
        chosen = []
        for e in reversed(pool):
            if len(chosen) >= n_cand:
                break
            if e[0] != p:
                continue
            L = min(len(e), cand_len, len(ra.draft))
            rows = tuple(e[1:L])
            if not rows or tuple(e[:L]) == tuple(ra.draft[:L]) or rows in chosen:
                continue
            chosen.append(rows)
        for rows in chosen:
            segs.append(tree.Segment(len(tokens), len(rows), 0, tree.ROLE_CAND, 0))
            tokens += list(rows)
        # ---- forward + verify ------------------------------------------
        g, parent = backend.step(tokens, segs)
        m = tree.verify(tokens, g, parent, segs)
        win, path = tree.winner_path(segs, m, parent)
        a = min(len(path), max_new - len(out))
        path = path[:a]
        backend.commit(path)
        committed = [int(tokens[i]) for i in path]
        out += committed
        p_new = int(g[path[-1]])
        trace.append(dict(R=len(tokens), segs=segs, m=list(m), winner=win, a=a,
                          committed=committed))
        if len(out) >= max_new:
            break
        C = backend.length
        # ---- RA tail update + pool ---------------------------------------
        a_ra = 1 + m[0]
        rejected = ra.draft[a_ra:]
        if len(rejected) >= 2:
            pool.append(tuple(int(t) for t in rejected))
            if len(pool) > pool_cap:
                pool.pop(0)
        ra.acc += committed
        left = n - len(ra.acc)
        ws = segs[win]
        branch = list(range(ws.n_rows)) if win == 0 else [0] + list(range(ws.first, ws.first + ws.n_rows))
        nxt = [int(g[i]) for i in branch[a - 1:]]
        nxt += [pad_id(pad_seed, C + i, V) for i in range(len(nxt), left)]
        ra.draft = nxt[:left]
        # ---- pseudo blocks -------------------------------------------------
        for bi, b in enumerate(pseudo):
            sg = segs[1 + bi]
            mb = m[1 + bi]
            b.acc += b.draft[:mb]
            b.draft = [int(g[parent[sg.first + i]]) for i in range(len(b.acc), n)]
        # ---- spawn ---------------------------------------------------------
        blocks = [ra] + pseudo
        if len(blocks) < K and any(len(b.acc) >= s_thr for b in blocks):
            start = blocks[-1].start + n
            d = list(ra.draft) + [pad_id(pad_seed, start + i, V) for i in range(len(ra.draft), n)]
            pseudo.append(Block(start, [], d[:n]))
        # ---- promote -------------------------------------------------------
        if len(ra.acc) >= n:
            if pseudo:
                b = pseudo.pop(0)
                rows = b.acc + b.draft
                ra = Block(b.start, [], [p_new] + rows[1:n])
            else:
                ra = Block(C, [], [p_new] + [pad_id(pad_seed, C + i, V) for i in range(1, n)])
        p = p_new
    return out, trace
