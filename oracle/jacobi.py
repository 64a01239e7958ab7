"""Greedy AR decoding, the Jacobi iteration and its drivers (oracle).

Notation of Sec. 2.1: prompt x, block of n tokens y_1..y_n.

* Eq. 1: AR greedy, y_i = argmax p(y | y_<i, x), one forward per token.
* Eq. 3: Jacobi update, y_i^(j+1) = argmax p(y | y_<i^(j), x) for all i in
  one forward pass; the fixed point y* equals the AR output (Sec. 2.1, citing
  Song et al. 2021), and the iteration stops when y^(k) = y^(k-1).
* Eq. 4: blocks of n are solved one after another until max_new.

The step computed here keeps an exact KV cache of committed tokens.  Its
first draft row is the *pending* token p: the argmax of the last committed
row, hence already correct (the i = 1 line of Eq. 3 depends on x alone).  For
a draft d[0..n-1] with d[0] = p at positions C..C+n-1:

    g[i] = argmax_v logits(prefix, d[0..i])[v]        (lowest v on ties)
    a    = 1 + max{m : d[k] = g[k-1] for all 1 <= k <= m}
    commit d[0..a-1] and their K/V;  new pending p' = g[a-1]

which is the greedy acceptance of Sec. 3.2 / App. A Alg. 1 ("accept longest
matching prefix").  The next draft is the Jacobi update of the rest,
[g[a-1], g[a], ...]: truncated to what is left of the block (block mode,
Eq. 4) or padded back to n (running window, Sec. 4.2).

Draft initialisation (random, Sec. 1 and Eq. 3) draws
pad_id(seed, pos) = splitmix64(seed XOR pos * 0x9E3779B97F4A7C15) mod V, the
first output of a splitmix64 generator (Steele, Lea & Flood 2014) whose
state is that value.
"""
from __future__ import annotations

import numpy as np

from . import tree

MASK64 = (1 << 64) - 1
GOLDEN = 0x9E3779B97F4A7C15


def splitmix64(state: int) -> int:
    """First output of splitmix64 seeded with ``state``."""
    z = (state + GOLDEN) & MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


def pad_id(seed: int, pos: int, vocab: int) -> int:
    """Random draft token for absolute position ``pos``."""
    return splitmix64((seed ^ ((pos * GOLDEN) & MASK64)) & MASK64) % vocab


def argmax_first(z) -> int:
    """argmax with the lowest index on ties (numpy's rule)."""
    return int(np.argmax(z))


def top2_gap(z) -> float:
    """Difference between the largest and second-largest logit."""
    t = np.partition(np.asarray(z, dtype=np.float64), -2)[-2:]
    return float(t[1] - t[0])


class TransformerBackend:
    """Runs steps of the oracle decoder and commits chosen rows."""

    def __init__(self, model):
        self.m = model
        self.last = None
        self.log = []

    @property
    def length(self):
        return self.m.length

    @property
    def vocab(self):
        return self.m.V

    def prefill(self, prompt, chunk: int = 0) -> int:
        z = self.m.prefill(prompt, chunk)
        self.prefill_logits = z
        return argmax_first(z)

    def step(self, tokens, segs):
        """One forward pass over the rows; returns g (argmax of every row)."""
        R = len(tokens)
        parent, pos, vis = tree.build(segs, R, self.m.length)
        logits, kv = self.m.forward(np.asarray(tokens), pos, vis)
        g = np.array([argmax_first(z) for z in logits], dtype=np.int64)
        self.last = (kv, logits, parent)
        self.log.append(dict(tokens=list(map(int, tokens)), segs=list(segs), g=g.copy(),
                             gap=np.array([top2_gap(z) for z in logits]), C=self.m.length))
        return g, parent

    def commit(self, rows):
        self.m.commit(self.last[0], rows)


def linear_segments(n: int):
    return [tree.Segment(0, n, -1, tree.ROLE_RA, 1)]


def accept_linear(draft, g) -> int:
    """a = 1 + longest prefix of draft[1:] equal to the preceding predictions."""
    a = 1
    while a < len(draft) and int(draft[a]) == int(g[a - 1]):
        a += 1
    return a


def generate_ar(backend, prompt, max_new: int):
    """Eq. 1: one forward per token; returns the generated tokens."""
    p = backend.prefill(prompt)
    out = []
    while len(out) < max_new:
        out.append(p)
        if len(out) == max_new:
            break
        g, _ = backend.step([p], linear_segments(1))
        backend.commit([0])
        p = int(g[0])
    return out


def jacobi_step(backend, draft):
    """One Jacobi iteration on a linear draft (draft[0] is the pending token).

    Returns (g, a); the caller commits rows 0..a-1.
    """
    g, _ = backend.step(draft, linear_segments(len(draft)))
    return g, accept_linear(draft, g)


def generate_jacobi(backend, prompt, n: int, max_new: int, mode: str = "block",
                    pad_seed: int = 2):
    """Jacobi decoding with KV commits.

    mode 'block'  : Eq. 4, block by block; a block's draft shrinks as its
                    tokens are accepted and a new block starts from
                    [p, pad, ...].
    mode 'window' : running window; the draft is refilled to n with pads.
    Returns (tokens, per-iteration accept counts).
    """
    V = backend.vocab
    p = backend.prefill(prompt)
    out, accepts = [], []
    left = 0
    draft = []
    while len(out) < max_new:
        C = backend.length
        if mode == "block" and left == 0:
            left = n
            draft = [p] + [pad_id(pad_seed, C + i, V) for i in range(1, n)]
        elif mode == "window" and not draft:
            draft = [p] + [pad_id(pad_seed, C + i, V) for i in range(1, n)]
        g, a = jacobi_step(backend, draft)
        a = min(a, max_new - len(out))
        backend.commit(range(a))
        out += [int(t) for t in draft[:a]]
        accepts.append(a)
        p = int(g[a - 1])
        C = backend.length
        if mode == "block":
            left -= a
            draft = [int(t) for t in g[a - 1:a - 1 + left]]
        else:
            nxt = [int(t) for t in g[a - 1:]]
            draft = nxt + [pad_id(pad_seed, C + i, V) for i in range(len(nxt), n)]
    return out, accepts


def generate_eq3(backend, prompt, n: int, max_new: int, pad_seed: int = 2):
    """Eq. 3 taken literally, block by block: no commit inside a block.

    y^(0) is random; y^(j+1) = [p, g_0 .. g_{n-2}] where p is the committed
    prefix's prediction of y_1 and g_i the prediction after y_i^(j); stop at
    y^(k) = y^(k-1), commit the whole block (Eq. 4).  Returns (tokens,
    iterations per block).
    """
    V = backend.vocab
    p = backend.prefill(prompt)
    out, iters = [], []
    while len(out) < max_new:
        C = backend.length
        y = [pad_id(pad_seed, C + i, V) for i in range(n)]
        k = 0
        while True:
            g, _ = backend.step(y, linear_segments(n))
            k += 1
            y_new = [p] + [int(t) for t in g[:n - 1]]
            if y_new == y:
                break
            y = y_new
        take = min(n, max_new - len(out))
        backend.commit(range(take))
        out += y[:take]
        iters.append(k)
        p = int(g[n - 1])
    return out, iters
