"""Deterministic next-token backends (oracle test doubles).

A greedy causal LM is, for the decoding algorithms, a function from a context
(the token sequence up to and including a row) to the next token.  These
backends implement that function directly, so the Jacobi and multi-block
state machines can be exercised -- including long accepted runs and recycled
candidates, which a random transformer almost never produces -- and checked
against sequential greedy decoding (Eq. 1).
"""
from __future__ import annotations

import numpy as np

from . import tree


class FunctionBackend:
    """next token = f(context), context = committed tokens + ancestors + row."""

    def __init__(self, f, vocab: int):
        self.f = f
        self.V = vocab
        self.ctx = []
        self.last = None
        self.log = []

    @property
    def vocab(self):
        return self.V

    @property
    def length(self):
        return len(self.ctx)

    def prefill(self, prompt, chunk: int = 0) -> int:
        self.ctx = [int(t) for t in prompt]
        return int(self.f(tuple(self.ctx)))

    def step(self, tokens, segs):
        R = len(tokens)
        parent, _, _ = tree.build(segs, R, len(self.ctx))
        g = np.zeros(R, dtype=np.int64)
        for r in range(R):
            chain = []
            x = r
            while x >= 0:
                chain.append(int(tokens[x]))
                x = parent[x]
            g[r] = self.f(tuple(self.ctx + chain[::-1]))
        self.last = list(tokens)
        self.log.append(dict(tokens=list(map(int, tokens)), segs=list(segs), g=g.copy()))
        return g, parent

    def commit(self, rows):
        self.ctx += [int(self.last[i]) for i in rows]


def ar_reference(f, prompt, max_new):
    """Sequential greedy decoding with a next-token function (Eq. 1)."""
    ctx = [int(t) for t in prompt]
    out = []
    for _ in range(max_new):
        t = int(f(tuple(ctx)))
        out.append(t)
        ctx.append(t)
    return out


def hash_fn(vocab, order=3, salt=0):
    """Next token = hash of the last ``order`` tokens."""
    def f(ctx):
        h = 1469598103934665603 ^ salt
        for t in ctx[-order:]:
            h = ((h ^ t) * 1099511628211) & ((1 << 64) - 1)
        return h % vocab
    return f


def copy_fn(offset=3):
    """Next token = the token ``offset`` places back (periodic output)."""
    return lambda ctx: ctx[-offset]


def const_fn(token=5):
    return lambda ctx: token


def cycle_fn(vocab, period=7):
    """Next token = (last + 1) mod period: a short deterministic cycle."""
    return lambda ctx: (ctx[-1] + 1) % min(period, vocab)


def mixed_fn(vocab, salt=0):
    """Alternates long repetitive stretches with hashed ones (pool hits)."""
    h = hash_fn(vocab, 2, salt)

    def f(ctx):
        if (len(ctx) // 23) % 2 == 0:
            return ctx[-5]
        return h(ctx)
    return f
