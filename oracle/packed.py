"""Sequence packing with the noise-aware causal mask (oracle).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Sec. 3.1 ("Noise-aware Causal Attention") and App. C: one training
sequence interleaves, for every block i of a response, a noisy block (the
trajectory point selected for the schedule's t_i) with its clean block (the
fixed point): [x, noisy_1, clean_1, ..., noisy_N, clean_N], 2N blocks, so
that a single forward yields the logits of both losses.  The two masks of
the packing figure:

* noisy-context (the noise-aware mask, used for L_pc of Eq. 8): a token of
  noisy block i sees the prompt, the noisy blocks before i and the earlier
  tokens of its own block; Eq. 8's student distribution is conditioned on
  x and the earlier blocks' noisy points;
* clean-context (CLLM's consistency setting, L_c of Eq. 5): a token of
  noisy block i sees the prompt, the clean blocks before i and the earlier
  tokens of its own block;

and under both, a token of clean block i sees the prompt, the clean blocks
before i and the earlier tokens of its own block (the teacher / AR side).

Readings: both copies of block i sit at the block's own positions in the
response (|x| + i n + k), not at their packed offsets, since each copy
stands for that stretch of the response; the figure itself is not in the
text available here, so the masks are taken from the prose above.

``packed_logits`` is the plain definition: a causal forward over each
chain of blocks that some row's context follows, reading every row's logits
at its position.  No attention mask is built here.
"""
from __future__ import annotations

import numpy as np

NOISY_CONTEXT = 0
CLEAN_CONTEXT = 1


def packed_tokens(noisy, clean):
    """[noisy_1, clean_1, ..., noisy_N, clean_N] as one token list."""
    if len(noisy) != len(clean) or not noisy:
        raise ValueError("need N >= 1 noisy and N clean blocks")
    n = len(noisy[0])
    out = []
    for a, b in zip(noisy, clean):
        if len(a) != n or len(b) != n:
            raise ValueError("all blocks must have n tokens")
        out += [int(t) for t in a] + [int(t) for t in b]
    return out


def row_of(i: int, copy: int, k: int, n: int) -> int:
    """Packed row of token k of block i; copy 0 = noisy, 1 = clean."""
    return (2 * i + copy) * n + k


def causal_logits(model, tokens):
    """Logits of every position of a plain causal forward over tokens, from
    an empty cache (the model's committed prefix is cleared)."""
    model.reset()
    R = len(tokens)
    logits, _ = model.forward(np.asarray(tokens), np.arange(R), np.tri(R, dtype=bool))
    return logits


def packed_logits(model, prompt, noisy, clean, mask: int):
    """Logits [2 N n][V] of the packed rows, each row conditioned on exactly
    the context its mask gives it."""
    N, n = len(noisy), len(noisy[0])
    P = len(prompt)
    x = [int(t) for t in prompt]
    out = None

    def put(i, copy, logits_of_seq):
        nonlocal out
        if out is None:
            out = np.zeros((2 * N * n, logits_of_seq.shape[1]), logits_of_seq.dtype)
        for k in range(n):
            out[row_of(i, copy, k, n)] = logits_of_seq[P + i * n + k]

    clean_seq = x + sum(([int(t) for t in b] for b in clean), [])
    Lc = causal_logits(model, clean_seq)
    for i in range(N):
        put(i, 1, Lc)
    if mask == NOISY_CONTEXT:
        Ln = causal_logits(model, x + sum(([int(t) for t in b] for b in noisy), []))
        for i in range(N):
            put(i, 0, Ln)
    elif mask == CLEAN_CONTEXT:
        for i in range(N):
            seq = x + sum(([int(t) for t in b] for b in clean[:i]), []) + [int(t) for t in noisy[i]]
            put(i, 0, causal_logits(model, seq))
    else:
        raise ValueError("mask must be NOISY_CONTEXT or CLEAN_CONTEXT")
    return out


def packed_logits_after_prefix(model, noisy, clean, mask: int):
    """packed_logits with the prompt already committed in the model's cache
    (length P): the chains are run after it, and the cache is cut back to P
    after each.  The same definition, without recomputing the prompt."""
    P = model.length
    N, n = len(noisy), len(noisy[0])

    def chain(blocks):
        toks = np.asarray(sum(([int(t) for t in b] for b in blocks), []))
        T = len(toks)
        z, _ = model.forward(toks, P + np.arange(T), np.tri(T, dtype=bool))
        model.truncate(P)
        return z

    zc = chain(clean)
    out = np.zeros((2 * N * n, zc.shape[1]), zc.dtype)
    for i in range(N):
        out[row_of(i, 1, 0, n):row_of(i, 1, 0, n) + n] = zc[i * n:(i + 1) * n]
    if mask == NOISY_CONTEXT:
        zn = chain(noisy)
        for i in range(N):
            out[row_of(i, 0, 0, n):row_of(i, 0, 0, n) + n] = zn[i * n:(i + 1) * n]
    elif mask == CLEAN_CONTEXT:
        for i in range(N):
            z = chain(list(clean[:i]) + [noisy[i]])
            out[row_of(i, 0, 0, n):row_of(i, 0, 0, n) + n] = z[i * n:(i + 1) * n]
    else:
        raise ValueError("mask must be NOISY_CONTEXT or CLEAN_CONTEXT")
    return out
