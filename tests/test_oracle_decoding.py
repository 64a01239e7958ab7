"""Pins for the oracle's step structure and decoding drivers (CPU).

What the paper fixes and these tests check:
* Sec. 2.1: the Jacobi fixed point equals greedy AR output (Eq. 1), and the
  first row of every iteration is always correct, so each iteration accepts
  >= 1 token and an n-block needs <= n iterations;
* Sec. 3.2 / App. A: rejection recycling and multi-block decoding are
  lossless -- their output equals greedy AR output.
"""
import itertools

import numpy as np
import pytest

import jf_inputs
from oracle import jacobi, mock, multiblock, tree
from oracle.model import DecoderOracle

MICRO = dict(n_layers=1, d_model=16, n_heads=2, n_kv_heads=1, head_dim=8,
             d_ffn=24, vocab=8, rope_base=10000.0, rms_eps=1e-6, dtype="f32")


def tiny_model(seed, vocab=64, layers=1, d=16, heads=2, kv=1, hd=8, ffn=32):
    shape = dict(n_layers=layers, d_model=d, n_heads=heads, n_kv_heads=kv, head_dim=hd,
                 d_ffn=ffn, vocab=vocab, rope_base=10000.0, rms_eps=1e-6, dtype="f32")
    w = jf_inputs.model_weights(shape, seed=seed)
    # larger weights than N(0, 0.02) so that tiny random models are not
    # degenerate (near-uniform logits would make every argmax a coin toss)
    w = {k: (v * 40.0 if v.ndim == 2 else v) for k, v in w.items()}
    return shape, w


def backend(shape, w):
    return jacobi.TransformerBackend(DecoderOracle(shape, w))


# ---------------------------------------------------------------- tree
def test_single_segment_is_causal_triangle():
    parent, pos, vis = tree.build(jacobi.linear_segments(6), 6, 10)
    np.testing.assert_array_equal(vis, np.tri(6, dtype=bool))
    np.testing.assert_array_equal(pos, 10 + np.arange(6))
    np.testing.assert_array_equal(parent, [-1, 0, 1, 2, 3, 4])


def test_visibility_is_ancestor_closure_brute_force():
    rng = np.random.default_rng(0)
    for _ in range(200):
        segs, first = [], 0
        for i in range(rng.integers(1, 7)):
            nr = int(rng.integers(1, 6))
            att = -1 if i == 0 else int(rng.integers(-1, first))
            segs.append(tree.Segment(first, nr, att, tree.ROLE_CAND, 0))
            first += nr
        parent, pos, vis = tree.build(segs, first, 3)
        # brute force: reachability along parent edges (transitive closure)
        A = np.eye(first, dtype=int)
        for r in range(first):
            if parent[r] >= 0:
                A[r, parent[r]] = 1
        Rch = np.linalg.matrix_power(A, first) > 0
        np.testing.assert_array_equal(vis, Rch)
        np.testing.assert_array_equal(pos - 3, Rch.sum(axis=1) - 1)


def test_check_segments_rejects_bad_forests():
    S = tree.Segment
    with pytest.raises(ValueError):
        tree.build([S(0, 2, -1, 0, 1), S(3, 1, 0, 1, 0)], 4, 0)      # gap
    with pytest.raises(ValueError):
        tree.build([S(0, 2, -1, 0, 1), S(2, 2, 2, 1, 0)], 4, 0)      # attaches to itself
    with pytest.raises(ValueError):
        tree.build([S(0, 2, 0, 0, 1)], 2, 0)                         # first not a root
    with pytest.raises(ValueError):
        tree.build([S(0, 2, -1, 0, 1)], 3, 0)                        # rows uncovered


def test_candidate_branch_equals_separate_linear_step():
    """Sec. 3.2 verifies candidates 'along the batch dimension'; the tree pass
    must give every branch exactly the logits of its own linear step."""
    shape, w = tiny_model(1, vocab=50)
    prompt = jf_inputs.prompt(2, 9, 50)
    m = DecoderOracle(shape, w)
    m.prefill(prompt)
    draft, c1, c2 = [7, 3, 9, 11], [21, 4], [8, 8, 30]
    toks = draft + c1 + c2
    segs = [tree.Segment(0, 4, -1, 0, 1), tree.Segment(4, 2, 0, 1, 0), tree.Segment(6, 3, 0, 1, 0)]
    parent, pos, vis = tree.build(segs, len(toks), m.length)
    lt, _ = m.forward(toks, pos, vis)
    for rows, lin in (([0, 1, 2, 3], draft), ([0, 4, 5], [7] + c1), ([0, 6, 7, 8], [7] + c2)):
        ll, _ = m.forward(lin, m.length + np.arange(len(lin)), np.tri(len(lin), dtype=bool))
        assert np.array_equal(lt[rows], ll)


def test_verify_and_winner_handcrafted():
    S = tree.Segment
    segs = [S(0, 4, -1, 0, 1), S(4, 3, 0, 1, 0), S(7, 2, 0, 1, 0), S(9, 3, 3, 2, 1)]
    toks = [5, 6, 1, 2, 6, 9, 3, 6, 9, 0, 4, 4]
    parent, _, _ = tree.build(segs, 12, 0)
    g = np.zeros(12, int)
    g[0] = 6; g[1] = 0; g[4] = 9; g[5] = 7; g[7] = 9; g[8] = 1; g[3] = 0; g[9] = 1; g[10] = 4
    m = tree.verify(toks, g, parent, segs)
    assert m == [1, 2, 2, 0]            # RA: 6 ok, 1 != 0; cand1: 6,9 ok, 3 != 7; cand2: 6,9
    win, path = tree.winner_path(segs, m, parent)
    assert win == 1 and path == [0, 4, 5]      # tie 2 vs 2: lowest candidate wins
    m2 = [3, 2, 3, 0]
    win, path = tree.winner_path(segs, m2, parent)
    assert win == 0 and path == [0, 1, 2, 3]   # tie with the RA draft: RA wins


# ---------------------------------------------------------------- Jacobi
def test_exhaustive_drafts_micro_model_closed_form():
    """V = 8, n = 4: every draft d[1..3] (512) accepts exactly 1 + the longest
    prefix of d[1:] that equals the AR continuation, and the new pending
    token is the next AR token."""
    w = jf_inputs.model_weights(MICRO, seed=5)
    w = {k: (v * 40.0 if v.ndim == 2 else v) for k, v in w.items()}
    prompt = jf_inputs.prompt(6, 5, 8)
    ar = jacobi.generate_ar(backend(MICRO, w), prompt, 5)
    be = backend(MICRO, w)
    p = be.prefill(prompt)
    assert p == ar[0]
    for tail in itertools.product(range(8), repeat=3):
        d = [p] + list(tail)
        g, a = jacobi.jacobi_step(be, d)
        k = 0
        while k < 3 and d[1 + k] == ar[1 + k]:
            k += 1
        assert a == 1 + k
        assert g[a - 1] == ar[a]


@pytest.mark.parametrize("seed", range(100))
def test_jacobi_equals_ar_random_tiny_models(seed):
    rng = np.random.default_rng(seed)
    vocab = int(rng.choice([8, 16, 64, 256, 1024]))
    layers = int(rng.integers(1, 3))
    n = int(rng.choice([1, 2, 3, 5, 8, 16]))
    shape, w = tiny_model(100 + seed, vocab=vocab, layers=layers)
    prompt = jf_inputs.prompt(seed, 6, vocab)
    max_new = 24
    ar = jacobi.generate_ar(backend(shape, w), prompt, max_new)
    for mode in ("block", "window"):
        out, acc = jacobi.generate_jacobi(backend(shape, w), prompt, n, max_new, mode, pad_seed=seed)
        assert out == ar, mode
        assert all(a >= 1 for a in acc)
        if n == 1:
            assert acc == [1] * max_new
    if seed % 4 == 0:
        out, iters = jacobi.generate_eq3(backend(shape, w), prompt, n, max_new, pad_seed=seed)
        assert out == ar
        assert all(k <= n + 1 for k in iters)    # n updates + the confirming pass


def test_block_mode_at_most_n_iterations_per_block():
    shape, w = tiny_model(7, vocab=16)
    be = backend(shape, w)
    out, acc = jacobi.generate_jacobi(be, jf_inputs.prompt(1, 4, 16), 5, 40, "block")
    # consecutive accepts fill blocks of exactly n = 5
    it, s = 0, 0
    for a in acc:
        s += a; it += 1
        assert it <= 5
        if s == 5:
            s, it = 0, 0
        assert s < 5


def test_perturbed_draft_accepts_up_to_perturbation():
    """A draft built from the AR tokens is accepted whole; changing the token
    at position p (1 <= p < n) makes exactly p tokens accepted."""
    shape, w = tiny_model(9, vocab=256)
    prompt = jf_inputs.prompt(3, 7, 256)
    n = 10
    ar = jacobi.generate_ar(backend(shape, w), prompt, n + 1)
    be = backend(shape, w)
    be.prefill(prompt)
    g, a = jacobi.jacobi_step(be, ar[:n])
    assert a == n and list(g) == ar[1:n + 1]
    for p in range(1, n):
        d = list(ar[:n]); d[p] = (d[p] + 1) % 256
        g, a = jacobi.jacobi_step(be, d)
        assert a == p


# ---------------------------------------------------------------- multi-block
FUNCS = {
    "hash": lambda V: mock.hash_fn(V, 3, 1),
    "copy": lambda V: mock.copy_fn(3),
    "const": lambda V: mock.const_fn(5),
    "cycle": lambda V: mock.cycle_fn(V, 7),
    "mixed": lambda V: mock.mixed_fn(V, 2),
}


@pytest.mark.parametrize("fname", sorted(FUNCS))
@pytest.mark.parametrize("n,K,r", [(4, 2, 0.5), (8, 4, 0.85), (16, 4, 0.85), (5, 3, 0.3)])
def test_multiblock_lossless_mock(fname, n, K, r):
    V = 50
    f = FUNCS[fname](V)
    prompt = [int(t) for t in jf_inputs.prompt(4, 12, V)]
    ar = mock.ar_reference(f, prompt, 120)
    out, trace = multiblock.generate_multiblock(mock.FunctionBackend(f, V), prompt, n, K, r, 120)
    assert out == ar
    assert all(t["a"] >= 1 for t in trace)
    assert max(t["R"] for t in trace) <= n * K + 8 * 15


def test_multiblock_exercises_its_state_machine():
    """On a repetitive next-token function, candidates win, pseudo blocks are
    spawned and promoted, and more than one token is accepted per pass."""
    V = 40
    f = mock.mixed_fn(V, 3)
    prompt = [int(t) for t in jf_inputs.prompt(5, 24, V)]
    out, trace = multiblock.generate_multiblock(mock.FunctionBackend(f, V), prompt, 8, 3, 0.5, 200)
    assert out == mock.ar_reference(f, prompt, 200)
    assert any(t["winner"] > 0 for t in trace)                      # recycled n-gram won
    assert any(any(s.role == tree.ROLE_PSEUDO for s in t["segs"]) for t in trace)
    assert sum(t["a"] for t in trace) / len(trace) > 1.5
    # copy-from-far-back contexts converge a whole block per pass or two
    f2 = mock.copy_fn(13)
    out2, tr2 = multiblock.generate_multiblock(mock.FunctionBackend(f2, V), prompt, 16, 4, 0.5, 200)
    assert out2 == mock.ar_reference(f2, prompt, 200)
    assert max(t["a"] for t in tr2) == 16


def test_multiblock_single_block_no_pool_is_block_jacobi():
    """K = 1 with no candidates is block-mode Jacobi decoding (Eq. 3-4)."""
    shape, w = tiny_model(11, vocab=32)
    prompt = jf_inputs.prompt(8, 6, 32)
    out_j, acc_j = jacobi.generate_jacobi(backend(shape, w), prompt, 6, 30, "block")
    out_m, tr = multiblock.generate_multiblock(backend(shape, w), prompt, 6, 1, 0.85, 30, n_cand=0)
    assert out_m == out_j
    assert [t["a"] for t in tr] == acc_j


@pytest.mark.parametrize("seed", range(6))
def test_multiblock_lossless_transformer(seed):
    shape, w = tiny_model(200 + seed, vocab=24)
    prompt = jf_inputs.prompt(seed, 6, 24)
    ar = jacobi.generate_ar(backend(shape, w), prompt, 40)
    out, tr = multiblock.generate_multiblock(backend(shape, w), prompt, 4, 4, 0.5, 40, pad_seed=seed)
    assert out == ar
