"""Pins of the packed-sequence oracle (oracle/packed.py):

* layout by hand;
* clean rows are the AR teacher: on the greedy continuation (Eq. 1) every
  clean row's argmax is the next token of the continuation;
* clean-context noisy rows are the Jacobi update (Eq. 3): with block i's
  noisy copy a point y^(j) of its trajectory (collected against the clean
  fixed points of the blocks before it), the noisy rows' argmaxes are
  y^(j+1) shifted by one -- checked against the trajectory oracle, which
  runs the step against a committed cache instead;
* the two masks agree on block 0, and on every block whose earlier noisy
  blocks equal their clean ones.
"""
import numpy as np
import pytest

import jf_inputs
from oracle import jacobi as ojac
from oracle import packed as opk
from oracle import trajectory as otr
from oracle.model import DecoderOracle

SHAPE = jf_inputs.MODEL_SHAPES["tiny"]


@pytest.fixture(scope="module")
def tiny():
    w = jf_inputs.model_weights(SHAPE, seed=0)
    return w, DecoderOracle(SHAPE, w)


def test_layout_by_hand():
    assert opk.packed_tokens([[1, 2], [5, 6]], [[3, 4], [7, 8]]) == [1, 2, 3, 4, 5, 6, 7, 8]
    assert [opk.row_of(i, c, k, 2) for i in range(2) for c in range(2) for k in range(2)] == list(range(8))
    with pytest.raises(ValueError):
        opk.packed_tokens([[1, 2]], [[3]])


def test_clean_rows_are_the_ar_teacher(tiny):
    w, m = tiny
    prompt = jf_inputs.prompt(2, 20, SHAPE["vocab"])
    N, n = 3, 6
    ar = ojac.generate_ar(ojac.TransformerBackend(DecoderOracle(SHAPE, w)), prompt, N * n + 1)
    clean = [ar[i * n:(i + 1) * n] for i in range(N)]
    noisy = [list(jf_inputs.token_ids(3, i, n, SHAPE["vocab"])) for i in range(N)]
    for mask in (opk.NOISY_CONTEXT, opk.CLEAN_CONTEXT):
        z = opk.packed_logits(m, prompt, noisy, clean, mask)
        for i in range(N):
            for k in range(n):
                assert int(np.argmax(z[opk.row_of(i, 1, k, n)])) == ar[i * n + k + 1]


def test_clean_context_noisy_rows_are_the_jacobi_update(tiny):
    w, m = tiny
    prompt = jf_inputs.prompt(4, 24, SHAPE["vocab"])
    N, n = 3, 8
    trajs = otr.collect_trajectories(ojac.TransformerBackend(DecoderOracle(SHAPE, w)), prompt, n, N)
    clean = [t[-1] for t in trajs]
    for j in range(3):
        idx = [min(j, len(t) - 2) for t in trajs]        # a non-final point of every block
        noisy = [t[x] for t, x in zip(trajs, idx)]
        z = opk.packed_logits(m, prompt, noisy, clean, opk.CLEAN_CONTEXT)
        for i in range(N):
            g = [int(np.argmax(z[opk.row_of(i, 0, k, n)])) for k in range(n)]
            assert g[:n - 1] == trajs[i][idx[i] + 1][1:], (j, i)


def test_masks_agree_where_the_contexts_do(tiny):
    w, m = tiny
    prompt = jf_inputs.prompt(5, 16, SHAPE["vocab"])
    N, n, V = 3, 5, SHAPE["vocab"]
    clean = [list(jf_inputs.token_ids(6, i, n, V)) for i in range(N)]
    noisy = [list(jf_inputs.token_ids(7, i, n, V)) for i in range(N)]
    a = opk.packed_logits(m, prompt, noisy, clean, opk.NOISY_CONTEXT)
    b = opk.packed_logits(m, prompt, noisy, clean, opk.CLEAN_CONTEXT)
    rows0 = [opk.row_of(0, 0, k, n) for k in range(n)]
    assert np.abs(a[rows0] - b[rows0]).max() < 1e-12
    rows1 = [opk.row_of(1, 0, k, n) for k in range(n)]
    assert np.abs(a[rows1] - b[rows1]).max() > 1e-3          # block 1's contexts differ
    noisy2 = [clean[0], clean[1], noisy[2]]                  # earlier noisy blocks = clean
    a2 = opk.packed_logits(m, prompt, noisy2, clean, opk.NOISY_CONTEXT)
    b2 = opk.packed_logits(m, prompt, noisy2, clean, opk.CLEAN_CONTEXT)
    assert np.abs(a2 - b2).max() < 1e-12


@pytest.mark.parametrize("mask", [opk.NOISY_CONTEXT, opk.CLEAN_CONTEXT])
def test_after_prefix_form_equals_the_full_form(tiny, mask):
    w, m = tiny
    prompt = jf_inputs.prompt(8, 18, SHAPE["vocab"])
    N, n, V = 3, 4, SHAPE["vocab"]
    clean = [list(jf_inputs.token_ids(9, i, n, V)) for i in range(N)]
    noisy = [list(jf_inputs.token_ids(10, i, n, V)) for i in range(N)]
    full = opk.packed_logits(m, prompt, noisy, clean, mask)
    m2 = DecoderOracle(SHAPE, w)
    m2.prefill(np.asarray(prompt))
    cached = opk.packed_logits_after_prefix(m2, noisy, clean, mask)
    assert m2.length == len(prompt)
    assert np.abs(full - cached).max() < 1e-10
