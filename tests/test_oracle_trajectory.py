"""Pins of the trajectory oracle (oracle/trajectory.py) against what the paper
and the mathematics fix: a hand-worked selection example, Eq. 7's values,
the closed-form trajectory of a successor "model", the fixed point of
Eq. 3 equals greedy AR decoding (Sec. 2.1), the one-position-per-iteration
convergence bound, and where the two wordings of the selection rule agree.
"""
from fractions import Fraction

import numpy as np
import pytest

import jf_inputs
from oracle import jacobi as ojac
from oracle import mock
from oracle import trajectory as otr
from oracle.model import DecoderOracle

# n = 4; fixed point [5, 7, 8, 9]; unconverged counts 3, 2, 1, 0, 0
HAND = [[5, 1, 1, 1], [5, 7, 2, 1], [5, 7, 8, 3], [5, 7, 8, 9], [5, 7, 8, 9]]


def test_unconverged_counts_by_hand():
    assert [otr.unconverged(y, HAND[-1]) for y in HAND] == [3, 2, 1, 0, 0]


@pytest.mark.parametrize("t,j", [
    (0, 3),                    # first point with no noisy token
    (Fraction(1, 4), 2),       # u = 1
    (Fraction(1, 2), 1),       # u = 2
    (Fraction(3, 4), 0),       # u = 3
    (1, 0),                    # nothing is fully noisy: the closest is u = 3
    (Fraction(3, 8), 1),       # u = 1 and u = 2 tie at 1/8: earliest point
    (Fraction(1, 8), 2),       # u = 0 and u = 1 tie: earliest of (j=2, j=3, j=4)
])
def test_select_point_by_hand(t, j):
    assert otr.select_point(HAND, t) == j


def test_noise_ratio_eq7():
    w = 16
    assert otr.noise_ratio(0, w) == 0
    assert otr.noise_ratio(1, w) == Fraction(1, 16)
    assert otr.noise_ratio(15, w) == Fraction(15, 16)
    assert otr.noise_ratio(16, w) == 0          # cyclic with period w
    assert otr.noise_ratio(33, w) == Fraction(1, 16)
    assert otr.noise_ratio(7, 8) == Fraction(7, 8)
    assert all(otr.noise_ratio(i, w) < 1 for i in range(100))
    with pytest.raises(ValueError):
        otr.noise_ratio(1, 0)


def successor(V):
    return lambda ctx: (ctx[-1] + 1) % V


def test_block_trajectory_successor_by_hand():
    """next token = last + 1: y^(j+1)_i = y^(j)_{i-1} + 1, written out."""
    V = 100
    be = mock.FunctionBackend(successor(V), V)
    p = be.prefill([3, 9])
    assert p == 10
    traj, g = otr.block_trajectory(be, [10, 50, 60, 70], p)
    assert traj == [[10, 50, 60, 70],
                    [10, 11, 51, 61],
                    [10, 11, 12, 52],
                    [10, 11, 12, 13],
                    [10, 11, 12, 13]]
    assert int(g[3]) == 14


def test_schedule_selection_closed_form():
    """Successor model, n = w = 16: point j has n - 1 - j noisy tokens, so
    block i (t_i = (i mod 16)/16, target i mod 16 noisy tokens) selects
    j = 15 - (i mod 16)."""
    V, n, w = 1 << 20, 16, 16
    be = mock.FunctionBackend(successor(V), V)
    trajs = otr.collect_trajectories(be, [1, 2, 3], n, 40, pad_seed=11)
    for traj in trajs:
        assert len(traj) == n + 1
        assert [otr.unconverged(y, traj[-1]) for y in traj] == [max(n - 1 - j, 0) for j in range(n + 1)]
    assert otr.select_points(trajs, w) == [15 - (i % 16) for i in range(40)]


@pytest.mark.parametrize("fn", ["hash", "mixed", "cycle"])
def test_fixed_points_equal_greedy_ar(fn):
    """Sec. 2.1: the fixed point of Eq. 3 is the greedy AR output; blocks
    concatenate (Eq. 4).  Also: position j is converged after iteration j
    (at least one more position per iteration, so k <= n), the last two
    points are equal and no earlier consecutive pair is."""
    V, n, nb = 64, 8, 5
    f = {"hash": mock.hash_fn(V, salt=3), "mixed": mock.mixed_fn(V, salt=1),
         "cycle": mock.cycle_fn(V)}[fn]
    prompt = [7, 1, 30, 2, 11, 5]
    trajs = otr.collect_trajectories(mock.FunctionBackend(f, V), prompt, n, nb, pad_seed=5)
    ar = mock.ar_reference(f, prompt, n * nb)
    assert sum((t[-1] for t in trajs), []) == ar
    for traj in trajs:
        k = len(traj) - 1
        assert 1 <= k <= n
        assert traj[-1] == traj[-2]
        assert all(traj[j] != traj[j + 1] for j in range(k - 1))
        for j, y in enumerate(traj):
            m = min(j + 1, n)
            assert y[:m] == traj[-1][:m]


def test_fixed_points_equal_greedy_ar_transformer():
    """The same theorem on the tiny decoder (fp64 oracle forward)."""
    shape = jf_inputs.MODEL_SHAPES["tiny"]
    w = jf_inputs.model_weights(shape, seed=0)
    prompt = jf_inputs.prompt(1, 24, shape["vocab"])
    trajs = otr.collect_trajectories(ojac.TransformerBackend(DecoderOracle(shape, w)), prompt, 8, 3)
    ar = ojac.generate_ar(ojac.TransformerBackend(DecoderOracle(shape, w)), prompt, 24)
    assert sum((t[-1] for t in trajs), []) == ar
    assert all(len(t) - 1 <= 8 for t in trajs)


def random_trajectory(rng, n, V=50):
    """A plausible trajectory: the converged prefix grows by 1..3 per step,
    the tail is random; ends with the fixed point twice."""
    y_star = list(rng.integers(0, V, n))
    traj, m = [], 1
    while m < n:
        traj.append(y_star[:m] + list(rng.integers(0, V, n - m)))
        m += int(rng.integers(1, 4))
    traj += [y_star, y_star]
    return traj


@pytest.mark.parametrize("n,w", [(16, 16), (32, 8), (16, 4), (64, 16)])
def test_count_wording_agrees_when_tn_is_integral(n, w):
    rng = np.random.default_rng(n * 100 + w)
    for i in range(300):
        traj = random_trajectory(rng, n)
        t = otr.noise_ratio(i, w)
        assert (t * n).denominator == 1
        assert otr.select_point(traj, t) == otr.select_point_by_count(traj, t)


def test_count_wording_can_differ_otherwise():
    """n = 10, t = 1/4: the fraction rule aims at 2.5 noisy tokens, the count
    rule at ceil(2.5) = 3; with counts 10, 4, 2, 0, 0 they pick different
    points."""
    y_star = list(range(10))
    traj = [[99] * 10, [99] * 4 + y_star[4:], [99] * 2 + y_star[2:], y_star, y_star]
    assert [otr.unconverged(y, y_star) for y in traj] == [10, 4, 2, 0, 0]
    assert otr.select_point(traj, Fraction(1, 4)) == 2
    assert otr.select_point_by_count(traj, Fraction(1, 4)) == 1


def test_select_points_with_a_table():
    trajs = [HAND] * 4
    assert otr.select_points(trajs, 4) == [3, 2, 1, 0]
    assert otr.select_points(trajs, 4, t_num=[3, 3, 0, 2]) == [0, 0, 3, 1]
