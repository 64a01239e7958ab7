"""Jacobi trajectories and the noise-schedule point selection (oracle).

TEST INFRASTRUCTURE ONLY (see the package docstring).

* Trajectory (Sec. 2.1, after Eq. 3): for one block of n tokens, the iterates
  J = {y^(0), ..., y^(k)} of the Jacobi update, where the iteration stops at
  the first k with y^(k) = y^(k-1); y* := y^(k) is the fixed point, so J ends
  with the fixed point twice.  A long response is decoded block after block
  (Eq. 4): the next block's context is the previous blocks' fixed points.
* Unconverged tokens (Sec. 3.1, the footnote to Eq. 6 on "noisy" tokens): the positions of an
  iterate that differ from the fixed point at the same position.
* Noise schedule (Sec. 3.1, Eq. 7): W = {0, 1/w, ..., (w-1)/w} and block i
  takes t_i = W[i mod w].
* Point selection (App. C, sequence packing): for block i, the trajectory
  point whose unconverged fraction (unconverged count / n) is closest to t_i.

Readings where the paper leaves a choice open:

* Block index i counts from 0, so each window of w blocks starts clean
  (t = 0) and ends at (w-1)/w; the text says the ratio rises from 0 within
  each window.
* Ties in |u/n - t| go to the earliest point of the trajectory.
* y^(0) of a block is [p, pad(C+1), ..., pad(C+n-1)]: its first position
  already holds p, the prediction of the committed context (the i = 1 line
  of Eq. 3 depends on the context alone, so y^(1) would hold p there for any
  initialisation); the rest is the seeded draft initialisation.  The
  iteration itself is Eq. 3 over all n positions, with no acceptance and no
  commit inside a block.
* The progressive-loss paragraph of Sec. 3.1 (Eq. 8) states the target as a noisy-token count closest
  to ceil(t_i n); it selects the same point as the fraction rule whenever
  t_i n is an integer (n = 16, w = 16 and n = 32, w = 8 in Sec. 4.1).
  ``select_point_by_count`` implements that wording for the comparison.
"""
from __future__ import annotations

from fractions import Fraction
from math import ceil

from .jacobi import linear_segments, pad_id


def noise_ratio(i: int, w: int) -> Fraction:
    """Eq. 7: t_i = W[i mod w], W[j] = j / w (exact)."""
    if w < 1:
        raise ValueError("window w must be >= 1")
    return Fraction(i % w, w)


def unconverged(y, y_star) -> int:
    """Number of positions where y differs from the fixed point y*."""
    if len(y) != len(y_star):
        raise ValueError("iterate and fixed point differ in length")
    return sum(1 for a, b in zip(y, y_star) if int(a) != int(b))


def select_point(traj, t) -> int:
    """Index j of the point of one block's trajectory whose unconverged
    fraction is closest to t (earliest on ties).  The fixed point is the last
    point of traj."""
    if not traj:
        raise ValueError("empty trajectory")
    n = len(traj[-1])
    t = Fraction(t)
    best, best_d = 0, None
    for j, y in enumerate(traj):
        d = abs(Fraction(unconverged(y, traj[-1]), n) - t)
        if best_d is None or d < best_d:
            best, best_d = j, d
    return best


def select_point_by_count(traj, t) -> int:
    """The count wording: noisy-token count closest to ceil(t n) (earliest on
    ties)."""
    n = len(traj[-1])
    target = ceil(Fraction(t) * n)
    best, best_d = 0, None
    for j, y in enumerate(traj):
        d = abs(unconverged(y, traj[-1]) - target)
        if best_d is None or d < best_d:
            best, best_d = j, d
    return best


def select_points(trajs, w: int, t_num=None):
    """Selected point per block: block i uses t_i = W[i mod w] (Eq. 7), or
    t_num[i] / w when a per-block table of numerators is given (another
    schedule, e.g. the random or reversed ones of Sec. 4.3, on the same
    denominator)."""
    out = []
    for i, traj in enumerate(trajs):
        t = noise_ratio(i, w) if t_num is None else Fraction(int(t_num[i]), w)
        out.append(select_point(traj, t))
    return out


def block_trajectory(backend, y0, p, max_iters: int = 0):
    """Eq. 3 on one block against the backend's committed context, from the
    initial iterate y0 (y0[0] is ignored by the update: position 0 always
    becomes p, the context's prediction).  Returns (trajectory, g of the
    last iteration); the last g[n-1] predicts the token after the block."""
    n = len(y0)
    y = [int(t) for t in y0]
    traj = [list(y)]
    it = 0
    while True:
        g, _ = backend.step(y, linear_segments(n))
        nxt = [int(p)] + [int(t) for t in g[:n - 1]]
        traj.append(nxt)
        it += 1
        if nxt == y:
            return traj, g
        if max_iters and it >= max_iters:
            raise RuntimeError("no fixed point within max_iters iterations")
        y = nxt


def collect_trajectories(backend, prompt, n: int, n_blocks: int, pad_seed: int = 2):
    """Decode n_blocks blocks of n tokens after the prompt (Eq. 4) and
    return every block's trajectory (Sec. 2.1).  The converged block is
    committed before the next block starts."""
    V = backend.vocab
    p = backend.prefill(prompt)
    trajs = []
    for _ in range(n_blocks):
        C = backend.length
        y0 = [p] + [pad_id(pad_seed, C + i, V) for i in range(1, n)]
        traj, g = block_trajectory(backend, y0, p)
        backend.commit(range(n))
        trajs.append(traj)
        p = int(g[n - 1])
    return trajs
