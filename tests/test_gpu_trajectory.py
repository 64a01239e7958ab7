"""GPU parity of trajectory recording and noise-schedule point selection
(jf_trajectory_record, jf_trajectory_select) against the oracle
(oracle/trajectory.py).  Everything is integer work: results must be
bit-exact.
"""
from fractions import Fraction

import numpy as np
import pytest

import jf_inputs
from oracle import jacobi as ojac
from oracle import trajectory as otr
from oracle.model import DecoderOracle

pytestmark = pytest.mark.gpu

SHAPE = jf_inputs.MODEL_SHAPES["tiny"]
# the full-size selection workload: 2^18 blocks of 16 tokens (up to 17
# points each), Eq. 7 with w = 16
FULL_BLOCKS, FULL_N, FULL_W = 1 << 18, 16, 16


@pytest.fixture(scope="module")
def torch_jf():
    import torch
    from paper_2512_14681_amd import jf
    assert torch.cuda.is_available()
    return torch, jf


def test_record_update_rule(torch_jf):
    """Every rows in [1, n], written to a separate buffer and in place."""
    torch, jf = torch_jf
    n = 300                                  # more than one workgroup of 256
    prev = jf_inputs.token_ids(3, 1, n, 1000)
    g = jf_inputs.token_ids(3, 2, n, 1000)
    d_prev = torch.as_tensor(prev, device="cuda")
    d_g = torch.as_tensor(g, device="cuda")
    for rows in (1, 2, 17, 255, 256, 299, 300):
        want = np.concatenate([prev[:n - rows + 1], g[:rows - 1]])
        d_out = torch.full((n,), -7, dtype=torch.int32, device="cuda")
        jf.trajectory_record(d_prev, d_g, n, rows, d_out)
        assert np.array_equal(d_out.cpu().numpy(), want), rows
        d_io = d_prev.clone()
        jf.trajectory_record(d_io, d_g, n, rows, d_io)
        assert np.array_equal(d_io.cpu().numpy(), want), rows
    with pytest.raises(jf.JfError):
        jf.trajectory_record(d_prev, d_g, n, n + 1, d_prev)
    with pytest.raises(jf.JfError):
        jf.trajectory_record(d_prev, d_g, n, 0, d_prev)


@pytest.mark.parametrize("n,blocks", [(8, 4), (16, 3)])
def test_trajectories_equal_oracle_eq3(torch_jf, n, blocks):
    """Block-mode decoding with commits on the GPU records exactly the
    trajectories of Eq. 3 iterated over the whole block without commits."""
    torch, jf = torch_jf
    from paper_2512_14681_amd import decode
    w = jf_inputs.model_weights(SHAPE, seed=0)
    prompt = jf_inputs.prompt(1, 32, SHAPE["vocab"])
    model = jf.Model(SHAPE, w, max_rows=64, max_ctx=256)
    d_traj, lengths = decode.Decoder(model).collect_trajectories(prompt, n, blocks, pad_seed=4)
    got = d_traj.cpu().numpy()
    want = otr.collect_trajectories(ojac.TransformerBackend(DecoderOracle(SHAPE, w)), prompt, n, blocks,
                                    pad_seed=4)
    assert [len(t) for t in want] == lengths.tolist()
    for b, traj in enumerate(want):
        assert got[b, :lengths[b]].tolist() == traj, b
        assert (got[b, lengths[b]:] == -1).all()


def select_on_gpu(torch, jf, traj, lengths, w, t_num=None, unconv=True):
    nb, P, n = traj.shape
    d_traj = torch.as_tensor(traj, device="cuda")
    d_len = torch.as_tensor(lengths, device="cuda")
    d_sel = torch.full((nb,), -9, dtype=torch.int32, device="cuda")
    d_u = torch.full((nb, P), -9, dtype=torch.int32, device="cuda") if unconv else None
    d_t = torch.as_tensor(np.asarray(t_num, np.int32), device="cuda") if t_num is not None else None
    jf.trajectory_select(d_traj, d_len, nb, n, P, w, d_sel, d_t_num=d_t, d_unconv=d_u)
    return d_sel.cpu().numpy(), (d_u.cpu().numpy() if unconv else None)


def oracle_select(traj, lengths, w, t_num=None, blocks=None):
    blocks = range(len(lengths)) if blocks is None else blocks
    sel, unc = {}, {}
    for b in blocks:
        L = int(lengths[b])
        if not 1 <= L <= traj.shape[1]:
            sel[b], unc[b] = -1, [-1] * traj.shape[1]
            continue
        pts = traj[b, :L].tolist()
        t = otr.noise_ratio(b, w) if t_num is None else Fraction(int(t_num[b]), w)
        sel[b] = otr.select_point(pts, t)
        unc[b] = [otr.unconverged(y, pts[-1]) for y in pts] + [-1] * (traj.shape[1] - L)
    return sel, unc


# (n, blocks, w, max_points - n): the launch takes 4 blocks per wave when
# all points fit 8 loads of floor(64 / n) points, 2 blocks per wave up to 17
# loads, else one block per wave
@pytest.mark.parametrize("n,nb,w,extra", [
    (1, 300, 4, 3), (5, 1000, 3, 3), (16, 3001, 16, 3), (21, 800, 16, 1),   # 4 per wave, <= 5 loads
    (16, 1001, 16, 16), (8, 999, 16, 56),                                  # 4 per wave, 8 loads
    (16, 501, 16, 17), (32, 2000, 8, 1),                                   # 2 per wave
    (1, 200, 4, 64),                                                       # more than 64 points
    (16, 300, 1 << 21, 1),                                                 # n w >= 2^25
    (32, 500, 8, 3), (48, 500, 16, 3), (64, 700, 16, 3), (65, 300, 16, 3), (200, 120, 8, 3)])
def test_select_equals_oracle(torch_jf, n, nb, w, extra):
    """Ragged trajectories (every length from 2 to n + 1), lengths outside
    [1, max_points] (-1) next to valid blocks of the same wave, a ragged
    last workgroup."""
    torch, jf = torch_jf
    P = n + extra
    traj, lengths = jf_inputs.trajectories(7 + n, nb, n, 152064, max_points=P)
    lengths[5] = 0
    lengths[6] = P + 1
    lengths[7] = P                           # the last point: -1 rows are the fixed point
    sel, unc = select_on_gpu(torch, jf, traj, lengths, w)
    want_sel, want_unc = oracle_select(traj, lengths, w)
    assert sel.tolist() == [want_sel[b] for b in range(nb)]
    assert unc.tolist() == [want_unc[b] for b in range(nb)]


def test_select_with_a_schedule_table(torch_jf):
    """Per-block targets t_num / w (e.g. the reversed schedule), including
    t = 1 and out-of-range numerators."""
    torch, jf = torch_jf
    n, nb, w = 16, 999, 16
    traj, lengths = jf_inputs.trajectories(21, nb, n, 1000)
    t_num = (jf_inputs.uniform_int(21, 3, nb, -2, w + 3)).astype(np.int32)
    t_num[:w] = np.arange(w)[::-1]           # reversed progressive on the first window
    t_num[w:w + 4] = [-(1 << 30), 1 << 30, -(1 << 31), (1 << 31) - 1]
    sel, _ = select_on_gpu(torch, jf, traj, lengths, w, t_num=t_num, unconv=False)
    want, _ = oracle_select(traj, lengths, w, t_num=t_num)
    assert sel.tolist() == [want[b] for b in range(nb)]


def test_select_empty_and_errors(torch_jf):
    torch, jf = torch_jf
    d = torch.zeros(16, dtype=torch.int32, device="cuda")
    jf.trajectory_select(d, d, 0, 4, 4, 16, d)           # n_blocks = 0: nothing to do
    with pytest.raises(jf.JfError):
        jf.trajectory_select(d, d, 1, 0, 4, 16, d)
    with pytest.raises(jf.JfError):
        jf.trajectory_select(d, d, 1, 4, 4, 0, d)
    with pytest.raises(jf.JfError):
        jf.trajectory_select(None, d, 1, 4, 4, 16, d)


def test_select_full_size_sampled(torch_jf):
    """The benchmarked workload (2^18 blocks of 16 tokens, w = 16) in the
    same launch; 2000 sampled blocks checked against the oracle, and every
    selected index within its block's trajectory."""
    torch, jf = torch_jf
    traj, lengths = jf_inputs.trajectories(5, FULL_BLOCKS, FULL_N, 152064)
    sel, _ = select_on_gpu(torch, jf, traj, lengths, FULL_W, unconv=False)
    assert ((sel >= 0) & (sel < lengths)).all()
    rng = np.random.default_rng(0)
    sample = sorted(set(rng.integers(0, FULL_BLOCKS, 2000).tolist()) | {0, FULL_BLOCKS - 1})
    want, _ = oracle_select(traj, lengths, FULL_W, blocks=sample)
    assert [int(sel[b]) for b in sample] == [want[b] for b in sample]
