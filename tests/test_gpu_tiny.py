"""GPU parity on the tiny fp32 decoder (2 layers, d 128, 4 heads of 32,
FFN 512, V 1024): every call goes through the C ABI of libjf and is checked
against the CPU oracle on the same seeded inputs.

Tolerances: the model is fp32 end to end, so logits must agree with the
oracle's fp64 values within 1e-4 absolute; tokens must be identical except
where the oracle's top-2 logit gap is below 1e-3.
"""
import numpy as np
import pytest

import jf_inputs
from oracle import jacobi as ojac
from oracle import multiblock as omb
from oracle.model import DecoderOracle

pytestmark = pytest.mark.gpu

SHAPE = jf_inputs.MODEL_SHAPES["tiny"]
LOGIT_TOL = 1e-4
GAP_EXEMPT = 1e-3


@pytest.fixture(scope="module")
def env():
    import torch
    from paper_2512_14681_amd import decode, jf
    assert torch.cuda.is_available()
    w = jf_inputs.model_weights(SHAPE, seed=0)
    prompt = jf_inputs.prompt(1, 32, SHAPE["vocab"])
    model = jf.Model(SHAPE, w, max_rows=64, max_ctx=512)
    return dict(w=w, prompt=prompt, model=model, dec=decode.Decoder(model), jf=jf, torch=torch)


def oracle(env):
    return ojac.TransformerBackend(DecoderOracle(SHAPE, env["w"]))


def test_prefill_pending_matches(env):
    env["dec"].reset()
    p = env["dec"].prefill(env["prompt"])
    be = oracle(env)
    assert p == be.prefill(env["prompt"])


@pytest.mark.parametrize("n", [1, 5, 16, 17, 33, 64])
def test_step_logits_and_argmax(env, n):
    """One linear step of n rows (several 16-row tiles and a ragged tail)."""
    import torch
    dec, jf_ = env["dec"], env["jf"]
    dec.reset()
    p = dec.prefill(env["prompt"])
    draft = [p] + [ojac.pad_id(7, 32 + i, SHAPE["vocab"]) for i in range(1, n)]
    d_draft = torch.tensor(draft, dtype=torch.int32, device="cuda")
    d_next = torch.zeros(n, dtype=torch.int32, device="cuda")
    d_logits = torch.empty((n, SHAPE["vocab"]), dtype=torch.float32, device="cuda")
    env["model"].jf_jacobi_step(d_draft, n, 1, 7, dec.d_argmax, dec.d_result, d_next, d_logits)
    torch.cuda.synchronize()
    z = d_logits.cpu().numpy()
    g = dec.d_argmax[:n].cpu().numpy()
    res = dec.d_result.cpu().numpy()
    be = oracle(env)
    be.prefill(env["prompt"])
    gz, _ = be.step(draft, ojac.linear_segments(n))
    zo = be.last[1]
    assert np.abs(z - zo).max() < LOGIT_TOL
    gap = be.log[-1]["gap"]
    ok = (g == gz) | (gap < GAP_EXEMPT)
    assert ok.all()
    a = ojac.accept_linear(draft, gz)
    assert res[0] == a and res[2] == gz[a - 1] and res[3] == 0
    # window-mode next draft: Jacobi update then pad ids after the new length
    nxt = list(gz[a - 1:]) + [ojac.pad_id(7, 32 + a + i, SHAPE["vocab"]) for i in range(n - a + 1, n)]
    assert list(d_next.cpu().numpy()) == nxt


def test_block_mode_64_tokens_equals_ar(env):
    """Configuration 1: block n = 8, random draft init, 64 new tokens."""
    dec = env["dec"]
    dec.reset()
    got, acc = dec.generate_jacobi(env["prompt"], 8, 64, mode="block", pad_seed=2)
    want = ojac.generate_ar(oracle(env), env["prompt"], 64)
    assert got == want
    _, acc_o = ojac.generate_jacobi(oracle(env), env["prompt"], 8, 64, "block", pad_seed=2)
    assert acc == acc_o
    assert all(a >= 1 for a in acc)


@pytest.mark.parametrize("n,mode", [(1, "window"), (8, "window"), (16, "window"), (3, "block")])
def test_other_modes_equal_ar(env, n, mode):
    dec = env["dec"]
    dec.reset()
    got, acc = dec.generate_jacobi(env["prompt"], n, 40, mode=mode, pad_seed=5)
    want = ojac.generate_ar(oracle(env), env["prompt"], 40)
    assert got == want
    _, acc_o = ojac.generate_jacobi(oracle(env), env["prompt"], n, 40, mode, pad_seed=5)
    assert acc == acc_o


def test_gpu_ar_driver(env):
    dec = env["dec"]
    dec.reset()
    assert dec.generate_ar(env["prompt"], 20) == ojac.generate_ar(oracle(env), env["prompt"], 20)


def test_multiblock_lockstep(env):
    """Same policy, same model: the GPU and oracle multi-block runs take the
    same steps (rows, per-segment accepts, winner, committed tokens)."""
    dec = env["dec"]
    dec.reset()
    got, tr = dec.generate_multiblock(env["prompt"], 8, 3, 0.5, 48, pad_seed=3)
    want, tro = omb.generate_multiblock(oracle(env), env["prompt"], 8, 3, 0.5, 48, pad_seed=3)
    assert got == want == ojac.generate_ar(oracle(env), env["prompt"], 48)
    assert len(tr) == len(tro)
    for a, b in zip(tr, tro):
        assert (a["R"], a["m"], a["winner"], a["a"], a["committed"]) == \
               (b["R"], b["m"], b["winner"], b["a"], b["committed"])
    assert max(t["R"] for t in tr) > 8  # pseudo blocks were in play


def test_prefill_chunks_longer_than_max_rows(env):
    import torch
    from paper_2512_14681_amd import decode, jf
    prompt = jf_inputs.prompt(11, 100, SHAPE["vocab"])
    m = jf.Model(SHAPE, env["w"], max_rows=16, max_ctx=256)
    dec = decode.Decoder(m)
    got = dec.generate_jacobi(prompt, 16, 24, mode="window")[0]
    assert got == ojac.generate_ar(oracle(env), prompt, 24)
    assert dec.length() == 100 + 24


def test_permuted_page_table_same_tokens(env):
    from paper_2512_14681_amd import decode, jf
    m = jf.Model(SHAPE, env["w"], max_rows=16, max_ctx=256)
    m.jf_kv_set_page_table(np.array([3, 1, 0, 2], dtype=np.int32))
    dec = decode.Decoder(m)
    got = dec.generate_jacobi(env["prompt"], 8, 64, mode="window")[0]
    assert got == ojac.generate_ar(oracle(env), env["prompt"], 64)


def test_error_paths(env):
    import torch
    jf_ = env["jf"]
    from paper_2512_14681_amd import decode, jf
    m = jf.Model(SHAPE, env["w"], max_rows=16, max_ctx=128)
    dec = decode.Decoder(m)
    d = torch.zeros(32, dtype=torch.int32, device="cuda")
    with pytest.raises(jf.JfError) as e:
        m.jf_jacobi_step(d, 4, 1, 0, dec.d_argmax, dec.d_result, dec.d_next)
    assert e.value.status == jf.JF_E_STATE          # no prefill yet
    with pytest.raises(jf.JfError) as e:
        m.jf_commit_kv(None, dec.d_result)
    assert e.value.status == jf.JF_E_STATE          # nothing to commit
    dec.prefill(env["prompt"])
    with pytest.raises(jf.JfError) as e:
        m.jf_jacobi_step(d, 17, 1, 0, dec.d_argmax, dec.d_result, dec.d_next)
    assert e.value.status == jf.JF_E_CAPACITY       # n > max_rows
    with pytest.raises(jf.JfError) as e:
        m.jf_jacobi_step(d, 4, 4, 0, dec.d_argmax, dec.d_result, dec.d_next)
    assert e.value.status == jf.JF_E_INVAL          # bad mode
    bad = [[(0, 3, -1, 0, 1), (4, 1, 0, 1, 0)],     # gap in rows
           [(0, 3, 0, 0, 1)],                       # first not a root
           [(0, 2, -1, 1, 1)],                      # first not real-active
           [(0, 2, -1, 0, 1), (2, 2, 2, 1, 0)]]     # attaches forward
    for segs in bad:
        R = sum(s[1] for s in segs)
        with pytest.raises(jf.JfError) as e:
            m.jf_multiblock_step(d, R, segs, dec.d_argmax, dec.d_seg, dec.d_result, dec.d_path)
        assert e.value.status == jf.JF_E_INVAL
    with pytest.raises(jf.JfError) as e:
        m.jf_kv_truncate(1000)
    assert e.value.status == jf.JF_E_STATE
    # capacity: perfect drafts (the AR tokens) commit all 16 rows per step;
    # 32 + 6 * 16 = 128 = max_ctx, so a seventh step has no room
    ar = ojac.generate_ar(oracle(env), env["prompt"], 112)
    for i in range(6):
        d[:16] = torch.tensor(ar[16 * i:16 * i + 16], dtype=torch.int32)
        m.jf_jacobi_step(d, 16, 1, 0, dec.d_argmax, dec.d_result, dec.d_next)
        m.jf_commit_kv(None, dec.d_result)
        assert dec.d_result.cpu()[0] == 16
    assert m.jf_kv_length() == 128
    with pytest.raises(jf.JfError) as e:
        m.jf_jacobi_step(d, 16, 1, 0, dec.d_argmax, dec.d_result, dec.d_next)
    assert e.value.status == jf.JF_E_CAPACITY
    # max_commit caps what a commit keeps
    m.jf_kv_truncate(32)
    d[:16] = torch.tensor(ar[:16], dtype=torch.int32)
    m.jf_jacobi_step(d, 16, 1, 0, dec.d_argmax, dec.d_result, dec.d_next)
    m.jf_commit_kv(None, dec.d_result, 5)
    assert m.jf_kv_length() == 37
    # out-of-range token ids are flagged by the device, never read out of bounds
    m.jf_kv_truncate(32)
    d[:4] = torch.tensor([5, 2000, -3, 7], dtype=torch.int32)
    m.jf_jacobi_step(d, 4, 1, 0, dec.d_argmax, dec.d_result, dec.d_next)
    res = dec.d_result.cpu().numpy()
    assert res[3] & jf.JF_FLAG_BAD_TOKEN


@pytest.mark.parametrize("m_len", [1, 5, 8])
def test_tree_commit_moves_winning_candidate(env, m_len):
    """A recycled candidate that holds the oracle's greedy continuation wins
    the step; the commit moves its rows' K/V from their in-step slots to
    C + 1 .. C + m (source != destination), and the next step, run on the
    moved cache, matches an oracle that committed the same rows (Sec. 3.2:
    only the winning branch is committed; App. A Alg. 1 drops the rest)."""
    import torch
    from oracle import tree as otree
    dec, jf_, model = env["dec"], env["jf"], env["model"]
    V = SHAPE["vocab"]
    n = 8
    prompt = env["prompt"]
    ar = ojac.generate_ar(oracle(env), prompt, n + 1)       # ar[0] = pending token
    rng = np.random.default_rng(100 + m_len)
    rand = lambda k: [int(t) for t in rng.integers(0, V, k)]
    ra = [ar[0]] + rand(n - 1)
    ra[1] = (ar[1] + 1) % V                                  # the Jacobi draft fails at once
    cand_a = rand(n)
    cand_b = ar[1:1 + m_len] + rand(n - m_len)
    if m_len < n:
        cand_b[m_len] = (ar[1 + m_len] + 1) % V              # stops after m_len rows
    pseudo = rand(n)
    tokens = ra + pseudo + cand_a + cand_b
    segs = [(0, n, -1, jf_.JF_ROLE_RA, 1), (n, n, n - 1, jf_.JF_ROLE_PSEUDO, 0),
            (2 * n, n, 0, jf_.JF_ROLE_CAND, 0), (3 * n, n, 0, jf_.JF_ROLE_CAND, 0)]
    R = len(tokens)
    dec.reset()
    p = dec.prefill(prompt)
    assert p == ar[0]
    d_tok = torch.tensor(tokens, dtype=torch.int32, device="cuda")
    d_log = torch.empty((R, V), dtype=torch.float32, device="cuda")
    model.jf_multiblock_step(d_tok, R, segs, dec.d_argmax, dec.d_seg, dec.d_result, dec.d_path, d_log)
    # oracle: the same step, its verification and winner
    be = oracle(env)
    be.prefill(prompt)
    osegs = [otree.Segment(*s) for s in segs]
    go, parent = be.step(tokens, osegs)
    assert np.abs(d_log.cpu().numpy() - be.last[1]).max() < LOGIT_TOL
    m = otree.verify(tokens, go, parent, osegs)
    win, path = otree.winner_path(osegs, m, parent)
    assert win == 3 and path == [0] + list(range(3 * n, 3 * n + m_len))
    res = dec.d_result.cpu().numpy()
    assert list(dec.d_seg.cpu().numpy()[:4]) == m
    assert res[0] == len(path) and res[1] == win and res[2] == go[path[-1]]
    assert list(dec.d_path.cpu().numpy()[:len(path)]) == path
    # commit the winning path (its candidate rows move down to C + 1 ..)
    model.jf_commit_kv(dec.d_path, dec.d_result)
    be.commit(path)
    assert dec.length() == be.length == len(prompt) + 1 + m_len
    # next step on the moved cache
    p2 = int(go[path[-1]])
    draft = [p2] + [ojac.pad_id(9, be.length + i, V) for i in range(1, n)]
    d_draft = torch.tensor(draft, dtype=torch.int32, device="cuda")
    d_next = torch.zeros(n, dtype=torch.int32, device="cuda")
    d_log2 = torch.empty((n, V), dtype=torch.float32, device="cuda")
    model.jf_jacobi_step(d_draft, n, 1, 9, dec.d_argmax, dec.d_result, d_next, d_log2)
    g2, _ = be.step(draft, ojac.linear_segments(n))
    err = np.abs(d_log2.cpu().numpy() - be.last[1]).max()
    assert err < LOGIT_TOL, err
    gap = be.log[-1]["gap"]
    assert ((dec.d_argmax[:n].cpu().numpy() == g2) | (gap < GAP_EXEMPT)).all()
    # and the committed tokens are the greedy continuation
    assert ar[:1 + m_len] == [tokens[r] for r in path]


@pytest.mark.parametrize("mode", [0, 1])
def test_step_commit_flag_equals_step_then_commit(env, mode):
    """jf_jacobi_step with JF_STEP_COMMIT (argmax reduction, acceptance and
    commit in one launch) against the step followed by jf_commit_kv: the same
    argmax, result, next draft and committed length at every iteration of a
    decode; no jf_commit_kv may follow a committing step."""
    import torch
    from paper_2512_14681_amd import decode, jf
    V, n = SHAPE["vocab"], 8
    runs = []
    for fused in (False, True):
        m = jf.Model(SHAPE, env["w"], max_rows=16, max_ctx=256)
        dec = decode.Decoder(m)
        p = dec.prefill(env["prompt"])
        C = len(env["prompt"])
        d_tok = torch.tensor([p] + [decode.pad_token(3, C + i, V) for i in range(1, n)], dtype=torch.int32,
                             device="cuda")
        rec = []
        for it in range(12):
            if fused:
                m.jf_jacobi_step(d_tok, n, mode | jf.JF_STEP_COMMIT, 3, dec.d_argmax, dec.d_result, d_tok)
            else:
                m.jf_jacobi_step(d_tok, n, mode, 3, dec.d_argmax, dec.d_result, d_tok)
                m.jf_commit_kv(None, dec.d_result)
            rec.append((dec.d_result.cpu().numpy().copy(), dec.d_argmax[:n].cpu().numpy().copy(),
                        d_tok.cpu().numpy().copy(), m.jf_kv_length()))
            if mode == 0:   # block mode: restart the block from the new pending token
                res = rec[-1][0]
                d_tok[0] = int(res[2])
        if fused:
            with pytest.raises(jf.JfError) as e:
                m.jf_commit_kv(None, dec.d_result)
            assert e.value.status == jf.JF_E_STATE
        runs.append(rec)
    for (r0, g0, t0, c0), (r1, g1, t1, c1) in zip(*runs):
        assert (r0 == r1).all() and (g0 == g1).all() and c0 == c1
        assert (t0 == t1).all() if mode == 1 else (t0[0] == t1[0])
