"""GPU parity of the attention and LM-head components through the C ABI.

Attention (the attention inside Eq. 3's forward pass) is compared with the
oracle's masked softmax attention; the LM head + argmax + acceptance (Eq. 3 /
Alg. 1 verification) with the plain fp64 product and numpy's argmax.

Tolerances, from the arithmetic:
* LM head: inputs are exact bf16/fp32 values, accumulation is fp32, so the
  logits differ from fp64 by the fp32 summation error, < 1e-3 absolute for
  these sizes (K <= 3584, |x w| < 0.1); tokens must match except where the
  oracle's top-2 gap is below 1e-3.
* attention: activations (q, output) travel as bf16 hi+lo planes (~16
  significant bits) and the softmax weights enter the PV contraction as a
  hi+lo bf16 pair, so |gpu - oracle| <= 2^-14 |oracle| + 1e-4 (bf16 cache);
  fp32 models: 1e-5.
"""
import numpy as np
import pytest

import jf_inputs
from oracle.model import DecoderOracle
from oracle.numerics import bf16_bits_to_float, round_bf16

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    assert torch.cuda.is_available()
    return torch


def to_dev(a):
    torch = _torch()
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).to("cuda")


def bf16_bits(x):
    """float64 -> bf16 bit patterns (round to nearest even) for test inputs."""
    r = round_bf16(np.asarray(x, np.float64)).astype(np.float32)
    return (r.view(np.uint32) >> 16).astype(np.uint16)


def planes(bits):
    """Activation planes of bf16 values: hi = the values, lo = 0."""
    return np.stack([bits, np.zeros_like(bits)])


def from_planes(a):
    """hi + lo of a [2, ...] uint16 plane pair, as float64."""
    return bf16_bits_to_float(a[0]) + bf16_bits_to_float(a[1])


# ------------------------------------------------------------------ LM head
def run_lm_head(x_bits_or_f32, w, R, d, V, dtype, draft=None, want_logits=True):
    torch = _torch()
    from paper_2512_14681_amd import jf
    L = jf.lib()
    dt = jf.JF_BF16 if dtype == "bf16" else jf.JF_F32
    d_w = to_dev(w)
    d_wp = torch.empty(L.jf_packed_matrix_bytes(V, d, dt), dtype=torch.uint8, device="cuda")
    st = jf._stream()
    jf.check(L.jf_pack_matrix(V, d, dt, jf._ptr(d_w), jf._ptr(d_wp), st))
    del d_w
    xl = jf.act_layout(x_bits_or_f32)          # GEMM-input layout, rows padded to 16
    d_x = to_dev(planes(xl) if dtype == "bf16" else xl)
    d_g = torch.zeros(R, dtype=torch.int32, device="cuda")
    d_res = torch.zeros(4, dtype=torch.int32, device="cuda")
    d_log = torch.empty((R, V), dtype=torch.float32, device="cuda") if want_logits else None
    d_ws = torch.empty(L.jf_lm_head_ws_bytes(R, V), dtype=torch.uint8, device="cuda")
    d_draft = to_dev(np.asarray(draft, np.int32)) if draft is not None else None
    jf.check(L.jf_lm_head_accept(R, d, V, dt, jf._ptr(d_x), jf._ptr(d_wp), jf._ptr(d_draft),
                                 jf._ptr(d_g), jf._ptr(d_res) if draft is not None else None,
                                 jf._ptr(d_log), jf._ptr(d_ws), st))
    torch.cuda.synchronize()
    return (d_g.cpu().numpy(), d_res.cpu().numpy(),
            d_log.cpu().numpy() if want_logits else None)


def top2(z):
    s = np.sort(z, axis=1)
    return s[:, -1] - s[:, -2]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("R", [1, 16, 17, 64, 200])
def test_lm_head_small(dtype, R):
    d, V = 256, 1024
    x = jf_inputs.normal(3, 1, R * d, dtype=dtype).reshape(R, d)
    w = jf_inputs.normal(3, 2, V * d, std=0.02, dtype=dtype).reshape(V, d)
    xf = bf16_bits_to_float(x) if dtype == "bf16" else x.astype(np.float64)
    wf = bf16_bits_to_float(w) if dtype == "bf16" else w.astype(np.float64)
    z = xf @ wf.T
    gz = np.argmax(z, axis=1)
    g, _, logits = run_lm_head(x, w, R, d, V, dtype)
    assert np.abs(logits - z).max() < 1e-4
    assert ((g == gz) | (top2(z) < 1e-3)).all()


def test_lm_head_acceptance_closed_form():
    """Draft = shifted argmax (self-consistent) perturbed at p: accept == p."""
    d, V, R = 256, 2048, 48
    x = jf_inputs.normal(4, 1, R * d, dtype="bf16").reshape(R, d)
    w = jf_inputs.normal(4, 2, V * d, std=0.02, dtype="bf16").reshape(V, d)
    g0, _, _ = run_lm_head(x, w, R, d, V, "bf16", want_logits=False)
    for p in (1, 7, 16, 47):
        draft = np.concatenate([[5], g0[:-1]]).astype(np.int32)
        draft[p] = (draft[p] + 1) % V
        g, res, _ = run_lm_head(x, w, R, d, V, "bf16", draft=draft, want_logits=False)
        assert res[0] == p and res[2] == g[p - 1]
    draft = np.concatenate([[5], g0[:-1]]).astype(np.int32)
    _, res, _ = run_lm_head(x, w, R, d, V, "bf16", draft=draft, want_logits=False)
    assert res[0] == R


@pytest.mark.parametrize("R", [25, 32, 48, 80, 96, 128, 144, 192, 256, 384, 512])
def test_lm_head_column_slice_chunks(R):
    """A vocabulary wide enough for the column-slice GEMM (2048 tiles of 16
    columns, K = 1024): 32-, 64-, 96- and 128-row chunks, one to four of
    them (128 and 256 rows: two and four 64-row chunks; 384 rows: four
    96-row chunks; 512 rows: four 128-row chunks), with ragged last chunks
    (25 = 32 - 7, 80 = 96 - 16, 144 = 96 + 48).  bf16 values, plain fp64
    product and argmax."""
    d, V = 1024, 32768
    x = jf_inputs.normal(5, 1, R * d, dtype="bf16").reshape(R, d)
    w = jf_inputs.normal(5, 2, V * d, std=0.02, dtype="bf16").reshape(V, d)
    z = bf16_bits_to_float(x) @ bf16_bits_to_float(w).T
    g, _, logits = run_lm_head(x, w, R, d, V, "bf16")
    assert np.abs(logits - z).max() < 1e-3
    assert ((g == np.argmax(z, axis=1)) | (top2(z) < 1e-3)).all()


def test_lm_head_full_size_config3():
    """LM head of the 7B shape: hidden [64, 3584] ~ N(0,1), W [152064, 3584] ~
    N(0, 0.02), bf16; per-row argmax and the perturbed-draft acceptance."""
    R, d, V = 64, 3584, 152064
    w = jf_inputs.normal(0, 3000, V * d, std=0.02, dtype="bf16").reshape(V, d)
    wf32 = bf16_bits_to_float(w, np.float32)
    for t in range(3):
        x = jf_inputs.normal(1000 + t, 1, R * d, dtype="bf16").reshape(R, d)
        xf = bf16_bits_to_float(x)
        z = np.empty((R, V))
        for s in range(0, V, 16384):      # plain fp64 product, in vocab chunks
            z[:, s:s + 16384] = xf @ wf32[s:s + 16384].astype(np.float64).T
        gz = np.argmax(z, axis=1)
        p = int(jf_inputs.uniform_int(1000 + t, 2, 1, 1, R)[0])
        draft = np.concatenate([[0], gz[:-1]]).astype(np.int32)
        draft[p] = (draft[p] + 1) % V
        g, res, logits = run_lm_head(x, w, R, d, V, "bf16", draft=draft)
        assert np.abs(logits - z).max() < 1e-3
        ok = (g == gz) | (top2(z) < 1e-3)
        assert ok.all()
        if (g[:p] == gz[:p]).all():
            assert res[0] == p


# ---------------------------------------------------------------- attention
def pages_from(K, Vv, G, hd, perm, bits):
    """Paged layout of one layer: page = K [G][64][hd], then V^T [G][hd][64]."""
    S = K.shape[0]
    n_pages = len(perm)
    dt = np.uint16 if bits else np.float32
    buf = np.zeros((n_pages, 2, G, 64 * hd), dtype=dt)
    for p in range(n_pages):
        lo, hi = p * 64, min(S, p * 64 + 64)
        if lo >= S:
            continue
        kp = np.zeros((64, G, hd), dt); vp = np.zeros((64, G, hd), dt)
        kp[:hi - lo] = K[lo:hi]; vp[:hi - lo] = Vv[lo:hi]
        buf[perm[p], 0] = kp.transpose(1, 0, 2).reshape(G, 64 * hd)
        buf[perm[p], 1] = vp.transpose(1, 2, 0).reshape(G, 64 * hd)
    return buf


def run_attention(H, G, hd, dtype, C, R, seed, tree=False):
    torch = _torch()
    from paper_2512_14681_amd import jf
    L = jf.lib()
    dt = jf.JF_BF16 if dtype == "bf16" else jf.JF_F32
    S = C + R
    q = jf_inputs.normal(seed, 1, R * H * hd, dtype=dtype).reshape(R, H, hd)
    K = jf_inputs.normal(seed, 2, S * G * hd, dtype=dtype).reshape(S, G, hd)
    Vv = jf_inputs.normal(seed, 3, S * G * hd, dtype=dtype).reshape(S, G, hd)
    n_pages = (S + 63) // 64
    perm = np.random.default_rng(seed).permutation(n_pages).astype(np.int32)
    buf = pages_from(K, Vv, G, hd, perm, dtype == "bf16")
    vis = np.tri(R, dtype=bool)
    if tree:   # a random forest: each row hangs under a random earlier row
        rng = np.random.default_rng(seed + 1)
        parent = [-1] + [int(rng.integers(-1, r)) for r in range(1, R)]
        vis = np.zeros((R, R), bool)
        for r in range(R):
            vis[r, r] = True
            if parent[r] >= 0:
                vis[r] |= vis[parent[r]]
    words = np.zeros((R, jf.JF_VIS_WORDS), np.uint64)
    for r in range(R):
        for j in np.nonzero(vis[r])[0]:
            words[r, j // 64] |= np.uint64(1) << np.uint64(j % 64)
    d_q = to_dev(planes(q) if dtype == "bf16" else q)
    d_kv, d_pt = to_dev(buf), to_dev(perm)
    d_vis = to_dev(words.view(np.int64)) if tree else None
    Rp = (R + 15) // 16 * 16                    # out: GEMM-input layout of [R][H*hd]
    oshape = (2, Rp * H * hd) if dtype == "bf16" else (Rp * H * hd,)
    d_out = torch.empty(oshape, dtype=torch.int16 if dtype == "bf16" else torch.float32, device="cuda")
    d_ws = torch.empty(L.jf_attention_ws_bytes(H, hd, R), dtype=torch.uint8, device="cuda")
    jf.check(L.jf_attention(H, G, hd, dt, C, R, jf._ptr(d_q), jf._ptr(d_kv), jf._ptr(d_pt),
                            jf._ptr(d_vis), jf._ptr(d_out), jf._ptr(d_ws), jf._stream()))
    torch.cuda.synchronize()
    out = d_out.cpu().numpy()
    if dtype == "bf16":
        u = out.view(np.uint16)
        out = from_planes(np.stack([jf.act_unlayout(u[p], R, H * hd) for p in (0, 1)]))
    else:
        out = jf.act_unlayout(out, R, H * hd).astype(np.float64)
    out = out.reshape(q.shape)
    # oracle: masked softmax attention over [prefix; visible rows]
    dec = lambda a: bf16_bits_to_float(a) if dtype == "bf16" else a.astype(np.float64)
    shape = dict(n_layers=1, d_model=H * hd, n_heads=H, n_kv_heads=G, head_dim=hd, d_ffn=128,
                 vocab=16, rope_base=10000.0, rms_eps=1e-6, dtype="f32")
    m = DecoderOracle(shape, {})
    m.K[0], m.Vc[0] = dec(K[:C]), dec(Vv[:C])
    want = m.attention(0, dec(q), dec(K[C:]), dec(Vv[C:]), vis)
    return out, want


def check_attn(out, want, dtype):
    if dtype == "bf16":
        assert (np.abs(out - want) <= 2.0 ** -14 * np.abs(want) + 1e-4).all(), np.abs(out - want).max()
    else:
        assert np.abs(out - want).max() < 1e-5


@pytest.mark.parametrize("H,G,hd,dtype", [(4, 4, 32, "f32"), (8, 2, 64, "bf16"), (28, 4, 128, "bf16"),
                                          (28, 4, 128, "f32")])
@pytest.mark.parametrize("C,R", [(0, 1), (5, 16), (100, 17), (600, 64), (130, 200), (40, 512)])
def test_attention_small(H, G, hd, dtype, C, R):
    out, want = run_attention(H, G, hd, dtype, C, R, seed=C * 7 + R)
    check_attn(out, want, dtype)


@pytest.mark.parametrize("R", [9, 64, 192, 320, 512])
def test_attention_tree_mask(R):
    out, want = run_attention(28, 4, 128, "bf16", 300, R, seed=R, tree=True)
    check_attn(out, want, "bf16")


@pytest.mark.parametrize("P", [512, 2048, 8192])
@pytest.mark.parametrize("n", [16, 32, 64])
def test_attention_config2(P, n):
    """Attention workload: 28 q / 4 kv heads, hd 128, N(0,1) bf16 Q/K/V,
    prefix P, n draft queries causal within the block."""
    out, want = run_attention(28, 4, 128, "bf16", P, n, seed=10 + P + n)
    check_attn(out, want, "bf16")
