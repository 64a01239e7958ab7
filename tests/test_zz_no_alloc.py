"""The allocation-free LM-head entry point (jf_lm_head_accept_noalloc, for
callers that cannot allocate device memory) against jf_lm_head_accept with a
caller workspace: identical argmax, acceptance and logits, on two calls in a
row through the C ABI, the second with fewer rows and a smaller vocabulary
(the shared fixed scratch keeps the first call's contents)."""
import numpy as np
import pytest

import jf_inputs

pytestmark = pytest.mark.gpu


def _run(L, jf, torch, R, d, V, seed, noalloc):
    st = jf._stream()
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    w = (torch.randn(V, d, device="cuda", generator=g) * 0.02).to(torch.bfloat16)
    wp = torch.empty(L.jf_packed_matrix_bytes(V, d, jf.JF_BF16), dtype=torch.uint8, device="cuda")
    jf.check(L.jf_pack_matrix(V, d, jf.JF_BF16, jf._ptr(w.view(torch.int16)), jf._ptr(wp), st))
    Rp = (R + 15) // 16 * 16
    x = torch.zeros(2, Rp * d, dtype=torch.int16, device="cuda")
    xr = torch.randn(R, d, device="cuda", generator=g).to(torch.bfloat16).view(torch.int16).cpu().numpy()
    x[0].copy_(torch.from_numpy(jf.act_layout(xr).astype(np.int16)))
    am = torch.zeros(R, dtype=torch.int32, device="cuda")
    res = torch.full((4,), -7, dtype=torch.int32, device="cuda")
    logits = torch.empty((R, V), dtype=torch.float32, device="cuda")
    # drafts: first the plain argmax (no acceptance), then a shifted copy
    # perturbed at p, which must accept exactly p
    jf.check(L.jf_lm_head_accept(R, d, V, jf.JF_BF16, jf._ptr(x), jf._ptr(wp), None, jf._ptr(am), None, None,
                                 jf._ptr(torch.empty(L.jf_lm_head_ws_bytes(R, V), dtype=torch.uint8,
                                                     device="cuda")), st))
    g0 = am.cpu().numpy()
    p = R // 2
    draft = np.concatenate([[3], g0[:-1]]).astype(np.int32)
    draft[p] = (draft[p] + 1) % V
    d_draft = torch.as_tensor(draft, device="cuda")
    am.zero_()
    if noalloc:
        jf.check(L.jf_lm_head_accept_noalloc(R, d, V, jf.JF_BF16, jf._ptr(x), jf._ptr(wp), jf._ptr(d_draft),
                                             jf._ptr(am), jf._ptr(res), jf._ptr(logits), st))
    else:
        ws = torch.empty(L.jf_lm_head_ws_bytes(R, V), dtype=torch.uint8, device="cuda")
        jf.check(L.jf_lm_head_accept(R, d, V, jf.JF_BF16, jf._ptr(x), jf._ptr(wp), jf._ptr(d_draft),
                                     jf._ptr(am), jf._ptr(res), jf._ptr(logits), jf._ptr(ws), st))
    torch.cuda.synchronize()
    return am.cpu().numpy(), res.cpu().numpy(), logits.cpu().numpy(), p


def test_noalloc_matches_workspace_entry_point_twice():
    import torch
    from paper_2512_14681_amd import jf
    assert torch.cuda.is_available()
    L = jf.lib()
    for R, d, V, seed in ((64, 1024, 32768, 11), (17, 512, 4096, 12)):
        g_ref, r_ref, z_ref, p = _run(L, jf, torch, R, d, V, seed, noalloc=False)
        g, r, z, _ = _run(L, jf, torch, R, d, V, seed, noalloc=True)
        assert (g == g_ref).all()
        assert (r == r_ref).all() and r[0] == p and r[2] == g[p - 1]
        assert np.array_equal(z, z_ref)


def test_noalloc_rejects_sizes_beyond_the_scratch():
    import torch
    from paper_2512_14681_amd import jf
    L = jf.lib()
    d = torch.zeros(16, dtype=torch.int32, device="cuda")
    st = jf._stream()
    # 256 rows over a 152064 vocabulary need ~19.5 MB of keys: more than the fixed scratch
    s = L.jf_lm_head_accept_noalloc(256, 3584, 152064, jf.JF_BF16, jf._ptr(d), jf._ptr(d), None, jf._ptr(d),
                                    None, None, st)
    assert s == jf.JF_E_CAPACITY and b"scratch" in L.jf_last_error()
