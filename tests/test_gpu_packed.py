"""GPU parity of the packed noisy/clean forward (jf_packed_forward) against
the oracle (oracle/packed.py), which conditions every row on exactly the
context its mask gives it by plain causal forwards over each chain.

Tolerances as for the step: fp32 logits within 1e-4 of the oracle's fp64
values, bf16 within 2e-2; argmax equal except where the oracle's top-2
gap is below 1e-3.
"""
import numpy as np
import pytest

import jf_inputs
from oracle import packed as opk
from oracle.model import DecoderOracle

pytestmark = pytest.mark.gpu

TINY = jf_inputs.MODEL_SHAPES["tiny"]
MID = dict(n_layers=2, d_model=2048, n_heads=16, n_kv_heads=4, head_dim=128, d_ffn=8192,
           vocab=4096, rope_base=10000.0, rms_eps=1e-6, dtype="bf16")
GAP_EXEMPT = 1e-3


def blocks(seed, N, n, V):
    return [list(jf_inputs.token_ids(seed, i, n, V)) for i in range(N)]


def run(shape, w, prompt, noisy, clean, mask, max_rows=256):
    import torch
    from paper_2512_14681_amd import decode, jf
    model = jf.Model(shape, w, max_rows=max_rows, max_ctx=512)
    dec = decode.Decoder(model)
    dec.prefill(prompt)
    N, n = len(noisy), len(noisy[0])
    R = 2 * N * n
    d_tok = torch.tensor(opk.packed_tokens(noisy, clean), dtype=torch.int32, device="cuda")
    d_arg = torch.zeros(R, dtype=torch.int32, device="cuda")
    d_log = torch.empty((R, shape["vocab"]), dtype=torch.float32, device="cuda")
    model.jf_packed_forward(d_tok, N, n, mask, d_arg, d_log)
    torch.cuda.synchronize()
    return d_arg.cpu().numpy(), d_log.cpu().numpy(), model


def check(z_gpu, g_gpu, z_ref, tol):
    err = np.abs(z_gpu - z_ref).max()
    assert err < tol, err
    top = np.sort(z_ref, axis=1)
    gap = top[:, -1] - top[:, -2]
    ok = (g_gpu == np.argmax(z_ref, axis=1)) | (gap < GAP_EXEMPT)
    assert ok.all(), np.nonzero(~ok)
    return err


@pytest.mark.parametrize("mask", [opk.NOISY_CONTEXT, opk.CLEAN_CONTEXT])
@pytest.mark.parametrize("N,n", [(1, 1), (3, 5), (4, 8), (8, 16)])
def test_packed_tiny(mask, N, n):
    """fp32 tiny decoder: 1 to 8 blocks, ragged 16-row tiles (n = 5), the
    maximum of 256 rows (8 blocks of 16)."""
    w = jf_inputs.model_weights(TINY, seed=0)
    prompt = jf_inputs.prompt(1, 24, TINY["vocab"])
    noisy = blocks(11, N, n, TINY["vocab"])
    clean = blocks(12, N, n, TINY["vocab"])
    g, z, _ = run(TINY, w, prompt, noisy, clean, mask)
    ref = opk.packed_logits(DecoderOracle(TINY, w), prompt, noisy, clean, mask)
    check(z, g, ref, 1e-4)


def test_packed_mid_bf16():
    """bf16 decoder (d 2048), 4 blocks of 16 (128 rows, four 32-row chunks),
    noise-aware mask."""
    w = jf_inputs.model_weights(MID, seed=5)
    prompt = jf_inputs.prompt(6, 40, MID["vocab"])
    noisy = blocks(13, 4, 16, MID["vocab"])
    clean = blocks(14, 4, 16, MID["vocab"])
    g, z, _ = run(MID, w, prompt, noisy, clean, opk.NOISY_CONTEXT, max_rows=128)
    ref = opk.packed_logits(DecoderOracle(MID, w), prompt, noisy, clean, opk.NOISY_CONTEXT)
    check(z, g, ref, 2e-2)


def test_packed_errors_and_no_commit():
    import torch
    from paper_2512_14681_amd import jf
    w = jf_inputs.model_weights(TINY, seed=0)
    model = jf.Model(TINY, w, max_rows=64, max_ctx=256)
    d = torch.zeros(64, dtype=torch.int32, device="cuda")
    g = torch.zeros(64, dtype=torch.int32, device="cuda")
    with pytest.raises(jf.JfError):                       # nothing prefilled
        model.jf_packed_forward(d, 2, 8, 0, g)
    model.jf_prefill(d[:10], g[:1])
    for args in [(2, 8, 2), (0, 8, 0), (2, 0, 0), (3, 11, 0)]:   # bad mask, empty, too many rows
        with pytest.raises(jf.JfError):
            model.jf_packed_forward(d, *args, g)
    model.jf_packed_forward(d, 2, 8, 0, g)
    r = torch.zeros(4, dtype=torch.int32, device="cuda")
    with pytest.raises(jf.JfError):                       # a packed pass is not a step
        model.jf_commit_kv(None, r)
    assert model.jf_kv_length() == 10
