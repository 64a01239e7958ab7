#!/usr/bin/env python3
"""Jacobi-step benchmark on one MI355X.

Workload: one Jacobi iteration (Eq. 3 of Jacobi Forcing, arXiv 2512.14681)
of a Qwen2.5-7B-shaped decoder in bf16 -- 28 layers, d 3584, 28 query / 4
KV heads of 128, SwiGLU FFN 18944, vocab 152064 -- with random-init weights,
a 1024-token random prompt prefilled into the paged KV cache, and a running
window of n = 16 draft rows (Sec. 4.2).  A step is the whole hot path:
forward over the 16 rows against the cache, fused vocabulary argmax, greedy
acceptance with the next draft, and the KV commit.  Inputs are resident in
HBM before timing; the timed loop enqueues steps back to back (the draft and
the committed length stay on the device) and reads the accept counts after.

Prints one JSON line (stdout); progress goes to stderr.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "Jacobi-step latency (µs) + accepted tokens/s, 7B-shaped bf16, n=16..64, 1 GPU"
HBM_PEAK_GBS = 8000.0
COPY_PROBE_BYTES = 256 << 20
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "gemm_gateup_7b_n16_hbm_traffic.md")


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def step_bytes(shape, n, C):
    """Algorithmic HBM bytes of one step: every weight once, the prefix KV
    read, the draft rows' KV written, the embedding rows read."""
    d, F, V = shape["d_model"], shape["d_ffn"], shape["vocab"]
    H, G, hd, L = shape["n_heads"], shape["n_kv_heads"], shape["head_dim"], shape["n_layers"]
    per_layer = ((H + 2 * G) * hd * d + d * H * hd + 2 * F * d + d * F) * 2
    kv_tok = L * 2 * G * hd * 2
    return L * per_layer + V * d * 2 + C * kv_tok + n * kv_tok + n * d * 2


def gateup_bytes(shape, n):
    d, F = shape["d_model"], shape["d_ffn"]
    return 2 * F * d * 2 + n * d * 2 + n * F * 2


def measured_traffic():
    """HBM bytes per gate/up launch from the committed hardware-counter
    summary (FETCH_SIZE + WRITE_SIZE, scaled by a copy kernel's readings),
    or None when the summary is missing or the GEMM sources changed since
    the counters were taken (the summary records their SHA-256)."""
    import hashlib
    try:
        text = open(TRAFFIC_SUMMARY).read()
    except OSError:
        return None
    fields = dict(line[2:].split(": ", 1) for line in text.splitlines()
                  if line.startswith("- ") and ": " in line)
    try:
        for rel, digest in (f.split("=") for f in fields["source_sha256"].split()):
            if hashlib.sha256(open(os.path.join(ROOT, rel), "rb").read()).hexdigest() != digest:
                return None
        return int(fields["hbm_bytes_per_launch"])
    except (KeyError, ValueError, OSError):
        return None


def cpu_baseline(shape, n, C, tpf, budget_s=20.0):
    """The CPU oracle timed on the host on one Jacobi step of the same shape.

    Sample: weights are generated for 2 of the 28 layers (layer l reuses
    layer l % 2's tensors) and the prefix K/V are random bf16 values instead
    of a CPU prefill; the oracle then runs the full 28-layer step over n rows
    against C cached positions in float32 BLAS with the bf16 rounding points.
    Repeated until ~budget_s of CPU time; tokens/s uses the GPU run's TPF.
    """
    import numpy as np
    import threadpoolctl

    import jf_inputs
    from oracle.model import DecoderOracle
    from oracle.numerics import round_bf16

    names = ["embed", "final_norm", "lm_head"] + [f"layers.{l}.{k}" for l in (0, 1) for k in
                                                  ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm",
                                                   "w_gate", "w_up", "w_down")]
    from oracle.numerics import bf16_bits_to_float
    w = jf_inputs.model_weights(shape, seed=0, names=set(names))
    w = {k: bf16_bits_to_float(v, np.float32) for k, v in w.items()}  # once, outside the timing
    for l in range(2, shape["n_layers"]):
        for k in ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down"):
            w[f"layers.{l}.{k}"] = w[f"layers.{l % 2}.{k}"]
    m = DecoderOracle(shape, w, compute=np.float32, row_invariant=False, cache_weights=False)
    G, hd = shape["n_kv_heads"], shape["head_dim"]
    kv = round_bf16(jf_inputs.normal(9, 1, C * G * hd).reshape(C, G, hd))
    m.K = [kv] * shape["n_layers"]
    m.Vc = [kv] * shape["n_layers"]
    toks = jf_inputs.token_ids(9, 2, n, shape["vocab"])
    pos = C + np.arange(n)
    vis = np.tri(n, dtype=bool)
    info = threadpoolctl.threadpool_info()
    threads = max([i.get("num_threads", 1) for i in info] or [1])
    m.forward(toks, pos, vis)  # warm-up (not timed)
    times = []
    t_all = time.perf_counter()
    while time.perf_counter() - t_all < budget_s or not times:
        t0 = time.perf_counter()
        m.forward(toks, pos, vis)
        times.append(time.perf_counter() - t0)
        if len(times) >= 50:
            break
    t = float(np.mean(times))
    return {"value": tpf / t, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": (f"{len(times)} oracle Jacobi steps (28 layers, n={n} rows, {C} cached "
                       f"positions, float32 BLAS with bf16 rounding points) on the host, "
                       f"{t * 1e3:.0f} ms/step; weights of 2 layers reused across depth, random "
                       f"prefix K/V; tokens/s = GPU TPF {tpf:.3f} / oracle step time"),
            "s_per_step": t, "affinity_cores": len(os.sched_getaffinity(0))}



def host_info():
    """CPU model, core counts and the BLAS numpy runs on (threadpoolctl)."""
    import threadpoolctl
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    blas = [{"api": i.get("internal_api"), "library": os.path.basename(i.get("filepath", "")),
             "version": i.get("version"), "threads": i.get("num_threads")}
            for i in threadpoolctl.threadpool_info() if i.get("user_api") == "blas"]
    return {"cpu_model": model, "nproc": os.cpu_count(), "affinity_cores": len(os.sched_getaffinity(0)),
            "blas": blas}


def cpu_oracle_configs(shape7b):
    """The oracle on the other configurations, each a bounded sample timed
    once on the host (a reported baseline, like cpu_baseline):
      config 1: the tiny fp32 decoder's block Jacobi decode (n = 8, 64 tokens);
      config 2: attention at P = 2048, n = 16 and P = 8192, n = 64;
      config 3: the LM head [64, 3584] x [152064, 3584] in fp64, argmax and
                the perturbed-draft acceptance;
      config 5: one 192-row step of the 7B shape after 2048 cached positions
                (weights of 2 layers reused across depth, random prefix K/V).
    """
    import numpy as np

    import jf_inputs
    from oracle import jacobi as ojac
    from oracle.model import DecoderOracle
    from oracle.numerics import bf16_bits_to_float, round_bf16
    out = {}
    # config 1
    tiny = jf_inputs.MODEL_SHAPES["tiny"]
    be = ojac.TransformerBackend(DecoderOracle(tiny, jf_inputs.model_weights(tiny, seed=0)))
    prompt = jf_inputs.prompt(1, 32, tiny["vocab"])
    t0 = time.perf_counter()
    toks, acc = ojac.generate_jacobi(be, prompt, 8, 64, "block", pad_seed=2)
    t = time.perf_counter() - t0
    out["config1_tiny"] = {"sample": "the whole decode (64 tokens, fp64)", "iterations": len(acc),
                           "s": round(t, 3), "us_per_iteration": round(t / len(acc) * 1e6, 1)}
    # config 2
    H, G, hd = 28, 4, 128
    att = {}
    for P, n in ((2048, 16), (8192, 64)):
        S = P + n
        K = bf16_bits_to_float(jf_inputs.normal(20 + P + n, 1, S * G * hd, dtype="bf16")).reshape(S, G, hd)
        Vv = bf16_bits_to_float(jf_inputs.normal(20 + P + n, 2, S * G * hd, dtype="bf16")).reshape(S, G, hd)
        q = bf16_bits_to_float(jf_inputs.normal(20 + P + n, 3, n * H * hd, dtype="bf16")).reshape(n, H, hd)
        m = DecoderOracle(dict(n_layers=1, d_model=H * hd, n_heads=H, n_kv_heads=G, head_dim=hd, d_ffn=128,
                               vocab=16, rope_base=10000.0, rms_eps=1e-6, dtype="f32"), {})
        m.K[0], m.Vc[0] = K[:P], Vv[:P]
        t0 = time.perf_counter()
        m.attention(0, q, K[P:], Vv[P:], np.tri(n, dtype=bool))
        att[f"P{P}_n{n}_us"] = round((time.perf_counter() - t0) * 1e6, 1)
    out["config2_attention"] = dict(att, sample="one call per shape, fp64, vectorised definition")
    # config 3
    R, d, V = 64, 3584, 152064
    w = bf16_bits_to_float(jf_inputs.normal(0, 3000, V * d, std=0.02, dtype="bf16"), np.float32).reshape(V, d)
    x = bf16_bits_to_float(jf_inputs.normal(1000, 1, R * d, dtype="bf16")).reshape(R, d)
    t0 = time.perf_counter()
    z = np.empty((R, V))
    for s0 in range(0, V, 16384):
        z[:, s0:s0 + 16384] = x @ w[s0:s0 + 16384].astype(np.float64).T
    g = np.argmax(z, axis=1)
    draft = np.concatenate([[0], g[:-1]])
    draft[R // 2] = (draft[R // 2] + 1) % V
    ojac.accept_linear(list(draft), list(g))
    t = time.perf_counter() - t0
    out["config3_lm_head_accept"] = {"sample": "one call, fp64 product", "us": round(t * 1e6, 1)}
    del w, z
    # config 5
    names = ["embed", "final_norm", "lm_head"] + [f"layers.{l}.{k}" for l in (0, 1) for k in
                                                  ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm",
                                                   "w_gate", "w_up", "w_down")]
    wts = jf_inputs.model_weights(shape7b, seed=0, names=set(names))
    wts = {k: bf16_bits_to_float(v, np.float32) for k, v in wts.items()}
    C, Rm = 2048, 192
    G7, hd7 = shape7b["n_kv_heads"], shape7b["head_dim"]
    kv = round_bf16(jf_inputs.normal(9, 1, C * G7 * hd7).reshape(C, G7, hd7))
    toks = jf_inputs.token_ids(9, 2, Rm, shape7b["vocab"])
    t_layers = {}
    for nl in (0, 2):          # the step without layers (embedding, final norm, LM head), then 2 layers
        m = DecoderOracle(dict(shape7b, n_layers=nl), wts, compute=np.float32, row_invariant=False,
                          cache_weights=False)
        m.K = [kv] * nl
        m.Vc = [kv] * nl
        t0 = time.perf_counter()
        m.forward(toks, C + np.arange(Rm), np.tri(Rm, dtype=bool))
        t_layers[nl] = time.perf_counter() - t0
    per_layer = (t_layers[2] - t_layers[0]) / 2
    out["config5_step_r192"] = {
        "sample": ("192 rows after 2048 cached positions (float32 BLAS with bf16 rounding points, random "
                   "prefix K/V), timed without layers and with 2 of the 28 layers; the 28-layer step is "
                   "scaled from those"),
        "s_head": round(t_layers[0], 3), "s_per_layer": round(per_layer, 3),
        "s_step_28_layers": round(t_layers[0] + shape7b["n_layers"] * per_layer, 3)}
    return out


def _bits(t):
    """A torch bf16 tensor's bit patterns as int16 (the ABI's bf16 storage)."""
    return t.contiguous().view(__import__("torch").int16)


def _time_calls(fn, iters, stream):
    import torch
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for i in range(iters):
        fn(i)
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / iters * 1e3  # us per call


def bench_attention(sets=32):
    """Attention workload: 28 q / 4 KV heads of 128, N(0,1) bf16 Q/K/V, prefix
    P, n draft queries causal within the block.  Each call reads a different
    one of `sets` buffer sets (> 256 MB in total for P = 8192), so the K/V
    come from HBM as in a decode step, not from the last-level cache."""
    import torch
    from paper_2512_14681_amd import jf
    L = jf.lib()
    H, G, hd = 28, 4, 128
    st = torch.cuda.current_stream()
    g = torch.Generator(device="cuda")
    out = []
    for P in (512, 2048, 8192):
        for n in (16, 32, 64):
            g.manual_seed(10 + P + n)
            keys = P + n
            pages = (keys + 63) // 64
            page_elems = 2 * G * 64 * hd
            kv = torch.randn(sets, pages * page_elems, device="cuda", generator=g).to(torch.bfloat16)
            q = torch.randn(sets, 2, n * H * hd, device="cuda", generator=g).to(torch.bfloat16)
            q[:, 1].zero_()                      # lo plane of a bf16 activation: exact
            pt = torch.arange(pages, dtype=torch.int32, device="cuda")
            Rp = (n + 15) // 16 * 16
            o = torch.empty(2, Rp * H * hd, dtype=torch.int16, device="cuda")
            ws = torch.empty(L.jf_attention_ws_bytes(H, hd, n), dtype=torch.uint8, device="cuda")
            kvb, qb = _bits(kv), _bits(q)

            def call(i):
                jf.check(L.jf_attention(H, G, hd, jf.JF_BF16, P, n, jf._ptr(qb[i % sets]), jf._ptr(kvb[i % sets]),
                                        jf._ptr(pt), None, jf._ptr(o), jf._ptr(ws), jf._stream(st)))
            for i in range(4):
                call(i)
            us = _time_calls(call, 2 * sets, st)
            nbytes = keys * G * hd * 2 * 2 + n * H * hd * 2 + n * H * hd * 4
            flops = 4 * H * hd * (n * P + n * (n + 1) // 2)
            out.append({"P": P, "n": n, "us": round(us, 2), "GB_s": round(nbytes / us / 1e3, 1),
                        "hbm_frac": round(nbytes / us / 1e3 / HBM_PEAK_GBS, 4),
                        "TFLOP_s": round(flops / us / 1e6, 2)})
            del kv, q, kvb, qb
    log("attention: " + ", ".join(f"P{r['P']}/n{r['n']} {r['us']}us" for r in out))
    return {"workload": "attention, 28 q / 4 kv heads x 128, bf16, prefix P + n causal draft rows, "
                        f"{sets} rotating buffer sets", "calls": out}


def bench_lm_head(trials=100):
    """LM head + acceptance: hidden [64, 3584] N(0,1), W [152064, 3584]
    N(0,0.02) bf16; per-row argmax, then the longest prefix with
    draft[i] == argmax[i-1], drafts = the shifted argmax perturbed at one
    random position p per trial (accept must equal p)."""
    import numpy as np
    import torch
    from paper_2512_14681_amd import jf
    L = jf.lib()
    R, d, V = 64, 3584, 152064
    st = torch.cuda.current_stream()
    g = torch.Generator(device="cuda")
    g.manual_seed(1000)
    w = torch.randn(V, d, device="cuda", generator=g).mul_(0.02).to(torch.bfloat16)
    wp = torch.empty(L.jf_packed_matrix_bytes(V, d, jf.JF_BF16), dtype=torch.uint8, device="cuda")
    jf.check(L.jf_pack_matrix(V, d, jf.JF_BF16, jf._ptr(_bits(w)), jf._ptr(wp), jf._stream(st)))
    del w
    x = torch.randn(R, d, device="cuda", generator=g).to(torch.bfloat16)
    # GEMM-input layout of include/jf.h: hi plane = the bf16 values, lo plane = 0
    xl = x.view(torch.int16).reshape(R // 16, 16, d // 128, 4, 4, 8).permute(0, 2, 4, 3, 1, 5).reshape(-1)
    xp = torch.zeros(2, R * d, dtype=torch.int16, device="cuda")
    xp[0].copy_(xl)
    am = torch.zeros(R, dtype=torch.int32, device="cuda")
    res = torch.zeros(trials, 4, dtype=torch.int32, device="cuda")
    ws = torch.empty(L.jf_lm_head_ws_bytes(R, V), dtype=torch.uint8, device="cuda")
    jf.check(L.jf_lm_head_accept(R, d, V, jf.JF_BF16, jf._ptr(xp), jf._ptr(wp), None, jf._ptr(am), None, None,
                                 jf._ptr(ws), jf._stream(st)))
    g0 = am.cpu().numpy()
    rng = np.random.default_rng(1000)
    ps = rng.integers(1, R, trials)
    drafts = np.zeros((trials, R), np.int32)
    for t, pp in enumerate(ps):
        dr = np.concatenate([[5], g0[:-1]]).astype(np.int32)
        dr[pp] = (dr[pp] + 1) % V
        drafts[t] = dr
    d_dr = torch.as_tensor(drafts, device="cuda")

    def call(i):
        jf.check(L.jf_lm_head_accept(R, d, V, jf.JF_BF16, jf._ptr(xp), jf._ptr(wp), jf._ptr(d_dr[i]), jf._ptr(am),
                                     jf._ptr(res[i]), None, jf._ptr(ws), jf._stream(st)))
    us = _time_calls(call, trials, st)
    acc = res[:, 0].cpu().numpy()
    nbytes = V * d * 2 + R * d * 4
    out = {"workload": "LM head + acceptance, hidden [64, 3584], W [152064, 3584] bf16, "
                       f"{trials} trials", "us": round(us, 2), "GB_s": round(nbytes / us / 1e3, 1),
           "hbm_frac": round(nbytes / us / 1e3 / HBM_PEAK_GBS, 4),
           "accept_equals_p": bool((acc == ps).all())}
    log(f"lm head + acceptance: {us:.1f} us, accept == p in all trials: {out['accept_equals_p']}")
    return out


def bench_tiny():
    """Tiny fp32 decoder (2 layers, d 128, vocab 1024): 32-token prompt, block
    Jacobi decoding with n = 8, 64 new tokens (wall clock per iteration,
    including the per-iteration result read)."""
    import jf_inputs
    from paper_2512_14681_amd import decode, jf
    shape = jf_inputs.MODEL_SHAPES["tiny"]
    model = jf.Model(shape, jf_inputs.model_weights(shape, seed=0), max_rows=16, max_ctx=128)
    dec = decode.Decoder(model)
    prompt = jf_inputs.prompt(1, 32, shape["vocab"])
    dec.generate_jacobi(prompt, 8, 64, mode="block", pad_seed=2)      # warm-up
    dec.reset()
    t0 = time.perf_counter()
    toks, acc = dec.generate_jacobi(prompt, 8, 64, mode="block", pad_seed=2)
    t = time.perf_counter() - t0
    out = {"workload": "tiny fp32 decoder, block Jacobi n=8, 64 new tokens", "iterations": len(acc),
           "tpf": round(len(toks) / len(acc), 3), "us_per_iteration_wall": round(t / len(acc) * 1e6, 1)}
    log(f"tiny: {out}")
    return out


def bench_window(model, dec, shape, n, prompt_len=1024, steps=10, warmup=3):
    import torch
    from paper_2512_14681_amd import decode, jf
    import jf_inputs
    V = shape["vocab"]
    dec.reset()
    p = dec.prefill(jf_inputs.prompt(1, prompt_len, V))
    d_draft = torch.tensor([p] + [decode.pad_token(2, prompt_len + i, V) for i in range(1, n)],
                           dtype=torch.int32, device="cuda")
    d_arg = torch.zeros(n, dtype=torch.int32, device="cuda")
    d_res = torch.zeros((warmup + steps, 4), dtype=torch.int32, device="cuda")
    st = torch.cuda.current_stream()

    def step(i):  # window step with its commit (one fused argmax / acceptance / commit launch)
        model.jf_jacobi_step(d_draft, n, 1 | jf.JF_STEP_COMMIT, 2, d_arg, d_res[i], d_draft)
    for i in range(warmup):
        step(i)
    us = _time_calls(lambda i: step(warmup + i), steps, st)
    acc = d_res[warmup:, 0].cpu().numpy()
    sb = step_bytes(shape, n, prompt_len + int(acc.sum()) // 2)
    out = {"workload": f"7B-shaped decoder, Jacobi step n={n} running window, 1024-token prefix",
           "step_us": round(us, 1), "tpf": round(float(acc.mean()), 4),
           "tokens_s": round(float(acc.mean()) / us * 1e6, 2),
           "step_hbm_frac": round(sb / us / 1e3 / HBM_PEAK_GBS, 4)}
    log(f"n={n}: {out}")
    return out


def bench_decode(model, dec, shape, n, new_tokens=256, prompt_len=1024):
    """Greedy Jacobi decoding, running window of n, 256 new tokens after a
    1024-token prompt: wall clock per iteration (prefill subtracted),
    including the host loop and its per-iteration result read."""
    import torch
    import jf_inputs
    V = shape["vocab"]
    prompt = jf_inputs.prompt(1, prompt_len, V)
    dec.reset()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    dec.prefill(prompt)
    t_prefill = time.perf_counter() - t0
    dec.reset()
    t0 = time.perf_counter()
    toks, acc = dec.generate_jacobi(prompt, n, new_tokens, mode="window", pad_seed=2)
    t = time.perf_counter() - t0 - t_prefill
    out = {"workload": f"7B-shaped decoder, greedy Jacobi decoding, n={n} running window, {new_tokens} new "
                       f"tokens after a {prompt_len}-token prompt",
           "new_tokens": len(toks), "iterations": len(acc), "tpf": round(len(toks) / len(acc), 3),
           "ms_per_iteration_wall": round(t / len(acc) * 1e3, 3), "tokens_s_wall": round(len(toks) / t, 1)}
    log(f"decode n={n}: {out}")
    return out


def bench_multiblock(model, dec, shape, prefix=2048, new_tokens=256, reps=10):
    """Multi-block decoding with rejection recycling (K = 4 blocks of n = 16,
    r = 0.85, up to 8 recycled 16-token candidates) after a 2048-token
    prompt; and the largest step of that configuration, R = 192 rows (the
    real-active draft, 3 pseudo-active blocks, 8 candidates) under the tree
    mask, timed without committing."""
    import numpy as np
    import torch
    import jf_inputs
    from paper_2512_14681_amd import decode, jf
    V = shape["vocab"]
    prompt = jf_inputs.prompt(3, prefix, V)
    dec.reset()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    dec.prefill(prompt)
    t_prefill = time.perf_counter() - t0
    dec.reset()
    t0 = time.perf_counter()
    toks, trace = dec.generate_multiblock(prompt, 16, 4, 0.85, new_tokens, n_cand=8, cand_len=16)
    t = time.perf_counter() - t0 - t_prefill
    Rs = [tr["R"] for tr in trace]
    natural = {"new_tokens": len(toks), "iterations": len(trace), "tpf": round(len(toks) / len(trace), 3),
               "rows_per_step_mean": round(float(np.mean(Rs)), 1), "rows_per_step_max": int(max(Rs)),
               "ms_per_iteration_wall": round(t / len(trace) * 1e3, 3),
               "note": "wall clock per iteration (prefill subtracted), incl. the host-side policy "
                       "and the per-iteration result read"}
    # the largest step shape, timed on the device
    dec.reset()
    p = dec.prefill(prompt)
    n, R = 16, 192
    segs = [(0, n, -1, jf.JF_ROLE_RA, 1)]
    for b in range(1, 4):
        segs.append((b * n, n, b * n - 1, jf.JF_ROLE_PSEUDO, 0))
    for c in range(8):
        segs.append((64 + c * n, n, 0, jf.JF_ROLE_CAND, 0))
    rng = np.random.default_rng(5)
    tokens = [p] + [int(t) for t in rng.integers(0, V, R - 1)]
    d_tok = torch.tensor(tokens, dtype=torch.int32, device="cuda")
    d_arg = torch.zeros(R, dtype=torch.int32, device="cuda")
    d_seg = torch.zeros(jf.JF_MAX_SEGMENTS, dtype=torch.int32, device="cuda")
    d_res = torch.zeros(4, dtype=torch.int32, device="cuda")
    d_path = torch.zeros(R, dtype=torch.int32, device="cuda")
    st = torch.cuda.current_stream()
    call = lambda i: model.jf_multiblock_step(d_tok, R, segs, d_arg, d_seg, d_res, d_path)
    for i in range(3):
        call(i)
    us = _time_calls(call, reps, st)
    d, F, H, G, hd, Lr = (shape[k] for k in ("d_model", "d_ffn", "n_heads", "n_kv_heads", "head_dim", "n_layers"))
    params = Lr * ((H + 2 * G) * hd * d + d * H * hd + 3 * F * d) + V * d
    flops = 2 * params * R + Lr * 4 * R * (prefix + R) * hd * H
    sb = step_bytes(shape, R, prefix)
    step = {"rows": R, "step_us": round(us, 1), "mfma_frac_bf16": round(flops / us / 1e6 / 2.5e3, 4),
            "step_hbm_frac": round(sb / us / 1e3 / HBM_PEAK_GBS, 4), "tflop_s": round(flops / us / 1e6, 1)}
    out = {"workload": "7B-shaped decoder, multi-block K=4 x n=16 + up to 8 recycled candidates, "
                       "2048-token prefix", "decode": natural, "largest_step": step}
    log(f"multi-block: {out}")
    return out

def bench_trajectory_select(n=16, sel_blocks=1 << 18, w=16, copies=4, reps=20):
    """Noise-schedule point selection (Eq. 7, App. C) over 2^18 synthetic
    16-token trajectories (up to 17 points each), timed over `copies`
    rotating device copies so that no launch finds its input in the 256 MB
    last-level cache.  Algorithmic bytes: every valid point once (L_b n 4
    bytes per block) + the length read + the selection write (8 bytes per
    block)."""
    import numpy as np
    import torch
    import jf_inputs
    from paper_2512_14681_amd import jf
    t1 = time.time()
    traj, lens = jf_inputs.trajectories(5, sel_blocks, n, 152064)
    log(f"trajectory inputs: {time.time() - t1:.1f}s")
    P = traj.shape[1]
    d_src = torch.as_tensor(traj, device="cuda")
    bufs = [d_src] + [d_src.clone() for _ in range(copies - 1)]
    d_len = torch.as_tensor(lens, device="cuda")
    d_sel = torch.zeros(sel_blocks, dtype=torch.int32, device="cuda")
    st = torch.cuda.current_stream()
    call = lambda i: jf.trajectory_select(bufs[i % copies], d_len, sel_blocks, n, P, w, d_sel)
    for i in range(copies):
        call(i)
    us = _time_calls(call, reps, st)
    nbytes = int(lens.astype(np.int64).sum()) * n * 4 + 8 * sel_blocks
    gbs = nbytes / us / 1e3
    out = {"workload": f"noise-schedule point selection, {sel_blocks} trajectories of {n}-token blocks "
                       f"(up to {P} points), w={w}", "blocks": sel_blocks, "n": n, "w": w, "max_points": P,
           "mean_points": round(float(lens.mean()), 2), "us": round(us, 2), "bytes_per_launch": nbytes,
           "GB_s": round(gbs, 1), "hbm_frac": round(gbs / HBM_PEAK_GBS, 4)}
    log(f"trajectory select: {out}")
    return out


def bench_trajectory(model, dec, shape, prefix=1024, n=16, blocks=2):
    """Trajectory collection (Sec. 2.1) on the 7B-shaped decoder: block-mode
    decoding of `blocks` blocks of n = 16 after a 1024-token prompt with every
    iterate recorded on the device; and the point selection."""
    import torch
    import jf_inputs
    from paper_2512_14681_amd import jf
    V = shape["vocab"]
    prompt = jf_inputs.prompt(1, prefix, V)
    dec.reset()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    dec.prefill(prompt)
    t_prefill = time.perf_counter() - t0
    dec.reset()
    t0 = time.perf_counter()
    d_traj, lengths = dec.collect_trajectories(prompt, n, blocks)
    torch.cuda.synchronize()
    t = time.perf_counter() - t0 - t_prefill
    iters = int((lengths - 1).sum())
    st = torch.cuda.current_stream()
    d_a, d_b = torch.zeros(n, dtype=torch.int32, device="cuda"), torch.zeros(n, dtype=torch.int32, device="cuda")
    rec_us = _time_calls(lambda i: jf.trajectory_record(d_a, d_b, n, n - (i % n), d_a), 200, st)
    collect = {"blocks": blocks, "n": n, "iterations": iters, "points_recorded": int(lengths.sum()),
               "ms_per_iteration_wall": round(t / iters * 1e3, 3), "record_call_us": round(rec_us, 2),
               "note": "wall clock per iteration (prefill subtracted): step + record + commit + the "
                       "per-iteration result read; record_call_us is back-to-back calls (host-bound)"}
    out = {"workload": "trajectory collection: 7B-shaped decoder, block Jacobi n=16 after a 1024-token "
                       "prefix, every iterate recorded; point selection over 2^18 synthetic 16-token "
                       "trajectories (Eq. 7, w=16)", "collect": collect, "select": bench_trajectory_select()}
    log(f"trajectory: {out}")
    return out


def bench_packed(model, dec, shape, prefix=1024, N=8, n=16, reps=10):
    """Forward over a packed training sequence (Sec. 3.1 noise-aware causal
    attention, App. C packing): N = 8 noisy + 8 clean blocks of n = 16
    (R = 256 rows) after a 1024-token prompt, noise-aware mask; next to the
    cost of the 2N separate n-row causal forwards the packing replaces."""
    import torch
    import jf_inputs
    from paper_2512_14681_amd import jf
    V = shape["vocab"]
    dec.reset()
    dec.prefill(jf_inputs.prompt(1, prefix, V))
    R = 2 * N * n
    d_tok = torch.as_tensor(jf_inputs.token_ids(8, 1, R, V), device="cuda")
    d_arg = torch.zeros(R, dtype=torch.int32, device="cuda")
    st = torch.cuda.current_stream()
    call = lambda i: model.jf_packed_forward(d_tok, N, n, jf.JF_MASK_NOISY_CONTEXT, d_arg)
    for i in range(2):
        call(i)
    us = _time_calls(call, reps, st)
    d_res = torch.zeros(4, dtype=torch.int32, device="cuda")
    one = lambda i: model.jf_jacobi_step(d_tok, n, 0, 2, d_arg, d_res, d_arg)
    for i in range(2):
        one(i)
    us_n = _time_calls(one, reps, st)
    d, F, H, G, hd, Lr = (shape[k] for k in ("d_model", "d_ffn", "n_heads", "n_kv_heads", "head_dim", "n_layers"))
    params = Lr * ((H + 2 * G) * hd * d + d * H * hd + 3 * F * d) + V * d
    flops = 2 * params * R + Lr * 4 * R * (prefix + N * n) * hd * H
    out = {"workload": f"packed noisy/clean forward, 7B-shaped decoder, {N}+{N} blocks of {n} "
                       f"(R={R}) after a {prefix}-token prompt, noise-aware mask",
           "us": round(us, 1), "rows_per_s": round(R / us * 1e6, 1),
           "mfma_frac_bf16": round(flops / us / 1e6 / 2.5e3, 4), "tflop_s": round(flops / us / 1e6, 1),
           "separate_forwards_us": round(2 * N * us_n, 1),
           "note": f"separate_forwards_us = 2N x one {n}-row step ({us_n:.1f} us), the unpacked cost"}
    log(f"packed: {out}")
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--n", type=int, default=16)
    ap.add_argument("--prompt", type=int, default=1024)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-kernel-profile", action="store_true",
                    help="skip the per-kernel event pass (for hardware-counter runs)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="first copy 256 MiB device-to-device 3 times (counter calibration)")
    ap.add_argument("--only", choices=["trajectory_select", "attention", "lm_head"],
                    help="run one component workload alone and print its JSON object")
    ap.add_argument("--headline-only", action="store_true",
                    help="skip the other workloads (configs 1, 2, 3, 4 at n=32 and 64, 5)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: the Jacobi step runs on a single MI355X and the "
              "library has no multi-GPU path (--gpus must be 1)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import jf_inputs
    from paper_2512_14681_amd import decode, jf

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.copy_probe:
        # A plain copy kernel of known size: its FETCH_SIZE / WRITE_SIZE
        # readings give the scale from counter units to HBM bytes.
        a = torch.ones(COPY_PROBE_BYTES // 4, dtype=torch.float32, device="cuda")
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        del a, b
        log(f"copy probe: 3 x {COPY_PROBE_BYTES} bytes")
    if args.only == "trajectory_select":
        print(json.dumps(bench_trajectory_select()), flush=True)
        return
    if args.only == "attention":
        print(json.dumps(bench_attention()), flush=True)
        return
    if args.only == "lm_head":
        print(json.dumps(bench_lm_head()), flush=True)
        return
    shape = jf_inputs.MODEL_SHAPES["7b"]
    n, K, W = args.n, args.steps, args.warmup
    t0 = time.time()
    w = jf_inputs.model_weights(shape, seed=0)
    log(f"weights generated in {time.time() - t0:.1f}s")
    max_ctx = ((max(args.prompt + n * (W + 2 * K + 4), 2048 + 64 + 256 + 256) + 63) // 64) * 64
    model = jf.Model(shape, w, max_rows=256, max_ctx=max_ctx)
    del w
    log(f"model loaded ({time.time() - t0:.1f}s)")
    dec = decode.Decoder(model)
    prompt = jf_inputs.prompt(1, args.prompt, shape["vocab"])
    torch.cuda.synchronize()
    t1 = time.time()
    p = dec.prefill(prompt)
    log(f"prefill of {args.prompt} tokens: {time.time() - t1:.3f}s")

    V = shape["vocab"]
    seed = 2
    d_draft = torch.tensor([p] + [decode.pad_token(seed, args.prompt + i, V) for i in range(1, n)],
                           dtype=torch.int32, device="cuda")
    d_argmax = torch.zeros(n, dtype=torch.int32, device="cuda")
    total = W + 2 * K
    d_res = torch.zeros((total, 4), dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()

    def step(i):  # window step with its commit (one fused argmax / acceptance / commit launch)
        model.jf_jacobi_step(d_draft, n, 1 | jf.JF_STEP_COMMIT, seed, d_argmax, d_res[i], d_draft)

    for i in range(W):
        step(i)
    torch.cuda.synchronize()
    C0 = model.jf_kv_length()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(K + 1)]
    ev[0].record(stream)
    for i in range(W, W + K):
        step(i)
        ev[i - W + 1].record(stream)
    torch.cuda.synchronize()
    ms = ev[0].elapsed_time(ev[K])
    per_step_us = np.array([ev[i].elapsed_time(ev[i + 1]) for i in range(K)]) * 1e3
    res = d_res.cpu().numpy()
    acc = res[W:W + K, 0]
    assert (acc >= 1).all() and (res[W:W + K, 3] == 0).all(), res[W:W + K]
    ms_step = ms / K
    tpf = float(acc.mean())
    tok_s = float(acc.sum()) / (ms / 1e3)
    log(f"timed {K} steps: {ms_step * 1e3:.1f} us/step, TPF {tpf:.3f}, {tok_s:.1f} tokens/s")

    # Per-kernel durations from HIP events on the library's stream, over a
    # second run of K steps (events around every launch of one class).
    kern = {}
    classes = () if args.no_kernel_profile else (
        (jf.JF_KERNEL_GATEUP, "gateup"), (jf.JF_KERNEL_DOWN, "down"), (jf.JF_KERNEL_QKV, "qkv"),
        (jf.JF_KERNEL_O, "o"), (jf.JF_KERNEL_ATTN, "attn"), (jf.JF_KERNEL_ATTN_BLOCK, "attn_block"),
        (jf.JF_KERNEL_LMHEAD, "lmhead"))
    for cls, name in classes:
        model.jf_profile_begin(cls)
        for i in range(K // 2):
            step(W + K + (i % K))
        t, cnt = model.jf_profile_end()
        if cnt:          # a class the step does not launch (fused away) records nothing
            kern[name] = dict(avg_us=t / cnt * 1e3, launches=cnt)
        model.jf_kv_truncate(C0 + int(acc.sum()))
    if not kern:
        log("per-kernel pass skipped; no roofline object")
        return
    log("kernel averages (us): " + ", ".join(f"{k} {v['avg_us']:.1f}" for k, v in kern.items()))
    C_mid = C0 + int(acc.sum()) // 2
    gu = gateup_bytes(shape, n)
    avg_s = kern["gateup"]["avg_us"] / 1e6
    achieved = gu / avg_s / 1e9
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": measured_traffic(),
                "kernel": "k_gemm gate/up projection + SwiGLU (28 launches per step)",
                "bytes_per_launch": gu, "avg_us": round(kern["gateup"]["avg_us"], 2)}
    sb = step_bytes(shape, n, C_mid)
    out = {
        "metric": METRIC, "value": round(tok_s, 2), "unit": "tokens/s", "n_gpus": 1,
        "steps": K, "warmup": W, "ms_per_step": round(ms_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (random-init weights N(0,0.02), uniform random prompt)",
        "config": {"workload": "7B-shaped decoder, one Jacobi step: n=16 running window, "
                               "1024-token prefix, bf16, greedy acceptance + KV commit",
                   "n": n, "prefix": args.prompt, "layers": shape["n_layers"],
                   "d_model": shape["d_model"], "vocab": shape["vocab"]},
        "step_us": round(ms_step * 1e3, 1), "tpf": round(tpf, 4),
        "step_us_p10_p50_p90": [round(float(np.percentile(per_step_us, q)), 1) for q in (10, 50, 90)],
        "step_hbm_bytes": sb, "step_hbm_frac": round(sb / (ms_step / 1e3) / (HBM_PEAK_GBS * 1e9), 4),
        "kernels_us": {k: round(v["avg_us"], 2) for k, v in kern.items()},
        "roofline": roofline,
    }
    if not args.headline_only:
        others = {}
        others["config4_n32"] = bench_window(model, dec, shape, 32)
        others["config4_n64"] = bench_window(model, dec, shape, 64)
        others["config4_decode_n16"] = bench_decode(model, dec, shape, 16)
        others["config4_decode_n32"] = bench_decode(model, dec, shape, 32)
        others["config5_multiblock"] = bench_multiblock(model, dec, shape)
        others["next2_trajectory"] = bench_trajectory(model, dec, shape)
        others["next3_packed"] = bench_packed(model, dec, shape)
        del model, dec
        torch.cuda.empty_cache()
        others["config2_attention"] = bench_attention()
        others["config3_lm_head_accept"] = bench_lm_head()
        others["config1_tiny"] = bench_tiny()
        out["other_workloads"] = others
    if not args.no_cpu_baseline:
        t2 = time.time()
        out["cpu_baseline"] = cpu_baseline(shape, n, args.prompt, tpf)
        out["cpu_baseline"]["host"] = host_info()
        log(f"cpu baseline: {out['cpu_baseline']['s_per_step']:.2f} s/step ({time.time() - t2:.0f}s)")
        if not args.headline_only:
            t2 = time.time()
            out["cpu_baseline"]["other_configs"] = cpu_oracle_configs(shape)
            log(f"cpu oracle on configs 1, 2, 3, 5: {out['cpu_baseline']['other_configs']} "
                f"({time.time() - t2:.0f}s)")
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
