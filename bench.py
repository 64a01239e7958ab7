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


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--n", type=int, default=16)
    ap.add_argument("--prompt", type=int, default=1024)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: the Jacobi step runs on a single MI355X and this "
              "build has no multi-GPU path (--gpus must be 1)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import jf_inputs
    from paper_2512_14681_amd import decode, jf

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    shape = jf_inputs.MODEL_SHAPES["7b"]
    n, K, W = args.n, args.steps, args.warmup
    t0 = time.time()
    w = jf_inputs.model_weights(shape, seed=0)
    log(f"weights generated in {time.time() - t0:.1f}s")
    max_ctx = ((args.prompt + n * (W + 2 * K + 4) + 63) // 64) * 64
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

    def step(i):
        model.jf_jacobi_step(d_draft, n, 1, seed, d_argmax, d_res[i], d_draft)
        model.jf_commit_kv(None, d_res[i])

    for i in range(W):
        step(i)
    torch.cuda.synchronize()
    C0 = model.jf_kv_length()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for i in range(W, W + K):
        step(i)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
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
    for cls, name in ((jf.JF_KERNEL_GATEUP, "gateup"), (jf.JF_KERNEL_DOWN, "down"),
                      (jf.JF_KERNEL_QKV, "qkv"), (jf.JF_KERNEL_O, "o"),
                      (jf.JF_KERNEL_ATTN, "attn"), (jf.JF_KERNEL_LMHEAD, "lmhead")):
        model.jf_profile_begin(cls)
        for i in range(K // 2):
            step(W + K + (i % K))
        t, cnt = model.jf_profile_end()
        kern[name] = dict(avg_us=t / cnt * 1e3, launches=cnt)
        model.jf_kv_truncate(C0 + int(acc.sum()))
    log("kernel averages (us): " + ", ".join(f"{k} {v['avg_us']:.1f}" for k, v in kern.items()))
    C_mid = C0 + int(acc.sum()) // 2
    gu = gateup_bytes(shape, n)
    avg_s = kern["gateup"]["avg_us"] / 1e6
    achieved = gu / avg_s / 1e9
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
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
        "step_hbm_bytes": sb, "step_hbm_frac": round(sb / (ms_step / 1e3) / (HBM_PEAK_GBS * 1e9), 4),
        "kernels_us": {k: round(v["avg_us"], 2) for k, v in kern.items()},
        "roofline": roofline,
    }
    if not args.no_cpu_baseline:
        t2 = time.time()
        out["cpu_baseline"] = cpu_baseline(shape, n, args.prompt, tpf)
        log(f"cpu baseline: {out['cpu_baseline']['s_per_step']:.2f} s/step ({time.time() - t2:.0f}s)")
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
