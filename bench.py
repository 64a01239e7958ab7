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
        (jf.JF_KERNEL_O, "o"), (jf.JF_KERNEL_ATTN, "attn"), (jf.JF_KERNEL_LMHEAD, "lmhead"))
    for cls, name in classes:
        model.jf_profile_begin(cls)
        for i in range(K // 2):
            step(W + K + (i % K))
        t, cnt = model.jf_profile_end()
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
    if not args.no_cpu_baseline:
        t2 = time.time()
        out["cpu_baseline"] = cpu_baseline(shape, n, args.prompt, tpf)
        log(f"cpu baseline: {out['cpu_baseline']['s_per_step']:.2f} s/step ({time.time() - t2:.0f}s)")
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
