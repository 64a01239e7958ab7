"""Latency of one Jacobi iteration against the number of parallel rows, and
decoding speed at a fixed number of accepted tokens per iteration.

    python -m paper_2512_14681_amd.sweep [--prefix 1024] [--rows 1,2,4,...]

On the 7B-shaped bf16 decoder (random-init weights, a random prompt):

* linear steps of R draft rows (one causal block, Eq. 3) and tree steps of
  R = 16 + 16 c rows (the real-active draft plus c recycled 16-token
  candidates under its root, the verification pass of App. A Alg. 1), each
  timed on the device without committing (the prefix stays fixed): the
  paper's per-iteration cost against parallel tokens (App. D, Fig. 4a), and
  the knee where the step stops being bound by streaming the weights;
* fixed fast-forward emulation (the methodology behind the paper's
  speedup-at-fixed-TPF profiling): the model's own greedy continuation is
  decoded first with one-row steps; then a block of n = 16 is decoded with
  drafts that hold the next k - 1 greedy tokens followed by a wrong one, so
  each iteration accepts k tokens.  Tokens/s at each k are reported next to
  the one-row (autoregressive) rate.

* with --packed, the packed noisy/clean forward (8 + 8 blocks of 16 after
  the prefix, noise-aware mask; App. C packing);

* with --grid, the configuration grid of App. E on latency only: block size
  n x verification size v (entries verified in parallel, each n tokens) x
  concurrent blocks K; one step holds the real-active draft, v - 1 recycled
  n-token entries under its root and K - 1 chained pseudo-active blocks,
  R = (v + K - 1) n rows.  Points beyond the engine's 512 rows are reported
  as such.  Tokens/s needs the TPF of trained weights and is not reported.

Prints one JSON object (stdout); progress on stderr.
"""
from __future__ import annotations

import argparse
import json
import sys
import time


def log(*a):
    print("[sweep]", *a, file=sys.stderr, flush=True)


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--prefix", type=int, default=1024)
    ap.add_argument("--rows", default="1,2,4,8,16,24,32,48,64,96,128,160,192,224,256")
    ap.add_argument("--cands", default="0,1,2,4,6,8,10,12,15")
    ap.add_argument("--k", default="1,2,3,4,5,8", help="accepted tokens per iteration ('' : no emulation)")
    ap.add_argument("--reps", type=int, default=10)
    ap.add_argument("--grid", action="store_true", help="the (n, verification size, K) grid")
    ap.add_argument("--packed", action="store_true", help="also time the packed noisy/clean forward")
    ap.add_argument("--grid-n", default="8,16,32,64,128")
    ap.add_argument("--grid-v", default="1,2,4,8,12")
    ap.add_argument("--grid-k", default="2", help="concurrent blocks K of the grid")
    args = ap.parse_args(argv)

    import numpy as np
    import torch

    import jf_inputs
    from paper_2512_14681_amd import decode, jf

    assert torch.cuda.is_available(), "the sweep needs a GPU"
    shape = jf_inputs.MODEL_SHAPES["7b"]
    V, P = shape["vocab"], args.prefix
    rows = [int(r) for r in args.rows.split(",")]
    t0 = time.time()
    model = jf.Model(shape, jf_inputs.model_weights(shape, seed=0), max_rows=jf.JF_MAX_ROWS,
                     max_ctx=((P + 512 + 63) // 64) * 64)
    dec = decode.Decoder(model)
    prompt = jf_inputs.prompt(1, P, V)
    p = dec.prefill(prompt)
    log(f"model ready ({time.time() - t0:.0f}s)")
    st = torch.cuda.current_stream()
    Rmax = jf.JF_MAX_ROWS
    d_tok = torch.tensor([p] + [decode.pad_token(2, P + i, V) for i in range(1, Rmax)], dtype=torch.int32,
                         device="cuda")
    d_arg = torch.zeros(Rmax, dtype=torch.int32, device="cuda")
    d_res = torch.zeros(4, dtype=torch.int32, device="cuda")
    d_nxt = torch.zeros(Rmax, dtype=torch.int32, device="cuda")
    d_seg = torch.zeros(jf.JF_MAX_SEGMENTS, dtype=torch.int32, device="cuda")
    d_path = torch.zeros(Rmax, dtype=torch.int32, device="cuda")

    def timed(call, reps):
        for _ in range(3):
            call()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(st)
        for _ in range(reps):
            call()
        e1.record(st)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps * 1e3

    d, F, H, G, hd, L = (shape[k] for k in ("d_model", "d_ffn", "n_heads", "n_kv_heads", "head_dim",
                                            "n_layers"))
    params = L * ((H + 2 * G) * hd * d + d * H * hd + 3 * F * d) + V * d
    weight_bytes = 2 * params
    kv_tok = L * 2 * G * hd * 2

    def costs(R, us):
        nbytes = weight_bytes + (P + R) * kv_tok + R * d * 2
        flops = 2 * params * R + L * 4 * R * (P + R) * hd * H
        return {"rows": R, "us": round(us, 1), "hbm_frac": round(nbytes / us / 1e3 / 8000.0, 4),
                "mfma_frac_bf16": round(flops / us / 1e6 / 2.5e3, 4)}

    linear = []
    for R in rows:
        us = timed(lambda: model.jf_jacobi_step(d_tok, R, 1, 2, d_arg, d_res, d_nxt), args.reps)
        linear.append(costs(R, us))
        log(f"linear R={R}: {us:.1f} us")
    tree = []
    for c in (int(x) for x in args.cands.split(",")):
        R = 16 + 16 * c
        segs = [(0, 16, -1, jf.JF_ROLE_RA, 1)] + [(16 + 16 * i, 16, 0, jf.JF_ROLE_CAND, 0) for i in range(c)]
        us = timed(lambda: model.jf_multiblock_step(d_tok, R, segs, d_arg, d_seg, d_res, d_path), args.reps)
        tree.append(dict(costs(R, us), candidates=c))
        log(f"tree R={R}: {us:.1f} us")

    grid = []
    if args.grid:
        for K in (int(x) for x in args.grid_k.split(",")):
            for n_ in (int(x) for x in args.grid_n.split(",")):
                for v in (int(x) for x in args.grid_v.split(",")):
                    R = (v + K - 1) * n_
                    if R > Rmax:
                        grid.append({"n": n_, "v": v, "K": K, "rows": R, "us": None,
                                     "note": f"exceeds {Rmax} rows"})
                        continue
                    segs = [(0, n_, -1, jf.JF_ROLE_RA, 1)]
                    for c in range(v - 1):
                        segs.append((n_ * (1 + c), n_, 0, jf.JF_ROLE_CAND, 0))
                    for b in range(K - 1):                   # pseudo-active blocks, chained
                        first = n_ * (v + b)
                        segs.append((first, n_, n_ - 1 if b == 0 else first - 1, jf.JF_ROLE_PSEUDO, 0))
                    if len(segs) > jf.JF_MAX_SEGMENTS:
                        grid.append({"n": n_, "v": v, "K": K, "rows": R, "us": None,
                                     "note": f"more than {jf.JF_MAX_SEGMENTS} segments"})
                        continue
                    us = timed(lambda: model.jf_multiblock_step(d_tok, R, segs, d_arg, d_seg, d_res, d_path),
                               args.reps)
                    grid.append(dict(costs(R, us), n=n_, v=v, K=K))
                    log(f"grid K={K} n={n_} v={v} R={R}: {us:.1f} us")

    packed = []
    if args.packed:
        # the packed noisy/clean forward (App. C packing, noise-aware mask): 8 +
        # 8 blocks of 16 after the prefix, as bench.py's packed workload
        d_pk = torch.as_tensor(jf_inputs.token_ids(8, 1, 256, V), device="cuda")
        us = timed(lambda: model.jf_packed_forward(d_pk, 8, 16, jf.JF_MASK_NOISY_CONTEXT, d_arg), args.reps)
        packed.append(dict(costs(256, us), blocks=8, n=16))
        log(f"packed R=256: {us:.1f} us")

    # fixed fast-forward emulation (none with --k '')
    ks = [int(k) for k in args.k.split(",") if k]
    n, iters = 16, 12
    fixed = []
    C0 = None
    if ks:
        dec.reset()
        ar = dec.generate_ar(prompt, max(ks) * iters + 1)   # one-row steps: the greedy continuation
        C0 = model.jf_kv_length()
    for k in ks:
        dec.reset()
        dec.prefill(prompt)
        drafts = np.zeros((iters, n), np.int32)
        for j in range(iters):
            base = j * k
            row = [ar[base + i] for i in range(k)]
            wrong = (ar[base + k] + 1) % V if base + k < len(ar) else 0
            row += [wrong] + [decode.pad_token(2, P + base + k + 1 + i, V) for i in range(n - k - 1)]
            drafts[j] = row[:n]
        d_dr = torch.as_tensor(drafts, device="cuda")
        d_r = torch.zeros((iters, 4), dtype=torch.int32, device="cuda")
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(st)
        for j in range(iters):
            model.jf_jacobi_step(d_dr[j], n, 0, 2, d_arg, d_r[j], d_nxt)
            model.jf_commit_kv(None, d_r[j])
        e1.record(st)
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) / iters * 1e3
        acc = d_r[:, 0].cpu().numpy()
        fixed.append({"k": k, "tpf_measured": round(float(acc.mean()), 3), "step_us": round(us, 1),
                      "tokens_s": round(float(acc.sum()) / (us * iters) * 1e6, 1)})
        log(f"fixed k={k}: accepts {acc.tolist()}, {us:.1f} us/iteration")
    ar_us = next((r["us"] for r in linear if r["rows"] == 1), None)
    if ar_us:
        for f in fixed:
            f["speedup_vs_one_row_steps"] = round(f["tokens_s"] / (1e6 / ar_us), 3)
    out = {"workload": f"7B-shaped bf16 decoder, {P}-token prefix, random-init weights",
           "linear": linear, "tree": tree, "packed": packed, "fixed_tpf_block16": fixed, "config_grid": grid,
           "note": f"one-row step {ar_us} us; C0 after greedy continuation {C0}"}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
