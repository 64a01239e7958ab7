"""Summaries of rocprofv3 CSV output for libjf runs (``rocprofv3 -f csv``).

    python -m paper_2512_14681_amd.profiling stats DIR
        kernel-time table from DIR's *_kernel_stats.csv (``--kernel-trace --stats``)

    python -m paper_2512_14681_amd.profiling traffic --fetch DIR1 --write DIR2 \
        --kernel REGEX --copy-bytes N
        HBM bytes per dispatch of the kernels matching REGEX from a FETCH_SIZE
        run (DIR1) and a WRITE_SIZE run (DIR2).  Both counters read in KiB per
        dispatch and are scaled by what they read for the first three dispatches
        whose name contains "copy" (a plain device copy of N bytes that the
        profiled program runs first, e.g. ``bench.py --copy-probe``).

    python -m paper_2512_14681_amd.profiling step-mfma DIR --rows R --ctx C [--select REGEX]
        MFMA load of every phase of the forwards in a --pmc run of
        SQ_INSTS_VALU_MFMA_MOPS_BF16, SQ_VALU_MFMA_BUSY_CYCLES and
        GRBM_GUI_ACTIVE (one pass): issued bf16 flops, the matrix cores' busy
        fraction, and the algorithmic flops of R rows at committed length C;
        forwards are kept when one of their kernels matches REGEX
        (default accept: the Jacobi steps; k_tree_packed: the packed forward).

    python -m paper_2512_14681_amd.profiling attn-traffic --fetch DIR1 --write DIR2 --copy-bytes N
        HBM bytes per call of the attention workload (``bench.py --only
        attention --copy-probe``: 9 shapes P x n, 68 calls each, each call the
        attention kernel and, when it splits the keys, its merge), per shape,
        against the shape's algorithmic bytes.

    python -m paper_2512_14681_amd.profiling ceiling [--gib G] [--reps K]
        HBM rates that plain library kernels reach on the device (GPU
        required): a full read of a G GiB bf16 tensor (torch's sum, fp32
        accumulation) and a device-to-device copy of it, each timed with
        events over K calls after a warm-up.  G well above the 256 MB
        Infinity Cache keeps both in HBM.  Also the library GEMM (torch's
        matmul) on the 7B gate/up shape, 16 x 3584 x 37888 bf16.

    python -m paper_2512_14681_amd.profiling library-gemms [--rows R] [--reps K]
        The projections of one 7B-shaped step as library GEMMs (torch's
        matmul, bf16): per layer QKV, O, gate/up and down over 28 layers of
        distinct weights, then the LM head; no attention, norms, epilogues
        or argmax.  Timed with events over K passes after a warm-up.

All print Markdown; ``traffic`` ends with ``- key: value`` lines that
bench.py reads back (the SHA-256 of the GEMM sources pins the figure to the
kernel it was measured on).
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import os
import re
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GEMM_SOURCES = ("paper_2512_14681_amd/csrc/gemm.hip", "paper_2512_14681_amd/csrc/jf_epilogue.h",
                "paper_2512_14681_amd/csrc/jf_device.h", "paper_2512_14681_amd/csrc/jf_internal.h")


def _rows(directory, suffix):
    paths = sorted(glob.glob(os.path.join(directory, "**", "*" + suffix), recursive=True))
    if not paths:
        raise FileNotFoundError(f"no *{suffix} under {directory}")
    out = []
    for p in paths:
        with open(p, newline="") as f:
            out.extend({k.lower(): v for k, v in r.items()} for r in csv.DictReader(f))
    return out


def short_name(name):
    """'void jf::k_gemm<unsigned short, 1, 4, 2, 1>(...)' -> 'k_gemm<bf16,1,4,2,1>'."""
    name = name.replace("(anonymous namespace)::", "")
    name = re.sub(r"\(.*", "", name).replace("void ", "").replace("jf::", "")
    return name.replace("unsigned short", "bf16").replace(" ", "")


def stats(directory, top=25):
    rows = _rows(directory, "kernel_stats.csv")
    total = sum(float(r["totaldurationns"]) for r in rows)
    lines = ["| kernel | calls | avg us | total ms | % |", "|---|---:|---:|---:|---:|"]
    for r in sorted(rows, key=lambda r: -float(r["totaldurationns"]))[:top]:
        lines.append(f"| `{short_name(r['name'])[:90]}` | {int(r['calls'])} | "
                     f"{float(r['averagens']) / 1e3:.2f} | {float(r['totaldurationns']) / 1e6:.2f} | "
                     f"{100 * float(r['totaldurationns']) / total:.1f} |")
    return "\n".join(lines)


def stats_by_grid(directory, pattern, top=40):
    """Per (kernel, grid of workgroups) from the kernel trace: the launches of
    one kernel at different shapes kept apart.  pattern: regex on the
    short kernel name."""
    pat = re.compile(pattern)
    groups = {}
    for r in _rows(directory, "kernel_trace.csv"):
        name = short_name(r["kernel_name"])
        if not pat.search(name):
            continue
        wg = tuple(int(r[f"workgroup_size_{a}"]) for a in "xyz")
        grid = tuple(int(r[f"grid_size_{a}"]) // w for a, w in zip("xyz", wg))
        dur = int(r["end_timestamp"]) - int(r["start_timestamp"])
        groups.setdefault((name, grid), []).append(dur)
    lines = ["| kernel | workgroups (x, y, z) | calls | avg us | min us |", "|---|---|---:|---:|---:|"]
    for (name, grid), d in sorted(groups.items(), key=lambda kv: -sum(kv[1]))[:top]:
        lines.append(f"| `{name[:60]}` | {grid[0]} x {grid[1]} x {grid[2]} | {len(d)} | "
                     f"{sum(d) / len(d) / 1e3:.2f} | {min(d) / 1e3:.2f} |")
    return "\n".join(lines)


def _per_dispatch(directory, counter):
    """[(dispatch id, kernel name, value)] of one counter, in dispatch order."""
    out = []
    for r in _rows(directory, "counter_collection.csv"):
        if r.get("counter_name") == counter:
            out.append((int(r["dispatch_id"]), r["kernel_name"], float(r["counter_value"])))
    return sorted(out)


def traffic(fetch_dir, write_dir, kernel_regex, copy_bytes, sources=None):
    pat = re.compile(kernel_regex)
    res = {}
    for label, directory, counter in (("fetch", fetch_dir, "FETCH_SIZE"), ("write", write_dir, "WRITE_SIZE")):
        rows = _per_dispatch(directory, counter)
        copies = [v for _, k, v in rows if "copy" in k.lower()][:3]
        if len(copies) < 3:
            raise RuntimeError(f"{counter}: fewer than 3 copy dispatches in {directory}")
        scale = copy_bytes / (sum(copies) / 3 * 1024)
        vals = [v for _, k, v in rows if pat.search(k)]
        if not vals:
            raise RuntimeError(f"{counter}: no dispatch matches {kernel_regex!r}")
        res[label] = dict(kib=sum(vals) / len(vals), n=len(vals), copy_kib=sum(copies) / 3, scale=scale,
                          bytes=sum(vals) / len(vals) * 1024 * scale)
    digests = " ".join(f"{p}={hashlib.sha256(open(os.path.join(ROOT, p), 'rb').read()).hexdigest()}"
                       for p in (sources or GEMM_SOURCES))
    f, w = res["fetch"], res["write"]
    return "\n".join([
        "| counter | dispatches | KiB per dispatch | copy probe KiB | scale (bytes per counted byte) "
        "| HBM bytes per dispatch |",
        "|---|---:|---:|---:|---:|---:|",
        f"| FETCH_SIZE | {f['n']} | {f['kib']:.0f} | {f['copy_kib']:.0f} | {f['scale']:.3f} | {f['bytes']:.0f} |",
        f"| WRITE_SIZE | {w['n']} | {w['kib']:.0f} | {w['copy_kib']:.0f} | {w['scale']:.3f} | {w['bytes']:.0f} |",
        "",
        f"- kernel_regex: {kernel_regex}",
        f"- copy_probe_bytes: {copy_bytes}",
        f"- fetch_bytes_per_launch: {f['bytes']:.0f}",
        f"- write_bytes_per_launch: {w['bytes']:.0f}",
        f"- hbm_bytes_per_launch: {f['bytes'] + w['bytes']:.0f}",
        f"- source_sha256: {digests}",
    ])


def algo_bytes_7b(n, ctx):
    """Algorithmic HBM bytes per dispatch of each phase of a 7B-shaped step of
    n rows at committed length ctx: weights once (bf16), activations in and
    outputs out at bf16, the attention's prefix and in-step K/V."""
    d, F, V, H, G, hd = 3584, 18944, 152064, 28, 4, 128
    qkv_n = (H + 2 * G) * hd
    return {
        "qkv": qkv_n * d * 2 + n * d * 2 + n * qkv_n * 2,
        "o": d * H * hd * 2 + n * H * hd * 2 + n * d * 2,
        "gateup": 2 * F * d * 2 + n * d * 2 + n * F * 2,
        "down": d * F * 2 + n * F * 2 + n * d * 2,
        "attn": (ctx + n) * 2 * G * hd * 2 + 2 * n * H * hd * 2,
        "lm_head": V * d * 2 + n * d * 2,
    }


def _step_phases(rows, layers):
    """Labels the dispatches of the Jacobi steps in rows [(id, name, value)]
    by phase, from the launch order of one forward: k_embed, then per layer
    the QKV projection, attention (+ its split merge), the O projection, the
    gate/up and the down projection, then the LM head and its tail.  A
    forward is kept when it ends in an acceptance kernel (k_accept_*, or the
    fused k_argmax_accept_*: a step, not a prefill chunk).  Returns {phase:
    [values]}."""
    forwards, cur = [], None
    for did, name, v in rows:
        n = short_name(name)
        if n.startswith("k_embed"):
            cur = []
            forwards.append(cur)
        if cur is not None:
            cur.append((n, v))
    gemm_phase = ("qkv", "o", "gateup", "down")
    out = {}
    for f in forwards:
        if not any(n.startswith(("k_accept", "k_argmax_accept")) for n, _ in f):
            continue
        gi = 0
        for n, v in f:
            if n.startswith("k_gemm"):
                lab = "lm_head" if gi == 4 * layers else gemm_phase[gi % 4]
                gi += 1
            elif n.startswith("k_attn_combine"):
                lab = "attn_combine"
            elif n.startswith("k_attn"):
                lab = "attn"
            else:
                lab = re.sub(r"<.*", "", n)
            out.setdefault(lab, []).append(v)
    return out


def step_traffic(fetch_dir, write_dir, copy_bytes, layers=28, algo=None):
    """HBM bytes per dispatch of every phase of the Jacobi steps in a
    rocprofv3 --pmc run (FETCH_SIZE and WRITE_SIZE in separate runs), scaled
    by a copy probe of copy_bytes (FETCH_SIZE counts half the bytes a copy
    moves, WRITE_SIZE all of them, on this device)."""
    per = {}
    for label, directory, counter in (("fetch", fetch_dir, "FETCH_SIZE"), ("write", write_dir, "WRITE_SIZE")):
        rows = _per_dispatch(directory, counter)
        copies = [v for _, k, v in rows if "copy" in k.lower()][:3]
        if len(copies) < 3:
            raise RuntimeError(f"{counter}: fewer than 3 copy dispatches in {directory}")
        scale = copy_bytes / (sum(copies) / 3 * 1024)
        for ph, vals in _step_phases(rows, layers).items():
            per.setdefault(ph, {})[label] = (sum(vals) / len(vals) * 1024 * scale, len(vals), scale)
    lines = ["| phase | dispatches | FETCH bytes | WRITE bytes | HBM bytes per dispatch | algorithmic bytes | ratio |",
             "|---|---:|---:|---:|---:|---:|---:|"]
    order = ["qkv", "attn", "attn_combine", "o", "gateup", "down", "lm_head"]
    for ph in order + sorted(k for k in per if k not in order):
        if ph not in per or "fetch" not in per[ph] or "write" not in per[ph]:
            continue
        fb, n, _ = per[ph]["fetch"]
        wb, _, _ = per[ph]["write"]
        a = (algo or {}).get(ph)
        lines.append(f"| {ph} | {n} | {fb:,.0f} | {wb:,.0f} | {fb + wb:,.0f} | "
                     f"{f'{a:,}' if a else '—'} | {f'{(fb + wb) / a:.3f}' if a else '—'} |")
    return "\n".join(lines)


ATTN_SHAPES = [(P, n) for P in (512, 2048, 8192) for n in (16, 32, 64)]  # bench.py's order


def attn_traffic(fetch_dir, write_dir, copy_bytes, shapes=None, calls=68, H=28, G=4, hd=128):
    """HBM bytes per call of each shape of the attention workload: the
    dispatches of the attention kernels in order, a call being one attention
    launch (k_attn / k_attn_lds) plus its merge (k_attn_combine) if any,
    `calls` calls a shape; FETCH_SIZE and WRITE_SIZE scaled by the copy
    probe as in traffic().  Algorithmic bytes: K and V of the P + n keys, q
    in and the output out at bf16 (the workload's own figure)."""
    shapes = shapes or ATTN_SHAPES
    per = {}
    for label, directory, counter in (("fetch", fetch_dir, "FETCH_SIZE"), ("write", write_dir, "WRITE_SIZE")):
        rows = _per_dispatch(directory, counter)
        copies = [v for _, k, v in rows if "copy" in k.lower()][:3]
        if len(copies) < 3:
            raise RuntimeError(f"{counter}: fewer than 3 copy dispatches in {directory}")
        scale = copy_bytes / (sum(copies) / 3 * 1024)
        main = -1
        for _, name, v in rows:
            n = short_name(name)
            if not n.startswith("k_attn"):
                continue
            if not n.startswith("k_attn_combine"):
                main += 1
            si = main // calls
            if si < 0 or si >= len(shapes):
                continue
            d = per.setdefault(si, {"fetch": 0.0, "write": 0.0, "kernels": set()})
            d[label] += v * 1024 * scale
            d["kernels"].add(re.sub(r"<.*", "", n))
    lines = ["| P | n | kernels | FETCH bytes per call | WRITE bytes per call | HBM bytes per call "
             "| algorithmic bytes | ratio |", "|---:|---:|---|---:|---:|---:|---:|---:|"]
    for si, (P, n) in enumerate(shapes):
        if si not in per:
            continue
        d = per[si]
        fb, wb = d["fetch"] / calls, d["write"] / calls
        algo = (P + n) * G * hd * 2 * 2 + n * H * hd * 2 + n * H * hd * 4
        lines.append(f"| {P} | {n} | {', '.join(sorted(d['kernels']))} | {fb:,.0f} | {wb:,.0f} | {fb + wb:,.0f} | "
                     f"{algo:,} | {(fb + wb) / algo:.2f} |")
    return "\n".join(lines)


MFMA_COUNTERS = ("SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_VALU_MFMA_BUSY_CYCLES", "GRBM_GUI_ACTIVE")


def _forwards_by_dispatch(directory, select):
    """{counter: {phase: [values]}} and {phase: [durations ns]} over the
    forwards of a --pmc run, each from its mask builder (k_tree*) to the
    next, kept when one of its kernels matches the regex select."""
    pat = re.compile(select)
    by_id = {}
    for r in _rows(directory, "counter_collection.csv"):
        d = by_id.setdefault(int(r["dispatch_id"]), {"name": short_name(r["kernel_name"]), "c": {},
                                                     "ns": int(r["end_timestamp"]) - int(r["start_timestamp"])})
        d["c"][r["counter_name"]] = float(r["counter_value"])
    forwards, cur = [], None
    for did in sorted(by_id):
        d = by_id[did]
        if d["name"].startswith("k_tree"):
            cur = []
            forwards.append(cur)
        if cur is not None:
            cur.append(d)
    return [f for f in forwards if any(pat.search(d["name"]) for d in f)]


def _label_forward(f, layers):
    gemm_phase = ("qkv", "o", "gateup", "down")
    gi = 0
    for d in f:
        n = d["name"]
        if n.startswith("k_gemm"):
            lab = "lm_head" if gi == 4 * layers else gemm_phase[gi % 4]
            gi += 1
        elif n.startswith("k_mr_reduce"):
            # the split-K reduction of the projection launched just before
            lab = ("lm_head" if gi == 4 * layers + 1 else gemm_phase[(gi - 1) % 4]) + "_reduce" if gi > 0 else "reduce"
        elif n.startswith("k_attn_combine"):
            lab = "attn_combine"
        elif n.startswith("k_attn"):
            lab = "attn"
        else:
            lab = re.sub(r"<.*", "", n)
        yield lab, d


def step_mfma(directory, select, rows, ctx, layers=28, clock_ghz=2.4, simds=1024, xcds=8):
    """MFMA load of every phase of the forwards in a rocprofv3 --pmc run of
    MFMA_COUNTERS: issued bf16 work (SQ_INSTS_VALU_MFMA_MOPS_BF16, 512 flops
    a unit), the matrix cores' busy fraction (SQ_VALU_MFMA_BUSY_CYCLES over
    all SIMDs against GRBM_GUI_ACTIVE, which the CSV sums over the XCDs), and
    the algorithmic flops of the phase (2 R N K for a projection, 4 R keys hd
    H for attention at the committed length ctx)."""
    d, F, V, H, G, hd = 3584, 18944, 152064, 28, 4, 128
    algo = {"qkv": 2 * rows * (H + 2 * G) * hd * d, "o": 2 * rows * d * H * hd, "gateup": 2 * rows * 2 * F * d,
            "down": 2 * rows * d * F, "lm_head": 2 * rows * V * d, "attn": 4 * rows * (ctx + rows) * hd * H}
    per = {}
    fw = _forwards_by_dispatch(directory, select)
    for f in fw:
        for lab, dd in _label_forward(f, layers):
            p = per.setdefault(lab, {"n": 0, "ns": 0.0, "mops": 0.0, "busy": 0.0, "grbm": 0.0})
            p["n"] += 1
            p["ns"] += dd["ns"]
            p["mops"] += dd["c"].get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0)
            p["busy"] += dd["c"].get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0)
            p["grbm"] += dd["c"].get("GRBM_GUI_ACTIVE", 0.0)
    lines = [f"{len(fw)} forwards matched {select!r}; per dispatch:", "",
             "| phase | dispatches | us (counter run) | issued bf16 GFLOP | algorithmic GFLOP | issued / algorithmic "
             "| issued TFLOP/s | MFMA busy |",
             "|---|---:|---:|---:|---:|---:|---:|---:|"]
    order = ["qkv", "qkv_reduce", "attn", "attn_combine", "o", "o_reduce", "gateup", "down", "down_reduce",
             "lm_head"]
    tot = {"ns": 0.0, "mops": 0.0, "algo": 0.0, "busy": 0.0, "grbm": 0.0}
    for lab in order + sorted(k for k in per if k not in order):
        if lab not in per:
            continue
        p = per[lab]
        n = p["n"]
        us = p["ns"] / n / 1e3
        gf = p["mops"] / n * 512 / 1e9
        a = algo.get(lab)
        busy = p["busy"] / (p["grbm"] / xcds * simds) if p["grbm"] else 0.0
        tot["ns"] += p["ns"]
        tot["mops"] += p["mops"]
        tot["busy"] += p["busy"]
        tot["grbm"] += p["grbm"]
        if a:
            tot["algo"] += a * n
        lines.append(f"| {lab} | {n} | {us:.1f} | {gf:.1f} | {f'{a / 1e9:.1f}' if a else '—'} | "
                     f"{f'{gf * 1e9 / a:.2f}' if a else '—'} | {gf / us * 1e3:.1f} | {busy:.3f} |")
    nf = max(1, len(fw))
    lines += ["", f"- per forward: {tot['ns'] / nf / 1e3:.1f} us in the counter run, "
              f"{tot['mops'] * 512 / nf / 1e12:.3f} TFLOP issued, {tot['algo'] / nf / 1e12:.3f} TFLOP algorithmic, "
              f"MFMA busy {tot['busy'] / (tot['grbm'] / xcds * simds) if tot['grbm'] else 0:.3f} "
              f"(cycle-weighted over the forward's dispatches)"]
    return "\n".join(lines)


def ceiling(gib=2.0, reps=20, peak_tbs=8.0):
    import torch
    n = int(gib * (1 << 30)) // 2
    x = torch.ones(n, dtype=torch.bfloat16, device="cuda")
    y = torch.empty_like(x)

    def timed(fn):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        b.synchronize()
        return a.elapsed_time(b) / reps * 1e-3

    rows = [("read (sum)", n * 2, timed(lambda: x.sum(dtype=torch.float32))),
            ("copy (read + write)", n * 4, timed(lambda: y.copy_(x)))]
    del x, y
    # The library GEMM on the 7B gate/up shape (16 rows, K 3584, N 37888),
    # rotating over four weight copies so that no call finds its weights in
    # the Infinity Cache; bytes are the weights' alone, as for k_gemm.
    K, N = 3584, 37888
    ws = [torch.ones(N, K, dtype=torch.bfloat16, device="cuda") for _ in range(4)]
    xa = torch.ones(16, K, dtype=torch.bfloat16, device="cuda")
    it = [0]

    def gemm():
        it[0] += 1
        return torch.matmul(xa, ws[it[0] % 4].t())

    rows.append(("library GEMM 16 x 3584 x 37888 (torch.matmul)", N * K * 2, timed(gemm)))
    out = [f"{gib:g} GiB bf16 tensor, {reps} calls each after 3 warm-up calls, HIP events",
           "", "| kernel | HBM bytes per call | us per call | TB/s | of " + f"{peak_tbs:g} TB/s |",
           "|---|---:|---:|---:|---:|"]
    for name, nbytes, t in rows:
        out.append(f"| {name} | {nbytes:,} | {t * 1e6:.1f} | {nbytes / t / 1e12:.2f} | "
                   f"{nbytes / t / 1e12 / peak_tbs:.3f} |")
    return "\n".join(out)


def library_gemms(rows=16, reps=10):
    import torch
    d, qkv, F, V, L = 3584, 4608, 18944, 152064, 28
    shapes = [(qkv, d), (d, d), (2 * F, d), (d, F)]
    layers = [[torch.ones(n, k, dtype=torch.bfloat16, device="cuda") for n, k in shapes] for _ in range(L)]
    lm = torch.ones(V, d, dtype=torch.bfloat16, device="cuda")
    x = torch.ones(rows, d, dtype=torch.bfloat16, device="cuda")
    a = torch.ones(rows, F, dtype=torch.bfloat16, device="cuda")

    def step():
        for wq, wo, wgu, wd in layers:
            torch.matmul(x, wq.t())
            torch.matmul(x, wo.t())
            torch.matmul(x, wgu.t())
            torch.matmul(a, wd.t())
        return torch.matmul(x, lm.t())

    for _ in range(2):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        step()
    e1.record()
    e1.synchronize()
    t = e0.elapsed_time(e1) / reps * 1e-3
    nbytes = sum(n * k for n, k in shapes) * L * 2 + V * d * 2
    return "\n".join([
        f"7B-shaped step projections as library GEMMs, {rows} rows, {L} layers + LM head, "
        f"{reps} passes after 2 warm-up passes, HIP events", "",
        "| what | weight bytes per pass | ms per pass | TB/s | of 8 TB/s |", "|---|---:|---:|---:|---:|",
        f"| {4 * L + 1} library GEMMs | {nbytes:,} | {t * 1e3:.3f} | {nbytes / t / 1e12:.2f} | "
        f"{nbytes / t / 1e12 / 8.0:.3f} |"])


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("dir")
    s.add_argument("--top", type=int, default=25)
    s.add_argument("--by-grid", metavar="REGEX",
                   help="kernels matching REGEX, one line per grid of workgroups (from the kernel trace)")
    t = sub.add_parser("traffic")
    t.add_argument("--fetch", required=True)
    t.add_argument("--write", required=True)
    t.add_argument("--kernel", required=True)
    t.add_argument("--copy-bytes", type=int, required=True)
    t.add_argument("--sources", nargs="*", help="source files whose hashes the summary records "
                   "(default: the GEMM sources)")
    stt = sub.add_parser("step-traffic", help="HBM bytes of every phase of the Jacobi steps in a --pmc run")
    stt.add_argument("--fetch", required=True)
    stt.add_argument("--write", required=True)
    stt.add_argument("--copy-bytes", type=int, required=True)
    stt.add_argument("--layers", type=int, default=28)
    stt.add_argument("--n", type=int, default=16, help="rows of the steps (for the algorithmic bytes)")
    stt.add_argument("--ctx", type=int, default=1024, help="committed length (for the attention bytes)")
    at = sub.add_parser("attn-traffic", help="HBM bytes per call of each attention workload shape")
    at.add_argument("--fetch", required=True)
    at.add_argument("--write", required=True)
    at.add_argument("--copy-bytes", type=int, required=True)
    at.add_argument("--calls", type=int, default=68, help="calls per shape (bench.py: 4 warm-up + 64 timed)")
    sm = sub.add_parser("step-mfma", help="MFMA load of every phase of the forwards in a --pmc run")
    sm.add_argument("dir")
    sm.add_argument("--select", default="accept", help="regex: keep forwards with a matching kernel "
                    "(default: the steps, which end in an acceptance kernel)")
    sm.add_argument("--rows", type=int, required=True)
    sm.add_argument("--ctx", type=int, required=True, help="committed length the forwards attend over")
    c = sub.add_parser("ceiling")
    c.add_argument("--gib", type=float, default=2.0)
    c.add_argument("--reps", type=int, default=20)
    lg = sub.add_parser("library-gemms")
    lg.add_argument("--rows", type=int, default=16)
    lg.add_argument("--reps", type=int, default=10)
    a = ap.parse_args(argv)
    if a.cmd == "library-gemms":
        print(library_gemms(a.rows, a.reps), flush=True)
    elif a.cmd == "ceiling":
        print(ceiling(a.gib, a.reps), flush=True)
    elif a.cmd == "step-mfma":
        print(step_mfma(a.dir, a.select, a.rows, a.ctx))
    elif a.cmd == "attn-traffic":
        print(attn_traffic(a.fetch, a.write, a.copy_bytes, calls=a.calls))
    elif a.cmd == "step-traffic":
        print(step_traffic(a.fetch, a.write, a.copy_bytes, a.layers, algo_bytes_7b(a.n, a.ctx)))
    elif a.cmd == "stats":
        print(stats_by_grid(a.dir, a.by_grid, a.top) if a.by_grid else stats(a.dir, a.top))
    else:
        print(traffic(a.fetch, a.write, a.kernel, a.copy_bytes, a.sources))


if __name__ == "__main__":
    sys.exit(main())
