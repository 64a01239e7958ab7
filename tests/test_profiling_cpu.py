"""The rocprofv3 summaries of profiling.py on synthetic counter CSVs (no
GPU): forwards are cut at the mask builder, kept by the selecting kernel,
and their dispatches labelled by phase from the launch order of a forward."""
import csv
import os

from paper_2512_14681_amd import profiling

COLS = ["Correlation_Id", "Dispatch_Id", "Agent_Id", "Queue_Id", "Process_Id", "Thread_Id", "Grid_Size",
        "Kernel_Id", "Kernel_Name", "Workgroup_Size", "LDS_Block_Size", "Scratch_Size", "VGPR_Count",
        "Accum_VGPR_Count", "SGPR_Count", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]


def forward(layers, tail):
    names = ["void jf::k_tree(int)", "jf::k_embed(int)"]
    for _ in range(layers):
        names += ["void jf::k_gemm<unsigned short, 1, 4, 2, 1, false>(int)", "jf::k_attn_lds(jf::AttnArgs)",
                  "void jf::k_attn_combine<unsigned short, 128, 8>(jf::AttnArgs)",
                  "void jf::k_gemm<unsigned short, 1, 4, 8, 1, false>(int)",
                  "void jf::k_gemm_mr<4, 2, 2>(int)", "void jf::k_gemm_mr<4, 2, 2>(int)",
                  "jf::k_mr_reduce(jf::MrPlan, jf::Epi)"]
    return names + ["void jf::k_gemm_mr<4, 2, 2>(int)"] + tail


def write_run(path, names):
    os.makedirs(path, exist_ok=True)
    with open(os.path.join(path, "x_counter_collection.csv"), "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(COLS)
        t = 1000
        for i, n in enumerate(names):
            for c, v in (("SQ_INSTS_VALU_MFMA_MOPS_BF16", 1000.0 * (i + 1)),
                         ("SQ_VALU_MFMA_BUSY_CYCLES", 1024.0 * 100), ("GRBM_GUI_ACTIVE", 8 * 400.0)):
                w.writerow([i, i, "Agent 1", 1, 1, 1, 512, 1, n, 256, 0, 0, 64, 0, 32, c, v, t, t + 2000])
            t += 3000


def test_step_mfma_labels_and_fractions(tmp_path):
    layers = 2
    prefill = forward(layers, [])                           # no acceptance: not a step
    step = forward(layers, ["jf::k_argmax_reduce(int)", "jf::k_accept_linear(int)"])
    write_run(str(tmp_path), prefill + step)
    fw = profiling._forwards_by_dispatch(str(tmp_path), "k_accept")
    assert len(fw) == 1
    labels = [lab for lab, _ in profiling._label_forward(fw[0], layers)]
    assert labels[:2] == ["k_tree", "k_embed"]
    assert labels[2:9] == ["qkv", "attn", "attn_combine", "o", "gateup", "down", "down_reduce"]
    assert labels.count("lm_head") == 1 and labels[-3] == "lm_head"
    out = profiling.step_mfma(str(tmp_path), "k_accept", rows=16, ctx=1024, layers=layers)
    # busy: 1024 SIMDs x 100 cycles over 400 active cycles an XCD (8 XCDs summed)
    assert "| qkv | 2 | 2.0 |" in out
    assert out.count("| 0.250 |") >= 6


def write_counter(path, counter, named_values):
    os.makedirs(path, exist_ok=True)
    with open(os.path.join(path, "x_counter_collection.csv"), "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(COLS)
        for i, (n, v) in enumerate(named_values):
            w.writerow([i, i, "Agent 1", 1, 1, 1, 512, 1, n, 256, 0, 0, 64, 0, 32, counter, v, 0, 1000])


def test_attn_traffic_splits_calls_by_shape(tmp_path):
    """Two shapes of two calls: the first runs the split kernel and its merge,
    the second the LDS-shared kernel alone; counters scale by the copy probe
    (FETCH_SIZE reads half a copy's bytes here: 1 KiB counted per 2 KiB)."""
    copy = [("__amd_rocclr_copyBuffer", 2.0)] * 3               # 2 KiB counted per 4 KiB copied
    calls = [("void jf::k_attn<unsigned short, 128, 1>(jf::AttnArgs)", 10.0),
             ("void jf::k_attn_combine<unsigned short, 128, 8>(jf::AttnArgs)", 2.0)] * 2 + \
            [("jf::k_attn_lds(jf::AttnArgs)", 6.0)] * 2
    write_counter(str(tmp_path / "f"), "FETCH_SIZE", copy + calls)
    write_counter(str(tmp_path / "w"), "WRITE_SIZE", copy + [(n, 1.0) for n, _ in calls])
    out = profiling.attn_traffic(str(tmp_path / "f"), str(tmp_path / "w"), 4096, shapes=[(512, 16), (512, 32)],
                                 calls=2)
    lines = out.splitlines()
    # scale 4096 / 2048 = 2: shape 1 fetches (10 + 2) KiB x 2 per call, writes 2 KiB x 2
    assert lines[2].startswith("| 512 | 16 | k_attn, k_attn_combine | 24,576 | 4,096 | 28,672 |")
    assert lines[3].startswith("| 512 | 32 | k_attn_lds | 12,288 | 2,048 | 14,336 |")
