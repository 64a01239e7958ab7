"""ctypes binding of libjf (include/jf.h) -- argument marshalling only.

Every function of the C ABI is exposed under its own name on ``lib()``; the
``Model`` class is a thin owner of the device buffers the ABI asks for
(allocated with torch, which is used here only for device memory and
streams).  No step of the decoding path runs in Python: each call below is
one ABI call that enqueues HIP kernels.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libjf.so")

JF_OK, JF_E_INVAL, JF_E_SHAPE, JF_E_CAPACITY, JF_E_DTYPE, JF_E_HIP, JF_E_STATE = 0, -1, -2, -3, -4, -5, -6
JF_F32, JF_BF16 = 0, 1
JF_ROLE_RA, JF_ROLE_CAND, JF_ROLE_PSEUDO = 0, 1, 2
JF_MAX_SEGMENTS = 16
JF_MAX_ROWS = 512      # rows of one step at most
JF_STEP_COMMIT = 2     # jf_jacobi_step mode bit: commit the accepted rows in the step
JF_VIS_WORDS = 8       # u64 words of a row's in-step visibility mask
JF_FLAG_BAD_TOKEN, JF_FLAG_CAPACITY, JF_FLAG_SYNC = 1, 2, 4
JF_OPT_FUSED_ATTENTION = 1
JF_MASK_NOISY_CONTEXT, JF_MASK_CLEAN_CONTEXT = 0, 1
(JF_KERNEL_QKV, JF_KERNEL_ATTN, JF_KERNEL_O, JF_KERNEL_GATEUP, JF_KERNEL_DOWN, JF_KERNEL_LMHEAD,
 JF_KERNEL_STEP, JF_KERNEL_ATTN_BLOCK) = range(1, 9)
STATUS_NAMES = {0: "JF_OK", -1: "JF_E_INVAL", -2: "JF_E_SHAPE", -3: "JF_E_CAPACITY",
                -4: "JF_E_DTYPE", -5: "JF_E_HIP", -6: "JF_E_STATE"}


def act_layout(x):
    """[R][K] row-major -> the GEMM-input activation layout of include/jf.h.

    Rows are padded to a multiple of 16 (padding rows are zero); the result
    is flat, ceil(R/16)*16*K elements.  K must be a multiple of 128.
    """
    x = np.asarray(x)
    R, K = x.shape
    Rp = (R + 15) // 16 * 16
    xp = np.zeros((Rp, K), x.dtype)
    xp[:R] = x
    # [tile, r, kc, q, j, e] -> [tile, kc, j, q, r, e]  (lane = 16 q + r)
    return np.ascontiguousarray(
        xp.reshape(Rp // 16, 16, K // 128, 4, 4, 8).transpose(0, 2, 4, 3, 1, 5)).reshape(-1)


def act_unlayout(a, R, K):
    """Inverse of act_layout: the first R rows as an [R][K] array."""
    a = np.asarray(a)
    Rp = (R + 15) // 16 * 16
    t = a[:Rp * K].reshape(Rp // 16, K // 128, 4, 4, 16, 8).transpose(0, 4, 1, 3, 2, 5)
    return np.ascontiguousarray(t).reshape(Rp, K)[:R]


class JfConfig(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("d_ffn", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("rope_base", ctypes.c_float),
                ("rms_eps", ctypes.c_float), ("dtype", ctypes.c_int32),
                ("max_rows", ctypes.c_int32), ("max_ctx", ctypes.c_int32)]


class JfSegment(ctypes.Structure):
    _fields_ = [("first_row", ctypes.c_int32), ("n_rows", ctypes.c_int32),
                ("attach_row", ctypes.c_int32), ("role", ctypes.c_int32),
                ("verify_from", ctypes.c_int32)]


class JfError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


_LIB = None
P, I32, U64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint64, ctypes.c_size_t
_SIGS = {
    "jf_query_sizes": (I32, [ctypes.POINTER(JfConfig), ctypes.POINTER(SZ), ctypes.POINTER(SZ), ctypes.POINTER(SZ)]),
    "jf_model_load": (I32, [ctypes.POINTER(JfConfig), ctypes.POINTER(P), I32, P, P, P, P, ctypes.POINTER(P)]),
    "jf_model_free": (I32, [P]),
    "jf_last_error": (ctypes.c_char_p, []),
    "jf_prefill": (I32, [P, P, I32, P, P]),
    "jf_jacobi_step": (I32, [P, P, I32, I32, U64, P, P, P, P, P]),
    "jf_multiblock_step": (I32, [P, P, I32, ctypes.POINTER(JfSegment), I32, P, P, P, P, P, P]),
    "jf_commit_kv": (I32, [P, P, P, I32, P]),
    "jf_kv_length": (I32, [P, ctypes.POINTER(I32), P]),
    "jf_kv_truncate": (I32, [P, I32, P]),
    "jf_kv_set_page_table": (I32, [P, ctypes.POINTER(I32), I32, P]),
    "jf_model_set_option": (I32, [P, I32, I32]),
    "jf_profile_begin": (I32, [P, I32]),
    "jf_profile_end": (I32, [P, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(I32)]),
    "jf_attention_ws_bytes": (SZ, [I32, I32, I32]),
    "jf_attention": (I32, [I32, I32, I32, I32, I32, I32, P, P, P, P, P, P, P]),
    "jf_packed_matrix_bytes": (SZ, [I32, I32, I32]),
    "jf_pack_matrix": (I32, [I32, I32, I32, P, P, P]),
    "jf_lm_head_ws_bytes": (SZ, [I32, I32]),
    "jf_lm_head_accept": (I32, [I32, I32, I32, I32, P, P, P, P, P, P, P, P]),
    "jf_lm_head_accept_noalloc": (I32, [I32, I32, I32, I32, P, P, P, P, P, P, P]),
    "jf_packed_forward": (I32, [P, P, I32, I32, I32, P, P, P]),
    "jf_trajectory_record": (I32, [P, P, I32, I32, P, P]),
    "jf_trajectory_select": (I32, [P, P, I32, I32, I32, I32, P, P, P, P]),
}
EXPORTS = tuple(_SIGS)


def lib():
    """The loaded libjf; raises if it has not been built (no fallback)."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2512_14681_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype, f.argtypes = res, args
        _LIB = L
    return _LIB


def check(status):
    if status != JF_OK:
        raise JfError(status, lib().jf_last_error().decode())
    return status


def config(shape: dict, max_rows: int, max_ctx: int) -> JfConfig:
    return JfConfig(shape["n_layers"], shape["d_model"], shape["n_heads"], shape["n_kv_heads"],
                    shape["head_dim"], shape["d_ffn"], shape["vocab"], float(shape["rope_base"]),
                    float(shape["rms_eps"]), JF_BF16 if shape["dtype"] == "bf16" else JF_F32,
                    int(max_rows), int(max_ctx))


def query_sizes(cfg: JfConfig):
    a, b, c = SZ(), SZ(), SZ()
    check(lib().jf_query_sizes(ctypes.byref(cfg), ctypes.byref(a), ctypes.byref(b), ctypes.byref(c)))
    return a.value, b.value, c.value


def weight_names(shape: dict):
    """Weight tensors in the order jf_model_load takes them."""
    names = ["embed"]
    for l in range(shape["n_layers"]):
        names += [f"layers.{l}.{k}" for k in ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm",
                                               "w_gate", "w_up", "w_down")]
    return names + ["final_norm", "lm_head"]


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def segments(segs):
    """Host array of jf_segment from (first, n_rows, attach, role, verify_from) tuples."""
    arr = (JfSegment * len(segs))()
    for i, s in enumerate(segs):
        arr[i] = JfSegment(*[int(v) for v in s])
    return arr


class Model:
    """Device buffers of one libjf model (one sequence) and its ABI calls."""

    def __init__(self, shape: dict, weights: dict, max_rows: int, max_ctx: int, device="cuda",
                 stream=None):
        import torch
        self.torch = torch
        self.shape = dict(shape)
        self.cfg = config(shape, max_rows, max_ctx)
        self.stream = stream
        packed, kv, ws = query_sizes(self.cfg)
        self.packed = torch.empty(packed, dtype=torch.uint8, device=device)
        self.kv = torch.empty(kv, dtype=torch.uint8, device=device)
        self.ws = torch.empty(ws, dtype=torch.uint8, device=device)
        names = weight_names(shape)
        dev = []
        for n in names:
            a = np.ascontiguousarray(weights[n])
            t = torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a).to(device)
            dev.append(t)
        ptrs = (ctypes.c_void_p * len(dev))(*[t.data_ptr() for t in dev])
        h = ctypes.c_void_p()
        check(lib().jf_model_load(ctypes.byref(self.cfg), ptrs, len(dev), _ptr(self.packed),
                                  _ptr(self.kv), _ptr(self.ws), _stream(stream), ctypes.byref(h)))
        self.h = h
        del dev
        self.V = shape["vocab"]

    def __del__(self):
        try:
            if getattr(self, "h", None):
                lib().jf_model_free(self.h)
                self.h = None
        except Exception:
            pass

    # ---- ABI calls (device tensors in, device tensors out) ----------------
    def jf_prefill(self, d_tokens, d_pending):
        check(lib().jf_prefill(self.h, _ptr(d_tokens), int(d_tokens.numel()), _ptr(d_pending),
                               _stream(self.stream)))

    def jf_jacobi_step(self, d_draft, n, mode, pad_seed, d_argmax, d_result, d_next, d_logits=None):
        check(lib().jf_jacobi_step(self.h, _ptr(d_draft), int(n), int(mode), int(pad_seed),
                                   _ptr(d_argmax), _ptr(d_result), _ptr(d_next), _ptr(d_logits),
                                   _stream(self.stream)))

    def jf_multiblock_step(self, d_tokens, R, segs, d_argmax, d_seg_accept, d_result, d_path,
                           d_logits=None):
        arr = segments(segs)
        check(lib().jf_multiblock_step(self.h, _ptr(d_tokens), int(R), arr, len(segs), _ptr(d_argmax),
                                       _ptr(d_seg_accept), _ptr(d_result), _ptr(d_path),
                                       _ptr(d_logits), _stream(self.stream)))

    def jf_packed_forward(self, d_tokens, n_blocks, n, mask, d_argmax, d_logits=None):
        check(lib().jf_packed_forward(self.h, _ptr(d_tokens), int(n_blocks), int(n), int(mask),
                                      _ptr(d_argmax), _ptr(d_logits), _stream(self.stream)))

    def jf_commit_kv(self, d_path, d_result, max_commit=0):
        check(lib().jf_commit_kv(self.h, _ptr(d_path), _ptr(d_result), int(max_commit),
                                 _stream(self.stream)))

    def jf_kv_length(self):
        v = ctypes.c_int32()
        check(lib().jf_kv_length(self.h, ctypes.byref(v), _stream(self.stream)))
        return v.value

    def jf_kv_truncate(self, n):
        check(lib().jf_kv_truncate(self.h, int(n), _stream(self.stream)))

    def jf_model_set_option(self, option, value):
        check(lib().jf_model_set_option(self.h, int(option), int(value)))

    def jf_profile_begin(self, kernel_class):
        check(lib().jf_profile_begin(self.h, int(kernel_class)))

    def jf_profile_end(self):
        t, n = ctypes.c_double(), ctypes.c_int32()
        check(lib().jf_profile_end(self.h, ctypes.byref(t), ctypes.byref(n)))
        return t.value, n.value

    def jf_kv_set_page_table(self, table):
        t = np.ascontiguousarray(table, dtype=np.int32)
        check(lib().jf_kv_set_page_table(self.h, t.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                         len(t), _stream(self.stream)))


# ---- trajectories (component calls, no model) ------------------------------------
def trajectory_record(d_prev, d_argmax, n, rows, d_out, stream=None):
    check(lib().jf_trajectory_record(_ptr(d_prev), _ptr(d_argmax), int(n), int(rows), _ptr(d_out),
                                     _stream(stream)))


def trajectory_select(d_traj, d_len, n_blocks, n, max_points, w, d_sel, d_t_num=None, d_unconv=None,
                      stream=None):
    check(lib().jf_trajectory_select(_ptr(d_traj), _ptr(d_len), int(n_blocks), int(n), int(max_points),
                                     int(w), _ptr(d_t_num), _ptr(d_sel), _ptr(d_unconv), _stream(stream)))
