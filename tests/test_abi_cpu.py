"""The C ABI without a GPU: libjf loads, exports every function include/jf.h
declares, and its host-side validation rejects bad arguments before any HIP
call (so these run on a CPU-only host)."""
import ctypes
import os
import re
import threading

import pytest

from paper_2512_14681_amd import jf

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "jf.h")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(jf.LIB_PATH):
        pytest.skip("libjf.so not built (python -m paper_2512_14681_amd.build)")
    return jf.lib()


def declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(jf_[a-z_0-9]+)\s*\(", text)))


def test_every_declared_function_is_exported(L):
    names = declared()
    assert len(names) >= 17
    for n in names:
        assert hasattr(L, n), n
    assert sorted(jf.EXPORTS) == names


def tiny_cfg(**kw):
    c = jf.config(dict(n_layers=2, d_model=128, n_heads=4, n_kv_heads=4, head_dim=32, d_ffn=512,
                       vocab=1024, rope_base=10000.0, rms_eps=1e-6, dtype="f32"), 16, 256)
    for k, v in kw.items():
        setattr(c, k, v)
    return c


def test_query_sizes_valid(L):
    packed, kv, ws = jf.query_sizes(tiny_cfg())
    # packed holds every weight once (plus the embedding copy), fp32
    n_w = 2 * (3 * 128 * 128 + 128 * 128 + 3 * 512 * 128) + 2 * 1024 * 128
    assert packed >= n_w * 4
    assert kv == 2 * (256 // 64) * 2 * 4 * 64 * 32 * 4
    assert ws > 0


@pytest.mark.parametrize("field,value,status", [
    ("dtype", 7, jf.JF_E_DTYPE),
    ("d_model", 100, jf.JF_E_SHAPE),
    ("head_dim", 48, jf.JF_E_SHAPE),
    ("n_kv_heads", 3, jf.JF_E_SHAPE),
    ("vocab", 1000, jf.JF_E_SHAPE),
    ("max_rows", 0, jf.JF_E_SHAPE),
    ("max_rows", jf.JF_MAX_ROWS + 1, jf.JF_E_SHAPE),
    ("max_ctx", 100, jf.JF_E_SHAPE),
    ("rms_eps", 0.0, jf.JF_E_INVAL),
])
def test_query_sizes_rejects(L, field, value, status):
    with pytest.raises(jf.JfError) as e:
        jf.query_sizes(tiny_cfg(**{field: value}))
    assert e.value.status == status
    assert L.jf_last_error().decode()


def test_null_arguments_rejected_without_hip(L):
    P = ctypes.c_void_p
    cfg = tiny_cfg()
    h = P()
    assert L.jf_model_load(ctypes.byref(cfg), None, 21, None, None, None, None, ctypes.byref(h)) == jf.JF_E_INVAL
    ptrs = (P * 3)()
    assert L.jf_model_load(ctypes.byref(cfg), ptrs, 3, P(1), P(1), P(1), None, ctypes.byref(h)) == jf.JF_E_INVAL
    assert "n_weights" in L.jf_last_error().decode()
    assert L.jf_jacobi_step(None, P(1), 4, 1, 0, P(1), P(1), P(1), None, None) == jf.JF_E_INVAL
    assert L.jf_multiblock_step(None, P(1), 4, None, 1, P(1), P(1), P(1), P(1), None, None) == jf.JF_E_INVAL
    assert L.jf_commit_kv(None, None, None, 0, None) == jf.JF_E_INVAL
    assert L.jf_prefill(None, P(1), 4, P(1), None) == jf.JF_E_INVAL
    assert L.jf_model_free(None) == jf.JF_E_INVAL
    assert L.jf_kv_truncate(None, 0, None) == jf.JF_E_INVAL
    assert L.jf_attention(4, 4, 48, 1, 0, 4, P(1), P(1), P(1), None, P(1), P(1), None) == jf.JF_E_SHAPE
    assert L.jf_attention(4, 4, 32, 5, 0, 4, P(1), P(1), P(1), None, P(1), P(1), None) == jf.JF_E_DTYPE
    assert L.jf_attention(4, 4, 32, 1, 0, jf.JF_MAX_ROWS + 1, P(1), P(1), P(1), None, P(1), P(1), None) == jf.JF_E_CAPACITY
    assert L.jf_pack_matrix(20, 128, 1, P(1), P(1), None) == jf.JF_E_SHAPE
    assert L.jf_lm_head_accept(4, 100, 1024, 1, P(1), P(1), None, P(1), None, None, P(1), None) == jf.JF_E_SHAPE
    assert L.jf_lm_head_accept(4, 128, 1024, 1, P(1), P(1), P(1), P(1), None, None, P(1), None) == jf.JF_E_INVAL
    # the allocation-free LM head: same checks, plus its fixed scratch capacity
    assert L.jf_lm_head_accept_noalloc(4, 100, 1024, 1, P(1), P(1), None, P(1), None, None, None) == jf.JF_E_SHAPE
    assert L.jf_lm_head_accept_noalloc(4, 128, 1024, 1, None, P(1), None, P(1), None, None, None) == jf.JF_E_INVAL
    assert L.jf_lm_head_accept_noalloc(jf.JF_MAX_ROWS + 1, 128, 1024, 1, P(1), P(1), None, P(1), None, None,
                                       None) == jf.JF_E_CAPACITY
    assert L.jf_lm_head_accept_noalloc(256, 3584, 152064, 1, P(1), P(1), None, P(1), None, None,
                                       None) == jf.JF_E_CAPACITY
    assert "scratch" in L.jf_last_error().decode()
    # packed forward and trajectories: argument checks happen before any HIP call
    assert L.jf_packed_forward(None, P(1), 2, 8, 0, P(1), None, None) == jf.JF_E_INVAL
    assert L.jf_trajectory_record(None, P(1), 16, 4, P(1), None) == jf.JF_E_INVAL
    assert L.jf_trajectory_record(P(1), P(1), 16, 17, P(1), None) == jf.JF_E_SHAPE
    assert L.jf_trajectory_record(P(1), P(1), 16, 0, P(1), None) == jf.JF_E_SHAPE
    assert L.jf_trajectory_select(P(1), None, 4, 16, 17, 16, None, P(1), None, None) == jf.JF_E_INVAL
    assert L.jf_trajectory_select(P(1), P(1), 4, 0, 17, 16, None, P(1), None, None) == jf.JF_E_SHAPE
    assert L.jf_trajectory_select(P(1), P(1), 4, 16, 17, 0, None, P(1), None, None) == jf.JF_E_SHAPE
    assert L.jf_trajectory_select(P(1), P(1), -1, 16, 17, 16, None, P(1), None, None) == jf.JF_E_SHAPE
    assert L.jf_trajectory_select(P(1), P(1), 0, 16, 17, 16, None, P(1), None, None) == jf.JF_OK


def test_last_error_is_thread_local(L):
    jf.query_sizes(tiny_cfg())
    with pytest.raises(jf.JfError):
        jf.query_sizes(tiny_cfg(dtype=9))
    msg = L.jf_last_error().decode()
    seen = []
    t = threading.Thread(target=lambda: seen.append(L.jf_last_error().decode()))
    t.start(); t.join()
    assert msg and seen == [""]


def test_workspace_size_helpers(L):
    assert L.jf_attention_ws_bytes(28, 128, 64) >= 32 * 64 * 28 * 130 * 4
    assert L.jf_lm_head_ws_bytes(64, 152064) >= 152064 // 16 * 64 * 8
    assert L.jf_packed_matrix_bytes(152064, 3584, 1) == 152064 * 3584 * 2
    assert L.jf_attention_ws_bytes(0, 128, 64) == 0


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    # No fallback: without the built library every call raises.
    monkeypatch.setattr(jf, "_LIB", None)
    monkeypatch.setattr(jf, "LIB_PATH", str(tmp_path / "libjf.so"))
    with pytest.raises(RuntimeError, match="is missing"):
        jf.lib()
    with pytest.raises(RuntimeError, match="is missing"):
        jf.query_sizes(tiny_cfg())
