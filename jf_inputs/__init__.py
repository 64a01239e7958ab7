"""Seeded synthetic inputs for the Jacobi-step engine and its CPU oracle.

This module turns seeds into data and nothing else: it holds none of the
decoding method's arithmetic.  Both the GPU path's callers (tests, bench) and
the oracle's callers draw their inputs from here, so the two sides see the same
bytes without sharing any code that computes a result.

Generator (fully specified, so the bytes do not depend on a library version):

* splitmix64 (Steele, Lea & Flood, OOPSLA 2014; Vigna's public-domain
  reference): ``mix64(z)`` is its output finaliser and element ``i`` of stream
  ``key`` is ``mix64(key + i * 0x9E3779B97F4A7C15)``.
* normals by the Box-Muller transform of two 24-bit fields of one draw:
  ``u1 = (bits 40..63 + 0.5) / 2**24``, ``u2 = (bits 0..23 + 0.5) / 2**24``,
  ``z = sqrt(-2 ln u1) * cos(2 pi u2)`` in float32, then scaled and, for bf16
  tensors, rounded to bf16 (nearest-even) and kept as uint16 bit patterns.
* uniform token ids by Lemire's multiply-shift: ``((x >> 32) * V) >> 32``.

Model recipe (the paper's backbone shape, random init):
projection and embedding weights ~ N(0, 0.02); RMSNorm gains ~ 1 + 0.1 N(0,1)
(non-trivial so that a dropped gain is visible); layout [out, in] row-major.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

GOLDEN = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)

# Model shapes named in the workloads.  "tiny" is the 2-layer fp32 decoder;
# "7b" is the Qwen2.5-7B-shaped bf16 decoder (the paper's backbone shape).
MODEL_SHAPES = {
    "tiny": dict(n_layers=2, d_model=128, n_heads=4, n_kv_heads=4, head_dim=32,
                 d_ffn=512, vocab=1024, rope_base=10000.0, rms_eps=1e-6, dtype="f32"),
    "7b": dict(n_layers=28, d_model=3584, n_heads=28, n_kv_heads=4, head_dim=128,
               d_ffn=18944, vocab=152064, rope_base=1000000.0, rms_eps=1e-6, dtype="bf16"),
}

_CHUNK = 1 << 18


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def mix64(z: np.ndarray) -> np.ndarray:
    """splitmix64 output finaliser on a uint64 array (wrapping arithmetic)."""
    with np.errstate(over="ignore"):
        z = (z ^ (z >> np.uint64(30))) * _M1
        z = (z ^ (z >> np.uint64(27))) * _M2
        return z ^ (z >> np.uint64(31))


def stream_key(seed: int, stream: int) -> np.uint64:
    """Key of an independent stream: mix64 of (seed, stream) packed in 64 bits."""
    z = np.array([(int(seed) * 0x100000001B3 + int(stream) * 0x9E3779B97F4A7C15 + 1)
                  & 0xFFFFFFFFFFFFFFFF], dtype=np.uint64)
    return mix64(z)[0]


def _draws(key: np.uint64, start: int, count: int) -> np.ndarray:
    i = np.arange(start, start + count, dtype=np.uint64)
    with np.errstate(over="ignore"):
        return mix64(key + i * GOLDEN)


def _f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit pattern, round to nearest even (finite inputs)."""
    b = x.view(np.uint32)
    lsb = (b >> np.uint32(16)) & np.uint32(1)
    return ((b + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)


def _normal_chunk(key, start, count, std, mean, dtype, out):
    x = _draws(key, start, count)
    u1 = ((x >> np.uint64(40)).astype(np.float32) + np.float32(0.5)) * np.float32(2.0 ** -24)
    u2 = ((x & np.uint64(0xFFFFFF)).astype(np.float32) + np.float32(0.5)) * np.float32(2.0 ** -24)
    z = np.sqrt(np.float32(-2.0) * np.log(u1)) * np.cos(np.float32(2.0 * np.pi) * u2)
    v = (z * np.float32(std) + np.float32(mean)).astype(np.float32)
    out[start:start + count] = _f32_to_bf16_bits(v) if dtype == "bf16" else v


def normal(seed: int, stream: int, n: int, std: float = 1.0, mean: float = 0.0,
           dtype: str = "f32") -> np.ndarray:
    """n draws of N(mean, std^2); float32 array, or uint16 bf16 bits if dtype == 'bf16'."""
    key = stream_key(seed, stream)
    out = np.empty(n, dtype=np.uint16 if dtype == "bf16" else np.float32)
    starts = list(range(0, n, _CHUNK))

    def job(s):
        _normal_chunk(key, s, min(_CHUNK, n - s), std, mean, dtype, out)

    if len(starts) > 4:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(job, starts))
    else:
        for s in starts:
            job(s)
    return out


def token_ids(seed: int, stream: int, n: int, vocab: int) -> np.ndarray:
    """n uniform token ids in [0, vocab) as int32."""
    x = _draws(stream_key(seed, stream), 0, n)
    with np.errstate(over="ignore"):
        return (((x >> np.uint64(32)) * np.uint64(vocab)) >> np.uint64(32)).astype(np.int32)


def uniform_int(seed: int, stream: int, n: int, lo: int, hi: int) -> np.ndarray:
    """n uniform integers in [lo, hi) as int64."""
    return token_ids(seed, stream, n, hi - lo).astype(np.int64) + lo


def weight_specs(shape: dict) -> list:
    """Tensor names, shapes and kinds in fixture order ('normal' or 'gain')."""
    d, H, G, hd = shape["d_model"], shape["n_heads"], shape["n_kv_heads"], shape["head_dim"]
    F, V = shape["d_ffn"], shape["vocab"]
    specs = [("embed", (V, d), "normal")]
    for l in range(shape["n_layers"]):
        p = f"layers.{l}."
        specs += [(p + "attn_norm", (d,), "gain"),
                  (p + "wq", (H * hd, d), "normal"),
                  (p + "wk", (G * hd, d), "normal"),
                  (p + "wv", (G * hd, d), "normal"),
                  (p + "wo", (d, H * hd), "normal"),
                  (p + "ffn_norm", (d,), "gain"),
                  (p + "w_gate", (F, d), "normal"),
                  (p + "w_up", (F, d), "normal"),
                  (p + "w_down", (d, F), "normal")]
    specs += [("final_norm", (d,), "gain"), ("lm_head", (V, d), "normal")]
    return specs


def model_weights(shape: dict, seed: int = 0, names=None) -> dict:
    """Random-init weights of a decoder shape, in fixture order.

    Values are float32 arrays for dtype 'f32' models and uint16 bf16 bit
    patterns for 'bf16' models.  ``names`` restricts generation to a subset
    (each tensor's values do not depend on which others are generated).
    """
    out = {}
    dtype = shape["dtype"]
    for t, (name, shp, kind) in enumerate(weight_specs(shape)):
        if names is not None and name not in names:
            continue
        n = int(np.prod(shp))
        if kind == "gain":
            a = normal(seed, 1000 + t, n, std=0.1, mean=1.0, dtype=dtype)
        else:
            a = normal(seed, 1000 + t, n, std=0.02, dtype=dtype)
        out[name] = a.reshape(shp)
    return out


def prompt(seed: int, length: int, vocab: int) -> np.ndarray:
    """A prompt of uniform-random token ids."""
    return token_ids(seed, 7, length, vocab)


def trajectories(seed: int, n_blocks: int, n: int, vocab: int, max_points: int = 0,
                 chunk: int = 1 << 16):
    """Synthetic Jacobi trajectories of n-token blocks, shaped like the data
    collection's: block b takes k_b uniform in [1, n] iterations, so it has
    k_b + 1 points (int32 lengths), the last two equal to a random fixed
    point y*.  Before them, point j keeps the first m_j = 1 + j (n-1) //
    (k_b-1) tokens of y*, has a token different from y* at position m_j,
    and beyond it each token is y*'s with probability 1/4 (tokens that
    settled early), else uniform.  Returns (traj [n_blocks][max_points][n]
    int32, with -1 in unused points; lengths [n_blocks] int32).
    max_points defaults to n + 1."""
    P = max_points or n + 1
    if P < n + 1:
        raise ValueError("max_points must be at least n + 1")
    traj = np.full((n_blocks, P, n), -1, np.int32)
    lengths = np.zeros(n_blocks, np.int32)
    V = np.uint64(vocab)
    for b0 in range(0, n_blocks, chunk):
        B = min(chunk, n_blocks - b0)
        k = (((_draws(stream_key(seed, 40), b0, B) >> np.uint64(32)) * np.uint64(n)) >> np.uint64(32))
        k = k.astype(np.int64) + 1
        lengths[b0:b0 + B] = k + 1
        ys = (((_draws(stream_key(seed, 41), b0 * n, B * n) >> np.uint64(32)) * V) >> np.uint64(32))
        ys = ys.astype(np.int64).reshape(B, 1, n)
        cnt = B * P * n
        r = _draws(stream_key(seed, 42), b0 * P * n, cnt).reshape(B, P, n)
        rnd = ((r >> np.uint64(32)) * V >> np.uint64(32)).astype(np.int64)
        keep = (r & np.uint64(3)) == 0
        j = np.arange(P).reshape(1, P, 1)
        p = np.arange(n).reshape(1, 1, n)
        kk = k.reshape(B, 1, 1)
        m = 1 + (j * (n - 1)) // np.maximum(kk - 1, 1)
        off = 1 + (rnd % max(vocab - 1, 1))
        out = np.where(p < m, ys, np.where(p == m, (ys + off) % vocab, np.where(keep, ys, rnd)))
        out = np.where(j >= kk - 1, ys, out)
        out = np.where(j >= kk + 1, -1, out)
        traj[b0:b0 + B] = out.astype(np.int32)
    return traj, lengths
