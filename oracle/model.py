"""Decoder forward pass over the rows of one Jacobi iteration (oracle).

Sec. 2.1 ("Jacobi Decoding"): all n maximisation problems of Eq. 3 are solved
by ONE forward pass of the causal LM, because row i only attends to the
prompt/prefix and to rows before it.  The paper's backbone is a pretrained
causal decoder (Qwen2.5-7B family, Sec. 4.1) reusing an exact KV cache of the
committed prefix (Sec. 1).  This module is that decoder written out plainly:

    h     = E[token]
    per layer:
      xn  = RMSNorm(h) * g_attn
      q,k,v = xn Wq^T, xn Wk^T, xn Wv^T
      q,k = RoPE(q, pos), RoPE(k, pos)             (rotate-half pairing i, i+hd/2)
      k,v are what the cache stores (rounded to bf16 in bf16 mode)
      o   = softmax(q k^T / sqrt(hd)) v over the visible keys, GQA with query
            head j reading KV head floor(j / (H/G))
      h   = h + o Wo^T
      u   = RMSNorm(h) * g_ffn
      m   = silu(u Wg^T) * (u Wu^T)
      h   = h + m Wd^T
    logits = (RMSNorm(h) * g_final) W_lm^T

bf16 mode means bf16 weights and a bf16 KV cache; every other value is
computed in the oracle's precision (fp64 by default).  Rounding activations
to bf16 as well would make any two correct implementations disagree by
random 1-ulp flips that compound layer after layer (the logits of a
2-layer d=2048 model then differ by up to 2e-2 between fp32 and fp64
arithmetic), so the engine carries activations in fp32.

Visible keys of a row: the whole committed prefix [0, C) plus the in-step
rows marked in its visibility row (its ancestors and itself).

Weights arrive as the fixture's arrays: float32 for 'f32' models, uint16 bf16
bit patterns for 'bf16' models, layout [out, in].
"""
from __future__ import annotations

import numpy as np

from .numerics import bf16_bits_to_float, round_bf16


class DecoderOracle:
    """Causal decoder with an exact, append-only KV cache of committed rows."""

    def __init__(self, shape: dict, weights: dict, compute=np.float64,
                 row_invariant: bool = True, cache_weights: bool = True):
        self.s = dict(shape)
        self.L = shape["n_layers"]
        self.d = shape["d_model"]
        self.H = shape["n_heads"]
        self.G = shape["n_kv_heads"]
        self.hd = shape["head_dim"]
        self.V = shape["vocab"]
        self.eps = float(shape["rms_eps"])
        self.base = float(shape["rope_base"])
        self.bf16 = shape["dtype"] == "bf16"
        self.ct = compute
        self.row_invariant = row_invariant
        self.cache_weights = cache_weights
        self._raw = weights
        self._w = {}
        half = self.hd // 2
        # inverse frequencies base^(-2i/hd), i in [0, hd/2), in float64
        self.inv_freq = self.base ** (-(2.0 * np.arange(half, dtype=np.float64)) / self.hd)
        self.reset()

    # ---- weights -------------------------------------------------------
    def w(self, name):
        if name in self._w:
            return self._w[name]
        a = self._raw[name]
        if a.dtype == np.uint16:
            a = bf16_bits_to_float(a, self.ct)
        else:
            a = np.asarray(a, dtype=self.ct)
        if self.cache_weights:
            self._w[name] = a
        return a

    # ---- cache ---------------------------------------------------------
    def reset(self):
        self.K = [np.zeros((0, self.G, self.hd), self.ct) for _ in range(self.L)]
        self.Vc = [np.zeros((0, self.G, self.hd), self.ct) for _ in range(self.L)]

    @property
    def length(self) -> int:
        return self.K[0].shape[0]

    def truncate(self, n: int):
        self.K = [k[:n] for k in self.K]
        self.Vc = [v[:n] for v in self.Vc]

    def commit(self, kv_rows, rows):
        """Append the K/V of the listed in-step rows, in the given order."""
        rows = list(rows)
        for l in range(self.L):
            k, v = kv_rows[l]
            self.K[l] = np.concatenate([self.K[l], k[rows]], axis=0)
            self.Vc[l] = np.concatenate([self.Vc[l], v[rows]], axis=0)

    # ---- pieces --------------------------------------------------------
    def rnd(self, x):
        return round_bf16(x) if self.bf16 else x

    def mm(self, x, W):
        """x [R, in] times W^T (W is [out, in]); per row when row_invariant."""
        if self.row_invariant:
            return np.stack([W @ xr for xr in x]) if len(x) else np.zeros((0, W.shape[0]), self.ct)
        return x @ W.T

    def rmsnorm(self, h, gain):
        ms = np.mean(h * h, axis=-1, keepdims=True)
        return h / np.sqrt(ms + self.eps) * gain

    def rope(self, x, pos):
        """Rotate-half RoPE: x [R, heads, hd], pos [R]."""
        half = self.hd // 2
        ang = np.asarray(pos, dtype=np.float64)[:, None] * self.inv_freq[None, :]
        c = np.cos(ang).astype(self.ct)[:, None, :]
        s = np.sin(ang).astype(self.ct)[:, None, :]
        x1, x2 = x[..., :half], x[..., half:]
        return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)

    def attention(self, l, q, k, v, vis):
        """q [R, H, hd]; k, v [R, G, hd] of this step's rows; vis [R, R] bool."""
        R = q.shape[0]
        grp = self.H // self.G
        scale = 1.0 / np.sqrt(self.hd)
        out = np.zeros((R, self.H, self.hd), self.ct)
        Kp, Vp = self.K[l], self.Vc[l]
        if not self.row_invariant:
            # Same definition, vectorised over rows and heads (large shapes).
            keys = np.concatenate([Kp, k], axis=0)            # [C + R, G, hd]
            vals = np.concatenate([Vp, v], axis=0)
            C = Kp.shape[0]
            mask = np.concatenate([np.ones((R, C), bool), vis], axis=1)  # [R, C + R]
            for g in range(self.G):
                qg = q[:, g * grp:(g + 1) * grp, :]           # [R, grp, hd]
                s = np.einsum("rjd,td->jrt", qg, keys[:, g, :]) * self.ct(scale)
                s = np.where(mask[None], s, -np.inf)
                p = np.exp(s - s.max(axis=-1, keepdims=True))
                p = p / p.sum(axis=-1, keepdims=True)
                out[:, g * grp:(g + 1) * grp, :] = np.einsum("jrt,td->rjd", p, vals[:, g, :])
            return out
        for r in range(R):
            sel = np.nonzero(vis[r])[0]
            keys = np.concatenate([Kp, k[sel]], axis=0)      # [C + |vis|, G, hd]
            vals = np.concatenate([Vp, v[sel]], axis=0)
            for j in range(self.H):
                g = j // grp
                s = keys[:, g, :] @ q[r, j] * self.ct(scale)
                p = np.exp(s - s.max())
                p = p / p.sum()
                out[r, j] = p @ vals[:, g, :]
        return out

    # ---- forward -------------------------------------------------------
    def forward(self, tokens, pos, vis):
        """Logits of R in-step rows, plus their per-layer (k, v) for a commit.

        tokens [R] ids, pos [R] absolute positions, vis [R, R] bool (row r sees
        in-step row j iff vis[r, j]; the committed prefix is always visible).
        """
        tokens = np.asarray(tokens, dtype=np.int64)
        vis = np.asarray(vis, dtype=bool)
        R = len(tokens)
        H, G, hd = self.H, self.G, self.hd
        h = self.w("embed")[tokens].astype(self.ct)
        kv_rows = []
        for l in range(self.L):
            p = f"layers.{l}."
            xn = self.rmsnorm(h, self.w(p + "attn_norm"))
            q = self.mm(xn, self.w(p + "wq")).reshape(R, H, hd)
            k = self.mm(xn, self.w(p + "wk")).reshape(R, G, hd)
            v = self.mm(xn, self.w(p + "wv")).reshape(R, G, hd)
            q = self.rope(q, pos)
            k = self.rnd(self.rope(k, pos))     # the cache holds bf16 K/V
            v = self.rnd(v)
            kv_rows.append((k, v))
            o = self.attention(l, q, k, v, vis).reshape(R, H * hd)
            h = h + self.mm(o, self.w(p + "wo"))
            u = self.rmsnorm(h, self.w(p + "ffn_norm"))
            gt = self.mm(u, self.w(p + "w_gate"))
            up = self.mm(u, self.w(p + "w_up"))
            m = gt / (1.0 + np.exp(-gt)) * up
            h = h + self.mm(m, self.w(p + "w_down"))
        xf = self.rmsnorm(h, self.w("final_norm"))
        logits = self.mm(xf, self.w("lm_head"))
        return logits, kv_rows

    def prefill(self, tokens, chunk: int = 0):
        """Run and commit the prompt; returns the logits of its last row.

        ``chunk`` > 0 processes it in causal chunks (same result).
        """
        tokens = np.asarray(tokens)
        n = len(tokens)
        step = chunk if chunk > 0 else n
        logits = None
        for s in range(0, n, step):
            t = tokens[s:s + step]
            R = len(t)
            C = self.length
            logits, kv = self.forward(t, C + np.arange(R), np.tri(R, dtype=bool))
            self.commit(kv, range(R))
        return logits[-1]
