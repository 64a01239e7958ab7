"""Host-side decoding loops over the libjf C ABI.

Each iteration is one ABI step (forward + argmax + acceptance on the GPU),
one commit, and one small device-to-host read (the 16-byte step result and
the row argmaxes) that the loop needs for control.  The loops follow the
paper's procedures:

* ``generate_ar``        -- Eq. 1, one token per forward (n = 1 steps).
* ``generate_jacobi``    -- Eq. 3 with commits; block mode (Eq. 4) or the
                            running window of Sec. 4.2.
* ``generate_multiblock`` -- multi-block decoding with rejection recycling,
                            App. A Alg. 1, with the readings documented in
                            the design doc (same policy as the CPU oracle's).
* ``collect_trajectories`` -- block-mode decoding that records every Jacobi
                            iterate of every block on the device (the
                            trajectories J of Sec. 2.1 that Jacobi Forcing
                            trains on).
"""
from __future__ import annotations

import math

import numpy as np

from . import jf

_MASK = (1 << 64) - 1
_GOLD = 0x9E3779B97F4A7C15


def pad_token(seed: int, pos: int, vocab: int) -> int:
    """Draft-initialisation token for absolute position pos: the first
    splitmix64 output for state seed ^ (pos * 0x9E3779B97F4A7C15), mod V."""
    z = ((seed ^ ((pos * _GOLD) & _MASK)) + _GOLD) & _MASK
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK
    return (z ^ (z >> 31)) % vocab


class Decoder:
    """Drives one jf.Model (one sequence)."""

    def __init__(self, model: jf.Model):
        import torch
        self.t = torch
        self.m = model
        self.V = model.V
        R = model.cfg.max_rows
        dev = "cuda"
        i32 = torch.int32
        self.d_tokens = torch.zeros(R, dtype=i32, device=dev)
        self.d_next = torch.zeros(R, dtype=i32, device=dev)
        # result (4 ints), argmax (R), per-segment counts and the committed
        # path adjacent in one buffer: one device-to-host read per iteration
        S = jf.JF_MAX_SEGMENTS
        self.d_io = torch.zeros(4 + R + S + R, dtype=i32, device=dev)
        self.d_result = self.d_io[:4]
        self.d_argmax = self.d_io[4:4 + R]
        self.d_seg = self.d_io[4 + R:4 + R + S]
        self.d_path = self.d_io[4 + R + S:]
        self._seg_at, self._path_at = 4 + R, 4 + R + S
        # pinned staging of host-built drafts: the upload is ordered on the
        # stream and needs no synchronisation (the buffer is rewritten only
        # after the next result read, when that upload has long completed)
        self.h_stage = torch.zeros(R, dtype=i32, pin_memory=True)
        self.d_pending = torch.zeros(1, dtype=i32, device=dev)
        self.trace = []

    def length(self) -> int:
        return self.m.jf_kv_length()

    def reset(self):
        self.m.jf_kv_truncate(0)
        self.trace = []

    def prefill(self, prompt) -> int:
        toks = self.t.as_tensor(np.asarray(prompt, dtype=np.int32), device="cuda")
        self.m.jf_prefill(toks, self.d_pending)
        return int(self.d_pending.cpu()[0])

    def _put(self, buf, values):
        k = len(values)
        self.h_stage[:k].copy_(self.t.from_numpy(np.asarray(values, dtype=np.int32)))
        buf[:k].copy_(self.h_stage[:k], non_blocking=True)

    # ---- Eq. 1 -----------------------------------------------------------------
    def generate_ar(self, prompt, max_new: int):
        p = self.prefill(prompt)
        out = [p]
        while len(out) < max_new:
            self._put(self.d_tokens, [p])
            self.m.jf_jacobi_step(self.d_tokens, 1, 0, 0, self.d_argmax, self.d_result, self.d_next)
            self.m.jf_commit_kv(None, self.d_result)
            p = int(self.d_io[:5].cpu()[2])
            out.append(p)
        return out

    # ---- Eq. 3 / Eq. 4 / running window ------------------------------------------
    def generate_jacobi(self, prompt, n: int, max_new: int, mode: str = "window",
                        pad_seed: int = 2, logits=None):
        """Returns (tokens, accept counts).  ``logits`` (optional list) gets,
        per iteration, the fp32 logits of the rows whose predictions were
        committed: rows 0 .. a-1, row j predicting the token after draft[j]."""
        m, V = self.m, self.V
        p = self.prefill(prompt)
        C = len(prompt)
        out, accepts = [], []
        cur = 0          # rows of the current draft (block mode shrinks it)
        d_logits = None
        while len(out) < max_new:
            if cur == 0:
                cur = n
                self._put(self.d_tokens, [p] + [pad_token(pad_seed, C + i, V) for i in range(1, n)])
            if logits is not None:
                d_logits = self.t.empty((cur, V), dtype=self.t.float32, device="cuda")
            left = max_new - len(out)
            m.jf_jacobi_step(self.d_tokens, cur, 1 if mode == "window" else 0, pad_seed,
                             self.d_argmax, self.d_result, self.d_tokens, d_logits)
            m.jf_commit_kv(None, self.d_result, left)
            io = self.d_io[:4 + cur].cpu().numpy()
            a = min(int(io[0]), left)
            g = io[4:4 + cur]
            out += [p] + [int(x) for x in g[:a - 1]]
            accepts.append(a)
            self.trace.append(dict(R=cur, a=a, g=g.copy()))
            if logits is not None:
                logits.append(d_logits[:a].cpu().numpy())
            p = int(g[a - 1])
            C += a
            if mode == "block":
                cur -= a
        return out[:max_new], accepts

    # ---- Sec. 2.1 trajectories ----------------------------------------------------
    def collect_trajectories(self, prompt, n: int, n_blocks: int, pad_seed: int = 2):
        """Block-mode Jacobi decoding (Eq. 4) of n_blocks blocks of n tokens
        after the prompt, recording every iterate on the device
        (jf_trajectory_record).  y^(0) of a block is [p, pad, ...]; each step
        feeds the block's unaccepted tail and commits the accepted rows, and
        the block ends when its last step accepts every row it fed (then
        y^(k) = y^(k-1)).  Returns (d_traj, lengths): d_traj is a device
        int32 tensor [n_blocks][n + 1][n] (-1 in unused points) and block b's
        trajectory is d_traj[b, :lengths[b]]."""
        t, m, V = self.t, self.m, self.V
        if n > m.cfg.max_rows:
            raise ValueError(f"block of {n} tokens exceeds max_rows {m.cfg.max_rows}")
        d_traj = t.full((n_blocks, n + 1, n), -1, dtype=t.int32, device="cuda")
        lengths = np.zeros(n_blocks, np.int32)
        p = self.prefill(prompt)
        C = len(prompt)
        for b in range(n_blocks):
            self._put(self.d_tokens, [p] + [pad_token(pad_seed, C + i, V) for i in range(1, n)])
            d_traj[b, 0].copy_(self.d_tokens[:n])
            cur, j = n, 0
            while cur > 0:
                m.jf_jacobi_step(self.d_tokens, cur, 0, pad_seed, self.d_argmax, self.d_result,
                                 self.d_tokens)
                jf.trajectory_record(d_traj[b, j], self.d_argmax, n, cur, d_traj[b, j + 1],
                                     stream=m.stream)
                m.jf_commit_kv(None, self.d_result)
                io = self.d_io[:4 + cur].cpu().numpy()
                a = int(io[0])
                p = int(io[4 + a - 1])
                cur -= a
                j += 1
            lengths[b] = j + 1
            C += n
        return d_traj, lengths

    # ---- App. A Alg. 1 ------------------------------------------------------------
    def generate_multiblock(self, prompt, n: int, K: int, r: float, max_new: int,
                            n_cand: int = 8, cand_len: int = 16, pool_cap: int = 64,
                            pad_seed: int = 2, logits=None):
        """Multi-block decoding with rejection recycling; returns (tokens, trace).
        ``logits`` (optional list) gets, per iteration, the fp32 logits of the
        committed path's rows path[0 .. a-1], row path[j] predicting the
        token committed after it."""
        m, V = self.m, self.V
        thr = math.ceil(r * n)
        p = self.prefill(prompt)
        C = len(prompt)
        # blocks: [start, accepted list, draft list]; index 0 is real-active
        blocks = [[C, [], [p] + [pad_token(pad_seed, C + i, V) for i in range(1, n)]]]
        pool = []
        out, trace = [], []
        while len(out) < max_new:
            ra = blocks[0]
            toks = list(ra[2])
            segs = [(0, len(ra[2]), -1, jf.JF_ROLE_RA, 1)]
            tail = len(toks) - 1
            for b in blocks[1:]:
                rows = b[1] + b[2]
                segs.append((len(toks), len(rows), tail, jf.JF_ROLE_PSEUDO, len(b[1])))
                toks += rows
                tail = len(toks) - 1
            picked = []
            for e in pool[::-1]:
                if len(picked) == n_cand:
                    break
                if e[0] != p:
                    continue
                L = min(len(e), cand_len, len(ra[2]))
                body = tuple(e[1:L])
                if body and tuple(e[:L]) != tuple(ra[2][:L]) and body not in picked:
                    picked.append(body)
            for body in picked:
                segs.append((len(toks), len(body), 0, jf.JF_ROLE_CAND, 0))
                toks += list(body)
            R = len(toks)
            self._put(self.d_tokens, toks)
            d_logits = None
            if logits is not None:
                d_logits = self.t.empty((R, V), dtype=self.t.float32, device="cuda")
            m.jf_multiblock_step(self.d_tokens, R, segs, self.d_argmax, self.d_seg, self.d_result,
                                 self.d_path, d_logits)
            left = max_new - len(out)
            m.jf_commit_kv(self.d_path, self.d_result, left)
            io = self.d_io.cpu().numpy()
            seg_m = io[self._seg_at:self._seg_at + len(segs)]
            path = io[self._path_at:self._path_at + int(io[0])]
            g = io[4:4 + R]
            a = min(int(io[0]), left)
            win = int(io[1])
            committed = [toks[i] for i in path[:a]]
            out += committed
            if logits is not None:
                logits.append(d_logits[self.t.as_tensor(path[:a].astype(np.int64), device="cuda")].cpu().numpy())
            trace.append(dict(R=R, segs=list(segs), m=[int(x) for x in seg_m], winner=win, a=a,
                              committed=committed))
            p_new = int(g[path[a - 1]])
            if len(out) >= max_new:
                break
            C += a
            # real-active tail and pool
            a_ra = 1 + int(seg_m[0])
            rej = ra[2][a_ra:]
            if len(rej) >= 2:
                pool.append(tuple(rej))
                if len(pool) > pool_cap:
                    del pool[0]
            ra[1] += committed
            left_blk = n - len(ra[1])
            s0 = segs[win]
            branch = list(range(s0[1])) if win == 0 else [0] + list(range(s0[0], s0[0] + s0[1]))
            nxt = [int(g[i]) for i in branch[a - 1:]]
            while len(nxt) < left_blk:
                nxt.append(pad_token(pad_seed, C + len(nxt), V))
            ra[2] = nxt[:left_blk]
            # pseudo-active blocks: grow accepted prefix, Jacobi-update the rest
            for bi, b in enumerate(blocks[1:], start=1):
                first, _, att, _, vf = segs[bi]
                mb = int(seg_m[bi])
                b[1] += b[2][:mb]
                newd = []
                for i in range(len(b[1]), n):
                    row = first + i
                    par = att if i == 0 else row - 1
                    newd.append(int(g[par]))
                b[2] = newd
            # spawn
            if len(blocks) < K and any(len(b[1]) >= thr for b in blocks):
                start = blocks[-1][0] + n
                d = list(ra[2])
                while len(d) < n:
                    d.append(pad_token(pad_seed, start + len(d), V))
                blocks.append([start, [], d[:n]])
            # promote
            if len(ra[1]) >= n:
                if len(blocks) > 1:
                    b = blocks[1]
                    rows = b[1] + b[2]
                    blocks = [[b[0], [], [p_new] + rows[1:n]]] + blocks[2:]
                else:
                    blocks = [[C, [], [p_new] + [pad_token(pad_seed, C + i, V) for i in range(1, n)]]]
            p = p_new
        return out[:max_new], trace
