// The GEMM epilogues of the decoder's projections (shared by the
// weight-streaming kernel of gemm.hip and the many-row kernel of gemm_mr.hip):
// store, residual add (+ the next RMSNorm's input and row sums of squares),
// QKV with RoPE and the K/V cache write, SwiGLU, per-block vocabulary argmax.
#pragma once

#include "jf_device.h"
#include "jf_internal.h"

namespace jf {

// Operands of the residual-add epilogue that do not depend on the product
// (the residual and the next norm's gain), loaded when the kernel starts so
// that their latency hides behind the weight stream instead of adding a
// memory round trip after it (16-row step: down 29.8 -> 29.1 us, O 12.6 ->
// 12.1 us; the same for QKV's RoPE tables and cache pages, a chain of two
// loads at its start, made QKV 0.8 us slower).  Entry k of a thread is its
// k-th element e = tid + k nth of the R x cols outputs, the order of the
// epilogue's loops; elements past kEpiPre load in the epilogue as before.
// The values read are not written by the launch before its epilogue (the
// residual of a column tile is updated by that tile's epilogue alone).
constexpr int kEpiPre = 2;
struct EpiPre {
  float a[kEpiPre], b[kEpiPre];   // residual, gain
};
__device__ __forceinline__ void epilogue_prefetch(EpiPre& p, int cols, int col0, const Epi& ep, int tid, int nth,
                                                  int r0, int R) {
  if (ep.kind == EPI_RESID && ep.gain_next) {
#pragma unroll
    for (int k = 0; k < kEpiPre; ++k) {
      const int e = min(tid + k * nth, R * cols - 1);
      const int row = r0 + e / cols, col = col0 + e % cols;
      p.a[k] = ep.f32[(size_t)row * ep.ldf + col];
      p.b[k] = ep.gain_next[col];
    }
  }
}

// Runs on output rows r0 .. r0 + R - 1 of the columns col0 .. col0 + cols - 1
// (cols a multiple of 16, col0 of 32 for the SwiGLU pairs), held in
// tile[(row - r0) * tld + c], with threads tid = 0..nth-1 sharing the work.
// part_idx: the slot of these columns' per-row argmax keys (EPI_ARGMAX).
// pre: the operands epilogue_prefetch loaded for the same rows, columns and
// threads, or null.
template <typename T>
__device__ __forceinline__ void epilogue(float* tile, int tld, int cols, int col0, const Epi& ep, int part_idx,
                                         int tid, int nth, int r0, int R, const EpiPre* pre = nullptr) {
  if (ep.kind == EPI_RESID && ep.gain_next) {
    // Residual add, then the next RMSNorm's input: (new h) * gain as
    // activation planes, and the row's sum of squares over these columns.
    T* xg = reinterpret_cast<T*>(ep.xg);
    int k = 0;
    for (int e = tid; e < R * cols; e += nth, ++k) {
      const int row = r0 + e / cols, c = e % cols;
      const int col = col0 + c;
      float* dst = ep.f32 + (size_t)row * ep.ldf + col;
      const bool have = pre && k < kEpiPre;
      const float hn = (have ? pre->a[k] : *dst) + tile[(row - r0) * tld + c];
      *dst = hn;
      act_store<T>(xg + act_offset(row, col, ep.ldf), ep.xg_plane, hn * (have ? pre->b[k] : ep.gain_next[col]));
      tile[(row - r0) * tld + c] = hn * hn;
    }
    __syncthreads();
    for (int row = r0 + tid; row < r0 + R; row += nth) {
      float p = 0.f;
      for (int c = 0; c < cols; ++c) p += tile[(row - r0) * tld + c];
      ss_add(ep.ss_out, ep.ss_stride, row, p);
    }
  } else if (ep.kind == EPI_STORE || ep.kind == EPI_RESID) {
    for (int e = tid; e < R * cols; e += nth) {
      int row = r0 + e / cols, c = e % cols;
      float v = tile[(row - r0) * tld + c];
      float* dst = ep.f32 + (size_t)row * ep.ldf + (size_t)col0 + c;
      if (ep.kind == EPI_RESID) *dst += v; else *dst = v;
    }
  } else if (ep.kind == EPI_SWIGLU) {
    const int half_cols = cols / 2;  // features per block
    T* act = reinterpret_cast<T*>(ep.act);
    for (int e = tid; e < R * half_cols; e += nth) {
      int row = r0 + e / half_cols, f = e % half_cols;
      int p = f >> 4, c = f & 15;
      float gt = tile[(row - r0) * tld + (2 * p) * 16 + c];
      float up = tile[(row - r0) * tld + (2 * p + 1) * 16 + c];
      float s = gt / (1.0f + __expf(-gt));
      act_store<T>(act + act_offset(row, col0 / 2 + f, ep.act_k), ep.act_plane, s * up);
    }
  } else if (ep.kind == EPI_ARGMAX) {
    for (int row = r0 + tid; row < r0 + R; row += nth) {
      uint64_t best = 0;
      for (int c = 0; c < cols; ++c) {
        uint64_t k = argmax_key(tile[(row - r0) * tld + c], (uint32_t)(col0 + c));
        best = k > best ? k : best;
      }
      ep.part[(size_t)part_idx * ep.part_stride + row] = best;
    }
    if (ep.logits) {
      for (int e = tid; e < R * cols; e += nth) {
        int row = r0 + e / cols, c = e % cols;
        ep.logits[(size_t)row * ep.ldl + (size_t)col0 + c] = tile[(row - r0) * tld + c];
      }
    }
  } else if (ep.kind == EPI_QKV) {
    const int hd = ep.hd, half = hd >> 1, H = ep.H, G = ep.G;
    const int C = ep.state[0];
    T* q = reinterpret_cast<T*>(ep.q);
    T* kv = reinterpret_cast<T*>(ep.kv);
    const size_t page_elems = (size_t)2 * G * kPage * hd;
    for (int e = tid; e < R * cols; e += nth) {
      int row = r0 + e / cols, c = e % cols;
      int pr = col0 + c;              // packed row
      int head = pr / hd, w = pr - head * hd;
      float x = tile[(row - r0) * tld + c];
      float out;
      int dim;
      if (head < H + G) {
        int t = w >> 4, cc = w & 15;
        int i = 8 * t + (cc & 7);
        dim = cc < 8 ? i : half + i;
        float y = tile[(row - r0) * tld + (c ^ 8)];
        int pos = ep.pos[row];
        float cs = ep.rope_cos[(size_t)pos * half + i];
        float sn = ep.rope_sin[(size_t)pos * half + i];
        out = cc < 8 ? (x * cs - y * sn) : (x * cs + y * sn);
      } else {
        dim = w;
        out = x;
      }
      if (head < H) {
        act_store<T>(q + ((size_t)row * H + head) * hd + dim, ep.q_plane, out);
      } else {
        const T v = from_f32<T>(out);
        int slot = C + row;
        if (slot >= ep.max_ctx) {
          if (ep.flags) atomicOr(ep.flags, 2);
          continue;
        }
        int phys = ep.page_table[slot / kPage];
        T* page = kv + (size_t)phys * page_elems;
        int s = slot % kPage;
        if (head < H + G) {
          int kh = head - H;
          page[((size_t)kh * kPage + s) * hd + dim] = v;
        } else {
          int vh = head - H - G;
          page[(size_t)G * kPage * hd + ((size_t)vh * hd + dim) * kPage + s] = v;
        }
      }
    }
  }
}

}  // namespace jf
