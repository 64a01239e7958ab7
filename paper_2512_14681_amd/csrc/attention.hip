// Block-causal grouped-query attention of one Jacobi iteration (the attention
// inside the single forward pass of Eq. 3): every draft row attends to the
// whole committed prefix [0, C) and to the in-step rows its visibility mask
// marks (its ancestors and itself: a causal triangle for a linear draft, a
// tree for multi-block / recycled candidates, Sec. 3.2 and App. A Alg. 1).
//
// Work split: block (kv head g, 16-query tile, key split), or two query
// tiles per block for bf16 when query tiles x keys is large (each key chunk
// then serves both tiles).  The query rows of a KV head are its
// n_heads/n_kv_heads query heads times R rows, 16 per MFMA tile.  The key splits are laid out over the host's upper bound of
// C + R, so no address waits on the device's committed length (which only
// masks), and the split's page-table entries are read once into LDS.  The
// block's 4 waves take interleaved 32-key chunks with the next chunk's K/V
// loads in flight: S^T = K Q^T (keys x queries), an fp32 online softmax per
// query column, then O^T += V^T P^T.  The score tiles' rows are the chunk's
// keys in the order 8 (i / 4) + 4 kt + i % 4, so each lane's 8 softmax
// weights are 8 consecutive keys and its V^T operand is one contiguous load
// from the transposed V of the page.  For bf16, Q and P enter the matrix
// cores as two bf16 terms (hi + lo), keeping ~16 significant bits.  The
// waves' (max, sum, O) states merge in LDS; with several splits each block
// writes its partial state and k_attn_combine merges them in split order
// (deterministic).
#include <algorithm>

#include "jf_device.h"
#include "jf_internal.h"

namespace jf {

// Softmax weights as the B operand of the P.V contraction.  bf16: two terms,
// hi = bf16(p) and lo = bf16(p - hi), so the product keeps ~16 significant
// bits of the weights instead of 8.
template <typename T> struct PFrag;
template <> struct PFrag<bf16_t> { Frag<bf16_t> hi, lo; };
template <> struct PFrag<float> { Frag<float> v; };

__device__ __forceinline__ void split2(float a, float b, uint32_t& hi, uint32_t& lo) {
  hi = pack_bf16x2(a, b);
  lo = pack_bf16x2(a - __uint_as_float(hi << 16), b - __uint_as_float(hi & 0xFFFF0000u));
}
template <typename T> __device__ __forceinline__ PFrag<T> pfrag(const float* p);
template <> __device__ __forceinline__ PFrag<bf16_t> pfrag<bf16_t>(const float* p) {
  PFrag<bf16_t> f;
  split2(p[0], p[1], f.hi.v.x, f.lo.v.x);
  split2(p[2], p[3], f.hi.v.y, f.lo.v.y);
  split2(p[4], p[5], f.hi.v.z, f.lo.v.z);
  split2(p[6], p[7], f.hi.v.w, f.lo.v.w);
  return f;
}
template <> __device__ __forceinline__ PFrag<float> pfrag<float>(const float* p) {
  PFrag<float> f;
  f.v.lo = make_float4(p[0], p[1], p[2], p[3]);
  f.v.hi = make_float4(p[4], p[5], p[6], p[7]);
  return f;
}

constexpr int kAttnMaxPages = 256;  // pages of one key split (LDS page-table copy)

// Bits j0 .. j0 + 7 of a row's in-step visibility mask (kVisWords words;
// bits outside [0, kMaxRows) read as 0), branch-free.
__device__ __forceinline__ uint32_t vis_bits8(const uint64_t (&vw)[kVisWords], int j0) {
  const int jc = min(max(j0, 0), kMaxRows - 1);
  const int wi = jc >> 6, sh = jc & 63;
  uint64_t lo = 0, hi = 0;
#pragma unroll
  for (int i = 0; i < kVisWords; ++i) {
    lo = wi == i ? vw[i] : lo;
    hi = wi + 1 == i ? vw[i] : hi;
  }
  const uint64_t win = sh ? (lo >> sh) | (hi << (64 - sh)) : lo;
  uint32_t b = (uint32_t)win & 0xFFu;
  if (j0 < 0) b = j0 > -8 ? ((uint32_t)vw[0] << (-j0)) & 0xFFu : 0u;
  return j0 >= kMaxRows ? 0u : b;
}

// The visibility words of in-step row r: from vis ([R][kVisWords]), or the
// causal mask (rows 0..r) when vis is null.
__device__ __forceinline__ void vis_words(const uint64_t* vis, int r, uint64_t (&vw)[kVisWords]) {
#pragma unroll
  for (int i = 0; i < kVisWords; ++i) {
    if (vis) {
      vw[i] = vis[(size_t)r * kVisWords + i];
    } else {
      const int lo = i * 64;
      vw[i] = r < lo ? 0ull : (r - lo >= 63 ? ~0ull : ((2ull << (r - lo)) - 1ull));
    }
  }
}

// Low n bits set, n clamped to [0, 8].
__device__ __forceinline__ uint32_t low_bits8(int n) {
  return n >= 8 ? 0xFFu : (n <= 0 ? 0u : (1u << n) - 1u);
}

// QT query tiles per block (QT = 1, or 2 for many query tiles over long
// prefixes, see attn_plan): each key chunk's K and V^T fragments, loaded
// once, serve all QT tiles of the wave, so the keys are read once per QT
// tiles.  With QT = 2 one chunk is in
// flight per wave instead of two (the register budget of two blocks per
// CU), and the waves' states merge tile after tile.
template <typename T, int HD, int QT>
__global__ void __launch_bounds__(256, 2) k_attn(AttnArgs a) {
  constexpr int NW = 4;  // waves per block
  __shared__ float s_m[NW][16], s_l[NW][16];
  __shared__ float s_o[NW][16][HD + 4];
  __shared__ float s_f[NW][16], s_M[16], s_den[16];
  __shared__ int s_pt[kAttnMaxPages];
  const int g = blockIdx.x;
  const int tile0 = blockIdx.y * QT;
  const int split = blockIdx.z, S = gridDim.z;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int grp = a.H / a.G;
  const int R = a.R;
  const int nq = grp * R;
  // This split's keys [k0, k1), 32-aligned, from the host's bound of C + R.
  int per = (a.keys_ub + S - 1) / S;
  per = (per + 31) & ~31;
  const int k0 = split * per;
  const int k1 = min(a.keys_ub, k0 + per);
  const int p0 = k0 / kPage;
  const int np = k1 > k0 ? (k1 - 1) / kPage - p0 + 1 : 0;
  for (int i = threadIdx.x; i < np; i += 64 * NW) s_pt[i] = a.page_table[p0 + i];
  const int C = a.state ? a.state[0] : a.C_host;
  const int lim = min(k1, C + R);                 // keys at or past lim are not visible here
  // Chunks up to lim only: when the host's bound runs ahead of the committed
  // length, the masked keys past C + R are neither loaded nor computed, and a
  // split that starts past them does no work.
  const int nch = lim > k0 ? (lim - k0 + 31) / 32 : 0;

  const int ql = lane & 15, kg = lane >> 4;
  const T* kv = reinterpret_cast<const T*>(a.kv);
  const size_t page_elems = (size_t)2 * a.G * kPage * HD;
  const size_t k_off = (size_t)g * kPage * HD;
  const size_t vt_off = (size_t)a.G * kPage * HD + (size_t)g * HD * kPage;

  ActFrag<T> qf[QT][HD / 32];
  uint64_t vw[QT][kVisWords];
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    const int qr = (tile0 + t) * 16 + ql;
    const bool qvalid = qr < nq;
    const int hl = qvalid ? qr / R : 0;
    const int r = qvalid ? qr - hl * R : 0;
    const int head = g * grp + hl;
    const T* qp = reinterpret_cast<const T*>(a.q) + ((size_t)r * a.H + head) * HD + 8 * kg;
#pragma unroll
    for (int c = 0; c < HD / 32; ++c) qf[t][c] = qvalid ? act_load<T>(qp + 32 * c, a.q_plane) : act_zero<T>();
    vis_words(a.vis, r, vw[t]);
  }
  __syncthreads();  // s_pt

  const float scale = 1.4426950408889634f / sqrtf((float)HD);  // log2(e) / sqrt(hd)
  float m_run[QT], l_run[QT];
  f32x4_t o[QT][HD / 16];
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    m_run[t] = -INFINITY;
    l_run[t] = 0.f;
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) o[t][dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  }

  // One 32-key chunk (inside one page): K rows of the two score tiles, row i
  // of tile kt being key 8 (i / 4) + 4 kt + i % 4, and the V^T fragments
  // holding keys 8 kg .. 8 kg + 7 for dims dt * 16 + ql.
  auto load = [&](int c, Frag<T> (&kf)[2][HD / 32], Frag<T> (&vf)[HD / 16]) {
    const int kb = k0 + 32 * c;
    const T* page = kv + (size_t)s_pt[kb / kPage - p0] * page_elems;
    const int ko = kb % kPage;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      const T* kp = page + k_off + (size_t)(ko + 8 * (ql >> 2) + 4 * kt + (ql & 3)) * HD + 8 * kg;
#pragma unroll
      for (int cc = 0; cc < HD / 32; ++cc) kf[kt][cc] = frag_load<T>(kp + 32 * cc);
    }
    const T* vp = page + vt_off + (size_t)ql * kPage + ko + 8 * kg;
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) vf[dt] = frag_load<T>(vp + (size_t)dt * 16 * kPage);
  };
  auto compute = [&](int c, const Frag<T> (&kf)[2][HD / 32], const Frag<T> (&vf)[HD / 16]) {
    const int key0 = k0 + 32 * c + 8 * kg;  // key of p[0]; p[e] is key0 + e
#pragma unroll
    for (int t = 0; t < QT; ++t) {
      f32x4_t sc[2];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        if constexpr (sizeof(T) == 2) {
          // Q = hi + lo: four independent accumulation chains
          f32x4_t sh = f32x4_t{0.f, 0.f, 0.f, 0.f}, sl = sh;
#pragma unroll
          for (int cc = 0; cc < HD / 32; ++cc) {
            mfma(sh, kf[kt][cc], qf[t][cc].hi);
            mfma(sl, kf[kt][cc], qf[t][cc].lo);
          }
          sc[kt] = sh + sl;
        } else {
          sc[kt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int cc = 0; cc < HD / 32; ++cc) mfma(sc[kt], kf[kt][cc], qf[t][cc]);
        }
      }
      // visible: below lim, and either in the prefix or marked in the row's mask
      const uint32_t vis = low_bits8(lim - key0) & (low_bits8(C - key0) | vis_bits8(vw[t], key0 - C));
      float p[8];
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int e = kt * 4 + i;
          const float v = ((vis >> e) & 1u) ? sc[kt][i] * scale : -INFINITY;
          p[e] = v;
          mx = fmaxf(mx, v);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run[t], mx);
      // No branch: the MFMAs need every lane.  A query with nothing visible
      // yet keeps p = 0 and m = -inf.
      const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
      // exponents are <= 0 (or -inf): the bare hardware exp2 suffices
      const float alpha = __builtin_amdgcn_exp2f(m_run[t] - m_use);
      float psum = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        p[e] = __builtin_amdgcn_exp2f(p[e] - m_use);
        psum += p[e];
      }
      l_run[t] = l_run[t] * alpha + psum;
      m_run[t] = m_new;
      const PFrag<T> pf = pfrag<T>(p);
#pragma unroll
      for (int dt = 0; dt < HD / 16; ++dt) o[t][dt] *= alpha;
      if constexpr (sizeof(T) == 2) {
#pragma unroll
        for (int dt = 0; dt < HD / 16; ++dt) mfma(o[t][dt], vf[dt], pf.hi);
#pragma unroll
        for (int dt = 0; dt < HD / 16; ++dt) mfma(o[t][dt], vf[dt], pf.lo);
      } else {
#pragma unroll
        for (int dt = 0; dt < HD / 16; ++dt) mfma(o[t][dt], vf[dt], pf.v);
      }
    }
  };

  // Chunks wave, wave + NW, ... (mine of them).  QT = 1: two at a time, both
  // loads issued (unconditionally; past the end they re-read the last
  // chunk, unused), then both chunks consumed; the launch plan gives each
  // wave at most two chunks, i.e. one memory round trip.  QT = 2: one at a
  // time.
  const int mine = wave < nch ? (nch - wave + NW - 1) / NW : 0;
  if constexpr (QT == 1) {
    Frag<T> kA[2][HD / 32], kB[2][HD / 32];
    Frag<T> vA[HD / 16], vB[HD / 16];
    for (int i = 0; i < mine; i += 2) {
      const int cA = wave + i * NW, cB = min(cA + NW, nch - 1);
      load(cA, kA, vA);
      load(cB, kB, vB);
      compute(cA, kA, vA);
      if (i + 1 < mine) compute(cA + NW, kB, vB);
    }
  } else {
    Frag<T> kA[2][HD / 32];
    Frag<T> vA[HD / 16];
    for (int i = 0; i < mine; ++i) {
      const int c = wave + i * NW;
      load(c, kA, vA);
      compute(c, kA, vA);
    }
  }

  // Merge the waves' partial softmax states in LDS, one query tile at a
  // time: per query row the waves' weights 2^(m_w - M) and the sum once,
  // then every element.
  const size_t nrow = (size_t)R * a.H;
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    float lr = l_run[t];
    lr += __shfl_xor(lr, 16);
    lr += __shfl_xor(lr, 32);
    if (t > 0) __syncthreads();  // the previous tile's reads of s_o are done
    if (kg == 0) {
      s_m[wave][ql] = m_run[t];
      s_l[wave][ql] = lr;
    }
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) s_o[wave][ql][dt * 16 + 4 * kg + i] = o[t][dt][i];
    __syncthreads();
    if (threadIdx.x < 16) {
      const int q = threadIdx.x;
      float M = -INFINITY;
#pragma unroll
      for (int w = 0; w < NW; ++w) M = fmaxf(M, s_m[w][q]);
      float den = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        const float f = s_m[w][q] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(s_m[w][q] - M);
        s_f[w][q] = f;
        den += s_l[w][q] * f;
      }
      s_M[q] = M;
      s_den[q] = den;
    }
    __syncthreads();
    for (int e = threadIdx.x; e < 16 * HD; e += 64 * NW) {
      const int q = e / HD, dim = e - q * HD;
      const int qq = (tile0 + t) * 16 + q;
      if (qq >= nq) continue;
      float num = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) num += s_o[w][q][dim] * s_f[w][q];
      const int hq = qq / R, rr = qq - hq * R;
      if (S == 1) {
        act_store<T>(reinterpret_cast<T*>(a.out) + act_offset(rr, (g * grp + hq) * HD + dim, a.H * HD),
                     a.out_plane, num / s_den[q]);
      } else {
        const size_t qidx = (size_t)rr * a.H + g * grp + hq;
        a.o_part[((size_t)split * nrow + qidx) * HD + dim] = num;
        if (dim == 0) {
          a.ml_part[((size_t)split * nrow + qidx) * 2 + 0] = s_M[q];
          a.ml_part[((size_t)split * nrow + qidx) * 2 + 1] = s_den[q];
        }
      }
    }
  }
}

// Merges the splits' (max, sum, O) states of 16 query rows x 32 dims per
// block in split order; every load of a thread is issued at once (SMAX >= S
// splits unrolled, the extra ones re-reading split S - 1 with weight 0).
template <typename T, int HD, int SMAX>
__global__ void __launch_bounds__(256) k_attn_combine(AttnArgs a) {
  const int g = blockIdx.x, tile = blockIdx.y, d0 = blockIdx.z * 32;
  const int S = a.splits;
  const int grp = a.H / a.G, R = a.R, nq = grp * R;
  const size_t nrow = (size_t)R * a.H;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int e = threadIdx.x + 256 * j;
    const int q = e >> 5, dim = d0 + (e & 31);
    const int qq = min(tile * 16 + q, nq - 1);
    const int hq = qq / R, rr = qq - hq * R;
    const size_t qidx = (size_t)rr * a.H + g * grp + hq;
    float m[SMAX], l[SMAX], ov[SMAX];
#pragma unroll
    for (int sp = 0; sp < SMAX; ++sp) {
      const size_t i = (size_t)min(sp, S - 1) * nrow + qidx;
      m[sp] = a.ml_part[i * 2];
      l[sp] = a.ml_part[i * 2 + 1];
      ov[sp] = a.o_part[i * HD + dim];
    }
    float M = -INFINITY;
#pragma unroll
    for (int sp = 0; sp < SMAX; ++sp) M = fmaxf(M, m[sp]);
    float num = 0.f, den = 0.f;
#pragma unroll
    for (int sp = 0; sp < SMAX; ++sp) {
      const float w = (sp >= S || m[sp] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m[sp] - M);
      num += ov[sp] * w;
      den += l[sp] * w;
    }
    if (tile * 16 + q < nq)
      act_store<T>(reinterpret_cast<T*>(a.out) + act_offset(rr, (g * grp + hq) * HD + dim, a.H * HD), a.out_plane,
                   num / den);
  }
}

// ---- K/V pages shared through LDS (bf16, head_dim 128) ----------------------------
// Block (kv head g, query group, key split): up to 8 query tiles of the KV
// head, one per wave, over the split's keys.  Each 64-key page's K rows
// (16 KB) and V^T rows (16 KB) are staged in LDS once per block and read by
// every wave, so the keys are fetched once per query group instead of once
// per query tile.  Pages stream through a register ring two pages deep into
// two LDS buffers; the per-wave maths (S^T = K Q^T, online softmax, O^T +=
// V^T P^T, Q and P as hi + lo bf16 terms) is that of k_attn.  Each wave owns
// its query tile's state, so there is no merge across waves; with several
// splits the states go to the combine kernel.
//
// LDS layout, in 16-byte slots, swizzled so that a fragment read touches 16
// distinct bank groups per 16 lanes: K row r (a key) piece c at
// 16 r + (c ^ kswz(r)); V^T row d (a dim) piece p (8 keys) at
// 8 d + (p ^ ((d >> 1) & 7)).
constexpr int kAttnLdsHD = 128;
constexpr int kAttnLdsPieces = 16 * kAttnLdsHD / 512;  // 16-byte pieces a thread stages per page
constexpr int kAttnLdsPageElems = 2 * kPage * kAttnLdsHD;

__device__ __forceinline__ int kswz(int r) { return (r & 3) | (((r >> 3) & 3) << 2); }

__global__ void __launch_bounds__(512, 1) k_attn_lds(AttnArgs a) {
  constexpr int HD = kAttnLdsHD;
  extern __shared__ float lds_raw[];
  bf16_t* s_kv = reinterpret_cast<bf16_t*>(lds_raw);  // two pages: K (64 x HD) then V^T (HD x 64)
  __shared__ int s_pt[kAttnMaxPages];
  const int g = blockIdx.x, qgrp = blockIdx.y;
  const int split = blockIdx.z, S = gridDim.z;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int grp = a.H / a.G;
  const int R = a.R;
  const int nq = grp * R;
  const int ntiles = (nq + 15) / 16;
  const int tile = qgrp * a.qg + wave;
  const bool active = wave < a.qg && tile < ntiles;     // wave-uniform
  // this split's keys [k0, k1): whole pages, from the host's bound of C + R
  int per = (a.keys_ub + S - 1) / S;
  per = (per + kPage - 1) / kPage * kPage;
  const int k0 = split * per;
  const int k1 = min(a.keys_ub, k0 + per);
  const int p0 = k0 / kPage;
  const int np = k1 > k0 ? (k1 - 1) / kPage - p0 + 1 : 0;
  for (int i = threadIdx.x; i < np; i += 512) s_pt[i] = a.page_table[p0 + i];
  const int C = a.state ? a.state[0] : a.C_host;
  const int lim = min(k1, C + R);                       // keys at or past lim are not visible here
  const int npg = lim > k0 ? (lim - k0 + kPage - 1) / kPage : 0;  // pages with visible keys

  const int ql = lane & 15, kg = lane >> 4;
  const bf16_t* kv = reinterpret_cast<const bf16_t*>(a.kv);
  const size_t page_elems = (size_t)2 * a.G * kPage * HD;
  const size_t k_off = (size_t)g * kPage * HD;
  const size_t vt_off = (size_t)a.G * kPage * HD + (size_t)g * HD * kPage;

  ActFrag<bf16_t> qf[HD / 32];
  uint64_t vw[kVisWords];
  int r = 0, head = 0;
  {
    const int qr = tile * 16 + ql;
    const bool qvalid = active && qr < nq;
    const int hl = qvalid ? qr / R : 0;
    r = qvalid ? qr - hl * R : 0;
    head = g * grp + hl;
    const bf16_t* qp = reinterpret_cast<const bf16_t*>(a.q) + ((size_t)r * a.H + head) * HD + 8 * kg;
#pragma unroll
    for (int c = 0; c < HD / 32; ++c) qf[c] = qvalid ? act_load<bf16_t>(qp + 32 * c, a.q_plane) : act_zero<bf16_t>();
    vis_words(a.vis, r, vw);
  }
  __syncthreads();  // s_pt
  {
    // first use of the query fragments and masks ahead of the page loop, so
    // that the compiler waits for their loads here: waited for inside the
    // loop, their count would merge with the page ring's and drain it
    uint32_t use = 0;
#pragma unroll
    for (int c = 0; c < HD / 32; ++c)
      use |= qf[c].hi.v.x | qf[c].hi.v.y | qf[c].hi.v.z | qf[c].hi.v.w | qf[c].lo.v.x | qf[c].lo.v.y |
             qf[c].lo.v.z | qf[c].lo.v.w;
#pragma unroll
    for (int i = 0; i < kVisWords; ++i) use |= (uint32_t)vw[i] | (uint32_t)(vw[i] >> 32);
    asm volatile("" ::"v"(use));
  }

  // page i of the split into ring registers (clamped: a short split re-reads
  // its last page) and from there into LDS buffer b
  auto load_page = [&](u32x4_t (&st)[kAttnLdsPieces], int i) {
    const bf16_t* page = kv + (size_t)s_pt[min(i, np - 1)] * page_elems;
#pragma unroll
    for (int j = 0; j < kAttnLdsPieces; ++j) {
      const int e = threadIdx.x + 512 * j;
      const bf16_t* src = j < kAttnLdsPieces / 2 ? page + k_off + (size_t)e * 8
                                                 : page + vt_off + (size_t)(e - 8 * HD) * 8;
      st[j] = *reinterpret_cast<const u32x4_t*>(src);
    }
  };
  auto store_page = [&](const u32x4_t (&st)[kAttnLdsPieces], int b) {
    u32x4_t* dst = reinterpret_cast<u32x4_t*>(s_kv + (size_t)b * kAttnLdsPageElems);
#pragma unroll
    for (int j = 0; j < kAttnLdsPieces; ++j) {
      const int e = threadIdx.x + 512 * j;
      if (j < kAttnLdsPieces / 2) {
        const int rr = e >> 4, c = e & 15;
        dst[16 * rr + (c ^ kswz(rr))] = st[j];
      } else {
        const int ev = e - 8 * HD, d = ev >> 3, pc = ev & 7;
        dst[8 * HD + 8 * d + (pc ^ ((d >> 1) & 7))] = st[j];
      }
    }
  };

  const float scale = 1.4426950408889634f / sqrtf((float)HD);  // log2(e) / sqrt(hd)
  float m_run = -INFINITY, l_run = 0.f;
  f32x4_t o[HD / 16];
#pragma unroll
  for (int dt = 0; dt < HD / 16; ++dt) o[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // one 32-key half h of the page in LDS buffer b (keys kp0 + 32 h ..)
  auto compute = [&](int b, int kp0, int h) {
    const uint4* lk = reinterpret_cast<const uint4*>(s_kv + (size_t)b * kAttnLdsPageElems);
    const uint4* lv = lk + 8 * HD;
    Frag<bf16_t> kf[2][HD / 32], vf[HD / 16];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      const int rr = 32 * h + 8 * (ql >> 2) + 4 * kt + (ql & 3);
#pragma unroll
      for (int cc = 0; cc < HD / 32; ++cc) kf[kt][cc].v = lk[16 * rr + ((kg + 4 * cc) ^ kswz(rr))];
    }
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) {
      const int d = dt * 16 + ql, pc = 4 * h + kg;
      vf[dt].v = lv[8 * d + (pc ^ ((d >> 1) & 7))];
    }
    const int key0 = kp0 + 32 * h + 8 * kg;  // key of p[0]; p[e] is key0 + e
    f32x4_t sc[2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      f32x4_t sh = f32x4_t{0.f, 0.f, 0.f, 0.f}, sl = sh;
#pragma unroll
      for (int cc = 0; cc < HD / 32; ++cc) {
        mfma(sh, kf[kt][cc], qf[cc].hi);
        mfma(sl, kf[kt][cc], qf[cc].lo);
      }
      sc[kt] = sh + sl;
    }
    const uint32_t vis = low_bits8(lim - key0) & (low_bits8(C - key0) | vis_bits8(vw, key0 - C));
    float p[8];
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int e = kt * 4 + i;
        const float v = ((vis >> e) & 1u) ? sc[kt][i] * scale : -INFINITY;
        p[e] = v;
        mx = fmaxf(mx, v);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
    float psum = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      p[e] = __builtin_amdgcn_exp2f(p[e] - m_use);
      psum += p[e];
    }
    l_run = l_run * alpha + psum;
    m_run = m_new;
    const PFrag<bf16_t> pf = pfrag<bf16_t>(p);
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) o[dt] *= alpha;
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) mfma(o[dt], vf[dt], pf.hi);
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) mfma(o[dt], vf[dt], pf.lo);
  };

  // pages through a two-deep register ring and two LDS buffers; waves
  // without a query tile stage pages and keep the barriers in step
  if (npg > 0) {
    u32x4_t ring[2][kAttnLdsPieces];
    load_page(ring[0], 0);
    load_page(ring[1], 1);
    store_page(ring[0], 0);
    __syncthreads();
    // two pages an iteration, so the ring slots are static, and no condition
    // inside: the loads and stores run unconditionally (past the end: the
    // split's last page again, unused), so the compiler's count of
    // outstanding loads stays exact
    int i = 0;
    for (; i + 2 <= npg; i += 2) {
#pragma unroll
      for (int slot = 0; slot < 2; ++slot) {
        if (active) {
          compute(slot, k0 + (i + slot) * kPage, 0);
          compute(slot, k0 + (i + slot) * kPage, 1);
        }
        load_page(ring[slot], i + slot + 2);
        store_page(ring[slot ^ 1], slot ^ 1);
        __syncthreads();
      }
    }
    if (i < npg && active) {                               // an odd last page, in buffer 0
      compute(0, k0 + i * kPage, 0);
      compute(0, k0 + i * kPage, 1);
    }
  }
  if (!active) return;

  // the tile's state: (max, sum) per query, O^T columns per lane
  float lr = l_run;
  lr += __shfl_xor(lr, 16);
  lr += __shfl_xor(lr, 32);
  const int qr = tile * 16 + ql;
  if (qr >= nq) return;
  const size_t nrow = (size_t)R * a.H;
  const size_t qidx = (size_t)r * a.H + head;
  if (S == 1) {
    const float inv = 1.f / lr;
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        act_store<bf16_t>(reinterpret_cast<bf16_t*>(a.out) + act_offset(r, head * HD + dt * 16 + 4 * kg + i, a.H * HD),
                          a.out_plane, o[dt][i] * inv);
  } else {
    float* op = a.o_part + ((size_t)split * nrow + qidx) * HD + 4 * kg;
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt)
      *reinterpret_cast<float4*>(op + dt * 16) = make_float4(o[dt][0], o[dt][1], o[dt][2], o[dt][3]);
    if (kg == 0) {
      a.ml_part[((size_t)split * nrow + qidx) * 2 + 0] = m_run;
      a.ml_part[((size_t)split * nrow + qidx) * 2 + 1] = lr;
    }
  }
}

// Launch shape: key splits such that each of a block's 4 waves gets at most
// kAttnChunksPerWave 32-key chunks (one memory round trip), at most
// kAttnMaxSplits splits, and at most kAttnMaxPages - 2 pages per split.
// Two query tiles per block from this many (query tiles x keys) on: measured
// on the attention workloads (28 q / 4 kv heads of 128), two tiles won at
// 57k and more (P = 8192, n = 16: -17%; P = 2048, n = 64: -15%) and lost at
// 29k (P = 2048, n = 32: +5%), where the one-chunk-in-flight loop costs more
// than the halved key traffic saves.
constexpr long kAttnQt2Work = 50000;

// The LDS-shared form: query groups of up to 8 tiles (balanced), and key
// splits of at least 3 pages up to about 256 blocks in all.  Splits of one
// or two pages cost more in partials and their merge than the extra blocks
// gain inside a step (1024-token prefix: 64 rows 5182 -> 5066 us, 128 rows
// 7171 -> 6943 us; 192 and 256 rows unchanged; the attention workload at
// P = 2048 / n = 64 21.7 -> 21.2 us, at P = 512 / n = 64 15.6 -> 16.6 us).
static void attn_lds_plan(AttnArgs& a) {
  const int ntiles = ((a.H / a.G) * a.R + 15) / 16;
  const int groups = (ntiles + 7) / 8;
  a.qg = (ntiles + groups - 1) / groups;
  const int pages = (a.keys_ub + kPage - 1) / kPage;
  int s = (256 + a.G * groups - 1) / (a.G * groups);
  s = std::min(s, (pages + 2) / 3);
  const int min_s = (pages + kAttnMaxPages - 3) / (kAttnMaxPages - 2);
  a.splits = std::max(1, std::min(kAttnMaxSplits, std::max(s, min_s)));
}

// The LDS-shared form from this many query tiles per KV head, or this much
// (query tiles x keys) work.  Measured on the attention workloads (28 q / 4
// kv heads of 128, us, one-tile form -> LDS-shared form): P = 512: n = 16
// 12.8 -> 13.1, n = 64 17.2 -> 15.3; P = 2048: n = 16 15.0 -> 20.5, n = 32
// 19.1 -> 21.9, n = 64 26.9 -> 21.2; P = 8192: n = 16 27.9 -> 27.0, n = 32
// 35.5 -> 29.2, n = 64 47.7 -> 35.2; the n = 16 step's attention (C ~ 1100)
// 14.1 -> 17.3.  With few query tiles the LDS-shared form needs many key
// splits to spread the keys, and merging them costs more than sharing the
// pages saves.
constexpr int kAttnLdsTiles = 20;
constexpr long kAttnLdsWork = 50000;

void attn_plan(AttnArgs& a) {
  a.qg = 0;
  const long qtiles = ((long)(a.H / a.G) * a.R + 15) / 16;
  if (a.lds_ok && a.hd == kAttnLdsHD && (qtiles >= kAttnLdsTiles || qtiles * a.keys_ub >= kAttnLdsWork)) {
    attn_lds_plan(a);
    return;
  }
  const int chunks = (a.keys_ub + 31) / 32;
  a.waves = 4;
  int s = (chunks + kAttnChunksPerWave * a.waves - 1) / (kAttnChunksPerWave * a.waves);
  const int min_s = (a.keys_ub + (kAttnMaxPages - 2) * kPage - 1) / ((kAttnMaxPages - 2) * kPage);
  if (s < min_s) s = min_s;
  a.splits = s < 1 ? 1 : (s > kAttnMaxSplits ? kAttnMaxSplits : s);
  // Many query tiles over long prefixes: two query tiles per block share
  // each key chunk.
  a.qt = qtiles >= 2 && qtiles * a.keys_ub >= kAttnQt2Work ? 2 : 1;
}

template <typename T, int HD>
static hipError_t launch_attn_t(const AttnArgs& a, hipStream_t st) {
  const int nq = (a.H / a.G) * a.R;
  const int ntiles = (nq + 15) / 16;
  // two query tiles per block: bf16 only (measured there; the fp32 kernel
  // has no registers to spare)
  bool two = false;
  if constexpr (sizeof(T) == 2) two = a.qt == 2;
  if (two) {
    if constexpr (sizeof(T) == 2)
      hipLaunchKernelGGL((k_attn<T, HD, 2>), dim3(a.G, (ntiles + 1) / 2, a.splits), dim3(256), 0, st, a);
  } else {
    hipLaunchKernelGGL((k_attn<T, HD, 1>), dim3(a.G, ntiles, a.splits), dim3(256), 0, st, a);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.splits == 1) return e;
  const dim3 grid(a.G, ntiles, HD / 32);
  if (a.splits <= 4)
    hipLaunchKernelGGL((k_attn_combine<T, HD, 4>), grid, dim3(256), 0, st, a);
  else if (a.splits <= 8)
    hipLaunchKernelGGL((k_attn_combine<T, HD, 8>), grid, dim3(256), 0, st, a);
  else if (a.splits <= 16)
    hipLaunchKernelGGL((k_attn_combine<T, HD, 16>), grid, dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL((k_attn_combine<T, HD, 32>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

static hipError_t launch_checked(int dtype, const AttnArgs& a, hipStream_t st) {
  if (a.R < 1 || a.R > kMaxRows || a.splits < 1 || a.splits > kAttnMaxSplits || a.H % a.G || a.keys_ub < a.R ||
      a.keys_ub > a.max_ctx)
    return hipErrorInvalidValue;
  // the LDS page-table copy must hold one split's pages
  {
    int per = (a.keys_ub + a.splits - 1) / a.splits;
    per = (per + 31) & ~31;
    if (per / kPage + 2 > kAttnMaxPages) return hipErrorInvalidValue;
  }
  if (a.splits > 1 && (!a.o_part || !a.ml_part)) return hipErrorInvalidValue;
  switch (a.hd) {
    case 32: return dtype == 1 ? launch_attn_t<bf16_t, 32>(a, st) : launch_attn_t<float, 32>(a, st);
    case 64: return dtype == 1 ? launch_attn_t<bf16_t, 64>(a, st) : launch_attn_t<float, 64>(a, st);
    case 128: return dtype == 1 ? launch_attn_t<bf16_t, 128>(a, st) : launch_attn_t<float, 128>(a, st);
    default: return hipErrorInvalidValue;
  }
}

// The two-tile form (bf16): its key splits are halved while the grid has
// more than kAttnQt2Blocks blocks.  Measured on the attention workloads at
// P = 8192 (32 splits from the one-tile plan): the wider combine of many
// splits costs more than the extra blocks gain once the grid is that large.
// Best were 16 splits at n = 16 (256 blocks, -9%) and n = 32 (448 blocks,
// -29%), 8 at n = 64 (448 blocks, -41%); 256 or 512 as the bound each lost
// one of them.
constexpr int kAttnQt2Blocks = 448;

static hipError_t launch_attn_lds(const AttnArgs& a, hipStream_t st) {
  if (a.R < 1 || a.R > kMaxRows || a.splits < 1 || a.splits > kAttnMaxSplits || a.H % a.G || a.keys_ub < a.R ||
      a.keys_ub > a.max_ctx || a.qg < 1 || a.qg > 8 || a.hd != kAttnLdsHD)
    return hipErrorInvalidValue;
  {
    int per = (a.keys_ub + a.splits - 1) / a.splits;
    per = (per + kPage - 1) / kPage * kPage;
    if (per / kPage + 1 > kAttnMaxPages) return hipErrorInvalidValue;
  }
  if (a.splits > 1 && (!a.o_part || !a.ml_part)) return hipErrorInvalidValue;
  const int ntiles = ((a.H / a.G) * a.R + 15) / 16;
  const int groups = (ntiles + a.qg - 1) / a.qg;
  hipLaunchKernelGGL(k_attn_lds, dim3(a.G, groups, a.splits), dim3(512),
                     (size_t)2 * kAttnLdsPageElems * sizeof(bf16_t), st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.splits == 1) return e;
  constexpr int HD = kAttnLdsHD;
  const dim3 grid(a.G, ntiles, HD / 32);
  if (a.splits <= 4)
    hipLaunchKernelGGL((k_attn_combine<bf16_t, HD, 4>), grid, dim3(256), 0, st, a);
  else if (a.splits <= 8)
    hipLaunchKernelGGL((k_attn_combine<bf16_t, HD, 8>), grid, dim3(256), 0, st, a);
  else if (a.splits <= 16)
    hipLaunchKernelGGL((k_attn_combine<bf16_t, HD, 16>), grid, dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL((k_attn_combine<bf16_t, HD, 32>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_attention(int dtype, const AttnArgs& a, hipStream_t st) {
  if (a.qg > 0) return dtype == 1 ? launch_attn_lds(a, st) : hipErrorInvalidValue;
  if (dtype == 1 && a.qt == 2) {
    AttnArgs b = a;
    const long pairs = ((long)((a.H / a.G) * a.R + 15) / 16 + 1) / 2;
    const int min_s = (a.keys_ub + (kAttnMaxPages - 2) * kPage - 1) / ((kAttnMaxPages - 2) * kPage);
    while (b.splits > 1 && (long)a.G * pairs * b.splits > kAttnQt2Blocks && (b.splits + 1) / 2 >= min_s)
      b.splits = (b.splits + 1) / 2;
    return launch_checked(dtype, b, st);
  }
  return launch_checked(dtype, a, st);
}

}  // namespace jf
