// Block-causal grouped-query attention of one Jacobi iteration (the attention
// inside the single forward pass of Eq. 3): every draft row attends to the
// whole committed prefix [0, C) and to the in-step rows its visibility mask
// marks (its ancestors and itself: a causal triangle for a linear draft, a
// tree for multi-block / recycled candidates, Sec. 3.2 and App. A Alg. 1).
//
// Work split: block (kv head g, 16-query tile, key split).  The query rows
// of a KV head are its n_heads/n_kv_heads query heads times R rows, 16 per
// MFMA tile.  The block's 4 waves take interleaved 32-key chunks with the
// next chunk's K/V loads in flight:  S^T = K Q^T (keys x queries) with K rows
// read straight from the page, an fp32 online softmax per query column, then
// O^T += V^T P^T with V stored transposed in the page, so both operands are
// contiguous loads and P never leaves registers (for bf16, P is split into
// two bf16 terms so the weights keep ~16 significant bits).  The waves' (max, sum, O)
// states merge in LDS; a context longer than one split writes partials that
// k_attn_combine merges.
#include "jf_device.h"
#include "jf_internal.h"

namespace jf {

template <typename T> __device__ __forceinline__ Frag<T> frag_from_p(const float* p);
template <> __device__ __forceinline__ Frag<bf16_t> frag_from_p<bf16_t>(const float* p) {
  Frag<bf16_t> f;
  f.v.x = (uint32_t)f32_to_bf16(p[0]) | ((uint32_t)f32_to_bf16(p[1]) << 16);
  f.v.y = (uint32_t)f32_to_bf16(p[2]) | ((uint32_t)f32_to_bf16(p[3]) << 16);
  f.v.z = (uint32_t)f32_to_bf16(p[4]) | ((uint32_t)f32_to_bf16(p[5]) << 16);
  f.v.w = (uint32_t)f32_to_bf16(p[6]) | ((uint32_t)f32_to_bf16(p[7]) << 16);
  return f;
}
template <> __device__ __forceinline__ Frag<float> frag_from_p<float>(const float* p) {
  Frag<float> f;
  f.lo = make_float4(p[0], p[1], p[2], p[3]);
  f.hi = make_float4(p[4], p[5], p[6], p[7]);
  return f;
}

// Two runs of 4 consecutive elements (the transposed-V operand).
template <typename T> __device__ __forceinline__ Frag<T> frag_load_4x2(const T* a, const T* b);
template <> __device__ __forceinline__ Frag<bf16_t> frag_load_4x2<bf16_t>(const bf16_t* a,
                                                                       const bf16_t* b) {
  uint2 x = *reinterpret_cast<const uint2*>(a), y = *reinterpret_cast<const uint2*>(b);
  Frag<bf16_t> f; f.v = make_uint4(x.x, x.y, y.x, y.y); return f;
}
template <> __device__ __forceinline__ Frag<float> frag_load_4x2<float>(const float* a,
                                                                     const float* b) {
  Frag<float> f;
  f.lo = *reinterpret_cast<const float4*>(a);
  f.hi = *reinterpret_cast<const float4*>(b);
  return f;
}

template <typename T, int HD>
__global__ void __launch_bounds__(256) k_attn(AttnArgs a) {
  constexpr int NW = 4;  // waves per block
  __shared__ float s_m[NW][16], s_l[NW][16];
  __shared__ float s_o[NW][16][HD + 4];
  const int g = blockIdx.x;
  const int tile = blockIdx.y;
  const int split = blockIdx.z;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int grp = a.H / a.G;
  const int R = a.R;
  const int nq = grp * R;
  const int C = a.state ? a.state[0] : a.C_host;
  const int total = C + R;
  int per = (total + a.splits - 1) / a.splits;
  per = (per + 31) & ~31;
  const int k0 = split * per;
  const int k1 = min(total, k0 + per);
  const int nch = k1 > k0 ? (k1 - k0 + 31) / 32 : 0;

  const int ql = lane & 15, kg = lane >> 4;
  const int qr = tile * 16 + ql;
  const bool qvalid = qr < nq;
  const int hl = qvalid ? qr / R : 0;
  const int r = qvalid ? qr - hl * R : 0;
  const int head = g * grp + hl;

  const T* kv = reinterpret_cast<const T*>(a.kv);
  const size_t page_elems = (size_t)2 * a.G * kPage * HD;
  const size_t vt_off = (size_t)a.G * kPage * HD + (size_t)g * HD * kPage;

  ActFrag<T> qf[HD / 32];
  const T* qp = reinterpret_cast<const T*>(a.q) + ((size_t)r * a.H + head) * HD + 8 * kg;
#pragma unroll
  for (int c = 0; c < HD / 32; ++c) qf[c] = qvalid ? act_load<T>(qp + 32 * c, a.q_plane) : act_zero<T>();

  uint64_t vw[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if (a.vis) {
      vw[i] = a.vis[r * 4 + i];
    } else {  // causal: rows 0..r
      int lo = i * 64;
      vw[i] = r < lo ? 0ull : (r - lo >= 63 ? ~0ull : ((2ull << (r - lo)) - 1ull));
    }
  }

  const float scale = 1.4426950408889634f / sqrtf((float)HD);  // log2(e) / sqrt(hd)
  float m_run = -INFINITY, l_run = 0.f;
  f32x4_t o[HD / 16];
#pragma unroll
  for (int dt = 0; dt < HD / 16; ++dt) o[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // K rows of the two 16-key tiles and the transposed-V fragments of one
  // 32-key chunk.
  auto load = [&](int c, Frag<T> (&kf)[2][HD / 32], Frag<T> (&vf)[HD / 16]) {
    const int kb = k0 + 32 * c;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      int key = min(kb + kt * 16 + ql, total - 1);
      const T* kp = kv + (size_t)a.page_table[key / kPage] * page_elems +
                    ((size_t)g * kPage + key % kPage) * HD + 8 * kg;
#pragma unroll
      for (int cc = 0; cc < HD / 32; ++cc) kf[kt][cc] = frag_load<T>(kp + 32 * cc);
    }
    const T* vpage = kv + (size_t)a.page_table[kb / kPage] * page_elems + vt_off + (kb % kPage);
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) {
      const T* vp = vpage + (size_t)(dt * 16 + ql) * kPage + 4 * kg;
      vf[dt] = frag_load_4x2<T>(vp, vp + 16);
    }
  };
  auto compute = [&](int c, const Frag<T> (&kf)[2][HD / 32], const Frag<T> (&vf)[HD / 16]) {
    const int kb = k0 + 32 * c;
    f32x4_t sc[2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      sc[kt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int cc = 0; cc < HD / 32; ++cc) mfma(sc[kt], kf[kt][cc], qf[cc]);
    }
    float p[8];
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        int key = kb + kt * 16 + 4 * kg + i;
        bool vis = key < k1;
        if (vis && key >= C) {
          int j = key - C;
          vis = (vw[j >> 6] >> (j & 63)) & 1ull;
        }
        float v = vis ? sc[kt][i] * scale : -INFINITY;
        p[kt * 4 + i] = v;
        mx = fmaxf(mx, v);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    // No branch: the MFMAs need every lane.  A query with nothing visible
    // yet keeps p = 0 and m = -inf.
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    const float alpha = exp2f(m_run - m_use);
    float psum = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      p[e] = exp2f(p[e] - m_use);
      psum += p[e];
    }
    l_run = l_run * alpha + psum;
    m_run = m_new;
    const Frag<T> pf = frag_from_p<T>(p);
    if constexpr (sizeof(T) == 2) {
      // bf16 operands: P = hi + lo with both halves bf16, so the product
      // keeps ~16 significant bits of the softmax weights instead of 8.
      float lo[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) lo[e] = p[e] - bf16_to_f32(f32_to_bf16(p[e]));
      const Frag<T> pl = frag_from_p<T>(lo);
#pragma unroll
      for (int dt = 0; dt < HD / 16; ++dt) {
        o[dt] *= alpha;
        mfma(o[dt], vf[dt], pf);
        mfma(o[dt], vf[dt], pl);
      }
    } else {
#pragma unroll
      for (int dt = 0; dt < HD / 16; ++dt) {
        o[dt] *= alpha;
        mfma(o[dt], vf[dt], pf);
      }
    }
  };

  // Chunks wave, wave + NW, ... with the next chunk's K/V in flight.
  Frag<T> kA[2][HD / 32], kB[2][HD / 32];
  Frag<T> vA[HD / 16], vB[HD / 16];
  int c = wave;
  if (c < nch) load(c, kA, vA);
  while (c < nch) {
    if (c + NW < nch) load(c + NW, kB, vB);
    compute(c, kA, vA);
    c += NW;
    if (c >= nch) break;
    if (c + NW < nch) load(c + NW, kA, vA);
    compute(c, kB, vB);
    c += NW;
  }
  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);

  // Merge the waves' partial softmax states in LDS.
  if (kg == 0) {
    s_m[wave][ql] = m_run;
    s_l[wave][ql] = l_run;
  }
#pragma unroll
  for (int dt = 0; dt < HD / 16; ++dt)
#pragma unroll
    for (int i = 0; i < 4; ++i) s_o[wave][ql][dt * 16 + 4 * kg + i] = o[dt][i];
  __syncthreads();
  const size_t nrow = (size_t)R * a.H;
  for (int e = threadIdx.x; e < 16 * HD; e += 64 * NW) {
    const int q = e / HD, dim = e - q * HD;
    const int qq = tile * 16 + q;
    if (qq >= nq) continue;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < NW; ++w) M = fmaxf(M, s_m[w][q]);
    float num = 0.f, den = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      if (s_m[w][q] == -INFINITY) continue;
      const float f = exp2f(s_m[w][q] - M);
      num += s_o[w][q][dim] * f;
      den += s_l[w][q] * f;
    }
    const int hq = qq / R, rr = qq - hq * R;
    const size_t qidx = (size_t)rr * a.H + g * grp + hq;
    if (a.splits == 1) {
      act_store<T>(reinterpret_cast<T*>(a.out) + act_offset(rr, (g * grp + hq) * HD + dim, a.H * HD), a.out_plane,
                   num / den);
    } else {
      a.o_part[((size_t)split * nrow + qidx) * HD + dim] = num;
      if (dim == 0) {
        a.ml_part[((size_t)split * nrow + qidx) * 2 + 0] = M;
        a.ml_part[((size_t)split * nrow + qidx) * 2 + 1] = den;
      }
    }
  }
}

template <typename T, int HD>
__global__ void k_attn_combine(AttnArgs a) {
  const size_t qidx = blockIdx.x;
  const int dim = threadIdx.x;
  const size_t nrow = (size_t)a.R * a.H;
  float M = -INFINITY;
  for (int s = 0; s < a.splits; ++s) M = fmaxf(M, a.ml_part[((size_t)s * nrow + qidx) * 2]);
  float num = 0.f, den = 0.f;
  for (int s = 0; s < a.splits; ++s) {
    float m = a.ml_part[((size_t)s * nrow + qidx) * 2];
    if (m == -INFINITY) continue;
    float w = exp2f(m - M);
    num += a.o_part[((size_t)s * nrow + qidx) * HD + dim] * w;
    den += a.ml_part[((size_t)s * nrow + qidx) * 2 + 1] * w;
  }
  const int rr = (int)(qidx / a.H), head = (int)(qidx - (size_t)rr * a.H);
  act_store<T>(reinterpret_cast<T*>(a.out) + act_offset(rr, head * HD + dim, a.H * HD), a.out_plane, num / den);
}

// Number of key splits: enough blocks to cover the machine (>= 256 blocks
// over kv heads x query tiles x splits), at least 128 keys per split, and at
// most 2048 keys per split.  The split ranges are derived on the device from
// the committed length, so any count is correct.
int attn_splits(int max_keys, int n_kv_heads, int n_qtiles) {
  int blocks = n_kv_heads * n_qtiles;
  int s = (256 + blocks - 1) / blocks;
  int by_len = max_keys / 128;
  if (s > by_len) s = by_len;
  int min_s = (max_keys + 2047) / 2048;
  if (s < min_s) s = min_s;
  return s < 1 ? 1 : (s > 32 ? 32 : s);
}

template <typename T, int HD>
static hipError_t launch_attn_t(const AttnArgs& a, hipStream_t st) {
  const int nq = (a.H / a.G) * a.R;
  const int ntiles = (nq + 15) / 16;
  dim3 grid(a.G, ntiles, a.splits), block(256);
  hipLaunchKernelGGL((k_attn<T, HD>), grid, block, 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.splits == 1) return e;
  hipLaunchKernelGGL((k_attn_combine<T, HD>), dim3(a.R * a.H), dim3(HD), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_attention(int dtype, const AttnArgs& a, hipStream_t st) {
  if (a.R < 1 || a.R > 256 || a.splits < 1 || a.H % a.G) return hipErrorInvalidValue;
  switch (a.hd) {
    case 32: return dtype == 1 ? launch_attn_t<bf16_t, 32>(a, st) : launch_attn_t<float, 32>(a, st);
    case 64: return dtype == 1 ? launch_attn_t<bf16_t, 64>(a, st) : launch_attn_t<float, 64>(a, st);
    case 128: return dtype == 1 ? launch_attn_t<bf16_t, 128>(a, st) : launch_attn_t<float, 128>(a, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace jf
