// Block-causal grouped-query attention of one Jacobi iteration (the attention
// inside the single forward pass of Eq. 3): every draft row attends to the
// whole committed prefix [0, C) and to the in-step rows its visibility mask
// marks (its ancestors and itself: a causal triangle for a linear draft, a
// tree for multi-block / recycled candidates, Sec. 3.2 and App. A Alg. 1).
//
// Work split: block (kv head g, key split, group of 4 query tiles).  The
// query rows of a KV head are its n_heads/n_kv_heads query heads times R
// rows, taken 16 at a time as one MFMA tile per wave.  Keys are visited 32 at
// a time:  S^T = K Q^T (keys x queries) with K rows read straight from the
// page, an fp32 online softmax per query column, then O^T += V^T P^T with V
// stored transposed in the page, so both operands are contiguous loads and P
// never leaves registers.  Splits write (max, sum, unnormalised O) partials
// that k_attn_combine merges.
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
  const int g = blockIdx.x;
  const int split = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int tile = blockIdx.z * 4 + wave;
  const int grp = a.H / a.G;
  const int R = a.R;
  const int nq = grp * R;
  if (tile * 16 >= nq) return;
  const int C = a.state ? a.state[0] : a.C_host;
  const int total = C + R;
  int per = (total + a.splits - 1) / a.splits;
  per = (per + 31) & ~31;
  const int k0 = split * per;
  const int k1 = min(total, k0 + per);

  const int ql = lane & 15, kg = lane >> 4;
  const int qr = tile * 16 + ql;
  const bool qvalid = qr < nq;
  const int hl = qvalid ? qr / R : 0;
  const int r = qvalid ? qr - hl * R : 0;
  const int head = g * grp + hl;

  const T* kv = reinterpret_cast<const T*>(a.kv);
  const size_t page_elems = (size_t)2 * a.G * kPage * HD;
  const size_t vt_off = (size_t)a.G * kPage * HD + (size_t)g * HD * kPage;

  Frag<T> qf[HD / 32];
  const T* qp = reinterpret_cast<const T*>(a.q) + ((size_t)r * a.H + head) * HD + 8 * kg;
#pragma unroll
  for (int c = 0; c < HD / 32; ++c) qf[c] = qvalid ? frag_load<T>(qp + 32 * c) : frag_zero<T>();

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

  for (int kb = k0; kb < k1; kb += 32) {
    f32x4_t s[2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      s[kt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      int key = min(kb + kt * 16 + ql, total - 1);
      const T* kp = kv + (size_t)a.page_table[key / kPage] * page_elems +
                    ((size_t)g * kPage + key % kPage) * HD + 8 * kg;
#pragma unroll
      for (int c = 0; c < HD / 32; ++c) mfma(s[kt], frag_load<T>(kp + 32 * c), qf[c]);
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
        float v = vis ? s[kt][i] * scale : -INFINITY;
        p[kt * 4 + i] = v;
        mx = fmaxf(mx, v);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    // No branch here: the MFMAs below need every lane of the wave.  A query
    // with nothing visible yet keeps p = 0 and m = -inf.
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    const float alpha = exp2f(m_run - m_use);  // m_run = -inf gives 0
    float psum = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      p[e] = exp2f(p[e] - m_use);
      psum += p[e];
    }
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) o[dt] *= alpha;
    const Frag<T> pf = frag_from_p<T>(p);
    const T* vpage = kv + (size_t)a.page_table[kb / kPage] * page_elems + vt_off + (kb % kPage);
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) {
      const T* vp = vpage + (size_t)(dt * 16 + ql) * kPage + 4 * kg;
      mfma(o[dt], frag_load_4x2<T>(vp, vp + 16), pf);
    }
  }
  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);

  if (!qvalid) return;
  const size_t qidx = (size_t)r * a.H + head;
  const size_t nrow = (size_t)R * a.H;
  if (kg == 0) {
    a.ml_part[((size_t)split * nrow + qidx) * 2 + 0] = m_run;
    a.ml_part[((size_t)split * nrow + qidx) * 2 + 1] = l_run;
  }
  float* op = a.o_part + ((size_t)split * nrow + qidx) * HD;
#pragma unroll
  for (int dt = 0; dt < HD / 16; ++dt)
#pragma unroll
    for (int i = 0; i < 4; ++i) op[dt * 16 + 4 * kg + i] = o[dt][i];
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
  reinterpret_cast<T*>(a.out)[qidx * HD + dim] = from_f32<T>(num / den);
}

int attn_splits(int max_keys) {
  int s = (max_keys + 127) / 128;
  return s < 1 ? 1 : (s > 32 ? 32 : s);
}

template <typename T, int HD>
static hipError_t launch_attn_t(const AttnArgs& a, hipStream_t st) {
  const int nq = (a.H / a.G) * a.R;
  const int ntiles = (nq + 15) / 16;
  dim3 grid(a.G, a.splits, (ntiles + 3) / 4), block(256);
  hipLaunchKernelGGL((k_attn<T, HD>), grid, block, 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
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
