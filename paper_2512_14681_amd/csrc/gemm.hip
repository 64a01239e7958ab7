// Small-M weight-streaming GEMM for the decoder's projections:
//   Y[R][N] = X[R][K] * W[N][K]^T,  R = rows of one Jacobi step (1..256).
//
// The step is bound by reading W once (Sec. 4.2 / App. D of the paper: the
// extra draft rows of a Jacobi iteration are nearly free until the hardware
// knee), so the kernel is organised around streaming the packed weight
// blocks: one block of 16 output rows x 128 inputs is 4 KB (bf16) that a
// wave reads with 4 fully coalesced 1 KB loads, then issues 4 MFMA steps per
// 16-row tile of X.  A workgroup owns NT adjacent 16-column tiles and splits
// K over WK waves; the waves' partial tiles are summed in LDS in a fixed
// order (deterministic) and the epilogue runs on the reduced tile.
#include "jf_device.h"
#include "jf_internal.h"

namespace jf {

template <typename T>
__device__ __forceinline__ void epilogue(const float* tile, int tld, int RT, int NT, const Epi& ep) {
  const int tid = threadIdx.x, nth = blockDim.x;
  const int ng = blockIdx.x;
  const int cols = NT * 16;
  const int R = ep.R;
  if (ep.kind == EPI_STORE || ep.kind == EPI_RESID) {
    for (int e = tid; e < R * cols; e += nth) {
      int row = e / cols, c = e - row * cols;
      float v = tile[row * tld + c];
      float* dst = ep.f32 + (size_t)row * ep.ldf + (size_t)ng * cols + c;
      if (ep.kind == EPI_RESID) *dst += v; else *dst = v;
    }
  } else if (ep.kind == EPI_SWIGLU) {
    const int half_cols = cols / 2;  // features per block
    T* act = reinterpret_cast<T*>(ep.act);
    for (int e = tid; e < R * half_cols; e += nth) {
      int row = e / half_cols, f = e - row * half_cols;
      int p = f >> 4, c = f & 15;
      float gt = tile[row * tld + (2 * p) * 16 + c];
      float up = tile[row * tld + (2 * p + 1) * 16 + c];
      float s = gt / (1.0f + __expf(-gt));
      act[(size_t)row * ep.lda + (size_t)ng * half_cols + f] = from_f32<T>(s * up);
    }
  } else if (ep.kind == EPI_ARGMAX) {
    for (int row = tid; row < R; row += nth) {
      uint64_t best = 0;
      for (int c = 0; c < cols; ++c) {
        uint64_t k = argmax_key(tile[row * tld + c], (uint32_t)(ng * cols + c));
        best = k > best ? k : best;
      }
      ep.part[(size_t)ng * ep.part_stride + row] = best;
    }
    if (ep.logits) {
      for (int e = tid; e < R * cols; e += nth) {
        int row = e / cols, c = e - row * cols;
        ep.logits[(size_t)row * ep.ldl + (size_t)ng * cols + c] = tile[row * tld + c];
      }
    }
  } else if (ep.kind == EPI_QKV) {
    const int hd = ep.hd, half = hd >> 1, H = ep.H, G = ep.G;
    const int C = ep.state[0];
    T* q = reinterpret_cast<T*>(ep.q);
    T* kv = reinterpret_cast<T*>(ep.kv);
    const size_t page_elems = (size_t)2 * G * kPage * hd;
    for (int e = tid; e < R * cols; e += nth) {
      int row = e / cols, c = e - row * cols;
      int pr = ng * cols + c;         // packed row
      int head = pr / hd, w = pr - head * hd;
      float x = tile[row * tld + c];
      float out;
      int dim;
      if (head < H + G) {
        int t = w >> 4, cc = w & 15;
        int i = 8 * t + (cc & 7);
        dim = cc < 8 ? i : half + i;
        float y = tile[row * tld + (c ^ 8)];
        int pos = ep.pos[row];
        float cs = ep.rope_cos[(size_t)pos * half + i];
        float sn = ep.rope_sin[(size_t)pos * half + i];
        out = cc < 8 ? (x * cs - y * sn) : (x * cs + y * sn);
      } else {
        dim = w;
        out = x;
      }
      T v = from_f32<T>(out);
      if (head < H) {
        q[((size_t)row * H + head) * hd + dim] = v;
      } else {
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

template <typename T, int RT, int NT, int WK>
__global__ void __launch_bounds__(64 * WK)
k_gemm(const T* __restrict__ X, int ldx, const T* __restrict__ Wp, int KC, Epi ep) {
  extern __shared__ float lds[];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int ng = blockIdx.x;
  const int R = ep.R;
  const int kc0 = (KC * wave) / WK, kc1 = (KC * (wave + 1)) / WK;

  f32x4_t acc[RT][NT];
#pragma unroll
  for (int mt = 0; mt < RT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int lrow = lane & 15;
  const int koff = (lane >> 4) * 32;
  const T* wb = Wp + (size_t)(ng * NT) * KC * kBlockElems + lane * 8;


  for (int kc = kc0; kc < kc1; ++kc) {
    Frag<T> b[NT][4];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        b[nt][j] = frag_load_nt<T>(wb + ((size_t)nt * KC + kc) * kBlockElems + j * 512);
#pragma unroll
    for (int mt = 0; mt < RT; ++mt) {
      const int row = mt * 16 + lrow;
      const T* xp = X + (size_t)row * ldx + kc * 128 + koff;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        Frag<T> a = row < R ? frag_load<T>(xp + j * 8) : frag_zero<T>();
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) mfma(acc[mt][nt], a, b[nt][j]);
      }
    }
  }

  // Output tile [RT*16][NT*16] in LDS after the partials (if any).
  const int tld = NT * 16 + 1;
  constexpr int PART = RT * NT * 256;  // floats per wave partial
  float* tile = lds + (WK > 1 ? WK * PART : 0);
  if (WK == 1) {
#pragma unroll
    for (int mt = 0; mt < RT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          tile[(mt * 16 + 4 * (lane >> 4) + i) * tld + nt * 16 + lrow] = acc[mt][nt][i];
  } else {
    float* mine = lds + wave * PART;
#pragma unroll
    for (int mt = 0; mt < RT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i) mine[((mt * NT + nt) * 4 + i) * 64 + lane] = acc[mt][nt][i];
    __syncthreads();
    for (int e = threadIdx.x; e < PART; e += 64 * WK) {
      float s = 0.f;
#pragma unroll
      for (int w = 0; w < WK; ++w) s += lds[w * PART + e];
      int l = e & 63, i = (e >> 6) & 3, mn = e >> 8;
      int mt = mn / NT, nt = mn - mt * NT;
      tile[(mt * 16 + 4 * (l >> 4) + i) * tld + nt * 16 + (l & 15)] = s;
    }
  }
  __syncthreads();
  epilogue<T>(tile, tld, RT, NT, ep);
}

static int round_rt(int R) {
  int rt = (R + 15) / 16;
  if (rt <= 2) return rt;
  if (rt <= 4) return 4;
  if (rt <= 8) return 8;
  if (rt <= 12) return 12;
  return 16;
}

static size_t lds_bytes(int RT, int NT, int WK) {
  size_t part = (size_t)RT * NT * 256;
  size_t tile = (size_t)RT * 16 * (NT * 16 + 1);
  return ((WK > 1 ? WK * part : 0) + tile) * sizeof(float);
}

void gemm_plan(GemmShape& s, int epi_kind) {
  const int KC = s.K / 128;
  const int RT = round_rt(s.R);
  s.NT = (epi_kind == EPI_SWIGLU) ? 2 : 1;
  const int groups = s.N / (16 * s.NT);
  // Aim for >= ~2048 waves in flight (256 CUs) while keeping >= 2 K-blocks
  // per wave, and stay inside 64 KB of LDS for the partial tiles.
  int wk = 1;
  while (wk < 16 && groups * wk < 2048 && KC / (wk * 2) >= 2) wk *= 2;
  while (wk > 1 && lds_bytes(RT, s.NT, wk) > 65536) wk /= 2;
  s.WK = wk;
}

size_t gemm_blocks(const GemmShape& s) { return (size_t)s.N / (16 * s.NT); }

template <typename T, int RT, int NT, int WK>
static hipError_t launch_t(const void* X, int ldx, const void* Wp, const GemmShape& s, const Epi& ep,
                           hipStream_t st) {
  size_t lds = lds_bytes(RT, NT, WK);
  dim3 grid((unsigned)(s.N / (16 * NT))), block(64 * WK);
  hipLaunchKernelGGL((k_gemm<T, RT, NT, WK>), grid, block, lds, st, reinterpret_cast<const T*>(X),
                     ldx, reinterpret_cast<const T*>(Wp), s.K / 128, ep);
  return hipGetLastError();
}

template <typename T, int RT, int NT>
static hipError_t launch_wk(const void* X, int ldx, const void* Wp, const GemmShape& s, const Epi& ep,
                            hipStream_t st) {
  switch (s.WK) {
    case 1: return launch_t<T, RT, NT, 1>(X, ldx, Wp, s, ep, st);
    case 2: return launch_t<T, RT, NT, 2>(X, ldx, Wp, s, ep, st);
    case 4: if constexpr (RT * NT <= 12) return launch_t<T, RT, NT, 4>(X, ldx, Wp, s, ep, st); break;
    case 8: if constexpr (RT * NT <= 6) return launch_t<T, RT, NT, 8>(X, ldx, Wp, s, ep, st); break;
    case 16: if constexpr (RT * NT <= 2) return launch_t<T, RT, NT, 16>(X, ldx, Wp, s, ep, st); break;
    default: break;
  }
  return hipErrorInvalidValue;
}

template <typename T, int RT>
static hipError_t launch_nt(const void* X, int ldx, const void* Wp, const GemmShape& s, const Epi& ep,
                            hipStream_t st) {
  if (s.NT == 1) return launch_wk<T, RT, 1>(X, ldx, Wp, s, ep, st);
  if (s.NT == 2) return launch_wk<T, RT, 2>(X, ldx, Wp, s, ep, st);
  return hipErrorInvalidValue;
}

template <typename T>
static hipError_t launch_rt(const void* X, int ldx, const void* Wp, const GemmShape& s, const Epi& ep,
                            hipStream_t st) {
  switch (round_rt(s.R)) {
    case 1: return launch_nt<T, 1>(X, ldx, Wp, s, ep, st);
    case 2: return launch_nt<T, 2>(X, ldx, Wp, s, ep, st);
    case 4: return launch_nt<T, 4>(X, ldx, Wp, s, ep, st);
    case 8: return launch_nt<T, 8>(X, ldx, Wp, s, ep, st);
    case 12: return launch_nt<T, 12>(X, ldx, Wp, s, ep, st);
    case 16: return launch_nt<T, 16>(X, ldx, Wp, s, ep, st);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_gemm(int dtype, const void* X, int ldx, const void* Wp, const GemmShape& s,
                       const Epi& ep, hipStream_t st) {
  if (s.R < 1 || s.R > 256 || s.K % 128 || s.N % (16 * s.NT)) return hipErrorInvalidValue;
  if (lds_bytes(round_rt(s.R), s.NT, s.WK) > 65536) return hipErrorInvalidValue;
  return dtype == 1 ? launch_rt<bf16_t>(X, ldx, Wp, s, ep, st)
                    : launch_rt<float>(X, ldx, Wp, s, ep, st);
}

// ---- weight packing ------------------------------------------------------------
template <typename T>
__global__ void k_pack(int rows, int cols, const T* s0, const T* s1, const T* s2, const T* s3,
                       const int32_t* rowmap, T* dst) {
  const int KC = cols / 128;
  const size_t total = (size_t)rows * cols;
  for (size_t o = (size_t)blockIdx.x * blockDim.x + threadIdx.x; o < total;
       o += (size_t)gridDim.x * blockDim.x) {
    size_t blk = o / kBlockElems;
    int r = (int)(o - blk * kBlockElems);
    int j = r >> 9, lane = (r >> 3) & 63, e = r & 7;
    int nt = (int)(blk / KC), kc = (int)(blk - (size_t)nt * KC);
    int row = nt * 16 + (lane & 15);
    int col = kc * 128 + 32 * (lane >> 4) + 8 * j + e;
    int src = 0, srow = row;
    if (rowmap) {
      int32_t m = rowmap[row];
      src = m >> 24;
      srow = m & 0xFFFFFF;
    }
    const T* sp = src == 0 ? s0 : src == 1 ? s1 : src == 2 ? s2 : s3;
    dst[o] = sp[(size_t)srow * cols + col];
  }
}

hipError_t launch_pack(int dtype, int rows, int cols, const void* const* srcs, int n_srcs,
                       const int32_t* d_rowmap, void* dst, hipStream_t st) {
  if (rows % 16 || cols % 128 || n_srcs < 1 || n_srcs > 4) return hipErrorInvalidValue;
  const void* s[4] = {srcs[0], n_srcs > 1 ? srcs[1] : srcs[0], n_srcs > 2 ? srcs[2] : srcs[0],
                      n_srcs > 3 ? srcs[3] : srcs[0]};
  dim3 grid(4096), block(256);
  if (dtype == 1)
    hipLaunchKernelGGL(k_pack<bf16_t>, grid, block, 0, st, rows, cols, (const bf16_t*)s[0],
                       (const bf16_t*)s[1], (const bf16_t*)s[2], (const bf16_t*)s[3], d_rowmap,
                       (bf16_t*)dst);
  else
    hipLaunchKernelGGL(k_pack<float>, grid, block, 0, st, rows, cols, (const float*)s[0],
                       (const float*)s[1], (const float*)s[2], (const float*)s[3], d_rowmap,
                       (float*)dst);
  return hipGetLastError();
}

}  // namespace jf
