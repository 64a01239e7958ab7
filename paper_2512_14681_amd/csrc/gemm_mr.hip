// Many-row GEMM of the decoder's wide projections (gate/up and the LM
// head), Y[R][N] = X[R][K] * W[N][K]^T, for the wide Jacobi steps:
// multi-block drafts with recycled candidates (Sec. 3.2, App. A Alg. 1), the
// packed training forward and the block-size sweeps: 33 .. 64 rows in one
// chunk, more as 128-row chunks.
//
// What bounds these launches is the bytes each compute unit requests (its
// share of the weights plus the activations it re-reads), so the kernel asks
// for every weight byte exactly once per compute unit and re-reads the
// activations as rarely as the register file allows:
//   * a workgroup of 8 waves owns a column group (one pass of up to 8B
//     16-column tiles; wider groups take several passes) and all K;
//   * the activations of all the chunk's rows for half a 128-wide K-block
//     (2 of its 4 fragment steps) are staged in LDS, double-buffered, and
//     read by every wave; each wave multiplies all row tiles by its own
//     column tiles (B of them, or none), so no two waves fetch the same
//     weights;
//   * each wave streams its tiles' packed weights from HBM into a register
//     ring D half-stages deep, and the activation loads run in a ring of the
//     same depth in step with them (the counter of outstanding loads retires
//     them in issue order, so a stage's activations must not queue behind
//     later weights); the workgroup barrier that hands over an LDS stage
//     waits only for LDS traffic.
// Epilogues are those of the weight-streaming kernel (jf_epilogue.h), run on
// an LDS tile one row half at a time.
#include <algorithm>

#include "jf_device.h"
#include "jf_epilogue.h"
#include "jf_internal.h"

namespace jf {

constexpr int kMrWaves = 8;
constexpr int kMrThreads = 64 * kMrWaves;

// LDS writes of this wave are complete, then the workgroup barrier.
// Outstanding global loads stay in flight (no vmcnt wait); written as
// mnemonics so the assembler encodes them for the target.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Column tiles [lo, hi) of part p of n over units of gr tiles in [u0, u1).
__device__ __forceinline__ void split_units(int u0, int u1, int n, int p, int gr, int& lo, int& hi) {
  lo = (u0 + (int)(((long)(u1 - u0) * p) / n)) * gr;
  hi = (u0 + (int)(((long)(u1 - u0) * (p + 1)) / n)) * gr;
}

// Stage h of a pass (K-block kb0 + h / 2, fragment steps 2 (h % 2), + 1) of
// the chunk's 2A row tiles x 2 planes: A 16-byte pieces per thread.
template <int A>
__device__ __forceinline__ void mr_load_act(u32x4_t (&stg)[A], const bf16_t* __restrict__ xrow, size_t xplane, int KC,
                                            int kb0, int rtiles, int h) {
  const int kb = kb0 + (h >> 1), jh = h & 1;
#pragma unroll
  for (int i = 0; i < A; ++i) {
    const int e = threadIdx.x + kMrThreads * i;              // 16-byte piece of the stage
    const int rt = e >> 8, pl = (e >> 7) & 1, q = e & 127;   // row tile, plane, piece of the 2 KB half
    const int rtc = min(rt, rtiles - 1);
    stg[i] = *reinterpret_cast<const u32x4_t*>(xrow + (size_t)pl * xplane + (((size_t)rtc * KC + kb) << 11) +
                                               (size_t)jh * 1024 + q * 8);
  }
}
template <int A>
__device__ __forceinline__ void mr_store_act(const u32x4_t (&stg)[A], bf16_t* lbuf) {
  u32x4_t* dst = reinterpret_cast<u32x4_t*>(lbuf);
#pragma unroll
  for (int i = 0; i < A; ++i) dst[threadIdx.x + kMrThreads * i] = stg[i];
}
// The wave's weight fragments of stage h: B tiles x 2 fragment steps.
template <int B>
__device__ __forceinline__ void mr_load_w(Frag<bf16_t> (&w)[B][2], const bf16_t* const (&wb)[B], size_t kstride,
                                          int h) {
  const size_t off = (size_t)(h >> 1) * kstride + (size_t)(h & 1) * 1024;
#pragma unroll
  for (int t = 0; t < B; ++t)
#pragma unroll
    for (int jj = 0; jj < 2; ++jj) w[t][jj] = frag_load<bf16_t>(wb[t] + off + jj * 512);
}
// acc[r][t] += rows (row tile r of the chunk, from the LDS stage) x weights
// (tile t), for all 2A row tiles.
template <int A, int B>
__device__ __forceinline__ void mr_compute(f32x4_t (&acc)[2 * A][B], const bf16_t* la, const Frag<bf16_t> (&w)[B][2]) {
#pragma unroll
  for (int jj = 0; jj < 2; ++jj)
#pragma unroll
    for (int r = 0; r < 2 * A; ++r) {
      ActFrag<bf16_t> x;
      x.hi.v = *reinterpret_cast<const uint4*>(la + (size_t)(r * 2 + 0) * 1024 + jj * 512);
      x.lo.v = *reinterpret_cast<const uint4*>(la + (size_t)(r * 2 + 1) * 1024 + jj * 512);
#pragma unroll
      for (int t = 0; t < B; ++t) mfma(acc[r][t], x, w[t][jj]);
    }
}

constexpr int kStageElems(int A) { return 2 * A * 2 * 1024; }  // 2A row tiles x 2 planes x 1024 bf16

// The K loop of one pass over nst half-K-block stages.  kW: the wave has
// column tiles (else it only stages activations and keeps the barriers in
// step).  Straight-line prologue and steady state, so that the compiler's
// count of outstanding loads stays exact and both rings stay in flight.
template <int A, int B, int D, bool kW>
__device__ __forceinline__ void mr_kloop(f32x4_t (&acc)[2 * A][B], const bf16_t* __restrict__ xrow, size_t xplane,
                                         int KC, int kb0, int rtiles, int nst, const bf16_t* const (&wb)[B],
                                         size_t kstride, bf16_t* lact, const bf16_t* lane_lds) {
  constexpr int SE = kStageElems(A);
  Frag<bf16_t> wr[D][B][2];
  u32x4_t ar[D][A];
  // a pass shorter than the ring re-reads its last stage
#pragma unroll
  for (int d = 0; d < D; ++d) {
    mr_load_act<A>(ar[d], xrow, xplane, KC, kb0, rtiles, min(d, nst - 1));
    if constexpr (kW) mr_load_w<B>(wr[d], wb, kstride, min(d, nst - 1));
  }
  mr_store_act<A>(ar[0], lact);
  lds_barrier();
  int hb = 0;
  for (; hb + 2 * D <= nst; hb += D) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const int h = hb + d;
      if constexpr (kW) mr_compute<A, B>(acc, lane_lds + (size_t)(h & 1) * SE, wr[d]);
      mr_load_act<A>(ar[d], xrow, xplane, KC, kb0, rtiles, h + D);
      if constexpr (kW) mr_load_w<B>(wr[d], wb, kstride, h + D);
      mr_store_act<A>(ar[(d + 1) % D], lact + (size_t)((h + 1) & 1) * SE);
      lds_barrier();
    }
  }
  // tail: fewer than 2 D stages left
#pragma unroll
  for (int d = 0; d < 2 * D; ++d) {
    const int h = hb + d;
    if (h < nst) {
      if constexpr (kW) mr_compute<A, B>(acc, lane_lds + (size_t)(h & 1) * SE, wr[d % D]);
      if (h + D < nst) {
        mr_load_act<A>(ar[d % D], xrow, xplane, KC, kb0, rtiles, h + D);
        if constexpr (kW) mr_load_w<B>(wr[d % D], wb, kstride, h + D);
      }
      if (h + 1 < nst) mr_store_act<A>(ar[(d + 1) % D], lact + (size_t)((h + 1) & 1) * SE);
      lds_barrier();
    }
  }
}

template <int A, int B, int D>
__global__ void __launch_bounds__(kMrThreads, 1)
k_gemm_mr(const bf16_t* __restrict__ X, size_t xplane, const bf16_t* __restrict__ Wp, MrPlan m, Epi ep) {
  extern __shared__ float lds[];
  bf16_t* lact = reinterpret_cast<bf16_t*>(lds);           // two activation stages
  __shared__ float s_rs[16 * A];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = blockIdx.x, z = blockIdx.z;
  const int KC = m.KC, P = m.P;
  // rows of this chunk
  const int r0 = z * 32 * A;
  const int Rz = min(32 * A, m.R - r0);
  const int rtiles = (Rz + 15) / 16;                       // valid row tiles
  const int U = m.T / m.gr;
  const int u0 = (int)(((long)U * g) / m.n_cg), u1 = (int)(((long)U * (g + 1)) / m.n_cg);
  const int np = m.passes;
  const size_t kstride = (size_t)P * kBlockElems;
  const int nst = 2 * KC;                                  // half-K-block stages of a pass

  // the pass's column tiles [pl, ph); wave w takes tiles pl + B w .. (up to
  // B of them), so every wave but one has B tiles or none
  auto pass_tiles = [&](int p, int& pl, int& ph) { split_units(u0, u1, np, p, m.gr, pl, ph); };
  auto toff = [&](int t) { return ((size_t)(t / P) * KC * P + t % P) * kBlockElems; };

  const bf16_t* xrow = X + ((size_t)(r0 / 16) * KC << 11);  // the chunk's first row tile
  // the other RMSNorm accumulator (filled by the next producer) is cleared
  // by the first workgroup, as in the weight-streaming kernel
  if (ep.ss_clear && g == 0 && z == 0)
    for (int i = threadIdx.x; i < 3 * ep.ss_stride; i += kMrThreads)
      __hip_atomic_store(ep.ss_clear + i, (uint64_t)0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);

  f32x4_t acc[2 * A][B];
  const bf16_t* lane_lds = lact + lane * 8;
  for (int p = 0; p < np; ++p) {
    int pl, ph;
    pass_tiles(p, pl, ph);
    const int c_lo = pl + B * wave;
    const int nb = max(0, min(B, ph - c_lo));              // wave-uniform
    // a partly filled wave re-reads its last tile in the empty slots (an L2
    // hit; those products are not used)
    const bf16_t* wb[B];
#pragma unroll
    for (int t = 0; t < B; ++t)
      wb[t] = Wp + toff(min(c_lo + min(t, max(nb - 1, 0)), m.T - 1)) + lane * 8;
#pragma unroll
    for (int r = 0; r < 2 * A; ++r)
#pragma unroll
      for (int t = 0; t < B; ++t) acc[r][t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    if (nb > 0)
      mr_kloop<A, B, D, true>(acc, xrow, xplane, KC, 0, rtiles, nst, wb, kstride, lact, lane_lds);
    else
      mr_kloop<A, B, D, false>(acc, xrow, xplane, KC, 0, rtiles, nst, wb, kstride, lact, lane_lds);

    // epilogue through an LDS tile aliased over the activation stages, one
    // row half (16 A rows) at a time
    const int cols = (ph - pl) * 16, tld = cols + 1;
    float* tile = lds;
    for (int half = 0; half < 2; ++half) {
      const int hr0 = r0 + half * 16 * A;
      const int hR = min(16 * A, m.R - hr0);
      if (hR <= 0) break;                                  // block-uniform
      __syncthreads();
#pragma unroll
      for (int i = 0; i < A; ++i)
#pragma unroll
        for (int t = 0; t < B; ++t)
          if (t < nb)
#pragma unroll
            for (int k = 0; k < 4; ++k)
              tile[(i * 16 + 4 * (lane >> 4) + k) * tld + (c_lo - pl + t) * 16 + (lane & 15)] =
                  acc[half * A + i][t][k];
      if (ep.ss_in)
        for (int r = threadIdx.x; r < hR; r += kMrThreads) {
          uint64_t w[3];
          ss_load(ep.ss_in, ep.ss_stride, hr0 + r, w);
          s_rs[r] = ss_rstd(w, ep.norm_inv_d, ep.norm_eps);
        }
      __syncthreads();
      if (ep.ss_in)
        for (int e = threadIdx.x; e < hR * cols; e += kMrThreads) {
          const int r = e / cols, c = e - r * cols;
          tile[r * tld + c] *= s_rs[r];
        }
      __syncthreads();
      epilogue<bf16_t>(tile, tld, cols, pl * 16, ep, g * np + p, threadIdx.x, kMrThreads, hr0, hR);
    }
    __syncthreads();
  }
}

// ---- plans ------------------------------------------------------------------------
int mr_row_tiles_half(int R) {
  // above 128 rows: 128-row chunks (each re-reads the weights, but a wider
  // chunk leaves registers for one column tile a wave, and re-reading the
  // activations once per 8 tiles costs more)
  return R <= 64 ? 2 : 4;
}

// Most column tiles one pass of a group holds (groups of ceil(U / n_cg)
// units split into `passes` parts).
static long mr_max_pass_tiles(const MrPlan& m) {
  const long U = m.T / m.gr;
  const long group = (U + m.n_cg - 1) / m.n_cg;
  return (group + m.passes - 1) / m.passes * m.gr;
}

// Column tiles per wave that the register file holds next to the rings, per
// row-tile count: accumulators 4 x 2A x B, weight ring 8 x B x D and
// activation ring 4 x A x D registers a lane (D = 2), within the 256 of a
// wave at two waves per SIMD (checked: no spills).
static int mr_max_cols(int A) { return A <= 2 ? 4 : 2; }

bool gemm_mr_plan(MrPlan& m, int R, int N, int K, int epi_kind, int n_cus) {
  if (R <= 32 || N % 16 || K % 128) return false;
  const int A = mr_row_tiles_half(R);
  m.R = R;
  m.A = A;
  m.KC = K / 128;
  m.P = pack_group(N);
  m.T = N / 16;
  m.gr = epi_kind == EPI_SWIGLU ? 2 : 1;
  if (m.T % m.gr) return false;
  m.chunks = (R + 32 * A - 1) / (32 * A);
  m.S = 1;
  const int U = m.T / m.gr;
  const int per_chunk = std::max(1, std::max(1, n_cus) / m.chunks);  // workgroups per row chunk
  // only matrices wide enough to give every compute unit a full wave's
  // worth of columns; narrower ones stay on the weight-streaming kernel
  if (m.T < 8 * per_chunk) return false;
  m.n_cg = std::min(per_chunk, U);
  // the fewest passes (each re-reads the activations), then the fewest tiles
  // a wave that holds a pass (idle waves fetch nothing)
  m.B = mr_max_cols(A);
  m.passes = 1;
  while (mr_max_pass_tiles(m) > 8L * m.B) ++m.passes;
  m.B = (int)((mr_max_pass_tiles(m) + 7) / 8);
  return true;
}

size_t gemm_mr_lds_bytes(const MrPlan& m) {
  const size_t stages = (size_t)2 * kStageElems(m.A) * 2;                  // bytes
  const int max_cols = 8 * m.B * 16;
  const size_t tile = (size_t)16 * m.A * (max_cols + 1) * 4;
  return std::max(stages, tile);
}

template <int A, int B, int D>
static hipError_t launch_mr_t(const void* X, size_t xplane, const void* Wp, const MrPlan& m, const Epi& ep,
                              hipStream_t st) {
  hipLaunchKernelGGL((k_gemm_mr<A, B, D>), dim3(m.n_cg, 1, m.chunks), dim3(kMrThreads), gemm_mr_lds_bytes(m), st,
                     reinterpret_cast<const bf16_t*>(X), xplane, reinterpret_cast<const bf16_t*>(Wp), m, ep);
  return hipGetLastError();
}

template <int A>
static hipError_t launch_mr_b(const void* X, size_t xplane, const void* Wp, const MrPlan& m, const Epi& ep,
                              hipStream_t st) {
  switch (m.B) {
    case 1: return launch_mr_t<A, 1, 2>(X, xplane, Wp, m, ep, st);
    case 2: return launch_mr_t<A, 2, 2>(X, xplane, Wp, m, ep, st);
    case 3: if constexpr (A <= 2) return launch_mr_t<A, 3, 2>(X, xplane, Wp, m, ep, st); break;
    case 4: if constexpr (A <= 2) return launch_mr_t<A, 4, 2>(X, xplane, Wp, m, ep, st); break;
    default: break;
  }
  return hipErrorInvalidValue;
}

hipError_t launch_gemm_mr(const void* X, size_t xplane, const void* Wp, const MrPlan& m, const Epi& ep,
                          hipStream_t st) {
  if (m.R <= 32 || m.T < 1 || m.KC < 1 || m.n_cg < 1 || m.S != 1 || m.passes < 1 || m.gr < 1 || m.B < 1 ||
      m.B > mr_max_cols(m.A) || m.T % m.gr || m.chunks != (m.R + 32 * m.A - 1) / (32 * m.A) || ep.row0 != 0)
    return hipErrorInvalidValue;
  // every pass must fit the waves' column tiles (8 waves of at most B)
  if (mr_max_pass_tiles(m) > 8L * m.B) return hipErrorInvalidValue;
  if (gemm_mr_lds_bytes(m) > 160 * 1024) return hipErrorInvalidValue;
  switch (m.A) {
    case 2: return launch_mr_b<2>(X, xplane, Wp, m, ep, st);
    case 4: return launch_mr_b<4>(X, xplane, Wp, m, ep, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace jf
