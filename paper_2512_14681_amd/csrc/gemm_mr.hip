// Column-slice GEMM of the decoder's projections, Y[R][N] = X[R][K] *
// W[N][K]^T, for the wide Jacobi steps (more than 24 rows: multi-block
// drafts with recycled candidates, Sec. 3.2 and App. A Alg. 1; the packed
// training forward; the block-size sweeps): the wide projections (gate/up,
// LM head) and the long-K narrow one (down), and from 65 rows QKV and O.
// Rows go in chunks of 32, 64, 96 or 128.
//
// What bounds these launches is the bytes each compute unit requests (its
// share of the weights plus the activations it re-reads), so the kernel asks
// for every weight byte exactly once per compute unit and for the
// activations once per pass:
//   * a workgroup of 8 waves owns a column group (one pass of up to 8B
//     16-column tiles; wider groups take several passes) and a K-range;
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
//     waits only for LDS traffic;
//   * split K (long-K narrow matrices): each workgroup writes its raw
//     partial tile and a second kernel sums the partials in split order
//     (deterministic) and runs the epilogue.
// Epilogues are those of the weight-streaming kernel (jf_epilogue.h), run on
// an LDS tile.
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
// the chunk's RT row tiles x 2 planes, 256 RT 16-byte pieces: RT / 2 a
// thread.
template <int RT> constexpr int mr_pieces() {
  static_assert(RT % 2 == 0, "an even number of row tiles");
  return 256 * RT / kMrThreads;
}
template <int RT>
__device__ __forceinline__ void mr_load_act(u32x4_t (&stg)[mr_pieces<RT>()], const bf16_t* __restrict__ xrow,
                                            size_t xplane, int KC, int kb0, int rtiles, int h) {
  const int kb = kb0 + (h >> 1), jh = h & 1;
#pragma unroll
  for (int i = 0; i < mr_pieces<RT>(); ++i) {
    const int e = threadIdx.x + kMrThreads * i;              // 16-byte piece of the stage
    const int rt = e >> 8, pl = (e >> 7) & 1, q = e & 127;   // row tile, plane, piece of the 2 KB half
    const int rtc = min(rt, rtiles - 1);
    stg[i] = *reinterpret_cast<const u32x4_t*>(xrow + (size_t)pl * xplane + (((size_t)rtc * KC + kb) << 11) +
                                               (size_t)jh * 1024 + q * 8);
  }
}
template <int RT>
__device__ __forceinline__ void mr_store_act(const u32x4_t (&stg)[mr_pieces<RT>()], bf16_t* lbuf) {
  u32x4_t* dst = reinterpret_cast<u32x4_t*>(lbuf);
#pragma unroll
  for (int i = 0; i < mr_pieces<RT>(); ++i) dst[threadIdx.x + kMrThreads * i] = stg[i];
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
// (tile t), for all RT row tiles.
template <int RT, int B>
__device__ __forceinline__ void mr_compute(f32x4_t (&acc)[RT][B], const bf16_t* la, const Frag<bf16_t> (&w)[B][2]) {
#pragma unroll
  for (int jj = 0; jj < 2; ++jj)
#pragma unroll
    for (int r = 0; r < RT; ++r) {
      ActFrag<bf16_t> x;
      x.hi.v = *reinterpret_cast<const uint4*>(la + (size_t)(r * 2 + 0) * 1024 + jj * 512);
      x.lo.v = *reinterpret_cast<const uint4*>(la + (size_t)(r * 2 + 1) * 1024 + jj * 512);
#pragma unroll
      for (int t = 0; t < B; ++t) mfma(acc[r][t], x, w[t][jj]);
    }
}

constexpr int kStageElems(int RT) { return RT * 2 * 1024; }  // RT row tiles x 2 planes x 1024 bf16

// The K loop of one pass over nst half-K-block stages.  kW: the wave has
// column tiles (else it only stages activations and keeps the barriers in
// step).  Straight-line prologue and steady state, so that the compiler's
// count of outstanding loads stays exact and both rings stay in flight.
template <int RT, int B, int D, bool kW>
__device__ __forceinline__ void mr_kloop(f32x4_t (&acc)[RT][B], const bf16_t* __restrict__ xrow, size_t xplane,
                                         int KC, int kb0, int rtiles, int nst, const bf16_t* const (&wb)[B],
                                         size_t kstride, bf16_t* lact, const bf16_t* lane_lds) {
  constexpr int SE = kStageElems(RT);
  Frag<bf16_t> wr[D][B][2];
  u32x4_t ar[D][mr_pieces<RT>()];
  // a pass shorter than the ring re-reads its last stage
#pragma unroll
  for (int d = 0; d < D; ++d) {
    mr_load_act<RT>(ar[d], xrow, xplane, KC, kb0, rtiles, min(d, nst - 1));
    if constexpr (kW) mr_load_w<B>(wr[d], wb, kstride, min(d, nst - 1));
  }
  mr_store_act<RT>(ar[0], lact);
  lds_barrier();
  int hb = 0;
  for (; hb + 2 * D <= nst; hb += D) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const int h = hb + d;
      if constexpr (kW) mr_compute<RT, B>(acc, lane_lds + (size_t)(h & 1) * SE, wr[d]);
      mr_load_act<RT>(ar[d], xrow, xplane, KC, kb0, rtiles, h + D);
      if constexpr (kW) mr_load_w<B>(wr[d], wb, kstride, h + D);
      mr_store_act<RT>(ar[(d + 1) % D], lact + (size_t)((h + 1) & 1) * SE);
      lds_barrier();
    }
  }
  // tail: fewer than 2 D stages left
#pragma unroll
  for (int d = 0; d < 2 * D; ++d) {
    const int h = hb + d;
    if (h < nst) {
      if constexpr (kW) mr_compute<RT, B>(acc, lane_lds + (size_t)(h & 1) * SE, wr[d % D]);
      if (h + D < nst) {
        mr_load_act<RT>(ar[d % D], xrow, xplane, KC, kb0, rtiles, h + D);
        if constexpr (kW) mr_load_w<B>(wr[d % D], wb, kstride, h + D);
      }
      if (h + 1 < nst) mr_store_act<RT>(ar[(d + 1) % D], lact + (size_t)((h + 1) & 1) * SE);
      lds_barrier();
    }
  }
}

// Row tiles per epilogue round: the LDS tile holds ER x 16 rows of a pass.
constexpr int mr_epi_tiles(int RT) { return RT / 2; }

template <int RT, int B, int D>
__global__ void __launch_bounds__(kMrThreads, 1)
k_gemm_mr(const bf16_t* __restrict__ X, size_t xplane, const bf16_t* __restrict__ Wp, MrPlan m, Epi ep) {
  constexpr int ER = mr_epi_tiles(RT);
  extern __shared__ float lds[];
  bf16_t* lact = reinterpret_cast<bf16_t*>(lds);           // two activation stages
  __shared__ float s_rs[16 * ER];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = blockIdx.x, sk = blockIdx.y, z = blockIdx.z;
  const int KC = m.KC, P = m.P;
  // rows of this chunk
  const int r0 = z * 16 * RT;
  const int Rz = min(16 * RT, m.R - r0);
  const int rtiles = (Rz + 15) / 16;                       // valid row tiles
  const int U = m.T / m.gr;
  const int u0 = (int)(((long)U * g) / m.n_cg), u1 = (int)(((long)U * (g + 1)) / m.n_cg);
  const int np = m.passes;
  const size_t kstride = (size_t)P * kBlockElems;
  const int kb0 = (KC * sk) / m.S, kb1 = (KC * (sk + 1)) / m.S;
  const int nst = 2 * (kb1 - kb0);                         // half-K-block stages of a pass

  auto toff = [&](int t) { return ((size_t)(t / P) * KC * P + t % P) * kBlockElems; };

  const bf16_t* xrow = X + ((size_t)(r0 / 16) * KC << 11);  // the chunk's first row tile
  // the other RMSNorm accumulator (filled by the next producer) is cleared
  // by the first workgroup, as in the weight-streaming kernel
  if (ep.ss_clear && g == 0 && sk == 0 && z == 0)
    for (int i = threadIdx.x; i < 3 * ep.ss_stride; i += kMrThreads)
      __hip_atomic_store(ep.ss_clear + i, (uint64_t)0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);

  f32x4_t acc[RT][B];
  const bf16_t* lane_lds = lact + lane * 8;
  for (int p = 0; p < np; ++p) {
    // the pass's column tiles [pl, ph); wave w takes tiles pl + B w .. (up
    // to B of them), so every wave but one has B tiles or none
    int pl, ph;
    split_units(u0, u1, np, p, m.gr, pl, ph);
    const int c_lo = pl + B * wave;
    const int nb = max(0, min(B, ph - c_lo));              // wave-uniform
    // a partly filled wave re-reads its last tile in the empty slots (an L2
    // hit; those products are not used)
    const bf16_t* wb[B];
#pragma unroll
    for (int t = 0; t < B; ++t)
      wb[t] = Wp + toff(min(c_lo + min(t, max(nb - 1, 0)), m.T - 1)) + (size_t)kb0 * kstride + lane * 8;
#pragma unroll
    for (int r = 0; r < RT; ++r)
#pragma unroll
      for (int t = 0; t < B; ++t) acc[r][t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    if (nb > 0)
      mr_kloop<RT, B, D, true>(acc, xrow, xplane, KC, kb0, rtiles, nst, wb, kstride, lact, lane_lds);
    else
      mr_kloop<RT, B, D, false>(acc, xrow, xplane, KC, kb0, rtiles, nst, wb, kstride, lact, lane_lds);

    // epilogue through an LDS tile aliased over the activation stages, ER
    // row tiles at a time; with split K the tile goes out raw, row-major per
    // split, for the reduction kernel
    const int cols = (ph - pl) * 16, tld = cols + 1;
    const int N = m.T * 16;
    float* tile = lds;
    for (int er = 0; er < RT / ER; ++er) {
      const int hr0 = r0 + er * 16 * ER;
      const int hR = min(16 * ER, m.R - hr0);
      if (hR <= 0) break;                                  // block-uniform
      __syncthreads();
#pragma unroll
      for (int i = 0; i < ER; ++i)
#pragma unroll
        for (int t = 0; t < B; ++t)
          if (t < nb)
#pragma unroll
            for (int k = 0; k < 4; ++k)
              tile[(i * 16 + 4 * (lane >> 4) + k) * tld + (c_lo - pl + t) * 16 + (lane & 15)] =
                  acc[er * ER + i][t][k];
      if (m.S > 1) {
        __syncthreads();
        float* kp = ep.kpart + ((size_t)sk * m.R + hr0) * N + pl * 16;
        for (int e = threadIdx.x; e < hR * cols; e += kMrThreads) {
          const int r = e / cols, c = e - r * cols;
          kp[(size_t)r * N + c] = tile[r * tld + c];
        }
        continue;
      }
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

// Split-K reduction: block (x, y) sums the S partials of rows 16 y .. and
// columns 64 x .. in split order (deterministic), applies the folded RMSNorm
// and runs the epilogue (its per-block argmax slot is x).  Each thread owns
// 4 adjacent columns of one row and keeps 8 partial loads in flight.
constexpr int kRedRows = 16, kRedCols = 64, kRedThreads = 256;

__global__ void __launch_bounds__(kRedThreads) k_mr_reduce(MrPlan m, Epi ep) {
  constexpr int tld = kRedCols + 1;
  __shared__ float tile[kRedRows * tld];
  __shared__ float s_rs[kRedRows];
  const int N = m.T * 16;
  const int c0 = blockIdx.x * kRedCols, r0 = blockIdx.y * kRedRows;
  const int cols = min(kRedCols, N - c0), rows = min(kRedRows, m.R - r0);
  const size_t split = (size_t)m.R * N;
  if (ep.ss_in && threadIdx.x < rows) {
    uint64_t w[3];
    ss_load(ep.ss_in, ep.ss_stride, r0 + threadIdx.x, w);
    s_rs[threadIdx.x] = ss_rstd(w, ep.norm_inv_d, ep.norm_eps);
  }
  __syncthreads();
  const int r = threadIdx.x / (kRedCols / 4), c = 4 * (threadIdx.x % (kRedCols / 4));
  float4 v = {0.f, 0.f, 0.f, 0.f};
  if (r < rows && c < cols) {                               // cols is a multiple of 16
    const float4* p = reinterpret_cast<const float4*>(ep.kpart + (size_t)(r0 + r) * N + c0 + c);
    const size_t sp = split / 4;
    int s = 0;
    for (; s + 8 <= m.S; s += 8) {
      float4 x[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) x[j] = p[(size_t)(s + j) * sp];
#pragma unroll
      for (int j = 0; j < 8; ++j) { v.x += x[j].x; v.y += x[j].y; v.z += x[j].z; v.w += x[j].w; }
    }
    float4 x[8];
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (s + j < m.S) x[j] = p[(size_t)(s + j) * sp];
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (s + j < m.S) { v.x += x[j].x; v.y += x[j].y; v.z += x[j].z; v.w += x[j].w; }
    if (ep.ss_in) {
      const float k = s_rs[r];
      v.x *= k; v.y *= k; v.z *= k; v.w *= k;
    }
  }
  tile[r * tld + c + 0] = v.x;
  tile[r * tld + c + 1] = v.y;
  tile[r * tld + c + 2] = v.z;
  tile[r * tld + c + 3] = v.w;
  __syncthreads();
  epilogue<bf16_t>(tile, tld, cols, c0, ep, blockIdx.x, threadIdx.x, kRedThreads, r0, rows);
}

// ---- plans ------------------------------------------------------------------------
// Row tiles of a chunk: 4, 6 or 8 (64-, 96- and 128-row chunks), or 2 up
// to 32 rows, whichever the cost below rates cheapest.  Each chunk streams
// the weights again, and a pass re-reads the chunk's activations, so wide
// chunks save weight bytes while narrow ones leave registers for more
// column tiles a wave (fewer passes): 192 rows run as two 96-row chunks in
// one pass each rather than a 128-row chunk in two passes plus a 64-row one.
static bool mr_rt_ok(int RT) { return RT == 2 || RT == 4 || RT == 6 || RT == 8; }

// Row ranges where a measured chunk size beats the cost's choice (7B-shaped
// steps after 1024 tokens, all projections at one row-tile count; us):
// 128 rows 7382 (8) -> 7029 (4), 256 rows 11340 (8) -> 10774 (4), 224 rows
// 10989 -> 10365 (4), 384 rows 14152 (8) -> 13937 (6).  The 64-row chunks
// win where the rows fill 2 or 4 of them: the chunks of a column group run
// on one XCD at the same time (their workgroup ids are congruent mod 8), so
// their weight re-reads hit L2, which the cost charges as full requests,
// while wider chunks re-read more activations per pass and load the matrix
// cores more.  0: the cost decides.
static int mr_measured_rt(int R) {
  if (R > 96 && R <= 128) return 4;
  if (R > 192 && R <= 256) return 4;
  if (R > 320 && R <= 384) return 6;
  return 0;
}

// Most column tiles one pass of a group holds (groups of ceil(U / n_cg)
// units split into `passes` parts).
static long mr_max_pass_tiles(const MrPlan& m) {
  const long U = m.T / m.gr;
  const long group = (U + m.n_cg - 1) / m.n_cg;
  return (group + m.passes - 1) / m.passes * m.gr;
}

// Column tiles per wave that the register file holds, per row-tile count:
// accumulators 4 RT B, weight ring 8 B D and activation ring 2 D RT
// registers a lane (ring depth D = 2 half K-blocks), within the 256 of a
// wave at two waves per SIMD (checked: no spills).
static int mr_max_cols(int RT) { return RT == 2 ? 6 : RT == 4 ? 4 : RT == 6 ? 3 : 2; }

// Plan cost, in compute-unit clocks: a workgroup's requested bytes (its
// weights, the activations of its K-range once per pass at half weight, as
// they come from L2, and its partial sums) at the rate one compute unit
// sustains on the weight streams (about 27 GB/s, 11 bytes a clock), or its
// matrix / LDS work if larger, times the rounds of workgroups; split K adds
// the reduction's traffic spread over the chip and its launch.
static double mr_cost(const MrPlan& m, int cus) {
  const double rows = std::min(m.R, 16 * m.RT);
  const double tiles = (double)mr_max_pass_tiles(m) * m.passes;
  const double kc = (m.KC + m.S - 1) / m.S;
  double bytes = tiles * kc * 4096 + m.passes * rows * kc * 256;
  if (m.S > 1) bytes += rows * tiles * 64;
  const double stages = 2.0 * kc * m.passes;
  const double work = stages * std::max(128.0 * m.RT * m.B, 256.0 * m.RT);
  const double rounds = std::ceil((double)m.n_cg * m.S * m.chunks / cus);
  double cost = rounds * std::max(bytes / 11.0, work);
  if (m.S > 1) cost += ((double)m.S + 1) * m.R * m.T * 64 / cus / 11.0 + 12000.0;
  return cost;
}

bool gemm_mr_plan(MrPlan& m, int R, int N, int K, int epi_kind, int n_cus, int max_splits) {
  // Up to 24 rows the weight-streaming kernel is faster on every 7B-shaped
  // projection: both run at the weight stream's rate per compute unit, and
  // its many small workgroups balance the chip better than one workgroup
  // per compute unit with a whole number of column tiles (measured: gate/up
  // 50.5 against 52.9 us, LM head 169 against 222 us at 16 rows; steps at
  // 17 / 20 / 24 rows +4.5 / +4.8 / +3.6% here).  From 25 rows its 2-row-tile
  // blocks re-read as many activation bytes as weight bytes, and the column
  // slices win (28 / 32 rows: -0.5 / -1.3%).
  if (R <= 24 || N % 16 || K % 128) return false;
  const int gr = epi_kind == EPI_SWIGLU ? 2 : 1;
  if ((N / 16) % gr) return false;
  const int cus = std::max(1, n_cus);
  double best = -1;
  const int rt_fixed = mr_measured_rt(R);
  for (int RT = R <= 32 ? 2 : 4; RT <= 8; RT += 2) {
    if (rt_fixed && RT != rt_fixed) continue;
    MrPlan t{};
    t.R = R;
    t.RT = RT;
    t.KC = K / 128;
    t.P = pack_group(N);
    t.T = N / 16;
    t.gr = gr;
    t.chunks = (R + 16 * RT - 1) / (16 * RT);
    const int U = t.T / t.gr;
    const int per_chunk = std::max(1, cus / t.chunks);     // workgroups per row chunk in one round
    // Measured on the 7B-shaped projections (64 to 256 rows): a matrix too
    // narrow to give every compute unit a wave's worth of columns needs
    // split K here, which pays (partials, a reduction launch) over a long K
    // (down: 64 K-blocks and more) at any row count, and over a short K
    // (QKV, O) from 65 rows, where the weight-streaming kernel's 32-row
    // chunks stream the weights three times or more (steps at 80 / 96 /
    // 192 / 256 rows: -4.6 / -3.4 / -2.7 / -7.2%; at 33 / 48 / 64 rows
    // +1.7 / +2.5 / +1.4%, so up to 64 rows they stay there); wide matrices
    // (gate/up, LM head) run faster without split K.  Narrowness is judged
    // at the widest chunk, so that the choice of chunk does not move a
    // matrix between kernels.
    const bool narrow = t.T < 8 * std::max(1, cus / ((R + 127) / 128));
    if (narrow && t.KC < 64 && R <= 64) return false;
    // at most 8 K splits: the cost below rates more splits cheaper than they
    // run (1024-token prefix, steps at 48 / 64 / 96 / 128 / 192 / 256 rows,
    // down with 17 / 17 / 17 / 17 / 9 / 9 splits and O with 10 at 96 rows ->
    // at most 8: -2.7 / -2.8 / -3.1 / -1.4 / -5.4 / -2.9%; capped at 6 or 4:
    // slower again)
    const int splits = narrow ? std::min(max_splits, 8) : 1;
    for (int S = 1; S <= std::min(t.KC, std::min(splits, 64)); ++S) {
      if (S > 1 && (size_t)S * R * N > kGemmPartFloats) break;
      t.S = S;
      t.n_cg = std::min(U, std::max(1, per_chunk / S));
      // the fewest passes (each re-reads the activations), then the fewest
      // tiles a wave that holds a pass (idle waves fetch nothing)
      t.B = mr_max_cols(RT);
      t.passes = 1;
      while (mr_max_pass_tiles(t) > 8L * t.B) ++t.passes;
      t.B = (int)((mr_max_pass_tiles(t) + 7) / 8);
      const double c = mr_cost(t, cus);
      if (best < 0 || c < best) {
        best = c;
        m = t;
      }
    }
  }
  return best >= 0;
}

size_t gemm_mr_lds_bytes(const MrPlan& m) {
  const size_t stages = (size_t)2 * kStageElems(m.RT) * 2;                  // bytes
  const int max_cols = 8 * m.B * 16;
  const size_t tile = (size_t)16 * mr_epi_tiles(m.RT) * (max_cols + 1) * 4;
  return std::max(stages, tile);
}

template <int RT, int B>
static hipError_t launch_mr_t(const void* X, size_t xplane, const void* Wp, const MrPlan& m, const Epi& ep,
                              hipStream_t st) {
  constexpr int D = 2;
  hipLaunchKernelGGL((k_gemm_mr<RT, B, D>), dim3(m.n_cg, m.S, m.chunks), dim3(kMrThreads), gemm_mr_lds_bytes(m), st,
                     reinterpret_cast<const bf16_t*>(X), xplane, reinterpret_cast<const bf16_t*>(Wp), m, ep);
  if (m.S > 1)
    hipLaunchKernelGGL(k_mr_reduce, dim3(gemm_mr_part_blocks(m), (m.R + kRedRows - 1) / kRedRows), dim3(kRedThreads),
                       0, st, m, ep);
  return hipGetLastError();
}

template <int RT>
static hipError_t launch_mr_b(const void* X, size_t xplane, const void* Wp, const MrPlan& m, const Epi& ep,
                              hipStream_t st) {
  switch (m.B) {
    case 1: return launch_mr_t<RT, 1>(X, xplane, Wp, m, ep, st);
    case 2: return launch_mr_t<RT, 2>(X, xplane, Wp, m, ep, st);
    case 3: if constexpr (RT <= 6) return launch_mr_t<RT, 3>(X, xplane, Wp, m, ep, st); break;
    case 4: if constexpr (RT <= 4) return launch_mr_t<RT, 4>(X, xplane, Wp, m, ep, st); break;
    case 5: if constexpr (RT == 2) return launch_mr_t<RT, 5>(X, xplane, Wp, m, ep, st); break;
    case 6: if constexpr (RT == 2) return launch_mr_t<RT, 6>(X, xplane, Wp, m, ep, st); break;
    default: break;
  }
  return hipErrorInvalidValue;
}

int gemm_mr_part_blocks(const MrPlan& m) {
  return m.S > 1 ? (m.T * 16 + kRedCols - 1) / kRedCols : m.n_cg * m.passes;
}

hipError_t launch_gemm_mr(const void* X, size_t xplane, const void* Wp, const MrPlan& m, const Epi& ep,
                          hipStream_t st) {
  if (m.R < 1 || m.T < 1 || m.KC < 1 || m.n_cg < 1 || m.S < 1 || m.S > m.KC || m.passes < 1 || m.gr < 1 || m.B < 1 ||
      !mr_rt_ok(m.RT) || m.B > mr_max_cols(m.RT) || m.T % m.gr ||
      m.chunks != (m.R + 16 * m.RT - 1) / (16 * m.RT) || ep.row0 != 0)
    return hipErrorInvalidValue;
  // every pass must fit the waves' column tiles (8 waves of at most B)
  if (mr_max_pass_tiles(m) > 8L * m.B) return hipErrorInvalidValue;
  if (gemm_mr_lds_bytes(m) > 160 * 1024) return hipErrorInvalidValue;
  if (m.S > 1 && (!ep.kpart || (size_t)m.S * m.R * m.T * 16 > kGemmPartFloats)) return hipErrorInvalidValue;
  switch (m.RT) {
    case 2: return launch_mr_b<2>(X, xplane, Wp, m, ep, st);
    case 4: return launch_mr_b<4>(X, xplane, Wp, m, ep, st);
    case 6: return launch_mr_b<6>(X, xplane, Wp, m, ep, st);
    case 8: return launch_mr_b<8>(X, xplane, Wp, m, ep, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace jf
