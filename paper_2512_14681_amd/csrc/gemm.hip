// Small-M weight-streaming GEMM for the decoder's projections:
//   Y[R][N] = X[R][K] * W[N][K]^T,  R = rows of one Jacobi step (1..512).
//
// The step is bound by reading W once (Sec. 4.2 / App. D of the paper: the
// extra draft rows of a Jacobi iteration are nearly free until the hardware
// knee), so the kernel is organised around streaming the packed weight
// blocks: one block of 16 output rows x 128 inputs is 4 KB (bf16) that a
// wave reads with 4 fully coalesced 1 KB loads, then issues 4 MFMA steps per
// 16-row tile of X.  A workgroup owns NT adjacent 16-column tiles and splits
// K over WK waves; the waves' partial tiles are summed in LDS in a fixed
// order (deterministic) and the epilogue runs on the reduced tile.
#include <algorithm>

#include "jf_device.h"
#include "jf_epilogue.h"
#include "jf_internal.h"

namespace jf {

// Register ring: D K-blocks of weights (and, for <= 32 rows, of
// activations) are in flight per wave.  The default depth is the largest
// (<= 4) that fits a register budget leaving room for two waves per SIMD
// (512 registers per lane per SIMD), or for the whole block when it has more
// than 8 waves.
template <typename T, int RT, int NT, int WK> struct Ring {
  static constexpr bool kPrefetchX = RT <= 2;
  static constexpr int kBudget = WK <= 8 ? 224 : 112;
  static constexpr int kFragRegs = sizeof(T) == 2 ? 4 : 8;
  static constexpr int kFixed = 48 + RT * NT * 4 + (kPrefetchX ? 0 : 4 * 8);
  static constexpr int kPerSlot = NT * 4 * kFragRegs + (kPrefetchX ? RT * 4 * 8 : 0);
  static constexpr int kD = (kBudget - kFixed) / kPerSlot;
  static constexpr int D = kD < 1 ? 1 : (kD > 4 ? 4 : kD);
};

// Grid: one block per (column group, K split, row chunk).  More than 32 rows
// are done in chunks of 32 (C of them), each by its own block with the
// weights of its unit (column group, K split) streamed again; the block
// order is XCD-aware so that those re-reads hit L2: linear block b runs on
// XCD b % 8 (round-robin dispatch), so the C chunks of a unit get ids
// congruent mod 8 and adjacent in dispatch order, i.e. the same XCD at the
// same time, and the unit's weights come from HBM once.
// CHUNKED (C > 1): the 1-D XCD-aware block order above, and the weights,
// read by the C chunk blocks of a unit, are loaded with the ordinary
// (L2-allocating) policy instead of the streaming hint.  Otherwise the grid
// is (column groups, K splits) and there is one chunk, or, with a tail split
// (full < groups), 1-D: blocks [0, full) take column groups [0, full) whole
// and the remaining groups take S blocks each, one K-range apiece.
template <typename T, int RT, int NT, int WK, int D = Ring<T, RT, NT, WK>::D, bool CHUNKED = false>
__global__ void __launch_bounds__(64 * WK)
k_gemm(const T* __restrict__ X, size_t xplane, const T* __restrict__ Wp, int KC, int P, int groups,
       int S, int C, int full, Epi ep) {
  extern __shared__ float lds[];
  constexpr bool PX = Ring<T, RT, NT, WK>::kPrefetchX;
  constexpr int RX = PX ? RT : 1;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  int z = 0, ng = blockIdx.x, ks = blockIdx.y;
  int Sb = S;                                      // K splits of this block's column group
  if constexpr (!CHUNKED) {
    if (full < groups) {
      const int b = blockIdx.x;
      if (b < full) {
        ks = 0;
        Sb = 1;
      } else {
        ng = full + (b - full) / S;
        ks = (b - full) % S;
      }
    }
  } else {
    const int b = blockIdx.x;
    z = (b >> 3) % C;                              // row chunk
    const int u = ((b >> 3) / C) * 8 + (b & 7);    // unit: column group + K split
    if (u >= groups * S) return;                   // ids past the last unit (block-uniform)
    ng = u % groups;
    ks = u / groups;
  }
  constexpr int CR = 16 * RT;                      // rows per chunk when chunked
  const int rb = CR * z;                           // the chunk's first output row
  const int Rs = CHUNKED ? CR : ep.R;              // rows per chunk (partial-tile stride)
  const int R = CHUNKED ? min(CR, ep.R - rb) : ep.R;  // rows of this chunk
  const int kb0 = (KC * ks) / Sb, kb1 = (KC * (ks + 1)) / Sb;  // this block's K-blocks
  const int kc0 = kb0 + ((kb1 - kb0) * wave) / WK;
  const int kc1 = kb0 + ((kb1 - kb0) * (wave + 1)) / WK;
  const int nk = kc1 - kc0;

  // Folded RMSNorm: the rows' fixed-point sums of squares are read now (one
  // row per thread) and only used by the epilogue, so their latency hides
  // behind the weight stream.
  const bool ss_early = ep.ss_in && R <= (int)blockDim.x;
  uint64_t ssw[3] = {0, 0, 0};
  if (ss_early && (int)threadIdx.x < R) ss_load(ep.ss_in, ep.ss_stride, ep.row0 + rb + threadIdx.x, ssw);
  if (ep.ss_clear && ng == 0 && ks == 0 && z == 0)
    for (int i = threadIdx.x; i < 3 * ep.ss_stride; i += blockDim.x)
      __hip_atomic_store(ep.ss_clear + i, (uint64_t)0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  // the residual-add epilogue's operands that do not depend on the product,
  // loaded now for the same reason; the 4-tile kernels with a 2-deep ring
  // have no registers to spare for them
  constexpr bool kPre = !(NT == 4 && D >= 2);
  EpiPre pre;
  if constexpr (kPre) epilogue_prefetch(pre, NT * 16, ng * NT * 16, ep, threadIdx.x, blockDim.x, rb, R);

  f32x4_t acc[RT][NT];
#pragma unroll
  for (int mt = 0; mt < RT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int lrow = lane & 15;
  const int koff = (lane >> 4) * 32;
  // Packed layout: tiles in groups of P, K-block-major inside a group, so a
  // wave whose NT tiles form (part of) one group streams one contiguous run.
  const T* wb = Wp + lane * 8;
  size_t toff[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int t = ng * NT + nt;
    toff[nt] = ((size_t)(t / P) * KC * P + t % P) * kBlockElems;
  }
  const size_t kstride = (size_t)P * kBlockElems;
  // Rows past R read row R-1 instead (no per-lane branch): MFMA rows are
  // independent and padding rows are never stored.
  auto xload = [&](int kc, int mt, ActFrag<T> (&x)[4]) {
    const int row = ep.row0 + rb + min(mt * 16 + lrow, R - 1);
    const T* xp = X + act_offset(row, kc * 128 + koff, KC * 128);
#pragma unroll
    for (int j = 0; j < 4; ++j) x[j] = act_load<T>(xp + j * 512, xplane);
  };

  // Slot d holds the weights (and activations) of one 128-wide K-block; it
  // is refilled with the block D ahead as soon as it has been consumed.
  Frag<T> wr[D][NT][4];
  ActFrag<T> xr[D][RX][4];
  auto load = [&](int kc, Frag<T> (&w)[NT][4], ActFrag<T> (&x)[RX][4]) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        w[nt][j] = CHUNKED ? frag_load<T>(wb + toff[nt] + kc * kstride + j * 512)
                          : frag_load_nt<T>(wb + toff[nt] + kc * kstride + j * 512);
    if constexpr (PX) {
#pragma unroll
      for (int mt = 0; mt < RT; ++mt) xload(kc, mt, x[mt]);
    }
  };
  auto compute = [&](int kc, const Frag<T> (&w)[NT][4], const ActFrag<T> (&x)[RX][4]) {
#pragma unroll
    for (int mt = 0; mt < RT; ++mt) {
      ActFrag<T> xt[4];
      if constexpr (PX) {
#pragma unroll
        for (int j = 0; j < 4; ++j) xt[j] = x[mt][j];
      } else {
        xload(kc, mt, xt);
      }
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) mfma(acc[mt][nt], xt[j], w[nt][j]);
    }
  };
#pragma unroll
  for (int d = 0; d < D; ++d)
    if (d < nk) load(kc0 + d, wr[d], xr[d]);
  int base = 0;
  // Steady state with no conditions inside, so the compiler keeps the other
  // D-1 slots' loads in flight while one slot is consumed.
  for (; base + 2 * D <= nk; base += D) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      compute(kc0 + base + d, wr[d], xr[d]);
      load(kc0 + base + D + d, wr[d], xr[d]);
    }
  }
  // Tail: fewer than 2D blocks left, the first min(D, nk - base) in flight.
#pragma unroll
  for (int d = 0; d < D; ++d) {
    if (base + d < nk) {
      compute(kc0 + base + d, wr[d], xr[d]);
      if (base + D + d < nk) load(kc0 + base + D + d, wr[d], xr[d]);
    }
  }
#pragma unroll
  for (int d = 0; d < D; ++d)
    if (base + D + d < nk) compute(kc0 + base + D + d, wr[d], xr[d]);

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
  if (Sb > 1) {
    // Split-K over blocks: publish this block's partial tile; the block that
    // arrives last for this column group sums all partials in split order
    // (deterministic) and runs the epilogue, then re-arms the counter.
    // Partials travel with device-coherent (agent-scope) stores and loads,
    // which bypass the per-XCD L2, so no L2 write-back / invalidate fence is
    // needed: the stores are complete (s_waitcnt) before the counter
    // increment, and the last block reads them after seeing the count.  A
    // release / acquire pair on the counter would say the same in the C++
    // memory model, but on gfx950 an agent-scope release writes back and an
    // acquire invalidates the whole L2 of the XCD, which costs more than the
    // split saves; the wait below is the one ordering the stores need.
    __shared__ int s_last;
    const int cols = NT * 16;
    const size_t unit_part = ((size_t)ng * C + z) * Sb;  // this chunk's Sb partial tiles
    float* mine = ep.kpart + (unit_part + ks) * (size_t)(Rs * cols);
    for (int e = threadIdx.x; e < R * cols; e += 64 * WK) {
      const int row = e / cols, c = e - row * cols;
      __hip_atomic_store(mine + e, tile[row * tld + c], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this thread's stores are done
    __syncthreads();
    if (threadIdx.x == 0)
      s_last = __hip_atomic_fetch_add(ep.kcount + ng * C + z, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == Sb - 1;
    __syncthreads();
    if (!s_last) return;
    // Loads are issued four splits at a time so that their latencies
    // overlap; the sum keeps split order.
    const float* all = ep.kpart + unit_part * (size_t)(Rs * cols);
    const size_t pstride = (size_t)Rs * cols;
    for (int e = threadIdx.x; e < R * cols; e += 64 * WK) {
      float sum = 0.f;
      int k = 0;
      for (; k + 4 <= Sb; k += 4) {
        float v[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
          v[i] = __hip_atomic_load(all + (k + i) * pstride + e, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
        for (int i = 0; i < 4; ++i) sum += v[i];
      }
      for (; k < Sb; ++k)
        sum += __hip_atomic_load(all + k * pstride + e, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const int row = e / cols, c = e - row * cols;
      tile[row * tld + c] = sum;
    }
    if (threadIdx.x == 0) __hip_atomic_store(ep.kcount + ng * C + z, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
  }
  if (ep.ss_in) {
    // Output row r times 1 / rms(h[row0 + rb + r]): the normalisation commutes
    // with the contraction (a per-row scale of X).
    __shared__ float s_rs[256];
    if (ss_early) {
      if ((int)threadIdx.x < R) s_rs[threadIdx.x] = ss_rstd(ssw, ep.norm_inv_d, ep.norm_eps);
    } else {
      for (int row = threadIdx.x; row < R; row += blockDim.x) {
        uint64_t w[3];
        ss_load(ep.ss_in, ep.ss_stride, ep.row0 + rb + row, w);
        s_rs[row] = ss_rstd(w, ep.norm_inv_d, ep.norm_eps);
      }
    }
    __syncthreads();
    const int cols = NT * 16;
    for (int e = threadIdx.x; e < R * cols; e += blockDim.x) {
      const int row = e / cols, c = e - row * cols;
      tile[row * tld + c] *= s_rs[row];
    }
    __syncthreads();
  }
  epilogue<T>(tile, tld, NT * 16, ng * NT * 16, ep, ng, threadIdx.x, blockDim.x, rb, R, kPre ? &pre : nullptr);
}

// Rows per chunk of a GEMM with more rows than that: 32 (2 row tiles per
// wave).  16-row chunks were measured slower on the 7B step (+0.6 ms at 32
// rows, +1.2 ms at 192).
constexpr int kChunkRows = 32;

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

// Few rows (R <= 32): the GEMM streams W once and is bound by HBM latency
// and bandwidth.  Measured on MI355X (7B-shaped projections, R = 16), the
// fastest plans keep about max(1024, weight bytes / 224 KB) waves in flight
// (fewer, longer waves stream better; small matrices still need enough
// waves to cover the chip), prefer wide column groups (an activation
// fragment then feeds more weight tiles) and avoid cross-block split-K
// unless K is long, where narrowing the column group would be worse.
static void plan_few_rows(GemmShape& s, int epi_kind) {
  const int KC = s.K / 128;
  const int RT = round_rt(s.R);
  const double target = std::max(1024.0, (double)s.N * s.K * 2 / (224.0 * 1024));
  const double enough = 0.9 * target;
  // SwiGLU pairs gate and up tiles inside a column group: NT must be even.
  const int narrowest = epi_kind == EPI_SWIGLU ? 2 : 1;
  for (int nt = 4; nt >= narrowest; nt /= 2) {
    if (s.N % (16 * nt)) continue;
    const double groups = s.N / (16 * nt);
    int wk = 1;
    while (wk < 8 && groups * wk < enough && KC >= 2 * wk && lds_bytes(RT, nt, 2 * wk) <= 65536) wk *= 2;
    int S = 1;
    if (groups * wk < enough) {
      const bool long_k = KC >= 64;
      if (!long_k && nt > narrowest) continue;  // short K: narrower column groups instead of split-K
      while (S < 16 && groups * wk * S < enough && KC / (wk * S * 2) >= 3 &&
             groups * 2 * S * s.R * nt * 16 <= (double)kGemmPartFloats && groups <= kGemmCounters)
        S *= 2;
    }
    s.NT = nt;
    s.WK = wk;
    s.S = S;
    // A deeper ring pays off once the grid outgrows one wave per slot.
    s.D = (nt == 4 && groups * wk * S > 2048) ? 2 : 0;
    return;
  }
}

// Residual projections (O and down) with <= 16 rows: 64-column groups of 8
// waves split K across 4 blocks when K allows 7+ K-blocks per block (step
// latency measured on the 7B shapes: the O projection gains ~0.6 us per call
// over the narrow-group plan; fewer blocks run the residual / next-norm
// epilogue).
static bool plan_residual(GemmShape& s) {
  const int KC = s.K / 128;
  if (s.R > 16 || s.N % 64 || KC < 28) return false;
  const int groups = s.N / 64;
  if (groups > (int)kGemmCounters || (size_t)groups * 4 * s.R * 64 > kGemmPartFloats) return false;
  s.NT = 4;
  s.WK = 8;
  s.S = 4;
  s.D = 0;
  return true;
}

// Plans measured at the step level for the 7B-shaped projections: with 17-32
// rows (2 row tiles per wave, one chunk), 33-64 rows (two 32-row chunks) and
// more (three or more chunks).  The rule above over-splits the long-K down
// projection and, once chunked, keeps too many waves per chunk: the C chunk
// blocks of a unit already multiply the waves in flight by C.
struct MeasuredPlan { int epi, N, K, NT, WK, S, D; };
static const MeasuredPlan kPlans32[] = {
    {EPI_RESID, 3584, 18944, 4, 4, 4, 0},    // down: -107 us per n = 32 step vs the rule
    {EPI_RESID, 3584, 3584, 2, 8, 2, 0},     // O: -29 us
    {EPI_SWIGLU, 37888, 3584, 4, 4, 1, 0},   // gate/up: -32 us
    {EPI_ARGMAX, 152064, 3584, 4, 4, 1, 0},  // LM head: -16 us
};
static const MeasuredPlan kPlans64[] = {     // per 32-row chunk, C = 2
    {EPI_RESID, 3584, 18944, 4, 4, 2, 0},    // down: -272 us per n = 64 step vs the rule
    {EPI_RESID, 3584, 3584, 2, 8, 1, 0},     // O: -195 us
    {EPI_QKV, 4608, 3584, 4, 4, 1, 0},       // QKV: -134 us
    {EPI_SWIGLU, 37888, 3584, 4, 2, 1, 2},   // gate/up: -115 us
    {EPI_ARGMAX, 152064, 3584, 4, 1, 1, 2},  // LM head: -26 us
};
static const MeasuredPlan kPlansMany[] = {   // per 32-row chunk, C >= 3 (measured at C = 6, R = 192)
    {EPI_RESID, 3584, 18944, 4, 4, 2, 0},    // down: -594 us per R = 192 step vs the rule
    {EPI_RESID, 3584, 3584, 2, 2, 1, 0},     // O: -520 us
    {EPI_QKV, 4608, 3584, 4, 2, 1, 0},       // QKV: -309 us
    {EPI_SWIGLU, 37888, 3584, 4, 1, 1, 2},   // gate/up: -569 us
    {EPI_ARGMAX, 152064, 3584, 4, 1, 1, 2},  // LM head: -77 us
};

void gemm_plan(GemmShape& s, int epi_kind) {
  // More than kChunkRows rows run as chunks of kChunkRows (see k_gemm), each
  // planned as a kChunkRows-row GEMM.
  const int R = s.R;
  s.R = std::min(R, kChunkRows);
  s.D = 0;
  s.NT = 0;
  bool measured = false;
  auto lookup = [&](const MeasuredPlan* t, size_t n) {
    for (size_t i = 0; i < n; ++i)
      if (t[i].epi == epi_kind && t[i].N == s.N && t[i].K == s.K) {
        s.NT = t[i].NT; s.WK = t[i].WK; s.S = t[i].S; s.D = t[i].D;
        measured = true;
      }
  };
  // each table only where it was measured (the 32-row plans measured no
  // better as chunk plans)
  if (R > 16 && R <= 32) lookup(kPlans32, sizeof kPlans32 / sizeof kPlans32[0]);
  if (R > 32 && R <= 64) lookup(kPlans64, sizeof kPlans64 / sizeof kPlans64[0]);
  if (R > 64) lookup(kPlansMany, sizeof kPlansMany / sizeof kPlansMany[0]);
  if (!measured && !(epi_kind == EPI_RESID && plan_residual(s))) plan_few_rows(s, epi_kind);
  s.R = R;
  s.C = R > kChunkRows ? (R + kChunkRows - 1) / kChunkRows : 1;
  // split-K scratch for all chunks (kChunkRows-row partial tiles when chunked)
  const size_t rows = s.C > 1 ? (size_t)kChunkRows * s.C : (size_t)R;
  if (s.S > 1 && ((size_t)s.N * s.S * rows > kGemmPartFloats ||
                  (size_t)(s.N / (16 * s.NT)) * s.C > kGemmCounters))
    s.S = 1;
}

size_t gemm_blocks(const GemmShape& s) { return (size_t)s.N / (16 * s.NT); }

// A launch of G whole-K workgroups on n compute units runs floor(G / n)
// even rounds and a last one that leaves most units idle, while the time is
// set by the units with the most weight bytes to stream (the rate each unit
// sustains is the bound).  Splitting only the last round's groups over K
// into S = n / (G mod n) blocks evens the units out: gate/up at 16 rows
// (592 groups) gives 80 units 3 groups and the rest 2; split, every unit
// streams at most 2 1/3 (48.1 against 50.7 us).  Only where the last round
// costs 15% or more: the partials and the last block's reduction at the
// end of the launch cost more than the LM head's 8% (2376 groups, 9.28
// rounds: 169 -> 172 us split).
void gemm_tail_split(GemmShape& s, int n_cus) {
  const int groups = s.N / (16 * s.NT);
  const int KC = s.K / 128;
  if (s.C != 1 || s.S != 1 || n_cus < 1 || groups <= n_cus) return;
  const int rem = groups % n_cus;
  if (rem == 0 || (double)(groups / n_cus + 1) * n_cus < 1.15 * groups) return;
  const int S = std::min(n_cus / rem, KC / s.WK);
  if (S < 2 || (size_t)s.N * S * s.R > kGemmPartFloats || (size_t)groups > kGemmCounters) return;
  s.full = groups - rem;
  s.S = S;
}

static unsigned grid_blocks(const GemmShape& s) {
  const int units = s.N / (16 * s.NT) * s.S;
  return (unsigned)((units + 7) / 8 * 8 * s.C);
}

template <typename T, int RT, int NT, int WK, int D>
static hipError_t launch_t(const void* X, size_t xplane, const void* Wp, const GemmShape& s,
                           const Epi& ep, hipStream_t st) {
  size_t lds = lds_bytes(RT, NT, WK);
  const int groups = s.N / (16 * NT);
  if (s.C > 1)
    hipLaunchKernelGGL((k_gemm<T, RT, NT, WK, D, true>), dim3(grid_blocks(s)), dim3(64 * WK), lds, st,
                       reinterpret_cast<const T*>(X), xplane, reinterpret_cast<const T*>(Wp), s.K / 128,
                       pack_group(s.N), groups, s.S, s.C, groups, ep);
  else if (s.full > 0)
    hipLaunchKernelGGL((k_gemm<T, RT, NT, WK, D, false>), dim3(s.full + (groups - s.full) * s.S), dim3(64 * WK),
                       lds, st, reinterpret_cast<const T*>(X), xplane, reinterpret_cast<const T*>(Wp), s.K / 128,
                       pack_group(s.N), groups, s.S, 1, s.full, ep);
  else
    hipLaunchKernelGGL((k_gemm<T, RT, NT, WK, D, false>), dim3(groups, s.S), dim3(64 * WK), lds, st,
                       reinterpret_cast<const T*>(X), xplane, reinterpret_cast<const T*>(Wp), s.K / 128,
                       pack_group(s.N), groups, s.S, 1, groups, ep);
  return hipGetLastError();
}

template <typename T, int RT, int NT, int WK>
static hipError_t launch_d(const void* X, size_t xplane, const void* Wp, const GemmShape& s,
                           const Epi& ep, hipStream_t st) {
  if constexpr (NT == 4)
    if (s.D == 2) return launch_t<T, RT, NT, WK, 2>(X, xplane, Wp, s, ep, st);
  if (s.D != 0) return hipErrorInvalidValue;
  return launch_t<T, RT, NT, WK, Ring<T, RT, NT, WK>::D>(X, xplane, Wp, s, ep, st);
}

template <typename T, int RT, int NT>
static hipError_t launch_wk(const void* X, size_t xplane, const void* Wp, const GemmShape& s,
                            const Epi& ep, hipStream_t st) {
  switch (s.WK) {
    case 1: return launch_d<T, RT, NT, 1>(X, xplane, Wp, s, ep, st);
    case 2: return launch_d<T, RT, NT, 2>(X, xplane, Wp, s, ep, st);
    case 4: if constexpr (RT * NT <= 12) return launch_d<T, RT, NT, 4>(X, xplane, Wp, s, ep, st); break;
    case 8: if constexpr (RT * NT <= 6) return launch_d<T, RT, NT, 8>(X, xplane, Wp, s, ep, st); break;
    default: break;
  }
  return hipErrorInvalidValue;
}

template <typename T, int RT>
static hipError_t launch_nt(const void* X, size_t xplane, const void* Wp, const GemmShape& s,
                            const Epi& ep, hipStream_t st) {
  if (s.NT == 1) return launch_wk<T, RT, 1>(X, xplane, Wp, s, ep, st);
  if (s.NT == 2) return launch_wk<T, RT, 2>(X, xplane, Wp, s, ep, st);
  if constexpr (RT <= 2)
    if (s.NT == 4) return launch_wk<T, RT, 4>(X, xplane, Wp, s, ep, st);
  return hipErrorInvalidValue;
}

template <typename T>
static hipError_t launch_rt(const void* X, size_t xplane, const void* Wp, const GemmShape& s,
                            const Epi& ep, hipStream_t st) {
  // row tiles per block: 1 or 2 (more rows are chunked)
  const int rt = s.C > 1 ? kChunkRows / 16 : (s.R > 16 ? 2 : 1);
  if (rt == 2) return launch_nt<T, 2>(X, xplane, Wp, s, ep, st);
  return launch_nt<T, 1>(X, xplane, Wp, s, ep, st);
}

hipError_t launch_gemm(int dtype, const void* X, size_t xplane, const void* Wp,
                       const GemmShape& s, const Epi& ep, hipStream_t st) {
  if (s.R < 1 || s.R > kMaxRows || s.K < 128 || s.K % 128 || s.N < 16 * s.NT || s.N % (16 * s.NT))
    return hipErrorInvalidValue;
  if (s.C != (s.R > kChunkRows ? (s.R + kChunkRows - 1) / kChunkRows : 1)) return hipErrorInvalidValue;
  if (s.S < 1 || s.S > s.K / 128) return hipErrorInvalidValue;
  if (s.full < 0 || (s.full > 0 && (s.C != 1 || s.S < 2 || s.full >= s.N / (16 * s.NT))))
    return hipErrorInvalidValue;
  const size_t rows = s.C > 1 ? (size_t)kChunkRows * s.C : (size_t)s.R;
  if (s.S > 1 && (!ep.kpart || !ep.kcount || (size_t)(s.N / (16 * s.NT)) * s.C > kGemmCounters ||
                  (size_t)s.N * s.S * rows > kGemmPartFloats))
    return hipErrorInvalidValue;
  if (s.C > 1 && ep.row0 != 0) return hipErrorInvalidValue;
  if (lds_bytes(s.C > 1 ? kChunkRows / 16 : round_rt(s.R), s.NT, s.WK) > 65536) return hipErrorInvalidValue;
  return dtype == 1 ? launch_rt<bf16_t>(X, xplane, Wp, s, ep, st)
                    : launch_rt<float>(X, xplane, Wp, s, ep, st);
}

// ---- weight packing ------------------------------------------------------------
template <typename T>
__global__ void k_pack(int rows, int cols, const T* s0, const T* s1, const T* s2, const T* s3,
                       const int32_t* rowmap, T* dst) {
  const int KC = cols / 128;
  const int P = pack_group(rows);
  const size_t total = (size_t)rows * cols;
  for (size_t o = (size_t)blockIdx.x * blockDim.x + threadIdx.x; o < total;
       o += (size_t)gridDim.x * blockDim.x) {
    size_t blk = o / kBlockElems;
    int r = (int)(o - blk * kBlockElems);
    int j = r >> 9, lane = (r >> 3) & 63, e = r & 7;
    // blk = ((t / P) * KC + kc) * P + t % P for 16-row tile t, K-block kc
    const size_t q = blk / P;
    int kc = (int)(q % KC);
    int t = (int)(q / KC) * P + (int)(blk % P);
    int row = t * 16 + (lane & 15);
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
