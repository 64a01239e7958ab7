// Jacobi trajectories (Sec. 2.1) and the noise-schedule point selection
// (Sec. 3.1, Eq. 7; App. C) -- the data-collection side of Jacobi Forcing.
//
// k_traj_record writes iterate y^(j+1) of an n-token block from y^(j) and the
// argmaxes of the step that fed y^(j)'s unaccepted tail: one HBM pass over n
// tokens.
//
// Point selection reads every point of every block once: HBM-bound, with
// little data per block (a 16-token block's 17 points are 1088 bytes), so
// the design goal is bytes in flight.  k_traj_select_multi gives each wave B
// blocks: one load of their B lengths, then every point of all B blocks and
// their fixed points y* loaded at once through range-checked buffer loads
// (when n <= 64 a load covers floor(64 / n) points: 4 points of a 16-token
// block per coalesced 256-byte load); lane j then owns point j (so
// max_points <= 64 there).
// k_traj_select (one block per wave, any n and length) is the general path.
// The unconverged count of a point is a popcount of the wave's mismatch
// ballot; the choice is exact integer arithmetic, |u w - t_num n| minimal
// (the fraction u / n closest to t_num / w), ties to the earliest point.
#include "jf_internal.h"

namespace jf {
namespace {

constexpr int kSelWaves = 4;   // waves (blocks of tokens) per workgroup
constexpr int kSelBatch = 8;   // loads issued back to back per wave
constexpr int kBufferFlags = 0x00020000;  // buffer descriptor word 3 (gfx9 family): 32-bit raw data

__global__ void __launch_bounds__(256) k_traj_record(const int32_t* prev, const int32_t* __restrict__ g,
                                                     int n, int rows, int32_t* out) {
  // positions < n - rows were accepted before the step; position n - rows is
  // the step's first row (the pending token): all of them stay.  Row r's
  // argmax is the update of position n - rows + 1 + r.
  const int keep = n - rows + 1;
  for (int i = blockIdx.x * 256 + threadIdx.x; i < n; i += gridDim.x * 256)
    out[i] = i < keep ? prev[i] : g[i - keep];
}

__global__ void __launch_bounds__(256) k_traj_select(const int32_t* __restrict__ traj,
                                                     const int32_t* __restrict__ len, int n_blocks, int n,
                                                     int max_points, int w, const int32_t* __restrict__ t_num,
                                                     int32_t* __restrict__ sel, int32_t* __restrict__ unconv) {
  const int lane = threadIdx.x & 63;
  const int b = blockIdx.x * kSelWaves + (threadIdx.x >> 6);
  if (b >= n_blocks) return;
  const int L = len[b];
  const size_t base = (size_t)b * max_points * n;
  int32_t* U = unconv ? unconv + (size_t)b * max_points : nullptr;
  if (L < 1 || L > max_points) {
    if (lane == 0) sel[b] = -1;
    if (U)
      for (int j = lane; j < max_points; j += 64) U[j] = -1;
    return;
  }
  const long long tn = (long long)(t_num ? t_num[b] : b % w) * n;
  const int32_t* T = traj + base;
  const int32_t* ys = T + (size_t)(L - 1) * n;
  long long best_d = -1;
  int best = 0;
  if (n <= 64) {
    const int per = 64 / n;                 // points per load
    const int used = per * n;
    const int sub = lane / n;
    const int pos = lane - sub * n;
    const bool active = lane < used;
    const int ystar = active ? ys[pos] : 0;
    const unsigned long long nmask = n == 64 ? ~0ull : ((1ull << n) - 1);
    for (int j0 = 0; j0 < L; j0 += per * kSelBatch) {
      int v[kSelBatch];
#pragma unroll
      for (int q = 0; q < kSelBatch; ++q) {
        const int j = j0 + q * per + sub;
        v[q] = (active && j < L) ? T[(size_t)j * n + pos] : ystar;
      }
#pragma unroll
      for (int q = 0; q < kSelBatch; ++q) {
        const int jq = j0 + q * per;
        if (jq >= L) break;
        const unsigned long long m = __ballot(v[q] != ystar);
        for (int s = 0; s < per; ++s) {
          const int j = jq + s;
          if (j >= L) break;
          const int u = __popcll((m >> (s * n)) & nmask);
          long long d = (long long)u * w - tn;
          d = d < 0 ? -d : d;
          if (best_d < 0 || d < best_d) { best_d = d; best = j; }
          if (U && lane == s) U[j] = u;
        }
      }
    }
  } else {
    for (int j = 0; j < L; ++j) {
      int u = 0;
      for (int c = 0; c < n; c += 64) {
        const int p = c + lane;
        const bool in = p < n;
        const bool diff = in && T[(size_t)j * n + p] != ys[p];
        u += __popcll(__ballot(diff));
      }
      long long d = (long long)u * w - tn;
      d = d < 0 ? -d : d;
      if (best_d < 0 || d < best_d) { best_d = d; best = j; }
      if (U && lane == 0) U[j] = u;
    }
  }
  if (U)
    for (int j = L + lane; j < max_points; j += 64) U[j] = -1;
  if (lane == 0) sel[b] = best;
}

// Minimum of a non-negative int over the 64 lanes: DPP within each row of
// 16 lanes (xor 1, xor 2, half-row mirror, row mirror), then the four row
// results through scalar registers.  All lanes must be active.
__device__ __forceinline__ int wave_min_nonneg(int x) {
  x = min(x, __builtin_amdgcn_update_dpp(0, x, 0xB1, 0xF, 0xF, false));   // quad_perm [1,0,3,2]
  x = min(x, __builtin_amdgcn_update_dpp(0, x, 0x4E, 0xF, 0xF, false));   // quad_perm [2,3,0,1]
  x = min(x, __builtin_amdgcn_update_dpp(0, x, 0x141, 0xF, 0xF, false));  // row_half_mirror
  x = min(x, __builtin_amdgcn_update_dpp(0, x, 0x140, 0xF, 0xF, false));  // row_mirror
  const int a = __builtin_amdgcn_readlane(x, 0), b = __builtin_amdgcn_readlane(x, 16);
  const int c = __builtin_amdgcn_readlane(x, 32), d = __builtin_amdgcn_readlane(x, 48);
  return min(min(a, b), min(c, d));
}

// B blocks per wave, all of their points held in K registers per block and
// the fixed point in one more (K * floor(64 / n) >= max_points, n <= 64,
// max_points <= 64, w < 2^24, n w < 2^25).
// Lane j takes point j's unconverged count u_j; a wave minimum over the key
// (d_j << 6) | j, d_j = |u_j w - t n|, picks the point, the earliest on
// ties.  The numerator t is clamped to [0, w] first: beyond that range d is
// monotone in u either way, so the choice is unchanged, and d <= n w keeps
// the key within 31 bits.
template <int B, int K>
__global__ void __launch_bounds__(256) k_traj_select_multi(const int32_t* __restrict__ traj,
                                                           const int32_t* __restrict__ len, int n_blocks,
                                                           int n, int max_points, int w,
                                                           const int32_t* __restrict__ t_num,
                                                           int32_t* __restrict__ sel,
                                                           int32_t* __restrict__ unconv) {
  const int lane = threadIdx.x & 63;
  // wave-uniform: a scalar register, so the buffer descriptors below are too
  const int b0 = __builtin_amdgcn_readfirstlane((blockIdx.x * kSelWaves + (threadIdx.x >> 6)) * B);
  if (b0 >= n_blocks) return;
  const int per = 64 / n;
  const int pos = lane % n;
  const bool active = lane < per * n;
  const unsigned long long nmask = n == 64 ? ~0ull : ((1ull << n) - 1);
  const bool mine = lane < B && b0 + lane < n_blocks;   // lane i carries block b0 + i's scalars
  const int Lr = mine ? len[b0 + lane] : 0;
  const int tr = mine ? (t_num ? min(max(t_num[b0 + lane], 0), w) : (b0 + lane) % w) : 0;
  // Loads through a buffer descriptor per block whose range is the block's
  // valid points (L n tokens): lanes past it read 0 from the hardware's range
  // check instead of branching.  Lane l of load q reads token l of the
  // per * n tokens that start at point q * per.
  // The fixed point y* (point L - 1) is one more load of the same batch.
  int v[B][K], ys[B];
#pragma unroll
  for (int i = 0; i < B; ++i) {
    const int L = __builtin_amdgcn_readlane(Lr, i);
    const int valid = (L >= 1 && L <= max_points) ? L * n * 4 : 0;
    __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int32_t*>(traj + (size_t)(b0 + i) * max_points * n), 0, valid, kBufferFlags);
#pragma unroll
    // whole offsets in the vector operand, the range-checked one
    for (int q = 0; q < K; ++q) v[i][q] = __builtin_amdgcn_raw_buffer_load_b32(rs, (q * per * n + lane) * 4, 0, 0);
    ys[i] = __builtin_amdgcn_raw_buffer_load_b32(rs, ((L - 1) * n + pos) * 4, 0, 0);
  }
  // this lane's own point (j = lane): load lq, slice lsl
  const int lq = lane / per;
  const int lsh = (lane - lq * per) * n;
  int res = 0;
#pragma unroll
  for (int i = 0; i < B; ++i) {
    const int b = b0 + i;
    if (b >= n_blocks) break;
    const int L = __builtin_amdgcn_readlane(Lr, i);
    int32_t* U = unconv ? unconv + (size_t)b * max_points : nullptr;
    if (L < 1 || L > max_points) {
      if (lane == i) res = -1;
      if (U && lane < max_points) U[lane] = -1;
      continue;
    }
    const int tn = __builtin_amdgcn_readlane(tr, i) * n;
    unsigned long long mine_m = 0;
#pragma unroll
    for (int q = 0; q < K; ++q) {
      if (q * per < L) {                                   // uniform: loads past L hold nothing
        const unsigned long long m = __builtin_amdgcn_ballot_w64(active && v[i][q] != ys[i]);
        mine_m = q == lq ? m : mine_m;
      }
    }
    const int u = __popcll((mine_m >> lsh) & nmask);
    const int d = abs((int)__umul24(u, w) - tn);   // u <= 64, w < 2^24: one 24-bit multiply
    const int key = lane < L ? (d << 6) | lane : 0x7FFFFFFF;
    const int best = wave_min_nonneg(key) & 63;
    if (U && lane < max_points) U[lane] = lane < L ? u : -1;
    if (lane == i) res = best;
  }
  if (mine) sel[b0 + lane] = res;
}

}  // namespace

hipError_t launch_traj_record(const int32_t* prev, const int32_t* g, int n, int rows, int32_t* out,
                              hipStream_t st) {
  const int blocks = (n + 255) / 256;
  hipLaunchKernelGGL(k_traj_record, dim3(blocks), dim3(256), 0, st, prev, g, n, rows, out);
  return hipGetLastError();
}

template <int B, int K>
static void launch_multi(const int32_t* traj, const int32_t* len, int n_blocks, int n, int max_points, int w,
                         const int32_t* t_num, int32_t* sel, int32_t* unconv, hipStream_t st) {
  const int blocks = (n_blocks + kSelWaves * B - 1) / (kSelWaves * B);
  hipLaunchKernelGGL((k_traj_select_multi<B, K>), dim3(blocks), dim3(64 * kSelWaves), 0, st, traj, len,
                     n_blocks, n, max_points, w, t_num, sel, unconv);
}

hipError_t launch_traj_select(const int32_t* traj, const int32_t* len, int n_blocks, int n, int max_points,
                              int w, const int32_t* t_num, int32_t* sel, int32_t* unconv, hipStream_t st) {
  const bool fast = n <= 64 && max_points <= 64 && w < (1 << 24) && (long long)n * w < (1 << 25);
  const int loads = fast ? (max_points + 64 / n - 1) / (64 / n) : 0;
  if (fast && loads <= 5)
    launch_multi<8, 5>(traj, len, n_blocks, n, max_points, w, t_num, sel, unconv, st);
  else if (fast && loads <= 8)
    launch_multi<4, 8>(traj, len, n_blocks, n, max_points, w, t_num, sel, unconv, st);
  else if (fast && loads <= 17)
    launch_multi<2, 17>(traj, len, n_blocks, n, max_points, w, t_num, sel, unconv, st);
  else
    hipLaunchKernelGGL(k_traj_select, dim3((n_blocks + kSelWaves - 1) / kSelWaves), dim3(64 * kSelWaves), 0,
                       st, traj, len, n_blocks, n, max_points, w, t_num, sel, unconv);
  return hipGetLastError();
}

}  // namespace jf
