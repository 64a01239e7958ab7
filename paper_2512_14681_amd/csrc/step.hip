// The non-GEMM kernels of one Jacobi iteration: the row forest of the step,
// the embedding gather, the vocabulary argmax reduction, greedy acceptance
// and the KV commit.  (The RMSNorms are folded into the projections: the
// residual adds write h * gain and the row sums of squares, the consumer
// GEMMs scale their output rows by 1 / rms.)
#include "jf_device.h"
#include "jf_internal.h"

namespace jf {

// ---- a1: rows of the step as a forest (Sec. 3.2, input assembly of App. A Alg. 1) ----
// parent[r]: row whose argmax r is checked against (-1: a root, predicted by
// the last committed row); pos[r] = C + depth(r); vis[r]: bit j set iff row j
// is r or an ancestor of r.  One thread per row walks its own ancestor chain
// (after par[] holds every row's parent).
__device__ void tree_walk(const int32_t* par, int r, int R, const int32_t* state, int32_t* parent,
                          int32_t* pos, uint64_t* vis) {
  if (r >= R) return;
  uint64_t w[kVisWords] = {};
  int depth = 0;
  int x = r;
  w[x >> 6] |= 1ull << (x & 63);
  while (par[x] >= 0) {
    x = par[x];
    w[x >> 6] |= 1ull << (x & 63);
    ++depth;
  }
  parent[r] = par[r];
  pos[r] = state[0] + depth;
  for (int i = 0; i < kVisWords; ++i) vis[r * kVisWords + i] = w[i];
}

__global__ void __launch_bounds__(kMaxRows) k_tree(SegArgs sg, int R, const int32_t* state, int32_t* flags,
                                                   int32_t* parent, int32_t* pos, uint64_t* vis) {
  __shared__ int32_t par[kMaxRows];
  const int r = threadIdx.x;
  if (r == 0 && flags) *flags = 0;  // flags are per step
  if (r < R) {
    int p = -1;
    for (int s = 0; s < sg.n; ++s) {
      if (r >= sg.first[s] && r < sg.first[s] + sg.nrows[s]) {
        p = (r == sg.first[s]) ? sg.attach[s] : r - 1;
        break;
      }
    }
    par[r] = p;
  }
  __syncthreads();
  tree_walk(par, r, R, state, parent, pos, vis);
}

hipError_t launch_tree(const SegArgs& segs, int R, const int32_t* state, int32_t* flags,
                       int32_t* parent, int32_t* pos, uint64_t* vis, hipStream_t st) {
  if (R < 1 || R > kMaxRows) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_tree, dim3(1), dim3(kMaxRows), 0, st, segs, R, state, flags, parent, pos, vis);
  return hipGetLastError();
}

// Packed training sequence (Sec. 3.1 noise-aware causal attention, App. C
// sequence packing): rows [noisy_0, clean_0, noisy_1, clean_1, ...], blocks
// of n.  Within a block copy each row follows the previous one; the first
// row of clean block i follows the last row of clean block i - 1, and the
// first row of noisy block i the last row of noisy block i - 1
// (noisy-context mask) or of clean block i - 1 (clean-context mask).  Both
// copies of block i get depths i n .. i n + n - 1, the block's own
// positions.
__global__ void __launch_bounds__(kMaxRows) k_tree_packed(int n_blocks, int n, int mask, const int32_t* state,
                                                          int32_t* flags, int32_t* parent, int32_t* pos,
                                                          uint64_t* vis) {
  __shared__ int32_t par[kMaxRows];
  const int R = 2 * n_blocks * n;
  const int r = threadIdx.x;
  if (r == 0 && flags) *flags = 0;
  if (r < R) {
    const int b = r / (2 * n), within = r - b * 2 * n;
    const int copy = within / n, k = within - copy * n;   // copy 0: noisy, 1: clean
    int p;
    if (k > 0) p = r - 1;
    else if (b == 0) p = -1;
    else if (copy == 1 || mask == kMaskCleanContext) p = 2 * b * n - 1;      // last row of clean b - 1
    else p = (2 * b - 1) * n - 1;                                            // last row of noisy b - 1
    par[r] = p;
  }
  __syncthreads();
  tree_walk(par, r, R, state, parent, pos, vis);
}

hipError_t launch_tree_packed(int n_blocks, int n, int mask, const int32_t* state, int32_t* flags,
                              int32_t* parent, int32_t* pos, uint64_t* vis, hipStream_t st) {
  if (n_blocks < 1 || n < 1 || 2 * n_blocks * n > kMaxRows) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_tree_packed, dim3(1), dim3(kMaxRows), 0, st, n_blocks, n, mask, state, flags, parent,
                     pos, vis);
  return hipGetLastError();
}

// ---- block reduction helper --------------------------------------------------
__device__ __forceinline__ float block_sum(float v, float* sh) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63, nw = blockDim.x >> 6;
  __syncthreads();
  if (l == 0) sh[w] = v;
  __syncthreads();
  float t = 0.f;
  for (int i = 0; i < nw; ++i) t += sh[i];  // fixed order: deterministic
  return t;
}

// ---- a2: embedding rows + the first RMSNorm's input -------------------------------
// h = E[token] (fp32); xg = h * gamma as activation planes in the GEMM-input
// layout; the row's sum of squares goes to the fixed-point accumulator ss
// (the QKV projection applies 1 / rms to its output rows).  Block 0 also
// zeroes ss_clear, the accumulator the first residual add fills.
template <typename T>
__global__ void __launch_bounds__(256)
    k_embed(const int32_t* __restrict__ tokens, const T* __restrict__ E, const float* __restrict__ gamma, int d,
            int V, float* __restrict__ h, T* __restrict__ xg, size_t xplane, uint64_t* ss, uint64_t* ss_clear,
            int ss_stride, int32_t* flags) {
  __shared__ float sh[16];
  const int r = blockIdx.x;
  if (r == 0 && ss_clear)
    for (int i = threadIdx.x; i < 3 * ss_stride; i += blockDim.x)
      __hip_atomic_store(ss_clear + i, (uint64_t)0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  int tok = tokens[r];
  if (tok < 0 || tok >= V) {
    if (threadIdx.x == 0 && flags) atomicOr(flags, 1);
    tok = 0;
  }
  const T* e = E + (size_t)tok * d;
  // d <= 4096: every thread's (at most 16) elements and gains are loaded at
  // once, then stored.
  float v[16], gm[16];
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const int i = threadIdx.x + 256 * k;
    v[k] = i < d ? to_f32<T>(e[i]) : 0.f;
    gm[k] = i < d ? gamma[i] : 0.f;
  }
  float ss_part = 0.f;
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const int i = threadIdx.x + 256 * k;
    if (i < d) {
      h[(size_t)r * d + i] = v[k];
      act_store<T>(xg + act_offset(r, i, d), xplane, v[k] * gm[k]);
    }
    ss_part += v[k] * v[k];
  }
  const float tot = block_sum(ss_part, sh);
  if (threadIdx.x == 0) {
    uint64_t w[3];
    ss_split(tot, w);
    for (int k = 0; k < 3; ++k)
      __hip_atomic_store(ss + (size_t)k * ss_stride + r, w[k], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

hipError_t launch_embed(int dtype, const int32_t* tokens, int R, const void* embed,
                        const float* gamma, int d, int V, float* h, void* xg, size_t xplane,
                        uint64_t* ss, uint64_t* ss_clear, int ss_stride, int32_t* flags,
                        hipStream_t st) {
  if (R < 1 || R > ss_stride || d > 16 * 256) return hipErrorInvalidValue;
  if (dtype == 1)
    hipLaunchKernelGGL(k_embed<bf16_t>, dim3(R), dim3(256), 0, st, tokens, (const bf16_t*)embed, gamma,
                       d, V, h, (bf16_t*)xg, xplane, ss, ss_clear, ss_stride, flags);
  else
    hipLaunchKernelGGL(k_embed<float>, dim3(R), dim3(256), 0, st, tokens, (const float*)embed, gamma, d,
                       V, h, (float*)xg, xplane, ss, ss_clear, ss_stride, flags);
  return hipGetLastError();
}

// ---- a7 tail: per-row maximum of the LM-head blocks' (value, index) keys ------
__global__ void k_argmax_reduce(const uint64_t* part, int nblocks, int stride, int32_t* g) {
  __shared__ uint64_t sh[16];
  const int r = blockIdx.x;
  uint64_t best = 0;
  for (int b = threadIdx.x; b < nblocks; b += blockDim.x) {
    uint64_t k = part[(size_t)b * stride + r];
    best = k > best ? k : best;
  }
  for (int o = 32; o > 0; o >>= 1) {
    uint64_t other = __shfl_xor(best, o);
    best = other > best ? other : best;
  }
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  if (l == 0) sh[w] = best;
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int i = 0; i < (int)(blockDim.x >> 6); ++i) best = sh[i] > best ? sh[i] : best;
    g[r] = (int32_t)argmax_key_index(best);
  }
}

hipError_t launch_argmax_reduce(const uint64_t* part, int nblocks, int stride, int R, int32_t* g,
                                hipStream_t st) {
  hipLaunchKernelGGL(k_argmax_reduce, dim3(R), dim3(1024), 0, st, part, nblocks, stride, g);
  return hipGetLastError();
}

// ---- a8: greedy acceptance of a linear draft + next draft --------------------------
// a = 1 + longest run of draft[k] == g[k-1]; pending = g[a-1]; next draft is
// the Jacobi update g[a-1], g[a], ... padded (mode 1) with pad ids at C+a+i.
__global__ void __launch_bounds__(kMaxRows) k_accept_linear(const int32_t* draft, const int32_t* g, int n, int mode,
                                uint64_t seed, int V, const int32_t* state, const int32_t* flags,
                                int32_t* result, int32_t* next_draft) {
  __shared__ int32_t s_a;
  __shared__ int32_t gs[kMaxRows];
  const int t = threadIdx.x;
  if (t < n) gs[t] = g[t];
  if (t == 0) s_a = n;
  __syncthreads();
  if (t >= 1 && t < n && draft[t] != gs[t - 1]) atomicMin(&s_a, t);
  __syncthreads();
  const int a = s_a;
  if (t == 0) {
    result[0] = a;
    result[1] = 0;
    result[2] = gs[a - 1];
    result[3] = flags ? flags[0] : 0;
  }
  if (next_draft && t < n) {
    int src = a - 1 + t;
    int v;
    if (src < n) v = gs[src];
    else v = mode == 1 ? pad_id(seed, (int64_t)state[0] + a + t, V) : 0;
    next_draft[t] = v;
  }
}

hipError_t launch_accept_linear(const int32_t* draft, const int32_t* g, int n, int mode,
                                uint64_t seed, int V, const int32_t* state, const int32_t* flags,
                                int32_t* result, int32_t* next_draft, hipStream_t st) {
  if (n < 1 || n > kMaxRows) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_accept_linear, dim3(1), dim3(kMaxRows), 0, st, draft, g, n, mode, seed, V, state,
                     flags, result, next_draft);
  return hipGetLastError();
}

// ---- a8 (tree): per-segment verification, winner and committed path ------------
// gv: the rows' argmax (global memory after a launch boundary, or a copy in
// LDS); m_sh: LDS scratch of JF_MAX_SEGMENTS counts.  Threads s < sg.n verify
// segment s, thread 0 picks the winner and walks its path.
__device__ void accept_tree(const SegArgs& sg, const int32_t* tokens, const int32_t* gv, const int32_t* parent,
                            const int32_t* flags, int32_t* seg_accept, int32_t* result, int32_t* path,
                            int32_t* m_sh) {
  const int s = threadIdx.x;
  if (s < sg.n) {
    int cnt = 0;
    for (int i = sg.verify_from[s]; i < sg.nrows[s]; ++i) {
      int r = sg.first[s] + i;
      int p = parent[r];
      if (p >= 0 && tokens[r] == gv[p]) ++cnt;
      else break;
    }
    m_sh[s] = cnt;
    seg_accept[s] = cnt;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int best = 0, bm = m_sh[0];
    for (int i = 1; i < sg.n; ++i)
      if (sg.role[i] == 1 && m_sh[i] > bm) { best = i; bm = m_sh[i]; }
    int k = sg.verify_from[best] + bm;
    int last = k > 0 ? sg.first[best] + k - 1 : sg.attach[best];
    if (last < 0) last = 0;  // unreachable for validated segments (row 0 is a root)
    int len = 0;
    for (int x = last; x >= 0; x = parent[x]) ++len;
    int i = len - 1;
    for (int x = last; x >= 0; x = parent[x]) path[i--] = x;
    result[0] = len;
    result[1] = best;
    result[2] = gv[last];
    result[3] = flags ? flags[0] : 0;
  }
}

__global__ void k_accept_tree(SegArgs sg, const int32_t* tokens, const int32_t* g,
                              const int32_t* parent, int R, const int32_t* flags,
                              int32_t* seg_accept, int32_t* result, int32_t* path) {
  __shared__ int32_t m[16];
  accept_tree(sg, tokens, g, parent, flags, seg_accept, result, path, m);
}

hipError_t launch_accept_tree(const SegArgs& segs, const int32_t* tokens, const int32_t* g,
                              const int32_t* parent, int R, const int32_t* flags,
                              int32_t* seg_accept, int32_t* result, int32_t* path,
                              hipStream_t st) {
  hipLaunchKernelGGL(k_accept_tree, dim3(1), dim3(64), 0, st, segs, tokens, g, parent, R, flags,
                     seg_accept, result, path);
  return hipGetLastError();
}

// ---- a7 tail + a8 (+ a9): argmax reduction, acceptance and commit in one launch ----
// Block r reduces row r's per-block keys to g[r] (as k_argmax_reduce) and
// publishes it; the last block to finish (counter state[2], re-armed by that
// block) reads all of g and runs the step's acceptance, and for a linear
// step asked to, its commit (C += a; the accepted rows' K/V are already in
// place).  g travels with device-coherent (L2-bypassing) stores and loads,
// each store complete before its block counts itself, so no L2 fence is
// needed (the split-K hand-off of the weight-streaming GEMM, the same way).
__device__ bool reduce_publish_last(const uint64_t* part, int nblocks, int stride, int R, int32_t* g,
                                    int32_t* count, uint64_t* sh, int* s_last) {
  const int r = blockIdx.x;
  uint64_t best = 0;
  for (int b = threadIdx.x; b < nblocks; b += blockDim.x) {
    uint64_t k = part[(size_t)b * stride + r];
    best = k > best ? k : best;
  }
  for (int o = 32; o > 0; o >>= 1) {
    uint64_t other = __shfl_xor(best, o);
    best = other > best ? other : best;
  }
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  if (l == 0) sh[w] = best;
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int i = 0; i < (int)(blockDim.x >> 6); ++i) best = sh[i] > best ? sh[i] : best;
    __hip_atomic_store(g + r, (int32_t)argmax_key_index(best), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // the store is done before the count
    const bool last = __hip_atomic_fetch_add(count, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == R - 1;
    if (last) __hip_atomic_store(count, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    *s_last = last;
  }
  __syncthreads();
  return *s_last;
}

__global__ void __launch_bounds__(1024)
    k_argmax_accept_linear(const uint64_t* part, int nblocks, int stride, const int32_t* draft, int n, int mode,
                           uint64_t seed, int V, int32_t* state, const int32_t* flags, int32_t* result,
                           int32_t* next_draft, int32_t* g, int commit, int max_ctx) {
  __shared__ uint64_t sh[16];
  __shared__ int32_t gs[kMaxRows];
  __shared__ int s_last, s_a, s_C;
  if (!reduce_publish_last(part, nblocks, stride, n, g, state + 2, sh, &s_last)) return;
  const int t = threadIdx.x;
  if (t < n) gs[t] = __hip_atomic_load(g + t, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (t == 0) {
    s_a = n;
    s_C = state[0];
  }
  __syncthreads();
  if (t >= 1 && t < n && draft[t] != gs[t - 1]) atomicMin(&s_a, t);
  __syncthreads();  // every read of draft is done (next_draft may be draft)
  const int a = s_a, C = s_C;
  if (t == 0) {
    result[0] = a;
    result[1] = 0;
    result[2] = gs[a - 1];
    result[3] = flags ? flags[0] : 0;
    if (commit) state[0] = C + a > max_ctx ? max_ctx : C + a;
  }
  if (next_draft && t < n) {
    const int src = a - 1 + t;
    next_draft[t] = src < n ? gs[src] : (mode == 1 ? pad_id(seed, (int64_t)C + a + t, V) : 0);
  }
}

__global__ void __launch_bounds__(1024)
    k_argmax_accept_tree(const uint64_t* part, int nblocks, int stride, SegArgs sg, const int32_t* tokens, int R,
                         const int32_t* parent, int32_t* state, const int32_t* flags, int32_t* seg_accept,
                         int32_t* result, int32_t* path, int32_t* g) {
  __shared__ uint64_t sh[16];
  __shared__ int32_t gs[kMaxRows];
  __shared__ int32_t m[16];
  __shared__ int s_last;
  if (!reduce_publish_last(part, nblocks, stride, R, g, state + 2, sh, &s_last)) return;
  for (int t = threadIdx.x; t < R; t += blockDim.x) gs[t] = __hip_atomic_load(g + t, __ATOMIC_RELAXED,
                                                                                __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  accept_tree(sg, tokens, gs, parent, flags, seg_accept, result, path, m);
}

hipError_t launch_argmax_accept_linear(const uint64_t* part, int nblocks, int stride, const int32_t* draft, int n,
                                       int mode, uint64_t seed, int V, int32_t* state, const int32_t* flags,
                                       int32_t* result, int32_t* next_draft, int32_t* g, int commit, int max_ctx,
                                       hipStream_t st) {
  if (n < 1 || n > kMaxRows || nblocks < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_argmax_accept_linear, dim3(n), dim3(1024), 0, st, part, nblocks, stride, draft, n, mode, seed,
                     V, state, flags, result, next_draft, g, commit, max_ctx);
  return hipGetLastError();
}

hipError_t launch_argmax_accept_tree(const uint64_t* part, int nblocks, int stride, const SegArgs& segs,
                                     const int32_t* tokens, int R, const int32_t* parent, int32_t* state,
                                     const int32_t* flags, int32_t* seg_accept, int32_t* result, int32_t* path,
                                     int32_t* g, hipStream_t st) {
  if (R < 1 || R > kMaxRows || nblocks < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_argmax_accept_tree, dim3(R), dim3(1024), 0, st, part, nblocks, stride, segs, tokens, R,
                     parent, state, flags, seg_accept, result, path, g);
  return hipGetLastError();
}

// ---- a9: KV commit ----------------------------------------------------------------
// The K/V of path row i moves from slot C + path[i] to slot C + i.  path is
// strictly increasing with path[i] >= i, so walking i upwards never
// overwrites a source that is still to be read; every (layer, kv head, K|V,
// dim) column is handled by one thread.
template <typename T>
__global__ void k_commit_move(T* kv, int n_pages, int G, int hd, const int32_t* page_table,
                              const int32_t* state, const int32_t* path, const int32_t* result,
                              int max_commit) {
  const int L_idx = blockIdx.y;
  const int col = blockIdx.x * blockDim.x + threadIdx.x;  // over G * 2 * hd
  if (col >= G * 2 * hd) return;
  const int kh = col / (2 * hd), rem = col - kh * 2 * hd, isv = rem / hd, dim = rem - isv * hd;
  int a = result[0];
  if (max_commit > 0 && a > max_commit) a = max_commit;
  const int C = state[0];
  const size_t page_elems = (size_t)2 * G * kPage * hd;
  T* base = kv + (size_t)L_idx * n_pages * page_elems;
  for (int i = 0; i < a; ++i) {
    int src = C + path[i], dst = C + i;
    if (src == dst) continue;
    T* ps = base + (size_t)page_table[src / kPage] * page_elems;
    T* pd = base + (size_t)page_table[dst / kPage] * page_elems;
    size_t os, od;
    if (!isv) {
      os = ((size_t)kh * kPage + src % kPage) * hd + dim;
      od = ((size_t)kh * kPage + dst % kPage) * hd + dim;
    } else {
      os = (size_t)G * kPage * hd + ((size_t)kh * hd + dim) * kPage + src % kPage;
      od = (size_t)G * kPage * hd + ((size_t)kh * hd + dim) * kPage + dst % kPage;
    }
    pd[od] = ps[os];
  }
}

// C += accepted count (capped), or += fixed_count when fixed_count > 0.
__global__ void k_commit_len(int32_t* state, const int32_t* result, int max_commit,
                             int fixed_count, int max_ctx) {
  int a = fixed_count > 0 ? fixed_count : result[0];
  if (max_commit > 0 && a > max_commit) a = max_commit;
  int c = state[0] + a;
  state[0] = c > max_ctx ? max_ctx : c;
}

hipError_t launch_commit(int dtype, void* kv, int L, int n_pages, int G, int hd,
                         const int32_t* page_table, int32_t* state, const int32_t* path,
                         const int32_t* result, int max_commit, int fixed_count, int max_ctx,
                         hipStream_t st) {
  if (path) {
    dim3 grid((G * 2 * hd + 255) / 256, L), block(256);
    if (dtype == 1)
      hipLaunchKernelGGL(k_commit_move<bf16_t>, grid, block, 0, st, (bf16_t*)kv, n_pages, G, hd,
                         page_table, state, path, result, max_commit);
    else
      hipLaunchKernelGGL(k_commit_move<float>, grid, block, 0, st, (float*)kv, n_pages, G, hd,
                         page_table, state, path, result, max_commit);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k_commit_len, dim3(1), dim3(1), 0, st, state, result, max_commit, fixed_count,
                     max_ctx);
  return hipGetLastError();
}

template <typename T>
__global__ void k_to_f32(const T* src, float* dst, int n) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
    dst[i] = to_f32<T>(src[i]);
}

hipError_t launch_to_f32(int dtype, const void* src, float* dst, int n, hipStream_t st) {
  dim3 grid((n + 255) / 256 < 1024 ? (n + 255) / 256 : 1024), block(256);
  if (dtype == 1)
    hipLaunchKernelGGL(k_to_f32<bf16_t>, grid, block, 0, st, (const bf16_t*)src, dst, n);
  else
    hipLaunchKernelGGL(k_to_f32<float>, grid, block, 0, st, (const float*)src, dst, n);
  return hipGetLastError();
}

__global__ void k_set_int(int32_t* p, int32_t v) { *p = v; }
__global__ void k_fill_int(int32_t* p, int n, int32_t v) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = v;
}
__global__ void k_copy_int(int32_t* d, const int32_t* s) { *d = *s; }

hipError_t launch_set_int(int32_t* p, int32_t v, hipStream_t st) {
  hipLaunchKernelGGL(k_set_int, dim3(1), dim3(1), 0, st, p, v);
  return hipGetLastError();
}

hipError_t launch_fill_int(int32_t* p, int n, int32_t v, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_fill_int, dim3((n + 255) / 256 < 64 ? (n + 255) / 256 : 64), dim3(256), 0, st, p, n, v);
  return hipGetLastError();
}
hipError_t launch_copy_int(int32_t* d, const int32_t* s, hipStream_t st) {
  hipLaunchKernelGGL(k_copy_int, dim3(1), dim3(1), 0, st, d, s);
  return hipGetLastError();
}

}  // namespace jf
