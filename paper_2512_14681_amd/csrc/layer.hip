// The attention half of one decoder layer for a Jacobi step of at most 16
// rows, as one persistent launch: QKV projection (+ folded RMSNorm, RoPE,
// K/V into the cache slots C + r), block-causal GQA attention over the paged
// prefix and the step's own rows, the merge of the key splits, and the O
// projection with the residual add (+ the FFN norm's input).  These are the
// steps of the single forward pass of Eq. 3 (and of the tree pass of
// Sec. 3.2 / App. A Alg. 1) up to the feed-forward block.
//
// Why one launch: at <= 16 rows every phase here is latency-bound (the QKV
// and O weights are 59 MB, ~9 us of HBM at full rate, but four dependent
// launches cost ~40 us).  Inside one launch the phases hand over through
// flags instead of kernel boundaries, and the O projection's weights are
// loaded into registers while the attention still runs.
//
// Grid: one workgroup of 8 waves per compute unit, all co-resident (the host
// checks occupancy), so every wait below is on work that is running or done.
// Phases, each over all workgroups in turn:
//   1. QKV: 16-column tiles (tile t on workgroup t mod NB); the 8 waves take
//      interleaved 128-wide K-blocks and reduce in LDS in a fixed order.  The
//      epilogue writes q and the cache K/V with device-coherent stores, then
//      sets the tile's flag to this launch's epoch.
//   2. Attention items (kv head g, 16-row query tile, key split s): wait for
//      the flags of the QKV tiles the item reads, then the 8 waves take the
//      split's 32-key chunks in turn (online softmax, S^T = K Q^T and
//      O^T += V^T P^T on the matrix cores, as in attention.hip) and merge in
//      LDS.  With several splits each item stores its (max, sum, O) state and
//      bumps a counter; the item that arrives last merges the splits of its
//      (g, tile) in split order and sets the tile's merge flag.
//   3. O projection: the waves' weights are loaded first, then the workgroup
//      waits for every merge flag, loads the merged attention output and
//      runs the residual epilogue of gemm.hip (h += y, next norm's input and
//      row sums of squares).
// Data that another workgroup of the same launch reads goes through
// agent-scope (L2-bypassing) stores and loads; a flag is stored only after
// the workgroup's stores have completed (vmcnt(0) and a barrier).  Every wait
// is bounded: on timeout it sets JF_FLAG_SYNC in the step flags and the
// workgroup stops, so the launch always ends.
#include "jf_device.h"
#include "jf_internal.h"

namespace jf {

constexpr int kSideWaves = 8;
constexpr int kSideThreads = 64 * kSideWaves;
constexpr int kSideSpin = 1 << 18;  // polls before a wait gives up (~0.3 s)

// ---- device-coherent accesses (agent scope: visible across the XCDs' L2s) ----
__device__ __forceinline__ uint32_t ld_coh32(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t ld_coh64(const void* p) {
  return __hip_atomic_load(reinterpret_cast<const uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_cohf(const float* p) {
  return __uint_as_float(__hip_atomic_load(reinterpret_cast<const uint32_t*>(p), __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT));
}
__device__ __forceinline__ void st_coh32(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_cohf(float* p, float v) {
  __hip_atomic_store(reinterpret_cast<uint32_t*>(p), __float_as_uint(v), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coh16(bf16_t* p, bf16_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// 8 bf16 (16 B) as two agent-scope 64-bit loads
__device__ __forceinline__ Frag<bf16_t> frag_load_coh(const bf16_t* p) {
  const uint64_t a = ld_coh64(p), b = ld_coh64(p + 4);
  Frag<bf16_t> f;
  f.v = make_uint4((uint32_t)a, (uint32_t)(a >> 32), (uint32_t)b, (uint32_t)(b >> 32));
  return f;
}
__device__ __forceinline__ ActFrag<bf16_t> act_load_coh(const bf16_t* p, size_t plane) {
  ActFrag<bf16_t> a;
  a.hi = frag_load_coh(p);
  a.lo = frag_load_coh(p + plane);
  return a;
}
__device__ __forceinline__ void act_store_coh(bf16_t* p, size_t plane, float v) {
  const bf16_t hi = f32_to_bf16(v);
  st_coh16(p, hi);
  st_coh16(p + plane, f32_to_bf16(v - bf16_to_f32(hi)));
}
// This thread's stores have completed (written through to the coherence
// point) before anything after it is issued.  Written as the mnemonic so the
// assembler encodes it for the target.
__device__ __forceinline__ void stores_done() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Workgroup-uniform wait until flag[i] == epoch for every i in the ranges
// [lo[k], hi[k]) (k < n): wave 0 polls (agent-scope loads, 64 flags a load),
// the workgroup follows.  False on timeout (JF_FLAG_SYNC set in *err), or at
// once when another workgroup of the step has timed out.
__device__ bool wait_flags(const uint32_t* flag, const int* lo, const int* hi, int n, uint32_t epoch, int32_t* err,
                           int* s_ok) {
  if (threadIdx.x < 64) {
    bool ok = false;
    for (int it = 0; it < kSideSpin; ++it) {
      // every load of a poll is issued before any is compared (no
      // short-circuit), so one poll costs one memory round trip; the host
      // bounds the ranges to at most 6 flags per lane (launch_attn_block)
      uint32_t seen[6];
      int m = 0;
      for (int k = 0; k < n; ++k)
        for (int i = lo[k] + (int)threadIdx.x; i < hi[k] && m < 6; i += 64) seen[m++] = ld_coh32(flag + i);
      const uint32_t e = ld_coh32(reinterpret_cast<const uint32_t*>(err));
      bool mine = true;
      for (int k = 0; k < m; ++k) mine &= seen[k] == epoch;
      if (__all(mine)) { ok = true; break; }
      if (e & JF_FLAG_SYNC_BIT) break;
      __builtin_amdgcn_s_sleep(2);
    }
    if (threadIdx.x == 0) {
      *s_ok = ok;
      if (!ok) atomicOr(err, JF_FLAG_SYNC_BIT);
    }
  }
  __syncthreads();
  const bool ok = *s_ok != 0;
  __syncthreads();
  return ok;
}
__device__ bool wait_range(const uint32_t* flag, int lo, int hi, uint32_t epoch, int32_t* err, int* s_ok) {
  return wait_flags(flag, &lo, &hi, 1, epoch, err, s_ok);
}

// Sum of the 8 waves' 16 x 16 partial tiles in LDS (fixed order) into
// tile[16][17]; acc is this wave's MFMA accumulator (rows 4 (lane / 16) + i,
// column lane % 16).
__device__ void reduce_tile(const f32x4_t& acc, float* part, float* tile) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int i = 0; i < 4; ++i) part[wave * 256 + i * 64 + lane] = acc[i];
  __syncthreads();
  if (threadIdx.x < 256) {
    const int e = threadIdx.x;
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < kSideWaves; ++w) s += part[w * 256 + e];
    const int l = e & 63, i = e >> 6;
    tile[(4 * (l >> 4) + i) * 17 + (l & 15)] = s;
  }
  __syncthreads();
}

// One wave's share of NT 16-column tiles of Y = X W^T (tile offsets toff[]):
// K-blocks wave, wave + 8, ... of kc, two in flight; the activation loads are
// shared by the NT tiles.  Rows past R read row R - 1 (never stored).
template <int NT>
__device__ __forceinline__ void tile_mma(const bf16_t* __restrict__ X, size_t xplane, int K, int R,
                                         const bf16_t* __restrict__ W, const size_t (&toff)[NT], size_t kstride,
                                         int kc, f32x4_t (&acc)[NT]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lrow = lane & 15, koff = (lane >> 4) * 32;
  const int row = min(lrow, R - 1);
  const bf16_t* wb = W + lane * 8;
#pragma unroll
  for (int t = 0; t < NT; ++t) acc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const int nk = wave < kc ? (kc - wave + kSideWaves - 1) / kSideWaves : 0;
  Frag<bf16_t> w0[NT][4], w1[NT][4];
  ActFrag<bf16_t> x0[4], x1[4];
  auto load = [&](int i, Frag<bf16_t> (&w)[NT][4], ActFrag<bf16_t> (&x)[4]) {
    const int kb = wave + kSideWaves * i;
    const bf16_t* xp = X + act_offset(row, kb * 128 + koff, K);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
#pragma unroll
      for (int t = 0; t < NT; ++t) w[t][j] = frag_load_nt<bf16_t>(wb + toff[t] + kb * kstride + j * 512);
      x[j] = act_load<bf16_t>(xp + j * 512, xplane);
    }
  };
  auto mma = [&](const Frag<bf16_t> (&w)[NT][4], const ActFrag<bf16_t> (&x)[4]) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int t = 0; t < NT; ++t) mfma(acc[t], x[j], w[t][j]);
  };
  if (nk > 0) load(0, w0, x0);
  int i = 0;
  for (; i + 2 <= nk; i += 2) {
    load(i + 1, w1, x1);
    mma(w0, x0);
    if (i + 2 < nk) load(i + 2, w0, x0);
    mma(w1, x1);
  }
  if (i < nk) mma(w0, x0);
}

// ---- phase 1: the QKV tiles of a workgroup (one, or two streamed together) ------
template <int HD>
__device__ void qkv_epilogue(const SideArgs& a, int t, const float* tile, const float* s_rs) {
  // RoPE on q/k (pairs (i, i + hd/2) sit at columns c and c ^ 8), q as
  // activation planes, k/v into the cache slot C + row
  const int H = a.H, G = a.G, half = HD / 2;
  const int C = a.state[0];
  bf16_t* q = reinterpret_cast<bf16_t*>(a.q);
  bf16_t* kv = reinterpret_cast<bf16_t*>(a.kv);
  const size_t page_elems = (size_t)2 * G * kPage * HD;
  if (threadIdx.x < 16 * 16) {
    const int row = threadIdx.x >> 4, c = threadIdx.x & 15;
    if (row < a.R) {
      const int pr = t * 16 + c;  // packed row
      const int head = pr / HD, w = pr - head * HD;
      const float x = tile[row * 17 + c] * s_rs[row];
      float out;
      int dim;
      if (head < H + G) {
        const int tt = w >> 4, cc = w & 15;
        const int i = 8 * tt + (cc & 7);
        dim = cc < 8 ? i : half + i;
        const float y = tile[row * 17 + (c ^ 8)] * s_rs[row];
        const int pos = a.pos[row];
        const float cs = a.rope_cos[(size_t)pos * half + i];
        const float sn = a.rope_sin[(size_t)pos * half + i];
        out = cc < 8 ? (x * cs - y * sn) : (x * cs + y * sn);
      } else {
        dim = w;
        out = x;
      }
      if (head < H) {
        act_store_coh(q + ((size_t)row * H + head) * HD + dim, a.q_plane, out);
      } else {
        const int slot = C + row;
        if (slot >= a.max_ctx) {
          atomicOr(a.flags, 2);
        } else {
          bf16_t* page = kv + (size_t)a.page_table[slot / kPage] * page_elems;
          const int s = slot % kPage;
          if (head < H + G)
            st_coh16(page + ((size_t)(head - H) * kPage + s) * HD + dim, f32_to_bf16(out));
          else
            st_coh16(page + (size_t)G * kPage * HD + ((size_t)(head - H - G) * HD + dim) * kPage + s,
                     f32_to_bf16(out));
        }
      }
    }
  }
}

template <int HD, int NT>
__device__ void qkv_tiles(const SideArgs& a, const int (&t)[NT], float* lds) {
  float* part = lds;
  float* tile = lds + kSideWaves * 256;
  __shared__ float s_rs[16];
  size_t toff[NT];
#pragma unroll
  for (int i = 0; i < NT; ++i) toff[i] = ((size_t)(t[i] / a.p_qkv) * a.kc_qkv * a.p_qkv + t[i] % a.p_qkv) * kBlockElems;
  f32x4_t acc[NT];
  tile_mma<NT>(reinterpret_cast<const bf16_t*>(a.x), a.x_plane, a.d, a.R, reinterpret_cast<const bf16_t*>(a.w_qkv),
               toff, (size_t)a.p_qkv * kBlockElems, a.kc_qkv, acc);
  if (threadIdx.x < a.R) {
    uint64_t w[3];
    ss_load(a.ss_in, a.ss_stride, threadIdx.x, w);
    s_rs[threadIdx.x] = ss_rstd(w, a.norm_inv_d, a.norm_eps);
  }
#pragma unroll
  for (int i = 0; i < NT; ++i) {
    reduce_tile(acc[i], part, tile);
    qkv_epilogue<HD>(a, t[i], tile, s_rs);
    stores_done();
    __syncthreads();
    if (threadIdx.x == 0) st_coh32(a.sync + t[i], a.epoch);
  }
}

// Bits j0 .. j0 + 7 of a row's in-step visibility (rows < 64: one word).
__device__ __forceinline__ uint32_t vis8(uint64_t v, int j0) {
  if (j0 >= 64 || j0 <= -8) return 0u;
  if (j0 >= 0) return (uint32_t)(v >> j0) & 0xFFu;
  return ((uint32_t)v << (-j0)) & 0xFFu;
}
__device__ __forceinline__ uint32_t lowbits8(int n) { return n >= 8 ? 0xFFu : (n <= 0 ? 0u : (1u << n) - 1u); }

// ---- phase 2: an attention item (kv head g, query tile qt, key split s) ----------
// The split merge: the (max, sum, O) states of S splits of 16 query rows; the
// thread (row q, dims 4 dg .. 4 dg + 3) issues all its loads at once (SMAX
// unrolled, splits past S re-read split S - 1 with weight 0), then combines
// them in split order.
template <int HD, int SMAX>
__device__ void merge_splits(const SideArgs& a, int g, int qt, int S) {
  const int grp = a.H / a.G, R = a.R, nq = grp * R;
  const size_t nrow = (size_t)R * a.H;
  bf16_t* out = reinterpret_cast<bf16_t*>(a.attn);
  for (int e = threadIdx.x; e < 16 * (HD / 4); e += kSideThreads) {
    const int qq = e / (HD / 4), dg = e - qq * (HD / 4);
    const int qi = qt * 16 + qq;
    if (qi >= nq) continue;
    const int hq = qi / R, rr = qi - hq * R;
    const size_t qidx = (size_t)rr * a.H + g * grp + hq;
    float m[SMAX], l[SMAX], o[SMAX][4];
#pragma unroll
    for (int sp = 0; sp < SMAX; ++sp) {
      const size_t i = (size_t)min(sp, S - 1) * nrow + qidx;
      const uint64_t ml = ld_coh64(a.ml_part + i * 2);
      m[sp] = __uint_as_float((uint32_t)ml);
      l[sp] = __uint_as_float((uint32_t)(ml >> 32));
      const uint64_t o01 = ld_coh64(a.o_part + i * HD + 4 * dg), o23 = ld_coh64(a.o_part + i * HD + 4 * dg + 2);
      o[sp][0] = __uint_as_float((uint32_t)o01);
      o[sp][1] = __uint_as_float((uint32_t)(o01 >> 32));
      o[sp][2] = __uint_as_float((uint32_t)o23);
      o[sp][3] = __uint_as_float((uint32_t)(o23 >> 32));
    }
    float M = -INFINITY;
#pragma unroll
    for (int sp = 0; sp < SMAX; ++sp) M = fmaxf(M, m[sp]);
    float num[4] = {0.f, 0.f, 0.f, 0.f}, den = 0.f;
#pragma unroll
    for (int sp = 0; sp < SMAX; ++sp) {
      const float w = (sp >= S || m[sp] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m[sp] - M);
      den += l[sp] * w;
#pragma unroll
      for (int k = 0; k < 4; ++k) num[k] += o[sp][k] * w;
    }
    const size_t base = act_offset(rr, (g * grp + hq) * HD + 4 * dg, a.H * HD);
#pragma unroll
    for (int k = 0; k < 4; ++k) act_store_coh(out + base + k, a.attn_plane, num[k] / den);
  }
}

template <int HD>
__device__ bool attn_item(const SideArgs& a, int item, float* lds, int* s_ok) {
  const int ngt = a.G * a.qtiles;
  const int gt = item % ngt, s = item / ngt;
  const int g = gt / a.qtiles, qt = gt % a.qtiles;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int grp = a.H / a.G, R = a.R, nq = grp * R;
  const int ql = lane & 15, kg = lane >> 4;
  const int C = a.state[0];
  const int per = a.split_keys;
  // splits that hold keys: those below C + R (the host laid the splits over
  // its upper bound of C + R); every item of the step computes the same
  // count from the device's C, the others leave at once
  const int S = min(a.splits, (min(a.keys_ub, C + R) + per - 1) / per);
  if (s >= S) return true;
  const int k0 = s * per;
  const int lim = min(min(a.keys_ub, k0 + per), C + R);
  const int nch = lim > k0 ? (lim - k0 + 31) / 32 : 0;
  const bf16_t* kv = reinterpret_cast<const bf16_t*>(a.kv);
  const size_t page_elems = (size_t)2 * a.G * kPage * HD;
  const size_t k_off = (size_t)g * kPage * HD;
  const size_t vt_off = (size_t)a.G * kPage * HD + (size_t)g * HD * kPage;
  // this lane's query row
  const int qr = qt * 16 + ql;
  const bool qvalid = qr < nq;
  const int hl = qvalid ? qr / R : 0;
  const int r = qvalid ? qr - hl * R : 0;
  const int head = g * grp + hl;
  const uint64_t vw = a.vis ? a.vis[(size_t)r * kVisWords] : (r >= 63 ? ~0ull : ((2ull << r) - 1ull));

  // K rows of the two score tiles of a 32-key chunk (row i of tile kt is key
  // 8 (i / 4) + 4 kt + i % 4) and the V^T fragments of keys 8 kg .. 8 kg + 7
  Frag<bf16_t> kf[2][HD / 32], vf[HD / 16];
  auto load_chunk = [&](int c, bool coh) {
    const int kb = k0 + 32 * c;
    const bf16_t* page = kv + (size_t)a.page_table[kb / kPage] * page_elems;
    const int ko = kb % kPage;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      const bf16_t* kp = page + k_off + (size_t)(ko + 8 * (ql >> 2) + 4 * kt + (ql & 3)) * HD + 8 * kg;
#pragma unroll
      for (int cc = 0; cc < HD / 32; ++cc)
        kf[kt][cc] = coh ? frag_load_coh(kp + 32 * cc) : frag_load<bf16_t>(kp + 32 * cc);
    }
    const bf16_t* vp = page + vt_off + (size_t)ql * kPage + ko + 8 * kg;
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt)
      vf[dt] = coh ? frag_load_coh(vp + (size_t)dt * 16 * kPage) : frag_load<bf16_t>(vp + (size_t)dt * 16 * kPage);
  };
  // The wave's first chunk, if it lies in the committed prefix, does not
  // depend on this launch's QKV tiles: its loads go out before the wait.
  const bool pre = wave < nch && k0 + 32 * wave + 32 <= C;
  if (pre) load_chunk(wave, false);
  {
    const int tph = HD / 16;
    const int hl0 = (qt * 16) / R, hl1 = min(qt * 16 + 15, nq - 1) / R;
    const int lo[3] = {(g * grp + hl0) * tph, (a.H + g) * tph, (a.H + a.G + g) * tph};
    const int hi[3] = {(g * grp + hl1 + 1) * tph, (a.H + g + 1) * tph, (a.H + a.G + g + 1) * tph};
    if (!wait_flags(a.sync, lo, hi, 3, a.epoch, a.flags, s_ok)) return false;
  }
  ActFrag<bf16_t> qf[HD / 32];
  {
    const bf16_t* qp = reinterpret_cast<const bf16_t*>(a.q) + ((size_t)r * a.H + head) * HD + 8 * kg;
#pragma unroll
    for (int c = 0; c < HD / 32; ++c) qf[c] = qvalid ? act_load_coh(qp + 32 * c, a.q_plane) : act_zero<bf16_t>();
  }
  const float scale = 1.4426950408889634f / sqrtf((float)HD);  // log2(e) / sqrt(hd)
  float m_run = -INFINITY, l_run = 0.f;
  f32x4_t o[HD / 16];
#pragma unroll
  for (int dt = 0; dt < HD / 16; ++dt) o[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  for (int c = wave; c < nch; c += kSideWaves) {
    const int kb = k0 + 32 * c;
    if (!(pre && c == wave)) load_chunk(c, kb + 32 > C);  // chunks with this step's keys: coherent
    f32x4_t sc[2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      f32x4_t sh = {0.f, 0.f, 0.f, 0.f}, sl = sh;
#pragma unroll
      for (int cc = 0; cc < HD / 32; ++cc) {
        mfma(sh, kf[kt][cc], qf[cc].hi);
        mfma(sl, kf[kt][cc], qf[cc].lo);
      }
      sc[kt] = sh + sl;
    }
    const int key0 = kb + 8 * kg;  // key of p[0]; p[e] is key0 + e
    const uint32_t vis = lowbits8(lim - key0) & (lowbits8(C - key0) | vis8(vw, key0 - C));
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
    Frag<bf16_t> phi, plo;
    {
      uint32_t h[4], l[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        h[e] = pack_bf16x2(p[2 * e], p[2 * e + 1]);
        l[e] = pack_bf16x2(p[2 * e] - __uint_as_float(h[e] << 16), p[2 * e + 1] - __uint_as_float(h[e] & 0xFFFF0000u));
      }
      phi.v = make_uint4(h[0], h[1], h[2], h[3]);
      plo.v = make_uint4(l[0], l[1], l[2], l[3]);
    }
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) o[dt] *= alpha;
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) mfma(o[dt], vf[dt], phi);
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt) mfma(o[dt], vf[dt], plo);
  }

  // merge the 8 waves' states in LDS (per query row: weights 2^(m_w - M))
  float* s_m = lds;                        // [8][16]
  float* s_l = s_m + kSideWaves * 16;      // [8][16]
  float* s_f = s_l + kSideWaves * 16;      // [8][16]
  float* s_M = s_f + kSideWaves * 16;      // [16]
  float* s_den = s_M + 16;                 // [16]
  float* s_o = s_den + 16;                 // [8][16][HD + 4]
  {
    float lr = l_run;
    lr += __shfl_xor(lr, 16);
    lr += __shfl_xor(lr, 32);
    if (kg == 0) {
      s_m[wave * 16 + ql] = m_run;
      s_l[wave * 16 + ql] = lr;
    }
#pragma unroll
    for (int dt = 0; dt < HD / 16; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) s_o[(wave * 16 + ql) * (HD + 4) + dt * 16 + 4 * kg + i] = o[dt][i];
  }
  __syncthreads();
  if (threadIdx.x < 16) {
    const int qq = threadIdx.x;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kSideWaves; ++w) M = fmaxf(M, s_m[w * 16 + qq]);
    float den = 0.f;
#pragma unroll
    for (int w = 0; w < kSideWaves; ++w) {
      const float mw = s_m[w * 16 + qq];
      const float f = mw == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mw - M);
      s_f[w * 16 + qq] = f;
      den += s_l[w * 16 + qq] * f;
    }
    s_M[qq] = M;
    s_den[qq] = den;
  }
  __syncthreads();
  const size_t nrow = (size_t)R * a.H;
  bf16_t* out = reinterpret_cast<bf16_t*>(a.attn);
  // thread (query row qq, dims 4 dg .. 4 dg + 3)
  for (int e = threadIdx.x; e < 16 * (HD / 4); e += kSideThreads) {
    const int qq = e / (HD / 4), dg = e - qq * (HD / 4);
    const int qi = qt * 16 + qq;
    if (qi >= nq) continue;
    float num[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      num[k] = 0.f;
#pragma unroll
      for (int w = 0; w < kSideWaves; ++w) num[k] += s_o[(w * 16 + qq) * (HD + 4) + 4 * dg + k] * s_f[w * 16 + qq];
    }
    const int hq = qi / R, rr = qi - hq * R;
    if (S == 1) {
      const size_t base = act_offset(rr, (g * grp + hq) * HD + 4 * dg, a.H * HD);
#pragma unroll
      for (int k = 0; k < 4; ++k) act_store_coh(out + base + k, a.attn_plane, num[k] / s_den[qq]);
    } else {
      const size_t qidx = (size_t)rr * a.H + g * grp + hq;
      uint64_t* op = reinterpret_cast<uint64_t*>(a.o_part + ((size_t)s * nrow + qidx) * HD + 4 * dg);
      __hip_atomic_store(op, (uint64_t)__float_as_uint(num[0]) | ((uint64_t)__float_as_uint(num[1]) << 32),
                         __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(op + 1, (uint64_t)__float_as_uint(num[2]) | ((uint64_t)__float_as_uint(num[3]) << 32),
                         __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (dg == 0)
        __hip_atomic_store(reinterpret_cast<uint64_t*>(a.ml_part + ((size_t)s * nrow + qidx) * 2),
                           (uint64_t)__float_as_uint(s_M[qq]) | ((uint64_t)__float_as_uint(s_den[qq]) << 32),
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  stores_done();
  __syncthreads();
  uint32_t* merge_flag = a.sync + a.qkv_tiles;
  if (S == 1) {
    if (threadIdx.x == 0) st_coh32(merge_flag + gt, a.epoch);
    return true;
  }
  // the item that arrives last for (g, qt) merges the splits in split order
  uint32_t* cnt = a.sync + a.qkv_tiles + ngt + (a.epoch & 1) * ngt;
  if (threadIdx.x == 0)
    *s_ok = __hip_atomic_fetch_add(cnt + gt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == (uint32_t)S - 1;
  __syncthreads();
  const bool last = *s_ok != 0;
  __syncthreads();
  if (!last) return true;
  if (S <= 4) merge_splits<HD, 4>(a, g, qt, S);
  else if (S <= 8) merge_splits<HD, 8>(a, g, qt, S);
  else if (S <= 16) merge_splits<HD, 16>(a, g, qt, S);
  else merge_splits<HD, 32>(a, g, qt, S);
  stores_done();
  __syncthreads();
  if (threadIdx.x == 0) st_coh32(merge_flag + gt, a.epoch);
  return true;
}

// ---- phase 3: an O-projection tile with the residual epilogue ---------------------
template <int HD>
__device__ bool o_tile(const SideArgs& a, int t, float* lds, int* s_ok) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int kc = a.kc_o, K = a.H * HD;
  const size_t toff = ((size_t)(t / a.p_o) * kc * a.p_o + t % a.p_o) * kBlockElems;
  const size_t kstride = (size_t)a.p_o * kBlockElems;
  const bf16_t* wb = reinterpret_cast<const bf16_t*>(a.w_o) + toff + lane * 8;
  // weights first (at most 4 K-blocks per wave), then the wait
  constexpr int kMaxK = 4;
  const int nk = wave < kc ? (kc - wave + kSideWaves - 1) / kSideWaves : 0;
  Frag<bf16_t> w[kMaxK][4];
#pragma unroll
  for (int i = 0; i < kMaxK; ++i)
    if (i < nk)
#pragma unroll
      for (int j = 0; j < 4; ++j) w[i][j] = frag_load_nt<bf16_t>(wb + (size_t)(wave + kSideWaves * i) * kstride + j * 512);
  // the residual rows and gains the epilogue adds to, also before the wait
  float h_old = 0.f, gain = 0.f;
  if (threadIdx.x < 256 && (int)(threadIdx.x >> 4) < a.R) {
    const int col = t * 16 + (threadIdx.x & 15);
    h_old = a.h[(size_t)(threadIdx.x >> 4) * a.d + col];
    gain = a.gain_next[col];
  }
  if (!wait_range(a.sync + a.qkv_tiles, 0, a.G * a.qtiles, a.epoch, a.flags, s_ok)) return false;
  const int lrow = lane & 15, koff = (lane >> 4) * 32;
  const int row = min(lrow, a.R - 1);
  const bf16_t* X = reinterpret_cast<const bf16_t*>(a.attn);
  f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
  // all of the wave's activation loads go out before the first MFMA
  ActFrag<bf16_t> x[kMaxK][4];
#pragma unroll
  for (int i = 0; i < kMaxK; ++i) {
    // slots past the wave's K-blocks re-read its last one (a valid block even
    // when the wave has none), and are not used
    const int kb = min(wave + kSideWaves * min(i, max(nk - 1, 0)), kc - 1);
    const bf16_t* xp = X + act_offset(row, kb * 128 + koff, K);
#pragma unroll
    for (int j = 0; j < 4; ++j) x[i][j] = act_load_coh(xp + j * 512, a.attn_plane);
  }
#pragma unroll
  for (int i = 0; i < kMaxK; ++i)
    if (i < nk)
#pragma unroll
      for (int j = 0; j < 4; ++j) mfma(acc, x[i][j], w[i][j]);
  float* part = lds;
  float* tile = lds + kSideWaves * 256;
  reduce_tile(acc, part, tile);
  // residual add, then the next RMSNorm's input (h * gain) and the rows'
  // sums of squares over these 16 columns
  bf16_t* xg = reinterpret_cast<bf16_t*>(a.xg);
  if (threadIdx.x < 256) {
    const int rr = threadIdx.x >> 4, c = threadIdx.x & 15;
    float sq = 0.f;
    if (rr < a.R) {
      const int col = t * 16 + c;
      const float hn = h_old + tile[rr * 17 + c];
      a.h[(size_t)rr * a.d + col] = hn;
      act_store<bf16_t>(xg + act_offset(rr, col, a.d), a.xg_plane, hn * gain);
      sq = hn * hn;
    }
    // row sum over the 16 columns (lanes 16 rr .. 16 rr + 15)
#pragma unroll
    for (int o = 8; o > 0; o >>= 1) sq += __shfl_xor(sq, o);
    if (c == 0 && rr < a.R) ss_add(a.ss_out, a.ss_stride, rr, sq);
  }
  __syncthreads();
  return true;
}

template <int HD>
__global__ void __launch_bounds__(kSideThreads, 1) k_attn_block(SideArgs a) {
  extern __shared__ float lds[];
  __shared__ int s_ok;
  const int NB = gridDim.x, b = blockIdx.x;
  const int ngt = a.G * a.qtiles;
  // the other parity's split counters are the next launch's: clear them
  if (b == 0) {
    uint32_t* nxt = a.sync + a.qkv_tiles + ngt + ((a.epoch + 1) & 1) * ngt;
    for (int i = threadIdx.x; i < ngt; i += kSideThreads) st_coh32(nxt + i, 0u);
  }
  // QKV: tiles b, b + NB, ...; two at a time share the activation loads
  {
    int t = b;
    for (; t + NB < a.qkv_tiles; t += 2 * NB) {
      const int tt[2] = {t, t + NB};
      qkv_tiles<HD, 2>(a, tt, lds);
    }
    if (t < a.qkv_tiles) {
      const int tt[1] = {t};
      qkv_tiles<HD, 1>(a, tt, lds);
    }
  }
  const int nitems = ngt * a.splits;
  for (int it = b; it < nitems; it += NB)
    if (!attn_item<HD>(a, it, lds, &s_ok)) return;
  for (int t = b; t < a.o_tiles; t += NB)
    if (!o_tile<HD>(a, t, lds, &s_ok)) return;
  // the attention norm's sums of squares have been read by every QKV tile
  // (every merge flag is set, so every QKV tile is done): clear them for the
  // next producer
  if (b == 0 && a.ss_clear) {
    if (a.o_tiles == 0 && !wait_range(a.sync + a.qkv_tiles, 0, ngt, a.epoch, a.flags, &s_ok)) return;
    for (int i = threadIdx.x; i < 3 * a.ss_stride; i += kSideThreads)
      __hip_atomic_store(a.ss_clear + i, (uint64_t)0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

size_t attn_block_lds_bytes(int hd) {
  const size_t gemm = (size_t)(kSideWaves * 256 + 16 * 17) * 4;
  const size_t attn = (size_t)(3 * kSideWaves * 16 + 32 + kSideWaves * 16 * (hd + 4)) * 4;
  return gemm > attn ? gemm : attn;
}

int attn_block_occupancy(int hd) {
  int occ = 0;
  if (hd != 128) return 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, (const void*)k_attn_block<128>, kSideThreads,
                                                   attn_block_lds_bytes(hd)) != hipSuccess)
    return 0;
  return occ;
}

void attn_block_plan(SideArgs& a) {
  const int nq = (a.H / a.G) * a.R;
  a.qtiles = (nq + 15) / 16;
  // key splits of one chunk per wave (256 keys), at most kAttnMaxSplits
  int per = 32 * kSideWaves;
  if ((a.keys_ub + per - 1) / per > kAttnMaxSplits) per = ((a.keys_ub + kAttnMaxSplits - 1) / kAttnMaxSplits + 31) & ~31;
  a.split_keys = per;
  a.splits = (a.keys_ub + per - 1) / per;
}

hipError_t launch_attn_block(const SideArgs& a, int n_blocks, hipStream_t st) {
  // the polls read at most 6 flags per lane: q of <= 16 heads (128 flags) +
  // k + v (8 each), or <= 256 merge flags
  if (a.R < 1 || a.R > kAttnBlockMaxRows || a.hd != 128 || a.H % a.G || a.kc_o > 4 * kSideWaves ||
      a.splits < 1 || a.splits > kAttnMaxSplits || a.G * a.qtiles > kAttnBlockMaxGT || n_blocks < 1 ||
      a.qkv_tiles > kAttnBlockMaxTiles)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_attn_block<128>, dim3(n_blocks), dim3(kSideThreads), attn_block_lds_bytes(a.hd), st, a);
  return hipGetLastError();
}

}  // namespace jf
