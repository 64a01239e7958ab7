// Device-side building blocks for gfx950 (CDNA4): element types, bf16
// rounding, MFMA fragments and the packed-weight layout shared by the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace jf {

typedef uint16_t bf16_t;  // bf16 storage (bit pattern)
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// ---- scalar conversions -----------------------------------------------------
__device__ __forceinline__ float bf16_to_f32(bf16_t b) {
  return __uint_as_float(((uint32_t)b) << 16);
}
// Round to nearest, ties to even (the hardware conversion, v_cvt_pk_bf16_f32).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) { return __builtin_bit_cast(bf16_t, (__bf16)f); }
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
// Two values rounded to bf16 in one instruction; a in the low half.
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  const f32x2_t v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}
template <typename T> __device__ __forceinline__ float to_f32(T v);
template <> __device__ __forceinline__ float to_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f32<bf16_t>(bf16_t v) { return bf16_to_f32(v); }
template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16_t from_f32<bf16_t>(float v) { return f32_to_bf16(v); }

// ---- MFMA fragments: 8 consecutive K-elements per lane ------------------------
// A 16x16 MFMA tile is built from lane l holding row/column (l % 16) and the
// K-group (l / 16).  Any fixed assignment of K indices to (group, element)
// gives the same contraction as long as both operands use it, which lets
// every lane load 8 (or 32) contiguous elements.
template <typename T> struct Frag;
template <> struct Frag<bf16_t> { uint4 v; };           // 8 x bf16 (16 B)
template <> struct Frag<float> { float4 lo, hi; };      // 8 x f32  (32 B)

template <typename T> __device__ __forceinline__ Frag<T> frag_zero();
template <> __device__ __forceinline__ Frag<bf16_t> frag_zero<bf16_t>() {
  Frag<bf16_t> f; f.v = make_uint4(0, 0, 0, 0); return f;
}
template <> __device__ __forceinline__ Frag<float> frag_zero<float>() {
  Frag<float> f; f.lo = make_float4(0, 0, 0, 0); f.hi = f.lo; return f;
}

template <typename T> __device__ __forceinline__ Frag<T> frag_load(const T* p);
template <> __device__ __forceinline__ Frag<bf16_t> frag_load<bf16_t>(const bf16_t* p) {
  Frag<bf16_t> f; f.v = *reinterpret_cast<const uint4*>(p); return f;
}
template <> __device__ __forceinline__ Frag<float> frag_load<float>(const float* p) {
  Frag<float> f;
  f.lo = reinterpret_cast<const float4*>(p)[0];
  f.hi = reinterpret_cast<const float4*>(p)[1];
  return f;
}
// Streaming load (weights are read once per step): non-temporal hint.
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4v_t __attribute__((ext_vector_type(4)));
template <typename T> __device__ __forceinline__ Frag<T> frag_load_nt(const T* p);
template <> __device__ __forceinline__ Frag<bf16_t> frag_load_nt<bf16_t>(const bf16_t* p) {
  u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
  Frag<bf16_t> f; f.v = make_uint4(v.x, v.y, v.z, v.w); return f;
}
template <> __device__ __forceinline__ Frag<float> frag_load_nt<float>(const float* p) {
  f32x4v_t a = __builtin_nontemporal_load(reinterpret_cast<const f32x4v_t*>(p));
  f32x4v_t b = __builtin_nontemporal_load(reinterpret_cast<const f32x4v_t*>(p) + 1);
  Frag<float> f;
  f.lo = make_float4(a.x, a.y, a.z, a.w);
  f.hi = make_float4(b.x, b.y, b.z, b.w);
  return f;
}

// acc += A * B for one 16x16 output tile over 32 K-elements (bf16: one
// v_mfma_f32_16x16x32_bf16) or over 32 K-elements in 8 steps of 4 (f32:
// v_mfma_f32_16x16x4_f32, element e of every lane in step e).
__device__ __forceinline__ void mfma(f32x4_t& acc, const Frag<bf16_t>& a, const Frag<bf16_t>& b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a.v),
                                                __builtin_bit_cast(bf16x8_t, b.v), acc, 0, 0, 0);
}
__device__ __forceinline__ void mfma(f32x4_t& acc, const Frag<float>& a, const Frag<float>& b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo.x, b.lo.x, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo.y, b.lo.y, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo.z, b.lo.z, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo.w, b.lo.w, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi.x, b.hi.x, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi.y, b.hi.y, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi.z, b.hi.z, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi.w, b.hi.w, acc, 0, 0, 0);
}

// ---- activations -----------------------------------------------------------------
// A bf16 model computes activations in fp32 and stores each one as two bf16
// planes, hi = bf16(v) and lo = bf16(v - hi) (plane stride in elements); the
// MFMA then runs once per plane, so the contraction sees ~16 significant bits
// of the activation instead of 8.  An fp32 model stores one fp32 plane.
// GEMM-input layout of an activation matrix X[R][K] (R padded to 16): 16-row
// tiles, each a run of 128-column K-blocks; inside a 16 x 128 block element
// (r, c) sits at j * 512 + lane * 8 + e with lane = r + 16 (c / 32),
// j = (c % 32) / 8, e = c % 8.  That is the MFMA operand order of the packed
// weights, so one activation fragment load is one contiguous 1 KB (bf16).
__host__ __device__ inline size_t act_offset(int row, int col, int K) {
  const int c = col & 127;
  return (((size_t)(row >> 4) * (size_t)(K >> 7) + (size_t)(col >> 7)) << 11) + (size_t)((c & 31) >> 3) * 512 +
         (size_t)((row & 15) + 16 * (c >> 5)) * 8 + (size_t)(c & 7);
}

template <typename T> struct ActFrag;
template <> struct ActFrag<bf16_t> { Frag<bf16_t> hi, lo; };
template <> struct ActFrag<float> { Frag<float> v; };

template <typename T> __device__ __forceinline__ ActFrag<T> act_load(const T* p, size_t plane);
template <> __device__ __forceinline__ ActFrag<bf16_t> act_load<bf16_t>(const bf16_t* p, size_t plane) {
  ActFrag<bf16_t> a; a.hi = frag_load<bf16_t>(p); a.lo = frag_load<bf16_t>(p + plane); return a;
}
template <> __device__ __forceinline__ ActFrag<float> act_load<float>(const float* p, size_t plane) {
  ActFrag<float> a; a.v = frag_load<float>(p); return a;
}
template <typename T> __device__ __forceinline__ ActFrag<T> act_zero();
template <> __device__ __forceinline__ ActFrag<bf16_t> act_zero<bf16_t>() {
  ActFrag<bf16_t> a; a.hi = frag_zero<bf16_t>(); a.lo = a.hi; return a;
}
template <> __device__ __forceinline__ ActFrag<float> act_zero<float>() {
  ActFrag<float> a; a.v = frag_zero<float>(); return a;
}
template <typename T> __device__ __forceinline__ void act_store(T* p, size_t plane, float v);
template <> __device__ __forceinline__ void act_store<bf16_t>(bf16_t* p, size_t plane, float v) {
  const bf16_t hi = f32_to_bf16(v);
  p[0] = hi;
  p[plane] = f32_to_bf16(v - bf16_to_f32(hi));
}
template <> __device__ __forceinline__ void act_store<float>(float* p, size_t plane, float v) { p[0] = v; }

// acc += A * B with an activation operand on either side.
__device__ __forceinline__ void mfma(f32x4_t& acc, const ActFrag<bf16_t>& a, const Frag<bf16_t>& b) {
  mfma(acc, a.hi, b);
  mfma(acc, a.lo, b);
}
__device__ __forceinline__ void mfma(f32x4_t& acc, const ActFrag<float>& a, const Frag<float>& b) {
  mfma(acc, a.v, b);
}
__device__ __forceinline__ void mfma(f32x4_t& acc, const Frag<bf16_t>& a, const ActFrag<bf16_t>& b) {
  mfma(acc, a, b.hi);
  mfma(acc, a, b.lo);
}
__device__ __forceinline__ void mfma(f32x4_t& acc, const Frag<float>& a, const ActFrag<float>& b) {
  mfma(acc, a, b.v);
}

// ---- packed weight layout --------------------------------------------------------
// W [N][K] (row-major, out x in) is stored as blocks of 16 rows x 128 columns.
// Block (nt, kc) = rows 16nt.., columns 128kc.., at element offset
// (nt * KC + kc) * 2048, KC = K / 128.  Inside a block, element
// [j][lane][e] (j < 4, lane < 64, e < 8) is W[16nt + lane%16][128kc + 32(lane/16) + 8j + e],
// so load j of a wave reads 64 lanes x 8 elements contiguously and yields the
// B fragment of one 32-wide MFMA step whose K indices match the A fragment
// X[row][128kc + 32(lane/16) + 8j + e].
constexpr int kBlockElems = 2048;


// Ordered 64-bit key for a (value, index) maximum: larger value wins, then
// the lower index.  Keys compare as unsigned integers.
__device__ __forceinline__ uint64_t argmax_key(float v, uint32_t idx) {
  uint32_t u = __float_as_uint(v);
  uint32_t o = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((uint64_t)o << 32) | (uint64_t)(0xFFFFFFFFu - idx);
}
__device__ __forceinline__ uint32_t argmax_key_index(uint64_t k) {
  return 0xFFFFFFFFu - (uint32_t)(k & 0xFFFFFFFFull);
}

// ---- RMSNorm row statistics ------------------------------------------------------
// Sums of squares of a row are accumulated across blocks as exact fixed-point
// words: a non-negative fp32 partial p is split into w0 = floor(p) and two
// 32-bit fraction words (p = w0 + w1 2^-32 + w2 2^-64, exact for p >= 2^-40;
// below that the tail is truncated).  Each word is added to its own 64-bit
// accumulator, so the total is the same whatever order the blocks arrive in
// (integer addition is associative) and no carry crosses words while adding.
// An accumulator of R rows is three word planes of `stride` entries.
__device__ __forceinline__ void ss_split(float p, uint64_t (&w)[3]) {
  double d = p < 1e18f ? (double)p : 1e18;  // non-finite or absurd partials saturate
  const double w0 = floor(d);
  d = (d - w0) * 4294967296.0;
  const double w1 = floor(d);
  d = (d - w1) * 4294967296.0;
  w[0] = (uint64_t)w0;
  w[1] = (uint64_t)w1;
  w[2] = (uint64_t)floor(d);
}
__device__ __forceinline__ void ss_add(uint64_t* acc, int stride, int row, float p) {
  uint64_t w[3];
  ss_split(p, w);
#pragma unroll
  for (int k = 0; k < 3; ++k)
    if (w[k]) __hip_atomic_fetch_add(acc + (size_t)k * stride + row, w[k], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void ss_load(const uint64_t* acc, int stride, int row, uint64_t (&w)[3]) {
#pragma unroll
  for (int k = 0; k < 3; ++k)
    w[k] = __hip_atomic_load(acc + (size_t)k * stride + row, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// 1 / sqrt(mean of squares + eps) of a row from its accumulated words.
__device__ __forceinline__ float ss_rstd(const uint64_t (&w)[3], double inv_d, double eps) {
  const double ss = (double)w[0] + (double)w[1] * 0x1p-32 + (double)w[2] * 0x1p-64;
  return (float)(1.0 / sqrt(ss * inv_d + eps));
}

// splitmix64 (Steele, Lea & Flood 2014): first output of the generator whose
// state is x.
__device__ __forceinline__ uint64_t splitmix64(uint64_t x) {
  uint64_t z = x + 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
__device__ __forceinline__ int32_t pad_id(uint64_t seed, int64_t pos, int32_t vocab) {
  return (int32_t)(splitmix64(seed ^ ((uint64_t)pos * 0x9E3779B97F4A7C15ull)) % (uint64_t)vocab);
}

}  // namespace jf
