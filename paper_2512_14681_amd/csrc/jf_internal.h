// Host-side interface between the C ABI and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace jf {

constexpr int kPage = 64;  // tokens per KV page
constexpr int kMaxRows = 512;             // rows of one step (draft, candidates, prefill chunk)
constexpr int kVisWords = kMaxRows / 64;  // u64 words of a row's in-step visibility mask

// Packed weight layout: 16-row tiles are stored in groups of P (4 when the
// row count allows, else 2, else 1), and inside a group K-block-major with
// the P tiles of one K-block adjacent: block index ((t / P) * KC + kc) * P +
// t % P for tile t and K-block kc.  A block is 16 rows x 128 inputs.
__host__ __device__ inline int pack_group(int rows) { return rows % 64 == 0 ? 4 : (rows % 32 == 0 ? 2 : 1); }

enum EpiKind { EPI_STORE = 0, EPI_RESID = 1, EPI_QKV = 2, EPI_SWIGLU = 3, EPI_ARGMAX = 4 };

// What a GEMM does with its output tile Y[R][N] (fp32 accumulators).
struct Epi {
  int kind;
  int R;
  // EPI_STORE: f32[row * ldf + col] = y;  EPI_RESID: f32[row * ldf + col] += y
  float* f32;
  int ldf;
  // EPI_SWIGLU: columns come in (gate tile, up tile) pairs of 16; writes the
  // activation act(row, f) = silu(gate) * up in the GEMM-input layout of an
  // [R][act_k] matrix (planes act_plane apart).
  void* act;
  int act_k;
  size_t act_plane;
  // EPI_QKV: packed rows are q heads, k heads, v heads (rope pairs (i, i+hd/2)
  // interleaved 8 by 8 inside each 16-row tile of q and k heads).
  void* q;                   // [R][H][hd] activation planes, q_plane apart
  size_t q_plane;
  void* kv;                  // this layer's pages
  const int32_t* page_table; // logical page -> physical page
  const int32_t* pos;        // [R] positions (RoPE)
  const int32_t* state;      // state[0] = committed length C
  const float* rope_cos;     // [max_ctx][hd/2]
  const float* rope_sin;
  int H, G, hd, max_ctx;
  int32_t* flags;
  // EPI_ARGMAX: part[blockIdx * R_stride + row] = packed (value, index) max over
  // the block's columns; optional logits[row * ldl + col] = y.
  uint64_t* part;
  int part_stride;
  float* logits;
  int ldl;
  // Split-K across blocks (gridDim.y > 1): each block stores its partial tile
  // in kpart; the last block of a column group (kcount) sums them in order.
  float* kpart;
  int32_t* kcount;
  // Input rows row0 .. row0 + R - 1 of X are read (the LM head of a prefill
  // chunk reads only its last row).
  int row0;
  // RMSNorm folded into the consumer: X holds activation planes of h * gain
  // and output row r is scaled by 1 / sqrt(mean(h[row0 + r]^2) + eps), read
  // from ss_in, the fixed-point sums of squares of h (ss_add; three word
  // planes of ss_stride entries).  Null: no scaling.
  const uint64_t* ss_in;
  int ss_stride;
  double norm_inv_d, norm_eps;
  // RMSNorm producer side (EPI_RESID): after f32 += y, also writes activation
  // planes of (new h) * gain_next into xg (GEMM-input layout of an [R][ldf]
  // matrix, planes xg_plane apart) and adds each row's sum of squares over
  // this block's columns to ss_out.  ss_clear (may be null) is zeroed by the
  // first block: the other accumulator, which the next producer fills.
  const float* gain_next;
  void* xg;
  size_t xg_plane;
  uint64_t* ss_out;
  uint64_t* ss_clear;
};

struct GemmShape {
  int R, N, K;   // Y[R][N] = X[R][K] * W[N][K]^T
  int NT, WK;    // 16-column tiles per block, waves splitting K per block
  int S;         // blocks splitting K per column group
  int D;         // register-ring depth (0: the kernel's default)
  int C;         // row chunks of at most 32 rows (blocks per column group and split)
  int full;      // tail split (C = 1, 0 < full < groups): column groups [0, full)
                 // run whole, the remaining ones split K over S blocks; 0: off
};

// Scratch a GEMM needs for split-K partials (floats) and counters (ints).
constexpr size_t kGemmPartFloats = (size_t)16 << 20;  // 64 MB
constexpr size_t kGemmCounters = 16384;

// Chooses NT / WK / S / C for a shape (NT fixed by the epilogue where it
// matters).
void gemm_plan(GemmShape& s, int epi_kind);
// Balances the last, partial round of a plan's workgroups over n_cus
// compute units by splitting its column groups over K (sets full and S);
// needs split-K scratch.
void gemm_tail_split(GemmShape& s, int n_cus);
// X: activation planes of an [R][K] matrix in the GEMM-input layout
// (act_offset; planes xplane elements apart for bf16 models).
hipError_t launch_gemm(int dtype, const void* X, size_t xplane, const void* Wp,
                       const GemmShape& s, const Epi& ep, hipStream_t stream);
size_t gemm_blocks(const GemmShape& s);

// Column-slice GEMM (gemm_mr.hip), bf16: 8-wave workgroups, each wave all
// row tiles of a chunk x its own column tiles, over LDS-staged activations
// (requested once per compute unit); split K writes partials that a second
// kernel reduces.
struct MrPlan {
  int R;            // rows
  int RT;           // row tiles per chunk (2, 4, 6, 8): 16 RT rows per chunk
  int B;            // column tiles per wave at most
  int KC;           // 128-wide K-blocks
  int P;            // pack group of the weight matrix
  int T;            // 16-column tiles of N
  int gr;           // column tiles per unit (2: SwiGLU pairs)
  int n_cg;         // column groups (workgroups along N)
  int passes;       // column passes per group
  int S;            // K splits (partials in Epi::kpart, S x R x N floats)
  int chunks;       // row chunks of 16 RT rows
};
// false if the shape is not for this kernel; max_splits 1: no split-K
// scratch
bool gemm_mr_plan(MrPlan& m, int R, int N, int K, int epi_kind, int n_cus, int max_splits);
size_t gemm_mr_lds_bytes(const MrPlan& m);
// per-block argmax slots (EPI_ARGMAX) the plan's epilogue writes
int gemm_mr_part_blocks(const MrPlan& m);
hipError_t launch_gemm_mr(const void* X, size_t xplane, const void* Wp, const MrPlan& m, const Epi& ep,
                          hipStream_t stream);

// Packs W[rows][cols] (row-major) into the kernels' block layout, reading
// source row rowmap[i] (or i if rowmap is null) from one of up to 4 source
// matrices: rowmap entries are (src << 24) | row.
hipError_t launch_pack(int dtype, int rows, int cols, const void* const* srcs, int n_srcs,
                       const int32_t* d_rowmap, void* dst, hipStream_t stream);

// Tree of one step: parent/pos/vis from segments (row 0 is a root).
struct SegArgs {
  int32_t n;
  int32_t first[16], nrows[16], attach[16], role[16], verify_from[16];
};
hipError_t launch_tree(const SegArgs& segs, int R, const int32_t* state, int32_t* flags,
                       int32_t* parent, int32_t* pos, uint64_t* vis, hipStream_t stream);
// the packed noisy/clean layout of a training sequence; mask as JF_MASK_* of jf.h
constexpr int kMaskNoisyContext = 0, kMaskCleanContext = 1;
hipError_t launch_tree_packed(int n_blocks, int n, int mask, const int32_t* state, int32_t* flags,
                              int32_t* parent, int32_t* pos, uint64_t* vis, hipStream_t stream);

// Embedding rows h[r] = E[token r] (fp32, row-major [R][d]) with the first
// RMSNorm's input: activation planes of h * gamma in the GEMM-input layout
// (xg) and each row's sum of squares stored into the fixed-point accumulator
// ss (three word planes of ss_stride entries); ss_clear is zeroed.
hipError_t launch_embed(int dtype, const int32_t* tokens, int R, const void* embed,
                        const float* gamma, int d, int V, float* h, void* xg, size_t xplane,
                        uint64_t* ss, uint64_t* ss_clear, int ss_stride, int32_t* flags,
                        hipStream_t stream);

constexpr int kAttnMaxSplits = 32;

struct AttnArgs {
  int H, G, hd, R, max_ctx;
  int splits;
  int waves;                 // waves per block (4)
  int qt;                    // query tiles per block (1 or 2)
  int lds_ok;                // bf16 K/V: the plan may choose the LDS-shared kernel
  int qg;                    // LDS-shared kernel: query tiles per block (0: not chosen)
  int keys_ub;               // host upper bound of C + R (<= max_ctx): the split layout
  const void* q;             // [R][H][hd] activation planes
  size_t q_plane;
  const void* kv;            // this layer's pages
  const int32_t* page_table;
  const int32_t* state;      // state[0] = C (device), or null: use C_host
  int C_host;
  const uint64_t* vis;       // [R][kVisWords] or null (causal)
  float* o_part;             // [splits][R*H][hd]
  float* ml_part;            // [splits][R*H][2]
  void* out;                 // [R][H*hd] activation planes, GEMM-input layout
  size_t out_plane;
};
// Sets a.waves, a.splits, a.qt and a.qg from a.keys_ub (and the head
// counts): the LDS-shared kernel (qg > 0) where a.lds_ok and head_dim 128.
void attn_plan(AttnArgs& a);
constexpr int kAttnChunksPerWave = 2;  // 32-key chunks per wave
hipError_t launch_attention(int dtype, const AttnArgs& a, hipStream_t stream);

// The attention half of a layer (QKV + attention + O) in one persistent
// launch, for bf16 steps of at most kAttnBlockMaxRows rows (layer.hip).
constexpr int kAttnBlockMaxRows = 16;
constexpr int kAttnBlockMaxGT = 256;      // kv heads x query tiles
constexpr int kAttnBlockMaxTiles = 1024;  // 16-column tiles of the QKV projection
constexpr int JF_FLAG_SYNC_BIT = 4;       // JF_FLAG_SYNC of jf.h
// uint32 words of the launch's flags and counters (caller-owned, zeroed once)
constexpr size_t kAttnBlockSyncWords = kAttnBlockMaxTiles + 3 * kAttnBlockMaxGT;
struct SideArgs {
  int R, d, H, G, hd, max_ctx;
  int qkv_tiles, o_tiles;       // 16-column tiles of the two projections
  int kc_qkv, kc_o;             // 128-wide K-blocks of the two projections
  int p_qkv, p_o;               // pack groups of the two packed matrices
  const void* x;                // attention norm's input (h * gain), GEMM-input layout
  size_t x_plane;
  const void* w_qkv;
  const uint64_t* ss_in;        // the rows' fixed-point sums of squares of h
  int ss_stride;
  double norm_inv_d, norm_eps;
  void* q;                      // [R][H][hd] activation planes
  size_t q_plane;
  void* kv;                     // this layer's pages
  const int32_t* page_table;
  const int32_t* pos;
  const int32_t* state;         // state[0] = committed length C
  const float* rope_cos;
  const float* rope_sin;
  int32_t* flags;               // step flags (JF_FLAG_*)
  const uint64_t* vis;          // [R][kVisWords] in-step visibility, or null (causal)
  int keys_ub;                  // host bound of C + R: the key-split layout
  int qtiles, splits, split_keys;
  float* o_part;                // [splits][R * H][hd]
  float* ml_part;               // [splits][R * H][2]
  void* attn;                   // merged attention output, GEMM-input layout [Rp][H * hd]
  size_t attn_plane;
  const void* w_o;
  float* h;                     // residual stream [R][d]
  const float* gain_next;       // next RMSNorm's gain
  void* xg;                     // its input planes (GEMM-input layout [Rp][d])
  size_t xg_plane;
  uint64_t* ss_out;             // row sums of squares of the new h
  uint64_t* ss_clear;           // zeroed after every QKV tile has read ss_in
  uint32_t* sync;               // kAttnBlockSyncWords words
  uint32_t epoch;               // this launch's number (never 0)
};
size_t attn_block_lds_bytes(int hd);
int attn_block_occupancy(int hd);   // workgroups per compute unit (0: cannot run)
void attn_block_plan(SideArgs& a);  // qtiles, splits, split_keys from R, H, G, keys_ub
hipError_t launch_attn_block(const SideArgs& a, int n_blocks, hipStream_t stream);

hipError_t launch_argmax_reduce(const uint64_t* part, int nblocks, int stride, int R,
                                int32_t* g, hipStream_t stream);
hipError_t launch_accept_linear(const int32_t* draft, const int32_t* g, int n, int mode,
                                uint64_t seed, int V, const int32_t* state, const int32_t* flags,
                                int32_t* result, int32_t* next_draft, hipStream_t stream);
hipError_t launch_accept_tree(const SegArgs& segs, const int32_t* tokens, const int32_t* g,
                              const int32_t* parent, int R, const int32_t* flags,
                              int32_t* seg_accept, int32_t* result, int32_t* path,
                              hipStream_t stream);
// The argmax reduction of the LM head's per-block keys, the acceptance and
// (linear steps, commit != 0) the commit, in one launch; state[2] is its
// counter (zero between launches).
hipError_t launch_argmax_accept_linear(const uint64_t* part, int nblocks, int stride, const int32_t* draft, int n,
                                       int mode, uint64_t seed, int V, int32_t* state, const int32_t* flags,
                                       int32_t* result, int32_t* next_draft, int32_t* g, int commit, int max_ctx,
                                       hipStream_t stream);
hipError_t launch_argmax_accept_tree(const uint64_t* part, int nblocks, int stride, const SegArgs& segs,
                                     const int32_t* tokens, int R, const int32_t* parent, int32_t* state,
                                     const int32_t* flags, int32_t* seg_accept, int32_t* result, int32_t* path,
                                     int32_t* g, hipStream_t stream);
hipError_t launch_commit(int dtype, void* kv, int L, int n_pages, int G, int hd,
                         const int32_t* page_table, int32_t* state, const int32_t* path,
                         const int32_t* result, int max_commit, int fixed_count, int max_ctx,
                         hipStream_t stream);
hipError_t launch_set_int(int32_t* p, int32_t v, hipStream_t stream);
hipError_t launch_fill_int(int32_t* p, int n, int32_t v, hipStream_t stream);  // p[0..n) = v
hipError_t launch_to_f32(int dtype, const void* src, float* dst, int n, hipStream_t stream);
hipError_t launch_copy_int(int32_t* dst, const int32_t* src, hipStream_t stream);

// trajectory.hip
hipError_t launch_traj_record(const int32_t* prev, const int32_t* g, int n, int rows, int32_t* out,
                              hipStream_t stream);
hipError_t launch_traj_select(const int32_t* traj, const int32_t* len, int n_blocks, int n, int max_points,
                              int w, const int32_t* t_num, int32_t* sel, int32_t* unconv, hipStream_t stream);

}  // namespace jf
