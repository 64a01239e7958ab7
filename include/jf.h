/*
 * jf.h -- C ABI of libjf, a Jacobi-step engine for causal decoders on
 * AMD Instinct MI355X (gfx950).
 *
 * One call of jf_jacobi_step / jf_multiblock_step is ONE Jacobi iteration
 * (Jacobi Forcing, arXiv 2512.14681, Sec. 2.1, Eq. 3): a single forward pass
 * of the decoder over the draft rows, causal against an exact KV cache of the
 * committed prefix, a greedy argmax over the vocabulary for every row, and
 * acceptance of the longest prefix of draft rows that reached their fixed
 * point (Sec. 3.2; the acceptance step of App. A Alg. 1).
 * jf_commit_kv then keeps the accepted rows' K/V and drops the rest (the
 * cache-trim step of Alg. 1).
 *
 * Conventions
 *  - Pointers named d_* are DEVICE pointers; everything else is host memory.
 *  - The caller owns every buffer: weights, the packed-weight buffer, the KV
 *    cache, the workspace and all outputs.  libjf owns only the opaque host
 *    object jf_model, and never allocates device memory.
 *  - Every call validates its arguments on the host before enqueuing any
 *    work.  On error it returns a negative jf_status, enqueues nothing and
 *    sets jf_last_error() (thread-local).  No exception crosses the ABI and
 *    the library never aborts.  HIP runtime failures return JF_E_HIP with the
 *    HIP error string in jf_last_error().
 *  - Step and commit calls only enqueue work on `stream` (a hipStream_t).
 *    The committed length C lives on the device, so step -> commit -> step
 *    needs no host round trip.  Conditions that only the device can see
 *    (a token id outside [0, V)) are reported in jf_step_result.flags.
 *    The host keeps an upper bound of C (it grows by the rows of each
 *    committed step); a step that would pass max_ctx by that bound first
 *    reads C back (one stream synchronisation) and fails with JF_E_CAPACITY
 *    only if the exact length leaves no room.
 *  - One jf_model decodes one sequence (batch 1).  Calls on one model must
 *    not overlap (one stream, or external ordering).
 */
#ifndef JF_H
#define JF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  JF_OK = 0,
  JF_E_INVAL = -1,    /* null pointer, bad enum, bad value             */
  JF_E_SHAPE = -2,    /* shape not supported (see jf_config)           */
  JF_E_CAPACITY = -3, /* rows > max_rows, or C + rows > max_ctx        */
  JF_E_DTYPE = -4,    /* unsupported dtype                             */
  JF_E_HIP = -5,      /* HIP runtime error                             */
  JF_E_STATE = -6     /* call not valid in the model's current state   */
} jf_status;

typedef enum { JF_F32 = 0, JF_BF16 = 1 } jf_dtype;

/* Decoder shape: RMSNorm (gain), RoPE (rotate-half pairs i, i + head_dim/2,
 * inverse frequency rope_base^(-2i/head_dim)), grouped-query attention with
 * query head j reading KV head j / (n_heads / n_kv_heads), SwiGLU FFN,
 * untied LM head, no biases.
 * Limits: d_model, d_ffn multiples of 128, d_model <= 4096; head_dim in
 * {32, 64, 128};
 * n_heads * head_dim a multiple of 128; n_heads a multiple of n_kv_heads;
 * vocab a multiple of 16; 1 <= max_rows <= JF_MAX_ROWS; max_ctx a multiple of 64. */
typedef struct {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ffn, vocab;
  float rope_base, rms_eps;
  int32_t dtype;     /* jf_dtype of the weights and the KV cache; all
                        activations are fp32 (see "activation planes")     */
  int32_t max_rows;  /* largest number of rows of any step / prefill chunk */
  int32_t max_ctx;   /* KV cache capacity in tokens                         */
} jf_config;

/* Activation planes: an activation tensor A[...] of a JF_BF16 model is kept
 * as two bf16 planes, hi = bf16(A) then lo = bf16(A - hi) (A ~= hi + lo to
 * about 16 significant bits); a JF_F32 model keeps one fp32 plane.  Either
 * way 4 bytes per element.  The component calls below take and return
 * activations in this form.
 *
 * GEMM-input layout: an activation matrix that feeds a projection, X[R][K]
 * (K a multiple of 128), is stored with R padded to Rp = 16 * ceil(R / 16)
 * rows as 16-row tiles, each a run of 128-column blocks; inside a 16 x 128
 * block, element (r, c) sits at j * 512 + lane * 8 + e, lane = r + 16 (c/32),
 * j = (c % 32) / 8, e = c % 8 (the matrix-core operand order, so one
 * fragment load is one contiguous 1 KB).  Element (row, col) of X is at
 *   ((row / 16) * (K / 128) + col / 128) * 2048 + that in-block offset,
 * and the lo plane follows the hi plane Rp * K elements later. */

/* One chain of rows in a multi-block step (the input-assembly step of App. A Alg. 1).
 * Rows first_row .. first_row+n_rows-1 form a chain; the first hangs under
 * attach_row (-1: a root, predicted by the last committed row) and every
 * other row under the row before it.  A row sees the committed prefix, its
 * ancestors and itself, and sits at position C + depth.  Rows
 * [first_row, first_row + verify_from) are context only; the rest are
 * verified against their parent's argmax (longest matching run).
 * Segment 0 must be the real-active draft: attach_row = -1, role JF_ROLE_RA,
 * verify_from = 1 (its root row is the pending token, always correct).
 * Segments tile rows 0..R-1 in order and attach backwards (a forest). */
typedef struct {
  int32_t first_row, n_rows, attach_row, role, verify_from;
} jf_segment;

enum { JF_ROLE_RA = 0, JF_ROLE_CAND = 1, JF_ROLE_PSEUDO = 2 };
#define JF_MAX_SEGMENTS 16
/* Rows of one step at most, and the u64 words of a row's in-step visibility
 * mask (bit j of word j / 64: in-step row j is visible). */
#define JF_MAX_ROWS 512
#define JF_VIS_WORDS 8

/* Result of one step, written on the device (16 bytes). */
typedef struct {
  int32_t accept;   /* tokens accepted = rows on the committed path (>= 1)  */
  int32_t winner;   /* segment that won (0: the Jacobi draft)               */
  int32_t pending;  /* argmax of the last accepted row: the next token      */
  int32_t flags;    /* JF_FLAG_* bits                                        */
} jf_step_result;

#define JF_FLAG_BAD_TOKEN 1 /* a token id was outside [0, V); read as 0       */
#define JF_FLAG_CAPACITY 2  /* C + rows exceeded max_ctx; cache writes dropped */
#define JF_FLAG_SYNC 4      /* a wait between the phases of a fused launch gave
                               up (the device did not run all its workgroups
                               at once); the step's outputs are invalid      */

typedef struct jf_model jf_model;
typedef void *jf_stream; /* hipStream_t; NULL is the null stream */

/* Bytes the caller must allocate (device memory) for a configuration.
 * packed: the weights in the kernels' layout; kv: the paged KV cache;
 * ws: workspace (activations, partial results, rope tables, page table). */
jf_status jf_query_sizes(const jf_config *cfg, size_t *packed_bytes,
                         size_t *kv_bytes, size_t *ws_bytes);

/* Bind buffers and pack the weights (Sec. 4.1: a pretrained causal decoder).
 * d_weights[n_weights]: device pointers in fixture order, each [out, in]
 * row-major of cfg->dtype:
 *   embed [V, d]; per layer l: attn_norm [d], wq [H*hd, d], wk [G*hd, d],
 *   wv [G*hd, d], wo [d, H*hd], ffn_norm [d], w_gate [F, d], w_up [F, d],
 *   w_down [d, F]; then final_norm [d], lm_head [V, d].
 * n_weights = 3 + 9 * n_layers.  After the call (and a stream sync) the
 * source tensors are no longer read.  The cache starts empty (C = 0).
 * KV cache layout (d_kv, cfg->dtype): [n_layers][max_ctx/64 pages] pages of
 * 64 tokens, page = K [G][64][hd] followed by V transposed [G][hd][64];
 * logical page p of every layer lives at physical page page_table[p]
 * (identity after load; see jf_kv_set_page_table). */
jf_status jf_model_load(const jf_config *cfg, const void *const *d_weights,
                        int32_t n_weights, void *d_packed, void *d_kv,
                        void *d_ws, jf_stream stream, jf_model **out);

/* Frees the host object only (device buffers stay the caller's). */
jf_status jf_model_free(jf_model *m);

/* Message of the last error on this thread ("" if none). */
const char *jf_last_error(void);

/* Run the prompt through the model in causal chunks of <= max_rows and
 * commit all of it (Sec. 2.1: prompt x; Eq. 1).  d_pending[0] receives the
 * argmax of the last prompt row: the first generated token. Requires C == 0
 * (host view) and n <= max_ctx. */
jf_status jf_prefill(jf_model *m, const int32_t *d_tokens, int32_t n,
                     int32_t *d_pending, jf_stream stream);

/* One Jacobi iteration on a linear draft (Eq. 3).  d_draft[n] holds the
 * draft at positions C..C+n-1; d_draft[0] must be the pending token.
 * Writes d_argmax[n] (g[i] = argmax of row i, lowest id on ties), d_result
 * (accept a = 1 + longest run of d_draft[k] == g[k-1], pending = g[a-1]) and
 * d_next_draft[n]: the Jacobi update g[a-1], g[a], ... ; mode 0 (block,
 * Eq. 4) leaves the n - a + 1 .. n tail unspecified (the next block step uses
 * n - a rows), mode 1 (running window) fills it with
 * pad_id(pad_seed, C + a + i) = splitmix64(pad_seed ^ (pos * 0x9E3779B97F4A7C15)) % V.
 * d_next_draft may equal d_draft.  d_logits (optional, may be NULL) receives
 * the fp32 logits [n][V].  The cache rows C..C+n-1 are overwritten with the
 * draft's K/V; jf_commit_kv keeps the accepted ones.  mode | JF_STEP_COMMIT
 * also commits them in the step (C += a, as jf_commit_kv(m, NULL, d_result,
 * 0, ...) would; no jf_commit_kv follows such a step).  The vocabulary
 * argmax reduction, the acceptance and that commit run in one launch. */
#define JF_STEP_COMMIT 2
jf_status jf_jacobi_step(jf_model *m, const int32_t *d_draft, int32_t n,
                         int32_t mode, uint64_t pad_seed, int32_t *d_argmax,
                         jf_step_result *d_result, int32_t *d_next_draft,
                         float *d_logits, jf_stream stream);

/* One multi-block / rejection-recycling iteration (Sec. 3.2, Alg. 1): R rows
 * d_tokens[R] arranged by segs[n_segs] (host array, n_segs <=
 * JF_MAX_SEGMENTS) into a forest, verified in one forward pass.
 * d_seg_accept[n_segs]: per segment, the longest run of verified rows that
 * match their parent's argmax.  The winner is the segment among 0 and the
 * JF_ROLE_CAND ones with the largest count (ties: segment 0, then the lowest
 * index); d_path[R] receives the committed path (rows from the root down to
 * the winner's last accepted row), d_result its length, winner and pending
 * token.  d_argmax[R] and d_logits (optional) as in jf_jacobi_step. */
jf_status jf_multiblock_step(jf_model *m, const int32_t *d_tokens, int32_t R,
                             const jf_segment *segs, int32_t n_segs,
                             int32_t *d_argmax, int32_t *d_seg_accept,
                             jf_step_result *d_result, int32_t *d_path,
                             float *d_logits, jf_stream stream);

/* Commit the accepted rows of the last step (cache-trim step of Alg. 1): the K/V
 * of path row i moves to position C + i, then C += accept (read from
 * d_result on the device), capped at max_commit if max_commit > 0.
 * d_path NULL means rows 0..accept-1 (a linear step: nothing moves).  Must
 * follow a step on the same model. */
jf_status jf_commit_kv(jf_model *m, const int32_t *d_path,
                       const jf_step_result *d_result, int32_t max_commit,
                       jf_stream stream);

/* Committed length C (synchronises the stream). */
jf_status jf_kv_length(jf_model *m, int32_t *out, jf_stream stream);

/* Drop committed tokens beyond new_len (rejected K/V removal of Alg. 1);
 * JF_E_STATE if new_len > C. Synchronises the stream. */
jf_status jf_kv_truncate(jf_model *m, int32_t new_len, jf_stream stream);

/* Replace the page table (max_ctx/64 entries, device memory copied in; each
 * entry a distinct physical page in [0, max_ctx/64)).  Checked on the host
 * from h_table, a host copy of the same table. */
jf_status jf_kv_set_page_table(jf_model *m, const int32_t *h_table,
                               int32_t n, jf_stream stream);

/* ---- measurement ---------------------------------------------------------
 * Kernel classes of one step; jf_profile_begin makes every following launch
 * of that class on this model bracketed by two HIP events on the launch
 * stream, jf_profile_end synchronises, returns the summed event time (ms)
 * and the number of launches, and stops recording. */
enum {
  JF_KERNEL_QKV = 1,    /* RMSNorm'd x times W_qkv, RoPE, K/V into the cache */
  JF_KERNEL_ATTN = 2,   /* attention + split combine                         */
  JF_KERNEL_O = 3,      /* O projection + residual                           */
  JF_KERNEL_GATEUP = 4, /* gate/up projection + SwiGLU                       */
  JF_KERNEL_DOWN = 5,   /* down projection + residual                        */
  JF_KERNEL_LMHEAD = 6, /* LM head + per-block argmax                        */
  JF_KERNEL_STEP = 7,   /* a whole jf_jacobi_step / jf_multiblock_step       */
  JF_KERNEL_ATTN_BLOCK = 8 /* QKV + attention + O of one layer in one launch
                              (bf16 steps of at most 16 rows)                  */
};
/* Options of a loaded model (host state; effective from the next call).
 * JF_OPT_FUSED_ATTENTION (default 0): 1 makes bf16 steps of at most 16 rows
 * run the QKV projection, the attention and the O projection of each layer
 * as one persistent launch (one workgroup per compute unit; the phases hand
 * over through device flags) instead of four launches.  Both compute the
 * same operation; on the 7B shape at 16 rows the fused launch measured
 * 44 us per layer against 40 us for the four launches, hence the default.
 * Returns JF_E_INVAL for an unknown option or value. */
enum { JF_OPT_FUSED_ATTENTION = 1 };
jf_status jf_model_set_option(jf_model *m, int32_t option, int32_t value);

jf_status jf_profile_begin(jf_model *m, int32_t kernel_class);
jf_status jf_profile_end(jf_model *m, double *total_ms, int32_t *launches);

/* ---- component calls (used by the attention and LM-head workloads) ---- */

/* Attention of one layer (the attention inside Eq. 3's forward pass):
 * q [R][n_heads][head_dim] activation planes, keys/values of positions
 * 0..C+R-1 in one layer's paged cache d_kv_layer (layout as in
 * jf_model_load; slots beyond C+R in a used page must hold finite values),
 * with the page table d_page_table.  Row r sees positions [0, C) and
 * in-step position C + j iff bit j of d_vis[r][JF_VIS_WORDS] is set (d_vis NULL:
 * j <= r, causal).  out: activation planes of the [R][n_heads * head_dim]
 * matrix in the GEMM-input layout (the O projection's input), Rp * n_heads *
 * head_dim elements per plane.  d_ws of at least jf_attention_ws_bytes(...). */
size_t jf_attention_ws_bytes(int32_t n_heads, int32_t head_dim, int32_t R);
jf_status jf_attention(int32_t n_heads, int32_t n_kv_heads, int32_t head_dim,
                       int32_t dtype, int32_t C, int32_t R, const void *d_q,
                       const void *d_kv_layer, const int32_t *d_page_table,
                       const uint64_t *d_vis, void *d_out, void *d_ws,
                       jf_stream stream);

/* LM head + greedy argmax + longest-prefix acceptance (Eq. 3; the
 * verification step of Alg. 1): x [R][d] activation planes in the GEMM-input layout
 * (Rp * d elements per plane) times lm_head^T (dtype), lm_head [V][d]
 * packed by jf_pack_matrix; g = argmax per row (lowest id on ties); accept as in
 * jf_jacobi_step against d_draft[R] (NULL: no acceptance, d_result unused).
 * d_ws of at least jf_lm_head_ws_bytes(R, V).
 * Packed weight layout (jf_pack_matrix): W[rows][cols] (rows % 16 == 0,
 * cols % 128 == 0) as 16 x 128 blocks in the same in-block order as the
 * GEMM-input layout (row r of the block = W row, c = W column); 16-row tiles
 * come in groups of P = 4 (rows % 64 == 0), else 2 (rows % 32 == 0), else 1,
 * and block (tile t, column block kc) is block number
 * ((t / P) * (cols / 128) + kc) * P + t % P. */
size_t jf_packed_matrix_bytes(int32_t rows, int32_t cols, int32_t dtype);
jf_status jf_pack_matrix(int32_t rows, int32_t cols, int32_t dtype,
                         const void *d_src, void *d_packed, jf_stream stream);
size_t jf_lm_head_ws_bytes(int32_t R, int32_t V);
jf_status jf_lm_head_accept(int32_t R, int32_t d, int32_t V, int32_t dtype,
                            const void *d_x, const void *d_w_packed,
                            const int32_t *d_draft, int32_t *d_argmax,
                            jf_step_result *d_result, float *d_logits,
                            void *d_ws, jf_stream stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * operation and outputs as jf_lm_head_accept, with no d_ws argument.  Its
 * scratch (per-block argmax keys and one zeroed word) is a fixed device array
 * inside libjf of JF_NOALLOC_SCRATCH_BYTES, one copy per GPU, held until the
 * process ends; the call performs no hipMalloc / hipFree and enqueues only
 * kernels.  R and V must satisfy jf_lm_head_ws_bytes(R, V) <=
 * JF_NOALLOC_SCRATCH_BYTES (e.g. R <= 64 at V = 152064), else JF_E_CAPACITY
 * and nothing is enqueued.  Every call on one GPU shares that GPU's array and
 * leaves its contents behind; calls that overlap on one GPU (other streams,
 * other threads) race and must be serialised by the caller.  The first call
 * on each device looks up the array's device address (hipGetSymbolAddress);
 * a failure there returns JF_E_HIP. */
#define JF_NOALLOC_SCRATCH_BYTES ((size_t)8 << 20)
jf_status jf_lm_head_accept_noalloc(int32_t R, int32_t d, int32_t V,
                                    int32_t dtype, const void *d_x,
                                    const void *d_w_packed,
                                    const int32_t *d_draft, int32_t *d_argmax,
                                    jf_step_result *d_result, float *d_logits,
                                    jf_stream stream);

/* ---- packed training sequences (forward only) -----------------------------
 * Sec. 3.1 (noise-aware causal attention) and App. C (sequence packing): a
 * training sequence interleaves, for each block i of a response, the noisy
 * block selected from its trajectory and its clean fixed point, so that one
 * forward pass gives the logits of both losses (Eq. 8 and the AR loss). */
enum {
  JF_MASK_NOISY_CONTEXT = 0, /* noisy block i sees the noisy blocks before it */
  JF_MASK_CLEAN_CONTEXT = 1  /* noisy block i sees the clean blocks before it */
};

/* One forward pass over d_tokens[R], R = 2 n_blocks n (R <= max_rows), laid
 * out [noisy_0, clean_0, noisy_1, clean_1, ...] in blocks of n, after the
 * committed prefix (the prompt, from jf_prefill).  Every row sees the
 * prefix and the earlier rows of its own block copy; beyond that a clean
 * block sees the clean blocks before it, and a noisy block sees the noisy
 * (JF_MASK_NOISY_CONTEXT) or the clean (JF_MASK_CLEAN_CONTEXT) blocks
 * before it.  Both copies of block i sit at positions C + i n + k.
 * Writes d_argmax[R] (lowest id on ties) and, if not NULL, the fp32 logits
 * d_logits[R][V].  The cache slots C .. C+R-1 are overwritten and nothing
 * is committed (a following jf_commit_kv fails with JF_E_STATE). */
jf_status jf_packed_forward(jf_model *m, const int32_t *d_tokens,
                            int32_t n_blocks, int32_t n, int32_t mask,
                            int32_t *d_argmax, float *d_logits,
                            jf_stream stream);

/* ---- trajectories (the data collection of Jacobi Forcing) -------------------
 * A block's Jacobi trajectory (Sec. 2.1) is the list of its iterates
 * y^(0), ..., y^(k), stopping at the first k with y^(k) = y^(k-1); y^(k) is
 * the fixed point.  Decoded in block mode (jf_jacobi_step mode 0, then
 * jf_commit_kv), a block of n tokens whose first n - rows positions are
 * accepted feeds its last `rows` tokens to a step, and the step's argmaxes
 * give the next iterate. */

/* Iterate y^(j+1) of an n-token block (Eq. 3) from y^(j) = d_prev[n] and the
 * argmaxes d_argmax[rows] of the step that fed y^(j)'s last rows tokens
 * (1 <= rows <= n):
 *   d_out[i] = d_prev[i]                     for i <= n - rows
 *   d_out[i] = d_argmax[i - (n - rows) - 1]  for i >  n - rows
 * (accepted positions and the pending token stay; each other position takes
 * the prediction made after its predecessor).  d_out may equal d_prev.
 * y^(0) is the caller's initial draft.  JF_E_SHAPE unless 1 <= rows <= n. */
jf_status jf_trajectory_record(const int32_t *d_prev, const int32_t *d_argmax,
                               int32_t n, int32_t rows, int32_t *d_out,
                               jf_stream stream);

/* Noise-schedule point selection (App. C with the schedule of Sec. 3.1,
 * Eq. 7).  d_traj[n_blocks][max_points][n]: block b's trajectory in its
 * first d_len[b] points, the last of them its fixed point y*; other points
 * are not read.  For each point, u = the number of positions that differ
 * from y* (unconverged tokens, Sec. 3.1).  Block b's target noise ratio is
 * t_b = (b mod w) / w (Eq. 7, blocks counted from 0), or d_t_num[b] / w
 * when d_t_num is not NULL (any other schedule on denominator w).
 * d_sel[b] = the point whose u / n is closest to t_b, the earliest on ties,
 * compared exactly in integers as |u w - t_num n| (t_num = b mod w or
 * d_t_num[b]); -1 when d_len[b] is outside
 * [1, max_points] (nothing of that block is read).  d_unconv (optional,
 * [n_blocks][max_points]) receives u per point, -1 beyond d_len[b].
 * n_blocks = 0 does nothing.  JF_E_SHAPE unless n, max_points, w >= 1. */
jf_status jf_trajectory_select(const int32_t *d_traj, const int32_t *d_len,
                               int32_t n_blocks, int32_t n, int32_t max_points,
                               int32_t w, const int32_t *d_t_num,
                               int32_t *d_sel, int32_t *d_unconv,
                               jf_stream stream);

#ifdef __cplusplus
}
#endif
#endif /* JF_H */
