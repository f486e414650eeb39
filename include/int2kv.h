/*
 * int2kv.h -- C ABI of the rotated, key-centered INT2 KV cache and its decode attention
 * for AMD Instinct MI355X (gfx950).
 *
 * What is computed (Yun et al., "Output-Aware Rotation for INT2 KV-Cache Quantization"):
 *   cache write  (Sec. 4.1 key reparameterization; Sec. 6 efficiency analysis; appendix
 *                 "Key-mean estimation and application"):
 *       k_R = Q_2((k - mu) R_K) = Q_2(k R_K - mu R_K),   v_R = Q_2(v R_V)
 *   decode       (eq:int2_attention, eq:int2_residual_readout; appendix "Rotated-query
 *                 implementation" and "Equivalent inference implementation"):
 *       a_s = (q R_K) k_R,s^T / sqrt(d),  p = softmax_s(a),  o = (sum_s p_s v_R,s) R_V^T,
 *       y = concat_j(o_j) W_O^T   (optional)
 *   Query head j reads KV head h(j) = floor(j / G_q), G_q = H_q / H_kv (GQA, Sec. 3).
 *
 * Q_2 is group-wise affine INT2 (Sec. 5 implementation details, Table A) over groups of G = 32
 * or G = 128 (the paper's setting) consecutive rotated channels of one token. The arithmetic, fixed for bit-exactness, is
 * (all fp32, no contraction, round-to-nearest-even throughout):
 *       mn = min x, mx = max x;   if clip != 1: mn = clip*mn, mx = clip*mx
 *       s  = fp16(fp32(mx - mn) / 3),   z = fp16(mn)
 *       inv = s > 0 ? 1 / s : 0;        code = clamp(rint((x - z) * inv), 0, 3)
 *       dequantized value = code * s + z
 *
 * Conventions for every call:
 *   - All tensor pointers are DEVICE pointers owned by the caller; the library allocates
 *     nothing and never synchronizes. Work is enqueued on `stream` (0 = null stream).
 *   - bf16 and fp16 tensors are passed as uint16_t bit patterns; row-major, densely packed.
 *   - Return value: INT2KV_OK or a negative int2kv_status. On an argument error nothing is
 *     launched; int2kv_last_error() (thread-local) describes the last failure.
 *   - head_dim = 128, block_size = 16, group_size = 32 or 128 are the supported shapes.
 *
 * Packed cache (part of the bit-exact contract): with NG = 128 / group_size groups per token,
 * the pool holds one record of R = 1024 + 128 * NG bytes (1536 at G = 32, 1152 at G = 128; see
 * int2kv_record_bytes) per (physical block, KV head) at pool + (block * num_kv_heads + h) * R,
 * 16-byte aligned. Token row t (0..15) of a block and rotated channel c (0..127) are stored as
 *     [   0,  512) K codes, token-major: 16-bit half m of token t at byte 32*t + 2*m
 *     [ 512, 1024) V codes, half-major : 16-bit half m of token t at byte 512 + 32*m + 2*t
 *     [1024, 1024 + 64 NG) K scale/zero: token t, group g at 1024 + 4*NG*t + 4*g (fp16 s, fp16 z)
 *     [1024 + 64 NG, ...)  V scales: group g, token t at 1024 + 64*NG + 32*g + 2*t (fp16)
 *     [1024 + 96 NG, R)    V zeros : group g, token t at 1024 + 96*NG + 32*g + 2*t (fp16)
 *   where channel c = 16*p + m sits in half m at bits 2p..2p+1 (little endian), i.e. 2 bits
 *   per element plus 32 metadata bits per group: 3.0 bits per cached element at G = 32, 2.25 at
 *   G = 128. A cache slot is block * 16 + t.
 */
#ifndef INT2KV_H
#define INT2KV_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define INT2KV_HEAD_DIM 128
#define INT2KV_BLOCK_SIZE 16
#define INT2KV_GROUP_SIZE 32    /* default group size; 128 is also supported */
#define INT2KV_RECORD_BYTES 1536 /* record bytes at the default group size   */

typedef enum {
  INT2KV_OK = 0,
  INT2KV_EINVAL = -1,       /* bad pointer, shape or alignment                         */
  INT2KV_EUNSUPPORTED = -2, /* a shape the library does not implement                 */
  INT2KV_EWORKSPACE = -3,   /* workspace missing or smaller than required              */
  INT2KV_EHIP = -4          /* a HIP launch reported an error                          */
} int2kv_status;

/* The paged INT2 cache. `pool` points to num_blocks * num_kv_heads * int2kv_record_bytes(group_size)
 * bytes (device, 16-byte aligned). The caller zero-fills it once; every slot is rewritten in full
 * by an append, so no clearing is needed when blocks are reused. */
typedef struct int2kv_cache {
  void* pool;
  int32_t num_blocks;
  int32_t num_kv_heads;
  int32_t block_size; /* must be 16  */
  int32_t head_dim;   /* must be 128 */
  int32_t group_size; /* 32 or 128   */
} int2kv_cache;

/* Thread-local description of the last non-OK status ("" if none). */
const char* int2kv_last_error(void);

/* Library version string. */
const char* int2kv_version(void);

/* Bytes of the pool for the given shape: num_blocks * num_kv_heads * int2kv_record_bytes(group_size)
 * (0 for a group size other than 32 or 128, or a non-positive count). */
size_t int2kv_pool_bytes(int num_blocks, int num_kv_heads, int group_size);

/* Bytes of one (block, KV head) record: 1536 at group size 32, 1152 at 128, 0 otherwise. */
size_t int2kv_record_bytes(int group_size);

/* Rotated key mean mu_h R_{K,h}, precomputed once per KV head and subtracted right after the
 * key rotation in the cache write (Sec. 6 efficiency analysis; appendix key-mean
 * application: (k - mu) R_K = k R_K - mu R_K).
 *   R_k   : fp32 [H_kv, 128, 128], row-major, the row-vector rotation z -> z R_K
 *   mu    : fp32 [H_kv, 128]
 *   mu_rk : fp32 [H_kv, 128] (output)
 * Accumulates in fp32 in channel order. */
int int2kv_prepare_mu_rot(const float* R_k, const float* mu, float* mu_rk, int num_kv_heads,
                          hipStream_t stream);

/* Folded output projection W-bar_{O,j} = W_{O,j} R_{V,h(j)} (appendix "Equivalent inference
 * implementation"), so that y = concat_j(o'_j) W-bar_O^T with o'_j = o_j R_V needs no
 * un-rotation.
 *   W_o        : bf16 [d_model, H_q*128] row-major (W_{O,j} = columns j*128 .. j*128+127)
 *   R_v        : fp32 [H_kv, 128, 128]
 *   W_o_folded : bf16 [d_model, H_q*128] (output; fp32 accumulation, rounded once to bf16) */
int int2kv_fold_wo(const uint16_t* W_o, const float* R_v, uint16_t* W_o_folded, int d_model,
                   int num_q_heads, int num_kv_heads, hipStream_t stream);

/* Output-projection weights in the form the decode's projection streams best: fp16, stored as
 * 128-row x 32-column operand tiles, each 8 KiB tile contiguous (row blocks padded with zero
 * rows to a multiple of 128). With R_v given, the value rotation is folded in first, as in
 * int2kv_fold_wo (W-bar_{O,j} = W_{O,j} R_{V,h(j)}, appendix "Equivalent inference
 * implementation"), accumulated in fp32 and rounded once to fp16; without it the bf16 weights
 * are converted exactly. Weights must lie within the fp16 range (|w| <= 65504); values below
 * 2^-14 keep the fp16 subnormal spacing 2^-24. Done once per layer, like the fold.
 *   W_o        : bf16 [d_model, H_q*128] row-major
 *   R_v        : fp32 [H_kv, 128, 128], or NULL (no fold)
 *   W_prepared : int2kv_prepared_wo_bytes(d_model, H_q) bytes, 16-byte aligned (output); must
 *                not overlap W_o */
size_t int2kv_prepared_wo_bytes(int d_model, int num_q_heads);
int int2kv_prepare_wo(const uint16_t* W_o, const float* R_v, uint16_t* W_prepared, int d_model,
                      int num_q_heads, int num_kv_heads, hipStream_t stream);

/* Weight formats of the output projection in int2kv_decode (wo_format). */
enum {
  INT2KV_WO_PLAIN = 0,          /* W_O, bf16 row-major; the merge un-rotates o by R_V          */
  INT2KV_WO_FOLDED = 1,         /* W-bar_O from int2kv_fold_wo, bf16 row-major                */
  INT2KV_WO_PREPARED = 2,       /* int2kv_prepare_wo output without R_V (merge un-rotates)    */
  INT2KV_WO_PREPARED_FOLDED = 3 /* int2kv_prepare_wo output with R_V folded in                */
};

/* Quantize already rotated rows and store them (the quantizer and packer alone; results are
 * bit-exact with the arithmetic above).
 *   k_rot, v_rot : fp32 [n, H_kv, 128]: (k - mu) R_K and v R_V
 *   slot_mapping : int32 [n]; a negative slot skips the token; slots must be distinct
 *   clip_k/clip_v: clip ratios c_K, c_V in (0, 1] (1 = no clipping) */
int int2kv_quantize_pack_rotated(const int2kv_cache* cache, const float* k_rot, const float* v_rot,
                                 const int32_t* slot_mapping, int num_tokens, float clip_k,
                                 float clip_v, hipStream_t stream);

/* Cache write (Sec. 4.1; Sec. 6): per token and KV head, k R_K - mu R_K and v R_V with fp32
 * accumulation, then INT2 group quantization and packing into the slot given by slot_mapping.
 *   k, v         : bf16 [n, H_kv, 128] (post-RoPE keys; values), 16-byte aligned
 *   slot_mapping : int32 [n]; negative = skip; distinct slots
 *   R_k, R_v     : fp32 [H_kv, 128, 128], 16-byte aligned;  mu_rk: fp32 [H_kv, 128] from
 *                  int2kv_prepare_mu_rot, 16-byte aligned
 * The rotation runs on the matrix cores with R split into three bf16 terms (exact products, fp32
 * accumulation starting from -mu R_K), so codes may differ from an exact-arithmetic rotation only
 * where x sits at a rounding boundary of the quantizer. */
int int2kv_quantize_append(const int2kv_cache* cache, const uint16_t* k, const uint16_t* v,
                           const int32_t* slot_mapping, int num_tokens, const float* R_k,
                           const float* R_v, const float* mu_rk, float clip_k, float clip_v,
                           hipStream_t stream);

/* Flags of int2kv_quantize_append_rope: rotate keys (values) by the normalized Sylvester Hadamard
 * matrix H_128 / sqrt(128), entry (i, c) = (-1)^popcount(i & c) / sqrt(128), instead of R_K (R_V),
 * the QuaRot base rotation (Sec. 2; Sec. 5 baselines). The library applies it without reading a
 * matrix: the +-1 entries are exact matrix-core operands (one pass instead of the three of a dense
 * fp32 R) and the fp32 sum is scaled by RN(1 / sqrt(128)). Readers (decode, fold, mu_rot) take the
 * dense fp32 matrix with entries +-RN(1 / sqrt(128)), which is the same rotation. */
#define INT2KV_HADAMARD_K 1
#define INT2KV_HADAMARD_V 2

/* Cache write fed with pre-RoPE keys (appendix, key-mean estimation and application: the mean is
 * subtracted from the post-RoPE key, then rotated and quantized), fused in one kernel:
 *     k_rope = bf16(RoPE(k, positions[i])),  stored: Q2((k_rope - mu) R_K) and Q2(v R_V),
 * RoPE with rotate-half pairs (i, i + 64), i < 64, from the caller's table:
 *     y_i = x_i cos_i - x_{i+64} sin_i,   y_{i+64} = x_{i+64} cos_i + x_i sin_i,
 * each evaluated exactly in fp64 (bf16 x fp32 products) and rounded once to bf16, nearest even.
 *   positions   : int32 [num_tokens], the tokens' positions; NULL = keys are already post-RoPE (the
 *                 write then equals int2kv_quantize_append, or its Hadamard form with flags)
 *   cos_sin     : fp32 [max_pos, 128], row p = (cos theta_{p,0..63}, sin theta_{p,0..63})
 *   flags       : INT2KV_HADAMARD_K / INT2KV_HADAMARD_V (the matching R may then be NULL)
 *   k_rope_out  : optional bf16 [num_tokens, H_kv, 128]: the post-RoPE keys (for the BF16 window)
 * A token whose position lies outside [0, max_pos) is skipped: no cache write and no k_rope_out row.
 * Other arguments as int2kv_quantize_append (mu_rk = mu R_K, with the dense Hadamard under
 * INT2KV_HADAMARD_K). */
int int2kv_quantize_append_rope(const int2kv_cache* cache, const uint16_t* k, const uint16_t* v,
                                const int32_t* slot_mapping, const int32_t* positions, int num_tokens,
                                const float* cos_sin, int max_pos, const float* R_k, const float* R_v,
                                const float* mu_rk, float clip_k, float clip_v, int flags, uint16_t* k_rope_out,
                                hipStream_t stream);

/* int2kv_quantize_append that also reports each token's reconstruction error, for the diagnostics of
 * Sec. 3.2 (E_rec, eq:raw_reconstruction_objective): err[(i * H_kv + h) * 2 + 0] = ||x - x^||^2 of
 * the key and [... + 1] of the value of token i, KV head h, where x is the library's fp32 rotated
 * (and, for keys, centered) row and x^ its dequantized INT2 row; since R_K, R_V are orthogonal this
 * is ||k - k~||^2 (k~ = k^ R_K^T + mu) and ||v - v~||^2 in the model's basis. err: fp32
 * [num_tokens, H_kv, 2], written for every token (also for skipped slots). Cache bytes are those of
 * int2kv_quantize_append. */
int int2kv_quantize_append_error(const int2kv_cache* cache, const uint16_t* k, const uint16_t* v,
                                 const int32_t* slot_mapping, int num_tokens, const float* R_k,
                                 const float* R_v, const float* mu_rk, float clip_k, float clip_v,
                                 float* err, hipStream_t stream);

/* Workspace bytes int2kv_decode needs for these sizes (d_model = 0 when W_O is not applied). */
size_t int2kv_decode_workspace_bytes(int batch, int num_q_heads, int num_kv_heads, int max_ctx,
                                     int d_model);

/* Decode attention over the INT2 cache for one new query per sequence.
 *   q            : bf16 [B, H_q, 128] (post-RoPE), 16-byte aligned
 *   block_table  : int32 [B, max_blocks_per_seq]; entry i of sequence b is the physical
 *                  block of tokens 16i .. 16i+15
 *   ctx_lens     : int32 [B] cached tokens to attend (the current token is appended first);
 *                  lengths are clamped to [0, min(max_ctx, 16*max_blocks_per_seq)], and blocks
 *                  outside [0, num_blocks) are skipped
 *   max_ctx      : host-side upper bound of ctx_lens (sizes the split-context grid)
 *   R_k, R_v     : fp32 [H_kv, 128, 128], 16-byte aligned (R_v may be NULL with a folded W_o)
 *   W_o          : output-projection weights in the format wo_format names, 16-byte aligned, or
 *                  NULL (no output projection). Row-major bf16 weights are applied on the matrix
 *                  cores with o split into two bf16 terms (fp32-like precision); prepared fp16
 *                  weights with o rounded once to fp16 (relative error <= 2^-11 per element). The
 *                  K range is split in fixed slices summed in a fixed order (deterministic)
 *   wo_format    : INT2KV_WO_PLAIN, _FOLDED, _PREPARED or _PREPARED_FOLDED (with a folded format
 *                  R_v is not applied); ignored when W_o is NULL
 *   out          : fp32 [B, H_q, 128] if W_o is NULL, else fp32 [B, d_model]
 *   workspace    : device scratch of at least int2kv_decode_workspace_bytes(...) bytes
 * The context is split into fixed-size chunks scanned in parallel (online softmax per chunk),
 * then merged with a log-sum-exp reduction; sequences with ctx_len 0 produce zeros. */
int int2kv_decode(const int2kv_cache* cache, const uint16_t* q, int batch, int num_q_heads,
                  const int32_t* block_table, int max_blocks_per_seq, const int32_t* ctx_lens,
                  int max_ctx, const float* R_k, const float* R_v, const uint16_t* W_o, int d_model,
                  int wo_format, float* out, void* workspace, size_t workspace_bytes,
                  hipStream_t stream);

/* One decode step of a serving loop: the cache write of the current tokens
 * (int2kv_quantize_append with k, v, slot_mapping, num_tokens, R_k, R_v, mu_rk, clip_k, clip_v)
 * followed by int2kv_decode with the remaining arguments; the results are bit-identical to those
 * two calls made in that order. With the matrix-core decode and at most 256 tokens, the cache
 * write runs as extra work-groups of the decode's first launch, beside the query preparation
 * (which does not read the cache), instead of as a launch of its own. R_v is required when
 * num_tokens > 0 (the cache write uses it); num_tokens = 0 makes this int2kv_decode. Errors as
 * for the two calls; nothing is launched on an argument error. */
int int2kv_append_decode(const int2kv_cache* cache, const uint16_t* k, const uint16_t* v,
                         const int32_t* slot_mapping, int num_tokens, const float* mu_rk, float clip_k,
                         float clip_v, const uint16_t* q, int batch, int num_q_heads,
                         const int32_t* block_table, int max_blocks_per_seq, const int32_t* ctx_lens,
                         int max_ctx, const float* R_k, const float* R_v, const uint16_t* W_o,
                         int d_model, int wo_format, float* out, void* workspace,
                         size_t workspace_bytes, hipStream_t stream);

/* Bytes of the static scratch behind int2kv_append_decode_noalloc (64 MiB per GPU). */
#define INT2KV_NOALLOC_SCRATCH_BYTES (64u << 20)

/* int2kv_append_decode without a workspace argument, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that forbid allocation).
 * The decode's workspace is a static device array of INT2KV_NOALLOC_SCRATCH_BYTES inside the
 * library, one copy per GPU, held until the process ends; its device address is looked up once per
 * device on the first call made there (hipGetSymbolAddress with that device current). The call
 * allocates nothing and calls no allocating routine. Results, arguments and errors as
 * int2kv_append_decode; in addition a call whose workspace (int2kv_decode_workspace_bytes of its
 * sizes) exceeds the scratch returns INT2KV_EWORKSPACE without launching. Every call on a GPU shares
 * that GPU's scratch and leaves its contents behind (nothing in it needs to start at zero): calls
 * that overlap on one GPU (concurrent streams, or threads) race and must be serialized by the
 * caller. */
int int2kv_append_decode_noalloc(const int2kv_cache* cache, const uint16_t* k, const uint16_t* v,
                                 const int32_t* slot_mapping, int num_tokens, const float* mu_rk, float clip_k,
                                 float clip_v, const uint16_t* q, int batch, int num_q_heads,
                                 const int32_t* block_table, int max_blocks_per_seq, const int32_t* ctx_lens,
                                 int max_ctx, const float* R_k, const float* R_v, const uint16_t* W_o, int d_model,
                                 int wo_format, float* out, hipStream_t stream);

/* BF16 sink and recent windows (Sec. 4.1; Sec. 5 implementation details: the paper keeps the
 * first 64 and the last 256 tokens of a sequence out of INT2). Window tokens keep the key
 * centering and are held in BF16; their values are held unchanged. The window store is a caller
 * buffer of rows, each row one token for every KV head: win[(row * H_kv + h) * 128 + c], bf16,
 * 16-byte aligned; row b * win_cap + t is token t of sequence b in int2kv_decode_window.
 *
 * int2kv_window_write stores num_tokens tokens: win_k[row] = bf16_rne(fp32(k - mu)) (the key
 * mean mu in the model's basis, fp32 [H_kv, 128]), win_v[row] = v (bit copy).
 *   k, v     : bf16 [num_tokens, H_kv, 128]
 *   rows     : int32 [num_tokens]; a negative row, or one >= num_rows, skips the token; rows must
 *              be distinct
 * num_tokens = 0 launches nothing. Returns INT2KV_EINVAL on NULL or misaligned pointers. */
int int2kv_window_write(const uint16_t* k, const uint16_t* v, const int32_t* rows, int num_tokens,
                        int num_kv_heads, const float* mu, uint16_t* win_k, uint16_t* win_v,
                        int num_rows, hipStream_t stream);

/* int2kv_decode over the INT2 tokens (block_table, ctx_lens) together with each sequence's window
 * tokens (win_lens[b], clamped to [0, win_cap], rows b * win_cap .. of win_k / win_v): one softmax
 * over both sets (eq:int2_attention, with the window tokens' keys and values as stored). The order
 * of tokens does not matter, so the window may be a ring. Other arguments, results, workspace and
 * errors as int2kv_decode; in addition R_v is required (the window's output joins the INT2 part in
 * the R_V basis), win_cap must be in [1, 512], and win_k, win_v must be 16-byte aligned. */
int int2kv_decode_window(const int2kv_cache* cache, const uint16_t* q, int batch, int num_q_heads,
                         const int32_t* block_table, int max_blocks_per_seq, const int32_t* ctx_lens,
                         int max_ctx, const float* R_k, const float* R_v, const uint16_t* W_o,
                         int d_model, int wo_format, const uint16_t* win_k, const uint16_t* win_v,
                         const int32_t* win_lens, int win_cap, float* out, void* workspace,
                         size_t workspace_bytes, hipStream_t stream);

/* Output-error diagnostics of the INT2 cache (Sec. 3.2; appendix output-space error metrics):
 * for every sequence b and query head j, with p the attention of q_j over the full-precision keys
 * k, p~ over the cache's effective INT2 keys k~ = k^ R_K^T + mu, V the full-precision values and V~
 * the effective INT2 values v^ R_V^T,
 *     dy_K = ((p~ - p)^T V) W_{O,j}^T,   dy_V = (p~^T (V~ - V)) W_{O,j}^T,
 * so that y~_j - y_j = dy_K + dy_V exactly (the key- and value-induced output errors), and
 *     stats[(b * H_q + j) * 4 + {0, 1, 2, 3}] = ||dy_K + dy_V||^2 (E_out), ||dy_K||^2, ||dy_V||^2,
 *                                              <dy_K, dy_V>.
 *   k_rows, v_rows : bf16 full-precision keys (raw, not centered) and values, row b * row_cap + t
 *                    holding token t of sequence b for every KV head ([rows, H_kv, 128]), the
 *                    tokens the cache holds at block_table / ctx_lens (lengths are also clamped to
 *                    row_cap)
 *   W_o            : bf16 [d_model, H_q * 128] row-major (required)
 *   dy             : fp32 [B, H_q, 2, d_model] (dy_K, dy_V) or NULL
 *   workspace      : int2kv_output_error_workspace_bytes(...) bytes, 256-byte aligned
 * Other arguments as int2kv_decode; up to 16 query heads per KV head. Scores and sums run in fp32
 * (INT2 scores with the rotated query, as the vector-ALU decode). */
size_t int2kv_output_error_workspace_bytes(int batch, int num_q_heads, int num_kv_heads, int max_ctx,
                                           int d_model);
int int2kv_output_error(const int2kv_cache* cache, const uint16_t* q, int batch, int num_q_heads,
                        const int32_t* block_table, int max_blocks_per_seq, const int32_t* ctx_lens,
                        int max_ctx, const float* R_k, const float* R_v, const uint16_t* k_rows,
                        const uint16_t* v_rows, int row_cap, const uint16_t* W_o, int d_model,
                        float* stats, float* dy, void* workspace, size_t workspace_bytes,
                        hipStream_t stream);

/* ---- OptR offline calibration (Sec. 4.2 - 4.5; Algorithm 1 of the appendix), fp64 on the GPU.
 * For every KV head h the corrected rotations R = R^0 exp(A - A^T) (eq:OptR_skew) are fitted to
 * calibration traces: first A_K on the key objective (eq:OptR_key_loss)
 *     L_K = mean over rows (t, j) of KL(p_t || p^K_t) + lambda_K ||((p^K_t - p_t)^T V) W_{O,j}^T||^2 / d_model,
 * then A_V on the value objective (eq:OptR_value_loss) under the selected key rotation's
 * probabilities p^K-hat:
 *     L_V = mean over rows of ||(p^K-hat_t^T (V~ - V)) W_{O,j}^T||^2 / d_model.
 * Rows: query heads j of the KV head's group at the final n_last positions t of each sequence,
 * attending causally (s <= t). Effective keys k~ = Q2((k - mu) R_K) R_K^T and values
 * v~ = Q2(v R_V) R_V^T use the cache's own quantizer on the fp32 rounding of the rotated rows
 * (group_size, clip ratios); tokens s < sink and s > t - recent stay in full precision (BF16
 * windows). Gradients pass the quantizer by the straight-through estimator of eq:OptR_ste: an
 * element's gradient passes when it lies inside its group's clipped range [c mn, c mx]; scale and
 * zero are held fixed. The optimizer is Adam (betas 0.9 / 0.999, eps 1e-8, learning rate lr); the
 * iterate with the lowest held-out objective among A = 0 and every eval_every-th step is kept.
 * All arithmetic is fp64; inputs stay as given (bf16 traces, fp32 R^0 and mu). Up to 16 query heads
 * per KV head. */
typedef struct int2kv_optr_traces {
  const uint16_t* k;          /* device bf16 [T, H_kv, 128]: keys (post-RoPE, raw); 16-byte aligned */
  const uint16_t* v;          /* device bf16 [T, H_kv, 128]: values; 16-byte aligned */
  const uint16_t* q;          /* device bf16 [T, H_q, 128]: queries (post-RoPE) */
  const int32_t* seq_starts;  /* HOST int32 [num_seqs + 1]: token offsets, seq_starts[0] = 0,
                                 sequences of 0 .. 4096 tokens */
  int num_seqs;
} int2kv_optr_traces;

typedef struct int2kv_optr_config {
  int num_kv_heads, num_q_heads, d_model, group_size; /* group_size 32 or 128 */
  float clip_k, clip_v;                               /* the paper's setting: 0.96, 0.92 */
  double lambda_k;                                    /* 1.0 */
  int n_last, sink, recent;                           /* 64, 64, 256 */
  int steps, eval_every;                              /* 80, 20 */
  double lr;                                          /* 0.02 */
} int2kv_optr_config;

/* Workspace bytes of the calls below (heldout may be NULL for the loss calls); 0 on bad arguments. */
size_t int2kv_optr_workspace_bytes(const int2kv_optr_config* cfg, const int2kv_optr_traces* calib,
                                   const int2kv_optr_traces* heldout);
/* Per-channel key mean per KV head (appendix, key-mean estimation): mu[h][c] = fp32(fp64 mean over
 * the num_tokens keys k [T, H_kv, 128] bf16). */
int int2kv_optr_key_mean(const uint16_t* k, int num_tokens, int num_kv_heads, float* mu, hipStream_t stream);
/* L_K of every KV head at generators A (device fp64 [H_kv, 128, 128]) into loss (device fp64 [H_kv]),
 * and dL_K/dA into grad (device fp64 [H_kv, 128, 128]) unless grad is NULL. R0_k: fp32 [H_kv, 128, 128];
 * mu: fp32 [H_kv, 128]; W_o: bf16 [d_model, H_q * 128]. */
int int2kv_optr_key_loss(const int2kv_optr_config* cfg, const int2kv_optr_traces* traces, const float* R0_k,
                         const float* mu, const uint16_t* W_o, const double* A, double* loss, double* grad,
                         void* workspace, size_t workspace_bytes, hipStream_t stream);
/* L_V at generators A_v under the key probabilities of generators A_k, and dL_V/dA_v. */
int int2kv_optr_value_loss(const int2kv_optr_config* cfg, const int2kv_optr_traces* traces, const float* R0_k,
                           const double* A_k, const float* mu, const float* R0_v, const uint16_t* W_o,
                           const double* A_v, double* loss, double* grad, void* workspace, size_t workspace_bytes,
                           hipStream_t stream);
/* Algorithm 1 for every KV head at once: R_k, R_v (device fp32 [H_kv, 128, 128]) receive the
 * selected R^0 exp(A - A^T); A_k, A_v (device fp64, may be NULL) the selected generators; history
 * (device fp64, may be NULL) [2][H_kv][steps + 1 + steps / eval_every]: for keys, then values, the
 * training objective before each step followed by the held-out objectives at A = 0 and every
 * eval_every-th step. The host tables of both trace sets are uploaded at the start (the call waits
 * for that copy); the rest runs asynchronously on stream. */
int int2kv_optr_calibrate(const int2kv_optr_config* cfg, const int2kv_optr_traces* calib,
                          const int2kv_optr_traces* heldout, const float* R0_k, const float* R0_v, const float* mu,
                          const uint16_t* W_o, float* R_k, float* R_v, double* A_k, double* A_v, double* history,
                          void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Measurement hook: when set (non-NULL), the calls this thread issues attach `before_scan` and
 * `after_scan` to the dispatch of their dominant kernel (hipExtLaunchKernel): the split-context scan
 * of int2kv_decode, int2kv_append_decode and int2kv_decode_window, the cache-write kernel of
 * int2kv_quantize_append(_error), the diagnostics scan of int2kv_output_error. They then mark that kernel's own start and end, and a caller can time it
 * alone with hipEventElapsedTime, without extra packets between the kernels. Pass NULLs to disable.
 * The setting is per calling thread. The events are owned by the caller and must outlive the calls
 * that record them. */
int int2kv_set_decode_events(hipEvent_t before_scan, hipEvent_t after_scan);

/* Tuning knobs for measurement sweeps: context chunk in tokens (multiple of 64, 0 = automatic)
 * and decode kernel variant (0 = automatic, 1 = vector ALU, 2 = matrix core; the matrix-core scan
 * serves at most 8 query heads per KV head, wider groups always use the vector-ALU scan). The
 * setting applies to the calls of the calling thread only (thread-local), including
 * int2kv_decode_workspace_bytes: size a workspace on the thread that decodes with it. Returns
 * INT2KV_EINVAL for out-of-range values. */
int int2kv_set_decode_tuning(int chunk_tokens, int variant);

#ifdef __cplusplus
}
#endif

#endif /* INT2KV_H */
