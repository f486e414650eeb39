// Internal launcher declarations shared by the C-ABI front end and the kernel files.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace int2kv {

struct CacheView {
  uint8_t* pool;
  int num_blocks;
  int num_kv_heads;
  int groups;  // groups per token: 4 (32 channels each) or 1 (128)
};

// ---- cache write (append.hip)
hipError_t launch_prepare_mu_rot(const float* R_k, const float* mu, float* mu_rk, int H, hipStream_t s);
hipError_t launch_fold_wo(const uint16_t* W_o, const float* R_v, uint16_t* W_f, int d_model, int Hq,
                          int H, hipStream_t s);
hipError_t launch_pack_rotated(CacheView c, const float* k_rot, const float* v_rot, const int32_t* slots,
                               int n, float clip_k, float clip_v, hipStream_t s);
// Optional stages of the cache write: RoPE of pre-RoPE keys (positions non-null) and the Hadamard
// rotation in place of R_K (hadamard bit 0) and / or R_V (bit 1).
struct AppendOptions {
  const int32_t* positions = nullptr;
  const float* cos_sin = nullptr;
  int max_pos = 0;
  uint16_t* k_rope_out = nullptr;
  int hadamard = 0;
};
// ev0 / ev1 (may be null): events that track the append kernel's own start and end
hipError_t launch_append_mfma(CacheView c, const uint16_t* k, const uint16_t* v, const int32_t* slots,
                              int n, const float* R_k, const float* R_v, const float* mu_rk, float clip_k,
                              float clip_v, hipStream_t s, hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr,
                              float* err = nullptr,  // err: [n, H, 2] squared reconstruction errors
                              const AppendOptions* opts = nullptr);

// ---- decode (decode.hip, decode_mfma.hip, wo_gemm.hip)
struct DecodePlan {
  int chunk_tokens;
  int n_chunks;
  int variant;        // 1 = vector ALU, 2 = matrix core
  int wo_ksplit;
  int grid_g;         // work-groups of the matrix-core scan
  int s1;             // slot ranges per sequence of the two-stage merge (0: one stage)
  size_t off_qrot, off_qop, off_prefix, off_wginfo, off_seqwg, off_pages, off_part, off_part2, off_win, off_o,
      off_wo, total;
};

struct DecodeArgs {
  const uint8_t* pool;
  int num_blocks, H;
  const uint16_t* q;
  int B, Hq, gq;
  const int32_t* block_table;
  int max_blocks;
  const int32_t* ctx_lens;
  int max_ctx;
  const float* R_k;
  const float* R_v;
  float* qrot;     // [B, Hq, 128] fp32
  uint8_t* qop;    // matrix-core query operands
  float* part;     // vector-ALU scan: [B, n_chunks, Hq, kPartStride]; matrix-core scan: [G + B, Hq, kPartStride]
  int chunk_tokens, n_chunks;
  int32_t* prefix; // [B + 1] page prefix sums (matrix-core scan)
  int32_t* wg_info;  // [grid_g + 1][4]: first sequence of each scan work-group, its page range, lo(g)
  int32_t* seq_wg;   // [B][2]: first and last scan work-group whose range meets each sequence
  uint32_t* pages;   // page list of the matrix-core scan: [total pages + padding][4]
  int grid_g;      // work-groups of the matrix-core scan
  int groups;      // groups per token of the cache (4 or 1)
  float* wpart;    // BF16-window partials [win_slices][B, Hq, kPartStride] folded in by the merge, or null
  float* part2;    // two-stage merge (few, long sequences): [B, s1, Hq, kPartStride] folded slot ranges
  int s1;          // slot ranges per sequence of the two-stage merge (0: one stage)
  int win_slices;  // window slices of kWinSliceTokens tokens (ceil(win_cap / kWinSliceTokens))
};

constexpr int kPartStride = 132;  // m, l, 2 pad, O[128]

// BF16 sink/recent window of each sequence: rows b * cap + t, each [H, 128] bf16
struct WindowArgs {
  const uint16_t *k, *v;
  const int32_t* lens;  // [B] tokens in each window (clamped to [0, cap])
  int cap;
};
constexpr int kWinMaxGq = 16;
constexpr int kWinMaxCap = 512;
constexpr int kWinSliceTokens = 96;                            // window tokens per partial
constexpr int kMerge2Ranges = 16;      // slot ranges per sequence in the two-stage merge
constexpr int kMerge2MaxUnits = 128;   // two-stage merge when batch x KV heads is below this
// window partials per (sequence, query head)
constexpr int kWinMaxSlices = (kWinMaxCap + kWinSliceTokens - 1) / kWinSliceTokens;
hipError_t launch_window_write(const uint16_t* k, const uint16_t* v, const int32_t* rows, int n, int H, const float* mu,
                               uint16_t* win_k, uint16_t* win_v, int num_rows, hipStream_t s);
// window partials into a.wpart (needs a.R_v)
hipError_t launch_window_attn(const DecodeArgs& a, const WindowArgs& w, hipStream_t s);

hipError_t launch_qrot(const DecodeArgs& a, hipStream_t s);
// ev0 / ev1 (may be null): events that track the scan kernel's own start and end
hipError_t launch_decode_split_valu(const DecodeArgs& a, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1);
// Cache write of the current tokens run inside the preparation launch (int2kv_append_decode).
struct AppendArgs {
  CacheView cv;
  const uint16_t *k, *v;
  const int32_t* slots;
  int n;
  const float *R_k, *R_v, *mu_rk;
  float clip_k, clip_v;
  int nbx;  // blocks per (KV head, K|V), set by the launcher
};
// ap (may be null): the cache write to run beside the query preparation
hipError_t launch_qprep(const DecodeArgs& a, const AppendArgs* ap, hipStream_t s);
hipError_t launch_decode_split_mfma(const DecodeArgs& a, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1);
size_t qop_bytes(int B, int H, int gq);
// Head-output formats of the merges: fp32 to `out`, or for the output projection (to `ob`) two bf16
// terms of each value (ob[0 .. B*Hq*128) = hi, ob[B*Hq*128 ..) = lo) or one fp16 term.
enum OutFmt { kOutF32 = 0, kOutBf16x2 = 1, kOutF16 = 2 };
hipError_t launch_merge(const DecodeArgs& a, bool unrotate, float* out, uint16_t* ob, int fmt, hipStream_t s);
hipError_t launch_merge_flat(const DecodeArgs& a, bool unrotate, float* out, uint16_t* ob, int fmt, hipStream_t s);
int num_cus();                        // compute units of the current device
int wo_slice(int K, int N, int B);    // K per work-group of the output projection
int wo_ksplit(int K, int N, int B);   // K slices of the output projection (partial products in the workspace)
// prepared: W is int2kv_prepare_wo output and ob one fp16 term; else W is bf16 row-major, ob two bf16 terms
hipError_t launch_wo_gemm(const uint16_t* ob, const uint16_t* W, bool prepared, float* y, float* partial, int B,
                          int K, int N, int ksplit, hipStream_t s);
size_t prepared_wo_elems(int N, int K);  // fp16 elements of the prepared weights (rows padded to 128)
hipError_t launch_prepare_wo(const uint16_t* W_o, const float* R_v, uint16_t* Wp, int N, int Hq, int H,
                             hipStream_t s);

// ---- output-error diagnostics (outerr.hip)
constexpr int kOePartStride = 4 + 3 * kHeadDim;  // m1, l1, m2, l2, A1[128], A2[128], A3[128]
constexpr int kOeRowTile = 128;  // W_O rows per output-error projection block (a statistics partial each)
struct OutErrArgs {
  DecodeArgs a;                 // cache, queries, block table, lengths, R_K, R_V, qrot, chunking
  const uint16_t *k_rows, *v_rows;  // full-precision keys and values, row b * row_cap + t, [H, 128]
  int row_cap;
  float* part;                  // [B, n_chunks, Hq, kOePartStride]
  uint16_t* dov;                // [3][B, Hq, 2, 128]: o2 - o1, o3 - o2 (model basis) as three bf16 terms
                                // whose sum is the fp32 value exactly
  float* spart;                 // [B, Hq, row tiles of kOeRowTile rows, 4]
};
// stats: [B, Hq, 4]; dy (may be null): [B, Hq, 2, d_model]; ev0 / ev1 track the scan kernel
hipError_t launch_output_error(const OutErrArgs& e, const uint16_t* W_o, int d_model, float* stats, float* dy,
                               hipStream_t s, hipEvent_t ev0, hipEvent_t ev1);

// ---- OptR offline calibration (optr.hip): fp64 throughout
constexpr int kCalMaxLen = 4096;  // tokens per calibration sequence
constexpr int kCalSplit = 16;     // token slices of the rotation-gradient reduction
constexpr int kCalScratch = 11;   // 128 x 128 scratch matrices per KV head of the matrix functions
struct CalSeq {
  int start, len, t0, row0;  // first token, length, first query position, first row
  long long p0;              // offset of the sequence's [rows][len] block of per-row token weights
};
// One trace set (calibration or held-out): inputs and its per-set buffers.
struct CalSet {
  const uint16_t *k, *v, *q;       // bf16 [T, H, 128], [T, H, 128], [T, Hq, 128]
  int T, nseq, nrows;              // nrows: query rows of one KV head
  int maxlen;                      // longest sequence
  int ntiles;                      // row tiles of the objective kernels
  int4* tiles;                     // [ntiles]: (sequence, first row, rows, position of the first row)
  long long pelems;                // per KV head: sum over sequences of rows * len
  CalSeq* seqs;                    // [nseq]
  int* row_seq;                    // [nrows]: sequence of each row
  double *zhat, *xeff, *gx, *gz;   // [H, T, 128]: dequantized rotated rows, effective rows, gradients
  uint8_t* mask;                   // [H, T, 128]: straight-through mask
  double* pd;                      // [H, pelems]: key probabilities, then logit gradients, on the tokens
                                   // read from INT2 (zero elsewhere, set once)
  double* pf;                      // [H, pelems]: scratch of the key-loss gradient
  double* fc;                      // [H, pelems]: full-precision logits f (rotation-independent, set once)
  double* pc;                      // [H, pelems]: full-precision probabilities p = softmax(f) (set once)
  double* rc;                      // [H, nrows, 2]: per row lse_f and LW (log-sum-exp of f over the row's
                                   // BF16-window tokens, -inf when none) (set once)
  double* wt;                      // [H, nrows, 128]: per row sum over its window tokens of exp(f - LW) v (set once)
  double* erow;                    // [H, nrows]: exp(LW - lse_k) of the latest key forward
  double* wrow;                    // [H, nrows, 128]: dO per row, then the value-loss row weights
  double* urow;                    // [H, nrows, 128]: M_j dO per row (key loss)
  double* lrow;                    // [H, nrows]: per-row losses
};
struct CalCfg {
  int H, Hq, gq, dm, ng;  // ng: quantizer groups per token (4 or 1)
  float clip_k, clip_v;
  double lam;
  int sink, recent, n_last;
  const float* mu;        // [H, 128]
  const float *R0k, *R0v; // fp32 [H, 128, 128]
  double* gram;           // [Hq, 128, 128]: W_{O,j}^T W_{O,j}
  double *R, *Rt;         // [H, 128, 128]: the current rotation and its transpose
  double* ex;             // [H, kCalScratch, 128, 128]
  double* drp;            // [kCalSplit, H, 128, 128]
  double* dr;             // [H, 128, 128]
};
size_t cal_set_bytes(int T, int nseq, int nrows, long long pelems, int H);
size_t cal_shared_bytes(int H, int Hq);
// carves a set's buffers from base and uploads its sequence and row tables (host starts [nseq + 1])
hipError_t cal_bind_set(CalSet& set, uint8_t* base, const uint16_t* k, const uint16_t* v, const uint16_t* q,
                        const int32_t* starts_host, int nseq, int H, int gq, int n_last, hipStream_t s);
void cal_bind_shared(CalCfg& c, uint8_t* base);
hipError_t cal_gram(const CalCfg& c, const uint16_t* W_o, hipStream_t s);
// loss[h] (device) of every KV head at generators A [H, 128, 128]; grad (may be null) receives dL/dA
// The rotation-independent part of the key objective for a bound set (after cal_bind_set, before any loss).
hipError_t cal_prepare_set(const CalCfg& c, CalSet& set, hipStream_t s);
hipError_t cal_key_loss(const CalCfg& c, CalSet& set, const double* A, double* loss, double* grad, hipStream_t s);
hipError_t cal_key_probs(const CalCfg& c, CalSet& set, const double* A, hipStream_t s);
hipError_t cal_value_loss(const CalCfg& c, CalSet& set, const double* A, double* loss, double* grad, hipStream_t s);
hipError_t cal_adam(double* A, const double* g, double* m, double* v, int n, int step, double lr, hipStream_t s);
// per head: when loss[h] < best[h], best[h] = loss[h] and A_best[h] = A[h]
hipError_t cal_select(const double* A, const double* loss, double* best, double* A_best, int H, hipStream_t s);
hipError_t cal_fill(double* p, size_t n, double v, hipStream_t s);
hipError_t cal_record(const double* loss, double* dst, int stride, int H, hipStream_t s);  // dst[h * stride] = loss[h]
// R0 exp(A - A^T) rounded to fp32
hipError_t cal_rotation_out(const CalCfg& c, const double* A, bool value, float* out, hipStream_t s);
hipError_t cal_key_mean(const uint16_t* k, int T, int H, float* mu, hipStream_t s);

}  // namespace int2kv
