// C-ABI front end: argument validation, workspace planning and kernel dispatch.
// Every entry point validates on the host and returns a negative status without launching on
// any argument error; nothing here allocates device memory or synchronizes.
#include <mutex>
#include <string>

#include "../../include/int2kv.h"
#include "common.h"
#include "kernels.h"

namespace int2kv {
bool mfma_decode_available();
}

using namespace int2kv;

namespace {

// Per-thread state: the last error message, the measurement knobs (int2kv_set_decode_tuning,
// int2kv_set_decode_events) of the calls this thread makes
thread_local std::string g_last_error;
thread_local int g_chunk_override = 0;
thread_local int g_variant_override = 0;
thread_local hipEvent_t g_ev_before = nullptr;
thread_local hipEvent_t g_ev_after = nullptr;

int fail(int status, const std::string& msg) {
  g_last_error = msg;
  return status;
}

int ok() {
  g_last_error.clear();
  return INT2KV_OK;
}

int hip_status(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(INT2KV_EHIP, std::string(what) + ": " + hipGetErrorString(e));
  return ok();
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

int check_cache(const int2kv_cache* c) {
  if (!c) return fail(INT2KV_EINVAL, "cache descriptor is NULL");
  if (!c->pool) return fail(INT2KV_EINVAL, "cache pool is NULL");
  if (!aligned(c->pool, 16)) return fail(INT2KV_EINVAL, "cache pool must be 16-byte aligned");
  if (c->num_blocks <= 0 || c->num_kv_heads <= 0) return fail(INT2KV_EINVAL, "cache has no blocks or heads");
  if (c->block_size != kBlock) return fail(INT2KV_EUNSUPPORTED, "block_size must be 16");
  if (c->head_dim != kHeadDim) return fail(INT2KV_EUNSUPPORTED, "head_dim must be 128");
  if (c->group_size != 32 && c->group_size != 128) return fail(INT2KV_EUNSUPPORTED, "group_size must be 32 or 128");
  if ((int64_t)c->num_blocks * kBlock > INT32_MAX) return fail(INT2KV_EUNSUPPORTED, "too many blocks for int32 slots");
  return INT2KV_OK;
}

bool valid_clip(float c) { return c > 0.0f && c <= 1.0f; }

CacheView view(const int2kv_cache* c) {
  return CacheView{static_cast<uint8_t*>(c->pool), c->num_blocks, c->num_kv_heads, kHeadDim / c->group_size};
}

}  // namespace

// Compute units of the current device (queried once per device; 256 when no device answers).
int int2kv::num_cus() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cached[dev] == 0) {
    hipDeviceProp_t prop;
    cached[dev] = hipGetDeviceProperties(&prop, dev) == hipSuccess && prop.multiProcessorCount > 0
                      ? prop.multiProcessorCount
                      : 256;
  }
  return cached[dev];
}

namespace {

DecodePlan make_plan(int B, int Hq, int H, int max_ctx, int d_model, int groups) {
  DecodePlan p{};
  const int gq = Hq / H;
  // the matrix-core scan serves up to 8 query heads per KV head; wider groups use the vector-ALU
  // scan (also when the tuning knob asks for the matrix-core one)
  (void)groups;
  const bool mfma_ok = gq <= 8 && mfma_decode_available();
  p.variant = g_variant_override == 1 || !mfma_ok ? 1 : 2;
  int chunk = g_chunk_override;
  if (chunk <= 0) {
    // the largest chunk (up to 4096 tokens) that still gives >= 1024 work-groups, so that 256 CUs
    // see several rounds of them; never below 512 tokens (per-group set-up and partials amortized)
    chunk = 4096;
    const long long units = (long long)B * H;
    while (chunk > 512 && units * ((max_ctx + chunk - 1) / chunk) < 1024) chunk /= 2;
  }
  if (p.variant == 2 && chunk > 4096) chunk = 4096;  // the matrix-core scan stages <= 256 pages
  p.chunk_tokens = chunk;
  p.n_chunks = max_ctx > 0 ? (max_ctx + chunk - 1) / chunk : 1;
  // matrix-core scan: persistent work-groups of min(H, 8) waves, enough to fill every CU
  const int nw = H < 8 ? H : 8;
  p.grid_g = num_cus() * (8 / nw);
  p.wo_ksplit = d_model > 0 ? wo_ksplit(Hq * kHeadDim, d_model, B) : 0;
  auto up = [](size_t x) { return (x + 255) & ~size_t(255); };
  size_t off = 0;
  p.off_qrot = off;
  off = up(off + (size_t)B * Hq * kHeadDim * sizeof(float));
  p.off_qop = off;
  off = up(off + qop_bytes(B, H, gq));
  p.off_prefix = off;
  off = up(off + (size_t)(B + 1) * sizeof(int32_t));
  p.off_wginfo = off;
  off = up(off + (size_t)(p.grid_g + 1) * 4 * sizeof(int32_t));
  p.off_seqwg = off;
  off = up(off + (size_t)B * 2 * sizeof(int32_t));
  // page list: one 16-byte entry per page of every sequence (lengths are clamped to max_ctx), plus
  // padding the scan may read (never use) one pair past the last page
  p.off_pages = off;
  off = up(off + ((size_t)B * (((size_t)max_ctx + kBlock - 1) / kBlock) + 8) * 16);
  p.off_part = off;
  const size_t part_rows = p.variant == 2 ? (size_t)(p.grid_g + B) : (size_t)B * p.n_chunks;
  off = up(off + part_rows * Hq * kPartStride * sizeof(float));
  // two-stage merge of the matrix-core scan for few, long sequences: folded slot ranges
  p.s1 = p.variant == 2 && (long long)B * H < kMerge2MaxUnits ? kMerge2Ranges : 0;
  p.off_part2 = off;
  off = up(off + (size_t)B * p.s1 * Hq * kPartStride * sizeof(float));
  p.off_win = off;  // BF16-window partials, [kWinMaxSlices][B, Hq, kPartStride]
  off = up(off + (size_t)kWinMaxSlices * B * Hq * kPartStride * sizeof(float));
  p.off_o = off;
  if (d_model > 0) off = up(off + (size_t)B * Hq * kHeadDim * sizeof(float));
  p.off_wo = off;
  if (d_model > 0 && p.wo_ksplit > 1) off = up(off + (size_t)p.wo_ksplit * B * d_model * sizeof(float));
  p.total = off;
  return p;
}

// Static scratch of the allocation-free decode step (int2kv_append_decode_noalloc): the decode's
// workspace as a file-scope device array, one copy per GPU, held until the process ends. Host code
// never uses the array's name as an address: the device address of each GPU's copy comes from
// hipGetSymbolAddress, taken once per device with that device current.
constexpr size_t kScratchBytes = (size_t)INT2KV_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The scratch's device address on the current device (looked up on the first call per device).
int scratch_for_current_device(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(INT2KV_EHIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(INT2KV_EUNSUPPORTED, "device index above 63");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return fail(INT2KV_EHIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
    if (!p) return fail(INT2KV_EHIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return INT2KV_OK;
}

}  // namespace

extern "C" {

const char* int2kv_last_error(void) { return g_last_error.c_str(); }

const char* int2kv_version(void) { return "int2kv 0.1 gfx950"; }

size_t int2kv_pool_bytes(int num_blocks, int num_kv_heads, int group_size) {
  if (num_blocks <= 0 || num_kv_heads <= 0) return 0;
  return (size_t)num_blocks * num_kv_heads * int2kv_record_bytes(group_size);
}

size_t int2kv_record_bytes(int group_size) {
  return group_size == 32 ? (size_t)Rec<4>::kBytes : group_size == 128 ? (size_t)Rec<1>::kBytes : 0;
}

int int2kv_set_decode_events(hipEvent_t before_scan, hipEvent_t after_scan) {
  if ((before_scan == nullptr) != (after_scan == nullptr))
    return fail(INT2KV_EINVAL, "pass both events or neither");
  g_ev_before = before_scan;
  g_ev_after = after_scan;
  return ok();
}

int int2kv_set_decode_tuning(int chunk_tokens, int variant) {
  if (chunk_tokens < 0 || chunk_tokens % 64 != 0 || chunk_tokens > (1 << 20))
    return fail(INT2KV_EINVAL, "chunk_tokens must be 0 or a positive multiple of 64");
  if (variant < 0 || variant > 2) return fail(INT2KV_EINVAL, "variant must be 0, 1 or 2");
  if (variant == 2 && !mfma_decode_available()) return fail(INT2KV_EUNSUPPORTED, "matrix-core decode not built");
  g_chunk_override = chunk_tokens;
  g_variant_override = variant;
  return ok();
}

int int2kv_prepare_mu_rot(const float* R_k, const float* mu, float* mu_rk, int num_kv_heads, hipStream_t stream) {
  if (!R_k || !mu || !mu_rk) return fail(INT2KV_EINVAL, "NULL pointer argument");
  if (num_kv_heads <= 0) return fail(INT2KV_EINVAL, "num_kv_heads must be positive");
  return hip_status(launch_prepare_mu_rot(R_k, mu, mu_rk, num_kv_heads, stream), "prepare_mu_rot");
}

int int2kv_fold_wo(const uint16_t* W_o, const float* R_v, uint16_t* W_o_folded, int d_model, int num_q_heads,
                   int num_kv_heads, hipStream_t stream) {
  if (!W_o || !R_v || !W_o_folded) return fail(INT2KV_EINVAL, "NULL pointer argument");
  if (d_model <= 0 || num_q_heads <= 0 || num_kv_heads <= 0 || num_q_heads % num_kv_heads)
    return fail(INT2KV_EINVAL, "bad d_model / head counts");
  if (W_o == W_o_folded) return fail(INT2KV_EINVAL, "W_o_folded must not alias W_o");
  return hip_status(launch_fold_wo(W_o, R_v, W_o_folded, d_model, num_q_heads, num_kv_heads, stream), "fold_wo");
}

size_t int2kv_prepared_wo_bytes(int d_model, int num_q_heads) {
  if (d_model <= 0 || num_q_heads <= 0) return 0;
  return prepared_wo_elems(d_model, num_q_heads * kHeadDim) * sizeof(uint16_t);
}

int int2kv_prepare_wo(const uint16_t* W_o, const float* R_v, uint16_t* W_prepared, int d_model, int num_q_heads,
                      int num_kv_heads, hipStream_t stream) {
  if (!W_o || !W_prepared) return fail(INT2KV_EINVAL, "NULL pointer argument");
  if (d_model <= 0 || num_q_heads <= 0 || num_kv_heads <= 0 || num_q_heads % num_kv_heads)
    return fail(INT2KV_EINVAL, "bad d_model / head counts");
  if (!aligned(W_prepared, 16)) return fail(INT2KV_EINVAL, "W_prepared must be 16-byte aligned");
  const uint8_t* src = reinterpret_cast<const uint8_t*>(W_o);
  const uint8_t* dst = reinterpret_cast<const uint8_t*>(W_prepared);
  if (dst < src + (size_t)d_model * num_q_heads * kHeadDim * 2 && src < dst + int2kv_prepared_wo_bytes(d_model, num_q_heads))
    return fail(INT2KV_EINVAL, "W_prepared must not overlap W_o");
  return hip_status(launch_prepare_wo(W_o, R_v, W_prepared, d_model, num_q_heads, num_kv_heads, stream), "prepare_wo");
}

int int2kv_quantize_pack_rotated(const int2kv_cache* cache, const float* k_rot, const float* v_rot,
                                 const int32_t* slot_mapping, int num_tokens, float clip_k, float clip_v,
                                 hipStream_t stream) {
  if (int st = check_cache(cache)) return st;
  if (num_tokens < 0) return fail(INT2KV_EINVAL, "num_tokens must be >= 0");
  if (num_tokens == 0) return ok();
  if (!k_rot || !v_rot || !slot_mapping) return fail(INT2KV_EINVAL, "NULL pointer argument");
  if (!valid_clip(clip_k) || !valid_clip(clip_v)) return fail(INT2KV_EINVAL, "clip ratios must be in (0, 1]");
  return hip_status(launch_pack_rotated(view(cache), k_rot, v_rot, slot_mapping, num_tokens, clip_k, clip_v, stream),
                    "quantize_pack_rotated");
}

int int2kv_quantize_append(const int2kv_cache* cache, const uint16_t* k, const uint16_t* v,
                           const int32_t* slot_mapping, int num_tokens, const float* R_k, const float* R_v,
                           const float* mu_rk, float clip_k, float clip_v, hipStream_t stream) {
  if (int st = check_cache(cache)) return st;
  if (num_tokens < 0) return fail(INT2KV_EINVAL, "num_tokens must be >= 0");
  if (num_tokens == 0) return ok();
  if (!k || !v || !slot_mapping || !R_k || !R_v || !mu_rk) return fail(INT2KV_EINVAL, "NULL pointer argument");
  if (!valid_clip(clip_k) || !valid_clip(clip_v)) return fail(INT2KV_EINVAL, "clip ratios must be in (0, 1]");
  if (!aligned(k, 16) || !aligned(v, 16) || !aligned(R_k, 16) || !aligned(R_v, 16) || !aligned(mu_rk, 16))
    return fail(INT2KV_EINVAL, "k, v, R_k, R_v and mu_rk must be 16-byte aligned");
  hipError_t e = launch_append_mfma(view(cache), k, v, slot_mapping, num_tokens, R_k, R_v, mu_rk, clip_k, clip_v,
                                    stream, g_ev_before, g_ev_after);
  return hip_status(e, "quantize_append");
}

int int2kv_quantize_append_rope(const int2kv_cache* cache, const uint16_t* k, const uint16_t* v,
                                const int32_t* slot_mapping, const int32_t* positions, int num_tokens,
                                const float* cos_sin, int max_pos, const float* R_k, const float* R_v,
                                const float* mu_rk, float clip_k, float clip_v, int flags, uint16_t* k_rope_out,
                                hipStream_t stream) {
  if (int st = check_cache(cache)) return st;
  if (num_tokens < 0) return fail(INT2KV_EINVAL, "num_tokens must be >= 0");
  if (flags & ~(INT2KV_HADAMARD_K | INT2KV_HADAMARD_V)) return fail(INT2KV_EINVAL, "unknown flags");
  if (num_tokens == 0) return ok();
  const bool had_k = flags & INT2KV_HADAMARD_K, had_v = flags & INT2KV_HADAMARD_V;
  if (!k || !v || !slot_mapping || !mu_rk || (!had_k && !R_k) || (!had_v && !R_v))
    return fail(INT2KV_EINVAL, "NULL pointer argument");
  if (positions && (!cos_sin || max_pos <= 0)) return fail(INT2KV_EINVAL, "RoPE needs cos_sin and max_pos > 0");
  if (k_rope_out && !positions) return fail(INT2KV_EINVAL, "k_rope_out needs positions");
  if (!valid_clip(clip_k) || !valid_clip(clip_v)) return fail(INT2KV_EINVAL, "clip ratios must be in (0, 1]");
  if (!aligned(k, 16) || !aligned(v, 16) || (!had_k && !aligned(R_k, 16)) || (!had_v && !aligned(R_v, 16)) ||
      !aligned(mu_rk, 16) || (cos_sin && !aligned(cos_sin, 16)) || (k_rope_out && !aligned(k_rope_out, 16)))
    return fail(INT2KV_EINVAL, "k, v, R_k, R_v, mu_rk, cos_sin and k_rope_out must be 16-byte aligned");
  AppendOptions o;
  o.positions = positions;
  o.cos_sin = positions ? cos_sin : nullptr;
  o.max_pos = positions ? max_pos : 0;
  o.k_rope_out = k_rope_out;
  o.hadamard = (had_k ? 1 : 0) | (had_v ? 2 : 0);
  hipError_t e = launch_append_mfma(view(cache), k, v, slot_mapping, num_tokens, had_k ? nullptr : R_k,
                                    had_v ? nullptr : R_v, mu_rk, clip_k, clip_v, stream, g_ev_before, g_ev_after,
                                    nullptr, &o);
  return hip_status(e, "quantize_append_rope");
}

int int2kv_quantize_append_error(const int2kv_cache* cache, const uint16_t* k, const uint16_t* v,
                                 const int32_t* slot_mapping, int num_tokens, const float* R_k, const float* R_v,
                                 const float* mu_rk, float clip_k, float clip_v, float* err, hipStream_t stream) {
  if (int st = check_cache(cache)) return st;
  if (num_tokens < 0) return fail(INT2KV_EINVAL, "num_tokens must be >= 0");
  if (num_tokens == 0) return ok();
  if (!k || !v || !slot_mapping || !R_k || !R_v || !mu_rk || !err) return fail(INT2KV_EINVAL, "NULL pointer argument");
  if (!valid_clip(clip_k) || !valid_clip(clip_v)) return fail(INT2KV_EINVAL, "clip ratios must be in (0, 1]");
  if (!aligned(k, 16) || !aligned(v, 16) || !aligned(R_k, 16) || !aligned(R_v, 16) || !aligned(mu_rk, 16))
    return fail(INT2KV_EINVAL, "k, v, R_k, R_v and mu_rk must be 16-byte aligned");
  if (!aligned(err, 4)) return fail(INT2KV_EINVAL, "err must be 4-byte aligned");
  hipError_t e = launch_append_mfma(view(cache), k, v, slot_mapping, num_tokens, R_k, R_v, mu_rk, clip_k, clip_v,
                                    stream, g_ev_before, g_ev_after, err);
  return hip_status(e, "quantize_append_error");
}

size_t int2kv_decode_workspace_bytes(int batch, int num_q_heads, int num_kv_heads, int max_ctx, int d_model) {
  if (batch <= 0 || num_q_heads <= 0 || num_kv_heads <= 0 || num_q_heads % num_kv_heads || max_ctx < 0 ||
      d_model < 0)
    return 0;
  // enough for either scan (the cache's group size picks one)
  const size_t a = make_plan(batch, num_q_heads, num_kv_heads, max_ctx, d_model, 4).total;
  const size_t b = make_plan(batch, num_q_heads, num_kv_heads, max_ctx, d_model, 1).total;
  return a > b ? a : b;
}

}  // extern "C"

namespace {

// Appends of at most this many tokens run inside the decode's preparation launch.
constexpr int kFusedAppendTokens = 256;

// The cache write of int2kv_append_decode: its arguments, validated, and whether there is one.
struct AppendStage {
  const uint16_t *k = nullptr, *v = nullptr;
  const int32_t* slots = nullptr;
  int n = 0;
  const float* mu_rk = nullptr;
  float clip_k = 1.0f, clip_v = 1.0f;
};

struct WindowStage {
  const uint16_t *k = nullptr, *v = nullptr;
  const int32_t* lens = nullptr;
  int cap = 0;
};

int decode_impl(const int2kv_cache* cache, const uint16_t* q, int batch, int num_q_heads,
                const int32_t* block_table, int max_blocks_per_seq, const int32_t* ctx_lens, int max_ctx,
                const float* R_k, const float* R_v, const uint16_t* W_o, int d_model, int wo_format, float* out,
                void* workspace, size_t workspace_bytes, hipStream_t stream, const AppendStage* ap,
                const WindowStage* win = nullptr) {
  if (int st = check_cache(cache)) return st;
  if (batch < 0) return fail(INT2KV_EINVAL, "batch must be >= 0");
  if (batch == 0) {
    if (!ap || ap->n == 0) return ok();
    return hip_status(launch_append_mfma(view(cache), ap->k, ap->v, ap->slots, ap->n, R_k, R_v, ap->mu_rk, ap->clip_k,
                                         ap->clip_v, stream),
                      "append_decode/append");
  }
  const int H = cache->num_kv_heads;
  if (num_q_heads <= 0 || num_q_heads % H) return fail(INT2KV_EINVAL, "num_q_heads must be a multiple of num_kv_heads");
  const int gq = num_q_heads / H;
  if (gq > 16) return fail(INT2KV_EUNSUPPORTED, "at most 16 query heads per KV head");
  if (max_blocks_per_seq <= 0 || max_ctx < 0) return fail(INT2KV_EINVAL, "bad max_blocks_per_seq / max_ctx");
  if (W_o && (wo_format < INT2KV_WO_PLAIN || wo_format > INT2KV_WO_PREPARED_FOLDED))
    return fail(INT2KV_EINVAL, "wo_format must be one of INT2KV_WO_*");
  const bool folded = W_o && (wo_format == INT2KV_WO_FOLDED || wo_format == INT2KV_WO_PREPARED_FOLDED);
  const bool prepared = W_o && wo_format >= INT2KV_WO_PREPARED;
  if (!q || !block_table || !ctx_lens || !R_k || !out || (!R_v && !folded))
    return fail(INT2KV_EINVAL, "NULL pointer argument");
  if (!aligned(q, 16) || !aligned(out, 16) || !aligned(R_k, 16) || (R_v && !aligned(R_v, 16)))
    return fail(INT2KV_EINVAL, "q, out, R_k and R_v must be 16-byte aligned");
  if (W_o) {
    if (d_model <= 0) return fail(INT2KV_EINVAL, "d_model must be positive when W_o is given");
    if (!aligned(W_o, 16)) return fail(INT2KV_EINVAL, "W_o must be 16-byte aligned");
  } else {
    d_model = 0;
  }
  const DecodePlan plan = make_plan(batch, num_q_heads, H, max_ctx, d_model, kHeadDim / cache->group_size);
  if (!workspace || workspace_bytes < plan.total)
    return fail(INT2KV_EWORKSPACE, "workspace smaller than int2kv_decode_workspace_bytes()");
  if (!aligned(workspace, 256)) return fail(INT2KV_EINVAL, "workspace must be 256-byte aligned");

  uint8_t* ws = static_cast<uint8_t*>(workspace);
  DecodeArgs a{};
  a.pool = static_cast<const uint8_t*>(cache->pool);
  a.num_blocks = cache->num_blocks;
  a.H = H;
  a.q = q;
  a.B = batch;
  a.Hq = num_q_heads;
  a.gq = gq;
  a.block_table = block_table;
  a.max_blocks = max_blocks_per_seq;
  a.ctx_lens = ctx_lens;
  a.max_ctx = max_ctx;
  a.R_k = R_k;
  a.R_v = R_v;
  a.qrot = reinterpret_cast<float*>(ws + plan.off_qrot);
  a.qop = ws + plan.off_qop;
  a.part = reinterpret_cast<float*>(ws + plan.off_part);
  a.s1 = plan.s1;
  a.part2 = plan.s1 ? reinterpret_cast<float*>(ws + plan.off_part2) : nullptr;
  a.chunk_tokens = plan.chunk_tokens;
  a.n_chunks = plan.n_chunks;
  a.prefix = reinterpret_cast<int32_t*>(ws + plan.off_prefix);
  a.wg_info = reinterpret_cast<int32_t*>(ws + plan.off_wginfo);
  a.seq_wg = reinterpret_cast<int32_t*>(ws + plan.off_seqwg);
  a.pages = reinterpret_cast<uint32_t*>(ws + plan.off_pages);
  a.grid_g = plan.grid_g;
  a.groups = kHeadDim / cache->group_size;
  a.wpart = win ? reinterpret_cast<float*>(ws + plan.off_win) : nullptr;
  a.win_slices = win ? (win->cap + kWinSliceTokens - 1) / kWinSliceTokens : 0;

  hipError_t e = hipSuccess;
  // the cache write (int2kv_append_decode): a few tokens per sequence run as extra blocks of the
  // matrix-core preparation launch, beside the query preparation (which does not read the cache);
  // otherwise (long appends, vector-ALU decode) as its own launch first
  AppendArgs apa{};
  const bool fused_append = ap && ap->n > 0 && plan.variant == 2 && ap->n <= kFusedAppendTokens;
  if (ap && ap->n > 0) {
    apa = AppendArgs{view(cache), ap->k, ap->v, ap->slots, ap->n, R_k, R_v, ap->mu_rk, ap->clip_k, ap->clip_v, 0};
    if (!fused_append) {
      e = launch_append_mfma(view(cache), ap->k, ap->v, ap->slots, ap->n, R_k, R_v, ap->mu_rk, ap->clip_k, ap->clip_v,
                             stream);
      if (e != hipSuccess) return hip_status(e, "append_decode/append");
    }
  }
  if (plan.variant != 2) {
    e = launch_qrot(a, stream);
    if (e != hipSuccess) return hip_status(e, "decode/qrot");
  } else {
    e = launch_qprep(a, fused_append ? &apa : nullptr, stream);
    if (e != hipSuccess) return hip_status(e, "decode/qprep");
  }
  // the measurement events (if set) ride on the scan's own dispatch: they mark its start and end
  e = plan.variant == 2 ? launch_decode_split_mfma(a, stream, g_ev_before, g_ev_after)
                        : launch_decode_split_valu(a, stream, g_ev_before, g_ev_after);
  if (e != hipSuccess) return hip_status(e, "decode/split");
  if (win) {
    e = launch_window_attn(a, WindowArgs{win->k, win->v, win->lens, win->cap}, stream);
    if (e != hipSuccess) return hip_status(e, "decode/window");
  }
  const bool unrotate = !folded;
  // with W_O the merge writes each head output as the projection's operand: two bf16 terms (hi, lo)
  // for row-major bf16 weights, one fp16 term for prepared weights
  uint16_t* ob = W_o ? reinterpret_cast<uint16_t*>(ws + plan.off_o) : nullptr;
  const int fmt = !W_o ? kOutF32 : (prepared ? kOutF16 : kOutBf16x2);
  e = plan.variant == 2 ? launch_merge_flat(a, unrotate, out, ob, fmt, stream)
                        : launch_merge(a, unrotate, out, ob, fmt, stream);
  if (e != hipSuccess) return hip_status(e, "decode/merge");
  if (W_o) {
    e = launch_wo_gemm(ob, W_o, prepared, out, reinterpret_cast<float*>(ws + plan.off_wo), batch,
                       num_q_heads * kHeadDim, d_model, plan.wo_ksplit, stream);
    if (e != hipSuccess) return hip_status(e, "decode/wo");
  }
  return ok();
}

}  // namespace

extern "C" {

int int2kv_decode(const int2kv_cache* cache, const uint16_t* q, int batch, int num_q_heads,
                  const int32_t* block_table, int max_blocks_per_seq, const int32_t* ctx_lens, int max_ctx,
                  const float* R_k, const float* R_v, const uint16_t* W_o, int d_model, int wo_format, float* out,
                  void* workspace, size_t workspace_bytes, hipStream_t stream) {
  return decode_impl(cache, q, batch, num_q_heads, block_table, max_blocks_per_seq, ctx_lens, max_ctx, R_k, R_v, W_o,
                     d_model, wo_format, out, workspace, workspace_bytes, stream, nullptr);
}

int int2kv_append_decode(const int2kv_cache* cache, const uint16_t* k, const uint16_t* v, const int32_t* slot_mapping,
                         int num_tokens, const float* mu_rk, float clip_k, float clip_v, const uint16_t* q, int batch,
                         int num_q_heads, const int32_t* block_table, int max_blocks_per_seq, const int32_t* ctx_lens,
                         int max_ctx, const float* R_k, const float* R_v, const uint16_t* W_o, int d_model,
                         int wo_format, float* out, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (int st = check_cache(cache)) return st;
  if (num_tokens < 0) return fail(INT2KV_EINVAL, "num_tokens must be >= 0");
  AppendStage ap;
  if (num_tokens > 0) {
    if (!k || !v || !slot_mapping || !R_k || !R_v || !mu_rk) return fail(INT2KV_EINVAL, "NULL pointer argument");
    if (!valid_clip(clip_k) || !valid_clip(clip_v)) return fail(INT2KV_EINVAL, "clip ratios must be in (0, 1]");
    if (!aligned(k, 16) || !aligned(v, 16) || !aligned(R_k, 16) || !aligned(R_v, 16) || !aligned(mu_rk, 16))
      return fail(INT2KV_EINVAL, "k, v, R_k, R_v and mu_rk must be 16-byte aligned");
    ap = AppendStage{k, v, slot_mapping, num_tokens, mu_rk, clip_k, clip_v};
  }
  return decode_impl(cache, q, batch, num_q_heads, block_table, max_blocks_per_seq, ctx_lens, max_ctx, R_k, R_v, W_o,
                     d_model, wo_format, out, workspace, workspace_bytes, stream, &ap);
}

int int2kv_append_decode_noalloc(const int2kv_cache* cache, const uint16_t* k, const uint16_t* v,
                                 const int32_t* slot_mapping, int num_tokens, const float* mu_rk, float clip_k,
                                 float clip_v, const uint16_t* q, int batch, int num_q_heads,
                                 const int32_t* block_table, int max_blocks_per_seq, const int32_t* ctx_lens,
                                 int max_ctx, const float* R_k, const float* R_v, const uint16_t* W_o, int d_model,
                                 int wo_format, float* out, hipStream_t stream) {
  if (int st = check_cache(cache)) return st;
  // the workspace this call needs must fit the static scratch (checked before any HIP call)
  const int H = cache->num_kv_heads;
  const int dm = W_o ? d_model : 0;
  if (batch > 0 && num_q_heads > 0 && num_q_heads % H == 0 && max_ctx >= 0 && dm >= 0) {
    const size_t need = make_plan(batch, num_q_heads, H, max_ctx, dm, kHeadDim / cache->group_size).total;
    if (need > kScratchBytes)
      return fail(INT2KV_EWORKSPACE, "this decode needs " + std::to_string(need) +
                                         " bytes of workspace, more than the static scratch holds (" +
                                         std::to_string(kScratchBytes) + "); use int2kv_append_decode");
  }
  void* ws = nullptr;
  if (int st = scratch_for_current_device(&ws)) return st;
  return int2kv_append_decode(cache, k, v, slot_mapping, num_tokens, mu_rk, clip_k, clip_v, q, batch, num_q_heads,
                              block_table, max_blocks_per_seq, ctx_lens, max_ctx, R_k, R_v, W_o, d_model, wo_format,
                              out, ws, kScratchBytes, stream);
}

int int2kv_decode_window(const int2kv_cache* cache, const uint16_t* q, int batch, int num_q_heads,
                         const int32_t* block_table, int max_blocks_per_seq, const int32_t* ctx_lens, int max_ctx,
                         const float* R_k, const float* R_v, const uint16_t* W_o, int d_model, int wo_format,
                         const uint16_t* win_k, const uint16_t* win_v, const int32_t* win_lens, int win_cap,
                         float* out, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (int st = check_cache(cache)) return st;
  if (!win_k || !win_v || !win_lens || !R_v) return fail(INT2KV_EINVAL, "NULL pointer argument");
  if (win_cap <= 0 || win_cap > kWinMaxCap) return fail(INT2KV_EINVAL, "win_cap must be in [1, 512]");
  if (!aligned(win_k, 16) || !aligned(win_v, 16)) return fail(INT2KV_EINVAL, "win_k and win_v must be 16-byte aligned");
  const WindowStage ws{win_k, win_v, win_lens, win_cap};
  return decode_impl(cache, q, batch, num_q_heads, block_table, max_blocks_per_seq, ctx_lens, max_ctx, R_k, R_v, W_o,
                     d_model, wo_format, out, workspace, workspace_bytes, stream, nullptr, &ws);
}

int int2kv_window_write(const uint16_t* k, const uint16_t* v, const int32_t* rows, int num_tokens, int num_kv_heads,
                        const float* mu, uint16_t* win_k, uint16_t* win_v, int num_rows, hipStream_t stream) {
  if (num_tokens < 0 || num_kv_heads <= 0 || num_rows < 0)
    return fail(INT2KV_EINVAL, "num_tokens, num_rows must be >= 0 and num_kv_heads > 0");
  if (num_tokens == 0) return ok();
  if (!k || !v || !rows || !mu || !win_k || !win_v) return fail(INT2KV_EINVAL, "NULL pointer argument");
  if (!aligned(k, 16) || !aligned(v, 16) || !aligned(mu, 16) || !aligned(win_k, 16) || !aligned(win_v, 16))
    return fail(INT2KV_EINVAL, "k, v, mu, win_k and win_v must be 16-byte aligned");
  return hip_status(launch_window_write(k, v, rows, num_tokens, num_kv_heads, mu, win_k, win_v, num_rows, stream),
                    "window_write");
}

}  // extern "C"

namespace {

// Workspace of int2kv_output_error: q R_K, the chunk partials, the output differences, the partial
// statistics of each W_O row tile; chunk as the vector-ALU decode's automatic choice.
struct OePlan {
  int chunk, n_chunks, ntiles;
  size_t off_qrot, off_part, off_dov, off_spart, total;
};

OePlan make_oe_plan(int B, int Hq, int H, int max_ctx, int d_model) {
  OePlan p{};
  int chunk = 4096;
  const long long units = (long long)B * H;
  while (chunk > 512 && units * ((max_ctx + chunk - 1) / chunk) < 1024) chunk /= 2;
  p.chunk = chunk;
  p.n_chunks = max_ctx > 0 ? (max_ctx + chunk - 1) / chunk : 1;
  p.ntiles = (d_model + kOeRowTile - 1) / kOeRowTile;
  auto up = [](size_t x) { return (x + 255) & ~size_t(255); };
  size_t off = 0;
  p.off_qrot = off;
  off = up(off + (size_t)B * Hq * kHeadDim * sizeof(float));
  p.off_part = off;
  off = up(off + (size_t)B * p.n_chunks * Hq * kOePartStride * sizeof(float));
  p.off_dov = off;
  off = up(off + 3 * (size_t)B * Hq * 2 * kHeadDim * sizeof(uint16_t));
  p.off_spart = off;
  off = up(off + (size_t)B * Hq * p.ntiles * 4 * sizeof(float));
  p.total = off;
  return p;
}

}  // namespace

extern "C" {

size_t int2kv_output_error_workspace_bytes(int batch, int num_q_heads, int num_kv_heads, int max_ctx, int d_model) {
  if (batch <= 0 || num_q_heads <= 0 || num_kv_heads <= 0 || num_q_heads % num_kv_heads || max_ctx < 0 ||
      d_model <= 0)
    return 0;
  return make_oe_plan(batch, num_q_heads, num_kv_heads, max_ctx, d_model).total;
}

int int2kv_output_error(const int2kv_cache* cache, const uint16_t* q, int batch, int num_q_heads,
                        const int32_t* block_table, int max_blocks_per_seq, const int32_t* ctx_lens, int max_ctx,
                        const float* R_k, const float* R_v, const uint16_t* k_rows, const uint16_t* v_rows,
                        int row_cap, const uint16_t* W_o, int d_model, float* stats, float* dy, void* workspace,
                        size_t workspace_bytes, hipStream_t stream) {
  if (int st = check_cache(cache)) return st;
  if (batch <= 0 || batch > 65535) return fail(INT2KV_EINVAL, "batch must be in [1, 65535]");
  const int H = cache->num_kv_heads;
  if (num_q_heads <= 0 || num_q_heads % H) return fail(INT2KV_EINVAL, "num_q_heads must be a multiple of num_kv_heads");
  const int gq = num_q_heads / H;
  if (gq > 16) return fail(INT2KV_EUNSUPPORTED, "at most 16 query heads per KV head");
  if (max_blocks_per_seq <= 0 || max_ctx < 0 || row_cap <= 0 || d_model <= 0)
    return fail(INT2KV_EINVAL, "bad max_blocks_per_seq / max_ctx / row_cap / d_model");
  if (!q || !block_table || !ctx_lens || !R_k || !R_v || !k_rows || !v_rows || !W_o || !stats)
    return fail(INT2KV_EINVAL, "NULL pointer argument");
  if (!aligned(q, 16) || !aligned(R_k, 16) || !aligned(R_v, 16) || !aligned(k_rows, 16) || !aligned(v_rows, 16) ||
      !aligned(W_o, 16) || !aligned(stats, 16) || (dy && !aligned(dy, 16)))
    return fail(INT2KV_EINVAL, "q, R_k, R_v, k_rows, v_rows, W_o, stats and dy must be 16-byte aligned");
  const OePlan plan = make_oe_plan(batch, num_q_heads, H, max_ctx, d_model);
  if (!workspace || workspace_bytes < plan.total)
    return fail(INT2KV_EWORKSPACE, "workspace smaller than int2kv_output_error_workspace_bytes()");
  if (!aligned(workspace, 256)) return fail(INT2KV_EINVAL, "workspace must be 256-byte aligned");
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  OutErrArgs e{};
  DecodeArgs& a = e.a;
  a.pool = static_cast<const uint8_t*>(cache->pool);
  a.num_blocks = cache->num_blocks;
  a.H = H;
  a.q = q;
  a.B = batch;
  a.Hq = num_q_heads;
  a.gq = gq;
  a.block_table = block_table;
  a.max_blocks = max_blocks_per_seq;
  a.ctx_lens = ctx_lens;
  a.max_ctx = max_ctx;
  a.R_k = R_k;
  a.R_v = R_v;
  a.qrot = reinterpret_cast<float*>(ws + plan.off_qrot);
  a.chunk_tokens = plan.chunk;
  a.n_chunks = plan.n_chunks;
  a.groups = kHeadDim / cache->group_size;
  e.k_rows = k_rows;
  e.v_rows = v_rows;
  e.row_cap = row_cap;
  e.part = reinterpret_cast<float*>(ws + plan.off_part);
  e.dov = reinterpret_cast<uint16_t*>(ws + plan.off_dov);
  e.spart = reinterpret_cast<float*>(ws + plan.off_spart);
  return hip_status(launch_output_error(e, W_o, d_model, stats, dy, stream, g_ev_before, g_ev_after), "output_error");
}

}  // extern "C"

// ---- OptR offline calibration
namespace {

struct OptrLayout {
  size_t shared, set_c, set_h, state, total;
};

struct SetDims {
  int T = 0, nseq = 0, nrows = 0;
  long long pel = 0;
};

int check_traces(const int2kv_optr_traces* t, const int2kv_optr_config* c, SetDims& d, const char* what) {
  if (!t || !t->k || !t->v || !t->q || !t->seq_starts || t->num_seqs <= 0)
    return fail(INT2KV_EINVAL, std::string(what) + ": NULL pointer or no sequences");
  if (t->seq_starts[0] != 0) return fail(INT2KV_EINVAL, std::string(what) + ": seq_starts[0] must be 0");
  const int gq = c->num_q_heads / c->num_kv_heads;
  d = SetDims{};
  for (int i = 0; i < t->num_seqs; ++i) {
    const int len = t->seq_starts[i + 1] - t->seq_starts[i];
    if (len < 0 || len > kCalMaxLen)
      return fail(INT2KV_EINVAL, std::string(what) + ": sequence lengths must be in [0, 4096]");
    const int rows = (len < c->n_last ? len : c->n_last) * gq;
    d.nrows += rows;
    d.pel += (long long)rows * len;
  }
  d.T = t->seq_starts[t->num_seqs];
  d.nseq = t->num_seqs;
  if (!aligned(t->k, 16) || !aligned(t->v, 16)) return fail(INT2KV_EINVAL, std::string(what) + ": k, v must be 16-byte aligned");
  return INT2KV_OK;
}

int check_config(const int2kv_optr_config* c) {
  if (!c) return fail(INT2KV_EINVAL, "config is NULL");
  if (c->num_kv_heads <= 0 || c->num_q_heads <= 0 || c->num_q_heads % c->num_kv_heads)
    return fail(INT2KV_EINVAL, "num_q_heads must be a positive multiple of num_kv_heads");
  if (c->num_q_heads / c->num_kv_heads > 16) return fail(INT2KV_EUNSUPPORTED, "at most 16 query heads per KV head");
  if (c->d_model <= 0) return fail(INT2KV_EINVAL, "d_model must be positive");
  if (c->group_size != 32 && c->group_size != 128) return fail(INT2KV_EUNSUPPORTED, "group_size must be 32 or 128");
  if (!valid_clip(c->clip_k) || !valid_clip(c->clip_v)) return fail(INT2KV_EINVAL, "clip ratios must be in (0, 1]");
  if (c->n_last <= 0 || c->sink < 0 || c->recent < 0) return fail(INT2KV_EINVAL, "bad n_last / sink / recent");
  if (c->steps < 0 || c->eval_every <= 0 || !(c->lr > 0.0) || !(c->lambda_k >= 0.0)) return fail(INT2KV_EINVAL, "bad steps / eval_every / lr");
  return INT2KV_OK;
}

OptrLayout optr_layout(const int2kv_optr_config* c, const SetDims& dc, const SetDims* dh) {
  OptrLayout L{};
  const int H = c->num_kv_heads;
  L.shared = cal_shared_bytes(H, c->num_q_heads);
  L.set_c = cal_set_bytes(dc.T, dc.nseq, dc.nrows, dc.pel, H);
  L.set_h = dh ? cal_set_bytes(dh->T, dh->nseq, dh->nrows, dh->pel, H) : 0;
  // optimizer state: A, A_best, m, v, grad ([H, 128, 128] each), best loss and loss ([H] each)
  L.state = 5 * (size_t)H * kHeadDim * kHeadDim * 8 + 2 * 256 + 2 * (size_t)H * 8;
  L.total = L.shared + L.set_c + L.set_h + L.state + 1024;
  return L;
}

CalCfg make_cal_cfg(const int2kv_optr_config* c, const float* mu, const float* R0k, const float* R0v) {
  CalCfg g{};
  g.H = c->num_kv_heads;
  g.Hq = c->num_q_heads;
  g.gq = g.Hq / g.H;
  g.dm = c->d_model;
  g.ng = kHeadDim / c->group_size;
  g.clip_k = c->clip_k;
  g.clip_v = c->clip_v;
  g.lam = c->lambda_k;
  g.sink = c->sink;
  g.recent = c->recent;
  g.n_last = c->n_last;
  g.mu = mu;
  g.R0k = R0k;
  g.R0v = R0v;
  return g;
}

uint8_t* align256(void* p) {
  return reinterpret_cast<uint8_t*>((reinterpret_cast<uintptr_t>(p) + 255) & ~uintptr_t(255));
}

}  // namespace

extern "C" {

size_t int2kv_optr_workspace_bytes(const int2kv_optr_config* cfg, const int2kv_optr_traces* calib,
                                   const int2kv_optr_traces* heldout) {
  if (check_config(cfg)) return 0;
  SetDims dc, dh;
  if (check_traces(calib, cfg, dc, "calib")) return 0;
  if (heldout && check_traces(heldout, cfg, dh, "heldout")) return 0;
  return optr_layout(cfg, dc, heldout ? &dh : nullptr).total;
}

int int2kv_optr_key_mean(const uint16_t* k, int num_tokens, int num_kv_heads, float* mu, hipStream_t stream) {
  if (!k || !mu || num_tokens <= 0 || num_kv_heads <= 0) return fail(INT2KV_EINVAL, "bad key-mean arguments");
  return hip_status(cal_key_mean(k, num_tokens, num_kv_heads, mu, stream), "optr_key_mean");
}

// Shared front part of the loss entry points: validation, layout, the set and the Gram matrices.
static int optr_setup(const int2kv_optr_config* cfg, const int2kv_optr_traces* tr, const float* mu,
                      const float* R0_k, const float* R0_v, const uint16_t* W_o, void* workspace,
                      size_t workspace_bytes, hipStream_t stream, CalCfg& g, CalSet& set, uint8_t*& state) {
  if (int st = check_config(cfg)) return st;
  SetDims d;
  if (int st = check_traces(tr, cfg, d, "traces")) return st;
  if (!mu || !R0_k || !R0_v || !W_o) return fail(INT2KV_EINVAL, "NULL pointer argument");
  const OptrLayout L = optr_layout(cfg, d, nullptr);
  if (!workspace || workspace_bytes < L.total) return fail(INT2KV_EWORKSPACE, "workspace smaller than int2kv_optr_workspace_bytes()");
  uint8_t* base = align256(workspace);
  g = make_cal_cfg(cfg, mu, R0_k, R0_v);
  cal_bind_shared(g, base);
  hipError_t e = cal_bind_set(set, base + L.shared, tr->k, tr->v, tr->q, tr->seq_starts, tr->num_seqs, g.H, g.gq,
                              g.n_last, stream);
  if (e == hipSuccess) e = cal_gram(g, W_o, stream);
  if (e == hipSuccess) e = cal_prepare_set(g, set, stream);
  state = base + L.shared + L.set_c;
  return hip_status(e, "optr setup");
}

int int2kv_optr_key_loss(const int2kv_optr_config* cfg, const int2kv_optr_traces* traces, const float* R0_k,
                         const float* mu, const uint16_t* W_o, const double* A, double* loss, double* grad,
                         void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (!A || !loss) return fail(INT2KV_EINVAL, "NULL pointer argument");
  CalCfg g;
  CalSet set;
  uint8_t* state;
  if (int st = optr_setup(cfg, traces, mu, R0_k, R0_k, W_o, workspace, workspace_bytes, stream, g, set, state)) return st;
  return hip_status(cal_key_loss(g, set, A, loss, grad, stream), "optr_key_loss");
}

int int2kv_optr_value_loss(const int2kv_optr_config* cfg, const int2kv_optr_traces* traces, const float* R0_k,
                           const double* A_k, const float* mu, const float* R0_v, const uint16_t* W_o,
                           const double* A_v, double* loss, double* grad, void* workspace, size_t workspace_bytes,
                           hipStream_t stream) {
  if (!A_k || !A_v || !loss) return fail(INT2KV_EINVAL, "NULL pointer argument");
  CalCfg g;
  CalSet set;
  uint8_t* state;
  if (int st = optr_setup(cfg, traces, mu, R0_k, R0_v, W_o, workspace, workspace_bytes, stream, g, set, state)) return st;
  hipError_t e = cal_key_probs(g, set, A_k, stream);
  if (e == hipSuccess) e = cal_value_loss(g, set, A_v, loss, grad, stream);
  return hip_status(e, "optr_value_loss");
}

int int2kv_optr_calibrate(const int2kv_optr_config* cfg, const int2kv_optr_traces* calib,
                          const int2kv_optr_traces* heldout, const float* R0_k, const float* R0_v, const float* mu,
                          const uint16_t* W_o, float* R_k, float* R_v, double* A_k, double* A_v, double* history,
                          void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (int st = check_config(cfg)) return st;
  SetDims dc, dh;
  if (int st = check_traces(calib, cfg, dc, "calib")) return st;
  if (int st = check_traces(heldout, cfg, dh, "heldout")) return st;
  if (!mu || !R0_k || !R0_v || !W_o || !R_k || !R_v) return fail(INT2KV_EINVAL, "NULL pointer argument");
  if (!aligned(R_k, 16) || !aligned(R_v, 16)) return fail(INT2KV_EINVAL, "R_k and R_v must be 16-byte aligned");
  const OptrLayout L = optr_layout(cfg, dc, &dh);
  if (!workspace || workspace_bytes < L.total) return fail(INT2KV_EWORKSPACE, "workspace smaller than int2kv_optr_workspace_bytes()");
  uint8_t* base = align256(workspace);
  CalCfg g = make_cal_cfg(cfg, mu, R0_k, R0_v);
  cal_bind_shared(g, base);
  CalSet sc, sh;
  hipError_t e = cal_bind_set(sc, base + L.shared, calib->k, calib->v, calib->q, calib->seq_starts, calib->num_seqs,
                              g.H, g.gq, g.n_last, stream);
  if (e == hipSuccess)
    e = cal_bind_set(sh, base + L.shared + L.set_c, heldout->k, heldout->v, heldout->q, heldout->seq_starts,
                     heldout->num_seqs, g.H, g.gq, g.n_last, stream);
  if (e == hipSuccess) e = cal_gram(g, W_o, stream);
  if (e == hipSuccess) e = cal_prepare_set(g, sc, stream);
  if (e == hipSuccess) e = cal_prepare_set(g, sh, stream);
  if (e != hipSuccess) return hip_status(e, "optr_calibrate setup");
  const size_t nA = (size_t)g.H * kHeadDim * kHeadDim;
  double* st = reinterpret_cast<double*>(base + L.shared + L.set_c + L.set_h);
  double *A = st, *Abest = st + nA, *m = st + 2 * nA, *v = st + 3 * nA, *gr = st + 4 * nA;
  double *best = st + 5 * nA, *loss = best + g.H;
  const int steps = cfg->steps, ev = cfg->eval_every, n_eval = 1 + steps / ev, hstride = steps + n_eval;
  auto record = [&](int phase, int idx) {
    return history ? cal_record(loss, history + (size_t)phase * g.H * hstride + idx, hstride, g.H, stream)
                   : hipSuccess;
  };
  for (int phase = 0; phase < 2 && e == hipSuccess; ++phase) {
    const bool value = phase == 1;
    auto eval = [&](CalSet& set, double* gradp) {
      return value ? cal_value_loss(g, set, A, loss, gradp, stream) : cal_key_loss(g, set, A, loss, gradp, stream);
    };
    if (value) {  // the selected key rotation's probabilities on both sets
      e = cal_key_probs(g, sc, A_k ? A_k : Abest, stream);
      if (e == hipSuccess) e = cal_key_probs(g, sh, A_k ? A_k : Abest, stream);
    }
    if (e == hipSuccess) e = cal_fill(A, 4 * nA, 0.0, stream);  // A, A_best, m, v
    if (e == hipSuccess) e = cal_fill(best, g.H, INFINITY, stream);
    if (e == hipSuccess) e = eval(sh, nullptr);
    if (e == hipSuccess) e = record(phase, steps);
    if (e == hipSuccess) e = cal_select(A, loss, best, Abest, g.H, stream);
    for (int i = 1; i <= steps && e == hipSuccess; ++i) {
      e = eval(sc, gr);
      if (e == hipSuccess) e = record(phase, i - 1);
      if (e == hipSuccess) e = cal_adam(A, gr, m, v, (int)nA, i, cfg->lr, stream);
      if (e == hipSuccess && i % ev == 0) {
        e = eval(sh, nullptr);
        if (e == hipSuccess) e = record(phase, steps + i / ev);
        if (e == hipSuccess) e = cal_select(A, loss, best, Abest, g.H, stream);
      }
    }
    if (e != hipSuccess) break;
    if (!value) {
      e = cal_rotation_out(g, Abest, false, R_k, stream);
      // the value phase reads the selected key generator from A_best before resetting it
      if (e == hipSuccess && A_k)
        e = hipMemcpyAsync(A_k, Abest, nA * sizeof(double), hipMemcpyDeviceToDevice, stream);
    } else {
      e = cal_rotation_out(g, Abest, true, R_v, stream);
      if (e == hipSuccess && A_v)
        e = hipMemcpyAsync(A_v, Abest, nA * sizeof(double), hipMemcpyDeviceToDevice, stream);
    }
  }
  return hip_status(e, "optr_calibrate");
}

}  // extern "C"
