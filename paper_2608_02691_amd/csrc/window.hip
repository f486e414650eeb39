// BF16 sink and recent windows (Sec. 4.1; Sec. 5 implementation details): a few tokens per
// sequence (the paper keeps the first 64 and the last 256) skip INT2. Their keys keep the key
// centering and are held in BF16, their values are held unchanged. Decode attends to the union of
// the window tokens and the INT2 tokens under one softmax: the window kernel below writes one more
// partial (m, l, o') per (sequence, query head) in the scan's units, which the merge folds in.
//
// Window store: row r = b * cap + t holds token t of sequence b for every KV head,
// win[(r * H + h) * 128 + c] (bf16). Keys are bf16_rne(fp32(k - mu)) in the model's basis (R_K is
// orthogonal, so the scores equal those of the rotated, centered keys); values are v's bits.
#include "common.h"
#include "kernels.h"

namespace int2kv {

namespace {

constexpr float kWinLogit2 = 1.4426950408889634f * 0.08838834764831845f;  // log2(e)/sqrt(128)

__device__ __forceinline__ float bf_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf_hi(uint32_t u) { return __uint_as_float(u & 0xFFFF0000u); }
__device__ __forceinline__ uint32_t bf16_rne_bits(float x) {
  const uint32_t u = __float_as_uint(x);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

}  // namespace

// One thread per 8 channels of one (token, KV head).
__global__ __launch_bounds__(256) void window_write_kernel(const uint16_t* __restrict__ k,
                                                           const uint16_t* __restrict__ v,
                                                           const int32_t* __restrict__ rows, int n, int H,
                                                           const float* __restrict__ mu, uint16_t* __restrict__ win_k,
                                                           uint16_t* __restrict__ win_v, int num_rows) {
  const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long long)n * H * 16) return;
  const int i = (int)(idx / (H * 16));
  const int h = (int)(idx / 16 % H), c8 = (int)(idx % 16);
  const int r = rows[i];
  if (r < 0 || r >= num_rows) return;
  const size_t src = ((size_t)i * H + h) * kHeadDim + 8 * c8;
  const size_t dst = ((size_t)r * H + h) * kHeadDim + 8 * c8;
  const uint4 kk = *reinterpret_cast<const uint4*>(k + src);
  const float4 m0 = *reinterpret_cast<const float4*>(mu + (size_t)h * kHeadDim + 8 * c8);
  const float4 m1 = *reinterpret_cast<const float4*>(mu + (size_t)h * kHeadDim + 8 * c8 + 4);
  uint4 o;
  o.x = bf16_rne_bits(bf_lo(kk.x) - m0.x) | (bf16_rne_bits(bf_hi(kk.x) - m0.y) << 16);
  o.y = bf16_rne_bits(bf_lo(kk.y) - m0.z) | (bf16_rne_bits(bf_hi(kk.y) - m0.w) << 16);
  o.z = bf16_rne_bits(bf_lo(kk.z) - m1.x) | (bf16_rne_bits(bf_hi(kk.z) - m1.y) << 16);
  o.w = bf16_rne_bits(bf_lo(kk.w) - m1.z) | (bf16_rne_bits(bf_hi(kk.w) - m1.w) << 16);
  *reinterpret_cast<uint4*>(win_k + dst) = o;
  *reinterpret_cast<uint4*>(win_v + dst) = *reinterpret_cast<const uint4*>(v + src);
}

hipError_t launch_window_write(const uint16_t* k, const uint16_t* v, const int32_t* rows, int n, int H, const float* mu,
                               uint16_t* win_k, uint16_t* win_v, int num_rows, hipStream_t s) {
  const long long threads = (long long)n * H * 16;
  if (threads == 0) return hipSuccess;
  hipLaunchKernelGGL(window_write_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s, k, v, rows, n, H,
                     mu, win_k, win_v, num_rows);
  return hipGetLastError();
}

// Block (sequence b, KV head h), 256 threads, up to kWinMaxGq query heads and kWinMaxCap tokens.
// Scores: thread per token (its 256-byte key row against the group's queries, broadcast from
// LDS), in base-2 units as the scan's; softmax statistics: 16 lanes per query head; values:
// thread (channel, token parity); then o' = o R_V, the scan's value basis.
__global__ __launch_bounds__(256) void window_attn_kernel(DecodeArgs a, WindowArgs w) {
  __shared__ float qs[kWinMaxGq][kHeadDim];
  __shared__ float sc[kWinMaxGq][kWinMaxCap];
  __shared__ float ow[2][kWinMaxGq][kHeadDim];
  const int b = blockIdx.x, h = blockIdx.y, tid = threadIdx.x, gq = a.gq;
  const int W = min(max(w.lens[b], 0), w.cap);
  for (int i = tid; i < gq * kHeadDim; i += 256)
    qs[i / kHeadDim][i % kHeadDim] = __uint_as_float((uint32_t)a.q[((size_t)b * a.Hq + h * gq) * kHeadDim + i] << 16);
  __syncthreads();
  for (int t = tid; t < W; t += 256) {
    const uint4* kr = reinterpret_cast<const uint4*>(w.k + (((size_t)b * w.cap + t) * a.H + h) * kHeadDim);
    float acc[kWinMaxGq];
#pragma unroll
    for (int j = 0; j < kWinMaxGq; ++j) acc[j] = 0.0f;
    // the key row in four quarters: the four 16-byte loads of a quarter are issued before its
    // arithmetic (register arrays with static indices only, so nothing goes to scratch)
    for (int c32 = 0; c32 < kHeadDim / 32; ++c32) {
      uint4 row[4];
#pragma unroll
      for (int u4 = 0; u4 < 4; ++u4) row[u4] = kr[4 * c32 + u4];
#pragma unroll
      for (int u4 = 0; u4 < 4; ++u4) {
        const uint4 u = row[u4];
        const float kf[8] = {bf_lo(u.x), bf_hi(u.x), bf_lo(u.y), bf_hi(u.y),
                             bf_lo(u.z), bf_hi(u.z), bf_lo(u.w), bf_hi(u.w)};
        const int c0 = 32 * c32 + 8 * u4;
#pragma unroll
        for (int j = 0; j < kWinMaxGq; ++j) {
          if (j < gq) {
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[j] = fmaf(qs[j][c0 + e], kf[e], acc[j]);
          }
        }
      }
    }
#pragma unroll
    for (int j = 0; j < kWinMaxGq; ++j)
      if (j < gq) sc[j][t] = acc[j] * kWinLogit2;
  }
  __syncthreads();
  const int jr = tid >> 4, lr = tid & 15;
  float m = -INFINITY, l = 0.0f;
  if (jr < gq) {
    for (int t = lr; t < W; t += 16) m = fmaxf(m, sc[jr][t]);
#pragma unroll
    for (int o = 8; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 16));
    for (int t = lr; t < W; t += 16) {
      const float p = exp2f(sc[jr][t] - m);
      sc[jr][t] = p;
      l += p;
    }
#pragma unroll
    for (int o = 8; o > 0; o >>= 1) l += __shfl_xor(l, o, 16);
  }
  __syncthreads();
  const int c = tid & 127, par = tid >> 7;
  float o[kWinMaxGq];
#pragma unroll
  for (int j = 0; j < kWinMaxGq; ++j) o[j] = 0.0f;
  // unrolled so that several value loads are in flight per thread
#pragma unroll 8
  for (int t = par; t < W; t += 2) {
    const float vv = __uint_as_float((uint32_t)w.v[(((size_t)b * w.cap + t) * a.H + h) * kHeadDim + c] << 16);
#pragma unroll
    for (int j = 0; j < kWinMaxGq; ++j)
      if (j < gq) o[j] = fmaf(sc[j][t], vv, o[j]);
  }
#pragma unroll
  for (int j = 0; j < kWinMaxGq; ++j)
    if (j < gq) ow[par][j][c] = o[j];
  __syncthreads();
  for (int i = tid; i < gq * kHeadDim; i += 256) ow[0][i / kHeadDim][i % kHeadDim] += ow[1][i / kHeadDim][i % kHeadDim];
  __syncthreads();
  // o'[j][c] = sum_i o[j][i] R_V[i][c]: thread (c, par) for query heads par, par + 2, ...
  float acc[kWinMaxGq / 2];
#pragma unroll
  for (int r = 0; r < kWinMaxGq / 2; ++r) acc[r] = 0.0f;
  const float* Rv = a.R_v + (size_t)h * kHeadDim * kHeadDim;
#pragma unroll 16
  for (int i = 0; i < kHeadDim; ++i) {
    const float rv = Rv[(size_t)i * kHeadDim + c];
#pragma unroll
    for (int r = 0; r < kWinMaxGq / 2; ++r)
      if (par + 2 * r < gq) acc[r] = fmaf(ow[0][par + 2 * r][i], rv, acc[r]);
  }
#pragma unroll
  for (int r = 0; r < kWinMaxGq / 2; ++r) {
    const int j = par + 2 * r;
    if (j < gq) a.wpart[((size_t)b * a.Hq + h * gq + j) * kPartStride + 4 + c] = acc[r];
  }
  if (jr < gq && lr == 0) {
    float* pp = a.wpart + ((size_t)b * a.Hq + h * gq + jr) * kPartStride;
    pp[0] = W > 0 ? m : -INFINITY;
    pp[1] = l;
  }
}

hipError_t launch_window_attn(const DecodeArgs& a, const WindowArgs& w, hipStream_t s) {
  if (a.gq > kWinMaxGq || w.cap > kWinMaxCap) return hipErrorNotSupported;
  hipLaunchKernelGGL(window_attn_kernel, dim3(a.B, a.H), dim3(256), 0, s, a, w);
  return hipGetLastError();
}

}  // namespace int2kv
