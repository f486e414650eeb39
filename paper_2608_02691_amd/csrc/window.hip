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

// Window attention. The window of every sequence is cut into slices of kWinSliceTokens tokens; a
// block covers one slice of one sequence for eight KV heads, wave w taking KV head w, so the block
// reads the slice's rows whole (a token's eight head rows are one contiguous 2 KiB span) and every
// wave writes the (m, l, o) partial of its (sequence, KV head, slice) with no exchange between waves.
// Up to kWinMaxGq query heads and kWinMaxCap window tokens. A wave runs its slice in passes of
// kWinPass tokens:
//  * scores on the matrix cores: S[j][t] = q_j . k_t over the 128 channels, one 16 x 16 x 32 bf16
//    product per 16 tokens and 32 channels (query rows are the A operand, 16 bytes of each key row
//    per lane the B operand; bf16 products are exact, fp32 accumulation), in the scan's base-2 units;
//  * online softmax over the passes (row maxima and sums over the 16 lanes of a DPP row);
//  * o_j = sum_t p_jt v_t on the vector ALU: lane l owns channels 2l, 2l + 1 (one 4-byte load per
//    value row, so each row is read by the wave in one coalesced 256-byte access), p broadcast from
//    LDS.
// All of a pass's key and value loads are issued before its arithmetic. The partials are in the
// model's basis: the merges fold the slices of a (sequence, query head) into the INT2 result in the
// basis of the output (adding o after the INT2 part's un-rotation, or rotating o by R_V when the
// output projection is folded with R_V).
constexpr int kWinPass = 32;  // tokens per pass of a wave (two 16-token tiles)
constexpr int kWinTiles = kWinPass / 16;
constexpr int kWinWaves = 8;  // KV heads per block
static_assert(kWinSliceTokens % kWinPass == 0 && kWinMaxSlices * kWinSliceTokens >= kWinMaxCap, "window slices");

typedef __bf16 win_bf16x8_t __attribute__((ext_vector_type(8)));
typedef float win_f4_t __attribute__((ext_vector_type(4)));

// LDS of a block: p[t][j] of each wave's current pass (the 16 rows of the score tile) and the rescale
// factor of each row's running sums
struct WinLds {
  float p[kWinWaves][kWinPass][kWinMaxGq];
  float alpha[kWinWaves][kWinMaxGq];
};

// One wave: KV head h of sequence b, window slice `slice`. NJ4 = ceil(gq / 4): groups of four query
// rows the arithmetic covers (rows >= gq are zero).
template <int NJ4>
__device__ void window_wave(const DecodeArgs& a, const WindowArgs& w, int b, int h, int slice, int wave, int l,
                            WinLds& L) {
  constexpr int NJ = 4 * NJ4;
  const int lo = l & 15, hi = l >> 4;
  const int gq = a.gq, H = a.H;
  const int W = min(max(w.lens[b], 0), w.cap);
  const int t0 = min(W, slice * kWinSliceTokens), t1 = min(W, t0 + kWinSliceTokens);
  const size_t row_stride = (size_t)H * kHeadDim;  // elements between consecutive window rows
  const uint16_t* kbase = w.k + ((size_t)b * w.cap * H + h) * kHeadDim;
  const uint16_t* vbase = w.v + ((size_t)b * w.cap * H + h) * kHeadDim;
  float run_m[4], run_l[4];  // rows 4 hi + i (lanes of a DPP row agree)
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    run_m[i] = -INFINITY;
    run_l[i] = 0.0f;
  }
  float oacc[NJ][2];
#pragma unroll
  for (int j = 0; j < NJ; ++j) oacc[j][0] = oacc[j][1] = 0.0f;
  for (int p0 = t0; p0 < t1; p0 += kWinPass) {
    const int nt = min(kWinPass, t1 - p0);
    // every key and value load of the pass first (tokens past the slice read the window's last
    // row and get p = 0), then the query operand
    win_bf16x8_t kr[kWinTiles][4];
#pragma unroll
    for (int u = 0; u < kWinTiles; ++u) {
      const int t = min(p0 + 16 * u + lo, W - 1);
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
        kr[u][ks] = *reinterpret_cast<const win_bf16x8_t*>(kbase + (size_t)t * row_stride + 32 * ks + 8 * hi);
    }
    uint32_t vr[kWinPass];
#pragma unroll
    for (int i = 0; i < kWinPass; ++i)
      vr[i] = *reinterpret_cast<const uint32_t*>(vbase + (size_t)min(p0 + i, W - 1) * row_stride + 2 * l);
    // query operand: lane (row lo, k block hi) holds q_lo[32 ks + 8 hi .. + 7]; rows >= gq are zero
    win_bf16x8_t qa[4];
    {
      const int j = min(lo, gq - 1);
      const uint16_t* qr = a.q + ((size_t)b * a.Hq + h * gq + j) * kHeadDim + 8 * hi;
      const uint32_t keep = lo < gq ? ~0u : 0u;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const uint4 v = *reinterpret_cast<const uint4*>(qr + 32 * ks);
        qa[ks] = __builtin_bit_cast(win_bf16x8_t, make_uint4(v.x & keep, v.y & keep, v.z & keep, v.w & keep));
      }
    }
    // scores of rows 4 hi + r for token 16 u + lo of the pass, base-2 units, -inf past the slice
    float sc[kWinTiles][4];
#pragma unroll
    for (int u = 0; u < kWinTiles; ++u) {
      win_f4_t d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[ks], kr[u][ks], d, 0, 0, 0);
      const bool valid = 16 * u + lo < nt;
#pragma unroll
      for (int r = 0; r < 4; ++r) sc[u][r] = valid ? d[r] * kWinLogit2 : -INFINITY;
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float pm = sc[0][r];
#pragma unroll
      for (int u = 1; u < kWinTiles; ++u) pm = fmaxf(pm, sc[u][r]);
      pm = row_max16(pm);
      const float mnew = fmaxf(run_m[r], pm);  // pm is finite: the pass holds a valid token
      const float al = __builtin_amdgcn_exp2f(run_m[r] - mnew);
      float rs = 0.0f;
#pragma unroll
      for (int u = 0; u < kWinTiles; ++u) {
        const float p = __builtin_amdgcn_exp2f(sc[u][r] - mnew);
        rs += p;
        L.p[wave][16 * u + lo][4 * hi + r] = p;
      }
      run_l[r] = al * run_l[r] + row_sum16(rs);
      run_m[r] = mnew;
      if (lo == 0) L.alpha[wave][4 * hi + r] = al;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // o_j = alpha_j o_j + sum_t p_jt v_t on this lane's two channels (p = 0 past the slice)
#pragma unroll
    for (int j4 = 0; j4 < NJ4; ++j4) {
      const win_f4_t al = *reinterpret_cast<const win_f4_t*>(&L.alpha[wave][4 * j4]);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        oacc[4 * j4 + r][0] *= al[r];
        oacc[4 * j4 + r][1] *= al[r];
      }
    }
#pragma unroll
    for (int i = 0; i < kWinPass; ++i) {
      const float v0 = __uint_as_float(vr[i] << 16), v1 = __uint_as_float(vr[i] & 0xFFFF0000u);
#pragma unroll
      for (int j4 = 0; j4 < NJ4; ++j4) {
        const win_f4_t pt = *reinterpret_cast<const win_f4_t*>(&L.p[wave][i][4 * j4]);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          oacc[4 * j4 + r][0] = fmaf(pt[r], v0, oacc[4 * j4 + r][0]);
          oacc[4 * j4 + r][1] = fmaf(pt[r], v1, oacc[4 * j4 + r][1]);
        }
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
  // the partial of (b, h, slice): an empty slice leaves m = -inf, l = 0, o = 0
  float* wp = a.wpart + (((size_t)slice * a.B + b) * a.Hq + h * gq) * kPartStride;
#pragma unroll
  for (int j = 0; j < NJ; ++j)
    if (j < gq) *reinterpret_cast<float2*>(wp + (size_t)j * kPartStride + 4 + 2 * l) = make_float2(oacc[j][0], oacc[j][1]);
  if (lo == 0) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int j = 4 * hi + r;
      if (j < gq) {
        wp[(size_t)j * kPartStride] = run_m[r];
        wp[(size_t)j * kPartStride + 1] = run_l[r];
      }
    }
  }
}

// Block (window slice, sequence, group of eight KV heads); four waves per SIMD (registers <= 128).
template <int NJ4>
__global__ __launch_bounds__(64 * kWinWaves) __attribute__((amdgpu_waves_per_eu(4)))
void window_attn_kernel(DecodeArgs a, WindowArgs w) {
  __shared__ __attribute__((aligned(16))) WinLds lds;
  const int wave = threadIdx.x >> 6, h = blockIdx.z * kWinWaves + wave;
  if (h >= a.H) return;
  window_wave<NJ4>(a, w, blockIdx.y, h, blockIdx.x, wave, threadIdx.x & 63, lds);
}

hipError_t launch_window_attn(const DecodeArgs& a, const WindowArgs& w, hipStream_t s) {
  if (a.gq > kWinMaxGq || w.cap > kWinMaxCap) return hipErrorNotSupported;
  const dim3 grid(a.win_slices, a.B, (a.H + kWinWaves - 1) / kWinWaves), block(64 * kWinWaves);
  switch ((a.gq + 3) / 4) {
    case 1: hipLaunchKernelGGL(window_attn_kernel<1>, grid, block, 0, s, a, w); break;
    case 2: hipLaunchKernelGGL(window_attn_kernel<2>, grid, block, 0, s, a, w); break;
    case 3: hipLaunchKernelGGL(window_attn_kernel<3>, grid, block, 0, s, a, w); break;
    default: hipLaunchKernelGGL(window_attn_kernel<4>, grid, block, 0, s, a, w); break;
  }
  return hipGetLastError();
}

}  // namespace int2kv
