// Output projection y = concat_j(o_j) W_O^T (eq:residual_readout; eq:int2_residual_readout).
// y: fp32 [B, N]; K = H_q * 128. Two weight formats:
//  * row-major bf16 W_O [N, K] as the model holds it (or folded by int2kv_fold_wo); o enters as two
//    bf16 terms (hi = bf16(o), lo = bf16(o - hi), written by the merge) so the product keeps
//    fp32-like precision (|o - hi - lo| <= 2^-16 |o|);
//  * prepared (int2kv_prepare_wo): fp16 weights stored tile by tile in the order the loads below
//    consume them, so every k step of a work-group reads one contiguous 8 KiB block; o enters as
//    one fp16 term (relative rounding <= 2^-11), which halves the o traffic and the MFMAs.
//
// Matrix-core GEMM, HBM-bound on the weights (read once). Work-group = 128 rows of W x one K slice
// x 64 batch rows, four waves of 32 rows. Every 32-wide k step of the weights and of o is staged in
// LDS with LDS-DMA loads (global_load_lds: lane i's 16 bytes land at M0 + 16 i), kWoStages - 1 steps
// ahead, with no registers held for data in flight; each lane fetches exactly the 16 bytes it later
// reads as its MFMA operand, so the LDS reads are conflict-free. The o tiles are shared by the four
// waves: each wave waits for its own DMA, then one barrier makes the whole step visible.
//
// K slices: each work-group writes its partial tile [slice][B][N]; a second kernel sums the slices
// in slice order (deterministic). With a single slice the GEMM writes y itself. (Letting the last
// work-group of a tile sum the slices needs a device-scope release in every work-group, i.e. an L2
// write-back per work-group, which measured slower than the second launch.)
#include "common.h"
#include "kernels.h"

namespace int2kv {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float wo_f4_t __attribute__((ext_vector_type(4)));

constexpr int kWoTileN = 128;  // rows of W (output columns) per work-group
constexpr int kWoBatch = 64;   // batch rows per work-group (four 16-column B tiles)
constexpr int kWoKStep = 32;
constexpr int kWoTileElems = kWoTileN * kWoKStep;  // one prepared tile: 128 rows x 32 k (8 KiB)

__device__ __forceinline__ void wo_dma(const void* base, uint32_t voff, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2" ::"s"(lds_addr), "v"(voff), "s"(base)
               : "memory", "m0");
}

#ifndef INT2KV_WO_PREP_STAGES
#define INT2KV_WO_PREP_STAGES 8
#endif
template <bool PREP>
struct WoCfg {
  static constexpr int kOTiles = PREP ? 4 : 8;                  // 1 KiB o tiles per step (terms x batch tiles)
  static constexpr int kStageBytes = 8192 + 1024 * kOTiles;     // W: 4 waves x 2 tiles x 1 KiB, then o
  static constexpr int kDmaPerStep = 2 + kOTiles / 4;           // DMA instructions per wave and step
  static constexpr int kStages = PREP ? INT2KV_WO_PREP_STAGES : 8;  // LDS stages; kStages - 1 steps in flight
};

template <bool PREP>
__global__ __launch_bounds__(256) void wo_mfma_kernel(const uint16_t* __restrict__ ob, const uint16_t* __restrict__ W,
                                                      float* __restrict__ partial, float* __restrict__ y, int B,
                                                      int K, int N, int slice, int ksplit) {
  using C = WoCfg<PREP>;
  constexpr int kWoStages = C::kStages;
  __shared__ __attribute__((aligned(16))) uint8_t stage[kWoStages][C::kStageBytes];
  const int n0 = blockIdx.x * kWoTileN, ks = blockIdx.y, b0 = blockIdx.z * kWoBatch;
  const int tid = threadIdx.x, w = __builtin_amdgcn_readfirstlane(tid >> 6), l = tid & 63;
  const int lo = l & 15, hi = l >> 4;
  const int k_begin = ks * slice;
  const int nsteps = (min(K, k_begin + slice) - k_begin) / kWoKStep;
  const int last = nsteps - 1;

  // Per-lane byte offsets (the step's k offset rides in the scalar base).
  // W tile a of this wave: rows n0 + 32 w + 16 a + lo, k + 8 hi
  uint32_t woff[2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
    woff[a] = PREP ? (uint32_t)((2 * w + a) * 1024 + 16 * l)
                   : (uint32_t)(((size_t)min(n0 + 32 * w + 16 * a + lo, N - 1) * K + 8 * hi) * 2);
  // o tile q of the work-group (q = w for one term; q = 2 w + u, term q / 4, batch tile q % 4 for two)
  constexpr int kOPerWave = C::kOTiles / 4;
  uint32_t ooff[kOPerWave];
#pragma unroll
  for (int u = 0; u < kOPerWave; ++u) {
    const int q = kOPerWave * w + u, term = q >> 2, t = q & 3;
    ooff[u] = (uint32_t)(((size_t)term * B * K + (size_t)min(b0 + 16 * t + lo, B - 1) * K + 8 * hi) * 2);
  }
  const uint16_t* wtile = W + (size_t)blockIdx.x * (K / kWoKStep) * kWoTileElems;  // prepared: this row block
  const uint32_t stage0 = (uint32_t)(uintptr_t)&stage[0][0];
  auto issue = [&](int s) {  // DMA of step min(s, last) into stage s % kWoStages
    const int sc = min(s, last);
    const uint32_t dst = stage0 + (uint32_t)((s % kWoStages) * C::kStageBytes);
    const int kk = k_begin + sc * kWoKStep;
    const uint16_t* wb = PREP ? wtile + (size_t)(kk / kWoKStep) * kWoTileElems : W + kk;
    const uint16_t* obb = ob + kk;
#pragma unroll
    for (int a = 0; a < 2; ++a) wo_dma(wb, woff[a], dst + (uint32_t)((2 * w + a) * 1024));
#pragma unroll
    for (int u = 0; u < kOPerWave; ++u) wo_dma(obb, ooff[u], dst + (uint32_t)(8192 + (kOPerWave * w + u) * 1024));
  };

  wo_f4_t acc[2][4];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int t = 0; t < 4; ++t) acc[a][t] = wo_f4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < kWoStages - 1; ++s) issue(s);
  for (int s = 0; s < nsteps; ++s) {
    // this wave's DMA of step s is done once at most (kWoStages - 2) younger steps are in flight;
    // the barrier then certifies every wave's DMA of step s, and that every wave has finished
    // reading step s - 1, whose stage is refilled right after
    asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"((kWoStages - 2) * C::kDmaPerStep) : "memory");
    issue(s + kWoStages - 1);
    const uint8_t* st = &stage[s % kWoStages][0];
    if constexpr (PREP) {
      f16x8_t A[2], Bt[4];
#pragma unroll
      for (int a = 0; a < 2; ++a) A[a] = *reinterpret_cast<const f16x8_t*>(st + (2 * w + a) * 1024 + 16 * l);
#pragma unroll
      for (int t = 0; t < 4; ++t) Bt[t] = *reinterpret_cast<const f16x8_t*>(st + 8192 + t * 1024 + 16 * l);
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int a = 0; a < 2; ++a) acc[a][t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(A[a], Bt[t], acc[a][t], 0, 0, 0);
    } else {
      bf16x8_t A[2], Bt[2][4];
#pragma unroll
      for (int a = 0; a < 2; ++a) A[a] = *reinterpret_cast<const bf16x8_t*>(st + (2 * w + a) * 1024 + 16 * l);
#pragma unroll
      for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int t = 0; t < 4; ++t)
          Bt[x][t] = *reinterpret_cast<const bf16x8_t*>(st + 8192 + (4 * x + t) * 1024 + 16 * l);
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int a = 0; a < 2; ++a) {
          acc[a][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A[a], Bt[0][t], acc[a][t], 0, 0, 0);
          acc[a][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A[a], Bt[1][t], acc[a][t], 0, 0, 0);
        }
    }
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // drain the clamped tail DMAs before exit
  // D[m][n] sits in lane n + 16 (m / 4), register m % 4: m = W row in the A tile, n = batch row; the
  // four registers are four consecutive output columns of one batch row. One slice writes y itself.
  float* dst_base = ksplit == 1 ? y : partial + (size_t)ks * B * N;
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int n = n0 + 32 * w + 16 * a + 4 * hi, b = b0 + 16 * t + lo;
      if (b >= B) continue;
      float* dst = dst_base + (size_t)b * N + n;
      if (n + 3 < N && (N & 3) == 0) {
        // non-temporal: the slices go out to memory now, while the weights stream, instead of staying
        // dirty in the caches until the next step's scan evicts them (measured: scan 3 us faster)
        __builtin_nontemporal_store(acc[a][t], reinterpret_cast<wo_f4_t*>(dst));
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (n + r < N) dst[r] = acc[a][t][r];
      }
    }
}

// y = sum over slices, in slice order, of partial[s] (B x N, fp32). Four consecutive elements per
// thread; the loads of all slices are issued before the sums (no load waits behind an add).
constexpr int kWoMaxUnroll = 8;
__global__ __launch_bounds__(256) void wo_reduce_kernel(const float* __restrict__ partial, float* __restrict__ y,
                                                         size_t total, int ksplit) {
  const size_t i = 4 * ((size_t)blockIdx.x * 256 + threadIdx.x);
  if (i >= total) return;
  if (i + 3 < total && (total & 3) == 0) {
    float4 sum = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int s0 = 0; s0 < ksplit; s0 += kWoMaxUnroll) {
      float4 p[kWoMaxUnroll];
#pragma unroll
      for (int u = 0; u < kWoMaxUnroll; ++u)
        if (s0 + u < ksplit) p[u] = *reinterpret_cast<const float4*>(partial + (size_t)(s0 + u) * total + i);
#pragma unroll
      for (int u = 0; u < kWoMaxUnroll; ++u)
        if (s0 + u < ksplit) {
          sum.x += p[u].x;
          sum.y += p[u].y;
          sum.z += p[u].z;
          sum.w += p[u].w;
        }
    }
    *reinterpret_cast<float4*>(y + i) = sum;
  } else {
    for (size_t e = i; e < i + 4 && e < total; ++e) {
      float acc = 0.0f;
      for (int s = 0; s < ksplit; ++s) acc += partial[(size_t)s * total + e];
      y[e] = acc;
    }
  }
}

hipError_t launch_wo_gemm(const uint16_t* ob, const uint16_t* W, bool prepared, float* y, float* partial, int B,
                          int K, int N, int ksplit, hipStream_t s) {
  // 32-bit per-lane DMA offsets: the row-major weights and both o terms must span less than 4 GiB
  if (K % kWoKStep != 0 || B <= 0 || N <= 0 || ksplit != wo_ksplit(K, N, B) ||
      (!prepared && (size_t)N * K * 2 >= (1ull << 32)) || (size_t)2 * B * K * 2 >= (1ull << 32))
    return hipErrorInvalidValue;
  dim3 grid((N + kWoTileN - 1) / kWoTileN, ksplit, (B + kWoBatch - 1) / kWoBatch);
  if (prepared)
    hipLaunchKernelGGL(wo_mfma_kernel<true>, grid, dim3(256), 0, s, ob, W, partial, y, B, K, N, wo_slice(K, N, B),
                       ksplit);
  else
    hipLaunchKernelGGL(wo_mfma_kernel<false>, grid, dim3(256), 0, s, ob, W, partial, y, B, K, N, wo_slice(K, N, B),
                       ksplit);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || ksplit == 1) return e;
  const size_t total = (size_t)B * N, threads = (total + 3) / 4;
  hipLaunchKernelGGL(wo_reduce_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s, partial, y, total,
                     ksplit);
  return hipGetLastError();
}

// K per work-group: the K range is split so that the grid holds about one work-group per CU (a
// work-group's stages fill most of the LDS), in whole 32-wide steps.
int wo_slice(int K, int N, int B) {
  const int tiles = ((N + kWoTileN - 1) / kWoTileN) * ((B + kWoBatch - 1) / kWoBatch);
  const int want = max(1, num_cus() / max(1, tiles));
  const int steps = (K + kWoKStep - 1) / kWoKStep;
  return kWoKStep * ((steps + want - 1) / want);
}
int wo_ksplit(int K, int N, int B) {
  const int sl = wo_slice(K, N, B);
  return (K + sl - 1) / sl;
}

// ---------------------------------------------------------------------------------------------
// Prepared weights: element (n, k) of W_O (or of W-bar_O = W_O R_V per head block) as fp16 at
//   ((n / 128) (K / 32) + k / 32) 4096 + 512 ((n % 128) / 16) + 8 ((n % 16) + 16 ((k % 32) / 8)) + k % 8,
// i.e. for each 128-row block and 32-wide k step, eight 16 x 32 operand tiles in lane order (lane
// l = row + 16 (k / 8) holds 8 consecutive k). Rows past N in the last block are zero. One block per
// (kPrepRows rows, query head j); thread c computes column j*128 + c.
constexpr int kPrepRows = 16;

__global__ __launch_bounds__(128) void prepare_wo_kernel(const uint16_t* __restrict__ W, const float* __restrict__ R_v,
                                                         uint16_t* __restrict__ Wp, int N, int Hq, int gq) {
  __shared__ float rows[kPrepRows][kHeadDim];
  const int j = blockIdx.y, c = threadIdx.x;
  const int n0 = blockIdx.x * kPrepRows;
  const int K = Hq * kHeadDim;
  for (int r = 0; r < kPrepRows; ++r) {
    const int n = n0 + r;
    rows[r][c] = n < N ? bf16_bits_to_f32(W[(size_t)n * K + (size_t)j * kHeadDim + c]) : 0.0f;
  }
  __syncthreads();
  float col[kHeadDim];
  if (R_v) {
    const float* R = R_v + (size_t)(j / gq) * kHeadDim * kHeadDim;
#pragma unroll
    for (int i = 0; i < kHeadDim; ++i) col[i] = R[i * kHeadDim + c];
  }
  const int k = j * kHeadDim + c;
  for (int r = 0; r < kPrepRows; ++r) {
    const int n = n0 + r;
    float v = rows[r][c];
    if (R_v) {
      float acc = 0.0f;
#pragma unroll
      for (int i = 0; i < kHeadDim; ++i) acc = fmaf(rows[r][i], col[i], acc);
      v = acc;
    }
    const size_t at = ((size_t)(n / kWoTileN) * (K / kWoKStep) + k / kWoKStep) * kWoTileElems +
                      512 * ((n % kWoTileN) / 16) + 8 * ((n % 16) + 16 * ((k % kWoKStep) / 8)) + k % 8;
    Wp[at] = __half_as_ushort(__float2half_rn(v));
  }
}

size_t prepared_wo_elems(int N, int K) { return (size_t)((N + kWoTileN - 1) / kWoTileN) * kWoTileN * K; }

hipError_t launch_prepare_wo(const uint16_t* W_o, const float* R_v, uint16_t* Wp, int N, int Hq, int H,
                             hipStream_t s) {
  const int Npad = (N + kWoTileN - 1) / kWoTileN * kWoTileN;
  dim3 grid(Npad / kPrepRows, Hq);
  hipLaunchKernelGGL(prepare_wo_kernel, grid, dim3(128), 0, s, W_o, R_v, Wp, N, Hq, Hq / H);
  return hipGetLastError();
}

}  // namespace int2kv
