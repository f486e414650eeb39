// Output projection y = concat_j(o_j) W_O^T (eq:residual_readout; eq:int2_residual_readout).
// o: [B, K] as two bf16 terms (hi = bf16(o), lo = bf16(o - hi), written by the merge), W_O: bf16
// [N, K] row-major, y: fp32 [B, N].
//
// Matrix-core GEMM, HBM-bound on the weights (N x K bf16, read once). Both terms of o are
// multiplied against the bf16 weights, which keeps the product at fp32-like precision
// (|o - hi - lo| <= 2^-16 |o|). Work-group (128 rows of W, one K slice, 64 batch rows), four waves
// of 32 rows. Every 32-wide k step of the weights and of o is staged in LDS with LDS-DMA loads
// (global_load_lds: lane i's 16 bytes land at M0 + 16 i), kWoStages - 1 steps ahead, with no
// registers held for data in flight; each lane fetches exactly the 16 bytes it later reads as its
// MFMA operand, so the LDS reads are conflict-free. The o tile is shared by the four waves: each
// wave waits for its own DMA, then one barrier makes the whole step visible. Slices write partial
// products [slice][B][N]; a second kernel sums them in slice order (deterministic).
#include "common.h"
#include "kernels.h"

namespace int2kv {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float wo_f4_t __attribute__((ext_vector_type(4)));

constexpr int kWoTileN = 128;   // rows of W (output columns) per work-group
constexpr int kWoBatch = 64;    // batch rows per work-group (four 16-column B tiles)
constexpr int kWoKStep = 32;
constexpr int kWoStages = 8;    // LDS stages; kWoStages - 1 steps in flight (112 KiB per work-group)
constexpr int kWoStageBytes = 16384;  // W: 4 waves x 2 tiles x 1 KiB; o: 2 terms x 4 tiles x 1 KiB
constexpr int kWoDmaPerStep = 4;      // DMA instructions per wave and step (2 of W, 2 of o)

__device__ __forceinline__ void wo_dma(const void* base, uint32_t voff, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2" ::"s"(lds_addr), "v"(voff), "s"(base)
               : "memory", "m0");
}

__global__ __launch_bounds__(256) void wo_mfma_kernel(const uint16_t* __restrict__ ob, const uint16_t* __restrict__ W,
                                                      float* __restrict__ partial, int B, int K, int N,
                                                      int slice) {
  __shared__ __attribute__((aligned(16))) uint8_t stage[kWoStages][kWoStageBytes];
  const int n0 = blockIdx.x * kWoTileN, ks = blockIdx.y, b0 = blockIdx.z * kWoBatch;
  const int tid = threadIdx.x, w = __builtin_amdgcn_readfirstlane(tid >> 6), l = tid & 63;
  const int lo = l & 15, hi = l >> 4;
  const int k_begin = ks * slice;
  const int nsteps = (min(K, k_begin + slice) - k_begin) / kWoKStep;
  const int last = nsteps - 1;

  // Per-lane byte offsets (the step's k offset rides in the scalar base):
  // W tile a of this wave: row n0 + 32 w + 16 a + lo (clamped), k + 8 hi
  uint32_t woff[2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
    woff[a] = (uint32_t)(((size_t)min(n0 + 32 * w + 16 * a + lo, N - 1) * K + 8 * hi) * 2);
  // o tile q = 2 w + u of the work-group: term q / 4 (hi, lo), batch tile q % 4
  uint32_t ooff[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int q = 2 * w + u, term = q >> 2, t = q & 3;
    ooff[u] = (uint32_t)(((size_t)term * B * K + (size_t)min(b0 + 16 * t + lo, B - 1) * K + 8 * hi) * 2);
  }
  const uint32_t stage0 = (uint32_t)(uintptr_t)&stage[0][0];
  auto issue = [&](int s) {  // DMA of step min(s, last) into stage s % kWoStages
    const int sc = min(s, last);
    const uint32_t dst = stage0 + (uint32_t)((s % kWoStages) * kWoStageBytes);
    const uint16_t* wb = W + k_begin + sc * kWoKStep;
    const uint16_t* obb = ob + k_begin + sc * kWoKStep;
#pragma unroll
    for (int a = 0; a < 2; ++a) wo_dma(wb, woff[a], dst + (uint32_t)((2 * w + a) * 1024));
#pragma unroll
    for (int u = 0; u < 2; ++u) wo_dma(obb, ooff[u], dst + (uint32_t)(8192 + (2 * w + u) * 1024));
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
    asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"((kWoStages - 2) * kWoDmaPerStep) : "memory");
    issue(s + kWoStages - 1);
    const uint8_t* st = &stage[s % kWoStages][0];
    bf16x8_t A[2], Bt[2][4];
#pragma unroll
    for (int a = 0; a < 2; ++a) A[a] = *reinterpret_cast<const bf16x8_t*>(st + (2 * w + a) * 1024 + 16 * l);
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
      for (int t = 0; t < 4; ++t) Bt[x][t] = *reinterpret_cast<const bf16x8_t*>(st + 8192 + (4 * x + t) * 1024 + 16 * l);
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int a = 0; a < 2; ++a) {
        acc[a][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A[a], Bt[0][t], acc[a][t], 0, 0, 0);
        acc[a][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A[a], Bt[1][t], acc[a][t], 0, 0, 0);
      }
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // drain the clamped tail DMAs before exit
  // D[m][n] sits in lane n + 16 (m / 4), register m % 4: m = W row in the A tile, n = batch row; the
  // four registers are four consecutive output columns of one batch row
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int n = n0 + 32 * w + 16 * a + 4 * hi, b = b0 + 16 * t + lo;
      if (b >= B) continue;
      float* dst = partial + ((size_t)ks * B + b) * N + n;
      if (n + 3 < N && (N & 3) == 0) {
        *reinterpret_cast<float4*>(dst) = make_float4(acc[a][t][0], acc[a][t][1], acc[a][t][2], acc[a][t][3]);
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (n + r < N) dst[r] = acc[a][t][r];
      }
    }
}

// y[i] = sum over slices, in slice order, of partial[s][i] (i = b N + n): one element per thread.
__global__ __launch_bounds__(256) void wo_reduce_kernel(const float* __restrict__ partial, float* __restrict__ y,
                                                         size_t total, int ksplit) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= total) return;
  float acc = 0.0f;
  for (int s = 0; s < ksplit; ++s) acc += partial[(size_t)s * total + i];
  y[i] = acc;
}

hipError_t launch_wo_gemm(const uint16_t* ob, const uint16_t* W, float* y, float* partial, int B, int K, int N,
                          int ksplit, hipStream_t s) {
  // 32-bit per-lane DMA offsets: the weights and both o terms must span less than 4 GiB
  if (K % kWoKStep != 0 || B <= 0 || N <= 0 || ksplit != wo_ksplit(K, N, B) || (size_t)N * K * 2 >= (1ull << 32) ||
      (size_t)2 * B * K * 2 >= (1ull << 32))
    return hipErrorInvalidValue;
  dim3 grid((N + kWoTileN - 1) / kWoTileN, ksplit, (B + kWoBatch - 1) / kWoBatch);
  hipLaunchKernelGGL(wo_mfma_kernel, grid, dim3(256), 0, s, ob, W, partial, B, K, N, wo_slice(K, N, B));
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t total = (size_t)B * N;
  hipLaunchKernelGGL(wo_reduce_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, partial, y, total,
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

}  // namespace int2kv
