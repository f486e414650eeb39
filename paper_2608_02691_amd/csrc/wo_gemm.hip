// Output projection y = concat_j(o_j) W_O^T (eq:residual_readout; eq:int2_residual_readout).
// o: [B, K] as two bf16 terms (hi = bf16(o), lo = bf16(o - hi), written by the merge), W_O: bf16
// [N, K] row-major, y: fp32 [B, N].
//
// Matrix-core GEMM, HBM-bound on the weights (N x K bf16, read once). Both terms of o are
// multiplied against the bf16 weights, which keeps the product at fp32-like precision
// (|o - hi - lo| <= 2^-16 |o|). Each wave owns a 64 x 64 output tile (four 16-row A tiles of W,
// four 16-column B tiles of o) over one k chunk and reads both operands straight from memory
// (W from HBM, o from L2, equal byte counts), two k steps ahead; the four waves of a work-group
// take consecutive k chunks of the same rows and add their tiles through LDS in wave order.
// Work-group slices write partial products [slice][B][N]; a second kernel sums them in slice
// order, so the result does not depend on scheduling (deterministic).
#include "common.h"
#include "kernels.h"

namespace int2kv {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float wo_f4_t __attribute__((ext_vector_type(4)));

constexpr int kWoRows = 64;     // rows of W (output columns) per wave and work-group
constexpr int kWoBatch = 64;    // batch rows per work-group
constexpr int kWoWaves = 4;     // waves per work-group: consecutive k chunks of the same rows
constexpr int kWoChunk = 320;   // k per wave (10 steps)
constexpr int kWoSlice = kWoWaves * kWoChunk;  // k per work-group
constexpr int kWoKStep = 32;
constexpr int kWoRing = 2;      // k steps of operands in flight per wave
constexpr int kWoRedRow = 68;   // floats per LDS row of the reduction tile (64 + 4 pad)

__global__ __launch_bounds__(256) void wo_mfma_kernel(const uint16_t* __restrict__ ob, const uint16_t* __restrict__ W,
                                                      float* __restrict__ partial, int B, int K, int N) {
  __shared__ __attribute__((aligned(16))) float red[kWoWaves][kWoBatch][kWoRedRow];
  const int n0 = blockIdx.x * kWoRows, ks = blockIdx.y, b0 = blockIdx.z * kWoBatch;
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, lo = l & 15, hi = l >> 4;
  const int k0 = ks * kWoSlice + w * kWoChunk;
  const int nsteps = max(0, min(K - k0, kWoChunk)) / kWoKStep;  // even (K is a multiple of 64)

  // A operand: W rows n0 + 16 a + lo; B operand: o rows b0 + 16 t + lo (hi and lo terms);
  // 8 consecutive k per lane; rows past N or B are clamped (computed, never stored)
  const uint16_t* pa[4];
  const uint16_t* pb[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    pa[i] = W + (size_t)min(n0 + 16 * i + lo, N - 1) * K + k0 + 8 * hi;
    pb[i] = ob + (size_t)min(b0 + 16 * i + lo, B - 1) * K + k0 + 8 * hi;
  }
  const size_t lo_term = (size_t)B * K;  // offset of the lo array
  struct Ops {
    bf16x8_t a[4], bh[4], bl[4];
  };
  auto load = [&](int s, Ops& o) {
    const int off = s * kWoKStep;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      o.a[i] = *reinterpret_cast<const bf16x8_t*>(pa[i] + off);
      o.bh[i] = *reinterpret_cast<const bf16x8_t*>(pb[i] + off);
      o.bl[i] = *reinterpret_cast<const bf16x8_t*>(pb[i] + lo_term + off);
    }
  };

  wo_f4_t acc[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int t = 0; t < 4; ++t) acc[a][t] = wo_f4_t{0.f, 0.f, 0.f, 0.f};
  if (nsteps > 0) {
    // branch-free body (loads past the end re-read the last step), so the compiler counts the
    // loads in flight exactly
    const int last = nsteps - 1;
    Ops ring[kWoRing];
#pragma unroll
    for (int i = 0; i < kWoRing; ++i) load(min(i, last), ring[i]);
    for (int s0 = 0; s0 < nsteps; s0 += kWoRing) {
#pragma unroll
      for (int i = 0; i < kWoRing; ++i) {
        const Ops& o = ring[i];
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            acc[a][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(o.a[a], o.bh[t], acc[a][t], 0, 0, 0);
            acc[a][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(o.a[a], o.bl[t], acc[a][t], 0, 0, 0);
          }
        load(min(s0 + i + kWoRing, last), ring[i]);
      }
    }
  }
  // D[m][n] sits in lane n + 16 (m / 4), register m % 4: m = W row in the A tile, n = batch row
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int t = 0; t < 4; ++t)
      *reinterpret_cast<float4*>(&red[w][16 * t + lo][16 * a + 4 * hi]) =
          make_float4(acc[a][t][0], acc[a][t][1], acc[a][t][2], acc[a][t][3]);
  __syncthreads();
  // sum of the four chunks in wave order; thread -> (batch row, four consecutive columns)
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int e = tid + 256 * u, bl = e >> 4, c4 = 4 * (e & 15);
    float4 s = *reinterpret_cast<const float4*>(&red[0][bl][c4]);
#pragma unroll
    for (int v = 1; v < kWoWaves; ++v) {
      const float4 x = *reinterpret_cast<const float4*>(&red[v][bl][c4]);
      s.x += x.x;
      s.y += x.y;
      s.z += x.z;
      s.w += x.w;
    }
    const int b = b0 + bl, n = n0 + c4;
    if (b >= B) continue;
    float* dst = partial + ((size_t)ks * B + b) * N + n;
    if (n + 3 < N && (N & 3) == 0) {
      *reinterpret_cast<float4*>(dst) = s;
    } else {
      const float sv[4] = {s.x, s.y, s.z, s.w};
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (n + r < N) dst[r] = sv[r];
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
  static_assert(kWoChunk % (kWoKStep * kWoRing) == 0, "chunks hold whole rings of k steps");
  if (K % (kWoKStep * kWoRing) != 0 || B <= 0 || N <= 0 || ksplit != wo_ksplit(K)) return hipErrorInvalidValue;
  dim3 grid((N + kWoRows - 1) / kWoRows, ksplit, (B + kWoBatch - 1) / kWoBatch);
  hipLaunchKernelGGL(wo_mfma_kernel, grid, dim3(256), 0, s, ob, W, partial, B, K, N);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t total = (size_t)B * N;
  hipLaunchKernelGGL(wo_reduce_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, partial, y, total,
                     ksplit);
  return hipGetLastError();
}

int wo_ksplit(int K) { return (K + kWoSlice - 1) / kWoSlice; }

}  // namespace int2kv
