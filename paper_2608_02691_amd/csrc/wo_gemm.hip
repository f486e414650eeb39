// Output projection y = concat_j(o_j) W_O^T (eq:residual_readout; eq:int2_residual_readout).
// o: fp32 [B, K], W_O: bf16 [N, K] row-major, y: fp32 [B, N]. Split over K into fixed slices
// whose partial products are summed in a fixed order (deterministic).
#include "common.h"
#include "kernels.h"

namespace int2kv {

constexpr int kWoN = 64;      // output columns per block
constexpr int kWoB = 16;      // batch rows per block
constexpr int kWoK = 32;      // k step staged in LDS
constexpr int kWoSlice = 512;  // k per split

__global__ __launch_bounds__(256) void wo_partial_kernel(const float* __restrict__ o, const uint16_t* __restrict__ W,
                                                          float* __restrict__ partial, int B, int K, int N) {
  __shared__ float ws[kWoK][kWoN + 1];
  __shared__ float xs[kWoB][kWoK + 1];
  const int n0 = blockIdx.x * kWoN, b0 = blockIdx.y * kWoB, ks = blockIdx.z;
  const int k_begin = ks * kWoSlice, k_end = min(K, k_begin + kWoSlice);
  const int tid = threadIdx.x, nl = tid & 63, bg = tid >> 6;  // 4 batch rows per thread
  float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int k0 = k_begin; k0 < k_end; k0 += kWoK) {
    for (int i = tid; i < kWoN * kWoK; i += 256) {
      const int r = i / kWoK, kk = i % kWoK;
      const int n = n0 + r, k = k0 + kk;
      ws[kk][r] = (n < N && k < k_end) ? bf16_bits_to_f32(W[(size_t)n * K + k]) : 0.0f;
    }
    for (int i = tid; i < kWoB * kWoK; i += 256) {
      const int r = i / kWoK, kk = i % kWoK;
      const int bb = b0 + r, k = k0 + kk;
      xs[r][kk] = (bb < B && k < k_end) ? o[(size_t)bb * K + k] : 0.0f;
    }
    __syncthreads();
#pragma unroll 8
    for (int kk = 0; kk < kWoK; ++kk) {
      const float wv = ws[kk][nl];
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[r] = fmaf(xs[bg * 4 + r][kk], wv, acc[r]);
    }
    __syncthreads();
  }
  const int n = n0 + nl;
  if (n < N) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int bb = b0 + bg * 4 + r;
      if (bb < B) partial[((size_t)ks * B + bb) * N + n] = acc[r];
    }
  }
}

__global__ __launch_bounds__(256) void wo_reduce_kernel(const float* __restrict__ partial, float* __restrict__ y,
                                                         int B, int N, int ksplit) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (size_t)B * N) return;
  float acc = 0.0f;
  for (int s = 0; s < ksplit; ++s) acc += partial[(size_t)s * B * N + i];
  y[i] = acc;
}

hipError_t launch_wo_gemm(const float* o, const uint16_t* W, float* y, float* partial, int B, int K, int N,
                          int ksplit, hipStream_t s) {
  dim3 grid((N + kWoN - 1) / kWoN, (B + kWoB - 1) / kWoB, ksplit);
  hipLaunchKernelGGL(wo_partial_kernel, grid, dim3(256), 0, s, o, W, partial, B, K, N);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t total = (size_t)B * N;
  hipLaunchKernelGGL(wo_reduce_kernel, dim3((total + 255) / 256), dim3(256), 0, s, partial, y, B, N, ksplit);
  return hipGetLastError();
}

int wo_ksplit(int K) { return (K + kWoSlice - 1) / kWoSlice; }

}  // namespace int2kv
