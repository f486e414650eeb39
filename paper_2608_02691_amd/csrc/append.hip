// Cache write: rotate (and center) keys/values, group-quantize to INT2, pack into the paged pool.
//
// Sec. 4.1 (key reparameterization k -> k - mu before rotation), Sec. 6 efficiency analysis and
// the appendix key-mean application ((k - mu) R_K = k R_K - mu R_K, mu R_K precomputed), Sec. 5
// implementation details (group-wise affine INT2). The packed record layout is documented in
// include/int2kv.h.
#include "append_core.h"
#include "common.h"
#include "kernels.h"

namespace int2kv {

// ---------------------------------------------------------------------------------------------
// mu R_K per KV head: thread c accumulates sum_i mu[i] R[i][c] in fp32, channel order.
__global__ __launch_bounds__(128) void prepare_mu_rot_kernel(const float* __restrict__ R_k,
                                                              const float* __restrict__ mu,
                                                              float* __restrict__ mu_rk) {
  const int h = blockIdx.x, c = threadIdx.x;
  const float* R = R_k + (size_t)h * kHeadDim * kHeadDim;
  const float* m = mu + (size_t)h * kHeadDim;
  float acc = 0.0f;
  for (int i = 0; i < kHeadDim; ++i) acc = fmaf(m[i], R[i * kHeadDim + c], acc);
  mu_rk[(size_t)h * kHeadDim + c] = acc;
}

hipError_t launch_prepare_mu_rot(const float* R_k, const float* mu, float* mu_rk, int H, hipStream_t s) {
  hipLaunchKernelGGL(prepare_mu_rot_kernel, dim3(H), dim3(128), 0, s, R_k, mu, mu_rk);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------------------------
// W-bar_{O,j} = W_{O,j} R_{V,h(j)}: block (row tile, query head), thread c = output column.
constexpr int kFoldRows = 32;

__global__ __launch_bounds__(128) void fold_wo_kernel(const uint16_t* __restrict__ W,
                                                       const float* __restrict__ R_v,
                                                       uint16_t* __restrict__ Wf, int d_model, int Hq,
                                                       int gq) {
  __shared__ float rows[kFoldRows][kHeadDim];
  const int j = blockIdx.y, h = j / gq, c = threadIdx.x;
  const int n0 = blockIdx.x * kFoldRows;
  const size_t ld = (size_t)Hq * kHeadDim;
  for (int r = 0; r < kFoldRows; ++r) {
    const int n = n0 + r;
    rows[r][c] = n < d_model ? bf16_bits_to_f32(W[n * ld + (size_t)j * kHeadDim + c]) : 0.0f;
  }
  __syncthreads();
  const float* R = R_v + (size_t)h * kHeadDim * kHeadDim;
  float col[kHeadDim];
#pragma unroll
  for (int i = 0; i < kHeadDim; ++i) col[i] = R[i * kHeadDim + c];
  for (int r = 0; r < kFoldRows; ++r) {
    const int n = n0 + r;
    if (n >= d_model) break;
    float acc = 0.0f;
#pragma unroll
    for (int i = 0; i < kHeadDim; ++i) acc = fmaf(rows[r][i], col[i], acc);
    Wf[n * ld + (size_t)j * kHeadDim + c] = static_cast<uint16_t>(f32_to_bf16_rne(acc));
  }
}

hipError_t launch_fold_wo(const uint16_t* W_o, const float* R_v, uint16_t* W_f, int d_model, int Hq,
                          int H, hipStream_t s) {
  dim3 grid((d_model + kFoldRows - 1) / kFoldRows, Hq);
  hipLaunchKernelGGL(fold_wo_kernel, grid, dim3(128), 0, s, W_o, R_v, W_f, d_model, Hq, Hq / H);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------------------------
// Quantize one token row of K (threads 0..127) and V (threads 128..255) held one channel per
// thread, and store it, with NG groups per token. All 256 threads of the block must call it (it
// synchronizes).
template <int NG>
__device__ __forceinline__ void quantize_store_pair(float x, int slot, int h, float clip_k, float clip_v,
                                                    const CacheView& cv, uint8_t (*codes)[kHeadDim],
                                                    float (*ext)[2][2]) {
  using L = Rec<NG>;
  const int tid = threadIdx.x;
  const int row = tid >> 7;  // 0 = K, 1 = V
  const int c = tid & 127;
  float mn = x, mx = x;
  if constexpr (NG == 4) {
#pragma unroll
    for (int off = 16; off >= 1; off >>= 1) {
      mn = fminf(mn, __shfl_xor(mn, off, 32));
      mx = fmaxf(mx, __shfl_xor(mx, off, 32));
    }
  } else {
    // one group of 128 channels: the row's two waves reduce, then exchange through LDS
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      mn = fminf(mn, __shfl_xor(mn, off));
      mx = fmaxf(mx, __shfl_xor(mx, off));
    }
    if ((tid & 63) == 0) {
      ext[row][(tid >> 6) & 1][0] = mn;
      ext[row][(tid >> 6) & 1][1] = mx;
    }
    __syncthreads();
    mn = fminf(ext[row][0][0], ext[row][1][0]);
    mx = fmaxf(ext[row][0][1], ext[row][1][1]);
  }
  uint32_t s_bits, z_bits;
  float zf, inv;
  int2_group_params(mn, mx, row == 0 ? clip_k : clip_v, s_bits, z_bits, zf, inv);
  codes[row][c] = static_cast<uint8_t>(int2_code(x, zf, inv));
  __syncthreads();
  const bool ok = slot >= 0 && slot < cv.num_blocks * kBlock;
  if (ok) {
    const int blk = slot >> 4, t = slot & 15;
    uint8_t* rec = cv.pool + ((size_t)blk * cv.num_kv_heads + h) * L::kBytes;
    if (c < 16) {
      uint32_t half = 0;
#pragma unroll
      for (int p = 0; p < 8; ++p) half |= static_cast<uint32_t>(codes[row][16 * p + c]) << (2 * p);
      const int off = row == 0 ? kOffKCodes + 32 * t + 2 * c : kOffVCodes + 32 * c + 2 * t;
      *reinterpret_cast<uint16_t*>(rec + off) = static_cast<uint16_t>(half);
    }
    if ((c % L::kGroupSize) == 0) {
      const int g = c / L::kGroupSize;
      if (row == 0) {
        *reinterpret_cast<uint32_t*>(rec + L::kOffKMeta + 4 * NG * t + 4 * g) = s_bits | (z_bits << 16);
      } else {
        *reinterpret_cast<uint16_t*>(rec + L::kOffVScale + 32 * g + 2 * t) = static_cast<uint16_t>(s_bits);
        *reinterpret_cast<uint16_t*>(rec + L::kOffVZero + 32 * g + 2 * t) = static_cast<uint16_t>(z_bits);
      }
    }
  }
  __syncthreads();
}

// Quantize already rotated rows: block (token, KV head).
template <int NG>
__global__ __launch_bounds__(256) void pack_rotated_kernel(CacheView cv, const float* __restrict__ k_rot,
                                                            const float* __restrict__ v_rot,
                                                            const int32_t* __restrict__ slots, float clip_k,
                                                            float clip_v) {
  __shared__ uint8_t codes[2][kHeadDim];
  __shared__ float ext[2][2][2];
  const int n = blockIdx.x, h = blockIdx.y, tid = threadIdx.x;
  const size_t base = ((size_t)n * cv.num_kv_heads + h) * kHeadDim + (tid & 127);
  const float x = tid < 128 ? k_rot[base] : v_rot[base];
  quantize_store_pair<NG>(x, slots[n], h, clip_k, clip_v, cv, codes, ext);
}

hipError_t launch_pack_rotated(CacheView c, const float* k_rot, const float* v_rot, const int32_t* slots,
                               int n, float clip_k, float clip_v, hipStream_t s) {
  if (c.groups == 1)
    hipLaunchKernelGGL(pack_rotated_kernel<1>, dim3(n, c.num_kv_heads), dim3(256), 0, s, c, k_rot, v_rot, slots,
                       clip_k, clip_v);
  else
    hipLaunchKernelGGL(pack_rotated_kernel<4>, dim3(n, c.num_kv_heads), dim3(256), 0, s, c, k_rot, v_rot, slots,
                       clip_k, clip_v);
  return hipGetLastError();
}

// Standalone append kernel: grid (blocks per (h, K|V), KV heads, K|V) of kApWaves waves.
template <int kApTiles, int NG, bool ERR = false, bool ROPE = false>
__global__ __launch_bounds__(512) void append_mfma_kernel(CacheView cv, const uint16_t* __restrict__ k,
                                                           const uint16_t* __restrict__ v,
                                                           const int32_t* __restrict__ slots, int n,
                                                           const float* __restrict__ R_k,
                                                           const float* __restrict__ R_v,
                                                           const float* __restrict__ mu_rk, float clip_k,
                                                           float clip_v, float* __restrict__ err, ApOpts opt) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[kAppendLdsBytes];
  append_block<kApTiles, kApWaves, NG, ERR, ROPE>(cv, k, v, slots, n, R_k, R_v, mu_rk, clip_k, clip_v,
                                                  (int)blockIdx.x, (int)gridDim.x, (int)blockIdx.y, (int)blockIdx.z,
                                                  lds, err, opt);
}

hipError_t launch_append_mfma(CacheView c, const uint16_t* k, const uint16_t* v, const int32_t* slots, int n,
                              const float* R_k, const float* R_v, const float* mu_rk, float clip_k,
                              float clip_v, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1, float* err,
                              const AppendOptions* o) {
  ApOpts opt{};
  if (o) {
    opt.pos = o->positions;
    opt.cos_sin = o->cos_sin;
    opt.max_pos = o->max_pos;
    opt.k_out = o->k_rope_out;
    opt.had = o->hadamard;
  }
  if (n <= 0) return hipSuccess;
  // one work-group per CU (its R^T terms fill most of the LDS), each converting R once for many
  // steps; short appends take one tile per wave step
  const int per_head = max(1, 256 / (2 * c.num_kv_heads));
  const int tiles = (n + 15) / 16;
  const dim3 block(64 * kApWaves);
  // the instantiation: one or two tiles per wave step, 4 or 1 groups per token, with or without the
  // reconstruction error
  auto go = [&](auto tiles_tag, auto ng_tag, dim3 grid) {
    constexpr int T = decltype(tiles_tag)::value, NG = decltype(ng_tag)::value;
    if (opt.pos)
      hipExtLaunchKernelGGL((append_mfma_kernel<T, NG, false, true>), grid, block, 0, s, ev0, ev1, 0, c, k, v,
                            slots, n, R_k, R_v, mu_rk, clip_k, clip_v, err, opt);
    else if (err)
      hipExtLaunchKernelGGL((append_mfma_kernel<T, NG, true>), grid, block, 0, s, ev0, ev1, 0, c, k, v, slots, n,
                            R_k, R_v, mu_rk, clip_k, clip_v, err, opt);
    else
      hipExtLaunchKernelGGL((append_mfma_kernel<T, NG, false>), grid, block, 0, s, ev0, ev1, 0, c, k, v, slots, n,
                            R_k, R_v, mu_rk, clip_k, clip_v, err, opt);
  };
  using One = std::integral_constant<int, 1>;
  using Two = std::integral_constant<int, 2>;
  using Four = std::integral_constant<int, 4>;
  if (tiles <= kApWaves * per_head) {
    const dim3 grid((tiles + kApWaves - 1) / kApWaves, c.num_kv_heads, 2);
    if (c.groups == 1)
      go(One{}, One{}, grid);
    else
      go(One{}, Four{}, grid);
  } else {
    const int steps = (tiles + 1) / 2;
    const dim3 grid(min((steps + kApWaves - 1) / kApWaves, per_head), c.num_kv_heads, 2);
    if (c.groups == 1)
      go(Two{}, One{}, grid);
    else
      go(Two{}, Four{}, grid);
  }
  return hipGetLastError();
}

}  // namespace int2kv
