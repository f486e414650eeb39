// Decode attention over the paged INT2 cache: query rotation, split-context scan (vector-ALU
// variant), and the log-sum-exp merge with the R_V^T un-rotation.
//
// eq:int2_attention / eq:int2_residual_readout evaluated in the rotated coordinates of the
// appendix "Rotated-query implementation": a_s = (q R_K) k_R,s^T / sqrt(d), and the value
// readout o = (sum_s p_s v_R,s) R_V^T. Dequantized entries are code * s + z per group; the dot
// products factor the affine metadata out: q'.k_hat = sum_g s_g (q'_g . c_g) + z_g sum(q'_g).
#include "common.h"
#include "kernels.h"

namespace int2kv {

// log2(e) / sqrt(128): logits are kept in the base-2 domain so exp2 is the only transcendental.
constexpr float kLogitScale = 1.4426950408889634f * 0.08838834764831845f;

__device__ __forceinline__ int seq_len(const DecodeArgs& a, int b) {
  int L = a.ctx_lens[b];
  L = min(L, a.max_ctx);
  L = min(L, a.max_blocks * kBlock);
  return max(L, 0);
}

// ---------------------------------------------------------------------------------------------
// q' = q R_K per query head (fp32, channel order). Block (b, j), thread c.
__global__ __launch_bounds__(128) void qrot_kernel(DecodeArgs a) {
  __shared__ float qs[kHeadDim];
  const int bj = blockIdx.x, b = bj / a.Hq, j = bj % a.Hq, h = j / a.gq, c = threadIdx.x;
  qs[c] = bf16_bits_to_f32(a.q[(size_t)bj * kHeadDim + c]);
  __syncthreads();
  const float* R = a.R_k + (size_t)h * kHeadDim * kHeadDim;
  float acc = 0.0f;
  for (int i = 0; i < kHeadDim; ++i) acc = fmaf(qs[i], R[i * kHeadDim + c], acc);
  a.qrot[((size_t)b * a.Hq + j) * kHeadDim + c] = acc;
}

hipError_t launch_qrot(const DecodeArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(qrot_kernel, dim3(a.B * a.Hq), dim3(128), 0, s, a);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------------------------
// Vector-ALU split-context scan. Block (chunk, KV head, sequence) of 4 waves; wave w scans pages
// w, w+4, ... of the chunk with its own online-softmax state; the block merges the four states
// and writes one partial (m, l, O) per query head of the group.
constexpr int kWaves = 4;

__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// NG groups per token (4 or 1). A lane's 32-channel quarter gk always carries its own q' sum; with
// one group per token the four quarters share the token's (s, z), and the summed logit is the same.
template <int MAXG, int NG>
__global__ __launch_bounds__(256) void decode_split_valu_kernel(DecodeArgs a) {
  using Lay = Rec<NG>;
  __shared__ float qs[MAXG][kHeadDim];
  __shared__ float qsum[MAXG][kGroups];
  __shared__ float pbuf[kWaves][MAXG][kBlock];
  __shared__ float wstate[kWaves][MAXG][2];
  __shared__ float wout[kWaves][MAXG][kHeadDim];

  const int chunk = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int L = seq_len(a, b);
  const int t0 = chunk * a.chunk_tokens;
  if (t0 >= L) return;  // uniform for the whole block
  const int t1 = min(L, t0 + a.chunk_tokens);
  const int gq = a.gq;
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63;

  for (int i = tid; i < gq * kHeadDim; i += blockDim.x) {
    const int jj = i / kHeadDim, c = i % kHeadDim;
    qs[jj][c] = a.qrot[((size_t)b * a.Hq + h * gq + jj) * kHeadDim + c] * kLogitScale;
  }
  __syncthreads();
  if (tid < gq * kGroups) {
    const int jj = tid / kGroups, g = tid % kGroups;
    float acc = 0.0f;
    for (int c = 0; c < kGroup; ++c) acc += qs[jj][g * kGroup + c];
    qsum[jj][g] = acc;
  }
  __syncthreads();

  float m_run[MAXG], l_run[MAXG], o0[MAXG], o1[MAXG];
#pragma unroll
  for (int j = 0; j < MAXG; ++j) {
    m_run[j] = -INFINITY;
    l_run[j] = 0.0f;
    o0[j] = 0.0f;
    o1[j] = 0.0f;
  }

  // QK lane role: token tq = l / 4 of the page, group gk = l % 4.
  const int tq = l >> 2, gk = l & 3;
  // PV lane role: channels 2l, 2l+1 -> halves m0, m0+1 at bit position pv, group gv.
  const int c0 = 2 * l, m0 = c0 & 15, pv = c0 >> 4, gv = c0 >> 5;

  const int pg0 = t0 / kBlock, pg1 = (t1 + kBlock - 1) / kBlock;
  for (int pg = pg0 + w; pg < pg1; pg += kWaves) {
    const int blk = a.block_table[(size_t)b * a.max_blocks + pg];
    if (blk < 0 || blk >= a.num_blocks) continue;  // uniform per wave
    const uint8_t* rec = a.pool + ((size_t)blk * a.H + h) * Lay::kBytes;

    // ---- scores of token tq for every query head of the group
    const uint4* kc = reinterpret_cast<const uint4*>(rec + kOffKCodes + 32 * tq);
    const uint4 k0 = kc[0], k1 = kc[1];
    const uint32_t kw[8] = {k0.x, k0.y, k0.z, k0.w, k1.x, k1.y, k1.z, k1.w};
    const uint32_t meta =
        *reinterpret_cast<const uint32_t*>(rec + Lay::kOffKMeta + 4 * NG * tq + 4 * (NG == 4 ? gk : 0));
    const float ks = f16_bits_to_f32(meta & 0xFFFF), kz = f16_bits_to_f32(meta >> 16);
    const int pos = pg * kBlock + tq;
    const bool valid = pos >= t0 && pos < t1;
    float codes[kGroup];
#pragma unroll
    for (int mm = 0; mm < 16; ++mm) {
      const uint32_t half = (kw[mm >> 1] >> (16 * (mm & 1))) & 0xFFFF;
      codes[mm] = static_cast<float>((half >> (4 * gk)) & 3);        // channel 16*(2gk)+mm
      codes[16 + mm] = static_cast<float>((half >> (4 * gk + 2)) & 3);  // channel 16*(2gk+1)+mm
    }
    float alpha[MAXG];
#pragma unroll
    for (int j = 0; j < MAXG; ++j) {
      if (j >= gq) {
        alpha[j] = 1.0f;
        continue;
      }
      float dot = 0.0f;
#pragma unroll
      for (int mm = 0; mm < 16; ++mm) {
        dot = fmaf(qs[j][32 * gk + mm], codes[mm], dot);
        dot = fmaf(qs[j][32 * gk + 16 + mm], codes[16 + mm], dot);
      }
      float logit = ks * dot + kz * qsum[j][gk];
      logit += __shfl_xor(logit, 1);
      logit += __shfl_xor(logit, 2);
      logit = valid ? logit : -INFINITY;
      float pmax = logit;
#pragma unroll
      for (int off = 4; off < 64; off <<= 1) pmax = fmaxf(pmax, __shfl_xor(pmax, off));
      const float m_new = fmaxf(m_run[j], pmax);
      const float al = m_new == -INFINITY ? 1.0f : exp2f(m_run[j] - m_new);
      const float p = valid ? exp2f(logit - m_new) : 0.0f;
      float ps = gk == 0 ? p : 0.0f;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) ps += __shfl_xor(ps, off);
      l_run[j] = l_run[j] * al + ps;
      m_run[j] = m_new;
      alpha[j] = al;
      if (gk == 0) pbuf[w][j][tq] = p;
    }
    wave_lds_sync();

    // ---- value accumulation for channels c0, c0+1
    const uint4* vc = reinterpret_cast<const uint4*>(rec + kOffVCodes + 32 * m0);
    const uint4 va = vc[0], vb = vc[1], vc2 = vc[2], vd = vc[3];  // halves m0 (tokens 0..15), m0+1
    const uint32_t hv0[8] = {va.x, va.y, va.z, va.w, vb.x, vb.y, vb.z, vb.w};
    const uint32_t hv1[8] = {vc2.x, vc2.y, vc2.z, vc2.w, vd.x, vd.y, vd.z, vd.w};
    const uint4* vsp = reinterpret_cast<const uint4*>(rec + Lay::kOffVScale + 32 * (NG == 4 ? gv : 0));
    const uint4* vzp = reinterpret_cast<const uint4*>(rec + Lay::kOffVZero + 32 * (NG == 4 ? gv : 0));
    const uint4 s0 = vsp[0], s1 = vsp[1], z0 = vzp[0], z1 = vzp[1];
    const uint32_t sw[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
    const uint32_t zw[8] = {z0.x, z0.y, z0.z, z0.w, z1.x, z1.y, z1.z, z1.w};
#pragma unroll
    for (int j = 0; j < MAXG; ++j) {
      o0[j] *= alpha[j];
      o1[j] *= alpha[j];
    }
#pragma unroll
    for (int t = 0; t < kBlock; ++t) {
      const int sh = 16 * (t & 1);
      const float vs = f16_bits_to_f32((sw[t >> 1] >> sh) & 0xFFFF);
      const float vz = f16_bits_to_f32((zw[t >> 1] >> sh) & 0xFFFF);
      const float x0 = fmaf(static_cast<float>((hv0[t >> 1] >> (sh + 2 * pv)) & 3), vs, vz);
      const float x1 = fmaf(static_cast<float>((hv1[t >> 1] >> (sh + 2 * pv)) & 3), vs, vz);
#pragma unroll
      for (int j = 0; j < MAXG; ++j) {
        if (j < gq) {
          const float p = pbuf[w][j][t];
          o0[j] = fmaf(p, x0, o0[j]);
          o1[j] = fmaf(p, x1, o1[j]);
        }
      }
    }
    wave_lds_sync();
  }

  // ---- merge the four wave states of the block
#pragma unroll
  for (int j = 0; j < MAXG; ++j) {
    if (j < gq) {
      if (l == 0) {
        wstate[w][j][0] = m_run[j];
        wstate[w][j][1] = l_run[j];
      }
      wout[w][j][c0] = o0[j];
      wout[w][j][c0 + 1] = o1[j];
    }
  }
  __syncthreads();
  for (int i = tid; i < gq * kHeadDim; i += blockDim.x) {
    const int j = i / kHeadDim, c = i % kHeadDim;
    float M = -INFINITY;
#pragma unroll
    for (int ww = 0; ww < kWaves; ++ww) M = fmaxf(M, wstate[ww][j][0]);
    float lsum = 0.0f, osum = 0.0f;
#pragma unroll
    for (int ww = 0; ww < kWaves; ++ww) {
      const float mw = wstate[ww][j][0];
      const float f = mw == -INFINITY ? 0.0f : exp2f(mw - M);
      lsum = fmaf(f, wstate[ww][j][1], lsum);
      osum = fmaf(f, wout[ww][j][c], osum);
    }
    float* dst = a.part + (((size_t)b * a.n_chunks + chunk) * a.Hq + h * gq + j) * kPartStride;
    if (c == 0) {
      dst[0] = M;
      dst[1] = lsum;
    }
    dst[4 + c] = osum;
  }
}

template <int NG>
static void launch_valu_ng(const DecodeArgs& a, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  dim3 grid(a.n_chunks, a.H, a.B);
  if (a.gq <= 1)
    hipExtLaunchKernelGGL((decode_split_valu_kernel<1, NG>), grid, dim3(256), 0, s, ev0, ev1, 0, a);
  else if (a.gq <= 2)
    hipExtLaunchKernelGGL((decode_split_valu_kernel<2, NG>), grid, dim3(256), 0, s, ev0, ev1, 0, a);
  else if (a.gq <= 4)
    hipExtLaunchKernelGGL((decode_split_valu_kernel<4, NG>), grid, dim3(256), 0, s, ev0, ev1, 0, a);
  else if (a.gq <= 8)
    hipExtLaunchKernelGGL((decode_split_valu_kernel<8, NG>), grid, dim3(256), 0, s, ev0, ev1, 0, a);
  else
    hipExtLaunchKernelGGL((decode_split_valu_kernel<16, NG>), grid, dim3(256), 0, s, ev0, ev1, 0, a);
}

hipError_t launch_decode_split_valu(const DecodeArgs& a, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  if (a.groups == 1)
    launch_valu_ng<1>(a, s, ev0, ev1);
  else
    launch_valu_ng<4>(a, s, ev0, ev1);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------------------------
// Merge the chunk partials of each (sequence, query head) with a log-sum-exp reduction, then
// undo the value rotation: o = o' R_V^T (skipped when W_O arrives pre-folded with R_V).
// Block (sequence, KV head), thread c = channel.
__global__ __launch_bounds__(128) void merge_kernel(DecodeArgs a, int unrotate, float* __restrict__ out,
                                                    uint16_t* __restrict__ ob, int fmt) {
  __shared__ float os[kHeadDim];
  const int b = blockIdx.x, h = blockIdx.y, c = threadIdx.x;
  const int L = seq_len(a, b);
  const int nch = (L + a.chunk_tokens - 1) / a.chunk_tokens;
  const float* Rv = a.R_v + (size_t)h * kHeadDim * kHeadDim;
  for (int jj = 0; jj < a.gq; ++jj) {
    const int j = h * a.gq + jj;
    const float* part = a.part + ((size_t)b * a.n_chunks * a.Hq + j) * kPartStride;
    const size_t stride = (size_t)a.Hq * kPartStride;
    // the BF16-window partials (when there are some) join the chunk partials
    float wm[kWinMaxSlices], wl[kWinMaxSlices], wo[kWinMaxSlices];
    float M = -INFINITY;
#pragma unroll
    for (int s = 0; s < kWinMaxSlices; ++s) {
      wm[s] = -INFINITY;
      wl[s] = wo[s] = 0.0f;
      if (a.wpart && s < a.win_slices) {
        const float* wp = a.wpart + (((size_t)s * a.B + b) * a.Hq + j) * kPartStride;
        wm[s] = wp[0];
        wl[s] = wp[1];
        wo[s] = wp[4 + c];
      }
      M = fmaxf(M, wm[s]);
    }
    for (int i = 0; i < nch; ++i) M = fmaxf(M, part[i * stride]);
    float lsum = 0.0f, osum = 0.0f;  // osum: the INT2 part only (the window's o is in another basis)
#pragma unroll
    for (int s = 0; s < kWinMaxSlices; ++s)
      if (wm[s] != -INFINITY) lsum = fmaf(exp2f(wm[s] - M), wl[s], lsum);
    for (int i = 0; i < nch; ++i) {
      const float mi = part[i * stride];
      const float f = mi == -INFINITY ? 0.0f : exp2f(mi - M);
      lsum = fmaf(f, part[i * stride + 1], lsum);
      osum = fmaf(f, part[i * stride + 4 + c], osum);
    }
    const float val = lsum > 0.0f ? osum / lsum : 0.0f;
    float res = val;
    if (a.wpart) {
      // the window part (model basis) joins in the output's basis: o = o_int2 R_V^T + o_win, or
      // o' = o_int2 + o_win R_V for a folded W_O
      float ow = 0.0f;
#pragma unroll
      for (int s = 0; s < kWinMaxSlices; ++s)
        if (wm[s] != -INFINITY) ow = fmaf(exp2f(wm[s] - M), wo[s], ow);
      ow = lsum > 0.0f ? ow / lsum : 0.0f;
      const float oi = val;
      os[c] = unrotate ? oi : ow;
      __syncthreads();
      float acc = unrotate ? ow : oi;
      if (unrotate) {
        const float4* row = reinterpret_cast<const float4*>(Rv + (size_t)c * kHeadDim);
#pragma unroll 8
        for (int i = 0; i < kHeadDim / 4; ++i) {
          const float4 r = row[i];
          acc = fmaf(os[4 * i], r.x, acc);
          acc = fmaf(os[4 * i + 1], r.y, acc);
          acc = fmaf(os[4 * i + 2], r.z, acc);
          acc = fmaf(os[4 * i + 3], r.w, acc);
        }
      } else {
#pragma unroll 8
        for (int i = 0; i < kHeadDim; ++i) acc = fmaf(os[i], Rv[(size_t)i * kHeadDim + c], acc);
      }
      res = acc;
      __syncthreads();
    } else if (unrotate) {
      os[c] = val;
      __syncthreads();
      const float4* row = reinterpret_cast<const float4*>(Rv + (size_t)c * kHeadDim);
      float acc = 0.0f;
#pragma unroll 8
      for (int i = 0; i < kHeadDim / 4; ++i) {
        const float4 r = row[i];
        acc = fmaf(os[4 * i], r.x, acc);
        acc = fmaf(os[4 * i + 1], r.y, acc);
        acc = fmaf(os[4 * i + 2], r.z, acc);
        acc = fmaf(os[4 * i + 3], r.w, acc);
      }
      res = acc;
      __syncthreads();
    }
    store_head_out(res, out, ob, fmt, ((size_t)b * a.Hq + j) * kHeadDim + c, (size_t)a.B * a.Hq * kHeadDim);
  }
}

hipError_t launch_merge(const DecodeArgs& a, bool unrotate, float* out, uint16_t* ob, int fmt, hipStream_t s) {
  hipLaunchKernelGGL(merge_kernel, dim3(a.B, a.H), dim3(128), 0, s, a, unrotate ? 1 : 0, out, ob, fmt);
  return hipGetLastError();
}

}  // namespace int2kv
