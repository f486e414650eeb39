// Output-error diagnostics of the INT2 cache (Sec. 3.2; appendix output-space error metrics).
//
// For every sequence b and query head j, against the full-precision keys and values the cache was
// written from:
//   o1 = p^T V         full-precision keys and values (p = softmax of q.k / sqrt(d)),
//   o2 = p~^T V        INT2 keys (p~ = softmax of q.k~ / sqrt(d)), full-precision values,
//   o3 = p~^T V~       INT2 keys and values (the INT2 decode),
// then dy_K = (o2 - o1) W_{O,j}^T and dy_V = (o3 - o2) W_{O,j}^T (so y~ - y = dy_K + dy_V), and the
// four statistics (||dy_K + dy_V||^2, ||dy_K||^2, ||dy_V||^2, <dy_K, dy_V>).
//
// Kernels: a split-context scan (block = context chunk x KV head x sequence, four waves, a page of
// 16 tokens per wave step) that runs both softmaxes over the chunk and accumulates the three value
// sums; a merge of the chunk partials that also undoes the value rotation of o3 (o3 = o3' R_V^T);
// the per-head projection by W_{O,j} (block = query head x 128 rows of W_O, all sequences) with
// partial statistics per row tile; and the sum of those partials. The INT2 scores use the rotated
// query (q R_K) . k^, the full-precision ones q . k with the raw keys: both softmaxes are invariant
// to the key offset mu, which the effective keys k~ = k^ R_K^T + mu carry.
#include "common.h"
#include "kernels.h"

namespace int2kv {

namespace {

constexpr float kOeLogit2 = 1.4426950408889634f * 0.08838834764831845f;  // log2(e)/sqrt(128)
constexpr int kOeWaves = 4;

__device__ __forceinline__ int oe_seq_len(const OutErrArgs& e, int b) {
  int L = e.a.ctx_lens[b];
  L = min(L, e.a.max_ctx);
  L = min(L, e.a.max_blocks * kBlock);
  L = min(L, e.row_cap);
  return max(L, 0);
}

// sum over the 4 lanes of a DPP quad (quad_perm [1, 0, 3, 2] then [2, 3, 0, 1]); every lane gets it
__device__ __forceinline__ float quad_sum4(float x) {
  x += dppf<0xB1>(x);
  return x + dppf<0x4E>(x);
}
// max over the four tokens of a DPP row (lanes 4 tq + gk; rotations by 4 and 8 lanes)
__device__ __forceinline__ float row_max_tokens(float x) {
  x = fmaxf(x, dppf<0x124>(x));
  return fmaxf(x, dppf<0x128>(x));
}
// max over the four DPP rows of values that are already uniform within each row (lanes 0, 16, 32
// and 48 read out as scalars)
__device__ __forceinline__ float rows_max4(float x) {
  const float a = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 0));
  const float b = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 16));
  const float c = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 32));
  const float d = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 48));
  return fmaxf(fmaxf(a, b), fmaxf(c, d));
}
__device__ __forceinline__ float rows_sum4(float x) {
  const float a = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 0));
  const float b = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 16));
  const float c = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 32));
  const float d = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 48));
  return (a + b) + (c + d);
}

__device__ __forceinline__ void oe_wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

}  // namespace

// Block (chunk, KV head h, sequence b). Lane roles as in the vector-ALU decode scan: for the scores,
// token tq = l / 4 of the page and 32-channel quarter gk = l % 4; for the values, channels 2l, 2l+1.
template <int MAXG, int NG>
__global__ __launch_bounds__(256, MAXG <= 4 ? 4 : 1) void outerr_scan_kernel(OutErrArgs e) {
  using Lay = Rec<NG>;
  const DecodeArgs& a = e.a;
  __shared__ float qf[MAXG][kHeadDim];       // q (model basis), base-2 logit units
  __shared__ float qr[MAXG][kHeadDim];       // q R_K, base-2 logit units
  __shared__ float qsum[MAXG][kGroups];      // sums of q R_K over each 32-channel quarter
  __shared__ float pb[kOeWaves][2][kBlock][MAXG];   // p of both softmaxes for the page (token-major)
  __shared__ float wst[kOeWaves][MAXG][4];
  __shared__ float wout[kOeWaves][3][MAXG][kHeadDim];

  const int chunk = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int L = oe_seq_len(e, b);
  const int t0 = chunk * a.chunk_tokens;
  const int gq = a.gq, tid = threadIdx.x, w = tid >> 6, l = tid & 63;
  if (t0 >= L) {
    // a chunk past the context: an empty partial (m = -inf) that the merge drops
    for (int i = tid; i < gq; i += blockDim.x) {
      float* dst = e.part + (((size_t)b * a.n_chunks + chunk) * a.Hq + h * gq + i) * kOePartStride;
      dst[0] = -INFINITY;
      dst[2] = -INFINITY;
    }
    return;
  }
  const int t1 = min(L, t0 + a.chunk_tokens);
  for (int i = tid; i < gq * kHeadDim; i += blockDim.x) {
    const int jj = i / kHeadDim, c = i % kHeadDim;
    const size_t q = ((size_t)b * a.Hq + h * gq + jj) * kHeadDim + c;
    qr[jj][c] = a.qrot[q] * kOeLogit2;
    qf[jj][c] = bf16_bits_to_f32(a.q[q]) * kOeLogit2;
  }
  __syncthreads();
  if (tid < gq * kGroups) {
    const int jj = tid / kGroups, g = tid % kGroups;
    float acc = 0.0f;
    for (int c = 0; c < kGroup; ++c) acc += qr[jj][g * kGroup + c];
    qsum[jj][g] = acc;
  }
  __syncthreads();

  // running states: (m, l) of both softmaxes, and the three value sums of channels 2l, 2l+1
  float m1[MAXG], l1[MAXG], m2[MAXG], l2[MAXG], o[3][MAXG][2];
#pragma unroll
  for (int j = 0; j < MAXG; ++j) {
    m1[j] = m2[j] = -INFINITY;
    l1[j] = l2[j] = 0.0f;
#pragma unroll
    for (int r = 0; r < 3; ++r) o[r][j][0] = o[r][j][1] = 0.0f;
  }
  const int tq = l >> 2, gk = l & 3;
  const int c0 = 2 * l, m0 = c0 & 15, pv = c0 >> 4, gv = c0 >> 5;
  const size_t row_stride = (size_t)a.H * kHeadDim;
  const uint16_t* krow0 = e.k_rows + ((size_t)b * e.row_cap * a.H + h) * kHeadDim;
  const uint16_t* vrow0 = e.v_rows + ((size_t)b * e.row_cap * a.H + h) * kHeadDim;

  const int pg0 = t0 / kBlock, pg1 = (t1 + kBlock - 1) / kBlock;
  for (int pg = pg0 + w; pg < pg1; pg += kOeWaves) {
    const int blk = a.block_table[(size_t)b * a.max_blocks + pg];
    if (blk < 0 || blk >= a.num_blocks) continue;  // uniform per wave
    const uint8_t* rec = a.pool + ((size_t)blk * a.H + h) * Lay::kBytes;
    const int pos = pg * kBlock + tq;
    const bool valid = pos >= t0 && pos < t1;
    const int posc = min(max(pos, t0), t1 - 1);  // a row inside the caller's store

    // ---- INT2 and full-precision scores of token tq over the lane's channel quarter gk: half mm of the
    // token's code words holds channels 32 gk + mm (bits 4 gk) and 32 gk + 16 + mm (bits 4 gk + 2); the
    // codes and the raw key values are unpacked four halves at a time, each chunk feeding every head
    const uint4* kc = reinterpret_cast<const uint4*>(rec + kOffKCodes + 32 * tq);
    const uint4 k0 = kc[0], k1 = kc[1];
    const uint32_t kw[8] = {k0.x, k0.y, k0.z, k0.w, k1.x, k1.y, k1.z, k1.w};
    const uint32_t meta =
        *reinterpret_cast<const uint32_t*>(rec + Lay::kOffKMeta + 4 * NG * tq + 4 * (NG == 4 ? gk : 0));
    const float ks = f16_bits_to_f32(meta & 0xFFFF), kz = f16_bits_to_f32(meta >> 16);
    uint32_t kraw[16];  // the token's raw key row, channels 32 gk .. 32 gk + 31 (two per word)
    {
      const uint4* kp = reinterpret_cast<const uint4*>(krow0 + (size_t)posc * row_stride + 32 * gk);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const uint4 x = kp[u];
        kraw[4 * u] = x.x;
        kraw[4 * u + 1] = x.y;
        kraw[4 * u + 2] = x.z;
        kraw[4 * u + 3] = x.w;
      }
    }
    auto kf = [&](int c) {  // raw key value of channel 32 gk + c
      return __uint_as_float((c & 1) ? (kraw[c >> 1] & 0xFFFF0000u) : (kraw[c >> 1] << 16));
    };
    float d1[MAXG], d2[MAXG];
#pragma unroll
    for (int j = 0; j < MAXG; ++j) d1[j] = d2[j] = 0.0f;
#pragma unroll
    for (int mc = 0; mc < 16; mc += 4) {
      float cl[4], chi[4], fl[4], fh[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int mm = mc + i;
        const uint32_t half = (kw[mm >> 1] >> (16 * (mm & 1))) & 0xFFFF;
        cl[i] = static_cast<float>((half >> (4 * gk)) & 3);       // channel 32 gk + mm
        chi[i] = static_cast<float>((half >> (4 * gk + 2)) & 3);  // channel 32 gk + 16 + mm
        fl[i] = kf(mm);
        fh[i] = kf(16 + mm);
      }
#pragma unroll
      for (int j = 0; j < MAXG; ++j) {
        if (j >= gq) continue;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int mm = mc + i;
          d2[j] = fmaf(qr[j][32 * gk + mm], cl[i], d2[j]);
          d2[j] = fmaf(qr[j][32 * gk + 16 + mm], chi[i], d2[j]);
          d1[j] = fmaf(qf[j][32 * gk + mm], fl[i], d1[j]);
          d1[j] = fmaf(qf[j][32 * gk + 16 + mm], fh[i], d1[j]);
        }
      }
    }
    float al1[MAXG], al2[MAXG];
#pragma unroll
    for (int j = 0; j < MAXG; ++j) {
      al1[j] = al2[j] = 1.0f;
      if (j >= gq) continue;
      // the token's scores: sums over its four quarter lanes (a DPP quad)
      float s2 = quad_sum4(ks * d2[j] + kz * qsum[j][gk]);
      float s1 = quad_sum4(d1[j]);
      s1 = valid ? s1 : -INFINITY;
      s2 = valid ? s2 : -INFINITY;
      // page maxima: over the four tokens of each DPP row, then the rows
      const float x1 = rows_max4(row_max_tokens(s1)), x2 = rows_max4(row_max_tokens(s2));
      const float n1 = fmaxf(m1[j], x1), n2 = fmaxf(m2[j], x2);
      al1[j] = n1 == -INFINITY ? 1.0f : exp2f(m1[j] - n1);
      al2[j] = n2 == -INFINITY ? 1.0f : exp2f(m2[j] - n2);
      const float p1 = valid ? exp2f(s1 - n1) : 0.0f, p2 = valid ? exp2f(s2 - n2) : 0.0f;
      // page sums of p: one lane per token (gk = 0), over each DPP row, then the rows
      const float ps1 = rows_sum4(row_sum16(gk == 0 ? p1 : 0.0f));
      const float ps2 = rows_sum4(row_sum16(gk == 0 ? p2 : 0.0f));
      l1[j] = l1[j] * al1[j] + ps1;
      l2[j] = l2[j] * al2[j] + ps2;
      m1[j] = n1;
      m2[j] = n2;
      if (gk == 0) {
        pb[w][0][tq][j] = p1;
        pb[w][1][tq][j] = p2;
      }
    }
    oe_wave_sync();

    // ---- values of channels c0, c0 + 1: INT2 (R_V basis) and full precision (model basis), in two
    // halves of eight tokens (the loads of a half, then its arithmetic)
    const uint4* vc = reinterpret_cast<const uint4*>(rec + kOffVCodes + 32 * m0);  // halves m0, m0 + 1
    const uint4* vsp = reinterpret_cast<const uint4*>(rec + Lay::kOffVScale + 32 * (NG == 4 ? gv : 0));
    const uint4* vzp = reinterpret_cast<const uint4*>(rec + Lay::kOffVZero + 32 * (NG == 4 ? gv : 0));
#pragma unroll
    for (int j = 0; j < MAXG; ++j) {
#pragma unroll
      for (int cc = 0; cc < 2; ++cc) {
        o[0][j][cc] *= al1[j];
        o[1][j][cc] *= al2[j];
        o[2][j][cc] *= al2[j];
      }
    }
#pragma unroll
    for (int H = 0; H < 2; ++H) {
      const uint4 ca = vc[H], cb = vc[2 + H], s4 = vsp[H], z4 = vzp[H];  // tokens 8 H .. 8 H + 7
      const uint32_t hv0[4] = {ca.x, ca.y, ca.z, ca.w}, hv1[4] = {cb.x, cb.y, cb.z, cb.w};
      const uint32_t sw[4] = {s4.x, s4.y, s4.z, s4.w}, zw[4] = {z4.x, z4.y, z4.z, z4.w};
      uint32_t vf[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int pt = min(max(pg * kBlock + 8 * H + i, t0), t1 - 1);
        vf[i] = *reinterpret_cast<const uint32_t*>(vrow0 + (size_t)pt * row_stride + c0);
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int t = 8 * H + i, sh = 16 * (i & 1);
        const float vs = f16_bits_to_f32((sw[i >> 1] >> sh) & 0xFFFF);
        const float vz = f16_bits_to_f32((zw[i >> 1] >> sh) & 0xFFFF);
        const float x0 = fmaf(static_cast<float>((hv0[i >> 1] >> (sh + 2 * pv)) & 3), vs, vz);
        const float x1 = fmaf(static_cast<float>((hv1[i >> 1] >> (sh + 2 * pv)) & 3), vs, vz);
        const float r0 = __uint_as_float(vf[i] << 16), r1 = __uint_as_float(vf[i] & 0xFFFF0000u);
#pragma unroll
        for (int j = 0; j < MAXG; ++j) {
          if (j < gq) {
            const float p1 = pb[w][0][t][j], p2 = pb[w][1][t][j];
            o[0][j][0] = fmaf(p1, r0, o[0][j][0]);
            o[0][j][1] = fmaf(p1, r1, o[0][j][1]);
            o[1][j][0] = fmaf(p2, r0, o[1][j][0]);
            o[1][j][1] = fmaf(p2, r1, o[1][j][1]);
            o[2][j][0] = fmaf(p2, x0, o[2][j][0]);
            o[2][j][1] = fmaf(p2, x1, o[2][j][1]);
          }
        }
      }
    }
    oe_wave_sync();
  }

  // ---- merge the four wave states into the chunk's partial
#pragma unroll
  for (int j = 0; j < MAXG; ++j) {
    if (j < gq) {
      if (l == 0) {
        wst[w][j][0] = m1[j];
        wst[w][j][1] = l1[j];
        wst[w][j][2] = m2[j];
        wst[w][j][3] = l2[j];
      }
#pragma unroll
      for (int r = 0; r < 3; ++r) {
        wout[w][r][j][c0] = o[r][j][0];
        wout[w][r][j][c0 + 1] = o[r][j][1];
      }
    }
  }
  __syncthreads();
  for (int i = tid; i < gq * kHeadDim; i += blockDim.x) {
    const int j = i / kHeadDim, c = i % kHeadDim;
    float M1 = -INFINITY, M2 = -INFINITY;
#pragma unroll
    for (int ww = 0; ww < kOeWaves; ++ww) {
      M1 = fmaxf(M1, wst[ww][j][0]);
      M2 = fmaxf(M2, wst[ww][j][2]);
    }
    float L1 = 0.0f, L2 = 0.0f, A[3] = {0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int ww = 0; ww < kOeWaves; ++ww) {
      const float f1 = wst[ww][j][0] == -INFINITY ? 0.0f : exp2f(wst[ww][j][0] - M1);
      const float f2 = wst[ww][j][2] == -INFINITY ? 0.0f : exp2f(wst[ww][j][2] - M2);
      L1 = fmaf(f1, wst[ww][j][1], L1);
      L2 = fmaf(f2, wst[ww][j][3], L2);
      A[0] = fmaf(f1, wout[ww][0][j][c], A[0]);
      A[1] = fmaf(f2, wout[ww][1][j][c], A[1]);
      A[2] = fmaf(f2, wout[ww][2][j][c], A[2]);
    }
    float* dst = e.part + (((size_t)b * a.n_chunks + chunk) * a.Hq + h * gq + j) * kOePartStride;
    if (c == 0) {
      dst[0] = M1;
      dst[1] = L1;
      dst[2] = M2;
      dst[3] = L2;
    }
#pragma unroll
    for (int r = 0; r < 3; ++r) dst[4 + r * kHeadDim + c] = A[r];
  }
}

// Block (sequence b, query head j), thread c: the chunk partials of the head merged into o1, o2
// (model basis) and o3' (R_V basis), o3 = o3' R_V^T, then do = (o2 - o1, o3 - o2).
__global__ __launch_bounds__(128) void outerr_merge_kernel(OutErrArgs e) {
  const DecodeArgs& a = e.a;
  __shared__ float os[kHeadDim];
  const int b = blockIdx.x, j = blockIdx.y, c = threadIdx.x, h = j / a.gq;
  const int L = oe_seq_len(e, b);
  const int nch = (L + a.chunk_tokens - 1) / a.chunk_tokens;
  const float* Rv = a.R_v + (size_t)h * kHeadDim * kHeadDim;
  const float* part = e.part + ((size_t)b * a.n_chunks * a.Hq + j) * kOePartStride;
  const size_t stride = (size_t)a.Hq * kOePartStride;
  float M1 = -INFINITY, M2 = -INFINITY;
  for (int i = 0; i < nch; ++i) {
    M1 = fmaxf(M1, part[i * stride]);
    M2 = fmaxf(M2, part[i * stride + 2]);
  }
  float L1 = 0.0f, L2 = 0.0f, A0 = 0.0f, A1 = 0.0f, A2 = 0.0f;
  for (int i = 0; i < nch; ++i) {
    const float* p = part + i * stride;
    const float f1 = p[0] == -INFINITY ? 0.0f : exp2f(p[0] - M1);
    const float f2 = p[2] == -INFINITY ? 0.0f : exp2f(p[2] - M2);
    L1 = fmaf(f1, p[1], L1);
    L2 = fmaf(f2, p[3], L2);
    A0 = fmaf(f1, p[4 + c], A0);
    A1 = fmaf(f2, p[4 + kHeadDim + c], A1);
    A2 = fmaf(f2, p[4 + 2 * kHeadDim + c], A2);
  }
  const float o1 = L1 > 0.0f ? A0 / L1 : 0.0f;
  const float o2 = L2 > 0.0f ? A1 / L2 : 0.0f;
  os[c] = L2 > 0.0f ? A2 / L2 : 0.0f;
  __syncthreads();
  const float4* row = reinterpret_cast<const float4*>(Rv + (size_t)c * kHeadDim);
  float o3 = 0.0f;
#pragma unroll 8
  for (int i = 0; i < kHeadDim / 4; ++i) {
    const float4 r = row[i];
    o3 = fmaf(os[4 * i], r.x, o3);
    o3 = fmaf(os[4 * i + 1], r.y, o3);
    o3 = fmaf(os[4 * i + 2], r.z, o3);
    o3 = fmaf(os[4 * i + 3], r.w, o3);
  }
  // do as three bf16 terms (the projection's matrix-core operands): truncation leaves each remainder
  // exact, and the third takes the last 8 significant bits, so t0 + t1 + t2 = do exactly
  const size_t plane = (size_t)a.B * a.Hq * 2 * kHeadDim;
  uint16_t* d = e.dov + ((size_t)b * a.Hq + j) * 2 * kHeadDim;
  const float dv[2] = {o2 - o1, o3 - o2};
#pragma unroll
  for (int kv = 0; kv < 2; ++kv) {
    const uint32_t b0 = __float_as_uint(dv[kv]) & 0xFFFF0000u;
    const float r1 = dv[kv] - __uint_as_float(b0);
    const uint32_t b1 = __float_as_uint(r1) & 0xFFFF0000u;
    const float r2 = r1 - __uint_as_float(b1);
    d[kv * kHeadDim + c] = (uint16_t)(b0 >> 16);
    d[plane + kv * kHeadDim + c] = (uint16_t)(b1 >> 16);
    d[2 * plane + kv * kHeadDim + c] = (uint16_t)(__float_as_uint(r2) >> 16);
  }
}

typedef float oe_f4_t __attribute__((ext_vector_type(4)));

// Block (query head j, tile of kOeRowTile rows of W_O), four waves: dy[b][j][{K, V}][row] =
// do[b][j][{K, V}] . W_O[row][j * 128 ..] for every sequence, and the tile's partial statistics, on
// the bf16 matrix cores with do as three exact bf16 terms (fp32 products and accumulation, as an
// fp32 product would give): 16 x 16 x 32 steps, lane l holds A[l % 16][8 (l / 16) ..] and
// B[8 (l / 16) ..][l % 16], D[4 (l / 16) + v][l % 16] is element v of its accumulator. M: the 2B rows
// m = 2 b + {0: K, 1: V} of do, 16 at a time; N: wave w's two 16-row tiles of the block's rows; K:
// the head's 128 channels in four blocks of 32 (lane: channels 32 i + 8 (l / 16) .. + 7 of its do
// and W_O rows).
constexpr int kOeNT = kOeRowTile / 64;  // 16-row N tiles per wave
typedef __bf16 oe_bf16x8_t __attribute__((ext_vector_type(8)));
__global__ __launch_bounds__(256) void outerr_proj_kernel(OutErrArgs e, const uint16_t* __restrict__ W_o,
                                                          int d_model, float* __restrict__ dy,
                                                          float* __restrict__ spart, int ntiles) {
  const DecodeArgs& a = e.a;
  __shared__ float red[4][8][4];  // [wave][sequence of the M tile][statistic]
  const int j = blockIdx.x, tile = blockIdx.y, tid = threadIdx.x;
  const int w = tid >> 6, l = tid & 63, li = l & 15, lk = l >> 4;
  int n[kOeNT];
  bool have[kOeNT];
  oe_bf16x8_t wb[kOeNT][4];
#pragma unroll
  for (int nt = 0; nt < kOeNT; ++nt) {
    n[nt] = tile * kOeRowTile + 16 * (kOeNT * w + nt) + li;  // this lane's W_O row of N tile nt
    have[nt] = n[nt] < d_model;
    const uint4* wp = reinterpret_cast<const uint4*>(W_o + (size_t)(have[nt] ? n[nt] : 0) * a.Hq * kHeadDim +
                                                     (size_t)j * kHeadDim + 8 * lk);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      wb[nt][i] = __builtin_bit_cast(oe_bf16x8_t, have[nt] ? wp[4 * i] : make_uint4(0, 0, 0, 0));
  }
  const int M = 2 * a.B;
  const size_t plane = (size_t)a.B * a.Hq * 2 * kHeadDim;
  for (int m0 = 0; m0 < M; m0 += 16) {
    const int m = m0 + li, mc = m < M ? m : 0;
    oe_bf16x8_t da[3][4];
    {
      const uint16_t* dp = e.dov + (((size_t)(mc >> 1) * a.Hq + j) * 2 + (mc & 1)) * kHeadDim + 8 * lk;
#pragma unroll
      for (int t = 0; t < 3; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          da[t][i] = __builtin_bit_cast(
              oe_bf16x8_t, m < M ? *reinterpret_cast<const uint4*>(dp + t * plane + 32 * i) : make_uint4(0, 0, 0, 0));
    }
    oe_f4_t acc[kOeNT];
#pragma unroll
    for (int nt = 0; nt < kOeNT; ++nt) acc[nt] = oe_f4_t{0.f, 0.f, 0.f, 0.f};
    // smallest term first
#pragma unroll
    for (int t = 2; t >= 0; --t)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int nt = 0; nt < kOeNT; ++nt)
          acc[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(da[t][i], wb[nt][i], acc[nt], 0, 0, 0);
    // acc[nt][v]: do row m0 + 4 lk + v, i.e. sequence m0 / 2 + 2 lk + v / 2, K (v even) or V (v odd)
#pragma unroll
    for (int hb = 0; hb < 2; ++hb) {
      const int b = m0 / 2 + 2 * lk + hb;
      float st[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int nt = 0; nt < kOeNT; ++nt) {
        const float yk = acc[nt][2 * hb], yv = acc[nt][2 * hb + 1];  // 0 past d_model or past the batch
        if (dy && have[nt] && b < a.B) {
          float* o = dy + ((size_t)b * a.Hq + j) * 2 * d_model;
          o[n[nt]] = yk;
          o[d_model + n[nt]] = yv;
        }
        st[0] += (yk + yv) * (yk + yv);
        st[1] += yk * yk;
        st[2] += yv * yv;
        st[3] += yk * yv;
      }
#pragma unroll
      for (int k = 0; k < 4; ++k)
#pragma unroll
        for (int off = 1; off < 16; off <<= 1) st[k] += __shfl_xor(st[k], off);
      if (li == 0)
#pragma unroll
        for (int k = 0; k < 4; ++k) red[w][2 * lk + hb][k] = st[k];
    }
    __syncthreads();
    if (tid < 32) {
      const int bb = tid >> 2, k = tid & 3, b = m0 / 2 + bb;
      if (b < a.B)
        spart[(((size_t)b * a.Hq + j) * ntiles + tile) * 4 + k] =
            ((red[0][bb][k] + red[1][bb][k]) + red[2][bb][k]) + red[3][bb][k];
    }
    __syncthreads();
  }
}

// Wave per (b, j): lane t sums the row tiles t, t + 64, ... in order, then a fixed butterfly over
// the lanes (deterministic).
__global__ __launch_bounds__(256) void outerr_stats_kernel(const float* __restrict__ spart, float* __restrict__ stats,
                                                           int n, int ntiles) {
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6), l = threadIdx.x & 63;
  if (i >= n) return;  // uniform over the wave
  float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int t = l; t < ntiles; t += 64) {
    const float4 x = *reinterpret_cast<const float4*>(spart + ((size_t)i * ntiles + t) * 4);
    s.x += x.x;
    s.y += x.y;
    s.z += x.z;
    s.w += x.w;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    s.x += __shfl_xor(s.x, off);
    s.y += __shfl_xor(s.y, off);
    s.z += __shfl_xor(s.z, off);
    s.w += __shfl_xor(s.w, off);
  }
  if (l == 0) {  // the caller's stats need only 4-byte alignment
    stats[(size_t)i * 4] = s.x;
    stats[(size_t)i * 4 + 1] = s.y;
    stats[(size_t)i * 4 + 2] = s.z;
    stats[(size_t)i * 4 + 3] = s.w;
  }
}

template <int NG>
static void launch_oe_scan(const OutErrArgs& e, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  const DecodeArgs& a = e.a;
  dim3 grid(a.n_chunks, a.H, a.B);
  if (a.gq <= 1)
    hipExtLaunchKernelGGL((outerr_scan_kernel<1, NG>), grid, dim3(256), 0, s, ev0, ev1, 0, e);
  else if (a.gq <= 2)
    hipExtLaunchKernelGGL((outerr_scan_kernel<2, NG>), grid, dim3(256), 0, s, ev0, ev1, 0, e);
  else if (a.gq <= 4)
    hipExtLaunchKernelGGL((outerr_scan_kernel<4, NG>), grid, dim3(256), 0, s, ev0, ev1, 0, e);
  else if (a.gq <= 8)
    hipExtLaunchKernelGGL((outerr_scan_kernel<8, NG>), grid, dim3(256), 0, s, ev0, ev1, 0, e);
  else
    hipExtLaunchKernelGGL((outerr_scan_kernel<16, NG>), grid, dim3(256), 0, s, ev0, ev1, 0, e);
}

hipError_t launch_output_error(const OutErrArgs& e, const uint16_t* W_o, int d_model, float* stats, float* dy,
                               hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  const DecodeArgs& a = e.a;
  hipError_t err = launch_qrot(a, s);
  if (err != hipSuccess) return err;
  if (a.groups == 1)
    launch_oe_scan<1>(e, s, ev0, ev1);
  else
    launch_oe_scan<4>(e, s, ev0, ev1);
  hipLaunchKernelGGL(outerr_merge_kernel, dim3(a.B, a.Hq), dim3(128), 0, s, e);
  const int ntiles = (d_model + kOeRowTile - 1) / kOeRowTile;
  hipLaunchKernelGGL(outerr_proj_kernel, dim3(a.Hq, ntiles), dim3(256), 0, s, e, W_o, d_model, dy, e.spart,
                     ntiles);
  const int n = a.B * a.Hq;
  hipLaunchKernelGGL(outerr_stats_kernel, dim3((n + 3) / 4), dim3(256), 0, s, e.spart, stats, n, ntiles);
  return hipGetLastError();
}

}  // namespace int2kv
