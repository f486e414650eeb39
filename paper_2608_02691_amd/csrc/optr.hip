// OptR offline calibration on the GPU (Sec. 4.2 - 4.5; Algorithm 1 of the appendix), in fp64.
//
// Per KV head h, with R = R^0 exp(A - A^T):
//   rows:        x_s = k_s - mu (keys) or v_s (values), bf16 inputs, exact in fp64
//   rotation:    z_s = x_s R, rounded to fp32 and quantized by the cache's quantizer (codes, fp16
//                scale and zero); zhat_s = code * s + z (exact); mask = element inside its group's
//                clipped range [c mn, c mx] (the straight-through estimator of eq:OptR_ste)
//   effective:   xeff_s = zhat_s R^T
//   key loss:    rows (t, j) over the final n_last positions; logits over s <= t with xeff for
//                tokens read from INT2 (sink <= s <= t - recent) and x otherwise;
//                KL(p || p^K) + lambda ||(p^K - p)^T V W_{O,j}^T||^2 / d_model, averaged over rows,
//                the output term as dO^T M_j dO with the Gram matrix M_j = W_{O,j}^T W_{O,j}
//   value loss:  ||p^Khat^T (Veff - V) W_{O,j}^T||^2 / d_model under fixed key probabilities
// Gradients by hand: dL/dlogit, then dL/dxeff (per token, summed over its rows), dL/dzhat =
// G R masked, dL/dR = X^T (mask . G R) + G^T Zhat, dL/dE = R0^T dL/dR for E = exp(S), dL/dS as the
// Frechet derivative of exp at S^T applied to dL/dE (the upper-right block of the exponential of
// [[S^T, dL/dE], [0, S^T]]), and dL/dA = dL/dS - dL/dS^T.
// exp: scaling by 2^-s until ||S||_1 <= 1/2, a Taylor polynomial of 14 terms (truncation below
// 1e-17 relative), then s squarings; one work-group per KV head, products through LDS tiles.
#include <vector>

#include "common.h"
#include "kernels.h"

namespace int2kv {

namespace {

constexpr int kD = kHeadDim;
constexpr int kMat = kD * kD;
constexpr int kExpTerms = 14;
constexpr int kExpThreads = 1024;

typedef double f64x4 __attribute__((ext_vector_type(4)));

// fp64 matrix-core step D += A B for 16 x 4 by 4 x 16 operands: lane l holds A[l % 16][l / 16] and
// B[l / 16][l % 16]; D[l / 16 + 4 v][l % 16] is element v of its accumulator.
__device__ __forceinline__ f64x4 mfma64(double a, double b, f64x4 d) {
  return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, d, 0, 0, 0);
}
constexpr double kInvSqrtD = 0.08838834764831845;  // 1 / sqrt(128)

__device__ __forceinline__ double bf16d(uint16_t b) { return (double)__uint_as_float((uint32_t)b << 16); }

__device__ __forceinline__ double wave_sum(double x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off);
  return x;
}

// block-wide reductions over blockDim.x threads (a multiple of 64, at most 1024); red: 16 doubles
__device__ double block_sum(double x, double* red) {
  x = wave_sum(x);
  const int w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = x;
  __syncthreads();
  double t = 0.0;
  for (int i = 0; i < nw; ++i) t += red[i];  // fixed order: deterministic
  return t;
}

__device__ double block_max(double x, double* red) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x = fmax(x, __shfl_xor(x, off));
  const int w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = x;
  __syncthreads();
  double t = red[0];
  for (int i = 1; i < nw; ++i) t = fmax(t, red[i]);
  return t;
}

// Offset of token s, KV head h in the per-head rows of the workspace ([H, T, 128]: each head's
// rows contiguous), as against the traces' [T, H, 128].
__device__ __forceinline__ size_t hrow(const CalSet& S, int s, int h) { return ((size_t)h * S.T + s) * kD; }

__device__ __forceinline__ bool int2_token(int s, int t, int sink, int recent) {
  return s >= sink && s <= t - recent;
}

__device__ __forceinline__ void bf16x8_to_f64(uint4 u, double (&d)[8]) {
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    d[2 * i] = (double)__uint_as_float(w[i] << 16);
    d[2 * i + 1] = (double)__uint_as_float(w[i] & 0xFFFF0000u);
  }
}

// ---------------------------------------------------------------------------------------------
// Rows times a 128 x 128 matrix on the fp64 matrix cores, as out^T = Bm^T y^T: M = the 128 output
// channels (eight 16-row tiles), N = the wave's 16 rows y (lane l holds row l % 16), K = the 128
// input channels. The lane's B operand at step s is ya[s] = y[row][k(s)], k(4 q + d) = 32 (l / 16) +
// 4 q + d (KMAP 0: each lane reads 32 contiguous channels of its row) or 16 q + 4 d + l / 16 (KMAP 1:
// the channels this layout leaves in a lane, see below); Bm goes through Bs (LDS, 16 rows x
// kBsStride) 16 rows at a time. Result element v of acc[ct]: channel 16 ct + l / 16 + 4 v of row
// l % 16. Contains block barriers: every thread of the block calls it.
constexpr int kBsStride = 132;  // doubles per staged row (lane groups l / 16 two banks apart)
template <int KMAP>
__device__ __forceinline__ void mat_t_rows(const double (&ya)[32], const double* __restrict__ Bm, double* Bs,
                                           f64x4 (&acc)[8]) {
  const int tid = threadIdx.x, l = tid & 63, li = l & 15, lk = l >> 4;
#pragma unroll
  for (int q = 0; q < 8; ++q) {  // unrolled: ya is indexed by q
    __syncthreads();
    for (int e = tid; e < 16 * kD; e += blockDim.x) {
      const int rr = e >> 7, col = e & 127;
      const int krow = KMAP == 0 ? 32 * (rr >> 2) + 4 * q + (rr & 3) : 16 * q + rr;
      Bs[rr * kBsStride + col] = Bm[krow * kD + col];
    }
    __syncthreads();
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      const double b = ya[4 * q + d];
      const double* br = Bs + (KMAP == 0 ? 4 * lk + d : 4 * d + lk) * kBsStride + li;
#pragma unroll
      for (int ct = 0; ct < 8; ++ct) acc[ct] = mfma64(br[16 * ct], b, acc[ct]);
    }
  }
}

// y's 32 channels 32 (l / 16) .. + 31 of a row of fp64 storage (zero when !ok).
__device__ __forceinline__ void row_operand_f64(const double* row, bool ok, double (&ya)[32]) {
  const double2* r2 = reinterpret_cast<const double2*>(row + 32 * ((threadIdx.x & 63) >> 4));
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const double2 x = ok ? r2[i] : make_double2(0.0, 0.0);
    ya[2 * i] = x.x;
    ya[2 * i + 1] = x.y;
  }
}

// Rotation and quantization: zhat (the dequantized codes of (x - mu) R, fp64), the in-range mask, and
// the effective rows zhat R^T. Block (128 tokens, KV head), wave w: tokens 16 w .. + 15 (one per lane
// l % 16), every lane group l / 16 a quarter of the channels. A token's quantization group is spread
// over its four lane groups: min / max through two cross-group exchanges.
constexpr int kRotTile = 128;  // tokens per rotation work-group (eight waves of 16)
__global__ __launch_bounds__(512) void cal_rotq_kernel(CalSet S, CalCfg c, int value) {
  __shared__ double Bs[16 * kBsStride];
  const int h = blockIdx.y, tid = threadIdx.x, w = tid >> 6, l = tid & 63, li = l & 15, lk = l >> 4;
  const int tok = blockIdx.x * kRotTile + 16 * w + li;
  const bool ok = tok < S.T;
  const size_t xo = ((size_t)(ok ? tok : 0) * c.H + h) * kD, rowo = hrow(S, ok ? tok : 0, h);
  const uint16_t* X = value ? S.v : S.k;
  double ya[32];
  {
    const uint4* xr = reinterpret_cast<const uint4*>(X + xo + 32 * lk);
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      double d[8];
      bf16x8_to_f64(ok ? xr[g] : make_uint4(0, 0, 0, 0), d);
#pragma unroll
      for (int i = 0; i < 8; ++i)
        ya[8 * g + i] = ok ? d[i] - (value ? 0.0 : (double)c.mu[h * kD + 32 * lk + 8 * g + i]) : 0.0;
    }
  }
  f64x4 acc[8];
#pragma unroll
  for (int ct = 0; ct < 8; ++ct) acc[ct] = f64x4{0.0, 0.0, 0.0, 0.0};
  mat_t_rows<0>(ya, c.R + (size_t)h * kMat, Bs, acc);  // z = (x - mu) R: channel 16 ct + lk + 4 v
  const float clip = value ? c.clip_v : c.clip_k;
  // groups: 32 channels (tiles 2 g, 2 g + 1) or all 128 (one group)
  const int ng = c.ng, tpg = 8 / ng;
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    if (g >= ng) break;
    float mn = INFINITY, mx = -INFINITY;
#pragma unroll
    for (int ct = 0; ct < 8; ++ct) {
      if (ct / tpg != g) continue;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const float x = (float)acc[ct][v];
        mn = fminf(mn, x);
        mx = fmaxf(mx, x);
      }
    }
    mn = fminf(mn, __shfl_xor(mn, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mn = fminf(mn, __shfl_xor(mn, 32));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    uint32_t s_bits, z_bits;
    float zf, inv;
    int2_group_params(mn, mx, clip, s_bits, z_bits, zf, inv);
    const double sd = (double)__half2float(__ushort_as_half((unsigned short)s_bits));
    float lo = mn, hi = mx;
    if (clip != 1.0f) {
#pragma clang fp contract(off)
      lo = clip * mn;
      hi = clip * mx;
    }
#pragma unroll
    for (int ct = 0; ct < 8; ++ct) {
      if (ct / tpg != g) continue;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const float x = (float)acc[ct][v];
        const double zh = (double)int2_code(x, zf, inv) * sd + (double)zf;
        ya[4 * ct + v] = zh;  // the B operand of the second product (KMAP 1)
        if (ok) {
          const size_t o = rowo + 16 * ct + lk + 4 * v;
          S.zhat[o] = zh;
          S.mask[o] = (x >= lo && x <= hi) ? 1 : 0;
        }
      }
    }
  }
#pragma unroll
  for (int ct = 0; ct < 8; ++ct) acc[ct] = f64x4{0.0, 0.0, 0.0, 0.0};
  mat_t_rows<1>(ya, c.Rt + (size_t)h * kMat, Bs, acc);  // effective rows zhat R^T
  if (ok)
#pragma unroll
    for (int ct = 0; ct < 8; ++ct)
#pragma unroll
      for (int v = 0; v < 4; ++v) S.xeff[rowo + 16 * ct + lk + 4 * v] = acc[ct][v];
}

// ---------------------------------------------------------------------------------------------
// The objectives over row tiles.

// The tile kernels take a tile of up to kTileRows rows: 16 / G_q consecutive query positions of
// one sequence with all their query heads (tiles[i] = (sequence, first row, rows, position of the
// first row)), so each key and value row is loaded once for the whole tile. Row r of a tile is
// position t_first + r / G_q, query head h G_q + r % G_q. The row x token and row x channel
// products run on the fp64 matrix cores with the tile's 16 rows as the M dimension.
constexpr int kTileRows = 16;
constexpr int kTileThreads = 256;  // four waves; one token per thread in the softmax passes
constexpr int kDlStride = 18;      // doubles per token of the staged row weights (16-byte rows)


// Row operand of a tile in matrix-core form: lane (li, lk) holds x[row li][32 lk + m], m = 0..31, for
// the contraction over 128 channels taken as 32 steps m whose 4-deep slices are channels 32 k + m
// (k = 0..3); rows li >= nr are zero. From bf16 (queries) or fp64 (row vectors) storage.
__device__ __forceinline__ void rows_operand_bf16(const uint16_t* row, bool ok, int lk, double (&x)[32]) {
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    double d[8];
    bf16x8_to_f64(ok ? *reinterpret_cast<const uint4*>(row + 32 * lk + 8 * g) : make_uint4(0, 0, 0, 0), d);
#pragma unroll
    for (int i = 0; i < 8; ++i) x[8 * g + i] = d[i];
  }
}

// Logits of 16 rows against the 16 tokens of a tile (token li of this lane's B operand): acc +=
// x . y_token with y the token's bf16 row; the same slice convention as rows_operand_*.
__device__ __forceinline__ f64x4 dot_tokens_bf16(const double (&x)[32], const uint16_t* yrow, bool ok, int lk) {
  f64x4 acc = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    double d[8];
    bf16x8_to_f64(ok ? *reinterpret_cast<const uint4*>(yrow + 32 * lk + 8 * g) : make_uint4(0, 0, 0, 0), d);
#pragma unroll
    for (int i = 0; i < 8; ++i) acc = mfma64(x[8 * g + i], d[i], acc);
  }
  return acc;
}
__device__ __forceinline__ f64x4 dot_tokens_f64(const double (&x)[32], const double* yrow, bool ok, int lk) {
  f64x4 acc = {0.0, 0.0, 0.0, 0.0};
  const double2* y2 = reinterpret_cast<const double2*>(yrow + 32 * lk);
#pragma unroll
  for (int g = 0; g < 16; ++g) {
    const double2 y = ok ? y2[g] : make_double2(0.0, 0.0);
    acc = mfma64(x[2 * g], y.x, acc);
    acc = mfma64(x[2 * g + 1], y.y, acc);
  }
  return acc;
}

// Row x channel accumulation: acc[t] (t = 0..7) += A B with A[row li][token lk] = a and
// B[token lk][column li] = y[t], the token's channel 8 li + t. Result element v of acc[t]: row
// lk + 4 v, channel 8 li + t.
__device__ __forceinline__ void acc_channels(f64x4 (&acc)[8], double a, const double (&y)[8]) {
#pragma unroll
  for (int t = 0; t < 8; ++t) acc[t] = mfma64(a, y[t], acc[t]);
}

// Sums the four waves' channel accumulators in the fixed order (w0 + w2) + (w1 + w3) through buf
// (32 KiB of LDS, free on entry) and stores rows r < nr at out + r 128 (row lk + 4 v, channel 8 li + t),
// plus add_w[r] times row r of add when add is given (add_w visible to wave 0 at entry).
__device__ __forceinline__ void sum_waves_store(f64x4 (&acc)[8], double* buf, double* out, int nr,
                                                const double* add = nullptr, const double* add_w = nullptr) {
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63, li = l & 15, lk = l >> 4;
  __syncthreads();
  if (w >= 2)
#pragma unroll
    for (int t = 0; t < 8; ++t)
#pragma unroll
      for (int v = 0; v < 4; ++v) buf[((w - 2) * 32 + 4 * t + v) * 64 + l] = acc[t][v];
  __syncthreads();
  if (w < 2)
#pragma unroll
    for (int t = 0; t < 8; ++t)
#pragma unroll
      for (int v = 0; v < 4; ++v) acc[t][v] += buf[(w * 32 + 4 * t + v) * 64 + l];
  __syncthreads();
  if (w == 1)
#pragma unroll
    for (int t = 0; t < 8; ++t)
#pragma unroll
      for (int v = 0; v < 4; ++v) buf[(4 * t + v) * 64 + l] = acc[t][v];
  __syncthreads();
  if (w == 0)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int r = lk + 4 * v;
      double o[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) o[t] = acc[t][v] + buf[(4 * t + v) * 64 + l];
      if (r < nr && add)
#pragma unroll
        for (int t = 0; t < 8; ++t) o[t] = fma(add_w[r], add[(size_t)r * kD + 8 * li + t], o[t]);
      if (r < nr) {
        double2* dst = reinterpret_cast<double2*>(out + (size_t)r * kD + 8 * li);
#pragma unroll
        for (int i = 0; i < 4; ++i) dst[i] = make_double2(o[2 * i], o[2 * i + 1]);
      }
    }
}

// Row maxima from the matrix-core layout (m4[v]: this lane's value for row lk + 4 v): over the 16
// lanes of each lk group, then over the four waves through red4 ([4][16] doubles). Returns the
// maxima of rows 4 w .. 4 w + 3, the rows wave w owns in the softmax passes.
__device__ __forceinline__ void rows_max(const double (&m4)[4], double* red4, double (&m)[4]) {
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63, li = l & 15, lk = l >> 4;
  double x[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    x[v] = m4[v];
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) x[v] = fmax(x[v], __shfl_xor(x[v], off));
  }
  __syncthreads();
  if (li == 0)
#pragma unroll
    for (int v = 0; v < 4; ++v) red4[w * 16 + lk + 4 * v] = x[v];
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = 4 * w + i;
    m[i] = fmax(fmax(red4[r], red4[16 + r]), fmax(red4[32 + r], red4[48 + r]));
  }
}

// The tile's 4-token steps of a 256-token chunk for wave w: tokens 64 w + k4 + lk, k4 = 0, 4, ..., 60,
// those below end.

// The rotation-independent part of the key objective, once per set: for every row the full-precision
// logits f_s = q.(k_s - mu)/sqrt(d) over its tokens s <= t_r (fc; q.(k - mu) = q.k - q.mu with q.mu once
// per row), p = softmax(f) (pc), lse_f and LW = log-sum-exp of f over the row's tokens held in BF16
// windows (-inf when none) (rc), and W~ = sum over those tokens of exp(f_s - LW) v_s (wt). A window
// token keeps g_s = f_s under every rotation, so the key forward needs only these sums for them.
// Block (tile, KV head), the layout of the key forward.
__global__ __launch_bounds__(kTileThreads) void cal_const_kernel(CalSet S, CalCfg c) {
  constexpr int R = kTileRows;
  __shared__ double qmu[R];
  __shared__ double red4[4 * R];
  __shared__ __align__(16) double dl[kTileThreads * kDlStride];
  const int h = blockIdx.y, tid = threadIdx.x, gq = c.gq;
  const int w = tid >> 6, l = tid & 63, li = l & 15, lk = l >> 4;
  const int4 tile = S.tiles[blockIdx.x];
  const CalSeq sq = S.seqs[tile.x];
  const int row0 = tile.y, nr = tile.z, tf = tile.w, a0 = sq.start, L = sq.len;
  const int tmax = tf + (nr - 1) / gq;
  const size_t pb = (size_t)h * S.pelems + sq.p0 + (size_t)(row0 - sq.row0) * L;  // row r at + r L
  double *fcb = S.fc + pb, *pcb = S.pc + pb;
  double qa[32];
  rows_operand_bf16(S.q + ((size_t)(a0 + tf + li / gq) * c.Hq + h * gq + li % gq) * kD, li < nr, lk, qa);
  {
    double t = 0.0;
#pragma unroll
    for (int m = 0; m < 32; ++m) t = fma(qa[m], (double)c.mu[h * kD + 32 * lk + m], t);
    t += __shfl_xor(t, 16);
    t += __shfl_xor(t, 32);
    if (w == 0 && lk == 0) qmu[li] = t;
  }
  __syncthreads();
  double m4f[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) m4f[v] = -INFINITY;
  for (int tt = w; 16 * tt <= tmax; tt += 4) {
    const int s = 16 * tt + li;
    const bool ok = s <= tmax;
    const f64x4 af = dot_tokens_bf16(qa, S.k + ((size_t)(a0 + s) * c.H + h) * kD, ok, lk);
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int r = lk + 4 * v, tr = tf + r / gq;
      if (r < nr && s <= tr) {
        const double f = (af[v] - qmu[r]) * kInvSqrtD;
        fcb[(size_t)r * L + s] = f;
        m4f[v] = fmax(m4f[v], f);
      }
    }
  }
  const int rb = 4 * w;
  double mf[4];
  rows_max(m4f, red4, mf);  // its barriers also make the logits visible to the whole block
  int tr4[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) tr4[i] = rb + i < nr ? tf + (rb + i) / gq : -1;
  double zf[4], zw[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) zf[i] = zw[i] = 0.0;
  for (int s = l; s <= tmax; s += 64)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (s > tr4[i]) continue;
      const double e = exp(fcb[(size_t)(rb + i) * L + s] - mf[i]);
      zf[i] += e;
      if (!int2_token(s, tr4[i], c.sink, c.recent)) zw[i] += e;
    }
  double lse[4], lw[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    zf[i] = wave_sum(zf[i]);
    zw[i] = wave_sum(zw[i]);
    lse[i] = mf[i] + log(zf[i]);
    lw[i] = zw[i] > 0.0 ? mf[i] + log(zw[i]) : -INFINITY;
  }
  // p, and W~ from the window tokens' weights exp(f - LW) staged in LDS by 256-token chunk
  f64x4 acc[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) acc[t] = f64x4{0.0, 0.0, 0.0, 0.0};
  for (int base = 0; base <= tmax; base += kTileThreads) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int j = 64 * q + l, s = base + j;
      double d[4] = {0.0, 0.0, 0.0, 0.0};
      if (s <= tmax) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if (s > tr4[i]) continue;
          const size_t o = (size_t)(rb + i) * L + s;
          const double f = fcb[o];
          pcb[o] = exp(f - lse[i]);
          if (!int2_token(s, tr4[i], c.sink, c.recent)) d[i] = exp(f - lw[i]);  // lw finite: a window token
        }
      }
      double2* dj = reinterpret_cast<double2*>(dl + j * kDlStride + rb);
      dj[0] = make_double2(d[0], d[1]);
      dj[1] = make_double2(d[2], d[3]);
    }
    __syncthreads();
    const int end = min(kTileThreads, tmax + 1 - base);
    for (int k4 = 0; k4 < 64 && 64 * w + k4 < end; k4 += 4) {
      const int j = 64 * w + k4 + lk;
      const bool ok = j < end;
      double y[8];
      bf16x8_to_f64(ok ? *reinterpret_cast<const uint4*>(S.v + ((size_t)(a0 + base + j) * c.H + h) * kD + 8 * li)
                       : make_uint4(0, 0, 0, 0),
                    y);
      acc_channels(acc, ok ? dl[j * kDlStride + li] : 0.0, y);
    }
    __syncthreads();
  }
  sum_waves_store(acc, dl, S.wt + ((size_t)h * S.nrows + row0) * kD, nr);
  if (l == 0)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (rb + i < nr) {
        S.rc[((size_t)h * S.nrows + row0 + rb + i) * 2] = lse[i];
        S.rc[((size_t)h * S.nrows + row0 + rb + i) * 2 + 1] = lw[i];
      }
}

// Forward of the key objective on a tile, with the rotation-independent part from cal_const_kernel.
// Logits g = q.x~/sqrt(d) on the tokens read from INT2 (elsewhere g = f); the softmax p^K over all
// tokens, the window tokens entering as one term exp(LW - mk); KL(p || p^K) = sum_INT2 p (f - g) +
// lse_k - lse_f into lrow (p sums to one); p^K on the INT2 tokens into pd (the rest of pd stays zero);
// dO = sum_INT2 (p^K - p) v + (exp(LW - lse_k) - exp(LW - lse_f)) W~ into wrow and exp(LW - lse_k)
// into erow. With probs_only: pd only. Block (tile, KV head); every pass covers only the tokens
// s_lo .. s_hi some row of the tile reads from INT2.
__global__ __launch_bounds__(kTileThreads) void cal_pos_fwd_kernel(CalSet S, CalCfg c, int probs_only) {
  constexpr int R = kTileRows;
  __shared__ double red4[4 * R];
  __shared__ double dw[R];  // exp(LW - lse_k) - exp(LW - lse_f) per row
  __shared__ __align__(16) double dl[kTileThreads * kDlStride];
  const int h = blockIdx.y, tid = threadIdx.x, gq = c.gq;
  const int w = tid >> 6, l = tid & 63, li = l & 15, lk = l >> 4;
  const int4 tile = S.tiles[blockIdx.x];
  const CalSeq sq = S.seqs[tile.x];
  const int row0 = tile.y, nr = tile.z, tf = tile.w, a0 = sq.start, L = sq.len;
  const int tmax = tf + (nr - 1) / gq;
  const int s_lo = c.sink, s_hi = tmax - c.recent;
  const size_t pb = (size_t)h * S.pelems + sq.p0 + (size_t)(row0 - sq.row0) * L;  // row r at + r L
  double* pdb = S.pd + pb;
  const double *fcb = S.fc + pb, *pcb = S.pc + pb;
  double qa[32];
  rows_operand_bf16(S.q + ((size_t)(a0 + tf + li / gq) * c.Hq + h * gq + li % gq) * kD, li < nr, lk, qa);
  // logits on the INT2 tokens: wave w takes the 16-token tiles w, w + 4, ... that meet s_lo .. s_hi;
  // lane (li, lk) ends with rows lk + 4 v of token 16 tt + li
  double m4k[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) m4k[v] = -INFINITY;
  for (int tt = w; 16 * tt <= s_hi; tt += 4) {
    if (16 * tt + 15 < s_lo) continue;  // uniform over the wave
    const int s = 16 * tt + li;
    const bool ok = s <= tmax;
    const f64x4 ak = dot_tokens_f64(qa, S.xeff + hrow(S, ok ? a0 + s : a0, h), ok, lk);
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int r = lk + 4 * v, tr = tf + r / gq;
      if (r < nr && int2_token(s, tr, c.sink, c.recent)) {
        const double g = ak[v] * kInvSqrtD;
        pdb[(size_t)r * L + s] = g;
        m4k[v] = fmax(m4k[v], g);
      }
    }
  }
  // softmax passes: wave w owns rows rb .. rb + 3 (rb = 4 w), lane l the tokens s_lo + l, + 64, ...
  const int rb = 4 * w;
  double mk[4];
  rows_max(m4k, red4, mk);  // its barriers also make the logits visible to the whole block
  int tr4[4];
  double lsf[4], lw[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const bool ok = rb + i < nr;
    tr4[i] = ok ? tf + (rb + i) / gq : -1;
    const size_t ro = ((size_t)h * S.nrows + row0 + (ok ? rb + i : 0)) * 2;
    lsf[i] = S.rc[ro];
    lw[i] = S.rc[ro + 1];
    mk[i] = fmax(mk[i], lw[i]);  // finite: a row has INT2 or window tokens
  }
  // e = exp(g - mk) in place of the logits, the row sums and sum_INT2 p (f - g)
  double zk[4], klp[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) zk[i] = klp[i] = 0.0;
  for (int s = s_lo + l; s <= s_hi; s += 64)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (tr4[i] < 0 || !int2_token(s, tr4[i], c.sink, c.recent)) continue;
      const size_t o = (size_t)(rb + i) * L + s;
      const double g = pdb[o], e = exp(g - mk[i]);
      pdb[o] = e;  // this lane's own elements
      zk[i] += e;
      klp[i] = fma(pcb[o], fcb[o] - g, klp[i]);
    }
  double kl[4], er[4], rden[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    zk[i] = wave_sum(zk[i]);
    klp[i] = wave_sum(klp[i]);
    const bool win = lw[i] != -INFINITY;
    const double den = zk[i] + (win ? exp(lw[i] - mk[i]) : 0.0);
    const double lsk = mk[i] + log(den);
    kl[i] = klp[i] + (lsk - lsf[i]);
    er[i] = win ? exp(lw[i] - lsk) : 0.0;
    if (l == 0 && rb + i < nr) dw[rb + i] = er[i] - (win ? exp(lw[i] - lsf[i]) : 0.0);
    rden[i] = 1.0 / den;
  }
  // p^K = e / den on the INT2 tokens by 256-token chunk (four tokens per lane); dO over them from the
  // differences p^K - p staged in LDS
  f64x4 acc[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) acc[t] = f64x4{0.0, 0.0, 0.0, 0.0};
  for (int base = s_lo; base <= s_hi; base += kTileThreads) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int j = 64 * q + l, s = base + j;
      double d[4] = {0.0, 0.0, 0.0, 0.0};
      if (s <= s_hi) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if (tr4[i] < 0 || !int2_token(s, tr4[i], c.sink, c.recent)) continue;
          const size_t o = (size_t)(rb + i) * L + s;
          const double pk = pdb[o] * rden[i];
          pdb[o] = pk;
          d[i] = pk - pcb[o];
        }
      }
      if (!probs_only) {
        double2* dj = reinterpret_cast<double2*>(dl + j * kDlStride + rb);
        dj[0] = make_double2(d[0], d[1]);
        dj[1] = make_double2(d[2], d[3]);
      }
    }
    if (probs_only) continue;  // uniform
    __syncthreads();
    const int end = min(kTileThreads, s_hi + 1 - base);
    for (int k4 = 0; k4 < 64 && 64 * w + k4 < end; k4 += 4) {
      const int j = 64 * w + k4 + lk;
      const bool ok = j < end;
      double y[8];
      bf16x8_to_f64(ok ? *reinterpret_cast<const uint4*>(S.v + ((size_t)(a0 + base + j) * c.H + h) * kD + 8 * li)
                       : make_uint4(0, 0, 0, 0),
                    y);
      acc_channels(acc, ok ? dl[j * kDlStride + li] : 0.0, y);
    }
    __syncthreads();
  }
  if (probs_only) return;  // uniform
  sum_waves_store(acc, dl, S.wrow + ((size_t)h * S.nrows + row0) * kD, nr, S.wt + ((size_t)h * S.nrows + row0) * kD,
                  dw);  // + dw W~ per row
  if (l == 0)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (rb + i < nr) {
        S.lrow[(size_t)h * S.nrows + row0 + rb + i] = kl[i];
        S.erow[(size_t)h * S.nrows + row0 + rb + i] = er[i];
      }
}

// Value objective on a tile: dO_V = sum_s p^K-hat_s (v~_s - v_s) into wrow (pd holds p^K-hat on the
// tokens read from INT2, 0 elsewhere). Block (tile, KV head); pd is staged through LDS by token chunk
// over the tokens s_lo .. s_hi some row of the tile reads from INT2.
__global__ __launch_bounds__(kTileThreads) void cal_pos_val_kernel(CalSet S, CalCfg c) {
  constexpr int R = kTileRows;
  __shared__ __align__(16) double dl[kTileThreads * kDlStride];
  const int h = blockIdx.y, tid = threadIdx.x, gq = c.gq;
  const int w = tid >> 6, l = tid & 63, li = l & 15, lk = l >> 4;
  const int4 tile = S.tiles[blockIdx.x];
  const CalSeq sq = S.seqs[tile.x];
  const int row0 = tile.y, nr = tile.z, tf = tile.w, a0 = sq.start, L = sq.len;
  const int tmax = tf + (nr - 1) / gq;
  const int s_lo = c.sink, s_hi = tmax - c.recent;
  const double* pdb = S.pd + (size_t)h * S.pelems + sq.p0 + (size_t)(row0 - sq.row0) * L;
  f64x4 acc[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) acc[t] = f64x4{0.0, 0.0, 0.0, 0.0};
  for (int base = s_lo; base <= s_hi; base += kTileThreads) {
    const int end = min(kTileThreads, s_hi + 1 - base);
    for (int e = tid; e < R * kTileThreads; e += kTileThreads) {
      const int r = e / kTileThreads, j = e % kTileThreads;
      dl[j * kDlStride + r] = r < nr && j < end ? pdb[(size_t)r * L + base + j] : 0.0;
    }
    __syncthreads();
    for (int k4 = 0; k4 < 64 && 64 * w + k4 < end; k4 += 4) {
      const int j = 64 * w + k4 + lk;
      const bool ok = j < end;
      const size_t o = ((size_t)(a0 + base + j) * c.H + h) * kD + 8 * li;
      double y[8];
      bf16x8_to_f64(ok ? *reinterpret_cast<const uint4*>(S.v + o) : make_uint4(0, 0, 0, 0), y);
      const double2* x2 = reinterpret_cast<const double2*>(S.xeff + hrow(S, ok ? a0 + base + j : a0, h) + 8 * li);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const double2 x = ok ? x2[i] : make_double2(0.0, 0.0);
        y[2 * i] = x.x - y[2 * i];
        y[2 * i + 1] = x.y - y[2 * i + 1];
      }
      acc_channels(acc, ok ? dl[j * kDlStride + li] : 0.0, y);
    }
    __syncthreads();
  }
  sum_waves_store(acc, dl, S.wrow + ((size_t)h * S.nrows + row0) * kD, nr);
}

// u = M_j dO for the rows of query head j (M_j = W_{O,j}^T W_{O,j}, symmetric), E = dO . u / d_model.
// Keys: urow = u, lrow += lambda E. Values: wrow = 2 u / (d_model rows), lrow = E. Block (query head j,
// 64 positions), the layout of the rotation kernel with positions as rows (a row's four lane groups
// are in one wave, each reads dO at its own output channels before writing them).
constexpr int kUTile = 64;
__global__ __launch_bounds__(256) void cal_u_kernel(CalSet S, CalCfg c, int value) {
  __shared__ double Bs[16 * kBsStride];
  const int j = blockIdx.x, h = j / c.gq, jj = j % c.gq, tid = threadIdx.x;
  const int w = tid >> 6, l = tid & 63, li = l & 15, lk = l >> 4;
  const int npos = S.nrows / c.gq, pp = blockIdx.y * kUTile + 16 * w + li;
  const bool ok = pp < npos;
  const size_t row = (size_t)h * S.nrows + (size_t)(ok ? pp : 0) * c.gq + jj;
  double ya[32];
  row_operand_f64(S.wrow + row * kD, ok, ya);
  f64x4 acc[8];
#pragma unroll
  for (int ct = 0; ct < 8; ++ct) acc[ct] = f64x4{0.0, 0.0, 0.0, 0.0};
  mat_t_rows<0>(ya, c.gram + (size_t)j * kMat, Bs, acc);
  double e = 0.0;
  if (ok)
#pragma unroll
    for (int ct = 0; ct < 8; ++ct)
#pragma unroll
      for (int v = 0; v < 4; ++v) e = fma(S.wrow[row * kD + 16 * ct + lk + 4 * v], acc[ct][v], e);
  e += __shfl_xor(e, 16);
  e += __shfl_xor(e, 32);
  if (!ok) return;
  const double dm = (double)c.dm;
#pragma unroll
  for (int ct = 0; ct < 8; ++ct)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const size_t o = row * kD + 16 * ct + lk + 4 * v;
      if (value)
        S.wrow[o] = 2.0 * acc[ct][v] / (dm * (double)S.nrows);
      else
        S.urow[o] = acc[ct][v];
    }
  if (lk == 0) {
    if (value)
      S.lrow[row] = e / dm;
    else
      S.lrow[row] += c.lam * e / dm;
  }
}

// Logit gradients of the key objective on a tile: G_s = 2 u . v_s / d_model, gbar = sum over all tokens of
// p^K_s G_s (the window tokens as exp(LW - lse_k) 2 u . W~ / d_model), and on the tokens read from INT2
// pd = ((p^K - p) + lambda p^K (G - gbar)) / rows (zero elsewhere, untouched). Block (tile, KV head);
// u . v_s on the fp64 matrix cores (16-token tiles per wave) over the INT2 span s_lo .. s_hi only.
__global__ __launch_bounds__(kTileThreads) void cal_pos_grad_kernel(CalSet S, CalCfg c) {
  constexpr int R = kTileRows;
  __shared__ double red[16 * R];
  __shared__ double gbw[R];  // window part of gbar per row
  const int h = blockIdx.y, tid = threadIdx.x, gq = c.gq;
  const int w = tid >> 6, l = tid & 63, li = l & 15, lk = l >> 4;
  const int4 tile = S.tiles[blockIdx.x];
  const CalSeq sq = S.seqs[tile.x];
  const int row0 = tile.y, nr = tile.z, tf = tile.w, a0 = sq.start, L = sq.len;
  const int tmax = tf + (nr - 1) / gq;
  const int s_lo = c.sink, s_hi = tmax - c.recent;
  const size_t pb = (size_t)h * S.pelems + sq.p0 + (size_t)(row0 - sq.row0) * L;
  double* pdb = S.pd + pb;
  double* pfb = S.pf + pb;
  const double* pcb = S.pc + pb;
  const double* urw = S.urow + ((size_t)h * S.nrows + row0) * kD;
  const double two_dm = 2.0 / (double)c.dm;
  {
    // u . W~ for row tid / 16, eight channels per lane, reduced over the row's 16 lanes
    const int r = tid >> 4, c8 = 8 * (tid & 15);
    double d = 0.0;
    if (r < nr) {
      const double* wtr = S.wt + ((size_t)h * S.nrows + row0 + r) * kD + c8;
#pragma unroll
      for (int m = 0; m < 8; ++m) d = fma(urw[(size_t)r * kD + c8 + m], wtr[m], d);
    }
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) d += __shfl_xor(d, off);
    if ((tid & 15) == 0) gbw[r] = r < nr ? S.erow[(size_t)h * S.nrows + row0 + r] * two_dm * d : 0.0;
  }
  double ua[32];
  {
    const bool ok = li < nr;
    const double* ur = urw + (size_t)(ok ? li : 0) * kD + 32 * lk;
#pragma unroll
    for (int m = 0; m < 32; ++m) ua[m] = ok ? ur[m] : 0.0;
  }
  double gb4[4] = {0.0, 0.0, 0.0, 0.0};
  for (int tt = w; 16 * tt <= s_hi; tt += 4) {
    if (16 * tt + 15 < s_lo) continue;  // uniform over the wave
    const int s = 16 * tt + li;
    const bool ok = s <= tmax;
    const f64x4 g = dot_tokens_bf16(ua, S.v + ((size_t)(a0 + (ok ? s : 0)) * c.H + h) * kD, ok, lk);
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int r = lk + 4 * v;
      if (r < nr && int2_token(s, tf + r / gq, c.sink, c.recent)) {
        const size_t o = (size_t)r * L + s;
        const double pk = pdb[o], gs = two_dm * g[v];
        gb4[v] = fma(pk, gs, gb4[v]);
        pfb[o] = (pk - pcb[o]) + c.lam * pk * gs;
      }
    }
  }
  // gbar per row: over the 16 lanes of each lk group, then the four waves (fixed order), then the window
#pragma unroll
  for (int v = 0; v < 4; ++v)
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) gb4[v] += __shfl_xor(gb4[v], off);
  if (li == 0)
#pragma unroll
    for (int v = 0; v < 4; ++v) red[w * 16 + lk + 4 * v] = gb4[v];
  __syncthreads();  // also makes the pf updates and gbw visible to the whole block
  double gb[R];
#pragma unroll
  for (int r = 0; r < R; ++r) gb[r] = ((red[r] + red[32 + r]) + (red[16 + r] + red[48 + r])) + gbw[r];
  const double inv_rows = 1.0 / (double)S.nrows;
  for (int s = s_lo + tid; s <= s_hi; s += kTileThreads) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if (r >= nr || !int2_token(s, tf + r / gq, c.sink, c.recent)) continue;
      const size_t o = (size_t)r * L + s;
      pdb[o] = (pfb[o] - c.lam * pdb[o] * gb[r]) * inv_rows;
    }
  }
}

// Gradient w.r.t. the effective rows: gx[s] = sum over the rows r of s's sequence of pd[r][s] y_r
// with y_r = q_r / sqrt(d) (keys) or the row weight (values): per sequence the product
// P^T Y of its [rows x len] weights and [rows x 128] row vectors, on the fp64 matrix cores. Block
// (64-token tile, KV head) of four waves, wave w: tokens 16 w .. + 15 x all 128 channels (eight
// 16 x 16 tiles); 16 rows at a time through LDS, the next chunk fetched into registers while the
// matrix cores run on the current one.
constexpr int kGxTok = 64, kGxRows = 16;
constexpr int kGxPs = kGxTok + 16, kGxYs = kD + 16;  // padded LDS rows: lane groups l / 16 on other banks
__global__ __launch_bounds__(256) void cal_gx_kernel(CalSet S, CalCfg c, int value) {
  __shared__ double ps[kGxRows][kGxPs];
  __shared__ double ys[kGxRows][kGxYs];
  const int h = blockIdx.y, tid = threadIdx.x, s0 = blockIdx.x * kGxTok;
  const int w = tid >> 6, l = tid & 63, li = l & 15, lk = l >> 4;
  f64x4 acc[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) acc[t] = f64x4{0.0, 0.0, 0.0, 0.0};
  int lo = 0, hi = S.nseq - 1;  // the sequence holding token s0
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (S.seqs[mid].start <= s0) lo = mid; else hi = mid - 1;
  }
  // chunk (sequence n, rows r0 .. r0 + 15) into registers: 4 weights and 8 row entries per thread
  double pr[4], yr[8];
  auto fetch = [&](const CalSeq& sq, int nr, int r0) {
    const double* pd = S.pd + (size_t)h * S.pelems + sq.p0;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int e = tid + 256 * u, i = e / kGxTok, x = e % kGxTok, sl = s0 + x - sq.start;
      pr[u] = (r0 + i < nr && sl >= 0 && sl < sq.len) ? pd[(size_t)(r0 + i) * sq.len + sl] : 0.0;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = tid + 256 * u, i = e / kD, col = e % kD, lr = r0 + i;
      double y = 0.0;
      if (lr < nr) {
        if (value) {
          y = S.wrow[((size_t)h * S.nrows + sq.row0 + lr) * kD + col];
        } else {
          const int t = sq.t0 + lr / c.gq, j = h * c.gq + lr % c.gq;
          y = bf16d(S.q[((size_t)(sq.start + t) * c.Hq + j) * kD + col]) * kInvSqrtD;
        }
      }
      yr[u] = y;
    }
  };
  int n = lo, r0 = 0;
  CalSeq sq = S.seqs[n];
  int nr = (sq.len - sq.t0) * c.gq;
  // the chunks: rows of every sequence that meets the tile, in order
  auto valid = [&]() { return n < S.nseq && sq.start < s0 + kGxTok; };
  auto advance = [&]() {
    r0 += kGxRows;
    while (valid() && r0 >= nr) {
      if (++n >= S.nseq) break;
      sq = S.seqs[n];
      nr = (sq.len - sq.t0) * c.gq;
      r0 = 0;
    }
  };
  if (valid() && nr == 0) {  // a sequence without query rows contributes nothing
    r0 = -kGxRows;
    advance();
  }
  if (valid()) fetch(sq, nr, r0);
  while (valid()) {
    __syncthreads();
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int e = tid + 256 * u;
      ps[e / kGxTok][e % kGxTok] = pr[u];
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = tid + 256 * u;
      ys[e / kD][e % kD] = yr[u];
    }
    __syncthreads();
    advance();
    if (valid()) fetch(sq, nr, r0);
#pragma unroll
    for (int k4 = 0; k4 < kGxRows; k4 += 4) {
      const double a = ps[k4 + lk][16 * w + li];
#pragma unroll
      for (int t = 0; t < 8; ++t) acc[t] = mfma64(a, ys[k4 + lk][16 * t + li], acc[t]);
    }
  }
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int s = s0 + 16 * w + lk + 4 * v;
    if (s < S.T) {
      double* out = S.gx + hrow(S, s, h) + li;
#pragma unroll
      for (int t = 0; t < 8; ++t) out[16 * t] = acc[t][v];
    }
  }
}

// gz = mask . (gx R): block (64 tokens, KV head), the layout of the rotation kernel.
constexpr int kGzTile = 64;
__global__ __launch_bounds__(256) void cal_gz_kernel(CalSet S, CalCfg c) {
  __shared__ double Bs[16 * kBsStride];
  const int h = blockIdx.y, tid = threadIdx.x, w = tid >> 6, l = tid & 63, li = l & 15, lk = l >> 4;
  const int tok = blockIdx.x * kGzTile + 16 * w + li;
  const bool ok = tok < S.T;
  const size_t rowo = hrow(S, ok ? tok : 0, h);
  double ya[32];
  row_operand_f64(S.gx + rowo, ok, ya);
  f64x4 acc[8];
#pragma unroll
  for (int ct = 0; ct < 8; ++ct) acc[ct] = f64x4{0.0, 0.0, 0.0, 0.0};
  mat_t_rows<0>(ya, c.R + (size_t)h * kMat, Bs, acc);
  if (ok)
#pragma unroll
    for (int ct = 0; ct < 8; ++ct)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const size_t o = rowo + 16 * ct + lk + 4 * v;
        S.gz[o] = S.mask[o] ? acc[ct][v] : 0.0;
      }
}

// Partial dL/dR over a token slice: sum_s x_s[a] gz_s[b] + gx_s[a] zhat_s[b] on the fp64 matrix
// cores (M = a, N = b, K = the slice's tokens, four per step). Block (KV head, slice) of eight
// waves, wave w: rows a = 16 w .. + 15 and all 128 columns; 16-token chunks of the four operands
// staged in LDS.
constexpr int kDrChunk = 16, kDrStride = 132;
__global__ __launch_bounds__(512) void cal_dr_kernel(CalSet S, CalCfg c, int value) {
  __shared__ double xs[kDrChunk][kDrStride], gxs[kDrChunk][kDrStride];
  __shared__ double gzs[kDrChunk][kDrStride], zs[kDrChunk][kDrStride];
  const int h = blockIdx.x, sp = blockIdx.y, tid = threadIdx.x;
  const int w = tid >> 6, l = tid & 63, li = l & 15, lk = l >> 4;
  const int s_lo = (int)((long long)S.T * sp / kCalSplit), s_hi = (int)((long long)S.T * (sp + 1) / kCalSplit);
  const uint16_t* X = value ? S.v : S.k;
  f64x4 acc[8];
#pragma unroll
  for (int ct = 0; ct < 8; ++ct) acc[ct] = f64x4{0.0, 0.0, 0.0, 0.0};
  for (int s0 = s_lo; s0 < s_hi; s0 += kDrChunk) {
    __syncthreads();
    for (int e = tid; e < kDrChunk * kD; e += blockDim.x) {
      const int t = e >> 7, col = e & 127, s = s0 + t;
      const bool ok = s < s_hi;
      const size_t o = ((size_t)(ok ? s : s_lo) * c.H + h) * kD + col, io = hrow(S, ok ? s : s_lo, h) + col;
      xs[t][col] = ok ? bf16d(X[o]) - (value ? 0.0 : (double)c.mu[h * kD + col]) : 0.0;
      gxs[t][col] = ok ? S.gx[io] : 0.0;
      gzs[t][col] = ok ? S.gz[io] : 0.0;
      zs[t][col] = ok ? S.zhat[io] : 0.0;
    }
    __syncthreads();
#pragma unroll
    for (int k4 = 0; k4 < kDrChunk; k4 += 4) {
      const int t = k4 + lk;
      const double ax = xs[t][16 * w + li], ag = gxs[t][16 * w + li];
#pragma unroll
      for (int ct = 0; ct < 8; ++ct) {
        acc[ct] = mfma64(ax, gzs[t][16 * ct + li], acc[ct]);
        acc[ct] = mfma64(ag, zs[t][16 * ct + li], acc[ct]);
      }
    }
  }
  // element v of acc[ct]: row a = 16 w + lk + 4 v, column b = 16 ct + li
  double* out = c.drp + ((size_t)sp * c.H + h) * kMat;
#pragma unroll
  for (int ct = 0; ct < 8; ++ct)
#pragma unroll
    for (int v = 0; v < 4; ++v) out[(16 * w + lk + 4 * v) * kD + 16 * ct + li] = acc[ct][v];
}

__global__ __launch_bounds__(256) void cal_dr_reduce_kernel(CalCfg c) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x, n = (size_t)c.H * kMat;
  if (i >= n) return;
  double acc = 0.0;
  for (int sp = 0; sp < kCalSplit; ++sp) acc += c.drp[(size_t)sp * n + i];
  c.dr[i] = acc;
}

// ---------------------------------------------------------------------------------------------
// Matrix functions: one work-group of 1024 threads per KV head; 128 x 128 products on the fp64
// matrix cores, operands staged through LDS in 16-deep slices.
struct ExpLds {
  double at[16][kD];  // op(A)^T chunk: at[k][r] = op(A)[r][k0 + k]
  double bs[16][kD];  // B chunk: bs[k][c] = B[k0 + k][c]
  double red[16];
};

// Output fragment of wg_gemm: a thread's acc[t][v] is the element (frag_row(v), frag_col(t)) of the
// 128 x 128 product. Wave w covers rows 16 (w / 2) .. + 15 and columns 64 (w % 2) .. + 63 as four
// 16 x 16 matrix-core tiles; lane l holds rows l / 16 + 4 v, column l % 16 of tile t.
__device__ __forceinline__ int frag_row(int v) {
  return 16 * (threadIdx.x >> 7) + ((threadIdx.x & 63) >> 4) + 4 * v;
}
__device__ __forceinline__ int frag_col(int t) {
  return 64 * ((threadIdx.x >> 6) & 1) + 16 * t + (threadIdx.x & 15);
}

// Fragment element (t, v) sits at offset frag_base() + frag_step(t, v) of a row-major 128 x 128 matrix.
__device__ __forceinline__ unsigned frag_base() { return (unsigned)(frag_row(0) * kD + frag_col(0)); }
constexpr unsigned frag_step(int t, int v) { return (unsigned)(4 * v * kD + 16 * t); }

// M[fragment] = acc * scale (+ I when add_identity).
__device__ __forceinline__ void frag_store(double* __restrict__ M, const f64x4 (&acc)[4], double scale,
                                           bool add_identity) {
  unsigned fb = frag_base();
  // computed here, at the store: hoisted out of the callers' loops, the 32 addresses would not
  // fit the register budget of a 1024-thread block
  asm volatile("" : "+v"(fb));
  double* __restrict__ Mf = M + fb;
  const int r0 = frag_row(0), c0 = frag_col(0);
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int v = 0; v < 4; ++v)
      Mf[frag_step(t, v)] = (add_identity && r0 + 4 * v == c0 + 16 * t ? 1.0 : 0.0) + acc[t][v] * scale;
}

// M[fragment] = acc + c0 I + c1 A1 + c2 A2 + c3 A3, the A's read at the thread's own fragment elements.
__device__ __forceinline__ void frag_store_lin(double* __restrict__ M, const f64x4 (&acc)[4], double c0,
                                               const double* A1, double c1, const double* A2, double c2,
                                               const double* A3, double c3) {
  unsigned fb = frag_base();
  asm volatile("" : "+v"(fb));  // as in frag_store
  const int r0 = frag_row(0), c0c = frag_col(0);
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const unsigned o = fb + frag_step(t, v);
      M[o] = (r0 + 4 * v == c0c + 16 * t ? c0 : 0.0) + acc[t][v] + c1 * A1[o] + c2 * A2[o] + c3 * A3[o];
    }
}

// Truncated Taylor series of exp (degree kExpTerms = 14) in Paterson-Stockmeyer form: with Y = X^4,
// sum_k X^k / k! = ((B_3 Y + B_2) Y + B_1) Y + B_0, B_i = sum_{j<4} X^j / (4 i + j)! (1/15! taken as 0),
// so the powers X^2, X^3, X^4 and three Horner steps take six products instead of fourteen.
__device__ __forceinline__ void taylor_coeffs(double (&cf)[16]) {
  cf[0] = 1.0;
#pragma unroll
  for (int k = 1; k <= kExpTerms; ++k) cf[k] = cf[k - 1] / (double)k;
  cf[15] = 0.0;
}

// acc += op(A) B for 128 x 128 fp64 matrices in global memory (op(A) = A or A^T) on the fp64
// matrix cores (16 x 16 x 4 steps), 16-deep chunks of A and B staged through LDS. Ends with a
// barrier, so the caller may overwrite A or B right after.
__device__ __forceinline__ void wg_gemm(const double* A, bool ta, const double* B, f64x4 (&acc)[4], ExpLds& sm) {
  const int tid = threadIdx.x, l = tid & 63;
  const int ar = 16 * (tid >> 7) + (l & 15), kl = l >> 4, bc = 64 * ((tid >> 6) & 1) + (l & 15);
#pragma unroll 1
  for (int k0 = 0; k0 < kD; k0 += 16) {
    for (int e = tid; e < kD * 16; e += kExpThreads) {
      const int kk = e >> 7, r = e & 127;
      sm.at[kk][r] = ta ? A[(k0 + kk) * kD + r] : A[r * kD + k0 + kk];
      sm.bs[kk][r] = B[(k0 + kk) * kD + r];
    }
    __syncthreads();
#pragma unroll
    for (int k4 = 0; k4 < 16; k4 += 4) {
      const double av = sm.at[k4 + kl][ar];
#pragma unroll
      for (int t = 0; t < 4; ++t)
        acc[t] = mfma64(av, sm.bs[k4 + kl][bc + 16 * t], acc[t]);
    }
    __syncthreads();
  }
}

__device__ __forceinline__ void zero4(f64x4 (&a)[4]) {
#pragma unroll
  for (int t = 0; t < 4; ++t) a[t] = f64x4{0.0, 0.0, 0.0, 0.0};
}

// X <- (A - A^T) * 2^-sc with sc the smallest scaling giving ||X||_1 <= 1/2 (returned); with
// transpose, X <- (A - A^T)^T * 2^-sc.
__device__ int wg_skew_scaled(const double* A, double* X, bool transpose, ExpLds& sm) {
  const int tid = threadIdx.x;
  double colsum = 0.0;
  if (tid < kD)
    for (int r = 0; r < kD; ++r) colsum += fabs(A[r * kD + tid] - A[tid * kD + r]);
  const double nrm = block_max(tid < kD ? colsum : 0.0, sm.red);
  int sc = 0;
  while (sc < 60 && ldexp(nrm, -sc) > 0.5) ++sc;
  const double f = ldexp(1.0, -sc);
  for (int e = tid; e < kMat; e += kExpThreads) {
    const int r = e >> 7, cc = e & 127;
    const double s = A[r * kD + cc] - A[cc * kD + r];
    X[e] = (transpose ? -s : s) * f;
  }
  __syncthreads();
  return sc;
}

// Forward: R = R0 exp(A - A^T) and Rt = R^T (fp64) for every head.
__global__ __launch_bounds__(kExpThreads) void cal_expm_kernel(CalCfg c, const double* __restrict__ Aall, int value) {
  __shared__ ExpLds sm;
  const int h = blockIdx.x, tid = threadIdx.x;
  double* ex = c.ex + (size_t)h * kCalScratch * kMat;
  double *X = ex, *P = ex + kMat, *R0 = ex + 2 * kMat;
  double *X2 = ex + 5 * kMat, *X3 = ex + 6 * kMat, *X4 = ex + 7 * kMat;
  const float* R0f = (value ? c.R0v : c.R0k) + (size_t)h * kMat;
  for (int e = tid; e < kMat; e += kExpThreads) R0[e] = (double)R0f[e];
  const int sc = wg_skew_scaled(Aall + (size_t)h * kMat, X, false, sm);
  double cf[16];
  taylor_coeffs(cf);
  f64x4 acc[4];
  zero4(acc);
  wg_gemm(X, false, X, acc, sm);
  frag_store(X2, acc, 1.0, false);
  __syncthreads();
  zero4(acc);
  wg_gemm(X2, false, X, acc, sm);
  frag_store(X3, acc, 1.0, false);
  zero4(acc);
  wg_gemm(X2, false, X2, acc, sm);
  frag_store(X4, acc, 1.0, false);
  __syncthreads();
  for (int e = tid; e < kMat; e += kExpThreads)  // P = B_3
    P[e] = ((e >> 7) == (e & 127) ? cf[12] : 0.0) + cf[13] * X[e] + cf[14] * X2[e] + cf[15] * X3[e];
  __syncthreads();
  for (int i = 2; i >= 0; --i) {  // P <- P X^4 + B_i
    zero4(acc);
    wg_gemm(P, false, X4, acc, sm);
    frag_store_lin(P, acc, cf[4 * i], X, cf[4 * i + 1], X2, cf[4 * i + 2], X3, cf[4 * i + 3]);
    __syncthreads();
  }
  for (int i = 0; i < sc; ++i) {  // P <- P P
    zero4(acc);
    wg_gemm(P, false, P, acc, sm);
    frag_store(P, acc, 1.0, false);
    __syncthreads();
  }
  zero4(acc);
  wg_gemm(R0, false, P, acc, sm);
  double* R = c.R + (size_t)h * kMat;
  double* Rt = c.Rt + (size_t)h * kMat;
  frag_store(R, acc, 1.0, false);
  const int r0 = frag_row(0), c0 = frag_col(0);
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int v = 0; v < 4; ++v) Rt[(unsigned)((c0 + 16 * t) * kD + r0 + 4 * v)] = acc[t][v];
}

// Backward: grad = dS - dS^T with dS = L_exp(S^T, R0^T dR), S = A - A^T, for every head: the top
// right block of exp([[X, G], [0, X]]) (X = S^T, G = R0^T dR, both scaled by 2^-sc), whose powers
// are [[X^k, D_k], [0, X^k]] with D_{a+b} = X^a D_b + D_a X^b; the Taylor polynomial of the block
// matrix in the Paterson-Stockmeyer form above, then sc squarings.
__global__ __launch_bounds__(kExpThreads) void cal_expm_grad_kernel(CalCfg c, const double* __restrict__ Aall,
                                                                   int value, double* __restrict__ grad) {
  __shared__ ExpLds sm;
  const int h = blockIdx.x, tid = threadIdx.x;
  double* ex = c.ex + (size_t)h * kCalScratch * kMat;
  double *X = ex, *P1 = ex + kMat, *R0 = ex + 2 * kMat, *P2 = ex + 3 * kMat, *Gs = ex + 4 * kMat;
  double *X2 = ex + 5 * kMat, *X3 = ex + 6 * kMat, *X4 = ex + 7 * kMat;
  double *D2 = ex + 8 * kMat, *D3 = ex + 9 * kMat, *D4 = ex + 10 * kMat;
  const float* R0f = (value ? c.R0v : c.R0k) + (size_t)h * kMat;
  for (int e = tid; e < kMat; e += kExpThreads) R0[e] = (double)R0f[e];
  const int sc = wg_skew_scaled(Aall + (size_t)h * kMat, X, true, sm);
  const double f = ldexp(1.0, -sc);
  double cf[16];
  taylor_coeffs(cf);
  f64x4 acc[4], t1[4];
  zero4(acc);
  wg_gemm(R0, true, c.dr + (size_t)h * kMat, acc, sm);  // G_E = R0^T dR, scaled like X
  frag_store(Gs, acc, f, false);
  __syncthreads();
  // M^2: (X^2, X G + G X)
  zero4(acc);
  wg_gemm(X, false, X, acc, sm);
  frag_store(X2, acc, 1.0, false);
  zero4(acc);
  wg_gemm(X, false, Gs, acc, sm);
  wg_gemm(Gs, false, X, acc, sm);
  frag_store(D2, acc, 1.0, false);
  __syncthreads();
  // M^3 = M^2 M: (X^2 X, X^2 G + D_2 X); M^4 = M^2 M^2: (X^2 X^2, X^2 D_2 + D_2 X^2)
  zero4(acc);
  wg_gemm(X2, false, X, acc, sm);
  frag_store(X3, acc, 1.0, false);
  zero4(acc);
  wg_gemm(X2, false, Gs, acc, sm);
  wg_gemm(D2, false, X, acc, sm);
  frag_store(D3, acc, 1.0, false);
  zero4(acc);
  wg_gemm(X2, false, X2, acc, sm);
  frag_store(X4, acc, 1.0, false);
  zero4(acc);
  wg_gemm(X2, false, D2, acc, sm);
  wg_gemm(D2, false, X2, acc, sm);
  frag_store(D4, acc, 1.0, false);
  __syncthreads();
  for (int e = tid; e < kMat; e += kExpThreads) {  // (P1, P2) = B_3
    P1[e] = ((e >> 7) == (e & 127) ? cf[12] : 0.0) + cf[13] * X[e] + cf[14] * X2[e] + cf[15] * X3[e];
    P2[e] = cf[13] * Gs[e] + cf[14] * D2[e] + cf[15] * D3[e];
  }
  __syncthreads();
  for (int i = 2; i >= 0; --i) {  // (P1, P2) <- (P1 X^4, P1 D_4 + P2 X^4) + B_i
    zero4(t1);
    wg_gemm(P1, false, X4, t1, sm);
    zero4(acc);
    wg_gemm(P1, false, D4, acc, sm);
    wg_gemm(P2, false, X4, acc, sm);
    frag_store_lin(P2, acc, 0.0, Gs, cf[4 * i + 1], D2, cf[4 * i + 2], D3, cf[4 * i + 3]);
    frag_store_lin(P1, t1, cf[4 * i], X, cf[4 * i + 1], X2, cf[4 * i + 2], X3, cf[4 * i + 3]);
    __syncthreads();
  }
  for (int i = 0; i < sc; ++i) {  // (P1, P2) <- (P1 P1, P1 P2 + P2 P1)
    zero4(t1);
    wg_gemm(P1, false, P1, t1, sm);
    zero4(acc);
    wg_gemm(P1, false, P2, acc, sm);
    wg_gemm(P2, false, P1, acc, sm);
    frag_store(P2, acc, 1.0, false);
    frag_store(P1, t1, 1.0, false);
    __syncthreads();
  }
  double* g = grad + (size_t)h * kMat;
  for (int e = tid; e < kMat; e += kExpThreads) {
    const int r = e >> 7, cc = e & 127;
    g[e] = P2[r * kD + cc] - P2[cc * kD + r];
  }
}

// ---------------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void cal_loss_kernel(const double* __restrict__ lrow, int nrows,
                                                       double* __restrict__ loss) {
  __shared__ double red[16];
  const int h = blockIdx.x;
  double acc = 0.0;
  for (int r = threadIdx.x; r < nrows; r += blockDim.x) acc += lrow[(size_t)h * nrows + r];
  acc = block_sum(acc, red);
  if (threadIdx.x == 0) loss[h] = acc / (double)nrows;
}

// Adam as torch.optim.Adam (betas 0.9, 0.999, eps 1e-8, no weight decay): m <- m + (1 - b1)(g - m),
// v <- b2 v + (1 - b2) g^2, A <- A - (lr / (1 - b1^t)) m / (sqrt(v) / sqrt(1 - b2^t) + eps).
__global__ __launch_bounds__(256) void cal_adam_kernel(double* A, const double* g, double* m, double* v, int n,
                                                       double step_size, double bc2_sqrt, double lr) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  (void)lr;
  const double gi = g[i];
  const double mi = m[i] + (1.0 - 0.9) * (gi - m[i]);
  const double vi = v[i] * 0.999 + (1.0 - 0.999) * gi * gi;
  m[i] = mi;
  v[i] = vi;
  A[i] -= step_size * mi / (sqrt(vi) / bc2_sqrt + 1e-8);
}

__global__ __launch_bounds__(1024) void cal_select_kernel(const double* A, const double* loss, double* best,
                                                          double* A_best) {
  const int h = blockIdx.x;
  const bool take = loss[h] < best[h];
  __syncthreads();  // every thread has read best[h] before thread 0 may replace it
  if (!take) return;
  for (int e = threadIdx.x; e < kMat; e += blockDim.x) A_best[(size_t)h * kMat + e] = A[(size_t)h * kMat + e];
  if (threadIdx.x == 0) best[h] = loss[h];
}

__global__ __launch_bounds__(64) void cal_record_kernel(const double* __restrict__ loss, double* __restrict__ dst,
                                                        int stride, int H) {
  const int h = threadIdx.x;
  if (h < H) dst[(size_t)h * stride] = loss[h];
}

__global__ __launch_bounds__(256) void cal_fill_kernel(double* p, size_t n, double v) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

__global__ __launch_bounds__(256) void cal_to_f32_kernel(const double* __restrict__ src, float* __restrict__ dst,
                                                         size_t n) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = (float)src[i];
}

// W_{O,j}^T W_{O,j} on the fp64 matrix cores: block = query head j, eight waves; wave w owns output rows
// 16 w .. 16 w + 15 (all eight 16-column tiles). The head's d_model x 128 slice of W_O goes through LDS
// 16 rows at a time (bf16 -> fp64, exact); K = those rows, 4 per step.
constexpr int kGramRows = 16;
__global__ __launch_bounds__(512) void cal_gram_kernel(const uint16_t* __restrict__ W, int dm, int Hq,
                                                       double* __restrict__ gram) {
  __shared__ double xs[kGramRows][kD + 2];
  const int j = blockIdx.x, tid = threadIdx.x, w = tid >> 6, l = tid & 63, lo = l & 15, lk = l >> 4;
  const size_t ld = (size_t)Hq * kD;
  f64x4 acc[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) acc[t] = f64x4{0.0, 0.0, 0.0, 0.0};
  for (int r0 = 0; r0 < dm; r0 += kGramRows) {
    for (int e = tid; e < kGramRows * kD; e += 512) {
      const int rr = e / kD, c = e % kD;
      xs[rr][c] = r0 + rr < dm ? bf16d(W[(size_t)(r0 + rr) * ld + (size_t)j * kD + c]) : 0.0;
    }
    __syncthreads();
#pragma unroll
    for (int k4 = 0; k4 < kGramRows; k4 += 4) {
      // A[m][k] = X[k][16 w + m], B[k][n] = X[k][16 t + n]: lane l holds A[lo][lk] and B[lk][lo]
      const double av = xs[k4 + lk][16 * w + lo];
#pragma unroll
      for (int t = 0; t < 8; ++t) acc[t] = mfma64(av, xs[k4 + lk][16 * t + lo], acc[t]);
    }
    __syncthreads();
  }
  // element v of tile t: row 16 w + lk + 4 v, column 16 t + lo
#pragma unroll
  for (int t = 0; t < 8; ++t)
#pragma unroll
    for (int v = 0; v < 4; ++v) gram[((size_t)j * kD + 16 * w + lk + 4 * v) * kD + 16 * t + lo] = acc[t][v];
}

// Per-channel mean of the keys: block = KV head, thread = channel (sequential fp64 sum).
__global__ __launch_bounds__(128) void cal_key_mean_kernel(const uint16_t* __restrict__ k, int T, int H,
                                                           float* __restrict__ mu) {
  const int h = blockIdx.x, col = threadIdx.x;
  double acc = 0.0;
  for (int s = 0; s < T; ++s) acc += bf16d(k[((size_t)s * H + h) * kD + col]);
  mu[h * kD + col] = (float)(acc / (double)T);
}

size_t up256(size_t x) { return (x + 255) & ~size_t(255); }

}  // namespace

size_t cal_set_bytes(int T, int nseq, int nrows, long long pelems, int H) {
  const size_t rows = (size_t)T * H * kD;
  return up256(sizeof(CalSeq) * (size_t)nseq) + up256(sizeof(int4) * (size_t)nrows) + up256(sizeof(int) * (size_t)nrows) + 4 * up256(rows * 8) +
         up256(rows) + 4 * up256((size_t)H * pelems * 8) + 3 * up256((size_t)H * nrows * kD * 8) +
         up256((size_t)H * nrows * 16) + 2 * up256((size_t)H * nrows * 8);
}

size_t cal_shared_bytes(int H, int Hq) {
  return up256((size_t)Hq * kMat * 8) + 2 * up256((size_t)H * kMat * 8) + up256((size_t)H * kCalScratch * kMat * 8) +
         up256((size_t)kCalSplit * H * kMat * 8) + up256((size_t)H * kMat * 8);
}

hipError_t cal_bind_set(CalSet& set, uint8_t* base, const uint16_t* k, const uint16_t* v, const uint16_t* q,
                        const int32_t* starts_host, int nseq, int H, int gq, int n_last, hipStream_t s) {
  std::vector<CalSeq> seqs(nseq);
  std::vector<int> row_seq;
  long long pel = 0;
  int rows = 0, maxlen = 0;
  for (int i = 0; i < nseq; ++i) {
    CalSeq& c = seqs[i];
    c.start = starts_host[i];
    c.len = starts_host[i + 1] - starts_host[i];
    c.t0 = c.len > n_last ? c.len - n_last : 0;
    c.row0 = rows;
    c.p0 = pel;
    maxlen = c.len > maxlen ? c.len : maxlen;
    const int nr = (c.len - c.t0) * gq;
    for (int r = 0; r < nr; ++r) row_seq.push_back(i);
    rows += nr;
    pel += (long long)nr * c.len;
  }
  set.k = k;
  set.v = v;
  set.q = q;
  set.T = starts_host[nseq] - starts_host[0];
  set.nseq = nseq;
  set.nrows = rows;
  set.pelems = pel;
  set.maxlen = maxlen;
  // tiles of up to kTileRows rows: 16 / gq positions of one sequence at a time
  std::vector<int4> tiles;
  const int per = gq >= kTileRows ? 1 : kTileRows / gq;
  for (int i = 0; i < nseq; ++i) {
    const CalSeq& cs = seqs[i];
    const int npos = cs.len - cs.t0;
    for (int pp = 0; pp < npos; pp += per)
      tiles.push_back(make_int4(i, cs.row0 + pp * gq, min(per, npos - pp) * gq, cs.t0 + pp));
  }
  set.ntiles = (int)tiles.size();
  const size_t nrow_el = (size_t)set.T * H * kD;
  uint8_t* p = base;
  set.seqs = reinterpret_cast<CalSeq*>(p);
  p += up256(sizeof(CalSeq) * (size_t)nseq);
  set.tiles = reinterpret_cast<int4*>(p);
  p += up256(sizeof(int4) * (size_t)rows);
  set.row_seq = reinterpret_cast<int*>(p);
  p += up256(sizeof(int) * (size_t)rows);
  set.zhat = reinterpret_cast<double*>(p);
  p += up256(nrow_el * 8);
  set.xeff = reinterpret_cast<double*>(p);
  p += up256(nrow_el * 8);
  set.gx = reinterpret_cast<double*>(p);
  p += up256(nrow_el * 8);
  set.gz = reinterpret_cast<double*>(p);
  p += up256(nrow_el * 8);
  set.mask = p;
  p += up256(nrow_el);
  set.pd = reinterpret_cast<double*>(p);
  p += up256((size_t)H * pel * 8);
  set.pf = reinterpret_cast<double*>(p);
  p += up256((size_t)H * pel * 8);
  set.fc = reinterpret_cast<double*>(p);
  p += up256((size_t)H * pel * 8);
  set.pc = reinterpret_cast<double*>(p);
  p += up256((size_t)H * pel * 8);
  set.rc = reinterpret_cast<double*>(p);
  p += up256((size_t)H * rows * 16);
  set.wt = reinterpret_cast<double*>(p);
  p += up256((size_t)H * rows * kD * 8);
  set.erow = reinterpret_cast<double*>(p);
  p += up256((size_t)H * rows * 8);
  set.wrow = reinterpret_cast<double*>(p);
  p += up256((size_t)H * rows * kD * 8);
  set.urow = reinterpret_cast<double*>(p);
  p += up256((size_t)H * rows * kD * 8);
  set.lrow = reinterpret_cast<double*>(p);
  hipError_t e = hipMemcpyAsync(set.seqs, seqs.data(), sizeof(CalSeq) * nseq, hipMemcpyHostToDevice, s);
  if (e == hipSuccess && rows > 0)
    e = hipMemcpyAsync(set.row_seq, row_seq.data(), sizeof(int) * rows, hipMemcpyHostToDevice, s);
  if (e == hipSuccess && !tiles.empty())
    e = hipMemcpyAsync(set.tiles, tiles.data(), sizeof(int4) * tiles.size(), hipMemcpyHostToDevice, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);  // the host tables go out of scope
  return e;
}

void cal_bind_shared(CalCfg& c, uint8_t* base) {
  uint8_t* p = base;
  c.gram = reinterpret_cast<double*>(p);
  p += up256((size_t)c.Hq * kMat * 8);
  c.R = reinterpret_cast<double*>(p);
  p += up256((size_t)c.H * kMat * 8);
  c.Rt = reinterpret_cast<double*>(p);
  p += up256((size_t)c.H * kMat * 8);
  c.ex = reinterpret_cast<double*>(p);
  p += up256((size_t)c.H * kCalScratch * kMat * 8);
  c.drp = reinterpret_cast<double*>(p);
  p += up256((size_t)kCalSplit * c.H * kMat * 8);
  c.dr = reinterpret_cast<double*>(p);
}

hipError_t cal_gram(const CalCfg& c, const uint16_t* W_o, hipStream_t s) {
  hipLaunchKernelGGL(cal_gram_kernel, dim3(c.Hq), dim3(512), 0, s, W_o, c.dm, c.Hq, c.gram);
  return hipGetLastError();
}

static void rot_and_quant(const CalCfg& c, CalSet& set, const double* A, int value, hipStream_t s) {
  hipLaunchKernelGGL(cal_expm_kernel, dim3(c.H), dim3(kExpThreads), 0, s, c, A, value);
  if (set.T > 0)
    hipLaunchKernelGGL(cal_rotq_kernel, dim3((set.T + kRotTile - 1) / kRotTile, c.H), dim3(512), 0, s, set, c, value);
}

static void backward(const CalCfg& c, CalSet& set, const double* A, int value, double* grad, hipStream_t s) {
  if (set.T > 0) {
    hipLaunchKernelGGL(cal_gx_kernel, dim3((set.T + kGxTok - 1) / kGxTok, c.H), dim3(256), 0, s, set, c, value);
    hipLaunchKernelGGL(cal_gz_kernel, dim3((set.T + kGzTile - 1) / kGzTile, c.H), dim3(256), 0, s, set, c);
    hipLaunchKernelGGL(cal_dr_kernel, dim3(c.H, kCalSplit), dim3(512), 0, s, set, c, value);
  } else {
    hipLaunchKernelGGL(cal_fill_kernel, dim3((unsigned)((kCalSplit * (size_t)c.H * kMat + 255) / 256)), dim3(256), 0,
                       s, c.drp, kCalSplit * (size_t)c.H * kMat, 0.0);
  }
  hipLaunchKernelGGL(cal_dr_reduce_kernel, dim3((unsigned)(((size_t)c.H * kMat + 255) / 256)), dim3(256), 0, s, c);
  hipLaunchKernelGGL(cal_expm_grad_kernel, dim3(c.H), dim3(kExpThreads), 0, s, c, A, value, grad);
}

// the tile kernels: one block per (tile, KV head)
#define CAL_POS_LAUNCH(KERNEL, ...) \
  hipLaunchKernelGGL(KERNEL, dim3(set.ntiles, c.H), dim3(kTileThreads), 0, s, __VA_ARGS__)

static void u_launch(const CalCfg& c, const CalSet& set, int value, hipStream_t s) {
  const int npos = set.nrows / c.gq;
  hipLaunchKernelGGL(cal_u_kernel, dim3(c.Hq, (npos + kUTile - 1) / kUTile), dim3(256), 0, s, set, c, value);
}

hipError_t cal_prepare_set(const CalCfg& c, CalSet& set, hipStream_t s) {
  if (set.nrows == 0) return hipSuccess;
  const size_t n = (size_t)c.H * set.pelems;
  hipLaunchKernelGGL(cal_fill_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, set.pd, n, 0.0);
  CAL_POS_LAUNCH(cal_const_kernel, set, c);
  return hipGetLastError();
}

hipError_t cal_key_loss(const CalCfg& c, CalSet& set, const double* A, double* loss, double* grad, hipStream_t s) {
  rot_and_quant(c, set, A, 0, s);
  if (set.nrows > 0) {
    CAL_POS_LAUNCH(cal_pos_fwd_kernel, set, c, 0);
    u_launch(c, set, 0, s);
    if (grad) CAL_POS_LAUNCH(cal_pos_grad_kernel, set, c);
    hipLaunchKernelGGL(cal_loss_kernel, dim3(c.H), dim3(256), 0, s, set.lrow, set.nrows, loss);
  } else {
    hipLaunchKernelGGL(cal_fill_kernel, dim3(1), dim3(256), 0, s, loss, (size_t)c.H, 0.0);
  }
  if (grad) {
    if (set.nrows == 0) {
      hipLaunchKernelGGL(cal_fill_kernel, dim3((unsigned)(((size_t)c.H * kMat + 255) / 256)), dim3(256), 0, s, grad,
                         (size_t)c.H * kMat, 0.0);
      return hipGetLastError();
    }
    backward(c, set, A, 0, grad, s);
  }
  return hipGetLastError();
}

hipError_t cal_key_probs(const CalCfg& c, CalSet& set, const double* A, hipStream_t s) {
  rot_and_quant(c, set, A, 0, s);
  if (set.nrows > 0) CAL_POS_LAUNCH(cal_pos_fwd_kernel, set, c, 1);
  return hipGetLastError();
}

hipError_t cal_value_loss(const CalCfg& c, CalSet& set, const double* A, double* loss, double* grad, hipStream_t s) {
  rot_and_quant(c, set, A, 1, s);
  if (set.nrows > 0) {
    CAL_POS_LAUNCH(cal_pos_val_kernel, set, c);
    u_launch(c, set, 1, s);
    hipLaunchKernelGGL(cal_loss_kernel, dim3(c.H), dim3(256), 0, s, set.lrow, set.nrows, loss);
  } else {
    hipLaunchKernelGGL(cal_fill_kernel, dim3(1), dim3(256), 0, s, loss, (size_t)c.H, 0.0);
  }
  if (grad) {
    if (set.nrows == 0) {
      hipLaunchKernelGGL(cal_fill_kernel, dim3((unsigned)(((size_t)c.H * kMat + 255) / 256)), dim3(256), 0, s, grad,
                         (size_t)c.H * kMat, 0.0);
      return hipGetLastError();
    }
    backward(c, set, A, 1, grad, s);
  }
  return hipGetLastError();
}

hipError_t cal_adam(double* A, const double* g, double* m, double* v, int n, int step, double lr, hipStream_t s) {
  const double bc1 = 1.0 - pow(0.9, (double)step), bc2 = 1.0 - pow(0.999, (double)step);
  hipLaunchKernelGGL(cal_adam_kernel, dim3((n + 255) / 256), dim3(256), 0, s, A, g, m, v, n, lr / bc1, sqrt(bc2), lr);
  return hipGetLastError();
}

hipError_t cal_select(const double* A, const double* loss, double* best, double* A_best, int H, hipStream_t s) {
  hipLaunchKernelGGL(cal_select_kernel, dim3(H), dim3(1024), 0, s, A, loss, best, A_best);
  return hipGetLastError();
}

hipError_t cal_record(const double* loss, double* dst, int stride, int H, hipStream_t s) {
  for (int h0 = 0; h0 < H; h0 += 64)
    hipLaunchKernelGGL(cal_record_kernel, dim3(1), dim3(64), 0, s, loss + h0, dst + (size_t)h0 * stride, stride,
                       min(64, H - h0));
  return hipGetLastError();
}

hipError_t cal_fill(double* p, size_t n, double v, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(cal_fill_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, p, n, v);
  return hipGetLastError();
}

hipError_t cal_rotation_out(const CalCfg& c, const double* A, bool value, float* out, hipStream_t s) {
  hipLaunchKernelGGL(cal_expm_kernel, dim3(c.H), dim3(kExpThreads), 0, s, c, A, value ? 1 : 0);
  const size_t n = (size_t)c.H * kMat;
  hipLaunchKernelGGL(cal_to_f32_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, c.R, out, n);
  return hipGetLastError();
}

hipError_t cal_key_mean(const uint16_t* k, int T, int H, float* mu, hipStream_t s) {
  hipLaunchKernelGGL(cal_key_mean_kernel, dim3(H), dim3(kD), 0, s, k, T, H, mu);
  return hipGetLastError();
}

}  // namespace int2kv
