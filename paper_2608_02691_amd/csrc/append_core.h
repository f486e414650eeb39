// Append on the matrix cores (shared by the append kernel and the decode's preparation kernel).
#pragma once
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace int2kv {

// Append on the matrix cores: x R (x bf16 [n, H, 128], R fp32 [128, 128]) as bf16 MFMA with R split
// into three bf16 terms (R = R_1 + R_2 + R_3 + O(2^-27 |R|): every product is exact and the sum is
// an fp32 accumulation, like an fp32 GEMM), starting from - mu R_K for keys; then the group
// quantizer and the packed stores. Work-group (KV head h, K or V, a stride of 16-token
// tiles); R^T of the work-group's (h, K|V) is converted once into LDS as the B operand.
// Tile layout: the product is formed transposed, D^T = R^T x^T, with R^T fragments as the A operand
// and token rows as the B operand. D^T[channel][token] of m-tile p (channels 16p .. 16p + 15) sits
// in lane token + 16 ((channel % 16) / 4), register channel % 4: lane (token, hi) holds channels
// 16 p + 4 hi + j, so register j of tiles p = 0..7 gives the eight 2-bit codes of half 4 hi + j of
// the packed layout, and the 32 channels of group g (tiles 2g, 2g + 1) sit in the four lanes of
// one token, eight in each. The group parameters are then computed once per (token, group).
typedef __bf16 ap_bf16x8_t __attribute__((ext_vector_type(8)));
typedef float ap_f4_t __attribute__((ext_vector_type(4)));

constexpr int kApWaves = 8;
constexpr int kApDepth = 6;   // R^T fragments in flight
constexpr int kApRow = 144;   // bf16 per LDS row of R^T (128 + 16 pad: conflict-free 16-byte reads)

// x / 3 correctly rounded, as a product with RN(1/3) and one FMA correction: checked against the
// correctly rounded quotient for every fp32 significand (so for every x whose intermediate values
// stay normal: x == 0 or x >= 2^-100; the caller routes other x to a division).
__device__ __forceinline__ float div3_rn(float x) {
#pragma clang fp contract(off)
  const float c = 0x1.555556p-2f;  // RN(1/3)
  const float q0 = x * c;
  const float r = __builtin_fmaf(-q0, 3.0f, x);
  return __builtin_fmaf(r, c, q0);
}

// The quantizer's group parameters (bit-identical to int2_group_params): s = fp16((mx - mn) / 3)
// with the division above, and 1/s from a table of the correctly rounded reciprocals of the 1024
// normal fp16 significands (exact after the power-of-two scaling); zero, fp16-subnormal and
// infinite scales and tiny ranges take the division.
__device__ __forceinline__ void int2_group_params_fast(float mn, float mx, float clip, const float* recip_tab,
                                                       uint32_t& s_bits, uint32_t& z_bits, float& zf, float& inv) {
#pragma clang fp contract(off)
  if (clip != 1.0f) {
    mn = clip * mn;
    mx = clip * mx;
  }
  const float range = mx - mn;
  float s32;
  if (range != 0.0f && range < 0x1p-100f)
    s32 = range / 3.0f;
  else
    s32 = div3_rn(range);
  const __half s = __float2half_rn(s32);
  const __half z = __float2half_rn(mn);
  s_bits = __half_as_ushort(s);
  z_bits = __half_as_ushort(z);
  zf = __half2float(z);
  const uint32_t e16 = (s_bits >> 10) & 31u;
  if (e16 == 0u || e16 == 31u) {  // zero, fp16-subnormal or infinite scale
    const float sf = __half2float(s);
    inv = sf > 0.0f ? 1.0f / sf : 0.0f;
  } else {
    inv = __builtin_ldexpf(recip_tab[s_bits & 1023u], 15 - (int)e16);
  }
}

// Cross-lane exchanges of the group reductions on the vector ALU (no LDS round trip).
// lane_swap32(a, b): lanes 32-63 of a trade places with lanes 0-31 of b, so afterwards lane l < 32
// holds (a[l], a[l + 32]) and lane l >= 32 holds (b[l - 32], b[l]). lane_swap16: the same between
// the odd 16-lane rows of a and the even rows of b, so a lane of an even row holds (a[l], a[l + 16])
// and a lane of an odd row (b[l - 16], b[l]).
struct LanePair {
  float a, b;
};
__device__ __forceinline__ LanePair lane_swap32(float a, float b) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(a), __float_as_uint(b), false, false);
  return LanePair{__uint_as_float(r[0]), __uint_as_float(r[1])};
}
__device__ __forceinline__ LanePair lane_swap16(float a, float b) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(a), __float_as_uint(b), false, false);
  return LanePair{__uint_as_float(r[0]), __uint_as_float(r[1])};
}

// Packed output of one lane for one 16-token tile: halves 4 hi .. 4 hi + 3 of its token (two per
// word) and the scale / zero of group hi.
struct ApOut {
  uint32_t w01, w23, meta;
  float err;  // with ERR: squared reconstruction error of the token's 128 channels (every lane of it)
};

// Group quantizer of one 16-token tile held in the transposed layout above.
// With ERR, also the token's squared reconstruction error sum_c (x_c - (code_c s + z))^2 in fp32
// (the rotated basis, where it equals the model basis' ||k - k~||^2: R is orthogonal).
template <int NG, bool ERR = false>
__device__ __forceinline__ ApOut quantize_tile(const ap_f4_t (&acc)[8], float clip, const float* recip_tab, int lo,
                                               int hi) {
  if constexpr (NG == 1) {
    // one group of 128 channels: the lane's 32 values, then the token's four lanes (xor 16, 32)
    float mn = acc[0][0], mx = acc[0][0];
#pragma unroll
    for (int p = 0; p < 8; ++p)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        mn = __builtin_elementwise_minimum(mn, acc[p][j]);
        mx = __builtin_elementwise_maximum(mx, acc[p][j]);
      }
    {
      const auto n16 = lane_swap16(mn, mn), x16 = lane_swap16(mx, mx);
      mn = __builtin_elementwise_minimum(n16.a, n16.b);
      mx = __builtin_elementwise_maximum(x16.a, x16.b);
      const auto n32 = lane_swap32(mn, mn), x32 = lane_swap32(mx, mx);
      mn = __builtin_elementwise_minimum(n32.a, n32.b);
      mx = __builtin_elementwise_maximum(x32.a, x32.b);
    }
    uint32_t s_bits, z_bits;
    float zf, inv;
    int2_group_params_fast(mn, mx, clip, recip_tab, s_bits, z_bits, zf, inv);
    float hf[4] = {0.f, 0.f, 0.f, 0.f};
    float e = 0.0f;
    const float sf = __half2float(__ushort_as_half((unsigned short)s_bits));
#pragma unroll
    for (int p = 0; p < 8; ++p)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
#pragma clang fp contract(off)
        const float t = (acc[p][j] - zf) * inv;
        const float c = __builtin_rintf(__builtin_amdgcn_fmed3f(t, 0.0f, 3.0f));
        hf[j] = __builtin_fmaf(c, (float)(1 << (2 * p)), hf[j]);
        if constexpr (ERR) {
          const float d = acc[p][j] - __builtin_fmaf(c, sf, zf);
          e = __builtin_fmaf(d, d, e);
        }
      }
    if constexpr (ERR) {
      e += __shfl_xor(e, 16);
      e += __shfl_xor(e, 32);
    }
    const uint32_t q0 = (uint32_t)hf[0], q1 = (uint32_t)hf[1], q2 = (uint32_t)hf[2], q3 = (uint32_t)hf[3];
    return ApOut{q0 | (q1 << 16), q2 | (q3 << 16), s_bits | (z_bits << 16), e};
  }
  // group g = tiles 2g, 2g + 1: lane-local min/max of its eight values, then a reduce-scatter
  // over the four lanes of the token (xor 32, then xor 16) leaves group hi's extremes in lane hi
  float pmn[4], pmx[4];
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    float a = __builtin_elementwise_minimum(acc[2 * g][0], acc[2 * g][1]), b = __builtin_elementwise_maximum(acc[2 * g][0], acc[2 * g][1]);
    a = __builtin_elementwise_minimum(a, __builtin_elementwise_minimum(acc[2 * g][2], acc[2 * g][3]));
    b = __builtin_elementwise_maximum(b, __builtin_elementwise_maximum(acc[2 * g][2], acc[2 * g][3]));
    a = __builtin_elementwise_minimum(a, __builtin_elementwise_minimum(acc[2 * g + 1][0], acc[2 * g + 1][1]));
    b = __builtin_elementwise_maximum(b, __builtin_elementwise_maximum(acc[2 * g + 1][0], acc[2 * g + 1][1]));
    pmn[g] = __builtin_elementwise_minimum(a, __builtin_elementwise_minimum(acc[2 * g + 1][2], acc[2 * g + 1][3]));
    pmx[g] = __builtin_elementwise_maximum(b, __builtin_elementwise_maximum(acc[2 * g + 1][2], acc[2 * g + 1][3]));
  }
  float mn, mx;
  {
    // lanes 0-31 keep groups 0 and 1, lanes 32-63 groups 2 and 3: one swap of (group g, group
    // g + 2) leaves both lanes' halves of the kept group in the swap's two results
    const auto n0 = lane_swap32(pmn[0], pmn[2]), n1 = lane_swap32(pmn[1], pmn[3]);
    const auto x0 = lane_swap32(pmx[0], pmx[2]), x1 = lane_swap32(pmx[1], pmx[3]);
    const float kn0 = __builtin_elementwise_minimum(n0.a, n0.b), kn1 = __builtin_elementwise_minimum(n1.a, n1.b);
    const float kx0 = __builtin_elementwise_maximum(x0.a, x0.b), kx1 = __builtin_elementwise_maximum(x1.a, x1.b);
    // even rows (hi 0, 2) keep the first of the two, odd rows the second: the same with rows of 16
    const auto n = lane_swap16(kn0, kn1), x = lane_swap16(kx0, kx1);
    mn = __builtin_elementwise_minimum(n.a, n.b);
    mx = __builtin_elementwise_maximum(x.a, x.b);
  }
  uint32_t s_bits, z_bits;
  float zf, inv;
  int2_group_params_fast(mn, mx, clip, recip_tab, s_bits, z_bits, zf, inv);
  // every lane of the token gathers the four groups' zero and reciprocal scale: a swap of rows of
  // 16 gives each lane (group 2 h1, group 2 h1 + 1), swaps of halves of 32 then give (group 0,
  // group 2) and (group 1, group 3) in every lane
  float zg[4], ig[4], sg[4];
  const float sfo = __half2float(__ushort_as_half((unsigned short)s_bits));
  auto gather4 = [](float v, float(&out)[4]) {
    const LanePair r = lane_swap16(v, v);
    const LanePair e = lane_swap32(r.a, r.a), o = lane_swap32(r.b, r.b);
    out[0] = e.a;
    out[1] = o.a;
    out[2] = e.b;
    out[3] = o.b;
  };
  gather4(zf, zg);
  gather4(inv, ig);
  if constexpr (ERR) gather4(sfo, sg);
  // codes: half 4 hi + j of the token collects tiles p = 0..7 of register j at bits 2p, summed as
  // exact small integers in fp32
  float hf[4] = {0.f, 0.f, 0.f, 0.f};
  float e = 0.0f;
#pragma unroll
  for (int p = 0; p < 8; ++p)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
#pragma clang fp contract(off)
      const float t = (acc[p][j] - zg[p >> 1]) * ig[p >> 1];
      const float c = __builtin_rintf(__builtin_amdgcn_fmed3f(t, 0.0f, 3.0f));
      hf[j] = __builtin_fmaf(c, (float)(1 << (2 * p)), hf[j]);
      if constexpr (ERR) {
        const float d = acc[p][j] - __builtin_fmaf(c, sg[p >> 1], zg[p >> 1]);
        e = __builtin_fmaf(d, d, e);
      }
    }
  if constexpr (ERR) {
    e += __shfl_xor(e, 16);
    e += __shfl_xor(e, 32);
  }
  const uint32_t q0 = (uint32_t)hf[0], q1 = (uint32_t)hf[1], q2 = (uint32_t)hf[2], q3 = (uint32_t)hf[3];
  return ApOut{q0 | (q1 << 16), q2 | (q3 << 16), s_bits | (z_bits << 16), e};
}

// Stores of one lane's ApOut into the record of its token's slot (skipped for slots out of range).
// With one group per token (NG = 1) the four lanes of a token hold the same metadata; lane hi = 0
// stores it.
template <int NG>
__device__ __forceinline__ void store_tile(const ApOut& o, int slot, const CacheView& cv, int h, int kv, int nslots,
                                           int hi) {
  using L = Rec<NG>;
  if (slot >= 0 && slot < nslots) {
    const int blk = slot >> 4, t = slot & 15;
    uint8_t* rec = cv.pool + ((size_t)blk * cv.num_kv_heads + h) * L::kBytes;
    const bool meta = NG == 4 || hi == 0;
    const int g = NG == 4 ? hi : 0;
    if (kv == 0) {
      *reinterpret_cast<uint2*>(rec + kOffKCodes + 32 * t + 8 * hi) = make_uint2(o.w01, o.w23);
      if (meta) *reinterpret_cast<uint32_t*>(rec + L::kOffKMeta + 4 * NG * t + 4 * g) = o.meta;
    } else {
      uint8_t* vc = rec + kOffVCodes + 32 * 4 * hi + 2 * t;
      *reinterpret_cast<uint16_t*>(vc) = (uint16_t)o.w01;
      *reinterpret_cast<uint16_t*>(vc + 32) = (uint16_t)(o.w01 >> 16);
      *reinterpret_cast<uint16_t*>(vc + 64) = (uint16_t)o.w23;
      *reinterpret_cast<uint16_t*>(vc + 96) = (uint16_t)(o.w23 >> 16);
      if (meta) {
        *reinterpret_cast<uint16_t*>(rec + L::kOffVScale + 32 * g + 2 * t) = (uint16_t)o.meta;
        *reinterpret_cast<uint16_t*>(rec + L::kOffVZero + 32 * g + 2 * t) = (uint16_t)(o.meta >> 16);
      }
    }
  }
}

// Optional stages of the cache write. RoPE (with ROPE): the keys arrive pre-RoPE and each token is
// turned at its position into its post-RoPE bf16 row first (rotate-half pairs (i, i + 64); each
// output evaluated in fp64, where both products are exact, and rounded once to bf16), optionally
// stored to k_out. Hadamard (bit 0 of had for keys, bit 1 for values): the rotation is
// H_128 / sqrt(128) instead of R; its +-1 entries are exact bf16 operands, so one matrix-core pass
// replaces the three-term split, and the fp32 sum is scaled by RN(2^-3.5) afterwards.
struct ApOpts {
  const int32_t* pos = nullptr;    // token positions (ROPE)
  const float* cos_sin = nullptr;  // fp32 [max_pos, 128]: cos of the 64 angles, then their sines
  int max_pos = 0;
  uint16_t* k_out = nullptr;       // post-RoPE keys, bf16 [n, H, 128], or null
  int had = 0;
};

constexpr float kHadScale = 0x1.6a09e6p-4f;  // RN(1 / sqrt(128))

// fp64 to bf16, nearest even, in two steps that cannot double-round: to fp32 by rounding to odd
// (round toward zero, then set the last bit when inexact; Boldo and Melquiond's rounding to odd),
// then to bf16 by nearest even, which is exact rounding because fp32 keeps 16 more bits.
__device__ __forceinline__ uint32_t f64_to_bf16_rne(double d) {
  float r = (float)d;
  if ((double)r != d) {
    uint32_t b = __float_as_uint(r);
    if (fabs((double)r) > fabs(d)) b -= 1u;  // rounded away from zero: one ulp back toward it
    r = __uint_as_float(b | 1u);
  }
  return f32_to_bf16_rne(r);
}

// RoPE of one lane's slice of a token row in place: X[ks] holds channels 32 ks + 8 hi + e
// (e = 0..7), so pairs (i, i + 64) are (X[ks][e], X[ks + 2][e]) for ks = 0, 1; cs points at the
// token's table row.
__device__ __forceinline__ void rope_lane(ap_bf16x8_t (&X)[4], const float* __restrict__ cs, int hi) {
#pragma clang fp contract(off)
  float c[2][8], sn[2][8];
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
    const float4* cp = reinterpret_cast<const float4*>(cs + 32 * ks + 8 * hi);
    const float4* sp = reinterpret_cast<const float4*>(cs + 64 + 32 * ks + 8 * hi);
    const float4 c0 = cp[0], c1 = cp[1], s0 = sp[0], s1 = sp[1];
    c[ks][0] = c0.x; c[ks][1] = c0.y; c[ks][2] = c0.z; c[ks][3] = c0.w;
    c[ks][4] = c1.x; c[ks][5] = c1.y; c[ks][6] = c1.z; c[ks][7] = c1.w;
    sn[ks][0] = s0.x; sn[ks][1] = s0.y; sn[ks][2] = s0.z; sn[ks][3] = s0.w;
    sn[ks][4] = s1.x; sn[ks][5] = s1.y; sn[ks][6] = s1.z; sn[ks][7] = s1.w;
  }
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
    uint4 a = __builtin_bit_cast(uint4, X[ks]), b = __builtin_bit_cast(uint4, X[ks + 2]);
    uint32_t aw[4] = {a.x, a.y, a.z, a.w}, bw[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      uint32_t oa = 0u, ob = 0u;
#pragma unroll
      for (int hlf = 0; hlf < 2; ++hlf) {
        const int e = 2 * q + hlf;
        const double x1 = (double)__uint_as_float((aw[q] >> (16 * hlf)) << 16);
        const double x2 = (double)__uint_as_float((bw[q] >> (16 * hlf)) << 16);
        const double cc = (double)c[ks][e], ss = (double)sn[ks][e];
        const double y1 = x1 * cc - x2 * ss;  // exact products, one rounding
        const double y2 = x2 * cc + x1 * ss;
        oa |= f64_to_bf16_rne(y1) << (16 * hlf);
        ob |= f64_to_bf16_rne(y2) << (16 * hlf);
      }
      aw[q] = oa;
      bw[q] = ob;
    }
    X[ks] = __builtin_bit_cast(ap_bf16x8_t, make_uint4(aw[0], aw[1], aw[2], aw[3]));
    X[ks + 2] = __builtin_bit_cast(ap_bf16x8_t, make_uint4(bw[0], bw[1], bw[2], bw[3]));
  }
}

// Each wave takes kApTiles consecutive 16-token tiles per step, so every R^T fragment read from
// LDS feeds kApTiles products (two for long appends; one for short ones, which spreads the few
// tiles over more waves).
// LDS of one append work-group: R^T as three bf16 terms, then the reciprocal table.
constexpr int kAppendLdsBytes = 3 * kHeadDim * kApRow * 2 + 1024 * 4;

// One append work-group of kWaves waves: KV head h, K (kv = 0) or V (kv = 1), block bx of nbx
// striding over the 16-token tiles; lds holds kAppendLdsBytes (16-byte aligned). Every thread of
// the block must call it (it synchronizes once).
// With ERR, err[(token * H + h) * 2 + kv] receives each token's squared reconstruction error.
// With ROPE, opt carries the positions and table (keys only); opt.had selects the Hadamard rotation.
template <int kApTiles, int kWaves, int NG, bool ERR = false, bool ROPE = false>
__device__ __forceinline__ void append_block(const CacheView& cv, const uint16_t* __restrict__ k,
                                             const uint16_t* __restrict__ v, const int32_t* __restrict__ slots,
                                             int n, const float* __restrict__ R_k, const float* __restrict__ R_v,
                                             const float* __restrict__ mu_rk, float clip_k, float clip_v, int bx,
                                             int nbx, int h, int kv, uint8_t* lds, float* __restrict__ err = nullptr,
                                             const ApOpts& opt = ApOpts{}) {
  uint16_t(*rt)[kHeadDim][kApRow] = reinterpret_cast<uint16_t(*)[kHeadDim][kApRow]>(lds);  // [term][c][i] = R[i][c]
  float* recip_tab = reinterpret_cast<float*>(lds + 3 * kHeadDim * kApRow * 2);  // RN(1 / (1 + m / 1024))
  const int H = cv.num_kv_heads, tid = threadIdx.x;
  const bool had = ((opt.had >> kv) & 1) != 0;
  const float* R = had ? nullptr : (kv == 0 ? R_k : R_v) + (size_t)h * kHeadDim * kHeadDim;
  const bool rope = ROPE && kv == 0;
  const int w = tid >> 6, l = tid & 63, lo = l & 15, hi = l >> 4;
  const uint16_t* X = kv == 0 ? k : v;
  constexpr int kStep = 16 * kApTiles;  // tokens per wave step
  // the first step's operands and slots are fetched before R, so their latency overlaps R's
  const int step0 = bx * kWaves + w;
  ap_bf16x8_t X8[kApTiles][4];
  int slot[kApTiles], pos[kApTiles];
#pragma unroll
  for (int u = 0; u < kApTiles; ++u) {
    const int tok = step0 * kStep + 16 * u + lo, tc = min(tok, n - 1);
    const uint16_t* xrow = X + ((size_t)tc * H + h) * kHeadDim + 8 * hi;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) X8[u][ks] = *reinterpret_cast<const ap_bf16x8_t*>(xrow + 32 * ks);
    slot[u] = slots[tc];
    if (tok >= n) slot[u] = -1;
    pos[u] = rope ? opt.pos[tc] : 0;
  }
  if (had) {
    // H^T = H: thread (c, i0) writes entries (i0 .. i0 + 7, c) = (-1)^popcount(i & c) as bf16 +-1
    constexpr int kIb = kWaves / 2;
    const int c = tid & 127, ib = tid >> 7;
#pragma unroll
    for (int u = 0; u < 16 / kIb; ++u) {
      const int i0 = 8 * (ib + kIb * u);
      uint32_t t16[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) t16[q] = (__builtin_popcount((i0 + q) & c) & 1) ? 0xBF80u : 0x3F80u;
      *reinterpret_cast<uint4*>(&rt[0][c][i0]) =
          make_uint4(t16[0] | (t16[1] << 16), t16[2] | (t16[3] << 16), t16[4] | (t16[5] << 16), t16[6] | (t16[7] << 16));
    }
  } else {
    // R^T as three bf16 terms: thread (c, i0) reads R[i0 .. i0 + 7][c] (coalesced over c) and
    // splits each value by truncation: r = t0 + t1 + t2 exactly (t0 and t1 take the leading 8
    // significant bits of r and of r - t0, the remainder has at most 8 left), then writes one
    // 16-byte row piece per term (conflict-free)
    constexpr int kIb = kWaves / 2;  // threads per channel c
    const int c = tid & 127, ib = tid >> 7;
#pragma unroll
    for (int u = 0; u < 16 / kIb; ++u) {
      const int i0 = 8 * (ib + kIb * u);
      uint32_t t16[3][8];
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const float r = R[(i0 + q) * kHeadDim + c];
        const uint32_t b0 = __float_as_uint(r) & 0xFFFF0000u;
        const float r1 = r - __uint_as_float(b0);
        const uint32_t b1 = __float_as_uint(r1) & 0xFFFF0000u;
        const float r2 = r1 - __uint_as_float(b1);
        t16[0][q] = b0 >> 16;
        t16[1][q] = b1 >> 16;
        t16[2][q] = __float_as_uint(r2) >> 16;
      }
#pragma unroll
      for (int term = 0; term < 3; ++term)
        *reinterpret_cast<uint4*>(&rt[term][c][i0]) =
            make_uint4(t16[term][0] | (t16[term][1] << 16), t16[term][2] | (t16[term][3] << 16),
                       t16[term][4] | (t16[term][5] << 16), t16[term][6] | (t16[term][7] << 16));
    }
  }
  for (int m = tid; m < 1024; m += 64 * kWaves) recip_tab[m] = 1.0f / (1.0f + (float)m * 0x1p-10f);
  __syncthreads();
  // lane (token lo, hi) holds channels 16 p + 4 hi + j of its token in register j of tile p
  ap_f4_t sub[8];
#pragma unroll
  for (int p = 0; p < 8; ++p)
    sub[p] = kv == 0 ? -*reinterpret_cast<const ap_f4_t*>(mu_rk + (size_t)h * kHeadDim + 16 * p + 4 * hi)
                     : ap_f4_t{0.f, 0.f, 0.f, 0.f};
  const float clip = kv == 0 ? clip_k : clip_v;
  const int nslots = cv.num_blocks * kBlock;
  // software pipeline over the wave's steps: the next step's operands and slots are fetched while
  // this one is computed (indexes clamped, so the fetch past the last step stays in bounds)
  const int sstride = nbx * kWaves;
  for (int st = step0; st * kStep < n; st += sstride) {
    if (rope) {
      // this step's keys become post-RoPE rows; a position outside the table skips the token
#pragma unroll
      for (int u = 0; u < kApTiles; ++u) {
        const int tok = st * kStep + 16 * u + lo;
        const bool ok = pos[u] >= 0 && pos[u] < opt.max_pos;
        if (!ok) slot[u] = -1;
        rope_lane(X8[u], opt.cos_sin + (size_t)(ok ? pos[u] : 0) * kHeadDim, hi);
        if (opt.k_out && ok && tok < n) {
          uint16_t* orow = opt.k_out + ((size_t)tok * H + h) * kHeadDim + 8 * hi;
#pragma unroll
          for (int ks = 0; ks < 4; ++ks) *reinterpret_cast<ap_bf16x8_t*>(orow + 32 * ks) = X8[u][ks];
        }
      }
    }
    ap_bf16x8_t Xn[kApTiles][4];
    int slotn[kApTiles], posn[kApTiles];
#pragma unroll
    for (int u = 0; u < kApTiles; ++u) {
      const int tok = (st + sstride) * kStep + 16 * u + lo, tc = min(tok, n - 1);
      const uint16_t* xrow = X + ((size_t)tc * H + h) * kHeadDim + 8 * hi;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) Xn[u][ks] = *reinterpret_cast<const ap_bf16x8_t*>(xrow + 32 * ks);
      slotn[u] = slots[tc];
      posn[u] = rope ? opt.pos[tc] : 0;
    }
    ap_f4_t acc[kApTiles][8];  // start at - mu R_K (keys) or 0 (values); 0 for the Hadamard product
#pragma unroll
    for (int u = 0; u < kApTiles; ++u)
#pragma unroll
      for (int p = 0; p < 8; ++p) acc[u][p] = had ? ap_f4_t{0.f, 0.f, 0.f, 0.f} : sub[p];
    // the R^T fragments are the same for every step: an opaque offset keeps the compiler from
    // hoisting all 96 of them into registers (which would cap occupancy at one wave per SIMD)
    int boff = (lo * kApRow + 8 * hi) * 2;
    asm volatile("" : "+v"(boff));
    const uint8_t* rb = reinterpret_cast<const uint8_t*>(&rt[0][0][0]) + boff;
    // fragment f = (term 2 - f / 32, k-step (f / 8) % 4, m-tile f % 8): smallest term first. The
    // LDS reads run kApDepth fragments ahead of the matrix cores (the schedule is pinned below).
    auto frag = [&](int f) {
      const int term = 2 - f / 32, ks = (f / 8) % 4, p = f % 8;
      return *reinterpret_cast<const ap_bf16x8_t*>(rb + ((term * kHeadDim + 16 * p) * kApRow + 32 * ks) * 2);
    };
    // fragments F0 .. 95: all three terms (F0 = 0) or the Hadamard's single +-1 term (F0 = 64)
    auto mfma_pass = [&](auto f0_tag) {
      constexpr int F0 = decltype(f0_tag)::value;
      ap_bf16x8_t fr[kApDepth];
#pragma unroll
      for (int f = 0; f < kApDepth; ++f) fr[f] = frag(F0 + f);
#pragma unroll
      for (int f = F0; f < 96; ++f) {
        const ap_bf16x8_t a = fr[(f - F0) % kApDepth];
        const int ks = (f / 8) % 4, p = f % 8;
#pragma unroll
        for (int u = 0; u < kApTiles; ++u)
          acc[u][p] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, X8[u][ks], acc[u][p], 0, 0, 0);
        if (f + kApDepth < 96) fr[(f - F0) % kApDepth] = frag(f + kApDepth);
      }
#pragma unroll
      for (int f = 0; f < kApDepth; ++f) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
#pragma unroll
      for (int f = F0; f < 96; ++f) {
        __builtin_amdgcn_sched_group_barrier(0x008, kApTiles, 0);  // MFMA
        if (f + kApDepth < 96) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
    };
    // a wave in its matrix-core phase is issued first: the other wave of the SIMD fills the gaps
    // between its products with quantizer instructions
    __builtin_amdgcn_s_setprio(1);
    if (had) {
      mfma_pass(std::integral_constant<int, 64>{});
#pragma unroll
      for (int u = 0; u < kApTiles; ++u)
#pragma unroll
        for (int p = 0; p < 8; ++p)
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[u][p][j] = __builtin_fmaf(acc[u][p][j], kHadScale, sub[p][j]);
    } else {
      mfma_pass(std::integral_constant<int, 0>{});
    }
    __builtin_amdgcn_s_setprio(0);
    ApOut out[kApTiles];
#pragma unroll
    for (int u = 0; u < kApTiles; ++u) out[u] = quantize_tile<NG, ERR>(acc[u], clip, recip_tab, lo, hi);
    // the next step's loads are waited for here, before this step's stores: a wait placed after
    // the (lane-conditional) stores would also wait for the stores to complete
#pragma unroll
    for (int u = 0; u < kApTiles; ++u) {
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) asm volatile("" : "+v"(Xn[u][ks])::"memory");
      asm volatile("" : "+v"(slotn[u])::"memory");
      if (rope) asm volatile("" : "+v"(posn[u])::"memory");
    }
#pragma unroll
    for (int u = 0; u < kApTiles; ++u) store_tile<NG>(out[u], slot[u], cv, h, kv, nslots, hi);
    if constexpr (ERR) {
#pragma unroll
      for (int u = 0; u < kApTiles; ++u) {
        const int tok = st * kStep + 16 * u + lo;
        if (hi == 0 && tok < n) err[((size_t)tok * H + h) * 2 + kv] = out[u].err;
      }
    }
#pragma unroll
    for (int u = 0; u < kApTiles; ++u) {
      const int tok = (st + sstride) * kStep + 16 * u + lo;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) X8[u][ks] = Xn[u][ks];
      slot[u] = tok < n ? slotn[u] : -1;
      pos[u] = posn[u];
    }
  }
}

}  // namespace int2kv
