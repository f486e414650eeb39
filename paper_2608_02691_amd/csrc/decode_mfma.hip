// Matrix-core split-context scan of the INT2 decode attention (gfx950, v_mfma_f32_16x16x32_f16).
//
// What is computed is the same as the vector-ALU scan (eq:int2_attention in the rotated-query
// form of the appendix): a_s = (q R_K) . (c_s * s + z) / sqrt(d) per group (32 or 128 channels), an
// online softmax, and O' = sum_s p_s (c_s * s + z) in R_V coordinates. The affine metadata is
// factored out of both contractions so the 2-bit codes enter the matrix cores unchanged:
//
//   scores : D[(j,g), t] = sum_{k in g} q'_jk c_tk          (MFMA, rows = head x group)
//            a_jt = sum_g s_tg D[(j,g), t] + sum_g z_tg sum_{k in g} q'_jk
//   values : O'[c, (j,g)] = sum_t (p_jt s_tg) c_tc + sum_t p_jt z_tg   (MFMA, K = tokens)
//
// A 2-bit code c sitting at bits 2x..2x+1 of a 16-bit half becomes the fp16 number 1 + c*2^-e
// with one AND-OR (after at most one shift): the code lands in mantissa bits 4..9 of the fp16 1.0
// pattern. e in {2, 4, 6} depends only on x. For the scores the constant 1 and the factor 2^-e
// are folded into the query operand (scaled by 2^e per channel, with sum_k A_k subtracted through
// the accumulator's initial value); for the values they are removed from the accumulator at the
// end (O = 2^e (D - sum_t w_t)), using the exact fp16 weights the matrix core multiplied.
#include "append_core.h"
#include "common.h"
#include "kernels.h"

namespace int2kv {

typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef float float4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr float kLogit2 = 1.4426950408889634f * 0.08838834764831845f;  // log2(e)/sqrt(128)
constexpr int kWavesM = 4;
constexpr float kRescaleTau = 8.0f;  // lazy rescaling: keep the running max until exceeded by 2^8
// Starting reference max: finite, so a segment whose tokens are all masked (-inf scores) still gives
// p = exp2(-inf - m0) = 0 rather than NaN; any real score exceeds it by more than 2^tau.
constexpr float kMaxInit = -1.0e30f;
constexpr int kQopTile = 4096 + 512;  // A operands (4 blocks x 64 lanes x 16 B) + constants

bool mfma_decode_available() { return true; }

size_t qop_bytes(int B, int H, int gq) {
  (void)gq;
  return (size_t)B * H * kQopTile;
}

// Class e of bit position x after the landing shift: the fp16 value is 1 + code * 2^-e.
__host__ __device__ constexpr int land_e(int x) {
  return (x == 4 || x == 7) ? 2 : ((x == 1 || x == 3 || x == 6) ? 4 : 6);
}

// Landing constants held in registers: the masks of code positions 2, 3, 4 (SGPRs) and the fp16
// 1.0 pattern (VGPR). They pass through empty asm statements (no instruction) so the compiler cannot
// fold them into literals; with all three operands in registers a landing selects one v_and_or_b32
// instead of a v_and_b32 / v_or_b32 pair with literals.
struct LandK {
  uint32_t m[3];  // 0x00030003 << 2 pos, pos = 2, 3, 4
  uint32_t one;   // 0x3C003C00
};
__device__ __forceinline__ LandK land_constants() {
  LandK k{{0x00300030u, 0x00C000C0u, 0x03000300u}, 0x3C003C00u};
  asm volatile("" : "+s"(k.m[0]), "+s"(k.m[1]), "+s"(k.m[2]), "+v"(k.one));
  return k;
}

// The codes at position X of both 16-bit halves of w, as an fp16 pair (1 + c_lo 2^-e, 1 + c_hi 2^-e):
// one AND-OR after at most one shift. Plain C, not inline asm: the compiler sees the VGPR write and
// keeps the matrix-core operand hazards around it (an asm landing placed right after an MFMA that
// still has to read the same registers corrupts that MFMA's inputs).
template <int X>
__device__ __forceinline__ uint32_t land(uint32_t w, const LandK& k) {
  constexpr int pos = X >= 5 ? X - 3 : (X <= 1 ? X + 2 : X);
  const uint32_t v = X >= 5 ? (w >> 6) : (X <= 1 ? (w << 4) : w);
  return (v & k.m[pos - 2]) | k.one;
}

__device__ __forceinline__ void lds_sync_wave() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ half2_t as_h2(uint32_t u) { return __builtin_bit_cast(half2_t, u); }
__device__ __forceinline__ uint32_t as_u(half2_t h) { return __builtin_bit_cast(uint32_t, h); }

__device__ __forceinline__ int seq_len_m(const DecodeArgs& a, int b) {
  int L = a.ctx_lens[b];
  L = min(L, a.max_ctx);
  L = min(L, a.max_blocks * kBlock);
  return max(L, 0);
}

// ---------------------------------------------------------------------------------------------
// Query operands of one (sequence, KV head): q' = q R_K (fp32) scaled by log2(e)/sqrt(d) and a
// per-head power of two sigma, laid out as the MFMA A operand of the score contraction: a row holds
// q'_j on the channels of one group, times 2^e of the channel's code position, as fp16 (row layouts:
// see the scan below). Constants: -sum_k A_k per row (accumulator start), sum_{k in g} q'_jk (for the
// zero term) and 1/sigma. sigma comes from the row's norm, which bounds every |q'_c| (R_K orthogonal):
// sigma |q'|_2 < 512, so every A value stays below 2^15 at the largest code factor 2^6.
// One block serves KV head h of kQpSeqs sequences and 128 / SPLIT channels of q' (whole groups:
// the operand block of group g and the group's constants only need its channels): those columns of
// R_K[h] go into LDS as the B operand of a bf16 matrix-core product (split into two bf16 terms, as in
// the cache write: error below 2^-17 |R|); the query rows are exact in bf16. Rows s * 8 + jj = query
// head jj of sequence b0 + s (16-row tiles, wave w owns tile w).
constexpr int kQpSeqs = 8;
constexpr int kQpRow = 136;   // bf16 per LDS row of R^T (128 + 8 pad: conflict-free 16-byte reads)
typedef __bf16 qp_bf16x8_t __attribute__((ext_vector_type(8)));

// LDS of the query-operand role with SPLIT blocks per (KV head, sequences): the block's columns of
// R^T as bf16 hi / lo, its q' columns, the per-row scale (the largest size, SPLIT = 1).
constexpr int qp_lds_bytes(int split) {
  return 2 * (kHeadDim / split) * kQpRow * 2 + 8 * kQpSeqs * (kHeadDim / split + 4) * 4 + 8 * kQpSeqs * 4;
}
constexpr int kQpLdsBytes = qp_lds_bytes(1);
static_assert(qp_lds_bytes(4) >= 512 * 4, "the page-prefix block's two 256-entry scans fit the query role's LDS");

template <int SPLIT>
__device__ void qprep_block(const DecodeArgs& a, int blk, bool wide, uint8_t* lds) {
  constexpr int kQpSplit = SPLIT, kQpCols = kHeadDim / SPLIT;
  uint16_t(*Rt)[kQpCols][kQpRow] = reinterpret_cast<uint16_t(*)[kQpCols][kQpRow]>(lds);  // [hi, lo][c][k] = R[k][32 g + c]
  float(*qb)[kQpCols + 4] = reinterpret_cast<float(*)[kQpCols + 4]>(lds + 2 * kQpCols * kQpRow * 2);  // q' rows
  float* sig = reinterpret_cast<float*>(lds + 2 * kQpCols * kQpRow * 2 + 8 * kQpSeqs * (kQpCols + 4) * 4);
  const int H = a.H, gq = a.gq, tid = threadIdx.x;
  constexpr int kGpb = kQpCols / 32;  // groups per block
  const int g0 = (blk % kQpSplit) * kGpb, hb = blk / kQpSplit;
  const int h = hb % H, b0 = kQpSeqs * (hb / H), nseq = min(kQpSeqs, a.B - b0);
  const int w = tid >> 6, l = tid & 63, lo = l & 15, hi = l >> 4;
  // A operand (query rows 16 w + lo, 8 consecutive channels per lane), fetched before R so the
  // two latencies overlap; absent rows are zero
  qp_bf16x8_t A[4];
  float ss = 0.0f;  // sum of squares of the lane's 32 channels
  {
    const int row = 16 * w + lo, sq = row >> 3, jj = row & 7;
    const bool ok = sq < nseq && jj < gq;
    const uint16_t* qr = a.q + ((size_t)(b0 + (ok ? sq : 0)) * a.Hq + h * gq + (ok ? jj : 0)) * kHeadDim + 8 * hi;
    const uint32_t keep = ok ? ~0u : 0u;  // a mask, not a select: the loads stay unconditional
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const uint4 v = *reinterpret_cast<const uint4*>(qr + 32 * ks);
      const uint32_t u[4] = {v.x & keep, v.y & keep, v.z & keep, v.w & keep};
      A[ks] = __builtin_bit_cast(qp_bf16x8_t, make_uint4(u[0], u[1], u[2], u[3]));
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float x0 = __uint_as_float(u[e] << 16), x1 = __uint_as_float(u[e] & 0xFFFF0000u);
        ss = fmaf(x0, x0, fmaf(x1, x1, ss));
      }
    }
  }
  {
    // the block's columns of R as bf16 hi/lo rows of R^T: thread (c, kb) reads R[k0 .. k0 + 7][32 g0 + c]
    // for k0 = 8 (kb + kKb u) (coalesced over c) and writes one 16-byte row piece per term
    constexpr int kKb = 256 / kQpCols, kNu = 16 / kKb;
    const float* R = a.R_k + (size_t)h * kHeadDim * kHeadDim + 32 * g0;
    const int c = tid & (kQpCols - 1), kb = tid / kQpCols;
    float rall[kNu][8];
#pragma unroll
    for (int u = 0; u < kNu; ++u)
#pragma unroll
      for (int q = 0; q < 8; ++q) rall[u][q] = R[(8 * (kb + kKb * u) + q) * kHeadDim + c];
#pragma unroll
    for (int u = 0; u < kNu; ++u) {
      const int k0 = 8 * (kb + kKb * u);
      const float* r8 = rall[u];
      uint32_t hw[4], lw[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t h0 = f32_to_bf16_rne(r8[2 * q]), h1 = f32_to_bf16_rne(r8[2 * q + 1]);
        hw[q] = h0 | (h1 << 16);
        lw[q] = f32_to_bf16_rne(r8[2 * q] - __uint_as_float(h0 << 16)) |
                (f32_to_bf16_rne(r8[2 * q + 1] - __uint_as_float(h1 << 16)) << 16);
      }
      *reinterpret_cast<uint4*>(&Rt[0][c][k0]) = make_uint4(hw[0], hw[1], hw[2], hw[3]);
      *reinterpret_cast<uint4*>(&Rt[1][c][k0]) = make_uint4(lw[0], lw[1], lw[2], lw[3]);
    }
  }
  // sigma of row 16 w + lo from |q|_2 (the four lanes hi of the row hold its 128 channels):
  // max_c |q'_c| <= log2(e)/sqrt(d) |q|_2 (with a 2^-10 margin for the rounding of the sum and of
  // the product's terms), sigma = 2^(9 - ex) for that bound below 2^ex
  ss += __shfl_xor(ss, 16);
  ss += __shfl_xor(ss, 32);
  if (hi == 0) {
    const float m = sqrtf(ss) * (kLogit2 * (1.0f + 0x1p-10f));
    int ex = 0;
    frexpf(m, &ex);
    sig[16 * w + lo] = m > 0.0f ? ldexpf(1.0f, max(-100, min(100, 9 - ex))) : 1.0f;
  }
  __syncthreads();
  // D[row][c] of n-tile p sits in lane (c % 16) + 16 (row / 4), register row % 4
#pragma unroll
  for (int p = 0; p < kQpCols / 16; ++p) {
    float4_t d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const qp_bf16x8_t bh = *reinterpret_cast<const qp_bf16x8_t*>(&Rt[0][16 * p + lo][32 * ks + 8 * hi]);
      const qp_bf16x8_t bl = *reinterpret_cast<const qp_bf16x8_t*>(&Rt[1][16 * p + lo][32 * ks + 8 * hi]);
      d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A[ks], bh, d, 0, 0, 0);
      d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A[ks], bl, d, 0, 0, 0);
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) qb[16 * w + 4 * hi + r][16 * p + lo] = d[r] * kLogit2;
  }
  __syncthreads();
  // A operand chunks of the block's groups g: (sequence, g, lane l) -> 8 fp16 values. Lane l = m + 16 q
  // holds row m, which belongs to query head jj and is nonzero only in the blocks of its group slot:
  // narrow rows (j, g) = 4 j + g in block g; wide rows (j, gg) = 2 j + gg in the blocks i with
  // i % 2 = gg. Its eight values are channels 32 g + 4 q + 0..3 (code position x = 2 g) and
  // 32 g + 16 + 4 q + 0..3 (x = 2 g + 1), scaled by sigma and 2^e(x).
  for (int cidx = tid; cidx < nseq * kGpb * 64; cidx += 256) {
    const int sq = cidx / (kGpb * 64), gi = (cidx / 64) % kGpb, l = cidx & 63, g = g0 + gi;
    const int m = l & 15, q = l >> 4;
    const int jj = wide ? m >> 1 : m >> 2;
    // with one group per token every block sits in row (j, 0) (the scan then reads one dense dot)
    const int gs = a.groups == 1 ? 0 : g;
    const bool on = wide ? (m & 1) == (gs & 1) : (m & 3) == gs;
    const int row = 8 * sq + jj;
    uint32_t packed[4] = {0u, 0u, 0u, 0u};
    if (on && jj < gq) {
      const float4 lo4 = *reinterpret_cast<const float4*>(&qb[row][32 * gi + 4 * q]);
      const float4 hi4 = *reinterpret_cast<const float4*>(&qb[row][32 * gi + 16 + 4 * q]);
      const float s0 = sig[row] * (float)(1 << land_e(2 * g)), s1 = sig[row] * (float)(1 << land_e(2 * g + 1));
      const float v[8] = {lo4.x * s0, lo4.y * s0, lo4.z * s0, lo4.w * s0, hi4.x * s1, hi4.y * s1, hi4.z * s1, hi4.w * s1};
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const _Float16 h0 = (_Float16)v[2 * u], h1 = (_Float16)v[2 * u + 1];
        packed[u] = (uint32_t)__builtin_bit_cast(uint16_t, h0) | ((uint32_t)__builtin_bit_cast(uint16_t, h1) << 16);
      }
    }
    uint8_t* out = a.qop + ((size_t)(b0 + sq) * H + h) * kQopTile;
    *reinterpret_cast<uint4*>(out + (g * 64 + l) * 16) = make_uint4(packed[0], packed[1], packed[2], packed[3]);
  }
  // Per (query head jj, group g): -sum of the row's 32 fp16 A values in block g (the accumulator
  // start of that row's tile), sum of q' over group g, and 1/sigma (group 0); thread -> (row, g), a
  // sequential sum over the group's channels. Narrow layout after the 4096 bytes of A operands:
  // start[4 jj + g], qsum[16 + 4 jj + g], 1/sigma[32 + jj]; wide: start of D01 [2 jj + g] (g < 2)
  // and of D23 [16 + 2 jj + g - 2] (g >= 2), qsum[32 + 4 jj + g], 1/sigma[64 + jj] (floats).
  if (tid < 8 * kQpSeqs * kGpb) {
    const int row = tid % (8 * kQpSeqs), gi = tid / (8 * kQpSeqs), g = g0 + gi, sq = row >> 3, jj = row & 7;
    if (sq < nseq && jj < (wide ? 8 : 4)) {
      float csum = 0.0f, qsum = 0.0f;
      if (jj < gq) {
        const float s0 = sig[row] * (float)(1 << land_e(2 * g)), s1 = sig[row] * (float)(1 << land_e(2 * g + 1));
#pragma unroll
        for (int c4 = 0; c4 < 8; ++c4) {
          const float4 v = *reinterpret_cast<const float4*>(&qb[row][32 * gi + 4 * c4]);
          const float sc = c4 < 4 ? s0 : s1;  // channels 32 g + 0..15 sit at code position 2 g
          csum += (float)(_Float16)(v.x * sc) + (float)(_Float16)(v.y * sc) + (float)(_Float16)(v.z * sc) +
                  (float)(_Float16)(v.w * sc);
          qsum += v.x + v.y + v.z + v.w;
        }
      }
      const float isg = jj < gq ? 1.0f / sig[row] : 0.0f;
      float* cst = reinterpret_cast<float*>(a.qop + ((size_t)(b0 + sq) * H + h) * kQopTile + 4096);
      if (wide) {
        cst[16 * (g >> 1) + 2 * jj + (g & 1)] = -csum;
        cst[32 + 4 * jj + g] = qsum;
        if (g == 0) cst[64 + jj] = isg;
      } else {
        cst[4 * jj + g] = -csum;
        cst[16 + 4 * jj + g] = qsum;
        if (g == 0) cst[32 + jj] = isg;
      }
    }
  }
}

// ---------------------------------------------------------------------------------------------
// Row layouts (groups of 32 channels; with one 128-channel group per token every k block of the
// query sits in row (j, 0), all four accumulate into tile 0, and the score is s D + z sum_k q'_jk with
// no zero-term product). The matrix cores contract over 32 channels, one quant group, while a group's scale
// multiplies only that group's partial dot product, so a score row serves one group: it is
// nonzero only in that group's k block.
//  * narrow (up to 4 query heads per KV head): row (j, g) = 4 j + g; the four k blocks accumulate
//    into one 16-row tile D[(j, g), t];
//  * wide (5 to 8 query heads): row (j, gg) = 2 j + gg, nonzero in the blocks g with g % 2 = gg;
//    blocks 0, 1 accumulate into tile D01 and blocks 2, 3 into D23, so eight query heads take
//    four MFMAs per page where two narrow tiles would take eight.
// The value contraction mirrors this: its columns are (j, g) (narrow) or (j, gg) (wide) and hold
// the weights p_jt s_tg of the column's group; channel tile mt (group mt / 2) uses the columns of
// its group.
template <bool WIDE>
struct PairLoads {
  uint2 kc[2];  // K codes of this lane's token (lo), chunk hi: halves 4hi..4hi+3
  uint4 km[2];  // K scale/zero of token lo, groups 0..3
  uint2 vc[2];  // V codes of half lo, tokens 4hi..4hi+3
  uint2 vs[2][WIDE ? 2 : 1];  // V scales, tokens 4hi..4hi+3: group lo&3 (narrow); lo&1, 2+(lo&1) (wide)
  uint2 vz[2];  // (Z, l) operand rows: V zeros of group lo (lo < 4), 1.0 (lo 4..7), 0 (lo 8..15)
  uint32_t nv[2];  // wave-uniform: cached tokens of each page (16 for a full page)
};

// Page records are staged in LDS by the wave that consumes them, with LDS-DMA loads
// (global_load_lds: lane i's bytes land at M0 + 16 i), so that several page pairs are in flight per
// wave without holding registers. A pair takes three dwordx4 loads: the 1024 B of codes of each
// page, then both pages' 512 B of metadata in one load (lanes 0..31 read page 0's, lanes 32..63
// page 1's, through per-lane 64-bit addresses). Issued through inline asm because the compiler
// would otherwise wait for every outstanding DMA before any LDS read; the waits are explicit instead
// (vmcnt counts this wave's loads in issue order). Slot layout: codes of page 0 | codes of page 1 |
// metadata of page 0 | metadata of page 1.
constexpr int kDmaPerPair = 3;
// Page list: one 16-byte entry per page of the concatenated sequences, written by the query-prep
// kernel: {address of the page's record of KV head 0 (low, high word), cached tokens in the page,
// 0}. A page whose block id lies outside the pool holds 0 tokens and points at block 0.
struct PageEnt {
  uint32_t lo, hi, nv, pad;
};
typedef const __attribute__((address_space(4))) PageEnt* ent_ptr;

__device__ __forceinline__ PageEnt load_ent(ent_ptr p, int i) {
  return PageEnt{p[i].lo, p[i].hi, p[i].nv, 0u};
}

// DMA of one page pair into the staging slot at lds_addr. (a_lo, a_hi), (b_lo, b_hi): records of KV
// head 0 of the two pages; voff16 = 16 l + R h (R the record size) selects head h for the codes;
// moff = (the record of page 0 or, for lanes 32..63, page 1) + R h + 1024 + 16 (l % 32) is the
// lane's metadata address.
// With one group per token (NG = 1) a page has 128 B of metadata: one dword load, lanes 0..31 and
// 32..63 reading 4 bytes of page 0 and page 1.
template <int NG>
__device__ __forceinline__ void dma_pair(uint32_t a_lo, uint32_t a_hi, uint32_t b_lo, uint32_t b_hi, uint32_t lds_addr,
                                         uint32_t voff16, uint64_t moff_head, uint64_t upper_mask) {
  const uint8_t* ra = reinterpret_cast<const uint8_t*>(((uint64_t)a_hi << 32) | a_lo);
  const uint8_t* rb = reinterpret_cast<const uint8_t*>(((uint64_t)b_hi << 32) | b_lo);
  // lanes 32..63 address page b: a + ((b - a) & mask) with the wave-uniform difference formed on the
  // scalar unit and a loop-invariant per-lane mask (two ANDs and two adds on the vector unit)
  const uint64_t a64 = ((uint64_t)a_hi << 32) | a_lo, d64 = (((uint64_t)b_hi << 32) | b_lo) - a64;
  const uint64_t maddr = a64 + ((d64 & upper_mask) + moff_head);
  if constexpr (NG == 4) {
    asm volatile(
        "s_mov_b32 m0, %0\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %3, %4 nt\n\t"
        "s_mov_b32 m0, %1\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %3, %5 nt\n\t"
        "s_mov_b32 m0, %2\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %6, off nt" ::"s"(lds_addr),
        "s"(lds_addr + 1024), "s"(lds_addr + 2048), "v"(voff16), "s"(ra), "s"(rb), "v"(maddr)
        : "memory", "m0");
  } else {
    asm volatile(
        "s_mov_b32 m0, %0\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %3, %4 nt\n\t"
        "s_mov_b32 m0, %1\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %3, %5 nt\n\t"
        "s_mov_b32 m0, %2\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dword %6, off nt" ::"s"(lds_addr),
        "s"(lds_addr + 1024), "s"(lds_addr + 2048), "v"(voff16), "s"(ra), "s"(rb), "v"(maddr)
        : "memory", "m0");
  }
}

// Operands of one page pair read back from its staging slot. Tokens a page does not hold (past the
// sequence's end, or the whole page for a block id outside the pool or a stand-in past the segment)
// get scores of -inf, so p = 0 multiplies their (finite) codes and metadata and they add nothing.
// An empty asm that uses every register read_pair filled: the compiler places its wait for those
// LDS reads here, ahead of the scalar block-id loads that follow (a later wait would have to
// wait for those loads too, since scalar loads return out of order).
// With one group per token only the first metadata word and the first scale pair are used (and
// pinned); the other slots hold copies the compiler drops.
template <bool WIDE, int NG>
__device__ __forceinline__ void pin_pair(PairLoads<WIDE>& p) {
  typedef uint32_t u2v __attribute__((ext_vector_type(2)));
  typedef uint32_t u4v __attribute__((ext_vector_type(4)));
#pragma unroll
  for (int P = 0; P < 2; ++P) {
    u2v kc = __builtin_bit_cast(u2v, p.kc[P]), vc = __builtin_bit_cast(u2v, p.vc[P]);
    u2v vs0 = __builtin_bit_cast(u2v, p.vs[P][0]), vz = __builtin_bit_cast(u2v, p.vz[P]);
    if constexpr (NG == 1) {
      asm volatile("" : "+v"(kc), "+v"(vc), "+v"(p.km[P].x), "+v"(vs0), "+v"(vz));
    } else {
      u4v km = __builtin_bit_cast(u4v, p.km[P]);
      asm volatile("" : "+v"(kc), "+v"(vc), "+v"(km), "+v"(vs0), "+v"(vz));
      p.km[P] = __builtin_bit_cast(uint4, km);
    }
    p.kc[P] = __builtin_bit_cast(uint2, kc);
    p.vc[P] = __builtin_bit_cast(uint2, vc);
    p.vs[P][0] = __builtin_bit_cast(uint2, vs0);
    p.vz[P] = __builtin_bit_cast(uint2, vz);
    if constexpr (WIDE && NG != 1) {
      u2v vs1 = __builtin_bit_cast(u2v, p.vs[P][1]);
      asm volatile("" : "+v"(vs1));
      p.vs[P][1] = __builtin_bit_cast(uint2, vs1);
    }
  }
}
// With one group per token (NG = 1) the token's single (s, z) is read into the group slots: the score
// is s D + z Q over the 128 channels, and the one value-weight operand uses the token's scale and zero.
template <bool WIDE, int NG>
__device__ __forceinline__ void read_pair(const uint8_t* slot, uint32_t nv0, uint32_t nv1, int lo, int hi,
                                          const uint8_t* czb, PairLoads<WIDE>& p) {
  using L = Rec<NG>;
#pragma unroll
  for (int P = 0; P < 2; ++P) {
    const uint8_t* rec = slot + P * 1024;                    // codes of page P (record offsets < 1024)
    const uint8_t* met = slot + 2048 + P * 128 * NG - 1024;  // metadata of page P (record offsets >= 1024)
    p.nv[P] = P == 0 ? nv0 : nv1;
    p.kc[P] = *reinterpret_cast<const uint2*>(rec + kOffKCodes + 32 * lo + 8 * hi);
    if constexpr (NG == 4) {
      p.km[P] = *reinterpret_cast<const uint4*>(met + L::kOffKMeta + 16 * lo);
    } else {
      const uint32_t m = *reinterpret_cast<const uint32_t*>(met + L::kOffKMeta + 4 * lo);
      p.km[P] = make_uint4(m, m, m, m);
    }
    p.vc[P] = *reinterpret_cast<const uint2*>(rec + kOffVCodes + 32 * lo + 8 * hi);
    constexpr int gs = NG == 4 ? 32 : 0;  // bytes between the V metadata of consecutive groups
    if constexpr (WIDE) {
      p.vs[P][0] = *reinterpret_cast<const uint2*>(met + L::kOffVScale + gs * (lo & 1) + 8 * hi);
      p.vs[P][1] = *reinterpret_cast<const uint2*>(met + L::kOffVScale + gs * (2 + (lo & 1)) + 8 * hi);
    } else {
      p.vs[P][0] = *reinterpret_cast<const uint2*>(met + L::kOffVScale + gs * (lo & 3) + 8 * hi);
    }
    // lanes 0..3: the zeros of group lo; lanes 4..15 read the constant rows of the (Z, l) operand
    const uint8_t* vzb = lo < 4 ? slot + 2048 - 1024 + L::kOffVZero + gs * (lo & 3) + 8 * hi : czb;
    p.vz[P] = *reinterpret_cast<const uint2*>(vzb + P * 128 * NG);
  }
}
template <int X>
__device__ __forceinline__ half8_t k_operand(uint2 w, const LandK& k) {
  // instruction i = X/2 ... called with X = 2i: registers (d0,x), (d1,x), (d0,x+1), (d1,x+1)
  return __builtin_bit_cast(half8_t,
                            u32x4_t{land<X>(w.x, k), land<X>(w.y, k), land<X + 1>(w.x, k), land<X + 1>(w.y, k)});
}

template <int MT>
__device__ __forceinline__ half8_t v_operand(uint2 w0, uint2 w1, const LandK& k) {
  return __builtin_bit_cast(half8_t,
                            u32x4_t{land<MT>(w0.x, k), land<MT>(w0.y, k), land<MT>(w1.x, k), land<MT>(w1.y, k)});
}

__device__ __forceinline__ float4_t mfma16(half8_t a, half8_t b, float4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// Per-wave scan state. Lane (lo, hi) serves, in the score tiles, token lo and the query heads
// jq(hi, u): narrow j = hi (u = 0); wide j = 2 hi + u (u = 0, 1).
template <bool WIDE>
struct ScanState {
  static constexpr int NJ = WIDE ? 2 : 1;   // query heads per lane in the score tiles
  static constexpr int NT = WIDE ? 2 : 1;   // score tiles (narrow D; wide D01, D23)
  half8_t A[4];                 // query operand of k block i
  float4_t cinit[NT];           // accumulator start of the score tiles (rows 4hi..4hi+3)
  half8_t Azq;                  // zero-term operand: row (j, 0) holds sum_{k in g} q'_jk, g = 0..3, as
                                // two fp16 terms (k = 0..3 high, 4..7 low); every other entry zero
  float invsig[NJ];              // 1 / sigma of query head jq(hi, u) (1 for absent heads)
  float thr[NJ];                 // (mref + tau) sigma: the lazy-rescale threshold on the scaled logits
  float4_t acc[8];              // O' tiles: channels 16 mt + 4hi + r, column lo
  float4_t wsum[NT];            // sum_t w_t of each column (every row); wide: groups gg, 2 + gg
  float4_t zl;                  // rows 0..3: sum_t p_t z_tg (row = group); rows 4..7: sum_t p_t
  float mref[NJ];
  float Qz[NJ];                 // sigma sum_k q'_jk of query head jq(hi, u) (used with one group per token)
  LandK lk;                     // landing constants
};

// Scores of one page pair, base-2 logits times sigma (the query operand's scale), -inf where masked:
// a2[P][u] for token lo of page P and query head jq(hi, u). The accumulation chains of both pages are issued interleaved so that each
// hides the others' latency.
template <bool WIDE, int NG>
__device__ __forceinline__ void qk_pair(const ScanState<WIDE>& st, const PairLoads<WIDE>& cur, int lo,
                                        float (&a2)[2][ScanState<WIDE>::NJ]) {
  constexpr int NT = ScanState<WIDE>::NT, NJ = ScanState<WIDE>::NJ;
  half8_t B[2][4];
#pragma unroll
  for (int P = 0; P < 2; ++P) {
    B[P][0] = k_operand<0>(cur.kc[P], st.lk);
    B[P][1] = k_operand<2>(cur.kc[P], st.lk);
    B[P][2] = k_operand<4>(cur.kc[P], st.lk);
    B[P][3] = k_operand<6>(cur.kc[P], st.lk);
  }
  float4_t d[2][NT];
#pragma unroll
  for (int P = 0; P < 2; ++P)
#pragma unroll
    for (int t = 0; t < NT; ++t) d[P][t] = st.cinit[t];
  if constexpr (WIDE && NG != 1) {
    // blocks 0, 2 then 1, 3: four independent chains (page x tile) of two
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int P = 0; P < 2; ++P)
#pragma unroll
        for (int t = 0; t < 2; ++t) d[P][t] = mfma16(st.A[2 * t + i], B[P][2 * t + i], d[P][t]);
  } else {
    // every block into tile 0 (with one group per token the query rows are dense: see qprep_block)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int P = 0; P < 2; ++P) d[P][0] = mfma16(st.A[i], B[P][i], d[P][0]);
  }
  if constexpr (NG == 1) {
    // one (s, z) per token: score = s D + z Q_j, D (all 128 channels) in row (j, 0) of tile 0
#pragma unroll
    for (int P = 0; P < 2; ++P) {
      const half2_t m = as_h2(cur.km[P].x);
#pragma unroll
      for (int u = 0; u < NJ; ++u) {
        const float Ds = d[P][0][WIDE ? 2 * u : 0];
        a2[P][u] = fmaf((float)m.x, Ds, (float)m.y * st.Qz[u]);
      }
    }
  } else {
  // Zero term on the matrix cores: rows (j, 0) of zd = sum_g Q_jg z_tg, with z_tg exact in fp16 (the
  // B operand is the token's (s, z) pairs as loaded; the query operand is zero at the s positions)
  float4_t zd[2];
#pragma unroll
  for (int P = 0; P < 2; ++P)
    zd[P] = mfma16(st.Azq, __builtin_bit_cast(half8_t, cur.km[P]), float4_t{0.f, 0.f, 0.f, 0.f});
#pragma unroll
  for (int P = 0; P < 2; ++P) {
    const half2_t m[4] = {as_h2(cur.km[P].x), as_h2(cur.km[P].y), as_h2(cur.km[P].z), as_h2(cur.km[P].w)};
#pragma unroll
    for (int u = 0; u < NJ; ++u) {
      // D of group g for query head jq(hi, u): narrow register g of D; wide register 2u + g % 2
      // of tile g / 2; its zero term sits in register 2u (wide) or 0 (narrow) of zd
      float Dg[4];
#pragma unroll
      for (int g = 0; g < 4; ++g) Dg[g] = WIDE ? d[P][g >> 1][2 * u + (g & 1)] : d[P][0][g];
      float sd = fmaf((float)m[0].x, Dg[0], zd[P][WIDE ? 2 * u : 0]);
      sd = fmaf((float)m[1].x, Dg[1], sd);
      sd = fmaf((float)m[2].x, Dg[2], sd);
      a2[P][u] = fmaf((float)m[3].x, Dg[3], sd);
    }
  }
  }
  // tokens a page does not hold get -inf (a wave-uniform branch, taken only for partial pages)
  if (cur.nv[0] < (uint32_t)kBlock || cur.nv[1] < (uint32_t)kBlock) {
#pragma unroll
    for (int P = 0; P < 2; ++P) {
      const float mk = (uint32_t)lo < cur.nv[P] ? 0.0f : -INFINITY;
#pragma unroll
      for (int u = 0; u < NJ; ++u) a2[P][u] += mk;
    }
  }
}

// Lazy online softmax of one pair: the reference max only moves when a score exceeds it by 2^tau
// (detected by a wave-wide vote, no row reduction in the common case). Writes p (fp16) to LDS as
// p_w[page][query head][token].
template <bool WIDE>
__device__ __forceinline__ void softmax_pair(ScanState<WIDE>& st, const float (&a2)[2][ScanState<WIDE>::NJ], int lo,
                                             int hi, _Float16 (*p_w)[8][kBlock], float* al_w) {
  constexpr int NJ = ScanState<WIDE>::NJ, NT = ScanState<WIDE>::NT;
  bool need = false;
#pragma unroll
  for (int P = 0; P < 2; ++P)
#pragma unroll
    for (int u = 0; u < NJ; ++u) need |= a2[P][u] > st.thr[u];
  if (__any(need)) {
#pragma unroll
    for (int u = 0; u < NJ; ++u) {
      const float pm = row_max16(fmaxf(a2[0][u], a2[1][u])) * st.invsig[u];  // exact: a power of two
      const float mnew = pm > st.mref[u] + kRescaleTau ? pm : st.mref[u];
      const float al = __builtin_amdgcn_exp2f(st.mref[u] - mnew);
      st.mref[u] = mnew;
      st.thr[u] = (mnew + kRescaleTau) / st.invsig[u];
      if (lo == 0) al_w[NJ * hi + u] = al;
    }
    lds_sync_wave();
    // every accumulator column (j, .) belongs to query head j = lo / 4 (narrow), lo / 2 (wide)
    const float alc = al_w[WIDE ? lo >> 1 : lo >> 2];
#pragma unroll
    for (int mt = 0; mt < 8; ++mt) st.acc[mt] *= alc;
#pragma unroll
    for (int t = 0; t < NT; ++t) st.wsum[t] *= alc;
    st.zl *= alc;
  }
#pragma unroll
  for (int P = 0; P < 2; ++P) {
#pragma unroll
    for (int u = 0; u < NJ; ++u) {
      const float p = __builtin_amdgcn_exp2f(fmaf(a2[P][u], st.invsig[u], -st.mref[u]));
      p_w[P][NJ * hi + u][lo] = (_Float16)p;
    }
  }
}

// Value accumulation of one pair: K = the pair's 32 tokens, N = the 16 columns, M = 8 tiles of 16
// channels; p comes back from LDS in the layout of the B operand.
//
// The weights w = p s enter the matrix cores as fp16. Lazy rescaling keeps p <= 2^tau = 256, so
// w is finite for every scale s < 256; a larger V scale (a rotated value range above 768) can make
// it overflow to inf, which then shows in the weight sums. The scaled form (big, uniform over the
// wave) keeps every weight finite: the codes land on the fp16 pattern of 256 instead of 1.0
// (A' = 256 (1 + c 2^-e), exact), the weights are w' = fp16(p s / 256) formed in fp32 and the
// weight sums add 256 w'. The products A' w' are those of the plain form and the final correction
// (O = 2^e (D - sum w) + Z) is unchanged. The scan runs a segment in the plain form and repeats it
// in the scaled form only when its sums came out non-finite.
template <bool WIDE, int NG, bool big>
__device__ __forceinline__ void pv_pair(ScanState<WIDE>& st, const PairLoads<WIDE>& cur, int lo, int hi,
                                        const _Float16 (*p_w)[8][kBlock]) {
  // with one group per token every group column has the same weights: one weight operand (and one
  // weight sum) serves all tiles
  constexpr int NT = NG == 1 ? 1 : ScanState<WIDE>::NT;
  LandK lk = st.lk;
  if constexpr (big) lk.one = 0x5C005C00u;  // fp16 256.0, twice
  // A operand of the (Z, l) contraction: rows 0..3 hold z of group `row`, rows 4..7 hold 1.0, rows
  // 8..15 zero, all as read from LDS (see read_pair)
  const half8_t Azl = __builtin_bit_cast(half8_t, u32x4_t{cur.vz[0].x, cur.vz[0].y, cur.vz[1].x, cur.vz[1].y});
  const half8_t Aones = __builtin_bit_cast(half8_t, u32x4_t{lk.one, lk.one, lk.one, lk.one});
  // column lo: query head jc, probabilities of tokens 4hi..4hi+3 of both pages
  const int jc = WIDE ? lo >> 1 : lo >> 2;
  const uint2 pp0 = *reinterpret_cast<const uint2*>(&p_w[0][jc][4 * hi]);
  const uint2 pp1 = *reinterpret_cast<const uint2*>(&p_w[1][jc][4 * hi]);
  const half8_t Bp = __builtin_bit_cast(half8_t, u32x4_t{pp0.x, pp0.y, pp1.x, pp1.y});
  uint32_t wv[NT][4];
  const uint32_t pw[4] = {pp0.x, pp0.y, pp1.x, pp1.y};
  if constexpr (big) {
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint2 sv = cur.vs[i >> 1][t];
        const half2_t p = as_h2(pw[i]), s = as_h2(i & 1 ? sv.y : sv.x);
        wv[t][i] = as_u(half2_t{(_Float16)((float)p.x * (float)s.x * 0x1p-8f),
                                (_Float16)((float)p.y * (float)s.y * 0x1p-8f)});
      }
  } else {
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint2 sv = cur.vs[i >> 1][t];
        wv[t][i] = as_u(as_h2(pw[i]) * as_h2(i & 1 ? sv.y : sv.x));
      }
  }
  half8_t Bw[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    Bw[t] = __builtin_bit_cast(half8_t, u32x4_t{wv[t][0], wv[t][1], wv[t][2], wv[t][3]});
    st.wsum[t] = mfma16(Aones, Bw[t], st.wsum[t]);
  }
  st.zl = mfma16(Azl, Bp, st.zl);
  // the value MFMAs issue at raised wave priority, so the other wave of the SIMD fills the vector
  // ALU beside them (measured: -2 % scan time at 5 query heads per KV head)
  __builtin_amdgcn_s_setprio(1);
#define INT2KV_PV_TILE(MT)                                                                        \
  st.acc[MT] = mfma16(v_operand<MT>(cur.vc[0], cur.vc[1], lk), Bw[WIDE && NT == 2 ? (MT) >> 2 : 0], st.acc[MT]);
  INT2KV_PV_TILE(0)
  INT2KV_PV_TILE(1)
  INT2KV_PV_TILE(2)
  INT2KV_PV_TILE(3)
  INT2KV_PV_TILE(4)
  INT2KV_PV_TILE(5)
  INT2KV_PV_TILE(6)
  INT2KV_PV_TILE(7)
#undef INT2KV_PV_TILE
  __builtin_amdgcn_s_setprio(0);
}

#ifndef INT2KV_SCAN_STAGES
#define INT2KV_SCAN_STAGES 3
#endif
constexpr int kStages = INT2KV_SCAN_STAGES;  // page pairs staged (in flight) per wave
constexpr int kUnroll = kStages % 2 ? 2 * kStages : kStages;  // steps per unrolled group: slots and X / Y repeat

// f(integral_constant<0>), ..., f(integral_constant<N - 1>) in order
template <int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (N > 0) {
    static_for<N - 1>(f);
    f(std::integral_constant<int, N - 1>{});
  }
}
constexpr int kWavesPerWG = 8;   // one wave per KV head of a head group

typedef __attribute__((address_space(4))) const int32_t* cint_ptr;  // read through the scalar cache

// Work split of the scan. Every sequence a work-group starts costs a prologue and a pipeline
// refill (measured: about 4 us per extra segment, the time of ~6 pages; 8 units measured best in a
// sweep of 3 to 10 on the ragged 64-sequence batch), so the pages are split
// evenly along a cost axis on which each non-empty sequence b occupies [c0(b), c1(b)): kSegCost
// units of lead-in, then one unit per page (c1 - c0 = kSegCost + pages; empty sequences take no
// room). Group g of G starts at cost x(g) = floor(g W / G), W = P + kSegCost * (non-empty
// sequences); a start inside a lead-in maps to the sequence's first page. Ranges that take on
// extra sequence starts thus get fewer pages.
#ifndef INT2KV_SCAN_SEG_COST
#define INT2KV_SCAN_SEG_COST 8
#endif
constexpr int kSegCost = INT2KV_SCAN_SEG_COST;

// Pages of every sequence and their exclusive prefix sums (prefix[B] = total pages), and for each
// scan work-group g the sequence b holding the first page of its range with that sequence's page
// range: wg_info[g] = {b, prefix[b], prefix[b + 1], lo(g)}, wg_info[G].w = P, and for every sequence
// the first and last group whose range meets it (seq_wg[b] = {ga, gb}, {0, -1} when empty), so that
// no later wave divides or searches. With x(g) <= T  <=>  g <= ceil((T + 1) G / W) - 1, the groups
// starting in b's span are ceil(c0 G / W) .. ceil(c1 G / W) - 1, the group holding b's first page
// is the last one with x(g) <= c0 + kSegCost, the one holding its last page the last with
// x(g) <= c1 - 1. Every group below G starts in exactly one span (the spans tile [0, W)), so every
// entry is written once, by the thread owning that sequence. One block of 256 threads.
__device__ void page_prefix_block(const DecodeArgs& a, uint8_t* lds) {
  int* sums = reinterpret_cast<int*>(lds);
  int* cnts = sums + 256;
  const int tid = threadIdx.x;
  const int per = (a.B + 255) / 256;
  const int b0 = min(a.B, tid * per), b1 = min(a.B, b0 + per);
  int s = 0, c = 0;
  for (int b = b0; b < b1; ++b) {
    const int n = (seq_len_m(a, b) + kBlock - 1) >> 4;
    s += n;
    c += n > 0;
  }
  sums[tid] = s;
  cnts[tid] = c;
  __syncthreads();
  for (int off = 1; off < 256; off <<= 1) {
    const int v = tid >= off ? sums[tid - off] : 0, u = tid >= off ? cnts[tid - off] : 0;
    __syncthreads();
    sums[tid] += v;
    cnts[tid] += u;
    __syncthreads();
  }
  const int P = sums[255], G = a.grid_g;
  const long long W = (long long)P + (long long)kSegCost * cnts[255];
  // few sequences: their group entries are filled by the whole block below (a long sequence spans
  // hundreds of groups, too many for one thread)
  const bool coop = a.B <= 8;
  int run = tid > 0 ? sums[tid - 1] : 0, cnt = tid > 0 ? cnts[tid - 1] : 0;
  for (int b = b0; b < b1; ++b) {
    const int n = (seq_len_m(a, b) + kBlock - 1) >> 4;
    a.prefix[b] = run;
    int ga = 0, gb = -1;
    if (n > 0) {
      const long long c0 = run + (long long)kSegCost * cnt, c1 = c0 + kSegCost + n;
      const int g1 = min(G - 1, (int)((c1 * G + W - 1) / W) - 1);
      // x(g) = floor(g W / G), stepped by quotient and remainder: one division for the whole loop
      // (a long sequence spans every group, and a 64-bit division per group costs microseconds)
      int g = coop ? g1 + 1 : (int)((c0 * G + W - 1) / W);
      const long long wq = W / G, wr = W % G;
      long long xq = (long long)g * wq + ((long long)g * wr) / G, xr = ((long long)g * wr) % G;
      for (; g <= g1; ++g) {
        const int lo = run + (int)min((long long)n - 1, max(0LL, xq - c0 - kSegCost));
        *reinterpret_cast<int4*>(a.wg_info + 4 * g) = make_int4(b, run, run + n, lo);
        xq += wq;
        xr += wr;
        if (xr >= G) {
          xr -= G;
          ++xq;
        }
      }
      ga = min(G - 1, (int)(((c0 + kSegCost + 1) * G + W - 1) / W) - 1);
      gb = g1;
      ++cnt;
    }
    a.seq_wg[2 * b] = ga;
    a.seq_wg[2 * b + 1] = gb;
    run += n;
  }
  if (coop) {
    // per = 1 here, so the exclusive prefixes of sequence b are the scan's entries at b - 1
    for (int b = 0; b < a.B; ++b) {
      const int n = (seq_len_m(a, b) + kBlock - 1) >> 4;
      if (n == 0) continue;  // uniform
      const int rb = b > 0 ? sums[b - 1] : 0, cb = b > 0 ? cnts[b - 1] : 0;
      const long long c0 = rb + (long long)kSegCost * cb, c1 = c0 + kSegCost + n;
      const int g1 = min(G - 1, (int)((c1 * G + W - 1) / W) - 1);
      for (int g = (int)((c0 * G + W - 1) / W) + tid; g <= g1; g += 256) {
        const long long x = (long long)g * W / G;
        const int lo = rb + (int)min((long long)n - 1, max(0LL, x - c0 - kSegCost));
        *reinterpret_cast<int4*>(a.wg_info + 4 * g) = make_int4(b, rb, rb + n, lo);
      }
    }
  }
  if (tid == 255) {
    a.prefix[a.B] = P;
    a.wg_info[4 * G + 3] = P;  // range start of the group after the last
  }
}

// Page list entries of pages [p0, p0 + kPlPages) of sequence b (four per thread, every block-table
// load issued before the first store). The list position of page 0 of b, the pages of the
// sequences before b, is summed by the block itself (the same prefix the page-prefix block
// computes). Entry: address of the record of KV head 0, cached tokens of the page (0, with the
// address of block 0, for a block id outside the pool).
constexpr int kPlPages = 1024;
static_assert(kPlPages == 4 * 256, "page_list_block writes four entries per thread of its 256");

__device__ void page_list_block(const DecodeArgs& a, int b, int p0, uint8_t* lds) {
  int* red = reinterpret_cast<int*>(lds);
  const int tid = threadIdx.x;
  const int L = seq_len_m(a, b), np = (L + kBlock - 1) >> 4;
  if (p0 >= np) return;  // uniform over the block
  int s = 0;
  for (int bb = tid; bb < b; bb += 256) s += (seq_len_m(a, bb) + kBlock - 1) >> 4;
  red[tid] = s;
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if (tid < off) red[tid] += red[tid + off];
    __syncthreads();
  }
  const size_t base = (size_t)red[0] + p0;
  const int32_t* row = a.block_table + (size_t)b * a.max_blocks + p0;
  const int n = min(kPlPages, np - p0);
  int id[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) id[u] = 4 * tid + u < n ? row[4 * tid + u] : 0;
  const uint64_t pool = (uint64_t)(uintptr_t)a.pool;
  const uint64_t stride = (uint64_t)a.H * (1024 + 128 * a.groups);
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int i = 4 * tid + u;
    if (i < n) {
      const bool ok = (uint32_t)id[u] < (uint32_t)a.num_blocks;
      const uint64_t rec = pool + (ok ? (uint64_t)(uint32_t)id[u] * stride : 0ull);
      const int t = kBlock * (p0 + i);
      *reinterpret_cast<uint4*>(a.pages + 4 * (base + i)) =
          make_uint4((uint32_t)rec, (uint32_t)(rec >> 32), ok ? (uint32_t)min(kBlock, L - t) : 0u, 0u);
    }
  }
}

// Blocks 0 .. nap - 1 (int2kv_append_decode): the cache write of the current tokens, one block per
// (block of ap.nbx, KV head, K|V), four waves; it runs beside the roles below, which do not read
// the cache. Then block nap: page prefix sums; nap + 1 .. nap + nq: query operands of KV head h for
// kQpSeqs sequences; the rest: the page list, kPlPages pages of one sequence per block (nseg blocks
// per sequence). Lower block ids are dispatched first. The roles share one LDS buffer.
constexpr int kPrepLdsBytes = kAppendLdsBytes > kQpLdsBytes ? kAppendLdsBytes : kQpLdsBytes;

// AP: the launch carries append blocks (their LDS sets the block's size; without them the roles
// below fit several blocks per CU).
// The query role runs as one block per (KV head, 8 sequences) beside append blocks (whose LDS allows
// one block per CU: fewer blocks keep the launch in one round) and as four (one per 32-channel group
// of q', shorter chains) otherwise.
constexpr int qp_split(bool ap) { return ap ? 1 : 4; }
template <bool AP>
__global__ __launch_bounds__(256) void qprep_kernel(DecodeArgs a, int wide, int nq, int nseg, AppendArgs ap, int nap) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[AP ? kPrepLdsBytes : qp_lds_bytes(qp_split(false))];
  int blk = blockIdx.x;
  if (AP && blk < nap) {
    const int bx = blk % ap.nbx, r = blk / ap.nbx;
    if (ap.cv.groups == 1)
      append_block<1, 4, 1>(ap.cv, ap.k, ap.v, ap.slots, ap.n, ap.R_k, ap.R_v, ap.mu_rk, ap.clip_k, ap.clip_v, bx,
                            ap.nbx, r % ap.cv.num_kv_heads, r / ap.cv.num_kv_heads, lds);
    else
      append_block<1, 4, 4>(ap.cv, ap.k, ap.v, ap.slots, ap.n, ap.R_k, ap.R_v, ap.mu_rk, ap.clip_k, ap.clip_v, bx,
                            ap.nbx, r % ap.cv.num_kv_heads, r / ap.cv.num_kv_heads, lds);
    return;
  }
  blk -= nap;
  if (blk == 0)
    page_prefix_block(a, lds);
  else if (blk <= nq)
    qprep_block<qp_split(AP)>(a, blk - 1, wide != 0, lds);
  else
    page_list_block(a, (blk - 1 - nq) / nseg, ((blk - 1 - nq) % nseg) * kPlPages, lds);
}

__device__ __forceinline__ void wait_vm_all() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// One wave: KV head h of sequence b, global pages [gs, ge) (all of sequence b), with its partial
// (m, l, O') per query head written to partial slot `slot`.
// big: every pair in the scaled value form (see pv_pair). Returns whether the segment's sums are
// finite (uniform over the wave); with big they always are.
template <bool WIDE, int NG, bool BIG>
__device__ __forceinline__ bool scan_segment(const DecodeArgs& a, int b, int h, int gs, int ge, int slot, int l,
                                             uint8_t* stage_w, _Float16 (*p_w)[2][8][kBlock], float* al_w,
                                             uint8_t* cz_w, bool all_waves) {
  constexpr int NJ = ScanState<WIDE>::NJ, NT = ScanState<WIDE>::NT;
  const int lo = l & 15, hi = l >> 4;
  const int n = ge - gs;             // pages
  const int npairs = (n + 1) >> 1;   // the last pair may hold one page
  const int nfull = n >> 1;          // pairs of two pages
  const uint32_t stage_base = (uint32_t)(uintptr_t)stage_w;

  // ---- query operands of (b, h): plain loads, issued ahead of the first page DMAs so that both
  // latencies overlap (the first use waits for every load in flight, which the prologue does anyway)
  const uint8_t* qop = a.qop + ((size_t)b * a.H + h) * kQopTile;
  const float* cst = reinterpret_cast<const float*>(qop + 4096);
  ScanState<WIDE> st;
#pragma unroll
  for (int i = 0; i < 4; ++i) st.A[i] = *reinterpret_cast<const half8_t*>(qop + (i * 64 + l) * 16);
  if constexpr (WIDE && NG == 1) {
    // dense rows (j, 0): the accumulator start of row 2 j is the sum of its four group entries
    const float4_t c01 = *reinterpret_cast<const float4_t*>(cst + 4 * hi);
    const float4_t c23 = *reinterpret_cast<const float4_t*>(cst + 16 + 4 * hi);
    st.cinit[0] = float4_t{(c01[0] + c01[1]) + (c23[0] + c23[1]), 0.0f, (c01[2] + c01[3]) + (c23[2] + c23[3]), 0.0f};
    st.cinit[1] = float4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int u = 0; u < 2; ++u) st.invsig[u] = cst[64 + 2 * hi + u] > 0.0f ? cst[64 + 2 * hi + u] : 1.0f;
  } else if constexpr (WIDE) {
    st.cinit[0] = *reinterpret_cast<const float4_t*>(cst + 4 * hi);       // D01 rows 4hi..4hi+3
    st.cinit[1] = *reinterpret_cast<const float4_t*>(cst + 16 + 4 * hi);  // D23 rows 4hi..4hi+3
#pragma unroll
    for (int u = 0; u < 2; ++u) st.invsig[u] = cst[64 + 2 * hi + u] > 0.0f ? cst[64 + 2 * hi + u] : 1.0f;
  } else {
    st.cinit[0] = *reinterpret_cast<const float4_t*>(cst + 4 * hi);
    if constexpr (NG == 1)  // dense row (j, 0): the sum of its four group entries
      st.cinit[0] = float4_t{((st.cinit[0][0] + st.cinit[0][1]) + st.cinit[0][2]) + st.cinit[0][3], 0.f, 0.f, 0.f};
    st.invsig[0] = cst[32 + hi] > 0.0f ? cst[32 + hi] : 1.0f;
  }
  {
    // zero-term operand against the token's metadata as it sits in registers (B rows k = 8 q + i:
    // s_0, z_0, s_1, z_1, .., z_3 for every q): the rows (j, 0) carry the group sums of q'_j at the z
    // positions, the high fp16 term in lanes 0..15 (k 1, 3, 5, 7), the low term in lanes 16..31
    // (k 9, 11, 13, 15); every other entry zero
    const int m = l & 15, j = WIDE ? m >> 1 : m >> 2;
    const bool zrow = l < 32 && (WIDE ? (m & 1) == 0 : (m & 3) == 0);
    const float4_t Q = *reinterpret_cast<const float4_t*>(cst + (WIDE ? 32 : 16) + 4 * j);
    const float isj = cst[(WIDE ? 64 : 32) + j], sg = isj > 0.0f ? 1.0f / isj : 1.0f;  // sigma: a power of two
    half8_t z;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const float qs = Q[g] * sg;
      const _Float16 qh = (_Float16)qs;
      const _Float16 term = l < 16 ? qh : (_Float16)(qs - (float)qh);
      z[2 * g] = (_Float16)0.0f;
      z[2 * g + 1] = zrow ? term : (_Float16)0.0f;
    }
    st.Azq = z;
  }
#pragma unroll
  for (int mt = 0; mt < 8; ++mt) st.acc[mt] = float4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int t = 0; t < NT; ++t) st.wsum[t] = float4_t{0.f, 0.f, 0.f, 0.f};
  st.zl = float4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int u = 0; u < NJ; ++u) {
    st.mref[u] = kMaxInit;
    st.thr[u] = (kMaxInit + kRescaleTau) / st.invsig[u];  // -inf or below every real scaled score
  }
#pragma unroll
  for (int u = 0; u < NJ; ++u) {  // q' sums of the lane's score heads (rows of absent heads are zero)
    const float4_t Q = *reinterpret_cast<const float4_t*>(cst + (WIDE ? 32 : 16) + 4 * (NJ * hi + u));
    st.Qz[u] = (((Q[0] + Q[1]) + Q[2]) + Q[3]) / st.invsig[u];
  }
  st.lk = land_constants();
  // the wave's constant rows of the (Z, l) operand, at both page offsets: fp16 1.0 x 4, then 0 x 4
  if (l < 4)
    *reinterpret_cast<uint2*>(cz_w + (l >> 1) * 128 * NG + 8 * (l & 1)) =
        (l & 1) ? make_uint2(0u, 0u) : make_uint2(0x3C003C00u, 0x3C003C00u);
  lds_sync_wave();
  const uint8_t* czb = cz_w + (lo < 8 ? 0 : 8);

  // ---- pipeline over the segment's page pairs (global pages gs + 2k, gs + 2k + 1; the second page
  // of a last pair of one page is a stand-in: block 0, no tokens). Pair k sits in slot k % kStages.
  const ent_ptr ent = (ent_ptr)(uintptr_t)(a.pages) + gs;
  const uint32_t voff16 = 16 * l + h * Rec<NG>::kBytes;
  const uint64_t moff = (uint64_t)(h * Rec<NG>::kBytes + 1024 + (NG == 4 ? 16 : 4) * (l & 31));
  uint64_t upper = l >= 32 ? ~0ull : 0ull;  // lanes reading page b's metadata
  asm volatile("" : "+v"(upper));             // an opaque mask: ANDs, not selects
  const uint32_t pool_lo = (uint32_t)(uintptr_t)a.pool, pool_hi = (uint32_t)((uintptr_t)a.pool >> 32);
  uint32_t nv[kStages][2];  // cached tokens of the two pages staged in each slot
  // entries of pair k with the bounds check of the last pair (paths outside the steady loop): both
  // loads are unconditional (the second index clamped into the segment), and a second page past
  // the segment becomes the stand-in afterwards, by scalar selects
  auto entries = [&](int k, PageEnt& e0, PageEnt& e1) {
    const bool two = 2 * k + 1 < n;
    e0 = load_ent(ent, 2 * k);
    e1 = load_ent(ent, two ? 2 * k + 1 : 2 * k);
    e1.lo = two ? e1.lo : pool_lo;
    e1.hi = two ? e1.hi : pool_hi;
    e1.nv = two ? e1.nv : 0u;
  };
  auto stage = [&](auto slot_tag, const PageEnt& e0, const PageEnt& e1) {
    constexpr int SL = decltype(slot_tag)::value;
    const uint32_t sa = stage_base + SL * 2 * kRecord;
    dma_pair<NG>(e0.lo, e0.hi, e1.lo, e1.hi, sa, voff16, moff, upper);
    nv[SL][0] = e0.nv;
    nv[SL][1] = e1.nv;
  };
  auto pin_ent = [](PageEnt& e0, PageEnt& e1) {
    asm volatile("" : "+s"(e0.lo), "+s"(e0.hi), "+s"(e0.nv), "+s"(e1.lo), "+s"(e1.hi), "+s"(e1.nv));
  };
  static_for<kStages>([&](auto I) {
    constexpr int k = decltype(I)::value;
    if (k == 0 || k < npairs) {
      PageEnt e0, e1;
      entries(k, e0, e1);
      stage(I, e0, e1);
    }
  });
  // entries of the next pair the steady loop stages, read one step ahead of their use so that the
  // scalar loads overlap the step's arithmetic (only full pairs inside the segment are read)
  PageEnt n0{0u, 0u, 0u, 0u}, n1 = n0;
  if (kStages + 1 < nfull) {
    n0 = load_ent(ent, 2 * (kStages + 1));
    n1 = load_ent(ent, 2 * (kStages + 1) + 1);
  }
  PairLoads<WIDE> X, Y;
  {
    if (kStages - 1 < npairs)
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(kDmaPerPair * (kStages - 1)) : "memory");
    else
      wait_vm_all();
    read_pair<WIDE, NG>(stage_w, nv[0][0], nv[0][1], lo, hi, czb, X);
    pin_pair<WIDE, NG>(X);
    if (kStages < npairs) {
      PageEnt e0, e1;
      entries(kStages, e0, e1);
      stage(std::integral_constant<int, 0>{}, e0, e1);
    }
    float a2[2][NJ];
    qk_pair<WIDE, NG>(st, X, lo, a2);
    softmax_pair<WIDE>(st, a2, lo, hi, p_w[0], al_w);
  }
  // Step J of an unrolled group that starts at pair k (k % kUnroll = 0): read pair kk + 1 =
  // k + J + 1 (staged kStages pairs ago, slot SL), refill its slot with pair kk + 1 + kStages,
  // scores of pair kk + 1 beside the value accumulation of pair kk, then the softmax of pair
  // kk + 1. STEADY: pair kk + 1 + kStages is a full pair inside the segment.
  auto step = [&](auto j_tag, auto steady_tag, const PairLoads<WIDE>& cur, PairLoads<WIDE>& nxt, int k) {
    constexpr int J = decltype(j_tag)::value;
    constexpr bool STEADY = decltype(steady_tag)::value;
    constexpr int SL = (J + 1) % kStages;
    const int kk = k + J;
    const bool more = STEADY || kk + 1 < npairs;
    if (more) {
      // the pair's LDS reads and the next DMA go first on the SIMD (the other wave's landing and
      // softmax fill in behind them)
      __builtin_amdgcn_s_setprio(1);
      if (STEADY || kk + kStages < npairs)
        asm volatile("s_waitcnt vmcnt(%0)" ::"n"(kDmaPerPair * (kStages - 1)) : "memory");
      else
        wait_vm_all();
      read_pair<WIDE, NG>(stage_w + SL * 2 * kRecord, nv[SL][0], nv[SL][1], lo, hi, czb, nxt);
      pin_pair<WIDE, NG>(nxt);
      if (STEADY) {
        // The entries read one step ago are pinned (their wait placed) before the next loads issue:
        // scalar loads return out of order, so a wait placed after those would wait for them too.
        // The new loads sit between the empty asm and the DMA (both memory barriers), so they
        // issue before the DMA and have the step to return.
        pin_ent(n0, n1);
        const PageEnt m0 = load_ent(ent, 2 * (kk + 2 + kStages)), m1 = load_ent(ent, 2 * (kk + 2 + kStages) + 1);
        stage(std::integral_constant<int, SL>{}, n0, n1);
        n0 = m0;
        n1 = m1;
      } else if (kk + 1 + kStages < npairs) {
        PageEnt e0, e1;
        entries(kk + 1 + kStages, e0, e1);
        stage(std::integral_constant<int, SL>{}, e0, e1);
      }
      __builtin_amdgcn_s_setprio(0);
    }
    float a2[2][NJ];
    if (more) qk_pair<WIDE, NG>(st, nxt, lo, a2);
    lds_sync_wave();
    pv_pair<WIDE, NG, BIG>(st, cur, lo, hi, p_w[kk & 1]);
    if (more) softmax_pair<WIDE>(st, a2, lo, hi, p_w[(kk + 1) & 1], al_w);
  };
  using T = std::true_type;
  using F = std::false_type;
  int k = 0;
  // steady groups of kUnroll steps (the slot and the X / Y register set repeat with that period)
  for (; k + kUnroll + kStages < nfull; k += kUnroll) {
    // one barrier per group keeps the 8 waves (the 8 head records of each block, 12 KiB of
    // contiguous memory) streaming close together in time: 1-2 us faster than free-running waves.
    // Every wave of the work-group runs the same segments and trip counts (same page ranges); the
    // barrier is skipped in work-groups where some waves have no KV head (all_waves is uniform).
    if (all_waves) __builtin_amdgcn_s_barrier();
    static_for<kUnroll>([&](auto J) {
      if constexpr (decltype(J)::value % 2 == 0)
        step(J, T{}, X, Y, k);
      else
        step(J, T{}, Y, X, k);
    });
  }
  for (; k < npairs; k += kUnroll) {
    bool go = true;
    static_for<kUnroll>([&](auto J) {
      constexpr int j = decltype(J)::value;
      if (go && (j == 0 || k + j < npairs)) {
        if constexpr (j % 2 == 0)
          step(J, F{}, X, Y, k);
        else
          step(J, F{}, Y, X, k);
      } else {
        go = false;
      }
    });
    if (!go) break;
  }

  // ---- partial (m, l, O') of every query head of this KV head
  const int gq = a.gq;
  float* part = a.part + ((size_t)slot * a.Hq + h * gq) * kPartStride;
  // m and l of query heads jq(hi, u): l_j sits in rows 4..7 of the (Z, l) tile, column of j, so in
  // lane (first column of j, hi = 1)
#pragma unroll
  for (int u = 0; u < NJ; ++u) {
    const int j = NJ * hi + u;
    const float ls = __shfl(st.zl[0], 16 + (WIDE ? 2 * j : 4 * j));
    if (lo == 0 && j < gq) {
      float* dst = part + (size_t)j * kPartStride;
      dst[0] = st.mref[u];
      dst[1] = ls;
    }
  }
  // O' of column lo = (jc, g) (narrow) or (jc, gg) (wide): W from any row of the column's weight
  // sum; Z[jc][g] from lane (lo, hi = 0), register g
  const int jc = WIDE ? lo >> 1 : lo >> 2;
  float zc[2], wc[2];
  if constexpr (WIDE) {
    const bool odd = lo & 1;
    zc[0] = __shfl(odd ? st.zl[1] : st.zl[0], lo);  // group lo & 1
    zc[1] = __shfl(odd ? st.zl[3] : st.zl[2], lo);  // group 2 + (lo & 1)
    wc[0] = st.wsum[0][0];
    wc[1] = st.wsum[NG == 1 ? 0 : NT - 1][0];
  } else {
    const int g = lo & 3;
    const float zown = g == 0 ? st.zl[0] : g == 1 ? st.zl[1] : g == 2 ? st.zl[2] : st.zl[3];
    zc[0] = zc[1] = __shfl(zown, lo);
    wc[0] = wc[1] = st.wsum[0][0];
  }
  float* dst = part + (size_t)jc * kPartStride + 4;
#define INT2KV_OUT_TILE(MT)                                                                         \
  if ((WIDE ? (lo & 1) == (((MT) >> 1) & 1) : (lo & 3) == ((MT) >> 1)) && jc < gq) {                \
    const float sc = (float)(1 << land_e(MT));                                                      \
    const float wa = wc[(MT) >> 2], za = zc[(MT) >> 2];                                             \
    float4 o;                                                                                       \
    o.x = fmaf(sc, st.acc[MT][0] - wa, za);                                                         \
    o.y = fmaf(sc, st.acc[MT][1] - wa, za);                                                         \
    o.z = fmaf(sc, st.acc[MT][2] - wa, za);                                                         \
    o.w = fmaf(sc, st.acc[MT][3] - wa, za);                                                         \
    *reinterpret_cast<float4*>(dst + 16 * (MT) + 4 * hi) = o;                                      \
  }
  INT2KV_OUT_TILE(0)
  INT2KV_OUT_TILE(1)
  INT2KV_OUT_TILE(2)
  INT2KV_OUT_TILE(3)
  INT2KV_OUT_TILE(4)
  INT2KV_OUT_TILE(5)
  INT2KV_OUT_TILE(6)
  INT2KV_OUT_TILE(7)
#undef INT2KV_OUT_TILE
  wait_vm_all();
  bool fin = true;
#pragma unroll
  for (int t = 0; t < NT; ++t) fin = fin && __builtin_isfinite(st.wsum[t][0]);
  return __any(!fin) == 0;
}

// Persistent, head-grouped scan: work-group g covers pages [lo(g), lo(g+1)) of the concatenation
// of all sequences (even split, so every group streams the same number of page records); wave w
// handles KV head 8*blockIdx.y + w of those pages, so the eight waves read the adjacent records
// of one block together. A range crossing sequence boundaries is scanned segment by segment; the
// partial of (group g, sequence b) goes to slot g + b, which is unique because the (g, b) pairs
// that meet form a monotone staircase.
template <bool WIDE, int NG>
__global__ __launch_bounds__(512, 1) void decode_scan_flat_kernel(DecodeArgs a) {
  __shared__ __attribute__((aligned(16))) uint8_t stage[kWavesPerWG][kStages][2][kRecord];
  __shared__ _Float16 p_lds[kWavesPerWG][2][2][8][kBlock];
  __shared__ float al_lds[kWavesPerWG][8];
  __shared__ __attribute__((aligned(16))) uint8_t cz_lds[kWavesPerWG][128 * NG + 16];

  // Work-groups are dispatched round-robin over the 8 XCDs (each with its own L2). Range g goes to
  // the work-group dispatched as blockIdx.x with g = (x % 8) (G / 8) + x / 8, so that each XCD scans
  // one contiguous eighth of the pages: the few work-groups sharing a sequence then share that
  // sequence's query operands and page-list entries through one L2.
  const int G = gridDim.x;
  const int g = G % 8 == 0 ? (int)(blockIdx.x % 8) * (G / 8) + (int)(blockIdx.x / 8) : (int)blockIdx.x;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), l = threadIdx.x & 63;
  const int h = blockIdx.y * kWavesPerWG + w;
  const bool all_waves = a.H < kWavesPerWG || (int)(blockIdx.y + 1) * kWavesPerWG <= a.H;
  if (h >= a.H) return;
  const cint_ptr prefix = (cint_ptr)(uintptr_t)(a.prefix);
  const int P = prefix[a.B];
  if (P == 0) return;
  const cint_ptr info = (cint_ptr)(uintptr_t)(a.wg_info + 4 * g);
  const int s = info[3], e = info[7];  // lo(g), lo(g + 1)
  if (s >= e) return;
  int b = info[0], Sb = info[1], Sb1 = info[2];  // prefix[b] <= s < prefix[b + 1]
  for (int pos = s;;) {
    const int seg_end = min(e, Sb1);
    const int Sb2 = seg_end < e ? prefix[b + 2] : 0;  // next sequence's end, fetched ahead
    // a segment whose value sums overflowed fp16 (V scales of 256 and more) is scanned again by this
    // wave in the scaled form, without the steady loop's work-group barriers: every wave still
    // executes the same number of barriers, so the others only wait for it at their next one
    if (!scan_segment<WIDE, NG, false>(a, b, h, pos, seg_end, g + b, l, &stage[w][0][0][0], p_lds[w], al_lds[w],
                                       cz_lds[w], all_waves))
      scan_segment<WIDE, NG, true>(a, b, h, pos, seg_end, g + b, l, &stage[w][0][0][0], p_lds[w], al_lds[w],
                                   cz_lds[w], false);
    pos = seg_end;
    if (pos >= e) break;
    ++b;
    Sb = Sb1;
    Sb1 = Sb2;
    while (Sb1 <= pos) Sb1 = prefix[++b + 1];  // skip empty sequences
  }
}

// Merge the partials of each (sequence, query head) over the work-groups whose ranges met the
// sequence (and the BF16-window partial, when there is one), then undo the value rotation (o = o' R_V^T, unless W_O arrives pre-folded).
// Block (sequence, KV head) of kMergeSlots x 128 threads: slot s merges the work-groups ga + s,
// ga + s + kMergeSlots, ... (one round of loads for up to kMergeSlots work-groups), thread c of a
// slot owns channel c; the slots are then combined in a fixed order through LDS (deterministic),
// thread (c, s) finishing query heads s, s + kMergeSlots, ... The un-rotation has the 128 threads of slot 0 share one
// pass over R_V (row c of R_V per thread) for all query heads.

// First stage of the two-stage merge (few, long sequences): block (sequence b, KV head h, range z)
// folds the work-group slots ga + z n .. ga + z n + n - 1 of the sequence (n = ceil(G / s1)) into
// one partial per query head, in slot order, and writes it to part2 (m = -inf for an empty range).
// Thread (channel c, slot lane sl) takes every eighth slot; the lanes are combined in a fixed order.
__global__ __launch_bounds__(1024) void merge_stage1_kernel(DecodeArgs a, int G) {
  __shared__ float ms[8][8], ls[8][8];
  __shared__ float os[8][8][kHeadDim];
  const int b = blockIdx.x, h = blockIdx.y, z = blockIdx.z, c = threadIdx.x & 127, sl = threadIdx.x >> 7;
  const int gq = a.gq, per = (G + a.s1 - 1) / a.s1;
  const int ga = a.seq_wg[2 * b], gb = a.seq_wg[2 * b + 1];
  const int lo = ga + z * per, hi = min(gb, lo + per - 1);
  float M[8], lsum[8], osum[8];
#pragma unroll
  for (int jj = 0; jj < 8; ++jj) {
    M[jj] = -INFINITY;
    lsum[jj] = 0.0f;
    osum[jj] = 0.0f;
  }
  for (int gg = lo + sl; gg <= hi; gg += 8) {
    const int r0 = a.wg_info[4 * gg + 3], r1 = a.wg_info[4 * gg + 7];
    const float* base = a.part + ((size_t)(gg + b) * a.Hq + h * gq) * kPartStride;
    float mv[8], lv[8], ov[8];
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) {
      const float* pp = base + min(jj, gq - 1) * kPartStride;
      mv[jj] = pp[0];
      lv[jj] = pp[1];
      ov[jj] = pp[4 + c];
    }
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) {
      const bool valid = r0 < r1 && mv[jj] != -INFINITY;
      const float Mn = valid ? fmaxf(M[jj], mv[jj]) : M[jj];
      const float fa = valid ? __builtin_amdgcn_exp2f(M[jj] - Mn) : 1.0f;
      const float fb = valid ? __builtin_amdgcn_exp2f(mv[jj] - Mn) : 0.0f;
      lsum[jj] = fmaf(lsum[jj], fa, valid ? fb * lv[jj] : 0.0f);
      osum[jj] = fmaf(osum[jj], fa, valid ? fb * ov[jj] : 0.0f);
      M[jj] = Mn;
    }
  }
  if (c == 0) {
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) {
      ms[sl][jj] = M[jj];
      ls[sl][jj] = lsum[jj];
    }
  }
#pragma unroll
  for (int jj = 0; jj < 8; ++jj) os[sl][jj][c] = osum[jj];
  __syncthreads();
  const int jj = sl;  // thread (c, sl) finishes query head sl
  if (jj >= gq) return;
  float Mx = -INFINITY;
#pragma unroll
  for (int t = 0; t < 8; ++t) Mx = fmaxf(Mx, ms[t][jj]);
  float L = 0.0f, O = 0.0f;
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    const float f = ms[t][jj] == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(ms[t][jj] - Mx);
    L = fmaf(f, ls[t][jj], L);
    O = fmaf(f, os[t][jj][c], O);
  }
  float* dst = a.part2 + ((size_t)(b * a.s1 + z) * a.Hq + h * gq + jj) * kPartStride;
  if (c == 0) {
    dst[0] = Mx;
    dst[1] = L;
  }
  dst[4 + c] = O;
}

template <int kMergeSlots>
__global__ __launch_bounds__(128 * kMergeSlots) void merge_flat_kernel(DecodeArgs a, int G, int unrotate,
                                                                       float* __restrict__ out,
                                                                       uint16_t* __restrict__ ob, int fmt) {
  __shared__ float ms[kMergeSlots][8], ls[kMergeSlots][8];
  __shared__ float os[kMergeSlots][8][kHeadDim];
  __shared__ float vs[8][kHeadDim];
  __shared__ float wsh[8][kHeadDim];  // BF16-window part of each head output (model basis)
  const int b = blockIdx.x, h = blockIdx.y, c = threadIdx.x & 127, sl = threadIdx.x >> 7, gq = a.gq;
  // the BF16-window partials of this thread's query heads (model basis, one per window slice), all
  // loaded first (slices past win_slices read slice 0 and are dropped), folded in below
  constexpr int kR = 8 / kMergeSlots;
  float wm[kR][kWinMaxSlices], wl[kR][kWinMaxSlices], wo[kR][kWinMaxSlices];
  if (a.wpart) {
#pragma unroll
    for (int r = 0; r < kR; ++r)
#pragma unroll
      for (int s = 0; s < kWinMaxSlices; ++s) {
        const int ss = s < a.win_slices ? s : 0;
        const float* pp =
            a.wpart + (((size_t)ss * a.B + b) * a.Hq + h * gq + min(sl + kMergeSlots * r, gq - 1)) * kPartStride;
        wm[r][s] = s < a.win_slices ? pp[0] : -INFINITY;
        wl[r][s] = pp[1];
        wo[r][s] = pp[4 + c];
      }
  }
  // groups whose ranges meet the sequence, from the page-prefix block; in the second stage of the
  // two-stage merge, the sequence's folded slot ranges instead
  const bool st2 = a.s1 > 0;
  const int ga = st2 ? 0 : a.seq_wg[2 * b], gb = st2 ? a.s1 - 1 : a.seq_wg[2 * b + 1];
  auto slot_base = [&](int gg) {
    return st2 ? a.part2 + ((size_t)(b * a.s1 + gg) * a.Hq + h * gq) * kPartStride
               : a.part + ((size_t)(gg + b) * a.Hq + h * gq) * kPartStride;
  };
  float M[8], lsum[8], osum[8];
#pragma unroll
  for (int jj = 0; jj < 8; ++jj) {
    M[jj] = -INFINITY;
    lsum[jj] = 0.0f;
    osum[jj] = 0.0f;
  }
  // rounds of kMergeSlots slots; a long sequence (many groups) loads two rounds per trip
  auto merge_round = [&](const float (&mv)[8], const float (&lv)[8], const float (&ov)[8], bool nonempty) {
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) {
      // a partial with no cached token has m = -inf (or the scan's finite floor) and l = 0
      const bool valid = nonempty && mv[jj] != -INFINITY;
      const float Mn = valid ? fmaxf(M[jj], mv[jj]) : M[jj];
      const float fa = valid ? __builtin_amdgcn_exp2f(M[jj] - Mn) : 1.0f;
      const float fb = valid ? __builtin_amdgcn_exp2f(mv[jj] - Mn) : 0.0f;
      lsum[jj] = fmaf(lsum[jj], fa, valid ? fb * lv[jj] : 0.0f);
      osum[jj] = fmaf(osum[jj], fa, valid ? fb * ov[jj] : 0.0f);
      M[jj] = Mn;
    }
  };
  for (int gg = ga + sl; gg <= gb; gg += 2 * kMergeSlots) {
    // the range bounds and the partials are loaded together (one round trip): slot gg + b exists
    // for every group, and an empty range (which wrote nothing, so the slot holds stale values) is
    // dropped by selects below, never multiplied; a second slot past gb is loaded as slot gg and
    // dropped
    const int g2 = gg + kMergeSlots <= gb ? gg + kMergeSlots : gg;
    // stage-2 ranges are never stale (an empty one was written with m = -inf)
    const int r0 = st2 ? 0 : a.wg_info[4 * gg + 3], r1 = st2 ? 1 : a.wg_info[4 * gg + 7];
    const int r2 = st2 ? 0 : a.wg_info[4 * g2 + 3], r3 = st2 ? 1 : a.wg_info[4 * g2 + 7];
    const float* base = slot_base(gg);
    const float* base2 = slot_base(g2);
    float mv[8], lv[8], ov[8], mv2[8], lv2[8], ov2[8];
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) {  // every load first, then the arithmetic (no load behind a test)
      const float* pp = base + min(jj, gq - 1) * kPartStride;
      const float* p2 = base2 + min(jj, gq - 1) * kPartStride;
      mv[jj] = pp[0];
      lv[jj] = pp[1];
      ov[jj] = pp[4 + c];
      mv2[jj] = p2[0];
      lv2[jj] = p2[1];
      ov2[jj] = p2[4 + c];
    }
    merge_round(mv, lv, ov, r0 < r1);
    merge_round(mv2, lv2, ov2, g2 != gg && r2 < r3);
  }
  if (c == 0) {
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) {
      ms[sl][jj] = M[jj];
      ls[sl][jj] = lsum[jj];
    }
  }
#pragma unroll
  for (int jj = 0; jj < 8; ++jj) os[sl][jj][c] = osum[jj];
  __syncthreads();
  // thread (c, s): query heads s, s + kMergeSlots, ..., channel c, the slots in a fixed order
  float val[8 / kMergeSlots], wval[8 / kMergeSlots];
#pragma unroll
  for (int r = 0; r < 8 / kMergeSlots; ++r) {
    const int jj = sl + kMergeSlots * r;
    float Mx = -INFINITY;
#pragma unroll
    for (int t = 0; t < kMergeSlots; ++t) Mx = fmaxf(Mx, ms[t][jj]);
    if (a.wpart) {
#pragma unroll
      for (int s = 0; s < kWinMaxSlices; ++s) Mx = fmaxf(Mx, wm[r][s]);
    }
    float L = 0.0f, O = 0.0f, Ow = 0.0f;
#pragma unroll
    for (int t = 0; t < kMergeSlots; ++t) {
      const float mt = ms[t][jj];
      const float f = mt == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(mt - Mx);
      L = fmaf(f, ls[t][jj], L);
      O = fmaf(f, os[t][jj][c], O);
    }
    if (a.wpart) {
#pragma unroll
      for (int s = 0; s < kWinMaxSlices; ++s) {
        const float f = wm[r][s] == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(wm[r][s] - Mx);
        L = fmaf(f, wl[r][s], L);
        Ow = fmaf(f, wo[r][s], Ow);
      }
    }
    val[r] = L > 0.0f ? O / L : 0.0f;
    wval[r] = L > 0.0f ? Ow / L : 0.0f;
  }
  if (!a.wpart && !unrotate) {
#pragma unroll
    for (int r = 0; r < 8 / kMergeSlots; ++r) {
      const int jj = sl + kMergeSlots * r;
      if (jj < gq)
        store_head_out(val[r], out, ob, fmt, ((size_t)b * a.Hq + h * gq + jj) * kHeadDim + c,
                       (size_t)a.B * a.Hq * kHeadDim);
    }
    return;
  }
  // The output's basis: o = o_int2 R_V^T (+ o_win, model basis) when the merge un-rotates, or
  // o' = o_int2 + o_win R_V when the output projection is folded with R_V. Every thread (c, slot)
  // sums the channels i of its slot's part of the product for all heads (all of its R_V loads issued
  // together), and the parts are added through LDS.
#pragma unroll
  for (int r = 0; r < 8 / kMergeSlots; ++r) {
    vs[sl + kMergeSlots * r][c] = val[r];
    wsh[sl + kMergeSlots * r][c] = wval[r];
  }
  __syncthreads();
  constexpr int kPart = kHeadDim / kMergeSlots;
  const float* R = a.R_v + (size_t)h * kHeadDim * kHeadDim;
  float rv[kPart];
  if (unrotate) {
    const float4* row = reinterpret_cast<const float4*>(R + (size_t)c * kHeadDim + sl * kPart);  // R_V[c][i]
#pragma unroll
    for (int i4 = 0; i4 < kPart / 4; ++i4) {
      const float4 q4 = row[i4];
      rv[4 * i4] = q4.x;
      rv[4 * i4 + 1] = q4.y;
      rv[4 * i4 + 2] = q4.z;
      rv[4 * i4 + 3] = q4.w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < kPart; ++i) rv[i] = R[(size_t)(sl * kPart + i) * kHeadDim + c];  // R_V[i][c]
  }
  float acc[8];
#pragma unroll
  for (int j2 = 0; j2 < 8; ++j2) acc[j2] = 0.0f;
  const float(*src)[kHeadDim] = unrotate ? vs : wsh;
#pragma unroll
  for (int i = 0; i < kPart; ++i)
#pragma unroll
    for (int j2 = 0; j2 < 8; ++j2) acc[j2] = fmaf(src[j2][sl * kPart + i], rv[i], acc[j2]);
#pragma unroll
  for (int j2 = 0; j2 < 8; ++j2) os[sl][j2][c] = acc[j2];  // the slots' partials are no longer needed
  __syncthreads();
  const float(*add)[kHeadDim] = unrotate ? wsh : vs;
#pragma unroll
  for (int r = 0; r < 8 / kMergeSlots; ++r) {
    const int jj = sl + kMergeSlots * r;
    float o = a.wpart ? add[jj][c] : 0.0f;
#pragma unroll
    for (int t = 0; t < kMergeSlots; ++t) o += os[t][jj][c];
    if (jj < gq)
      store_head_out(o, out, ob, fmt, ((size_t)b * a.Hq + h * gq + jj) * kHeadDim + c,
                     (size_t)a.B * a.Hq * kHeadDim);
  }
}

hipError_t launch_qprep(const DecodeArgs& a, const AppendArgs* ap, hipStream_t s) {
  if (a.gq > 8) return hipErrorNotSupported;
  AppendArgs none{};
  int nap = 0;
  if (ap && ap->n > 0) {
    none = *ap;
    none.nbx = (ap->n + 16 * 4 - 1) / (16 * 4);  // one 16-token tile per wave and step
    nap = none.nbx * ap->cv.num_kv_heads * 2;
  }
  const int nq = a.H * ((a.B + kQpSeqs - 1) / kQpSeqs) * qp_split(nap > 0);
  const long long maxlen = min((long long)a.max_ctx, (long long)a.max_blocks * kBlock);
  const int maxp = (int)((maxlen + kBlock - 1) / kBlock);
  const int nseg = max(1, (maxp + kPlPages - 1) / kPlPages);
  if (nap > 0)
    hipLaunchKernelGGL(qprep_kernel<true>, dim3(nap + 1 + nq + a.B * nseg), dim3(256), 0, s, a, a.gq > 4 ? 1 : 0, nq,
                       nseg, none, nap);
  else
    hipLaunchKernelGGL(qprep_kernel<false>, dim3(1 + nq + a.B * nseg), dim3(256), 0, s, a, a.gq > 4 ? 1 : 0, nq, nseg,
                       none, 0);
  return hipGetLastError();
}

hipError_t launch_decode_split_mfma(const DecodeArgs& a, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  if (a.gq > 8) return hipErrorNotSupported;
  dim3 grid(a.grid_g, (a.H + kWavesPerWG - 1) / kWavesPerWG);
  const int threads = 64 * min(a.H, kWavesPerWG);
  if (a.gq > 4 && a.groups == 1)
    hipExtLaunchKernelGGL((decode_scan_flat_kernel<true, 1>), grid, dim3(threads), 0, s, ev0, ev1, 0, a);
  else if (a.gq > 4)
    hipExtLaunchKernelGGL((decode_scan_flat_kernel<true, 4>), grid, dim3(threads), 0, s, ev0, ev1, 0, a);
  else if (a.groups == 1)
    hipExtLaunchKernelGGL((decode_scan_flat_kernel<false, 1>), grid, dim3(threads), 0, s, ev0, ev1, 0, a);
  else
    hipExtLaunchKernelGGL((decode_scan_flat_kernel<false, 4>), grid, dim3(threads), 0, s, ev0, ev1, 0, a);
  return hipGetLastError();
}

hipError_t launch_merge_flat(const DecodeArgs& a, bool unrotate, float* out, uint16_t* ob, int fmt, hipStream_t s) {
  if (a.gq > 8) return hipErrorNotSupported;
  // four slots when many sequences share the work-groups (short spans; fewer idle waves to
  // dispatch), eight for few, long sequences (fewer rounds of loads)
  if (a.s1 > 0) {
    // few, long sequences: every range of slots folded by its own block first, so that the
    // partials stream through B x H x s1 blocks instead of B x H
    DecodeArgs a1 = a;
    hipLaunchKernelGGL(merge_stage1_kernel, dim3(a.B, a.H, a.s1), dim3(1024), 0, s, a1, a.grid_g);
    hipLaunchKernelGGL(merge_flat_kernel<8>, dim3(a.B, a.H), dim3(128 * 8), 0, s, a, a.grid_g, unrotate ? 1 : 0, out,
                       ob, fmt);
  } else if (a.B >= 32)
    hipLaunchKernelGGL(merge_flat_kernel<4>, dim3(a.B, a.H), dim3(128 * 4), 0, s, a, a.grid_g, unrotate ? 1 : 0, out,
                       ob, fmt);
  else
    hipLaunchKernelGGL(merge_flat_kernel<8>, dim3(a.B, a.H), dim3(128 * 8), 0, s, a, a.grid_g, unrotate ? 1 : 0, out,
                       ob, fmt);
  return hipGetLastError();
}

}  // namespace int2kv
