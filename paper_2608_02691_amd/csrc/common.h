// Shared device helpers of the INT2 KV-cache library (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>
#include <stdint.h>

namespace int2kv {

constexpr int kHeadDim = 128;
constexpr int kBlock = 16;
constexpr int kGroup = 32;
constexpr int kGroups = kHeadDim / kGroup;
constexpr int kRecord = 1536;
// byte offsets inside one (block, KV head) record
constexpr int kOffKCodes = 0;     // [16 tok][16 halves]
constexpr int kOffVCodes = 512;   // [16 halves][16 tok]
constexpr int kOffKMeta = 1024;   // [16 tok][4 groups] (fp16 s, fp16 z)
constexpr int kOffVScale = 1280;  // [4 groups][16 tok] fp16
constexpr int kOffVZero = 1408;   // [4 groups][16 tok] fp16

// Record layout for NG groups per token: NG = 4 (groups of 32 channels, the constants above,
// 1536-byte records) or NG = 1 (one group of 128 channels, 1152-byte records). Codes as above;
// K (s, z) of token t and group g at kOffKMeta + 4 NG t + 4 g; V scale and zero of group g and
// token t at kOffVScale + 32 g + 2 t and kOffVZero + 32 g + 2 t.
template <int NG>
struct Rec {
  static constexpr int kGroupSize = kHeadDim / NG;
  static constexpr int kOffKMeta = 1024;
  static constexpr int kOffVScale = 1024 + 64 * NG;
  static constexpr int kOffVZero = 1024 + 96 * NG;
  static constexpr int kBytes = 1024 + 128 * NG;
};
static_assert(Rec<4>::kBytes == kRecord && Rec<4>::kOffVScale == kOffVScale && Rec<4>::kOffVZero == kOffVZero,
              "the 32-channel layout");

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b) { return __uint_as_float(b << 16); }
// round to nearest even on the upper 16 bits (finite inputs)
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float x) {
  const uint32_t u = __float_as_uint(x);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}
// One head-output value, either as fp32 (out) or as two bf16 terms for the output projection:
// hi = bf16(v) at ob[idx], lo = bf16(v - hi) at ob[total + idx].
// Head output v at index idx: fp32 to out (fmt 0), two bf16 terms hi, lo = bf16(v - hi) at idx and
// total + idx of ob (fmt 1), or one fp16 term (fmt 2).
__device__ __forceinline__ void store_head_out(float v, float* out, uint16_t* ob, int fmt, size_t idx, size_t total) {
  if (fmt == 1) {
    const uint32_t h = f32_to_bf16_rne(v);
    ob[idx] = (uint16_t)h;
    ob[total + idx] = (uint16_t)f32_to_bf16_rne(v - __uint_as_float(h << 16));
  } else if (fmt == 2) {
    ob[idx] = __half_as_ushort(__float2half_rn(v));
  } else {
    out[idx] = v;
  }
}
__device__ __forceinline__ float f16_bits_to_f32(uint32_t h) {
  return __half2float(__ushort_as_half(static_cast<unsigned short>(h)));
}

// Group parameters of the group-wise affine INT2 quantizer: scale and zero rounded to fp16,
// and the fp32 values the codes are computed with. Fixed rounding sequence, no contraction.
__device__ __forceinline__ void int2_group_params(float mn, float mx, float clip, uint32_t& s_bits,
                                                  uint32_t& z_bits, float& zf, float& inv) {
#pragma clang fp contract(off)
  if (clip != 1.0f) {
    mn = clip * mn;
    mx = clip * mx;
  }
  const float s32 = (mx - mn) / 3.0f;
  const __half s = __float2half_rn(s32);
  const __half z = __float2half_rn(mn);
  s_bits = __half_as_ushort(s);
  z_bits = __half_as_ushort(z);
  const float sf = __half2float(s);
  zf = __half2float(z);
  inv = sf > 0.0f ? 1.0f / sf : 0.0f;
}

__device__ __forceinline__ uint32_t int2_code(float x, float zf, float inv) {
#pragma clang fp contract(off)
  const float d = x - zf;
  const float t = d * inv;
  const float r = fminf(fmaxf(rintf(t), 0.0f), 3.0f);
  return static_cast<uint32_t>(r);
}

// DPP lane move inside rows of 16 lanes (CTRL = row_ror:n is 0x120 + n)
template <int CTRL>
__device__ __forceinline__ float dppf(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}

// max / min / sum over the 16 lanes of a DPP row (every lane gets the result)
__device__ __forceinline__ float row_max16(float x) {
  x = fmaxf(x, dppf<0x128>(x));
  x = fmaxf(x, dppf<0x124>(x));
  x = fmaxf(x, dppf<0x122>(x));
  x = fmaxf(x, dppf<0x121>(x));
  return x;
}
__device__ __forceinline__ float row_min16(float x) {
  x = fminf(x, dppf<0x128>(x));
  x = fminf(x, dppf<0x124>(x));
  x = fminf(x, dppf<0x122>(x));
  x = fminf(x, dppf<0x121>(x));
  return x;
}
__device__ __forceinline__ float row_sum16(float x) {
  x += dppf<0x128>(x);
  x += dppf<0x124>(x);
  x += dppf<0x122>(x);
  x += dppf<0x121>(x);
  return x;
}

}  // namespace int2kv
