// Pieces shared by the attention kernels read from the packed caches: partial
// layout, LDS row pitches, wavefront reductions and the value-code MFMA operands.
#pragma once
#include "device_common.hpp"

namespace spectra_dev {

constexpr int PART = 136;  // floats per (chunk, query head): m, l, Z[4], pad[2], acc[128]
constexpr int WROW = 72;  // bf16 per weight row (64 tokens + pad: spreads rows over LDS banks)
constexpr float RESCALE_SLACK = 4.0f;  // log2 units: weights exp2(score - m) stay <= 16
constexpr int AROW = D + 4;  // floats per row of merged value sums (rows of one wave spread over banks)
constexpr int TROW = 68;  // uint32 per staged record-word row (64 tokens + pad: distinct words of one
                          // token group fall on distinct LDS banks)

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = __builtin_fmaxf(v, __shfl_xor(v, o));
  return v;
}

// DPP lane moves (row = 16 lanes): quad_perm [1,0,3,2] 0xB1 and [2,3,0,1] 0x4E,
// row_half_mirror 0x141, row_mirror 0x140, row_bcast:15 0x142, row_bcast:31 0x143.
// Lanes outside ROWMASK, or with no source, receive IDENT.
template <int CTRL, int ROWMASK>
__device__ __forceinline__ float dpp(float v, float ident) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, ident), __builtin_bit_cast(int, v),
                                                               CTRL, ROWMASK, 0xF, false));
}
// Sum over the 64 lanes, valid in lane 63: butterflies within each row of 16,
// then the row totals are chained through row broadcasts.
__device__ __forceinline__ float wave_sum_lane63(float v) {
  v += dpp<0xB1, 0xF>(v, 0.0f);
  v += dpp<0x4E, 0xF>(v, 0.0f);
  v += dpp<0x141, 0xF>(v, 0.0f);
  v += dpp<0x140, 0xF>(v, 0.0f);
  v += dpp<0x142, 0xA>(v, 0.0f);
  v += dpp<0x143, 0xC>(v, 0.0f);
  return v;
}
// Maximum over the 64 lanes, returned in every lane.
__device__ __forceinline__ float wave_max_all(float v) {
  v = __builtin_fmaxf(v, dpp<0xB1, 0xF>(v, v));
  v = __builtin_fmaxf(v, dpp<0x4E, 0xF>(v, v));
  v = __builtin_fmaxf(v, dpp<0x141, 0xF>(v, v));
  v = __builtin_fmaxf(v, dpp<0x140, 0xF>(v, v));
  const float r0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 0));
  const float r1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 16));
  const float r2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 32));
  const float r3 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 48));
  return __builtin_fmaxf(__builtin_fmaxf(r0, r1), __builtin_fmaxf(r2, r3));
}

// ---------------------------------------------------------------------------
// Value-code operands: the codes of in-group coefficients n and n + 1 (bit
// offsets off = n*b and off + b in the group payload at record word `pay`) for
// 8 consecutive tokens, as bf16 pairs. CLS 0: b in {1,2,4} (both codes in one
// byte: one byte gather per token pair); CLS 1: b in {3,5,6,7} (one 32-bit
// funnel-shift window per token holds both). Both give 1 + c 2^-b: the code in
// the top b bits of the 7-bit mantissa under the exponent of 1.0 (`magic`,
// 0x3F80 in both halves, held in a VGPR), so the offset 1 removed afterwards (a
// product against -1) is at most 2^b times the code's weight and costs no
// precision; the caller scales the sums by 2^b. CLS 2: b = 8, exact c.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t rotr32(uint32_t x, uint32_t s) { return __builtin_amdgcn_alignbit(x, x, s); }

template <int CLS>
__device__ __forceinline__ void value_codes2(const uint32_t* __restrict__ vt, int pay, int used, int b, int off,
                                             int tok0, uint32_t magic, u32x4& r0, u32x4& r1) {
  // offsets fit in 24 bits: full-rate 24-bit multiplies instead of 32-bit ones
  const int w = pay + (off >> 5), o = off & 31;
  const uint32_t* row = vt + __umul24(w, TROW) + tok0;
  const u32x4 a0 = *reinterpret_cast<const u32x4*>(row);
  const u32x4 a1 = *reinterpret_cast<const u32x4*>(row + 4);
  const uint32_t M = ((1u << b) - 1u) << (7 - b);  // the code's bits at the top of the mantissa
  const uint32_t MM = M | (M << 16);
  if constexpr (CLS == 0) {
    // byte k of two tokens' words in both bytes of each half (bytes k, k, 4 + k, 4 + k,
    // a byte broadcast, not a 32-bit multiply); the copy in the upper byte of a half,
    // shifted right, puts a code at mantissa bits 7 - b .. 6 of that half
    const uint32_t k = (uint32_t)o >> 3, sh = (uint32_t)o & 7u;
    const uint32_t sel = __builtin_amdgcn_perm(k, k, 0u) | 0x04040000u;
    const uint32_t s0 = sh + 1 + b, s1 = s0 + b;
    uint32_t y[4];
    y[0] = __builtin_amdgcn_perm(a0[1], a0[0], sel);
    y[1] = __builtin_amdgcn_perm(a0[3], a0[2], sel);
    y[2] = __builtin_amdgcn_perm(a1[1], a1[0], sel);
    y[3] = __builtin_amdgcn_perm(a1[3], a1[2], sel);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      r0[i] = ((y[i] >> s0) & MM) | magic;
      r1[i] = ((y[i] >> s1) & MM) | magic;
    }
  } else {
    const int wn = (w + 1 < used) ? w + 1 : w;  // the next word only matters when a code straddles
    const uint32_t* rown = vt + __umul24(wn, TROW) + tok0;
    const u32x4 b0 = *reinterpret_cast<const u32x4*>(rown);
    const u32x4 b1 = *reinterpret_cast<const u32x4*>(rown + 4);
    uint32_t c[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      c[i] = __builtin_amdgcn_alignbit(b0[i], a0[i], o);
      c[4 + i] = __builtin_amdgcn_alignbit(b1[i], a1[i], o);
    }
    if constexpr (CLS == 2) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        r0[i] = int_to_bf16_pair(c[2 * i] & 0xFFu, c[2 * i + 1] & 0xFFu);
        r1[i] = int_to_bf16_pair((c[2 * i] >> 8) & 0xFFu, (c[2 * i + 1] >> 8) & 0xFFu);
      }
    } else {
      // codes at bits 0.. and b.. of each half; rotations (either direction, bits that
      // wrap land outside the mask) move them to bits 7 - b .. 6
      const uint32_t s0 = (uint32_t)(32 - (7 - b)) & 31u, s1 = (uint32_t)(32 + 2 * b - 7) & 31u;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint32_t y = __builtin_amdgcn_perm(c[2 * i + 1], c[2 * i], 0x05040100u);
        r0[i] = (rotr32(y, s0) & MM) | magic;
        r1[i] = (rotr32(y, s1) & MM) | magic;
      }
    }
  }
}

}  // namespace spectra_dev
