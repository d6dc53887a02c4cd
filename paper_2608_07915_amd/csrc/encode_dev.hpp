// Per-group encode steps shared by the encode kernel and the decode-step kernel
// (Sec. 3.2-3.3): projection of staged token rows onto the kept group's basis
// columns on MFMA, centering, per-token group metadata, quantization, packing.
#pragma once
#include "device_common.hpp"

namespace spectra_dev {

// ---------------------------------------------------------------------------
// Quantization of 16 centered coefficients of one token (one lane half); the
// two halves of a group exchange min/max. Returns the metadata word; q[j] holds
// code j in its low B bits (the bits above are not zero: callers mask).
//   z = fp16(min), s = fp16(max(max - z, 0) / (2^B - 1)), both RNE, saturating;
//   code = clamp(rne((c - z) / s), 0, 2^B - 1), 0 when s = 0.
// The rounding to an integer is one fused multiply-add onto 1.5 * 2^23, where
// fp32 values are spaced one apart, so the sum's low mantissa bits are the
// rounded quotient (ties to even); a clamp on the sum gives the code range.
// 1/(2^B - 1) and 1/s are fp32 reciprocals: both quotients are within a few
// fp32 ulps of the exact ones, so results differ from exact arithmetic only
// at rounding ties.
// ---------------------------------------------------------------------------
constexpr float QROUND = 12582912.0f;  // 1.5 * 2^23

// The value of lane l ^ 32 (one lane swap between the wave's halves).
__device__ __forceinline__ uint32_t other_half_u(uint32_t v) {
  // the swap exchanges lanes 32..63 of the first operand with lanes 0..31 of the
  // second: r[0] holds v[0..31] in both halves, r[1] holds v[32..63] in both
  const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return (threadIdx.x & 32) ? r[0] : r[1];
}
__device__ __forceinline__ float other_half(float v) { return __uint_as_float(other_half_u(__float_as_uint(v))); }

template <int B>
__device__ __forceinline__ uint32_t quantize16(const float (&c)[16], uint32_t (&q)[16]) {
  float lo = c[0], hi = c[0];
#pragma unroll
  for (int j = 1; j < 16; ++j) {
    lo = __builtin_fminf(lo, c[j]);
    hi = __builtin_fmaxf(hi, c[j]);
  }
  lo = __builtin_fminf(lo, other_half(lo));
  hi = __builtin_fmaxf(hi, other_half(hi));
  constexpr float LEV = (float)((1 << B) - 1);
  constexpr float INV_LEV = 1.0f / LEV;
  const uint32_t z16 = f2h_sat(lo);
  const float z = h2f(z16);
  const uint32_t s16 = f2h_sat(__builtin_fmaxf(hi - z, 0.0f) * INV_LEV);
  const float s = h2f(s16);
  const float rinv = s > 0.0f ? __builtin_amdgcn_rcpf(s) : 0.0f;
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    const float v = __builtin_fmaf(c[j] - z, rinv, QROUND);
    q[j] = __float_as_uint(__builtin_amdgcn_fmed3f(v, QROUND, QROUND + LEV));
  }
  return s16 | (z16 << 16);
}

// ---------------------------------------------------------------------------
// Basis columns of kept group grp as MFMA A operands: row r of the 32x32 tile is
// in-group coefficient jj(r), so that after the product lane half h holds
// coefficients 16h..16h+15. The fp32 basis is split into three bf16 parts.
// Also loads the 16 coefficient means of the lane half, negated (the projection's
// starting accumulator).
// ---------------------------------------------------------------------------
__device__ __forceinline__ void load_group_operands(const float* __restrict__ Vs, const float* __restrict__ ms, int grp,
                                                    int col, int h, bf16x8 (&Va)[3][8], f32x16& nm) {
  const int r = col;
  const int jj = 16 * ((r & 7) >> 2) + 4 * (r >> 3) + (r & 3);
  const int cidx = G * grp + jj;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    uint32_t p0[8], p1[8], p2[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) split3(Vs[(16 * k + 8 * h + i) * D + cidx], p0[i], p1[i], p2[i]);
    Va[0][k] = as_bf16x8(u32x4{pack2(p0[0], p0[1]), pack2(p0[2], p0[3]), pack2(p0[4], p0[5]), pack2(p0[6], p0[7])});
    Va[1][k] = as_bf16x8(u32x4{pack2(p1[0], p1[1]), pack2(p1[2], p1[3]), pack2(p1[4], p1[5]), pack2(p1[6], p1[7])});
    Va[2][k] = as_bf16x8(u32x4{pack2(p2[0], p2[1]), pack2(p2[2], p2[3]), pack2(p2[4], p2[5]), pack2(p2[6], p2[7])});
  }
  const float* m = ms + G * grp + 16 * h;
#pragma unroll
  for (int j = 0; j < 16; ++j) nm[j] = -m[j];
}

// ---------------------------------------------------------------------------
// Projection of the 32 token rows of MFMA block beta of a staged tile (LDS rows
// of ROWB bytes, bf16 or fp32) onto the group's basis columns, accumulated onto
// `init` (the negated coefficient means, so the result is centered): after it,
// lane (h, col) holds coefficients 16h..16h+15 of row 32 beta + col. The operand for
// K step k and part p is PART(p, k) (a bf16x8); both encode paths below issue
// the same MFMAs in the same order, so their results are bit-identical.
// ---------------------------------------------------------------------------
// ROWB = 0 selects the swizzled bf16 layout of the bulk encode: 256-byte rows
// whose 16-byte chunk c sits at chunk position c ^ (row % 16).
template <bool F32IN, int ROWB, bool SERIAL_K = false, typename PartFn>
__device__ __forceinline__ f32x16 project_block(const uint8_t* __restrict__ xs, int beta, int col, int h,
                                                const f32x16& init, PartFn&& part) {
  f32x16 acc = init;
  const int row = 32 * beta + col;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    if constexpr (!F32IN) {
      const int off = ROWB == 0 ? row * 256 + (((2 * k + h) ^ (row & 15)) << 4) : row * ROWB + (16 * k + 8 * h) * 2;
      const bf16x8 xb8 = as_bf16x8(*reinterpret_cast<const u32x4*>(xs + off));
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(part(0, k), xb8, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(part(1, k), xb8, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(part(2, k), xb8, acc, 0, 0, 0);
    } else {
      const float* xr = reinterpret_cast<const float*>(xs + row * ROWB) + 16 * k + 8 * h;
      uint32_t q0[8], q1[8], q2[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) split3(xr[i], q0[i], q1[i], q2[i]);
      const bf16x8 x0 = as_bf16x8(u32x4{pack2(q0[0], q0[1]), pack2(q0[2], q0[3]), pack2(q0[4], q0[5]), pack2(q0[6], q0[7])});
      const bf16x8 x1 = as_bf16x8(u32x4{pack2(q1[0], q1[1]), pack2(q1[2], q1[3]), pack2(q1[4], q1[5]), pack2(q1[6], q1[7])});
      const bf16x8 x2 = as_bf16x8(u32x4{pack2(q2[0], q2[1]), pack2(q2[2], q2[3]), pack2(q2[4], q2[5]), pack2(q2[6], q2[7])});
      const bf16x8 v0 = part(0, k), v1 = part(1, k), v2 = part(2, k);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(v0, x0, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(v0, x1, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(v1, x0, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(v0, x2, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(v1, x1, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(v2, x0, acc, 0, 0, 0);
    }
    // SERIAL_K: nothing moves across K steps, so operands are formed step by
    // step (few registers live) instead of all up front
    if constexpr (SERIAL_K) __builtin_amdgcn_sched_barrier(0);
  }
  return acc;
}

// Quantize and pack one lane's 16 centered coefficients at width B; P holds the
// lane half's 16B payload bits, the return value the group's metadata word.
template <int B>
__device__ __forceinline__ uint32_t quantize_pack(const f32x16& acc, uint32_t (&P)[4]) {
  float c[16];
#pragma unroll
  for (int j = 0; j < 16; ++j) c[j] = acc[j];
  uint32_t q[16];
  const uint32_t meta = quantize16<B>(c, q);
  pack16<B>(q, P);
  return meta;
}

// Record words of one token into LDS staging without branches: every lane
// issues the same stores. Both lane halves write the (identical) metadata word;
// for odd B the upper half's first store goes to `dummy` (a per-wave scratch
// word) instead of a record word.
template <int B>
__device__ __forceinline__ void stage_record_words(uint32_t* rec, uint32_t* dummy, int h, int slot, int gpay,
                                                   uint32_t meta, const uint32_t (&P)[4]) {
  rec[slot * TILE] = meta;
  if constexpr ((B & 1) == 0) {
#pragma unroll
    for (int i = 0; i < B / 2; ++i) rec[(gpay + h * (B / 2) + i) * TILE] = P[i];
  } else {
    // lower half: words 0..N1-1 (its last word shares 16 bits with the upper half);
    // upper half: words N1..B-1 from its bits shifted by 16
    constexpr int N1 = (B + 1) / 2;
    uint32_t S[N1];
    S[0] = P[0] << 16;
#pragma unroll
    for (int i = 1; i < N1; ++i) S[i] = (P[i] << 16) | (P[i - 1] >> 16);
    const uint32_t from_upper = other_half_u(h ? S[0] : 0u);  // lower half: the upper half's first 16 bits
#pragma unroll
    for (int i = 0; i < N1; ++i) {
      uint32_t v;
      uint32_t* dst;
      if (i == 0) {
        v = h ? 0u : (N1 == 1 ? (P[0] | from_upper) : P[0]);
        dst = h ? dummy : rec + gpay * TILE;
      } else {
        v = h ? S[i] : (i == N1 - 1 ? (P[i] | from_upper) : P[i]);
        dst = rec + (gpay + (h ? (B - 1) / 2 + i : i)) * TILE;
      }
      *dst = v;
    }
  }
}

// Quantize, pack and store the projected (centered) block: `rec` is record word 0
// of this lane's token; writes the group's metadata word and payload when `valid`.
// gbits, gpay and slot are wave-uniform.
__device__ __forceinline__ void store_block(const f32x16& acc, uint32_t* __restrict__ rec, bool valid, int h, int slot,
                                            int gbits, int gpay) {
  float c[16];
#pragma unroll
  for (int j = 0; j < 16; ++j) c[j] = acc[j];
  with_bits(gbits, [&](auto bc) {
    constexpr int B = decltype(bc)::value;
    uint32_t q[16], P[4];
    const uint32_t meta = quantize16<B>(c, q);
    pack16<B>(q, P);
    if (h == 0 && valid) rec[slot * TILE] = meta;
    store_payload<B>(rec, 0, gpay, P, h, valid);
  });
}

// Encode one block for one kept group, the basis held as split operands.
template <bool F32IN, int ROWB>
__device__ __forceinline__ void encode_block(const uint8_t* __restrict__ xs, int beta, int col, int h,
                                             const bf16x8 (&Va)[3][8], const f32x16& nm, int64_t slot0,
                                             int64_t t_lo, int64_t t_hi, int64_t sbase, int W, int slot, int gbits,
                                             int gpay, uint32_t* __restrict__ packed) {
  const f32x16 acc = project_block<F32IN, ROWB>(xs, beta, col, h, nm, [&](int p, int k) { return Va[p][k]; });
  const int64_t t = slot0 + 32 * beta + col;
  store_block(acc, packed + rec_word(sbase, t, W, 0), t >= t_lo && t < t_hi, h, slot, gbits, gpay);
}

// Same, with the basis columns streamed from memory K step by K step (a ring of
// PF steps in flight) and split as they arrive: few registers, for callers that
// encode a single block.
template <bool F32IN, int ROWB, int PF = 4>
__device__ __forceinline__ void encode_block_streamed(const uint8_t* __restrict__ xs, int beta, int col, int h,
                                                      const float* __restrict__ Vs, int grp, const f32x16& nm,
                                                      int64_t slot0, int64_t t_lo, int64_t t_hi, int64_t sbase, int W,
                                                      int slot, int gbits, int gpay, uint32_t* __restrict__ packed) {
  const int r = col;
  const int jj = 16 * ((r & 7) >> 2) + 4 * (r >> 3) + (r & 3);
  const float* src = Vs + (8 * h) * D + G * grp + jj;  // row 16k + 8h + i of this lane's column
  float ring[PF][8];
#pragma unroll
  for (int k = 0; k < PF; ++k)
#pragma unroll
    for (int i = 0; i < 8; ++i) ring[k][i] = src[(16 * k + i) * D];
  bf16x8 cur[3];
  const f32x16 acc = project_block<F32IN, ROWB, true>(xs, beta, col, h, nm, [&](int p, int k) {
    if (p == 0) {
      uint32_t p0[8], p1[8], p2[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) split3(ring[k % PF][i], p0[i], p1[i], p2[i]);
      cur[0] = as_bf16x8(u32x4{pack2(p0[0], p0[1]), pack2(p0[2], p0[3]), pack2(p0[4], p0[5]), pack2(p0[6], p0[7])});
      cur[1] = as_bf16x8(u32x4{pack2(p1[0], p1[1]), pack2(p1[2], p1[3]), pack2(p1[4], p1[5]), pack2(p1[6], p1[7])});
      cur[2] = as_bf16x8(u32x4{pack2(p2[0], p2[1]), pack2(p2[2], p2[3]), pack2(p2[4], p2[5]), pack2(p2[6], p2[7])});
      if (k + PF < 8) {
#pragma unroll
        for (int i = 0; i < 8; ++i) ring[k % PF][i] = src[(16 * (k + PF) + i) * D];
      }
    }
    return cur[p];
  });
  const int64_t t = slot0 + 32 * beta + col;
  store_block(acc, packed + rec_word(sbase, t, W, 0), t >= t_lo && t < t_hi, h, slot, gbits, gpay);
}

}  // namespace spectra_dev
