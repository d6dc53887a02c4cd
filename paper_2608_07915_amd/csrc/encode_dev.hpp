// Per-group encode steps shared by the encode kernel and the decode-step kernel
// (Sec. 3.2-3.3): projection of staged token rows onto the kept group's basis
// columns on MFMA, centering, per-token group metadata, quantization, packing.
#pragma once
#include "device_common.hpp"

namespace spectra_dev {

// ---------------------------------------------------------------------------
// Quantization of 16 centered coefficients of one token (one lane half); the
// two halves of a group exchange min/max. Returns codes and the metadata word.
// ---------------------------------------------------------------------------
template <int B>
__device__ __forceinline__ uint32_t quantize16(const float (&c)[16], uint32_t (&q)[16]) {
  float lo = c[0], hi = c[0];
#pragma unroll
  for (int j = 1; j < 16; ++j) {
    lo = __builtin_fminf(lo, c[j]);
    hi = __builtin_fmaxf(hi, c[j]);
  }
  lo = __builtin_fminf(lo, __shfl_xor(lo, 32));
  hi = __builtin_fmaxf(hi, __shfl_xor(hi, 32));
  constexpr float LEV = (float)((1 << B) - 1);
  const uint32_t z16 = f2h_sat(lo);
  const float z = h2f(z16);
  const uint32_t s16 = f2h_sat(__builtin_fmaxf(hi - z, 0.0f) / LEV);
  const float s = h2f(s16);
  const float rinv = s > 0.0f ? 1.0f / s : 0.0f;
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    float u = __builtin_rintf((c[j] - z) * rinv);
    u = __builtin_fminf(__builtin_fmaxf(u, 0.0f), LEV);
    q[j] = (uint32_t)u;
  }
  return s16 | (z16 << 16);
}

// ---------------------------------------------------------------------------
// Basis columns of kept group grp as MFMA A operands: row r of the 32x32 tile is
// in-group coefficient jj(r), so that after the product lane half h holds
// coefficients 16h..16h+15. The fp32 basis is split into three bf16 parts.
// Also loads the 16 coefficient means of the lane half.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void load_group_operands(const float* __restrict__ Vs, const float* __restrict__ ms, int grp,
                                                    int col, int h, bf16x8 (&Va)[3][8], float (&mv)[16]) {
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
  for (int j = 0; j < 16; ++j) mv[j] = m[j];
}

// ---------------------------------------------------------------------------
// Projection of the 32 token rows of MFMA block beta of a staged tile (LDS rows
// of ROWB bytes, bf16 or fp32) onto the group's basis columns: after it, lane
// (h, col) holds coefficients 16h..16h+15 of row 32 beta + col. The operand for
// K step k and part p is PART(p, k) (a bf16x8); both encode paths below issue
// the same MFMAs in the same order, so their results are bit-identical.
// ---------------------------------------------------------------------------
template <bool F32IN, int ROWB, bool SERIAL_K = false, typename PartFn>
__device__ __forceinline__ f32x16 project_block(const uint8_t* __restrict__ xs, int beta, int col, int h, PartFn&& part) {
  f32x16 acc = {};
  const int row = 32 * beta + col;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    if constexpr (!F32IN) {
      const bf16x8 xb8 = as_bf16x8(*reinterpret_cast<const u32x4*>(xs + row * ROWB + (16 * k + 8 * h) * 2));
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

// Center, quantize, pack and store the projected block: writes the group's
// metadata word and payload of the tokens slot0 + 32 beta + col in [t_lo, t_hi).
__device__ __forceinline__ void store_block(const f32x16& acc, const float (&mv)[16], int beta, int col, int h,
                                            int64_t slot0, int64_t t_lo, int64_t t_hi, int64_t sbase, int W, int slot,
                                            int gbits, int gpay, uint32_t* __restrict__ packed) {
  float c[16];
#pragma unroll
  for (int j = 0; j < 16; ++j) c[j] = acc[j] - mv[j];
  const int64_t t = slot0 + 32 * beta + col;
  const bool valid = t >= t_lo && t < t_hi;
  const int64_t base = rec_word(sbase, t, W, 0);
  with_bits(gbits, [&](auto bc) {
    constexpr int B = decltype(bc)::value;
    uint32_t q[16], P[4];
    const uint32_t meta = quantize16<B>(c, q);
    pack16<B>(q, P);
    if (h == 0 && valid) packed[base + (int64_t)slot * TILE] = meta;
    store_payload<B>(packed, base, gpay, P, h, valid);
  });
}

// Encode one block for one kept group, the basis held as split operands.
template <bool F32IN, int ROWB>
__device__ __forceinline__ void encode_block(const uint8_t* __restrict__ xs, int beta, int col, int h,
                                             const bf16x8 (&Va)[3][8], const float (&mv)[16], int64_t slot0,
                                             int64_t t_lo, int64_t t_hi, int64_t sbase, int W, int slot, int gbits,
                                             int gpay, uint32_t* __restrict__ packed) {
  const f32x16 acc = project_block<F32IN, ROWB>(xs, beta, col, h, [&](int p, int k) { return Va[p][k]; });
  store_block(acc, mv, beta, col, h, slot0, t_lo, t_hi, sbase, W, slot, gbits, gpay, packed);
}

// Same, with the basis columns streamed from memory K step by K step (a ring of
// PF steps in flight) and split as they arrive: few registers, for callers that
// encode a single block.
template <bool F32IN, int ROWB, int PF = 4>
__device__ __forceinline__ void encode_block_streamed(const uint8_t* __restrict__ xs, int beta, int col, int h,
                                                      const float* __restrict__ Vs, int grp, const float (&mv)[16],
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
  const f32x16 acc = project_block<F32IN, ROWB, true>(xs, beta, col, h, [&](int p, int k) {
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
  store_block(acc, mv, beta, col, h, slot0, t_lo, t_hi, sbase, W, slot, gbits, gpay, packed);
}

}  // namespace spectra_dev
