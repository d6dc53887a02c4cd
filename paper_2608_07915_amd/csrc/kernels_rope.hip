// Decode-step attention for rotary models (Sec. 3.3, Mode A): the cache holds
// latents of pre-RoPE keys, so each key is reconstructed and then rotated at its
// own position before its dot product with the rotated query; this is what keeps
// Mode A exact under RoPE. Values need no rotation and stay in the latent space:
// their weighted sums run over the kept value coefficients and the chunk combine
// (log-sum-exp merge, + m_V, one inverse rotation) is the latent kernel's.
//
// Two kernels. rope_attn4_kernel (at most eight query heads per KV head, records of at
// most 16 words; described further down) keeps the reconstructed keys in registers.
// rope_attn_kernel serves the wider shapes: one workgroup of eight wavefronts per
// (token chunk, KV head, sequence), 64-token tiles, three workgroup barriers per tile. While tile tt is processed, the record
// words of tile tt + 1 are staged and its key codes unpacked, once for the whole
// workgroup, into a bf16 tile in LDS:
//   1. wavefront w reconstructs key dimensions 16w..16w+15 of the 64 tokens,
//      k = sum_G (s_tG codes_tG + z_tG) V_G^T + m_K V^T, on v_mfma_f32_16x16x32_bf16
//      (one kept group per MFMA; codes are exact in bf16, the basis enters as three
//      bf16 parts whose products are exact in fp32), into LDS;
//   2. each thread rotates eight dimension pairs (i, i + 64) of one token by its
//      in-tile offset t w_i (a 64 x 64 table) and takes their dot products with the
//      queries rotated by (p_q - 64 tt) w_i, an angle reduced in fp64 once per tile;
//      the product is the query at p_q against the key at 64 tt + t, since rotations
//      compose and are orthogonal. The same threads unpack the next tile's key codes;
//   3. online softmax (lane = token), identical in every wavefront; wavefront w adds
//      the softmax-weighted codes of kept value slot w mod 4 over token half w / 4 on
//      v_mfma_f32_16x16x32_bf16 exactly as the latent kernel does, and the last
//      wavefront rotates the queries for the next tile.
#include "attn_common.hpp"
#include "device_common.hpp"
#include "encode_dev.hpp"
#include "kernels.hpp"

namespace spectra_dev {

constexpr int RTT = 64;           // tokens per tile
constexpr int RKROW = RTT + 4;    // floats per reconstructed-key row (dimension x token, 16-byte rows)
constexpr int RCS2 = 2 * 64 + 2;  // floats per row of the interleaved in-tile cos/sin table
constexpr int RCP = 136;          // bf16 per token row of the unpacked key codes (4 kept groups + pad)
constexpr int RWMAX = 32;         // record words per tensor staged for this kernel
constexpr int RWAVES = 8;         // wavefronts per workgroup
constexpr int RTHREADS = 64 * RWAVES;
constexpr int RPP = 64 / RWAVES;  // dimension pairs per thread in the score step

// LDS layout (bytes) for NH query heads per KV head
__host__ __device__ constexpr int rope_off_rv() { return RWMAX * TROW * 4; }
__host__ __device__ constexpr int rope_off_codes() { return 2 * RWMAX * TROW * 4; }
__host__ __device__ constexpr int rope_off_kmeta() { return rope_off_codes() + RTT * RCP * 2; }
__host__ __device__ constexpr int rope_off_kh() { return rope_off_kmeta() + NG * RTT * 2 * 4; }
__host__ __device__ constexpr int rope_off_tcs() { return rope_off_kh() + D * RKROW * 4; }
__host__ __device__ constexpr int rope_off_qs(int) { return rope_off_tcs() + RTT * RCS2 * 4; }
__host__ __device__ constexpr int rope_off_qpp(int nh) { return rope_off_qs(nh) + nh * D * 4; }
__host__ __device__ constexpr int rope_off_red(int nh) { return rope_off_qpp(nh) + 64 * nh * 2 * 4; }
__host__ __device__ constexpr int rope_off_wt(int nh) { return rope_off_red(nh) + RWAVES * nh * RTT * 4; }
__host__ __device__ constexpr int rope_lds_bytes(int nh) { return rope_off_wt(nh) + RWAVES * 2 * nh * WROW * 2; }
static_assert(rope_off_kmeta() % 16 == 0 && rope_off_kh() % 16 == 0 && rope_off_qpp(4) % 16 == 0, "16-byte reads");
static_assert(rope_off_wt(4) % 16 == 0 && (WROW * 2) % 16 == 0, "weight rows are read 16 bytes at a time");
static_assert(2 * (2 * 4) * AROW * 4 <= D * RKROW * 4, "value sums of both token halves reuse the key rows");
static_assert(rope_lds_bytes(4) <= 160 * 1024 && rope_lds_bytes(8) <= 160 * 1024, "LDS of one CU");
static_assert(rope_off_qpp(8) % 16 == 0 && rope_off_wt(8) % 16 == 0, "16-byte reads");

// cos and sin of an angle given exactly in fp64 (a position below 2^28 times an
// fp32 frequency needs at most 52 significant bits). Cody-Waite reduction by pi/2
// (two-term split, fused multiply-adds), then the Taylor series of sin and cos on
// [-pi/4, pi/4] to degree 15 and 16 (truncation below 2e-17) in fp64, then the
// quadrant's signs and swap; the results are rounded to fp32.
__device__ __forceinline__ void sincos_reduced(double ang, float* c, float* s) {
  constexpr double PIO2_HI = 1.5707963267948966;     // pi/2 rounded to fp64
  constexpr double PIO2_LO = 6.123233995736766e-17;  // pi/2 - PIO2_HI
  constexpr double TWO_OVER_PI = 0.6366197723675814;
  const double k = __builtin_rint(ang * TWO_OVER_PI);
  double y = __builtin_fma(-k, PIO2_HI, ang);
  y = __builtin_fma(-k, PIO2_LO, y);
  const double y2 = y * y;
  // 1/n! for n = 2..16
  double sp = 1.0 / 1307674368000.0;                         // 1/15!
  sp = __builtin_fma(sp, -y2, 1.0 / 6227020800.0);           // 1/13!
  sp = __builtin_fma(sp, -y2, 1.0 / 39916800.0);             // 1/11!
  sp = __builtin_fma(sp, -y2, 1.0 / 362880.0);               // 1/9!
  sp = __builtin_fma(sp, -y2, 1.0 / 5040.0);                 // 1/7!
  sp = __builtin_fma(sp, -y2, 1.0 / 120.0);                  // 1/5!
  sp = __builtin_fma(sp, -y2, 1.0 / 6.0);                    // 1/3!
  sp = __builtin_fma(sp, -y2, 1.0);
  const double sy = sp * y;                                  // y - y^3/3! + ... - y^15/15!
  double cp = 1.0 / 20922789888000.0;                        // 1/16!
  cp = __builtin_fma(cp, -y2, 1.0 / 87178291200.0);          // 1/14!
  cp = __builtin_fma(cp, -y2, 1.0 / 479001600.0);            // 1/12!
  cp = __builtin_fma(cp, -y2, 1.0 / 3628800.0);              // 1/10!
  cp = __builtin_fma(cp, -y2, 1.0 / 40320.0);                // 1/8!
  cp = __builtin_fma(cp, -y2, 1.0 / 720.0);                  // 1/6!
  cp = __builtin_fma(cp, -y2, 1.0 / 24.0);                   // 1/4!
  cp = __builtin_fma(cp, -y2, 0.5);                          // 1/2!
  const double cy = __builtin_fma(cp, -y2, 1.0);             // 1 - y^2/2! + ... + y^16/16!
  const int q = (int)((int64_t)k & 3);
  const double sv = (q == 0) ? sy : (q == 1) ? cy : (q == 2) ? -sy : -cy;
  const double cv = (q == 0) ? cy : (q == 1) ? -sy : (q == 2) ? -cy : sy;
  *s = (float)sv;
  *c = (float)cv;
}

template <int NQ>
__global__ __launch_bounds__(RTHREADS, 1) void rope_attn_kernel(AttnArgs a) {
  constexpr int NH = 4 * NQ;
  static_assert(2 * NH <= 16, "stacked hi/lo weight rows");
  extern __shared__ __attribute__((aligned(16))) uint8_t rsm[];
  uint32_t* recK = reinterpret_cast<uint32_t*>(rsm);
  uint32_t* recV = reinterpret_cast<uint32_t*>(rsm + rope_off_rv());
  uint16_t* codes = reinterpret_cast<uint16_t*>(rsm + rope_off_codes());
  float* kmeta = reinterpret_cast<float*>(rsm + rope_off_kmeta());
  float* khat = reinterpret_cast<float*>(rsm + rope_off_kh());
  float* tcs = reinterpret_cast<float*>(rsm + rope_off_tcs());
  float* qs = reinterpret_cast<float*>(rsm + rope_off_qs(NH));
  float* qpp = reinterpret_cast<float*>(rsm + rope_off_qpp(NH));
  float* red = reinterpret_cast<float*>(rsm + rope_off_red(NH));
  __shared__ float mst[NH], lst[NH], zst[NH][NG];

  const int chunk = blockIdx.x, kv = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar slot and role selection
  const int s = b * a.n_kv_heads + kv;
  const int nqh = a.n_qh;
  const int Wk = a.Wk, Wv = a.Wv;
  const Kept Kk = read_kept(a.bits_k + (int64_t)s * NG);
  const Kept Kv = read_kept(a.bits_v + (int64_t)s * NG);
  const bool ok = Kk.ok && Kv.ok && Kk.used <= Wk && Kv.used <= Wv;
  const int64_t n_tiles = (a.n_tokens + 63) >> 6;
  const int64_t tile_begin = (int64_t)chunk * a.tiles_per_chunk;
  const int64_t tile_end = tile_begin + a.tiles_per_chunk < n_tiles ? tile_begin + a.tiles_per_chunk : n_tiles;

  // ---- prologue: in-tile rotation table, scaled queries, key-basis operands ----
  for (int e = tid; e < RTT * 64; e += RTHREADS) {
    const int r = e >> 6, i = e & 63;
    float c, sn;
    sincos_reduced((double)r * (double)a.inv_freq[i], &c, &sn);
    tcs[r * RCS2 + 2 * i] = c;
    tcs[r * RCS2 + 2 * i + 1] = sn;
  }
  for (int e = tid; e < NH * 64; e += RTHREADS) {
    const int h = e >> 6, i = e & 63;
    float q0 = 0.0f, q1 = 0.0f;
    if (h < nqh) {
      const int64_t qi = ((int64_t)b * a.n_q_heads + kv * nqh + h) * D + i;
      q0 = a.q_f32 ? reinterpret_cast<const float*>(a.q)[qi] : bf2f(reinterpret_cast<const uint16_t*>(a.q)[qi]);
      q1 = a.q_f32 ? reinterpret_cast<const float*>(a.q)[qi + 64] : bf2f(reinterpret_cast<const uint16_t*>(a.q)[qi + 64]);
    }
    qs[h * D + i] = q0 * a.scale_log2;
    qs[h * D + 64 + i] = q1 * a.scale_log2;
  }
  // Key reconstruction operands of this lane (16x16x32 layout): output dimension
  // ch = 16 wave + (lane & 15), in-group coefficients 8 kg .. 8 kg + 7 (kg = lane >> 4)
  // of each kept key slot, as three bf16 parts.
  const int kg = lane >> 4;
  const int ch = 16 * wave + (lane & 15);
  const float* Vk = a.basis_k + (int64_t)s * D * D;
  bf16x8 Vb[NG][3];
  float vsum[NG];
#pragma unroll
  for (int sl = 0; sl < NG; ++sl) {
    vsum[sl] = 0.0f;
    if (sl < Kk.n) {
      const float* vr = Vk + (int64_t)ch * D + G * Kk.grp[sl];
      uint32_t p0[8], p1[8], p2[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) split3(vr[8 * kg + i], p0[i], p1[i], p2[i]);
      Vb[sl][0] = as_bf16x8(u32x4{pack2(p0[0], p0[1]), pack2(p0[2], p0[3]), pack2(p0[4], p0[5]), pack2(p0[6], p0[7])});
      Vb[sl][1] = as_bf16x8(u32x4{pack2(p1[0], p1[1]), pack2(p1[2], p1[3]), pack2(p1[4], p1[5]), pack2(p1[6], p1[7])});
      Vb[sl][2] = as_bf16x8(u32x4{pack2(p2[0], p2[1]), pack2(p2[2], p2[3]), pack2(p2[4], p2[5]), pack2(p2[6], p2[7])});
      float acc = 0.0f;
      for (int j = 0; j < G; ++j) acc += vr[j];
      vsum[sl] = acc;
    } else {
#pragma unroll
      for (int p = 0; p < 3; ++p) Vb[sl][p] = bf16x8{};
    }
  }
  float bias = 0.0f;  // (m_K V^T)_ch
  {
    const float* ms = a.mean_k + (int64_t)s * D;
    const float* vr = Vk + (int64_t)ch * D;
    for (int j = 0; j < D; ++j) bias = __builtin_fmaf(ms[j], vr[j], bias);
  }

  // value path of this wavefront: kept value slot wave mod 4 over tokens 32 (wave / 4) ..
  const int vsl = wave & 3, vhalf = wave >> 2;
  const bool vslot = vsl < Kv.n;
  const int vB = vslot ? pick4(Kv.bits, vsl) : 0, vpay = vslot ? pick4(Kv.pay, vsl) : 0;
  const int vgrp = vslot ? pick4(Kv.grp, vsl) : 0;
  const int col16 = lane & 15, kq = lane >> 4;
  const int voff = 2 * col16 * vB;
  uint16_t* ws = reinterpret_cast<uint16_t*>(rsm + rope_off_wt(NH)) + wave * (2 * NH * WROW);

  float m_run[NH], l_run[NH], zacc[NH];
#pragma unroll
  for (int h = 0; h < NH; ++h) {
    m_run[h] = -__builtin_inff();
    l_run[h] = 0.0f;
    zacc[h] = 0.0f;
  }
  f32x4 vacc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};

  // record words of one tile (64 W contiguous words per tensor), two per thread
  const uint32_t* kps = a.packed_k + (int64_t)s * a.t_cap * Wk;
  const uint32_t* vps = a.packed_v + (int64_t)s * a.t_cap * Wv;
  constexpr int PFR = 64 * RWMAX / RTHREADS;
  uint32_t pk[PFR], pv[PFR];
  auto load_k = [&](int64_t tt) {
#pragma unroll
    for (int i = 0; i < PFR; ++i) {
      const int k = tid + RTHREADS * i;
      pk[i] = k < 64 * Wk ? kps[tt * 64 * Wk + k] : 0u;
    }
  };
  auto load_v = [&](int64_t tt) {
#pragma unroll
    for (int i = 0; i < PFR; ++i) {
      const int k = tid + RTHREADS * i;
      pv[i] = k < 64 * Wv ? vps[tt * 64 * Wv + k] : 0u;
    }
  };
  auto stage_k = [&]() {
#pragma unroll
    for (int i = 0; i < PFR; ++i) {
      const int k = tid + RTHREADS * i;
      if (k < 64 * Wk) recK[(k >> 6) * TROW + (k & 63)] = pk[i];
    }
  };
  // codes of the staged key words as bf16 [token][slot * 32 + coefficient] and the
  // per-token scale and zero point [slot][token]: thread (token lane, eight
  // coefficients of one slot); the slot is uniform in a wavefront
  auto unpack_k = [&]() {
#pragma unroll
    for (int r = 0; r < (NG * 4 * 64) / RTHREADS; ++r) {
      const int g8 = wave + RWAVES * r, sl = g8 >> 2, k8 = g8 & 3;
      if (sl < Kk.n) {
        const int pay = pick4(Kk.pay, sl);
        const uint32_t* rt = recK + lane;
        with_bits(pick4(Kk.bits, sl), [&](auto bc) {
          constexpr int B = decltype(bc)::value;
          uint32_t cd[8];
          extract8<B>([&](int i) { return rt[(pay + i) * TROW]; }, 8 * k8, cd);
          *reinterpret_cast<u32x4*>(codes + lane * RCP + sl * G + 8 * k8) =
              u32x4{int_to_bf16_pair(cd[0], cd[1]), int_to_bf16_pair(cd[2], cd[3]), int_to_bf16_pair(cd[4], cd[5]),
                    int_to_bf16_pair(cd[6], cd[7])};
        });
        if (k8 == 0) {
          const uint32_t m = rt[sl * TROW];
          *reinterpret_cast<f32x2*>(kmeta + 2 * (sl * RTT + lane)) = f32x2{h2f(m), h2f(m >> 16)};
        }
      }
    }
  };
  // queries rotated by (p_q - 64 tt) w_i for tile tt, [pair i][head][2] (lane = pair)
  auto rotate_queries = [&](int64_t tt) {
    float c, sn;
    sincos_reduced((double)(a.q_pos - tt * 64) * (double)a.inv_freq[lane], &c, &sn);
#pragma unroll
    for (int h = 0; h < NH; h += 2) {
      const float a0 = qs[h * D + lane], a1 = qs[h * D + 64 + lane];
      const float b0 = qs[(h + 1) * D + lane], b1 = qs[(h + 1) * D + 64 + lane];
      *reinterpret_cast<f32x4*>(qpp + (lane * NH + h) * 2) =
          f32x4{a0 * c - a1 * sn, a1 * c + a0 * sn, b0 * c - b1 * sn, b1 * c + b0 * sn};
    }
  };
  if (ok && tile_begin < tile_end) {
    load_k(tile_begin);
    stage_k();
    __syncthreads();  // staged words, the query and table writes visible
    unpack_k();
    if (wave == RWAVES - 1) rotate_queries(tile_begin);
    if (tile_begin + 1 < tile_end) load_k(tile_begin + 1);
    load_v(tile_begin);
  }

  for (int64_t tt = tile_begin; ok && tt < tile_end; ++tt) {
    __syncthreads();  // the previous tile's LDS reads done; this tile's codes and rotated queries visible
    if (tt + 1 < tile_end) stage_k();
#pragma unroll
    for (int i = 0; i < PFR; ++i) {
      const int k = tid + RTHREADS * i;
      if (k < 64 * Wv) recV[(k >> 6) * TROW + (k & 63)] = pv[i];
    }
    if (tt + 2 < tile_end) load_k(tt + 2);
    if (tt + 1 < tile_end) load_v(tt + 1);
    // keep the loop-invariant LDS operands (rotation table) as LDS reads inside
    // the loop rather than registers held across it
    asm volatile("" ::: "memory");

    // ---- 1. key dimension ch of the 64 tokens: four 16-token MFMA blocks, two at a time ----
#pragma unroll
    for (int pass = 0; pass < 2; ++pass) {
      const int tok0 = 32 * pass;
      float out[2][4];
#pragma unroll
      for (int blk = 0; blk < 2; ++blk)
#pragma unroll
        for (int j = 0; j < 4; ++j) out[blk][j] = bias;
#pragma unroll
      for (int sl = 0; sl < NG; ++sl) {
        if (sl < Kk.n) {
          const bf16x8 A0 = as_bf16x8(*reinterpret_cast<const u32x4*>(codes + (tok0 + (lane & 15)) * RCP + sl * G + 8 * kg));
          const bf16x8 A1 =
              as_bf16x8(*reinterpret_cast<const u32x4*>(codes + (tok0 + 16 + (lane & 15)) * RCP + sl * G + 8 * kg));
          f32x4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int part = 0; part < 3; ++part) {
            acc0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A0, Vb[sl][part], acc0, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A1, Vb[sl][part], acc1, 0, 0, 0);
          }
          // acc_b[j]: token tok0 + 16 b + 4 kg + j of the tile, dimension ch
          const float* mt0 = kmeta + 2 * (sl * RTT + tok0 + 4 * kg);
          const f32x4 m00 = *reinterpret_cast<const f32x4*>(mt0), m01 = *reinterpret_cast<const f32x4*>(mt0 + 4);
          const f32x4 m10 = *reinterpret_cast<const f32x4*>(mt0 + 32), m11 = *reinterpret_cast<const f32x4*>(mt0 + 36);
          out[0][0] += m00[0] * acc0[0] + m00[1] * vsum[sl];
          out[0][1] += m00[2] * acc0[1] + m00[3] * vsum[sl];
          out[0][2] += m01[0] * acc0[2] + m01[1] * vsum[sl];
          out[0][3] += m01[2] * acc0[3] + m01[3] * vsum[sl];
          out[1][0] += m10[0] * acc1[0] + m10[1] * vsum[sl];
          out[1][1] += m10[2] * acc1[1] + m10[3] * vsum[sl];
          out[1][2] += m11[0] * acc1[2] + m11[1] * vsum[sl];
          out[1][3] += m11[2] * acc1[3] + m11[3] * vsum[sl];
        }
      }
#pragma unroll
      for (int blk = 0; blk < 2; ++blk)
        *reinterpret_cast<f32x4*>(khat + ch * RKROW + tok0 + 16 * blk + 4 * kg) =
            f32x4{out[blk][0], out[blk][1], out[blk][2], out[blk][3]};
    }
    __syncthreads();

    // ---- 2. in-tile rotation and the dot products with the tile's rotated queries:
    // thread (token lane, pairs RPP wave ..); then the next tile's key codes ----
    {
      const int t = lane;
      float sc[NH];
#pragma unroll
      for (int h = 0; h < NH; ++h) sc[h] = 0.0f;
#pragma unroll 4
      for (int ii = 0; ii < RPP; ++ii) {
        const int i = RPP * wave + ii;
        const float x0 = khat[i * RKROW + t], x1 = khat[(i + 64) * RKROW + t];
        const f32x2 cs = *reinterpret_cast<const f32x2*>(tcs + t * RCS2 + 2 * i);
        const float r0 = x0 * cs[0] - x1 * cs[1], r1 = x1 * cs[0] + x0 * cs[1];
#pragma unroll
        for (int h = 0; h < NH; h += 2) {
          const f32x4 qv = *reinterpret_cast<const f32x4*>(qpp + (i * NH + h) * 2);
          sc[h] = __builtin_fmaf(qv[0], r0, __builtin_fmaf(qv[1], r1, sc[h]));
          sc[h + 1] = __builtin_fmaf(qv[2], r0, __builtin_fmaf(qv[3], r1, sc[h + 1]));
        }
      }
#pragma unroll
      for (int h = 0; h < NH; ++h) red[(wave * NH + h) * RTT + t] = sc[h];
    }
    if (tt + 1 < tile_end) unpack_k();
    __syncthreads();
    // the next tile's rotated queries, by the last wavefront
    if (wave == RWAVES - 1 && tt + 1 < tile_end) rotate_queries(tt + 1);

    // ---- 3. online softmax over the tile (lane = token) and value sums ----
    const bool valid = tt * 64 + lane < a.n_tokens;
    float x[NH];
    bool over = false;
#pragma unroll
    for (int h = 0; h < NH; ++h) {
      float acc = 0.0f;
#pragma unroll
      for (int w = 0; w < RWAVES; ++w) acc += red[(w * NH + h) * RTT + lane];
      x[h] = (valid && h < nqh) ? acc : -__builtin_inff();
      over = over || x[h] > m_run[h] + RESCALE_SLACK;
    }
    if (__any(over)) {
#pragma unroll
      for (int h = 0; h < NH; ++h) {
        if (__any(x[h] > m_run[h] + RESCALE_SLACK)) {
          const float mn = __builtin_fmaxf(m_run[h], wave_max_all(x[h]));
          const float alpha = (m_run[h] == -__builtin_inff()) ? 0.0f : __builtin_amdgcn_exp2f(m_run[h] - mn);
          l_run[h] *= alpha;
          zacc[h] *= alpha;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int row = 4 * kq + j;
            const float f = (row == h || row == NH + h) ? alpha : 1.0f;
            vacc[0][j] *= f;
            vacc[1][j] *= f;
          }
          m_run[h] = mn;
        }
      }
    }
    float p[NH];
#pragma unroll
    for (int h = 0; h < NH; ++h) {
      p[h] = x[h] != -__builtin_inff() ? __builtin_amdgcn_exp2f(x[h] - m_run[h]) : 0.0f;
      l_run[h] += p[h];
    }
    if (vslot) {
      const uint32_t meta = valid ? recV[vsl * TROW + lane] : 0u;
      const float sv = h2f(meta), zv = h2f(meta >> 16);
#pragma unroll
      for (int h = 0; h < NH; h += 2) {  // two heads per packed conversion
        if (vhalf == 0) {  // zero-point sums over the whole tile once per slot
          zacc[h] = __builtin_fmaf(p[h], zv, zacc[h]);
          zacc[h + 1] = __builtin_fmaf(p[h + 1], zv, zacc[h + 1]);
        }
        const float w0 = p[h] * sv, w1 = p[h + 1] * sv;
        const uint32_t hb2 = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{w0, w1}, bf16x2));
        const float h0 = __builtin_bit_cast(float, hb2 << 16), h1 = __builtin_bit_cast(float, hb2 & 0xFFFF0000u);
        const uint32_t lb = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{w0 - h0, w1 - h1}, bf16x2));
        ws[h * WROW + lane] = (uint16_t)hb2;
        ws[(h + 1) * WROW + lane] = (uint16_t)(hb2 >> 16);
        ws[(NH + h) * WROW + lane] = (uint16_t)lb;
        ws[(NH + h + 1) * WROW + lane] = (uint16_t)(lb >> 16);
      }
      __builtin_amdgcn_wave_barrier();
      // rows 0..NH-1: hi weights of the heads, NH..2NH-1: lo; MFMA rows past them
      // re-read a weight row and are never read back
      const int arow = col16 < 2 * NH ? col16 : col16 - 2 * NH;
      const bf16x8 negone = as_bf16x8(u32x4{0xBF80BF80u, 0xBF80BF80u, 0xBF80BF80u, 0xBF80BF80u});
      uint32_t vmagic = 0x3F803F80u;  // exponent of 1.0 in both halves (see value_codes2)
      asm volatile("" : "+v"(vmagic));
      const int tok0 = 32 * vhalf + 8 * kq;
      auto body = [&](auto cls) {
        constexpr int CLS = decltype(cls)::value;
        const bf16x8 aw = as_bf16x8(*reinterpret_cast<const u32x4*>(ws + arow * WROW + tok0));
        u32x4 vc[2];
        value_codes2<CLS>(recV, vpay, Kv.used, vB, voff, tok0, vmagic, vc[0], vc[1]);
#pragma unroll
        for (int c2 = 0; c2 < 2; ++c2) {
          f32x4 acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aw, as_bf16x8(vc[c2]), vacc[c2], 0, 0, 0);
          if constexpr (CLS != 2) acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aw, negone, acc, 0, 0, 0);
          vacc[c2] = acc;
        }
      };
      if (vB == 8)
        body(std::integral_constant<int, 2>{});
      else if (vB == 1 || vB == 2 || vB == 4)
        body(std::integral_constant<int, 0>{});
      else
        body(std::integral_constant<int, 1>{});
      __builtin_amdgcn_wave_barrier();
    }
  }

  // ---- chunk partial: m, l and the zero-point sums per head, value sums per coefficient ----
#pragma unroll
  for (int h = 0; h < NH; ++h) {
    const float l = wave_sum_lane63(l_run[h]);
    const float z = wave_sum_lane63(zacc[h]);
    if (wave == 0 && lane == 63) {
      mst[h] = ok ? m_run[h] : -__builtin_inff();
      lst[h] = l;
#pragma unroll
      for (int g = 0; g < NG; ++g) zst[h][g] = 0.0f;
    }
    __syncthreads();
    if (vslot && vhalf == 0 && lane == 63) zst[h][vgrp] = z;
  }
  __syncthreads();  // all tile buffers are free: the key rows hold the value sums of both token halves now
  float* accw = khat + vhalf * (2 * NH * AROW);
  if (vslot) {
    // codes below 8 bits entered as 1 + c 2^-b (see value_codes2)
    const float vscale = vB < 8 ? (float)(1u << vB) : 1.0f;
#pragma unroll
    for (int c2 = 0; c2 < 2; ++c2)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int row = 4 * kq + j;
        if (row < 2 * NH) accw[row * AROW + G * vgrp + 2 * col16 + c2] = vacc[c2][j] * vscale;
      }
  }
  uint32_t kept_groups = 0u;
#pragma unroll
  for (int sl = 0; sl < NG; ++sl)
    if (sl < Kv.n) kept_groups |= 1u << pick4(Kv.grp, sl);
  __syncthreads();
  const float* acc_lo = khat;
  const float* acc_hi = khat + 2 * NH * AROW;
  float* part = a.partial + ((int64_t)b * a.n_q_heads + kv * nqh) * a.n_chunks * PART + (int64_t)chunk * PART;
  for (int e = tid; e < nqh * D; e += RTHREADS) {
    const int h = e >> 7, j = e & 127;
    const bool kept = ok && ((kept_groups >> (j >> 5)) & 1u);
    float* ph = part + (int64_t)h * a.n_chunks * PART;
    ph[8 + j] = kept ? (acc_lo[h * AROW + j] + acc_lo[(NH + h) * AROW + j]) +
                           (acc_hi[h * AROW + j] + acc_hi[(NH + h) * AROW + j])
                     : 0.0f;
    if (j == 0) {
      ph[0] = mst[h];
      ph[1] = lst[h];
    }
    if (j < NG) ph[2 + j] = zst[h][j];
  }
}

// ---------------------------------------------------------------------------
// Four-wavefront form (at most eight query heads per KV head, records of at most 16
// words): two workgroups per CU, two workgroup barriers per tile, the reconstructed
// keys never leave the registers.
//   1. wavefront w reconstructs dimensions 16w..16w+15 and 64+16w..64+16w+15 of the
//      tile's 64 tokens on v_mfma_f32_32x32x16_bf16 (rows m and m + 16 of its 32-row
//      output are the pair (i, i + 64) with i = 16w + m, so a lane holds both
//      members of eight pairs of one token), rotates them by the token's in-tile
//      offset r (cos and sin of r w_i from a table), dots them with the tile's
//      rotated queries and leaves its partial scores in LDS;
//      it also stages the next tile's key words and this tile's value words;
//   2. online softmax (lane = token) in every wavefront; wavefront w adds the
//      softmax-weighted codes of kept value slot w over the whole tile; the next tile's
//      key codes are unpacked and its queries rotated.
// ---------------------------------------------------------------------------
constexpr int R4W = 16;  // record words per tensor
constexpr int R4T = 256;  // threads
// In-tile rotation table: with four heads one row of (cos, sin) of r w_i per in-tile
// offset r (64 rows); with eight heads (whose query buffers take the room) two tables of
// eight rows, b w_i and 8a w_i, composed per use (r = 8a + b). Rows hold 64 frequencies
// + a pad, so the rows of the 32 tokens of one read start on distinct banks.
constexpr int R4TP = 65;
__host__ __device__ constexpr int r4_tab_rows(int nh) { return nh <= 4 ? 64 : 16; }
__host__ __device__ constexpr int r4_off_reck() { return 0; }                                   // [R4W][TROW] u32
__host__ __device__ constexpr int r4_off_recv() { return R4W * TROW * 4; }                      // [R4W][TROW] u32
__host__ __device__ constexpr int r4_off_codes() { return 2 * R4W * TROW * 4; }                 // [64][RCP] bf16
__host__ __device__ constexpr int r4_off_kmeta() { return r4_off_codes() + RTT * RCP * 2; }     // [NG][64] (s, z)
__host__ __device__ constexpr int r4_off_tab() { return r4_off_kmeta() + NG * RTT * 8; }       // [rows][R4TP] (cos, sin)
__host__ __device__ constexpr int r4_off_vsum(int nh) { return r4_off_tab() + r4_tab_rows(nh) * R4TP * 8; }  // [NG + 1][128]
__host__ __device__ constexpr int r4_off_qs(int nh) { return r4_off_vsum(nh) + (NG + 1) * D * 4; }          // [nh][128]
__host__ __device__ constexpr int r4_off_qpp(int nh) { return r4_off_qs(nh) + nh * D * 4; }                 // [64][nh][2]
__host__ __device__ constexpr int r4_off_red(int nh) { return r4_off_qpp(nh) + 64 * nh * 2 * 4; }           // [4][nh][64]
__host__ __device__ constexpr int r4_off_wt(int nh) { return r4_off_red(nh) + 4 * nh * 64 * 4; }            // [4][2nh][WROW]
__host__ __device__ constexpr int r4_lds_bytes(int nh) { return r4_off_wt(nh) + 4 * 2 * nh * WROW * 2; }
static_assert(r4_off_codes() % 16 == 0 && r4_off_kmeta() % 16 == 0 && r4_off_tab() % 16 == 0, "16-byte reads");
static_assert(r4_off_vsum(4) % 16 == 0 && r4_off_qpp(4) % 16 == 0 && r4_off_wt(4) % 16 == 0, "16-byte reads");
static_assert(r4_off_vsum(8) % 16 == 0 && r4_off_qpp(8) % 16 == 0 && r4_off_wt(8) % 16 == 0, "16-byte reads");
static_assert(2 * r4_lds_bytes(4) <= 160 * 1024 && 2 * r4_lds_bytes(8) <= 160 * 1024, "two workgroups per CU");
static_assert(16 * AROW * 4 <= RTT * RCP * 2, "the value sums of the merge fit the code rows");

template <int NQ>
__global__ __launch_bounds__(R4T, 2) void rope_attn4_kernel(AttnArgs a) {
  constexpr int NH = 4 * NQ;
  constexpr bool FULL_TAB = NH <= 4;
  extern __shared__ __attribute__((aligned(16))) uint8_t rsm[];
  uint32_t* recK = reinterpret_cast<uint32_t*>(rsm + r4_off_reck());
  uint32_t* recV = reinterpret_cast<uint32_t*>(rsm + r4_off_recv());
  uint16_t* codes = reinterpret_cast<uint16_t*>(rsm + r4_off_codes());
  f32x2* kmeta = reinterpret_cast<f32x2*>(rsm + r4_off_kmeta());
  f32x2* tab = reinterpret_cast<f32x2*>(rsm + r4_off_tab());
  float* vsum = reinterpret_cast<float*>(rsm + r4_off_vsum(NH));  // [sl][dim], row NG: m V^T
  float* qs = reinterpret_cast<float*>(rsm + r4_off_qs(NH));
  float* qpp = reinterpret_cast<float*>(rsm + r4_off_qpp(NH));
  float* red = reinterpret_cast<float*>(rsm + r4_off_red(NH));
  __shared__ float lst[NH], zst[NH][NG];

  const int chunk = blockIdx.x, kv = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = lane >> 5, c32 = lane & 31;
  const int s = b * a.n_kv_heads + kv;
  const int nqh = a.n_qh;
  const int Wk = a.Wk, Wv = a.Wv;
  const Kept Kk = read_kept(a.bits_k + (int64_t)s * NG);
  const Kept Kv = read_kept(a.bits_v + (int64_t)s * NG);
  const bool ok = Kk.ok && Kv.ok && Kk.used <= Wk && Kv.used <= Wv;
  const int64_t n_tiles = (a.n_tokens + 63) >> 6;
  const int64_t tile_begin = (int64_t)chunk * a.tiles_per_chunk;
  const int64_t tile_end = tile_begin + a.tiles_per_chunk < n_tiles ? tile_begin + a.tiles_per_chunk : n_tiles;
  const float* Vk = a.basis_k + (int64_t)s * D * D;

  // ---- prologue: in-tile rotation table(s), scaled queries, group sums and m V^T of the key basis ----
  for (int e = tid; e < r4_tab_rows(NH) * 64; e += R4T) {
    const int r = e >> 6, i = e & 63;
    const int off = FULL_TAB ? r : (r < 8 ? r : 8 * (r - 8));  // rows 0..7: b w_i, rows 8..15: 8a w_i
    float c, sn;
    sincos_reduced((double)off * (double)a.inv_freq[i], &c, &sn);
    tab[r * R4TP + i] = f32x2{c, sn};
  }
  for (int e = tid; e < NH * 64; e += R4T) {
    const int hh = e >> 6, i = e & 63;
    float q0 = 0.0f, q1 = 0.0f;
    if (hh < nqh) {
      const int64_t qi = ((int64_t)b * a.n_q_heads + kv * nqh + hh) * D + i;
      q0 = a.q_f32 ? reinterpret_cast<const float*>(a.q)[qi] : bf2f(reinterpret_cast<const uint16_t*>(a.q)[qi]);
      q1 = a.q_f32 ? reinterpret_cast<const float*>(a.q)[qi + 64] : bf2f(reinterpret_cast<const uint16_t*>(a.q)[qi + 64]);
    }
    qs[hh * D + i] = q0 * a.scale_log2;
    qs[hh * D + 64 + i] = q1 * a.scale_log2;
  }
  if (tid < D) {
    const float* vr = Vk + (int64_t)tid * D;
    const float* ms = a.mean_k + (int64_t)s * D;
    float bias = 0.0f;
    for (int j = 0; j < D; ++j) bias = __builtin_fmaf(ms[j], vr[j], bias);
    vsum[NG * D + tid] = bias;
#pragma unroll
    for (int sl = 0; sl < NG; ++sl) {
      float acc = 0.0f;
      if (sl < Kk.n)
        for (int j = 0; j < G; ++j) acc += vr[G * pick4(Kk.grp, sl) + j];
      vsum[sl * D + tid] = acc;
    }
  }
  // reconstruction operands of this lane (32x32x16 layout): row m = lane % 32 is
  // dimension 16 wave + m (m < 16) or 48 + 16 wave + m (m >= 16); K = in-group
  // coefficients 16 ks + 8 h .. + 7 of each kept key slot, as three bf16 parts
  const int dimA = c32 < 16 ? 16 * wave + c32 : 48 + 16 * wave + c32;
  bf16x8 Va[NG][2][3];
#pragma unroll
  for (int sl = 0; sl < NG; ++sl) {
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      if (sl < Kk.n) {
        const float* vr = Vk + (int64_t)dimA * D + G * pick4(Kk.grp, sl) + 16 * ks + 8 * h;
        uint32_t p0[8], p1[8], p2[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) split3(vr[i], p0[i], p1[i], p2[i]);
        Va[sl][ks][0] = as_bf16x8(u32x4{pack2(p0[0], p0[1]), pack2(p0[2], p0[3]), pack2(p0[4], p0[5]), pack2(p0[6], p0[7])});
        Va[sl][ks][1] = as_bf16x8(u32x4{pack2(p1[0], p1[1]), pack2(p1[2], p1[3]), pack2(p1[4], p1[5]), pack2(p1[6], p1[7])});
        Va[sl][ks][2] = as_bf16x8(u32x4{pack2(p2[0], p2[1]), pack2(p2[2], p2[3]), pack2(p2[4], p2[5]), pack2(p2[6], p2[7])});
      } else {
#pragma unroll
        for (int p = 0; p < 3; ++p) Va[sl][ks][p] = bf16x8{};
      }
    }
  }

  // value path of this wavefront: kept value slot `wave` over the whole tile
  const bool vslot = wave < Kv.n;
  const int vB = vslot ? pick4(Kv.bits, wave) : 0, vpay = vslot ? pick4(Kv.pay, wave) : 0;
  const int vgrp = vslot ? pick4(Kv.grp, wave) : 0;
  const int col16 = lane & 15, kq = lane >> 4;
  const int voff = 2 * col16 * vB;
  uint16_t* ws = reinterpret_cast<uint16_t*>(rsm + r4_off_wt(NH)) + wave * (2 * NH * WROW);

  float m_run[NH], l_run[NH], zacc[NH];
#pragma unroll
  for (int hh = 0; hh < NH; ++hh) {
    m_run[hh] = -__builtin_inff();
    l_run[hh] = 0.0f;
    zacc[hh] = 0.0f;
  }
  f32x4 vacc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};

  // record words of one tile, a quarter per thread and tensor: word w of token t is
  // element 64 w + t of the tile (tid + 256 i)
  const uint32_t* kps = a.packed_k + (int64_t)s * a.t_cap * Wk;
  const uint32_t* vps = a.packed_v + (int64_t)s * a.t_cap * Wv;
  constexpr int PF = 64 * R4W / R4T;
  uint32_t pk[PF], pv[PF];
  auto load_k = [&](int64_t tt) {
#pragma unroll
    for (int i = 0; i < PF; ++i) {
      const int k = tid + R4T * i;
      pk[i] = k < 64 * Wk ? kps[tt * 64 * Wk + k] : 0u;
    }
  };
  auto load_v = [&](int64_t tt) {
#pragma unroll
    for (int i = 0; i < PF; ++i) {
      const int k = tid + R4T * i;
      pv[i] = k < 64 * Wv ? vps[tt * 64 * Wv + k] : 0u;
    }
  };
  auto stage = [&](uint32_t* rec, const uint32_t (&pr)[PF], int W) {
#pragma unroll
    for (int i = 0; i < PF; ++i) {
      const int k = tid + R4T * i;
      if (k < 64 * W) rec[(k >> 6) * TROW + (k & 63)] = pr[i];
    }
  };
  // codes of the staged key words as bf16 [token][slot * 32 + coefficient] and each
  // token's scale and zero point [slot][token]: thread (token lane, eight coefficients
  // of one slot); slot and coefficient octet uniform in a wavefront
  auto unpack_k = [&]() {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int sl = r, k8 = wave;
      if (sl < Kk.n) {
        const int pay = pick4(Kk.pay, sl);
        const uint32_t* rt = recK + lane;
        with_bits(pick4(Kk.bits, sl), [&](auto bc) {
          constexpr int B = decltype(bc)::value;
          uint32_t cd[8];
          extract8<B>([&](int i) { return rt[(pay + i) * TROW]; }, 8 * k8, cd);
          *reinterpret_cast<u32x4*>(codes + lane * RCP + sl * G + 8 * k8) =
              u32x4{int_to_bf16_pair(cd[0], cd[1]), int_to_bf16_pair(cd[2], cd[3]), int_to_bf16_pair(cd[4], cd[5]),
                    int_to_bf16_pair(cd[6], cd[7])};
        });
        if (k8 == 0) {
          const uint32_t m = rt[sl * TROW];
          kmeta[sl * RTT + lane] = f32x2{h2f(m), h2f(m >> 16)};
        }
      }
    }
  };
  // queries rotated by (p_q - 64 tt) w_i, [pair i][head][2] (lane = pair), by the last wavefront
  auto rotate_queries = [&](int64_t tt) {
    float c, sn;
    sincos_reduced((double)(a.q_pos - tt * 64) * (double)a.inv_freq[lane], &c, &sn);
#pragma unroll
    for (int hh = 0; hh < NH; hh += 2) {
      const float a0 = qs[hh * D + lane], a1 = qs[hh * D + 64 + lane];
      const float b0 = qs[(hh + 1) * D + lane], b1 = qs[(hh + 1) * D + 64 + lane];
      *reinterpret_cast<f32x4*>(qpp + (lane * NH + hh) * 2) =
          f32x4{a0 * c - a1 * sn, a1 * c + a0 * sn, b0 * c - b1 * sn, b1 * c + b0 * sn};
    }
  };
  __syncthreads();  // tables, queries and sums visible
  if (ok && tile_begin < tile_end) {
    load_k(tile_begin);
    stage(recK, pk, Wk);
    if (wave == 3) rotate_queries(tile_begin);
    __syncthreads();
    unpack_k();
    if (tile_begin + 1 < tile_end) load_k(tile_begin + 1);
    load_v(tile_begin);
    __syncthreads();  // codes, scales and rotated queries of the first tile visible
  }

  for (int64_t tt = tile_begin; ok && tt < tile_end; ++tt) {
    const bool more = tt + 1 < tile_end;
    // keep the loop-invariant LDS operands (sums, angle tables) as reads inside the
    // loop rather than registers held across it
    asm volatile("" ::: "memory");
    // this tile's value words and the next tile's key words to LDS, the loads after them
    stage(recV, pv, Wv);
    if (more) stage(recK, pk, Wk);
    if (tt + 2 < tile_end) load_k(tt + 2);
    if (more) load_v(tt + 1);

    // ---- 1. reconstruction, in-tile rotation and dot products, 32 tokens at a time ----
#pragma unroll 1
    for (int tb = 0; tb < 2; ++tb) {
      const int tok = 32 * tb + c32;  // the lane's token (output column)
      f32x16 o;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int m0 = 8 * q + 4 * h;
        const int d0 = m0 < 16 ? 16 * wave + m0 : 48 + 16 * wave + m0;
        const f32x4 bv = *reinterpret_cast<const f32x4*>(&vsum[NG * D + d0]);
#pragma unroll
        for (int r = 0; r < 4; ++r) o[4 * q + r] = bv[r];
      }
#pragma unroll
      for (int sl = 0; sl < NG; ++sl) {
        if (sl < Kk.n) {
          f32x16 acc = {};
#pragma unroll
          for (int ks = 0; ks < 2; ++ks) {
            const bf16x8 C = as_bf16x8(*reinterpret_cast<const u32x4*>(codes + tok * RCP + sl * G + 16 * ks + 8 * h));
#pragma unroll
            for (int p = 0; p < 3; ++p) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(Va[sl][ks][p], C, acc, 0, 0, 0);
          }
          const f32x2 sz = kmeta[sl * RTT + tok];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int m0 = 8 * q + 4 * h;
            const int d0 = m0 < 16 ? 16 * wave + m0 : 48 + 16 * wave + m0;
            const f32x4 v4 = *reinterpret_cast<const f32x4*>(&vsum[sl * D + d0]);
#pragma unroll
            for (int r = 0; r < 4; ++r) o[4 * q + r] = __builtin_fmaf(sz[0], acc[4 * q + r], __builtin_fmaf(sz[1], v4[r], o[4 * q + r]));
          }
        }
      }
      // pairs: row m < 16 (entry j < 8) with row m + 16 (entry j + 8), i = 16 wave + m
      const f32x2* tr = tab + (FULL_TAB ? tok : (tok & 7)) * R4TP;
      const f32x2* ta = tab + (8 + (tok >> 3)) * R4TP;  // eight heads: angle 8a w_i, r = 8a + b
      float sc[NH];
#pragma unroll
      for (int hh = 0; hh < NH; ++hh) sc[hh] = 0.0f;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int i = 16 * wave + 8 * (j >> 2) + 4 * h + (j & 3);
        float c, sn;
        if constexpr (FULL_TAB) {
          const f32x2 cs = tr[i];
          c = cs[0];
          sn = cs[1];
        } else {
          const f32x2 cb = tr[i], ca = ta[i];
          c = ca[0] * cb[0] - ca[1] * cb[1];
          sn = ca[1] * cb[0] + ca[0] * cb[1];
        }
        const float x0 = o[j], x1 = o[j + 8];
        const float r0 = x0 * c - x1 * sn, r1 = x1 * c + x0 * sn;
#pragma unroll
        for (int hh = 0; hh < NH; hh += 2) {
          const f32x4 qv = *reinterpret_cast<const f32x4*>(qpp + (i * NH + hh) * 2);
          sc[hh] = __builtin_fmaf(qv[0], r0, __builtin_fmaf(qv[1], r1, sc[hh]));
          sc[hh + 1] = __builtin_fmaf(qv[2], r0, __builtin_fmaf(qv[3], r1, sc[hh + 1]));
        }
      }
      // the other half of the wavefront holds the other eight pairs of the same token
#pragma unroll
      for (int hh = 0; hh < NH; ++hh) sc[hh] += other_half(sc[hh]);
      if (h == 0) {
#pragma unroll
        for (int hh = 0; hh < NH; ++hh) red[(wave * NH + hh) * 64 + tok] = sc[hh];
      }
    }
    __syncthreads();  // partial scores, value words and the next tile's key words visible

    // ---- 2. online softmax over the tile (lane = token) and value sums ----
    const bool valid = tt * 64 + lane < a.n_tokens;
    float x[NH];
    bool over = false;
#pragma unroll
    for (int hh = 0; hh < NH; ++hh) {
      const float acc = (red[(0 * NH + hh) * 64 + lane] + red[(1 * NH + hh) * 64 + lane]) +
                        (red[(2 * NH + hh) * 64 + lane] + red[(3 * NH + hh) * 64 + lane]);
      x[hh] = (valid && hh < nqh) ? acc : -__builtin_inff();
      over = over || x[hh] > m_run[hh] + RESCALE_SLACK;
    }
    if (__any(over)) {
#pragma unroll
      for (int hh = 0; hh < NH; ++hh) {
        if (__any(x[hh] > m_run[hh] + RESCALE_SLACK)) {
          const float mn = __builtin_fmaxf(m_run[hh], wave_max_all(x[hh]));
          const float alpha = (m_run[hh] == -__builtin_inff()) ? 0.0f : __builtin_amdgcn_exp2f(m_run[hh] - mn);
          l_run[hh] *= alpha;
          zacc[hh] *= alpha;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int row = 4 * kq + j;
            const float f = (row == hh || row == NH + hh) ? alpha : 1.0f;
            vacc[0][j] *= f;
            vacc[1][j] *= f;
          }
          m_run[hh] = mn;
        }
      }
    }
    float pw[NH];
#pragma unroll
    for (int hh = 0; hh < NH; ++hh) {
      pw[hh] = x[hh] != -__builtin_inff() ? __builtin_amdgcn_exp2f(x[hh] - m_run[hh]) : 0.0f;
      l_run[hh] += pw[hh];
    }
    if (vslot) {
      const uint32_t meta = valid ? recV[wave * TROW + lane] : 0u;
      const float sv = h2f(meta), zv = h2f(meta >> 16);
#pragma unroll
      for (int hh = 0; hh < NH; hh += 2) {  // two heads per packed conversion
        zacc[hh] = __builtin_fmaf(pw[hh], zv, zacc[hh]);
        zacc[hh + 1] = __builtin_fmaf(pw[hh + 1], zv, zacc[hh + 1]);
        const float w0 = pw[hh] * sv, w1 = pw[hh + 1] * sv;
        const uint32_t hb2 = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{w0, w1}, bf16x2));
        const float h0 = __builtin_bit_cast(float, hb2 << 16), h1 = __builtin_bit_cast(float, hb2 & 0xFFFF0000u);
        const uint32_t lb = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{w0 - h0, w1 - h1}, bf16x2));
        ws[hh * WROW + lane] = (uint16_t)hb2;
        ws[(hh + 1) * WROW + lane] = (uint16_t)(hb2 >> 16);
        ws[(NH + hh) * WROW + lane] = (uint16_t)lb;
        ws[(NH + hh + 1) * WROW + lane] = (uint16_t)(lb >> 16);
      }
      __builtin_amdgcn_wave_barrier();
      // rows 0..NH-1: hi weights of the heads, NH..2NH-1: lo; MFMA rows past them
      // re-read a weight row and are never read back
      const int arow = col16 < 2 * NH ? col16 : col16 - 2 * NH;
      const bf16x8 negone = as_bf16x8(u32x4{0xBF80BF80u, 0xBF80BF80u, 0xBF80BF80u, 0xBF80BF80u});
      uint32_t vmagic = 0x3F803F80u;  // exponent of 1.0 in both halves (see value_codes2)
      asm volatile("" : "+v"(vmagic));
      auto body = [&](auto cls) {
        constexpr int CLS = decltype(cls)::value;
#pragma unroll
        for (int th = 0; th < 2; ++th) {
          const int tok0 = 32 * th + 8 * kq;
          const bf16x8 aw = as_bf16x8(*reinterpret_cast<const u32x4*>(ws + arow * WROW + tok0));
          u32x4 vc[2];
          value_codes2<CLS>(recV, vpay, Kv.used, vB, voff, tok0, vmagic, vc[0], vc[1]);
#pragma unroll
          for (int c2 = 0; c2 < 2; ++c2) {
            f32x4 acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aw, as_bf16x8(vc[c2]), vacc[c2], 0, 0, 0);
            if constexpr (CLS != 2) acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aw, negone, acc, 0, 0, 0);
            vacc[c2] = acc;
          }
        }
      };
      if (vB == 8)
        body(std::integral_constant<int, 2>{});
      else if (vB == 1 || vB == 2 || vB == 4)
        body(std::integral_constant<int, 0>{});
      else
        body(std::integral_constant<int, 1>{});
    }
    if (more) {
      unpack_k();
      if (wave == 3) rotate_queries(tt + 1);
    }
    __syncthreads();  // the tile's LDS reads done; the next tile's codes and queries visible
  }

  // ---- chunk partial: m, l and the zero-point sums per head, value sums per coefficient ----
  // (every wavefront holds the same m and l: the softmax runs in all of them)
  float zs[NH];
#pragma unroll
  for (int hh = 0; hh < NH; ++hh) {
    const float l = wave_sum_lane63(l_run[hh]);
    zs[hh] = wave_sum_lane63(zacc[hh]);
    if (wave == 0 && lane == 63) lst[hh] = l;
  }
  if (tid < NH * NG) zst[tid / NG][tid % NG] = 0.0f;
  __syncthreads();
  if (vslot && lane == 63) {
#pragma unroll
    for (int hh = 0; hh < NH; ++hh) zst[hh][vgrp] = zs[hh];
  }
  float* accw = reinterpret_cast<float*>(codes);  // [2NH][AROW]: hi-weight rows, then lo
  if (vslot) {
    // codes below 8 bits entered as 1 + c 2^-b (see value_codes2)
    const float vscale = vB < 8 ? (float)(1u << vB) : 1.0f;
#pragma unroll
    for (int c2 = 0; c2 < 2; ++c2)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int row = 4 * kq + j;
        if (row < 2 * NH) accw[row * AROW + G * vgrp + 2 * col16 + c2] = vacc[c2][j] * vscale;
      }
  }
  uint32_t kept_groups = 0u;
#pragma unroll
  for (int sl = 0; sl < NG; ++sl)
    if (sl < Kv.n) kept_groups |= 1u << pick4(Kv.grp, sl);
  __syncthreads();
  float* part = a.partial + ((int64_t)b * a.n_q_heads + kv * nqh) * a.n_chunks * PART + (int64_t)chunk * PART;
  const bool any = ok && tile_begin < tile_end;
  for (int e = tid; e < nqh * D; e += R4T) {
    const int hh = e >> 7, j = e & 127;
    const bool kept = any && ((kept_groups >> (j >> 5)) & 1u);
    float* ph = part + (int64_t)hh * a.n_chunks * PART;
    ph[8 + j] = kept ? accw[hh * AROW + j] + accw[(NH + hh) * AROW + j] : 0.0f;
    if (j == 0) {
      ph[0] = any ? m_run[hh] : -__builtin_inff();
      ph[1] = any ? lst[hh] : 0.0f;
    }
    if (j < NG) ph[2 + j] = any ? zst[hh][j] : 0.0f;
  }
}

}  // namespace spectra_dev

namespace spectra {
using namespace spectra_dev;

// About per_cu workgroups per CU in one round, at least four tiles per chunk.
int32_t rope_attention_chunks(int32_t batch, int32_t n_kv_heads, int64_t n_tokens, int32_t* tiles_per_chunk,
                              int32_t per_cu) {
  const int64_t n_tiles = (n_tokens + 63) / 64;
  const int64_t groups = (int64_t)batch * n_kv_heads;
  const int64_t want = (256 * (int64_t)per_cu + groups - 1) / groups;
  int64_t tpc = (n_tiles + want - 1) / want;
  if (tpc < 4) tpc = 4;
  *tiles_per_chunk = (int32_t)tpc;
  return (int32_t)((n_tiles + tpc - 1) / tpc);
}

// The four-wavefront kernel (two workgroups per CU) for at most eight query heads per
// KV head and records of at most 16 words; the eight-wavefront kernel otherwise.
hipError_t launch_attention_rope(const AttnArgs& a, hipStream_t st) {
  int dev = 0, lds = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
  if (e != hipSuccess) return e;
  const int nq = a.n_qh <= 4 ? 1 : 2;
  const bool four = a.n_qh <= 8 && a.Wk <= R4W && a.Wv <= R4W && lds >= r4_lds_bytes(4 * nq);
  AttnArgs g = a;
  g.n_chunks = rope_attention_chunks(a.batch, a.n_kv_heads, a.n_tokens, &g.tiles_per_chunk, four ? 2 : 1);
  const dim3 grid(g.n_chunks, g.n_kv_heads, g.batch);
  if (four) {
    if (nq == 1)
      hipLaunchKernelGGL(rope_attn4_kernel<1>, grid, dim3(R4T), r4_lds_bytes(4), st, g);
    else
      hipLaunchKernelGGL(rope_attn4_kernel<2>, grid, dim3(R4T), r4_lds_bytes(8), st, g);
  } else {
    // the tile buffers need more than 64 KB of LDS: refuse a device that has less
    const int nh = a.n_qh <= 4 ? 4 : 8;
    if (lds < rope_lds_bytes(nh)) return hipErrorInvalidConfiguration;
    if (nh == 4)
      hipLaunchKernelGGL(rope_attn_kernel<1>, grid, dim3(RTHREADS), rope_lds_bytes(4), st, g);
    else
      hipLaunchKernelGGL(rope_attn_kernel<2>, grid, dim3(RTHREADS), rope_lds_bytes(8), st, g);
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_combine(g, st);
}

}  // namespace spectra
