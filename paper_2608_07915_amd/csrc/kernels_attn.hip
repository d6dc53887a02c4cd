// Decode-step attention read straight from the packed caches (App. E, Mode B).
//
//   q'_h   = scale * log2(e) * q_h V_K              (workgroup prologue)
//   score  = sum_G s_tG <q'_G, code_tG> + z_tG sum_{j in G} q'_j
//            (the constant q' . m_K cancels in the softmax and is dropped)
//   a_h    = sum_t p_ht (z_tG + s_tG code_tj)       over kept value coefficients
//   out_h  = (a_h / l_h + m_V) V_V^T                (combine_kernel)
//
// The per-token contractions over the kept latent coefficients are the two
// matrix products of latent attention; they run on MFMA:
//   * scores: v_mfma_f32_4x4x4f16 (16 blocks), lane = token, block rows = four
//     query heads; codes are exact in fp16; q' enters as two fp16 parts (hi+lo)
//     pre-scaled by a power of two, so the dot products are ~fp32-accurate;
//   * values: v_mfma_f32_16x16x32_bf16, rows = query heads (softmax weights p*s as
//     bf16 hi and lo parts, stacked in the otherwise unused rows when there are
//     at most 8 heads), K = 32 tokens, columns = 16 coefficients. Codes of width
//     <= 7 enter as bf16 (128 + c), built with one byte-gather permute and a mask;
//     a second MFMA against the constant -128 removes the offset tile by tile.
// Work: one workgroup of four wavefronts per (token chunk, KV head, sequence);
// each wavefront streams 64-token record tiles with the next tile's words
// prefetched into registers; the four wavefronts merge their online-softmax
// states in LDS and write one partial per chunk; combine_kernel merges chunks.
#include "device_common.hpp"
#include "kernels.hpp"

namespace spectra_dev {

constexpr int PART = 136;                    // floats per (chunk, query head): m, l, Z[4], pad[2], acc[128]
constexpr int QA_QUAD = 4 * 8 * 2 * 4 * 2;   // uint32 of score-MFMA A operands per head quad
constexpr int QP = 4 + 16 * 4 + 4 * QA_QUAD;  // floats per (sequence, kv head) of prepared query data
constexpr int WAVES = 4;
constexpr int WROW = 72;  // bf16 per weight row (64 tokens + pad: spreads rows over LDS banks)

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = __builtin_fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}


// ---------------------------------------------------------------------------
// Query preparation, once per step: one workgroup per (kv head, sequence) writes
// E2 = 2^-E, Qbar[h][g] = sum_{j in g} q'_hj and the score-MFMA A operands
// [quad][g][k][part][r] = fp16 parts of q'_{4quad+r}[32g + 4k + i] * 2^E.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void qprep_kernel(AttnArgs a) {
  __shared__ float qs[16][D];
  __shared__ float part_s[2][16][D];
  __shared__ float red_s[4];
  const int kv = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  const int s = b * a.n_kv_heads + kv;
  const int nqh = a.n_qh;
  for (int e = tid; e < 16 * D; e += 256) {
    const int h = e >> 7, c = e & 127;
    float v = 0.0f;
    if (h < nqh) {
      const int64_t qi = ((int64_t)b * a.n_q_heads + kv * nqh + h) * D + c;
      v = a.q_f32 ? reinterpret_cast<const float*>(a.q)[qi] : bf2f(reinterpret_cast<const uint16_t*>(a.q)[qi]);
    }
    qs[h][c] = v;
  }
  // column j of V_K, rows [64 half, 64 half + 64): all loads issued before use
  const int j = tid & 127, half = tid >> 7;
  const float* Vk = a.basis_k + (int64_t)s * D * D + (int64_t)(64 * half) * D + j;
  float v[64];
#pragma unroll
  for (int i = 0; i < 64; ++i) v[i] = Vk[i * D];
  __syncthreads();
  for (int h = 0; h < nqh; ++h) {
    float acc = 0.0f;
#pragma unroll
    for (int i = 0; i < 64; ++i) acc = __builtin_fmaf(qs[h][64 * half + i], v[i], acc);
    part_s[half][h][j] = acc;
  }
  __syncthreads();
  float amax = 0.0f;
  for (int e = tid; e < 16 * D; e += 256) {
    const int h = e >> 7, c = e & 127;
    const float q = h < nqh ? (part_s[0][h][c] + part_s[1][h][c]) * a.scale_log2 : 0.0f;
    qs[h][c] = q;
    amax = __builtin_fmaxf(amax, __builtin_fabsf(q));
  }
  amax = wave_max(amax);
  if ((tid & 63) == 0) red_s[tid >> 6] = amax;
  __syncthreads();
  amax = __builtin_fmaxf(__builtin_fmaxf(red_s[0], red_s[1]), __builtin_fmaxf(red_s[2], red_s[3]));
  // 2^E brings max |q'| into [2^13, 2^14): both fp16 parts stay normal and finite.
  int e2 = 0;
  if (amax > 0.0f) (void)__builtin_frexpf(amax, &e2);
  const int E = amax > 0.0f ? 14 - e2 : 0;
  const float scl = __builtin_ldexpf(1.0f, E);
  float* qp = a.qprep + (int64_t)s * QP;
  if (tid == 0) {
    qp[0] = __builtin_ldexpf(1.0f, -E);
    qp[1] = qp[2] = qp[3] = 0.0f;
  }
  if (tid < 64) {
    const int h = tid >> 2, g = tid & 3;
    float acc = 0.0f;
    for (int i = 0; i < G; ++i) acc += qs[h][G * g + i];
    qp[4 + tid] = acc;
  }
  // K order of the score MFMA: for widths dividing 32 the kernel pairs codes
  // i and i + 16/b of each payload word (one shift and one mask per pair), so
  // step k, slot (2u + v) is coefficient word*(32/b) + i + v*(16/b) of pair
  // 2k + u; other widths keep the natural order 4k + slot.
  const uint32_t bwk = *reinterpret_cast<const uint32_t*>(a.bits_k + (int64_t)s * NG);
  uint32_t* qa = reinterpret_cast<uint32_t*>(qp + 4 + 64);
  for (int e = tid; e < 4 * 128; e += 256) {
    const int r = e & 3, k = (e >> 2) & 7, g = (e >> 5) & 3, quad = e >> 7;
    const int h = 4 * quad + r;
    const int B = (int)((bwk >> (8 * g)) & 0xFFu);
    const bool fast = B == 1 || B == 2 || B == 4 || B == 8;
    uint32_t hi[4], lo[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int jj = 4 * k + i;
      if (fast) {
        const int half = 16 / B, pair = 2 * k + (i >> 1);
        jj = (pair / half) * (32 / B) + (pair % half) + (i & 1) * half;
      }
      const float x = qs[h][G * g + jj] * scl;
      const _Float16 xh = (_Float16)x;
      const _Float16 xl = (_Float16)(x - (float)xh);
      hi[i] = __builtin_bit_cast(uint16_t, xh);
      lo[i] = __builtin_bit_cast(uint16_t, xl);
    }
    const int base = ((((quad * 4 + g) * 8 + k) * 2) * 4 + r) * 2;
    qa[base + 0] = hi[0] | (hi[1] << 16);
    qa[base + 1] = hi[2] | (hi[3] << 16);
    qa[base + 8] = lo[0] | (lo[1] << 16);
    qa[base + 9] = lo[2] | (lo[3] << 16);
  }
}

// Bytes of LDS holding the softmax-weight rows of all wavefronts: per wave and kept
// slot, 2*NH rows (hi parts of the NH heads, then lo parts) of 64 bf16 tokens.
__host__ __device__ constexpr int attn_wt_bytes(int nq) { return WAVES * NG * (8 * nq) * WROW * 2; }

// ---------------------------------------------------------------------------
// Value-code operand: 8 codes of in-group coefficient n (bit offset off = n*b in
// the group payload starting at record word `pay`) for 8 consecutive tokens, as
// bf16. CLS 0: b in {1,2,4} (a code never crosses a byte); CLS 1: b in {3,5,6,7};
// both give 128 + c. CLS 2: b = 8, exact c.
// ---------------------------------------------------------------------------
template <int CLS>
__device__ __forceinline__ u32x4 value_codes(const uint32_t* __restrict__ vt, int pay, int used, int b, int off,
                                             int tok0) {
  const int w = pay + (off >> 5), o = off & 31;
  const u32x4 a0 = *reinterpret_cast<const u32x4*>(vt + w * 64 + tok0);
  const u32x4 a1 = *reinterpret_cast<const u32x4*>(vt + w * 64 + tok0 + 4);
  const uint32_t M = (1u << b) - 1u;
  const uint32_t MM = M | (M << 16);
  u32x4 r;
  if constexpr (CLS == 0) {
    // gather byte k of two tokens' words with one permute, then shift and mask
    const uint32_t k = (uint32_t)o >> 3, sh = (uint32_t)o & 7u;
    const uint32_t sel = k * 0x00000101u + (4u + k) * 0x01010000u;
    r[0] = ((__builtin_amdgcn_perm(a0[1], a0[0], sel) >> sh) & MM) | 0x43004300u;
    r[1] = ((__builtin_amdgcn_perm(a0[3], a0[2], sel) >> sh) & MM) | 0x43004300u;
    r[2] = ((__builtin_amdgcn_perm(a1[1], a1[0], sel) >> sh) & MM) | 0x43004300u;
    r[3] = ((__builtin_amdgcn_perm(a1[3], a1[2], sel) >> sh) & MM) | 0x43004300u;
  } else {
    const int wn = (w + 1 < used) ? w + 1 : w;  // the next word only matters when the code straddles
    const u32x4 b0 = *reinterpret_cast<const u32x4*>(vt + wn * 64 + tok0);
    const u32x4 b1 = *reinterpret_cast<const u32x4*>(vt + wn * 64 + tok0 + 4);
    uint32_t c[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      c[i] = __builtin_amdgcn_alignbit(b0[i], a0[i], o);
      c[4 + i] = __builtin_amdgcn_alignbit(b1[i], a1[i], o);
    }
    if constexpr (CLS == 2) {
#pragma unroll
      for (int i = 0; i < 4; ++i) r[i] = int_to_bf16_pair(c[2 * i] & 0xFFu, c[2 * i + 1] & 0xFFu);
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) r[i] = (__builtin_amdgcn_perm(c[2 * i + 1], c[2 * i], 0x05040100u) & MM) | 0x43004300u;
    }
  }
  return r;
}

// ---------------------------------------------------------------------------
// Split-K partial. NQ = query-head quads (n_qh <= 4 NQ); PW = prefetched record
// words per tile (>= max(W_k, W_v)).
// ---------------------------------------------------------------------------
template <int NQ, int PW>
__global__ __launch_bounds__(256, 2) void attn_kernel(AttnArgs a) {
  constexpr int NH = 4 * NQ;
  constexpr bool STACK = NQ <= 2;  // 2*NH <= 16: hi and lo weight rows share one MFMA
  extern __shared__ __attribute__((aligned(16))) uint32_t smem[];
  __shared__ __attribute__((aligned(16))) uint32_t qa_s[NQ * QA_QUAD];
  __shared__ float qbar_s[16 * 4];
  __shared__ float mst[WAVES][NH], lst[WAVES][NH], zst[WAVES][NH][NG];

  const int chunk = blockIdx.x, kv = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int s = b * a.n_kv_heads + kv;
  const int nqh = a.n_qh;
  const Kept Kk = read_kept(a.bits_k + (int64_t)s * NG);
  const Kept Kv = read_kept(a.bits_v + (int64_t)s * NG);
  const int Wk = a.Wk, Wv = a.Wv;
  const bool ok = Kk.ok && Kv.ok && Kk.used <= Wk && Kv.used <= Wv;

  // ---- prologue: prepared query data of this (sequence, kv head) ----
  const float* qp = a.qprep + (int64_t)s * QP;
  for (int i = tid; i < NQ * QA_QUAD; i += 256) qa_s[i] = reinterpret_cast<const uint32_t*>(qp + 4 + 64)[i];
  if (tid < 64) qbar_s[tid] = qp[4 + tid];
  const float E2 = qp[0];

  // ---- per-wave streaming over this chunk's tiles ----
  const int wk_rows = PW > 0 ? PW : Wk, wv_rows = PW > 0 ? PW : Wv;  // staged words per token
  const int wpw = wk_rows + wv_rows;
  uint32_t* kt = smem + wave * wpw * 64;
  uint32_t* vt = kt + wk_rows * 64;
  uint16_t* wt = reinterpret_cast<uint16_t*>(smem + WAVES * wpw * 64) + wave * (NG * 2 * NH * WROW);
  const int64_t kbase = (int64_t)s * a.t_cap * Wk;
  const int64_t vbase = (int64_t)s * a.t_cap * Wv;
  const int64_t n_tiles = (a.n_tokens + 63) >> 6;
  const int64_t tile_begin = (int64_t)chunk * a.tiles_per_chunk;
  int64_t tile_end = tile_begin + a.tiles_per_chunk;
  if (tile_end > n_tiles) tile_end = n_tiles;

  float m_run[NH], l_run[NH], zacc[NH][NG];
#pragma unroll
  for (int h = 0; h < NH; ++h) {
    m_run[h] = -__builtin_inff();
    l_run[h] = 0.0f;
#pragma unroll
    for (int g = 0; g < NG; ++g) zacc[h][g] = 0.0f;
  }
  f32x4 vacc[NG][2];
#pragma unroll
  for (int g = 0; g < NG; ++g) vacc[g][0] = vacc[g][1] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int r4 = lane & 3;    // score MFMA: A row (query head within a quad)
  const int col = lane & 15;  // value MFMA: coefficient column / A row
  const int kq = lane >> 4;   // value MFMA: 8-token group of K

  // register prefetch of one tile's record words (K and V); PW = 0: none
  constexpr int PWR = PW > 0 ? PW : 1;
  uint32_t pk[PWR], pv[PWR];
  auto load_tile = [&](int64_t tt) {
    // every lane loads in-bounds words (word index clamped to the record, token
    // to the tile); values of tokens past n_tokens are zeroed afterwards
    const uint32_t* kp = a.packed_k + kbase + tt * (64 * Wk) + lane;  // word w at kp[64 w]
    const uint32_t* vp = a.packed_v + vbase + tt * (64 * Wv) + lane;
#pragma unroll
    for (int w = 0; w < PW; ++w) {
      pk[w] = kp[64 * (w < Wk ? w : Wk - 1)];
      pv[w] = vp[64 * (w < Wv ? w : Wv - 1)];
    }
  };
  int64_t tt = tile_begin + wave;
  if (ok && tt < tile_end) load_tile(tt);
  __syncthreads();  // prepared query data in LDS

  Kept kk = Kk, kvv = Kv;
  for (; ok && tt < tile_end; tt += WAVES) {
    // keep per-tile LDS reads (operand tables) inside the loop instead of in registers,
    // and make the slot tables opaque so their derived scalars are not hoisted out of it
    asm volatile("" ::: "memory");
#pragma unroll
    for (int i = 0; i < NG; ++i) {
      kk.grp[i] = __builtin_amdgcn_readfirstlane(kk.grp[i]);
      kk.bits[i] = __builtin_amdgcn_readfirstlane(kk.bits[i]);
      kk.pay[i] = __builtin_amdgcn_readfirstlane(kk.pay[i]);
      kvv.grp[i] = __builtin_amdgcn_readfirstlane(kvv.grp[i]);
      kvv.bits[i] = __builtin_amdgcn_readfirstlane(kvv.bits[i]);
      kvv.pay[i] = __builtin_amdgcn_readfirstlane(kvv.pay[i]);
      asm volatile("" : "+s"(kk.grp[i]), "+s"(kk.bits[i]), "+s"(kk.pay[i]));
      asm volatile("" : "+s"(kvv.grp[i]), "+s"(kvv.bits[i]), "+s"(kvv.pay[i]));
    }
    kk.n = __builtin_amdgcn_readfirstlane(kk.n);
    kvv.n = __builtin_amdgcn_readfirstlane(kvv.n);
    kvv.used = __builtin_amdgcn_readfirstlane(kvv.used);
    asm volatile("" : "+s"(kk.n), "+s"(kvv.n), "+s"(kvv.used));
    const int64_t t = tt * 64 + lane;
    const bool valid = t < a.n_tokens;
    // stage this tile's words in LDS (lane = token), then prefetch the next tile
    if constexpr (PW > 0) {
#pragma unroll
      for (int w = 0; w < PW; ++w) {
        kt[w * 64 + lane] = valid ? pk[w] : 0u;
        vt[w * 64 + lane] = valid ? pv[w] : 0u;
      }
      if (tt + WAVES < tile_end) load_tile(tt + WAVES);
    } else {
      for (int w = 0; w < kk.used; ++w) kt[w * 64 + lane] = valid ? a.packed_k[rec_word(kbase, t, Wk, w)] : 0u;
      for (int w = 0; w < kvv.used; ++w) vt[w * 64 + lane] = valid ? a.packed_v[rec_word(vbase, t, Wv, w)] : 0u;
    }
    __builtin_amdgcn_wave_barrier();

    // ---- scores over the kept key coefficients (lane = token) ----
    float sc[NH];
#pragma unroll
    for (int h = 0; h < NH; ++h) sc[h] = 0.0f;
#pragma unroll
    for (int sl = 0; sl < NG; ++sl) {
      if (sl >= kk.n) continue;
      const int g = kk.grp[sl];
      const uint32_t meta = kt[sl * 64 + lane];
      f32x4 d[NQ];
#pragma unroll
      for (int q = 0; q < NQ; ++q) d[q] = f32x4{0.f, 0.f, 0.f, 0.f};
      {
        const int B = kk.bits[sl], pay = kk.pay[sl];
        typedef __attribute__((__vector_size__(2 * sizeof(_Float16)))) _Float16 f16x2;
        const f16x2 off = {(_Float16)1024.0f, (_Float16)1024.0f};
        const uint32_t MM = ((1u << B) - 1u) * 0x00010001u;
        if (B == 1 || B == 2 || B == 4 || B == 8) {
          // pair (c_i, c_{i+16/B}) of a payload word = (x >> B i) & MM: one shift, one and-or
          const int lg = B == 1 ? 0 : B == 2 ? 1 : B == 4 ? 2 : 3;  // log2 B
#pragma unroll 2
          for (int k = 0; k < 8; ++k) {
            const int pair = 2 * k, wsel = (pair << lg) >> 4, i0 = pair & ((16 >> lg) - 1);
            const uint32_t x = kt[(pay + wsel) * 64 + lane];
            const uint32_t v0 = ((x >> (i0 << lg)) & MM) | 0x64006400u;
            const uint32_t v1 = ((x >> ((i0 + 1) << lg)) & MM) | 0x64006400u;
            const f16x2 p01 = __builtin_bit_cast(f16x2, v0) - off;
            const f16x2 p23 = __builtin_bit_cast(f16x2, v1) - off;
            const f16x4 bop = {p01[0], p01[1], p23[0], p23[1]};
#pragma unroll
            for (int q = 0; q < NQ; ++q) {
              const int base = ((((q * 4 + g) * 8 + k) * 2) * 4 + r4) * 2;
              const f16x4 ahi = as_f16x4(*reinterpret_cast<const u32x2*>(qa_s + base));
              const f16x4 alo = as_f16x4(*reinterpret_cast<const u32x2*>(qa_s + base + 8));
              d[q] = __builtin_amdgcn_mfma_f32_4x4x4f16(ahi, bop, d[q], 0, 0, 0);
              d[q] = __builtin_amdgcn_mfma_f32_4x4x4f16(alo, bop, d[q], 0, 0, 0);
            }
          }
        } else {
#pragma unroll 2
          for (int k = 0; k < 8; ++k) {
            // codes 4k..4k+3 of this token: a 4B-bit window starting at bit 4kB
            const int p0 = 4 * k * B, w0 = pay + (p0 >> 5);
            const uint32_t lo = kt[w0 * 64 + lane];
            const uint32_t hi = ((p0 & 31) + 4 * B > 32) ? kt[(w0 + 1) * 64 + lane] : 0u;
            const uint32_t win = __builtin_amdgcn_alignbit(hi, lo, (uint32_t)(p0 & 31));
            const uint32_t c0 = __builtin_amdgcn_ubfe(win, 0, B), c1 = __builtin_amdgcn_ubfe(win, B, B);
            const uint32_t c2 = __builtin_amdgcn_ubfe(win, 2 * B, B), c3 = __builtin_amdgcn_ubfe(win, 3 * B, B);
            // 1024 + c as fp16 has c in the mantissa; subtracting 1024 is exact
            const f16x2 p01 = __builtin_bit_cast(f16x2, __builtin_amdgcn_perm(c1, c0, 0x05040100u) | 0x64006400u) - off;
            const f16x2 p23 = __builtin_bit_cast(f16x2, __builtin_amdgcn_perm(c3, c2, 0x05040100u) | 0x64006400u) - off;
            const f16x4 bop = {p01[0], p01[1], p23[0], p23[1]};
#pragma unroll
            for (int q = 0; q < NQ; ++q) {
              const int base = ((((q * 4 + g) * 8 + k) * 2) * 4 + r4) * 2;
              const f16x4 ahi = as_f16x4(*reinterpret_cast<const u32x2*>(qa_s + base));
              const f16x4 alo = as_f16x4(*reinterpret_cast<const u32x2*>(qa_s + base + 8));
              d[q] = __builtin_amdgcn_mfma_f32_4x4x4f16(ahi, bop, d[q], 0, 0, 0);
              d[q] = __builtin_amdgcn_mfma_f32_4x4x4f16(alo, bop, d[q], 0, 0, 0);
            }
          }
        }
      }
      const float sk = h2f(meta) * E2, zk = h2f(meta >> 16);
#pragma unroll
      for (int q = 0; q < NQ; ++q)
#pragma unroll
        for (int j = 0; j < 4; ++j) sc[4 * q + j] += sk * d[q][j] + zk * qbar_s[(4 * q + j) * 4 + g];
    }

    // ---- online softmax (log2 domain); the running max moves only when exceeded ----
    float p[NH];
#pragma unroll
    for (int h = 0; h < NH; ++h) {
      const bool live = valid && h < nqh;
      const float x = live ? sc[h] : -__builtin_inff();
      if (__any(x > m_run[h])) {
        const float mn = __builtin_fmaxf(m_run[h], wave_max(x));
        const float alpha = (m_run[h] == -__builtin_inff()) ? 0.0f : __builtin_amdgcn_exp2f(m_run[h] - mn);
        l_run[h] *= alpha;
#pragma unroll
        for (int g = 0; g < NG; ++g) zacc[h][g] *= alpha;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int row = 4 * kq + j;
          const float f = (row == h || (STACK && row == NH + h)) ? alpha : 1.0f;
#pragma unroll
          for (int g = 0; g < NG; ++g) {
            vacc[g][0][j] *= f;
            vacc[g][1][j] *= f;
          }
        }
        m_run[h] = mn;
      }
      p[h] = live ? __builtin_amdgcn_exp2f(x - m_run[h]) : 0.0f;
      l_run[h] += p[h];
    }
    // softmax weight times value scale, as bf16 hi/lo rows; zero-point terms per lane
#pragma unroll
    for (int sl = 0; sl < NG; ++sl) {
      if (sl >= kvv.n) continue;
      const uint32_t meta = vt[sl * 64 + lane];
      const float sv = h2f(meta), zv = h2f(meta >> 16);
      uint16_t* ws = wt + sl * 2 * NH * WROW;  // rows: hi of heads 0..NH-1, then lo
#pragma unroll
      for (int h = 0; h < NH; ++h) {
        zacc[h][sl] = __builtin_fmaf(p[h], zv, zacc[h][sl]);
        const float w = p[h] * sv;
        const __bf16 whi = (__bf16)w;
        const __bf16 wlo = (__bf16)(w - (float)whi);
        ws[h * WROW + lane] = __builtin_bit_cast(uint16_t, whi);
        ws[(NH + h) * WROW + lane] = __builtin_bit_cast(uint16_t, wlo);
      }
    }
    __builtin_amdgcn_wave_barrier();

    // ---- value accumulation over the kept value coefficients ----
    const bf16x8 neg128 = as_bf16x8(u32x4{0xC300C300u, 0xC300C300u, 0xC300C300u, 0xC300C300u});
#pragma unroll
    for (int sl = 0; sl < NG; ++sl) {
      if (sl >= kvv.n) continue;
      const uint16_t* ws = wt + sl * 2 * NH * WROW;
      const int B = kvv.bits[sl], pay = kvv.pay[sl];
      auto body = [&](auto cls) {
        constexpr int CLS = decltype(cls)::value;
#pragma unroll 1
        for (int th = 0; th < 2; ++th) {
          const int tok0 = 32 * th + 8 * kq;
          // stacked: rows 0..2NH-1 = hi then lo; otherwise hi rows and lo rows separately
          bf16x8 aw = bf16x8{};
          if (col < (STACK ? 2 * NH : NH)) aw = as_bf16x8(*reinterpret_cast<const u32x4*>(ws + col * WROW + tok0));
          bf16x8 awl = bf16x8{};
          if (!STACK && col < NH) awl = as_bf16x8(*reinterpret_cast<const u32x4*>(ws + (NH + col) * WROW + tok0));
#pragma unroll
          for (int c2 = 0; c2 < 2; ++c2) {
            const bf16x8 bop = as_bf16x8(value_codes<CLS>(vt, pay, kvv.used, B, (16 * c2 + col) * B, tok0));
            f32x4 acc = vacc[sl][c2];
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aw, bop, acc, 0, 0, 0);
            if constexpr (CLS != 2) acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aw, neg128, acc, 0, 0, 0);
            if constexpr (!STACK) {
              acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(awl, bop, acc, 0, 0, 0);
              if constexpr (CLS != 2) acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(awl, neg128, acc, 0, 0, 0);
            }
            vacc[sl][c2] = acc;
          }
        }
      };
      if (B == 8)
        body(std::integral_constant<int, 2>{});
      else if (B == 1 || B == 2 || B == 4)
        body(std::integral_constant<int, 0>{});
      else
        body(std::integral_constant<int, 1>{});
    }
    __builtin_amdgcn_wave_barrier();
  }

  // ---- merge the four wavefronts and write this chunk's partial ----
#pragma unroll
  for (int h = 0; h < NH; ++h) {
    const float l = wave_sum(l_run[h]);
    float z[NG];
#pragma unroll
    for (int g = 0; g < NG; ++g) z[g] = wave_sum(zacc[h][g]);
    if (lane == 0) {
      mst[wave][h] = ok ? m_run[h] : -__builtin_inff();
      lst[wave][h] = l;
#pragma unroll
      for (int g = 0; g < NG; ++g) zst[wave][h][g] = z[g];
    }
  }
  __syncthreads();  // all waves done with their tile buffers: reuse smem for the value sums
  float* accw = reinterpret_cast<float*>(smem) + wave * NH * D;  // [NH][128] per wave
  for (int i = lane; i < NH * D; i += 64) accw[i] = 0.0f;
  __builtin_amdgcn_wave_barrier();
  // rows 4*kq + j: heads (hi rows) then, when stacked, the lo rows of the same heads
#pragma unroll
  for (int pass = 0; pass < (STACK ? 2 : 1); ++pass) {
#pragma unroll
    for (int sl = 0; sl < NG; ++sl) {
      if (sl >= Kv.n) continue;
#pragma unroll
      for (int c2 = 0; c2 < 2; ++c2)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int row = 4 * kq + j;
          const int h = pass == 0 ? row : row - NH;
          if ((pass == 0 && row < NH) || (pass == 1 && row >= NH && row < 2 * NH)) {
            float* dst = accw + h * D + G * Kv.grp[sl] + 16 * c2 + col;
            *dst += vacc[sl][c2][j];
          }
        }
    }
    __builtin_amdgcn_wave_barrier();
  }
  __syncthreads();
  float* part = a.partial + ((int64_t)b * a.n_q_heads + kv * nqh) * a.n_chunks * PART + (int64_t)chunk * PART;
  for (int e = tid; e < nqh * D; e += 256) {
    const int h = e >> 7, j = e & 127;
    float M = -__builtin_inff();
#pragma unroll
    for (int w = 0; w < WAVES; ++w) M = __builtin_fmaxf(M, mst[w][h]);
    float acc = 0.0f, l = 0.0f, z = 0.0f;
#pragma unroll
    for (int w = 0; w < WAVES; ++w) {
      const float f = (mst[w][h] == -__builtin_inff()) ? 0.0f : __builtin_amdgcn_exp2f(mst[w][h] - M);
      acc += f * (reinterpret_cast<float*>(smem) + w * NH * D)[h * D + j];
      l += f * lst[w][h];
      if (j < NG) z += f * zst[w][h][j];
    }
    float* ph = part + (int64_t)h * a.n_chunks * PART;
    ph[8 + j] = acc;
    if (j == 0) {
      ph[0] = M;
      ph[1] = l;
    }
    if (j < NG) ph[2 + j] = z;
  }
}

// ---------------------------------------------------------------------------
// Combine chunk partials and inverse-rotate: one workgroup per (query head,
// sequence); 8 thread groups of 128 split the chunks, then reduce in LDS.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(1024) void combine_kernel(AttnArgs a) {
  __shared__ float accs[8][D];
  __shared__ float chat[D];
  __shared__ float red[32];
  const int hq = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  const int j = tid & 127, grp = tid >> 7;
  const int kv = hq / a.n_qh;
  const int s = b * a.n_kv_heads + kv;
  const float* ph = a.partial + ((int64_t)b * a.n_q_heads + hq) * a.n_chunks * PART;
  const int nch = a.n_chunks;
  float mx = -__builtin_inff();
  for (int c = tid; c < nch; c += 1024) mx = __builtin_fmaxf(mx, ph[(int64_t)c * PART]);
  mx = wave_max(mx);
  if ((tid & 63) == 0) red[tid >> 6] = mx;
  __syncthreads();
  mx = red[0];
#pragma unroll
  for (int i = 1; i < 16; ++i) mx = __builtin_fmaxf(mx, red[i]);
  const uint32_t bw = *reinterpret_cast<const uint32_t*>(a.bits_v + (int64_t)s * NG);
  const int g = j >> 5;
  const bool kept = ((bw >> (8 * g)) & 0xFFu) != 0u;
  float acc = 0.0f, l = 0.0f;
#pragma unroll 4
  for (int c = grp; c < nch; c += 8) {
    const float* pc = ph + (int64_t)c * PART;
    const float mc = pc[0];
    const float w = (mc == -__builtin_inff()) ? 0.0f : __builtin_amdgcn_exp2f(mc - mx);
    l += w * pc[1];
    if (kept) acc += w * (pc[2 + g] + pc[8 + j]);
  }
  accs[grp][j] = acc;
  __syncthreads();
  if (j == 0) red[16 + grp] = l;
  __syncthreads();
  if (tid < D) {
    float sacc = 0.0f, sl = 0.0f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      sacc += accs[i][tid];
      sl += red[16 + i];
    }
    chat[tid] = sacc / sl + a.mean_v[(int64_t)s * D + tid];
  }
  __syncthreads();
  if (tid < D) {
    const float* Vv = a.basis_v + (int64_t)s * D * D + (int64_t)tid * D;
    float o = 0.0f;
#pragma unroll 16
    for (int i = 0; i < D; ++i) o = __builtin_fmaf(chat[i], Vv[i], o);
    a.out[((int64_t)b * a.n_q_heads + hq) * D + tid] = o;
  }
}

}  // namespace spectra_dev

namespace spectra {
using namespace spectra_dev;

size_t attention_qprep_floats(int32_t batch, int32_t, int32_t n_kv_heads) { return (size_t)batch * n_kv_heads * QP; }
size_t attention_partial_floats(int32_t batch, int32_t n_q_heads, int32_t n_chunks) {
  return (size_t)batch * n_q_heads * n_chunks * PART;
}
int32_t attention_chunks(int32_t batch, int32_t n_kv_heads, int64_t n_tokens, int32_t* tiles_per_chunk) {
  const int64_t n_tiles = (n_tokens + 63) / 64;
  const int64_t groups = (int64_t)batch * n_kv_heads;
  const int64_t want = (768 + groups - 1) / groups;   // ~768 workgroups of 4 wavefronts
  int64_t tpc = (n_tiles + want - 1) / want;
  if (tpc < 16) tpc = 16;                              // >= 4 tiles per wavefront
  if (tpc > n_tiles) tpc = n_tiles > 0 ? n_tiles : 1;
  const int64_t nch = n_tiles > 0 ? (n_tiles + tpc - 1) / tpc : 1;
  *tiles_per_chunk = (int32_t)tpc;
  return (int32_t)nch;
}

template <int NQ, int PW>
static void launch_nq_pw(const AttnArgs& a, hipStream_t st) {
  const int wpw = PW > 0 ? 2 * PW : a.Wk + a.Wv;
  size_t tiles = (size_t)WAVES * wpw * 64 * 4 + (size_t)attn_wt_bytes(NQ);
  size_t merge = (size_t)WAVES * 4 * NQ * D * 4;       // per-wave value sums
  size_t lds = tiles > merge ? tiles : merge;
  const dim3 grid(a.n_chunks, a.n_kv_heads, a.batch);
  hipLaunchKernelGGL((attn_kernel<NQ, PW>), grid, dim3(256), lds, st, a);
}

template <int NQ>
static void launch_nq(const AttnArgs& a, hipStream_t st) {
  const int w = a.Wk > a.Wv ? a.Wk : a.Wv;
  if (w <= 8)
    launch_nq_pw<NQ, 8>(a, st);
  else if (w <= 16)
    launch_nq_pw<NQ, 16>(a, st);
  else
    launch_nq_pw<NQ, 0>(a, st);
}

hipError_t launch_attention(const AttnArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(qprep_kernel, dim3(a.n_kv_heads, a.batch), dim3(256), 0, st, a);
  switch ((a.n_qh + 3) / 4) {
    case 1: launch_nq<1>(a, st); break;
    case 2: launch_nq<2>(a, st); break;
    case 3: launch_nq<3>(a, st); break;
    default: launch_nq<4>(a, st); break;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(combine_kernel, dim3(a.n_q_heads, a.batch), dim3(1024), 0, st, a);
  return hipGetLastError();
}

}  // namespace spectra
