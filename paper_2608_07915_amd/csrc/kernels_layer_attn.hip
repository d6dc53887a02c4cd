// Decode-step attention over per-layer latents (App. E, Mode B; the latent spans all
// KV heads of a layer, d = n_kv_heads x 128, groups of 64). For query head h on KV head
// kv, k_t[kv rows] = (c_t + m_K) V_K[kv rows]^T, so the score is c_t . q~_h plus a
// constant that cancels in the softmax, with q~_h = q_h V_K[kv rows] a d-dimensional
// latent query; the output is (sum_t p_t c^V_t / sum_t p_t + m_V) V_V[kv rows]^T.
// Every query head reads the same per-token record, so one tile of records serves all
// heads of a sequence.
//
//   layer_qprep_kernel    q~ (scale and log2 e folded in) and its per-group sums;
//   layer_scores_kernel   scores of all heads for a chunk of 64-token tiles: codes
//                         (exact in fp16) times q~ as two fp16 parts on
//                         v_mfma_f32_16x16x32_f16, one kept group at a time, the
//                         token's scale and zero point applied after; chunk max and sum;
//   layer_values_kernel   p = exp2(s - max over all chunks), then per kept value group
//                         sum_t p_t s_t q_t on v_mfma_f32_16x16x32_f16 (weights as two
//                         fp16 parts, codes of eight consecutive tokens read from the
//                         word-major tile) and sum_t p_t z_t;
//   layer_combine_kernel  sums the chunk partials, divides by the softmax sum, adds m_V
//                         and applies V_V[kv rows]^T.
#include "device_common.hpp"
#include "kernels.hpp"
#include "layer.hpp"

namespace spectra_dev {

typedef __attribute__((__vector_size__(8 * sizeof(_Float16)))) _Float16 f16x8v;

constexpr int LA_H = 32;     // query heads per sequence (at most)
constexpr int LA_ROW = 68;   // words per staged record row (64 tokens + pad)
constexpr int LA_WMAX = 64;  // record words per tensor

// kept groups of a per-layer stream in slot order: group, width, first payload word
__device__ __forceinline__ int layer_slots(const uint8_t* __restrict__ bits_s, int ng, int* grp, int* bw, int* pay) {
  int n = 0;
  for (int g = 0; g < ng; ++g)
    if (bits_s[g] > 0) ++n;
  int off = n;
  int k = 0;
  for (int g = 0; g < ng; ++g) {
    const int b = bits_s[g];
    if (b > 0) {
      grp[k] = g;
      bw[k] = b;
      pay[k] = off;
      off += 2 * b;
      ++k;
    }
  }
  return n;
}

__device__ __forceinline__ bool layer_bits_ok(const uint8_t* __restrict__ bits_s, int ng, int W) {
  int used = 0;
  for (int g = 0; g < ng; ++g) {
    const int b = bits_s[g];
    if (b > 8) return false;
    if (b > 0) used += 1 + 2 * b;
  }
  return used <= W;
}

// ---------------------------------------------------------------------------
// q~[b][h][j] = scale log2(e) sum_i q[b][h][i] V_K[b][kv 128 + i][j] on kept groups
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void layer_qprep_kernel(LayerAttnArgs a) {
  __shared__ float qv[128];
  __shared__ float qtl[1024];
  const int h = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  const int d = a.d, ng = d / 64;
  const int kv = h / (a.n_q_heads / a.n_kv_heads);
  const uint8_t* bits_s = a.bits_k + (int64_t)b * ng;
  if (tid < 128) {
    const int64_t qi = ((int64_t)b * a.n_q_heads + h) * 128 + tid;
    qv[tid] = (a.q_f32 ? reinterpret_cast<const float*>(a.q)[qi] : bf2f(reinterpret_cast<const uint16_t*>(a.q)[qi])) *
              a.scale_log2;
  }
  __syncthreads();
  const float* V = a.basis_k + (int64_t)b * d * d + (int64_t)kv * 128 * d;
  for (int j = tid; j < d; j += 256) {
    float acc = 0.0f;
    if (bits_s[j >> 6] > 0)
      for (int i = 0; i < 128; ++i) acc = __builtin_fmaf(qv[i], V[(int64_t)i * d + j], acc);
    qtl[j] = acc;
    a.qt[((int64_t)b * a.n_q_heads + h) * d + j] = acc;
  }
  __syncthreads();
  if (tid < 16) {
    float s = 0.0f;
    if (tid < ng)
      for (int j = 0; j < 64; ++j) s += qtl[64 * tid + j];
    a.qsum[((int64_t)b * a.n_q_heads + h) * 16 + tid] = s;
  }
}

// ---------------------------------------------------------------------------
// Scores
// ---------------------------------------------------------------------------
__host__ __device__ constexpr int la_qp(int d) { return d + 8; }  // fp16 per staged query row
__host__ __device__ constexpr int la_off_rec(int d) { return 2 * LA_H * la_qp(d) * 2; }
__host__ __device__ constexpr int la_off_qs(int d, int Wk) { return la_off_rec(d) + Wk * LA_ROW * 4; }
__host__ __device__ constexpr int la_scores_lds(int d, int Wk) { return la_off_qs(d, Wk) + LA_H * 16 * 4 + 4 * LA_H * 2 * 4; }

__global__ __launch_bounds__(512) void layer_scores_kernel(LayerAttnArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint8_t lsm[];
  const int d = a.d, ng = d / 64, QP = la_qp(d), Wk = a.Wk;
  uint16_t* qa = reinterpret_cast<uint16_t*>(lsm);                       // [2][LA_H][QP]
  uint32_t* rec = reinterpret_cast<uint32_t*>(lsm + la_off_rec(d));      // [Wk][LA_ROW]
  float* qs = reinterpret_cast<float*>(lsm + la_off_qs(d, Wk));          // [LA_H][16]
  float* red = qs + LA_H * 16;                                           // [4][LA_H][2]
  __shared__ int sgrp[16], sbw[16], spay[16], snk;
  const int chunk = blockIdx.x, b = blockIdx.y;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, kg = lane >> 4, c16 = lane & 15;
  const int Hq = a.n_q_heads;
  const uint8_t* bits_s = a.bits_k + (int64_t)b * ng;
  const bool ok = layer_bits_ok(bits_s, ng, Wk);
  if (tid == 0) snk = ok ? layer_slots(bits_s, ng, sgrp, sbw, spay) : 0;
  __syncthreads();
  const int nk = snk;
  // kept coefficients of q~ as two fp16 parts, compacted by slot; group sums
  for (int e = tid; e < LA_H * nk * 64; e += 512) {
    const int h = e / (nk * 64), jj = e - h * (nk * 64);
    const float v = h < Hq ? a.qt[((int64_t)b * Hq + h) * d + 64 * sgrp[jj >> 6] + (jj & 63)] : 0.0f;
    const _Float16 hi = (_Float16)v;
    const _Float16 lo = (_Float16)(v - (float)hi);
    qa[h * QP + jj] = __builtin_bit_cast(uint16_t, hi);
    qa[(LA_H + h) * QP + jj] = __builtin_bit_cast(uint16_t, lo);
  }
  for (int e = tid; e < LA_H * 16; e += 512) {
    const int h = e >> 4, sl = e & 15;
    qs[e] = (h < Hq && sl < nk) ? a.qsum[((int64_t)b * Hq + h) * 16 + sgrp[sl]] : 0.0f;
  }

  const int64_t n_tiles = (a.n_tokens + 63) >> 6;
  const int64_t t_begin = (int64_t)chunk * a.tiles_per_chunk;
  const int64_t t_end = t_begin + a.tiles_per_chunk < n_tiles ? t_begin + a.tiles_per_chunk : n_tiles;
  const uint32_t* kp = a.packed_k + (int64_t)b * a.t_cap * Wk;
  const int hb = wave & 1, tb = wave >> 1;  // head block (16 heads), token block (16 tokens)
  float mloc[4], lloc[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    mloc[j] = -__builtin_inff();
    lloc[j] = 0.0f;
  }
  for (int64_t tt = t_begin; tt < t_end; ++tt) {
    __syncthreads();  // previous tile's reads done (and the prologue's writes visible)
    for (int k = tid; k < 64 * Wk; k += 512) rec[(k >> 6) * LA_ROW + (k & 63)] = kp[tt * 64 * Wk + k];
    __syncthreads();
    const int u = 16 * tb + c16;
    f32x4 S = {0.f, 0.f, 0.f, 0.f};
    for (int sl = 0; sl < nk; ++sl) {
      const int pay = spay[sl];
      const uint32_t m = rec[sl * LA_ROW + u];
      const float st = h2f(m), zt = h2f(m >> 16);
      f32x4 g = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        f16x8v bop;
        with_bits(sbw[sl], [&](auto bc) {
          constexpr int B = decltype(bc)::value;
          uint32_t cd[8];
          extract8<B>([&](int i) { return rec[(pay + i) * LA_ROW + u]; }, 32 * ks + 8 * kg, cd);
#pragma unroll
          for (int i = 0; i < 8; ++i) bop[i] = (_Float16)(float)cd[i];
        });
        const int col = sl * 64 + 32 * ks + 8 * kg;
        const f16x8v a0 = __builtin_bit_cast(f16x8v, *reinterpret_cast<const u32x4*>(qa + (16 * hb + c16) * QP + col));
        const f16x8v a1 = __builtin_bit_cast(f16x8v, *reinterpret_cast<const u32x4*>(qa + (LA_H + 16 * hb + c16) * QP + col));
        g = __builtin_amdgcn_mfma_f32_16x16x32_f16(a0, bop, g, 0, 0, 0);
        g = __builtin_amdgcn_mfma_f32_16x16x32_f16(a1, bop, g, 0, 0, 0);
      }
      // lane: heads 16 hb + 4 kg + j, token u
#pragma unroll
      for (int j = 0; j < 4; ++j) S[j] += st * g[j] + zt * qs[(16 * hb + 4 * kg + j) * 16 + sl];
    }
    const int64_t t = tt * 64 + u;
    if (t < a.n_tokens) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int h = 16 * hb + 4 * kg + j;
        if (h < Hq) {
          a.scores[((int64_t)b * Hq + h) * a.n_tokens + t] = S[j];
          const float x = S[j];
          if (x > mloc[j]) {
            lloc[j] = lloc[j] * __builtin_amdgcn_exp2f(mloc[j] - x) + 1.0f;
            mloc[j] = x;
          } else {
            lloc[j] += __builtin_amdgcn_exp2f(x - mloc[j]);
          }
        }
      }
    }
  }
  // chunk statistics: merge the 16 token lanes, then the four token-block wavefronts
#pragma unroll
  for (int j = 0; j < 4; ++j) {
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) {
      const float mo = __shfl_xor(mloc[j], o), lo = __shfl_xor(lloc[j], o);
      const float mn = __builtin_fmaxf(mloc[j], mo);
      const float l = (mloc[j] == -__builtin_inff() ? 0.0f : lloc[j] * __builtin_amdgcn_exp2f(mloc[j] - mn)) +
                      (mo == -__builtin_inff() ? 0.0f : lo * __builtin_amdgcn_exp2f(mo - mn));
      mloc[j] = mn;
      lloc[j] = l;
    }
  }
  __syncthreads();
  if (c16 == 0) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int h = 16 * hb + 4 * kg + j;
      red[(tb * LA_H + h) * 2] = mloc[j];
      red[(tb * LA_H + h) * 2 + 1] = lloc[j];
    }
  }
  __syncthreads();
  if (tid < Hq) {
    float m = -__builtin_inff();
    for (int q = 0; q < 4; ++q) m = __builtin_fmaxf(m, red[(q * LA_H + tid) * 2]);
    float l = 0.0f;
    for (int q = 0; q < 4; ++q) {
      const float mq = red[(q * LA_H + tid) * 2];
      if (mq != -__builtin_inff()) l += red[(q * LA_H + tid) * 2 + 1] * __builtin_amdgcn_exp2f(mq - m);
    }
    float* st = a.stats + (((int64_t)b * a.n_chunks + chunk) * Hq + tid) * 2;
    st[0] = m;
    st[1] = l;
  }
}

// ---------------------------------------------------------------------------
// Values
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(512) void layer_values_kernel(LayerAttnArgs a) {
  __shared__ __attribute__((aligned(16))) uint32_t rec[LA_WMAX * LA_ROW];
  __shared__ __attribute__((aligned(16))) float pl[LA_H * LA_ROW];
  __shared__ float mh[LA_H];
  __shared__ int sgrp[16], sbw[16], spay[16], snk;
  const int chunk = blockIdx.x, b = blockIdx.y;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, kg = lane >> 4, c16 = lane & 15;
  const int d = a.d, ng = d / 64, Wv = a.Wv, Hq = a.n_q_heads;
  const uint8_t* bits_s = a.bits_v + (int64_t)b * ng;
  const bool ok = layer_bits_ok(bits_s, ng, Wv) && layer_bits_ok(a.bits_k + (int64_t)b * ng, ng, a.Wk);
  if (tid == 0) snk = ok ? layer_slots(bits_s, ng, sgrp, sbw, spay) : 0;
  if (tid < LA_H) {
    float m = -__builtin_inff();
    if (tid < Hq)
      for (int c = 0; c < a.n_chunks; ++c) m = __builtin_fmaxf(m, a.stats[(((int64_t)b * a.n_chunks + c) * Hq + tid) * 2]);
    mh[tid] = m;
  }
  __syncthreads();
  const int nk = snk;
  const int hb = wave & 1, q4 = wave >> 1;  // head block; value slots q4, q4 + 4, q4 + 8, q4 + 12
  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[i][c] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int zh = tid & 31, zsl = tid >> 5;  // zero-point sums: thread -> (head, slot)
  float zacc = 0.0f;

  const int64_t n_tiles = (a.n_tokens + 63) >> 6;
  const int64_t t_begin = (int64_t)chunk * a.tiles_per_chunk;
  const int64_t t_end = t_begin + a.tiles_per_chunk < n_tiles ? t_begin + a.tiles_per_chunk : n_tiles;
  const uint32_t* vp = a.packed_v + (int64_t)b * a.t_cap * Wv;
  for (int64_t tt = (ok ? t_begin : t_end); tt < t_end; ++tt) {
    __syncthreads();
    for (int k = tid; k < 64 * Wv; k += 512) rec[(k >> 6) * LA_ROW + (k & 63)] = vp[tt * 64 * Wv + k];
    for (int e = tid; e < LA_H * 64; e += 512) {
      const int h = e >> 6, t = e & 63;
      const int64_t tok = tt * 64 + t;
      float p = 0.0f;
      if (h < Hq && tok < a.n_tokens && mh[h] != -__builtin_inff())
        p = __builtin_amdgcn_exp2f(a.scores[((int64_t)b * Hq + h) * a.n_tokens + tok] - mh[h]);
      pl[h * LA_ROW + t] = p;
    }
    __syncthreads();
    if (zsl < nk && zh < Hq) {
      float z = 0.0f;
      for (int t = 0; t < 64; ++t) z = __builtin_fmaf(pl[zh * LA_ROW + t], h2f(rec[zsl * LA_ROW + t] >> 16), z);
      zacc += z;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int sl = q4 + 4 * i;
      if (sl < nk) {
        const int B = sbw[sl], pay = spay[sl];
        const uint32_t M = (1u << B) - 1u;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          const int tk0 = 32 * ks + 8 * kg;
          // weights p_t s_t of head 16 hb + c16 for tokens tk0 .. tk0 + 7, two fp16 parts
          f16x8v whi, wlo;
          {
            const float* pr = pl + (16 * hb + c16) * LA_ROW + tk0;
            const f32x4 p0 = *reinterpret_cast<const f32x4*>(pr), p1 = *reinterpret_cast<const f32x4*>(pr + 4);
            const u32x4 m0 = *reinterpret_cast<const u32x4*>(rec + sl * LA_ROW + tk0);
            const u32x4 m1 = *reinterpret_cast<const u32x4*>(rec + sl * LA_ROW + tk0 + 4);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              const float w = (e < 4 ? p0[e] : p1[e - 4]) * h2f(e < 4 ? m0[e] : m1[e - 4]);
              const _Float16 hi = (_Float16)w;
              whi[e] = hi;
              wlo[e] = (_Float16)(w - (float)hi);
            }
          }
#pragma unroll
          for (int cb = 0; cb < 4; ++cb) {
            // codes of coefficient 16 cb + c16 for tokens tk0 .. tk0 + 7
            const int bit = (16 * cb + c16) * B, w = pay + (bit >> 5), sh = bit & 31;
            const bool two = sh + B > 32;
            const u32x4 l0 = *reinterpret_cast<const u32x4*>(rec + w * LA_ROW + tk0);
            const u32x4 l1 = *reinterpret_cast<const u32x4*>(rec + w * LA_ROW + tk0 + 4);
            u32x4 h0 = {0u, 0u, 0u, 0u}, h1 = {0u, 0u, 0u, 0u};
            if (two) {
              h0 = *reinterpret_cast<const u32x4*>(rec + (w + 1) * LA_ROW + tk0);
              h1 = *reinterpret_cast<const u32x4*>(rec + (w + 1) * LA_ROW + tk0 + 4);
            }
            f16x8v cv;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              cv[e] = (_Float16)(float)(__builtin_amdgcn_alignbit(h0[e], l0[e], sh) & M);
              cv[4 + e] = (_Float16)(float)(__builtin_amdgcn_alignbit(h1[e], l1[e], sh) & M);
            }
            acc[i][cb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(whi, cv, acc[i][cb], 0, 0, 0);
            acc[i][cb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(wlo, cv, acc[i][cb], 0, 0, 0);
          }
        }
      }
    }
  }
  // partials: lane holds rows (heads 16 hb + 4 kg + j) of column (coefficient 16 cb + c16)
  float* pb = a.part + ((int64_t)b * a.n_chunks + chunk) * Hq * (d + 16);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int sl = q4 + 4 * i;
    if (sl < nk) {
#pragma unroll
      for (int cb = 0; cb < 4; ++cb)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int h = 16 * hb + 4 * kg + j;
          if (h < Hq) pb[(int64_t)h * (d + 16) + 64 * sgrp[sl] + 16 * cb + c16] = acc[i][cb][j];
        }
    }
  }
  if (zsl < nk && zh < Hq) pb[(int64_t)zh * (d + 16) + d + sgrp[zsl]] = zacc;
}

// ---------------------------------------------------------------------------
// Combine and inverse rotation
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void layer_combine_kernel(LayerAttnArgs a) {
  __shared__ float cf[1024];
  __shared__ float part_o[2][128];
  __shared__ float ml[2];
  const int h = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  const int d = a.d, ng = d / 64, Hq = a.n_q_heads;
  const int kv = h / (Hq / a.n_kv_heads);
  const uint8_t* bv = a.bits_v + (int64_t)b * ng;
  const bool ok = layer_bits_ok(bv, ng, a.Wv) && layer_bits_ok(a.bits_k + (int64_t)b * ng, ng, a.Wk);
  if (tid == 0) {
    float m = -__builtin_inff();
    for (int c = 0; c < a.n_chunks; ++c) m = __builtin_fmaxf(m, a.stats[(((int64_t)b * a.n_chunks + c) * Hq + h) * 2]);
    float l = 0.0f;
    for (int c = 0; c < a.n_chunks; ++c) {
      const float* st = a.stats + (((int64_t)b * a.n_chunks + c) * Hq + h) * 2;
      if (st[0] != -__builtin_inff()) l += st[1] * __builtin_amdgcn_exp2f(st[0] - m);
    }
    ml[0] = m;
    ml[1] = l;
  }
  __syncthreads();
  const float inv_l = ml[1] > 0.0f ? 1.0f / ml[1] : 0.0f;
  const float* mv = a.mean_v + (int64_t)b * d;
  for (int j = tid; j < d; j += 256) {
    const int g = j >> 6;
    float c = 0.0f;
    if (ok && bv[g] > 0) {
      float s = 0.0f, z = 0.0f;
      for (int ch = 0; ch < a.n_chunks; ++ch) {
        const float* pb = a.part + (((int64_t)b * a.n_chunks + ch) * Hq + h) * (d + 16);
        s += pb[j];
        z += pb[d + g];
      }
      c = (s + z) * inv_l;
    }
    cf[j] = c + mv[j];
  }
  __syncthreads();
  const int i = tid & 127, half = tid >> 7;
  const float* vr = a.basis_v + (int64_t)b * d * d + (int64_t)(kv * 128 + i) * d;
  float acc = 0.0f;
  for (int j = half * (d / 2); j < (half + 1) * (d / 2); ++j) acc = __builtin_fmaf(cf[j], vr[j], acc);
  part_o[half][i] = acc;
  __syncthreads();
  if (tid < 128) a.out[((int64_t)b * Hq + h) * 128 + tid] = part_o[0][tid] + part_o[1][tid];
}

}  // namespace spectra_dev

namespace spectra {
using namespace spectra_dev;

// About 256 workgroups per pass over all sequences, at least four tiles per chunk.
int32_t layer_attention_chunks(int32_t batch, int64_t n_tokens, int32_t* tiles_per_chunk) {
  const int64_t n_tiles = (n_tokens + 63) / 64;
  const int64_t want = (256 + batch - 1) / batch;
  int64_t tpc = (n_tiles + want - 1) / want;
  if (tpc < 4) tpc = 4;
  *tiles_per_chunk = (int32_t)tpc;
  return (int32_t)((n_tiles + tpc - 1) / tpc);
}

size_t layer_attention_ws_floats(int32_t batch, int32_t n_q_heads, int32_t d, int64_t n_tokens) {
  int32_t tpc;
  const int64_t nch = layer_attention_chunks(batch, n_tokens, &tpc);
  const int64_t B = batch, H = n_q_heads;
  auto r64 = [](int64_t n) { return (n + 63) / 64 * 64; };  // 256-byte aligned sections
  return (size_t)(r64(B * H * d) + r64(B * H * 16) + r64(B * H * n_tokens) + r64(B * nch * H * 2) +
                  r64(B * nch * H * (d + 16)));
}

void layer_attention_ws_layout(LayerAttnArgs& a, float* ws) {
  a.n_chunks = layer_attention_chunks(a.batch, a.n_tokens, &a.tiles_per_chunk);
  const int64_t B = a.batch, H = a.n_q_heads;
  auto r64 = [](int64_t n) { return (n + 63) / 64 * 64; };
  a.qt = ws;
  a.qsum = a.qt + r64(B * H * a.d);
  a.scores = a.qsum + r64(B * H * 16);
  a.stats = a.scores + r64(B * H * a.n_tokens);
  a.part = a.stats + r64(B * a.n_chunks * H * 2);
}

size_t layer_scores_lds_bytes(int32_t d, int32_t Wk) { return (size_t)la_scores_lds(d, Wk); }

hipError_t launch_layer_attention(const LayerAttnArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(layer_qprep_kernel, dim3(a.n_q_heads, a.batch), dim3(256), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(layer_scores_kernel, dim3(a.n_chunks, a.batch), dim3(512), la_scores_lds(a.d, a.Wk), st, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(layer_values_kernel, dim3(a.n_chunks, a.batch), dim3(512), 0, st, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(layer_combine_kernel, dim3(a.n_q_heads, a.batch), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace spectra
