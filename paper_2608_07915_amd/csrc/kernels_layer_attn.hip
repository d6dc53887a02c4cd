// Decode-step attention over per-layer latents (App. E, Mode B; the latent spans all
// KV heads of a layer, d = n_kv_heads x 128, groups of 64). For query head h on KV head
// kv, k_t[kv rows] = (c_t + m_K) V_K[kv rows]^T, so the score is c_t . q~_h plus a
// constant that cancels in the softmax, with q~_h = q_h V_K[kv rows] a d-dimensional
// latent query; the output is (sum_t p_t c^V_t / sum_t p_t + m_V) V_V[kv rows]^T.
// Every query head reads the same per-token record, so one tile of records serves all
// heads of a sequence. With the square-root split (Eq. gsvd) the cached coordinate is
// c'_j = c_j f_j: the keys' 1 / f_j folds into the latent query (q~'_j = q~_j / f_j) and
// the values' sums are divided by f_j before m_V is added.
//
//   layer_qprep_kernel    q~ (scale and log2 e folded in) and its per-group sums;
//   layer_scores_kernel   scores of all heads for a chunk of 64-token tiles: codes
//                         (exact in fp16) times q~ as two fp16 parts on
//                         v_mfma_f32_16x16x32_f16, one kept group at a time, the
//                         token's scale and zero point applied after; chunk max and sum;
//   layer_stats_kernel    softmax max and sum of every head over the chunks;
//   layer_values_kernel   p = exp2(s - max over all chunks), then per kept value group
//                         sum_t p_t s_t q_t on v_mfma_f32_16x16x32_bf16 (weights as two
//                         bf16 parts, codes of eight consecutive tokens read from the
//                         word-major tile) and sum_t p_t z_t;
//   layer_combine_kernel  sums the chunk partials, divides by the softmax sum, adds m_V;
//   layer_rotate_kernel   applies V_V[kv rows]^T.
#include "device_common.hpp"
#include "kernels.hpp"
#include "layer.hpp"

namespace spectra_dev {

typedef __attribute__((__vector_size__(8 * sizeof(_Float16)))) _Float16 f16x8v;

constexpr int LA_H = 32;     // query heads per sequence (at most)
constexpr int LA_ROW = 68;   // words per staged record row (64 tokens + pad)
constexpr int LA_WMAX = 128;  // record words per tensor
// record words per tile staged through registers: the kernels are instantiated for
// records of at most 64 words and of at most LA_WMAX words
__host__ __device__ constexpr int la_prefetch_words(int W) { return W <= 64 ? 64 : LA_WMAX; }

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
// grid (heads, sequences, d / 256): thread -> one coefficient j, four groups per workgroup
__global__ __launch_bounds__(256) void layer_qprep_kernel(LayerAttnArgs a) {
  __shared__ float qv[128];
  __shared__ float qtl[256];
  __shared__ int slot_of[16];  // kept rank of each group
  const int h = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  const int d = a.d, ng = d / 64;
  const int j = 256 * blockIdx.z + tid;
  const int kv = h / (a.n_q_heads / a.n_kv_heads);
  const uint8_t* bits_s = a.bits_k + (int64_t)b * ng;
  if (tid == 0) {
    int n = 0;
    for (int g = 0; g < ng; ++g) {
      slot_of[g] = n;
      n += bits_s[g] > 0 ? 1 : 0;
    }
  }
  if (tid < 128) {
    const int64_t qi = ((int64_t)b * a.n_q_heads + h) * 128 + tid;
    qv[tid] = (a.q_f32 ? reinterpret_cast<const float*>(a.q)[qi] : bf2f(reinterpret_cast<const uint16_t*>(a.q)[qi])) *
              a.scale_log2;
  }
  __syncthreads();
  const float* V = a.basis_k + (int64_t)b * d * d + (int64_t)kv * 128 * d + j;
  float acc = 0.0f;
  if (j < d && bits_s[j >> 6] > 0) {
    float part[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
    for (int i = 0; i < 128; i += 8)
#pragma unroll
      for (int r = 0; r < 8; ++r) part[r] = __builtin_fmaf(qv[i + r], V[(int64_t)(i + r) * d], part[r]);
    acc = ((part[0] + part[1]) + (part[2] + part[3])) + ((part[4] + part[5]) + (part[6] + part[7]));
    if (a.lscale_k) acc /= a.lscale_k[(int64_t)b * d + j];
  }
  qtl[tid] = acc;
  if (j < d) {
    a.qt[((int64_t)b * a.n_q_heads + h) * d + j] = acc;
    const int g = j >> 6;
    if (bits_s[g] > 0) {  // fp16 parts for the score pass, at the group's kept slot
      const int slot = slot_of[g];
      const _Float16 hi = (_Float16)acc;
      const _Float16 lo = (_Float16)(acc - (float)hi);
      uint16_t* qh = a.qh + (int64_t)b * 2 * LA_H * d;
      qh[(int64_t)h * d + 64 * slot + (j & 63)] = __builtin_bit_cast(uint16_t, hi);
      qh[(int64_t)(LA_H + h) * d + 64 * slot + (j & 63)] = __builtin_bit_cast(uint16_t, lo);
    }
  }
  __syncthreads();
  // group sums (only the groups of this workgroup's coefficients; the score pass reads kept groups only)
  if (tid < 4 && 4 * (int)blockIdx.z + tid < ng) {
    float s = 0.0f;
    for (int jj = 0; jj < 64; ++jj) s += qtl[64 * tid + jj];
    a.qsum[((int64_t)b * a.n_q_heads + h) * 16 + 4 * blockIdx.z + tid] = s;
  }
}

// ---------------------------------------------------------------------------
// Scores
// ---------------------------------------------------------------------------
// A score workgroup takes NHB blocks of 16 query heads: both (NHB = 2), or, when the
// latent queries of 32 heads and the record rows would not fit the LDS together
// (d = 1024 with records of more than ~100 words), one (NHB = 1, blockIdx.z selects it).
__host__ __device__ constexpr int la_qp(int d) { return d + 8; }  // fp16 per staged query row
constexpr int LA_QSP = 17;  // floats per row of the group sums (16 slots + pad: the rows of four heads read together lie on distinct banks)
__host__ __device__ constexpr int la_off_rec(int d, int nhb) { return 2 * 16 * nhb * la_qp(d) * 2; }
// the record rows also hold the slot halves' scores of a tile ([4][64][8] floats) once read
__host__ __device__ constexpr int la_rec_bytes(int Wk) { return Wk * LA_ROW * 4 > 4 * 64 * 8 * 4 ? Wk * LA_ROW * 4 : 4 * 64 * 8 * 4; }
__host__ __device__ constexpr int la_off_qs(int d, int Wk, int nhb) { return la_off_rec(d, nhb) + la_rec_bytes(Wk); }
__host__ __device__ constexpr int la_scores_lds(int d, int Wk, int nhb) {
  return la_off_qs(d, Wk, nhb) + LA_H * LA_QSP * 4 + 4 * LA_H * 2 * 4;
}

template <int NHB, int WP>
__global__ __launch_bounds__(512) void layer_scores_kernel(LayerAttnArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint8_t lsm[];
  const int d = a.d, ng = d / 64, QP = la_qp(d), Wk = a.Wk;
  uint16_t* qa = reinterpret_cast<uint16_t*>(lsm);                       // [2][16 NHB][QP]
  uint32_t* rec = reinterpret_cast<uint32_t*>(lsm + la_off_rec(d, NHB)); // [Wk][LA_ROW]
  float* qs = reinterpret_cast<float*>(lsm + la_off_qs(d, Wk, NHB));     // [LA_H][LA_QSP]
  float* red = qs + LA_H * LA_QSP;                                       // [4][LA_H][2]
  __shared__ int sgrp[16], sbw[16], spay[16], snk;
  const int chunk = blockIdx.x, b = blockIdx.y;
  const int hb0 = NHB == 2 ? 0 : (int)blockIdx.z;  // first head block of this workgroup
  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63, kg = lane >> 4, c16 = lane & 15;
  const int Hq = a.n_q_heads;
  const uint8_t* bits_s = a.bits_k + (int64_t)b * ng;
  const bool ok = layer_bits_ok(bits_s, ng, Wk);
  if (tid == 0) snk = ok ? layer_slots(bits_s, ng, sgrp, sbw, spay) : 0;
  __syncthreads();
  const int nk = __builtin_amdgcn_readfirstlane(snk);
  // kept coefficients of q~ as two fp16 parts, compacted by slot; group sums
  // copied as written by the query pass (16-byte pieces, eight in flight per thread);
  // rows of heads past n_q_heads are zero
  {
    // staged row = part * 16 NHB + local head; source row = part * LA_H + 16 hb0 + local head
    const uint16_t* qh = a.qh + (int64_t)b * 2 * LA_H * d;
    const int pieces = nk * 8;  // 16-byte pieces per row
    for (int i0 = 0; i0 < (2 * 16 * NHB * 16 * 8) / 512; i0 += 8) {
      u32x4 v[8];
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        const int e = tid + 512 * (i0 + r), row = e >> 7, pc = e & 127;
        const int part = row / (16 * NHB), h = 16 * hb0 + row % (16 * NHB);
        v[r] = (h < Hq && pc < pieces) ? *reinterpret_cast<const u32x4*>(qh + (int64_t)(part * LA_H + h) * d + 8 * pc)
                                       : u32x4{0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        const int e = tid + 512 * (i0 + r), row = e >> 7, pc = e & 127;
        if (pc < pieces) *reinterpret_cast<u32x4*>(qa + row * QP + 8 * pc) = v[r];
      }
    }
  }
  for (int e = tid; e < LA_H * 16; e += 512) {
    const int h = e >> 4, sl = e & 15;
    qs[h * LA_QSP + sl] = (h < Hq && sl < nk) ? a.qsum[((int64_t)b * Hq + h) * 16 + sgrp[sl]] : 0.0f;
  }

  const int64_t n_tiles = (a.n_tokens + 63) >> 6;
  const int64_t t_begin = (int64_t)chunk * a.tiles_per_chunk;
  const int64_t t_end = t_begin + a.tiles_per_chunk < n_tiles ? t_begin + a.tiles_per_chunk : n_tiles;
  const uint32_t* kp = a.packed_k + (int64_t)b * a.t_cap * Wk;
  // wavefront: token block tb (16 tokens), both head blocks, kept slots sh, sh + 2, ...
  const int tb = wave & 3, sh = wave >> 2;
  float mloc[8], lloc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    mloc[j] = -__builtin_inff();
    lloc[j] = 0.0f;
  }
  constexpr int PF = 64 * WP / 512;  // record words per thread and tile
  uint32_t pre[PF];
  auto load_tile = [&](int64_t tt) {
#pragma unroll
    for (int i = 0; i < PF; ++i) {
      const int k = tid + 512 * i;
      pre[i] = k < 64 * Wk ? kp[tt * 64 * Wk + k] : 0u;
    }
  };
  float* sred = reinterpret_cast<float*>(rec);  // [4 token blocks][64 lanes][8], after the tile's products
  if (t_begin < t_end) load_tile(t_begin);
  for (int64_t tt = t_begin; tt < t_end; ++tt) {
    __syncthreads();  // previous tile's reads done (and the prologue's writes visible)
#pragma unroll
    for (int i = 0; i < PF; ++i) {
      const int k = tid + 512 * i;
      if (k < 64 * Wk) rec[(k >> 6) * LA_ROW + (k & 63)] = pre[i];
    }
    __syncthreads();
    if (tt + 1 < t_end) load_tile(tt + 1);
    const int u = 16 * tb + c16;
    f32x4 S[NHB];
#pragma unroll
    for (int hb = 0; hb < NHB; ++hb) S[hb] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int sl = sh; sl < nk; sl += 2) {
      // slot tables are uniform: scalar registers, scalar branches on the width
      const int pay = __builtin_amdgcn_readfirstlane(spay[sl]);
      const int bw = __builtin_amdgcn_readfirstlane(sbw[sl]);
      const uint32_t m = rec[sl * LA_ROW + u];
      const float st = h2f(m), zt = h2f(m >> 16);
      f32x4 g[NHB];
#pragma unroll
      for (int hb = 0; hb < NHB; ++hb) g[hb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        f16x8v bop;
        with_bits(bw, [&](auto bc) {
          constexpr int B = decltype(bc)::value;
          uint32_t cd[8];
          extract8<B>([&](int i) { return rec[(pay + i) * LA_ROW + u]; }, 32 * ks + 8 * kg, cd);
#pragma unroll
          for (int i = 0; i < 8; ++i) bop[i] = (_Float16)(float)cd[i];
        });
        const int col = sl * 64 + 32 * ks + 8 * kg;
#pragma unroll
        for (int hb = 0; hb < NHB; ++hb) {
          const f16x8v a0 = __builtin_bit_cast(f16x8v, *reinterpret_cast<const u32x4*>(qa + (16 * hb + c16) * QP + col));
          const f16x8v a1 =
              __builtin_bit_cast(f16x8v, *reinterpret_cast<const u32x4*>(qa + (16 * NHB + 16 * hb + c16) * QP + col));
          g[hb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a0, bop, g[hb], 0, 0, 0);
          g[hb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a1, bop, g[hb], 0, 0, 0);
        }
      }
      // lane: heads 16 (hb0 + hb) + 4 kg + j, token u
#pragma unroll
      for (int hb = 0; hb < NHB; ++hb)
#pragma unroll
        for (int j = 0; j < 4; ++j) S[hb][j] += st * g[hb][j] + zt * qs[(16 * (hb0 + hb) + 4 * kg + j) * LA_QSP + sl];
    }
    // the two slot halves meet in LDS (over the record rows, whose reads are done)
    __syncthreads();
    if (sh == 1) {
#pragma unroll
      for (int hb = 0; hb < NHB; ++hb) *reinterpret_cast<f32x4*>(&sred[(tb * 64 + lane) * 8 + 4 * hb]) = S[hb];
    }
    __syncthreads();
    if (sh == 0) {
      const int64_t t = tt * 64 + u;
#pragma unroll
      for (int hb = 0; hb < NHB; ++hb) {
        const f32x4 o4 = *reinterpret_cast<const f32x4*>(&sred[(tb * 64 + lane) * 8 + 4 * hb]);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int h = 16 * (hb0 + hb) + 4 * kg + j;
          const float x = S[hb][j] + o4[j];
          if (t < a.n_tokens && h < Hq) {
            a.scores[((int64_t)b * Hq + h) * a.n_tokens + t] = x;
            const int q = 4 * hb + j;
            if (x > mloc[q]) {
              lloc[q] = lloc[q] * __builtin_amdgcn_exp2f(mloc[q] - x) + 1.0f;
              mloc[q] = x;
            } else {
              lloc[q] += __builtin_amdgcn_exp2f(x - mloc[q]);
            }
          }
        }
      }
    }
  }
  // chunk statistics: merge the 16 token lanes, then the four token-block wavefronts
#pragma unroll
  for (int j = 0; j < 8; ++j) {
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
  if (c16 == 0 && sh == 0) {
#pragma unroll
    for (int q = 0; q < 4 * NHB; ++q) {
      const int h = 16 * (hb0 + (q >> 2)) + 4 * kg + (q & 3);
      red[(tb * LA_H + h) * 2] = mloc[q];
      red[(tb * LA_H + h) * 2 + 1] = lloc[q];
    }
  }
  __syncthreads();
  // this workgroup's heads only (with NHB = 1 the other block is another workgroup's)
  if (tid < Hq && tid >= 16 * hb0 && tid < 16 * (hb0 + NHB)) {
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
// Softmax max and sum of every head over all chunks (one workgroup per head)
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void layer_stats_kernel(LayerAttnArgs a) {
  __shared__ float rm[4], rl[4];
  const int h = blockIdx.x, b = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int Hq = a.n_q_heads;
  float m = -__builtin_inff(), l = 0.0f;
  for (int c = tid; c < a.n_chunks; c += 256) {
    const float* st = a.stats + (((int64_t)b * a.n_chunks + c) * Hq + h) * 2;
    const float mc = st[0], lc = st[1];
    if (mc != -__builtin_inff()) {
      const float mn = __builtin_fmaxf(m, mc);
      l = (m == -__builtin_inff() ? 0.0f : l * __builtin_amdgcn_exp2f(m - mn)) + lc * __builtin_amdgcn_exp2f(mc - mn);
      m = mn;
    }
  }
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const float mo = __shfl_xor(m, o), lo = __shfl_xor(l, o);
    const float mn = __builtin_fmaxf(m, mo);
    l = (m == -__builtin_inff() ? 0.0f : l * __builtin_amdgcn_exp2f(m - mn)) +
        (mo == -__builtin_inff() ? 0.0f : lo * __builtin_amdgcn_exp2f(mo - mn));
    m = mn;
  }
  if (lane == 0) {
    rm[wave] = m;
    rl[wave] = l;
  }
  __syncthreads();
  if (tid == 0) {
    float mm = -__builtin_inff();
    for (int w = 0; w < 4; ++w) mm = __builtin_fmaxf(mm, rm[w]);
    float ll = 0.0f;
    for (int w = 0; w < 4; ++w)
      if (rm[w] != -__builtin_inff()) ll += rl[w] * __builtin_amdgcn_exp2f(rm[w] - mm);
    a.ml[((int64_t)b * Hq + h) * 2] = mm;
    a.ml[((int64_t)b * Hq + h) * 2 + 1] = ll;
  }
}

// ---------------------------------------------------------------------------
// Values: one workgroup per (token chunk, block of 16 query heads, sequence); wavefront w
// takes kept value slots w and w + 8
// ---------------------------------------------------------------------------
template <int WP>
__global__ __launch_bounds__(512) void layer_values_kernel(LayerAttnArgs a) {
  __shared__ __attribute__((aligned(16))) uint32_t rec[WP * LA_ROW];
  __shared__ __attribute__((aligned(16))) float pl[16 * LA_ROW];
  __shared__ float mh[LA_H];
  __shared__ int sgrp[16], sbw[16], spay[16], snk;
  const int chunk = blockIdx.x, hbk = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63, kg = lane >> 4, c16 = lane & 15;
  const int d = a.d, ng = d / 64, Wv = a.Wv, Hq = a.n_q_heads;
  const uint8_t* bits_s = a.bits_v + (int64_t)b * ng;
  const bool ok = layer_bits_ok(bits_s, ng, Wv) && layer_bits_ok(a.bits_k + (int64_t)b * ng, ng, a.Wk);
  if (tid == 0) snk = ok ? layer_slots(bits_s, ng, sgrp, sbw, spay) : 0;
  if (tid < LA_H) mh[tid] = tid < Hq ? a.ml[((int64_t)b * Hq + tid) * 2] : -__builtin_inff();
  __syncthreads();
  const int nk = __builtin_amdgcn_readfirstlane(snk);
  // workgroup: heads 16 hbk .. 16 hbk + 15; wavefront: kept slots wave, wave + 8
  const int hb = hbk;
  f32x4 acc[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[i][c] = f32x4{0.f, 0.f, 0.f, 0.f};
  // zero-point sums: thread -> (head 16 hbk + (tid & 15), slot (tid >> 4) & 15, tokens 32 (tid >> 8) ..)
  const int zhl = tid & 15, zh = 16 * hbk + zhl, zsl = (tid >> 4) & 15, zq = tid >> 8;
  __shared__ float zred[2][256];
  float zacc = 0.0f;

  const int64_t n_tiles = (a.n_tokens + 63) >> 6;
  const int64_t t_begin = (int64_t)chunk * a.v_tiles_per_chunk;
  const int64_t t_end = t_begin + a.v_tiles_per_chunk < n_tiles ? t_begin + a.v_tiles_per_chunk : n_tiles;
  const uint32_t* vp = a.packed_v + (int64_t)b * a.t_cap * Wv;
  constexpr int PF = 64 * WP / 512;            // record words per thread and tile
  constexpr int PS = 16 * 64 / 512;            // scores per thread and tile
  uint32_t pre[PF];
  float spre[PS];
  // Slots past n_tokens in the last tile get weight 0; their metadata words are
  // staged as 0 so that whatever the cache holds there (a NaN scale or zero-point)
  // never enters the products (0 * NaN would reach every head through the MFMA).
  auto load_tile = [&](int64_t tt) {
#pragma unroll
    for (int i = 0; i < PF; ++i) {
      const int k = tid + 512 * i;
      const bool meta_past_end = (k >> 6) < nk && tt * 64 + (k & 63) >= a.n_tokens;
      pre[i] = (k < 64 * Wv && !meta_past_end) ? vp[tt * 64 * Wv + k] : 0u;
    }
#pragma unroll
    for (int i = 0; i < PS; ++i) {
      const int e = tid + 512 * i, h = 16 * hbk + (e >> 6);
      const int64_t tok = tt * 64 + (e & 63);
      spre[i] = (h < Hq && tok < a.n_tokens) ? a.scores[((int64_t)b * Hq + h) * a.n_tokens + tok] : -__builtin_inff();
    }
  };
  if (ok && t_begin < t_end) load_tile(t_begin);
  for (int64_t tt = (ok ? t_begin : t_end); tt < t_end; ++tt) {
    __syncthreads();
#pragma unroll
    for (int i = 0; i < PF; ++i) {
      const int k = tid + 512 * i;
      if (k < 64 * Wv) rec[(k >> 6) * LA_ROW + (k & 63)] = pre[i];
    }
#pragma unroll
    for (int i = 0; i < PS; ++i) {
      const int e = tid + 512 * i, hl = e >> 6, h = 16 * hbk + hl;
      const float x = spre[i];
      pl[hl * LA_ROW + (e & 63)] = (x != -__builtin_inff() && mh[h] != -__builtin_inff()) ? __builtin_amdgcn_exp2f(x - mh[h]) : 0.0f;
    }
    __syncthreads();
    if (tt + 1 < t_end) load_tile(tt + 1);
    if (zsl < nk && zh < Hq) {
      const float* pr = pl + zhl * LA_ROW + 32 * zq;
      const uint32_t* mr = rec + zsl * LA_ROW + 32 * zq;
      float z = 0.0f;
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const f32x4 pv = *reinterpret_cast<const f32x4*>(pr + 4 * q);
        const u32x4 mv = *reinterpret_cast<const u32x4*>(mr + 4 * q);
#pragma unroll
        for (int e = 0; e < 4; ++e) z = __builtin_fmaf(pv[e], h2f(mv[e] >> 16), z);
      }
      zacc += z;
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int sl = wave + 8 * i;
      if (sl < nk) {
        const int B = __builtin_amdgcn_readfirstlane(sbw[sl]), pay = __builtin_amdgcn_readfirstlane(spay[sl]);
        const uint32_t M = (1u << B) - 1u;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          const int tk0 = 32 * ks + 8 * kg;
          // weights p_t s_t of head 16 hb + c16 for tokens tk0 .. tk0 + 7 as two bf16 parts:
          // the fp32 exponent range (p_t s_t spans many decades below 1) and 16 significant
          // bits (relative error below 2^-17 per weight; a third part changed the output by
          // 1e-6 relative and cost 7% of the call)
          bf16x8 wp[2];
          {
            const float* pr = pl + c16 * LA_ROW + tk0;
            const f32x4 p0 = *reinterpret_cast<const f32x4*>(pr), p1 = *reinterpret_cast<const f32x4*>(pr + 4);
            const u32x4 m0 = *reinterpret_cast<const u32x4*>(rec + sl * LA_ROW + tk0);
            const u32x4 m1 = *reinterpret_cast<const u32x4*>(rec + sl * LA_ROW + tk0 + 4);
            uint32_t q0[8], q1[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              const float wv = (e < 4 ? p0[e] : p1[e - 4]) * h2f(e < 4 ? m0[e] : m1[e - 4]);
              q0[e] = f2bf(wv);
              q1[e] = f2bf(wv - bf2f(q0[e]));
            }
            wp[0] = as_bf16x8(u32x4{pack2(q0[0], q0[1]), pack2(q0[2], q0[3]), pack2(q0[4], q0[5]), pack2(q0[6], q0[7])});
            wp[1] = as_bf16x8(u32x4{pack2(q1[0], q1[1]), pack2(q1[2], q1[3]), pack2(q1[4], q1[5]), pack2(q1[6], q1[7])});
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
            uint32_t cd[8];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              cd[e] = __builtin_amdgcn_alignbit(h0[e], l0[e], sh) & M;
              cd[4 + e] = __builtin_amdgcn_alignbit(h1[e], l1[e], sh) & M;
            }
            const bf16x8 cv = as_bf16x8(u32x4{int_to_bf16_pair(cd[0], cd[1]), int_to_bf16_pair(cd[2], cd[3]),
                                              int_to_bf16_pair(cd[4], cd[5]), int_to_bf16_pair(cd[6], cd[7])});
#pragma unroll
            for (int q = 0; q < 2; ++q)
              acc[i][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wp[q], cv, acc[i][cb], 0, 0, 0);
          }
        }
      }
    }
  }
  // partials: lane holds rows (heads 16 hb + 4 kg + j) of column (coefficient 16 cb + c16)
  float* pb = a.part + ((int64_t)b * a.nv_chunks + chunk) * Hq * (d + 16);
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int sl = wave + 8 * i;
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
  zred[zq][tid & 255] = zacc;
  __syncthreads();
  if (tid < 256 && zsl < nk && zh < Hq) pb[(int64_t)zh * (d + 16) + d + sgrp[zsl]] = zred[0][tid] + zred[1][tid];
}

// ---------------------------------------------------------------------------
// Combine: c[j] = (sum over value chunks of the coefficient sums + zero-point sums)
// / softmax sum + m_V[j], written over q~ (no longer needed); grid (heads, sequences,
// d / 64 groups)
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void layer_combine_kernel(LayerAttnArgs a) {
  // thread -> (coefficient 64 z + (tid & 63), every fourth chunk from tid >> 6): four short
  // chains of loads instead of one long one, summed in LDS in a fixed order
  __shared__ float ps[4][64], pz[4][64];
  const int h = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  const int d = a.d, ng = d / 64, Hq = a.n_q_heads;
  const int j = 64 * blockIdx.z + (tid & 63), part = tid >> 6;
  const uint8_t* bv = a.bits_v + (int64_t)b * ng;
  const bool ok = layer_bits_ok(bv, ng, a.Wv) && layer_bits_ok(a.bits_k + (int64_t)b * ng, ng, a.Wk);
  const int g = j >> 6;  // one group per workgroup
  const bool kept = ok && bv[g] > 0;
  float s0 = 0.f, s1 = 0.f, z0 = 0.f, z1 = 0.f;
  if (kept) {
    const float* pb = a.part + ((int64_t)b * a.nv_chunks * Hq + h) * (d + 16);
    const int64_t cstride = (int64_t)Hq * (d + 16);
    int ch = part;
#pragma unroll 2
    for (; ch + 4 < a.nv_chunks; ch += 8) {
      s0 += pb[ch * cstride + j];
      z0 += pb[ch * cstride + d + g];
      s1 += pb[(ch + 4) * cstride + j];
      z1 += pb[(ch + 4) * cstride + d + g];
    }
    if (ch < a.nv_chunks) {
      s0 += pb[ch * cstride + j];
      z0 += pb[ch * cstride + d + g];
    }
  }
  ps[part][tid & 63] = s0 + s1;
  pz[part][tid & 63] = z0 + z1;
  __syncthreads();
  if (tid < 64) {
    const float l = a.ml[((int64_t)b * Hq + h) * 2 + 1];
    const float inv_l = l > 0.0f ? 1.0f / l : 0.0f;
    float c = 0.0f;
    if (kept)
      c = (((ps[0][tid] + ps[1][tid]) + (ps[2][tid] + ps[3][tid])) + ((pz[0][tid] + pz[1][tid]) + (pz[2][tid] + pz[3][tid]))) *
          inv_l;
    if (a.lscale_v) c /= a.lscale_v[(int64_t)b * d + j];
    a.qt[((int64_t)b * Hq + h) * d + j] = c + a.mean_v[(int64_t)b * d + j];
  }
}

// ---------------------------------------------------------------------------
// Inverse rotation: out[i] = sum_j c[j] V_V[kv 128 + i][j]; grid (heads, sequences, 16):
// workgroup z takes rows 8 z .. 8 z + 7, two per wavefront, each row read by the whole
// wavefront (d / 64 values per lane), then a wavefront sum
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void layer_rotate_kernel(LayerAttnArgs a) {
  const int h = blockIdx.x, b = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int d = a.d, Hq = a.n_q_heads;
  const int kv = h / (Hq / a.n_kv_heads);
  const float* cfv = a.qt + ((int64_t)b * Hq + h) * d;
  float cl[16];
#pragma unroll
  for (int k = 0; k < 16; ++k) cl[k] = (64 * k + lane < d) ? cfv[64 * k + lane] : 0.0f;
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    const int i = 8 * blockIdx.z + 2 * wave + r;
    const float* vr = a.basis_v + (int64_t)b * d * d + (int64_t)(kv * 128 + i) * d;
    float acc = 0.0f;
#pragma unroll
    for (int k = 0; k < 16; ++k)
      if (64 * k + lane < d) acc = __builtin_fmaf(cl[k], vr[64 * k + lane], acc);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o);
    if (lane == 0) a.out[((int64_t)b * Hq + h) * 128 + i] = acc;
  }
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

// Value pass: about 256 workgroups over (chunk, head block of 16, sequence), at least 8
// tiles each.
int32_t layer_value_chunks(int32_t batch, int64_t n_tokens, int32_t* tiles_per_chunk) {
  const int64_t n_tiles = (n_tokens + 63) / 64;
  const int64_t want = (128 + batch - 1) / batch;
  int64_t tpc = (n_tiles + want - 1) / want;
  if (tpc < 8) tpc = 8;
  *tiles_per_chunk = (int32_t)tpc;
  return (int32_t)((n_tiles + tpc - 1) / tpc);
}

size_t layer_attention_ws_floats(int32_t batch, int32_t n_q_heads, int32_t d, int64_t n_tokens) {
  int32_t tpc;
  const int64_t nch = layer_attention_chunks(batch, n_tokens, &tpc);
  const int64_t nv = layer_value_chunks(batch, n_tokens, &tpc);
  const int64_t B = batch, H = n_q_heads;
  auto r64 = [](int64_t n) { return (n + 63) / 64 * 64; };  // 256-byte aligned sections
  return (size_t)(r64(B * H * d) + r64(B * LA_H * d) + r64(B * H * 16) + r64(B * H * 2) + r64(B * H * n_tokens) +
                  r64(B * nch * H * 2) + r64(B * nv * H * (d + 16)));
}

void layer_attention_ws_layout(LayerAttnArgs& a, float* ws) {
  a.n_chunks = layer_attention_chunks(a.batch, a.n_tokens, &a.tiles_per_chunk);
  a.nv_chunks = layer_value_chunks(a.batch, a.n_tokens, &a.v_tiles_per_chunk);
  const int64_t B = a.batch, H = a.n_q_heads;
  auto r64 = [](int64_t n) { return (n + 63) / 64 * 64; };
  a.qt = ws;
  a.qh = reinterpret_cast<uint16_t*>(a.qt + r64(B * H * a.d));  // 2 x 32 x d halves = 32 x d floats
  a.qsum = a.qt + r64(B * H * a.d) + r64(B * LA_H * a.d);
  a.ml = a.qsum + r64(B * H * 16);
  a.scores = a.ml + r64(B * H * 2);
  a.stats = a.scores + r64(B * H * a.n_tokens);
  a.part = a.stats + r64(B * a.n_chunks * H * 2);
}

// the score pass with one head block per workgroup (the smaller LDS footprint)
size_t layer_scores_lds_bytes(int32_t d, int32_t Wk) { return (size_t)la_scores_lds(d, Wk, 1); }

hipError_t launch_layer_attention(const LayerAttnArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(layer_qprep_kernel, dim3(a.n_q_heads, a.batch, (a.d + 255) / 256), dim3(256), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  int dev = 0, lds_max = 0;
  e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
  if (e != hipSuccess) return e;
  const bool k_wide = la_prefetch_words(a.Wk) > 64, v_wide = la_prefetch_words(a.Wv) > 64;
  if ((size_t)la_scores_lds(a.d, a.Wk, 2) <= (size_t)lds_max) {
    if (k_wide)
      hipLaunchKernelGGL((layer_scores_kernel<2, LA_WMAX>), dim3(a.n_chunks, a.batch), dim3(512),
                         la_scores_lds(a.d, a.Wk, 2), st, a);
    else
      hipLaunchKernelGGL((layer_scores_kernel<2, 64>), dim3(a.n_chunks, a.batch), dim3(512), la_scores_lds(a.d, a.Wk, 2),
                         st, a);
  } else {
    if (k_wide)
      hipLaunchKernelGGL((layer_scores_kernel<1, LA_WMAX>), dim3(a.n_chunks, a.batch, 2), dim3(512),
                         la_scores_lds(a.d, a.Wk, 1), st, a);
    else
      hipLaunchKernelGGL((layer_scores_kernel<1, 64>), dim3(a.n_chunks, a.batch, 2), dim3(512),
                         la_scores_lds(a.d, a.Wk, 1), st, a);
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(layer_stats_kernel, dim3(a.n_q_heads, a.batch), dim3(256), 0, st, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (v_wide)
    hipLaunchKernelGGL(layer_values_kernel<LA_WMAX>, dim3(a.nv_chunks, 2, a.batch), dim3(512), 0, st, a);
  else
    hipLaunchKernelGGL(layer_values_kernel<64>, dim3(a.nv_chunks, 2, a.batch), dim3(512), 0, st, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(layer_combine_kernel, dim3(a.n_q_heads, a.batch, a.d / 64), dim3(256), 0, st, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(layer_rotate_kernel, dim3(a.n_q_heads, a.batch, 16), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace spectra
