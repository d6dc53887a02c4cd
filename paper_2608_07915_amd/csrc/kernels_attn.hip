// Decode-step attention read straight from the packed caches (App. E, Mode B).
//
//   q'_h   = scale * log2(e) * q_h V_K          (once per step, qprep_kernel)
//   score  = sum_G s_tG <q'_G, code_tG> + z_tG sum_{j in G} q'_j
//            (the constant q' . m_K cancels in the softmax and is dropped)
//   a_h    = sum_t p_ht (z_tG + s_tG code_tj)     over kept value coefficients
//   out_h  = (a_h / l_h + m_V) V_V^T              (once per output, combine_kernel)
//
// The two per-token contractions over the kept latent coefficients are the
// products the paper calls the dominant matrix multiplies of latent attention;
// they run on MFMA:
//   * scores: v_mfma_f32_4x4x4f16 with 16 blocks; lane = token, block rows = 4 query
//     heads; codes are exact in fp16 and q' is split into two fp16 parts (hi + lo,
//     pre-scaled by a power of two) so the dot products are ~fp32-accurate;
//   * values: v_mfma_f32_16x16x32_bf16 with rows = query heads, K = 32 tokens,
//     columns = 16 coefficients; the softmax weights p*s go in as bf16 hi + lo.
// Work is split over token chunks (flash-decoding style); each wavefront streams
// one chunk of 64-token record tiles and writes a log-sum-exp partial.
#include "device_common.hpp"
#include "kernels.hpp"

namespace spectra_dev {

constexpr int PART = 136;  // floats per (chunk, query head) partial: m, l, Z[4], pad[2], acc[128]
constexpr int QA_QUAD = 4 * 8 * 2 * 4 * 2;   // uint32 of K-side MFMA A operands per head quad
constexpr int QP_QA = 4 * QA_QUAD;             // ... for up to 16 query heads per kv head
constexpr int QP = 4 + 16 * 4 + QP_QA;         // floats per (b, kv) in qprep: E2, pad, Qbar[16][4], qa

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
// Query preparation: one workgroup per (batch, kv head).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void qprep_kernel(AttnArgs a) {
  __shared__ float qs[16][D];
  __shared__ float qr[16][D];
  __shared__ float red[256];
  const int kv = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  const int s = b * a.n_kv_heads + kv;
  const int nqh = a.n_qh;
  for (int e = tid; e < 16 * D; e += 256) {
    const int h = e / D, c = e % D;
    float v = 0.0f;
    if (h < nqh) {
      const int64_t qi = ((int64_t)b * a.n_q_heads + kv * nqh + h) * D + c;
      v = a.q_f32 ? reinterpret_cast<const float*>(a.q)[qi] : bf2f(reinterpret_cast<const uint16_t*>(a.q)[qi]);
    }
    qs[h][c] = v;
  }
  __syncthreads();
  const float* Vk = a.basis_k + (int64_t)s * D * D;
  float amax = 0.0f;
  for (int e = tid; e < 16 * D; e += 256) {
    const int h = e / D, j = e % D;
    float acc = 0.0f;
    if (h < nqh)
      for (int i = 0; i < D; ++i) acc = __builtin_fmaf(qs[h][i], Vk[i * D + j], acc);
    acc *= a.scale_log2;
    qr[h][j] = acc;
    amax = __builtin_fmaxf(amax, __builtin_fabsf(acc));
  }
  red[tid] = amax;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (tid < o) red[tid] = __builtin_fmaxf(red[tid], red[tid + o]);
    __syncthreads();
  }
  amax = red[0];
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
    for (int j = 0; j < G; ++j) acc += qr[h][G * g + j];
    qp[4 + h * 4 + g] = acc;
  }
  // A operands of v_mfma_f32_4x4x4f16: entry [quad][g][k][part][r] holds the four
  // fp16 values q'_{4 quad + r}[32 g + 4 k + i] * 2^E, i = 0..3 (part 0 = hi, 1 = lo).
  uint32_t* qa = reinterpret_cast<uint32_t*>(qp + 4 + 64);
  for (int e = tid; e < 4 * 8 * 4 * 4; e += 256) {
    const int r = e & 3, quad = (e >> 2) & 3, k = (e >> 4) & 7, g = e >> 7;
    const int h = 4 * quad + r;
    uint32_t hi[4], lo[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float v = qr[h][G * g + 4 * k + i] * scl;
      const _Float16 vh = (_Float16)v;
      const _Float16 vl = (_Float16)(v - (float)vh);
      hi[i] = __builtin_bit_cast(uint16_t, vh);
      lo[i] = __builtin_bit_cast(uint16_t, vl);
    }
    const int base = ((((quad * 4 + g) * 8 + k) * 2) * 4 + r) * 2;
    qa[base + 0] = hi[0] | (hi[1] << 16);
    qa[base + 1] = hi[2] | (hi[3] << 16);
    qa[base + 8 + 0] = lo[0] | (lo[1] << 16);
    qa[base + 8 + 1] = lo[2] | (lo[3] << 16);
  }
}

// ---------------------------------------------------------------------------
// Split-K partial: one wavefront per (token chunk, kv head, batch).
// ---------------------------------------------------------------------------
template <int NQ>
__global__ __launch_bounds__(64) void attn_partial_kernel(AttnArgs a) {
  constexpr int NH = 4 * NQ;  // query-head rows handled (>= n_qh)
  __shared__ __attribute__((aligned(16))) uint32_t qa_s[NQ * QA_QUAD];
  __shared__ __attribute__((aligned(16))) uint16_t wt[NG][2][NH][64];    // p*s as bf16 hi/lo [slot][part][head][t]
  __shared__ float qbar_s[16 * 4];
  extern __shared__ __attribute__((aligned(16))) uint32_t vt[];          // value record tile [w][t], 64*Wv words

  const int chunk = blockIdx.x, kv = blockIdx.y, b = blockIdx.z;
  const int lane = threadIdx.x;
  const int s = b * a.n_kv_heads + kv;
  const int nqh = a.n_qh;
  const Kept Kk = read_kept(a.bits_k + (int64_t)s * NG);
  const Kept Kv = read_kept(a.bits_v + (int64_t)s * NG);
  const int Wk = a.Wk, Wv = a.Wv;
  float* part = a.partial + ((int64_t)b * a.n_q_heads + kv * nqh) * a.n_chunks * PART + (int64_t)chunk * PART;
  const bool ok = Kk.ok && Kv.ok && Kk.used <= Wk && Kv.used <= Wv;

  const float* qp = a.qprep + (int64_t)s * QP;
  const float E2 = qp[0];
  for (int i = lane; i < NQ * QA_QUAD; i += 64) qa_s[i] = reinterpret_cast<const uint32_t*>(qp + 4 + 64)[i];
  qbar_s[lane] = qp[4 + lane];
  __syncthreads();

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

  const int r4 = lane & 3;     // A-operand row (query head within a quad) of the score MFMA
  const int col = lane & 15;   // value MFMA: coefficient column / head row
  const int kq = lane >> 4;    // value MFMA: 8-token group of the K dimension

  for (int64_t tt = ok ? tile_begin : tile_end; tt < tile_end; ++tt) {
    const int64_t t = tt * 64 + lane;
    const bool valid = t < a.n_tokens;

    // ---- scores over the kept key coefficients (lane = token) ----
    float sc[NH];
#pragma unroll
    for (int h = 0; h < NH; ++h) sc[h] = 0.0f;
#pragma unroll
    for (int sl = 0; sl < NG; ++sl) {
      if (sl >= Kk.n) continue;
      const int g = Kk.grp[sl];
      const uint32_t meta = valid ? a.packed_k[rec_word(kbase, t, Wk, sl)] : 0u;
      f32x4 d[NQ];
#pragma unroll
      for (int q = 0; q < NQ; ++q) d[q] = f32x4{0.f, 0.f, 0.f, 0.f};
      with_bits(Kk.bits[sl], [&](auto bc) {
        constexpr int B = decltype(bc)::value;
        uint32_t pw[B + 1];
#pragma unroll
        for (int i = 0; i < B; ++i) pw[i] = valid ? a.packed_k[rec_word(kbase, t, Wk, Kk.pay[sl] + i)] : 0u;
        pw[B] = 0u;
        constexpr uint32_t M = (1u << B) - 1u;
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          uint32_t c[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int p = (4 * k + i) * B, w = p >> 5, o = p & 31;
            c[i] = (o + B <= 32) ? ((pw[w] >> o) & M) : (__builtin_amdgcn_alignbit(pw[w + 1], pw[w], o) & M);
          }
          // small integers -> fp16 exactly: 1024 + c has the code in the mantissa
          typedef __attribute__((__vector_size__(2 * sizeof(_Float16)))) _Float16 f16x2;
          const f16x2 off = {(_Float16)1024.0f, (_Float16)1024.0f};
          const f16x2 p01 = __builtin_bit_cast(f16x2, (c[0] | (c[1] << 16)) | 0x64006400u) - off;
          const f16x2 p23 = __builtin_bit_cast(f16x2, (c[2] | (c[3] << 16)) | 0x64006400u) - off;
          const f16x4 bop = {p01[0], p01[1], p23[0], p23[1]};
#pragma unroll
          for (int q = 0; q < NQ; ++q) {
            const int base = ((((q * 4 + g) * 8 + k) * 2) * 4 + r4) * 2;
            const f16x4 ahi = as_f16x4(u32x2{qa_s[base], qa_s[base + 1]});
            const f16x4 alo = as_f16x4(u32x2{qa_s[base + 8], qa_s[base + 9]});
            d[q] = __builtin_amdgcn_mfma_f32_4x4x4f16(ahi, bop, d[q], 0, 0, 0);
            d[q] = __builtin_amdgcn_mfma_f32_4x4x4f16(alo, bop, d[q], 0, 0, 0);
          }
        }
      });
      const float sk = h2f(meta) * E2, zk = h2f(meta >> 16);
#pragma unroll
      for (int q = 0; q < NQ; ++q)
#pragma unroll
        for (int j = 0; j < 4; ++j) sc[4 * q + j] += sk * d[q][j] + zk * qbar_s[(4 * q + j) * 4 + g];
    }

    // ---- stage the value record tile; lane = token ----
    __syncthreads();
    for (int w = 0; w < Kv.used; ++w) vt[w * 64 + lane] = valid ? a.packed_v[rec_word(vbase, t, Wv, w)] : 0u;
    // (the value tile holds only the words the kept groups use)

    // ---- online softmax (log2 domain), per query head ----
    float alpha[NH], p[NH];
#pragma unroll
    for (int h = 0; h < NH; ++h) {
      const float x = valid ? sc[h] : -__builtin_inff();
      const float mt = wave_max(x);
      const float mn = __builtin_fmaxf(m_run[h], mt);
      alpha[h] = (mn == -__builtin_inff()) ? 1.0f : __builtin_amdgcn_exp2f(m_run[h] - mn);
      p[h] = valid ? __builtin_amdgcn_exp2f(x - mn) : 0.0f;
      l_run[h] = l_run[h] * alpha[h] + p[h];
      m_run[h] = mn;
    }
    // softmax weights times value scales -> LDS as bf16 hi + lo; z terms per lane
#pragma unroll
    for (int sl = 0; sl < NG; ++sl) {
      if (sl >= Kv.n) continue;
      const uint32_t meta = vt[sl * 64 + lane];
      const float sv = h2f(meta), zv = h2f(meta >> 16);
#pragma unroll
      for (int h = 0; h < NH; ++h) {
        zacc[h][sl] = zacc[h][sl] * alpha[h] + p[h] * zv;
        const float w = p[h] * sv;
        const uint32_t whi = f2bf(w);
        const uint32_t wlo = f2bf(w - bf2f(whi));
        wt[sl][0][h][lane] = (uint16_t)whi;
        wt[sl][1][h][lane] = (uint16_t)wlo;
      }
    }
    // rescale value accumulators: lane holds heads 4*kq + j
    float al[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float v = 1.0f;
#pragma unroll
      for (int h = 0; h < NH; ++h)
        if (h == 4 * kq + j) v = alpha[h];
      al[j] = v;
    }
#pragma unroll
    for (int g = 0; g < NG; ++g)
#pragma unroll
      for (int c2 = 0; c2 < 2; ++c2)
#pragma unroll
        for (int j = 0; j < 4; ++j) vacc[g][c2][j] *= al[j];
    __syncthreads();

    // ---- value accumulation over the kept value coefficients ----
#pragma unroll
    for (int sl = 0; sl < NG; ++sl) {
      if (sl < Kv.n) {
        with_bits(Kv.bits[sl], [&](auto bc) {
          constexpr int B = decltype(bc)::value;
          constexpr uint32_t M = (1u << B) - 1u;
#pragma unroll
          for (int th = 0; th < 2; ++th) {
            const int tok0 = 32 * th + 8 * kq;
            bf16x8 whi = bf16x8{}, wlo = bf16x8{};
            if (col < nqh) {
              whi = as_bf16x8(*reinterpret_cast<const u32x4*>(&wt[sl][0][col][tok0]));
              wlo = as_bf16x8(*reinterpret_cast<const u32x4*>(&wt[sl][1][col][tok0]));
            }
#pragma unroll
            for (int c2 = 0; c2 < 2; ++c2) {
              const int jj = 16 * c2 + col;
              const int p0 = jj * B, w = Kv.pay[sl] + (p0 >> 5), o = p0 & 31;
              const u32x4 a0 = *reinterpret_cast<const u32x4*>(&vt[w * 64 + tok0]);
              const u32x4 a1 = *reinterpret_cast<const u32x4*>(&vt[w * 64 + tok0 + 4]);
              uint32_t cd[8];
              if (o + B <= 32) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                  cd[i] = (a0[i] >> o) & M;
                  cd[4 + i] = (a1[i] >> o) & M;
                }
              } else {
                const u32x4 b0 = *reinterpret_cast<const u32x4*>(&vt[(w + 1) * 64 + tok0]);
                const u32x4 b1 = *reinterpret_cast<const u32x4*>(&vt[(w + 1) * 64 + tok0 + 4]);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                  cd[i] = __builtin_amdgcn_alignbit(b0[i], a0[i], o) & M;
                  cd[4 + i] = __builtin_amdgcn_alignbit(b1[i], a1[i], o) & M;
                }
              }
              const bf16x8 bop = as_bf16x8(u32x4{int_to_bf16_pair(cd[0], cd[1]), int_to_bf16_pair(cd[2], cd[3]),
                                                 int_to_bf16_pair(cd[4], cd[5]), int_to_bf16_pair(cd[6], cd[7])});
              vacc[sl][c2] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(whi, bop, vacc[sl][c2], 0, 0, 0);
              vacc[sl][c2] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wlo, bop, vacc[sl][c2], 0, 0, 0);
            }
          }
        });
      }
    }
  }

  // ---- partial of this chunk: m, l, Z per group, acc per kept coefficient ----
#pragma unroll
  for (int h = 0; h < NH; ++h) {
    const float l = wave_sum(l_run[h]);
    float z[NG];
#pragma unroll
    for (int g = 0; g < NG; ++g) z[g] = wave_sum(zacc[h][g]);
    if (h < nqh && lane == 0) {
      float* ph = part + (int64_t)h * a.n_chunks * PART;
      ph[0] = ok ? m_run[h] : -__builtin_inff();
      ph[1] = ok ? l : 0.0f;
#pragma unroll
      for (int sl = 0; sl < NG; ++sl)
        if (sl < Kv.n) ph[2 + Kv.grp[sl]] = z[sl];
    }
  }
#pragma unroll
  for (int sl = 0; sl < NG; ++sl) {
    if (sl < Kv.n) {
#pragma unroll
      for (int c2 = 0; c2 < 2; ++c2)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int h = 4 * kq + j;
          if (h < nqh) part[(int64_t)h * a.n_chunks * PART + 8 + G * Kv.grp[sl] + 16 * c2 + col] = vacc[sl][c2][j];
        }
    }
  }
}

// ---------------------------------------------------------------------------
// Combine partials and inverse-rotate: one workgroup per (batch, query head).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(128) void combine_kernel(AttnArgs a) {
  __shared__ float chat[D];
  __shared__ float wsum[2];
  const int hq = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  const int kv = hq / a.n_qh;
  const int s = b * a.n_kv_heads + kv;
  const float* ph = a.partial + ((int64_t)b * a.n_q_heads + hq) * a.n_chunks * PART;
  float mx = -__builtin_inff();
  for (int c = 0; c < a.n_chunks; ++c) mx = __builtin_fmaxf(mx, ph[(int64_t)c * PART]);
  const uint32_t bw = *reinterpret_cast<const uint32_t*>(a.bits_v + (int64_t)s * NG);
  const int g = tid >> 5;
  const bool kept = ((bw >> (8 * g)) & 0xFFu) != 0u;
  float l = 0.0f, acc = 0.0f;
  for (int c = 0; c < a.n_chunks; ++c) {
    const float* pc = ph + (int64_t)c * PART;
    const float mc = pc[0];
    const float w = (mc == -__builtin_inff()) ? 0.0f : __builtin_amdgcn_exp2f(mc - mx);
    l += w * pc[1];
    if (kept) acc += w * (pc[2 + g] + pc[8 + tid]);
  }
  chat[tid] = acc / l + a.mean_v[(int64_t)s * D + tid];
  __syncthreads();
  const float* Vv = a.basis_v + (int64_t)s * D * D + (int64_t)tid * D;
  float o = 0.0f;
  for (int j = 0; j < D; ++j) o = __builtin_fmaf(chat[j], Vv[j], o);
  a.out[((int64_t)b * a.n_q_heads + hq) * D + tid] = o;
  (void)wsum;
}

}  // namespace spectra_dev

namespace spectra {
using namespace spectra_dev;

size_t attention_qprep_floats(int32_t batch, int32_t, int32_t n_kv_heads) {
  return (size_t)batch * n_kv_heads * QP;
}
size_t attention_partial_floats(int32_t batch, int32_t n_q_heads, int32_t n_chunks) {
  return (size_t)batch * n_q_heads * n_chunks * PART;
}
int32_t attention_chunks(int32_t batch, int32_t n_kv_heads, int64_t n_tokens, int32_t* tiles_per_chunk) {
  const int64_t n_tiles = (n_tokens + 63) / 64;
  const int64_t groups = (int64_t)batch * n_kv_heads;
  int64_t want = (1024 + groups - 1) / groups;   // ~1024 wavefronts in flight
  int64_t tpc = (n_tiles + want - 1) / want;
  if (tpc < 8) tpc = 8;                           // keep partial traffic small
  if (tpc > n_tiles) tpc = n_tiles > 0 ? n_tiles : 1;
  const int64_t nch = n_tiles > 0 ? (n_tiles + tpc - 1) / tpc : 1;
  *tiles_per_chunk = (int32_t)tpc;
  return (int32_t)nch;
}

hipError_t launch_attention(const AttnArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(qprep_kernel, dim3(a.n_kv_heads, a.batch), dim3(256), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 grid(a.n_chunks, a.n_kv_heads, a.batch);
  const int nq = (a.n_qh + 3) / 4;
  const size_t lds = (size_t)64 * a.Wv * sizeof(uint32_t);
  switch (nq) {
    case 1: hipLaunchKernelGGL(attn_partial_kernel<1>, grid, dim3(64), lds, st, a); break;
    case 2: hipLaunchKernelGGL(attn_partial_kernel<2>, grid, dim3(64), lds, st, a); break;
    case 3: hipLaunchKernelGGL(attn_partial_kernel<3>, grid, dim3(64), lds, st, a); break;
    default: hipLaunchKernelGGL(attn_partial_kernel<4>, grid, dim3(64), lds, st, a); break;
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(combine_kernel, dim3(a.n_q_heads, a.batch), dim3(128), 0, st, a);
  return hipGetLastError();
}

}  // namespace spectra
