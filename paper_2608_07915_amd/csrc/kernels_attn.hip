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
//     query heads. The B operand is the payload itself, cut by masks into bit
//     fields that each lie inside one code and inside bits 0..9 of a 16-bit half;
//     OR-ing in the exponent of 1024 and subtracting 1024 in fp16 (both exact)
//     turns a field into the normal fp16 integer it spells. A field at bit f0 of
//     its half holding code bits b0.. equals code-part * 2^(f0-b0), so the
//     matching A entry is q'_j * 2^(b0-f0). (Fields are not fed as fp16
//     subnormals: the matrix cores align such products by the subnormal's
//     nominal exponent and drop low bits.) q' enters as fp16 hi and 2^11-scaled
//     lo parts in two accumulators, so the dot products are ~fp32-accurate;
//   * values: v_mfma_f32_16x16x32_bf16, rows = query heads (softmax weights p*s as
//     bf16 hi and lo parts, stacked in the otherwise unused rows when there are
//     at most 8 heads), K = 32 tokens, columns = 16 coefficients. Codes of width
//     <= 7 enter as bf16 (128 + c), built with one byte-gather permute and a mask;
//     a second MFMA against the constant -128 removes the offset tile by tile.
// Work: one workgroup of four wavefronts per (token chunk, KV head, sequence);
// each wavefront streams 64-token record tiles with the next tile's words
// prefetched into registers; the four wavefronts merge their online-softmax
// states in LDS and write one partial per chunk; combine_kernel merges chunks.
#include "attn_common.hpp"
#include "device_common.hpp"
#include "encode_dev.hpp"
#include "kernels.hpp"
#include "kplan.hpp"

namespace spectra_dev {

constexpr int kplan_mfmas(int B) { return (make_kplan(B).n_ops + 1) / 2; }
constexpr int KM_MAX = 14;  // score MFMAs per slot, widest plan (B = 7)
static_assert(make_kplan(7).n_ops == KOPS_MAX && kplan_mfmas(7) == KM_MAX, "plan sizes");
static_assert(make_kplan(1).n_ops == 16 && make_kplan(5).n_ops == 20 && make_kplan(8).n_ops == 16, "plan sizes");
__device__ constexpr KGather KGATHER = make_kgather();
static_assert(KMFMA_MAX == KM_MAX, "plan sizes");

// score-MFMA A operands per (head quad, slot): [m][row r][hi k0..k3, lo k0..k3] as fp16
constexpr int QA_SLOT = KM_MAX * 4 * 4;  // uint32
constexpr int QA_QUAD = NG * QA_SLOT;
constexpr int WAVES = 4;

// ---------------------------------------------------------------------------
// Decode-step append, done by the workgroup whose chunk holds the last tile:
// the new key and value of stream s go into slot t_new exactly as the encode
// kernel would write them (same staging, same MFMA sequence per token). Wave w
// takes kept key slot w, then kept value slot w; the token sits in LDS row 0 of
// a 32-row block whose other rows are zero (their columns are discarded).
// `xs` is scratch LDS of at least append_stage_bytes(F32) bytes.
// ---------------------------------------------------------------------------
__host__ __device__ constexpr int append_rowb(bool f32) { return f32 ? (512 + 16) : (256 + 16); }
__host__ __device__ constexpr int append_stage_bytes(bool f32) { return 2 * 32 * append_rowb(f32); }

template <bool F32>
__device__ __forceinline__ void append_token(const AttnArgs& a, int s, int tid, uint8_t* xs) {
  constexpr int ESZ = F32 ? 4 : 2;
  constexpr int ROWB = append_rowb(F32);
  constexpr int CPR = (D * ESZ) / 16;
  constexpr int PER = (2 * 32 * CPR) / 256;  // staged 16-byte pieces per thread
  static_assert(PER * 256 == 2 * 32 * CPR, "staging split");
  const int wave = tid >> 6, lane = tid & 63, h = lane >> 5, col = lane & 31;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int e = tid + 256 * i;
    const int wh = e / (32 * CPR), row = (e / CPR) % 32, part = e % CPR;
    u32x4 v = u32x4{0u, 0u, 0u, 0u};
    if (row == 0) {
      const char* src = reinterpret_cast<const char*>(wh ? a.v_new : a.k_new);
      v = *reinterpret_cast<const u32x4*>(src + (int64_t)s * D * ESZ + part * 16);
    }
    *reinterpret_cast<u32x4*>(xs + wh * 32 * ROWB + row * ROWB + part * 16) = v;
  }
  __syncthreads();
#pragma unroll 1
  for (int which = 0; which < 2; ++which) {
    const Kept K = read_kept((which ? a.bits_v : a.bits_k) + (int64_t)s * NG);
    const int W = which ? a.Wv : a.Wk;
    if (!K.ok || K.used > W) continue;  // width table inconsistent with the record: write nothing
    uint32_t* packed = which ? a.app_v : a.app_k;
    const int64_t sbase = (int64_t)s * a.t_cap * W;
    const int slot = wave;
    if (slot < K.n) {
      const int grp = pick4(K.grp, slot);
      f32x16 nm;
      const float* m = (which ? a.mean_v : a.mean_k) + (int64_t)s * D + G * grp + 16 * h;
#pragma unroll
      for (int j = 0; j < 16; ++j) nm[j] = -m[j];
      encode_block_streamed<F32, ROWB>(xs + which * 32 * ROWB, 0, col, h, (which ? a.basis_v : a.basis_k) + (int64_t)s * D * D,
                                       grp, nm, a.t_new, a.t_new, a.t_new + 1, sbase, W, slot, pick4(K.bits, slot),
                                       pick4(K.pay, slot), packed);
    }
    // padding words of the record are zero
    if (wave == 0 && lane < W - K.used) packed[rec_word(sbase, a.t_new, W, K.used + lane)] = 0u;
  }
}

// ---------------------------------------------------------------------------
// Query preparation of one (sequence, kv head), done by every scan workgroup in
// its prologue (the result is identical in all of them): q' = scale * log2(e) *
// q V_K for the n_qh heads, Qbar[h][g] = sum_{j in g} q'_hj, and the score-MFMA
// A operands [quad][slot][m][row][hi k0..k3, lo k0..k3] (see score_slot) in
// qa_s. Returns E2 = 2^-E. `scratch` is LDS of at least qprep_scratch_bytes(NQ).
// ---------------------------------------------------------------------------
__host__ __device__ constexpr int qprep_scratch_bytes(int nq) {
  return (5 * 4 * nq * D) * 4 + (int)sizeof(KGather);
}

// `issue_more` is called once the loads this step needs are in flight (the caller
// puts its own, later-needed loads behind them).
template <int NQ, typename F>
__device__ __forceinline__ float prepare_query(const AttnArgs& a, int s, int b, int kv, int tid, uint8_t* scratch,
                                               uint32_t* __restrict__ qa_s, float* __restrict__ qbar_s, float* red_s,
                                               F&& issue_more) {
  constexpr int NH = 4 * NQ;
  constexpr int QPT = (NH * D) / 256;  // q values per thread
  float(*qs)[D] = reinterpret_cast<float(*)[D]>(scratch);                          // [NH][D]: q, then q'
  float(*part)[NH][D] = reinterpret_cast<float(*)[NH][D]>(scratch + NH * D * 4);  // [4][NH][D]
  KField(*gat)[KM_MAX][4] = reinterpret_cast<KField(*)[KM_MAX][4]>(scratch + 5 * NH * D * 4);  // [8][m][k]
  const int nqh = a.n_qh;
  const uint32_t bwk = *reinterpret_cast<const uint32_t*>(a.bits_k + (int64_t)s * NG);
  // Only the kept groups' q' are needed. Columns 0..63 (groups 0 and 1, kept in the
  // common case: widths fall with the variance) are requested before the width
  // table arrives; columns 64..127 only when groups 2 or 3 are kept. Thread
  // (quarter qt, column jj) takes rows [32 qt, 32 qt + 32).
  const int jj = tid & 63, qt = tid >> 6;
  const float* Vk = a.basis_k + (int64_t)s * D * D + (int64_t)(32 * qt) * D + jj;
  float v[32];
#pragma unroll
  for (int i = 0; i < 32; ++i) v[i] = Vk[i * D];
  float qv[QPT];
#pragma unroll
  for (int i = 0; i < QPT; ++i) {
    const int e = tid + 256 * i, h = e >> 7, c = e & 127;
    qv[i] = 0.0f;
    if (h < nqh) {
      const int64_t qi = ((int64_t)b * a.n_q_heads + kv * nqh + h) * D + c;
      qv[i] = a.q_f32 ? reinterpret_cast<const float*>(a.q)[qi] : bf2f(reinterpret_cast<const uint16_t*>(a.q)[qi]);
    }
  }
  constexpr int GW = (int)(sizeof(KGather) / 4);
  static_assert(sizeof(KGather) % 4 == 0 && GW <= 256, "gather table copy");
  const uint32_t gw = tid < GW ? reinterpret_cast<const uint32_t*>(&KGATHER)[tid] : 0u;
  issue_more();
#pragma unroll
  for (int i = 0; i < QPT; ++i) {
    const int e = tid + 256 * i;
    qs[e >> 7][e & 127] = qv[i];
  }
  if (tid < GW) reinterpret_cast<uint32_t*>(gat)[tid] = gw;
  __syncthreads();
  const int npass = (bwk >> 16) != 0u ? 2 : 1;  // groups 2 or 3 kept: columns 64..127 too
#pragma unroll 1
  for (int pass = 0; pass < npass; ++pass) {
    if (pass > 0) {
#pragma unroll
      for (int i = 0; i < 32; ++i) v[i] = Vk[i * D + 64];
    }
    float acc[NH];
#pragma unroll
    for (int h = 0; h < NH; ++h) acc[h] = 0.0f;
#pragma unroll
    for (int i = 0; i < 32; ++i)
#pragma unroll
      for (int h = 0; h < NH; ++h) acc[h] = __builtin_fmaf(qs[h][32 * qt + i], v[i], acc[h]);
#pragma unroll
    for (int h = 0; h < NH; ++h) part[qt][h][64 * pass + jj] = acc[h];
  }
  __syncthreads();
  float amax = 0.0f;
  for (int e = tid; e < NH * D; e += 256) {
    const int h = e >> 7, c = e & 127;
    const bool kept = ((bwk >> (8 * (c >> 5))) & 0xFFu) != 0u;
    const float q =
        (h < nqh && kept) ? ((part[0][h][c] + part[1][h][c]) + (part[2][h][c] + part[3][h][c])) * a.scale_log2 : 0.0f;
    qs[h][c] = q;
    amax = __builtin_fmaxf(amax, __builtin_fabsf(q));
  }
  amax = wave_max(amax);
  if ((tid & 63) == 0) red_s[tid >> 6] = amax;
  __syncthreads();
  amax = __builtin_fmaxf(__builtin_fmaxf(red_s[0], red_s[1]), __builtin_fmaxf(red_s[2], red_s[3]));
  // 2^E brings max |q'| into [2^8, 2^9), so every A entry x = q' * 2^(E + e) (e <= 6)
  // stays below 2^15. x is split into hi = fp16(x) and lo = fp16((x - hi) * 2^11):
  // lo is kept in the normal fp16 range by its 2^11 and accumulates separately.
  // E2 = 2^-E undoes the scaling.
  int e2 = 0;
  if (amax > 0.0f) (void)__builtin_frexpf(amax, &e2);
  const int E = amax > 0.0f ? 9 - e2 : 0;
  {
    // Qbar[h][g]: four lanes per (head, group), eight values each, then a lane reduction
    const int ent = tid >> 2, pt = tid & 3, h = ent >> 2, g = ent & 3;
    if (ent < NH * NG) {
      float sum = 0.0f;
#pragma unroll
      for (int i = 0; i < 8; ++i) sum += qs[h][G * g + 8 * pt + i];
      sum += __shfl_xor(sum, 1);
      sum += __shfl_xor(sum, 2);
      if (pt == 0) qbar_s[ent] = sum;
    }
  }
  // Score-MFMA A operands, entry (quad, slot, m, r): K element k is field
  // (op 2m + k/2, half k%2) of the slot's plan, i.e. q'_{4quad+r} of the field's
  // coefficient times 2^(E + e), as fp16 hi + lo.
  for (int e = tid; e < NQ * NG * KM_MAX * 4; e += 256) {
    const int r = e & 3, m = (e >> 2) % KM_MAX, slot = (e / (4 * KM_MAX)) & 3, quad = e / (4 * KM_MAX * NG);
    int g = -1, B = 0, c = 0;
#pragma unroll
    for (int gg = 0; gg < NG; ++gg) {
      const int bb = (int)((bwk >> (8 * gg)) & 0xFFu);
      const bool here = bb != 0 && c == slot;
      g = here ? gg : g;
      B = here ? bb : B;
      c += bb != 0 ? 1 : 0;
    }
    uint32_t hi[4] = {0u, 0u, 0u, 0u}, lo[4] = {0u, 0u, 0u, 0u};
    if (g >= 0 && B <= 8) {
      const int h = 4 * quad + r;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const KField f = gat[B - 1][m][k];
        const float x = f.code >= 0 ? __builtin_ldexpf(qs[h][G * g + f.code], E + f.e) : 0.0f;
        const _Float16 xh = (_Float16)x;
        const _Float16 xl = (_Float16)((x - (float)xh) * 2048.0f);
        hi[k] = __builtin_bit_cast(uint16_t, xh);
        lo[k] = __builtin_bit_cast(uint16_t, xl);
      }
    }
    uint32_t* dst = qa_s + ((((quad * NG + slot) * KM_MAX + m) * 4 + r) * 4);
    dst[0] = hi[0] | (hi[1] << 16);
    dst[1] = hi[2] | (hi[3] << 16);
    dst[2] = lo[0] | (lo[1] << 16);
    dst[3] = lo[2] | (lo[3] << 16);
  }
  return __builtin_ldexpf(1.0f, -E);
}

// Bytes of LDS holding the softmax-weight rows of all wavefronts: per wave and kept
// slot, 2*NH rows (hi parts of the NH heads, then lo parts) of 64 bf16 tokens.
__host__ __device__ constexpr int attn_wt_bytes(int nq) { return WAVES * NG * (8 * nq) * WROW * 2; }

// ---------------------------------------------------------------------------
// Score contributions of one kept key slot of width B for the lane's token:
// dh[q][j] += sum over the slot's fields of hi(4q + j, field) * field, and dl
// likewise with the lo parts (scaled by 2^11); fields are exact fp16 integers.
// qsl points at the slot's A operands of quad 0; quad q is QA_QUAD further.
// ---------------------------------------------------------------------------
template <int B, int NQ>
__device__ __forceinline__ void score_slot(const uint32_t* __restrict__ kt, int lane, int pay,
                                           const uint32_t* __restrict__ qsl, int r4, f32x4 (&dh)[NQ],
                                           f32x4 (&dl)[NQ]) {
  constexpr KPlan P = make_kplan(B);
  // the exponent of 1024 in both halves, kept in a VGPR so that mask-and-or is one
  // v_and_or_b32 (its mask then comes from an SGPR)
  uint32_t magic = 0x64006400u;
  asm volatile("" : "+v"(magic));
  uint32_t reg0 = 0u;
  int opi = 0;
#pragma unroll
  for (int w = 0; w < B; ++w) {
    const uint32_t x = kt[(pay + w) * TROW + lane];
    const uint32_t x6 = x >> 6;
#pragma unroll
    for (int i = 0; i < P.word_ops[w]; ++i, ++opi) {
      // (field | exponent of 1024) - 1024: the field as a normal fp16 integer, both halves
      const uint32_t v = __builtin_bit_cast(
          uint32_t, __builtin_bit_cast(f16x2, ((P.op[opi].shifted ? x6 : x) & P.op[opi].mask) | magic) -
                        f16x2{(_Float16)1024.0f, (_Float16)1024.0f});
      if ((opi & 1) == 0) {
        reg0 = v;
        if (opi + 1 < P.n_ops) continue;
      }
      // ops opi-1, opi (or opi and an empty register) form the B operand of MFMA m
      const int m = opi >> 1;
      const f16x4 bop = as_f16x4(u32x2{(opi & 1) ? reg0 : v, (opi & 1) ? v : 0u});
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        const u32x4 A = *reinterpret_cast<const u32x4*>(qsl + q * QA_QUAD + (m * 4 + r4) * 4);
        dh[q] = __builtin_amdgcn_mfma_f32_4x4x4f16(as_f16x4(u32x2{A[0], A[1]}), bop, dh[q], 0, 0, 0);
        dl[q] = __builtin_amdgcn_mfma_f32_4x4x4f16(as_f16x4(u32x2{A[2], A[3]}), bop, dl[q], 0, 0, 0);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Split-K partial. NQ = query-head quads (n_qh <= 4 NQ); PK, PV = prefetched key
// and value record words per tile (>= W_k, W_v; both 0: no prefetch); EXACT:
// W_k = PK and W_v = PV.
// ---------------------------------------------------------------------------
// ---------------------------------------------------------------------------
// Merge of the four wavefronts' online-softmax states of one scan workgroup in LDS
// and the chunk's partial (m, l, zero-point sums per group, value sums per
// coefficient) for every query head of the KV head. smem: the tile buffers, free
// once every wave has left its tile loop.
// ---------------------------------------------------------------------------
template <int NQ>
__device__ __forceinline__ void write_chunk_partial(const AttnArgs& a, int b, int kv, int chunk, int tid, int wave,
                                                    int lane, int kq, int col, bool ok, const Kept& Kv,
                                                    const float (&m_run)[4 * NQ], const float (&l_run)[4 * NQ],
                                                    const float (&zacc)[4 * NQ][NG], const f32x4 (&vacc)[NG][2],
                                                    uint32_t* smem) {
  constexpr int NH = 4 * NQ;
  constexpr bool STACK = NQ <= 2;
  __shared__ float mst[WAVES][NH], lst[WAVES][NH], zst[WAVES][NH][NG];
  const int nqh = a.n_qh;
#pragma unroll
  for (int h = 0; h < NH; ++h) {
    const float l = wave_sum_lane63(l_run[h]);
    float z[NG];
#pragma unroll
    for (int g = 0; g < NG; ++g) z[g] = g < Kv.n ? wave_sum_lane63(zacc[h][g]) : 0.0f;
    if (lane == 63) {
      mst[wave][h] = ok ? m_run[h] : -__builtin_inff();
      lst[wave][h] = l;
#pragma unroll
      for (int g = 0; g < NG; ++g) zst[wave][h][g] = 0.0f;
      // zero-point sums are kept per slot; the partial holds them per group
#pragma unroll
      for (int sl = 0; sl < NG; ++sl)
        if (sl < Kv.n) zst[wave][h][Kv.grp[sl]] = z[sl];
    }
  }
  __syncthreads();  // all waves done with their tile buffers: reuse smem for the value sums
  // per wave, MFMA row r of the value accumulators lands in row r of [ACC_ROWS][AROW]
  // (stacked: rows NH.. hold the lo-weight sums of the same heads); every kept
  // column of a row is written exactly once, so no read-modify-write is needed
  constexpr int ACC_ROWS = STACK ? 2 * NH : NH;
  float* accw = reinterpret_cast<float*>(smem) + wave * ACC_ROWS * AROW;
#pragma unroll
  for (int sl = 0; sl < NG; ++sl) {
    if (sl >= Kv.n) continue;
    // codes below 8 bits entered as 1 + c 2^-b (see value_codes2)
    const float vscale = Kv.bits[sl] < 8 ? (float)(1u << Kv.bits[sl]) : 1.0f;
#pragma unroll
    for (int c2 = 0; c2 < 2; ++c2)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int row = 4 * kq + j;
        if (row < ACC_ROWS) accw[row * AROW + G * Kv.grp[sl] + 2 * col + c2] = vacc[sl][c2][j] * vscale;
      }
  }
  uint32_t kept_groups = 0u;  // groups with no kept value coefficients have no sums
#pragma unroll
  for (int sl = 0; sl < NG; ++sl)
    if (sl < Kv.n) kept_groups |= 1u << Kv.grp[sl];
  __syncthreads();
  float* part = a.partial + ((int64_t)b * a.n_q_heads + kv * nqh) * a.n_chunks * PART + (int64_t)chunk * PART;
  for (int e = tid; e < nqh * D; e += 256) {
    const int h = e >> 7, j = e & 127;
    const bool kept = (kept_groups >> (j >> 5)) & 1u;
    float M = -__builtin_inff();
#pragma unroll
    for (int w = 0; w < WAVES; ++w) M = __builtin_fmaxf(M, mst[w][h]);
    float acc = 0.0f, l = 0.0f, z = 0.0f;
#pragma unroll
    for (int w = 0; w < WAVES; ++w) {
      const float f = (mst[w][h] == -__builtin_inff()) ? 0.0f : __builtin_amdgcn_exp2f(mst[w][h] - M);
      const float* aw = reinterpret_cast<const float*>(smem) + w * ACC_ROWS * AROW;
      float v = kept ? aw[h * AROW + j] : 0.0f;
      if constexpr (STACK) v += kept ? aw[(NH + h) * AROW + j] : 0.0f;
      acc += f * v;
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

template <int NQ, int PK, int PV, bool EXACT>
__global__ __launch_bounds__(256, 2) void attn_kernel(AttnArgs a) {
  constexpr int NH = 4 * NQ;
  constexpr bool STACK = NQ <= 2;  // 2*NH <= 16: hi and lo weight rows share one MFMA
  extern __shared__ __attribute__((aligned(16))) uint32_t smem[];
  __shared__ __attribute__((aligned(16))) uint32_t qa_s[NQ * QA_QUAD];
  __shared__ float qbar_s[16 * 4];

  // a.group_major: one-dimensional grid, workgroup i = chunk * groups + group, so that
  // (dispatched round-robin over the XCDs) every chunk of a (sequence, kv head) runs on
  // the same XCD and its L2 serves that head's key basis to all of them
  int chunk = blockIdx.x, kv = blockIdx.y, b = blockIdx.z;
  if (a.group_major) {
    const int ngr = a.n_kv_heads * a.batch, gid = (int)(blockIdx.x % (unsigned)ngr);
    chunk = (int)(blockIdx.x / (unsigned)ngr);
    kv = gid % a.n_kv_heads;
    b = gid / a.n_kv_heads;
  }
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int s = b * a.n_kv_heads + kv;
  const int nqh = a.n_qh;
  const int Wk = a.Wk, Wv = a.Wv;
  // ---- per-wave streaming over this chunk's tiles ----
  static_assert((PK > 0) == (PV > 0), "prefetch both tensors or neither");
  const int wk_rows = PK > 0 ? PK : Wk, wv_rows = PV > 0 ? PV : Wv;  // staged words per token
  const int wpw = wk_rows + wv_rows;
  uint32_t* kt = smem + wave * wpw * TROW;
  uint32_t* vt = kt + wk_rows * TROW;
  uint16_t* wt = reinterpret_cast<uint16_t*>(smem + WAVES * wpw * TROW) + wave * (NG * 2 * NH * WROW);
  const int64_t kbase = (int64_t)s * a.t_cap * Wk;
  const int64_t vbase = (int64_t)s * a.t_cap * Wv;
  // chunk c < n_chunks - 1 holds tiles [c * tpc, (c + 1) * tpc) of all but the last
  // tile; the last chunk holds the last tile alone
  const int64_t n_tiles = (a.n_tokens + 63) >> 6;
  const bool last_chunk = chunk == a.n_chunks - 1;
  const int64_t tile_begin = last_chunk ? n_tiles - 1 : (int64_t)chunk * a.tiles_per_chunk;
  int64_t tile_end = last_chunk ? n_tiles : tile_begin + a.tiles_per_chunk;
  if (!last_chunk && tile_end > n_tiles - 1) tile_end = n_tiles - 1;

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

  // register prefetch of one tile's record words (K and V); PK = PV = 0: none
  constexpr int PKR = PK > 0 ? PK : 1, PVR = PV > 0 ? PV : 1;
  uint32_t pk[PKR], pv[PVR];
  // every lane loads in-bounds words: the word index is clamped to the record (a
  // uniform offset folded into the per-word base pointer), the token to the tile;
  // tokens past n_tokens are never weighted (their value metadata is zeroed)
  const uint32_t* kps = a.packed_k + kbase;
  const uint32_t* vps = a.packed_v + vbase;
  auto load_tile = [&](int64_t tt) {
    const uint32_t ko = (uint32_t)tt * (uint32_t)(64 * Wk) + (uint32_t)lane;
    const uint32_t vo = (uint32_t)tt * (uint32_t)(64 * Wv) + (uint32_t)lane;
    if constexpr (EXACT) {  // Wk == PK, Wv == PV: no clamping, word offsets are immediates
      const uint32_t* kp = kps + ko;
      const uint32_t* vp = vps + vo;
#pragma unroll
      for (int w = 0; w < (PK > PV ? PK : PV); ++w) {
        if (w < PK) pk[w] = kp[64 * w];
        if (w < PV) pv[w] = vp[64 * w];
      }
    } else {
#pragma unroll
      for (int w = 0; w < (PK > PV ? PK : PV); ++w) {
        if (w < PK) pk[w] = (kps + 64 * (w < Wk ? w : Wk - 1))[ko];
        if (w < PV) pv[w] = (vps + 64 * (w < Wv ? w : Wv - 1))[vo];
      }
    }
  };
  // In a decode step the workgroup of the last chunk (the last tile) first appends
  // the new token of its stream (and makes the records visible to its own loads).
  int64_t tt = tile_begin + wave;
  if (a.app_k != nullptr && last_chunk) {
    if (a.app_f32)
      append_token<true>(a, s, tid, reinterpret_cast<uint8_t*>(smem));
    else
      append_token<false>(a, s, tid, reinterpret_cast<uint8_t*>(smem));
    __threadfence();
    __syncthreads();
  }

  // ---- prologue: query preparation of this (sequence, kv head) into LDS; the
  // first tile's loads (in bounds whatever the width tables hold) queue behind
  // its loads ----
  __shared__ float red_s[WAVES];
  __shared__ float e2_s;
  const float E2q = prepare_query<NQ>(a, s, b, kv, tid, reinterpret_cast<uint8_t*>(smem), qa_s, qbar_s, red_s, [&] {
    if (tt < tile_end) load_tile(tt);
  });
  const Kept Kk = read_kept(a.bits_k + (int64_t)s * NG);
  const Kept Kv = read_kept(a.bits_v + (int64_t)s * NG);
  const bool ok = Kk.ok && Kv.ok && Kk.used <= Wk && Kv.used <= Wv;
  if (tid == 0) e2_s = E2q;
  __syncthreads();  // prepared query data in LDS; the scratch may now hold tiles
  const float E2 = e2_s;

  Kept kk = Kk, kvv = Kv;
  // bit offset 2 col b (< 256) of the lane's first value code in each kept slot, one byte per slot
  uint32_t voffs = 0u;
#pragma unroll
  for (int sl = 0; sl < NG; ++sl) voffs |= (uint32_t)(2 * col * Kv.bits[sl]) << (8 * sl);
  for (; ok && tt < tile_end; tt += WAVES) {
    asm volatile("" : "+v"(voffs));
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
    if constexpr (PK > 0) {
#pragma unroll
      for (int w = 0; w < (PK > PV ? PK : PV); ++w) {
        if (w < PK) kt[w * TROW + lane] = pk[w];
        if (w < PV) vt[w * TROW + lane] = pv[w];
      }
      if (tt + WAVES < tile_end) load_tile(tt + WAVES);
    } else {
      const uint32_t ko = (uint32_t)tt * (uint32_t)(64 * Wk) + (uint32_t)lane;
      const uint32_t vo = (uint32_t)tt * (uint32_t)(64 * Wv) + (uint32_t)lane;
      for (int w = 0; w < kk.used; ++w) kt[w * TROW + lane] = (kps + 64 * w)[ko];
      for (int w = 0; w < kvv.used; ++w) vt[w * TROW + lane] = (vps + 64 * w)[vo];
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
      const uint32_t meta = kt[sl * TROW + lane];
      f32x4 dh[NQ], dl[NQ];
#pragma unroll
      for (int q = 0; q < NQ; ++q) dh[q] = dl[q] = f32x4{0.f, 0.f, 0.f, 0.f};
      const uint32_t* qsl = qa_s + sl * QA_SLOT;
      const int pay = kk.pay[sl];
      switch (kk.bits[sl]) {
        case 1: score_slot<1, NQ>(kt, lane, pay, qsl, r4, dh, dl); break;
        case 2: score_slot<2, NQ>(kt, lane, pay, qsl, r4, dh, dl); break;
        case 3: score_slot<3, NQ>(kt, lane, pay, qsl, r4, dh, dl); break;
        case 4: score_slot<4, NQ>(kt, lane, pay, qsl, r4, dh, dl); break;
        case 5: score_slot<5, NQ>(kt, lane, pay, qsl, r4, dh, dl); break;
        case 6: score_slot<6, NQ>(kt, lane, pay, qsl, r4, dh, dl); break;
        case 7: score_slot<7, NQ>(kt, lane, pay, qsl, r4, dh, dl); break;
        default: score_slot<8, NQ>(kt, lane, pay, qsl, r4, dh, dl); break;
      }
      const float sk = h2f(meta) * E2, zk = h2f(meta >> 16);
#pragma unroll
      for (int q = 0; q < NQ; ++q)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          sc[4 * q + j] += sk * __builtin_fmaf(dl[q][j], 1.0f / 2048.0f, dh[q][j]) + zk * qbar_s[(4 * q + j) * 4 + g];
    }

    // ---- online softmax (log2 domain) against a reference m that moves only when
    // a score exceeds it by more than RESCALE_SLACK: weights stay <= 2^RESCALE_SLACK,
    // and the rescale of the running sums is rare after the first tile ----
    float p[NH], x[NH];
    bool over = false;
#pragma unroll
    for (int h = 0; h < NH; ++h) {
      x[h] = (valid && h < nqh) ? sc[h] : -__builtin_inff();
      over = over || x[h] > m_run[h] + RESCALE_SLACK;
    }
    if (__any(over)) {  // rare after the first tile: one branch for all heads
#pragma unroll
      for (int h = 0; h < NH; ++h) {
        if (__any(x[h] > m_run[h] + RESCALE_SLACK)) {
          const float mn = __builtin_fmaxf(m_run[h], wave_max_all(x[h]));
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
      }
    }
#pragma unroll
    for (int h = 0; h < NH; ++h) {
      p[h] = x[h] != -__builtin_inff() ? __builtin_amdgcn_exp2f(x[h] - m_run[h]) : 0.0f;
      l_run[h] += p[h];
    }
    // softmax weight times value scale, as bf16 hi/lo rows; zero-point terms per lane
#pragma unroll
    for (int sl = 0; sl < NG; ++sl) {
      if (sl >= kvv.n) continue;
      // tokens past n_tokens hold whatever the cache holds there: zero their metadata
      const uint32_t meta = valid ? vt[sl * TROW + lane] : 0u;
      const float sv = h2f(meta), zv = h2f(meta >> 16);
      uint16_t* ws = wt + sl * 2 * NH * WROW;  // rows: hi of heads 0..NH-1, then lo
#pragma unroll
      for (int h = 0; h < NH; h += 2) {  // two heads per packed conversion
        zacc[h][sl] = __builtin_fmaf(p[h], zv, zacc[h][sl]);
        zacc[h + 1][sl] = __builtin_fmaf(p[h + 1], zv, zacc[h + 1][sl]);
        const float w0 = p[h] * sv, w1 = p[h + 1] * sv;
        const uint32_t hb = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{w0, w1}, bf16x2));
        const float h0 = __builtin_bit_cast(float, hb << 16), h1 = __builtin_bit_cast(float, hb & 0xFFFF0000u);
        const uint32_t lb = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{w0 - h0, w1 - h1}, bf16x2));
        ws[h * WROW + lane] = (uint16_t)hb;
        ws[(h + 1) * WROW + lane] = (uint16_t)(hb >> 16);
        ws[(NH + h) * WROW + lane] = (uint16_t)lb;
        ws[(NH + h + 1) * WROW + lane] = (uint16_t)(lb >> 16);
      }
    }
    __builtin_amdgcn_wave_barrier();

    // ---- value accumulation over the kept value coefficients ----
    const bf16x8 negone = as_bf16x8(u32x4{0xBF80BF80u, 0xBF80BF80u, 0xBF80BF80u, 0xBF80BF80u});
    constexpr int AR = STACK ? 2 * NH : NH;  // weight rows of one MFMA (8, 12 or 16)
    static_assert(AR >= 8 && AR <= 16, "rows past AR re-read row col - AR");
    uint32_t vmagic = 0x3F803F80u;  // exponent of 1.0 in both halves, in a VGPR (see value_codes2)
    asm volatile("" : "+v"(vmagic));
#pragma unroll
    for (int sl = 0; sl < NG; ++sl) {
      if (sl >= kvv.n) continue;
      const uint16_t* ws = wt + sl * 2 * NH * WROW;
      const int B = kvv.bits[sl], pay = kvv.pay[sl];
      auto body = [&](auto cls) {
        constexpr int CLS = decltype(cls)::value;
#pragma unroll
        for (int th = 0; th < 2; ++th) {
          const int tok0 = 32 * th + 8 * kq;
          // stacked: rows 0..2NH-1 = hi then lo; otherwise hi rows and lo rows separately.
          // Lanes of MFMA rows past the weight rows read a weight row again (no masked
          // load): those accumulator rows are never read.
          const int arow = col < AR ? col : col - AR;
          const bf16x8 aw = as_bf16x8(*reinterpret_cast<const u32x4*>(ws + arow * WROW + tok0));
          bf16x8 awl = bf16x8{};
          if constexpr (!STACK) awl = as_bf16x8(*reinterpret_cast<const u32x4*>(ws + (NH + arow) * WROW + tok0));
          // MFMA column col of block c2 is in-group coefficient 2 col + c2
          u32x4 vc[2];
          value_codes2<CLS>(vt, pay, kvv.used, B, (int)((voffs >> (8 * sl)) & 0xFFu), tok0, vmagic, vc[0], vc[1]);
#pragma unroll
          for (int c2 = 0; c2 < 2; ++c2) {
            const bf16x8 bop = as_bf16x8(vc[c2]);
            f32x4 acc = vacc[sl][c2];
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aw, bop, acc, 0, 0, 0);
            if constexpr (CLS != 2) acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aw, negone, acc, 0, 0, 0);
            if constexpr (!STACK) {
              acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(awl, bop, acc, 0, 0, 0);
              if constexpr (CLS != 2) acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(awl, negone, acc, 0, 0, 0);
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

  write_chunk_partial<NQ>(a, b, kv, chunk, tid, wave, lane, kq, col, ok, Kv, m_run, l_run, zacc, vacc, smem);
}

// ---------------------------------------------------------------------------
// Combine chunk partials and inverse-rotate: one workgroup per (query head,
// sequence). Every global load is issued before the first use: the V_V rows,
// m_V and bits, then the partials (eight thread groups of 128 take every eighth
// chunk, merged with a running maximum in batches of CB chunks); the group
// states are then merged in LDS.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(1024) void combine_kernel(AttnArgs a) {
  constexpr int CB = 12;  // 8 x 12 = 96 chunks per round: one round of loads for ~768 scan workgroups over 8 heads
  __shared__ float accs[8][D];
  __shared__ float chat[D];
  __shared__ float gm[8], gl[8];
  const int hq = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  const int j = tid & 127, grp = tid >> 7;
  const int kv = hq / a.n_qh;
  const int s = b * a.n_kv_heads + kv;
  // rotation operands: output row i = tid / 8, coefficients 16 (tid % 8) .. + 15
  const int ri = tid >> 3, rpart = tid & 7;
  const f32x4* Vr = reinterpret_cast<const f32x4*>(a.basis_v + (int64_t)s * D * D + (int64_t)ri * D + 16 * rpart);
  const f32x4 v0 = Vr[0], v1 = Vr[1], v2 = Vr[2], v3 = Vr[3];
  const float mv = tid < D ? a.mean_v[(int64_t)s * D + tid] : 0.0f;
  const uint32_t bw = *reinterpret_cast<const uint32_t*>(a.bits_v + (int64_t)s * NG);

  const float* ph = a.partial + ((int64_t)b * a.n_q_heads + hq) * a.n_chunks * PART;
  const int nch = a.n_chunks;
  const int g = j >> 5;
  float M = -__builtin_inff(), L = 0.0f, A = 0.0f;
  for (int c0 = grp; c0 < nch; c0 += 8 * CB) {
    float m[CB], l[CB], z[CB], x[CB];
#pragma unroll
    for (int k = 0; k < CB; ++k) {
      const int c = c0 + 8 * k;
      const float* pc = ph + (int64_t)(c < nch ? c : grp) * PART;
      m[k] = c < nch ? pc[0] : -__builtin_inff();
      l[k] = pc[1];
      z[k] = pc[2 + g];
      x[k] = pc[8 + j];
    }
    float mb = M;
#pragma unroll
    for (int k = 0; k < CB; ++k) mb = __builtin_fmaxf(mb, m[k]);
    if (mb != -__builtin_inff()) {
      const float r = (M == -__builtin_inff()) ? 0.0f : __builtin_amdgcn_exp2f(M - mb);
      L *= r;
      A *= r;
#pragma unroll
      for (int k = 0; k < CB; ++k) {
        const float w = (m[k] == -__builtin_inff()) ? 0.0f : __builtin_amdgcn_exp2f(m[k] - mb);
        L = __builtin_fmaf(w, l[k], L);
        A = __builtin_fmaf(w, z[k] + x[k], A);
      }
      M = mb;
    }
  }
  if (j == 0) {
    gm[grp] = M;
    gl[grp] = L;
  }
  __syncthreads();
  float Mx = gm[0];
#pragma unroll
  for (int i = 1; i < 8; ++i) Mx = __builtin_fmaxf(Mx, gm[i]);
  const float f = (M == -__builtin_inff()) ? 0.0f : __builtin_amdgcn_exp2f(M - Mx);
  accs[grp][j] = f * A;
  if (j == 0) gl[grp] = f * L;  // each group reads only its own entry above
  __syncthreads();
  if (tid < D) {
    float sacc = 0.0f, sl = 0.0f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      sacc += accs[i][tid];
      sl += gl[i];
    }
    const bool kept = ((bw >> (8 * (tid >> 5))) & 0xFFu) != 0u;
    chat[tid] = (kept ? sacc / sl : 0.0f) + mv;
  }
  __syncthreads();
  // out_i = sum_j chat_j V[i][j]: eight lanes per output row, 16 contiguous j each
  const float* ch = chat + 16 * rpart;
  float o = 0.0f;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    o = __builtin_fmaf(ch[k], v0[k], o);
    o = __builtin_fmaf(ch[4 + k], v1[k], o);
    o = __builtin_fmaf(ch[8 + k], v2[k], o);
    o = __builtin_fmaf(ch[12 + k], v3[k], o);
  }
  o += __shfl_xor(o, 1);
  o += __shfl_xor(o, 2);
  o += __shfl_xor(o, 4);
  if (rpart == 0) a.out[((int64_t)b * a.n_q_heads + hq) * D + ri] = o;
}

}  // namespace spectra_dev

namespace spectra {
using namespace spectra_dev;

size_t attention_partial_floats(int32_t batch, int32_t n_q_heads, int32_t n_chunks) {
  return (size_t)batch * n_q_heads * n_chunks * PART;
}
// Split of each (sequence, kv head) token range into chunks of whole tiles: about
// 768 workgroups of four wavefronts, >= 4 tiles per wavefront, over all tiles but
// the last; the last tile is a chunk of its own (in a decode step its workgroup
// also appends the new token).
int32_t attention_chunks(int32_t batch, int32_t n_kv_heads, int64_t n_tokens, int32_t* tiles_per_chunk) {
  const int64_t n_tiles = (n_tokens + 63) / 64;
  const int64_t body = n_tiles > 0 ? n_tiles - 1 : 0;
  const int64_t groups = (int64_t)batch * n_kv_heads;
  const int64_t want = (768 + groups - 1) / groups;
  int64_t tpc = (body + want - 1) / want;
  if (tpc < 16) tpc = 16;
  if (tpc > body) tpc = body > 0 ? body : 1;
  const int64_t nch = (body + tpc - 1) / tpc + 1;
  *tiles_per_chunk = (int32_t)tpc;
  return (int32_t)nch;
}

template <int NQ, int PK, int PV, bool EXACT>
static void launch_nq_pw(const AttnArgs& a, hipStream_t st) {
  const int wpw = PK > 0 ? PK + PV : a.Wk + a.Wv;
  size_t tiles = (size_t)WAVES * wpw * TROW * 4 + (size_t)attn_wt_bytes(NQ);
  size_t merge = (size_t)WAVES * (NQ <= 2 ? 8 * NQ : 4 * NQ) * AROW * 4;  // per-wave value sums
  size_t lds = tiles > merge ? tiles : merge;
  if ((size_t)qprep_scratch_bytes(NQ) > lds) lds = qprep_scratch_bytes(NQ);
  if (a.app_k && (size_t)append_stage_bytes(a.app_f32 != 0) > lds) lds = append_stage_bytes(a.app_f32 != 0);
  // more (sequence, kv head) groups than XCDs: chunks of a group kept on one XCD
  AttnArgs g = a;
  g.group_major = a.n_kv_heads * a.batch > 8 ? 1 : 0;
  const dim3 grid = g.group_major ? dim3(a.n_chunks * a.n_kv_heads * a.batch, 1, 1) : dim3(a.n_chunks, a.n_kv_heads, a.batch);
  hipLaunchKernelGGL((attn_kernel<NQ, PK, PV, EXACT>), grid, dim3(256), lds, st, g);
}

// Prefetch shapes. Up to eight query heads per KV head, records of unequal width
// get their own shapes: exact (4, 12) and (12, 4) (the 8x budget split a quarter
// or three quarters to the keys), otherwise (8, 16) or (16, 8); at most 24
// prefetch registers keep three wavefronts per SIMD.
template <int NQ>
static void launch_nq(const AttnArgs& a, hipStream_t st) {
  const int wk = a.Wk, wv = a.Wv;
  if constexpr (NQ <= 2) {
    if (wk == 4 && wv == 12) return launch_nq_pw<NQ, 4, 12, true>(a, st);
    if (wk == 12 && wv == 4) return launch_nq_pw<NQ, 12, 4, true>(a, st);
    if (wk <= 8 && wv > 8 && wv <= 16) return launch_nq_pw<NQ, 8, 16, false>(a, st);
    if (wv <= 8 && wk > 8 && wk <= 16) return launch_nq_pw<NQ, 16, 8, false>(a, st);
  }
  if (wk == 8 && wv == 8)
    launch_nq_pw<NQ, 8, 8, true>(a, st);
  else if (wk <= 8 && wv <= 8)
    launch_nq_pw<NQ, 8, 8, false>(a, st);
  else if (wk == 16 && wv == 16)
    launch_nq_pw<NQ, 16, 16, true>(a, st);
  else if (wk <= 16 && wv <= 16)
    launch_nq_pw<NQ, 16, 16, false>(a, st);
  else
    launch_nq_pw<NQ, 0, 0, false>(a, st);
}

hipError_t launch_combine(const AttnArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(combine_kernel, dim3(a.n_q_heads, a.batch), dim3(1024), 0, st, a);
  return hipGetLastError();
}

static hipError_t launch_scan_combine(const AttnArgs& a, hipStream_t st) {
  switch ((a.n_qh + 3) / 4) {
    case 1: launch_nq<1>(a, st); break;
    case 2: launch_nq<2>(a, st); break;
    case 3: launch_nq<3>(a, st); break;
    default: launch_nq<4>(a, st); break;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_combine(a, st);
}

// Decode-step attention; with a.app_k set, the decode step (append first): the
// scan kernel, then the chunk combine.
hipError_t launch_attention(const AttnArgs& a, hipStream_t st) { return launch_scan_combine(a, st); }

}  // namespace spectra
