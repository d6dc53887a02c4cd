// Per-layer cross-head latent (Sec. 3.1 applied to a layer's whole KV vector, the
// geometry of Sec. 4.1 and App. F: d = d_kv = n_kv_heads x 128, latent groups of
// g = 64 coefficients). A stream is one (sequence, layer, tensor) T x d matrix; the
// record format is the per-head one with 64-coefficient groups (one metadata word
// per kept group, then 2b payload words per kept group at b bits).
//
// Kernels:
//   layer_gram_kernel     fp64 second moment x^T x of every stream, split over
//                         token ranges (deterministic partial sums), 64 x 64 tiles;
//   layer_moments_kernel  sums the partials in a fixed order and adds the column sums;
//   layer_encode_kernel   c = x V - m on v_mfma_f32_32x32x16_bf16 (bf16 tokens exact,
//                         the fp32 basis as three bf16 parts staged through LDS), then
//                         per token and kept group fp16 zero-point and scale, codes,
//                         packing; one workgroup per (256 tokens, kept group, stream);
//   layer_decode_kernel   x_hat = sum_G (s_tG q_tG + z_tG 1) V_G^T + m V^T: codes
//                         unpacked once per workgroup into LDS as bf16, the basis
//                         columns of the group as three bf16 parts, the group's
//                         per-token scale applied after its product; one workgroup per
//                         (128 tokens, 128 channels, stream).
#include "device_common.hpp"
#include "kernels.hpp"
#include "layer.hpp"

namespace spectra_dev {

constexpr int LG = 64;  // latent group size of the per-layer geometry

// Kept group `slot` of a per-layer stream (widths bits_s[0..ng)): group index, width
// and first payload word; also the number of kept groups and the record words used.
struct LayerSlot {
  int grp, b, pay, n_kept, used;
  bool ok;  // every width in [0, 8]
};
__device__ __forceinline__ LayerSlot layer_slot(const uint8_t* __restrict__ bits_s, int ng, int slot) {
  LayerSlot r{-1, 0, 0, 0, 0, true};
  int n = 0, payw = 0;
  for (int g = 0; g < ng; ++g) {
    const int b = bits_s[g];
    if (b > 8) r.ok = false;
    if (b > 0) {
      if (n == slot) {
        r.grp = g;
        r.b = b;
        r.pay = payw;  // relative to the end of the metadata words
      }
      ++n;
      payw += 2 * b;
    }
  }
  r.n_kept = n;
  r.pay += n;
  r.used = n + payw;
  return r;
}

// ---------------------------------------------------------------------------
// Moments
// ---------------------------------------------------------------------------
template <bool F32IN>
__device__ __forceinline__ double load_x(const void* x, int64_t i) {
  if constexpr (F32IN)
    return (double)reinterpret_cast<const float*>(x)[i];
  else
    return (double)bf2f(reinterpret_cast<const uint16_t*>(x)[i]);
}

// partial[s][kc] = [sum over tokens [kc * ck, min(n, (kc + 1) ck)) of x_t^T x_t (d x d),
// then the column sums over the same tokens (d)], 64 x 64 output tile per workgroup,
// 16-token steps staged in LDS, 4 x 4 outputs per thread. The workgroups of the first
// tile column also sum their 64 channels: each thread over the tokens it stages (every
// 16th), then the 16 shares of a channel in order.
template <bool F32IN>
__global__ __launch_bounds__(256) void layer_gram_kernel(LayerGramArgs g) {
  __shared__ double As[16][65];
  __shared__ double Bs[16][65];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int i0 = blockIdx.x * 64, j0 = blockIdx.y * 64;
  const int s = blockIdx.z / g.k_split, kc = blockIdx.z % g.k_split;
  const int64_t t_begin = (int64_t)kc * g.chunk_tokens;
  const int64_t t_end = t_begin + g.chunk_tokens < g.n ? t_begin + g.chunk_tokens : g.n;
  const int64_t xb = (int64_t)s * g.stream_stride;
  const bool col_sums = blockIdx.y == 0;  // uniform over the workgroup
  double csum[4] = {0.0, 0.0, 0.0, 0.0};
  double acc[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[a][b] = 0.0;
  for (int64_t t0 = t_begin; t0 < t_end; t0 += 16) {
    // 16 tokens x 64 channels of each operand: thread -> (token tid >> 4, channels 4 (tid & 15) ..)
    {
      const int tk = tid >> 4, c4 = 4 * (tid & 15);
      const int64_t t = t0 + tk;
      const bool in = t < t_end;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const double xa = in ? load_x<F32IN>(g.x, xb + t * g.token_stride + i0 + c4 + e) : 0.0;
        As[tk][c4 + e] = xa;
        Bs[tk][c4 + e] = in ? load_x<F32IN>(g.x, xb + t * g.token_stride + j0 + c4 + e) : 0.0;
        if (col_sums) csum[e] += xa;
      }
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      double a[4], b[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) a[q] = As[k][ty + 16 * q];
#pragma unroll
      for (int q = 0; q < 4; ++q) b[q] = Bs[k][tx + 16 * q];
#pragma unroll
      for (int p = 0; p < 4; ++p)
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[p][q] = __builtin_fma(a[p], b[q], acc[p][q]);
    }
    __syncthreads();
  }
  const int64_t dd = (int64_t)g.d * g.d;
  double* out = g.partial + ((int64_t)s * g.k_split + kc) * (dd + g.d);
#pragma unroll
  for (int p = 0; p < 4; ++p)
#pragma unroll
    for (int q = 0; q < 4; ++q) out[(int64_t)(i0 + ty + 16 * p) * g.d + j0 + tx + 16 * q] = acc[p][q];
  if (col_sums) {
    const int tk = tid >> 4, c4 = 4 * (tid & 15);
#pragma unroll
    for (int e = 0; e < 4; ++e) As[tk][c4 + e] = csum[e];  // the loop ended with a barrier
    __syncthreads();
    if (tid < 64) {
      double cs = 0.0;
      for (int k = 0; k < 16; ++k) cs += As[k][tid];
      out[dd + i0 + tid] = cs;
    }
  }
}

// moments[s] = sum_kc partial[s][kc] ([d x d Gram, d column sums]), partials added in
// ascending kc.
template <bool F32IN>
__global__ __launch_bounds__(256) void layer_moments_kernel(LayerGramArgs g) {
  const int s = blockIdx.y;
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t dd = (int64_t)g.d * g.d;
  double* mom = g.moments + (int64_t)s * (dd + g.d);
  if (e < dd + g.d) {
    const double* p = g.partial + (int64_t)s * g.k_split * (dd + g.d) + e;
    double acc = 0.0;
    for (int kc = 0; kc < g.k_split; ++kc) acc += p[kc * (dd + g.d)];
    mom[e] = acc;
  }
}

// ---------------------------------------------------------------------------
// Encode
// ---------------------------------------------------------------------------
// Workgroups of a one-dimensional grid over (token range, block) are dispatched to the
// eight XCDs in turn (workgroup i to XCD i mod 8). Numbering them i = 8 (nb r + blk) + x
// with token range 8 r + x puts every block of a range on the same XCD, close together
// in time, so that XCD's L2 serves the range's rows to all of them instead of every XCD
// fetching them from HBM. Ranges past the last one (the grid is rounded up to whole
// groups of eight) get range = -1.
__host__ __device__ constexpr unsigned xcd_major_grid(int n_ranges, int nb) { return 8u * (unsigned)nb * (unsigned)((n_ranges + 7) / 8); }
__device__ __forceinline__ void xcd_major_block(int n_ranges, int nb, int& range, int& blk) {
  const int i = (int)blockIdx.x, x = i & 7, j = i >> 3;
  blk = j % nb;
  range = 8 * (j / nb) + x;
  if (range >= n_ranges) range = -1;
}

constexpr int LE_TOK = 256;       // tokens per workgroup (eight wavefronts of 32)
constexpr int LE_KC = 64;         // basis rows per staged chunk
constexpr int LE_KP = LE_KC + 8;  // bf16 per staged row (144-byte rows, 16-byte aligned)

// Row of the staged 64-row operand that holds group coefficient c: within each
// 32-row block, row r feeds coefficient 16 ((r >> 2) & 1) + (r & 3) + 4 (r >> 3), so
// that after the 32x32 product lane half h holds coefficients 16h .. 16h + 15.
__device__ __forceinline__ int le_row(int c) {
  const int cc = c & 31;
  return 32 * (c >> 5) + (cc & 3) + 4 * (cc >> 4) + 8 * ((cc >> 2) & 3);
}

__global__ __launch_bounds__(512, 4) void layer_encode_kernel(LayerEncodeArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t vs[3][64][LE_KP];
  const int s = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, col = lane & 31, h = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: the staging rows are scalar
  const int d = a.d, ng = d / LG;
  int range, slot;
  xcd_major_block((int)((a.n + LE_TOK - 1) / LE_TOK), ng, range, slot);
  if (range < 0) return;
  const LayerSlot ks = layer_slot(a.bits + (int64_t)s * ng, ng, slot);
  const int64_t sbase = (int64_t)s * a.t_cap * a.W;
  const int64_t wg_tok = (int64_t)range * LE_TOK;
  if (!ks.ok || ks.used > a.W) return;  // width table inconsistent with the record: write nothing

  // words past the used ones are zero: written by the slot-0 workgroup
  if (slot == 0 && ks.used < a.W) {
    const int nw = a.W - ks.used;
    for (int e = tid; e < LE_TOK * nw; e += 512) {
      const int64_t i = wg_tok + (e % LE_TOK);
      if (i < a.n) a.packed[rec_word(sbase, a.t0 + i, a.W, ks.used + e / LE_TOK)] = 0u;
    }
  }
  if (slot >= ks.n_kept) return;  // uniform over the workgroup

  const int64_t i_tok = wg_tok + 32 * wave + col;
  const bool valid = i_tok < a.n;
  const int64_t i_ld = valid ? i_tok : a.n - 1;
  const uint16_t* xr = reinterpret_cast<const uint16_t*>(a.x) + (int64_t)s * a.stream_stride + i_ld * a.token_stride;
  const float* V = a.basis + (int64_t)s * d * d + LG * ks.grp;

  // staging map: thread -> (group coefficient sc, basis rows sk .. sk + 7 of the chunk)
  const int sc = tid & 63, sk = 8 * wave, srow = le_row(sc);
  float pre[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) pre[i] = V[(int64_t)(sk + i) * d + sc];
  u32x4 xb[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) xb[k] = *reinterpret_cast<const u32x4*>(xr + 16 * k + 8 * h);

  // Accumulation order, for fp32 accuracy over d up to 1024 terms: the products with
  // the basis' high bf16 part are summed per 64-row chunk and the chunk sums added
  // into the running totals; the two low parts (2^-8 and 2^-16 of the value) go to a
  // separate accumulator whose rounding is correspondingly small.
  f32x16 acc0 = {}, acc1 = {}, sm0 = {}, sm1 = {};
  const int nk = d / LE_KC;
  for (int kc = 0; kc < nk; ++kc) {
    {
      uint32_t p0[8], p1[8], p2[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) split3(pre[i], p0[i], p1[i], p2[i]);
      *reinterpret_cast<u32x4*>(&vs[0][srow][sk]) = u32x4{pack2(p0[0], p0[1]), pack2(p0[2], p0[3]), pack2(p0[4], p0[5]), pack2(p0[6], p0[7])};
      *reinterpret_cast<u32x4*>(&vs[1][srow][sk]) = u32x4{pack2(p1[0], p1[1]), pack2(p1[2], p1[3]), pack2(p1[4], p1[5]), pack2(p1[6], p1[7])};
      *reinterpret_cast<u32x4*>(&vs[2][srow][sk]) = u32x4{pack2(p2[0], p2[1]), pack2(p2[2], p2[3]), pack2(p2[4], p2[5]), pack2(p2[6], p2[7])};
    }
    __syncthreads();
    if (kc + 1 < nk) {
#pragma unroll
      for (int i = 0; i < 8; ++i) pre[i] = V[(int64_t)((kc + 1) * LE_KC + sk + i) * d + sc];
    }
    f32x16 ch0 = {}, ch1 = {};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const bf16x8 xk = as_bf16x8(xb[k]);
#pragma unroll
      for (int p = 0; p < 3; ++p) {
        const bf16x8 a0 = as_bf16x8(*reinterpret_cast<const u32x4*>(&vs[p][col][16 * k + 8 * h]));
        const bf16x8 a1 = as_bf16x8(*reinterpret_cast<const u32x4*>(&vs[p][32 + col][16 * k + 8 * h]));
        if (p == 0) {
          ch0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, xk, ch0, 0, 0, 0);
          ch1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, xk, ch1, 0, 0, 0);
        } else {
          sm0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, xk, sm0, 0, 0, 0);
          sm1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, xk, sm1, 0, 0, 0);
        }
      }
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      acc0[i] += ch0[i];
      acc1[i] += ch1[i];
    }
    if (kc + 1 < nk) {
#pragma unroll
      for (int k = 0; k < 4; ++k) xb[k] = *reinterpret_cast<const u32x4*>(xr + (kc + 1) * LE_KC + 16 * k + 8 * h);
    }
    __syncthreads();
  }

  // lane (h, col): coefficients 16h + i (acc0) and 32 + 16h + i (acc1) of token col. The
  // lane's token and half are recomputed here rather than held in registers across the loop.
  int tid_e = tid;
  asm volatile("" : "+v"(tid_e));
  const int he = (tid_e & 63) >> 5;
  const int64_t i_tok_e = wg_tok + 32 * wave + (tid_e & 31);
  const bool valid_e = i_tok_e < a.n;
  const int64_t i_ld_e = valid_e ? i_tok_e : a.n - 1;
  const float* mg = a.mean + (int64_t)s * d + LG * ks.grp;
  float c[32];
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    c[i] = (acc0[i] + sm0[i]) - mg[16 * he + i];
    c[16 + i] = (acc1[i] + sm1[i]) - mg[32 + 16 * he + i];
  }
  if (a.lscale) {  // square-root split: the cached coordinate is (x V - m)_j f_j
    const float* fg = a.lscale + (int64_t)s * d + LG * ks.grp;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      c[i] *= fg[16 * he + i];
      c[16 + i] *= fg[32 + 16 * he + i];
    }
  }
  float lo = c[0], hi = c[0];
#pragma unroll
  for (int i = 1; i < 32; ++i) {
    lo = __builtin_fminf(lo, c[i]);
    hi = __builtin_fmaxf(hi, c[i]);
  }
  lo = __builtin_fminf(lo, __shfl_xor(lo, 32));
  hi = __builtin_fmaxf(hi, __shfl_xor(hi, 32));
  const int64_t base = rec_word(sbase, a.t0 + i_ld_e, a.W, 0);
  with_bits(ks.b, [&](auto bc) {
    constexpr int B = decltype(bc)::value;
    constexpr float LEV = (float)((1 << B) - 1);
    const uint32_t z16 = f2h_sat(lo);
    const float z = h2f(z16);
    const uint32_t s16 = f2h_sat(__builtin_fmaxf(hi - z, 0.0f) / LEV);
    const float sf = h2f(s16);
    const float rinv = sf > 0.0f ? 1.0f / sf : 0.0f;
    uint32_t q0[16], q1[16], P0[4], P1[4];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      q0[i] = (uint32_t)__builtin_fminf(__builtin_fmaxf(__builtin_rintf((c[i] - z) * rinv), 0.0f), LEV);
      q1[i] = (uint32_t)__builtin_fminf(__builtin_fmaxf(__builtin_rintf((c[16 + i] - z) * rinv), 0.0f), LEV);
    }
    pack16<B>(q0, P0);
    pack16<B>(q1, P1);
    if (he == 0 && valid_e) a.packed[base + (int64_t)slot * TILE] = s16 | (z16 << 16);
    store_payload<B>(a.packed, base, ks.pay, P0, he, valid_e);
    store_payload<B>(a.packed, base, ks.pay + B, P1, he, valid_e);
  });
}

// ---------------------------------------------------------------------------
// Decode (Mode A)
// ---------------------------------------------------------------------------
// One workgroup: LD_CH = 64 output channels x LD_NT = 2 tiles of 128 tokens. The
// group's basis operands and the mean term m V^T are built once per workgroup and
// serve both tiles (the L2 reads of basis rows per token are what bound this kernel).
// Registers are capped at 128 per lane so that two workgroups (four wavefronts per
// SIMD) share a CU and hide each other's load latency; per-piece shift amounts are
// scalar and record offsets are recomputed per slot, so almost nothing spills.
constexpr int LD_TOK = 128;       // tokens per tile
constexpr int LD_NT = 2;          // tiles per workgroup
constexpr int LD_CH = 64;         // output channels per workgroup
constexpr int LD_P = LG + 8;      // bf16 per LDS row (144 bytes)
constexpr int LD_R = 2 * LD_NT;   // staged (token, 8-code) pieces per thread

__global__ __launch_bounds__(512, 4) void layer_decode_kernel(LayerDecodeArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t vsl[3][LD_CH][LD_P];          // basis columns of the group, [channel][coef]
  __shared__ __attribute__((aligned(16))) uint16_t cod[LD_NT][LD_TOK][LD_P];     // codes, [tile][token][coef]
  __shared__ __attribute__((aligned(16))) float sl[LD_NT][LD_TOK], zl[LD_NT][LD_TOK], vsum[LD_CH], bias[LD_CH];
  const int s = blockIdx.z;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, col = lane & 31, h = lane >> 5;
  const int d = a.d, ng = d / LG;
  int range, cblk;
  xcd_major_block((int)((a.n + LD_TOK * LD_NT - 1) / (LD_TOK * LD_NT)), d / LD_CH, range, cblk);
  if (range < 0) return;
  const int ch0 = cblk * LD_CH;
  const int64_t tok0 = (int64_t)range * (LD_TOK * LD_NT);
  const int64_t sbase = (int64_t)s * a.t_cap * a.W;
  const float* Vs = a.basis + (int64_t)s * d * d;
  const uint8_t* bits_s = a.bits + (int64_t)s * ng;
  const LayerSlot k0 = layer_slot(bits_s, ng, 0);
  if (!k0.ok || k0.used > a.W) return;  // width table inconsistent with the record: write nothing
  const int n_kept = k0.n_kept;

  // per-thread shares of a slot's staging: basis row (channel tid >> 3) coefficients
  // 8 (tid & 7) .. + 7; piece r: token u_r = (tid + 512 r) & 127 of tile (tid + 512 r) >> 10,
  // coefficients 8 k8_r .. + 7 with k8_r = ((tid + 512 r) >> 7) & 7 (uniform in a wavefront)
  const int vc = tid >> 3, vq = tid & 7;
  // ((tid + 512 r) >> 7) & 7 = (kq + 4 r) & 7 with kq = tid >> 7, uniform in a wavefront:
  // held in a scalar register, so the shift amounts derived from it are scalar too
  const int kq = __builtin_amdgcn_readfirstlane(tid >> 7);
  float vpre[8];
  uint32_t wpre[LD_R][3], mpre[LD_R];
  auto prefetch = [&](const LayerSlot& ks, int slot) {
    const float* vr = Vs + (int64_t)(ch0 + vc) * d + LG * ks.grp + 8 * vq;
#pragma unroll
    for (int i = 0; i < 8; ++i) vpre[i] = vr[i];
    // record word 0 of the thread's token in each tile, recomputed per call rather than
    // held in registers across the slot loop
    int u = tid & (LD_TOK - 1);
    asm volatile("" : "+v"(u));
    int64_t tb[LD_NT];
#pragma unroll
    for (int t2 = 0; t2 < LD_NT; ++t2) {
      const int64_t i = tok0 + (int64_t)t2 * LD_TOK + u;
      tb[t2] = rec_word(sbase, a.t0 + (i < a.n ? i : a.n - 1), a.W, 0);
    }
#pragma unroll
    for (int r = 0; r < LD_R; ++r) {
      const int k8 = (kq + 4 * r) & 7, t2 = r >> 1;
      const int P = 8 * k8 * ks.b, w0 = P >> 5, wl = (P + 8 * ks.b - 1) >> 5;  // payload words extract8 reads
#pragma unroll
      for (int i = 0; i < 3; ++i) wpre[r][i] = (w0 + i <= wl) ? a.packed[tb[t2] + (int64_t)(ks.pay + w0 + i) * TILE] : 0u;
      mpre[r] = a.packed[tb[t2] + (int64_t)slot * TILE];
    }
  };

  // bias = m V^T over all d coefficients: wavefront w takes channels 8w .. 8w + 7,
  // each row read by the whole wavefront (16 values per lane), then a wavefront sum
  {
    const float* mr = a.mean + (int64_t)s * d;
    float mv[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) mv[i] = (64 * i + lane < d) ? mr[64 * i + lane] : 0.0f;
    float part[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      const float* vr = Vs + (int64_t)(ch0 + 8 * wave + c) * d;
      float acc = 0.0f;
#pragma unroll
      for (int i = 0; i < 16; ++i)
        if (64 * i + lane < d) acc = __builtin_fmaf(mv[i], vr[64 * i + lane], acc);
      part[c] = acc;
    }
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      float v = part[c];
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
      if (lane == c) bias[8 * wave + c] = v;
    }
  }

  // wavefront -> channel block cb (32 channels), tile tl, token blocks 2 tp, 2 tp + 1
  // (32 tokens each) of that tile
  const int cb = wave & 1, tl = (wave >> 1) >> 1, tp = (wave >> 1) & 1;
  f32x16 out[2] = {f32x16{}, f32x16{}};
  LayerSlot ks = k0;
  if (n_kept > 0) prefetch(ks, 0);
  for (int slot = 0; slot < n_kept; ++slot) {
    // stage the prefetched slot: codes as bf16 and metadata, basis parts and sums
    int kqs = kq;
    asm volatile("" : "+s"(kqs));  // shift amounts recomputed per slot (scalar), not hoisted
#pragma unroll
    for (int r = 0; r < LD_R; ++r) {
      const int u = tid & (LD_TOK - 1), k8 = (kqs + 4 * r) & 7, t2 = r >> 1;
      const int w0 = (8 * k8 * ks.b) >> 5;
      with_bits(ks.b, [&](auto bc) {
        constexpr int B = decltype(bc)::value;
        uint32_t cd[8];
        extract8<B>([&](int i) { return wpre[r][i - w0]; }, 8 * k8, cd);
        *reinterpret_cast<u32x4*>(&cod[t2][u][8 * k8]) =
            u32x4{int_to_bf16_pair(cd[0], cd[1]), int_to_bf16_pair(cd[2], cd[3]), int_to_bf16_pair(cd[4], cd[5]),
                  int_to_bf16_pair(cd[6], cd[7])};
      });
      if (k8 == 0) {
        sl[t2][u] = h2f(mpre[r]);
        zl[t2][u] = h2f(mpre[r] >> 16);
      }
    }
    {
      if (a.lscale) {  // square-root split: c_hat_j / f_j, folded into the basis columns
        const float* fr = a.lscale + (int64_t)s * d + LG * ks.grp + 8 * vq;
#pragma unroll
        for (int i = 0; i < 8; ++i) vpre[i] = vpre[i] * (1.0f / fr[i]);
      }
      float sum = 0.0f;
#pragma unroll
      for (int i = 0; i < 8; ++i) sum += vpre[i];
      sum += __shfl_xor(sum, 1);
      sum += __shfl_xor(sum, 2);
      sum += __shfl_xor(sum, 4);
      if (vq == 0) vsum[vc] = sum;
      uint32_t p0[8], p1[8], p2[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) split3(vpre[i], p0[i], p1[i], p2[i]);
      const int j = 8 * vq;
      *reinterpret_cast<u32x4*>(&vsl[0][vc][j]) = u32x4{pack2(p0[0], p0[1]), pack2(p0[2], p0[3]), pack2(p0[4], p0[5]), pack2(p0[6], p0[7])};
      *reinterpret_cast<u32x4*>(&vsl[1][vc][j]) = u32x4{pack2(p1[0], p1[1]), pack2(p1[2], p1[3]), pack2(p1[4], p1[5]), pack2(p1[6], p1[7])};
      *reinterpret_cast<u32x4*>(&vsl[2][vc][j]) = u32x4{pack2(p2[0], p2[1]), pack2(p2[2], p2[3]), pack2(p2[4], p2[5]), pack2(p2[6], p2[7])};
    }
    __syncthreads();
    if (slot + 1 < n_kept) {
      ks = layer_slot(bits_s, ng, slot + 1);
      prefetch(ks, slot + 1);
    }
    // D[channel][token] = sum_j V[channel][j] q[token][j] for this group
    f32x16 g[2] = {f32x16{}, f32x16{}};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const bf16x8 b0 = as_bf16x8(*reinterpret_cast<const u32x4*>(&cod[tl][64 * tp + col][16 * k + 8 * h]));
      const bf16x8 b1 = as_bf16x8(*reinterpret_cast<const u32x4*>(&cod[tl][64 * tp + 32 + col][16 * k + 8 * h]));
#pragma unroll
      for (int p = 0; p < 3; ++p) {
        const bf16x8 av = as_bf16x8(*reinterpret_cast<const u32x4*>(&vsl[p][32 * cb + col][16 * k + 8 * h]));
        g[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, b0, g[0], 0, 0, 0);
        g[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, b1, g[1], 0, 0, 0);
      }
    }
    // lane (h, col): rows 4h + (i & 3) + 8 (i >> 2) = channels, column col = token
#pragma unroll
    for (int tb = 0; tb < 2; ++tb) {
      const int u = 64 * tp + 32 * tb + col;
      const float st = sl[tl][u], zt = zl[tl][u];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const f32x4 vs4 = *reinterpret_cast<const f32x4*>(&vsum[32 * cb + 4 * h + 8 * q]);
#pragma unroll
        for (int j = 0; j < 4; ++j) out[tb][4 * q + j] += st * g[tb][4 * q + j] + zt * vs4[j];
      }
    }
    __syncthreads();
  }
  if (n_kept == 0) __syncthreads();  // bias visible
#pragma unroll
  for (int tb = 0; tb < 2; ++tb) {
    const int64_t i = tok0 + (int64_t)tl * LD_TOK + 64 * tp + 32 * tb + col;
    if (i < a.n) {
      float* o = a.out + ((int64_t)s * a.n + i) * d + ch0 + 32 * cb + 4 * h;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int r0 = 32 * cb + 4 * h + 8 * q;
        *reinterpret_cast<f32x4*>(o + 8 * q) =
            f32x4{out[tb][4 * q] + bias[r0], out[tb][4 * q + 1] + bias[r0 + 1], out[tb][4 * q + 2] + bias[r0 + 2],
                  out[tb][4 * q + 3] + bias[r0 + 3]};
      }
    }
  }
}

}  // namespace spectra_dev

namespace spectra {
using namespace spectra_dev;

// Token split of the second moment: enough workgroups to fill the chip, chunks of
// at least 256 tokens.
void layer_gram_layout(int32_t d, int64_t n_streams, int64_t n_tokens, int32_t* k_split, int64_t* chunk_tokens) {
  const int64_t tiles = (int64_t)(d / 64) * (d / 64) * n_streams;
  int64_t ks = (2048 + tiles - 1) / tiles;
  const int64_t max_ks = (n_tokens + 255) / 256;
  ks = ks < 1 ? 1 : (ks > max_ks ? max_ks : ks);
  int64_t ct = (n_tokens + ks - 1) / ks;
  ct = (ct + 15) / 16 * 16;
  *chunk_tokens = ct;
  *k_split = (int32_t)((n_tokens + ct - 1) / ct);
}

hipError_t launch_layer_moments(const LayerGramArgs& g, bool f32_in, hipStream_t st) {
  const dim3 grid(g.d / 64, g.d / 64, g.n_streams * g.k_split);
  if (f32_in)
    hipLaunchKernelGGL(layer_gram_kernel<true>, grid, dim3(256), 0, st, g);
  else
    hipLaunchKernelGGL(layer_gram_kernel<false>, grid, dim3(256), 0, st, g);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t per = (int64_t)g.d * g.d + g.d;
  const dim3 grid2((unsigned)((per + 255) / 256), g.n_streams);
  if (f32_in)
    hipLaunchKernelGGL(layer_moments_kernel<true>, grid2, dim3(256), 0, st, g);
  else
    hipLaunchKernelGGL(layer_moments_kernel<false>, grid2, dim3(256), 0, st, g);
  return hipGetLastError();
}

hipError_t launch_layer_encode(const LayerEncodeArgs& a, hipStream_t st) {
  const dim3 grid(xcd_major_grid((int)((a.n + LE_TOK - 1) / LE_TOK), a.d / LG), 1, a.n_streams);
  hipLaunchKernelGGL(layer_encode_kernel, grid, dim3(512), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_layer_decode(const LayerDecodeArgs& a, hipStream_t st) {
  const dim3 grid(xcd_major_grid((int)((a.n + LD_TOK * LD_NT - 1) / (LD_TOK * LD_NT)), a.d / LD_CH), 1, a.n_streams);
  hipLaunchKernelGGL(layer_decode_kernel, grid, dim3(512), 0, st, a);
  return hipGetLastError();
}

}  // namespace spectra
