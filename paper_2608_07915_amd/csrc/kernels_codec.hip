// Encode, decode, fit-moment and test pack/unpack kernels of libspectra (gfx950).
//
// Encode (Sec. 3.2-3.3): c = x V - m for the kept coefficient groups, per token and
// group min/max -> fp16 zero-point and scale, round-to-nearest-even codes, bit-packed
// records. The projection is the one dense contraction here and runs on MFMA
// (v_mfma_f32_32x32x16_bf16): bf16 inputs are exact in bf16 and the fp32 basis is
// split into three bf16 parts whose products are exact in fp32, so the result is
// fp32-accurate. Token tiles are staged in LDS and shared by the waves of a
// workgroup; each wave keeps the basis columns of one kept group in registers.
//
// Decode (Sec. 3.3, Mode A): x_hat = sum_G (z_G 1 + s_G q_G) V_G^T + m V^T, with the
// q_G V_G^T contraction on MFMA (codes are exact small integers in bf16).
#include "device_common.hpp"
#include "encode_dev.hpp"
#include "kernels.hpp"

namespace spectra_dev {

// ---------------------------------------------------------------------------
// Encode
// ---------------------------------------------------------------------------
template <bool F32IN>
__global__ __launch_bounds__(256, 2) void encode_kernel(EncodeArgs a) {
  constexpr int ST = F32IN ? 64 : 128;             // tokens per super-tile
  constexpr int ROWB = F32IN ? (512 + 16) : (256 + 16);  // padded LDS row (bank spread)
  __shared__ __attribute__((aligned(16))) uint8_t xs[ST * ROWB];

  const int s = blockIdx.y;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int h = lane >> 5, col = lane & 31;

  const int64_t first_tile = a.t0 >> 6;
  const int64_t end = a.t0 + a.n;                       // exclusive slot
  const int64_t n_tiles = ((end - 1) >> 6) - first_tile + 1;
  const int64_t n_st = (n_tiles * TILE + ST - 1) / ST;
  const char* xb = reinterpret_cast<const char*>(a.x);
  constexpr int ESZ = F32IN ? 4 : 2;
  constexpr int CPR = (D * ESZ) / 16;  // 16-byte chunks per token row
  // Super-tile st covers slots [slot0, slot0 + ST); rows [lo, hi) hold the call's
  // tokens and only the 32-row MFMA blocks [b_lo, b_hi) that meet them are
  // staged and projected.
  struct Span {
    int64_t slot0;
    int lo, hi, b_lo, b_hi;
  };
  auto span = [&](int64_t st) {
    Span sp;
    sp.slot0 = (first_tile << 6) + st * ST;
    sp.lo = (int)(a.t0 > sp.slot0 ? a.t0 - sp.slot0 : 0);
    sp.hi = (int)(end - sp.slot0 < ST ? end - sp.slot0 : ST);
    sp.b_lo = sp.lo >> 5;
    sp.b_hi = (sp.hi + 31) >> 5;
    return sp;
  };
  // The rows of those blocks are staged in LDS in 16-byte chunks (coalesced); rows
  // outside the call's token range are zero. A super-tile is PRE chunks per thread;
  // the next super-tile's chunks are loaded into registers while this one is
  // projected and quantized, then written to LDS.
  constexpr int PRE = (ST * CPR) / 256;
  static_assert(PRE * 256 == ST * CPR, "staging split");
  auto load_stage = [&](const Span& sp, u32x4 (&r)[PRE]) {
#pragma unroll
    for (int i = 0; i < PRE; ++i) {
      const int c = tid + 256 * i;
      const int row = c / CPR, part = c % CPR;
      const int64_t t = sp.slot0 + row - a.t0;
      r[i] = u32x4{0u, 0u, 0u, 0u};
      if (row >= 32 * sp.b_lo && row < 32 * sp.b_hi && t >= 0 && t < a.n)
        r[i] = *reinterpret_cast<const u32x4*>(xb + ((int64_t)s * a.stream_stride + t * a.token_stride) * ESZ + part * 16);
    }
  };
  auto store_stage = [&](const Span& sp, const u32x4 (&r)[PRE]) {
#pragma unroll
    for (int i = 0; i < PRE; ++i) {
      const int c = tid + 256 * i;
      const int row = c / CPR, part = c % CPR;
      if (row >= 32 * sp.b_lo && row < 32 * sp.b_hi) *reinterpret_cast<u32x4*>(xs + row * ROWB + part * 16) = r[i];
    }
  };
  int64_t st = blockIdx.x;
  if (st >= n_st) return;
  // The first rows are requested before the width table is needed, so their latency
  // overlaps the basis loads (which depend on it).
  u32x4 pre[PRE];
  load_stage(span(st), pre);

  const Kept K = read_kept(a.bits + (int64_t)s * NG);
  const int W = a.W;
  if (!K.ok || K.used > W) return;  // width table inconsistent with the record: write nothing
  const int64_t sbase = (int64_t)s * a.t_cap * W;

  // Wave roles: wpg waves per kept group, each taking every wpg-th 32-token block.
  const int wpg = K.n ? 4 / K.n : 0;
  const bool active = K.n > 0 && wave < K.n * wpg;
  const int slot = active ? wave / wpg : 0;
  const int phase = active ? wave % wpg : 0;
  const int grp = pick4(K.grp, slot);
  const int gbits = pick4(K.bits, slot);
  const int gpay = pick4(K.pay, slot);

  bf16x8 Va[3][8];
  float mv[16];
  if (active) load_group_operands(a.basis + (int64_t)s * D * D, a.mean + (int64_t)s * D, grp, col, h, Va, mv);

  for (;;) {
    const Span sp = span(st);
    const int64_t slot0 = sp.slot0;
    const int b_lo = sp.b_lo, b_hi = sp.b_hi, lo = sp.lo, hi = sp.hi;
    store_stage(sp, pre);
    __syncthreads();  // staged rows visible
    const int64_t st_next = st + gridDim.x;
    if (st_next < n_st) load_stage(span(st_next), pre);

    if (active) {
      for (int beta = b_lo + phase; beta < b_hi; beta += wpg)
        encode_block<F32IN, ROWB>(xs, beta, col, h, Va, mv, slot0, a.t0, end, sbase, W, slot, gbits, gpay, a.packed);
    }
    // Padding words of the record are zero.
    const int npad = W - K.used, nrow = hi - lo;
    for (int c = tid; c < nrow * npad; c += 256) {
      const int row = lo + c % nrow, w = K.used + c / nrow;
      a.packed[rec_word(sbase, slot0 + row, W, w)] = 0u;
    }
    st = st_next;
    if (st >= n_st) break;
    __syncthreads();  // every wave is done with the staged rows
  }
}

// ---------------------------------------------------------------------------
// Decode: wave w owns output channels 32w..32w+31 for every token of a super-tile.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void decode_kernel(DecodeArgs a) {
  constexpr int ST = 128;
  __shared__ uint32_t rec[2 * 64 * 64];  // two record tiles, W <= 64 words
  const int s = blockIdx.y;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int h = lane >> 5, col = lane & 31;
  const Kept K = read_kept(a.bits + (int64_t)s * NG);
  const int W = a.W;
  if (!K.ok || K.used > W) return;  // width table inconsistent with the record: write nothing
  const int64_t sbase = (int64_t)s * a.t_cap * W;
  const int ch = 32 * wave + col;  // this lane's output channel
  const float* Vs = a.basis + (int64_t)s * D * D;

  // B operands: column = channel ch, K = in-group coefficients 16k + 8h + i.
  bf16x8 Vb[NG][2][3];
  float vsum[NG];
#pragma unroll
  for (int sl = 0; sl < NG; ++sl) {
    vsum[sl] = 0.0f;
    if (sl < K.n) {
      const float* vr = Vs + (int64_t)ch * D + G * K.grp[sl];
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        uint32_t p0[8], p1[8], p2[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) split3(vr[16 * k + 8 * h + i], p0[i], p1[i], p2[i]);
        Vb[sl][k][0] = as_bf16x8(u32x4{pack2(p0[0], p0[1]), pack2(p0[2], p0[3]), pack2(p0[4], p0[5]), pack2(p0[6], p0[7])});
        Vb[sl][k][1] = as_bf16x8(u32x4{pack2(p1[0], p1[1]), pack2(p1[2], p1[3]), pack2(p1[4], p1[5]), pack2(p1[6], p1[7])});
        Vb[sl][k][2] = as_bf16x8(u32x4{pack2(p2[0], p2[1]), pack2(p2[2], p2[3]), pack2(p2[4], p2[5]), pack2(p2[6], p2[7])});
      }
      float acc = 0.0f;
      for (int j = 0; j < G; ++j) acc += vr[j];
      vsum[sl] = acc;
    } else {
#pragma unroll
      for (int k = 0; k < 2; ++k)
#pragma unroll
        for (int p = 0; p < 3; ++p) Vb[sl][k][p] = bf16x8{};
    }
  }
  float bias = 0.0f;
  {
    const float* ms = a.mean + (int64_t)s * D;
    const float* vr = Vs + (int64_t)ch * D;
    for (int j = 0; j < D; ++j) bias += ms[j] * vr[j];
  }

  const int64_t first_tile = a.t0 >> 6;
  const int64_t end = a.t0 + a.n;
  const int64_t last_tile = (end - 1) >> 6;
  const int64_t n_st = (last_tile - first_tile + 2) / 2;
  for (int64_t st = blockIdx.x; st < n_st; st += gridDim.x) {
    const int64_t tile0 = first_tile + 2 * st;
    const int ntile = (tile0 + 1 <= last_tile) ? 2 : 1;
    __syncthreads();
    for (int i = tid; i < ntile * 64 * W; i += 256) rec[i] = a.packed[sbase + tile0 * (int64_t)(64 * W) + i];
    __syncthreads();
    for (int beta = 0; beta < 2 * ntile; ++beta) {
      const int row = 32 * beta + col;  // token of this lane's A-operand row
      const uint32_t* rtok = rec + (row >> 6) * 64 * W + (row & 63);
      float out[16];
#pragma unroll
      for (int j = 0; j < 16; ++j) out[j] = bias;
#pragma unroll
      for (int sl = 0; sl < NG; ++sl) {
        if (sl < K.n) {
          f32x16 acc = {};
          with_bits(K.bits[sl], [&](auto bc) {
            constexpr int B = decltype(bc)::value;
            const int pay = K.pay[sl];
            auto word = [&](int i) { return rtok[(pay + i) * 64]; };
#pragma unroll
            for (int k = 0; k < 2; ++k) {
              uint32_t cd[8];
              extract8<B>(word, 16 * k + 8 * h, cd);
              const bf16x8 A = as_bf16x8(u32x4{int_to_bf16_pair(cd[0], cd[1]), int_to_bf16_pair(cd[2], cd[3]),
                                               int_to_bf16_pair(cd[4], cd[5]), int_to_bf16_pair(cd[6], cd[7])});
              acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A, Vb[sl][k][0], acc, 0, 0, 0);
              acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A, Vb[sl][k][1], acc, 0, 0, 0);
              acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A, Vb[sl][k][2], acc, 0, 0, 0);
            }
          });
          // acc[j]: token row 8(j/4) + 4h + j%4 of this block, channel ch
#pragma unroll
          for (int j = 0; j < 16; ++j) {
            const int tr = 32 * beta + 8 * (j >> 2) + 4 * h + (j & 3);
            const uint32_t m = rec[(tr >> 6) * 64 * W + sl * 64 + (tr & 63)];
            out[j] += h2f(m) * acc[j] + h2f(m >> 16) * vsum[sl];
          }
        }
      }
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int tr = 32 * beta + 8 * (j >> 2) + 4 * h + (j & 3);
        const int64_t t = (tile0 << 6) + tr;
        if (t >= a.t0 && t < end) a.out[((int64_t)s * a.n + (t - a.t0)) * D + ch] = out[j];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Test hooks: pack given codes / unpack records with the device code above.
// One wave per (64-token tile, stream); lane (h, col) handles token 32*beta + col.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(64) void pack_codes_kernel(PackArgs a) {
  const int s = blockIdx.y;
  const int lane = threadIdx.x, h = lane >> 5, col = lane & 31;
  const Kept K = read_kept(a.bits + (int64_t)s * NG);
  const int W = a.W;
  if (!K.ok || K.used > W) return;  // width table inconsistent with the record: write nothing
  const int64_t sbase = (int64_t)s * a.t_cap * W;
  for (int beta = 0; beta < 2; ++beta) {
    const int64_t t = (int64_t)blockIdx.x * TILE + 32 * beta + col;
    const bool valid = t < a.n;
    const int64_t base = rec_word(sbase, t, W, 0);
#pragma unroll
    for (int sl = 0; sl < NG; ++sl) {
      if (sl >= K.n) continue;
      const int g = K.grp[sl];
      uint32_t q[16];
#pragma unroll
      for (int j = 0; j < 16; ++j)
        q[j] = valid ? a.codes[((int64_t)s * a.n + t) * D + G * g + 16 * h + j] : 0u;
      with_bits(K.bits[sl], [&](auto bc) {
        constexpr int B = decltype(bc)::value;
        uint32_t P[4];
        pack16<B>(q, P);
        if (h == 0 && valid) a.packed[base + (int64_t)sl * TILE] = a.meta[((int64_t)s * a.n + t) * NG + g];
        store_payload<B>(a.packed, base, K.pay[sl], P, h, valid);
      });
    }
    for (int w = K.used + h; w < W; w += 2)
      if (valid) a.packed[rec_word(sbase, t, W, w)] = 0u;
  }
}

__global__ __launch_bounds__(64) void unpack_codes_kernel(PackArgs a) {
  const int s = blockIdx.y;
  const int lane = threadIdx.x, h = lane >> 5, col = lane & 31;
  const Kept K = read_kept(a.bits + (int64_t)s * NG);
  const int W = a.W;
  if (!K.ok || K.used > W) return;  // width table inconsistent with the record: write nothing
  const int64_t sbase = (int64_t)s * a.t_cap * W;
  for (int beta = 0; beta < 2; ++beta) {
    const int64_t t = (int64_t)blockIdx.x * TILE + 32 * beta + col;
    if (t >= a.n) continue;
    const uint32_t* rtok = a.packed_in + rec_word(sbase, t, W, 0);
    uint8_t* cd = a.codes_out + ((int64_t)s * a.n + t) * D;
    for (int j = 0; j < 64; ++j) cd[64 * h + j] = 0;
    if (h == 0)
      for (int g = 0; g < NG; ++g) a.meta_out[((int64_t)s * a.n + t) * NG + g] = 0u;
#pragma unroll
    for (int sl = 0; sl < NG; ++sl) {
      if (sl >= K.n) continue;
      const int g = K.grp[sl];
      if (h == 0) a.meta_out[((int64_t)s * a.n + t) * NG + g] = rtok[(int64_t)sl * TILE];
      with_bits(K.bits[sl], [&](auto bc) {
        constexpr int B = decltype(bc)::value;
        const int pay = K.pay[sl];
        auto word = [&](int i) { return rtok[(int64_t)(pay + i) * TILE]; };
        for (int k = 0; k < 2; ++k) {
          uint32_t c8[8];
          extract8<B>(word, 16 * k + 8 * h, c8);
          for (int i = 0; i < 8; ++i) cd[G * g + 16 * k + 8 * h + i] = (uint8_t)c8[i];
        }
      });
    }
  }
}

// ---------------------------------------------------------------------------
// Fit moments: per (stream, token chunk) fp64 partial sums of x^T x and x.
// Thread tau owns the 8x8 block (8*(tau/16), 8*(tau%16)) of the 128x128 Gram.
// ---------------------------------------------------------------------------
template <bool F32IN>
__global__ __launch_bounds__(256) void gram_kernel(GramArgs a) {
  __shared__ __attribute__((aligned(16))) float xs[64 * D];
  const int s = blockIdx.y, chunk = blockIdx.x;
  const int tid = threadIdx.x;
  const int I = tid >> 4, J = tid & 15;
  const int64_t t_begin = (int64_t)chunk * a.chunk_tokens;
  const int64_t t_end = t_begin + a.chunk_tokens < a.n ? t_begin + a.chunk_tokens : a.n;
  double acc[8][8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = 0.0;
  double cs = 0.0;
  for (int64_t t0 = t_begin; t0 < t_end; t0 += 64) {
    __syncthreads();
    for (int e = tid; e < 64 * D; e += 256) {
      const int r = e >> 7, c = e & 127;
      const int64_t t = t0 + r;
      float v = 0.0f;
      if (t < t_end) {
        const int64_t idx = (int64_t)s * a.stream_stride + t * a.token_stride + c;
        if constexpr (F32IN)
          v = reinterpret_cast<const float*>(a.x)[idx];
        else
          v = bf2f(reinterpret_cast<const uint16_t*>(a.x)[idx]);
      }
      xs[e] = v;
    }
    __syncthreads();
    const int nt = (int)((t_end - t0) < 64 ? (t_end - t0) : 64);
    for (int r = 0; r < nt; ++r) {
      const float* xr = xs + r * D;
      double xi[8], xj[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        xi[i] = (double)xr[8 * I + i];
        xj[i] = (double)xr[8 * J + i];
      }
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[i][j] = __builtin_fma(xi[i], xj[j], acc[i][j]);
      if (tid < D) cs += (double)xr[tid];
    }
  }
  double* out = a.partial + ((int64_t)s * a.n_chunks + chunk) * (D * D + D);
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) out[(8 * I + i) * D + 8 * J + j] = acc[i][j];
  if (tid < D) out[D * D + tid] = cs;
}

__global__ __launch_bounds__(256) void gram_reduce_kernel(GramArgs a) {
  const int s = blockIdx.y;
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e >= D * D + D) return;
  const double* p = a.partial + (int64_t)s * a.n_chunks * (D * D + D) + e;
  double acc = 0.0;
  for (int c = 0; c < a.n_chunks; ++c) acc += p[(int64_t)c * (D * D + D)];
  a.moments[(int64_t)s * (D * D + D) + e] = acc;
}

}  // namespace spectra_dev

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------
namespace spectra {
using namespace spectra_dev;

hipError_t launch_encode(const EncodeArgs& a, bool f32_input, hipStream_t st) {
  const int ST = f32_input ? 64 : 128;
  const int64_t first_tile = a.t0 >> 6, last_tile = (a.t0 + a.n - 1) >> 6;
  const int64_t n_st = ((last_tile - first_tile + 1) * 64 + ST - 1) / ST;
  // Enough workgroups to fill the GPU several times over, not more than super-tiles.
  int64_t per_stream = (2048 + a.n_streams - 1) / a.n_streams;
  if (per_stream > n_st) per_stream = n_st;
  if (per_stream < 1) per_stream = 1;
  dim3 grid((unsigned)per_stream, (unsigned)a.n_streams);
  if (f32_input)
    hipLaunchKernelGGL(encode_kernel<true>, grid, dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL(encode_kernel<false>, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_decode(const DecodeArgs& a, hipStream_t st) {
  const int64_t first_tile = a.t0 >> 6, last_tile = (a.t0 + a.n - 1) >> 6;
  const int64_t n_st = (last_tile - first_tile + 2) / 2;
  // one round of workgroups (two per CU): the basis operands are set up once per
  // workgroup, and each workgroup streams many super-tiles
  int64_t per_stream = (512 + a.n_streams - 1) / a.n_streams;
  if (per_stream > n_st) per_stream = n_st;
  if (per_stream < 1) per_stream = 1;
  hipLaunchKernelGGL(decode_kernel, dim3((unsigned)per_stream, (unsigned)a.n_streams), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_pack_codes(const PackArgs& a, bool unpack, hipStream_t st) {
  dim3 grid((unsigned)((a.n + 63) / 64), (unsigned)a.n_streams);
  if (unpack)
    hipLaunchKernelGGL(unpack_codes_kernel, grid, dim3(64), 0, st, a);
  else
    hipLaunchKernelGGL(pack_codes_kernel, grid, dim3(64), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_gram(const GramArgs& a, bool f32_input, hipStream_t st) {
  dim3 grid((unsigned)a.n_chunks, (unsigned)a.n_streams);
  if (f32_input)
    hipLaunchKernelGGL(gram_kernel<true>, grid, dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL(gram_kernel<false>, grid, dim3(256), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  dim3 g2((unsigned)((D * D + D + 255) / 256), (unsigned)a.n_streams);
  hipLaunchKernelGGL(gram_reduce_kernel, g2, dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace spectra
