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
// Super-tile st covers slots [slot0, slot0 + ST); rows [lo, hi) hold the call's
// tokens and only the 32-row MFMA blocks [b_lo, b_hi) that meet them are
// projected.
struct Span {
  int64_t slot0;
  int lo, hi, b_lo, b_hi;
};
__device__ __forceinline__ Span encode_span(const EncodeArgs& a, int64_t st, int ST) {
  const int64_t end = a.t0 + a.n;
  Span sp;
  sp.slot0 = ((a.t0 >> 6) << 6) + st * ST;
  sp.lo = (int)(a.t0 > sp.slot0 ? a.t0 - sp.slot0 : 0);
  sp.hi = (int)(end - sp.slot0 < ST ? end - sp.slot0 : ST);
  sp.b_lo = sp.lo >> 5;
  sp.b_hi = (sp.hi + 31) >> 5;
  return sp;
}

// Wave roles: wpg waves per kept group, each taking every wpg-th 32-token block.
// PIPE: the next block's MFMAs are issued before this block is quantized, so the
// matrix cores and the vector ALU work on two blocks at once.
// Records go to `out` + sbase, tile by tile as in HBM (out = a.packed, or the
// LDS staging of one super-tile with sbase = 0 and slot0 taken as tile 0).
template <bool F32IN, int ROWB, bool PIPE>
__device__ __forceinline__ void encode_span_blocks(const EncodeArgs& a, const uint8_t* xs, const Span& sp, int phase,
                                                   int wpg, int col, int h, const bf16x8 (&Va)[3][8],
                                                   const f32x16& nm, uint32_t* out, int64_t sbase, int slot, int gbits,
                                                   int gpay) {
  if (sp.b_lo + phase >= sp.b_hi) return;
  auto proj = [&](int beta) {
    return project_block<F32IN, ROWB>(xs, beta, col, h, nm, [&](int p, int k) { return Va[p][k]; });
  };
  // record word 0 of the super-tile's first tile; row r of the super-tile is at
  // (r / 64) * 64 W + r % 64 from it
  uint32_t* tile0 = out == a.packed ? a.packed + sbase + (sp.slot0 >> 6) * (int64_t)(TILE * a.W) : out;
  int beta = sp.b_lo + phase;
  f32x16 acc = proj(beta);
  for (;;) {
    const int nb = beta + wpg;
    const bool more = nb < sp.b_hi;
    f32x16 nacc = acc;
    if (PIPE && more) nacc = proj(nb);
    const int r = 32 * beta + col;
    store_block(acc, tile0 + (r >> 6) * (TILE * a.W) + (r & 63), r >= sp.lo && r < sp.hi, h, slot, gbits, gpay);
    if (!more) break;
    acc = PIPE ? nacc : proj(nb);
    beta = nb;
  }
}

// Staged variant: records go to the LDS staging of the super-tile (all rows,
// valid or not: only the call's rows are copied out). The loop is instantiated
// per code width, so a block's quantization is straight-line code that the
// scheduler interleaves with the next block's MFMA chain.
template <int B>
__device__ __forceinline__ void encode_span_blocks_staged(const uint8_t* xs, const Span& sp, int phase, int wpg,
                                                          int col, int h, const bf16x8 (&Va)[3][8], const f32x16& nm,
                                                          uint32_t* rs, uint32_t* dummy, int W, int slot, int gpay) {
  auto proj = [&](int beta) {
    return project_block<false, 0>(xs, beta, col, h, nm, [&](int p, int k) { return Va[p][k]; });
  };
  auto stage = [&](const f32x16& acc, int beta) {
    uint32_t P[4];
    const uint32_t meta = quantize_pack<B>(acc, P);
    const int r = 32 * beta + col;
    stage_record_words<B>(rs + (r >> 6) * (TILE * W) + (r & 63), dummy, h, slot, gpay, meta, P);
  };
  int beta = sp.b_lo + phase;
  f32x16 acc = proj(beta);
  for (int nb = beta + wpg; nb < sp.b_hi; nb += wpg) {
    const f32x16 nacc = proj(nb);
    stage(acc, beta);
    // interleave: each MFMA of the next block with a share of this block's VALU work
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // the K step's LDS operand read
#pragma unroll
      for (int p = 0; p < 3; ++p) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
        __builtin_amdgcn_sched_group_barrier(0x002, 5, 0);  // five VALU
      }
    }
    acc = nacc;
    beta = nb;
  }
  stage(acc, beta);
}

// Padding words of the records of rows [lo, hi) are zero.
__device__ __forceinline__ void encode_padding(const EncodeArgs& a, const Span& sp, int64_t sbase, int used, int tid) {
  const int npad = a.W - used, nrow = sp.hi - sp.lo;
  for (int c = tid; c < nrow * npad; c += 256) {
    const int row = sp.lo + c % nrow, w = used + c / nrow;
    a.packed[rec_word(sbase, sp.slot0 + row, a.W, w)] = 0u;
  }
}

// bf16 tokens: super-tiles of 128 tokens (32 KB) are copied straight from HBM
// into one of two LDS buffers (global_load_lds, 16 bytes per lane) while the
// other buffer is projected; rows are 256 bytes with the 16-byte chunks
// XOR-swizzled by the row index, so the MFMA operand reads of 32 rows spread
// over the LDS banks. Rows outside the call's tokens load a clamped in-range
// row (their blocks are not projected or their records not stored).
//
// STAGED: the super-tile's records (two 64-token tiles, word-major, the layout
// they have in HBM) are assembled in LDS and written with one coalesced
// 16-byte store per 4 tokens of a word; each wave then waits only for its
// loads of the next super-tile (the stores it issued after them are not
// waited for). Otherwise every lane stores its own record words.
constexpr int EST = 128;

__host__ __device__ constexpr size_t encode_bf16_lds_bytes(int W, bool staged) {
  return (size_t)2 * EST * 256 + (staged ? (size_t)(EST * W + 256) * 4 : 0);  // + a scratch word per lane
}

// s_waitcnt with vmcnt(n) (n < 64: low four bits at 3:0, high two at 15:14), expcnt
// and lgkmcnt not waited for
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt field");
  __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | ((N >> 4) << 14));
}

template <bool STAGED>
__global__ __launch_bounds__(256, 2) void encode_bf16_kernel(EncodeArgs a) {
  extern __shared__ __attribute__((aligned(1024))) uint8_t esmem[];
  uint8_t(*xs)[EST * 256] = reinterpret_cast<uint8_t(*)[EST * 256]>(esmem);
  uint32_t* rs = reinterpret_cast<uint32_t*>(esmem + 2 * EST * 256);  // STAGED: [2][W][64] record words, [4][64] scratch
  const int s = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: role selection stays scalar
  const int h = lane >> 5, col = lane & 31;
  const int64_t first_tile = a.t0 >> 6;
  const int64_t n_tiles = ((a.t0 + a.n - 1) >> 6) - first_tile + 1;
  const int64_t n_st = (n_tiles * TILE + EST - 1) / EST;
  const char* xb = reinterpret_cast<const char*>(a.x) + (int64_t)s * a.stream_stride * 2;
  // one global_load_lds fills 1 KB: rows 4m..4m+3 of the super-tile; lane i
  // brings chunk (i % 16) ^ (row % 16) of row 4m + i / 16. Wave w issues m = 8w..8w+7.
  const int lrow = lane >> 4;
  // A super-tile whose 128 rows all hold the call's tokens: uniform row base plus a
  // per-lane offset that does not change between super-tiles (row 32 wave + 4 i + lrow
  // has row % 16 = 4 (i % 4) + lrow), so the copies take no per-copy vector arithmetic.
  const int64_t ts2 = a.token_stride * 2;  // bytes from one token row to the next
  uint32_t voff[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) voff[k] = (uint32_t)(lrow * ts2) + ((uint32_t)((lane & 15) ^ (4 * k + lrow)) << 4);
  auto stage = [&](int64_t st, int b) {
    const int64_t slot0 = (first_tile << 6) + st * EST;
    if (slot0 >= a.t0 && slot0 + EST <= a.t0 + a.n) {
      const char* rb = xb + (slot0 - a.t0 + 32 * wave) * ts2;
#pragma unroll
      for (int i = 0; i < 8; ++i)
        __builtin_amdgcn_global_load_lds(rb + 4 * i * ts2 + voff[i & 3], &xs[b][(8 * wave + i) * 1024], 16, 0, 0);
      return;
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int m = 8 * wave + i, row = 4 * m + lrow;
      const int chunk = (lane & 15) ^ (row & 15);
      int64_t t = slot0 + row - a.t0;
      t = t < 0 ? 0 : (t >= a.n ? a.n - 1 : t);
      __builtin_amdgcn_global_load_lds(xb + t * ts2 + chunk * 16, &xs[b][m * 1024], 16, 0, 0);
    }
  };
  int64_t st = blockIdx.x;
  if (st >= n_st) return;
  stage(st, 0);

  const Kept K = read_kept(a.bits + (int64_t)s * NG);
  const int W = a.W;
  if (!K.ok || K.used > W) return;  // width table inconsistent with the record: write nothing
  const int64_t sbase = (int64_t)s * a.t_cap * W;
  const int wpg = K.n ? 4 / K.n : 0;
  const bool active = K.n > 0 && wave < K.n * wpg;
  const int slot = active ? wave / wpg : 0;
  const int phase = active ? wave % wpg : 0;
  const int grp = pick4(K.grp, slot);
  const int gbits = pick4(K.bits, slot);
  const int gpay = pick4(K.pay, slot);
  bf16x8 Va[3][8];
  f32x16 nm;
  if (active) load_group_operands(a.basis + (int64_t)s * D * D, a.mean + (int64_t)s * D, grp, col, h, Va, nm);
  if constexpr (STAGED) {
    // padding words stay zero: no wave writes words >= K.used
    for (int i = tid; i < EST * W; i += 256) rs[i] = 0u;
  }
  int buf = 0;
  wait_vmcnt<0>();  // this super-tile is in LDS
  __syncthreads();
  for (;;) {
    const int64_t st_next = st + gridDim.x;
    if (st_next < n_st) stage(st_next, buf ^ 1);
    const Span sp = encode_span(a, st, EST);
    if constexpr (STAGED) {
      if (active)
        with_bits(gbits, [&](auto bc) {
          encode_span_blocks_staged<decltype(bc)::value>(xs[buf], sp, phase, wpg, col, h, Va, nm, rs,
                                                         rs + EST * W + 64 * wave, W, slot, gpay);
        });
      __syncthreads();  // the records of the super-tile are in LDS
      uint32_t* dst = a.packed + sbase + (sp.slot0 >> 6) * (int64_t)(TILE * W);
      const bool full = sp.lo == 0 && sp.hi == EST;
      // 16-byte piece c = tid + 256 q of the 2 * 64 * W words; this wave's pieces
      // for q < nst (the first lane of each is in range), so the wave issues
      // exactly nst stores after its loads of the next super-tile
      const int nst = (32 * W - 64 * wave + 255) >> 8;
      if (full) {
        for (int q = 0; q < nst; ++q) {
          const int c = tid + 256 * q;
          if (c < 32 * W) *reinterpret_cast<u32x4*>(dst + 4 * c) = *reinterpret_cast<const u32x4*>(rs + 4 * c);
        }
      } else {
        for (int i = tid; i < EST * W; i += 256) {
          const int row = ((i / (TILE * W)) << 6) + (i & 63);
          if (row >= sp.lo && row < sp.hi) dst[i] = rs[i];
        }
      }
      st = st_next;
      if (st >= n_st) break;
      // wait for this wave's loads of the next super-tile; the nst stores issued
      // after them may still be in flight (vector memory operations complete in
      // issue order; nothing else in the loop touches vector memory)
      if (!full || nst <= 0 || nst > 5)
        wait_vmcnt<0>();
      else if (nst == 1)
        wait_vmcnt<1>();
      else if (nst == 2)
        wait_vmcnt<2>();
      else if (nst == 3)
        wait_vmcnt<3>();
      else if (nst == 4)
        wait_vmcnt<4>();
      else
        wait_vmcnt<5>();
    } else {
      if (active) encode_span_blocks<false, 0, true>(a, xs[buf], sp, phase, wpg, col, h, Va, nm, a.packed, sbase, slot,
                                                     gbits, gpay);
      encode_padding(a, sp, sbase, K.used, tid);
      st = st_next;
      if (st >= n_st) break;
      wait_vmcnt<0>();  // the next super-tile is in LDS
    }
    __syncthreads();  // ... for every wave; every wave is done with this super-tile
    buf ^= 1;
  }
}

// fp32 tokens: super-tiles of 64 tokens staged through registers into padded
// LDS rows; the next super-tile's rows are loaded into registers while this one
// is projected and quantized.
__global__ __launch_bounds__(256, 2) void encode_f32_kernel(EncodeArgs a) {
  constexpr int ST = 64;
  constexpr int ROWB = 512 + 16;  // padded LDS row (bank spread)
  __shared__ __attribute__((aligned(16))) uint8_t xs[ST * ROWB];
  const int s = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: role selection stays scalar
  const int h = lane >> 5, col = lane & 31;
  const int64_t first_tile = a.t0 >> 6;
  const int64_t n_tiles = ((a.t0 + a.n - 1) >> 6) - first_tile + 1;
  const int64_t n_st = (n_tiles * TILE + ST - 1) / ST;
  const char* xb = reinterpret_cast<const char*>(a.x);
  constexpr int CPR = (D * 4) / 16;  // 16-byte chunks per token row
  constexpr int PRE = (ST * CPR) / 256;
  static_assert(PRE * 256 == ST * CPR, "staging split");
  // rows of the projected blocks are staged (rows outside the call's tokens are zero)
  auto load_stage = [&](const Span& sp, u32x4 (&r)[PRE]) {
#pragma unroll
    for (int i = 0; i < PRE; ++i) {
      const int c = tid + 256 * i;
      const int row = c / CPR, part = c % CPR;
      const int64_t t = sp.slot0 + row - a.t0;
      r[i] = u32x4{0u, 0u, 0u, 0u};
      if (row >= 32 * sp.b_lo && row < 32 * sp.b_hi && t >= 0 && t < a.n)
        r[i] = *reinterpret_cast<const u32x4*>(xb + ((int64_t)s * a.stream_stride + t * a.token_stride) * 4 + part * 16);
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
  u32x4 pre[PRE];
  load_stage(encode_span(a, st, ST), pre);
  const Kept K = read_kept(a.bits + (int64_t)s * NG);
  const int W = a.W;
  if (!K.ok || K.used > W) return;  // width table inconsistent with the record: write nothing
  const int64_t sbase = (int64_t)s * a.t_cap * W;
  const int wpg = K.n ? 4 / K.n : 0;
  const bool active = K.n > 0 && wave < K.n * wpg;
  const int slot = active ? wave / wpg : 0;
  const int phase = active ? wave % wpg : 0;
  const int grp = pick4(K.grp, slot);
  const int gbits = pick4(K.bits, slot);
  const int gpay = pick4(K.pay, slot);
  bf16x8 Va[3][8];
  f32x16 nm;
  if (active) load_group_operands(a.basis + (int64_t)s * D * D, a.mean + (int64_t)s * D, grp, col, h, Va, nm);
  for (;;) {
    const Span sp = encode_span(a, st, ST);
    store_stage(sp, pre);
    __syncthreads();  // staged rows visible
    const int64_t st_next = st + gridDim.x;
    if (st_next < n_st) load_stage(encode_span(a, st_next, ST), pre);
    if (active)
      encode_span_blocks<true, ROWB, false>(a, xs, sp, phase, wpg, col, h, Va, nm, a.packed, sbase, slot, gbits, gpay);
    encode_padding(a, sp, sbase, K.used, tid);
    st = st_next;
    if (st >= n_st) break;
    __syncthreads();  // every wave is done with the staged rows
  }
}

// ---------------------------------------------------------------------------
// Decode: wave w owns output channels 32w..32w+31 for every token of a super-tile.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256, 2) void decode_kernel(DecodeArgs a) {
  // super-tile = two 64-token record tiles; records of W <= 32 words are double-buffered
  // (the next super-tile is copied HBM -> LDS by global_load_lds while this one is
  // decoded), wider ones go through one buffer
  __shared__ __attribute__((aligned(16))) uint32_t rec[2 * 64 * 64];
  __shared__ __attribute__((aligned(16))) float vsum_s[NG][D], bias_s[D];
  const int s = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = lane >> 5, col = lane & 31;
  const Kept K = read_kept(a.bits + (int64_t)s * NG);
  const int W = a.W;
  if (!K.ok || K.used > W) return;  // width table inconsistent with the record: write nothing
  const int64_t sbase = (int64_t)s * a.t_cap * W;
  const int ch = 32 * wave + col;  // channel of this lane's basis operand row
  const float* Vs = a.basis + (int64_t)s * D * D;

  const int64_t first_tile = a.t0 >> 6;
  const int64_t end = a.t0 + a.n;
  const int64_t last_tile = (end - 1) >> 6;
  const int64_t n_st = (last_tile - first_tile + 2) / 2;
  const bool db = W <= 32;
  // super-tile st into buffer b: its words are contiguous in HBM (tile-major), 16 bytes
  // per lane and copy; lanes past the super-tile's last word re-read its last piece
  // (their LDS slots are never read)
  auto issue = [&](int64_t st, int b) {
    const int64_t tile0 = first_tile + 2 * st;
    const int ntile = (tile0 + 1 <= last_tile) ? 2 : 1;
    const int np = ntile * 16 * W;  // 16-byte pieces
    const uint32_t* src = a.packed + sbase + tile0 * (int64_t)(64 * W);
    uint32_t* dst = rec + b * (64 * 64);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int p0 = 256 * i + 64 * wave;
      if (p0 < np) {
        const int pc = p0 + lane < np ? p0 + lane : np - 1;
        __builtin_amdgcn_global_load_lds(src + 4 * pc, dst + 4 * p0, 16, 0, 0);
      }
    }
  };
  int64_t st = blockIdx.x;
  if (st >= n_st) return;
  issue(st, 0);

  // A operands: row = channel ch, K = in-group coefficients 16k + 8h + i.
  bf16x8 Vb[NG][2][3];
#pragma unroll
  for (int sl = 0; sl < NG; ++sl) {
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
      if (h == 0) {
        float acc = 0.0f;
        for (int j = 0; j < G; ++j) acc += vr[j];
        vsum_s[sl][ch] = acc;
      }
    } else {
#pragma unroll
      for (int k = 0; k < 2; ++k)
#pragma unroll
        for (int p = 0; p < 3; ++p) Vb[sl][k][p] = bf16x8{};
    }
  }
  if (h == 0) {
    const float* ms = a.mean + (int64_t)s * D;
    const float* vr = Vs + (int64_t)ch * D;
    float bias = 0.0f;
    for (int j = 0; j < D; ++j) bias += ms[j] * vr[j];
    bias_s[ch] = bias;
  }
  wait_vmcnt<0>();  // this wave's copies of the first super-tile (and the operand loads) done
  __syncthreads();  // ... every wave's; vsum and bias visible

  int buf = 0;
  for (;;) {
    const int64_t st_next = st + gridDim.x;
    const bool more = st_next < n_st;
    if (db && more) issue(st_next, buf ^ 1);
    const int64_t tile0 = first_tile + 2 * st;
    const int ntile = (tile0 + 1 <= last_tile) ? 2 : 1;
    const bool full = ntile == 2 && (tile0 << 6) >= a.t0 && (tile0 << 6) + 128 <= end;
    const uint32_t* rb = rec + buf * (64 * 64);
    for (int beta = 0; beta < 2 * ntile; ++beta) {
      const int row = 32 * beta + col;  // token of this lane's B-operand column
      const uint32_t* rtok = rb + (row >> 6) * 64 * W + (row & 63);
      f32x16 out = {};
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
              const bf16x8 C = as_bf16x8(u32x4{int_to_bf16_pair(cd[0], cd[1]), int_to_bf16_pair(cd[2], cd[3]),
                                               int_to_bf16_pair(cd[4], cd[5]), int_to_bf16_pair(cd[6], cd[7])});
              acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(Vb[sl][k][0], C, acc, 0, 0, 0);
              acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(Vb[sl][k][1], C, acc, 0, 0, 0);
              acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(Vb[sl][k][2], C, acc, 0, 0, 0);
            }
          });
          // acc[4q + r]: channel 32 wave + 8q + 4h + r, token row (the lane's column)
          const uint32_t m = rtok[sl * 64];
          const float sc = h2f(m), zc = h2f(m >> 16);
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const f32x4 v4 = *reinterpret_cast<const f32x4*>(&vsum_s[sl][32 * wave + 8 * q + 4 * h]);
#pragma unroll
            for (int r = 0; r < 4; ++r) out[4 * q + r] = __builtin_fmaf(sc, acc[4 * q + r], __builtin_fmaf(zc, v4[r], out[4 * q + r]));
          }
        }
      }
      const int64_t t = (tile0 << 6) + row;
      float* o = a.out + ((int64_t)s * a.n + (t - a.t0)) * D + 32 * wave + 4 * h;
      if (full || (t >= a.t0 && t < end)) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const f32x4 b4 = *reinterpret_cast<const f32x4*>(&bias_s[32 * wave + 8 * q + 4 * h]);
          *reinterpret_cast<f32x4*>(o + 8 * q) =
              f32x4{out[4 * q] + b4[0], out[4 * q + 1] + b4[1], out[4 * q + 2] + b4[2], out[4 * q + 3] + b4[3]};
        }
      }
    }
    if (!more) break;
    if (db) {
      // this wave's copies of the next super-tile were issued before the 16 stores of a
      // full super-tile (vector memory operations complete in issue order)
      if (full)
        wait_vmcnt<16>();
      else
        wait_vmcnt<0>();
      __syncthreads();  // every wave's copies landed; every wave is done with rec[buf]
      buf ^= 1;
    } else {
      __syncthreads();  // every wave is done with the buffer
      issue(st_next, 0);
      wait_vmcnt<0>();
      __syncthreads();
    }
    st = st_next;
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
  if (f32_input) {
    hipLaunchKernelGGL(encode_f32_kernel, grid, dim3(256), 0, st, a);
  } else {
    // staged records (W <= 64 words: at most 96 KB of LDS) when the device has the LDS
    int dev = 0, lds_max = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
    if (e != hipSuccess) return e;
    const size_t lds = encode_bf16_lds_bytes(a.W, true);
    if (a.W <= 64 && lds <= (size_t)lds_max)
      hipLaunchKernelGGL(encode_bf16_kernel<true>, grid, dim3(256), lds, st, a);
    else
      hipLaunchKernelGGL(encode_bf16_kernel<false>, grid, dim3(256), encode_bf16_lds_bytes(a.W, false), st, a);
  }
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
