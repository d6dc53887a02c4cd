// Device helpers shared by the libspectra kernels (gfx950 / CDNA4, wave64).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace spectra_dev {

constexpr int D = 128;      // head_dim on the GPU path
constexpr int G = 32;       // group size on the GPU path
constexpr int NG = D / G;   // groups per head
constexpr int TILE = 64;    // tokens per record tile

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(_Float16)))) _Float16 f16x4;
typedef __attribute__((__vector_size__(2 * sizeof(_Float16)))) _Float16 f16x2;
typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(2 * sizeof(float)))) float f32x2;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// ---------------------------------------------------------------------------
// Number formats
// ---------------------------------------------------------------------------
__device__ __forceinline__ float h2f(uint32_t bits16) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)(bits16 & 0xFFFFu));
}
// fp32 -> fp16 bits, round to nearest even, saturating at +-65504.
__device__ __forceinline__ uint32_t f2h_sat(float x) {
  x = __builtin_fminf(__builtin_fmaxf(x, -65504.0f), 65504.0f);
  return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)x);
}
// fp32 -> bf16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint32_t f2bf(float x) {
  uint32_t u = __float_as_uint(x);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}
__device__ __forceinline__ float bf2f(uint32_t b) { return __uint_as_float(b << 16); }

// Exact 3-way split of an fp32 value into bf16 parts: v = p0 + p1 + p2 (+ <2^-24 |v|).
__device__ __forceinline__ void split3(float v, uint32_t& p0, uint32_t& p1, uint32_t& p2) {
  p0 = f2bf(v);
  const float r1 = v - bf2f(p0);
  p1 = f2bf(r1);
  const float r2 = r1 - bf2f(p1);
  p2 = f2bf(r2);
}

// Pack two bf16 bit patterns (low half = first) into one 32-bit register.
__device__ __forceinline__ uint32_t pack2(uint32_t lo16, uint32_t hi16) { return (lo16 & 0xFFFFu) | (hi16 << 16); }

// Small integer (< 256) -> bf16 bits, exact: the upper half of its fp32 value.
__device__ __forceinline__ uint32_t int_to_bf16_pair(uint32_t c0, uint32_t c1) {
  const uint32_t f0 = __float_as_uint((float)c0), f1 = __float_as_uint((float)c1);
  return __builtin_amdgcn_perm(f1, f0, 0x07060302u);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }
__device__ __forceinline__ f16x4 as_f16x4(u32x2 v) { return __builtin_bit_cast(f16x4, v); }

// ---------------------------------------------------------------------------
// Record geometry: word w of token t of stream s (tiles of 64 tokens, word-major).
// ---------------------------------------------------------------------------
__device__ __forceinline__ int64_t rec_word(int64_t stream_base, int64_t t, int W, int w) {
  return stream_base + (t >> 6) * (int64_t)(TILE * W) + (int64_t)w * TILE + (t & 63);
}

// Kept-group bookkeeping read from the per-stream width table (4 groups).
struct Kept {
  int n;           // number of kept groups
  int grp[NG];     // group index of kept slot k
  int bits[NG];    // width of kept slot k
  int pay[NG];     // first payload word of kept slot k (metadata words come first)
  int used;        // words used by the record
  bool ok;         // widths all in [0, 8]
};
__device__ __forceinline__ Kept read_kept(const uint8_t* bits_s) {
  Kept k;
  const uint32_t w = *reinterpret_cast<const uint32_t*>(bits_s);
  k.ok = true;
#pragma unroll
  for (int i = 0; i < NG; ++i) {
    k.grp[i] = 0;
    k.bits[i] = 0;
  }
  int cnt = 0;
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    const int b = (int)((w >> (8 * g)) & 0xFFu);
    if (b > 8) k.ok = false;
    // slot cnt takes group g when b > 0 (compile-time indices only)
#pragma unroll
    for (int i = 0; i < NG; ++i) {
      const bool here = (b > 0) && (i == cnt);
      k.grp[i] = here ? g : k.grp[i];
      k.bits[i] = here ? b : k.bits[i];
    }
    cnt += b > 0 ? 1 : 0;
  }
  k.n = cnt;
  int off = cnt;
#pragma unroll
  for (int i = 0; i < NG; ++i) {
    k.pay[i] = off;
    off += i < cnt ? k.bits[i] : 0;
  }
  k.used = off;
  return k;
}

// ---------------------------------------------------------------------------
// Packing of 16 codes held by one lane (lane half h of a 32x32 MFMA tile holds
// in-group coefficients 16h..16h+15 of one token). The group payload of b words
// takes the lower half's 16b bits first, then the upper half's. Code j is the
// low B bits of q[j] (higher bits are ignored).
// ---------------------------------------------------------------------------
template <int B>
__device__ __forceinline__ void pack16(const uint32_t (&q)[16], uint32_t (&P)[4]) {
  constexpr uint32_t M = (1u << B) - 1u;
#pragma unroll
  for (int i = 0; i < 4; ++i) P[i] = 0;
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    const int pos = j * B;
    const uint32_t c = q[j] & M;
    P[pos >> 5] |= c << (pos & 31);
    if ((pos & 31) + B > 32) P[(pos >> 5) + 1] |= c >> (32 - (pos & 31));
  }
}

// Store the group payload of one token. Both lane halves must call this (it
// contains a cross-half exchange). `base` is the record-word address of word 0
// of this token; `pay` the group's first payload word; `valid` masks stores.
template <int B>
__device__ __forceinline__ void store_payload(uint32_t* __restrict__ packed, int64_t base, int pay,
                                              const uint32_t (&P)[4], int h, bool valid) {
  if constexpr ((B & 1) == 0) {
#pragma unroll
    for (int i = 0; i < B / 2; ++i)
      if (valid) packed[base + (int64_t)(pay + h * (B / 2) + i) * TILE] = P[i];
  } else {
    constexpr int N1 = (B + 1) / 2;
    uint32_t S[N1];
    S[0] = P[0] << 16;
#pragma unroll
    for (int i = 1; i < N1; ++i) S[i] = (P[i] << 16) | (P[i - 1] >> 16);
    const uint32_t from_upper = __shfl_xor(h ? S[0] : 0u, 32);
    if (h == 0) {
#pragma unroll
      for (int i = 0; i < N1; ++i) {
        const uint32_t v = (i == N1 - 1) ? (P[i] | from_upper) : P[i];
        if (valid) packed[base + (int64_t)(pay + i) * TILE] = v;
      }
    } else {
#pragma unroll
      for (int i = 1; i < N1; ++i)
        if (valid) packed[base + (int64_t)(pay + (B - 1) / 2 + i) * TILE] = S[i];
    }
  }
}

// ---------------------------------------------------------------------------
// Unpacking of 8 consecutive in-group codes (j0 .. j0+7) of one token from its
// group payload. `word(i)` returns payload word i of the token (i < B).
// ---------------------------------------------------------------------------
template <int B, typename WordFn>
__device__ __forceinline__ void extract8(WordFn word, int j0, uint32_t (&c)[8]) {
  const int P = j0 * B;                 // first bit
  const int w0 = P >> 5, sh = P & 31;
  const int wl = (P + 8 * B - 1) >> 5;  // last payload word touched
  const uint32_t a0 = word(w0);
  const uint32_t a1 = (w0 + 1 <= wl) ? word(w0 + 1) : 0u;
  const uint32_t a2 = (w0 + 2 <= wl) ? word(w0 + 2) : 0u;
  const uint32_t lo = __builtin_amdgcn_alignbit(a1, a0, sh);
  const uint32_t hi = __builtin_amdgcn_alignbit(a2, a1, sh);
  constexpr uint32_t M = (1u << B) - 1u;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int o = i * B;
    if (o + B <= 32)
      c[i] = (lo >> o) & M;
    else if (o >= 32)
      c[i] = (hi >> (o - 32)) & M;
    else
      c[i] = __builtin_amdgcn_alignbit(hi, lo, o) & M;
  }
}

// a[i] for a wave-uniform runtime i without indexing a private array.
__device__ __forceinline__ int pick4(const int (&a)[NG], int i) {
  return i == 0 ? a[0] : i == 1 ? a[1] : i == 2 ? a[2] : a[3];
}

// Dispatch a runtime width 1..8 to a template (wave-uniform b).
template <typename F>
__device__ __forceinline__ void with_bits(int b, F&& f) {
  switch (b) {
    case 1: f(std::integral_constant<int, 1>{}); break;
    case 2: f(std::integral_constant<int, 2>{}); break;
    case 3: f(std::integral_constant<int, 3>{}); break;
    case 4: f(std::integral_constant<int, 4>{}); break;
    case 5: f(std::integral_constant<int, 5>{}); break;
    case 6: f(std::integral_constant<int, 6>{}); break;
    case 7: f(std::integral_constant<int, 7>{}); break;
    case 8: f(std::integral_constant<int, 8>{}); break;
    default: break;
  }
}

}  // namespace spectra_dev
