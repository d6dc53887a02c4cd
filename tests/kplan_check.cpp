// Host check of the score-operand bit-field plans (kplan.hpp): for every code
// width, the masked fields cover each payload bit once, lie in bits 0..9 of
// their 16-bit half, and with weights q_j * 2^e give exactly sum_j q_j * c_j.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <random>

#include "kplan.hpp"

using namespace spectra_dev;

int main() {
  std::mt19937_64 rng(7);
  int bad = 0;
  for (int B = 1; B <= 8; ++B) {
    const KPlan P = make_kplan(B);
    if (P.n_ops > KOPS_MAX) { std::printf("B=%d: %d ops > max\n", B, P.n_ops); ++bad; }
    // coverage: every payload bit of every word is in exactly one field
    int opi = 0;
    for (int w = 0; w < B; ++w) {
      int cover[32] = {};
      for (int i = 0; i < P.word_ops[w]; ++i, ++opi) {
        const KOp& op = P.op[opi];
        for (int hh = 0; hh < 2; ++hh) {
          const uint32_t m = (op.mask >> (16 * hh)) & 0xFFFFu;
          if (m & ~0x3FFu) { std::printf("B=%d w=%d op %d: field outside bits 0..9\n", B, w, i); ++bad; }
          if ((m == 0) != (op.f[hh].code < 0)) { std::printf("B=%d: empty-field mismatch\n", B); ++bad; }
          if (op.f[hh].code >= 0 && (op.f[hh].e < -9 || op.f[hh].e > 7)) { std::printf("B=%d: scale out of range\n", B); ++bad; }
          for (int bit = 0; bit < 16; ++bit)
            if (m >> bit & 1u) {
              const int src = bit + (op.shifted ? 6 : 0);   // bit position in the half before the shift
              if (src >= 16) { std::printf("B=%d: field reads the other half\n", B); ++bad; continue; }
              cover[16 * hh + src]++;
            }
        }
      }
      for (int b = 0; b < 32; ++b)
        if (cover[b] != 1) { std::printf("B=%d w=%d bit %d covered %d times\n", B, w, b, cover[b]); ++bad; }
    }
    if (opi != P.n_ops) { std::printf("B=%d: word_ops do not add up\n", B); ++bad; }
    // value identity on random payloads and integer weights (exact in double)
    for (int trial = 0; trial < 2000; ++trial) {
      uint32_t words[8] = {};
      for (int w = 0; w < B; ++w) words[w] = (uint32_t)rng();
      double q[32];
      for (int j = 0; j < 32; ++j) q[j] = (double)((int64_t)(rng() % 2001) - 1000);
      double want = 0.0;
      for (int j = 0; j < 32; ++j) {
        uint32_t c = 0;
        for (int b = 0; b < B; ++b) {
          const int p = B * j + b;
          c |= ((words[p >> 5] >> (p & 31)) & 1u) << b;
        }
        want += q[j] * (double)c;
      }
      double got = 0.0;
      opi = 0;
      for (int w = 0; w < B; ++w) {
        const uint32_t x = words[w], x6 = x >> 6;
        for (int i = 0; i < P.word_ops[w]; ++i, ++opi) {
          const KOp& op = P.op[opi];
          const uint32_t v = (op.shifted ? x6 : x) & op.mask;
          for (int hh = 0; hh < 2; ++hh)
            if (op.f[hh].code >= 0) got += q[op.f[hh].code] * std::ldexp((double)((v >> (16 * hh)) & 0xFFFFu), op.f[hh].e);
        }
      }
      if (got != want) { std::printf("B=%d trial %d: %.17g != %.17g\n", B, trial, got, want); ++bad; break; }
    }
  }
  if (bad == 0) std::printf("OK\n");
  return bad ? 1 : 0;
}
