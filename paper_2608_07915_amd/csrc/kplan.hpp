// Bit-field plans for the score operand of decode-step attention (plain C++17,
// shared by the device code and host-side checks).
//
// For code width B a group payload is B 32-bit words, codes LSB-first. Each word
// x is cut into fields by ops: a source (x, or x >> 6) and one AND mask, giving
// one field per 16-bit half. A field never crosses a code boundary and lies in
// bits 0..9 of its half, so the half is an integer below 1024 (the device turns
// it into an exact fp16 number). A field at bit f0 of its half that holds code
// bits b0.. equals (code part) * 2^(f0 - b0), so a weight of q_j * 2^(b0 - f0)
// on it reproduces q_j * (code part) exactly. Pieces that fit neither source
// are split in two fields.
#pragma once
#include <cstdint>

namespace spectra_dev {

struct KField {
  int8_t code;  // in-group coefficient index 0..31, -1 = empty half
  int8_t e;     // b0 - f0: log2 of the weight scale
};
struct KOp {
  uint32_t mask;
  uint8_t shifted;  // 0: from x, 1: from x >> 6
  KField f[2];      // low half, high half
};
constexpr int KOPS_MAX = 28;  // B = 7
struct KPlan {
  int n_ops;
  int word_ops[8];  // ops per payload word, in order
  KOp op[KOPS_MAX];
};

constexpr KPlan make_kplan(int B) {
  KPlan P{};
  for (int w = 0; w < B; ++w) {
    // fields per (source, half): code, b0, f0, length
    int cnt[2][2] = {{0, 0}, {0, 0}};
    int fc[2][2][16] = {}, fb[2][2][16] = {}, ff[2][2][16] = {}, fl[2][2][16] = {};
    for (int hh = 0; hh < 2; ++hh) {
      const int P0 = 32 * w + 16 * hh;
      for (int j = 0; j < 32; ++j) {
        const int a = B * j, b = B * j + B;
        const int lo = a > P0 ? a : P0, hi = b < P0 + 16 ? b : P0 + 16;
        if (lo >= hi) continue;
        const int p0 = lo - P0, p1 = hi - P0, b0 = lo - a;
        int src[2] = {0, 0}, f0[2] = {0, 0}, bb[2] = {0, 0}, len[2] = {0, 0};
        int n = 0;
        if (p1 <= 10) {
          src[0] = 0, f0[0] = p0, bb[0] = b0, len[0] = p1 - p0, n = 1;
        } else if (p0 >= 6) {
          src[0] = 1, f0[0] = p0 - 6, bb[0] = b0, len[0] = p1 - p0, n = 1;
        } else {
          src[0] = 0, f0[0] = p0, bb[0] = b0, len[0] = 10 - p0;
          src[1] = 1, f0[1] = 4, bb[1] = b0 + 10 - p0, len[1] = p1 - 10, n = 2;
        }
        for (int t = 0; t < n; ++t) {
          const int k = cnt[src[t]][hh]++;
          fc[src[t]][hh][k] = j;
          fb[src[t]][hh][k] = bb[t];
          ff[src[t]][hh][k] = f0[t];
          fl[src[t]][hh][k] = len[t];
        }
      }
    }
    int nw = 0;
    for (int sc = 0; sc < 2; ++sc) {
      const int n = cnt[sc][0] > cnt[sc][1] ? cnt[sc][0] : cnt[sc][1];
      for (int k = 0; k < n; ++k) {
        KOp op{};
        op.shifted = (uint8_t)sc;
        for (int hh = 0; hh < 2; ++hh) {
          if (k < cnt[sc][hh]) {
            op.mask |= (((1u << fl[sc][hh][k]) - 1u) << ff[sc][hh][k]) << (16 * hh);
            op.f[hh].code = (int8_t)fc[sc][hh][k];
            op.f[hh].e = (int8_t)(fb[sc][hh][k] - ff[sc][hh][k]);
          } else {
            op.f[hh].code = -1;
            op.f[hh].e = 0;
          }
        }
        P.op[P.n_ops++] = op;
        ++nw;
      }
    }
    P.word_ops[w] = nw;
  }
  return P;
}

// The same plans as MFMA operand gathers: score MFMA m of a width-B slot takes the
// fields of ops 2m and 2m + 1 (low half, high half of each) as its four K elements;
// entry [B - 1][m][k] is field (op 2m + k / 2, half k % 2), code -1 where empty.
constexpr int KMFMA_MAX = (KOPS_MAX + 1) / 2;
struct alignas(4) KGather {
  KField f[8][KMFMA_MAX][4];
};
constexpr KGather make_kgather() {
  KGather T{};
  for (int B = 1; B <= 8; ++B) {
    const KPlan P = make_kplan(B);
    for (int m = 0; m < KMFMA_MAX; ++m)
      for (int k = 0; k < 4; ++k) {
        const int i = 2 * m + k / 2;
        KField f{};
        f.code = -1;
        f.e = 0;
        if (i < P.n_ops) f = P.op[i].f[k % 2];
        T.f[B - 1][m][k] = f;
      }
  }
  return T;
}

}  // namespace spectra_dev
