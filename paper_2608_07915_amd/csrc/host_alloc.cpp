// Group bit allocation: exact integer optimum of the rate-distortion objective.
//
// App. D minimises sum_j v_j 2^{-2 b_j} at a fixed rate (reverse water-filling,
// Eq. waterfill); Sec. 3.2 lets g adjacent energy-ordered coefficients share one
// width chosen from the group's mean variance, drops zero-bit groups and charges
// one fp16 scale + zero-point per kept group per token; App. F counts that
// metadata in the effective rate. The paper rounds the continuous solution with
// an unspecified fix-up; here the same objective is minimised exactly over
// integer widths by dynamic programming over groups and remaining budget.
#include <cmath>
#include <cstring>
#include <vector>

#include "host_common.hpp"

namespace spectra {

namespace {
// w_G * 4^(8 - b): proportional to D_G 2^{-2b}; b = 0 leaves the whole energy.
inline uint64_t distortion(uint64_t w, int b) { return w << (2 * (8 - b)); }
}  // namespace

spectra_status allocate_bits(const double* var, const spectra_params& p, uint8_t* bits) {
  const int d = p.head_dim, g = p.group_size, nG = d / g;
  const int R = budget_bits(p);
  if (R < 0) return fail(SPECTRA_EINVAL, "negative bit budget");
  // Integer group energies: D_G summed in ascending index (fp64), negatives to 0,
  // w_G = floor(2^39 * D_G / max D); all zero when max D is not positive.
  std::vector<double> D(nG, 0.0);
  double dmax = 0.0;
  for (int G = 0; G < nG; ++G) {
    double acc = 0.0;
    for (int j = G * g; j < (G + 1) * g; ++j) acc += var[j];
    if (!std::isfinite(acc)) return fail(SPECTRA_ENUMERIC, "non-finite variance in group %d", G);
    D[G] = acc > 0.0 ? acc : 0.0;
    if (D[G] > dmax) dmax = D[G];
  }
  std::vector<uint64_t> w(nG, 0);
  if (dmax > 0.0)
    for (int G = 0; G < nG; ++G) w[G] = (uint64_t)std::floor((D[G] / dmax) * 549755813888.0);

  // Backward DP: for suffix G.., remaining budget r -> best (J, C) and width of group G.
  const int W1 = R + 1;
  std::vector<uint64_t> J_next(W1, 0), J_cur(W1);
  std::vector<int> C_next(W1, 0), C_cur(W1);
  std::vector<uint8_t> choice((size_t)nG * W1, 0);
  for (int G = nG - 1; G >= 0; --G) {
    for (int r = 0; r <= R; ++r) {
      bool have = false;
      uint64_t bestJ = 0;
      int bestC = 0, bestB = 0;
      for (int b = p.b_max; b >= 0; --b) {
        const int c = b == 0 ? 0 : g * b + p.meta_bits;
        if (c > r) continue;
        const uint64_t J = distortion(w[G], b) + J_next[r - c];
        const int C = c + C_next[r - c];
        if (!have || J < bestJ || (J == bestJ && C < bestC)) {
          have = true;
          bestJ = J;
          bestC = C;
          bestB = b;
        }
      }
      J_cur[r] = bestJ;
      C_cur[r] = bestC;
      choice[(size_t)G * W1 + r] = (uint8_t)bestB;
    }
    J_next.swap(J_cur);
    C_next.swap(C_cur);
  }
  int r = R;
  for (int G = 0; G < nG; ++G) {
    const int b = choice[(size_t)G * W1 + r];
    bits[G] = (uint8_t)b;
    r -= b == 0 ? 0 : g * b + p.meta_bits;
  }
  return SPECTRA_OK;
}

}  // namespace spectra
