// Fit of one stream from its first and second moments (Sec. 3.1), plus the
// parameter checks, error reporting and the C entry points that need no GPU.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <string>
#include <vector>

#include "host_common.hpp"

namespace spectra {

namespace {
thread_local std::string g_last_error;
}

void set_last_error(const std::string& msg) { g_last_error = msg; }

spectra_status fail(spectra_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

int32_t budget_bits(const spectra_params& p) {
  if (p.budget_bits > 0) return p.budget_bits;
  return (int32_t)std::floor(16.0 * (double)p.head_dim / p.ratio + 1e-6);
}

spectra_status check_params(const spectra_params& p) {
  if (p.head_dim <= 0 || p.head_dim > 1024) return fail(SPECTRA_EINVAL, "head_dim=%d out of range", p.head_dim);
  if (p.group_size <= 0 || p.head_dim % p.group_size != 0)
    return fail(SPECTRA_EINVAL, "group_size=%d must divide head_dim=%d", p.group_size, p.head_dim);
  if (p.head_dim / p.group_size > 128) return fail(SPECTRA_EINVAL, "more than 128 groups");
  if (p.b_max < 0 || p.b_max > 8) return fail(SPECTRA_EINVAL, "b_max=%d must be in [0, 8]", p.b_max);
  if (p.meta_bits < 0) return fail(SPECTRA_EINVAL, "meta_bits=%d negative", p.meta_bits);
  if (p.centered != 0 && p.centered != 1) return fail(SPECTRA_EINVAL, "centered must be 0 or 1");
  if (p.budget_bits < 0) return fail(SPECTRA_EINVAL, "budget_bits negative");
  if (p.budget_bits == 0 && !(p.ratio > 0.0 && std::isfinite(p.ratio)))
    return fail(SPECTRA_EINVAL, "ratio must be positive and finite when budget_bits is 0");
  if (budget_bits(p) > 65536) return fail(SPECTRA_EINVAL, "bit budget %d too large", budget_bits(p));
  return SPECTRA_OK;
}

bool layer_geometry(const spectra_params& p) {
  return p.head_dim >= 256 && p.head_dim <= 1024 && p.head_dim % 128 == 0 && p.group_size == 64;
}

spectra_status check_params_gpu(const spectra_params& p) {
  spectra_status st = check_params(p);
  if (st != SPECTRA_OK) return st;
  if (p.meta_bits != 32) return fail(SPECTRA_EUNSUPPORTED, "GPU path needs meta_bits=32 (got %d)", p.meta_bits);
  if (layer_geometry(p)) {
    if (record_words(p) > 128) return fail(SPECTRA_EUNSUPPORTED, "record of %d words exceeds 128", record_words(p));
    return SPECTRA_OK;
  }
  if (p.head_dim != 128)
    return fail(SPECTRA_EUNSUPPORTED, "GPU path needs head_dim=128, or a multiple of 128 in [256, 1024] with group_size=64 (got %d)",
                p.head_dim);
  if (p.group_size != 32) return fail(SPECTRA_EUNSUPPORTED, "GPU path needs group_size=32 at head_dim=128 (got %d)", p.group_size);
  if (record_words(p) > 64) return fail(SPECTRA_EUNSUPPORTED, "record of %d words exceeds 64", record_words(p));
  return SPECTRA_OK;
}

spectra_status fit_from_moments(const spectra_params& p, int64_t n_tokens, const double* gram,
                                const double* colsum, float* basis, float* mean, double* var,
                                uint8_t* bits, float* scale) {
  const int d = p.head_dim;
  if (n_tokens <= 0) return fail(SPECTRA_EINVAL, "fit needs at least one token");
  const double invT = 1.0 / (double)n_tokens;
  std::vector<double> mu(d), S((size_t)d * d), C((size_t)d * d), w(d), V((size_t)d * d);
  for (int i = 0; i < d; ++i) {
    mu[i] = colsum[i] * invT;
    if (!std::isfinite(mu[i])) return fail(SPECTRA_ENUMERIC, "non-finite token mean");
  }
  for (int i = 0; i < d; ++i)
    for (int j = 0; j < d; ++j) {
      const double s = gram[(size_t)i * d + j] * invT;
      if (!std::isfinite(s)) return fail(SPECTRA_ENUMERIC, "non-finite second moment");
      S[(size_t)i * d + j] = s;
      C[(size_t)i * d + j] = s - mu[i] * mu[j];
    }
  // Sec. 3.1: eigenbasis of the uncentered second moment (centered=1: covariance).
  spectra_status st = eigh_sym(p.centered ? C.data() : S.data(), d, w.data(), V.data());
  if (st != SPECTRA_OK) return st;
  std::vector<double> V32((size_t)d * d);
  for (size_t i = 0; i < (size_t)d * d; ++i) {
    basis[i] = (float)V[i];
    V32[i] = (double)basis[i];
  }
  // m = mu . V32 (coefficient-space mean), v_j = V32_j^T C V32_j (centered variance)
  std::vector<double> Cv(d);
  for (int j = 0; j < d; ++j) {
    double m = 0.0;
    for (int i = 0; i < d; ++i) m += mu[i] * V32[(size_t)i * d + j];
    mean[j] = (float)m;
    for (int i = 0; i < d; ++i) {
      double s = 0.0;
      for (int k = 0; k < d; ++k) s += C[(size_t)i * d + k] * V32[(size_t)k * d + j];
      Cv[i] = s;
    }
    double vj = 0.0;
    for (int i = 0; i < d; ++i) vj += V32[(size_t)i * d + j] * Cv[i];
    var[j] = vj;
  }
  if (scale) {
    // Eq. gsvd, square-root split: coordinate j of the orthonormal latent times
    // lambda_j^(-1/4) (lambda floored at lambda_0 2^-40); widths from the scaled variances
    const double floor_l = w[0] > 0.0 ? w[0] * std::ldexp(1.0, -40) : 0.0;
    for (int j = 0; j < d; ++j) {
      scale[j] = w[0] > 0.0 ? (float)std::pow(std::max(w[j], floor_l), -0.25) : 1.0f;
      const double f = (double)scale[j];
      var[j] *= f * f;
    }
  }
  return allocate_bits(var, p, bits);
}

}  // namespace spectra

using namespace spectra;

extern "C" {

spectra_status spectra_codec_init(spectra_codec* c, const spectra_params* p, int64_t n_streams) {
  if (!c || !p) return fail(SPECTRA_EINVAL, "null codec or params");
  spectra_status st = check_params(*p);
  if (st != SPECTRA_OK) return st;
  if (n_streams < 0) return fail(SPECTRA_EINVAL, "n_streams negative");
  c->p = *p;
  c->n_streams = n_streams;
  c->record_words = record_words(*p);
  c->reserved = 0;
  return SPECTRA_OK;
}

int32_t spectra_record_budget_bits(const spectra_params* p) { return p ? budget_bits(*p) : -1; }
int32_t spectra_record_words(const spectra_params* p) { return p ? record_words(*p) : -1; }

spectra_status spectra_split_budget(const spectra_params* p, double kappa, spectra_params* p_k, spectra_params* p_v) {
  if (!p || !p_k || !p_v) return fail(SPECTRA_EINVAL, "null argument");
  spectra_status st = check_params(*p);
  if (st != SPECTRA_OK) return st;
  if (!(kappa > 0.0 && kappa < 1.0)) return fail(SPECTRA_EINVAL, "kappa must lie in (0, 1)");
  // the two records' combined budget, keys' share rounded to whole words
  const int64_t total = 2 * (int64_t)budget_bits(*p);
  const int64_t rk = 32 * (int64_t)std::floor(kappa * (double)total / 32.0 + 0.5);
  const int64_t rv = total - rk;
  const int64_t one = (int64_t)p->group_size + p->meta_bits;
  if (rk < one || rv < one)
    return fail(SPECTRA_EINVAL, "kappa=%g leaves a tensor without a whole group (%lld + %lld bits)", kappa,
                (long long)rk, (long long)rv);
  *p_k = *p;
  *p_v = *p;
  p_k->budget_bits = (int32_t)rk;
  p_v->budget_bits = (int32_t)rv;
  return SPECTRA_OK;
}

int64_t spectra_packed_words(const spectra_codec* c, int64_t t_capacity) {
  if (!c || t_capacity < 0 || t_capacity % 64 != 0) return -1;
  return c->n_streams * t_capacity * (int64_t)c->record_words;
}

spectra_status spectra_allocate_bits(const double* var, const spectra_params* p, uint8_t* bits_out) {
  if (!var || !p || !bits_out) return fail(SPECTRA_EINVAL, "null argument");
  spectra_status st = check_params(*p);
  if (st != SPECTRA_OK) return st;
  return allocate_bits(var, *p, bits_out);
}

spectra_status spectra_eigh_host(const double* a, int32_t n, double* w, double* v) {
  if (!a || !w || !v) return fail(SPECTRA_EINVAL, "null argument");
  return eigh_sym(a, n, w, v);
}

spectra_status spectra_fit_from_moments_host(const spectra_params* p, int64_t n_tokens, const double* gram,
                                             const double* colsum, float* basis, float* mean, double* var,
                                             uint8_t* bits) {
  if (!p || !gram || !colsum || !basis || !mean || !var || !bits) return fail(SPECTRA_EINVAL, "null argument");
  spectra_status st = check_params(*p);
  if (st != SPECTRA_OK) return st;
  return fit_from_moments(*p, n_tokens, gram, colsum, basis, mean, var, bits);
}

const char* spectra_status_string(spectra_status s) {
  switch (s) {
    case SPECTRA_OK: return "ok";
    case SPECTRA_EINVAL: return "invalid argument";
    case SPECTRA_EUNSUPPORTED: return "unsupported on the GPU path";
    case SPECTRA_ENUMERIC: return "numerical failure";
    case SPECTRA_EWORKSPACE: return "workspace too small";
    case SPECTRA_EHIP: return "HIP runtime error";
  }
  return "unknown status";
}

const char* spectra_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
