// Shared host-side helpers of libspectra: error reporting and parameter checks.
#pragma once
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <string>

#include "spectra.h"

namespace spectra {

// Thread-local text of the last error; set by fail().
void set_last_error(const std::string& msg);
spectra_status fail(spectra_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

// Per-token bit budget R (metadata included) and record width W = floor(R / 32).
int32_t budget_bits(const spectra_params& p);
inline int32_t record_words(const spectra_params& p) { return budget_bits(p) / 32; }

// Host-side validation of parameters (any head_dim); GPU limits are checked separately.
spectra_status check_params(const spectra_params& p);
spectra_status check_params_gpu(const spectra_params& p);
// Per-layer geometry on the GPU: one stream per (sequence, layer, tensor), d = n_kv_heads x 128
// in [256, 1024], groups of 64 (fit, encode and decode only).
bool layer_geometry(const spectra_params& p);

// Exact integer allocation (App. D objective, Sec. 3.2 groups, App. F rate).
spectra_status allocate_bits(const double* var, const spectra_params& p, uint8_t* bits);

// Symmetric eigendecomposition, descending, sign-normalised columns.
spectra_status eigh_sym(const double* a, int n, double* w, double* v);

// Fit of one stream from its moments.
// scale: NULL, or the square-root split factors f_j to write (var then holds v_j f_j^2).
spectra_status fit_from_moments(const spectra_params& p, int64_t n_tokens, const double* gram,
                                const double* colsum, float* basis, float* mean, double* var,
                                uint8_t* bits, float* scale = nullptr);

}  // namespace spectra
