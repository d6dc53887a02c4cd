// Kernel argument blocks and launchers of the per-layer geometry (one stream per
// (sequence, layer, tensor), d = n_kv_heads x 128 in [256, 1024], latent groups of 64).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace spectra_dev {

struct LayerGramArgs {
  const void* x;
  int64_t stream_stride, token_stride, n;
  int64_t chunk_tokens;
  int32_t k_split;
  int32_t n_streams;
  int32_t d;
  double* partial;  // [n_streams][k_split][d*d]
  double* moments;  // [n_streams][d*d + d]
};

struct LayerEncodeArgs {
  const void* x;  // bf16
  int64_t stream_stride, token_stride;
  int64_t t0, n;
  const float* basis;
  const float* mean;
  const uint8_t* bits;
  uint32_t* packed;
  int64_t t_cap;
  int32_t W, d, n_streams;
  const float* lscale;  // NULL or [n_streams][d]: square-root split factors
};

struct LayerDecodeArgs {
  const uint32_t* packed;
  int64_t t_cap, t0, n;
  const float* basis;
  const float* mean;
  const uint8_t* bits;
  float* out;  // [n_streams][n][d]
  int32_t W, d, n_streams;
  const float* lscale;  // NULL or [n_streams][d]: square-root split factors
};

}  // namespace spectra_dev

namespace spectra {
void layer_gram_layout(int32_t d, int64_t n_streams, int64_t n_tokens, int32_t* k_split, int64_t* chunk_tokens);
hipError_t launch_layer_moments(const spectra_dev::LayerGramArgs& g, bool f32_in, hipStream_t st);
hipError_t launch_layer_encode(const spectra_dev::LayerEncodeArgs& a, hipStream_t st);
hipError_t launch_layer_decode(const spectra_dev::LayerDecodeArgs& a, hipStream_t st);
}  // namespace spectra
