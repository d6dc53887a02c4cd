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
  double* partial;  // [n_streams][k_split][d*d + d]: Gram, then column sums
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

namespace spectra_dev {

// Decode-step attention over per-layer latents (App. E, Mode B, with the latent spanning
// all KV heads of the layer): stream b of both codecs is sequence b.
struct LayerAttnArgs {
  const uint32_t* packed_k;
  const uint32_t* packed_v;
  int64_t t_cap, n_tokens;
  const float* basis_k;
  const float* basis_v;
  const float* mean_v;
  const uint8_t* bits_k;
  const uint8_t* bits_v;
  const float* lscale_k;  // NULL or [batch][d]: square-root split factors of the keys' latent
  const float* lscale_v;  // NULL or [batch][d]: of the values' latent
  const void* q;
  int32_t q_f32;
  int32_t batch, n_q_heads, n_kv_heads, d, Wk, Wv;
  float scale_log2;
  int32_t n_chunks, tiles_per_chunk;     // score pass: token chunks
  int32_t nv_chunks, v_tiles_per_chunk;  // value pass: token chunks (x 2 head blocks)
  float* qt;      // [batch][Hq][d]: scale log2(e) q_h V_K[kv rows], 0 on dropped groups
  float* ml;      // [batch][Hq][2]: softmax max and sum over all tokens
  uint16_t* qh;   // [batch][2][32][d] fp16: qt as high and low parts, kept groups in slot order
  float* qsum;    // [batch][Hq][16]: per group sums of qt
  float* scores;  // [batch][Hq][n_tokens] (log2 domain)
  float* stats;   // [batch][n_chunks][Hq][2]: chunk max, chunk sum of exp2(s - max)
  float* part;    // [batch][nv_chunks][Hq][d + 16]: value sums per coefficient, zero-point sums per group
  float* out;     // [batch][Hq][128]
};

}  // namespace spectra_dev

namespace spectra {
int32_t layer_attention_chunks(int32_t batch, int64_t n_tokens, int32_t* tiles_per_chunk);
size_t layer_attention_ws_floats(int32_t batch, int32_t n_q_heads, int32_t d, int64_t n_tokens);
void layer_attention_ws_layout(spectra_dev::LayerAttnArgs& a, float* ws);
size_t layer_scores_lds_bytes(int32_t d, int32_t Wk);
hipError_t launch_layer_attention(const spectra_dev::LayerAttnArgs& a, hipStream_t st);
}  // namespace spectra
