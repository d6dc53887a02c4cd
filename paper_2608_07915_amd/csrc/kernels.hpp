// Kernel argument blocks and launchers of libspectra (host and device visible).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace spectra_dev {

struct EncodeArgs {
  const void* x;
  int64_t stream_stride, token_stride;  // elements
  int64_t t0, n;                        // record slots [t0, t0 + n)
  const float* basis;
  const float* mean;
  const uint8_t* bits;
  uint32_t* packed;
  int64_t t_cap;
  int32_t W;
  int32_t n_streams;
};

struct DecodeArgs {
  const uint32_t* packed;
  int64_t t_cap, t0, n;
  const float* basis;
  const float* mean;
  const uint8_t* bits;
  float* out;  // [n_streams][n][128]
  int32_t W;
  int32_t n_streams;
};

struct PackArgs {
  const uint8_t* codes;  // pack input
  const uint32_t* meta;
  uint32_t* packed;      // pack output
  const uint32_t* packed_in;  // unpack input
  uint8_t* codes_out;
  uint32_t* meta_out;
  const uint8_t* bits;
  int64_t n, t_cap;
  int32_t W;
  int32_t n_streams;
};

struct GramArgs {
  const void* x;
  int64_t stream_stride, token_stride, n;
  int64_t chunk_tokens;
  int32_t n_chunks;
  int32_t n_streams;
  double* partial;  // [n_streams][n_chunks][128*128 + 128]
  double* moments;  // [n_streams][128*128 + 128]
};

struct AttnArgs {
  const uint32_t* packed_k;
  const uint32_t* packed_v;
  int64_t t_cap, n_tokens;
  const float* basis_k;
  const float* basis_v;
  const float* mean_v;
  const uint8_t* bits_k;
  const uint8_t* bits_v;
  const void* q;
  int32_t q_f32;
  int32_t batch, n_q_heads, n_kv_heads, n_qh;
  int32_t Wk, Wv;
  float scale_log2;      // softmax scale * log2(e)
  int32_t n_chunks;      // split of the token range per (batch, kv head)
  int32_t tiles_per_chunk;
  int32_t group_major;   // scan grid order: 0 = (chunk, kv head, sequence); 1 = 1-D, chunk-major over groups
  // decode step only: the new token of every stream is encoded into slot t_new
  // of app_k / app_v (the same caches as packed_k / packed_v) before attention
  const void* k_new;     // [batch][n_kv_heads][128], fp32 if app_f32 else bf16
  const void* v_new;
  const float* mean_k;
  uint32_t* app_k;
  uint32_t* app_v;
  int64_t t_new;
  int32_t app_f32;
  float* partial;        // workspace: per-chunk softmax partials
  float* out;            // [batch][n_q_heads][128]
  // attention with rotary position embeddings only: pair frequencies [64] (device)
  // and the query's position (key t sits at position t)
  const float* inv_freq;
  int64_t q_pos;
};

// Batched fp64 product C_b = A_{b / a_div} B_b, element strides; M, N multiples
// of 64, K of 16 (calibration from weights).
struct WgemmArgs {
  const void* A;
  const void* B;
  double* C;
  int32_t M, N, K;
  int64_t a_rs, a_cs, a_bs;
  int32_t a_div;
  int64_t b_rs, b_cs, b_bs;
  int64_t c_rs, c_bs;
};

}  // namespace spectra_dev

namespace spectra {
hipError_t launch_encode(const spectra_dev::EncodeArgs& a, bool f32_input, hipStream_t st);
hipError_t launch_decode(const spectra_dev::DecodeArgs& a, hipStream_t st);
hipError_t launch_pack_codes(const spectra_dev::PackArgs& a, bool unpack, hipStream_t st);
hipError_t launch_gram(const spectra_dev::GramArgs& a, bool f32_input, hipStream_t st);
// Decode-step attention; with a.app_k != nullptr the new token of every stream is
// appended first (the decode step).
hipError_t launch_attention(const spectra_dev::AttnArgs& a, hipStream_t st);
// Merge of the chunk partials in a.partial into a.out (+ m_V, inverse value rotation).
hipError_t launch_combine(const spectra_dev::AttnArgs& a, hipStream_t st);
// Attention with rotary position embeddings (Mode A keys, latent values), then the
// combine; chunk split from rope_attention_chunks.
hipError_t launch_attention_rope(const spectra_dev::AttnArgs& a, hipStream_t st);
int32_t rope_attention_chunks(int32_t batch, int32_t n_kv_heads, int64_t n_tokens, int32_t* tiles_per_chunk,
                              int32_t per_cu);
// Workspace layout of decode_attention (bytes), shared by the host API and launcher.
size_t attention_partial_floats(int32_t batch, int32_t n_q_heads, int32_t n_chunks);
int32_t attention_chunks(int32_t batch, int32_t n_kv_heads, int64_t n_tokens, int32_t* tiles_per_chunk);
// moments[s] = [W_s^T G W_s, hbar W_s] for W [n_streams][d_model][d] fp32 (d a multiple of 64)
// and per-layer G [layers][d_model][d_model], hbar [layers][d_model] fp64 (layer = s /
// streams_per_layer); scratch: n_streams * d_model * d doubles.
hipError_t launch_weights_moments(const float* W, const double* G, const double* hbar, int32_t d_model, int32_t d,
                                  int32_t n_streams, int32_t streams_per_layer, double* scratch, double* moments,
                                  int64_t mom_stride, hipStream_t st);
}  // namespace spectra
