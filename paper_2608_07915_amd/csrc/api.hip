// C entry points of libspectra that run on the GPU: argument checks, workspace
// layout and kernel launches. Host-only entry points live in host_fit.cpp.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <thread>
#include <vector>

#include "host_common.hpp"
#include "kernels.hpp"
#include "layer.hpp"

using namespace spectra;
using spectra_dev::AttnArgs;
using spectra_dev::DecodeArgs;
using spectra_dev::EncodeArgs;
using spectra_dev::GramArgs;
using spectra_dev::PackArgs;

namespace {

constexpr int kD = 128;
constexpr int64_t kMoments = (int64_t)kD * kD + kD;  // gram + column sums per stream

spectra_status hip_fail(hipError_t e, const char* what) {
  return fail(SPECTRA_EHIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

spectra_status check_codec(const spectra_codec* c, const char* name, bool layer_ok = false) {
  if (!c) return fail(SPECTRA_EINVAL, "%s: null codec", name);
  spectra_status st = check_params_gpu(c->p);
  if (st != SPECTRA_OK) return st;
  if (!layer_ok && layer_geometry(c->p))
    return fail(SPECTRA_EUNSUPPORTED, "%s: the per-layer geometry (head_dim %d, group_size 64) supports fit, encode and decode only",
                name, c->p.head_dim);
  if (c->record_words != record_words(c->p))
    return fail(SPECTRA_EINVAL, "%s: record_words %d does not match the parameters (%d); call spectra_codec_init",
                name, c->record_words, record_words(c->p));
  if (c->n_streams <= 0 || c->n_streams > 65535)
    return fail(SPECTRA_EINVAL, "%s: n_streams=%lld out of range [1, 65535]", name, (long long)c->n_streams);
  if (!c->basis || !c->mean || !c->var || !c->bits) return fail(SPECTRA_EINVAL, "%s: null codec array", name);
  if (c->lscale && !layer_geometry(c->p))
    return fail(SPECTRA_EUNSUPPORTED, "%s: the square-root latent split (lscale) runs in the per-layer geometry only", name);
  if (c->lscale && !aligned(c->lscale, 4)) return fail(SPECTRA_EINVAL, "%s: lscale must be 4-byte aligned", name);
  if (!aligned(c->basis, 16) || !aligned(c->mean, 4) || !aligned(c->var, 4) || !aligned(c->bits, 4))
    return fail(SPECTRA_EINVAL, "%s: basis must be 16-byte aligned, the other codec arrays 4-byte aligned", name);
  return SPECTRA_OK;
}

spectra_status check_slots(int64_t t0, int64_t n, int64_t t_cap) {
  if (t_cap <= 0 || t_cap % 64 != 0) return fail(SPECTRA_EINVAL, "t_capacity=%lld must be a positive multiple of 64", (long long)t_cap);
  if (t0 < 0 || n < 0 || t0 + n > t_cap)
    return fail(SPECTRA_EINVAL, "slots [%lld, %lld) exceed t_capacity %lld", (long long)t0, (long long)(t0 + n), (long long)t_cap);
  return SPECTRA_OK;
}

spectra_status check_input(const void* x, spectra_dtype dt, int64_t stream_stride, int64_t token_stride, int64_t n_streams,
                           int64_t n_tokens, int64_t d) {
  if (dt != SPECTRA_F32 && dt != SPECTRA_BF16) return fail(SPECTRA_EINVAL, "dtype %d not supported", (int)dt);
  if (!x) return fail(SPECTRA_EINVAL, "null input");
  const int64_t vec = dt == SPECTRA_F32 ? 4 : 8;  // elements per 16 bytes
  if (!aligned(x, 16)) return fail(SPECTRA_EINVAL, "input must be 16-byte aligned");
  if (stream_stride < 0 || token_stride < 0 || stream_stride % vec || token_stride % vec)
    return fail(SPECTRA_EINVAL, "strides must be non-negative multiples of %lld elements", (long long)vec);
  if (n_tokens > 1 && token_stride < d) return fail(SPECTRA_EINVAL, "token_stride must be >= head_dim");
  if (n_streams > 1 && stream_stride == 0) return fail(SPECTRA_EINVAL, "stream_stride is 0 for several streams");
  return SPECTRA_OK;
}

size_t round256(size_t b) { return (b + 255) / 256 * 256; }

void moments_layout(int64_t n_streams, int64_t n_tokens, int32_t* n_chunks, int64_t* chunk_tokens) {
  int64_t want = (1024 + n_streams - 1) / n_streams;
  const int64_t max_chunks = (n_tokens + 63) / 64;
  want = std::max<int64_t>(1, std::min(want, max_chunks));
  int64_t ct = (n_tokens + want - 1) / want;
  ct = (ct + 63) / 64 * 64;
  *chunk_tokens = ct;
  *n_chunks = (int32_t)((n_tokens + ct - 1) / ct);
}

size_t fit_ws_bytes(int64_t n_streams, int64_t n_tokens) {
  int32_t nch;
  int64_t ct;
  moments_layout(n_streams, n_tokens, &nch, &ct);
  return (size_t)n_streams * (size_t)(nch + 1) * (size_t)kMoments * sizeof(double);
}

// Per-layer geometry: moments [S][d*d + d], then the token-split partials [S][k_split][d*d + d].
size_t layer_fit_ws_bytes(int32_t d, int64_t n_streams, int64_t n_tokens) {
  int32_t ks;
  int64_t ct;
  layer_gram_layout(d, n_streams, n_tokens, &ks, &ct);
  const size_t dd = (size_t)d * d;
  return round256((size_t)n_streams * (dd + d) * sizeof(double)) + (size_t)n_streams * ks * (dd + d) * sizeof(double);
}

// Host half of a fit: eigenbasis, mean, variances and widths of every stream from
// its moments (gram, column sums over n_tokens), in parallel, then copied into the
// codec arrays. Synchronises hs.
spectra_status finish_fit(spectra_codec* c, const std::vector<double>& mom, int64_t n_tokens, hipStream_t hs) {
  const int64_t S = c->n_streams;
  const int d = c->p.head_dim;
  const int64_t mstride = (int64_t)d * d + d;
  hipError_t e = hipSuccess;
  std::vector<float> basis((size_t)S * d * d), mean((size_t)S * d), var32((size_t)S * d);
  std::vector<double> var((size_t)S * d);
  std::vector<float> scale(c->lscale ? (size_t)S * d : 0);
  const int nG = d / c->p.group_size;
  std::vector<uint8_t> bits((size_t)S * nG);
  std::vector<spectra_status> res((size_t)S, SPECTRA_OK);
  std::vector<std::string> msgs((size_t)S);
  const int nthreads = (int)std::max<int64_t>(1, std::min<int64_t>(S, std::min(16u, std::max(1u, std::thread::hardware_concurrency()))));
  std::vector<std::thread> pool;
  for (int w = 0; w < nthreads; ++w) {
    pool.emplace_back([&, w]() {
      for (int64_t s = w; s < S; s += nthreads) {
        const double* m = &mom[(size_t)(s * mstride)];
        res[(size_t)s] = fit_from_moments(c->p, n_tokens, m, m + (size_t)d * d, &basis[(size_t)s * d * d], &mean[(size_t)s * d],
                                          &var[(size_t)s * d], &bits[(size_t)s * nG],
                                          c->lscale ? &scale[(size_t)s * d] : nullptr);
        if (res[(size_t)s] != SPECTRA_OK) msgs[(size_t)s] = spectra_last_error();
      }
    });
  }
  for (auto& t : pool) t.join();
  for (int64_t s = 0; s < S; ++s)
    if (res[(size_t)s] != SPECTRA_OK) return fail(res[(size_t)s], "fit stream %lld: %s", (long long)s, msgs[(size_t)s].c_str());
  for (size_t i = 0; i < var.size(); ++i) var32[i] = (float)var[i];
  e = hipMemcpyAsync(c->basis, basis.data(), basis.size() * sizeof(float), hipMemcpyHostToDevice, hs);
  if (e == hipSuccess) e = hipMemcpyAsync(c->mean, mean.data(), mean.size() * sizeof(float), hipMemcpyHostToDevice, hs);
  if (e == hipSuccess) e = hipMemcpyAsync(c->var, var32.data(), var32.size() * sizeof(float), hipMemcpyHostToDevice, hs);
  if (e == hipSuccess) e = hipMemcpyAsync(c->bits, bits.data(), bits.size(), hipMemcpyHostToDevice, hs);
  if (e == hipSuccess && c->lscale)
    e = hipMemcpyAsync(c->lscale, scale.data(), scale.size() * sizeof(float), hipMemcpyHostToDevice, hs);
  if (e == hipSuccess) e = hipStreamSynchronize(hs);
  if (e != hipSuccess) return hip_fail(e, "fit result copy");
  return SPECTRA_OK;
}

}  // namespace

extern "C" {

size_t spectra_fit_workspace_bytes(const spectra_codec* c, int64_t n_tokens) {
  if (!c || n_tokens <= 0 || c->n_streams <= 0) return 0;
  if (layer_geometry(c->p)) return layer_fit_ws_bytes(c->p.head_dim, c->n_streams, n_tokens);
  return fit_ws_bytes(c->n_streams, n_tokens);
}

spectra_status spectra_fit_basis(spectra_codec* c, const void* x, spectra_dtype dt, int64_t n_tokens,
                                 int64_t stream_stride, int64_t token_stride, void* workspace, size_t ws_bytes,
                                 void* stream) {
  spectra_status st = check_codec(c, "fit_basis", true);
  if (st != SPECTRA_OK) return st;
  if (n_tokens <= 0) return fail(SPECTRA_EINVAL, "fit_basis needs n_tokens >= 1");
  st = check_input(x, dt, stream_stride, token_stride, c->n_streams, n_tokens, c->p.head_dim);
  if (st != SPECTRA_OK) return st;
  const int64_t S = c->n_streams;
  if (!workspace || !aligned(workspace, 256)) return fail(SPECTRA_EINVAL, "fit workspace must be 256-byte aligned");
  if (layer_geometry(c->p)) {
    const int d = c->p.head_dim;
    const size_t need = layer_fit_ws_bytes(d, S, n_tokens);
    if (ws_bytes < need) return fail(SPECTRA_EWORKSPACE, "fit workspace %zu < %zu bytes", ws_bytes, need);
    hipStream_t hs = (hipStream_t)stream;
    spectra_dev::LayerGramArgs g{};
    g.x = x;
    g.stream_stride = stream_stride;
    g.token_stride = token_stride;
    g.n = n_tokens;
    g.n_streams = (int32_t)S;
    g.d = d;
    layer_gram_layout(d, S, n_tokens, &g.k_split, &g.chunk_tokens);
    g.moments = reinterpret_cast<double*>(workspace);
    g.partial = reinterpret_cast<double*>(static_cast<char*>(workspace) +
                                          round256((size_t)S * ((size_t)d * d + d) * sizeof(double)));
    hipError_t e = launch_layer_moments(g, dt == SPECTRA_F32, hs);
    if (e != hipSuccess) return hip_fail(e, "fit moments launch");
    std::vector<double> mom((size_t)S * ((size_t)d * d + d));
    e = hipMemcpyAsync(mom.data(), g.moments, mom.size() * sizeof(double), hipMemcpyDeviceToHost, hs);
    if (e != hipSuccess) return hip_fail(e, "fit moments copy");
    e = hipStreamSynchronize(hs);
    if (e != hipSuccess) return hip_fail(e, "fit moments sync");
    return finish_fit(c, mom, n_tokens, hs);
  }
  if (ws_bytes < fit_ws_bytes(S, n_tokens))
    return fail(SPECTRA_EWORKSPACE, "fit workspace %zu < %zu bytes", ws_bytes, fit_ws_bytes(S, n_tokens));
  hipStream_t hs = (hipStream_t)stream;
  GramArgs g{};
  g.x = x;
  g.stream_stride = stream_stride;
  g.token_stride = token_stride;
  g.n = n_tokens;
  moments_layout(S, n_tokens, &g.n_chunks, &g.chunk_tokens);
  g.n_streams = (int32_t)S;
  g.moments = reinterpret_cast<double*>(workspace);
  g.partial = g.moments + S * kMoments;
  hipError_t e = launch_gram(g, dt == SPECTRA_F32, hs);
  if (e != hipSuccess) return hip_fail(e, "fit moments launch");
  std::vector<double> mom((size_t)(S * kMoments));
  e = hipMemcpyAsync(mom.data(), g.moments, mom.size() * sizeof(double), hipMemcpyDeviceToHost, hs);
  if (e != hipSuccess) return hip_fail(e, "fit moments copy");
  e = hipStreamSynchronize(hs);
  if (e != hipSuccess) return hip_fail(e, "fit moments sync");

  return finish_fit(c, mom, n_tokens, hs);
}

size_t spectra_fit_weights_workspace_bytes(const spectra_codec* c, int32_t d_model) {
  if (!c || c->n_streams <= 0 || d_model <= 0 || c->p.head_dim <= 0) return 0;
  const size_t d = (size_t)c->p.head_dim;
  return round256((size_t)c->n_streams * (d * d + d) * sizeof(double)) +
         (size_t)c->n_streams * (size_t)d_model * d * sizeof(double);
}

spectra_status spectra_fit_weights(spectra_codec* c, const float* W, int32_t d_model, const double* G,
                                   const double* hbar, int32_t streams_per_layer, void* workspace, size_t ws_bytes,
                                   void* stream) {
  spectra_status st = check_codec(c, "fit_weights", true);
  if (st != SPECTRA_OK) return st;
  if (!W || !G || !aligned(W, 4) || !aligned(G, 8) || (hbar && !aligned(hbar, 8)))
    return fail(SPECTRA_EINVAL, "fit_weights: W and G must be non-null and aligned (4 / 8 bytes)");
  if (d_model < 64 || d_model > 16384 || d_model % 64 != 0)
    return fail(SPECTRA_EINVAL, "fit_weights: d_model=%d must be a multiple of 64 in [64, 16384]", d_model);
  const int64_t S = c->n_streams;
  if (streams_per_layer < 1 || S % streams_per_layer != 0)
    return fail(SPECTRA_EINVAL, "fit_weights: streams_per_layer=%d must divide n_streams=%lld", streams_per_layer,
                (long long)S);
  if (!workspace || !aligned(workspace, 256)) return fail(SPECTRA_EINVAL, "fit_weights workspace must be 256-byte aligned");
  const size_t need = spectra_fit_weights_workspace_bytes(c, d_model);
  if (ws_bytes < need) return fail(SPECTRA_EWORKSPACE, "fit_weights workspace %zu < %zu bytes", ws_bytes, need);
  hipStream_t hs = (hipStream_t)stream;
  const int d = c->p.head_dim;  // 128 per head; d_kv in the per-layer geometry
  const int64_t mstride = (int64_t)d * d + d;
  double* moments = reinterpret_cast<double*>(workspace);
  double* scratch = reinterpret_cast<double*>(static_cast<char*>(workspace) +
                                              round256((size_t)S * (size_t)mstride * sizeof(double)));
  hipError_t e = launch_weights_moments(W, G, hbar, d_model, d, (int32_t)S, streams_per_layer, scratch, moments,
                                        mstride, hs);
  if (e != hipSuccess) return hip_fail(e, "fit_weights launch");
  std::vector<double> mom((size_t)(S * mstride));
  e = hipMemcpyAsync(mom.data(), moments, mom.size() * sizeof(double), hipMemcpyDeviceToHost, hs);
  if (e != hipSuccess) return hip_fail(e, "fit_weights moments copy");
  e = hipStreamSynchronize(hs);
  if (e != hipSuccess) return hip_fail(e, "fit_weights moments sync");
  return finish_fit(c, mom, 1, hs);  // moments are already expectations
}

spectra_status spectra_encode(const spectra_codec* c, const void* x, spectra_dtype dt, int64_t stream_stride,
                              int64_t token_stride, int64_t t0, int64_t n_tokens, uint32_t* packed, int64_t t_capacity,
                              void* stream) {
  spectra_status st = check_codec(c, "encode", true);
  if (st != SPECTRA_OK) return st;
  st = check_slots(t0, n_tokens, t_capacity);
  if (st != SPECTRA_OK) return st;
  if (n_tokens == 0) return SPECTRA_OK;
  st = check_input(x, dt, stream_stride, token_stride, c->n_streams, n_tokens, c->p.head_dim);
  if (st != SPECTRA_OK) return st;
  if (!packed || !aligned(packed, 4)) return fail(SPECTRA_EINVAL, "packed must be non-null and 4-byte aligned");
  if (c->record_words == 0) return SPECTRA_OK;
  if (layer_geometry(c->p)) {
    if (dt != SPECTRA_BF16) return fail(SPECTRA_EUNSUPPORTED, "encode: the per-layer geometry takes bf16 tokens");
    spectra_dev::LayerEncodeArgs a{};
    a.x = x;
    a.stream_stride = stream_stride;
    a.token_stride = token_stride;
    a.t0 = t0;
    a.n = n_tokens;
    a.basis = c->basis;
    a.mean = c->mean;
    a.bits = c->bits;
    a.packed = packed;
    a.t_cap = t_capacity;
    a.W = c->record_words;
    a.d = c->p.head_dim;
    a.n_streams = (int32_t)c->n_streams;
    a.lscale = c->lscale;
    hipError_t e = launch_layer_encode(a, (hipStream_t)stream);
    return e == hipSuccess ? SPECTRA_OK : hip_fail(e, "encode launch");
  }
  EncodeArgs a{};
  a.x = x;
  a.stream_stride = stream_stride;
  a.token_stride = token_stride;
  a.t0 = t0;
  a.n = n_tokens;
  a.basis = c->basis;
  a.mean = c->mean;
  a.bits = c->bits;
  a.packed = packed;
  a.t_cap = t_capacity;
  a.W = c->record_words;
  a.n_streams = (int32_t)c->n_streams;
  hipError_t e = launch_encode(a, dt == SPECTRA_F32, (hipStream_t)stream);
  return e == hipSuccess ? SPECTRA_OK : hip_fail(e, "encode launch");
}

spectra_status spectra_decode(const spectra_codec* c, const uint32_t* packed, int64_t t_capacity, int64_t t0,
                              int64_t n_tokens, float* out, void* stream) {
  spectra_status st = check_codec(c, "decode", true);
  if (st != SPECTRA_OK) return st;
  st = check_slots(t0, n_tokens, t_capacity);
  if (st != SPECTRA_OK) return st;
  if (n_tokens == 0) return SPECTRA_OK;
  if (!out || !aligned(out, 4)) return fail(SPECTRA_EINVAL, "out must be non-null and 4-byte aligned");
  if (c->record_words > 0 && (!packed || !aligned(packed, 4)))
    return fail(SPECTRA_EINVAL, "packed must be non-null and 4-byte aligned");
  if (layer_geometry(c->p)) {
    if (!aligned(out, 16)) return fail(SPECTRA_EINVAL, "decode: out must be 16-byte aligned for the per-layer geometry");
    spectra_dev::LayerDecodeArgs a{};
    a.packed = packed;
    a.t_cap = t_capacity;
    a.t0 = t0;
    a.n = n_tokens;
    a.basis = c->basis;
    a.mean = c->mean;
    a.bits = c->bits;
    a.out = out;
    a.W = c->record_words;
    a.d = c->p.head_dim;
    a.n_streams = (int32_t)c->n_streams;
    a.lscale = c->lscale;
    hipError_t e = launch_layer_decode(a, (hipStream_t)stream);
    return e == hipSuccess ? SPECTRA_OK : hip_fail(e, "decode launch");
  }
  DecodeArgs a{};
  a.packed = packed;
  a.t_cap = t_capacity;
  a.t0 = t0;
  a.n = n_tokens;
  a.basis = c->basis;
  a.mean = c->mean;
  a.bits = c->bits;
  a.out = out;
  a.W = c->record_words;
  a.n_streams = (int32_t)c->n_streams;
  hipError_t e = launch_decode(a, (hipStream_t)stream);
  return e == hipSuccess ? SPECTRA_OK : hip_fail(e, "decode launch");
}

size_t spectra_layer_attention_workspace_bytes(const spectra_codec* ck, int32_t batch, int32_t n_q_heads,
                                               int64_t n_tokens) {
  if (!ck || batch <= 0 || n_q_heads <= 0 || n_tokens <= 0) return 0;
  return layer_attention_ws_floats(batch, n_q_heads, ck->p.head_dim, n_tokens) * sizeof(float);
}

spectra_status spectra_layer_decode_attention(const spectra_codec* ck, const spectra_codec* cv, const uint32_t* packed_k,
                                              const uint32_t* packed_v, int64_t t_capacity, int64_t n_tokens,
                                              const void* q, spectra_dtype q_dt, int32_t batch, int32_t n_q_heads,
                                              int32_t n_kv_heads, float softmax_scale, float* out, void* workspace,
                                              size_t ws_bytes, void* stream) {
  const char* name = "layer_decode_attention";
  spectra_status st = check_codec(ck, name, true);
  if (st != SPECTRA_OK) return st;
  st = check_codec(cv, name, true);
  if (st != SPECTRA_OK) return st;
  if (!layer_geometry(ck->p) || !layer_geometry(cv->p) || ck->p.head_dim != cv->p.head_dim)
    return fail(SPECTRA_EINVAL, "%s: both codecs must use the same per-layer geometry", name);
  const int d = ck->p.head_dim;
  if (n_kv_heads <= 0 || n_kv_heads * 128 != d)
    return fail(SPECTRA_EINVAL, "%s: n_kv_heads * 128 must equal the latent width %d", name, d);
  if (n_q_heads <= 0 || n_q_heads % n_kv_heads != 0 || n_q_heads > 32)
    return fail(SPECTRA_EINVAL, "%s: n_q_heads must be a multiple of n_kv_heads, at most 32", name);
  if (batch <= 0 || batch > 65535 || batch > ck->n_streams || batch > cv->n_streams)
    return fail(SPECTRA_EINVAL, "%s: batch must be in [1, codec streams]", name);
  if (ck->record_words > 128 || cv->record_words > 128)
    return fail(SPECTRA_EUNSUPPORTED, "%s: records of at most 128 words", name);
  if (n_tokens <= 0) return fail(SPECTRA_EINVAL, "%s: attention needs n_tokens >= 1", name);
  st = check_slots(0, n_tokens, t_capacity);
  if (st != SPECTRA_OK) return st;
  if (q_dt != SPECTRA_F32 && q_dt != SPECTRA_BF16) return fail(SPECTRA_EINVAL, "%s: q dtype %d not supported", name, (int)q_dt);
  if (!q || !out || !aligned(q, 4) || !aligned(out, 4)) return fail(SPECTRA_EINVAL, "%s: q/out must be non-null and aligned", name);
  if ((ck->record_words > 0 && (!packed_k || !aligned(packed_k, 4))) ||
      (cv->record_words > 0 && (!packed_v || !aligned(packed_v, 4))))
    return fail(SPECTRA_EINVAL, "%s: packed_k / packed_v must be non-null and 4-byte aligned", name);
  if (!(softmax_scale == softmax_scale) || std::isinf(softmax_scale)) return fail(SPECTRA_EINVAL, "%s: softmax_scale not finite", name);
  const size_t need = spectra_layer_attention_workspace_bytes(ck, batch, n_q_heads, n_tokens);
  if (!workspace || !aligned(workspace, 256)) return fail(SPECTRA_EINVAL, "%s: workspace must be 256-byte aligned", name);
  if (ws_bytes < need) return fail(SPECTRA_EWORKSPACE, "%s: workspace %zu < %zu bytes", name, ws_bytes, need);
  int dev = 0, lds = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
  if (e != hipSuccess) return hip_fail(e, "device query");
  if ((size_t)lds < layer_scores_lds_bytes(d, ck->record_words))
    return fail(SPECTRA_EUNSUPPORTED, "%s: needs %zu bytes of LDS per workgroup", name, layer_scores_lds_bytes(d, ck->record_words));
  spectra_dev::LayerAttnArgs a{};
  a.packed_k = packed_k;
  a.packed_v = packed_v;
  a.t_cap = t_capacity;
  a.n_tokens = n_tokens;
  a.basis_k = ck->basis;
  a.basis_v = cv->basis;
  a.mean_v = cv->mean;
  a.bits_k = ck->bits;
  a.bits_v = cv->bits;
  a.lscale_k = ck->lscale;
  a.lscale_v = cv->lscale;
  a.q = q;
  a.q_f32 = q_dt == SPECTRA_F32;
  a.batch = batch;
  a.n_q_heads = n_q_heads;
  a.n_kv_heads = n_kv_heads;
  a.d = d;
  a.Wk = ck->record_words;
  a.Wv = cv->record_words;
  const float sc = softmax_scale > 0.0f ? softmax_scale : 1.0f / std::sqrt(128.0f);
  a.scale_log2 = sc * 1.4426950408889634f;
  a.out = out;
  layer_attention_ws_layout(a, reinterpret_cast<float*>(workspace));
  e = launch_layer_attention(a, (hipStream_t)stream);
  return e == hipSuccess ? SPECTRA_OK : hip_fail(e, "layer attention launch");
}

size_t spectra_attention_workspace_bytes(int32_t batch, int32_t n_q_heads, int32_t n_kv_heads, int64_t n_tokens) {
  if (batch <= 0 || n_q_heads <= 0 || n_kv_heads <= 0 || n_tokens <= 0) return 0;
  int32_t tpc;
  // one workspace serves both attention entry points (latent, and with rotary embeddings)
  const int32_t nch = std::max(attention_chunks(batch, n_kv_heads, n_tokens, &tpc),
                               rope_attention_chunks(batch, n_kv_heads, n_tokens, &tpc, 2));
  return attention_partial_floats(batch, n_q_heads, nch) * sizeof(float);
}

// Checks shared by decode_attention and decode_step; fills everything of AttnArgs
// except the decode-step append fields.
static spectra_status prepare_attention(const char* name, const spectra_codec* ck, const spectra_codec* cv,
                                        const uint32_t* packed_k, const uint32_t* packed_v, int64_t t_capacity,
                                        int64_t n_tokens, const void* q, spectra_dtype q_dt, int32_t batch,
                                        int32_t n_q_heads, int32_t n_kv_heads, float softmax_scale, float* out,
                                        void* workspace, size_t ws_bytes, AttnArgs* args) {
  spectra_status st = check_codec(ck, name);
  if (st != SPECTRA_OK) return st;
  st = check_codec(cv, name);
  if (st != SPECTRA_OK) return st;
  if (batch <= 0 || n_kv_heads <= 0 || n_q_heads <= 0 || n_q_heads % n_kv_heads != 0)
    return fail(SPECTRA_EINVAL, "%s: need batch > 0 and n_q_heads a positive multiple of n_kv_heads", name);
  if (n_q_heads / n_kv_heads > 16) return fail(SPECTRA_EUNSUPPORTED, "%s: more than 16 query heads per kv head", name);
  if (batch > 65535 || n_kv_heads > 65535) return fail(SPECTRA_EINVAL, "%s: batch or n_kv_heads too large", name);
  if ((int64_t)batch * n_kv_heads > ck->n_streams || (int64_t)batch * n_kv_heads > cv->n_streams)
    return fail(SPECTRA_EINVAL, "%s: batch * n_kv_heads exceeds the codec's streams", name);
  if (n_tokens <= 0) return fail(SPECTRA_EINVAL, "%s: attention needs n_tokens >= 1", name);
  st = check_slots(0, n_tokens, t_capacity);
  if (st != SPECTRA_OK) return st;
  if (t_capacity * (int64_t)std::max(ck->record_words, cv->record_words) >= ((int64_t)1 << 31))
    return fail(SPECTRA_EINVAL, "%s: t_capacity * record words must stay below 2^31 per stream", name);
  if (q_dt != SPECTRA_F32 && q_dt != SPECTRA_BF16) return fail(SPECTRA_EINVAL, "%s: q dtype %d not supported", name, (int)q_dt);
  if (!q || !out || !aligned(q, 4) || !aligned(out, 4)) return fail(SPECTRA_EINVAL, "%s: q/out must be non-null and aligned", name);
  if ((ck->record_words > 0 && (!packed_k || !aligned(packed_k, 4))) ||
      (cv->record_words > 0 && (!packed_v || !aligned(packed_v, 4))))
    return fail(SPECTRA_EINVAL, "%s: packed_k / packed_v must be non-null and 4-byte aligned", name);
  if (!(softmax_scale == softmax_scale) || std::isinf(softmax_scale))
    return fail(SPECTRA_EINVAL, "%s: softmax_scale not finite", name);
  const size_t need = spectra_attention_workspace_bytes(batch, n_q_heads, n_kv_heads, n_tokens);
  if (!workspace || !aligned(workspace, 256)) return fail(SPECTRA_EINVAL, "%s: workspace must be 256-byte aligned", name);
  if (ws_bytes < need) return fail(SPECTRA_EWORKSPACE, "%s: workspace %zu < %zu bytes", name, ws_bytes, need);
  AttnArgs a{};
  a.packed_k = packed_k;
  a.packed_v = packed_v;
  a.t_cap = t_capacity;
  a.n_tokens = n_tokens;
  a.basis_k = ck->basis;
  a.basis_v = cv->basis;
  a.mean_v = cv->mean;
  a.mean_k = ck->mean;
  a.bits_k = ck->bits;
  a.bits_v = cv->bits;
  a.q = q;
  a.q_f32 = q_dt == SPECTRA_F32;
  a.batch = batch;
  a.n_q_heads = n_q_heads;
  a.n_kv_heads = n_kv_heads;
  a.n_qh = n_q_heads / n_kv_heads;
  a.Wk = ck->record_words;
  a.Wv = cv->record_words;
  const float sc = softmax_scale > 0.0f ? softmax_scale : 1.0f / std::sqrt((float)kD);
  a.scale_log2 = sc * 1.4426950408889634f;
  a.n_chunks = attention_chunks(batch, n_kv_heads, n_tokens, &a.tiles_per_chunk);
  a.partial = reinterpret_cast<float*>(workspace);
  a.out = out;
  *args = a;
  return SPECTRA_OK;
}

spectra_status spectra_decode_attention(const spectra_codec* ck, const spectra_codec* cv, const uint32_t* packed_k,
                                        const uint32_t* packed_v, int64_t t_capacity, int64_t n_tokens, const void* q,
                                        spectra_dtype q_dt, int32_t batch, int32_t n_q_heads, int32_t n_kv_heads,
                                        float softmax_scale, float* out, void* workspace, size_t ws_bytes, void* stream) {
  AttnArgs a{};
  const spectra_status st = prepare_attention("decode_attention", ck, cv, packed_k, packed_v, t_capacity, n_tokens, q,
                                              q_dt, batch, n_q_heads, n_kv_heads, softmax_scale, out, workspace,
                                              ws_bytes, &a);
  if (st != SPECTRA_OK) return st;
  hipError_t e = launch_attention(a, (hipStream_t)stream);
  return e == hipSuccess ? SPECTRA_OK : hip_fail(e, "attention launch");
}

spectra_status spectra_decode_attention_rope(const spectra_codec* ck, const spectra_codec* cv, const uint32_t* packed_k,
                                             const uint32_t* packed_v, int64_t t_capacity, int64_t n_tokens, const void* q,
                                             spectra_dtype q_dt, int32_t batch, int32_t n_q_heads, int32_t n_kv_heads,
                                             float softmax_scale, const float* inv_freq, int64_t q_position, float* out,
                                             void* workspace, size_t ws_bytes, void* stream) {
  AttnArgs a{};
  const spectra_status st = prepare_attention("decode_attention_rope", ck, cv, packed_k, packed_v, t_capacity, n_tokens,
                                              q, q_dt, batch, n_q_heads, n_kv_heads, softmax_scale, out, workspace,
                                              ws_bytes, &a);
  if (st != SPECTRA_OK) return st;
  if (a.n_qh > 8) return fail(SPECTRA_EUNSUPPORTED, "decode_attention_rope: at most 8 query heads per kv head");
  if (a.Wk > 32 || a.Wv > 32) return fail(SPECTRA_EUNSUPPORTED, "decode_attention_rope: records of at most 32 words");
  if (!inv_freq || !aligned(inv_freq, 4)) return fail(SPECTRA_EINVAL, "decode_attention_rope: inv_freq must be non-null");
  if (q_position < 0) return fail(SPECTRA_EINVAL, "decode_attention_rope: q_position negative");
  a.inv_freq = inv_freq;
  a.q_pos = q_position;
  hipError_t e = launch_attention_rope(a, (hipStream_t)stream);  // sets the chunk split of the kernel it runs
  return e == hipSuccess ? SPECTRA_OK : hip_fail(e, "attention (rope) launch");
}

spectra_status spectra_decode_step(const spectra_codec* ck, const spectra_codec* cv, uint32_t* packed_k,
                                   uint32_t* packed_v, int64_t t_capacity, int64_t t, const void* k_new,
                                   const void* v_new, spectra_dtype kv_dt, const void* q, spectra_dtype q_dt,
                                   int32_t batch, int32_t n_q_heads, int32_t n_kv_heads, float softmax_scale, float* out,
                                   void* workspace, size_t ws_bytes, void* stream) {
  if (t < 0 || t >= t_capacity) return fail(SPECTRA_EINVAL, "decode_step: slot t=%lld outside [0, t_capacity)", (long long)t);
  AttnArgs a{};
  spectra_status st = prepare_attention("decode_step", ck, cv, packed_k, packed_v, t_capacity, t + 1, q, q_dt, batch,
                                        n_q_heads, n_kv_heads, softmax_scale, out, workspace, ws_bytes, &a);
  if (st != SPECTRA_OK) return st;
  if (kv_dt != SPECTRA_F32 && kv_dt != SPECTRA_BF16) return fail(SPECTRA_EINVAL, "decode_step: dtype %d not supported", (int)kv_dt);
  if (!k_new || !v_new || !aligned(k_new, 16) || !aligned(v_new, 16))
    return fail(SPECTRA_EINVAL, "decode_step: k_new / v_new must be non-null and 16-byte aligned");
  a.k_new = k_new;
  a.v_new = v_new;
  a.app_k = packed_k;
  a.app_v = packed_v;
  a.t_new = t;
  a.app_f32 = kv_dt == SPECTRA_F32;
  hipError_t e = launch_attention(a, (hipStream_t)stream);
  return e == hipSuccess ? SPECTRA_OK : hip_fail(e, "decode_step launch");
}

spectra_status spectra_pack_codes(const spectra_codec* c, const uint8_t* codes, const uint32_t* meta, int64_t n_tokens,
                                  uint32_t* packed, int64_t t_capacity, void* stream) {
  spectra_status st = check_codec(c, "pack_codes");
  if (st != SPECTRA_OK) return st;
  st = check_slots(0, n_tokens, t_capacity);
  if (st != SPECTRA_OK) return st;
  if (n_tokens == 0 || c->record_words == 0) return SPECTRA_OK;
  if (!codes || !meta || !packed || !aligned(meta, 4) || !aligned(packed, 4))
    return fail(SPECTRA_EINVAL, "null or misaligned pack buffer");
  PackArgs a{};
  a.codes = codes;
  a.meta = meta;
  a.packed = packed;
  a.bits = c->bits;
  a.n = n_tokens;
  a.t_cap = t_capacity;
  a.W = c->record_words;
  a.n_streams = (int32_t)c->n_streams;
  hipError_t e = launch_pack_codes(a, false, (hipStream_t)stream);
  return e == hipSuccess ? SPECTRA_OK : hip_fail(e, "pack launch");
}

spectra_status spectra_unpack_codes(const spectra_codec* c, const uint32_t* packed, int64_t t_capacity, int64_t n_tokens,
                                    uint8_t* codes, uint32_t* meta, void* stream) {
  spectra_status st = check_codec(c, "unpack_codes");
  if (st != SPECTRA_OK) return st;
  st = check_slots(0, n_tokens, t_capacity);
  if (st != SPECTRA_OK) return st;
  if (n_tokens == 0) return SPECTRA_OK;
  if (!codes || !meta || !aligned(meta, 4) || (c->record_words > 0 && (!packed || !aligned(packed, 4))))
    return fail(SPECTRA_EINVAL, "null or misaligned unpack buffer");
  PackArgs a{};
  a.packed_in = packed;
  a.codes_out = codes;
  a.meta_out = meta;
  a.bits = c->bits;
  a.n = n_tokens;
  a.t_cap = t_capacity;
  a.W = c->record_words;
  a.n_streams = (int32_t)c->n_streams;
  hipError_t e = launch_pack_codes(a, true, (hipStream_t)stream);
  return e == hipSuccess ? SPECTRA_OK : hip_fail(e, "unpack launch");
}

}  // extern "C"
