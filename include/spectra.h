/*
 * spectra.h - C ABI of the SPECTRA KV-cache codec hot path for AMD MI355X (gfx950).
 *
 * The codec follows arXiv 2608.07915 (SPECTRA):
 *   Sec. 3.1  cache a latent in a spectral basis fitted from second-moment
 *             statistics (Eqs. gsvd, second-moment-latent), centered by the
 *             measured coordinate means;
 *   Sec. 3.2  quantize the latent at rate-distortion optimal group widths
 *             (Eq. waterfill, App. D) with per-token min/max, one fp16 scale
 *             and zero-point per kept group and token; zero-bit groups are
 *             dropped (rank reduction);
 *   Sec. 3.3  Mode A: reconstruct K,V from the latent; App. E Mode B:
 *             attention carried out in the latent space (q' = q V once per
 *             step, scores and value accumulation over the kept coefficients,
 *             one inverse rotation per output);
 *   App. F    effective compression ratio 16 / b_eff, metadata included.
 *
 * Terminology. A *stream* is one (sequence, layer, KV head, tensor) matrix of
 * T tokens x head_dim channels. A *codec* holds the state of a set of streams
 * of one tensor kind (keys or values): per-stream basis, mean, variances and
 * group bit widths. Streams are independent; stream index s addresses every
 * per-stream array. For attention, stream s = b * n_kv_heads + kv_head.
 *
 * Record format. Each token of each stream is stored as a record of W 32-bit
 * words (W = floor(R / 32), R the per-token bit budget including metadata):
 *   words [0, k)   one metadata word per kept group (ascending group index):
 *                  bits 0..15 = fp16 scale s, bits 16..31 = fp16 zero-point z;
 *   then, per kept group at b bits, g*b/32 payload words: in-group code j
 *                  occupies payload bits [j*b, (j+1)*b), least significant
 *                  bit first (payload bit p = bit p%32 of payload word p/32);
 *   remaining words are 0.
 * Records are stored in tiles of 64 tokens, word-major inside a tile:
 *   packed[s*T_cap*W + (t/64)*64*W + w*64 + t%64]   (T_cap % 64 == 0),
 * so a wavefront reading word w of 64 consecutive tokens reads 256 contiguous
 * bytes. The dequantized coefficient is z + s*q; dropped groups decode to 0;
 * the reconstruction is x_hat = (c_hat + m) V^T.
 *
 * Ownership and errors. The caller owns every buffer (device memory for the
 * codec arrays, inputs, outputs, packed records and workspaces); the library
 * never allocates device memory and keeps no pointer after a call returns.
 * Every argument is checked on the host before anything is launched: a
 * non-zero return means nothing ran. Returns are negative spectra_status
 * values; the text of the last error of the calling thread is available from
 * spectra_last_error(). encode / decode / decode_attention / pack / unpack
 * are asynchronous on the given stream; fit_basis synchronizes it.
 * Buffers must stay alive until the stream has passed the work. Non-finite
 * inputs give unspecified (but in-bounds) codes.
 *
 * GPU support: head_dim = 128, group_size = 32, b_max <= 8, meta_bits = 32,
 * records of at most 64 words. Per-layer geometry (Sec. 4.1, App. F: one
 * transform over a layer's whole KV vector, a stream being one (sequence, layer,
 * tensor) matrix with head_dim = d_kv = n_kv_heads x 128): head_dim a multiple
 * of 128 in [256, 1024] with group_size = 64 and records of at most 128 words,
 * for spectra_fit_basis, spectra_encode (bf16 tokens), spectra_decode and
 * spectra_layer_decode_attention; the other GPU entry points return
 * SPECTRA_EUNSUPPORTED for it.
 * The host-only functions (allocation, eigensolver, fit from moments) accept
 * any head_dim <= 1024 that group_size divides.
 */
#ifndef SPECTRA_H
#define SPECTRA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SPECTRA_OK = 0,
  SPECTRA_EINVAL = -1,       /* bad argument (null pointer, size, alignment, range) */
  SPECTRA_EUNSUPPORTED = -2, /* valid parameters the GPU path does not implement */
  SPECTRA_ENUMERIC = -3,     /* non-finite moments or eigensolver non-convergence */
  SPECTRA_EWORKSPACE = -4,   /* workspace too small */
  SPECTRA_EHIP = -5          /* a HIP runtime call failed (message in spectra_last_error) */
} spectra_status;

typedef enum { SPECTRA_F32 = 0, SPECTRA_BF16 = 1 } spectra_dtype;

/* Parameters shared by all streams of a codec. */
typedef struct {
  int32_t head_dim;    /* d (128 on the GPU; 256..1024 for the per-layer geometry) */
  int32_t group_size;  /* g: adjacent energy-ordered coefficients sharing one width (32 on the GPU; 64 per layer) */
  int32_t b_max;       /* largest code width, <= 8 */
  int32_t meta_bits;   /* bits of metadata per kept group per token: 32 (fp16 s + fp16 z) */
  int32_t centered;    /* 0: basis of the uncentered second moment (Sec. 3.1); 1: of the covariance */
  double ratio;        /* effective compression vs fp16 (App. F); R = floor(16 d / ratio + 1e-6) bits */
  int32_t budget_bits; /* > 0 overrides ratio: R bits per token per stream, metadata included */
} spectra_params;

/* Codec state. Device arrays are caller-owned; a view of a subset of streams is
 * made by offsetting the four pointers and lowering n_streams. basis must be
 * 16-byte aligned, the other arrays 4-byte aligned (EINVAL otherwise). */
typedef struct {
  spectra_params p;
  int64_t n_streams;
  int32_t record_words; /* W, set by spectra_codec_init */
  int32_t reserved;
  float* basis;         /* device [n_streams][d][d] fp32: basis[s][i][j] = channel i of direction j,
                           directions in descending second-moment energy */
  float* mean;          /* device [n_streams][d] fp32: coefficient-space mean m = mean_t(x_t) V */
  float* var;           /* device [n_streams][d] fp32: centered marginal variance of coefficient j */
  uint8_t* bits;        /* device [n_streams][d/g]: group code widths (0 = dropped) */
  float* lscale;        /* device [n_streams][d] fp32, or NULL: square-root split of the latent
                           (Eq. gsvd; per-layer geometry only). When set, the fit writes
                           f_j = max(lambda_j, lambda_0 2^-40)^(-1/4) (lambda the descending
                           eigenvalues), var holds the scaled coordinates' variances v_j f_j^2
                           and the widths are allocated on them; encode caches (x V - m)_j f_j
                           and decode reconstructs (c_hat / f + m) V^T. */
} spectra_codec;

/* Validates p, fills c->p, c->n_streams and c->record_words. Host only. */
spectra_status spectra_codec_init(spectra_codec* c, const spectra_params* p, int64_t n_streams);

/* R (bits per token per stream, metadata included) and W = floor(R/32). Host only. */
int32_t spectra_record_budget_bits(const spectra_params* p);
int32_t spectra_record_words(const spectra_params* p);

/* Asymmetric key/value split (Sec. 3.1: ranks r_k = kappa B and r_v = (1 - kappa) B;
 * kappa = 1/2 and 1/4 in App. F). The allocation turns a bit budget into a kept
 * rank, so the split is applied to the two records' combined budget 2R (R from p):
 * keys get R_k = 32 * floor(kappa * 2R / 32 + 1/2) bits, values R_v = 2R - R_k.
 * Writes copies of *p with budget_bits = R_k into *p_k and R_v into *p_v (key and
 * value codecs then have different record widths). SPECTRA_EINVAL unless
 * 0 < kappa < 1 and both budgets hold at least one group (g + meta_bits). Host only. */
spectra_status spectra_split_budget(const spectra_params* p, double kappa, spectra_params* p_k,
                                    spectra_params* p_v);

/* Number of uint32 words of a packed cache holding t_capacity tokens per stream
 * (n_streams * t_capacity * W); t_capacity must be a multiple of 64. */
int64_t spectra_packed_words(const spectra_codec* c, int64_t t_capacity);

/* ---------------------------------------------------------------------------
 * Fit (Sec. 3.1 basis, Sec. 3.2 / App. D allocation). Off the per-token path.
 * x[s*stream_stride + i*token_stride + c], i < n_tokens, c < d, dtype dt, on the
 * device. Computes per stream mu = mean x, S = mean x^T x in fp64 on the GPU,
 * then on the host the eigenbasis of S (or of the covariance if centered),
 * sorted by descending eigenvalue with each direction's largest-|.| entry
 * positive, the coefficient mean m = mu V, the centered variances and the
 * bit allocation; writes basis/mean/var/bits of the codec. Synchronizes
 * `stream`. Workspace: device, spectra_fit_workspace_bytes bytes, 256-B aligned.
 * ------------------------------------------------------------------------- */
size_t spectra_fit_workspace_bytes(const spectra_codec* c, int64_t n_tokens);
spectra_status spectra_fit_basis(spectra_codec* c, const void* x, spectra_dtype dt, int64_t n_tokens,
                                 int64_t stream_stride, int64_t token_stride, void* workspace,
                                 size_t ws_bytes, void* stream);

/* Calibrate-once fit from weights (Sec. 3.1, Eqs. gweighted and gsvd; App. B). The
 * paper whitens a projection, M = G^{1/2} W = U S V^T, and keeps the top right
 * singular directions; for k = h W these are the eigenvectors of E[k^T k] = W^T G W,
 * so the basis, coefficient means, centered variances and widths are those of a
 * stream whose second moment is W^T G W and whose mean is hbar W (no data pass).
 * Both geometries: d = 128 (one KV head's projection) or the per-layer geometry (d =
 * d_kv, the layer's KV heads side by side: W is the layer's whole key or value
 * projection, the paper's own setting), where lscale, when set, receives the
 * square-root split as in spectra_fit_basis.
 *   W     device fp32 [n_streams][d_model][d]: stream s's projection (k = h W);
 *   G     device fp64 [n_streams / streams_per_layer][d_model][d_model]: E[h^T h] of
 *         the input of stream s's layer, layer = s / streams_per_layer;
 *   hbar  device fp64 [layers][d_model]: E[h]; NULL means zero mean.
 * d_model: a multiple of 64 in [64, 16384]. The products run in fp64 on the GPU
 * (P_s = G W_s in the workspace, then W_s^T P_s); the eigensolve as in
 * spectra_fit_basis. Synchronises `stream`. Workspace: device,
 * spectra_fit_weights_workspace_bytes bytes, 256-B aligned (n_streams * (d^2 + d +
 * d_model * d) doubles). Errors as spectra_fit_basis. */
size_t spectra_fit_weights_workspace_bytes(const spectra_codec* c, int32_t d_model);
spectra_status spectra_fit_weights(spectra_codec* c, const float* W, int32_t d_model, const double* G,
                                   const double* hbar, int32_t streams_per_layer, void* workspace,
                                   size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Encode (Sec. 3.2-3.3: every new token is projected, quantized and appended).
 * Token i < n_tokens of stream s is read from x[s*stream_stride + i*token_stride + c]
 * (16-byte aligned rows: token_stride and stream_stride multiples of 8 for bf16,
 * 4 for fp32) and written to record slot t0 + i of `packed` (device, layout in the
 * file header). Slots outside [t0, t0 + n_tokens) are not touched, so appends of
 * single tokens (n_tokens = 1) never disturb earlier records. The projection
 * c = x V - m is computed to fp32 accuracy; per kept group and token:
 * z = fp16(min), s = fp16((max - z)/(2^b - 1)) (round to nearest even, saturating),
 * q = clamp(rne((c - z)/s), 0, 2^b - 1), q = 0 when s = 0. Asynchronous.
 * ------------------------------------------------------------------------- */
spectra_status spectra_encode(const spectra_codec* c, const void* x, spectra_dtype dt,
                              int64_t stream_stride, int64_t token_stride, int64_t t0, int64_t n_tokens,
                              uint32_t* packed, int64_t t_capacity, void* stream);

/* ---------------------------------------------------------------------------
 * Decode (Sec. 3.3 Mode A: K and V reconstructed from the latent). Reads record slots
 * [t0, t0 + n_tokens) of every stream and writes out[s][i][c] (fp32, contiguous,
 * device) = ((z + s q) over kept groups, 0 elsewhere, + m) V^T. Asynchronous.
 * ------------------------------------------------------------------------- */
spectra_status spectra_decode(const spectra_codec* c, const uint32_t* packed, int64_t t_capacity,
                              int64_t t0, int64_t n_tokens, float* out, void* stream);

/* ---------------------------------------------------------------------------
 * Decode-step attention over per-layer latents (App. E Mode B with the latent of
 * Sec. 3.1 spanning all KV heads of a layer; the per-layer geometry, d = n_kv_heads x
 * 128). Stream b of both codecs is sequence b < batch (record slots [0, n_tokens));
 * q[b][h][c] (device, q_dt, contiguous, 128 channels per head), query head h reads KV
 * head kv = h / (n_q_heads / n_kv_heads), whose keys and values are channels
 * [128 kv, 128 kv + 128) of the reconstructed layer vectors. out[b][h][c] (fp32) =
 * sum_t softmax_t(scale q_h . k_hat_t[kv]) v_hat_t[kv], computed as q~_h = scale q_h
 * V_K[kv rows] (a d-wide latent query), scores over the kept key coefficients (the
 * constant q~_h . m_K cancels), softmax, value sums over the kept value coefficients,
 * then (a / sum + m_V) V_V[kv rows]^T. With the square-root split (lscale set) the
 * cached coordinates are c_j f_j: q~_j is divided by the keys' f_j and the value sums
 * by the values' f_j before m_V is added. n_q_heads <= 32, records of at most 128 words.
 * softmax_scale <= 0 selects 1/sqrt(128). Workspace: device,
 * spectra_layer_attention_workspace_bytes bytes, 256-byte aligned. Asynchronous.
 * ------------------------------------------------------------------------- */
size_t spectra_layer_attention_workspace_bytes(const spectra_codec* ck, int32_t batch, int32_t n_q_heads,
                                               int64_t n_tokens);
spectra_status spectra_layer_decode_attention(const spectra_codec* ck, const spectra_codec* cv,
                                              const uint32_t* packed_k, const uint32_t* packed_v,
                                              int64_t t_capacity, int64_t n_tokens, const void* q,
                                              spectra_dtype q_dt, int32_t batch, int32_t n_q_heads,
                                              int32_t n_kv_heads, float softmax_scale, float* out,
                                              void* workspace, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Decode-step attention read straight from the packed caches (App. E, Mode B).
 * q[b][h][c] (device, dtype q_dt, contiguous), b < batch, h < n_q_heads; query head
 * h reads KV head h / (n_q_heads / n_kv_heads) through streams
 * s = b*n_kv_heads + kv of both codecs (record slots [0, n_tokens)).
 * out[b][h][c] (fp32, device) = sum_t softmax_t(scale * q_h . k_hat_t) v_hat_t,
 * computed as q' = scale q V_K once, scores over the kept key coefficients
 * (the constant q' . m_K cancels in the softmax), value accumulation over the
 * kept value coefficients, then one inverse rotation (a + m_V) V_V^T.
 * softmax_scale <= 0 selects 1/sqrt(d). n_q_heads / n_kv_heads <= 16;
 * t_capacity * record_words < 2^31 for both codecs.
 * Workspace: device, spectra_attention_workspace_bytes bytes. Asynchronous.
 * ------------------------------------------------------------------------- */
size_t spectra_attention_workspace_bytes(int32_t batch, int32_t n_q_heads, int32_t n_kv_heads,
                                         int64_t n_tokens);
spectra_status spectra_decode_attention(const spectra_codec* ck, const spectra_codec* cv,
                                        const uint32_t* packed_k, const uint32_t* packed_v,
                                        int64_t t_capacity, int64_t n_tokens, const void* q,
                                        spectra_dtype q_dt, int32_t batch, int32_t n_q_heads,
                                        int32_t n_kv_heads, float softmax_scale, float* out,
                                        void* workspace, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Decode-step attention for rotary models (Sec. 3.3, Mode A): the cached latents are
 * of pre-RoPE keys, so each key is reconstructed, k_hat_t = (c_hat_t + m_K) V_K^T, and
 * rotated at its own position t (its record slot) before the dot product with the
 * query rotated at q_position:
 *   out[b][h] = sum_t softmax_t(scale * R(q_position) q_h . R(t) k_hat_t) v_hat_t,
 * where R(p) turns each dimension pair (i, i + d/2), i < d/2, by the angle
 * p * inv_freq[i] (x_i cos - x_{i+d/2} sin, x_{i+d/2} cos + x_i sin). Values are not
 * rotated; their sums run over the kept value coefficients as in
 * spectra_decode_attention. inv_freq: device fp32 [d/2], any frequencies (base^(-2i/d)
 * or a scaled set). Angles are reduced in fp64 before fp32 cos/sin. Other arguments,
 * the workspace (spectra_attention_workspace_bytes) and the errors as
 * spectra_decode_attention; SPECTRA_EUNSUPPORTED for more than 8 query heads per KV
 * head or records wider than 32 words. Asynchronous.
 * ------------------------------------------------------------------------- */
spectra_status spectra_decode_attention_rope(const spectra_codec* ck, const spectra_codec* cv,
                                             const uint32_t* packed_k, const uint32_t* packed_v,
                                             int64_t t_capacity, int64_t n_tokens, const void* q,
                                             spectra_dtype q_dt, int32_t batch, int32_t n_q_heads,
                                             int32_t n_kv_heads, float softmax_scale, const float* inv_freq,
                                             int64_t q_position, float* out, void* workspace, size_t ws_bytes,
                                             void* stream);

/* ---------------------------------------------------------------------------
 * One decode step (Sec. 3.3: append-only latent cache, then App. E attention):
 * the new key and value of every stream, k_new[b][kv][c] and v_new[b][kv][c]
 * (device, dtype kv_dt, contiguous, 16-byte aligned), are encoded into record
 * slot t of packed_k / packed_v with the fitted state (the records equal those
 * spectra_encode writes for the same token), then attention runs over slots
 * [0, t + 1) exactly as spectra_decode_attention with n_tokens = t + 1.
 * 0 <= t < t_capacity. Workspace: spectra_attention_workspace_bytes(batch,
 * n_q_heads, n_kv_heads, t + 1) bytes. Asynchronous.
 * ------------------------------------------------------------------------- */
spectra_status spectra_decode_step(const spectra_codec* ck, const spectra_codec* cv, uint32_t* packed_k,
                                   uint32_t* packed_v, int64_t t_capacity, int64_t t, const void* k_new,
                                   const void* v_new, spectra_dtype kv_dt, const void* q, spectra_dtype q_dt,
                                   int32_t batch, int32_t n_q_heads, int32_t n_kv_heads, float softmax_scale,
                                   float* out, void* workspace, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * spectra_decode_step for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same step, with the split-K partials in a file-scope device array of
 * SPECTRA_STATIC_SCRATCH_BYTES bytes that the library holds on every GPU it runs
 * on until the process ends, instead of a workspace. Calls no hipMalloc/hipFree
 * (the array's address is looked up once per device, on its first call there).
 * Returns SPECTRA_EWORKSPACE when spectra_attention_workspace_bytes(batch,
 * n_q_heads, n_kv_heads, t + 1) exceeds the array. Every call on one GPU shares
 * that GPU's array: calls that overlap on one GPU (other streams, other threads)
 * race and must be serialised by the caller. Other arguments and errors as
 * spectra_decode_step. Asynchronous.
 * ------------------------------------------------------------------------- */
#define SPECTRA_STATIC_SCRATCH_BYTES (8u << 20)
spectra_status spectra_decode_step_static(const spectra_codec* ck, const spectra_codec* cv, uint32_t* packed_k,
                                          uint32_t* packed_v, int64_t t_capacity, int64_t t, const void* k_new,
                                          const void* v_new, spectra_dtype kv_dt, const void* q,
                                          spectra_dtype q_dt, int32_t batch, int32_t n_q_heads,
                                          int32_t n_kv_heads, float softmax_scale, float* out, void* stream);

/* ---------------------------------------------------------------------------
 * Host-side pieces of the fit, exported so they can be checked without a GPU.
 * ------------------------------------------------------------------------- */

/* Group widths for centered variances var[d] (App. D objective, Sec. 3.2
 * groups, App. F rate): the exact integer minimiser of
 * J(b) = sum_G w_G 4^(8-b_G), w_G = floor(2^39 D_G / max D), D_G = sum of the
 * group's variances (ascending, fp64), subject to
 * sum_{b_G>0} (g b_G + meta_bits) <= R, b_G in [0, b_max]; ties go to the
 * smaller cost, then to the lexicographically largest b. bits_out[d/g]. */
spectra_status spectra_allocate_bits(const double* var, const spectra_params* p, uint8_t* bits_out);

/* Symmetric eigendecomposition of a[n][n] (fp64, row-major, host): eigenvalues
 * w[n] descending, eigenvectors as columns of v[n][n] (row-major), each with its
 * largest-|.| entry (lowest index on ties) positive. n <= 1024. */
spectra_status spectra_eigh_host(const double* a, int32_t n, double* w, double* v);

/* Fit of one stream from its moments (host): gram[d][d] = sum_t x_t^T x_t,
 * colsum[d] = sum_t x_t over n_tokens tokens. Writes basis[d][d] (fp32), mean[d]
 * (fp32), var[d] (fp64) and bits[d/g]. */
spectra_status spectra_fit_from_moments_host(const spectra_params* p, int64_t n_tokens,
                                             const double* gram, const double* colsum, float* basis,
                                             float* mean, double* var, uint8_t* bits);

/* ---------------------------------------------------------------------------
 * Test hooks: the packing and unpacking device code of encode/decode driven by
 * given codes. codes[s][i][d] uint8 and meta[s][i][d/g] uint32 (device, contiguous;
 * meta word = s16 | z16 << 16 for kept groups) for record slots [0, n_tokens).
 * Asynchronous.
 * ------------------------------------------------------------------------- */
spectra_status spectra_pack_codes(const spectra_codec* c, const uint8_t* codes, const uint32_t* meta,
                                  int64_t n_tokens, uint32_t* packed, int64_t t_capacity, void* stream);
spectra_status spectra_unpack_codes(const spectra_codec* c, const uint32_t* packed, int64_t t_capacity,
                                    int64_t n_tokens, uint8_t* codes, uint32_t* meta, void* stream);

/* Status text and the calling thread's last error message. */
const char* spectra_status_string(spectra_status s);
const char* spectra_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* SPECTRA_H */
