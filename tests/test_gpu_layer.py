"""GPU parity of the per-layer geometry (one transform over a layer's whole KV
vector, d = n_kv_heads x 128, latent groups of 64) against the oracle, through the
C ABI: fit, encode (ragged token counts, offsets, appends) and decode (Mode A).
Comparison rules are those of the per-head path (tests/gpu_parity.py), except that
codes are judged against the forward error bound of a d-term fp32 projection."""
import numpy as np
import pytest

import oracle as O
import paper_2608_07915_amd as S
import synth
from gpu_parity import ATTN_SAME_TOL, check_encoded_stream, codec_state, records_of, rel_l2, sparams, to_device, values_f64

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)


def _layers(name, tensor, T, n_layers=1, seed=0):
    w = synth.WORKLOADS[name]
    return w, np.stack([synth.numpy_layer_stream(w, 0, l, tensor, T, seed=seed) for l in range(n_layers)])


# The fit sees at least 2 d tokens: with fewer tokens than channels the second moment
# is rank-deficient and the trailing coefficients are pure rounding noise, whose codes
# no two correct implementations need to share.
T_FIT = 2304


def _fit(x_dev, p):
    codec = S.Codec(sparams(p), x_dev.shape[0])
    S.spectra_fit_basis(codec, x_dev)
    return codec


@pytest.mark.parametrize("name,tensor", [("qwen_layer_8x", 0), ("llama_layer_4x", 1)])
def test_layer_fit_matches_oracle(name, tensor):
    w, x = _layers(name, tensor, 3000)   # 3000 tokens: ragged 16-token steps and token split
    d = x.shape[2]
    p = O.Params(head_dim=d, group_size=64, ratio=8.0)
    codec = _fit(to_device(x, w.dtype), p)
    basis, mean, bits = codec_state(codec, 0)
    f = O.fit(values_f64(x[0], w.dtype), p)
    V = basis.astype(np.float64)
    assert np.abs(V.T @ V - np.eye(d)).max() <= 1e-5
    D = V.T @ f.second_moment @ V
    assert np.abs(D - np.diag(np.diag(D))).max() <= 1e-6 * f.eigvals[0]
    assert np.allclose(np.diag(D), f.eigvals, rtol=0, atol=1e-5 * f.eigvals[0])
    gap = np.minimum(np.abs(np.diff(f.eigvals, prepend=np.inf)), np.abs(np.diff(f.eigvals, append=-np.inf)))
    clear = gap > 1e-3 * f.eigvals[0]
    cos = np.sum(V * f.basis.astype(np.float64), axis=0)
    assert np.all(cos[clear] >= 1 - 1e-6)
    assert bits == O.allocate_bits(f.var, p)
    assert np.abs(mean - f.mean).max() <= 1e-5 * np.abs(f.mean).max() + 1e-6


CASES = [
    ("qwen_layer_8x", 0, 1000, 0, 8.0),      # d = 512, several 256-token blocks, ragged tail
    ("qwen_layer_8x", 1, 777, 64, 4.0),      # offset slots
    ("llama_layer_4x", 0, 600, 0, 8.0),      # d = 1024, 64 words per record
    ("llama_layer_4x", 1, 333, 128, 12.0),
    ("qwen_layer_8x", 0, 300, 0, 2.0),       # 128-word records, most groups at 7-8 bits
]


@pytest.mark.parametrize("name,tensor,T,t0,ratio", CASES)
def test_layer_encode_decode_parity(name, tensor, T, t0, ratio):
    w, xf = _layers(name, tensor, max(T_FIT, T), n_layers=2)
    x = np.ascontiguousarray(xf[:, :T])
    d = x.shape[2]
    p = O.Params(head_dim=d, group_size=64, ratio=ratio)
    x_dev = to_device(x, w.dtype)
    codec = _fit(to_device(xf, w.dtype), p)
    W = O.record_words(p)
    t_cap = (t0 + T + 63) // 64 * 64 + 64
    packed = codec.empty_packed(t_cap)
    packed.fill_(-1)
    S.spectra_encode(codec, x_dev, t0, packed, t_cap)
    dec_gpu = S.spectra_decode(codec, packed, t_cap, t0, T).cpu().numpy()
    words = packed.cpu().numpy().view(np.uint32)
    for s in range(x.shape[0]):
        basis, mean, bits = codec_state(codec, s)
        xs = values_f64(x[s], w.dtype)
        rec = records_of(packed, s, t0, T, t_cap, W)
        check_encoded_stream(xs, basis, mean, bits, p, rec, dot_bound=True)
        dec_same = O.decode(rec, basis, mean, bits, p)
        assert rel_l2(dec_gpu[s], dec_same) <= 1e-6
        rec_o, *_ = O.encode(xs, basis, mean, bits, p)
        dec_o = O.decode(rec_o, basis, mean, bits, p)
        assert rel_l2(dec_gpu[s], dec_o) <= 1e-3
        # slots outside [t0, t0 + T) untouched
        outside = np.concatenate([np.arange(0, t0), np.arange(t0 + T, t_cap)])
        for w_ in (0, W - 1):
            assert np.all(words[O.physical_index(s, outside, w_, t_cap, W)] == 0xFFFFFFFF)


def test_layer_appends_equal_one_shot_and_dropped_groups():
    w, xf = _layers("qwen_layer_8x", 0, T_FIT)
    x = np.ascontiguousarray(xf[:, :400])
    d = x.shape[2]
    p = O.Params(head_dim=d, group_size=64, ratio=8.0)
    x_dev = to_device(x, w.dtype)
    codec = _fit(to_device(xf, w.dtype), p)
    t_cap = 448
    one = codec.empty_packed(t_cap)
    S.spectra_encode(codec, x_dev, 0, one, t_cap)
    pieces = codec.empty_packed(t_cap)
    S.spectra_encode(codec, x_dev[:, :300], 0, pieces, t_cap)
    for i in range(300, 303):
        S.spectra_encode(codec, x_dev[:, i:i + 1], i, pieces, t_cap)
    S.spectra_encode(codec, x_dev[:, 303:], 303, pieces, t_cap)
    torch.cuda.synchronize()
    assert torch.equal(one, pieces)
    # groups kept out of order and everything dropped
    ng = d // 64
    for bits in ([0, 3, 0, 5, 0, 0, 2, 0], [0] * ng):
        codec.bits.copy_(torch.tensor([bits[:ng]], dtype=torch.uint8))
        packed = codec.empty_packed(t_cap)
        packed.fill_(-1)
        S.spectra_encode(codec, x_dev, 0, packed, t_cap)
        dec = S.spectra_decode(codec, packed, t_cap, 0, 400).cpu().numpy()[0]
        basis, mean, b = codec_state(codec, 0)
        rec = records_of(packed, 0, 0, 400, t_cap, O.record_words(p))
        xs = values_f64(x[0], w.dtype)
        check_encoded_stream(xs, basis, mean, b, p, rec, dot_bound=True)
        assert rel_l2(dec, O.decode(rec, basis, mean, b, p)) <= 1e-6
        if not any(bits):
            assert np.all(rec == 0)
            want = np.tile(mean.astype(np.float64) @ basis.astype(np.float64).T, (400, 1))
            assert rel_l2(dec, want) <= 1e-6


def test_layer_rejects_what_it_does_not_run():
    w, x = _layers("qwen_layer_8x", 0, 128)
    d = x.shape[2]
    p = O.Params(head_dim=d, group_size=64, ratio=8.0)
    codec = _fit(to_device(x, w.dtype), p)
    t_cap = 128
    packed = codec.empty_packed(t_cap)
    with pytest.raises(S.SpectraError):
        S.spectra_encode(codec, torch.from_numpy(synth.bf16_bits_to_f32(x)).cuda(), 0, packed, t_cap)  # fp32 tokens
    q = torch.zeros((1, 28, d), dtype=torch.float32, device="cuda")
    with pytest.raises((S.SpectraError, ValueError)):
        S.spectra_decode_attention(codec, codec, packed, packed, t_cap, 128, q, 1)


@pytest.mark.parametrize("name,ratio", [("qwen_layer_8x", 8.0), ("llama_layer_4x", 12.0)])
def test_layer_square_root_split(name, ratio):
    # Eq. gsvd's square-root split of the latent: factors, widths, records and
    # reconstruction against the oracle's scaled codec
    w, xf = _layers(name, 1, T_FIT)
    T = 500
    x = np.ascontiguousarray(xf[:, :T])
    d = x.shape[2]
    p = O.Params(head_dim=d, group_size=64, ratio=ratio)
    codec = S.Codec(sparams(p), 1, latent_scale=True)
    S.spectra_fit_basis(codec, to_device(xf, w.dtype))
    basis, mean, bits = codec_state(codec, 0)
    f_gpu = codec.lscale[0].cpu().numpy()
    fo = O.fit(values_f64(xf[0], w.dtype), p, latent_scale=True)
    assert np.allclose(f_gpu, fo.scale, rtol=2e-5)
    assert bits == O.allocate_bits(fo.var, p)
    t_cap = 576
    packed = codec.empty_packed(t_cap)
    x_dev = to_device(x, w.dtype)
    S.spectra_encode(codec, x_dev, 0, packed, t_cap)
    dec = S.spectra_decode(codec, packed, t_cap, 0, T).cpu().numpy()[0]
    rec = records_of(packed, 0, 0, T, t_cap, O.record_words(p))
    xs = values_f64(x[0], w.dtype)
    check_encoded_stream(xs, basis, mean, bits, p, rec, dot_bound=True, scale=f_gpu)
    assert rel_l2(dec, O.decode(rec, basis, mean, bits, p, f_gpu)) <= 1e-6
    rec_o, *_ = O.encode(xs, basis, mean, bits, p, f_gpu)
    assert rel_l2(dec, O.decode(rec_o, basis, mean, bits, p, f_gpu)) <= 1e-3
    # the per-head geometry refuses the split
    ph = O.Params(ratio=8.0)
    with pytest.raises(S.SpectraError):
        ch = S.Codec(sparams(ph), 1, latent_scale=True)
        S.spectra_fit_basis(ch, to_device(np.ascontiguousarray(x[:, :, :128]), w.dtype))


def _oracle_layer_attention(q64, kh, vh, n_kv):
    """Mode A over reconstructed layer vectors: kh, vh [T, n_kv * 128] -> heads of 128."""
    T = kh.shape[0]
    k = kh.reshape(T, n_kv, 128).transpose(1, 0, 2)
    v = vh.reshape(T, n_kv, 128).transpose(1, 0, 2)
    return O.attention_mode_a(q64, k, v)


@pytest.mark.parametrize("name,T,ratio,batch", [("qwen_layer_8x", 1000, 8.0, 1), ("llama_layer_4x", 777, 8.0, 2),
                                                 ("qwen_layer_8x", 300, 16.0, 2), ("qwen_layer_8x", 2500, 8.0, 1),
                                                 # 1024-wide latent at 4x: 128-word records, the score pass
                                                 # split over the two blocks of 16 query heads
                                                 ("llama_layer_4x", 600, 4.0, 1)])
def test_layer_decode_attention(name, T, ratio, batch):
    # Mode B over the per-layer latent against Mode A over the oracle's reconstruction of
    # the same bytes (arithmetic only) and of the oracle's own encoding
    w = synth.WORKLOADS[name]
    xk = np.stack([synth.numpy_layer_stream(w, b, 0, 0, max(T_FIT, T)) for b in range(batch)])
    xv = np.stack([synth.numpy_layer_stream(w, b, 0, 1, max(T_FIT, T)) for b in range(batch)])
    d = xk.shape[2]
    n_kv = d // 128
    p = O.Params(head_dim=d, group_size=64, ratio=ratio)
    ck, cv = S.Codec(sparams(p), batch), S.Codec(sparams(p), batch)
    S.spectra_fit_basis(ck, to_device(xk, w.dtype))
    S.spectra_fit_basis(cv, to_device(xv, w.dtype))
    t_cap = (T + 63) // 64 * 64 + 64
    pk, pv = ck.empty_packed(t_cap), cv.empty_packed(t_cap)
    pk.fill_(-1)  # slots past the tokens hold NaN metadata: they must not reach the output
    pv.fill_(-1)
    S.spectra_encode(ck, to_device(np.ascontiguousarray(xk[:, :T]), w.dtype), 0, pk, t_cap)
    S.spectra_encode(cv, to_device(np.ascontiguousarray(xv[:, :T]), w.dtype), 0, pv, t_cap)
    qs = np.stack([synth.numpy_query(w, b, 0, 0) for b in range(batch)])   # [batch, n_q_heads, 128]
    out = S.spectra_layer_decode_attention(ck, cv, pk, pv, t_cap, T, to_device(qs, w.dtype), n_kv).cpu().numpy()
    W = O.record_words(p)
    for b in range(batch):
        q64 = values_f64(qs[b], w.dtype)
        kb, km, kbits = codec_state(ck, b)
        vb, vm, vbits = codec_state(cv, b)
        rk, rv = records_of(pk, b, 0, T, t_cap, W), records_of(pv, b, 0, T, t_cap, W)
        ref = _oracle_layer_attention(q64, O.decode(rk, kb, km, kbits, p), O.decode(rv, vb, vm, vbits, p), n_kv)
        for h in range(q64.shape[0]):
            assert rel_l2(out[b, h], ref[h]) <= ATTN_SAME_TOL, (b, h, rel_l2(out[b, h], ref[h]))
        rko, *_ = O.encode(values_f64(xk[b, :T], w.dtype), kb, km, kbits, p)
        rvo, *_ = O.encode(values_f64(xv[b, :T], w.dtype), vb, vm, vbits, p)
        ref_o = _oracle_layer_attention(q64, O.decode(rko, kb, km, kbits, p), O.decode(rvo, vb, vm, vbits, p), n_kv)
        for h in range(q64.shape[0]):
            assert rel_l2(out[b, h], ref_o[h]) <= 2e-3


def test_layer_attention_three_heads_d384():
    # a latent width that is not a multiple of 256 (three KV heads side by side)
    w = synth.WORKLOADS["qwen_layer_8x"]
    T = 700
    xk = np.ascontiguousarray(synth.numpy_layer_stream(w, 0, 0, 0, T_FIT)[None, :, :384])
    xv = np.ascontiguousarray(synth.numpy_layer_stream(w, 0, 0, 1, T_FIT)[None, :, :384])
    p = O.Params(head_dim=384, group_size=64, ratio=8.0)
    ck, cv = S.Codec(sparams(p), 1), S.Codec(sparams(p), 1)
    S.spectra_fit_basis(ck, to_device(xk, w.dtype))
    S.spectra_fit_basis(cv, to_device(xv, w.dtype))
    t_cap = 768
    pk, pv = ck.empty_packed(t_cap), cv.empty_packed(t_cap)
    S.spectra_encode(ck, to_device(np.ascontiguousarray(xk[:, :T]), w.dtype), 0, pk, t_cap)
    S.spectra_encode(cv, to_device(np.ascontiguousarray(xv[:, :T]), w.dtype), 0, pv, t_cap)
    qs = np.ascontiguousarray(synth.numpy_query(w, 0, 0, 0)[None, :24])
    out = S.spectra_layer_decode_attention(ck, cv, pk, pv, t_cap, T, to_device(qs, w.dtype), 3).cpu().numpy()
    W = O.record_words(p)
    kb, km, kbits = codec_state(ck, 0)
    vb, vm, vbits = codec_state(cv, 0)
    ref = _oracle_layer_attention(values_f64(qs[0], w.dtype),
                                  O.decode(records_of(pk, 0, 0, T, t_cap, W), kb, km, kbits, p),
                                  O.decode(records_of(pv, 0, 0, T, t_cap, W), vb, vm, vbits, p), 3)
    for h in range(24):
        assert rel_l2(out[0, h], ref[h]) <= ATTN_SAME_TOL, (h, rel_l2(out[0, h], ref[h]))


def test_layer_attention_fp32_queries_and_softmax_scale():
    # fp32 queries and an explicit softmax scale take the same path as bf16 ones
    w = synth.WORKLOADS["qwen_layer_8x"]
    T = 640
    xk = synth.numpy_layer_stream(w, 0, 0, 0, T_FIT)[None]
    xv = synth.numpy_layer_stream(w, 0, 0, 1, T_FIT)[None]
    d = xk.shape[2]
    n_kv = d // 128
    p = O.Params(head_dim=d, group_size=64, ratio=8.0)
    ck, cv = S.Codec(sparams(p), 1), S.Codec(sparams(p), 1)
    S.spectra_fit_basis(ck, to_device(xk, w.dtype))
    S.spectra_fit_basis(cv, to_device(xv, w.dtype))
    t_cap = 704
    pk, pv = ck.empty_packed(t_cap), cv.empty_packed(t_cap)
    S.spectra_encode(ck, to_device(np.ascontiguousarray(xk[:, :T]), w.dtype), 0, pk, t_cap)
    S.spectra_encode(cv, to_device(np.ascontiguousarray(xv[:, :T]), w.dtype), 0, pv, t_cap)
    rng = np.random.default_rng(9)
    q32 = rng.standard_normal((1, w.n_q_heads, 128)).astype(np.float32) * 2.0
    scale = 0.05
    out = S.spectra_layer_decode_attention(ck, cv, pk, pv, t_cap, T, torch.from_numpy(q32).cuda(), n_kv,
                                           softmax_scale=scale).cpu().numpy()
    W = O.record_words(p)
    kb, km, kbits = codec_state(ck, 0)
    vb, vm, vbits = codec_state(cv, 0)
    kh = O.decode(records_of(pk, 0, 0, T, t_cap, W), kb, km, kbits, p)
    vh = O.decode(records_of(pv, 0, 0, T, t_cap, W), vb, vm, vbits, p)
    k = kh.reshape(T, n_kv, 128).transpose(1, 0, 2)
    v = vh.reshape(T, n_kv, 128).transpose(1, 0, 2)
    ref = O.attention_mode_a(q32[0].astype(np.float64), k, v, scale)
    for h in range(w.n_q_heads):
        assert rel_l2(out[0, h], ref[h]) <= ATTN_SAME_TOL, (h, rel_l2(out[0, h], ref[h]))


@pytest.mark.parametrize("T", [1, 65])
def test_layer_attention_tiny_caches(T):
    # one token (the softmax is 1: the output is that token's reconstructed value) and a
    # ragged second tile
    w = synth.WORKLOADS["qwen_layer_8x"]
    xk = synth.numpy_layer_stream(w, 0, 0, 0, T_FIT)[None]
    xv = synth.numpy_layer_stream(w, 0, 0, 1, T_FIT)[None]
    d = xk.shape[2]
    n_kv = d // 128
    p = O.Params(head_dim=d, group_size=64, ratio=8.0)
    ck, cv = S.Codec(sparams(p), 1), S.Codec(sparams(p), 1)
    S.spectra_fit_basis(ck, to_device(xk, w.dtype))
    S.spectra_fit_basis(cv, to_device(xv, w.dtype))
    t_cap = 128
    pk, pv = ck.empty_packed(t_cap), cv.empty_packed(t_cap)
    pk.fill_(-1)  # slots past the tokens hold NaN metadata: they must not reach the output
    pv.fill_(-1)
    S.spectra_encode(ck, to_device(np.ascontiguousarray(xk[:, :T]), w.dtype), 0, pk, t_cap)
    S.spectra_encode(cv, to_device(np.ascontiguousarray(xv[:, :T]), w.dtype), 0, pv, t_cap)
    qs = synth.numpy_query(w, 0, 0, 0)[None]
    out = S.spectra_layer_decode_attention(ck, cv, pk, pv, t_cap, T, to_device(qs, w.dtype), n_kv).cpu().numpy()
    W = O.record_words(p)
    kb, km, kbits = codec_state(ck, 0)
    vb, vm, vbits = codec_state(cv, 0)
    vh = O.decode(records_of(pv, 0, 0, T, t_cap, W), vb, vm, vbits, p)
    ref = _oracle_layer_attention(values_f64(qs[0], w.dtype),
                                  O.decode(records_of(pk, 0, 0, T, t_cap, W), kb, km, kbits, p), vh, n_kv)
    for h in range(w.n_q_heads):
        assert rel_l2(out[0, h], ref[h]) <= ATTN_SAME_TOL, (h, rel_l2(out[0, h], ref[h]))
    if T == 1:
        kvh = np.arange(w.n_q_heads) // (w.n_q_heads // n_kv)
        want = vh[0].reshape(n_kv, 128)[kvh]
        assert rel_l2(out[0], want) <= 1e-5


@pytest.mark.parametrize("name,T", [("qwen_layer_8x", 900), ("llama_layer_4x", 333)])
def test_layer_decode_attention_square_root_split(name, T):
    """Both latents cached with Eq. gsvd's square-root split (lscale): the attention over
    the scaled records equals Mode A over the oracle's reconstruction of the same bytes."""
    w = synth.WORKLOADS[name]
    xk = synth.numpy_layer_stream(w, 0, 0, 0, max(T_FIT, T))[None]
    xv = synth.numpy_layer_stream(w, 0, 0, 1, max(T_FIT, T))[None]
    d = xk.shape[2]
    n_kv = d // 128
    p = O.Params(head_dim=d, group_size=64, ratio=8.0)
    ck = S.Codec(sparams(p), 1, latent_scale=True)
    cv = S.Codec(sparams(p), 1, latent_scale=True)
    S.spectra_fit_basis(ck, to_device(xk, w.dtype))
    S.spectra_fit_basis(cv, to_device(xv, w.dtype))
    t_cap = (T + 63) // 64 * 64
    pk, pv = ck.empty_packed(t_cap), cv.empty_packed(t_cap)
    pk.fill_(-1)
    pv.fill_(-1)
    S.spectra_encode(ck, to_device(np.ascontiguousarray(xk[:, :T]), w.dtype), 0, pk, t_cap)
    S.spectra_encode(cv, to_device(np.ascontiguousarray(xv[:, :T]), w.dtype), 0, pv, t_cap)
    qs = synth.numpy_query(w, 0, 0, 0)[None]
    out = S.spectra_layer_decode_attention(ck, cv, pk, pv, t_cap, T, to_device(qs, w.dtype), n_kv).cpu().numpy()
    W = O.record_words(p)
    kb, km, kbits = codec_state(ck, 0)
    vb, vm, vbits = codec_state(cv, 0)
    fk, fv = ck.lscale[0].cpu().numpy(), cv.lscale[0].cpu().numpy()
    kh = O.decode(records_of(pk, 0, 0, T, t_cap, W), kb, km, kbits, p, fk)
    vh = O.decode(records_of(pv, 0, 0, T, t_cap, W), vb, vm, vbits, p, fv)
    ref = _oracle_layer_attention(values_f64(qs[0], w.dtype), kh, vh, n_kv)
    for h in range(w.n_q_heads):
        assert rel_l2(out[0, h], ref[h]) <= ATTN_SAME_TOL, (h, rel_l2(out[0, h], ref[h]))
