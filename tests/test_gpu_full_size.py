"""Parity at the benchmark's full size and launch configuration: one layer of the
Llama-3.1-8B 131k-token cache at 8x (8 KV heads, 32 query heads, 131072 bf16
prefill tokens), fitted and encoded as the benchmark does, then two decode
steps of spectra_decode_step. Sampled against the oracle: the records of two
KV heads (K and V streams, every token, including the appended ones) and the
attention outputs of their eight query heads, over the GPU's bytes and over the
oracle's own encoding (App. E, Mode A). Also at that size: the per-layer geometry
(1024-wide latents) and attention with rotary embeddings, as the benchmark runs them."""
import numpy as np
import pytest

import oracle as O
import paper_2608_07915_amd as S
import synth
from gpu_parity import (ATTN_SAME_TOL, check_encoded_stream, codec_state, host_values, records_of, rel_l2, sparams, to_device,
                         values_f64)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)


def test_full_size_layer_two_decode_steps_sampled():
    w = synth.WORKLOADS["llama_model_131k_8x"]
    dev = torch.device("cuda:0")
    layer, n_dec = 0, 2
    H, Hq, T = w.n_kv_heads, w.n_q_heads, w.n_tokens
    nqh = Hq // H
    t_cap = (T + n_dec + 63) // 64 * 64
    p = O.Params(ratio=w.ratio)
    xk = synth.device_streams(w, 0, layer, T + n_dec, dev)
    xv = synth.device_streams(w, 1, layer, T + n_dec, dev)
    ck, cv = S.Codec(sparams(p), H), S.Codec(sparams(p), H)
    S.spectra_fit_basis(ck, xk, n_tokens=T)
    S.spectra_fit_basis(cv, xv, n_tokens=T)
    pk, pv = ck.empty_packed(t_cap), cv.empty_packed(t_cap)
    S.spectra_encode(ck, xk, 0, pk, t_cap, n_tokens=T)
    S.spectra_encode(cv, xv, 0, pv, t_cap, n_tokens=T)
    ws = torch.empty(S.spectra_attention_workspace_bytes(1, Hq, H, t_cap), dtype=torch.uint8, device=dev)
    out = None
    q = None
    for i in range(n_dec):
        t = T + i
        q = synth.device_queries(w, layer, i, dev)                       # [1, Hq, 128]
        out = S.spectra_decode_step(ck, cv, pk, pv, t_cap, t, xk[:, t].reshape(1, H, 128).contiguous(),
                                    xv[:, t].reshape(1, H, 128).contiguous(), q, H, workspace=ws)
    torch.cuda.synchronize()
    n = T + n_dec
    out = out.cpu().numpy()
    q64 = host_values(q)[0]
    for kv in (0, H - 1):
        dec_same, dec_own = [], []
        for codec, packed, x in ((ck, pk, xk), (cv, pv, xv)):
            basis, mean, bits = codec_state(codec, kv)
            xs = host_values(x[kv, :n])
            rec = records_of(packed, kv, 0, n, t_cap, codec.record_words)
            check_encoded_stream(xs, basis, mean, bits, p, rec)       # every token, appended ones included
            dec_same.append(O.decode(rec, basis, mean, bits, p))
            rec_o, *_ = O.encode(xs, basis, mean, bits, p)
            dec_own.append(O.decode(rec_o, basis, mean, bits, p))
        heads = range(kv * nqh, (kv + 1) * nqh)
        qh = q64[kv * nqh:(kv + 1) * nqh]
        ref_same = O.attention_mode_a(qh, dec_same[0][None], dec_same[1][None], 0.0)
        ref_own = O.attention_mode_a(qh, dec_own[0][None], dec_own[1][None], 0.0)
        for i, h in enumerate(heads):
            assert rel_l2(out[0, h], ref_same[i]) <= ATTN_SAME_TOL, (kv, h, rel_l2(out[0, h], ref_same[i]))
            assert rel_l2(out[0, h], ref_own[i]) <= 2e-3, (kv, h)


def _gather_records(packed, t, t_cap, W):
    """Logical records [len(t), W] of stream 0 gathered on the device."""
    idx = np.stack([O.physical_index(0, t, k, t_cap, W) for k in range(W)], axis=1)
    got = packed[torch.from_numpy(idx.reshape(-1)).to(packed.device)].cpu().numpy().view(np.uint32)
    return got.reshape(len(t), W)


def test_largest_capacity_offsets():
    """Record offsets at the largest capacity the attention accepts: t_capacity x W just
    below 2^31 words per stream (W = 8, 2^28 - 64 slots, 8.6 GB per packed stream).
    Tokens are encoded at both ends of the range; the slots between hold zero records,
    which decode to the stream mean (z = s = 0). Attention over every slot is checked
    by a property that holds at any size: the n0 identical zero-record tokens enter
    the softmax as one term of multiplicity n0 (Mode A, App. E)."""
    w = synth.WORKLOADS["llama_layer_4x"]
    dev = torch.device("cuda:0")
    p = O.Params(ratio=8.0)
    W = O.record_words(p)
    t_cap = (1 << 28) - 64
    assert t_cap * W < (1 << 31)
    n_end = 1000
    xk = synth.numpy_stream(w, 0, 0, 0, 0, n_tokens=2 * n_end)[None]
    xv = synth.numpy_stream(w, 0, 0, 0, 1, n_tokens=2 * n_end)[None]
    ck, cv = S.Codec(sparams(p), 1), S.Codec(sparams(p), 1)
    dk, dv = to_device(xk, w.dtype), to_device(xv, w.dtype)
    S.spectra_fit_basis(ck, dk)
    S.spectra_fit_basis(cv, dv)
    pk, pv = ck.empty_packed(t_cap), cv.empty_packed(t_cap)
    for codec, packed, x in ((ck, pk, dk), (cv, pv, dv)):
        S.spectra_encode(codec, x[:, :n_end].contiguous(), 0, packed, t_cap)
        S.spectra_encode(codec, x[:, n_end:].contiguous(), t_cap - n_end, packed, t_cap)
    q = synth.device_queries(w, 0, 0, dev)[:, :w.n_qh].contiguous()    # the 4 query heads of KV head 0
    print("largest capacity: t_cap", t_cap, flush=True)
    out = S.spectra_decode_attention(ck, cv, pk, pv, t_cap, t_cap, q, 1).cpu().numpy()[0]
    torch.cuda.synchronize()
    dec = []
    for codec, packed, x in ((ck, pk, xk), (cv, pv, xv)):
        basis, mean, bits = codec_state(codec, 0)
        xs = values_f64(x[0], w.dtype)
        ends = np.concatenate([np.arange(n_end), np.arange(t_cap - n_end, t_cap)])
        rec = _gather_records(packed, ends, t_cap, W)          # device gather: the caches are 8.6 GB
        check_encoded_stream(xs, basis, mean, bits, p, rec)
        zero = O.decode(np.zeros((1, W), dtype=np.uint32), basis, mean, bits, p)[0]
        assert not _gather_records(packed, np.arange(t_cap // 2, t_cap // 2 + 64), t_cap, W).any()
        dec.append((O.decode(rec, basis, mean, bits, p), zero))
    (kh, k0), (vh, v0) = dec
    n0 = t_cap - 2 * n_end
    q64 = host_values(q)[0]
    scale = 1.0 / np.sqrt(128.0)
    for h in range(w.n_qh):
        s_end = scale * (kh @ q64[h])
        s_0 = scale * float(k0 @ q64[h])
        m = max(s_end.max(), s_0)
        e_end = np.exp(s_end - m)
        e_0 = n0 * np.exp(s_0 - m)
        want = (e_end @ vh + e_0 * v0) / (e_end.sum() + e_0)
        # fp32 running sums over ~1400 tiles per lane: rounding up to ~1400 * 2^-24 relative
        assert rel_l2(out[h], want) <= 2e-4, h


def test_full_size_per_layer_latent_sampled():
    # the per-layer geometry at the benchmark's size, as the bench runs it: one Llama layer's
    # keys and values as 1024-wide streams (131104 tokens), fitted on the first 8192 tokens,
    # encoded, decoded and attended by the 32 query heads; checked against the oracle on a
    # sample of tokens (records, reconstruction) and in full for the attention outputs
    w = synth.WORKLOADS["llama_model_131k_8x"]
    dev = torch.device("cuda:0")
    H, Hq = w.n_kv_heads, w.n_q_heads
    n = w.n_tokens + w.n_append
    t_cap = (n + 63) // 64 * 64
    d = H * 128
    p = O.Params(head_dim=d, group_size=64, ratio=w.ratio)
    xs_dev, codecs, packs = [], [], []
    for tensor in (0, 1):
        x = synth.device_layer_stream(w, 0, 0, tensor, n, dev)
        c = S.Codec(sparams(p), 1)
        S.spectra_fit_basis(c, x[:, :8192])
        pk = c.empty_packed(t_cap)
        S.spectra_encode(c, x, 0, pk, t_cap)
        xs_dev.append(x)
        codecs.append(c)
        packs.append(pk)
    q = synth.device_queries(w, 0, 0, dev)                                 # [1, Hq, 128]
    out = S.spectra_layer_decode_attention(codecs[0], codecs[1], packs[0], packs[1], t_cap, n, q, H).cpu().numpy()
    rng = np.random.default_rng(4)
    sample = np.sort(rng.choice(n, size=1500, replace=False))
    sample[-1] = n - 1
    dec_full = []
    for c, pk, x in zip(codecs, packs, xs_dev):
        basis, mean, bits = codec_state(c, 0)
        W = c.record_words
        words = pk.cpu().numpy().view(np.uint32)
        rec = np.stack([words[O.physical_index(0, np.arange(n), w_, t_cap, W)] for w_ in range(W)], axis=1)
        xs = host_values(x[0, sample])
        check_encoded_stream(xs, basis, mean, bits, p, rec[sample], dot_bound=True)
        dec = S.spectra_decode(c, pk, t_cap, 0, n).cpu().numpy()[0]
        dec_o = O.decode(rec, basis, mean, bits, p)
        assert rel_l2(dec[sample], dec_o[sample]) <= 1e-6
        dec_full.append(dec_o)
    q64 = host_values(q)[0]
    k = dec_full[0].reshape(n, H, 128).transpose(1, 0, 2)
    v = dec_full[1].reshape(n, H, 128).transpose(1, 0, 2)
    ref = O.attention_mode_a(q64, k, v)
    for h in range(Hq):
        assert rel_l2(out[0, h], ref[h]) <= ATTN_SAME_TOL, (h, rel_l2(out[0, h], ref[h]))


def test_full_size_rope_attention():
    # Mode A with RoPE at the benchmark's size and launch shape (one layer, 8 KV heads, 32
    # query heads, 131104 slots, rope base 500000): every output against the oracle's
    # rotary attention over the reconstruction of the GPU's bytes
    w = synth.WORKLOADS["llama_model_131k_8x"]
    dev = torch.device("cuda:0")
    H, Hq = w.n_kv_heads, w.n_q_heads
    n = w.n_tokens + w.n_append
    t_cap = (n + 63) // 64 * 64
    p = O.Params(ratio=w.ratio)
    inv_freq = (500000.0 ** (-np.arange(64, dtype=np.float64) / 64)).astype(np.float32)
    codecs, packs = [], []
    for tensor in (0, 1):
        x = synth.device_streams(w, tensor, 0, n, dev)
        c = S.Codec(sparams(p), H)
        S.spectra_fit_basis(c, x)
        pk = c.empty_packed(t_cap)
        S.spectra_encode(c, x, 0, pk, t_cap)
        codecs.append(c)
        packs.append(pk)
        del x
    q = synth.device_queries(w, 0, 0, dev)
    out = S.spectra_decode_attention_rope(codecs[0], codecs[1], packs[0], packs[1], t_cap, n, q, H,
                                          torch.from_numpy(inv_freq).to(dev)).cpu().numpy()
    hats = []
    for c, pk in zip(codecs, packs):
        rows = []
        for s in range(H):
            basis, mean, bits = codec_state(c, s)
            rows.append(O.decode(records_of(pk, s, 0, n, t_cap, c.record_words), basis, mean, bits, p))
        hats.append(np.stack(rows))
    ref = O.attention_mode_a_rope(host_values(q)[0], hats[0], hats[1], inv_freq, n - 1)
    for h in range(Hq):
        assert rel_l2(out[0, h], ref[h]) <= ATTN_SAME_TOL, (h, rel_l2(out[0, h], ref[h]))
