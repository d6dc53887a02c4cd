"""GPU parity of decode-step attention read from the packed caches (App. E,
Mode B on the GPU) against the oracle's Mode A over reconstructed caches."""
import math

import numpy as np
import pytest

import oracle as O
import paper_2608_07915_amd as S
import synth
from gpu_parity import ATTN_SAME_TOL, codec_state, fit_and_encode, records_of, rel_l2, sparams, to_device, values_f64

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)


def _workload_streams(w, T, batch):
    ks, vs = [], []
    for b in range(batch):
        for h in range(w.n_kv_heads):
            ks.append(synth.numpy_stream(w, b, 0, h, 0, n_tokens=T))
            vs.append(synth.numpy_stream(w, b, 0, h, 1, n_tokens=T))
    return np.stack(ks), np.stack(vs)


def _queries(w, batch, step=0):
    return np.stack([synth.numpy_query(w, b, 0, step) for b in range(batch)])


def _fit_encode_with_bits(x_dev, p, t_cap, bits):
    """Fit, then override every stream's width table before encoding."""
    codec = S.Codec(sparams(p), x_dev.shape[0])
    S.spectra_fit_basis(codec, x_dev)
    if bits is not None:
        codec.bits.copy_(torch.tensor([bits] * x_dev.shape[0], dtype=torch.uint8))
    return fit_and_encode(x_dev, p, t_cap, fit=False, codec=codec)


def run_and_check(w, T, batch, ratio, scale=0.0, n_tokens=None, check_heads=None, p=None, bits_k=None,
                  bits_v=None, p_v=None):
    """p: key params (and value params unless p_v is given)."""
    p = O.Params(ratio=ratio) if p is None else p
    p_v = p if p_v is None else p_v
    xk, xv = _workload_streams(w, T, batch)
    t_cap = (T + 63) // 64 * 64
    ck, pk = _fit_encode_with_bits(to_device(xk, w.dtype), p, t_cap, bits_k)
    cv, pv = _fit_encode_with_bits(to_device(xv, w.dtype), p_v, t_cap, bits_v)
    q = _queries(w, batch)
    n = T if n_tokens is None else n_tokens
    out = S.spectra_decode_attention(ck, cv, pk, pv, t_cap, n, to_device(q, w.dtype), w.n_kv_heads,
                                     softmax_scale=scale).cpu().numpy()
    assert np.all(np.isfinite(out))
    sc = scale if scale > 0 else 0.0
    worst_own, worst_same = 0.0, 0.0
    for b in range(batch):
        kh_same, vh_same, kh_own, vh_own = [], [], [], []
        for h in range(w.n_kv_heads):
            s = b * w.n_kv_heads + h
            for par, codec, packed, x, same, own in ((p, ck, pk, xk, kh_same, kh_own), (p_v, cv, pv, xv, vh_same, vh_own)):
                basis, mean, bits = codec_state(codec, s)
                rec = records_of(packed, s, 0, n, t_cap, O.record_words(par))
                same.append(O.decode(rec, basis, mean, bits, par))
                rec_o, *_ = O.encode(values_f64(x[s][:n], w.dtype), basis, mean, bits, par)
                own.append(O.decode(rec_o, basis, mean, bits, par))
        q64 = values_f64(q[b], w.dtype)
        ref_same = O.attention_mode_a(q64, np.stack(kh_same), np.stack(vh_same), sc)
        ref_own = O.attention_mode_a(q64, np.stack(kh_own), np.stack(vh_own), sc)
        for h in (range(w.n_q_heads) if check_heads is None else check_heads):
            e_same = rel_l2(out[b, h], ref_same[h])
            e_own = rel_l2(out[b, h], ref_own[h])
            worst_same = max(worst_same, e_same)
            worst_own = max(worst_own, e_own)
    assert worst_same <= ATTN_SAME_TOL, worst_same
    assert worst_own <= 2e-3, worst_own
    return worst_same, worst_own


def test_attention_tiny_one_head():
    run_and_check(synth.WORKLOADS["tiny"], 4096, 1, 8.0)


def test_attention_llama_gqa4_4x_ragged():
    run_and_check(synth.WORKLOADS["llama_layer_4x"], 1000, 1, 4.0)


def test_attention_qwen_gqa7_8x():
    run_and_check(synth.WORKLOADS["qwen_layer_8x"], 1300, 1, 8.0)


def test_attention_batched_12x():
    run_and_check(synth.WORKLOADS["llama_batch16_12x"], 700, 3, 12.0)


def test_attention_prefix_of_cache_and_explicit_scale():
    # attend over the first 333 slots only, with an explicit softmax scale
    run_and_check(synth.WORKLOADS["llama_model_131k_8x"], 640, 1, 8.0, scale=0.05, n_tokens=333)


def test_attention_single_token_returns_its_value():
    w = synth.WORKLOADS["llama_layer_4x"]
    p = O.Params(ratio=4.0)
    xk, xv = _workload_streams(w, 200, 1)
    ck, pk = fit_and_encode(to_device(xk, w.dtype), p, 256)
    cv, pv = fit_and_encode(to_device(xv, w.dtype), p, 256)
    q = to_device(_queries(w, 1), w.dtype)
    out = S.spectra_decode_attention(ck, cv, pk, pv, 256, 1, q, w.n_kv_heads)
    v0 = S.spectra_decode(cv, pv, 256, 0, 1)[:, 0]          # [n_kv, d]
    want = v0.repeat_interleave(w.n_qh, dim=0)[None]
    assert rel_l2(out.cpu().numpy(), want.cpu().numpy()) <= 1e-5


def test_attention_long_context_many_chunks():
    """More tiles than one wavefront's chunk: exercises the split-K combine."""
    run_and_check(synth.WORKLOADS["llama_layer_4x"], 20000, 1, 8.0, check_heads=[0, 5, 31])


@pytest.mark.parametrize("n_qh,ratio", [(1, 8.0), (3, 12.0), (8, 4.0), (12, 8.0), (16, 8.0), (4, 16.0 / 9.0),
                                        (12, 16.0 / 9.0)])
def test_attention_gqa_widths_and_wide_records(n_qh, ratio):
    """Every head-quad count (1..4), stacked and separate weight rows, and records
    wider than 16 words (the path without register prefetch)."""
    from dataclasses import replace
    base = synth.WORKLOADS["llama_layer_4x"]
    w = replace(base, n_kv_heads=2, n_q_heads=2 * n_qh)
    run_and_check(w, 900, 1, ratio)


@pytest.mark.parametrize("bits_k,bits_v", [([0, 3, 0, 4], [2, 0, 5, 0]), ([1, 1, 1, 0], [0, 0, 0, 7]),
                                           ([0, 0, 6, 0], [0, 4, 0, 3])])
def test_attention_non_prefix_kept_groups(bits_k, bits_v):
    """Width tables that keep non-adjacent groups: slot order differs from group order."""
    from dataclasses import replace
    w = replace(synth.WORKLOADS["llama_layer_4x"], n_kv_heads=2, n_q_heads=8)
    run_and_check(w, 700, 1, 0.0, p=O.Params(budget_bits=32 * 9), bits_k=bits_k, bits_v=bits_v)


@pytest.mark.parametrize("kappa,n_qh", [(0.25, 4), (0.75, 4), (0.3, 4), (0.7, 4), (0.25, 8), (0.7, 7)])
def test_attention_asymmetric_budget_split(kappa, n_qh):
    """Key and value records of different widths from the kappa split of the 8x
    budget (Sec. 3.1, App. F): kappa = 1/4 gives 4-word keys and 12-word values,
    0.3 gives 5 and 11 words (each prefetch shape of unequal widths)."""
    from dataclasses import replace
    w = replace(synth.WORKLOADS["llama_layer_4x"], n_kv_heads=2, n_q_heads=2 * n_qh)
    pk, pv = O.split_budget(O.Params(ratio=8.0), kappa)
    assert O.record_words(pk) + O.record_words(pv) == 16
    run_and_check(w, 1500, 1, 0.0, p=pk, p_v=pv)


def test_attention_zero_query_is_value_mean():
    """q = 0: every score is 0, the softmax is uniform and the output is the mean of
    the reconstructed values (App. E with a constant score)."""
    w = synth.WORKLOADS["llama_layer_4x"]
    T = 777
    xk, xv = _workload_streams(w, T, 1)
    p = O.Params(ratio=8.0)
    t_cap = (T + 63) // 64 * 64
    ck, pk = _fit_encode_with_bits(to_device(xk, w.dtype), p, t_cap, None)
    cv, pv = _fit_encode_with_bits(to_device(xv, w.dtype), p, t_cap, None)
    q = torch.zeros(1, w.n_q_heads, 128, dtype=torch.bfloat16, device="cuda")
    out = S.spectra_decode_attention(ck, cv, pk, pv, t_cap, T, q, w.n_kv_heads).cpu().numpy()[0]
    for h in range(w.n_kv_heads):
        basis, mean, bits = codec_state(cv, h)
        vh = O.decode(records_of(pv, h, 0, T, t_cap, O.record_words(p)), basis, mean, bits, p)
        want = vh.mean(axis=0)
        for hq in range(h * w.n_qh, (h + 1) * w.n_qh):
            assert rel_l2(out[hq], want) <= ATTN_SAME_TOL, (h, hq, rel_l2(out[hq], want))


def _width_signatures(words):
    """Every tuple of kept-slot widths (1..7) whose record fits `words` words:
    sum over slots of (b + 1) <= words, up to four slots (plus the empty one)."""
    out = [[]]
    for n in range(1, 5):
        for code in range(7 ** n):
            b = [code // 7 ** k % 7 + 1 for k in range(n)]
            if sum(x + 1 for x in b) <= words:
                out.append(b)
    return out


@pytest.mark.parametrize("words,n_qh", [(8, 4), (8, 7), (5, 4), (6, 8)])
def test_attention_every_width_signature(words, n_qh):
    """One KV head per width signature of records of at most 8 words (every order of
    kept-slot widths), keys and values with different signatures and kept groups at
    seeded, not necessarily adjacent, positions."""
    from dataclasses import replace
    sigs = _width_signatures(words)
    rng = np.random.default_rng(words * 10 + n_qh)
    n_kv = len(sigs)
    w = replace(synth.WORKLOADS["llama_layer_4x"], n_kv_heads=n_kv, n_q_heads=n_kv * n_qh)
    T = 300
    p = O.Params(budget_bits=32 * words)

    def table(sig):
        bits = [0, 0, 0, 0]
        for g, b in zip(sorted(rng.choice(4, size=len(sig), replace=False)), sig):
            bits[int(g)] = b
        return bits

    bits_k = [table(sigs[i]) for i in range(n_kv)]
    bits_v = [table(sigs[(i * 7 + 3) % n_kv]) for i in range(n_kv)]
    xk, xv = _workload_streams(w, T, 1)
    t_cap = 320
    codecs = []
    for x, bits in ((xk, bits_k), (xv, bits_v)):
        codec = S.Codec(sparams(p), n_kv)
        S.spectra_fit_basis(codec, to_device(x, w.dtype))
        codec.bits.copy_(torch.tensor(bits, dtype=torch.uint8))
        codecs.append(fit_and_encode(to_device(x, w.dtype), p, t_cap, fit=False, codec=codec))
    (ck, pk), (cv, pv) = codecs
    q = _queries(w, 1)
    out = S.spectra_decode_attention(ck, cv, pk, pv, t_cap, T, to_device(q, w.dtype), n_kv).cpu().numpy()[0]
    q64 = values_f64(q[0], w.dtype)
    W = O.record_words(p)
    for h in range(n_kv):
        kb, km, kbits = codec_state(ck, h)
        vb, vm, vbits = codec_state(cv, h)
        assert kbits == bits_k[h] and vbits == bits_v[h]
        kh = O.decode(records_of(pk, h, 0, T, t_cap, W), kb, km, kbits, p)
        vh = O.decode(records_of(pv, h, 0, T, t_cap, W), vb, vm, vbits, p)
        ref = O.attention_mode_a(q64[h * n_qh:(h + 1) * n_qh], kh[None], vh[None])
        for i in range(n_qh):
            e = rel_l2(out[h * n_qh + i], ref[i])
            assert e <= ATTN_SAME_TOL, (sigs[h], sigs[(h * 7 + 3) % n_kv], i, e)
