"""GPU parity of decode-step attention for rotary models (Sec. 3.3, Mode A with
RoPE): spectra_decode_attention_rope against the oracle's attention_mode_a_rope over
the reconstructed caches, on the GPU's bytes and on the oracle's own encoding."""
import numpy as np
import pytest

import oracle as O
import paper_2608_07915_amd as S
import synth
from gpu_parity import ATTN_SAME_TOL, codec_state, fit_and_encode, records_of, rel_l2, to_device, values_f64

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)


def _inv_freq(base=500000.0, d=128):
    return (base ** (-np.arange(d // 2, dtype=np.float64) / (d // 2))).astype(np.float32)


def _streams(w, T, tensor, batch=1):
    return np.stack([synth.numpy_stream(w, b, 0, h, tensor, n_tokens=T) for b in range(batch)
                     for h in range(w.n_kv_heads)])


def run_rope(w, T, p_k, p_v, q_pos=None, inv_freq=None, batch=1, check_own=True):
    inv_freq = _inv_freq() if inv_freq is None else inv_freq
    xk, xv = _streams(w, T, 0, batch), _streams(w, T, 1, batch)
    t_cap = (T + 63) // 64 * 64
    ck, pk = fit_and_encode(to_device(xk, w.dtype), p_k, t_cap)
    cv, pv = fit_and_encode(to_device(xv, w.dtype), p_v, t_cap)
    q = np.stack([synth.numpy_query(w, b, 0, 0) for b in range(batch)])
    pos = T - 1 if q_pos is None else q_pos
    out = S.spectra_decode_attention_rope(ck, cv, pk, pv, t_cap, T, to_device(q, w.dtype), w.n_kv_heads,
                                          torch.from_numpy(inv_freq).cuda(), q_position=pos).cpu().numpy()
    assert np.all(np.isfinite(out))
    worst_same = worst_own = 0.0
    for b in range(batch):
        ks, vs, ko, vo = [], [], [], []
        for h in range(w.n_kv_heads):
            s = b * w.n_kv_heads + h
            for par, codec, packed, x, same, own in ((p_k, ck, pk, xk, ks, ko), (p_v, cv, pv, xv, vs, vo)):
                basis, mean, bits = codec_state(codec, s)
                rec = records_of(packed, s, 0, T, t_cap, O.record_words(par))
                same.append(O.decode(rec, basis, mean, bits, par))
                if check_own:
                    rec_o, *_ = O.encode(values_f64(x[s], w.dtype), basis, mean, bits, par)
                    own.append(O.decode(rec_o, basis, mean, bits, par))
        q64 = values_f64(q[b], w.dtype)
        ref = O.attention_mode_a_rope(q64, np.stack(ks), np.stack(vs), inv_freq, pos)
        worst_same = max(worst_same, max(rel_l2(out[b, h], ref[h]) for h in range(w.n_q_heads)))
        if check_own:
            ref_o = O.attention_mode_a_rope(q64, np.stack(ko), np.stack(vo), inv_freq, pos)
            worst_own = max(worst_own, max(rel_l2(out[b, h], ref_o[h]) for h in range(w.n_q_heads)))
    assert worst_same <= ATTN_SAME_TOL, worst_same
    assert worst_own <= 2e-3, worst_own
    return worst_same, worst_own


def test_rope_attention_llama_layer_8x_ragged():
    w = synth.WORKLOADS["llama_layer_4x"]
    p = O.Params(ratio=8.0)
    run_rope(w, 1500, p, p)


def test_rope_attention_query_ahead_and_fp32_tiny():
    """The query at a later position than the last key (scores depend on q_position - t),
    fp32 inputs, one KV head."""
    w = synth.WORKLOADS["tiny"]
    p = O.Params(ratio=8.0)
    run_rope(w, 1000, p, p, q_pos=4000)


def test_rope_attention_asymmetric_split_and_batch():
    from dataclasses import replace
    w = replace(synth.WORKLOADS["llama_layer_4x"], n_kv_heads=2, n_q_heads=8)
    pk, pv = O.split_budget(O.Params(ratio=8.0), 0.25)      # 4-word keys, 12-word values
    run_rope(w, 700, pk, pv, batch=2)


def test_rope_attention_large_positions():
    """Positions near 2^27: the base angles are reduced in fp64 before cos/sin."""
    from dataclasses import replace
    w = replace(synth.WORKLOADS["llama_layer_4x"], n_kv_heads=1, n_q_heads=4)
    p = O.Params(ratio=8.0)
    run_rope(w, 3000, p, p, q_pos=(1 << 27) + 12345, inv_freq=_inv_freq(10000.0), check_own=False)


def test_zero_frequencies_match_latent_attention():
    """inv_freq = 0 is attention without rotation: the Mode A kernel and the latent
    (Mode B) kernel agree on the same caches."""
    w = synth.WORKLOADS["llama_layer_4x"]
    T = 2000
    p = O.Params(ratio=8.0)
    t_cap = (T + 63) // 64 * 64
    ck, pk = fit_and_encode(to_device(_streams(w, T, 0), w.dtype), p, t_cap)
    cv, pv = fit_and_encode(to_device(_streams(w, T, 1), w.dtype), p, t_cap)
    q = to_device(synth.numpy_query(w, 0, 0, 0)[None], w.dtype)
    a = S.spectra_decode_attention_rope(ck, cv, pk, pv, t_cap, T, q, w.n_kv_heads,
                                        torch.zeros(64, dtype=torch.float32, device="cuda")).cpu().numpy()
    b = S.spectra_decode_attention(ck, cv, pk, pv, t_cap, T, q, w.n_kv_heads).cpu().numpy()
    assert max(rel_l2(a[0, h], b[0, h]) for h in range(w.n_q_heads)) <= ATTN_SAME_TOL


def test_rope_attention_qwen_gqa7_8x():
    """Qwen2.5-7B's 28:4 grouping (seven query heads per KV head: two head quads) at 8x."""
    w = synth.WORKLOADS["qwen_layer_8x"]
    p = O.Params(ratio=8.0)
    run_rope(w, 1300, p, p)


@pytest.mark.parametrize("n_qh,ratio", [(8, 2.0), (5, 16.0 / 5.0)])
def test_rope_attention_wide_records(n_qh, ratio):
    """Records wider than 16 words (32 words at 2x, 20 at 3.2x) with five to eight query
    heads per KV head."""
    from dataclasses import replace
    w = replace(synth.WORKLOADS["llama_layer_4x"], n_kv_heads=2, n_q_heads=2 * n_qh)
    p = O.Params(ratio=ratio)
    assert O.record_words(p) in (32, 20)
    run_rope(w, 900, p, p)
