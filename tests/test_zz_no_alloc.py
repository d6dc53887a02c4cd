"""spectra_decode_step_static (the decode step with its partials in the library's
static device array, for callers that cannot allocate) against spectra_decode_step
with a caller workspace: records and outputs identical, on two calls in a row, the
second with a smaller input (fewer sequences and tokens), and the outputs within
the attention bar of the oracle over the same bytes."""
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


def _streams(w, T, batch, tensor):
    return np.stack([synth.numpy_stream(w, b, 0, h, tensor, n_tokens=T) for b in range(batch)
                     for h in range(w.n_kv_heads)])


def _step_pair(w, batch, T0, p):
    """One decode step at slot T0 through both entry points on copies of one cache."""
    H = w.n_kv_heads
    t_cap = (T0 + 1 + 63) // 64 * 64
    xk, xv = _streams(w, T0 + 1, batch, 0), _streams(w, T0 + 1, batch, 1)
    dk, dv = to_device(xk, w.dtype), to_device(xv, w.dtype)
    ck, pk = fit_and_encode(dk[:, :T0].contiguous(), p, t_cap)
    cv, pv = fit_and_encode(dv[:, :T0].contiguous(), p, t_cap)
    pk2, pv2 = pk.clone(), pv.clone()
    q = to_device(np.stack([synth.numpy_query(w, b, 0, 0) for b in range(batch)]), w.dtype)
    k_new = dk[:, T0].reshape(batch, H, 128).contiguous()
    v_new = dv[:, T0].reshape(batch, H, 128).contiguous()
    want = S.spectra_decode_step(ck, cv, pk, pv, t_cap, T0, k_new, v_new, q, H)
    got = S.spectra_decode_step_static(ck, cv, pk2, pv2, t_cap, T0, k_new, v_new, q, H)
    torch.cuda.synchronize()
    assert torch.equal(pk, pk2) and torch.equal(pv, pv2)
    assert torch.equal(got, want)
    # the bar of the attention parity tests: oracle Mode A over the same bytes
    W = O.record_words(p)
    out = got.cpu().numpy()
    for b in range(batch):
        kh, vh = [], []
        for h in range(H):
            s = b * H + h
            for codec, packed, dst in ((ck, pk2, kh), (cv, pv2, vh)):
                basis, mean, bits = codec_state(codec, s)
                dst.append(O.decode(records_of(packed, s, 0, T0 + 1, t_cap, W), basis, mean, bits, p))
        ref = O.attention_mode_a(values_f64(q[b].cpu().view(torch.int16).numpy().view(np.uint16), w.dtype),
                                 np.stack(kh), np.stack(vh))
        for hq in range(w.n_q_heads):
            assert rel_l2(out[b, hq], ref[hq]) <= ATTN_SAME_TOL, (b, hq)


def test_static_decode_step_equals_workspace_decode_step_twice():
    w = synth.WORKLOADS["llama_layer_4x"]
    p = O.Params(ratio=8.0)
    _step_pair(w, 2, 1500, p)   # a larger call first: the array keeps its partials
    _step_pair(w, 1, 300, p)    # then a smaller one (fewer sequences, tokens and chunks)
