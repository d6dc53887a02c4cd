"""spectra_decode_step (append the new key/value, then attend) against the two
separate calls it replaces: spectra_encode of the new token into slot t, then
spectra_decode_attention over t + 1 tokens. Records must be byte-identical and
outputs identical; both are checked against the oracle by the encode and
attention parity tests."""
import numpy as np
import pytest

import oracle as O
import paper_2608_07915_amd as S
import synth
from gpu_parity import fit_and_encode, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)


def _streams(w, T, batch, tensor):
    return np.stack([synth.numpy_stream(w, b, 0, h, tensor, n_tokens=T) for b in range(batch)
                     for h in range(w.n_kv_heads)])


@pytest.mark.parametrize("name,T0,batch,ratio,kappa", [("llama_layer_4x", 61, 2, 8.0, 0.5), ("tiny", 127, 1, 8.0, 0.5),
                                                       ("qwen_layer_8x", 700, 1, 12.0, 0.5),
                                                       ("llama_layer_4x", 500, 1, 16 / 9, 0.5),
                                                       ("llama_layer_4x", 61, 1, 8.0, 0.25),
                                                       ("qwen_layer_8x", 190, 1, 4.0, 0.7)])
def test_decode_step_equals_encode_then_attention(name, T0, batch, ratio, kappa):
    """kappa != 1/2: key and value records of different widths (asymmetric split)."""
    w = synth.WORKLOADS[name]
    n_steps = 5                                   # crosses a 64-token tile boundary for T0 = 61 / 127
    T = T0 + n_steps
    t_cap = (T + 63) // 64 * 64
    xk, xv = _streams(w, T, batch, 0), _streams(w, T, batch, 1)
    dk, dv = to_device(xk, w.dtype), to_device(xv, w.dtype)
    p_k = p_v = O.Params(ratio=ratio)
    if kappa != 0.5:
        p_k, p_v = O.split_budget(p_k, kappa)
    ck, pk = fit_and_encode(dk[:, :T0].contiguous(), p_k, t_cap)
    cv, pv = fit_and_encode(dv[:, :T0].contiguous(), p_v, t_cap)
    pk2, pv2 = pk.clone(), pv.clone()
    H, Hq = w.n_kv_heads, w.n_q_heads
    for i in range(n_steps):
        t = T0 + i
        q = to_device(np.stack([synth.numpy_query(w, b, 0, i) for b in range(batch)]), w.dtype)
        # separate calls
        S.spectra_encode(ck, dk[:, t:t + 1], t, pk, t_cap)
        S.spectra_encode(cv, dv[:, t:t + 1], t, pv, t_cap)
        want = S.spectra_decode_attention(ck, cv, pk, pv, t_cap, t + 1, q, H)
        # fused
        k_new = dk[:, t].reshape(batch, H, 128).contiguous()
        v_new = dv[:, t].reshape(batch, H, 128).contiguous()
        got = S.spectra_decode_step(ck, cv, pk2, pv2, t_cap, t, k_new, v_new, q, H)
        torch.cuda.synchronize()
        assert torch.equal(pk, pk2), (name, t)
        assert torch.equal(pv, pv2), (name, t)
        assert torch.equal(got, want), (name, t)
        assert got.shape == (batch, Hq, 128)
