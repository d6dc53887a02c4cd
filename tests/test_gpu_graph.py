"""Appends and decode-step attention captured in a HIP graph give, on every
replay, exactly the records and outputs of the same calls launched eagerly.
(No memset nodes: the library clears nothing with hipMemsetAsync.)"""
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


def test_graph_replays_match_eager():
    w = synth.WORKLOADS["llama_layer_4x"]
    T, n_app, t_cap = 2000, 3, 2048
    xk = np.stack([synth.numpy_stream(w, 0, 0, h, 0, n_tokens=T + n_app) for h in range(w.n_kv_heads)])
    xv = np.stack([synth.numpy_stream(w, 0, 0, h, 1, n_tokens=T + n_app) for h in range(w.n_kv_heads)])
    p = O.Params(ratio=8.0)
    dk, dv = to_device(xk, w.dtype), to_device(xv, w.dtype)
    ck, pk = fit_and_encode(dk[:, :T].contiguous(), p, t_cap)
    cv, pv = fit_and_encode(dv[:, :T].contiguous(), p, t_cap)
    q = to_device(np.stack([synth.numpy_query(w, 0, 0, 0)]), w.dtype)
    H = w.n_kv_heads
    ws = torch.empty(S.spectra_attention_workspace_bytes(1, w.n_q_heads, H, t_cap), dtype=torch.uint8,
                     device=q.device)
    out = torch.empty((1, w.n_q_heads, 128), dtype=torch.float32, device=q.device)

    def work():
        for i in range(n_app):
            t = T + i
            S.spectra_encode(ck, dk[:, t:t + 1], t, pk, t_cap)
            S.spectra_encode(cv, dv[:, t:t + 1], t, pv, t_cap)
        S.spectra_decode_attention(ck, cv, pk, pv, t_cap, T + n_app, q, H, out=out, workspace=ws)

    work()
    torch.cuda.synchronize()
    want_out, want_k, want_v = out.clone(), pk.clone(), pv.clone()

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        work()
    for rep in range(3):
        # eager work in between: clobber the outputs and the appended records
        out.fill_(float("nan"))
        S.spectra_encode(ck, dk[:, :1], T, pk, t_cap)   # overwrite slot T with another token
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, want_out), rep
        assert torch.equal(pk, want_k), rep
        assert torch.equal(pv, want_v), rep


def test_layer_geometry_graph_replays_match_eager():
    # per-layer geometry: single-token appends and the layer attention captured in a graph
    w = synth.WORKLOADS["qwen_layer_8x"]
    T, n_app, t_cap = 1500, 2, 1536
    xk = synth.numpy_layer_stream(w, 0, 0, 0, 2304)[None]
    xv = synth.numpy_layer_stream(w, 0, 0, 1, 2304)[None]
    d = xk.shape[2]
    p = S.Params(head_dim=d, group_size=64, ratio=8.0)
    dk, dv = to_device(xk, w.dtype), to_device(xv, w.dtype)
    ck, cv = S.Codec(p, 1), S.Codec(p, 1)
    S.spectra_fit_basis(ck, dk)
    S.spectra_fit_basis(cv, dv)
    pk, pv = ck.empty_packed(t_cap), cv.empty_packed(t_cap)
    S.spectra_encode(ck, dk[:, :T].contiguous(), 0, pk, t_cap)
    S.spectra_encode(cv, dv[:, :T].contiguous(), 0, pv, t_cap)
    q = to_device(np.stack([synth.numpy_query(w, 0, 0, 0)]), w.dtype)
    n_kv = d // 128
    ws = torch.empty(S.spectra_layer_attention_workspace_bytes(ck, 1, w.n_q_heads, T + n_app), dtype=torch.uint8,
                     device=q.device)
    out = torch.empty((1, w.n_q_heads, 128), dtype=torch.float32, device=q.device)

    def work():
        for i in range(n_app):
            t = T + i
            S.spectra_encode(ck, dk[:, t:t + 1], t, pk, t_cap)
            S.spectra_encode(cv, dv[:, t:t + 1], t, pv, t_cap)
        S.spectra_layer_decode_attention(ck, cv, pk, pv, t_cap, T + n_app, q, n_kv, out=out, workspace=ws)

    work()
    torch.cuda.synchronize()
    want_out, want_k, want_v = out.clone(), pk.clone(), pv.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        work()
    for rep in range(3):
        out.fill_(float("nan"))
        ws.fill_(255)                                    # garbage in the workspace between replays
        S.spectra_encode(ck, dk[:, :1], T, pk, t_cap)   # overwrite slot T with another token
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, want_out), rep
        assert torch.equal(pk, want_k), rep
        assert torch.equal(pv, want_v), rep
