"""Benchmark of the SPECTRA codec hot path on one MI355X.

One step = the whole hot path over one batch of the headline 8x workload
(Llama-3.1-8B KV geometry, 32 layers x 8 KV heads x head_dim 128, 131072
prefill tokens in bf16, ~17 GB uncompressed):
  1. encode the whole cache (keys and values) into packed records;
  2. 32 decode steps; in each, one spectra_decode_step call per layer: append
     the new token's key and value to the packed cache (encoded in the fitted
     bases), then decode-step attention (32 query heads, GQA 4:1) read
     straight from the packed records.
The basis fit (GPU moments + host eigensolve) is calibration, done once before
the timed region and reported separately as fit_ms. Each decode step (32
calls) is replayed from a HIP graph captured beforehand, as a serving loop
would run it; --eager launches every call from Python instead.

Prints one JSON line. `value` is the step's algorithmic bytes (inputs read,
records written and read, queries, outputs, codec state) divided by the step
time. `roofline` covers the dominant work, the decode-step calls (append,
query preparation, split-K scan, combine), timed with HIP events around the
32 calls of every decode step inside the timed region.
`cpu_baseline` is the CPU oracle on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
CALIB_BYTES = 256 << 20

# HBM bytes per decode-step call from rocprofv3 counters (FETCH_SIZE and WRITE_SIZE
# passes over `bench.py --steps 1 --warmup 0 --decode-steps 2 --no-cpu-baseline
# --eager --copy-calibration --skip-configs`), scaled by the counters' reading of the
# 256 MiB copy (FETCH_SIZE reads 131093 KiB for 256 MiB read: x2.0; WRITE_SIZE reads
# 262148 KiB for 256 MiB written: x1.0). Valid only for the kernel sources they
# were taken on (sha256 over DECODE_STEP_SOURCES); otherwise `traffic` is null.
DECODE_STEP_SOURCES = ("kernels_attn.hip", "attn_common.hpp", "kplan.hpp", "encode_dev.hpp", "device_common.hpp",
                       "kernels.hpp")
# sha256 -> fetch / write bytes per call; per_kernel: [fetch, write]
MEASURED_TRAFFIC = {
    "0dc6e80a2b7f61b0b562fde7cbff11884cbad20ea2f1c2a005395111734033e8": {
        "fetch_bytes": 74542716, "write_bytes": 1674244, "mfma_busy": 0.096,
        "per_kernel": {"attn_kernel<1,8,8,true>": [70734430, 1657860], "combine_kernel": [3808286, 16384]}},
}
# The same passes over the bulk encode of one codec (256 streams x 131072 tokens):
# HBM bytes per call and the matrix cores' busy fraction (SQ_VALU_MFMA_BUSY_CYCLES
# over GRBM_GUI_ACTIVE x 1024 SIMDs), keyed by sha256 over ENCODE_SOURCES.
ENCODE_SOURCES = ("kernels_codec.hip", "encode_dev.hpp", "device_common.hpp", "kernels.hpp")
MEASURED_ENCODE = {
    "39359687aa625a2fad9927ac1b89124751d52288a590f4d285f932dbf9896b21": {
        "fetch_bytes": 8665222080, "write_bytes": 1073741824, "mfma_busy": 0.368},
}


def sources_sha256(files):
    import hashlib
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2608_07915_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def decode_step_sources_sha256():
    return sources_sha256(DECODE_STEP_SOURCES)
METRIC = "KV encode GB/s + compressed decode-attn tokens/s, % of HBM peak, at 8x"


def _parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="llama_model_131k_8x")
    ap.add_argument("--decode-steps", type=int, default=None, help="decode steps per bench step (default: workload)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--fit-weights", action="store_true",
                    help="time the calibrate-once fit from weights (Llama-3.1-8B keys: 32 layers x 8 heads, "
                         "d_model 4096) instead of the hot path; prints its own JSON line")
    ap.add_argument("--skip-extras", action="store_true",
                    help="skip the measurements outside the step (Mode A decode, attention with rotary embeddings), "
                         "e.g. for counter passes over the step's kernels only")
    ap.add_argument("--kappa", type=float, default=0.5,
                    help="key share of the combined K+V budget (asymmetric split; 0.5 = symmetric records)")
    ap.add_argument("--check", action="store_true", help="compare sampled outputs with the oracle after timing")
    ap.add_argument("--eager", action="store_true", help="launch decode steps from Python instead of HIP graphs")
    ap.add_argument("--skip-configs", action="store_true",
                    help="skip the encode + attention measurements of the other layer workloads "
                         "(Llama 4x, Qwen 8x, Llama batch 16 at 12x)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 256 MiB device-to-device copy (reference for HBM byte counters)")
    return ap.parse_args()


def algorithmic_bytes(w, Wk, Wv, n_tokens_attended):
    """Bytes the method itself must move (no dense cache bytes it avoids)."""
    d = 128
    in_b = 2 if w.dtype == "bf16" else 4
    S_layer = w.n_seq * w.n_kv_heads
    state = S_layer * 2 * (d * d * 4 + d * 4)              # K and V bases + means read once per call
    enc_per_tok = in_b * d                                   # input read per token per stream
    att_records = S_layer * n_tokens_attended * (Wk + Wv) * 4
    att_qo = w.n_seq * w.n_q_heads * d * (in_b + 4)
    append = S_layer * 2 * in_b * d + S_layer * (Wk + Wv) * 4   # new key/value rows in, records out
    return {"enc_per_token_stream": enc_per_tok, "attn_call": att_records + att_qo + state,
            "step_call": att_records + att_qo + state + append}


def cpu_baseline(w, p, budget_s=20.0, p_v=None):
    """CPU oracle on a bounded sample: one layer's first KV head (K and V streams),
    encode of the prefill + one decode-step attention; throughput in the step's
    bytes/s units."""
    import numpy as np

    import oracle as O
    import synth
    p_v = p if p_v is None else p_v
    T = w.n_tokens
    t_start = time.perf_counter()
    xk = synth.numpy_stream(w, 0, 0, 0, 0, n_tokens=T)
    xv = synth.numpy_stream(w, 0, 0, 0, 1, n_tokens=T)
    gen_s = time.perf_counter() - t_start
    xk64 = synth.bf16_bits_to_f32(xk).astype(np.float64)
    xv64 = synth.bf16_bits_to_f32(xv).astype(np.float64)
    q = synth.bf16_bits_to_f32(synth.numpy_query(w, 0, 0, 0)).astype(np.float64)[: w.n_qh]
    t0 = time.perf_counter()
    fk, fv = O.fit(xk64, p), O.fit(xv64, p_v)
    bk, bv = O.allocate_bits(fk.var, p), O.allocate_bits(fv.var, p_v)
    t1 = time.perf_counter()
    rk, *_ = O.encode(xk64, fk.basis, fk.mean, bk, p)
    rv, *_ = O.encode(xv64, fv.basis, fv.mean, bv, p_v)
    t2 = time.perf_counter()
    kh = O.decode(rk, fk.basis, fk.mean, bk, p)
    vh = O.decode(rv, fv.basis, fv.mean, bv, p_v)
    O.attention_mode_a(q, kh[None], vh[None])
    t3 = time.perf_counter()
    Wk, Wv = O.record_words(p), O.record_words(p_v)
    enc_bytes = T * (2 * 2 * 128 + (Wk + Wv) * 4)
    att_bytes = T * (Wk + Wv) * 4
    secs = t3 - t1
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        threads = 1
    return {
        "value": (enc_bytes + att_bytes) / secs / 1e9,
        "unit": "GB/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": (f"1 layer x 1 KV head (K and V streams) of the workload: encode {T} tokens + one "
                   f"decode-step attention ({w.n_qh} query heads) from the packed records; fit excluded "
                   f"({t1 - t0:.1f} s); encode {t2 - t1:.2f} s, decode+attention {t3 - t2:.2f} s"),
        "host_cores_available": len(os.sched_getaffinity(0)),
    }


def fit_weights_bench(args):
    """Calibrate-once fit from weights at the Llama-3.1-8B key geometry: per layer a
    synthetic SPD input second moment G (4096 x 4096, fp64) and mean, per KV head a
    random fp32 projection W (4096 x 128). Times spectra_fit_weights (fp64 products
    on the GPU, eigensolve of 256 streams on the host)."""
    import torch

    import paper_2608_07915_amd as S
    dev = torch.device("cuda:0")
    L, H, dm = 32, 8, 4096
    g = torch.Generator(device=dev)
    g.manual_seed(0)
    lam = torch.arange(1, dm + 1, dtype=torch.float64, device=dev) ** -1.2
    lam *= dm / lam.sum()
    G = torch.empty(L, dm, dm, dtype=torch.float64, device=dev)
    for l in range(L):
        a = torch.randn(dm, dm, dtype=torch.float64, device=dev, generator=g) * lam.sqrt()[None, :]
        G[l] = a @ a.T / dm
    hbar = 0.5 * torch.randn(L, dm, dtype=torch.float64, device=dev, generator=g)
    W = (torch.randn(L * H, dm, 128, device=dev, generator=g) / dm ** 0.5).contiguous()
    codec = S.Codec(S.Params(ratio=8.0), L * H)
    ws = torch.empty(S.spectra_fit_weights_workspace_bytes(codec, dm), dtype=torch.uint8, device=dev)
    times = []
    for _ in range(args.warmup + args.steps):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        S.spectra_fit_weights(codec, W, G, hbar, streams_per_layer=H, workspace=ws)
        times.append(time.perf_counter() - t0)
    ms = 1e3 * min(times[args.warmup:])
    flops = L * H * (2.0 * dm * dm * 128 + 2.0 * dm * 128 * 128)
    print(json.dumps({"metric": "calibrate-once fit from weights, wall ms (GPU fp64 products + host eigensolve)",
                      "value": round(ms, 2), "unit": "ms", "higher_is_better": False, "steps": args.steps,
                      "warmup": args.warmup, "data": "synthetic",
                      "config": {"workload": "llama3.1-8b keys", "n_layers": L, "n_kv_heads": H, "d_model": dm},
                      "product_gflop": round(flops / 1e9, 1),
                      "bits_first_layer": codec.bits[:H].cpu().numpy().tolist()}))


def outside_step(S, torch, w, layer_ck, layer_cv, layer_pk, layer_pv, t_cap, n_rec, qs, ws, Wk, Wv, H, Hq, d, dev):
    """Timings outside the step on layer 0: Mode A reconstruction of the keys to fp32,
    and attention with rotary embeddings (keys reconstructed and rotated)."""
    import synth
    dec_out = torch.empty((H, n_rec, d), dtype=torch.float32, device=dev)
    dec_ev = []
    for _ in range(4):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        S.spectra_decode(layer_ck[0], layer_pk[0], t_cap, 0, n_rec, out=dec_out)
        e1.record()
        dec_ev.append((e0, e1))
    torch.cuda.synchronize()
    dec_ms = min(e0.elapsed_time(e1) for e0, e1 in dec_ev[1:])
    dec_bytes = H * n_rec * (Wk * 4 + d * 4) + H * (d * d * 4 + d * 4)
    del dec_out
    # ---- Mode A attention with rotary embeddings (outside the step): one layer call ----
    inv_freq = (500000.0 ** (-torch.arange(d // 2, dtype=torch.float64, device=dev) / (d // 2))).float()
    rope_out = torch.empty((1, Hq, d), dtype=torch.float32, device=dev)
    rope_ev = []
    for _ in range(4):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        S.spectra_decode_attention_rope(layer_ck[0], layer_cv[0], layer_pk[0], layer_pv[0], t_cap, n_rec, qs[0, 0],
                                        H, inv_freq, out=rope_out, workspace=ws)
        e1.record()
        rope_ev.append((e0, e1))
    torch.cuda.synchronize()
    rope_ms = min(e0.elapsed_time(e1) for e0, e1 in rope_ev[1:])
    rope_bytes = algorithmic_bytes(w, Wk, Wv, n_rec)["attn_call"]

    # ---- per-layer cross-head latent (outside the step): the keys (and values) of one
    # layer as one d_kv = 8 x 128 stream each, groups of 64, fitted on the first 8192 tokens ----
    dl = H * d
    pl = S.Params(head_dim=dl, group_size=64, ratio=w.ratio)
    xl = synth.device_layer_stream(w, 0, 0, 0, n_rec, dev)
    cl = S.Codec(pl, 1)
    S.spectra_fit_basis(cl, xl[:, :8192])
    pkl = cl.empty_packed(t_cap)
    outl = torch.empty((1, n_rec, dl), dtype=torch.float32, device=dev)
    xlv = synth.device_layer_stream(w, 0, 0, 1, n_rec, dev)
    clv = S.Codec(pl, 1)
    S.spectra_fit_basis(clv, xlv[:, :8192])
    pklv = clv.empty_packed(t_cap)
    S.spectra_encode(clv, xlv, 0, pklv, t_cap)
    del xlv
    lay_ev = []
    for _ in range(4):
        e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        e[0].record()
        S.spectra_encode(cl, xl, 0, pkl, t_cap)
        e[1].record()
        S.spectra_decode(cl, pkl, t_cap, 0, n_rec, out=outl)
        e[2].record()
        lay_ev.append(e)
    torch.cuda.synchronize()
    lenc_ms = min(e[0].elapsed_time(e[1]) for e in lay_ev[1:])
    ldec_ms = min(e[1].elapsed_time(e[2]) for e in lay_ev[1:])
    # Mode B attention of the 32 query heads over both per-layer caches
    lq = qs[0, 0].contiguous()  # [1, Hq, 128]
    lws = torch.empty(S.spectra_layer_attention_workspace_bytes(cl, 1, Hq, n_rec), dtype=torch.uint8, device=dev)
    lout = torch.empty((1, Hq, d), dtype=torch.float32, device=dev)
    latt_ev = []
    for _ in range(4):
        e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        e[0].record()
        S.spectra_layer_decode_attention(cl, clv, pkl, pklv, t_cap, n_rec, lq, H, out=lout, workspace=lws)
        e[1].record()
        latt_ev.append(e)
    torch.cuda.synchronize()
    latt_ms = min(e[0].elapsed_time(e[1]) for e in latt_ev[1:])
    Wl = cl.record_words
    # the same attention over per-layer caches at 4x (128-word records)
    pl4 = S.Params(head_dim=dl, group_size=64, ratio=4.0)
    c4 = []
    for tensor in (0, 1):
        x4 = synth.device_layer_stream(w, 0, 0, tensor, n_rec, dev)
        cc = S.Codec(pl4, 1)
        S.spectra_fit_basis(cc, x4[:, :8192])
        pp = cc.empty_packed(t_cap)
        S.spectra_encode(cc, x4, 0, pp, t_cap)
        del x4
        c4.append((cc, pp))
    lws4 = torch.empty(S.spectra_layer_attention_workspace_bytes(c4[0][0], 1, Hq, n_rec), dtype=torch.uint8, device=dev)
    latt4_ev = []
    for _ in range(4):
        e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        e[0].record()
        S.spectra_layer_decode_attention(c4[0][0], c4[1][0], c4[0][1], c4[1][1], t_cap, n_rec, lq, H, out=lout,
                                         workspace=lws4)
        e[1].record()
        latt4_ev.append(e)
    torch.cuda.synchronize()
    latt4_ms = min(e[0].elapsed_time(e[1]) for e in latt4_ev[1:])
    W4 = c4[0][0].record_words
    latt4_bytes = 2 * n_rec * W4 * 4 + 2 * (dl * dl * 4 + dl * 4) + Hq * d * 2 + Hq * d * 4
    del c4, lws4
    lenc_bytes = n_rec * dl * 2 + n_rec * Wl * 4 + dl * dl * 4 + dl * 4
    ldec_bytes = n_rec * Wl * 4 + n_rec * dl * 4 + dl * dl * 4 + dl * 4
    kept = int((cl.bits[0] > 0).sum().item())
    latt_bytes = 2 * n_rec * Wl * 4 + 2 * (dl * dl * 4 + dl * 4) + Hq * d * 2 + Hq * d * 4
    del xl, pkl, outl, cl, clv, pklv, lws

    return {
        "layer_latent": {"d": dl, "group_size": 64, "record_words": Wl, "kept_groups": kept, "tokens": n_rec,
                         "encode_ms": round(lenc_ms, 4), "encode_GBps": round(lenc_bytes / (lenc_ms * 1e-3) / 1e9, 1),
                         "decode_ms": round(ldec_ms, 4), "decode_GBps": round(ldec_bytes / (ldec_ms * 1e-3) / 1e9, 1),
                         "attention_us": round(latt_ms * 1e3, 1),
                         "attention_GBps": round(latt_bytes / (latt_ms * 1e-3) / 1e9, 1),
                         "attention_4x_record_words": W4,
                         "attention_4x_us": round(latt4_ms * 1e3, 1),
                         "attention_4x_GBps": round(latt4_bytes / (latt4_ms * 1e-3) / 1e9, 1),
                         "what": "per-layer cross-head latent: spectra_encode and spectra_decode of one layer's keys "
                                 "as one d_kv stream, and spectra_layer_decode_attention of the 32 query heads "
                                 "over that layer's keys and values (8x, and attention_4x_* over caches at 4x), "
                                 "outside the step"},
        "mode_a_rope_attention": {"us_per_layer_call": round(rope_ms * 1e3, 1),
                                  "GBps": round(rope_bytes / (rope_ms * 1e-3) / 1e9, 1),
                                  "what": "spectra_decode_attention_rope (keys reconstructed and rotated) over one "
                                          "layer, outside the step"},
        "mode_a_decode": {"ms_per_layer": round(dec_ms, 4), "GBps": round(dec_bytes / (dec_ms * 1e-3) / 1e9, 1),
                          "frac": round(dec_bytes / (dec_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
                          "what": "spectra_decode of one layer's keys (8 streams) to fp32, outside the step"},
    }


# The model-shaped layer workloads measured beside the headline one: encode of the whole
# layer, then decode-step attention read from the packed records (no appends).
CONFIG_WORKLOADS = ("llama_layer_4x", "qwen_layer_8x", "llama_batch16_12x")
MALL_BYTES = 256 << 20


def config_bench(S, torch, w, dev, reps=4):
    """Encode and decode-step attention of one layer workload. Attention steps cycle
    through enough copies of the packed caches (>= 2x the 256 MB MALL in total) that
    every step reads its records from HBM; the steps of one pass are replayed from a
    HIP graph, and HIP events around the replays give the time per step."""
    import synth
    H, Hq, d, B, T = w.n_kv_heads, w.n_q_heads, 128, w.n_seq, w.n_tokens
    Sn = B * H
    t_cap = (T + 63) // 64 * 64
    xk = synth.device_streams(w, 0, 0, T, dev)
    xv = synth.device_streams(w, 1, 0, T, dev)
    sp = S.Params(ratio=w.ratio)
    ck, cv = S.Codec(sp, Sn), S.Codec(sp, Sn)
    S.spectra_fit_basis(ck, xk)
    S.spectra_fit_basis(cv, xv)
    Wk, Wv = ck.record_words, cv.record_words
    pk, pv = ck.empty_packed(t_cap), cv.empty_packed(t_cap)
    ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731
    enc = []
    for _ in range(reps):
        e0, e1 = ev(), ev()
        e0.record()
        S.spectra_encode(ck, xk, 0, pk, t_cap)
        S.spectra_encode(cv, xv, 0, pv, t_cap)
        e1.record()
        enc.append((e0, e1))
    torch.cuda.synchronize()
    enc_ms = sum(e0.elapsed_time(e1) for e0, e1 in enc[1:]) / (reps - 1)
    in_b = 2 if w.dtype == "bf16" else 4
    state = Sn * 2 * (d * d * 4 + d * 4)
    enc_bytes = Sn * T * (2 * d * in_b + (Wk + Wv) * 4) + state
    del xk, xv
    rec_bytes = Sn * T * (Wk + Wv) * 4
    att_bytes = rec_bytes + state + B * Hq * d * (in_b + 4)
    copies = max(1, -(-2 * MALL_BYTES // rec_bytes))
    caches = [(pk, pv)] + [(pk.clone(), pv.clone()) for _ in range(copies - 1)]
    steps = max(w.attn_steps, copies)
    qs = [synth.device_queries(w, 0, s % max(w.attn_steps, 1), dev) for s in range(steps)]
    ws = torch.empty(S.spectra_attention_workspace_bytes(B, Hq, H, T), dtype=torch.uint8, device=dev)
    out = torch.empty((B, Hq, d), dtype=torch.float32, device=dev)

    def attend():
        for s in range(steps):
            kp, vp = caches[s % copies]
            S.spectra_decode_attention(ck, cv, kp, vp, t_cap, T, qs[s], H, out=out, workspace=ws)

    attend()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        attend()
    g.replay()
    torch.cuda.synchronize()
    runs = []
    for _ in range(reps):
        e0, e1 = ev(), ev()
        e0.record()
        g.replay()
        e1.record()
        runs.append((e0, e1))
    torch.cuda.synchronize()
    att_ms = sum(e0.elapsed_time(e1) for e0, e1 in runs) / (reps * steps)
    # Mode A with rotary embeddings over the same caches (keys reconstructed and rotated)
    theta = 1.0e6 if w.name.startswith("qwen") else 5.0e5
    inv_freq = (theta ** (-torch.arange(d // 2, dtype=torch.float64, device=dev) / (d // 2))).float()
    rope = []
    for i in range(reps + 1):
        kp, vp = caches[i % copies]
        e0, e1 = ev(), ev()
        e0.record()
        S.spectra_decode_attention_rope(ck, cv, kp, vp, t_cap, T, qs[i % steps], H, inv_freq, out=out, workspace=ws)
        e1.record()
        rope.append((e0, e1))
    torch.cuda.synchronize()
    rope_ms = min(e0.elapsed_time(e1) for e0, e1 in rope[1:])
    del caches, g
    enc_gbps = enc_bytes / (enc_ms * 1e-3) / 1e9
    att_gbps = att_bytes / (att_ms * 1e-3) / 1e9
    return {
        "description": w.description, "record_words": [Wk, Wv], "ratio_actual": round(16 * d / (32 * Wk), 2),
        "encode": {"ms": round(enc_ms, 4), "GBps": round(enc_gbps, 1), "frac": round(enc_gbps / HBM_PEAK_GBPS, 4),
                   "bytes": enc_bytes},
        "attention": {"us_per_step": round(att_ms * 1e3, 2), "GBps": round(att_gbps, 1),
                      "frac": round(att_gbps / HBM_PEAK_GBPS, 4), "bytes_per_step": att_bytes,
                      "cache_tokens_per_s": round(B * T / (att_ms * 1e-3), 1),
                      "sequences_per_s": round(B / (att_ms * 1e-3), 1),
                      "steps_timed": steps * reps, "distinct_cache_copies": copies},
        "mode_a_rope_attention": {"us_per_call": round(rope_ms * 1e3, 1),
                                  "GBps": round(att_bytes / (rope_ms * 1e-3) / 1e9, 1),
                                  "rope_theta": theta},
        "bits_k_first": ck.bits[0].cpu().numpy().tolist(), "bits_v_first": cv.bits[0].cpu().numpy().tolist(),
    }


def main():
    args = _parse()
    if args.gpus != 1:
        print(json.dumps({"error": "bench.py runs on one GPU only; multi-GPU runs are not implemented (codec streams are independent and shard without communication)",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    if args.fit_weights:
        return fit_weights_bench(args)
    import numpy as np
    import torch

    import oracle as O
    import paper_2608_07915_amd as S
    import synth

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = synth.WORKLOADS[args.workload]
    L, H, Hq, d = w.n_layers, w.n_kv_heads, w.n_q_heads, 128
    n_seq = w.n_seq
    T = w.n_tokens
    n_dec = w.n_append if args.decode_steps is None else args.decode_steps
    T_all = T + max(n_dec, 0)
    t_cap = (T_all + 63) // 64 * 64
    Sn = n_seq * L * H                      # streams per codec, index (seq*L + layer)*H + head
    sp = sp_v = S.Params(ratio=w.ratio)
    p = p_v = O.Params(ratio=w.ratio)
    if args.kappa != 0.5:
        sp, sp_v = S.spectra_split_budget(sp, args.kappa)
        p, p_v = O.split_budget(p, args.kappa)

    # ---- synthetic inputs (resident in HBM before timing) ----
    t_gen = time.perf_counter()
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    xk = torch.empty((Sn, T_all, d), dtype=dt, device=dev)
    xv = torch.empty((Sn, T_all, d), dtype=dt, device=dev)
    for layer in range(L):
        for tensor, x in ((0, xk), (1, xv)):
            blk = synth.device_streams(w, tensor, layer, T_all, dev)      # [n_seq*H, T, d]
            for seq in range(n_seq):
                dst = (seq * L + layer) * H
                x[dst:dst + H] = blk[seq * H:(seq + 1) * H]
            del blk
    qs = torch.stack([torch.stack([synth.device_queries(w, layer, step, dev) for layer in range(L)])
                      for step in range(max(n_dec, 1))])  # [steps][L][n_seq][Hq][d]
    torch.cuda.synchronize()
    gen_s = time.perf_counter() - t_gen

    # ---- calibration: fit once on the prefill ----
    ck, cv = S.Codec(sp, Sn), S.Codec(sp_v, Sn)
    t_fit = time.perf_counter()
    S.spectra_fit_basis(ck, xk, n_tokens=T)
    S.spectra_fit_basis(cv, xv, n_tokens=T)
    torch.cuda.synchronize()
    fit_s = time.perf_counter() - t_fit
    Wk, Wv = ck.record_words, cv.record_words
    pk, pv = ck.empty_packed(t_cap), cv.empty_packed(t_cap)
    # per-layer views (codec state and packed records)
    layer_ck = [ck.view(l * H, H) for l in range(L)]
    layer_cv = [cv.view(l * H, H) for l in range(L)]
    layer_pk = [pk[l * H * t_cap * Wk:(l + 1) * H * t_cap * Wk] for l in range(L)]
    layer_pv = [pv[l * H * t_cap * Wv:(l + 1) * H * t_cap * Wv] for l in range(L)]
    if n_seq != 1:
        raise SystemExit("the per-layer decode loop here expects one sequence")
    ws_bytes = S.spectra_attention_workspace_bytes(1, Hq, H, t_cap)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    outs = torch.empty((L, 1, Hq, d), dtype=torch.float32, device=dev)

    n_attn_calls = max(n_dec, 0) * L
    ev = lambda: torch.cuda.Event(enable_timing=True)  # noqa: E731

    # the new key / value rows of every decode step and layer, [1][H][d] contiguous
    k_new = [[xk[l * H:(l + 1) * H, T + s].contiguous().view(1, H, d) for l in range(L)] for s in range(n_dec)]
    v_new = [[xv[l * H:(l + 1) * H, T + s].contiguous().view(1, H, d) for l in range(L)] for s in range(n_dec)]

    def decode_steps(s):
        # one call per layer: append the new key and value at slot T + s, attend over T + s + 1 slots
        for l in range(L):
            S.spectra_decode_step(layer_ck[l], layer_cv[l], layer_pk[l], layer_pv[l], t_cap, T + s, k_new[s][l],
                                  v_new[s][l], qs[s, l], H, out=outs[l], workspace=ws)

    # Each decode step (L calls) runs as one HIP graph, as a serving loop would, so
    # host launch overhead is not timed; --eager launches every call from Python.
    graphs = None

    def step(record):
        e0, e1 = ev(), ev()
        e0.record()
        S.spectra_encode(ck, xk, 0, pk, t_cap, n_tokens=T)
        S.spectra_encode(cv, xv, 0, pv, t_cap, n_tokens=T)
        e1.record()
        att = []
        for s in range(n_dec):
            a0 = ev()
            a0.record()
            if graphs is None:
                decode_steps(s)
            else:
                graphs[s].replay()
            a1 = ev()
            a1.record()
            att.append((a0, a1, T + s + 1))
        if record is not None:
            record.append(((e0, e1), att))

    for _ in range(args.warmup):
        step(None)
    torch.cuda.synchronize()
    if not args.eager:
        graphs = []
        for s in range(n_dec):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                decode_steps(s)
            graphs.append(g)
        torch.cuda.synchronize()
        step(None)  # one untimed pass through the replays
        torch.cuda.synchronize()
    rec = []
    start, end = ev(), ev()
    start.record()
    for _ in range(args.steps):
        step(rec)
    end.record()
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(end)
    ms_per_step = total_ms / args.steps

    if args.copy_calibration:
        # A plain copy of known size: its FETCH_SIZE / WRITE_SIZE counters scale the
        # counters of the codec kernels to bytes.
        src = torch.empty(CALIB_BYTES // 2, dtype=torch.bfloat16, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # ---- Mode A reconstruction (a9), outside the step: one layer's keys to fp32 ----
    n_rec = T + max(n_dec, 0)
    extras = {}
    if not args.skip_extras:
        extras = outside_step(S, torch, w, layer_ck, layer_cv, layer_pk, layer_pv, t_cap, n_rec, qs, ws, Wk, Wv, H, Hq,
                              d, dev)

    # ---- derived throughput ----
    ab = lambda n: algorithmic_bytes(w, Wk, Wv, n)  # noqa: E731
    enc_bytes = Sn * T * 2 * d * (2 if w.dtype == "bf16" else 4) + Sn * T * (Wk + Wv) * 4 + Sn * 2 * (d * d * 4 + d * 4)
    att_bytes_calls = [ab(n)["step_call"] for s in range(n_dec) for n in [T + s + 1] for _ in range(L)]
    step_bytes = enc_bytes + sum(att_bytes_calls)
    enc_ms = float(np.mean([r[0][0].elapsed_time(r[0][1]) for r in rec]))
    att_ms_blocks = [a0.elapsed_time(a1) for r in rec for (a0, a1, _) in r[1]]
    att_call_ms = float(np.sum(att_ms_blocks)) / max(len(att_ms_blocks) * L, 1)
    att_call_bytes = float(np.mean(att_bytes_calls)) if att_bytes_calls else 0.0
    att_gbps = att_call_bytes / (att_call_ms * 1e-3) / 1e9 if att_call_ms > 0 else 0.0
    tokens_per_call = n_seq * float(np.mean([T + s + 1 for s in range(n_dec)])) if n_dec else 0.0
    value = step_bytes / (ms_per_step * 1e-3) / 1e9
    # counters were taken on the default workload with symmetric records
    headline = (w.name, args.kappa) == ("llama_model_131k_8x", 0.5)
    measured = MEASURED_TRAFFIC.get(decode_step_sources_sha256()) if headline else None
    traffic = (measured["fetch_bytes"] + measured["write_bytes"]) if measured else None
    enc_counters = MEASURED_ENCODE.get(sources_sha256(ENCODE_SOURCES)) if headline else None

    result = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": w.name, "description": w.description, "n_layers": L, "n_kv_heads": H, "n_q_heads": Hq,
            "head_dim": d, "batch": n_seq, "prefill_tokens": T, "decode_steps": n_dec,
            "ratio_nominal": w.ratio, "ratio_actual_k": round(16 * d / (32 * Wk), 3),
            "ratio_actual_v": round(16 * d / (32 * Wv), 3), "record_words": [Wk, Wv],
            "kappa": args.kappa,
        },
        "frac_of_hbm_peak": round(value / HBM_PEAK_GBPS, 4),
        "encode": {"ms": round(enc_ms, 3), "GBps": round(enc_bytes / (enc_ms * 1e-3) / 1e9, 1),
                   "frac": round(enc_bytes / (enc_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
                   "algorithmic_bytes": enc_bytes,
                   "traffic": (2 * (enc_counters["fetch_bytes"] + enc_counters["write_bytes"])
                               if enc_counters else None),
                   "mfma_busy": enc_counters["mfma_busy"] if enc_counters else None},
        "decode_step": {"ms_per_layer_call": round(att_call_ms, 4), "GBps": round(att_gbps, 1),
                             "frac": round(att_gbps / HBM_PEAK_GBPS, 4),
                             "cache_tokens_per_s": round(tokens_per_call / (att_call_ms * 1e-3), 1),
                             "generated_tokens_per_s": round(1.0 / (att_call_ms * 1e-3 * L), 2)},
        "roofline": {"bound": "hbm", "achieved": round(att_gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(att_gbps / HBM_PEAK_GBPS, 4), "traffic": traffic,
                     "mfma_busy": measured["mfma_busy"] if measured else None,
                     "kernel": "decode_step (split-K scan with in-kernel query prep and append, then combine), per layer call",
                     "algorithmic_bytes_per_launch": round(att_call_bytes)},
        "traffic_detail": measured,
        **extras,
        "decode_launch": "eager" if args.eager else "hip_graph",
        "fit_ms": round(fit_s * 1e3, 1),
        "input_generation_s": round(gen_s, 1),
        "bits_k_first_layer": ck.bits[:H].cpu().numpy().tolist(),
        "bits_v_first_layer": cv.bits[:H].cpu().numpy().tolist(),
    }
    if args.check:
        result["check"] = sampled_check(w, p, p_v, ck, cv, pk, pv, xk, xv, qs, outs, t_cap, T, n_dec, L, H)
    if not args.skip_configs:
        # the other layer workloads, after the headline one's buffers are released
        del xk, xv, pk, pv, k_new, v_new, layer_pk, layer_pv, graphs
        torch.cuda.empty_cache()
        result["configs"] = {}
        for name in CONFIG_WORKLOADS:
            result["configs"][name] = config_bench(S, torch, synth.WORKLOADS[name], dev)
            torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(w, p, p_v=p_v)
    print(json.dumps(result))


def sampled_check(w, p, p_v, ck, cv, pk, pv, xk, xv, qs, outs, t_cap, T, n_dec, L, H):
    """Oracle comparison of the last layer's head 0 after the timed steps."""
    import numpy as np

    import oracle as O
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    from gpu_parity import check_encoded_stream, codec_state, records_of, rel_l2, host_values
    l = L - 1
    n = T + n_dec
    s = l * H
    res = {}
    for name, par, codec, packed, x in (("k", p, ck, pk, xk), ("v", p_v, cv, pv, xv)):
        basis, mean, bits = codec_state(codec, s)
        rec = records_of(packed, s, 0, n, t_cap, codec.record_words)
        r = check_encoded_stream(host_values(x[s, :n]), basis, mean, bits, par, rec)
        res[name] = {"code_mismatch": r.code_mismatch, "meta_mismatch": r.meta_mismatch}
    return res


if __name__ == "__main__":
    main()
