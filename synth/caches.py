"""Seeded synthetic KV caches with a controlled spectrum.

Recipe (one *stream* = one (sequence, layer, KV head, tensor) T x d matrix):

* rng = numpy ``default_rng([seed, workload_id, seq, layer, head, tensor])``
  with tensor 0 = keys, 1 = values, 2 = queries (for queries the ``head`` slot
  carries the decode-step index).
* Draw order: (alpha, n_out when randomised) -> Haar orthogonal Q (QR of a
  Gaussian d x d, columns sign-fixed by sign(diag R)) -> mean mu ~ N(0,1)^d ->
  outlier channel indices (without replacement) -> Z ~ N(0,1)^{T x d}.
* lambda_i = i^-alpha (i = 1..d) normalised so sum(lambda) = d, i.e. unit
  mean channel variance, which keeps bf16 values O(1) like real caches.
* X = Z diag(sqrt(lambda)) Q^T + mu, then X[:, outliers] *= outlier_scale.
* Stored as fp32 or as bf16 (round-to-nearest-even). The stored values are
  the input of every consumer.

The model-shaped workloads follow the KV geometry of Llama-3.1-8B (32 query /
8 KV heads, head_dim 128) and Qwen2.5-7B (28 query / 4 KV heads, head_dim 128)
named in Sec. 4.1. Real activations and the LongBench/NIAH data are not used:
these synthetic caches stand in for them.

Two backends draw the same *distribution*:

* ``numpy_stream`` draws one stream exactly as above (bit-reproducible on any
  host); tests use it at small and medium sizes.
* ``device_streams`` draws the per-stream parameters (alpha, Q, mu, outliers)
  with numpy exactly as above but Z with a seeded torch generator on the GPU,
  for multi-gigabyte caches. Its values are not the numpy backend's; parity
  checks at those sizes copy the drawn input back to the host.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Optional, Tuple

import numpy as np

D = 128


@dataclass(frozen=True)
class StreamSpec:
    alpha: float
    n_out: int
    out_scale: float


@dataclass(frozen=True)
class Workload:
    """One synthetic workload: shapes, dtypes and spectra recipe."""
    wid: int
    name: str
    n_seq: int
    n_layers: int
    n_kv_heads: int
    n_q_heads: int
    n_tokens: int          # prefill tokens encoded in one pass
    n_append: int          # tokens appended one at a time afterwards
    dtype: str             # "f32" or "bf16"
    ratio: float           # effective compression vs fp16
    k_alpha: Optional[float]     # None -> alpha ~ U(1, 2) per stream
    k_out: Optional[int]         # None -> n_out ~ U{0..8} per stream
    k_out_scale: float
    v_alpha: Optional[float]
    v_out: int
    attn_steps: int
    description: str = ""

    @property
    def n_streams(self) -> int:
        return self.n_seq * self.n_layers * self.n_kv_heads

    @property
    def n_qh(self) -> int:
        return self.n_q_heads // self.n_kv_heads


WORKLOADS = {
    "tiny": Workload(0, "tiny", 1, 1, 1, 1, 4096, 0, "f32", 8.0,
                     1.5, 4, 10.0, 0.8, 0, 1,
                     "1 layer, 1 KV head, 4096 fp32 tokens, 8x"),
    "llama_layer_4x": Workload(1, "llama_layer_4x", 1, 1, 8, 32, 32768, 0, "bf16", 4.0,
                               1.5, 4, 10.0, 0.8, 0, 64,
                               "Llama-3.1-8B layer: 32 q / 8 kv heads, 32768 bf16 tokens, 4x"),
    "qwen_layer_8x": Workload(2, "qwen_layer_8x", 1, 1, 4, 28, 65536, 0, "bf16", 8.0,
                              2.0, 8, 20.0, 0.8, 0, 64,
                              "Qwen2.5-7B layer: 28 q / 4 kv heads, 65536 bf16 tokens, 8x"),
    "llama_batch16_12x": Workload(3, "llama_batch16_12x", 16, 1, 8, 32, 32768, 0, "bf16", 12.0,
                                  1.5, 4, 10.0, 0.8, 0, 1,
                                  "Llama-3.1-8B layer, batch 16 x 32768 bf16 tokens, 12x"),
    "llama_model_131k_8x": Workload(4, "llama_model_131k_8x", 1, 32, 8, 32, 131072, 32, "bf16", 8.0,
                                    None, None, 10.0, None, 0, 32,
                                    "Llama-3.1-8B cache, 32 layers x 8 kv heads, 131072 bf16 tokens "
                                    "+ 32 appended, 8x"),
}


def _rng(seed: int, wid: int, seq: int, layer: int, head: int, tensor: int):
    return np.random.default_rng([seed, wid, seq, layer, head, tensor])


def stream_spec(w: Workload, rng, tensor: int) -> StreamSpec:
    """Draw the spectrum parameters of one stream (first draws of its rng)."""
    if tensor == 0:
        alpha = w.k_alpha if w.k_alpha is not None else float(rng.uniform(1.0, 2.0))
        n_out = w.k_out if w.k_out is not None else int(rng.integers(0, 9))
        return StreamSpec(alpha, n_out, w.k_out_scale)
    alpha = w.v_alpha if w.v_alpha is not None else float(rng.uniform(1.0, 2.0))
    return StreamSpec(alpha, w.v_out, 1.0)


def _haar(rng, d: int) -> np.ndarray:
    a = rng.standard_normal((d, d))
    q, r = np.linalg.qr(a)
    return q * np.sign(np.diag(r))[None, :]


def _stream_params(w: Workload, seed: int, seq: int, layer: int, head: int, tensor: int):
    rng = _rng(seed, w.wid, seq, layer, head, tensor)
    spec = stream_spec(w, rng, tensor)
    q = _haar(rng, D)
    mu = rng.standard_normal(D)
    out_idx = rng.choice(D, size=spec.n_out, replace=False) if spec.n_out > 0 else np.zeros(0, np.int64)
    lam = np.arange(1, D + 1, dtype=np.float64) ** (-spec.alpha)
    lam *= D / lam.sum()
    mix = np.sqrt(lam)[:, None] * q.T          # diag(sqrt(lambda)) Q^T
    return rng, spec, mix, mu, out_idx


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round to nearest even; NaN kept NaN."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        r = np.where(nan, np.uint16(0x7FC0), r)
    return r


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def numpy_stream(w: Workload, seq: int, layer: int, head: int, tensor: int,
                 n_tokens: Optional[int] = None, seed: int = 0) -> np.ndarray:
    """One stream, [T, 128]: float32 array (f32 workloads) or uint16 bf16 bits."""
    T = (w.n_tokens + w.n_append) if n_tokens is None else n_tokens
    rng, spec, mix, mu, out_idx = _stream_params(w, seed, seq, layer, head, tensor)
    z = rng.standard_normal((T, D))
    x = z @ mix + mu
    if out_idx.size:
        x[:, out_idx] *= spec.out_scale
    x32 = x.astype(np.float32)
    return x32 if w.dtype == "f32" else f32_to_bf16_bits(x32)


def numpy_query(w: Workload, seq: int, layer: int, step: int, seed: int = 0) -> np.ndarray:
    """Queries of one (sequence, layer, decode step): [n_q_heads, 128], q ~ N(0,1)."""
    rng = _rng(seed, w.wid, seq, layer, step, 2)
    q = rng.standard_normal((w.n_q_heads, D)).astype(np.float32)
    return q if w.dtype == "f32" else f32_to_bf16_bits(q)


def device_streams(w: Workload, tensor: int, layer: int, n_tokens: int, device, seed: int = 0,
                   out=None):
    """All streams of one layer and tensor, drawn on the GPU: [n_seq*n_kv, T, 128].

    Per-stream parameters come from numpy as in ``numpy_stream``; the Gaussian
    Z comes from a torch generator seeded by (seed, workload, layer, tensor).
    Returns a torch tensor of the workload dtype (written into ``out`` if given).
    """
    import torch
    n = w.n_seq * w.n_kv_heads
    dt = torch.float32 if w.dtype == "f32" else torch.bfloat16
    if out is None:
        out = torch.empty((n, n_tokens, D), dtype=dt, device=device)
    gen = torch.Generator(device=device)
    gen.manual_seed(((seed * 1000003 + w.wid) * 1000003 + layer) * 4 + tensor)
    for seq in range(w.n_seq):
        for head in range(w.n_kv_heads):
            _, spec, mix, mu, out_idx = _stream_params(w, seed, seq, layer, head, tensor)
            i = seq * w.n_kv_heads + head
            mix_t = torch.from_numpy(mix.astype(np.float32)).to(device)
            mu_t = torch.from_numpy(mu.astype(np.float32)).to(device)
            step = 16384
            for t0 in range(0, n_tokens, step):
                t1 = min(n_tokens, t0 + step)
                z = torch.randn((t1 - t0, D), generator=gen, device=device, dtype=torch.float32)
                x = z @ mix_t + mu_t
                if out_idx.size:
                    x[:, torch.from_numpy(out_idx).to(device)] *= spec.out_scale
                out[i, t0:t1] = x.to(dt)
    return out


def device_queries(w: Workload, layer: int, step: int, device, seed: int = 0):
    """Queries for all sequences of one (layer, step): [n_seq, n_q_heads, 128] on device."""
    import torch
    qs = [numpy_query(w, s, layer, step, seed) for s in range(w.n_seq)]
    q = np.stack(qs)
    if w.dtype == "f32":
        return torch.from_numpy(q).to(device)
    return torch.from_numpy(q.view(np.int16)).to(device).view(torch.bfloat16)


def numpy_layer_stream(w: Workload, seq: int, layer: int, tensor: int, n_tokens: int, seed: int = 0,
                       shared_rank: int = 16, shared_frac: float = 0.3) -> np.ndarray:
    """One per-layer stream, [T, n_kv_heads * 128]: the layer's KV heads side by side
    (each drawn by ``numpy_stream``) plus a component shared across heads.

    Real layers correlate their heads, which is what a transform over the whole
    d_kv = n_kv_heads * 128 vector exploits and a per-head one cannot. Recipe: rng
    ``default_rng([seed, workload_id, seq, layer, 1000 + tensor])``; U ~ N(0,1)^{d_kv x r}
    scaled so the shared part carries ``shared_frac`` of the heads' mean channel
    energy, Z ~ N(0,1)^{T x r}; X = [X_1 .. X_H] + Z U^T, then rounded like the heads
    (fp32, or bf16 round-to-nearest-even). Returns float32 or uint16 bf16 bits.
    """
    heads = [numpy_stream(w, seq, layer, h, tensor, n_tokens=n_tokens, seed=seed) for h in range(w.n_kv_heads)]
    x = np.concatenate([hh if w.dtype == "f32" else bf16_bits_to_f32(hh) for hh in heads], axis=1).astype(np.float64)
    d_kv = x.shape[1]
    rng = np.random.default_rng([seed, w.wid, seq, layer, 1000 + tensor])
    u = rng.standard_normal((d_kv, shared_rank))
    energy = float(np.mean(x * x))
    u *= math.sqrt(shared_frac * energy / shared_rank)
    z = rng.standard_normal((n_tokens, shared_rank))
    x = (x + z @ u.T).astype(np.float32)
    return x if w.dtype == "f32" else f32_to_bf16_bits(x)


def device_layer_stream(w: Workload, seq: int, layer: int, tensor: int, n_tokens: int, device, seed: int = 0,
                        shared_rank: int = 16, shared_frac: float = 0.3):
    """Per-layer stream of ``numpy_layer_stream``'s distribution drawn on the GPU:
    [1, T, n_kv_heads * 128] in the workload dtype. The heads come from
    ``device_streams`` (sequence ``seq``), U from the same numpy rng as the numpy
    backend, Z from a torch generator; values differ from the numpy backend's."""
    import torch
    heads = device_streams(w, tensor, layer, n_tokens, device, seed=seed)[seq * w.n_kv_heads:(seq + 1) * w.n_kv_heads]
    x = heads.permute(1, 0, 2).reshape(n_tokens, -1).float()
    del heads
    d_kv = x.shape[1]
    rng = np.random.default_rng([seed, w.wid, seq, layer, 1000 + tensor])
    u = rng.standard_normal((d_kv, shared_rank))
    energy = float((x[: min(n_tokens, 8192)] ** 2).mean())
    u_t = torch.from_numpy((u * math.sqrt(shared_frac * energy / shared_rank)).astype(np.float32)).to(device)
    gen = torch.Generator(device=device)
    gen.manual_seed(((seed * 1000003 + w.wid) * 1000003 + layer) * 4 + tensor + 7919)
    step = 16384
    for t0 in range(0, n_tokens, step):
        t1 = min(n_tokens, t0 + step)
        z = torch.randn((t1 - t0, shared_rank), generator=gen, device=device, dtype=torch.float32)
        x[t0:t1] += z @ u_t.T
    dt = torch.float32 if w.dtype == "f32" else torch.bfloat16
    return x.to(dt).unsqueeze(0)
