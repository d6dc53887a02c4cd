"""Thin Python binding of libspectra: argument marshalling only.

Torch tensors provide device memory and the current stream; every step of the
codec runs in the HIP library. Function names match the C ABI in
``include/spectra.h``.
"""
from __future__ import annotations

import ctypes
import dataclasses
from dataclasses import dataclass
from typing import Optional, Tuple

import numpy as np

from . import _lib
from ._lib import check, spectra_codec, spectra_params

F32, BF16 = 0, 1


@dataclass(frozen=True)
class Params:
    head_dim: int = 128
    group_size: int = 32
    b_max: int = 8
    meta_bits: int = 32
    centered: bool = False
    ratio: float = 8.0
    budget_bits: int = 0

    def c(self) -> spectra_params:
        return spectra_params(self.head_dim, self.group_size, self.b_max, self.meta_bits, int(self.centered),
                              float(self.ratio), int(self.budget_bits))

    @property
    def n_groups(self) -> int:
        return self.head_dim // self.group_size


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _need(ok: bool, msg: str) -> None:
    """Shape and size checks the C ABI cannot make (it sees pointers only): a
    mismatched tensor raises here instead of reaching a kernel."""
    if not ok:
        raise ValueError(msg)


def _device_rows(codec: "Codec", x, name: str, n: int) -> None:
    """x [n_streams, >= n, head_dim] on the device, unit stride along head_dim."""
    _need(x.is_cuda, f"{name} must be a device tensor")
    d = codec.params.head_dim
    _need(x.dim() == 3 and x.shape[0] == codec.n_streams and x.shape[2] == d,
          f"{name} must be [n_streams={codec.n_streams}, T, {d}], got {tuple(x.shape)}")
    _need(x.stride(2) == 1, f"{name} needs unit stride along head_dim")
    _need(0 <= n <= x.shape[1], f"n_tokens={n} exceeds {name}.shape[1]={x.shape[1]}")


def _packed_words(codec: "Codec", packed, t_capacity: int, name: str) -> None:
    import torch
    _need(packed.is_cuda and packed.dtype == torch.int32 and packed.is_contiguous(),
          f"{name} must be a contiguous int32 device tensor")
    need = codec.packed_words(t_capacity)
    _need(packed.numel() >= need, f"{name} holds {packed.numel()} words, the codec needs {need}")


def _attention_shapes(ck: "Codec", cv: "Codec", packed_k, packed_v, t_capacity: int, q, n_kv_heads: int, out):
    import torch
    _need(q.is_cuda and q.dim() == 3 and q.is_contiguous(), "q must be a contiguous device tensor [batch, n_q_heads, d]")
    batch, n_q_heads, d = q.shape
    _need(d == ck.params.head_dim == cv.params.head_dim, f"q has head_dim {d}")
    _need(n_kv_heads > 0 and n_q_heads % n_kv_heads == 0, f"n_q_heads={n_q_heads} is not a multiple of n_kv_heads={n_kv_heads}")
    _need(ck.n_streams == cv.n_streams == batch * n_kv_heads,
          f"codecs hold {ck.n_streams} / {cv.n_streams} streams, batch x n_kv_heads = {batch * n_kv_heads}")
    _packed_words(ck, packed_k, t_capacity, "packed_k")
    _packed_words(cv, packed_v, t_capacity, "packed_v")
    if out is not None:
        _need(out.is_cuda and out.dtype == torch.float32 and out.is_contiguous() and tuple(out.shape) == (batch, n_q_heads, d),
              f"out must be a contiguous float32 device tensor {(batch, n_q_heads, d)}")
    return batch, n_q_heads, d


def _stream(stream=None):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


class Codec:
    """Per-stream codec state (basis, mean, variances, group widths) in device memory."""

    def __init__(self, params: Params, n_streams: int, device="cuda", _views=None, latent_scale: bool = False):
        """latent_scale: cache the square-root split of the latent (Eq. gsvd; per-layer
        geometry only): the fit then also writes ``lscale`` [n_streams, d]."""
        import torch
        self.params = params
        self.n_streams = int(n_streams)
        if _views is None:
            d, nG = params.head_dim, params.n_groups
            self.basis = torch.zeros((n_streams, d, d), dtype=torch.float32, device=device)
            self.mean = torch.zeros((n_streams, d), dtype=torch.float32, device=device)
            self.var = torch.zeros((n_streams, d), dtype=torch.float32, device=device)
            self.bits = torch.zeros((n_streams, nG), dtype=torch.uint8, device=device)
            self.lscale = torch.ones((n_streams, d), dtype=torch.float32, device=device) if latent_scale else None
        else:
            self.basis, self.mean, self.var, self.bits, self.lscale = _views
        self.struct = spectra_codec()
        check(_lib.get().spectra_codec_init(ctypes.byref(self.struct), ctypes.byref(params.c()), self.n_streams))
        self.struct.basis = self.basis.data_ptr()
        self.struct.mean = self.mean.data_ptr()
        self.struct.var = self.var.data_ptr()
        self.struct.bits = self.bits.data_ptr()
        self.struct.lscale = self.lscale.data_ptr() if self.lscale is not None else None

    @property
    def record_words(self) -> int:
        return int(self.struct.record_words)

    def view(self, start: int, count: int) -> "Codec":
        """Codec over streams [start, start + count) sharing this codec's memory."""
        sl = slice(start, start + count)
        return Codec(self.params, count, _views=(self.basis[sl], self.mean[sl], self.var[sl], self.bits[sl],
                                                 self.lscale[sl] if self.lscale is not None else None))

    def packed_words(self, t_capacity: int) -> int:
        return int(_lib.get().spectra_packed_words(ctypes.byref(self.struct), int(t_capacity)))

    def empty_packed(self, t_capacity: int):
        import torch
        n = max(self.packed_words(t_capacity), 1)
        return torch.zeros(n, dtype=torch.int32, device=self.basis.device)


def spectra_record_words(params: Params) -> int:
    return int(_lib.get().spectra_record_words(ctypes.byref(params.c())))


def spectra_record_budget_bits(params: Params) -> int:
    return int(_lib.get().spectra_record_budget_bits(ctypes.byref(params.c())))


def spectra_split_budget(params: Params, kappa: float) -> Tuple[Params, Params]:
    """Key and value params for the asymmetric split kappa of the combined budget."""
    pk, pv = spectra_params(), spectra_params()
    check(_lib.get().spectra_split_budget(ctypes.byref(params.c()), ctypes.c_double(kappa), ctypes.byref(pk),
                                          ctypes.byref(pv)))
    return dataclasses.replace(params, budget_bits=int(pk.budget_bits)), \
        dataclasses.replace(params, budget_bits=int(pv.budget_bits))


def spectra_fit_workspace_bytes(codec: Codec, n_tokens: int) -> int:
    return int(_lib.get().spectra_fit_workspace_bytes(ctypes.byref(codec.struct), int(n_tokens)))


def spectra_fit_basis(codec: Codec, x, n_tokens: Optional[int] = None, workspace=None, stream=None) -> None:
    """Fit every stream of ``codec`` on x [n_streams, T, d] (device; strides from the tensor)."""
    import torch
    n = x.shape[1] if n_tokens is None else int(n_tokens)
    _device_rows(codec, x, "x", n)
    need = spectra_fit_workspace_bytes(codec, n)
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=x.device)
    check(_lib.get().spectra_fit_basis(ctypes.byref(codec.struct), x.data_ptr(), _dtype_code(x), n, x.stride(0),
                                       x.stride(1), workspace.data_ptr(), workspace.numel(), _stream(stream)))


def spectra_fit_weights_workspace_bytes(codec: Codec, d_model: int) -> int:
    return int(_lib.get().spectra_fit_weights_workspace_bytes(ctypes.byref(codec.struct), int(d_model)))


def spectra_fit_weights(codec: Codec, W, G, hbar=None, streams_per_layer: int = 1, workspace=None,
                        stream=None) -> None:
    """Fit every stream from weights: W [n_streams, d_model, d] fp32, G [layers, d_model, d_model]
    fp64, hbar [layers, d_model] fp64 or None (device tensors, contiguous)."""
    import torch
    d_model = int(W.shape[1])
    for t, dt in ((W, torch.float32), (G, torch.float64)) + (((hbar, torch.float64),) if hbar is not None else ()):
        if t.dtype != dt or not t.is_contiguous() or not t.is_cuda:
            raise ValueError("W must be contiguous float32, G and hbar contiguous float64, all on the device")
    spl = int(streams_per_layer)
    _need(spl > 0 and codec.n_streams % spl == 0, f"streams_per_layer={spl} must divide n_streams={codec.n_streams}")
    layers = codec.n_streams // spl
    _need(tuple(W.shape) == (codec.n_streams, d_model, codec.params.head_dim),
          f"W must be [{codec.n_streams}, d_model, {codec.params.head_dim}], got {tuple(W.shape)}")
    _need(tuple(G.shape) == (layers, d_model, d_model), f"G must be [{layers}, {d_model}, {d_model}], got {tuple(G.shape)}")
    _need(hbar is None or tuple(hbar.shape) == (layers, d_model), f"hbar must be [{layers}, {d_model}]")
    if workspace is None:
        workspace = torch.empty(spectra_fit_weights_workspace_bytes(codec, d_model), dtype=torch.uint8,
                                device=W.device)
    check(_lib.get().spectra_fit_weights(ctypes.byref(codec.struct), W.data_ptr(), d_model, G.data_ptr(),
                                         hbar.data_ptr() if hbar is not None else None, int(streams_per_layer),
                                         workspace.data_ptr(), workspace.numel(), _stream(stream)))


def spectra_encode(codec: Codec, x, t0: int, packed, t_capacity: int, n_tokens: Optional[int] = None,
                   stream=None) -> None:
    """Encode tokens x[:, i] of every stream into record slots t0 + i of ``packed``."""
    n = x.shape[1] if n_tokens is None else int(n_tokens)
    _device_rows(codec, x, "x", n)
    _packed_words(codec, packed, t_capacity, "packed")
    check(_lib.get().spectra_encode(ctypes.byref(codec.struct), x.data_ptr(), _dtype_code(x), x.stride(0),
                                    x.stride(1), int(t0), n, packed.data_ptr(), int(t_capacity), _stream(stream)))


def spectra_decode(codec: Codec, packed, t_capacity: int, t0: int, n_tokens: int, out=None, stream=None):
    """Reconstruct record slots [t0, t0 + n_tokens) of every stream -> float32 [n_streams, n_tokens, d]."""
    import torch
    _packed_words(codec, packed, t_capacity, "packed")
    shape = (codec.n_streams, int(n_tokens), codec.params.head_dim)
    if out is None:
        out = torch.empty(shape, dtype=torch.float32, device=packed.device)
    _need(out.is_cuda and out.dtype == torch.float32 and out.is_contiguous() and tuple(out.shape) == shape,
          f"out must be a contiguous float32 device tensor {shape}")
    check(_lib.get().spectra_decode(ctypes.byref(codec.struct), packed.data_ptr(), int(t_capacity), int(t0),
                                    int(n_tokens), out.data_ptr(), _stream(stream)))
    return out


def spectra_attention_workspace_bytes(batch: int, n_q_heads: int, n_kv_heads: int, n_tokens: int) -> int:
    return int(_lib.get().spectra_attention_workspace_bytes(batch, n_q_heads, n_kv_heads, int(n_tokens)))


def spectra_decode_attention(ck: Codec, cv: Codec, packed_k, packed_v, t_capacity: int, n_tokens: int, q,
                             n_kv_heads: int, softmax_scale: float = 0.0, out=None, workspace=None, stream=None):
    """One decode step over the packed caches: q [batch, n_q_heads, d] -> float32 [batch, n_q_heads, d]."""
    import torch
    batch, n_q_heads, d = _attention_shapes(ck, cv, packed_k, packed_v, t_capacity, q, n_kv_heads, out)
    if out is None:
        out = torch.empty((batch, n_q_heads, d), dtype=torch.float32, device=q.device)
    if workspace is None:
        need = spectra_attention_workspace_bytes(batch, n_q_heads, n_kv_heads, n_tokens)
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    check(_lib.get().spectra_decode_attention(ctypes.byref(ck.struct), ctypes.byref(cv.struct), packed_k.data_ptr(),
                                              packed_v.data_ptr(), int(t_capacity), int(n_tokens), q.data_ptr(),
                                              _dtype_code(q), batch, n_q_heads, int(n_kv_heads), float(softmax_scale),
                                              out.data_ptr(), workspace.data_ptr(), workspace.numel(),
                                              _stream(stream)))
    return out


def spectra_layer_attention_workspace_bytes(ck: Codec, batch: int, n_q_heads: int, n_tokens: int) -> int:
    return int(_lib.get().spectra_layer_attention_workspace_bytes(ctypes.byref(ck.struct), int(batch), int(n_q_heads),
                                                                   int(n_tokens)))


def spectra_layer_decode_attention(ck: Codec, cv: Codec, packed_k, packed_v, t_capacity: int, n_tokens: int, q,
                                   n_kv_heads: int, softmax_scale: float = 0.0, out=None, workspace=None, stream=None):
    """Decode-step attention over per-layer latents: codecs of the per-layer geometry
    (stream b = sequence b), q [batch, n_q_heads, 128] -> float32 [batch, n_q_heads, 128]."""
    import torch
    _need(q.is_cuda and q.dim() == 3 and q.is_contiguous() and q.shape[2] == 128,
          "q must be a contiguous device tensor [batch, n_q_heads, 128]")
    batch, n_q_heads, _ = q.shape
    _need(ck.params.head_dim == cv.params.head_dim == 128 * int(n_kv_heads),
          f"the codecs' latent width must be n_kv_heads x 128 = {128 * int(n_kv_heads)}")
    _need(n_q_heads % n_kv_heads == 0, f"n_q_heads={n_q_heads} is not a multiple of n_kv_heads={n_kv_heads}")
    _need(ck.n_streams >= batch and cv.n_streams >= batch, "the codecs hold fewer streams than sequences")
    _packed_words(ck, packed_k, t_capacity, "packed_k")
    _packed_words(cv, packed_v, t_capacity, "packed_v")
    if out is None:
        out = torch.empty((batch, n_q_heads, 128), dtype=torch.float32, device=q.device)
    _need(out.is_cuda and out.dtype == torch.float32 and out.is_contiguous() and tuple(out.shape) == (batch, n_q_heads, 128),
          f"out must be a contiguous float32 device tensor {(batch, n_q_heads, 128)}")
    if workspace is None:
        need = spectra_layer_attention_workspace_bytes(ck, batch, n_q_heads, n_tokens)
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    check(_lib.get().spectra_layer_decode_attention(ctypes.byref(ck.struct), ctypes.byref(cv.struct), packed_k.data_ptr(),
                                                    packed_v.data_ptr(), int(t_capacity), int(n_tokens), q.data_ptr(),
                                                    _dtype_code(q), batch, n_q_heads, int(n_kv_heads),
                                                    float(softmax_scale), out.data_ptr(), workspace.data_ptr(),
                                                    workspace.numel(), _stream(stream)))
    return out


def spectra_decode_attention_rope(ck: Codec, cv: Codec, packed_k, packed_v, t_capacity: int, n_tokens: int, q,
                                  n_kv_heads: int, inv_freq, q_position: Optional[int] = None, softmax_scale: float = 0.0,
                                  out=None, workspace=None, stream=None):
    """Decode-step attention for rotary models: keys reconstructed and rotated at their slot
    positions, the query at q_position (default n_tokens - 1); inv_freq: float32 [d/2] device."""
    import torch
    batch, n_q_heads, d = _attention_shapes(ck, cv, packed_k, packed_v, t_capacity, q, n_kv_heads, out)
    _need(inv_freq.is_cuda and inv_freq.dtype == torch.float32 and inv_freq.is_contiguous()
          and tuple(inv_freq.shape) == (d // 2,), f"inv_freq must be a contiguous float32 device tensor [{d // 2}]")
    pos = int(n_tokens) - 1 if q_position is None else int(q_position)
    if out is None:
        out = torch.empty((batch, n_q_heads, d), dtype=torch.float32, device=q.device)
    if workspace is None:
        need = spectra_attention_workspace_bytes(batch, n_q_heads, n_kv_heads, n_tokens)
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    check(_lib.get().spectra_decode_attention_rope(ctypes.byref(ck.struct), ctypes.byref(cv.struct),
                                                   packed_k.data_ptr(), packed_v.data_ptr(), int(t_capacity),
                                                   int(n_tokens), q.data_ptr(), _dtype_code(q), batch, n_q_heads,
                                                   int(n_kv_heads), float(softmax_scale), inv_freq.data_ptr(), pos,
                                                   out.data_ptr(), workspace.data_ptr(), workspace.numel(),
                                                   _stream(stream)))
    return out


def spectra_decode_step(ck: Codec, cv: Codec, packed_k, packed_v, t_capacity: int, t: int, k_new, v_new, q,
                        n_kv_heads: int, softmax_scale: float = 0.0, out=None, workspace=None, stream=None):
    """Append k_new, v_new [batch, n_kv_heads, d] at record slot t, then attend over slots [0, t]:
    q [batch, n_q_heads, d] -> float32 [batch, n_q_heads, d]."""
    import torch
    batch, n_q_heads, d = _attention_shapes(ck, cv, packed_k, packed_v, t_capacity, q, n_kv_heads, out)
    _need(k_new.is_cuda and v_new.is_cuda and k_new.is_contiguous() and v_new.is_contiguous(),
          "k_new and v_new must be contiguous device tensors")
    _need(k_new.dtype == v_new.dtype and tuple(k_new.shape) == tuple(v_new.shape) == (batch, n_kv_heads, d),
          f"k_new and v_new must be [{batch}, {n_kv_heads}, {d}] of one dtype")
    if out is None:
        out = torch.empty((batch, n_q_heads, d), dtype=torch.float32, device=q.device)
    if workspace is None:
        need = spectra_attention_workspace_bytes(batch, n_q_heads, n_kv_heads, t + 1)
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    check(_lib.get().spectra_decode_step(ctypes.byref(ck.struct), ctypes.byref(cv.struct), packed_k.data_ptr(),
                                         packed_v.data_ptr(), int(t_capacity), int(t), k_new.data_ptr(),
                                         v_new.data_ptr(), _dtype_code(k_new), q.data_ptr(), _dtype_code(q), batch,
                                         n_q_heads, int(n_kv_heads), float(softmax_scale), out.data_ptr(),
                                         workspace.data_ptr(), workspace.numel(), _stream(stream)))
    return out



def spectra_decode_step_static(ck: Codec, cv: Codec, packed_k, packed_v, t_capacity: int, t: int, k_new, v_new, q,
                               n_kv_heads: int, softmax_scale: float = 0.0, out=None, stream=None):
    """spectra_decode_step with the partials in the library's static device array (no
    workspace, nothing allocated by the library; `out` is allocated here only when not
    given). Calls that overlap on one GPU race."""
    import torch
    batch, n_q_heads, d = _attention_shapes(ck, cv, packed_k, packed_v, t_capacity, q, n_kv_heads, out)
    _need(k_new.is_cuda and v_new.is_cuda and k_new.is_contiguous() and v_new.is_contiguous(),
          "k_new and v_new must be contiguous device tensors")
    _need(k_new.dtype == v_new.dtype and tuple(k_new.shape) == tuple(v_new.shape) == (batch, n_kv_heads, d),
          f"k_new and v_new must be [{batch}, {n_kv_heads}, {d}] of one dtype")
    if out is None:
        out = torch.empty((batch, n_q_heads, d), dtype=torch.float32, device=q.device)
    check(_lib.get().spectra_decode_step_static(ctypes.byref(ck.struct), ctypes.byref(cv.struct), packed_k.data_ptr(),
                                                packed_v.data_ptr(), int(t_capacity), int(t), k_new.data_ptr(),
                                                v_new.data_ptr(), _dtype_code(k_new), q.data_ptr(), _dtype_code(q),
                                                batch, n_q_heads, int(n_kv_heads), float(softmax_scale),
                                                out.data_ptr(), _stream(stream)))
    return out

def spectra_pack_codes(codec: Codec, codes, meta, packed, t_capacity: int, stream=None) -> None:
    import torch
    n = codes.shape[1]
    _need(codes.is_cuda and codes.dtype == torch.uint8 and codes.is_contiguous()
          and tuple(codes.shape) == (codec.n_streams, n, codec.params.head_dim), "codes must be contiguous uint8 [S, n, d]")
    _need(meta.is_cuda and meta.dtype == torch.int32 and meta.is_contiguous()
          and tuple(meta.shape) == (codec.n_streams, n, codec.params.n_groups), "meta must be contiguous int32 [S, n, d/g]")
    _packed_words(codec, packed, t_capacity, "packed")
    check(_lib.get().spectra_pack_codes(ctypes.byref(codec.struct), codes.data_ptr(), meta.data_ptr(),
                                        codes.shape[1], packed.data_ptr(), int(t_capacity), _stream(stream)))


def spectra_unpack_codes(codec: Codec, packed, t_capacity: int, n_tokens: int, stream=None):
    import torch
    _packed_words(codec, packed, t_capacity, "packed")
    dev = packed.device
    codes = torch.empty((codec.n_streams, n_tokens, codec.params.head_dim), dtype=torch.uint8, device=dev)
    meta = torch.empty((codec.n_streams, n_tokens, codec.params.n_groups), dtype=torch.int32, device=dev)
    check(_lib.get().spectra_unpack_codes(ctypes.byref(codec.struct), packed.data_ptr(), int(t_capacity),
                                          int(n_tokens), codes.data_ptr(), meta.data_ptr(), _stream(stream)))
    return codes, meta


# ---------------------------------------------------------------------------
# Host-only entry points (numpy in, numpy out)
# ---------------------------------------------------------------------------
def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def spectra_allocate_bits(var, params: Params) -> np.ndarray:
    v = np.ascontiguousarray(var, dtype=np.float64)
    out = np.zeros(params.n_groups, dtype=np.uint8)
    check(_lib.get().spectra_allocate_bits(_ptr(v), ctypes.byref(params.c()), _ptr(out)))
    return out


def spectra_eigh_host(a) -> tuple:
    a = np.ascontiguousarray(a, dtype=np.float64)
    n = a.shape[0]
    w = np.zeros(n)
    v = np.zeros((n, n))
    check(_lib.get().spectra_eigh_host(_ptr(a), n, _ptr(w), _ptr(v)))
    return w, v


def spectra_fit_from_moments_host(params: Params, n_tokens: int, gram, colsum) -> tuple:
    d = params.head_dim
    gram = np.ascontiguousarray(gram, dtype=np.float64)
    colsum = np.ascontiguousarray(colsum, dtype=np.float64)
    basis = np.zeros((d, d), dtype=np.float32)
    mean = np.zeros(d, dtype=np.float32)
    var = np.zeros(d, dtype=np.float64)
    bits = np.zeros(params.n_groups, dtype=np.uint8)
    check(_lib.get().spectra_fit_from_moments_host(ctypes.byref(params.c()), int(n_tokens), _ptr(gram), _ptr(colsum),
                                                   _ptr(basis), _ptr(mean), _ptr(var), _ptr(bits)))
    return basis, mean, var, bits
