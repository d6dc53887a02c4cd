"""SPECTRA KV-cache codec hot path for AMD MI355X (gfx950).

The codec (fit, encode, decode, decode-step attention from the packed cache)
runs in libspectra.so, hand-written HIP kernels behind a C ABI
(``include/spectra.h``). This package is a thin ctypes binding; torch supplies
device memory and streams.
"""
from ._lib import LibraryMissing, SpectraError, LIB_PATH  # noqa: F401
from .codec import (  # noqa: F401
    BF16, F32, Codec, Params,
    spectra_allocate_bits, spectra_attention_workspace_bytes, spectra_decode, spectra_decode_attention,
    spectra_decode_attention_rope, spectra_decode_step, spectra_decode_step_static,
    spectra_eigh_host, spectra_encode, spectra_fit_basis, spectra_fit_from_moments_host,
    spectra_fit_weights, spectra_fit_weights_workspace_bytes, spectra_fit_workspace_bytes, spectra_pack_codes, spectra_record_budget_bits, spectra_record_words,
    spectra_split_budget, spectra_unpack_codes, spectra_layer_attention_workspace_bytes,
    spectra_layer_decode_attention,
)
