"""ctypes loader for libspectra.so (built in-tree by ``build.py``).

The library is required: every entry point raises ``LibraryMissing`` if the
shared object has not been built. There is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "lib", "libspectra.so")


class LibraryMissing(RuntimeError):
    pass


class SpectraError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"spectra status {status}: {msg}")
        self.status = status


class spectra_params(ctypes.Structure):
    _fields_ = [("head_dim", ctypes.c_int32), ("group_size", ctypes.c_int32), ("b_max", ctypes.c_int32),
                ("meta_bits", ctypes.c_int32), ("centered", ctypes.c_int32), ("ratio", ctypes.c_double),
                ("budget_bits", ctypes.c_int32)]


class spectra_codec(ctypes.Structure):
    _fields_ = [("p", spectra_params), ("n_streams", ctypes.c_int64), ("record_words", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("basis", ctypes.c_void_p), ("mean", ctypes.c_void_p),
                ("var", ctypes.c_void_p), ("bits", ctypes.c_void_p), ("lscale", ctypes.c_void_p)]


_P = ctypes.c_void_p
_I32, _I64, _F32, _SZ = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_size_t
_PP = ctypes.POINTER(spectra_params)
_PC = ctypes.POINTER(spectra_codec)

_SIGNATURES = {
    "spectra_codec_init": (_I32, [_PC, _PP, _I64]),
    "spectra_layer_attention_workspace_bytes": (_SZ, [_PC, _I32, _I32, _I64]),
    "spectra_layer_decode_attention": (_I32, [_PC, _PC, _P, _P, _I64, _I64, _P, _I32, _I32, _I32, _I32, _F32, _P, _P,
                                              _SZ, _P]),
    "spectra_record_budget_bits": (_I32, [_PP]),
    "spectra_record_words": (_I32, [_PP]),
    "spectra_split_budget": (_I32, [_PP, ctypes.c_double, _PP, _PP]),
    "spectra_packed_words": (_I64, [_PC, _I64]),
    "spectra_fit_workspace_bytes": (_SZ, [_PC, _I64]),
    "spectra_fit_basis": (_I32, [_PC, _P, _I32, _I64, _I64, _I64, _P, _SZ, _P]),
    "spectra_fit_weights_workspace_bytes": (_SZ, [_PC, _I32]),
    "spectra_fit_weights": (_I32, [_PC, _P, _I32, _P, _P, _I32, _P, _SZ, _P]),
    "spectra_encode": (_I32, [_PC, _P, _I32, _I64, _I64, _I64, _I64, _P, _I64, _P]),
    "spectra_decode": (_I32, [_PC, _P, _I64, _I64, _I64, _P, _P]),
    "spectra_attention_workspace_bytes": (_SZ, [_I32, _I32, _I32, _I64]),
    "spectra_decode_attention": (_I32, [_PC, _PC, _P, _P, _I64, _I64, _P, _I32, _I32, _I32, _I32, _F32, _P, _P,
                                        _SZ, _P]),
    "spectra_decode_attention_rope": (_I32, [_PC, _PC, _P, _P, _I64, _I64, _P, _I32, _I32, _I32, _I32, _F32, _P, _I64,
                                              _P, _P, _SZ, _P]),
    "spectra_decode_step": (_I32, [_PC, _PC, _P, _P, _I64, _I64, _P, _P, _I32, _P, _I32, _I32, _I32, _I32, _F32,
                                   _P, _P, _SZ, _P]),
    "spectra_decode_step_static": (_I32, [_PC, _PC, _P, _P, _I64, _I64, _P, _P, _I32, _P, _I32, _I32, _I32, _I32,
                                          _F32, _P, _P]),
    "spectra_allocate_bits": (_I32, [_P, _PP, _P]),
    "spectra_eigh_host": (_I32, [_P, _I32, _P, _P]),
    "spectra_fit_from_moments_host": (_I32, [_PP, _I64, _P, _P, _P, _P, _P, _P]),
    "spectra_pack_codes": (_I32, [_PC, _P, _P, _I64, _P, _I64, _P]),
    "spectra_unpack_codes": (_I32, [_PC, _P, _I64, _I64, _P, _P, _P]),
    "spectra_status_string": (ctypes.c_char_p, [_I32]),
    "spectra_last_error": (ctypes.c_char_p, []),
}

_lib = None


def get():
    """The loaded library; raises LibraryMissing if it was not built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise LibraryMissing(f"{LIB_PATH} is not built; run `python -c 'import __graft_entry__ as g; g.build()'`")
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def check(status: int) -> None:
    if status != 0:
        lib = get()
        raise SpectraError(status, lib.spectra_last_error().decode(errors="replace"))
