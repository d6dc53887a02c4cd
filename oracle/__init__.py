"""CPU oracle for the SPECTRA KV-cache codec hot path.

TEST INFRASTRUCTURE ONLY. Nothing in the product path imports this package:
only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may call it. It is a plain, slow, obviously-correct numpy
implementation in float64 written from the paper, and it shares no code,
tables or helpers with the HIP library.

Every function is pinned by ``tests/test_oracle_pins.py`` against values the
mathematics fixes (closed forms, identities, brute force, hand-built records).
"""
from .codec import (  # noqa: F401
    Params, FitResult, record_budget_bits, record_words, split_budget,
    fit, fit_from_weights, latent_scale_factors, allocate_bits, allocate_bits_bruteforce,
    quantize, quantize_given_meta, dequantize, pack, unpack, physical_index, encode, decode,
    attention_mode_a, attention_mode_a_rope, rope, attention_mode_b, softmax_f64, fp16_rne_sat, fp16_bits,
    f16_bits_to_f64,
)
