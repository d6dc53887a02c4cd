"""CPU tests of libspectra: it loads, exports every declared symbol, and its
host-side pieces (allocation, eigensolver, fit from moments, argument checks)
agree with the oracle. No GPU compute is called here."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle as O
import paper_2608_07915_amd as S
from paper_2608_07915_amd import _lib
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_lib.LIB_PATH):
        pytest.fail("libspectra.so is not built (run __graft_entry__.build())")
    return _lib.get()


def _declared_symbols():
    txt = open(os.path.join(ROOT, "include", "spectra.h")).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(spectra_[a-z_]+)\s*\(", txt)))


def test_library_exports_every_declared_symbol(lib):
    names = _declared_symbols()
    assert len(names) >= 17
    for n in names:
        assert hasattr(lib, n), n
    # and the binding wraps each of them
    assert set(names) <= set(_lib._SIGNATURES)


def _o2s(p: O.Params) -> S.Params:
    return S.Params(p.head_dim, p.group_size, p.b_max, p.meta_bits, p.centered, p.ratio, p.budget_bits)


def test_allocation_bit_exact_random(lib):
    rng = np.random.default_rng(2024)
    n = 0
    for i in range(10000):
        kind = i % 4
        if kind == 0:
            v = np.exp(rng.uniform(-10, 4, 128))
        elif kind == 1:
            v = np.sort(np.exp(rng.uniform(-6, 3, 128)))[::-1] * rng.uniform(0.1, 10)
        elif kind == 2:
            v = np.arange(1, 129, dtype=np.float64) ** -rng.uniform(0.5, 2.5)
        else:
            v = rng.uniform(0, 1, 128) * (rng.uniform(size=128) < 0.5)
        ratio = float(rng.choice([3.0, 4.0, 6.0, 8.0, 10.0, 12.0, 16.0, 16.0 / 9.0]))
        p = O.Params(ratio=ratio, b_max=int(rng.choice([4, 6, 8])))
        got = S.spectra_allocate_bits(v, _o2s(p)).tolist()
        assert got == O.allocate_bits(v, p), (i, ratio)
        n += 1
    assert n == 10000


def test_allocation_bit_exact_small_dims(lib):
    rng = np.random.default_rng(5)
    for i in range(400):
        g = int(rng.choice([1, 2, 4, 8]))
        meta = int(rng.choice([0, 32]))
        R = int(rng.integers(0, 300))
        p = O.Params(head_dim=8, group_size=g, meta_bits=meta, budget_bits=max(R, 1), b_max=int(rng.choice([4, 8])))
        v = np.exp(rng.uniform(-5, 3, 8))
        assert S.spectra_allocate_bits(v, _o2s(p)).tolist() == O.allocate_bits(v, p)


def test_allocation_on_workload_variances(lib):
    for name in ("tiny", "llama_layer_4x", "qwen_layer_8x", "llama_batch16_12x", "llama_model_131k_8x"):
        w = synth.WORKLOADS[name]
        for tensor in (0, 1):
            x = synth.numpy_stream(w, 0, 0, 1 % w.n_kv_heads, tensor, n_tokens=4096)
            x = x if w.dtype == "f32" else synth.bf16_bits_to_f32(x)
            f = O.fit(x, O.Params(ratio=w.ratio))
            for ratio in (4.0, 8.0, 12.0):
                p = O.Params(ratio=ratio)
                assert S.spectra_allocate_bits(f.var, _o2s(p)).tolist() == O.allocate_bits(f.var, p)


def test_eigh_host_matches_numpy(lib):
    rng = np.random.default_rng(3)
    for n in (1, 2, 5, 64, 128):
        a = rng.standard_normal((n, n))
        a = a @ a.T + np.diag(rng.uniform(0, 1, n))
        w, v = S.spectra_eigh_host(a)
        wn = np.linalg.eigvalsh(a)[::-1]
        assert np.allclose(w, wn, rtol=0, atol=1e-12 * wn[0])
        assert np.abs(v.T @ v - np.eye(n)).max() < 1e-12
        assert np.abs(a @ v - v * w[None, :]).max() < 1e-11 * wn[0]
        idx = np.argmax(np.abs(v), axis=0)
        assert np.all(v[idx, np.arange(n)] > 0)
    # repeated eigenvalues and a diagonal input
    w, v = S.spectra_eigh_host(np.diag([3.0, 1.0, 3.0, 2.0]))
    assert w.tolist() == [3.0, 3.0, 2.0, 1.0]
    assert np.abs(np.abs(v) - np.abs(v).round()).max() < 1e-15


@pytest.mark.parametrize("tensor,centered", [(0, False), (1, False), (0, True)])
def test_fit_from_moments_matches_oracle(lib, tensor, centered):
    x = synth.numpy_stream(synth.WORKLOADS["tiny"], 0, 0, 0, tensor).astype(np.float64)
    op = O.Params(ratio=8.0, centered=centered)
    f = O.fit(x, op)
    basis, mean, var, bits = S.spectra_fit_from_moments_host(_o2s(op), x.shape[0], x.T @ x, x.sum(axis=0))
    # same directions (sign convention included) up to fp32 rounding where eigen-gaps are clear
    gap = np.minimum(np.abs(np.diff(f.eigvals, prepend=np.inf)), np.abs(np.diff(f.eigvals, append=-np.inf)))
    clear = gap > 1e-6 * f.eigvals[0]
    assert np.abs(basis - f.basis)[:, clear].max() <= 1e-5
    assert np.allclose(var, f.var, rtol=1e-6, atol=1e-12 * f.var.max())  # fp32 basis ulps
    assert np.abs(mean - f.mean).max() <= 1e-5 * np.abs(f.mean).max()
    assert bits.tolist() == O.allocate_bits(f.var, op)


def test_record_geometry(lib):
    for ratio, W in ((4.0, 16), (8.0, 8), (12.0, 5), (16.0 / 9.0, 36)):
        assert S.spectra_record_words(S.Params(ratio=ratio)) == W == O.record_words(O.Params(ratio=ratio))
    assert S.spectra_record_budget_bits(S.Params(budget_bits=1152)) == 1152


def test_argument_errors_return_before_any_launch(lib):
    c = _lib.spectra_codec()
    bad = S.Params(group_size=48).c()
    assert lib.spectra_codec_init(ctypes.byref(c), ctypes.byref(bad), 4) == -1
    assert b"group_size" in lib.spectra_last_error()
    ok = S.Params().c()
    assert lib.spectra_codec_init(ctypes.byref(c), ctypes.byref(ok), 4) == 0
    assert c.record_words == 8
    # null codec arrays -> EINVAL from encode / decode / attention, nothing launched
    assert lib.spectra_encode(ctypes.byref(c), None, 1, 0, 128, 0, 1, None, 64, None) == -1
    assert lib.spectra_decode(ctypes.byref(c), None, 64, 0, 1, None, None) == -1
    assert lib.spectra_decode_attention(ctypes.byref(c), ctypes.byref(c), None, None, 64, 1, None, 1, 1, 1, 1, 0.0,
                                        None, None, 0, None) == -1
    # head_dim other than 128 is host-only
    c2 = _lib.spectra_codec()
    p64 = S.Params(head_dim=64).c()
    assert lib.spectra_codec_init(ctypes.byref(c2), ctypes.byref(p64), 1) == 0
    c2.basis = c2.mean = c2.var = c2.bits = 256
    assert lib.spectra_encode(ctypes.byref(c2), 256, 1, 0, 128, 0, 1, 256, 64, None) == -2
    # slot range and t_capacity checks
    c.basis = c.mean = c.var = c.bits = 256
    assert lib.spectra_encode(ctypes.byref(c), 256, 1, 0, 128, 60, 8, 256, 64, None) == -1
    assert b"exceed" in lib.spectra_last_error()
    assert lib.spectra_encode(ctypes.byref(c), 256, 1, 0, 128, 0, 8, 256, 100, None) == -1
    # misaligned input / bad strides
    assert lib.spectra_encode(ctypes.byref(c), 258, 1, 0, 128, 0, 8, 256, 64, None) == -1
    assert lib.spectra_encode(ctypes.byref(c), 256, 1, 0, 100, 0, 8, 256, 64, None) == -1
    # workspace too small
    assert lib.spectra_decode_attention(ctypes.byref(c), ctypes.byref(c), 256, 256, 64, 8, 256, 1, 1, 4, 4, 0.0,
                                        256, 256, 16, None) == -4
    assert lib.spectra_status_string(-4) == b"workspace too small"
    # decode step: slot outside the capacity, misaligned new rows, too-small workspace
    ws = lib.spectra_attention_workspace_bytes(1, 4, 4, 9)
    assert lib.spectra_decode_step(ctypes.byref(c), ctypes.byref(c), 256, 256, 64, 64, 256, 256, 1, 256, 1, 1, 4, 4,
                                   0.0, 256, 256, ws, None) == -1
    assert lib.spectra_decode_step(ctypes.byref(c), ctypes.byref(c), 256, 256, 64, 8, 264, 256, 1, 256, 1, 1, 4, 4,
                                   0.0, 256, 256, ws, None) == -1
    assert b"16-byte" in lib.spectra_last_error()
    assert lib.spectra_decode_step(ctypes.byref(c), ctypes.byref(c), 256, 256, 64, 8, 256, 256, 1, 256, 1, 1, 4, 4,
                                   0.0, 256, 256, 16, None) == -4
    # decode step on the static array: slot outside the capacity, partials beyond the
    # array's size (both refused before any device call)
    assert lib.spectra_decode_step_static(ctypes.byref(c), ctypes.byref(c), 256, 256, 64, 64, 256, 256, 1, 256, 1, 1,
                                          4, 4, 0.0, 256, None) == -1
    big_t = 1 << 26
    assert lib.spectra_attention_workspace_bytes(256, 4096, 256, big_t + 1) > 8 << 20
    assert lib.spectra_decode_step_static(ctypes.byref(c), ctypes.byref(c), 256, 256, big_t + 64, big_t, 256, 256, 1,
                                          256, 1, 256, 4096, 256, 0.0, 256, None) == -4
    assert b"static" in lib.spectra_last_error()
    # fit from weights: d_model, layer grouping, alignment, workspace (c holds 4 streams)
    need = lib.spectra_fit_weights_workspace_bytes(ctypes.byref(c), 256)
    assert need == 4 * (128 * 128 + 128) * 8 + 4 * 256 * 128 * 8
    assert lib.spectra_fit_weights(ctypes.byref(c), 256, 200, 256, None, 1, 256, need, None) == -1
    assert b"multiple of 64" in lib.spectra_last_error()
    assert lib.spectra_fit_weights(ctypes.byref(c), 256, 256, 256, None, 3, 256, need, None) == -1
    assert b"streams_per_layer" in lib.spectra_last_error()
    assert lib.spectra_fit_weights(ctypes.byref(c), None, 256, 256, None, 1, 256, need, None) == -1
    assert lib.spectra_fit_weights(ctypes.byref(c), 256, 256, 260, None, 1, 256, need, None) == -1
    assert lib.spectra_fit_weights(ctypes.byref(c), 256, 256, 256, None, 2, 256, need - 8, None) == -4


def test_binding_fails_loudly_without_library(monkeypatch):
    monkeypatch.setattr(_lib, "_lib", None)
    monkeypatch.setattr(_lib, "LIB_PATH", "/nonexistent/libspectra.so")
    with pytest.raises(_lib.LibraryMissing):
        S.spectra_allocate_bits(np.ones(128), S.Params())


def test_layer_geometry_argument_errors(lib):
    # the per-layer geometry (d = heads x 128, groups of 64): accepted by fit / encode /
    # decode / layer attention only, checked on the host before anything is launched
    cl = _lib.spectra_codec()
    pl = S.Params(head_dim=1024, group_size=64, ratio=8.0).c()
    assert lib.spectra_codec_init(ctypes.byref(cl), ctypes.byref(pl), 2) == 0
    assert cl.record_words == 64
    cl.basis = cl.mean = cl.var = cl.bits = 256
    # the fit from weights takes it: products of d_kv-wide projections in the workspace
    assert lib.spectra_fit_weights_workspace_bytes(ctypes.byref(cl), 4096) == (2 * (1024 * 1024 + 1024) * 8
                                                                                + 2 * 4096 * 1024 * 8)
    # the per-head entry points refuse it
    assert lib.spectra_decode_attention(ctypes.byref(cl), ctypes.byref(cl), 256, 256, 64, 8, 256, 1, 1, 8, 8, 0.0,
                                        256, 256, 1 << 20, None) == -2
    assert b"per-layer geometry" in lib.spectra_last_error()
    # 1024-wide records beyond 128 words are not run on the GPU
    c4 = _lib.spectra_codec()
    p4 = S.Params(head_dim=1024, group_size=64, ratio=2.0).c()
    assert lib.spectra_codec_init(ctypes.byref(c4), ctypes.byref(p4), 1) == 0
    c4.basis = c4.mean = c4.var = c4.bits = 256
    assert lib.spectra_decode(ctypes.byref(c4), 256, 64, 0, 8, 256, None) == -2
    # encode takes bf16 tokens only in this geometry; fp32 is refused
    assert lib.spectra_encode(ctypes.byref(cl), 256, 0, 8192, 1024, 0, 8, 256, 64, None) == -2
    # layer attention: kv heads x 128 must equal the width, at most 32 query heads, workspace
    ws = lib.spectra_layer_attention_workspace_bytes(ctypes.byref(cl), 1, 32, 100)
    assert ws > 0
    args = lambda n_q, n_kv, wsb: (ctypes.byref(cl), ctypes.byref(cl), 256, 256, 128, 100, 256, 1, 1, n_q, n_kv, 0.0,
                                   256, 256, wsb, None)
    assert lib.spectra_layer_decode_attention(*args(32, 4, ws)) == -1
    assert lib.spectra_layer_decode_attention(*args(48, 8, ws)) == -1
    assert lib.spectra_layer_decode_attention(*args(32, 8, 1024)) == -4
    # the square-root split belongs to the per-layer geometry
    ch = _lib.spectra_codec()
    assert lib.spectra_codec_init(ctypes.byref(ch), ctypes.byref(S.Params().c()), 1) == 0
    ch.basis = ch.mean = ch.var = ch.bits = ch.lscale = 256
    assert lib.spectra_decode(ctypes.byref(ch), 256, 64, 0, 8, 256, None) == -2
    assert b"square-root" in lib.spectra_last_error()
