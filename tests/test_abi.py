"""The C ABI library without a GPU: it loads, exports every function the
header declares, sizes buffers as documented and rejects bad arguments on the
host before any device work."""

import ctypes
import os
import re

import pytest

from paper_2608_13076_amd import spade
from synth import workload

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    return spade.load_library()


def _declared():
    src = open(os.path.join(ROOT, "include", "spade.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(spade_[a-z_]+)\s*\(", src)))


def test_exports_every_declared_symbol(lib):
    names = _declared()
    assert len(names) >= 15
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(spade.EXPORTED)


def test_buffer_sizes(lib):
    for name in ("c1_tiny_greedy", "c2_7b_greedy", "c3_13b_sample", "c5_33b_commit"):
        m = workload(name).model
        cfg = spade.config_from(m)
        wb = lib.spade_weight_bytes(ctypes.byref(cfg))
        elt = 2 if m.weight_dtype == "bf16" else 4
        vpad = (m.vocab + 15) // 16 * 16
        mats = m.n_layers * (4 * m.d_model ** 2 + 3 * m.d_model * m.d_ffn) + (m.vocab + vpad) * m.d_model
        assert mats * elt <= wb <= mats * elt + (6 * m.n_layers + 8) * 256 + (2 * m.n_layers + 1) * m.d_model * 4
        kvb = lib.spade_kv_bytes(ctypes.byref(cfg), 4, 1000)
        kelt = 2 if m.kv_dtype == "bf16" else 4
        assert kvb >= 2 * m.n_layers * 4 * m.n_heads * 1000 * m.head_dim * kelt
        assert lib.spade_workspace_bytes(ctypes.byref(cfg), 4, 8, 1000) > 0
        assert lib.spade_workspace_bytes(ctypes.byref(cfg), 4, 16, 1000) == 0  # gamma + 1 > 16


def test_gqa_buffer_sizes(lib):
    m = workload("gqa_8b_greedy").model
    cfg = spade.config_from(m)
    assert cfg.n_kv_heads == 8
    wb = lib.spade_weight_bytes(ctypes.byref(cfg))
    d, f, v, dkv = m.d_model, m.d_ffn, m.vocab, m.kv_heads * m.head_dim
    vpad = (v + 15) // 16 * 16
    mats = m.n_layers * (2 * d * d + 2 * d * dkv + 3 * d * f) + (v + vpad) * d
    assert mats * 2 <= wb <= mats * 2 + (6 * m.n_layers + 8) * 256 + (2 * m.n_layers + 1) * d * 4
    # the cache holds the 8 K/V heads only
    kvb = lib.spade_kv_bytes(ctypes.byref(cfg), 2, 1024)
    assert 2 * m.n_layers * 2 * 8 * 1024 * m.head_dim * 2 <= kvb < 2 * m.n_layers * 2 * 9 * 1024 * m.head_dim * 2
    # 0 means one K/V head per query head; a non-divisor is rejected
    for kvh, ok in ((0, True), (32, True), (1, True), (3, False), (-1, False)):
        bad = m.__class__(**{**m.__dict__, "n_kv_heads": kvh})
        assert (lib.spade_weight_bytes(ctypes.byref(spade.config_from(bad))) > 0) == ok, kvh


def test_unsupported_configs(lib):
    base = workload("c2_7b_greedy").model
    for kw in (dict(head_dim=96, n_heads=32, d_model=3072), dict(d_model=4000, n_heads=40, head_dim=100),
               dict(d_ffn=11000), dict(vocab=1)):
        bad = base.__class__(**{**base.__dict__, **kw})
        assert lib.spade_weight_bytes(ctypes.byref(spade.config_from(bad))) == 0
        assert lib.spade_last_error().decode()


def test_host_validation_without_device(lib):
    cfg = spade.config_from(workload("c1_tiny_greedy").model)
    out = ctypes.c_void_p()
    assert lib.spade_model_create(ctypes.byref(cfg), None, None, 1, 4, 128, ctypes.byref(out)) == -1
    assert lib.spade_model_create(ctypes.byref(cfg), ctypes.c_void_p(256), ctypes.c_void_p(512), 1, 16, 128,
                                  ctypes.byref(out)) == -2
    assert lib.spade_model_create(ctypes.byref(cfg), ctypes.c_void_p(300), ctypes.c_void_p(512), 1, 4, 128,
                                  ctypes.byref(out)) == -1
    assert lib.spade_verify(None, None, 1, 4, None, None, None, None, 1.0, None, None, None, None) == -1
    assert lib.spade_kv_commit(None, 1, None, None, None) == -1
    assert lib.spade_prefill(None, None, 0, None, 3, None) == -1
    assert lib.spade_kv_create(None, None, 1, 8, None, None, ctypes.byref(out)) == -1
    assert "null" in lib.spade_last_error().decode()
