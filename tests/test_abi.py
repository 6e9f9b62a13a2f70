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


def _declared(header="spade.h"):
    src = open(os.path.join(ROOT, "include", header)).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(spade_[a-z_]+)\s*\(", src)))


def test_exports_every_declared_symbol(lib):
    names = _declared()
    assert len(names) >= 15
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(spade.EXPORTED)
    tuning = _declared("spade_tuning.h")
    for n in tuning:
        assert hasattr(lib, n), n
    assert set(tuning) == set(spade.EXPORTED_TUNING)
    assert not set(tuning) & set(names)


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
    assert lib.spade_model_set_wide_k_splits(None, 2) == -1
    assert lib.spade_model_set_attn_merge(None, 1) == -1
    assert lib.spade_model_set_correction_slices(None, 1) == -1
    assert lib.spade_model_set_attn_grouped(None, 1) == -1
    assert lib.spade_model_set_wide_tiles(None, 0, 0) == -1
    assert lib.spade_model_set_split_k(None, 0) == -1
    assert "null" in lib.spade_last_error().decode()


def test_wide_tiling_splits_narrow_projections(lib):
    """The wide-row tiling model cuts the down projection of the batched 7B
    shape (144 rows) and the O and down projections of the 33B shape (28
    rows) into k-splits -- their few panel groups would leave most compute
    units idle -- and never splits QKV, gate/up or the LM head.  The picks
    are the fastest tilings measured for those launches (7B O: 2 row tiles,
    no split; 7B down: 3 row tiles, 4 splits; 33B O and down: 2 row tiles,
    4 splits)."""
    want = {(144, "o"): (2, 1, 1), (144, "down"): (3, 1, 4), (28, "o"): (2, 1, 4), (28, "down"): (2, 1, 4)}
    for (M, d, F) in ((144, 4096, 11008), (28, 6656, 17920)):
        for kind, nu, K in (("o", d // 16, d), ("down", d // 16, F), ("qkv", 3 * d // 16, d),
                            ("gu", 2 * F // 16, d), ("lm", 2000, d)):
            rt, p, ks = spade.wide_tiling(kind, M, nu, K)
            assert 1 <= rt <= 3 and 1 <= p <= 2 and not (rt == 3 and p == 2)
            if kind in ("o", "down"):
                assert (rt, p, ks) == want[(M, kind)], (M, kind, rt, p, ks)
            else:
                assert ks == 1, (M, kind, rt, p, ks)
    # two k-splits only with at most two accumulators per lane
    for M in range(17, 257, 7):
        rt, p, ks = spade.wide_tiling("down", M, 256, 11008)
        assert ks != 2 or rt * p <= 2
    with pytest.raises(spade.SpadeError):
        spade.wide_tiling("o", 16, 256, 4096)
    with pytest.raises(spade.SpadeError):
        spade.wide_tiling("o", 64, 256, 4000)
