"""Medium-M projection GEMM (144 rows per workgroup, k-split) against the
wide-row GEMM.

Every engine sums a dot product over the same eight k-ranges in the same
order, so a verify call must give bit-identical logits and decisions whichever
engine runs its projections: here the medium-M engine forced onto calls of
35 rows (five requests of gamma + 1 = 7; k-blocks fewer than the eight ranges,
so some ranges and some k-splits are empty) with every k-split count, and at
its own size, 144 rows (sixteen requests of nine), where the default picks it.
The wide-row engine these are compared with is checked against the oracle by
the parity tests.
"""

import numpy as np
import pytest

from synth import ModelWeights, make_inputs, mini_workloads
from tests.helpers import gpu_setup, gpu_verify

pytestmark = pytest.mark.gpu

MINIS = {w.name: w for w in mini_workloads()}


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _two_caches(w):
    from paper_2608_13076_amd import spade
    weights = ModelWeights(w.model, w.seed)
    inp = make_inputs(w)
    prompts = [np.asarray(p) for p in inp.prompts]
    max_len = max(len(p) for p in prompts) + 2 * (w.gamma + 1) + 24
    model, kv1 = gpu_setup(w, weights, max_len=max_len)
    kv2 = spade.KVCache(model, w.batch, max_len)
    model.set_mid_gemm(1)
    kv1.prefill_batch(prompts)
    kv2.prefill_batch(prompts)
    return model, kv1, kv2, inp


def _same(r1, r2, what):
    diff = r1[0].view(np.uint32) != r2[0].view(np.uint32)
    assert not diff.any(), f"{what}: {int(diff.sum())} of {diff.size} logits differ, rows {np.argwhere(diff.any(-1))[:8].tolist()}"
    assert np.array_equal(r1[1], r2[1]) and np.array_equal(r1[2], r2[2]), what


@pytest.mark.parametrize("name", ["mini_bf16_wide_b5", "mini_gqa_mixed_b5"])
def test_mid_gemm_forced_bit_identical(name):
    """35 rows: the medium-M engine forced, k-splits 1, 2, 3, 5, 8 and the
    chosen count, against the wide-row engine; the caches written by its QKV
    epilogue are compared through a second verify call."""
    w = MINIS[name]
    model, kv1, kv2, inp = _two_caches(w)
    model.set_mid_gemm(1)
    ref = gpu_verify(model, kv1, inp)
    for ks in (1, 2, 3, 5, 8, 0):
        model.set_mid_gemm(2, ks)
        got = gpu_verify(model, kv2, inp)
        _same(ref, got, f"k-splits {ks}")
        assert model.device_error() == 0, f"k-splits {ks}"
    model.set_mid_gemm(0)


def test_mid_gemm_144_rows_bit_identical():
    """Sixteen requests of gamma + 1 = 9 rows (144, the engine's default
    range) on the wide mini shape: the default against the wide-row engine,
    then k-splits 1 and 4, then a second round of verify calls on caches whose
    new rows each engine's QKV epilogue wrote."""
    w = MINIS["mini_bf16_wide_b5"].with_(batch=16, gamma=8, ctx=(20, 400), seed=2011)
    model, kv1, kv2, inp = _two_caches(w)
    model.set_mid_gemm(1)
    ref = gpu_verify(model, kv1, inp)
    model.set_mid_gemm(0)
    got = gpu_verify(model, kv2, inp)
    _same(ref, got, "default")
    for ks in (1, 4):
        model.set_mid_gemm(2, ks)
        _same(ref, gpu_verify(model, kv2, inp), f"k-splits {ks}")
    assert model.device_error() == 0
    model.set_mid_gemm(0)


def test_mid_gemm_setter_rejects_bad_values():
    from paper_2608_13076_amd import spade
    w = MINIS["mini_bf16_mixed"]
    model, _ = gpu_setup(w)
    for mode, ks in ((3, 0), (-1, 0), (0, 9), (0, -1)):
        with pytest.raises(spade.SpadeError):
            model.set_mid_gemm(mode, ks)
    model.set_mid_gemm(0, 0)
