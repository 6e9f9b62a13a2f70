"""Stale and uninitialised cache rows, and the device error word.

Algorithm 1's context update (m <- m + k + 1) leaves the rejected drafts'
K/V rows in the cache past the new length; a fresh cache holds whatever the
allocation held.  Neither may change any result: a verify call reads only
positions below lens + gamma + 1 and masks the rest of its last chunk.  Here
every cache position is filled with NaN before the prefill and every
position at or past the committed length is filled with NaN again before the
second round; logits, n_accepted and corrections must equal, bit for bit, a
run on a zero-filled cache -- for each attention variant: the one-chunk
kernel with either merge, the grouped-query chunks, and the float32-cache
kernel.  Error paths forced from the host: a NaN gain flags
SPADE_DERR_NAN, an n_accepted outside [0, gamma] is clamped by the commit
and flags SPADE_DERR_COMMIT, a length written outside the library is clamped
and flags SPADE_DERR_CAPACITY.
"""

import numpy as np
import pytest

from synth import ModelWeights, make_inputs, mini_workloads
from tests.helpers import gpu_setup, gpu_verify, k_phys_index, kv_stride, kv_views, v_phys_index

pytestmark = pytest.mark.gpu

MINIS = {w.name: w for w in mini_workloads()}


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _views(kv, shape, max_len):
    """K and V as [layer][request][K/V head][region] over the cache buffer."""
    return kv_views(kv, shape, max_len)


def _nan_value(shape):
    return 0x7FC0 if shape.kv_dtype == "bf16" else float("nan")


def _two_rounds(w, weights, fill, merge, grouped):
    import torch
    from paper_2608_13076_amd import spade
    inp = make_inputs(w)
    max_len = int(inp.lens.max()) + 3 * (w.gamma + 1) + 8
    model, kv = gpu_setup(w, weights, max_len=max_len)
    model.set_attn_merge(merge)
    if w.model.kv_heads != w.model.n_heads:
        model.set_attn_grouped(grouped)
    k, v = _views(kv, w.model, max_len)
    vidx = v_phys_index(w.model, kv_stride(max_len))
    kidx = k_phys_index(w.model, kv_stride(max_len))
    if fill == "nan":
        k.fill_(_nan_value(w.model))
        v.fill_(_nan_value(w.model))
    else:
        kv.buf.zero_()
    kv.prefill_batch(inp.prompts)
    r1 = gpu_verify(model, kv, inp)
    buf = r1[3]
    kv.commit(buf.n, buf.corr)
    torch.cuda.synchronize()
    lens, _ = kv.get_state(w.batch)
    if fill == "nan":  # the rolled-back drafts' rows and everything after them
        for b in range(w.batch):
            kpast = torch.as_tensor(kidx[int(lens[b]):, :].reshape(-1), device=k.device)
            k[:, b, :, kpast] = _nan_value(w.model)
            past = torch.as_tensor(vidx[:, int(lens[b]):].reshape(-1), device=v.device)
            v[:, b, :, past] = _nan_value(w.model)
    inp2 = make_inputs(w, round_index=1)
    r2 = gpu_verify(model, kv, inp2)
    err = model.device_error()
    assert err == 0, (fill, err)
    assert isinstance(kv, spade.KVCache)
    return [r[:3] for r in (r1, r2)]


@pytest.mark.parametrize("name,merge,grouped", [
    ("mini_bf16_mixed", 1, 0),      # one-chunk kernel, merged by the last chunk to finish
    ("mini_bf16_mixed", 2, 0),      # one-chunk kernel, second-launch merge
    ("mini_bf16_wide_b5", 2, 0),    # wide-row projections, second-launch merge
    ("mini_gqa_mixed_b5", 2, 0),    # grouped-query chunks
    ("mini_gqa_mixed_b5", 2, 1),    # one workgroup per query head
    ("mini_f32_greedy", 0, 0),      # float32 cache, head_dim 64
])
def test_nan_poisoned_rows_change_nothing(name, merge, grouped):
    w = MINIS[name]
    weights = ModelWeights(w.model, w.seed)
    print(f"[{name}] merge {merge} grouped {grouped}: zero-filled cache", flush=True)
    ref = _two_rounds(w, weights, "zero", merge, grouped)
    print(f"[{name}] NaN-filled cache, NaN rows past the committed lengths", flush=True)
    got = _two_rounds(w, weights, "nan", merge, grouped)
    for rnd in range(2):
        assert np.isfinite(ref[rnd][0]).all()
        assert np.array_equal(got[rnd][0].view(np.uint32), ref[rnd][0].view(np.uint32)), rnd
        assert np.array_equal(got[rnd][1], ref[rnd][1]) and np.array_equal(got[rnd][2], ref[rnd][2]), rnd


def test_nan_gain_sets_nan_flag():
    """A NaN in the final RMSNorm gain makes every logit NaN: the LM head
    flags SPADE_DERR_NAN (NaN arithmetic does not trap)."""
    from paper_2608_13076_amd.spade import DERR_NAN
    w = MINIS["mini_bf16_greedy"]
    weights = ModelWeights(w.model, w.seed)
    inp = make_inputs(w)
    model, kv = gpu_setup(w, weights)
    g = weights.get("g_final").copy()
    g[3] = np.nan
    model.load_numpy("g_final", None, g)
    kv.prefill_batch(inp.prompts)
    gpu_verify(model, kv, inp)
    assert model.device_error() & DERR_NAN


def test_commit_clamps_and_flags():
    """spade_kv_commit clamps an n_accepted outside [0, gamma] of the last
    verify call (here a buffer the call did not write) and flags it; a commit
    without a verify since the last one is refused on the host."""
    import torch
    from paper_2608_13076_amd import spade
    w = MINIS["mini_bf16_mixed"]
    weights = ModelWeights(w.model, w.seed)
    inp = make_inputs(w)
    model, kv = gpu_setup(w, weights)
    kv.prefill_batch(inp.prompts)
    lens0, _ = kv.get_state(w.batch)
    _, n, c, buf = gpu_verify(model, kv, inp)
    assert model.device_error() == 0
    bad = torch.tensor([w.gamma + 5, -3, 0, w.gamma][: w.batch], dtype=torch.int32, device=model.device)
    kv.commit(bad, buf.corr)
    torch.cuda.synchronize()
    lens1, pend1 = kv.get_state(w.batch)
    expect = np.clip(bad.cpu().numpy(), 0, w.gamma) + 1
    np.testing.assert_array_equal(lens1, lens0 + expect)
    np.testing.assert_array_equal(pend1, c)
    assert model.device_error() & spade.DERR_COMMIT
    with pytest.raises(spade.SpadeError):
        kv.commit(buf.n, buf.corr)  # no verify since the last commit


def test_length_past_capacity_is_clamped_and_flagged():
    """A length written into the caller-owned lens array behind the library's
    back (so the host bound does not cover it) is clamped on the device
    before any cache access and the call is flagged SPADE_DERR_CAPACITY."""
    import torch
    from paper_2608_13076_amd import spade
    w = MINIS["mini_bf16_mixed"]
    weights = ModelWeights(w.model, w.seed)
    inp = make_inputs(w)
    max_len = int(inp.lens.max()) + 2 * (w.gamma + 1) + 8
    model, kv = gpu_setup(w, weights, max_len=max_len)
    kv.prefill_batch(inp.prompts)
    kv.lens[0] = max_len + 1000  # a value only the device sees
    torch.cuda.synchronize()
    gpu_verify(model, kv, inp)
    lens, _ = kv.get_state(w.batch)
    assert model.device_error() & spade.DERR_CAPACITY
    assert 0 <= lens[0] <= max_len - (w.gamma + 1)
