"""Batched verification on the wide-row GEMM (more than 16 rows, bf16).

Every tiling of the wide-row engine (1, 2 or 3 sixteen-row tiles per
workgroup with 1 weight panel per wave, 1 or 2 with 2 panels, and the
per-launch choice), each with the O and down projections unsplit or cut
into 2 or 4 k-splits, must give bit-for-bit the logits, n_accepted and
corrections of the skinny engine run once per 32 rows: all sum each dot
product over the same eight k-ranges in the same order.  The mini shape's O
projection has 4 k-blocks (empty k-ranges, splits without k-blocks) and its
down projection 11.  The per-launch choice is also compared with the oracle
to the usual bar, at 35 rows (B=5, gamma 6) and at 144 rows (B=16, gamma 8,
the batched-serving shape).
"""

import numpy as np
import pytest

from synth import ModelWeights, make_inputs, mini_workloads
from tests.helpers import LOGIT_TOL, compare, gpu_prefill, gpu_setup, gpu_verify, oracle_run

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _wide_workloads():
    base = {w.name: w for w in mini_workloads()}["mini_bf16_wide_b5"]
    return [base, base.with_(name="mini_bf16_wide_b16", batch=16, gamma=8, ctx=(20, 600), seed=2016)]


@pytest.mark.parametrize("w", _wide_workloads(), ids=lambda w: w.name)
def test_wide_tilings_bit_identical_and_match_oracle(w):
    weights = ModelWeights(w.model, w.seed)
    inp = make_inputs(w)
    orun = oracle_run(w, inp, weights=weights)  # also completes the chain drafts
    model, kv = gpu_setup(w, weights)
    gpu_prefill(kv, inp)
    runs = {}
    for tiles in ((-1, 0), (1, 1), (2, 1), (3, 1), (1, 2), (2, 2), (3, 2), (0, 0)):
        for ks in ((0,) if tiles[0] < 0 else (1, 2, 4, 0)):
            print(f"[{w.name}] M={w.batch * (w.gamma + 1)} wide (row tiles, panels) {tiles} k-splits {ks}",
                  flush=True)
            model.set_wide_tiles(*tiles)
            model.set_wide_k_splits(ks)
            runs[tiles + (ks,)] = gpu_verify(model, kv, inp)[:3]
    ref = runs[(-1, 0, 0)]
    for cfg, (lg, n, c) in runs.items():
        assert np.array_equal(lg.view(np.uint32), ref[0].view(np.uint32)), cfg
        assert np.array_equal(n, ref[1]) and np.array_equal(c, ref[2]), cfg
    p = compare(orun, *runs[(0, 0, 0)])
    print(f"[{w.name}] logit err {p.logit_err:.2e}, n {runs[(0, 0, 0)][1].tolist()}", flush=True)
    assert p.logit_err < LOGIT_TOL[w.model.weight_dtype]
    assert not p.stable_n_fail and not p.stable_corr_fail, p
    assert model.device_error() == 0



@pytest.mark.parametrize("batch", [1, 6])
def test_attention_merges_bit_identical_and_vs_oracle(batch):
    """The verify attention (one 256-key chunk per workgroup) with its chunk
    partials merged by the last chunk workgroup to finish, in a second launch,
    and by the per-call choice gives bit-for-bit the same logits, n_accepted
    and corrections (every chunk's partial and the chunk-order merge are the
    same whichever workgroup runs them), and matches the oracle.  Contexts up
    to 2100 keys (9 chunks); batch 1 runs the skinny projections, batch 6 the
    wide-row ones."""
    base = {w.name: w for w in mini_workloads()}["mini_bf16_wide_b5"]
    w = base.with_(name=f"mini_bf16_long_b{batch}", batch=batch, gamma=4,
                   ctx=(2000, 2100) if batch == 1 else (90, 2100), mode="greedy", draft_recipe="random",
                   seed=2018 + batch)
    weights = ModelWeights(w.model, w.seed)
    inp = make_inputs(w)
    orun = oracle_run(w, inp, weights=weights)
    model, kv = gpu_setup(w, weights)
    kv.prefill_batch(inp.prompts)
    from paper_2608_13076_amd import spade
    for bad in (-1, 3, 8):
        with pytest.raises(spade.SpadeError):
            model.set_wide_k_splits(bad)
    for bad in (-1, 3):
        with pytest.raises(spade.SpadeError):
            model.set_attn_merge(bad)
    runs = {}
    for merge in (1, 2, 0, 1):
        print(f"[{w.name}] lens {inp.lens.tolist()} attention merge {merge}", flush=True)
        model.set_attn_merge(merge)
        runs[merge] = gpu_verify(model, kv, inp)[:3]
    ref = runs[1]
    assert np.isfinite(ref[0]).all()
    for cfg, (lg, n, c) in runs.items():
        assert np.array_equal(lg.view(np.uint32), ref[0].view(np.uint32)), cfg
        assert np.array_equal(n, ref[1]) and np.array_equal(c, ref[2]), cfg
    p = compare(orun, *runs[2])
    print(f"[{w.name}] vs oracle: logit err {p.logit_err:.2e}, stable n/corr {p.stable_n}/{p.stable_corr}, "
          f"excluded n/corr {p.excluded_n}/{p.excluded_corr}", flush=True)
    assert p.logit_err < LOGIT_TOL[w.model.weight_dtype]
    assert not p.stable_n_fail and not p.stable_corr_fail, p
    assert model.device_error() == 0


@pytest.mark.parametrize("gamma,kv_heads", [(6, 2), (11, 2), (2, 2), (6, 4), (15, 4)])
def test_grouped_attention_bit_identical(gamma, kv_heads):
    """Grouped-query chunks (one workgroup computes a chunk for all G query
    heads of a K/V head, the G (gamma+1) rows packed into one to three 16-row
    tiles) give the per-head chunks' logits, n_accepted and corrections bit
    for bit, with the second-launch merge forced so both run: G = 4 and 2,
    rows per request 3 to 16, one to three tiles; both match the oracle."""
    import dataclasses
    base = {w.name: w for w in mini_workloads()}["mini_gqa_mixed_b5"]
    w = base.with_(name=f"mini_gqa_g{gamma}_kvh{kv_heads}", model=dataclasses.replace(base.model, n_kv_heads=kv_heads),
                   gamma=gamma, seed=3000 + gamma + kv_heads)
    weights = ModelWeights(w.model, w.seed)
    inp = make_inputs(w)
    orun = oracle_run(w, inp, weights=weights)  # also fills the chain drafts of inp
    model, kv = gpu_setup(w, weights)
    kv.prefill_batch(inp.prompts)
    from paper_2608_13076_amd import spade
    with pytest.raises(spade.SpadeError):
        model.set_attn_grouped(2)
    model.set_attn_merge(2)
    runs = {}
    for grouped in (1, 0):
        print(f"[{w.name}] lens {inp.lens.tolist()} grouped attention mode {grouped}", flush=True)
        model.set_attn_grouped(grouped)
        runs[grouped] = gpu_verify(model, kv, inp)[:3]
    a, b = runs[1], runs[0]
    assert np.isfinite(a[0]).all()
    assert np.array_equal(a[0].view(np.uint32), b[0].view(np.uint32))
    assert np.array_equal(a[1], b[1]) and np.array_equal(a[2], b[2])
    # and the grouped chunks against the oracle
    p = compare(orun, *b)
    print(f"[{w.name}] grouped vs oracle: logit err {p.logit_err:.2e}, stable n/corr {p.stable_n}/"
          f"{p.stable_corr}, excluded n/corr {p.excluded_n}/{p.excluded_corr}", flush=True)
    assert p.logit_err < LOGIT_TOL[w.model.weight_dtype]
    assert not p.stable_n_fail and not p.stable_corr_fail, p
    assert model.device_error() == 0
