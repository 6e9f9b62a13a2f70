"""The stored-results generator (tests/golden/make_golden.py) on scaled-down
workloads: its layer-by-layer driver over several requests and rounds gives
what the oracle gives request by request -- verify, the context update
m <- m + k + 1, and a second verify whose chain drafts come from the
committed state (Algorithm 1, Cloud step)."""

from dataclasses import replace

import numpy as np

from oracle import Decoder, verify as oracle_verify
from oracle.speculative import _argmax_f32, commit
from synth import ModelWeights, make_inputs
from synth.configs import MINI_BF16, Workload
from tests.golden import make_golden
from tests.helpers import chain_drafts, complete_drafts

W2 = Workload("mini_two_rounds", replace(MINI_BF16, n_layers=1),
              batch=3, gamma=4, ctx=(9, 40), mode="greedy", draft_recipe="chain_half",
              rounds=2, seed=2099)


def _reference(w):
    weights = ModelWeights(w.model, w.seed)
    dec = Decoder(w.model, weights.get, keep_f64=True)
    inp = make_inputs(w)
    G = w.gamma
    out = []
    for b in range(w.batch):
        c = dec.new_cache(int(inp.lens.max()) + 3 * (G + 1) + 1)
        dec.prefill(c, inp.prompts[b][:-1])
        complete_drafts(dec, inp, {b: c}, requests=[b])
        r1 = oracle_verify(dec, c, inp.pending[b], inp.drafts[b], None, inp.uniforms[b], 0)
        pend = commit(c, r1)
        i2 = make_inputs(w, round_index=1)
        i2.pending[b] = pend
        cc, cur, chain = c.copy(), pend, []
        for _ in range(i2.chain_slots + 1):
            cur = _argmax_f32(dec.forward(cc, [cur])[0])
            chain.append(cur)
        chain_drafts(i2, b, chain)
        r2 = oracle_verify(dec, c, pend, i2.drafts[b], None, i2.uniforms[b], 0)
        out.append((r1, r2, i2.drafts[b].copy()))
    return out


def test_layer_major_two_rounds_equal_request_by_request():
    ref = _reference(W2)
    rounds, logits = make_golden._rounds_layer_major("t", W2, make_inputs(W2), 0.0)
    for b, (r1, r2, d2) in enumerate(ref):
        for rnd, r in ((0, r1), (1, r2)):
            got = rounds[rnd]["requests"][b]
            assert (got["n_accepted"], got["correction"]) == (r.n_accepted, r.correction)
            assert got["lens"] == r.start_len
            np.testing.assert_allclose(logits[rnd, b], r.logits, rtol=0, atol=1e-5)
        assert rounds[1]["drafts"][b] == d2.tolist()
        assert rounds[1]["pending"][b] == r1.correction
    # the chain recipe makes the first drafts the argmax chain: they are accepted
    assert all(rd["requests"][b]["n_accepted"] >= 2 for rd in rounds for b in range(W2.batch))


def test_request_by_request_round_matches_batch_oracle():
    from tests.helpers import oracle_run
    w = W2.with_(rounds=1, mode="mixed")
    inp = make_inputs(w)
    rounds, logits = make_golden._one_round("t", w, inp, 0.0)
    orun = oracle_run(w, make_inputs(w))
    for b, r in enumerate(orun.results):
        got = rounds[0]["requests"][b]
        assert (got["n_accepted"], got["correction"]) == (r.n_accepted, r.correction)
        np.testing.assert_allclose(logits[0, b], r.logits, rtol=0, atol=1e-5)
    assert rounds[0]["drafts"] == orun.inputs.drafts.tolist()
