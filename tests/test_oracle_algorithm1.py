"""Pins of the oracle's Algorithm 1 loop (edge drafting, cloud verify, commit
and rollback on both sides) against what the paper fixes.

* Greedy speculative decoding emits exactly the verifier's own greedy
  continuation, whatever the draft model: every emitted token is either a
  draft the verifier's argmax agreed with or the verifier's argmax itself
  (Sec. III-A greedy selection, Sec. III-C).  Checked against plain
  autoregressive decoding with the verifier for drafts that always agree (the
  verifier itself), partly agree (its first layer, an early exit) and hardly
  agree (an unrelated model), for several draft lengths.
* A draft model equal to the verifier has every draft accepted in both modes
  (alpha = min(1, p/q) = 1), so each call emits gamma + 1 tokens and the run
  needs ceil(N / (gamma + 1)) calls.
* With an unrelated draft the greedy loop still needs at most N calls (every
  call emits at least one token: the correction).
"""

from dataclasses import replace

import numpy as np
import pytest

from oracle.decoder import Decoder
from oracle.speculative import GREEDY, SAMPLE, algorithm1, target_only
from synth import ModelWeights
from synth.configs import ModelShape

SHAPE = ModelShape("t-loop", n_layers=2, d_model=64, n_heads=2, head_dim=32, d_ffn=96, vocab=61,
                   weight_dtype="f32", kv_dtype="f32", init_std=0.3, gain_std=0.2)


def _models():
    mw = ModelWeights(SHAPE, 11)
    target = Decoder(SHAPE, mw.get, keep_f64=True)
    early = Decoder(replace(SHAPE, n_layers=1), mw.get, keep_f64=True)  # the verifier's first layer
    other = Decoder(SHAPE, ModelWeights(SHAPE, 12).get, keep_f64=True)
    return target, early, other


def _uniforms(seed):
    return iter(np.random.default_rng(seed).random(100000, dtype=np.float32).tolist())


@pytest.mark.parametrize("gamma", [1, 3, 4])
def test_greedy_loop_emits_the_verifiers_greedy_continuation(gamma):
    target, early, other = _models()
    prompt = np.random.default_rng(1).integers(0, SHAPE.vocab, 9)
    ref = target_only(target, prompt, 30, GREEDY, _uniforms(0)).tokens
    for draft in (target, early, other):
        res = algorithm1(target, draft, prompt, gamma, 30, GREEDY, _uniforms(0))
        assert res.tokens == ref
        assert res.calls <= 30 and sum(a + 1 for a in res.accepted) >= 30
    full = algorithm1(target, target, prompt, gamma, 30, GREEDY, _uniforms(0))
    assert full.accepted == [gamma] * full.calls
    assert full.calls == -(-30 // (gamma + 1))
    # the early exit agrees sometimes, the unrelated model less
    ex = algorithm1(target, early, prompt, gamma, 30, GREEDY, _uniforms(0))
    assert sum(ex.accepted) > 0


def test_sampling_loop_with_the_verifier_as_draft_accepts_everything():
    target, _, _ = _models()
    prompt = np.random.default_rng(2).integers(0, SHAPE.vocab, 7)
    res = algorithm1(target, target, prompt, 4, 25, SAMPLE, _uniforms(3), temperature=1.0)
    assert res.accepted == [4] * res.calls
    assert res.calls == 5
    assert len(res.tokens) == 25 and all(0 <= t < SHAPE.vocab for t in res.tokens)


def test_agreement_falls_with_draft_noise():
    """A draft built from the verifier's weights plus noise: the more noise,
    the fewer drafts accepted (the alignment knob of the gamma sweep)."""
    from synth import perturb_tensor
    mw = ModelWeights(SHAPE, 11)
    target = Decoder(SHAPE, mw.get, keep_f64=True)
    prompt = np.random.default_rng(4).integers(0, SHAPE.vocab, 9)
    acc = []
    for sigma in (0.0, 0.05, 3.0):
        get = (lambda s: (lambda k, l=None: perturb_tensor(SHAPE, k, l, mw.get(k, l), s, 99)))(sigma)
        draft = Decoder(SHAPE, get, keep_f64=True)
        r = algorithm1(target, draft, prompt, 4, 40, GREEDY, _uniforms(0))
        acc.append(np.mean(r.accepted))
    assert acc[0] == 4 and acc[0] > acc[1] > acc[2]
