"""Algorithm 1 end to end on the GPU (edge draft model + cloud verify, commit
and rollback on both sides), through the C ABI.

* Greedy: the speculative loop emits exactly what plain autoregressive
  decoding with the verifier emits on the GPU, token for token, whatever the
  draft (an early exit of the verifier, or the verifier itself) and draft
  length: the verify pass gives a position the same logits whether it is
  scored in a block or alone.
* A draft model equal to the verifier has every draft accepted (greedy and
  sampling).
* Against the oracle's loop (same prompt, same uniforms): the emitted tokens
  agree up to the first position whose decision is within the logit tolerance
  of a tie (greedy top-2 margin), which is reported.
"""

import numpy as np
import pytest

from oracle.decoder import Decoder
from oracle.speculative import GREEDY, SAMPLE, algorithm1
from synth import ModelWeights, mini_workloads

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _shape(name):
    return {w.name: w for w in mini_workloads()}[name].model


# a decision can flip where the top-2 margin is within twice the logit error:
# ~1e-6 for f32 weights, up to ~1.3e-2 measured for the bf16 mini shapes
CASES = [("mini_f32_greedy", 1e-4), ("mini_bf16_greedy", 0.03)]


@pytest.mark.parametrize("name,band", CASES, ids=[c[0] for c in CASES])
def test_greedy_loop_equals_target_only_and_oracle(name, band):
    from dataclasses import replace
    from paper_2608_13076_amd.algorithm1 import load_model, run_algorithm1, run_target_only
    shape = _shape(name)
    seed, n_new = 31, 40
    prompt = np.random.default_rng(5).integers(0, shape.vocab, 60).astype(np.int32)
    uniforms = np.random.default_rng(6).random(4000, dtype=np.float32)
    max_len = 60 + n_new + 32
    target = load_model(shape, seed, max_len, 6)
    early = load_model(shape, seed, max_len, 6, n_layers=1)
    base = run_target_only(target, prompt, n_new, GREEDY, uniforms)
    for draft, gamma in ((early, 2), (early, 5), (target, 4)):
        print(f"[{name}] greedy loop, draft layers {draft.shape.n_layers}, gamma {gamma}", flush=True)
        r = run_algorithm1(target, draft, prompt, gamma, n_new, GREEDY, uniforms)
        assert r.tokens == base.tokens, (gamma, r.tokens, base.tokens)
        if draft is target:
            assert r.accepted == [gamma] * r.calls
        print(f"  calls {r.calls} for {n_new} tokens, accepted {r.accepted}", flush=True)
    # the oracle's loop with the early-exit draft
    mw = ModelWeights(shape, seed)
    o_t = Decoder(shape, mw.get, keep_f64=True)
    o_d = Decoder(replace(shape, n_layers=1), mw.get, keep_f64=True)
    o = algorithm1(o_t, o_d, prompt.astype(np.int64), 5, n_new, GREEDY, iter(uniforms.tolist()))
    g = run_algorithm1(target, early, prompt, 5, n_new, GREEDY, uniforms)
    decided = next((i for i, m in enumerate(o.margins) if m <= band), n_new)
    print(f"[{name}] oracle agreement checked on the first {decided} of {n_new} tokens "
          f"(margins {np.round(o.margins[:decided + 1], 4).tolist()})", flush=True)
    assert decided >= 3
    assert g.tokens[:decided] == o.tokens[:decided]
    assert target.device_error() == 0 and early.device_error() == 0
    early.close()
    target.close()


def test_sampling_loop_with_the_verifier_as_draft():
    from paper_2608_13076_amd.algorithm1 import load_model, run_algorithm1
    shape = _shape("mini_f32_greedy")
    prompt = np.random.default_rng(7).integers(0, shape.vocab, 40).astype(np.int32)
    uniforms = np.random.default_rng(8).random(4000, dtype=np.float32)
    target = load_model(shape, 41, 120, 4)
    r = run_algorithm1(target, target, prompt, 4, 30, SAMPLE, uniforms, temperature=1.0)
    assert r.accepted == [4] * r.calls and r.calls == 6
    assert all(0 <= t < shape.vocab for t in r.tokens)
    assert target.device_error() == 0
    target.close()
