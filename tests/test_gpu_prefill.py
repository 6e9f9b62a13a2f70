"""Batched prefill (spade_prefill_batch) against per-request prefill.

All requests' next chunks run in one forward; a request whose prompt is used
up contributes placeholder rows past its length.  A cached key depends only
on its own token and the keys before it, so the cache contents, lengths and
pending tokens must be bit-identical to prefilling each request alone, and so
must the logits and decisions of the verify call that follows.  Ragged prompt
lengths (including a prompt of one token: nothing to cache) and both the
multi-head and the grouped-query mini shapes.
"""

import numpy as np
import pytest

from synth import ModelWeights, make_inputs, mini_workloads
from tests.helpers import gpu_setup, gpu_verify

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _cases():
    ws = {w.name: w for w in mini_workloads()}
    return [ws["mini_bf16_mixed"], ws["mini_gqa_mixed_b5"], ws["mini_f32_greedy"]]


@pytest.mark.parametrize("w", _cases(), ids=lambda w: w.name)
def test_batched_prefill_equals_per_request(w):
    import torch
    weights = ModelWeights(w.model, w.seed)
    inp = make_inputs(w)
    prompts = [np.asarray(p) for p in inp.prompts]
    prompts[0] = prompts[0][:1]  # nothing to cache for request 0
    inp.prompts = prompts
    max_len = max(len(p) for p in prompts) + 2 * (w.gamma + 1) + 24
    model, kv1 = gpu_setup(w, weights, max_len=max_len)
    from paper_2608_13076_amd import spade
    kv2 = spade.KVCache(model, w.batch, max_len)
    print(f"[{w.name}] prompts {[len(p) for p in prompts]}", flush=True)
    for b, p in enumerate(prompts):
        kv1.prefill(b, p)
    kv2.prefill_batch(prompts)
    l1, p1 = kv1.get_state(w.batch)
    l2, p2 = kv2.get_state(w.batch)
    np.testing.assert_array_equal(l1, l2)
    np.testing.assert_array_equal(p1, p2)
    # cache contents up to each request's length
    half = kv1.buf.numel() // 2
    s = model.shape
    stride = (max_len + 31) // 32 * 32
    elt = torch.int16 if s.kv_dtype == "bf16" else torch.float32
    n_el = s.n_layers * w.batch * s.kv_heads * stride * s.head_dim
    for which, part in (("k", slice(0, half)), ("v", slice(half, 2 * half))):
        a = kv1.buf[part].view(elt)[:n_el].view(s.n_layers, w.batch, s.kv_heads, stride * s.head_dim)
        c = kv2.buf[part].view(elt)[:n_el].view(s.n_layers, w.batch, s.kv_heads, stride * s.head_dim)
        for b in range(w.batch):
            n = int(l1[b])
            if which == "k":  # K rows [pos][hd]
                ka = a[:, b].reshape(s.n_layers, s.kv_heads, stride, s.head_dim)[:, :, :n]
                kc = c[:, b].reshape(s.n_layers, s.kv_heads, stride, s.head_dim)[:, :, :n]
            else:  # V stored transposed: [hd][stride] per head
                ka = a[:, b].reshape(s.n_layers, s.kv_heads, s.head_dim, stride)[..., :n]
                kc = c[:, b].reshape(s.n_layers, s.kv_heads, s.head_dim, stride)[..., :n]
            assert torch.equal(ka, kc), (which, b)
    r1 = gpu_verify(model, kv1, inp)
    r2 = gpu_verify(model, kv2, inp)
    assert np.array_equal(r1[0].view(np.uint32), r2[0].view(np.uint32))
    assert np.array_equal(r1[1], r2[1]) and np.array_equal(r1[2], r2[2])
    assert model.device_error() == 0
