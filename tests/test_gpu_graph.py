"""spade_verify captured in a HIP graph.

The verify call is stream-ordered kernel launches only (no memsets, no host
synchronisation while the cache's host length bound covers the call), so a
caller can capture it.  The graph is replayed several times with eager work
between the replays (the output buffers cleared, an eager verify call of the
same inputs, synchronisations); every replay must give the eager call's
logits and decisions bit for bit.  Shapes: multi-head, wide (the medium-M GEMM
forced, with its second launch), grouped-query, and the float32 cache.
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


@pytest.mark.parametrize("name,mid", [("mini_bf16_mixed", 0), ("mini_bf16_wide_b5", 2), ("mini_gqa_mixed_b5", 0),
                                      ("mini_f32_greedy", 0)])
def test_captured_verify_replays_match_eager(name, mid):
    import torch
    from paper_2608_13076_amd import spade
    w = MINIS[name]
    weights = ModelWeights(w.model, w.seed)
    inp = make_inputs(w)
    max_len = max(len(p) for p in inp.prompts) + 4 * (w.gamma + 1) + 16
    model, kv = gpu_setup(w, weights, max_len=max_len)
    if mid:
        model.set_mid_gemm(mid)
    kv.prefill_batch([np.asarray(p) for p in inp.prompts])
    ref = gpu_verify(model, kv, inp)
    buf = spade.VerifyBuffers(model, inp.drafts, inp.draft_probs, inp.uniforms, inp.modes, True)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        spade.verify(model, kv, buf, inp.temperature)  # the launch path once before the capture
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(graph, stream=s):
            spade.verify(model, kv, buf, inp.temperature)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for i in range(4):
        buf.logits.zero_()
        buf.n.fill_(-1)
        buf.corr.fill_(-1)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        lg = buf.logits.cpu().numpy()
        assert np.array_equal(lg.view(np.uint32), ref[0].view(np.uint32)), f"replay {i}: logits"
        assert np.array_equal(buf.n.cpu().numpy(), ref[1]), f"replay {i}: n"
        assert np.array_equal(buf.corr.cpu().numpy(), ref[2]), f"replay {i}: correction"
        eager = gpu_verify(model, kv, inp)
        assert np.array_equal(eager[0].view(np.uint32), ref[0].view(np.uint32)), f"eager call after replay {i}"
    assert model.device_error() == 0
    model.set_mid_gemm(0)
