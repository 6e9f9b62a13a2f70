"""spade_accept_from_logits_noalloc -- the accept/reject and correction
draw with the library's static device scratch instead of a model's workspace
-- against spade_accept_from_logits on the same logits, drafts, q rows and
uniforms: two calls in a row, the second with a smaller input (fewer
requests, drafts and vocabulary), n_accepted and corrections bit for bit;
the oracle's decisions where its bands pin them (identical float32 logits
on both sides)."""

import numpy as np
import pytest

from oracle import SAMPLE, speculative_rows
from tests.test_gpu_accept import _case

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def model():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_13076_amd import spade
    from synth.configs import ModelShape
    shape = ModelShape("acc-noalloc", n_layers=1, d_model=256, n_heads=2, head_dim=128, d_ffn=256,
                       vocab=40000, weight_dtype="f32", kv_dtype="f32")
    return spade.Model(shape, max_batch=64, max_gamma=15, max_len=64)


def test_noalloc_matches_workspace_entry_point(model):
    import torch
    from paper_2608_13076_amd import spade
    dev = model.device
    rng = np.random.default_rng(2024)
    for B, G, V, scale, T in ((64, 8, 40000, 1.3, 1.0), (5, 3, 5000, 2.0, 0.7)):
        logits, drafts, q, u, modes = _case(rng, B, G, V, scale, 0.6)
        args = [torch.from_numpy(x).to(dev) for x in (logits, drafts, q, u, modes)]
        print(f"noalloc B={B} gamma={G} V={V}", flush=True)
        ref_n, ref_c = model.accept_from_logits(*args, T)
        n = torch.full((B,), -1, dtype=torch.int32, device=dev)
        c = torch.full((B,), -1, dtype=torch.int32, device=dev)
        err = torch.zeros(1, dtype=torch.int32, device=dev)
        spade.accept_from_logits_noalloc(*args, T, n, c, err)
        torch.cuda.synchronize()
        assert int(err[0]) == 0
        assert model.device_error() == 0
        n, c = n.cpu().numpy(), c.cpu().numpy()
        np.testing.assert_array_equal(n, ref_n.cpu().numpy())
        np.testing.assert_array_equal(c, ref_c.cpu().numpy())
        band = 0
        for b in range(B):
            r = speculative_rows(logits[b].astype(np.float64), drafts[b],
                                 q[b].astype(np.float64) if modes[b] == SAMPLE else None, u[b], int(modes[b]), T)
            if r.pinned_n:
                band += 1
                assert n[b] == r.n_accepted, b
            if r.pinned_correction:
                assert c[b] == r.correction, b
        assert band > 0


def test_noalloc_rejects_beyond_its_limits(model):
    import torch
    from paper_2608_13076_amd import spade
    dev = model.device
    logits = torch.zeros((65, 2, 10), dtype=torch.float32, device=dev)
    drafts = torch.zeros((65, 1), dtype=torch.int32, device=dev)
    modes = torch.zeros(65, dtype=torch.uint8, device=dev)
    n = torch.empty(65, dtype=torch.int32, device=dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    with pytest.raises(spade.SpadeError):
        spade.accept_from_logits_noalloc(logits, drafts, None, None, modes, 1.0, n, n.clone(), err)
    with pytest.raises(spade.SpadeError):
        spade.accept_from_logits_noalloc(logits[:4], drafts[:4], None, None, modes[:4], 1.0, n[:4], n[:4].clone(),
                                         None)
