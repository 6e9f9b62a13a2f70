"""Accept / reject and correction draw alone (spade_accept_from_logits)
against the oracle's verification step on the same logits, drafts, q rows and
uniforms (Sec. III-C, Algorithm 1)."""

import numpy as np
import pytest

from oracle import GREEDY, SAMPLE, speculative_rows
from tests.helpers import report_parity

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def model():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_13076_amd import spade
    from synth.configs import ModelShape
    shape = ModelShape("acc", n_layers=1, d_model=256, n_heads=2, head_dim=128, d_ffn=256,
                       vocab=40000, weight_dtype="f32", kv_dtype="f32")
    return spade.Model(shape, max_batch=16, max_gamma=15, max_len=64)


def _case(rng, B, G, V, scale, mode_mix, T=1.0):
    logits = rng.standard_normal((B, G + 1, V)) * scale
    drafts = rng.integers(0, V, (B, G)).astype(np.int32)
    # make some drafts the argmax so chains of acceptances occur
    for b in range(B):
        for i in range(G):
            if rng.random() < 0.7:
                drafts[b, i] = int(np.argmax(logits[b, i].astype(np.float32)))
    q = rng.dirichlet(np.full(V, 0.3), (B, G)).astype(np.float32)
    for b in range(B):
        for i in range(G):
            if rng.random() < 0.5:  # draft drawn from q
                qq = q[b, i].astype(np.float64)
                drafts[b, i] = int(rng.choice(V, p=qq / qq.sum()))
    u = rng.random((B, G + 1)).astype(np.float32)
    modes = (rng.random(B) < mode_mix).astype(np.uint8)
    return logits.astype(np.float32), drafts, q, u, modes


@pytest.mark.parametrize("V,G,B,scale", [(7, 3, 16, 3.0), (1000, 5, 16, 2.0), (32000, 8, 4, 1.3),
                                         (40000, 15, 2, 4.0), (33, 0, 5, 1.0)])
def test_accept_matches_oracle(model, V, G, B, scale):
    import torch
    rng = np.random.default_rng(V + G)
    dev = model.device
    cnt = dict(total=0, band_n=0, band_c=0, excluded_n=0, excluded_c=0, excluded_mismatch=0)
    for rep in range(6):
        logits, drafts, q, u, modes = _case(rng, B, G, V, scale, 0.5)
        T = 1.0 if rep % 2 == 0 else 0.7
        print(f"accept case V={V} G={G} B={B} rep={rep}", flush=True)
        n, c = model.accept_from_logits(torch.from_numpy(logits).to(dev), torch.from_numpy(drafts).to(dev),
                                        torch.from_numpy(q).to(dev), torch.from_numpy(u).to(dev),
                                        torch.from_numpy(modes).to(dev), T)
        torch.cuda.synchronize()
        n, c = n.cpu().numpy(), c.cpu().numpy()
        for b in range(B):
            r = speculative_rows(logits[b].astype(np.float64), drafts[b],
                                 q[b].astype(np.float64) if modes[b] == SAMPLE else None,
                                 u[b], int(modes[b]), T)
            # identical float32 logits on both sides: the target's bands
            # (greedy top-2 margin 0.1, |u - p/q| 1e-3, draw gap 1e-3) are exact
            cnt["total"] += 1
            cnt["band_n"] += r.pinned_n
            cnt["band_c"] += r.pinned_correction
            cnt["excluded_n"] += not r.pinned_n
            cnt["excluded_c"] += not r.pinned_correction
            if r.pinned_n:
                assert n[b] == r.n_accepted, (b, n[b], r.n_accepted, modes[b], cnt)
            if r.pinned_correction:
                assert c[b] == r.correction, (b, c[b], r.correction, modes[b], cnt)
            if not r.pinned_correction and (n[b] != r.n_accepted or c[b] != r.correction):
                cnt["excluded_mismatch"] += 1
    report_parity(f"accept V={V} G={G} B={B}", cnt)
    assert cnt["band_n"] > 0
    assert model.device_error() == 0


def test_accept_error_flags(model):
    import torch
    dev = model.device
    V, G = 50, 2
    logits = np.zeros((1, G + 1, V), np.float32)
    logits[0, :, 3] = 1.0
    drafts = np.array([[3, 77]], np.int32)  # 77 out of range
    modes = np.zeros(1, np.uint8)
    n, c = model.accept_from_logits(torch.from_numpy(logits).to(dev), torch.from_numpy(drafts).to(dev),
                                    None, None, torch.from_numpy(modes).to(dev))
    torch.cuda.synchronize()
    assert int(n[0]) == 1 and int(c[0]) == 3
    from paper_2608_13076_amd.spade import DERR_TOKEN
    assert model.device_error() & DERR_TOKEN
    assert model.device_error() == 0  # cleared by the read


@pytest.mark.parametrize("V,G,B,scale", [(7, 3, 16, 3.0), (40000, 8, 6, 1.3), (33, 0, 5, 1.0),
                                         (300000, 2, 3, 2.0)])
def test_correction_slices_bit_identical(model, V, G, B, scale):
    """The correction draw over vocabulary slices (a second launch) gives the
    one-workgroup draw's n and correction bit for bit, every request sampling
    (1024 tokens a slice; 300000 tokens hit the 256-slice cap), and matches
    the oracle where the oracle pins it."""
    import torch
    rng = np.random.default_rng(7 * V + G)
    dev = model.device
    try:
        for rep in range(4):
            logits, drafts, q, u, modes = _case(rng, B, G, V, scale, 1.0)
            T = 1.0 if rep % 2 == 0 else 0.7
            print(f"correction slices V={V} G={G} B={B} rep={rep}", flush=True)
            args = (torch.from_numpy(logits).to(dev), torch.from_numpy(drafts).to(dev),
                    torch.from_numpy(q).to(dev), torch.from_numpy(u).to(dev), torch.from_numpy(modes).to(dev), T)
            out = {}
            for mode in (1, 2):
                model.set_correction_slices(mode)
                n, c = model.accept_from_logits(*args)
                torch.cuda.synchronize()
                out[mode] = (n.cpu().numpy(), c.cpu().numpy())
            assert np.array_equal(out[1][0], out[2][0]) and np.array_equal(out[1][1], out[2][1]), (out[1], out[2])
            n, c = out[2]
            for b in range(B):
                r = speculative_rows(logits[b].astype(np.float64), drafts[b], q[b].astype(np.float64), u[b],
                                     SAMPLE, T)
                if r.pinned_n:
                    assert n[b] == r.n_accepted, (b, n[b], r.n_accepted)
                if r.pinned_correction:
                    assert c[b] == r.correction, (b, c[b], r.correction)
        assert model.device_error() == 0
    finally:
        model.set_correction_slices(0)
    from paper_2608_13076_amd.spade import SpadeError
    with pytest.raises(SpadeError):
        model.set_correction_slices(3)
