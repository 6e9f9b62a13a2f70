"""Seeded input generators: determinism, shapes and distributions."""

import numpy as np

from synth import ModelWeights, bf16_bits_to_f32, make_inputs, mini_workloads, workload
from synth.weights import make_tensor, normal_table_bf16


def test_bf16_table_is_normal_quantiles():
    t = bf16_bits_to_f32(normal_table_bf16(0.02)).astype(np.float64)
    assert np.all(np.diff(t) >= 0)
    np.testing.assert_allclose(t, -t[::-1], atol=0)  # symmetric
    assert abs(t.std() - 0.02) < 2e-4 and abs(t.mean()) < 1e-6


def test_weights_deterministic_and_chunk_independent():
    w = workload("c1_tiny_greedy").model
    a = make_tensor(w, "wg", 1, 5)
    b = make_tensor(w, "wg", 1, 5)
    np.testing.assert_array_equal(a, b)
    assert not np.array_equal(a, make_tensor(w, "wg", 0, 5))
    assert a.dtype == np.float32 and a.shape == (1024, 256)
    assert abs(a.std() - 0.02) < 1e-3


def test_inputs_shapes():
    for wl in mini_workloads():
        inp = make_inputs(wl)
        B, G, V = wl.batch, wl.gamma, wl.model.vocab
        assert inp.drafts.shape == (B, G) and inp.uniforms.shape == (B, G + 1)
        assert all(len(p) == L + 1 for p, L in zip(inp.prompts, inp.lens))
        assert inp.drafts.min() >= 0 and inp.drafts.max() < V
        if inp.draft_probs is not None:
            s = inp.draft_probs.sum(-1)
            for b in range(B):
                if inp.recipe[b] == "noise_q":
                    np.testing.assert_allclose(s[b], 1.0, atol=1e-5)


def test_perturbed_weights():
    from synth import make_tensor, perturb_tensor
    from synth.configs import ModelShape
    sh = ModelShape("p", n_layers=1, d_model=256, n_heads=2, head_dim=128, d_ffn=512, vocab=300)
    t = make_tensor(sh, "wq", 0, 5)
    assert perturb_tensor(sh, "wq", 0, t, 0.0, 1) is t
    g = make_tensor(sh, "g_attn", 0, 5)
    assert perturb_tensor(sh, "g_attn", 0, g, 0.5, 1) is g
    from synth import bf16_bits_to_f32
    p1 = perturb_tensor(sh, "wq", 0, t, 0.25, 1)
    assert p1.dtype == np.uint16 and p1.shape == t.shape
    np.testing.assert_array_equal(p1, perturb_tensor(sh, "wq", 0, t, 0.25, 1))  # seeded
    diff = bf16_bits_to_f32(p1).astype(np.float64) - bf16_bits_to_f32(t)
    assert abs(diff.std() / (0.25 * sh.init_std) - 1) < 0.05 and abs(diff.mean()) < 1e-4
    assert not np.array_equal(p1, perturb_tensor(sh, "wq", 0, t, 0.25, 2))
