"""Seeded per-call inputs: prompts, cached lengths, drafts, q rows, uniforms.

Row convention of a verify call: request b's cache holds ``lens[b]`` tokens
and a pending token (the last prompt token, or the previous round's
correction) that has not been run through the verifier yet.  The call scores
the rows [pending, d_1 .. d_gamma] at positions lens[b] .. lens[b] + gamma.
A prompt therefore has lens[b] + 1 ids.

Draft recipes (no trained draft model exists here):
  random       uniform ids;
  chain_half   the first ceil(gamma/2) drafts are placeholders that the caller
               replaces with the verifier's own argmax chain, the rest uniform;
  noise_q      q_i = softmax(N(0,1) logits), d_i ~ q_i;
  draft_model  q_i = softmax(verifier logits_i / T + N(0,1)); the caller forms
               q_i from ``q_noise`` once it has the verifier logits, and draws
               d_i with ``draw_from`` and the uniform ``draft_u[b, i]``.
In "mixed" mode even requests are greedy and odd requests sample; sampling
requests of a chain_half workload use noise_q.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

from .configs import Workload

GREEDY = 0
SAMPLE = 1


@dataclass
class VerifyInputs:
    workload: Workload
    round: int
    prompts: List[np.ndarray]  # per request: lens[b] + 1 int32 ids
    lens: np.ndarray  # int32 [B] cached tokens
    pending: np.ndarray  # int32 [B]
    modes: np.ndarray  # uint8 [B]
    drafts: np.ndarray  # int32 [B, gamma]
    draft_probs: Optional[np.ndarray]  # float32 [B, gamma, V] or None
    uniforms: np.ndarray  # float32 [B, gamma + 1] in [0, 1)
    temperature: float
    recipe: List[str]  # per-request draft recipe
    chain_slots: int  # leading drafts of chain_half requests to be replaced
    q_noise: Optional[np.ndarray] = None  # float32 [B, gamma, V] for draft_model
    draft_u: Optional[np.ndarray] = None  # float64 [B, gamma] draws for d_i ~ q_i
    notes: dict = field(default_factory=dict)


def softmax64(z: np.ndarray) -> np.ndarray:
    """Draft-side softmax used to build q rows (input generation only)."""
    z = np.asarray(z, dtype=np.float64)
    m = z.max(axis=-1, keepdims=True)
    e = np.exp(z - m)
    return e / e.sum(axis=-1, keepdims=True)


def draw_from(q: np.ndarray, u: float) -> int:
    """Inverse-CDF draw of a draft token from a q row (float64)."""
    c = np.cumsum(np.asarray(q, dtype=np.float64))
    i = int(np.searchsorted(c, u * c[-1], side="right"))
    return min(i, len(c) - 1)


def _rng(seed: int, *key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=key)))


def make_inputs(w: Workload, round_index: int = 0, ctx_override: Optional[List[int]] = None) -> VerifyInputs:
    m = w.model
    B, G, V = w.batch, w.gamma, m.vocab
    r_len = _rng(w.seed, 1)
    lo, hi = w.ctx
    if ctx_override is not None:
        lens = np.asarray(ctx_override, dtype=np.int32)
    elif lo == hi:
        lens = np.full(B, lo, dtype=np.int32)
    else:
        lens = r_len.integers(lo, hi + 1, size=B).astype(np.int32)
    r_prompt = _rng(w.seed, 2)
    prompts = [r_prompt.integers(0, V, size=int(L) + 1).astype(np.int32) for L in lens]
    pending = np.array([p[-1] for p in prompts], dtype=np.int32)

    if w.mode == "greedy":
        modes = np.full(B, GREEDY, dtype=np.uint8)
    elif w.mode == "sample":
        modes = np.full(B, SAMPLE, dtype=np.uint8)
    else:
        modes = np.array([GREEDY if b % 2 == 0 else SAMPLE for b in range(B)], dtype=np.uint8)

    recipe = []
    for b in range(B):
        if modes[b] == SAMPLE and w.draft_recipe == "chain_half":
            recipe.append("noise_q")
        elif modes[b] == GREEDY and w.draft_recipe in ("noise_q", "draft_model"):
            recipe.append("random")
        else:
            recipe.append(w.draft_recipe)

    rd = _rng(w.seed, 3, round_index)
    drafts = rd.integers(0, V, size=(B, G)).astype(np.int32)
    uniforms = rd.random((B, G + 1), dtype=np.float32)
    draft_u = rd.random((B, G))
    any_sample = bool((modes == SAMPLE).any())
    draft_probs = np.zeros((B, G, V), dtype=np.float32) if any_sample else None
    q_noise = None
    for b in range(B):
        if recipe[b] == "noise_q":
            rq = _rng(w.seed, 4, round_index, b)
            q = softmax64(rq.standard_normal((G, V)))
            draft_probs[b] = q.astype(np.float32)
            for i in range(G):
                drafts[b, i] = draw_from(draft_probs[b, i], draft_u[b, i])
        elif recipe[b] == "draft_model":
            if q_noise is None:
                q_noise = np.zeros((B, G, V), dtype=np.float32)
            rq = _rng(w.seed, 5, round_index, b)
            q_noise[b] = rq.standard_normal((G, V)).astype(np.float32)
    chain_slots = (G + 1) // 2 if w.draft_recipe == "chain_half" else 0
    return VerifyInputs(w, round_index, prompts, lens, pending, modes, drafts, draft_probs,
                        uniforms, float(w.temperature), recipe, chain_slots, q_noise, draft_u)
