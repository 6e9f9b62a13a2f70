"""Algorithm 1 (edge drafting + cloud verification) on one GPU, through the C
ABI only.

The edge side runs a draft model autoregressively: one draft token is one
``spade_verify`` call with no drafts (its "bonus" token is the next token:
the argmax, or the Gumbel-max draw keyed by a uniform), followed by
``spade_softmax`` for the distribution q the token was drawn from (sampling)
and a commit.  The cloud side is one ``spade_verify`` over the pending token
and the gamma drafts, followed by ``spade_kv_commit`` (Algorithm 1: m <- m +
k + 1, on the device).  The draft's cache is then cut back to the same
accepted prefix plus the correction; when every draft was accepted the draft
model first runs its last draft, which it never appended.

Uniforms are consumed in a fixed order -- one per draft step, then gamma + 1
per cloud call -- from a device array, so a CPU run of the same loop
(``oracle.speculative.algorithm1``) can be fed the same values.

``python -m paper_2608_13076_amd.algorithm1`` measures cloud calls per
emitted token and time per token against plain autoregressive decoding with
the verifier, on the synthetic 7B-shaped verifier with early-exit drafts.
"""

from __future__ import annotations

import argparse
import json
import sys
import time
from dataclasses import dataclass, field, replace
from typing import List, Optional

import numpy as np
import torch

from . import spade

GREEDY, SAMPLE = 0, 1


@dataclass
class LoopStats:
    tokens: List[int]
    calls: int
    accepted: List[int] = field(default_factory=list)
    seconds: float = 0.0  # wall time of the decoding (prefill excluded), synchronised per call


class _Side:
    """One model's cache and reusable call buffers (batch 1)."""

    def __init__(self, model: spade.Model, max_len: int, gamma: int, mode: int):
        dev = model.device
        self.model = model
        self.kv = spade.KVCache(model, 1, max_len)
        self.mode = torch.tensor([mode], dtype=torch.uint8, device=dev)
        self.n = torch.zeros(1, dtype=torch.int32, device=dev)
        self.corr = torch.zeros(1, dtype=torch.int32, device=dev)
        self.logits = torch.empty((1, gamma + 1, model.shape.vocab), dtype=torch.float32, device=dev)

    def call(self, gamma: int, drafts: Optional[torch.Tensor], q: Optional[torch.Tensor],
             u: torch.Tensor, temperature: float) -> None:
        m = self.model
        spade._check(m.lib.spade_verify(m.handle, self.kv.handle, 1, gamma, spade._ptr(drafts), spade._ptr(q),
                                        spade._ptr(u), spade._ptr(self.mode), float(temperature),
                                        spade._ptr(self.n), spade._ptr(self.corr), spade._ptr(self.logits),
                                        spade._stream()))


def _step(side: _Side, u: torch.Tensor, temperature: float) -> None:
    """One autoregressive step: next token into side.corr, appended."""
    side.call(0, None, None, u, temperature)
    side.kv.commit(side.n, side.corr)


def run_algorithm1(target: spade.Model, draft: spade.Model, prompt, gamma: int, max_new: int, mode: int,
                   uniforms: np.ndarray, temperature: float = 1.0) -> LoopStats:
    """Speculative decoding of ``max_new`` tokens after ``prompt`` (its last
    id is the first pending token)."""
    dev = target.device
    prompt = np.asarray(prompt, dtype=np.int32)
    max_len = len(prompt) + max_new + 2 * gamma + 4
    t, d = _Side(target, max_len, gamma, mode), _Side(draft, max_len, gamma, mode)
    t.kv.prefill(0, prompt)
    d.kv.prefill(0, prompt)
    uni = torch.from_numpy(np.ascontiguousarray(uniforms, dtype=np.float32)).to(dev)
    half = torch.full((1,), 0.5, dtype=torch.float32, device=dev)
    drafts = torch.zeros((1, max(gamma, 1)), dtype=torch.int32, device=dev)
    q = torch.zeros((1, max(gamma, 1), target.shape.vocab), dtype=torch.float32, device=dev)
    start = len(prompt) - 1
    pos = 0  # next uniform
    out: List[int] = []
    acc: List[int] = []
    calls = 0
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    while len(out) < max_new:
        for j in range(gamma):  # edge
            _step(d, uni[pos:pos + 1], temperature)
            pos += 1
            drafts[0, j].copy_(d.corr[0])
            if mode == SAMPLE:
                spade.softmax_into(d.logits[0, 0], q[0, j], temperature)
        # cloud
        t.call(gamma, drafts, q if mode == SAMPLE else None, uni[pos:pos + gamma + 1], temperature)
        pos += gamma + 1
        calls += 1
        t.kv.commit(t.n, t.corr)  # m <- m + k + 1 on the device
        n = int(t.n.item())
        corr = int(t.corr.item())
        new_len = start + n + 1
        if n == gamma and gamma > 0:  # the draft never appended d_gamma: run it now
            d.call(0, None, None, half, temperature)
        d.kv.set_state(np.array([new_len], np.int32), np.array([corr], np.int32))
        toks = drafts[0, :n].cpu().tolist() if n > 0 else []
        out += toks + [corr]
        acc.append(n)
        start = new_len
    torch.cuda.synchronize()
    secs = time.perf_counter() - t0
    t.kv.close()
    d.kv.close()
    return LoopStats(out[:max_new], calls, acc, secs)


def run_target_only(target: spade.Model, prompt, max_new: int, mode: int, uniforms: np.ndarray,
                    temperature: float = 1.0) -> LoopStats:
    """Plain autoregressive decoding with the verifier: one call per token."""
    dev = target.device
    prompt = np.asarray(prompt, dtype=np.int32)
    t = _Side(target, len(prompt) + max_new + 2, 0, mode)
    t.kv.prefill(0, prompt)
    uni = torch.from_numpy(np.ascontiguousarray(uniforms, dtype=np.float32)).to(dev)
    toks = torch.zeros(max_new, dtype=torch.int32, device=dev)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(max_new):
        _step(t, uni[i:i + 1], temperature)
        toks[i].copy_(t.corr[0])
    torch.cuda.synchronize()
    secs = time.perf_counter() - t0
    t.kv.close()
    return LoopStats(toks.cpu().tolist(), max_new, [], secs)


def load_model(shape, seed: int, max_len: int, gamma: int, n_layers: Optional[int] = None,
               sigma: float = 0.0, noise_seed: int = 7) -> spade.Model:
    """A model of ``shape`` (or its first ``n_layers`` layers with the same
    embedding, final norm and LM head: an early-exit draft) with the seeded
    synthetic weights, every matrix perturbed by ``sigma`` (relative to the
    weights' scale; 0: none) for a draft of controlled agreement."""
    from synth import iter_weights_perturbed
    sh = shape if n_layers is None else replace(shape, n_layers=n_layers)
    m = spade.Model(sh, 1, gamma, max_len)
    for kind, layer, arr in iter_weights_perturbed(sh, seed, sigma, noise_seed):
        m.load_numpy(kind, layer, arr)
    return m


def main() -> int:
    from synth import workload
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--workload", default="c2_7b_greedy", help="verifier shape (and seed) of this workload")
    ap.add_argument("--prompt", type=int, default=1024)
    ap.add_argument("--tokens", type=int, default=96)
    ap.add_argument("--gammas", default="3,5,8")
    ap.add_argument("--draft-layers", default="2,8,16", help="early-exit drafts (comma list; empty: none)")
    ap.add_argument("--draft-noise", default="", help="full-depth drafts with perturbed weights: sigmas")
    ap.add_argument("--mode", default="greedy", choices=["greedy", "sample"])
    ap.add_argument("--temperature", type=float, default=1.0)
    a = ap.parse_args()
    w = workload(a.workload)
    mode = GREEDY if a.mode == "greedy" else SAMPLE
    gammas = [int(x) for x in a.gammas.split(",")]
    layers = [int(x) for x in a.draft_layers.split(",") if x]
    sigmas = [float(x) for x in a.draft_noise.split(",") if x]
    max_len = a.prompt + a.tokens + 2 * max(gammas) + 8
    prompt = np.random.default_rng(w.seed).integers(0, w.model.vocab, a.prompt + 1).astype(np.int32)
    uniforms = np.random.default_rng(w.seed + 1).random(8 * a.tokens * (max(gammas) + 2), dtype=np.float32)
    target = load_model(w.model, w.seed, max_len, max(gammas))
    base = run_target_only(target, prompt, a.tokens, mode, uniforms, a.temperature)
    rows = [{"draft_layers": None, "gamma": 0, "calls": base.calls, "tokens": a.tokens,
             "calls_per_token": 1.0, "ms_per_token": round(base.seconds * 1e3 / a.tokens, 3)}]
    print(json.dumps(rows[0]), flush=True)
    drafts = [("draft_layers", k, dict(n_layers=k)) for k in layers] + \
             [("draft_noise", sg, dict(sigma=sg)) for sg in sigmas]
    for key, val, kw in drafts:
        draft = load_model(w.model, w.seed, max_len, max(gammas), **kw)
        for g in gammas:
            r = run_algorithm1(target, draft, prompt, g, a.tokens, mode, uniforms, a.temperature)
            same = r.tokens == base.tokens if mode == GREEDY else None
            row = {key: val, "gamma": g, "calls": r.calls, "tokens": a.tokens,
                   "calls_per_token": round(r.calls / a.tokens, 4),
                   "accepted_per_call": round(float(np.mean(r.accepted)), 3),
                   "ms_per_token": round(r.seconds * 1e3 / a.tokens, 3), "same_as_target_only": same}
            rows.append(row)
            print(json.dumps(row), flush=True)
        draft.close()
    print(json.dumps({"workload": w.name, "mode": a.mode, "prompt_tokens": a.prompt, "rows": rows}))
    return 0


if __name__ == "__main__":
    sys.exit(main())
