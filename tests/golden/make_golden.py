"""Write the oracle's results for full-size workloads to tests/golden/.

    python -m tests.golden.make_golden c2_7b_greedy c4_7b_batched c5_33b_commit ...

Calls only the oracle (and the seeded input generators).  For each workload
it prefills the oracle's caches with the seeded prompts, fills the draft
slots that depend on the verifier (argmax chain, or q = softmax(logits/T +
noise) with drafts drawn from q), runs the verify call and, for two-round
workloads, the context update m <- m + k + 1 and a second verify call whose
chain drafts are taken at the committed state (Algorithm 1, Cloud step).

Files per workload:
  <name>.json        per round: drafts, uniforms, pending tokens and cached
                     lengths; per request: the decisions and how decided they
                     are (margins, ratios, the draw's score gap and its
                     error bound);
  <name>_logits.npy  float32 [rounds, B, gamma+1, V]: every logit row;
  <name>_q.npy       q rows of draft_model (sampling) workloads.

Single-round workloads run request by request (one cache alive at a time);
two-round workloads run layer by layer over all requests
(``Decoder.forward_many``), so each layer's weights are generated once per
pass and never held for the whole model.
"""

from __future__ import annotations

import json
import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

from oracle import GREEDY, SAMPLE, Decoder, verify as oracle_verify  # noqa: E402
from oracle.speculative import _argmax_f32, commit, speculative_rows  # noqa: E402
from synth import ModelWeights, make_inputs, make_tensor, workload  # noqa: E402
from tests.helpers import chain_drafts, complete_drafts  # noqa: E402


def _log(name, t0, msg):
    print(f"[{name} {time.time() - t0:7.0f}s] {msg}", flush=True)


def _record(r, inp, b) -> dict:
    """Decisions of request b and how far each is from a flip."""
    lg = r.logits
    draw = r.notes.get("draw")
    draw_bound = None
    if draw is not None:
        # score error of the draw per unit of (exp(2 eps / T) - 1): p_v / (p_v - q_v)
        # summed over the two best tokens for a residual draw, 0 for a bonus draw
        draw_bound = 0.0
        if draw["kind"] == "residual":
            z = lg[draw["row"]] / inp.temperature
            pz = np.exp(z - z.max())
            pz /= pz.sum()
            for v in (draw["top"], draw["second"]):
                wv = pz[v] - float(inp.draft_probs[b, draw["row"], v])
                draw_bound += float(pz[v] / wv) if wv > 0 else float("inf")
    return {"n_accepted": r.n_accepted, "correction": r.correction, "pinned_n": r.pinned_n,
            "pinned_correction": r.pinned_correction, "draw_margin": r.draw_margin,
            "row_margins": [x.margin for x in r.rows], "row_ratios": [x.ratio for x in r.rows],
            "draw": draw, "draw_bound": draw_bound, "fallback": r.fallback,
            "argmax": [int(_argmax_f32(row)) for row in lg],
            "lens": int(r.start_len), "mode": int(inp.modes[b])}


def _round_json(inp, recs) -> dict:
    return {"drafts": inp.drafts.tolist(), "uniforms": inp.uniforms.tolist(),
            "pending": [int(x) for x in inp.pending], "lens": [int(x) for x in inp.lens],
            "requests": recs}


def _one_round(name, w, inp, t0):
    """Request by request: prefill, verifier-dependent drafts, verify."""
    weights = ModelWeights(w.model, w.seed)
    dec = Decoder(w.model, weights.get, keep_f64=False)
    G, V = w.gamma, w.model.vocab
    logits = np.zeros((1, w.batch, G + 1, V), dtype=np.float32)
    recs = []
    for b in range(w.batch):
        c = dec.new_cache(int(inp.lens[b]) + 2 * (G + 1) + 1)
        dec.prefill(c, inp.prompts[b][:-1])
        _log(name, t0, f"request {b}: prefilled {int(inp.lens[b])} tokens")
        complete_drafts(dec, inp, {b: c}, requests=[b])
        q = inp.draft_probs[b] if inp.modes[b] == SAMPLE else None
        r = oracle_verify(dec, c, inp.pending[b], inp.drafts[b], q, inp.uniforms[b], int(inp.modes[b]),
                          inp.temperature)
        logits[0, b] = r.logits.astype(np.float32)
        recs.append(_record(r, inp, b))
        _log(name, t0, f"request {b}: n {r.n_accepted} correction {r.correction} "
                       f"pinned {r.pinned_n}/{r.pinned_correction}")
        del c
    weights.close()
    return [_round_json(inp, recs)], logits


def _rounds_layer_major(name, w, inp, t0):
    """All requests layer by layer, several rounds with commits between them."""
    pool = ThreadPoolExecutor(8)
    dec = Decoder(w.model, lambda kind, layer: make_tensor(w.model, kind, layer, w.seed, pool),
                  keep_f64=False)
    B, G, V = w.batch, w.gamma, w.model.vocab
    if any(r not in ("chain_half", "random") for r in inp.recipe) or (inp.modes != GREEDY).any():
        raise ValueError("the layer-major driver handles greedy chain_half / random workloads")
    cap = int(inp.lens.max()) + (w.rounds + 1) * (G + 1) + 1
    caches = [dec.new_cache(cap) for _ in range(B)]
    dec.forward_many(caches, [p[:-1] for p in inp.prompts], want_logits=False)
    _log(name, t0, f"prefilled {B} x {int(inp.lens.max())} tokens")
    logits = np.zeros((w.rounds, B, G + 1, V), dtype=np.float32)
    rounds = []
    pending = inp.pending.copy()
    for rnd in range(w.rounds):
        ri = inp if rnd == 0 else make_inputs(w, round_index=rnd)
        ri.pending = pending.copy()
        ri.lens = np.array([c.length for c in caches], dtype=np.int32)
        chain_b = [b for b in range(B) if ri.recipe[b] == "chain_half"]
        if chain_b and G > 0:
            # the verifier's own argmax chain from the current state; the rows it
            # appends are rolled back (the verify call below overwrites them)
            start = [caches[b].length for b in chain_b]
            cur = [int(pending[b]) for b in chain_b]
            chains = [[] for _ in chain_b]
            for step in range(min(ri.chain_slots + 1, G + 1)):
                lg = dec.forward_many([caches[b] for b in chain_b], [[t] for t in cur])
                cur = [_argmax_f32(x[0]) for x in lg]
                for j, t in enumerate(cur):
                    chains[j].append(t)
                _log(name, t0, f"round {rnd}: chain step {step}")
            for j, b in enumerate(chain_b):
                caches[b].length = start[j]
                chain_drafts(ri, b, chains[j])
        starts = [c.length for c in caches]
        lgs = dec.forward_many(caches, [np.concatenate([[int(pending[b])], ri.drafts[b]]) for b in range(B)])
        recs = []
        for b in range(B):
            r = speculative_rows(lgs[b], ri.drafts[b], None, ri.uniforms[b], int(ri.modes[b]), ri.temperature)
            r.logits, r.start_len = lgs[b], starts[b]
            logits[rnd, b] = lgs[b].astype(np.float32)
            recs.append(_record(r, ri, b))
            pending[b] = commit(caches[b], r)
            _log(name, t0, f"round {rnd} request {b}: n {r.n_accepted} correction {r.correction} "
                           f"pinned {r.pinned_n}/{r.pinned_correction}")
        rounds.append(_round_json(ri, recs))
    pool.shutdown()
    return rounds, logits


def make(name: str) -> dict:
    w = workload(name)
    t0 = time.time()
    inp = make_inputs(w)
    if w.rounds == 1:
        rounds, logits = _one_round(name, w, inp, t0)
    else:
        rounds, logits = _rounds_layer_major(name, w, inp, t0)
    out = {"workload": name, "seed": w.seed, "recipe": w.draft_recipe, "temperature": inp.temperature,
           "gamma": w.gamma, "vocab": w.model.vocab, "drafts": rounds[0]["drafts"], "rounds": rounds,
           "logits_file": f"{name}_logits.npy", "oracle": "float64 NumPy oracle (oracle/)",
           "seconds": round(time.time() - t0, 1)}
    if inp.draft_probs is not None and w.draft_recipe == "draft_model":
        np.save(os.path.join(HERE, f"{name}_q.npy"), inp.draft_probs)
        out["draft_probs_file"] = f"{name}_q.npy"
    np.save(os.path.join(HERE, out["logits_file"]), logits)
    with open(os.path.join(HERE, f"{name}.json"), "w") as f:
        json.dump(out, f)
    return out


if __name__ == "__main__":
    for n in sys.argv[1:]:
        o = make(n)
        print(n, [[(r["n_accepted"], r["correction"], r["pinned_n"]) for r in rd["requests"]]
                  for rd in o["rounds"]], o["seconds"], "s", flush=True)
