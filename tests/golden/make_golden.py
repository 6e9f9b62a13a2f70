"""Write the oracle's results for full-size workloads to tests/golden/.

    python -m tests.golden.make_golden c2_7b_greedy [c3_13b_sample ...]

Calls only the oracle (and the seeded input generators).  For each workload
it prefills the oracle's cache with the seeded prompt, fills the draft slots
that depend on the verifier (argmax chain, or q = softmax(logits/T + noise)
with drafts drawn from q), runs one verify, and stores: the drafts, q rows
(sampling workloads, as <name>_q.npy), the decisions and how decided they are,
the top-2 logits of every row, and the logits at a seeded sample of vocabulary
ids per row (plus the row argmax) for tolerance checks.
"""

from __future__ import annotations

import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

from synth import ModelWeights, make_inputs, workload  # noqa: E402
from tests.helpers import oracle_run  # noqa: E402

N_SAMPLED_IDS = 256


def make(name: str) -> dict:
    w = workload(name)
    t0 = time.time()
    inp = make_inputs(w)
    weights = ModelWeights(w.model, w.seed)
    orun = oracle_run(w, inp, weights=weights, keep_f64=False)
    rng = np.random.default_rng(w.seed + 77)
    reqs = []
    for b, r in enumerate(orun.results):
        lg = r.logits
        rows = []
        for i in range(lg.shape[0]):
            ids = np.unique(np.concatenate([rng.choice(w.model.vocab, N_SAMPLED_IDS, replace=False),
                                            [int(np.argmax(lg[i]))]]))
            top2 = np.sort(lg[i])[-2:]
            rows.append({"ids": ids.tolist(), "logits": lg[i, ids].tolist(),
                         "top2": top2[::-1].tolist(), "argmax": int(np.argmax(lg[i].astype(np.float32)))})
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
        reqs.append({"drafts": inp.drafts[b].tolist(), "n_accepted": r.n_accepted,
                     "correction": r.correction, "pinned_n": r.pinned_n,
                     "pinned_correction": r.pinned_correction, "draw_margin": r.draw_margin,
                     "row_margins": [x.margin for x in r.rows],
                     "row_ratios": [x.ratio for x in r.rows], "draw": draw, "draw_bound": draw_bound,
                     "fallback": r.fallback, "rows": rows,
                     "lens": int(inp.lens[b]), "mode": int(inp.modes[b])})
    out = {"workload": name, "seed": w.seed, "recipe": w.draft_recipe, "drafts": inp.drafts.tolist(),
           "uniforms": inp.uniforms.tolist(), "temperature": inp.temperature, "requests": reqs,
           "oracle": "float64 NumPy oracle (oracle/)", "seconds": round(time.time() - t0, 1)}
    if inp.draft_probs is not None:
        np.save(os.path.join(HERE, f"{name}_q.npy"), inp.draft_probs)
        out["draft_probs_file"] = f"{name}_q.npy"
    with open(os.path.join(HERE, f"{name}.json"), "w") as f:
        json.dump(out, f)
    weights.close()
    return out


if __name__ == "__main__":
    for n in sys.argv[1:]:
        o = make(n)
        print(n, [(r["n_accepted"], r["correction"], r["pinned_n"]) for r in o["requests"]], o["seconds"], "s",
              flush=True)
