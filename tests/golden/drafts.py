"""Stored draft tokens for the full-size workloads whose recipe needs the
verifier (written by tests/golden/make_golden.py, which calls only the
oracle).  Reading them needs no oracle."""

from __future__ import annotations

import json
import os

HERE = os.path.dirname(os.path.abspath(__file__))


def golden_path(name: str) -> str:
    return os.path.join(HERE, f"{name}.json")


def load_golden(name: str):
    p = golden_path(name)
    if not os.path.exists(p):
        return None
    with open(p) as f:
        return json.load(f)


def load_drafts(w, inp) -> str:
    """Replace inp.drafts (and the q rows of draft_model workloads) by the
    stored first-round drafts of workload w; returns a short description of
    where the drafts came from."""
    g = load_golden(w.name)
    if g is None or g.get("seed") != w.seed:
        return "uniform random ids (no stored chain drafts)"
    import numpy as np
    inp.drafts[:] = np.asarray(g["drafts"], dtype=np.int32)
    if g.get("draft_probs_file"):
        inp.draft_probs = np.load(os.path.join(HERE, g["draft_probs_file"]))
    return g.get("recipe", "stored")
