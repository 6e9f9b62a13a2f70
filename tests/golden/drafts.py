"""Stored draft tokens for the full-size workloads whose recipe needs the
verifier's own greedy chain (written by tests/golden/make_golden.py, which
calls only the oracle).  Reading them needs no oracle."""

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
    """Replace inp.drafts (and q rows when stored) by the golden drafts of
    workload w; returns a short description of where the drafts came from."""
    g = load_golden(w.name)
    if g is None or g.get("seed") != w.seed:
        return "uniform random ids (no stored chain drafts)"
    import numpy as np
    inp.drafts[:] = np.asarray(g["drafts"], dtype=np.int32)
    return g.get("recipe", "stored")
