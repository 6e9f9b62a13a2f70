"""Shared test helpers: build a workload's inputs with the oracle, run the
oracle verify, run the HIP verify through the C ABI, compare them."""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

from oracle import GREEDY, SAMPLE, Decoder, verify as oracle_verify
from oracle.speculative import _argmax_f32
from synth import ModelWeights, make_inputs
from synth.inputs import draw_from, softmax64

LOGIT_TOL = {"f32": 1e-4, "bf16": 5e-2}

# one JSON line per parity check (decided / excluded / in-band mismatch
# counts), printed as the check runs and again in pytest's terminal summary
PARITY_LINES: List[str] = []


def report_parity(name: str, counts: dict) -> None:
    import json
    line = json.dumps({"parity": name, **counts})
    PARITY_LINES.append(line)
    print(line, flush=True)


@dataclass
class OracleRun:
    inputs: object
    results: list
    caches: list
    chains: list = field(default_factory=list)


def chain_drafts(inp, b: int, chain) -> None:
    """chain_half recipe for request b: its first chain_slots drafts are the
    verifier's argmax chain; the next draft (a uniform id) is moved off the
    argmax of its row so the chain ends there."""
    k = inp.chain_slots
    G, V = inp.workload.gamma, inp.workload.model.vocab
    inp.drafts[b, :k] = chain[:k]
    if k < G and inp.drafts[b, k] == chain[k]:
        inp.drafts[b, k] = (chain[k] + 1) % V


def complete_drafts(dec: Decoder, inp, caches, requests=None) -> None:
    """Fill the draft slots that depend on the verifier (chain_half,
    draft_model recipes) using the oracle, in place.  ``caches[b]`` is
    request b's prefilled cache; ``requests`` limits the work to some b."""
    w = inp.workload
    G = w.gamma
    for b in (range(w.batch) if requests is None else requests):
        rec = inp.recipe[b]
        if rec == "chain_half" and G > 0:
            c = caches[b].copy()
            cur, chain = int(inp.pending[b]), []
            for _ in range(min(inp.chain_slots + 1, G + 1)):
                cur = _argmax_f32(dec.forward(c, [cur])[0])
                chain.append(cur)
            chain_drafts(inp, b, chain)
        elif rec == "draft_model":
            c = caches[b].copy()
            cur = int(inp.pending[b])
            for i in range(G):
                lg = dec.forward(c, [cur])[0]
                q = softmax64(lg / inp.temperature + inp.q_noise[b, i].astype(np.float64))
                inp.draft_probs[b, i] = q.astype(np.float32)
                cur = draw_from(inp.draft_probs[b, i], inp.draft_u[b, i])
                inp.drafts[b, i] = cur


def oracle_run(w, inp=None, weights: Optional[ModelWeights] = None, cap: Optional[int] = None,
               keep_f64: bool = True) -> OracleRun:
    shape = w.model
    weights = weights or ModelWeights(shape, w.seed)
    dec = Decoder(shape, weights.get, keep_f64=keep_f64)
    inp = inp or make_inputs(w)
    cap = cap or int(inp.lens.max()) + 2 * (w.gamma + 1) + 1
    caches = []
    for b in range(w.batch):
        c = dec.new_cache(cap)
        dec.prefill(c, inp.prompts[b][:-1])
        caches.append(c)
    complete_drafts(dec, inp, caches)
    results = []
    for b in range(w.batch):
        q = inp.draft_probs[b] if inp.modes[b] == SAMPLE else None
        results.append(oracle_verify(dec, caches[b], inp.pending[b], inp.drafts[b], q, inp.uniforms[b],
                                     int(inp.modes[b]), inp.temperature))
    return OracleRun(inp, results, caches)


@dataclass
class Parity:
    logit_err: float
    n_match_all: int
    corr_match_all: int
    pinned_n: int
    pinned_corr: int
    pinned_n_fail: List[int]
    pinned_corr_fail: List[int]
    excluded_n: int
    excluded_corr: int
    total: int
    stable_n: int = 0
    stable_corr: int = 0
    stable_n_fail: List[int] = field(default_factory=list)
    stable_corr_fail: List[int] = field(default_factory=list)


def stability(res, logits: np.ndarray, q: Optional[np.ndarray], mode: int, temperature: float,
              eps: float):
    """Whether n_accepted and the correction are decided beyond what logits
    off by at most eps (max abs) could change.

    greedy: a row's argmax cannot move when its top-2 margin exceeds 2 eps.
    sampling: z = logit / T moves by at most eps/T, so p(x) / q(x) moves by a
    factor within exp(+-2 eps / T); the test u q < p cannot flip when
    |u - p/q| > (p/q)(exp(2 eps/T) - 1).  A bonus / fallback draw scores
    z_v + G_v, each off by at most eps/T; a residual draw scores
    log(p_v - q_v) + G_v, off by at most p_v (exp(2 eps/T) - 1) / (p_v - q_v).
    Small constants cover the float32 evaluation of the same quantities."""
    if mode == GREEDY:
        n_ok = all(r.margin > 2 * eps + 1e-6 for r in res.rows)
        return n_ok, n_ok and res.draw_margin > 2 * eps + 1e-6
    f = float(np.expm1(2 * eps / temperature))
    n_ok = all((not np.isfinite(r.ratio)) or r.margin > r.ratio * f + 2e-6 for r in res.rows)
    d = res.notes["draw"]
    if d["kind"] == "residual":
        z = np.asarray(logits[d["row"]], dtype=np.float64) / temperature
        pz = np.exp(z - z.max())
        pz /= pz.sum()
        bound = 0.0
        for v in (d["top"], d["second"]):
            w = pz[v] - float(q[d["row"], v])
            bound += pz[v] * f / w if w > 0 else np.inf
        c_ok = res.draw_margin > bound + 1e-5
    else:
        c_ok = res.draw_margin > 2 * eps / temperature + 1e-5
    return n_ok, n_ok and c_ok


def compare(orun: OracleRun, gpu_logits: np.ndarray, gpu_n: np.ndarray, gpu_corr: np.ndarray) -> Parity:
    inp = orun.inputs
    errs = [np.abs(gpu_logits[b].astype(np.float64) - r.logits).max() for b, r in enumerate(orun.results)]
    p = Parity(float(max(errs)), 0, 0, 0, 0, [], [], 0, 0, len(orun.results))
    for b, r in enumerate(orun.results):
        nm = int(gpu_n[b]) == r.n_accepted
        cm = int(gpu_corr[b]) == r.correction
        p.n_match_all += nm
        p.corr_match_all += nm and cm
        if r.pinned_n:
            p.pinned_n += 1
            if not nm:
                p.pinned_n_fail.append(b)
        else:
            p.excluded_n += 1
        if r.pinned_correction:
            p.pinned_corr += 1
            if not (nm and cm):
                p.pinned_corr_fail.append(b)
        else:
            p.excluded_corr += 1
        q = inp.draft_probs[b] if inp.draft_probs is not None else None
        sn, sc = stability(r, r.logits, q, int(inp.modes[b]), inp.temperature, errs[b])
        if sn:
            p.stable_n += 1
            if not nm:
                p.stable_n_fail.append(b)
        if sc:
            p.stable_corr += 1
            if not (nm and cm):
                p.stable_corr_fail.append(b)
    return p


def gpu_setup(w, weights: Optional[ModelWeights] = None, max_len: Optional[int] = None, max_batch=None):
    from paper_2608_13076_amd import spade
    shape = w.model
    weights = weights or ModelWeights(shape, w.seed)
    max_len = max_len or (w.ctx[1] + 2 * (w.gamma + 1) + 8)
    model = spade.Model(shape, max_batch or w.batch, w.gamma, max_len)
    for layer in range(shape.n_layers):
        for kind in ("wq", "wk", "wv", "wo", "wg", "wu", "wd", "g_attn", "g_ffn"):
            model.load_numpy(kind, layer, weights.get(kind, layer))
    for kind in ("embed", "g_final", "lm_head"):
        model.load_numpy(kind, None, weights.get(kind))
    kv = spade.KVCache(model, max_batch or w.batch, max_len)
    return model, kv


def gpu_prefill(kv, inp) -> None:
    for b, pr in enumerate(inp.prompts):
        kv.prefill(b, pr)


def gpu_verify(model, kv, inp, want_logits=True):
    import torch
    from paper_2608_13076_amd import spade
    buf = spade.VerifyBuffers(model, inp.drafts, inp.draft_probs, inp.uniforms, inp.modes, want_logits)
    spade.verify(model, kv, buf, inp.temperature)
    torch.cuda.synchronize()
    lg = buf.logits.cpu().numpy() if want_logits else None
    return lg, buf.n.cpu().numpy(), buf.corr.cpu().numpy(), buf


def gpu_setup_streaming(w, max_len: int, max_batch: Optional[int] = None):
    """Model + KV on the GPU with weights generated and uploaded one tensor at
    a time (no host copy of the whole model)."""
    from paper_2608_13076_amd import spade
    from synth import iter_weights
    model = spade.Model(w.model, max_batch or w.batch, w.gamma, max_len)
    for kind, layer, arr in iter_weights(w.model, w.seed):
        model.load_numpy(kind, layer, arr)
        if kind == "wd" and layer is not None and layer % 8 == 7:
            print(f"  [{w.name}] weights of layer {layer} loaded", flush=True)
    kv = spade.KVCache(model, max_batch or w.batch, max_len)
    return model, kv


# The cache layout (include/spade.h, spade_kv_bytes): K and V in blocks of
# V_BLOCK positions.  bf16 K: the B operands of S = Q K^T in MFMA order, 1 KB
# fragments (16-position group, 32-feature step) whose lane 16 ((f / 8) % 4)
# + p % 16 holds features 8 ((f / 8) % 4) .. + 7; float32 K: [V_BLOCK][head_dim].
# bf16 V: the B operands of O = P V, 1 KB fragments (16-feature tile,
# 32-position step) whose lane 16 ((p / 8) % 4) + f % 16 holds positions
# 8 ((p / 8) % 4) .. + 7; float32 V: [head_dim][V_BLOCK].  Positions per
# (request, K/V head): max_len rounded up to a whole block.
V_BLOCK = 256


def kv_stride(max_len: int) -> int:
    return (max_len + V_BLOCK - 1) // V_BLOCK * V_BLOCK


def v_phys_index(shape, S: int) -> np.ndarray:
    """[head_dim, S]: the element offset of (feature, position) in a
    (request, K/V head) region of the V cache."""
    hd = shape.head_dim
    f = np.arange(hd)[:, None]
    pos = np.arange(S)[None, :]
    blk, p = pos // V_BLOCK, pos % V_BLOCK
    if shape.kv_dtype == "bf16":
        return blk * hd * V_BLOCK + (((f // 16) * (V_BLOCK // 32) + p // 32) * 64 + ((p // 8) % 4) * 16 + f % 16) * 8 + p % 8
    return (blk * hd + f) * V_BLOCK + p


def k_phys_index(shape, S: int) -> np.ndarray:
    """[S, head_dim]: the element offset of (position, feature) in a
    (request, K/V head) region of the K cache."""
    hd = shape.head_dim
    pos = np.arange(S)[:, None]
    f = np.arange(hd)[None, :]
    if shape.kv_dtype == "bf16":
        blk, p = pos // V_BLOCK, pos % V_BLOCK
        return blk * hd * V_BLOCK + (((p // 16) * (hd // 32) + f // 32) * 64 + ((f // 8) % 4) * 16 + p % 16) * 8 + f % 8
    return pos * hd + f


def kv_views(kv, shape, max_len: int):
    """K and V as [layer][request][K/V head][region] views of the cache
    (k_phys_index and v_phys_index map a region's elements)."""
    import torch
    S = kv_stride(max_len)
    dt = torch.int16 if shape.kv_dtype == "bf16" else torch.float32
    half = kv.buf.numel() // 2
    n = shape.n_layers * kv.max_batch * shape.kv_heads * S * shape.head_dim
    k = kv.buf[:half].view(dt)[:n].view(shape.n_layers, kv.max_batch, shape.kv_heads, S * shape.head_dim)
    v = kv.buf[half:].view(dt)[:n].view(shape.n_layers, kv.max_batch, shape.kv_heads, S * shape.head_dim)
    return k, v


def k_by_position(k, shape, max_len: int):
    """[..., region] -> [..., position, head_dim] (a copy)."""
    import torch
    S = kv_stride(max_len)
    idx = torch.as_tensor(k_phys_index(shape, S).reshape(-1), device=k.device)
    return k[..., idx].reshape(*k.shape[:-1], S, shape.head_dim)


def v_by_position(v, shape, max_len: int):
    """[..., region] -> [..., head_dim, position] (a copy)."""
    import torch
    S = kv_stride(max_len)
    idx = torch.as_tensor(v_phys_index(shape, S).reshape(-1), device=v.device)
    return v[..., idx].reshape(*v.shape[:-1], shape.head_dim, S)

