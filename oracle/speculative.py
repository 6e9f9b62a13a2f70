"""Oracle verification step -- test infrastructure only.

Follows the cloud side of Algorithm 1 and Sec. III-B/III-C of the paper:

1. one forward pass of the verifier over the d+1 positions m+1 .. m+d+1
   gives the distributions p_1 .. p_{d+1} (row i conditions on the context
   plus drafts d_1 .. d_{i-1});
2. the drafts are checked left to right.  Sampling: draft x ~ q is accepted
   with probability alpha(x) = min(1, p(x)/q(x)); with u ~ U[0,1) this is the
   test u * q(x) < p(x).  Greedy decoding (Sec. III-A, argmax selection):
   x is accepted iff it is the argmax of the verifier's logits;
3. k = the number accepted before the first rejection (the longest verified
   prefix);
4. if k < d the rejected draft is replaced by a draw from
   p'(x) = norm(max(0, p(x) - q(x))) of row k+1 (greedy: its argmax); if all d
   are accepted there is no q at row d+1 and the extra token is drawn from
   p_{d+1} itself (greedy: its argmax), so every call emits k+1 >= 1 tokens;
5. the context grows by the k accepted drafts and the corrected token
   (m <- m + k + 1); the correction is the new pending token.

Readings the paper leaves open:
* p = softmax(logits / T) with T the sampling temperature; q arrives already
  tempered and is used as given;
* the acceptance test, the greedy argmax and the Gumbel-max draw are decided
  on float32 values (the verify kernels' precision): p(x) and q(x) are
  rounded to float32 and compared as float32(u) * q(x) < p(x); argmax ties
  go to the lowest token id;
* if max(0, p - q) has no mass the draw falls back to p (flagged);
* uniforms[b, i], i < d, drives the test of draft i+1; uniforms[b, d] keys the
  Gumbel noise of the correction / bonus draw.

Besides the decisions, each row reports how far it is from a flip so parity
checks can tell decided positions from knife-edge ones: the top-2 logit margin
(greedy) and |u - p(x)/q(x)| (sampling), and the top-2 gap of the draw's
perturbed scores.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

from .decoder import Decoder, KVCache
from .sampling import gumbel_top2, uniform_seed

GREEDY = 0
SAMPLE = 1
GREEDY_MARGIN = 0.1
RATIO_MARGIN = 1e-3
DRAW_MARGIN = 1e-3


def accept_test(u: float, p_x: float, q_x: float) -> bool:
    """alpha(x) = min(1, p/q) realised as u * q(x) < p(x), in float32."""
    return bool(np.float32(u) * np.float32(q_x) < np.float32(p_x))


def residual_distribution(p: np.ndarray, q: np.ndarray):
    """p' = norm(max(0, p - q)); returns (p', unnormalised mass)."""
    w = np.maximum(0.0, np.asarray(p, dtype=np.float64) - np.asarray(q, dtype=np.float64))
    mass = float(w.sum())
    return (w / mass if mass > 0 else w), mass


def _log_softmax(z: np.ndarray) -> np.ndarray:
    m = np.max(z)
    return z - (m + np.log(np.sum(np.exp(z - m))))


def _argmax_f32(row: np.ndarray) -> int:
    return int(np.argmax(np.asarray(row, dtype=np.float64).astype(np.float32)))


def _top2_margin(row: np.ndarray) -> float:
    r = np.asarray(row, dtype=np.float64)
    if r.size < 2:
        return np.inf
    top2 = np.partition(r, -2)[-2:]
    return float(top2[1] - top2[0])


@dataclass
class RowDecision:
    accepted: bool
    margin: float  # greedy: top-2 logit margin; sampling: |u - p/q|
    ratio: float = float("nan")  # sampling: p(x) / q(x)


@dataclass
class VerifyResult:
    n_accepted: int
    correction: int
    rows: List[RowDecision]
    draw_margin: float  # greedy: top-2 margin of the drawn row; sampling: top-2 score gap
    fallback: bool = False
    logits: Optional[np.ndarray] = None
    start_len: int = 0
    pinned_n: bool = True
    pinned_correction: bool = True
    notes: dict = field(default_factory=dict)


def speculative_rows(logits: np.ndarray, drafts: np.ndarray, q: Optional[np.ndarray],
                     uniforms: np.ndarray, mode: int, temperature: float = 1.0) -> VerifyResult:
    """Decide one request from its d+1 logit rows (float64 [d+1, V])."""
    logits = np.asarray(logits, dtype=np.float64)
    d = len(drafts)
    rows: List[RowDecision] = []
    n = d
    if mode == GREEDY:
        for i in range(d):
            ok = int(drafts[i]) == _argmax_f32(logits[i])
            rows.append(RowDecision(ok, _top2_margin(logits[i])))
            if not ok:
                n = i
                break
        corr = _argmax_f32(logits[n])
        res = VerifyResult(n, corr, rows, _top2_margin(logits[n]))
        res.pinned_n = all(r.margin > GREEDY_MARGIN for r in rows)
        res.pinned_correction = res.pinned_n and res.draw_margin > GREEDY_MARGIN
        return res

    if temperature <= 0:
        raise ValueError("sampling needs temperature > 0")
    z = logits / temperature
    for i in range(d):
        x = int(drafts[i])
        p_i = np.exp(_log_softmax(z[i]))
        p_x, q_x = float(p_i[x]), float(q[i, x])
        ok = accept_test(uniforms[i], p_x, q_x)
        ratio = np.inf if q_x == 0.0 else p_x / q_x
        gap = np.inf if not np.isfinite(ratio) else abs(float(uniforms[i]) - ratio)
        rows.append(RowDecision(ok, gap, ratio))
        if not ok:
            n = i
            break
    seed = uniform_seed(uniforms[d])
    fallback = False
    kind = "bonus"
    if n < d:
        p_n = np.exp(_log_softmax(z[n]))
        w = np.maximum(0.0, p_n - np.asarray(q[n], dtype=np.float64))
        if w.sum() > 0:
            kind = "residual"
            with np.errstate(divide="ignore"):
                corr, second, gap = gumbel_top2(np.log(w), seed)
        else:
            fallback = True
            kind = "fallback"
            corr, second, gap = gumbel_top2(z[n], seed)
    else:
        corr, second, gap = gumbel_top2(z[d], seed)
    res = VerifyResult(n, corr, rows, gap, fallback)
    res.notes["draw"] = {"kind": kind, "row": n, "top": corr, "second": second}
    res.pinned_n = all(r.margin > RATIO_MARGIN for r in rows)
    res.pinned_correction = res.pinned_n and gap > DRAW_MARGIN and not fallback
    return res


def verify(model: Decoder, cache: KVCache, pending: int, drafts: np.ndarray,
           q: Optional[np.ndarray], uniforms: np.ndarray, mode: int,
           temperature: float = 1.0) -> VerifyResult:
    """One verify call: forward over [pending, d_1 .. d_gamma] appended to the
    cache, then the accept/reject chain.  The cache keeps all gamma+1 rows
    until ``commit`` rolls it back to the accepted prefix."""
    start = cache.length
    tokens = np.concatenate([[int(pending)], np.asarray(drafts, dtype=np.int64)])
    logits = model.forward(cache, tokens)
    res = speculative_rows(logits, drafts, q, uniforms, mode, temperature)
    res.logits = logits
    res.start_len = start
    return res


def commit(cache: KVCache, res: VerifyResult) -> int:
    """Context update m <- m + k + 1: keep the rows of the pending token and
    the k accepted drafts, drop the rest; returns the new pending token."""
    cache.length = res.start_len + res.n_accepted + 1
    return res.correction


@dataclass
class LoopResult:
    """Output of an Algorithm 1 run: the emitted tokens (after the prompt), the
    number of cloud verify calls, and the accepted drafts per call."""

    tokens: List[int]
    calls: int
    accepted: List[int]
    margins: List[float] = field(default_factory=list)  # greedy: top-2 margin behind each emitted token


def decode_step(model: Decoder, cache: KVCache, pending: int, u: float, mode: int,
                temperature: float = 1.0):
    """One autoregressive step (a verify call with no drafts): append
    ``pending``, draw the next token from the row's distribution (greedy: its
    argmax; sampling: the Gumbel-max draw keyed by ``u``).  Returns (token,
    logits row, margin of the draw)."""
    res = verify(model, cache, pending, np.zeros(0, dtype=np.int64), None, np.array([u]), mode, temperature)
    cache.length = res.start_len + 1
    return res.correction, res.logits[0], res.draw_margin


def algorithm1(target: Decoder, draft: Decoder, prompt: np.ndarray, gamma: int, max_new: int,
               mode: int, uniforms, temperature: float = 1.0, capacity: Optional[int] = None) -> LoopResult:
    """Algorithm 1 of the paper with both sides on one machine.

    Edge: the draft model continues the context autoregressively for
    ``gamma`` tokens, keeping the distribution q_j each token was drawn from.
    Cloud: one verify call scores them (``verify``: accept/reject, correction
    or bonus token).  Both sides keep the accepted prefix plus the correction
    (m <- m + k + 1); the draft's cache is cut back to the same length, and
    when every draft was accepted the draft first appends its last draft,
    which it never ran.  Stops after ``max_new`` emitted tokens.

    ``uniforms`` yields float32 values in [0, 1): one per draft step (its
    draw), then gamma + 1 per cloud call, in that order (greedy ignores them).
    The prompt's last id is the first pending token."""
    prompt = np.asarray(prompt, dtype=np.int64)
    cap = capacity or (len(prompt) + max_new + gamma + 2)
    tc, dc = target.new_cache(cap), draft.new_cache(cap)
    target.prefill(tc, prompt[:-1])
    draft.prefill(dc, prompt[:-1])
    pending = int(prompt[-1])
    out: List[int] = []
    accepted: List[int] = []
    margins: List[float] = []
    calls = 0
    while len(out) < max_new:
        start = tc.length
        # edge: gamma draft tokens and their distributions
        drafts = np.zeros(gamma, dtype=np.int64)
        q = np.zeros((gamma, target.shape.vocab))
        dp = pending
        for j in range(gamma):
            tok, row, _ = decode_step(draft, dc, dp, next(uniforms), mode, temperature)
            z = row / temperature if mode == SAMPLE else row
            q[j] = np.exp(_log_softmax(z)).astype(np.float32)
            drafts[j] = tok
            dp = tok
        # cloud: one verify call
        u = np.array([next(uniforms) for _ in range(gamma + 1)])
        res = verify(target, tc, pending, drafts, q if mode == SAMPLE else None, u, mode, temperature)
        calls += 1
        n = res.n_accepted
        new_pending = commit(tc, res)
        if mode == GREEDY:
            margins += [r.margin for r in res.rows[:n]] + [res.draw_margin]
        # edge: keep [pending, d_1 .. d_n]; with all accepted, run d_gamma first
        if n == gamma:
            draft.forward(dc, drafts[gamma - 1:], want_logits=False)
        dc.length = start + n + 1
        out += [int(t) for t in drafts[:n]] + [new_pending]
        accepted.append(n)
        pending = new_pending
    return LoopResult(out[:max_new], calls, accepted, margins[:max_new])


def target_only(target: Decoder, prompt: np.ndarray, max_new: int, mode: int, uniforms,
                temperature: float = 1.0) -> LoopResult:
    """Plain autoregressive decoding with the verifier (one call per token):
    the baseline Algorithm 1 is measured against."""
    prompt = np.asarray(prompt, dtype=np.int64)
    tc = target.new_cache(len(prompt) + max_new + 1)
    target.prefill(tc, prompt[:-1])
    pending = int(prompt[-1])
    out, margins = [], []
    for _ in range(max_new):
        pending, _, m = decode_step(target, tc, pending, next(uniforms), mode, temperature)
        out.append(pending)
        margins.append(m)
    return LoopResult(out, max_new, [0] * max_new, margins)
