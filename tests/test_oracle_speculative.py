"""Pins of the oracle's verification step (Sec. III-B/III-C, Algorithm 1).

* the acceptance test realises alpha(x) = min(1, p/q) exactly (its accepting
  set of u is [0, min(1, p/q)));
* exact enumeration on a table model: speculative decoding rounds, chained
  until T tokens are out, emit sequences with exactly the verifier's
  autoregressive probabilities (the paper's "statistically identical" claim);
* Monte Carlo chi-square of the full step (uniforms + Gumbel-max draw) and of
  both samplers against their target distributions;
* closed forms: P(accept) = sum_x min(p, q) = 1 - TV(p, q); q = p accepts
  everything; one-hot p and q reduce sampling to greedy; q = one-hot(x) with
  p(x) = 0 always rejects and the residual is p;
* published SplitMix64 outputs;
* on the transformer oracle: the verifier's own greedy chain is fully
  accepted, an adversarial first draft rejects at 0, a k-token chain prefix
  gives n = k; commit + second round equals a fresh prefill of the committed
  sequence, and poisoned rows past the committed length change nothing.
"""

import itertools

import numpy as np
import pytest
from scipy.stats import chisquare

from oracle import (GREEDY, SAMPLE, Decoder, accept_test, commit, gumbel_argmax,
                    inverse_cdf_draw, residual_distribution, speculative_rows,
                    splitmix64_stream, verify)
from oracle.sampling import gumbel_noise
from synth import ModelWeights
from synth.configs import ModelShape


def _threshold(p_x, q_x):
    """Measure of {u in [0,1): accept_test(u, p, q)}, by bisection."""
    if not accept_test(0.0, p_x, q_x):
        return 0.0
    if accept_test(np.nextafter(np.float32(1.0), np.float32(0.0)), p_x, q_x):
        return 1.0
    lo, hi = 0.0, 1.0
    for _ in range(60):
        mid = 0.5 * (lo + hi)
        if accept_test(mid, p_x, q_x):
            lo = mid
        else:
            hi = mid
    return lo


def test_splitmix64_published_outputs():
    assert [int(x) for x in splitmix64_stream(0, 3)] == [
        0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]
    assert [int(x) for x in splitmix64_stream(1234567, 3)] == [
        6457827717110365317, 3203168211198807973, 9817491932198370423]
    # counter form: output n of the stream does not depend on where we start
    assert int(splitmix64_stream(99, 1, start=5)[0]) == int(splitmix64_stream(99, 6)[5])


def test_accept_threshold_is_min_one_p_over_q():
    rng = np.random.default_rng(0)
    for _ in range(200):
        p, q = rng.random(), rng.random()
        if rng.random() < 0.2:
            p = q * 0.5
        t = _threshold(p, q)
        assert abs(t - min(1.0, p / q)) < 2e-7, (p, q, t)
    assert _threshold(0.0, 0.3) == 0.0  # p(x) = 0 always rejects
    assert _threshold(0.2, 0.0) == 1.0  # q(x) = 0 < p(x) always accepts


def test_residual_distribution():
    p = np.array([0.5, 0.2, 0.2, 0.1])
    q = np.array([0.1, 0.4, 0.2, 0.3])
    r, mass = residual_distribution(p, q)
    np.testing.assert_allclose(r, [1.0, 0, 0, 0])
    assert abs(mass - 0.4) < 1e-15
    p2 = np.array([0.3, 0.3, 0.4])
    r2, _ = residual_distribution(p2, np.array([0.0, 0.0, 1.0]))
    np.testing.assert_allclose(r2, [0.5, 0.5, 0.0])


class TableModel:
    """p(. | prefix) and q(. | prefix) as seeded Dirichlet tables."""

    def __init__(self, V, seed, alpha_p=0.7, alpha_q=0.7, mix=0.5):
        self.V, self.seed = V, seed
        self.ap, self.aq, self.mix = alpha_p, alpha_q, mix
        self._p, self._q = {}, {}

    def _rng(self, prefix, tag):
        return np.random.default_rng([self.seed, tag, len(prefix)] + list(prefix))

    def p(self, prefix):
        prefix = tuple(prefix)
        if prefix not in self._p:
            self._p[prefix] = self._rng(prefix, 1).dirichlet([self.ap] * self.V)
        return self._p[prefix]

    def q(self, prefix):
        prefix = tuple(prefix)
        if prefix not in self._q:
            own = self._rng(prefix, 2).dirichlet([self.aq] * self.V)
            self._q[prefix] = self.mix * own + (1 - self.mix) * self.p(prefix)
        return self._q[prefix]


def _round_outcomes(tm, prefix, d, exact_alpha=False):
    """Exact distribution of the tokens one verify round emits.  The
    acceptance probability is the measured threshold of ``accept_test``
    (float32 decision), or min(1, p/q) itself with ``exact_alpha``."""
    out = {}
    for drafts in itertools.product(range(tm.V), repeat=d):
        pd = 1.0
        for i, x in enumerate(drafts):
            pd *= tm.q(prefix + drafts[:i])[x]
        if pd == 0:
            continue
        reach = pd  # probability of reaching draft i with all before accepted
        for i, x in enumerate(drafts):
            ctx = prefix + drafts[:i]
            px, qx = tm.p(ctx)[x], tm.q(ctx)[x]
            a = min(1.0, px / qx) if exact_alpha else _threshold(px, qx)
            r, mass = residual_distribution(tm.p(ctx), tm.q(ctx))
            if a < 1.0:
                for y in range(tm.V):
                    if r[y] > 0:
                        e = drafts[:i] + (y,)
                        out[e] = out.get(e, 0.0) + reach * (1 - a) * r[y]
            reach *= a
            if reach == 0:
                break
        else:
            pb = tm.p(prefix + drafts)
            for y in range(tm.V):
                e = drafts + (y,)
                out[e] = out.get(e, 0.0) + reach * pb[y]
    return out


def _emit_dist(tm, prefix, d, T, exact_alpha=False):
    dist = {}
    for e, pr in _round_outcomes(tm, prefix, d, exact_alpha).items():
        if len(e) >= T:
            dist[e[:T]] = dist.get(e[:T], 0.0) + pr
        else:
            for rest, pr2 in _emit_dist(tm, prefix + e, d, T - len(e), exact_alpha).items():
                dist[e + rest] = dist.get(e + rest, 0.0) + pr * pr2
    return dist


@pytest.mark.parametrize("exact_alpha,tol", [(True, 1e-12), (False, 1e-6)])
@pytest.mark.parametrize("V,d,T", [(3, 1, 3), (3, 2, 3), (4, 2, 3), (3, 3, 4)])
def test_exact_enumeration_matches_verifier_distribution(V, d, T, exact_alpha, tol):
    """With alpha = min(1, p/q) the emitted sequences follow the verifier's
    autoregressive distribution to rounding; with the float32 acceptance test
    the deviation stays at the float32 rounding of p(x) and q(x)."""
    tm = TableModel(V, seed=10 * V + d)
    dist = _emit_dist(tm, (), d, T, exact_alpha)
    assert abs(sum(dist.values()) - 1.0) < tol
    for seq in itertools.product(range(V), repeat=T):
        target = 1.0
        for t in range(T):
            target *= tm.p(seq[:t])[seq[t]]
        assert abs(dist.get(seq, 0.0) - target) < tol, (seq, dist.get(seq), target)


def test_exact_acceptance_rate_is_one_minus_tv():
    tm = TableModel(6, seed=3)
    p, q = tm.p(()), tm.q(())
    acc = sum(q[x] * _threshold(p[x], q[x]) for x in range(6))
    # float32 decision: p(x) and q(x) are rounded to float32 before the test
    assert abs(acc - np.minimum(p, q).sum()) < 1e-7
    assert abs(np.minimum(p, q).sum() - (1 - 0.5 * np.abs(p - q).sum())) < 1e-12


def _logits_from(p):
    return np.log(np.maximum(p, 1e-300))


def test_monte_carlo_first_token_and_acceptance_rate():
    """Full step with uniforms and the Gumbel-max correction: the first
    emitted token is distributed as p(. | prefix) (chi-square), and the
    acceptance rate of draft 1 matches 1 - TV(p, q)."""
    V, d, N = 8, 3, 60000
    tm = TableModel(V, seed=42)
    rng = np.random.default_rng(7)
    counts = np.zeros(V)
    accepted1 = 0
    logit_rows = {}
    for _ in range(N):
        drafts = []
        for i in range(d):
            drafts.append(int(rng.choice(V, p=tm.q(tuple(drafts)))))
        rows = []
        for i in range(d + 1):
            ctx = tuple(drafts[:i])
            if ctx not in logit_rows:
                logit_rows[ctx] = _logits_from(tm.p(ctx))
            rows.append(logit_rows[ctx])
        q = np.stack([tm.q(tuple(drafts[:i])) for i in range(d)])
        u = rng.random(d + 1).astype(np.float32)
        res = speculative_rows(np.stack(rows), np.array(drafts), q, u, SAMPLE, 1.0)
        first = drafts[0] if res.n_accepted >= 1 else res.correction
        counts[first] += 1
        accepted1 += res.n_accepted >= 1
    exp = tm.p(()) * N
    assert chisquare(counts, exp).pvalue > 1e-3
    rate = accepted1 / N
    target = np.minimum(tm.p(()), tm.q(())).sum()
    assert abs(rate - target) < 4 * np.sqrt(target * (1 - target) / N)


def _block_chi_square(tm, d, N, seed, q_equals_p=False):
    """Monte Carlo of whole verify rounds through ``speculative_rows`` (the
    float32 acceptance test, the Gumbel-max residual and bonus draws keyed by
    the last uniform): the emitted block drafts[:n] + (correction,) against
    its exact distribution from ``_round_outcomes`` (chi-square, cells with
    small expectation pooled)."""
    V = tm.V
    rng = np.random.default_rng(seed)
    qf = tm.p if q_equals_p else tm.q
    exact = {}
    for e, pr in _round_outcomes_q(tm, qf, d).items():
        exact[e] = exact.get(e, 0.0) + pr
    counts = {}
    logit_rows = {}
    for _ in range(N):
        drafts = []
        for i in range(d):
            drafts.append(int(rng.choice(V, p=qf(tuple(drafts)))))
        rows = []
        for i in range(d + 1):
            ctx = tuple(drafts[:i])
            if ctx not in logit_rows:
                logit_rows[ctx] = _logits_from(tm.p(ctx))
            rows.append(logit_rows[ctx])
        q = np.stack([qf(tuple(drafts[:i])) for i in range(d)])
        u = rng.random(d + 1).astype(np.float32)
        res = speculative_rows(np.stack(rows), np.array(drafts), q, u, SAMPLE, 1.0)
        e = tuple(drafts[:res.n_accepted]) + (res.correction,)
        counts[e] = counts.get(e, 0) + 1
    assert set(counts) <= {e for e, pr in exact.items() if pr > 0}, "emitted a block of probability 0"
    keys = sorted(exact, key=lambda e: -exact[e])
    obs, exp, pool_o, pool_e = [], [], 0, 0.0
    for e in keys:
        if exact[e] * N >= 10:
            obs.append(counts.get(e, 0))
            exp.append(exact[e] * N)
        else:
            pool_o += counts.get(e, 0)
            pool_e += exact[e] * N
    if pool_e > 0:
        obs.append(pool_o)
        exp.append(pool_e)
    exp = np.asarray(exp) * (sum(obs) / sum(exp))
    return chisquare(obs, exp).pvalue, counts, exact


def _round_outcomes_q(tm, qf, d):
    """``_round_outcomes`` with q(. | prefix) given by ``qf`` and the float32
    acceptance threshold."""
    class _Q:
        V = tm.V
        p = staticmethod(tm.p)
        q = staticmethod(qf)
    return _round_outcomes(_Q, (), d)


def test_whole_block_chi_square():
    """Every position of the emitted block -- accepted drafts, the residual
    draw at whichever row rejects, and the bonus draw from the row after the
    last draft when all are accepted -- has the exact distribution of a
    verify round (Sec. III-C; Algorithm 1)."""
    tm = TableModel(4, seed=21, mix=0.6)
    pv, counts, exact = _block_chi_square(tm, d=2, N=40000, seed=8)
    assert pv > 1e-3, pv
    # each kind of ending was exercised: rejection at rows 0 and 1, and a bonus
    lens = {len(e) for e in counts}
    assert lens == {1, 2, 3}


def test_q_equal_p_bonus_follows_last_row():
    """q = p accepts every draft (Sec. III-C: min(1, p/q) = 1), so every
    round emits the d drafts plus a bonus token drawn from p(. | prefix,
    drafts): the block distribution is the verifier's chain probability."""
    tm = TableModel(5, seed=33)
    pv, counts, exact = _block_chi_square(tm, d=2, N=30000, seed=9, q_equals_p=True)
    assert pv > 1e-3, pv
    assert {len(e) for e in counts} == {3}


@pytest.mark.parametrize("sampler", ["gumbel", "inverse_cdf"])
def test_samplers_chi_square(sampler):
    rng = np.random.default_rng(11)
    w = rng.dirichlet([0.5] * 10)
    w[3] = 0.0
    N = 40000
    counts = np.zeros(10)
    seeds = rng.integers(0, 2 ** 32, N)
    with np.errstate(divide="ignore"):
        lw = np.log(w)
    for s in seeds:
        if sampler == "gumbel":
            v, _ = gumbel_argmax(lw, int(s))
        else:
            v = inverse_cdf_draw(w, rng.random())
        counts[v] += 1
    assert counts[3] == 0
    keep = w > 0
    assert chisquare(counts[keep], w[keep] / w[keep].sum() * N).pvalue > 1e-3


def test_gumbel_noise_is_standard_gumbel():
    g = gumbel_noise(12345, 200000)
    # mean = Euler-Mascheroni constant, variance = pi^2 / 6
    assert abs(g.mean() - 0.5772156649) < 0.01
    assert abs(g.var() - np.pi ** 2 / 6) < 0.03


def test_special_cases():
    rng = np.random.default_rng(5)
    V, d = 7, 4
    logits = rng.standard_normal((d + 1, V))
    p = np.exp(logits - logits.max(1, keepdims=True))
    p /= p.sum(1, keepdims=True)
    drafts = rng.integers(0, V, d)
    u = rng.random(d + 1).astype(np.float32)
    # q = p: every draft is accepted for any u < 1
    res = speculative_rows(logits, drafts, p[:d].astype(np.float64), u, SAMPLE)
    assert res.n_accepted == d
    # one-hot p and q: sampling reduces to greedy
    big = np.full((d + 1, V), -1e4)
    top = rng.integers(0, V, d + 1)
    big[np.arange(d + 1), top] = 0.0
    drafts2 = top[:d].copy()
    drafts2[2] = (top[2] + 1) % V
    q1 = np.zeros((d, V))
    q1[np.arange(d), drafts2] = 1.0
    rs = speculative_rows(big, drafts2, q1, u, SAMPLE)
    rg = speculative_rows(big, drafts2, None, u, GREEDY)
    assert (rs.n_accepted, rs.correction) == (rg.n_accepted, rg.correction) == (2, top[2])
    # q = one-hot(x) with p(x) = 0: rejected, the correction is drawn from p
    lg = np.log(np.array([[0.5, 0.5, 0.0, 0.0], [0.25] * 4]) + 1e-300)
    qx = np.array([[0.0, 0.0, 1.0, 0.0]])
    for s in range(50):
        r = speculative_rows(lg, np.array([2]), qx, np.array([0.0, s / 50.0], np.float32), SAMPLE)
        assert r.n_accepted == 0 and r.correction in (0, 1) and not r.fallback


MINI = ModelShape("spec-mini", n_layers=2, d_model=128, n_heads=2, head_dim=64, d_ffn=256,
                  vocab=173, init_std=0.08, gain_std=0.1)


def _greedy_chain(dec, cache, pending, n):
    c = cache.copy()
    toks, cur = [], pending
    for _ in range(n):
        cur = int(np.argmax(dec.forward(c, [cur])[0].astype(np.float32)))
        toks.append(cur)
    return np.array(toks)


def test_greedy_chain_adversarial_and_partial():
    mw = ModelWeights(MINI, 3)
    dec = Decoder(MINI, mw.get, keep_f64=True)
    rng = np.random.default_rng(9)
    prompt = rng.integers(0, MINI.vocab, 40)
    base = dec.new_cache(64)
    dec.prefill(base, prompt[:-1])
    gamma = 5
    chain = _greedy_chain(dec, base, prompt[-1], gamma + 1)
    u = np.zeros(gamma + 1, np.float32)
    r = verify(dec, base.copy(), prompt[-1], chain[:gamma], None, u, GREEDY)
    assert r.n_accepted == gamma and r.correction == chain[gamma]
    bad = chain[:gamma].copy()
    bad[0] = (chain[0] + 1) % MINI.vocab
    r = verify(dec, base.copy(), prompt[-1], bad, None, u, GREEDY)
    assert r.n_accepted == 0 and r.correction == chain[0]
    for k in range(gamma):
        part = chain[:gamma].copy()
        part[k] = (chain[k] + 7) % MINI.vocab
        r = verify(dec, base.copy(), prompt[-1], part, None, u, GREEDY)
        assert r.n_accepted == k and r.correction == chain[k]


@pytest.mark.parametrize("mode", [GREEDY, SAMPLE])
def test_commit_then_round_two_equals_fresh_prefill(mode):
    mw = ModelWeights(MINI, 4)
    dec = Decoder(MINI, mw.get, keep_f64=True)
    rng = np.random.default_rng(12)
    V, gamma = MINI.vocab, 4
    prompt = rng.integers(0, V, 30)
    cache = dec.new_cache(64)
    dec.prefill(cache, prompt[:-1])
    drafts = rng.integers(0, V, gamma)
    q = rng.dirichlet([1.0] * V, gamma) if mode == SAMPLE else None
    u = rng.random(gamma + 1).astype(np.float32)
    r1 = verify(dec, cache, prompt[-1], drafts, q, u, mode)
    pending = commit(cache, r1)
    assert cache.length == len(prompt) - 1 + r1.n_accepted + 1
    # poison every row past the committed length
    for l in range(MINI.n_layers):
        cache.k[l][:, cache.length:] = np.nan
        cache.v[l][:, cache.length:] = np.nan
    drafts2 = rng.integers(0, V, gamma)
    u2 = rng.random(gamma + 1).astype(np.float32)
    q2 = rng.dirichlet([1.0] * V, gamma) if mode == SAMPLE else None
    r2 = verify(dec, cache, pending, drafts2, q2, u2, mode)
    committed = np.concatenate([prompt, drafts[:r1.n_accepted], [pending]])
    fresh = dec.new_cache(64)
    dec.prefill(fresh, committed[:-1])
    r2f = verify(dec, fresh, committed[-1], drafts2, q2, u2, mode)
    np.testing.assert_allclose(r2.logits, r2f.logits, rtol=0, atol=1e-11)
    assert (r2.n_accepted, r2.correction) == (r2f.n_accepted, r2f.correction)
