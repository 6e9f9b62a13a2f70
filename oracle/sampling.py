"""Oracle samplers for the correction / bonus token -- test infrastructure only.

The paper replaces the first rejected draft by a draw from
p'(x) = norm(max(0, p(x) - q(x))) (Sec. III-C, Algorithm 1) and gives no
sampling method.  Two exact samplers are stated here:

* ``gumbel_argmax``: argmax_v (log w_v + G_v) with G_v independent standard
  Gumbel variables is distributed as w / sum(w).  This is the sampler the
  verify path uses.  Its noise is counter-based, so a single uniform per
  request keys the whole vocabulary-sized stream:
      seed  = the IEEE-754 bit pattern of that uniform (float32 -> uint32),
      x_v   = output number v of SplitMix64 started from ``seed``
              (Steele, Lea and Flood, OOPSLA 2014: the state advances by
              0x9E3779B97F4A7C15 and each output is the state passed through
              the variant-13 mixer 30/0xBF58476D1CE4E5B9/27/0x94D049BB133111EB/31),
      U_v   = ((x_v >> 41) + 0.5) * 2^-23   (exact in float32 and float64),
      G_v   = -log(-log(U_v)).
* ``inverse_cdf_draw``: the smallest v whose cumulative mass exceeds u * sum(w),
  in ascending token order -- the literal reading, used only as a second,
  independent sampler in the distribution tests.
"""

from __future__ import annotations

import numpy as np

_GOLDEN = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)


def splitmix64_stream(seed: int, n: int, start: int = 0) -> np.ndarray:
    """Outputs start .. start+n-1 of SplitMix64 seeded with ``seed`` (uint64)."""
    with np.errstate(over="ignore"):
        idx = np.arange(start + 1, start + n + 1, dtype=np.uint64)
        z = np.uint64(seed) + idx * _GOLDEN
        z = (z ^ (z >> np.uint64(30))) * _M1
        z = (z ^ (z >> np.uint64(27))) * _M2
        return z ^ (z >> np.uint64(31))


def uniform_seed(u: float) -> int:
    """Bit pattern of a float32 uniform, used as the stream seed."""
    return int(np.asarray(u, dtype=np.float32).view(np.uint32))


def gumbel_noise(seed: int, n: int) -> np.ndarray:
    """G_v, v < n, in float64."""
    x = splitmix64_stream(seed, n)
    U = ((x >> np.uint64(41)).astype(np.float64) + 0.5) * 2.0 ** -23
    return -np.log(-np.log(U))


def gumbel_top2(log_w: np.ndarray, seed: int):
    """Perturbed scores log_w[v] + G_v: the best token, the runner-up and the
    gap between their scores.  Ties go to the lowest id."""
    s = np.asarray(log_w, dtype=np.float64) + gumbel_noise(seed, len(log_w))
    v = int(np.argmax(s))
    rest = s.copy()
    rest[v] = -np.inf
    v2 = int(np.argmax(rest)) if rest.size > 1 else v
    second = float(rest[v2]) if rest.size > 1 else -np.inf
    return v, v2, float(s[v] - second)


def gumbel_argmax(log_w: np.ndarray, seed: int):
    """Draw v with probability proportional to exp(log_w[v]).

    Entries with log_w = -inf (zero weight) can never be drawn.  Returns the
    token and the gap between the best and second-best perturbed scores (the
    margin by which the draw is decided).
    """
    v, _, gap = gumbel_top2(log_w, seed)
    return v, gap


def inverse_cdf_draw(w: np.ndarray, u: float) -> int:
    """Smallest v with cumsum(w)[v] > u * sum(w)."""
    c = np.cumsum(np.asarray(w, dtype=np.float64))
    v = int(np.searchsorted(c, u * c[-1], side="right"))
    return min(v, len(c) - 1)
