"""CPU oracle for the speculative-verify path -- TEST INFRASTRUCTURE ONLY.

A plain, slow, float64 NumPy statement of what the verifier computes, written
from the SPADE paper (arXiv 2608.13076):

* ``decoder``      the verifier forward pass: embedding, L residual blocks
                   x_{l+1} = x_l + f_l(x_l), LM head, softmax (Sec. III-A);
* ``speculative``  verification of d draft tokens in one pass, the acceptance
                   rule alpha(x) = min(1, p(x)/q(x)), the residual
                   p'(x) = norm(max(0, p(x) - q(x))), the bonus token and the
                   context update (Sec. III-B, Sec. III-C, Algorithm 1);
* ``sampling``     the exact samplers used for the correction draw and the
                   SplitMix64 stream that feeds the Gumbel-max sampler.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The HIP library shares no code with it
and never calls it.
"""

from .decoder import Decoder, KVCache, bf16_round, rope_tables  # noqa: F401
from .speculative import (  # noqa: F401
    GREEDY,
    SAMPLE,
    RowDecision,
    VerifyResult,
    accept_test,
    residual_distribution,
    speculative_rows,
    verify,
    commit,
)
from .sampling import splitmix64_stream, gumbel_noise, gumbel_argmax, inverse_cdf_draw  # noqa: F401
