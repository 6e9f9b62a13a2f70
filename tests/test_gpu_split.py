"""Small-batch projections split along K (device_gemm_split.h).

Forcing 2 or 4 k-splits on every bf16 projection of the scaled-down shapes
(the automatic choice only splits where the whole operand does not fit in
LDS, as at the 7B down projection and the 13B shape) must give bit-for-bit
the logits, n_accepted and corrections of the unsplit engine, and match the
oracle to the usual bar.  Rows: 6 (B=1, gamma 5), 9 (gamma 8), 14 (B=2,
gamma 6) and 16 (B=4, gamma 3); k-blocks per projection from 2 to 11, so
some k-ranges are empty and some k-splits have an odd number of k-blocks.
"""

import numpy as np
import pytest

from synth import ModelWeights, make_inputs, mini_workloads
from tests.helpers import LOGIT_TOL, compare, gpu_prefill, gpu_setup, gpu_verify, oracle_run

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _split_workloads():
    ws = {w.name: w for w in mini_workloads()}
    out = [ws["mini_bf16_greedy"], ws["mini_bf16_sample"], ws["mini_bf16_mixed"]]
    out.append(ws["mini_bf16_wide_b5"].with_(name="mini_bf16_wide_b2", batch=2, gamma=6, seed=2017))
    return out


@pytest.mark.parametrize("w", _split_workloads(), ids=lambda w: w.name)
def test_split_k_bit_identical_and_matches_oracle(w):
    weights = ModelWeights(w.model, w.seed)
    inp = make_inputs(w)
    orun = oracle_run(w, inp, weights=weights)  # also completes the chain drafts
    model, kv = gpu_setup(w, weights)
    gpu_prefill(kv, inp)
    runs = {}
    for ks in (-1, 2, 4, 0):
        print(f"[{w.name}] M={w.batch * (w.gamma + 1)} k-splits {ks}", flush=True)
        model.set_split_k(ks)
        runs[ks] = gpu_verify(model, kv, inp)[:3]
    ref = runs[-1]
    for ks, (lg, n, c) in runs.items():
        assert np.array_equal(lg.view(np.uint32), ref[0].view(np.uint32)), ks
        assert np.array_equal(n, ref[1]) and np.array_equal(c, ref[2]), ks
    p = compare(orun, *runs[2])
    print(f"[{w.name}] logit err {p.logit_err:.2e}, n {runs[2][1].tolist()}", flush=True)
    assert p.logit_err < LOGIT_TOL[w.model.weight_dtype]
    assert not p.stable_n_fail and not p.stable_corr_fail, p
    assert model.device_error() == 0
