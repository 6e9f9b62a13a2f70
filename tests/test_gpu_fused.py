"""The single-launch verify pass against the oracle and against the
one-kernel-per-stage path, through the C ABI.

Eligible workloads (bf16 weights and cache, head_dim 128, multi-head
attention, B * (gamma+1) <= 16) run both paths on the same model, cache and inputs:
* each path meets the parity bar of test_gpu_parity.py against the oracle;
* the two paths agree bit for bit (logits, n_accepted, correction): they run
  the same GEMM engine, attention arithmetic and accept code;
* several calls in a row (the persistent kernel resets its barrier words and
  arrival counters on the way out) give identical results.
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


def _eligible(w):
    m = w.model
    return m.weight_dtype == "bf16" and m.kv_dtype == "bf16" and m.head_dim == 128 and \
        m.kv_heads == m.n_heads and w.batch * (w.gamma + 1) <= 16


FUSED_CASES = [w for w in mini_workloads() if _eligible(w)]


def _check_parity(w, orun, lg, n, c):
    p = compare(orun, lg, n, c)
    assert not p.stable_n_fail, p
    assert not p.stable_corr_fail, p
    if w.mode == "greedy":
        assert not p.pinned_n_fail and not p.pinned_corr_fail, p
    assert p.logit_err < LOGIT_TOL[w.model.weight_dtype], p.logit_err
    return p


@pytest.mark.parametrize("w", FUSED_CASES, ids=lambda w: w.name)
def test_fused_matches_oracle_and_stage_path(w):
    assert FUSED_CASES, "no eligible mini workload"
    weights = ModelWeights(w.model, w.seed)
    model, kv = gpu_setup(w, weights)
    for k in range(2):
        wk = w.with_(seed=w.seed * 1000 + 17 + k)
        inp = make_inputs(wk)
        orun = oracle_run(wk, inp, weights=weights)
        kv.set_state(np.zeros(w.batch, np.int32), np.zeros(w.batch, np.int32))
        gpu_prefill(kv, inp)
        results = {}
        for fused in (True, False, True):
            print(f"[{w.name}] round {k}: verify fused={fused}", flush=True)
            model.set_fused(fused)
            lg, n, c, _ = gpu_verify(model, kv, inp)
            p = _check_parity(w, orun, lg, n, c)
            assert model.device_error() == 0
            if fused in results:
                plg, pn, pc = results[fused]
                assert np.array_equal(plg, lg) and np.array_equal(pn, n) and np.array_equal(pc, c)
            results[fused] = (lg, n, c)
        (flg, fn, fc), (slg, sn, sc) = results[True], results[False]
        print(f"[{w.name}] round {k}: logit err {p.logit_err:.2e}, max |fused - staged| "
              f"{np.abs(flg - slg).max():.2e}", flush=True)
        assert np.array_equal(fn, sn) and np.array_equal(fc, sc)
        assert np.array_equal(flg, slg)
    model.set_fused(True)
