"""Score fidelity on synthetic states, oracle only (Appendix B; the GPU counterpart is
test_gpu_fidelity.py). Reduced contexts keep the CPU suite fast.

* App. B.2: the CompKV score ranks blocks by the exact residual T_b far better than the estimated mass
  (Spearman, residual capture at a 512-token budget of 16-token blocks), here where the logits are
  flat and within-block variation decides the residual;
* App. B.1: selecting by the exact residual instead of the exact mass, both with Mean compensation,
  lowers the attention KL of every head on these units.
"""
import numpy as np
import pytest

import oracle
from fidelity_case import FidelityUnit
from oracle import diagnostics as dg
from workloads import WORKLOADS


@pytest.mark.parametrize("wl", ["fidelity_16k", "fidelity_lognormal_16k"])
def test_compkv_score_tracks_exact_residual(wl):
    w = WORKLOADS[wl].with_(context=4096)
    sp = {"mass": [], "compkv": []}
    cap = {"mass": [], "compkv": []}
    for h in range(2):
        u = FidelityUnit(w, h)
        km, dv, vm = oracle.block_stats(u.K, u.V, u.n, u.B, 4)
        for name, kind in (("mass", oracle.SCORE_MASS), ("compkv", oracle.SCORE_COMPKV)):
            s, c = u.judge(oracle.block_scores(u.q, km, dv, u.n, u.B, 4, u.scale, kind=kind)["score"])
            sp[name].append(s)
            cap[name].append(c)
    assert np.mean(sp["compkv"]) > 0.9 and np.mean(cap["compkv"]) > 0.8
    assert np.mean(sp["compkv"]) > np.mean(sp["mass"]) + 0.5
    assert np.mean(cap["compkv"]) > np.mean(cap["mass"])


def test_exact_residual_selection_lowers_kl_against_exact_mass():
    """App. B.1 on synthetic units: the same Mean compensator, the same budget; residual-ranked
    selection gives a lower KL(P-hat || P) = lse_dense - lse_compensated for every head."""
    w = WORKLOADS["fidelity_lognormal_16k"].with_(context=4096)
    for h in range(2):
        u = FidelityUnit(w, h)
        km, dv, vm = oracle.block_stats(u.K, u.V, u.n, u.B, 4)
        od, ld = oracle.dense_decode(u.q, u.K, u.V, u.n, u.scale)
        kl = {}
        for name, score in (("mass", u.bx["p"].sum(axis=0)), ("residual", u.T)):
            sel = np.sort(np.concatenate([u.F, dg.top_blocks(score, u.kk, exclude=u.F)])).astype(np.int32)
            o, l = oracle.sparse_decode(u.q, u.K, u.V, km, vm, u.n, u.B, u.scale, sel)
            kl[name] = ld - l
            assert np.all(kl[name] >= -1e-12)
        assert np.all(kl["residual"] < kl["mass"])
