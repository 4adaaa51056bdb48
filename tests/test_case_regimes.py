"""The GPU parity cases meant to stress large logit spreads reach that regime (oracle, CPU only).

* high_spread_8k: for most query heads the blocks the mass score selects hold more than 90% of the
  head's estimated attention mass (the selected blocks dominate, so the fused step's compensation is
  mostly taken back out by its exact items);
* span_98nats: some unit's per-head log weights log|b| + zbar + sig2/2 span more than 80 nats.
Both keep the selection cut clear of ties (the next candidate at least 1e-4 relative below the cut),
so their GPU parity tests exercise the arithmetic, not the tie band.
"""
import math

import numpy as np
import pytest

import oracle
from workloads import WORKLOADS, gen_layer

LLAMA = WORKLOADS["llama8b_32k"]
HIGH = LLAMA.with_(context=8192, offset_frac=0.05, offset_logit=8.0, peaky_frac=0.25, peaky_scale=16.0, seed=69)
SPAN = LLAMA.with_(context=4096, offset_frac=0.05, offset_logit=8.0, peaky_frac=0.125, peaky_scale=128.0,
                   budget_blocks=20, seed=55)


def _units(w, kind):
    K, V, q = gen_layer(w, 0)
    s = 1.0 / math.sqrt(w.head_dim)
    G = w.group
    for h in range(w.n_kv_heads):
        km, dv, vm = oracle.block_stats(K[0, h], V[0, h], w.context, w.block_size, w.n_var_groups)
        sc = oracle.block_scores(q[0, h * G:(h + 1) * G], km, dv, w.context, w.block_size, w.n_var_groups, s,
                                 kind=kind)
        X = km.shape[0]
        logw = np.log(np.minimum(w.block_size, w.context - np.arange(X) * w.block_size)) + sc["zbar"] + \
            0.5 * sc["sig2"]
        yield sc, logw


def _cut_gap(score, K):
    X = len(score)
    cand = sorted(range(1, X - 2), key=lambda b: (-score[b], b))
    kk = K - 3
    return (score[cand[kk - 1]] - score[cand[kk]]) / score[cand[kk - 1]]


@pytest.mark.parametrize("kind", [oracle.SCORE_COMPKV, oracle.SCORE_MASS])
def test_high_spread_selected_blocks_hold_the_mass(kind):
    dominated = 0
    for sc, _ in _units(HIGH, kind):
        sel = oracle.select(sc["score"], HIGH.budget_blocks)
        dominated += int((sc["phat"][:, sel].sum(axis=1) > 0.9).sum())
        assert _cut_gap(sc["score"], HIGH.budget_blocks) > 1e-4
    if kind == oracle.SCORE_MASS:
        assert dominated > HIGH.n_q_heads // 2


@pytest.mark.parametrize("kind", [oracle.SCORE_COMPKV, oracle.SCORE_MASS])
def test_span_case_exceeds_80_nats(kind):
    spans = []
    for sc, logw in _units(SPAN, kind):
        spans.append(float((logw.max(axis=1) - logw.min(axis=1)).max()))
        assert _cut_gap(sc["score"], SPAN.budget_blocks) > 1e-4
    assert max(spans) > 80.0
