"""Score fidelity of the GPU scores on synthetic states (Appendix B.2 setting; needs an MI355X).

For every unit of the two fidelity workloads (32 query / 8 KV heads, 16K tokens, 16-token blocks,
512-token budget), the GPU scores of estimated-mass selection (r = 4), CompKV (r = 4) and CompKV
(r = 128) are judged against the exact residual T_b (oracle diagnostics): Spearman over the
non-mandatory blocks and residual capture of each score's own selection. Each metric must match the
one computed from the oracle's scores within 0.01, and the GPU selection must be the score's top
K - |F| blocks (tie band aside). The means are printed (run with -s to see them).
"""
import numpy as np
import pytest

import oracle
import paper_2609_26300_amd as P
from fidelity_case import FidelityUnit
from gpu_case import Case, check_selection
from workloads import WORKLOADS

pytestmark = pytest.mark.gpu

METHODS = (("estimated mass, r = 4", 4, P.COMPKV_SCORE_MASS), ("CompKV, r = 4", 4, P.COMPKV_SCORE_COMPKV),
           ("CompKV, r = 128", 128, P.COMPKV_SCORE_COMPKV))


@pytest.mark.parametrize("wl", ["fidelity_16k", "fidelity_lognormal_16k"])
def test_gpu_score_fidelity(wl):
    w = WORKLOADS[wl]
    units = [FidelityUnit(w, h) for h in range(w.n_kv_heads)]
    lines = []
    for name, r, kind in METHODS:
        c = Case(w, r=r)
        c.score_kind = kind
        c.build_stats()
        c.score_select()
        scores, sel, nsel = (x.cpu().numpy() for x in (c.scores, c.sel, c.n_sel))
        got, ref = [], []
        for h, u in enumerate(units):
            km, dv, vm = oracle.block_stats(u.K, u.V, u.n, u.B, r)
            osc = oracle.block_scores(u.q, km, dv, u.n, u.B, r, u.scale, kind=kind)["score"]
            check_selection(sel[0, h, :nsel[0, h]], osc, c.budget)
            got.append(u.judge(scores[0, h]))
            ref.append(u.judge(osc))
        got, ref = np.array(got), np.array(ref)
        assert np.all(np.abs(got - ref) <= 0.01), (name, got, ref)
        lines.append(f"{wl} {name}: Spearman {got[:, 0].mean():.4f}, capture {got[:, 1].mean():.4f}")
    print("\n" + "\n".join(lines), flush=True)
