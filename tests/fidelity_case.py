"""Score fidelity against the exact residual (Appendix B), shared by the CPU and GPU fidelity tests.

For one (layer 0, batch 0) unit of a workload: the exact per-block residual T_b = sum_g rho_{g,b} from
all keys (oracle diagnostics), the non-mandatory blocks, and the exact-residual selection S_rho of
K - |F| blocks; a score vector is then judged by its Spearman correlation with T over the
non-mandatory blocks and by the residual capture of its own top K - |F| blocks.
"""
from __future__ import annotations

import math

import numpy as np

from oracle import diagnostics as dg
from workloads import gen_queries, gen_unit_kv


class FidelityUnit:
    def __init__(self, w, h: int):
        self.w, self.h = w, h
        self.n, self.B, self.G = w.context, w.block_size, w.group
        self.scale = 1.0 / math.sqrt(w.head_dim)
        self.K, self.V = gen_unit_kv(w, 0, 0, h)
        self.q = gen_queries(w, 0, 0, 0)[h * self.G:(h + 1) * self.G]
        self.z = dg.exact_logits(self.q, self.K, self.n, self.scale)
        self.bx = dg.block_exact(self.z, self.n, self.B)
        self.T = self.bx["rho"].sum(axis=0)
        X = len(self.T)
        self.F = [0, X - 2, X - 1]
        self.free = np.setdiff1d(np.arange(X), self.F)
        self.kk = w.budget_blocks - len(self.F)
        self.S_rho = dg.top_blocks(self.T, self.kk, exclude=self.F)

    def judge(self, score):
        """(Spearman with T over the non-mandatory blocks, residual capture of the score's selection)."""
        score = np.asarray(score, np.float64)[:len(self.T)]
        sel = dg.top_blocks(score, self.kk, exclude=self.F)
        return dg.spearman(score[self.free], self.T[self.free]), dg.capture(self.T, sel, self.S_rho)
