"""Helpers for GPU parity tests: upload a seeded workload, run the library through the C ABI, and
compare with the CPU oracle under the parity rules.

Parity rules (bf16 inputs, fp32 accumulation on the GPU, fp64 in the oracle):
  * floating-point results: max_i |x_i - y_i| / max(|y_i|, tau) <= 2e-3 with tau = 1e-3 * RMS(y)
    over the compared row (an output row, a mean-key / mean-value row) or tensor (grouped
    variances, scores);
  * selected ids: same count, ascending, mandatory blocks present, and identical outside the band
    of blocks whose oracle score is within 1e-5 (relative) of the oracle's (K-|F|)-th candidate
    score -- several selections are correct when scores tie up to rounding.
"""
from __future__ import annotations

import math

import numpy as np
import torch

import oracle
import paper_2609_26300_amd as P
from workloads import WORKLOADS, Workload, gen_layer

TOL = 2e-3
BAND = 1e-5


def dev_bf16(bits: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to("cuda")


def bits_of(t: torch.Tensor) -> np.ndarray:
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def rel_err(x, y, axis=None) -> float:
    """Max relative error with the RMS floor, rows along ``axis`` (None: whole tensor)."""
    x = np.asarray(x, np.float64)
    y = np.asarray(y, np.float64)
    if axis is None:
        rms = math.sqrt(float(np.mean(y * y))) if y.size else 0.0
        tau = 1e-3 * rms if rms > 0 else 1e-12
        return float(np.max(np.abs(x - y) / np.maximum(np.abs(y), tau))) if y.size else 0.0
    rms = np.sqrt(np.mean(y * y, axis=axis, keepdims=True))
    tau = np.where(rms > 0, 1e-3 * rms, 1e-12)
    return float(np.max(np.abs(x - y) / np.maximum(np.abs(y), tau))) if y.size else 0.0


def mandatory(X, n_sink=1, n_recent=2):
    return {b for b in range(X) if b < n_sink or b >= X - n_recent}


def check_selection(sel_gpu, score_oracle, K, n_sink=1, n_recent=2, band=BAND):
    """Selection parity under the tie band; returns the oracle's selection."""
    sel_gpu = [int(s) for s in sel_gpu]
    X = len(score_oracle)
    sel_or = oracle.select(score_oracle, K, n_sink, n_recent).tolist()
    assert len(sel_gpu) == len(sel_or) == min(K, X), (len(sel_gpu), len(sel_or))
    assert sel_gpu == sorted(set(sel_gpu)), "selection not ascending/unique"
    F = mandatory(X, n_sink, n_recent)
    assert F <= set(sel_gpu)
    if K >= X:
        assert sel_gpu == sel_or
        return sel_or
    cand = sorted((b for b in range(X) if b not in F), key=lambda b: (-score_oracle[b], b))
    kk = K - len(F)
    if kk == 0:
        assert sel_gpu == sel_or
        return sel_or
    s_k = score_oracle[cand[kk - 1]]
    A = {b for b in range(X) if abs(score_oracle[b] - s_k) <= band * abs(s_k)}
    assert set(sel_gpu) - A == set(sel_or) - A, (sorted(set(sel_gpu) ^ set(sel_or)), sorted(A))
    return sel_or


class Case:
    """One seeded workload resident on the GPU (layer 0) plus its library outputs."""

    def __init__(self, w: Workload, seq_lens=None, r=None, layout=0, budget=None, n_sink=1, n_recent=2,
                 capacity=None, max_seq_len=None):
        self.w = w
        self.K_bits, self.V_bits, self.q_bits = gen_layer(w, 0)
        self.seq_lens = np.array(seq_lens if seq_lens is not None else [w.context] * w.batch, np.int32)
        self.r = w.n_var_groups if r is None else r
        self.layout = layout
        self.budget = w.budget_blocks if budget is None else budget
        self.n_sink, self.n_recent = n_sink, n_recent
        self.scale = 1.0 / math.sqrt(w.head_dim)
        cap = w.capacity if capacity is None else capacity
        self.dims = P.make_dims(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.block_size, self.r, cap,
                                max_seq_len=int(max_seq_len or max(1, self.seq_lens.max())),
                                group_layout=layout)
        self.K = dev_bf16(self.K_bits[:, :, :cap])
        self.V = dev_bf16(self.V_bits[:, :, :cap])
        self.q = dev_bf16(self.q_bits)
        self.sl = torch.from_numpy(self.seq_lens).to("cuda")
        self.ws = P.alloc_workspace(self.dims, self.budget)
        self.G = w.group
        self._orc = {}  # oracle results per (kind, unit, length)
        self.select_path = P.COMPKV_SELECT_AUTO
        self.score_kind = P.COMPKV_SCORE_COMPKV
        self.compensation = P.COMPKV_COMP_MEAN

    def one_group_ok(self) -> bool:
        """Whether the one-workgroup-per-unit selection accepts these dims (G * blocks <= 8192)."""
        return self.G * self.dims.xmax <= 8192

    def params(self):
        return P.CompkvSelectParams(self.budget, self.n_sink, self.n_recent, self.scale, self.select_path,
                                    self.score_kind, self.compensation)

    # ---------------------------------------------------------------- library calls
    def build_stats(self):
        self.summ = P.alloc_summaries(self.dims)
        P.compkv_build_stats(self.dims, self.K, self.V, self.sl, self.summ.kmean, self.summ.dvar, self.summ.vmean)
        return self.summ

    def score_select(self, q=None):
        d = self.dims
        units = (d.batch, d.n_kv_heads)
        self.sel = torch.full((*units, self.budget), -7, dtype=torch.int32, device="cuda")
        self.n_sel = torch.zeros(units, dtype=torch.int32, device="cuda")
        self.blk_logit = torch.zeros((*units, self.G, d.xcap), dtype=torch.float32, device="cuda")
        self.scores = torch.zeros((*units, d.xcap), dtype=torch.float32, device="cuda")
        P.compkv_score_select(d, self.params(), self.q if q is None else q, self.summ.kmean, self.summ.dvar, self.sl,
                              self.sel, self.n_sel, self.blk_logit, self.scores, self.ws)

    def sparse_decode(self, sel=None, n_sel=None, from_kmean=False):
        """compkv_sparse_decode; the Drop decode when this case's compensation is COMPKV_COMP_DROP. With
        from_kmean the block logits are not passed: the library recomputes them from the mean keys."""
        d = self.dims
        self.out = torch.zeros((d.batch, d.n_q_heads, d.head_dim), dtype=torch.float32, device="cuda")
        self.lse = torch.zeros((d.batch, d.n_q_heads), dtype=torch.float32, device="cuda")
        drop = self.compensation == P.COMPKV_COMP_DROP
        P.compkv_sparse_decode(d, self.scale, self.q, self.K, self.V, None if drop else self.summ.vmean,
                               None if drop or from_kmean else self.blk_logit, self.sl,
                               self.sel if sel is None else sel, self.n_sel if n_sel is None else n_sel,
                               self.out, self.lse, self.ws, kmean=self.summ.kmean if from_kmean else None)
        return self.out, self.lse

    def decode_step(self, k_new=None, v_new=None, sl=None, summ=None, K=None, V=None, ws=None):
        """compkv_decode_step on this case's tensors (or the given ones); returns its outputs."""
        d = self.dims
        units = (d.batch, d.n_kv_heads)
        summ = self.summ if summ is None else summ
        r = dict(
            sel=torch.full((*units, self.budget), -7, dtype=torch.int32, device="cuda"),
            n_sel=torch.zeros(units, dtype=torch.int32, device="cuda"),
            blk_logit=torch.zeros((*units, self.G, d.xcap), dtype=torch.float32, device="cuda"),
            scores=torch.zeros((*units, d.xcap), dtype=torch.float32, device="cuda"),
            out=torch.zeros((d.batch, d.n_q_heads, d.head_dim), dtype=torch.float32, device="cuda"),
            lse=torch.zeros((d.batch, d.n_q_heads), dtype=torch.float32, device="cuda"))
        P.compkv_decode_step(d, self.params(), self.q, self.K if K is None else K, self.V if V is None else V, k_new, v_new,
                             self.sl if sl is None else sl, summ.kmean, summ.dvar, summ.vmean, r["sel"], r["n_sel"],
                             r["blk_logit"], r["scores"], r["out"], r["lse"], self.ws if ws is None else ws)
        return r

    def dense_decode(self):
        d = self.dims
        out = torch.zeros((d.batch, d.n_q_heads, d.head_dim), dtype=torch.float32, device="cuda")
        lse = torch.zeros((d.batch, d.n_q_heads), dtype=torch.float32, device="cuda")
        P.compkv_dense_decode(d, self.scale, self.q, self.K, self.V, self.sl, out, lse, self.ws)
        return out, lse

    def run_all(self):
        self.build_stats()
        self.score_select()
        self.sparse_decode()
        torch.cuda.synchronize()

    # ---------------------------------------------------------------- oracle side
    def unit_inputs(self, b, h):
        G = self.G
        return self.q_bits[b, h * G:(h + 1) * G], self.K_bits[b, h], self.V_bits[b, h], int(self.seq_lens[b])

    def oracle_stats(self, b, h):
        q, K, V, n = self.unit_inputs(b, h)
        key = ("stats", b, h, n)
        if key not in self._orc:
            self._orc[key] = oracle.block_stats(K, V, n, self.w.block_size, self.r, self.layout)
        return self._orc[key]

    def oracle_scores(self, b, h, stats=None):
        q, K, V, n = self.unit_inputs(b, h)
        if stats is not None:
            km, dv, vm = stats
            return oracle.block_scores(q, km, dv, n, self.w.block_size, self.r, self.scale, self.layout,
                                       kind=self.score_kind)
        key = ("scores", b, h, n, self.score_kind)
        if key not in self._orc:
            km, dv, vm = self.oracle_stats(b, h)
            self._orc[key] = oracle.block_scores(q, km, dv, n, self.w.block_size, self.r, self.scale,
                                                 self.layout, kind=self.score_kind)
        return self._orc[key]

    def prefetch_oracle(self, units=None, threads=8):
        """Oracle summaries and scores of the given units (all by default), computed on a thread pool (the C
        oracle releases the interpreter lock)."""
        from concurrent.futures import ThreadPoolExecutor

        with ThreadPoolExecutor(max_workers=threads) as ex:
            list(ex.map(lambda u: self.oracle_scores(*u), units or self.units()))

    def check_stats(self, kmean, dvar, vmean, units=None):
        """Summaries (device tensors) against the oracle's, unit by unit."""
        km_g, dv_g, vm_g = (x.cpu().numpy() for x in (kmean, dvar, vmean))
        for b, h in units or self.units():
            okm, odv, ovm = self.oracle_stats(b, h)
            X = okm.shape[0]
            assert rel_err(km_g[b, h, :X], okm, axis=1) <= TOL, ("kmean", b, h)
            assert rel_err(vm_g[b, h, :X], ovm, axis=1) <= TOL, ("vmean", b, h)
            assert rel_err(dv_g[b, h, :X], odv) <= TOL, ("dvar", b, h)

    def check_step(self, sel, n_sel, out, lse=None, units=None):
        """Selection (tie band) and compensated output / lse against the oracle recomputed on the GPU's
        selection, unit by unit."""
        sel, nsel, out = (x.cpu().numpy() for x in (sel, n_sel, out))
        lse = None if lse is None else lse.cpu().numpy()
        G = self.G
        compensate = self.compensation != P.COMPKV_COMP_DROP
        for b, h in units or self.units():
            q, K, V, n = self.unit_inputs(b, h)
            km, dv, vm = self.oracle_stats(b, h)
            sc = self.oracle_scores(b, h)
            s = sel[b, h, :nsel[b, h]]
            check_selection(s, sc["score"], self.budget, self.n_sink, self.n_recent)
            assert np.all(sel[b, h, nsel[b, h]:] == -1)
            o, l = oracle.sparse_decode(q, K, V, km, vm, n, self.w.block_size, self.scale, s, compensate)
            assert rel_err(out[b, h * G:(h + 1) * G], o, axis=1) <= TOL, ("out", b, h)
            if lse is not None:
                got = lse[b, h * G:(h + 1) * G]
                fin = np.isfinite(l)
                assert np.array_equal(fin, np.isfinite(got)), ("lse finiteness", b, h)
                if fin.any():
                    assert np.max(np.abs(got[fin] - l[fin])) <= TOL * max(1.0, float(np.max(np.abs(l[fin])))), \
                        ("lse", b, h)

    def check_dense(self, out, lse, units=None):
        out, lse = out.cpu().numpy(), lse.cpu().numpy()
        G = self.G
        for b, h in units or self.units():
            q, K, V, n = self.unit_inputs(b, h)
            o, l = oracle.dense_decode(q, K, V, n, self.scale)
            assert rel_err(out[b, h * G:(h + 1) * G], o, axis=1) <= TOL, ("dense out", b, h)
            assert np.max(np.abs(lse[b, h * G:(h + 1) * G] - l)) <= TOL * max(1.0, np.max(np.abs(l))), \
                ("dense lse", b, h)

    def units(self):
        return [(b, h) for b in range(self.w.batch) for h in range(self.w.n_kv_heads)]


# selection paths under test; a case the one-group path does not accept runs on the chunked path only
PATHS = {"chunked": P.COMPKV_SELECT_CHUNKED, "one_group": P.COMPKV_SELECT_ONE_GROUP,
         "chunked_exact": P.COMPKV_SELECT_CHUNKED_EXACT, "stream": P.COMPKV_SELECT_STREAM}


def make_case(name: str, path: str) -> Case:
    """Parity case ``name`` with its selection path set; skips an ineligible one-group variant."""
    import pytest

    c = CASES[name]()
    c.select_path = PATHS[path]
    if path == "one_group" and not c.one_group_ok():
        pytest.skip("the one-group selection needs G * blocks <= 8192")
    return c


TINY = WORKLOADS["tiny_4k"]
LLAMA = WORKLOADS["llama8b_32k"]

# Parity cases: the tiny 4K workload, the Llama-3-8B-shaped 32K layer at full size, and edge cases.
CASES = {
    "tiny_4k": lambda: Case(TINY),
    "llama8b_32k": lambda: Case(LLAMA),
    "partial_tail": lambda: Case(TINY.with_(context=4001, seed=7)),
    "block1": lambda: Case(TINY.with_(context=300, block_size=1, budget_blocks=40, seed=8)),
    "r_eq_d": lambda: Case(TINY.with_(n_var_groups=128, seed=9)),
    "interleaved_r8": lambda: Case(TINY.with_(n_var_groups=8, seed=10), layout=1),
    # variance groups of every width: one group of all 64 pairs, and 64 groups of one pair
    "r1": lambda: Case(TINY.with_(n_var_groups=1, seed=28)),
    "interleaved_r64": lambda: Case(TINY.with_(n_var_groups=64, seed=29), layout=1),
    "d64": lambda: Case(TINY.with_(head_dim=64, seed=11)),
    "d64_b64": lambda: Case(TINY.with_(head_dim=64, block_size=64, context=4000, budget_blocks=8, seed=30)),
    "g1": lambda: Case(TINY.with_(n_q_heads=2, seed=12)),
    "g2_b32": lambda: Case(TINY.with_(n_q_heads=4, block_size=32, budget_blocks=9, seed=13)),
    "g8_b64": lambda: Case(TINY.with_(n_q_heads=16, block_size=64, context=8000, budget_blocks=12, seed=14)),
    "varlen": lambda: Case(TINY.with_(batch=4, seed=15), seq_lens=[4096, 1000, 17, 49]),
    "short": lambda: Case(TINY.with_(batch=4, seed=16), seq_lens=[1, 10, 16, 40], budget=3),
    "budget_ge_x": lambda: Case(TINY.with_(context=1000, budget_blocks=80, seed=17)),
    "wide_gqa_8k": lambda: Case(WORKLOADS["wide_gqa_64k"].with_(batch=2, context=8192, seed=18)),
    "long_16k_lognormal": lambda: Case(WORKLOADS["long_128k"].with_(batch=1, context=16384, budget_blocks=32,
                                                                    seed=19)),
    # more mean-value rows than selected tokens per unit (the fused launch's form with compensation
    # workgroups); the cases above with a budget of at least X / B blocks take its one-selector form
    "long_16k_b8": lambda: Case(WORKLOADS["long_128k"].with_(batch=2, context=16384, budget_blocks=8, seed=31)),
    # selection paths: > 8192 blocks (keys outside registers), ~1000 candidates ranked by brute force,
    # and ~2000 candidates (radix select fallback)
    "block1_9000": lambda: Case(TINY.with_(context=9000, block_size=1, budget_blocks=40, seed=25)),
    "budget300_x1000": lambda: Case(TINY.with_(context=16000, budget_blocks=300, seed=26)),
    "budget300_x2000": lambda: Case(TINY.with_(context=32000, budget_blocks=300, seed=27)),
    # high logit spread: 8 of 32 query heads scaled by 16 and offset blocks 8 nats up along the unit's mean
    # query, so that in most units the selected blocks hold most of the attention mass; and a 4K layer with
    # 4 query heads scaled by 128, whose units' log weights span up to 98 nats (seeds chosen so the cut
    # is at least 2.5e-4 relative away from the next candidate: the case tests the arithmetic at large
    # spreads, not ties)
    "high_spread_8k": lambda: Case(LLAMA.with_(context=8192, offset_frac=0.05, offset_logit=8.0, peaky_frac=0.25,
                                               peaky_scale=16.0, seed=69)),
    "span_98nats": lambda: Case(LLAMA.with_(context=4096, offset_frac=0.05, offset_logit=8.0, peaky_frac=0.125,
                                            peaky_scale=128.0, budget_blocks=20, seed=55)),
    # mandatory sets other than (1, 2): none, (2, 1) and (3, 3), on long contexts and on contexts of a few
    # blocks where the sink and recent ranges overlap or cover every block
    "sink0_recent0": lambda: Case(TINY.with_(context=2000, seed=50), n_sink=0, n_recent=0),
    "sink2_recent1": lambda: Case(TINY.with_(context=3000, seed=51), n_sink=2, n_recent=1),
    "sink3_recent3": lambda: Case(TINY.with_(context=4000, seed=52), n_sink=3, n_recent=3),
    "sink3_recent3_short": lambda: Case(TINY.with_(batch=4, seed=53), seq_lens=[16, 48, 80, 100], budget=6,
                                        n_sink=3, n_recent=3),
    "sink2_recent1_short": lambda: Case(TINY.with_(batch=4, seed=54), seq_lens=[1, 20, 33, 64], budget=3,
                                        n_sink=2, n_recent=1),
    "sink0_recent0_short": lambda: Case(TINY.with_(batch=3, seed=56), seq_lens=[5, 40, 70], budget=2,
                                        n_sink=0, n_recent=0),
}
