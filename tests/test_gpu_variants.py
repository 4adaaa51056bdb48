"""GPU parity of the ablation variants (Section 5.4, Appendix A.5) against the oracle (needs an MI355X).

* score kinds: the mass-only score and the first-order mass estimate, on both selection paths, through
  compkv_score_select and the fused step: scores within the parity tolerance, selections identical
  outside the tie band, outputs matching the oracle on the selected set;
* the Drop decode (no compensation) through compkv_sparse_decode (vmean = blk_logit = NULL) and the
  fused step (compensation = COMPKV_COMP_DROP), with and without an append;
* on the Llama-shaped 32K layer the mass-only score selects every high-mass, low-variance offset block
  and the CompKV score none, as the oracle does.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_26300_amd as P
from gpu_case import CASES, PATHS, TOL, check_selection, make_case, rel_err
from workloads import offset_blocks

pytestmark = pytest.mark.gpu

KINDS = {"mass": P.COMPKV_SCORE_MASS, "first_order": P.COMPKV_SCORE_FIRST_ORDER}
VARIANT_CASES = ["tiny_4k", "llama8b_32k", "partial_tail", "g8_b64", "short", "budget_ge_x", "interleaved_r8",
                 "high_spread_8k", "span_98nats", "sink0_recent0", "sink2_recent1_short"]


def _gpu(t):
    return t.cpu().numpy()


def _oracle_output_check(c, sel, nsel, out, lse, compensate):
    G = c.G
    for b, h in c.units():
        q, K, V, n = c.unit_inputs(b, h)
        st = c.oracle_stats(b, h)
        s = sel[b, h, :nsel[b, h]]
        o, l = oracle.sparse_decode(q, K, V, st[0], st[2], n, c.w.block_size, c.scale, s, compensate=compensate)
        if n == 0:
            continue
        assert rel_err(out[b, h * G:(h + 1) * G], o, axis=1) <= TOL
        assert np.max(np.abs(lse[b, h * G:(h + 1) * G] - l)) <= TOL * max(1.0, np.max(np.abs(l)))


@pytest.mark.parametrize("path", sorted(PATHS))
@pytest.mark.parametrize("kind", sorted(KINDS))
@pytest.mark.parametrize("name", VARIANT_CASES)
def test_score_kind_parity(name, kind, path):
    c = make_case(name, path)
    c.score_kind = KINDS[kind]
    print(f"\n[variant {name} / {kind} / {path}]", flush=True)
    c.run_all()
    step = c.decode_step()
    torch.cuda.synchronize()
    sel, nsel, scores = _gpu(c.sel), _gpu(c.n_sel), _gpu(c.scores)
    for b, h in c.units():
        sc = c.oracle_scores(b, h)
        X = sc["score"].shape[0]
        assert rel_err(scores[b, h, :X], sc["score"]) <= TOL
        check_selection(sel[b, h, :nsel[b, h]], sc["score"], c.budget, c.n_sink, c.n_recent)
    # the fused step selects exactly what the separate calls select, for the same score kind
    for key, ref in (("sel", c.sel), ("n_sel", c.n_sel), ("scores", c.scores), ("blk_logit", c.blk_logit)):
        assert torch.equal(step[key], ref), key
    _oracle_output_check(c, sel, nsel, _gpu(c.out), _gpu(c.lse), True)
    _oracle_output_check(c, sel, nsel, _gpu(step["out"]), _gpu(step["lse"]), True)


@pytest.mark.parametrize("path", sorted(PATHS))
@pytest.mark.parametrize("name", ["tiny_4k", "llama8b_32k", "partial_tail", "short", "block1", "g8_b64"])
def test_drop_decode_parity(name, path):
    """Drop: attention over the selected tokens alone, renormalized (Appendix A.5)."""
    c = make_case(name, path)
    c.compensation = P.COMPKV_COMP_DROP
    print(f"\n[drop {name} / {path}]", flush=True)
    c.run_all()  # separate calls: score_select, then sparse_decode without vmean / blk_logit
    step = c.decode_step()
    torch.cuda.synchronize()
    sel, nsel = _gpu(c.sel), _gpu(c.n_sel)
    _oracle_output_check(c, sel, nsel, _gpu(c.out), _gpu(c.lse), False)
    assert torch.equal(step["sel"], c.sel)
    _oracle_output_check(c, sel, nsel, _gpu(step["out"]), _gpu(step["lse"]), False)
    assert rel_err(_gpu(step["out"]), _gpu(c.out), axis=-1) <= TOL


@pytest.mark.parametrize("path", sorted(PATHS))
def test_drop_decode_with_append(path):
    """The fused step with an append and the Drop decode: the appended row and the refreshed summary
    are used, and the output matches the oracle's Drop output on the full context."""
    from test_gpu_step import _prefix_state

    c = make_case("llama8b_32k", path)
    c.compensation = P.COMPKV_COMP_DROP
    c.run_all()
    K2, V2, kn, vn, summ2 = _prefix_state(c)
    r = c.decode_step(kn, vn, summ=summ2, K=K2, V=V2)
    torch.cuda.synchronize()
    assert torch.equal(K2, c.K) and torch.equal(summ2.kmean, c.summ.kmean)
    assert torch.equal(r["sel"], c.sel)
    _oracle_output_check(c, _gpu(r["sel"]), _gpu(r["n_sel"]), _gpu(r["out"]), _gpu(r["lse"]), False)


@pytest.mark.parametrize("path", sorted(PATHS))
def test_offset_blocks_mass_vs_compkv_on_gpu(path):
    """Llama-shaped 32K layer: the mass-only score picks every offset block of every unit, the CompKV
    score none (the oracle's counts, Sections 3.2 and 4.1)."""
    counts = {}
    for kind in (P.COMPKV_SCORE_COMPKV, P.COMPKV_SCORE_MASS):
        c = make_case("llama8b_32k", path)
        c.score_kind = kind
        c.run_all()
        sel, nsel = _gpu(c.sel), _gpu(c.n_sel)
        counts[kind] = [len(set(offset_blocks(c.w, 0, b, h).tolist()) & set(sel[b, h, :nsel[b, h]].tolist()))
                        for b, h in c.units()]
        offs = [len(offset_blocks(c.w, 0, b, h)) for b, h in c.units()]
    assert counts[P.COMPKV_SCORE_MASS] == offs
    assert counts[P.COMPKV_SCORE_COMPKV] == [0] * len(offs)
