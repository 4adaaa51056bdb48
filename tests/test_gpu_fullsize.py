"""Full-size parity of the fused decode step (needs an MI355X).

The long-context 128K layer (batch 4; budgets 32, 64 and 128 blocks), the wide-GQA 64K layer (batch 8,
G = 8) and the streaming layer's first appending step (131072 + 1 tokens, so the last block holds one
token), each run exactly as bench.py times them: summaries built over n tokens, then one
compkv_decode_step on the automatic launch shape that appends row n - 1 (rewriting it with the same
values, which also refreshes the active block's summary). The oracle is too slow for every unit at these
sizes, so three units per workload (first, middle, last) are checked one by one: their summaries, the
selection (bit-exact outside the tie band), the compensated output and lse.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_26300_amd as P
from gpu_case import TOL, Case, check_selection, rel_err
from workloads import WORKLOADS

pytestmark = pytest.mark.gpu

# (workload, tokens in the cache after the step, budgets)
FULL = {
    "long_128k": (WORKLOADS["long_128k"], None, (32, 64, 128)),
    "wide_gqa_64k": (WORKLOADS["wide_gqa_64k"], None, (None,)),
    "streaming_128k": (WORKLOADS["streaming_128k"], WORKLOADS["streaming_128k"].context + 1, (None,)),
}
PATH_NAMES = {P.COMPKV_SELECT_CHUNKED: "chunked", P.COMPKV_SELECT_ONE_GROUP: "one group",
              P.COMPKV_SELECT_CHUNKED_EXACT: "chunked + fused selection/exact"}

_cases = {}


def _case(name):
    if name not in _cases:
        _cases.clear()  # one full-size workload resident at a time
        torch.cuda.empty_cache()
        w, n, _ = FULL[name]
        print(f"\n[full-size {name}] generating and building summaries", flush=True)
        c = Case(w, seq_lens=None if n is None else [n] * w.batch)
        c.build_stats()
        torch.cuda.synchronize()
        _cases[name] = c
    return _cases[name]


def _sample_units(c):
    units = c.units()
    return [units[0], units[len(units) // 2], units[-1]]


@pytest.mark.parametrize("name,budget", [(n, k) for n, (_, _, ks) in FULL.items() for k in ks],
                         ids=lambda x: str(x))
def test_fullsize_fused_step(name, budget):
    c = _case(name)
    c.budget = budget or c.w.budget_blocks
    c.select_path = P.COMPKV_SELECT_AUTO
    d = c.dims
    path = P.compkv_decode_step_path(d, c.params())
    print(f"[full-size {name} K={c.budget}] launch shape: {PATH_NAMES.get(path, path)}", flush=True)
    n = int(c.seq_lens[0])
    k_new = c.K[:, :, n - 1].contiguous()
    v_new = c.V[:, :, n - 1].contiguous()
    ws = P.alloc_workspace(d, c.budget)
    r = c.decode_step(k_new, v_new, ws=ws)
    torch.cuda.synchronize()
    sel, nsel = r["sel"].cpu().numpy(), r["n_sel"].cpu().numpy()
    out, lse = r["out"].cpu().numpy(), r["lse"].cpu().numpy()
    G = c.G
    for b, h in _sample_units(c):
        q, K, V, nn = c.unit_inputs(b, h)
        km, dv, vm = c.oracle_stats(b, h)
        X = km.shape[0]
        for got, ref, what in ((c.summ.kmean, km, "kmean"), (c.summ.dvar, dv, "dvar"), (c.summ.vmean, vm, "vmean")):
            g = got[b, h, :X].cpu().numpy()
            err = rel_err(g, ref, axis=None if what == "dvar" else 1)
            assert err <= TOL, (name, b, h, what, err)
        sc = c.oracle_scores(b, h, (km, dv, vm))
        s = sel[b, h, :nsel[b, h]]
        check_selection(s, sc["score"], c.budget, c.n_sink, c.n_recent)
        o, l = oracle.sparse_decode(q, K, V, km, vm, nn, c.w.block_size, c.scale, s)
        assert rel_err(out[b, h * G:(h + 1) * G], o, axis=1) <= TOL, (name, b, h)
        assert np.max(np.abs(lse[b, h * G:(h + 1) * G] - l)) <= TOL * max(1.0, float(np.max(np.abs(l)))), (name, b, h)


@pytest.mark.parametrize("name", ["long_128k", "wide_gqa_64k"])
def test_fullsize_graph_replays_match_eager(name):
    """At full size the chunk grid exceeds one resident round (the last-block workgroups then trail the
    grid) and the exact items are sized to one round: a captured step reproduces the eager step bit for
    bit on every replay."""
    c = _case(name)
    c.budget = c.w.budget_blocks
    c.select_path = P.COMPKV_SELECT_AUTO
    d = c.dims
    n = int(c.seq_lens[0])
    k_new = c.K[:, :, n - 1].contiguous()
    v_new = c.V[:, :, n - 1].contiguous()
    ws = P.alloc_workspace(d, c.budget)
    ref = c.decode_step(k_new, v_new, ws=ws)
    torch.cuda.synchronize()
    outs = {k: torch.empty_like(v) for k, v in ref.items()}
    params = c.params()

    def call():
        P.compkv_decode_step(d, params, c.q, c.K, c.V, k_new, v_new, c.sl, c.summ.kmean, c.summ.dvar, c.summ.vmean,
                             outs["sel"], outs["n_sel"], outs["blk_logit"], outs["scores"], outs["out"], outs["lse"],
                             ws)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        call()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call()
    for rep in range(3):
        for t in outs.values():
            t.fill_(-3)
        g.replay()
        torch.cuda.synchronize()
        for k in ref:
            assert torch.equal(outs[k], ref[k]), f"{name} replay {rep}: {k} differs"
    print(f"[full-size {name}] {rep + 1} graph replays match the eager step", flush=True)
