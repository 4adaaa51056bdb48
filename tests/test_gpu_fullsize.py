"""Full-size parity of the fused decode step (needs an MI355X).

The long-context 128K layer (batch 4; budgets 32, 64 and 128 blocks), the wide-GQA 64K layer (batch 8,
G = 8) and the streaming layer's first appending step (131072 + 1 tokens, so the last block holds one
token), each run exactly as bench.py times them: summaries built over n tokens, then one
compkv_decode_step on the automatic launch shape that appends row n - 1 (rewriting it with the same
values, which also refreshes the active block's summary). Every unit is checked against the oracle: its
summaries, the selection (bit-exact outside the tie band), the compensated output and lse. The streaming
layer is also run through 40 appending steps from its 131072-token prefill (a block completes and the
next one starts), and the last step is checked the same way.
"""
import numpy as np
import pytest
import torch

import paper_2609_26300_amd as P
from gpu_case import Case
from workloads import WORKLOADS

pytestmark = pytest.mark.gpu

# (workload, tokens in the cache after the step, budgets)
FULL = {
    "long_128k": (WORKLOADS["long_128k"], None, (32, 64, 128)),
    "wide_gqa_64k": (WORKLOADS["wide_gqa_64k"], None, (None,)),
    "streaming_128k": (WORKLOADS["streaming_128k"], WORKLOADS["streaming_128k"].context + 1, (None,)),
}
PATH_NAMES = {P.COMPKV_SELECT_CHUNKED: "chunked", P.COMPKV_SELECT_ONE_GROUP: "one group",
              P.COMPKV_SELECT_CHUNKED_EXACT: "chunked + fused selection/exact",
              P.COMPKV_SELECT_STREAM: "one launch"}

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
    print(f"[full-size {name} K={c.budget}] oracle over all {len(c.units())} units", flush=True)
    c.prefetch_oracle()
    c.check_stats(c.summ.kmean, c.summ.dvar, c.summ.vmean)
    c.check_step(r["sel"], r["n_sel"], r["out"], r["lse"])


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


@pytest.mark.parametrize("name", ["long_128k", "wide_gqa_64k"])
def test_fullsize_repeated_steps_bit_identical(name):
    """The fused launch's last workgroup of each unit merges the unit's partials in index order, whichever
    workgroup arrives last: 200 eager steps and 200 graph replays of the same full-size step (no append)
    all give the same output and lse bits."""
    c = _case(name)
    c.budget = c.w.budget_blocks
    c.select_path = P.COMPKV_SELECT_AUTO
    d = c.dims
    ws = P.alloc_workspace(d, c.budget)
    ref = c.decode_step(ws=ws)
    torch.cuda.synchronize()
    outs = {k: torch.empty_like(v) for k, v in ref.items()}
    params = c.params()

    def call():
        P.compkv_decode_step(d, params, c.q, c.K, c.V, None, None, c.sl, c.summ.kmean, c.summ.dvar, c.summ.vmean,
                             outs["sel"], outs["n_sel"], outs["blk_logit"], outs["scores"], outs["out"], outs["lse"],
                             ws)

    bad = 0
    for rep in range(200):
        call()
        if rep % 20 == 19:
            torch.cuda.synchronize()
            bad += int(not (torch.equal(outs["out"], ref["out"]) and torch.equal(outs["lse"], ref["lse"])))
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        call()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(20):
            call()
    for rep in range(10):
        outs["out"].fill_(-3)
        g.replay()
        torch.cuda.synchronize()
        bad += int(not (torch.equal(outs["out"], ref["out"]) and torch.equal(outs["lse"], ref["lse"])))
    assert bad == 0, f"{bad} of 20 checks differ"


def test_fullsize_streaming_forty_appends():
    """The streaming layer (batch 2, 8 KV heads, K = 128) prefilled with 131072 tokens, then 40 fused steps
    that each append the next token and score / select / decode with fresh queries (Appendix E.2's
    decode phase). Block 4096 fills and block 4097 opens on the way. After the last step every summary
    equals a prefill build over the final cache bit for bit, and every unit's summaries, selection and
    output match the oracle over 131112 tokens."""
    from workloads import gen_queries
    from gpu_case import dev_bf16

    _cases.clear()
    torch.cuda.empty_cache()
    w = WORKLOADS["streaming_128k"]
    n0, T = w.context, 40
    c = Case(w, seq_lens=[n0 + T] * w.batch, max_seq_len=w.capacity)
    c.select_path = P.COMPKV_SELECT_AUTO
    d = c.dims
    c.K[:, :, n0:] = 0
    c.V[:, :, n0:] = 0
    summ = P.alloc_summaries(d)
    P.compkv_build_stats(d, c.K, c.V, torch.full((w.batch,), n0, dtype=torch.int32, device="cuda"), summ.kmean,
                         summ.dvar, summ.vmean)
    Kn = dev_bf16(c.K_bits[:, :, n0:n0 + T])
    Vn = dev_bf16(c.V_bits[:, :, n0:n0 + T])
    ws = P.alloc_workspace(d, c.budget)
    path = P.compkv_decode_step_path(d, c.params())
    print(f"[full-size streaming] 40 appending steps, launch shape {PATH_NAMES.get(path, path)}", flush=True)
    for t in range(T):
        c.q = dev_bf16(np.stack([gen_queries(w, 0, b, t) for b in range(w.batch)]))
        sl = torch.full((w.batch,), n0 + t + 1, dtype=torch.int32, device="cuda")
        r = c.decode_step(Kn[:, :, t].contiguous(), Vn[:, :, t].contiguous(), sl=sl, summ=summ, ws=ws)
    torch.cuda.synchronize()
    c.q_bits = np.stack([gen_queries(w, 0, b, T - 1) for b in range(w.batch)])
    ref = P.alloc_summaries(d)
    P.compkv_build_stats(d, c.K, c.V, sl, ref.kmean, ref.dvar, ref.vmean)
    for f in ("kmean", "dvar", "vmean"):
        assert torch.equal(getattr(ref, f), getattr(summ, f)), f
    assert np.array_equal(c.K.view(torch.int16).cpu().numpy().view(np.uint16)[:, :, :n0 + T], c.K_bits[:, :, :n0 + T])
    c.prefetch_oracle()
    c.check_stats(summ.kmean, summ.dvar, summ.vmean)
    c.check_step(r["sel"], r["n_sel"], r["out"], r["lse"])
