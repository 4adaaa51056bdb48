"""The allocation-free decode step (compkv_decode_step_noalloc) against compkv_decode_step (needs an
MI355X).

Two calls in a row through the C ABI, the second on a smaller input (fewer sequences, a shorter context,
another budget), so the second runs on the scratch as the first left it. Each call must give exactly the
outputs, cache rows and summaries of compkv_decode_step with a workspace on the same inputs (same kernels
and launch shapes, so bit for bit).
"""
import pytest
import torch

import paper_2609_26300_amd as P
from gpu_case import LLAMA, TINY, Case

pytestmark = pytest.mark.gpu


def _inputs(c: Case):
    """Cache and summaries holding n - 1 tokens, and the rows the step appends."""
    d = c.dims
    n = int(c.seq_lens[0])
    kn = c.K[:, :, n - 1].contiguous()
    vn = c.V[:, :, n - 1].contiguous()
    c.K[:, :, n - 1:] = 0
    c.V[:, :, n - 1:] = 0
    before = torch.full((d.batch,), n - 1, dtype=torch.int32, device="cuda")
    summ = P.alloc_summaries(d)
    P.compkv_build_stats(d, c.K, c.V, before, summ.kmean, summ.dvar, summ.vmean)
    return kn, vn, summ


def _outputs(c: Case):
    d = c.dims
    units = (d.batch, d.n_kv_heads)
    return dict(sel=torch.full((*units, c.budget), -7, dtype=torch.int32, device="cuda"),
                n_sel=torch.zeros(units, dtype=torch.int32, device="cuda"),
                blk_logit=torch.zeros((*units, c.G, d.xcap), dtype=torch.float32, device="cuda"),
                scores=torch.zeros((*units, d.xcap), dtype=torch.float32, device="cuda"),
                out=torch.zeros((d.batch, d.n_q_heads, d.head_dim), dtype=torch.float32, device="cuda"),
                lse=torch.zeros((d.batch, d.n_q_heads), dtype=torch.float32, device="cuda"))


def _compare(c: Case):
    """One allocation-free step and one workspace step from the same state; everything bitwise equal."""
    kn, vn, summ = _inputs(c)
    K0, V0 = c.K.clone(), c.V.clone()
    summ2 = P.Summaries(summ.kmean.clone(), summ.dvar.clone(), summ.vmean.clone())
    params = c.params()
    r1 = _outputs(c)
    print(f"[no-alloc] {c.w.name} batch {c.w.batch} context {c.w.context} K {c.budget}", flush=True)
    P.compkv_decode_step_noalloc(c.dims, params, c.q, c.K, c.V, kn, vn, c.sl, summ.kmean, summ.dvar, summ.vmean,
                                 r1["sel"], r1["n_sel"], r1["blk_logit"], r1["scores"], r1["out"], r1["lse"])
    r2 = _outputs(c)
    ws = P.alloc_workspace(c.dims, c.budget)
    P.compkv_decode_step(c.dims, params, c.q, K0, V0, kn, vn, c.sl, summ2.kmean, summ2.dvar, summ2.vmean,
                         r2["sel"], r2["n_sel"], r2["blk_logit"], r2["scores"], r2["out"], r2["lse"], ws)
    torch.cuda.synchronize()
    for k in r1:
        assert torch.equal(r1[k], r2[k]), k
    assert torch.equal(c.K, K0) and torch.equal(c.V, V0)
    for k in ("kmean", "dvar", "vmean"):
        assert torch.equal(getattr(summ, k), getattr(summ2, k)), k
    assert int(r1["n_sel"].min()) == min(c.budget, -(-int(c.seq_lens[0]) // c.w.block_size))


def test_noalloc_matches_workspace_step_twice():
    """A 32K layer of 8 units, then a smaller 4K case of 2 units on the scratch it left behind."""
    _compare(Case(LLAMA.with_(context=32768, seed=41)))
    _compare(Case(TINY.with_(context=3000, budget_blocks=24, seed=42)))
