"""Offload tier: K/V caches in pinned host memory read and written by the kernels across the host link
(needs an MI355X). Every call gives bit-identical results to a device-memory cache, and the fused step's
append lands in the host cache. The host-memory results are also checked against the CPU oracle directly
(summaries, selection under the tie band, compensated and dense outputs)."""
import pytest
import torch

import paper_2609_26300_amd as P
from gpu_case import PATHS, make_case
from test_gpu_step import _prefix_state

pytestmark = pytest.mark.gpu


def _pinned(t):
    h = torch.empty(t.shape, dtype=t.dtype, pin_memory=True)
    h.copy_(t.cpu())
    return h


@pytest.mark.parametrize("path", sorted(PATHS))
@pytest.mark.parametrize("name", ["tiny_4k", "llama8b_32k", "varlen"])
def test_host_cache_bitwise(name, path):
    print(f"\n[host cache {name} / {path}]", flush=True)
    c = make_case(name, path)
    c.run_all()
    ref_dense = c.dense_decode()
    Kh, Vh = _pinned(c.K), _pinned(c.V)
    d = c.dims
    units = (d.batch, d.n_kv_heads)
    # separate calls on the host cache
    summ = P.alloc_summaries(d)
    P.compkv_build_stats(d, Kh, Vh, c.sl, summ.kmean, summ.dvar, summ.vmean)
    torch.cuda.synchronize()
    for f in ("kmean", "dvar", "vmean"):
        assert torch.equal(getattr(summ, f), getattr(c.summ, f)), f
    out = torch.zeros_like(c.out)
    lse = torch.zeros_like(c.lse)
    P.compkv_sparse_decode(d, c.scale, c.q, Kh, Vh, c.summ.vmean, c.blk_logit, c.sl, c.sel, c.n_sel, out, lse, c.ws)
    dout, dlse = torch.zeros_like(c.out), torch.zeros_like(c.lse)
    P.compkv_dense_decode(d, c.scale, c.q, Kh, Vh, c.sl, dout, dlse, c.ws)
    torch.cuda.synchronize()
    assert torch.equal(out, c.out) and torch.equal(lse, c.lse)
    assert torch.equal(dout, ref_dense[0]) and torch.equal(dlse, ref_dense[1])
    c.check_stats(summ.kmean, summ.dvar, summ.vmean)
    c.check_step(c.sel, c.n_sel, out, lse)
    c.check_dense(dout, dlse)
    # the fused step with an append, from n - 1 cached tokens
    K2, V2, kn, vn, summ2 = _prefix_state(c)
    ref = c.decode_step(kn, vn, summ=summ2, K=K2, V=V2)
    K3, V3, _, _, summ3 = _prefix_state(c)
    K3h, V3h = _pinned(K3), _pinned(V3)
    r = c.decode_step(kn, vn, summ=summ3, K=K3h, V=V3h)
    torch.cuda.synchronize()
    for k in ref:
        assert torch.equal(r[k], ref[k]), k
    assert torch.equal(K3h, K2.cpu()) and torch.equal(V3h, V2.cpu())
    for f in ("kmean", "dvar", "vmean"):
        assert torch.equal(getattr(summ3, f), getattr(summ2, f)), f
    c.check_stats(summ3.kmean, summ3.dvar, summ3.vmean)
    c.check_step(r["sel"], r["n_sel"], r["out"], r["lse"])


@pytest.mark.parametrize("path", sorted(PATHS))
@pytest.mark.parametrize("name", ["tiny_4k", "llama8b_32k"])
def test_host_summaries_bitwise(name, path):
    """The paper's deployment layout: K/V and the fp32 summaries both in pinned host memory. Prefill,
    scoring, decode and the fused step (with its append and refresh) read and write them across the host
    link and give bit-identical results to device memory."""
    from types import SimpleNamespace

    print(f"\n[host summaries {name} / {path}]", flush=True)
    c = make_case(name, path)
    c.run_all()
    d = c.dims
    Kh, Vh = _pinned(c.K), _pinned(c.V)
    hs = SimpleNamespace(**{f: _pinned(torch.zeros_like(getattr(c.summ, f))) for f in ("kmean", "dvar", "vmean")})
    P.compkv_build_stats(d, Kh, Vh, c.sl, hs.kmean, hs.dvar, hs.vmean)
    torch.cuda.synchronize()
    for f in ("kmean", "dvar", "vmean"):
        assert torch.equal(getattr(hs, f), getattr(c.summ, f).cpu()), f
    units = (d.batch, d.n_kv_heads)
    sel = torch.full((*units, c.budget), -7, dtype=torch.int32, device="cuda")
    n_sel = torch.zeros(units, dtype=torch.int32, device="cuda")
    blk = torch.zeros_like(c.blk_logit)
    scores = torch.zeros_like(c.scores)
    P.compkv_score_select(d, c.params(), c.q, hs.kmean, hs.dvar, c.sl, sel, n_sel, blk, scores, c.ws)
    out, lse = torch.zeros_like(c.out), torch.zeros_like(c.lse)
    P.compkv_sparse_decode(d, c.scale, c.q, Kh, Vh, hs.vmean, blk, c.sl, sel, n_sel, out, lse, c.ws)
    torch.cuda.synchronize()
    for got, ref in ((sel, c.sel), (n_sel, c.n_sel), (blk, c.blk_logit), (scores, c.scores), (out, c.out),
                     (lse, c.lse)):
        assert torch.equal(got, ref)
    # the fused step with an append, from n - 1 cached tokens
    K2, V2, kn, vn, summ2 = _prefix_state(c)
    ref = c.decode_step(kn, vn, summ=summ2, K=K2, V=V2)
    K3, V3, _, _, summ3 = _prefix_state(c)
    hs3 = SimpleNamespace(**{f: _pinned(getattr(summ3, f)) for f in ("kmean", "dvar", "vmean")})
    r = c.decode_step(kn, vn, summ=hs3, K=_pinned(K3), V=_pinned(V3))
    torch.cuda.synchronize()
    for k in ref:
        assert torch.equal(r[k], ref[k]), k
    for f in ("kmean", "dvar", "vmean"):
        assert torch.equal(getattr(hs3, f), getattr(summ2, f).cpu()), f
    c.check_stats(hs3.kmean, hs3.dvar, hs3.vmean)
    c.check_step(r["sel"], r["n_sel"], r["out"], r["lse"])
