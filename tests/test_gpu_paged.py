"""Paged KV caches (block-table indirection) on the GPU (needs an MI355X).

Every case's cache is scattered over randomly permuted physical pages; every call then runs on the
paged cache and must give bit-identical results to the contiguous cache: the summaries of the prefill
build, the selection and outputs of score_select / sparse_decode / dense_decode, and the fused step on
every launch shape with an append whose row lands in the right page. The paged results are also
checked against the CPU oracle directly (summaries, the selection under the tie band, the compensated
and dense outputs), so they do not rest on the contiguous path alone.
"""
import numpy as np
import pytest
import torch

import paper_2609_26300_amd as P
from gpu_case import CASES, PATHS, make_case
from test_gpu_step import _prefix_state

pytestmark = pytest.mark.gpu

# case -> tokens per page (a multiple of the case's block size)
PAGED = {"tiny_4k": 16, "llama8b_32k": 64, "varlen": 48, "block1": 16, "partial_tail": 32, "g8_b64": 128,
         "short": 16}


def _paginate(c, page, seed):
    """Physical pages for c's caches: [num_pages][hkv][page][d] and the int32 block table."""
    d = c.dims
    pps = -(-d.capacity_tokens // page)
    rng = np.random.default_rng(seed)
    num_pages = d.batch * pps + 3  # spare pages stay unused
    perm = rng.permutation(num_pages)[:d.batch * pps].reshape(d.batch, pps).astype(np.int32)
    table = torch.from_numpy(perm).cuda()
    cap = pps * page

    def pack(X):
        Xp = torch.zeros((num_pages, d.n_kv_heads, page, d.head_dim), dtype=X.dtype, device="cuda")
        Xc = torch.zeros((d.batch, d.n_kv_heads, cap, d.head_dim), dtype=X.dtype, device="cuda")
        Xc[:, :, :d.capacity_tokens] = X
        for b in range(d.batch):
            for lp in range(pps):
                Xp[perm[b, lp]] = Xc[b, :, lp * page:(lp + 1) * page]
        return Xp

    def unpack(Xp):
        out = torch.empty((d.batch, d.n_kv_heads, cap, d.head_dim), dtype=Xp.dtype, device="cuda")
        for b in range(d.batch):
            for lp in range(pps):
                out[b, :, lp * page:(lp + 1) * page] = Xp[perm[b, lp]]
        return out[:, :, :d.capacity_tokens]

    dims = P.make_dims(d.batch, d.n_q_heads, d.n_kv_heads, d.head_dim, d.block_size, d.n_var_groups, cap,
                       max_seq_len=d.max_seq_len, group_layout=d.group_layout, block_table=table,
                       page_tokens=page, num_pages=num_pages)
    return dims, pack, unpack


def _run(c, dims, K, V, path):
    """score_select + sparse_decode + dense_decode on (dims, K, V), with c's summaries rebuilt there."""
    units = (dims.batch, dims.n_kv_heads)
    summ = P.alloc_summaries(dims)
    P.compkv_build_stats(dims, K, V, c.sl, summ.kmean, summ.dvar, summ.vmean)
    ws = P.alloc_workspace(dims, c.budget)
    c.select_path = path
    r = dict(sel=torch.full((*units, c.budget), -7, dtype=torch.int32, device="cuda"),
             n_sel=torch.zeros(units, dtype=torch.int32, device="cuda"),
             blk=torch.zeros((*units, c.G, dims.xcap), dtype=torch.float32, device="cuda"),
             scores=torch.zeros((*units, dims.xcap), dtype=torch.float32, device="cuda"),
             out=torch.zeros((dims.batch, dims.n_q_heads, dims.head_dim), dtype=torch.float32, device="cuda"),
             lse=torch.zeros((dims.batch, dims.n_q_heads), dtype=torch.float32, device="cuda"),
             dout=torch.zeros((dims.batch, dims.n_q_heads, dims.head_dim), dtype=torch.float32, device="cuda"),
             dlse=torch.zeros((dims.batch, dims.n_q_heads), dtype=torch.float32, device="cuda"))
    P.compkv_score_select(dims, c.params(), c.q, summ.kmean, summ.dvar, c.sl, r["sel"], r["n_sel"], r["blk"],
                          r["scores"], ws)
    P.compkv_sparse_decode(dims, c.scale, c.q, K, V, summ.vmean, r["blk"], c.sl, r["sel"], r["n_sel"], r["out"],
                           r["lse"], ws)
    P.compkv_dense_decode(dims, c.scale, c.q, K, V, c.sl, r["dout"], r["dlse"], ws)
    torch.cuda.synchronize()
    return summ, r


@pytest.mark.parametrize("name", sorted(PAGED))
def test_paged_separate_calls_bitwise(name):
    c = make_case(name, "chunked")
    dims, pack, _ = _paginate(c, PAGED[name], seed=len(name))
    s0, r0 = _run(c, c.dims, c.K, c.V, P.COMPKV_SELECT_CHUNKED)
    s1, r1 = _run(c, dims, pack(c.K), pack(c.V), P.COMPKV_SELECT_CHUNKED)
    X = c.dims.xcap
    for f in ("kmean", "dvar", "vmean"):
        assert torch.equal(getattr(s0, f)[:, :, :X], getattr(s1, f)[:, :, :X]), f
    for k in r0:
        a, b = r0[k], r1[k]
        if k in ("blk", "scores"):
            a, b = a[..., :X], b[..., :X]
        assert torch.equal(a, b), k
    c.check_stats(s1.kmean, s1.dvar, s1.vmean)
    c.check_step(r1["sel"], r1["n_sel"], r1["out"], r1["lse"])
    c.check_dense(r1["dout"], r1["dlse"])


@pytest.mark.parametrize("path", sorted(PATHS))
@pytest.mark.parametrize("name", sorted(PAGED))
def test_paged_decode_step_with_append_bitwise(name, path):
    c = make_case(name, path)
    c.run_all()
    dims, pack, unpack = _paginate(c, PAGED[name], seed=7 + len(name))
    # contiguous reference: the fused step appending token n - 1
    K2, V2, kn, vn, summ2 = _prefix_state(c)
    ref = c.decode_step(kn, vn, summ=summ2, K=K2, V=V2)
    torch.cuda.synchronize()
    # the same on the paged cache (prefix state rebuilt there)
    Kp, Vp = pack(_prefix_state(c)[0]), pack(_prefix_state(c)[1])
    summ = P.alloc_summaries(dims)
    before = torch.clamp(c.sl - 1, min=0).to(torch.int32)
    P.compkv_build_stats(dims, Kp, Vp, before, summ.kmean, summ.dvar, summ.vmean)
    units = (dims.batch, dims.n_kv_heads)
    r = {k: torch.full_like(v, -3) for k, v in ref.items()}
    r["blk_logit"] = torch.zeros((*units, c.G, dims.xcap), dtype=torch.float32, device="cuda")
    r["scores"] = torch.zeros((*units, dims.xcap), dtype=torch.float32, device="cuda")
    ws = P.alloc_workspace(dims, c.budget)
    P.compkv_decode_step(dims, c.params(), c.q, Kp, Vp, kn, vn, c.sl, summ.kmean, summ.dvar, summ.vmean, r["sel"],
                         r["n_sel"], r["blk_logit"], r["scores"], r["out"], r["lse"], ws)
    torch.cuda.synchronize()
    X = c.dims.xcap
    for k in ("sel", "n_sel", "out", "lse"):
        assert torch.equal(r[k], ref[k]), k
    assert torch.equal(r["blk_logit"][..., :X], ref["blk_logit"]) and torch.equal(r["scores"][..., :X], ref["scores"])
    for f in ("kmean", "dvar", "vmean"):
        assert torch.equal(getattr(summ, f)[:, :, :X], getattr(summ2, f)), f
    assert torch.equal(unpack(Kp), K2) and torch.equal(unpack(Vp), V2)  # the appended rows, in their pages
    c.check_stats(summ.kmean, summ.dvar, summ.vmean)
    c.check_step(r["sel"], r["n_sel"], r["out"], r["lse"])
