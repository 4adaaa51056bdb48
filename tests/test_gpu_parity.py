"""GPU parity: every call of the C ABI against the CPU oracle on seeded inputs (needs an MI355X).

Cases span the tiny 4K workload, the Llama-3-8B-shaped 32K layer at full size, and edge cases:
partial last blocks, block size 1, per-coordinate groups (r = d), the interleaved group layout,
head_dim 64, group sizes 1/2/8, variable sequence lengths, contexts of 1-3 blocks (mandatory set
overlap) and budgets at or above the block count.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_case import CASES, LLAMA, PATHS, TINY, TOL, Case, check_selection, dev_bf16, make_case, rel_err

pytestmark = pytest.mark.gpu

_cache = {}


def _get(name, path):
    if (name, path) not in _cache:
        print(f"\n[case {name} / {path} selection] generating + running", flush=True)
        c = make_case(name, path)
        c.run_all()
        _cache[name, path] = c
    return _cache[name, path]


@pytest.fixture(params=sorted(CASES), scope="module")
def case(request):
    """A case for the calls that do not depend on the selection path (chunked selection run)."""
    return _get(request.param, "chunked")


@pytest.fixture(params=[(n, p) for n in sorted(CASES) for p in PATHS], ids=lambda x: f"{x[0]}-{x[1]}",
                scope="module")
def case_p(request):
    """A case on each selection path."""
    return _get(*request.param)


def _gpu(t):
    return t.cpu().numpy()


def test_build_stats_parity(case):
    km, dv, vm = (_gpu(x) for x in (case.summ.kmean, case.summ.dvar, case.summ.vmean))
    for b, h in case.units():
        okm, odv, ovm = case.oracle_stats(b, h)
        X = okm.shape[0]
        assert rel_err(km[b, h, :X], okm, axis=1) <= TOL
        assert rel_err(vm[b, h, :X], ovm, axis=1) <= TOL
        assert rel_err(dv[b, h, :X], odv) <= TOL


def test_score_select_parity(case_p):
    case = case_p
    sel, nsel = _gpu(case.sel), _gpu(case.n_sel)
    scores, zbar = _gpu(case.scores), _gpu(case.blk_logit)
    for b, h in case.units():
        sc = case.oracle_scores(b, h)
        X = sc["score"].shape[0]
        assert rel_err(scores[b, h, :X], sc["score"]) <= TOL
        assert rel_err(zbar[b, h, :, :X], sc["zbar"]) <= TOL
        assert nsel[b, h] == min(case.budget, X)
        check_selection(sel[b, h, :nsel[b, h]], sc["score"], case.budget, case.n_sink, case.n_recent)
        assert np.all(sel[b, h, nsel[b, h]:] == -1)


@pytest.mark.parametrize("from_kmean", [False, True], ids=["blk_logit", "kmean"])
def test_sparse_decode_with_oracle_selection(case, from_kmean):
    """Eq. compkv-output on the oracle's own selected set (decode tested apart from selection), with the
    block-mean logits passed in (blk_logit) or recomputed by the library from the mean keys."""
    d = case.dims
    sel = np.full((d.batch, d.n_kv_heads, case.budget), -1, np.int32)
    nsel = np.zeros((d.batch, d.n_kv_heads), np.int32)
    stats = {}
    for b, h in case.units():
        stats[b, h] = case.oracle_stats(b, h)
        s = oracle.select(case.oracle_scores(b, h, stats[b, h])["score"], case.budget, case.n_sink, case.n_recent)
        sel[b, h, :len(s)] = s
        nsel[b, h] = len(s)
    out, lse = case.sparse_decode(torch.from_numpy(sel).cuda(), torch.from_numpy(nsel).cuda(), from_kmean)
    out, lse = _gpu(out), _gpu(lse)
    G = case.G
    for b, h in case.units():
        q, K, V, n = case.unit_inputs(b, h)
        km, dv, vm = stats[b, h]
        o, l = oracle.sparse_decode(q, K, V, km, vm, n, case.w.block_size, case.scale, sel[b, h, :nsel[b, h]])
        assert rel_err(out[b, h * G:(h + 1) * G], o, axis=1) <= TOL
        assert np.max(np.abs(lse[b, h * G:(h + 1) * G] - l)) <= TOL * max(1.0, np.max(np.abs(l)))
    case.sparse_decode()  # restore the pipeline's own output


def test_score_select_without_block_logits(case_p):
    """blk_logit is optional: without it the selection outputs are the same, bit for bit."""
    case = case_p
    import paper_2609_26300_amd as P
    sel = torch.full_like(case.sel, -7)
    n_sel = torch.zeros_like(case.n_sel)
    scores = torch.zeros_like(case.scores)
    P.compkv_score_select(case.dims, case.params(), case.q, case.summ.kmean, case.summ.dvar, case.sl, sel, n_sel,
                          None, scores, case.ws)
    torch.cuda.synchronize()
    assert torch.equal(sel, case.sel) and torch.equal(n_sel, case.n_sel) and torch.equal(scores, case.scores)


def test_end_to_end_parity(case_p):
    """Whole step: once the GPU's selection passes the band rule, the oracle output recomputed on
    that same selection must match the GPU output."""
    case = case_p
    sel, nsel = _gpu(case.sel), _gpu(case.n_sel)
    out, lse = _gpu(case.out), _gpu(case.lse)
    G = case.G
    for b, h in case.units():
        q, K, V, n = case.unit_inputs(b, h)
        st = case.oracle_stats(b, h)
        sc = case.oracle_scores(b, h, st)
        s = sel[b, h, :nsel[b, h]]
        check_selection(s, sc["score"], case.budget, case.n_sink, case.n_recent)
        o, l = oracle.sparse_decode(q, K, V, st[0], st[2], n, case.w.block_size, case.scale, s)
        assert rel_err(out[b, h * G:(h + 1) * G], o, axis=1) <= TOL


def test_dense_decode_parity(case):
    out, lse = case.dense_decode()
    out, lse = _gpu(out), _gpu(lse)
    G = case.G
    for b, h in case.units():
        q, K, V, n = case.unit_inputs(b, h)
        o, l = oracle.dense_decode(q, K, V, n, case.scale)
        assert rel_err(out[b, h * G:(h + 1) * G], o, axis=1) <= TOL
        assert np.max(np.abs(lse[b, h * G:(h + 1) * G] - l)) <= TOL * max(1.0, np.max(np.abs(l)))


def test_rerun_is_bit_identical(case_p):
    """No float atomics: a second run reproduces every output bit."""
    case = case_p
    before = [x.clone() for x in (case.summ.kmean, case.summ.dvar, case.summ.vmean, case.sel, case.n_sel,
                                  case.scores, case.out, case.lse)]
    case.run_all()
    after = (case.summ.kmean, case.summ.dvar, case.summ.vmean, case.sel, case.n_sel, case.scores, case.out, case.lse)
    for x, y in zip(before, after):
        assert torch.equal(x, y)


# ---------------------------------------------------------------- special cases pinned by the paper

def test_budget_all_blocks_equals_dense_on_gpu():
    """K >= X: Eq. compkv-output has no omitted block, so sparse decode is dense attention."""
    c = Case(TINY.with_(context=777, budget_blocks=64, seed=21))
    c.run_all()
    o_sp, l_sp = _gpu(c.out), _gpu(c.lse)
    o_de, l_de = (_gpu(x) for x in c.dense_decode())
    assert rel_err(o_sp, o_de, axis=-1) <= TOL and np.max(np.abs(l_sp - l_de)) <= 1e-4


def test_block_size_one_equals_dense_on_gpu():
    """B = 1: every pseudo-token is its token, so any budget reproduces dense attention."""
    c = Case(TINY.with_(context=500, block_size=1, budget_blocks=20, seed=22))
    c.run_all()
    assert np.all(_gpu(c.scores)[:, :, :500] == 0.0)
    # all scores tie at zero: the stable Top-K takes the lowest candidate ids
    assert np.all(_gpu(c.sel) == np.array(list(range(18)) + [498, 499], np.int32))
    o_de, l_de = (_gpu(x) for x in c.dense_decode())
    assert rel_err(_gpu(c.out), o_de, axis=-1) <= TOL and np.max(np.abs(_gpu(c.lse) - l_de)) <= 1e-4


def test_append_matches_build_bitwise():
    """Streaming appends (Appendix E.1) give the same summaries, bit for bit, as a prefill build over
    the final cache; completed blocks never change; the cache rows hold the appended tokens."""
    w = TINY.with_(batch=2, context=1000, decode_steps=40, block_size=16, seed=23)
    c = Case(w, max_seq_len=w.capacity)
    n0 = 1000
    torch.cuda.synchronize()
    # cache holding only the prefix: zero the rows that the appends will write
    c.K[:, :, n0:] = 0
    c.V[:, :, n0:] = 0
    c.build_stats()
    km0 = c.summ.kmean.clone()
    Kn = dev_bf16(c.K_bits[:, :, n0:n0 + 40])
    Vn = dev_bf16(c.V_bits[:, :, n0:n0 + 40])
    import paper_2609_26300_amd as P
    for t in range(40):
        sl = torch.full((w.batch,), n0 + t, dtype=torch.int32, device="cuda")
        P.compkv_append_stats(c.dims, c.K, c.V, Kn[:, :, t].contiguous(), Vn[:, :, t].contiguous(), sl,
                              c.summ.kmean, c.summ.dvar, c.summ.vmean)
    torch.cuda.synchronize()
    assert np.array_equal(c.K.view(torch.int16).cpu().numpy().view(np.uint16)[:, :, :n0 + 40],
                          c.K_bits[:, :, :n0 + 40])
    assert torch.equal(c.summ.kmean[:, :, :n0 // 16], km0[:, :, :n0 // 16])
    ref = P.alloc_summaries(c.dims)
    sl = torch.full((w.batch,), n0 + 40, dtype=torch.int32, device="cuda")
    P.compkv_build_stats(c.dims, c.K, c.V, sl, ref.kmean, ref.dvar, ref.vmean)
    X = -(-(n0 + 40) // 16)
    assert torch.equal(ref.kmean[:, :, :X], c.summ.kmean[:, :, :X])
    assert torch.equal(ref.dvar[:, :, :X], c.summ.dvar[:, :, :X])
    assert torch.equal(ref.vmean[:, :, :X], c.summ.vmean[:, :, :X])
    # and against the oracle
    for b in range(w.batch):
        for h in range(w.n_kv_heads):
            okm, odv, ovm = oracle.block_stats(c.K_bits[b, h], c.V_bits[b, h], n0 + 40, 16, w.n_var_groups)
            assert rel_err(c.summ.kmean[b, h, :X].cpu().numpy(), okm, axis=1) <= TOL
            assert rel_err(c.summ.dvar[b, h, :X].cpu().numpy(), odv) <= TOL


@pytest.mark.parametrize("path", sorted(PATHS))
def test_graph_replays_match_eager(path):
    """The library enqueues no memsets and leaves its arrival counters at zero after each call, so a
    captured HIP graph of score_select + sparse_decode reproduces the eager outputs on every replay."""
    c = Case(LLAMA.with_(batch=1, context=8192, seed=24))
    c.select_path = PATHS[path]
    c.run_all()
    ref = [x.clone() for x in (c.sel, c.n_sel, c.blk_logit, c.out, c.lse)]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        c.score_select()
        c.sparse_decode()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    sel, n_sel, blk, out, lse = c.sel, c.n_sel, c.blk_logit, c.out, c.lse
    import paper_2609_26300_amd as P
    params = c.params()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        P.compkv_score_select(c.dims, params, c.q, c.summ.kmean, c.summ.dvar, c.sl, sel, n_sel, blk, None, c.ws)
        P.compkv_sparse_decode(c.dims, c.scale, c.q, c.K, c.V, c.summ.vmean, blk, c.sl, sel, n_sel, out, lse, c.ws)
    for rep in range(4):
        for t in (sel, n_sel, blk, out, lse):
            t.fill_(-3)
        g.replay()
        torch.cuda.synchronize()
        for x, y in zip((sel, n_sel, blk, out, lse), ref):
            assert torch.equal(x, y), f"replay {rep} differs"
        c.dense_decode()  # unrelated eager work on the same workspace between replays
        torch.cuda.synchronize()
