"""GPU parity of the fused decode step (compkv_decode_step) on every parity case (needs an MI355X).

For each case the separate calls (build, score/select, sparse decode) run first on the full context.
The fused step must then
  * without an append: reproduce the separate selection outputs bit for bit and the compensated
    output within the parity tolerance, and match the oracle end to end;
  * with an append from n - 1 cached tokens: store the new rows, leave summaries bit-identical to a
    prefill build over n tokens (Appendix E.1: only the active block changes), select exactly what the
    separate calls select, and match the oracle end to end.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_26300_amd as P
from gpu_case import CASES, LLAMA, PATHS, TINY, TOL, Case, bits_of, check_selection, dev_bf16, make_case, rel_err

pytestmark = pytest.mark.gpu

_cache = {}


def _prefix_state(c: Case):
    """Cache and summaries holding n - 1 tokens per sequence, plus the rows that the step appends."""
    d = c.dims
    K2, V2 = c.K.clone(), c.V.clone()
    kn = torch.zeros((d.batch, d.n_kv_heads, d.head_dim), dtype=torch.bfloat16, device="cuda")
    vn = torch.zeros_like(kn)
    for b, n in enumerate(c.seq_lens.tolist()):
        if n >= 1:
            kn[b] = c.K[b, :, n - 1]
            vn[b] = c.V[b, :, n - 1]
            K2[b, :, n - 1] = 0
            V2[b, :, n - 1] = 0
    before = torch.clamp(c.sl - 1, min=0).to(torch.int32)
    summ = P.alloc_summaries(d)
    P.compkv_build_stats(d, K2, V2, before, summ.kmean, summ.dvar, summ.vmean)
    return K2, V2, kn.contiguous(), vn.contiguous(), summ


@pytest.fixture(params=[(n, p) for n in sorted(CASES) for p in PATHS], ids=lambda x: f"{x[0]}-{x[1]}",
                scope="module")
def step(request):
    """Separate calls and fused steps (plain and appended) on one selection path."""
    name = request.param
    if name not in _cache:
        print(f"\n[step case {name[0]} / {name[1]} selection] generating + running", flush=True)
        c = make_case(*name)
        c.run_all()
        plain = c.decode_step()
        K2, V2, kn, vn, summ2 = _prefix_state(c)
        appended = c.decode_step(kn, vn, summ=summ2, K=K2, V=V2)
        torch.cuda.synchronize()
        _cache[name] = (c, plain, (K2, V2, summ2, appended))
    return _cache[name]


def _gpu(t):
    return t.cpu().numpy()


def _selection_equal(c: Case, r):
    for key, ref in (("sel", c.sel), ("n_sel", c.n_sel), ("blk_logit", c.blk_logit), ("scores", c.scores)):
        assert torch.equal(r[key], ref), key


def _oracle_end_to_end(c: Case, r):
    c.check_step(r["sel"], r["n_sel"], r["out"], r["lse"])


def test_step_selection_matches_separate_calls(step):
    c, plain, _ = step
    _selection_equal(c, plain)


def test_step_output_matches_separate_decode(step):
    c, plain, _ = step
    assert rel_err(_gpu(plain["out"]), _gpu(c.out), axis=-1) <= TOL
    assert np.max(np.abs(_gpu(plain["lse"]) - _gpu(c.lse))) <= 1e-4 * max(1.0, float(c.lse.abs().max()))


def test_step_end_to_end_parity(step):
    c, plain, _ = step
    _oracle_end_to_end(c, plain)


def test_step_append_state_bitwise(step):
    """The stored rows are the new tokens; every summary equals the prefill build over n tokens."""
    c, _, (K2, V2, summ2, _) = step
    assert torch.equal(K2, c.K) and torch.equal(V2, c.V)
    for name in ("kmean", "dvar", "vmean"):
        assert torch.equal(getattr(summ2, name), getattr(c.summ, name)), name


def test_step_append_outputs(step):
    c, _, (_, _, _, appended) = step
    _selection_equal(c, appended)
    _oracle_end_to_end(c, appended)


@pytest.mark.parametrize("path", sorted(PATHS))
def test_step_streaming_appends_match_build(path):
    """Forty fused steps, each appending one token: summaries stay bit-identical to a rebuild, and the
    last step's output matches the oracle."""
    w = TINY.with_(batch=2, context=1000, decode_steps=40, block_size=16, seed=31)
    c = Case(w, max_seq_len=w.capacity)
    c.select_path = PATHS[path]
    n0, T = 1000, 40
    c.K[:, :, n0:] = 0
    c.V[:, :, n0:] = 0
    c.build_stats()
    Kn = dev_bf16(c.K_bits[:, :, n0:n0 + T])
    Vn = dev_bf16(c.V_bits[:, :, n0:n0 + T])
    for t in range(T):
        sl = torch.full((w.batch,), n0 + t + 1, dtype=torch.int32, device="cuda")
        r = c.decode_step(Kn[:, :, t].contiguous(), Vn[:, :, t].contiguous(), sl=sl)
    torch.cuda.synchronize()
    assert np.array_equal(bits_of(c.K)[:, :, :n0 + T], c.K_bits[:, :, :n0 + T])
    ref = P.alloc_summaries(c.dims)
    P.compkv_build_stats(c.dims, c.K, c.V, sl, ref.kmean, ref.dvar, ref.vmean)
    for name in ("kmean", "dvar", "vmean"):
        assert torch.equal(getattr(ref, name), getattr(c.summ, name)), name
    c.seq_lens = np.full(w.batch, n0 + T, np.int32)
    _oracle_end_to_end(c, r)


@pytest.mark.parametrize("path", sorted(PATHS))
def test_step_graph_replays_match_eager(path):
    """A captured fused step (with its append, which rewrites the same row and block each time)
    reproduces the eager outputs on every replay."""
    c = Case(LLAMA.with_(batch=1, context=8192, seed=32))
    c.select_path = PATHS[path]
    c.build_stats()
    K2, V2, kn, vn, summ2 = _prefix_state(c)
    ref = c.decode_step(kn, vn, summ=summ2, K=K2, V=V2)
    torch.cuda.synchronize()
    d = c.dims
    outs = {k: torch.empty_like(v) for k, v in ref.items()}
    params = c.params()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())

    def call():
        P.compkv_decode_step(d, params, c.q, K2, V2, kn, vn, c.sl, summ2.kmean, summ2.dvar, summ2.vmean,
                             outs["sel"], outs["n_sel"], outs["blk_logit"], outs["scores"], outs["out"],
                             outs["lse"], c.ws)

    with torch.cuda.stream(side):
        call()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call()
    for rep in range(4):
        for t in outs.values():
            t.fill_(-3)
        g.replay()
        torch.cuda.synchronize()
        for k in ref:
            assert torch.equal(outs[k], ref[k]), f"replay {rep}: {k} differs"
        assert torch.equal(summ2.kmean, c.summ.kmean)
        c.dense_decode()  # unrelated eager work on the same workspace between replays
        torch.cuda.synchronize()


@pytest.mark.parametrize("path", sorted(PATHS))
def test_step_length_beyond_max_seq_appends_nothing(path):
    """A sequence whose length exceeds max_seq_len appends nothing: its cache rows and every block
    summary stay bit-identical, and the step's outputs equal a step without an append (the unit is
    decoded over max_seq_len tokens, like in every other call)."""
    w = TINY.with_(batch=2, context=1000, decode_steps=8, seed=34)
    c = Case(w, seq_lens=[1001, 700], max_seq_len=1000)
    c.select_path = PATHS[path]
    c.build_stats()
    K0, V0 = c.K.clone(), c.V.clone()
    summ0 = {k: getattr(c.summ, k).clone() for k in ("kmean", "dvar", "vmean")}
    ref = c.decode_step()
    kn = dev_bf16(c.K_bits[:, :, 1003])
    vn = dev_bf16(c.V_bits[:, :, 1004])
    r = c.decode_step(kn.contiguous(), vn.contiguous())
    torch.cuda.synchronize()
    # sequence 0 (1001 > max_seq_len): nothing stored, no summary touched
    assert torch.equal(c.K[0], K0[0]) and torch.equal(c.V[0], V0[0])
    for k, v in summ0.items():
        assert torch.equal(getattr(c.summ, k)[0], v[0]), k
    for k in ("sel", "n_sel", "out", "lse"):
        assert torch.equal(r[k][0], ref[k][0]), k
    # sequence 1 (700 tokens) did append row 699
    assert torch.equal(c.K[1, :, 699], kn[1]) and torch.equal(c.V[1, :, 699], vn[1])


@pytest.mark.parametrize("path", sorted(PATHS))
def test_empty_sequence_in_batch(path):
    """A sequence with no tokens has no blocks: nothing is selected, its output is zero and its lse is
    -inf, in the separate calls and in the fused step (which appends nothing for it); the other
    sequences of the batch are unaffected."""
    c = Case(TINY.with_(batch=3, seed=33), seq_lens=[0, 700, 1500], max_seq_len=1500)
    c.select_path = PATHS[path]
    c.run_all()
    for r in (dict(sel=c.sel, n_sel=c.n_sel, out=c.out, lse=c.lse), c.decode_step()):
        torch.cuda.synchronize()
        assert int(r["n_sel"][0].max()) == 0 and bool((r["sel"][0] == -1).all())
        assert float(r["out"][0].abs().max()) == 0.0
        assert bool(torch.isinf(r["lse"][0]).all()) and float(r["lse"][0].max()) < 0
    # the non-empty sequences against the oracle
    G = c.G
    for b, h in c.units():
        if b == 0:
            continue
        q, K, V, n = c.unit_inputs(b, h)
        st = c.oracle_stats(b, h)
        sc = c.oracle_scores(b, h, st)
        for sel, nsel, out in ((c.sel, c.n_sel, c.out),):
            s = _gpu(sel)[b, h, :int(_gpu(nsel)[b, h])]
            check_selection(s, sc["score"], c.budget, c.n_sink, c.n_recent)
            o, _ = oracle.sparse_decode(q, K, V, st[0], st[2], n, c.w.block_size, c.scale, s)
            assert rel_err(_gpu(out)[b, h * G:(h + 1) * G], o, axis=1) <= TOL


@pytest.mark.parametrize("path", sorted(PATHS))
@pytest.mark.parametrize("name", ["tiny_4k", "llama8b_32k", "wide_gqa_8k", "block1", "budget300_x2000"])
def test_step_stays_within_workspace(name, path):
    """Given exactly compkv_workspace_bytes(..., COMPKV_WS_DECODE_STEP) bytes, the fused step writes
    nothing past them (a guard region after the workspace keeps its pattern) and gives the outputs of a
    step on an oversized workspace. Only the per-unit words at the start of the workspace (16 bytes per
    unit, rounded up to 256) need initial contents (zero); the step leaves them zero, and the rest of
    the workspace may hold anything."""
    c = make_case(name, path)
    c.build_stats()
    d = c.dims
    need = P.compkv_workspace_bytes(d, c.budget, P.COMPKV_WS_DECODE_STEP)
    state = -(-16 * d.batch * d.n_kv_heads // 256) * 256
    guard = 1 << 16
    buf = torch.full((need + guard,), 0xA5, dtype=torch.uint8, device="cuda")
    buf[:state] = 0
    r = c.decode_step(ws=buf[:need])
    ref = c.decode_step(ws=P.alloc_workspace(d, c.budget))
    torch.cuda.synchronize()
    assert bool((buf[need:] == 0xA5).all()), "the step wrote past its workspace"
    assert bool((buf[:state] == 0).all()), "the step left its per-unit words non-zero"
    for k in ref:
        assert torch.equal(r[k], ref[k]), k
