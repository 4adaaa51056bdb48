"""C ABI contract checks that need no GPU: the library loads, exports every function the header
declares, sizes workspaces, and rejects invalid arguments on the host before enqueuing anything
(every call below returns from host-side validation; no kernel is launched)."""
import ctypes
import json
import os

import pytest

import paper_2609_26300_amd as P

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
EINVAL, EUNSUP, EBUDGET, EWS = -1, -2, -3, -4
FAKE = ctypes.c_void_p(4096)  # never dereferenced: validation fails before any device access


def dims(**kw):
    base = dict(batch=1, n_q_heads=8, n_kv_heads=2, head_dim=128, block_size=16, n_var_groups=4,
                capacity_tokens=4096, max_seq_len=4096)
    base.update(kw)
    layout = base.pop("group_layout", 0)
    return P.make_dims(group_layout=layout, **base)


def test_library_exports_every_declared_function():
    L = P.library()
    names = P.exported_symbols()
    assert {"compkv_build_stats", "compkv_append_stats", "compkv_score_select", "compkv_sparse_decode",
            "compkv_dense_decode", "compkv_decode_step", "compkv_workspace_bytes", "compkv_status_string",
            "compkv_version"} <= set(names)
    for name in names:
        assert hasattr(L, name), name


def test_status_strings_and_version():
    assert P.compkv_version() >= 100
    for code in (0, EINVAL, EUNSUP, EBUDGET, EWS, -5):
        assert P.compkv_status_string(code).startswith("COMPKV_")
    assert "unknown" in P.compkv_status_string(-99)


def test_workspace_sizing():
    d = dims()
    for which in range(5):
        assert P.compkv_workspace_bytes(d, 16, which) > 0
    assert P.compkv_workspace_bytes(d, 16, 5) == 0
    all_ = P.compkv_workspace_bytes(d, 16, 0)
    assert all(all_ >= P.compkv_workspace_bytes(d, 16, w) for w in (1, 2, 3, 4))
    # the fused step holds the scoring region plus its decode partials
    assert P.compkv_workspace_bytes(d, 16, P.COMPKV_WS_DECODE_STEP) > P.compkv_workspace_bytes(
        d, 16, P.COMPKV_WS_SCORE_SELECT)
    assert P.compkv_workspace_bytes(d, 0, 0) == 0
    assert P.compkv_workspace_bytes(dims(head_dim=96), 16, 0) == 0
    # grows with context
    assert P.compkv_workspace_bytes(dims(capacity_tokens=131072, max_seq_len=131072), 64, 0) > all_


@pytest.mark.parametrize("bad,code", [
    (dict(n_q_heads=6, n_kv_heads=4), EINVAL),
    (dict(batch=0), EINVAL),
    (dict(max_seq_len=5000), EINVAL),
    (dict(max_seq_len=0), EINVAL),
    (dict(head_dim=96), EUNSUP),
    (dict(n_q_heads=24, n_kv_heads=2), EUNSUP),  # G = 12
    (dict(block_size=0), EUNSUP),
    (dict(n_var_groups=3), EUNSUP),
    (dict(n_var_groups=128, head_dim=64), EUNSUP),
    (dict(group_layout=2), EUNSUP),
])
def test_invalid_dims_rejected(bad, code):
    d = dims(**bad)
    L = P.library()
    assert L.compkv_build_stats(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None) == code
    assert L.compkv_dense_decode(ctypes.byref(d), 0.1, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, 1 << 30,
                                 None) == code


def test_null_pointers_rejected():
    d = dims()
    L = P.library()
    assert L.compkv_build_stats(ctypes.byref(d), None, FAKE, FAKE, FAKE, FAKE, FAKE, None) == EINVAL
    assert L.compkv_append_stats(ctypes.byref(d), FAKE, FAKE, None, FAKE, FAKE, FAKE, FAKE, FAKE, None) == EINVAL
    p = P.CompkvSelectParams(16, 1, 2, 0.088)
    assert L.compkv_score_select(ctypes.byref(d), ctypes.byref(p), FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE,
                                 None, FAKE, 1 << 30, None) == EINVAL  # n_sel required
    # blk_logit is optional: a NULL one gets past the pointer checks (to the workspace check)
    assert L.compkv_score_select(ctypes.byref(d), ctypes.byref(p), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None,
                                 None, FAKE, 1, None) == EWS
    assert L.compkv_sparse_decode(ctypes.byref(d), 0.1, None, FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE,
                                  16, FAKE, None, FAKE, 1 << 30, None) == EINVAL  # q required


def test_misaligned_vector_arrays_rejected():
    """Arrays read with 16-byte vector loads must be 16-byte aligned: a pointer 4 bytes off is EINVAL
    on the host for every call that reads it (the rest of each call's arguments are valid)."""
    d = dims()
    L = P.library()
    OFF = ctypes.c_void_p(4100)
    assert L.compkv_build_stats(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, OFF, FAKE, None) == EINVAL  # dvar
    assert L.compkv_build_stats(ctypes.byref(d), OFF, FAKE, FAKE, FAKE, FAKE, FAKE, None) == EINVAL  # k_cache
    assert L.compkv_append_stats(ctypes.byref(d), FAKE, FAKE, OFF, FAKE, FAKE, FAKE, FAKE, FAKE, None) == EINVAL
    p = P.CompkvSelectParams(16, 1, 2, 0.088)
    assert L.compkv_score_select(ctypes.byref(d), ctypes.byref(p), OFF, FAKE, FAKE, FAKE, FAKE, FAKE, None,
                                 None, FAKE, 1 << 30, None) == EINVAL  # q
    assert L.compkv_score_select(ctypes.byref(d), ctypes.byref(p), FAKE, FAKE, OFF, FAKE, FAKE, FAKE, None,
                                 None, FAKE, 1 << 30, None) == EINVAL  # dvar
    assert L.compkv_sparse_decode(ctypes.byref(d), 0.1, FAKE, FAKE, FAKE, FAKE, OFF, FAKE, FAKE, FAKE, FAKE,
                                  16, FAKE, None, FAKE, 1 << 30, None) == EINVAL  # vmean
    for name in ("q", "k_cache", "v_cache", "k_new", "v_new", "kmean", "dvar", "vmean"):
        assert _step(L, d, p, **{name: OFF}) == EINVAL, name


def test_budget_below_mandatory_set_rejected():
    """Section 4.2: the sink and recent blocks count inside the budget, so K < n_sink + n_recent
    cannot be honoured."""
    d = dims()
    L = P.library()
    for K, ns, nr in ((2, 1, 2), (0, 0, 0), (4, 3, 2)):
        p = P.CompkvSelectParams(K, ns, nr, 0.088)
        rc = L.compkv_score_select(ctypes.byref(d), ctypes.byref(p), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                                   None, FAKE, 1 << 30, None)
        assert rc == (EINVAL if K < 1 else EBUDGET)


def test_workspace_checks():
    d = dims()
    L = P.library()
    p = P.CompkvSelectParams(16, 1, 2, 0.088)
    need = P.compkv_workspace_bytes(d, 16, P.COMPKV_WS_SCORE_SELECT)
    args = [FAKE] * 6 + [FAKE, None]
    assert L.compkv_score_select(ctypes.byref(d), ctypes.byref(p), *args, FAKE, need - 1, None) == EWS
    assert L.compkv_score_select(ctypes.byref(d), ctypes.byref(p), *args, None, need, None) == EWS
    assert L.compkv_score_select(ctypes.byref(d), ctypes.byref(p), *args, ctypes.c_void_p(4100), need,
                                 None) == EWS  # misaligned
    need = P.compkv_workspace_bytes(d, 1, P.COMPKV_WS_DENSE_DECODE)
    assert L.compkv_dense_decode(ctypes.byref(d), 0.1, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, need - 1,
                                 None) == EWS


def test_summary_layout_matches_paper():
    """Section 4.2: a block summary holds 2d + r + 1 scalars; the library stores the mean key (d),
    grouped variances (r) and mean value (d) per block, and derives |b| from the sequence length."""
    fx = json.load(open(os.path.join(GOLDEN, "summary_size.json")))
    for case in fx["cases"]:
        d = dims(head_dim=fx["head_dim"], n_var_groups=case["r"])
        per_block = d.head_dim + d.n_var_groups + d.head_dim + 1
        assert per_block == case["scalars_per_block"]


def test_product_path_fails_loudly_without_library(monkeypatch, tmp_path):
    """No CPU fallback: a missing library makes every call raise."""
    from paper_2609_26300_amd import binding
    monkeypatch.setattr(binding, "_lib", None)
    monkeypatch.setattr(binding, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(binding.CompkvError):
        binding.library()


def _step(L, d, p, ws=FAKE, ws_bytes=1 << 30, k_new=FAKE, v_new=FAKE, **null):
    args = dict(q=FAKE, k_cache=FAKE, v_cache=FAKE, k_new=k_new, v_new=v_new, seq_lens=FAKE, kmean=FAKE,
                dvar=FAKE, vmean=FAKE, sel=FAKE, n_sel=FAKE, blk_logit=FAKE, scores=None, out=FAKE, lse=None)
    args.update(null)
    return L.compkv_decode_step(ctypes.byref(d), ctypes.byref(p), *args.values(), ws, ws_bytes, None)


def test_decode_step_validation():
    d = dims()
    L = P.library()
    p = P.CompkvSelectParams(16, 1, 2, 0.088)
    for name in ("q", "k_cache", "v_cache", "seq_lens", "kmean", "dvar", "vmean", "sel", "n_sel",
                 "blk_logit", "out"):
        assert _step(L, d, p, **{name: None}) == EINVAL, name
    assert _step(L, d, p, k_new=None) == EINVAL  # k_new and v_new come together
    assert _step(L, d, p, v_new=None) == EINVAL
    assert _step(L, dims(head_dim=96), p) == EUNSUP
    assert _step(L, d, P.CompkvSelectParams(2, 1, 2, 0.088)) == EBUDGET
    need = P.compkv_workspace_bytes(d, 16, P.COMPKV_WS_DECODE_STEP)
    assert _step(L, d, p, ws_bytes=need - 1) == EWS
    assert _step(L, d, p, ws=ctypes.c_void_p(4100), ws_bytes=need) == EWS
    assert _step(L, d, p, ws=None, ws_bytes=need) == EWS
    # more partials than one merge holds: the separate calls remain available for such shapes
    huge = dims(block_size=1, capacity_tokens=1 << 20, max_seq_len=1 << 20)
    assert _step(L, huge, P.CompkvSelectParams(64, 1, 2, 0.088)) == EUNSUP


def test_score_select_block_count_limit():
    """Above 128 * (4096 / G - 1) blocks per unit the selection's partial merge does not fit: the call says
    so before enqueuing anything."""
    L = P.library()
    p = P.CompkvSelectParams(64, 1, 2, 0.088)
    args = [FAKE] * 6 + [FAKE, None]
    ok = dims(block_size=1, capacity_tokens=65536, max_seq_len=65536)  # G = 4: 512 chunks of 128
    big = dims(block_size=1, capacity_tokens=1 << 20, max_seq_len=(1 << 20))
    need = P.compkv_workspace_bytes(big, 64, P.COMPKV_WS_SCORE_SELECT)
    assert L.compkv_score_select(ctypes.byref(big), ctypes.byref(p), *args, FAKE, need, None) == EUNSUP
    need = P.compkv_workspace_bytes(ok, 64, P.COMPKV_WS_SCORE_SELECT)
    assert L.compkv_score_select(ctypes.byref(ok), ctypes.byref(p), *args, FAKE, need - 1, None) == EWS


def test_select_path_validation():
    """select_path: an unknown value is EINVAL; the one-group path is refused (before anything is
    enqueued) when G * blocks exceeds 8192, and accepted up to that bound; the one-launch step is
    accepted by both calls (the scoring call runs it chunked)."""
    L = P.library()
    args = [FAKE] * 6 + [FAKE, None]

    def score(d, path, ws_bytes=None):
        p = P.CompkvSelectParams(64, 1, 2, 0.088, path)
        need = P.compkv_workspace_bytes(d, 64, P.COMPKV_WS_SCORE_SELECT)
        return L.compkv_score_select(ctypes.byref(d), ctypes.byref(p), *args, FAKE,
                                     need - 1 if ws_bytes is None else ws_bytes, None)

    fits = dims(block_size=16, capacity_tokens=2048 * 16, max_seq_len=2048 * 16)  # G = 4: 4 * 2048 = 8192
    over = dims(block_size=16, capacity_tokens=2049 * 16, max_seq_len=2049 * 16)
    for bad in (-1, 5):
        assert score(fits, bad) == EINVAL
        assert _step(L, fits, P.CompkvSelectParams(64, 1, 2, 0.088, bad)) == EINVAL
    assert score(over, P.COMPKV_SELECT_ONE_GROUP) == EUNSUP
    assert _step(L, over, P.CompkvSelectParams(64, 1, 2, 0.088, P.COMPKV_SELECT_ONE_GROUP)) == EUNSUP
    # accepted: the calls get as far as the workspace check
    for path in (P.COMPKV_SELECT_AUTO, P.COMPKV_SELECT_CHUNKED, P.COMPKV_SELECT_ONE_GROUP,
                 P.COMPKV_SELECT_CHUNKED_EXACT, P.COMPKV_SELECT_STREAM):
        assert score(fits, path) == EWS
    for path in (P.COMPKV_SELECT_AUTO, P.COMPKV_SELECT_CHUNKED, P.COMPKV_SELECT_CHUNKED_EXACT,
                 P.COMPKV_SELECT_STREAM):
        assert score(over, path) == EWS
    # one workspace size serves the fused step on every path
    need = P.compkv_workspace_bytes(fits, 64, P.COMPKV_WS_DECODE_STEP)
    for path in (P.COMPKV_SELECT_CHUNKED, P.COMPKV_SELECT_ONE_GROUP, P.COMPKV_SELECT_CHUNKED_EXACT,
                 P.COMPKV_SELECT_STREAM):
        assert _step(L, fits, P.CompkvSelectParams(64, 1, 2, 0.088, path), ws_bytes=need - 1) == EWS


def test_score_kind_and_compensation_validation():
    """Unknown score kinds and compensation modes are EINVAL; the sparse decode takes vmean and
    blk_logit together (both NULL: the Drop decode) -- all checked before anything is enqueued."""
    L = P.library()
    d = dims()
    args = [FAKE] * 6 + [FAKE, None]
    need = P.compkv_workspace_bytes(d, 16, P.COMPKV_WS_SCORE_SELECT)
    for kind, rc in ((-1, EINVAL), (3, EINVAL), (P.COMPKV_SCORE_MASS, EWS), (P.COMPKV_SCORE_FIRST_ORDER, EWS)):
        p = P.CompkvSelectParams(16, 1, 2, 0.088, 0, kind)
        assert L.compkv_score_select(ctypes.byref(d), ctypes.byref(p), *args, FAKE, need - 1, None) == rc
        assert _step(L, d, p, ws_bytes=1) == rc
    for comp, rc in ((-1, EINVAL), (2, EINVAL), (P.COMPKV_COMP_DROP, EWS), (P.COMPKV_COMP_MEAN, EWS)):
        assert _step(L, d, P.CompkvSelectParams(16, 1, 2, 0.088, 0, 0, comp), ws_bytes=1) == rc

    def sparse(vmean, blk, kmean=None):
        return L.compkv_sparse_decode(ctypes.byref(d), 0.1, FAKE, FAKE, FAKE, kmean, vmean, blk, FAKE, FAKE, FAKE,
                                      16, FAKE, None, FAKE, 1, None)

    # Mean needs the block logits or the mean keys to form them; Drop takes neither vmean nor blk_logit
    assert sparse(FAKE, None) == EINVAL and sparse(None, FAKE) == EINVAL and sparse(None, FAKE, FAKE) == EINVAL
    assert sparse(None, None) == EWS and sparse(FAKE, FAKE) == EWS
    assert sparse(FAKE, None, FAKE) == EWS and sparse(None, None, FAKE) == EWS


def test_decode_step_path_resolution():
    """compkv_decode_step_path reports the launch shape without enqueuing anything: explicit paths as
    requested (the fused selection + exact launch and the two-launch step whenever their limits
    hold), AUTO as one group or the chunked launches, and errors as statuses."""
    small = dims(block_size=16, capacity_tokens=4096, max_seq_len=4096)  # 256 blocks
    big = dims(block_size=32, capacity_tokens=32768, max_seq_len=32768)  # 1024 blocks
    prm = lambda path, K=16: P.CompkvSelectParams(K, 1, 2, 0.088, path)
    assert P.compkv_decode_step_path(big, prm(P.COMPKV_SELECT_ONE_GROUP)) == P.COMPKV_SELECT_ONE_GROUP
    for d in (small, big):
        assert P.compkv_decode_step_path(d, prm(P.COMPKV_SELECT_CHUNKED)) == P.COMPKV_SELECT_CHUNKED
        assert P.compkv_decode_step_path(d, prm(P.COMPKV_SELECT_CHUNKED_EXACT)) == P.COMPKV_SELECT_CHUNKED_EXACT
        assert P.compkv_decode_step_path(d, prm(P.COMPKV_SELECT_STREAM)) == P.COMPKV_SELECT_STREAM
    assert P.compkv_decode_step_path(small, prm(P.COMPKV_SELECT_AUTO)) in (P.COMPKV_SELECT_ONE_GROUP,
                                                                           P.COMPKV_SELECT_CHUNKED_EXACT)
    assert P.compkv_decode_step_path(big, prm(P.COMPKV_SELECT_AUTO)) in (P.COMPKV_SELECT_CHUNKED,
                                                                         P.COMPKV_SELECT_CHUNKED_EXACT)
    # past the fused kernels' budget limit the chunked-exact and one-launch requests run chunked
    assert P.compkv_decode_step_path(big, prm(P.COMPKV_SELECT_CHUNKED_EXACT, 1025)) == P.COMPKV_SELECT_CHUNKED
    assert P.compkv_decode_step_path(big, prm(P.COMPKV_SELECT_STREAM, 1025)) == P.COMPKV_SELECT_CHUNKED
    # past 8192 blocks per unit AUTO falls back to the chunked launches
    long_ = dims(block_size=16, capacity_tokens=8193 * 16, max_seq_len=8193 * 16)
    assert P.compkv_decode_step_path(long_, prm(P.COMPKV_SELECT_AUTO)) in (P.COMPKV_SELECT_CHUNKED,
                                                                           P.COMPKV_SELECT_CHUNKED_EXACT)
    with pytest.raises(P.CompkvError):
        P.compkv_decode_step_path(big, prm(7))
    with pytest.raises(P.CompkvError):
        P.compkv_decode_step_path(dims(head_dim=96), prm(0))


def test_paged_dims_validation():
    """Paged caches: the page size must be a multiple of the block size (else EUNSUPPORTED), and
    num_pages, pages_per_seq and the table must be given with capacity = pages_per_seq * page_tokens
    (else EINVAL) -- checked before anything is enqueued."""
    import torch

    L = P.library()
    table = torch.zeros((1, 4), dtype=torch.int32)  # never read: every case fails validation or the ws check
    need = lambda d: P.compkv_workspace_bytes(d, 16, P.COMPKV_WS_ALL)

    def dense(d):
        return L.compkv_dense_decode(ctypes.byref(d), 0.1, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, 1, None)

    ok = dims(capacity_tokens=128, max_seq_len=128, block_table=table, page_tokens=32, num_pages=9)
    assert need(ok) > 0 and dense(ok) == EWS
    bad = dims(capacity_tokens=96, max_seq_len=96, block_table=table, page_tokens=24, num_pages=9)
    assert dense(bad) == EUNSUP  # 24 is not a multiple of block_size 16
    assert dense(dims(capacity_tokens=100, max_seq_len=100, block_table=table, page_tokens=32, num_pages=9)) == EINVAL
    assert dense(dims(capacity_tokens=128, max_seq_len=128, block_table=table, page_tokens=32, num_pages=0)) == EINVAL
    nul = dims(capacity_tokens=128, max_seq_len=128, block_table=table, page_tokens=32, num_pages=9)
    nul.block_table = None
    assert dense(nul) == EINVAL
    neg = dims()
    neg.page_tokens = -1
    assert dense(neg) == EINVAL


def test_host_cache_pointer_rejects_unmapped_memory():
    """The offload tier's pointer query refuses null arguments and memory that is not pinned and mapped
    (a plain host buffer), so such a cache never reaches a kernel."""
    L = P.library()
    out = ctypes.c_void_p()
    assert L.compkv_host_cache_pointer(None, ctypes.byref(out)) == EINVAL
    buf = ctypes.create_string_buffer(4096)
    assert L.compkv_host_cache_pointer(ctypes.cast(buf, ctypes.c_void_p), None) == EINVAL
    assert L.compkv_host_cache_pointer(ctypes.cast(buf, ctypes.c_void_p), ctypes.byref(out)) == EINVAL
    assert not out.value
    import torch

    with pytest.raises(P.CompkvError):  # unpinned host tensors are refused by the binding
        d = dims()
        K = torch.zeros((1, 2, 4096, 128), dtype=torch.bfloat16)
        P.compkv_dense_decode(d, 0.1, K, K, K, K, K, None, K)


def test_noalloc_step_rejects_oversized_workspace():
    """The allocation-free step refuses, before enqueuing anything, a step whose workspace would exceed
    its fixed scratch (here 256 units of 65536 blocks: over 1 GiB of score terms)."""
    L = P.library()
    limit = P.compkv_decode_step_noalloc_limit()
    assert limit == 32 << 20
    d = dims(batch=16, n_q_heads=128, n_kv_heads=16, block_size=16, capacity_tokens=1 << 20, max_seq_len=1 << 20)
    assert P.compkv_workspace_bytes(d, 64, P.COMPKV_WS_DECODE_STEP) > limit
    p = P.CompkvSelectParams(64, 1, 2, 0.088)
    assert L.compkv_decode_step_noalloc(ctypes.byref(d), ctypes.byref(p), *([FAKE] * 15), None) == -6
    assert "scratch" in P.compkv_status_string(-6)
