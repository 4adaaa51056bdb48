"""ctypes binding of libcompkv.so: argument marshalling only (see include/compkv.h for semantics)."""
from __future__ import annotations

import ctypes
import math
import os
import re
from dataclasses import dataclass

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libcompkv.so")
HEADER_PATH = os.path.join(os.path.dirname(_PKG), "include", "compkv.h")

COMPKV_GROUPS_ROTATE_HALF = 0
COMPKV_GROUPS_INTERLEAVED = 1
COMPKV_WS_ALL = 0
COMPKV_WS_SCORE_SELECT = 1
COMPKV_WS_SPARSE_DECODE = 2
COMPKV_WS_DENSE_DECODE = 3
COMPKV_WS_DECODE_STEP = 4
COMPKV_SELECT_AUTO = 0
COMPKV_SELECT_CHUNKED = 1
COMPKV_SELECT_ONE_GROUP = 2
COMPKV_SELECT_CHUNKED_EXACT = 3
COMPKV_SELECT_STREAM = 4
COMPKV_SCORE_COMPKV = 0
COMPKV_SCORE_MASS = 1
COMPKV_SCORE_FIRST_ORDER = 2
COMPKV_COMP_MEAN = 0
COMPKV_COMP_DROP = 1


class CompkvError(RuntimeError):
    pass


class CompkvDims(ctypes.Structure):
    _fields_ = [(name, ctypes.c_int32) for name in (
        "batch", "n_q_heads", "n_kv_heads", "head_dim", "block_size", "n_var_groups", "group_layout",
        "capacity_tokens", "max_seq_len", "page_tokens", "num_pages", "pages_per_seq")] + [
        ("block_table", ctypes.c_void_p)]

    @property
    def paged(self) -> bool:
        return self.page_tokens > 0

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def xcap(self) -> int:
        return -(-self.capacity_tokens // self.block_size)

    @property
    def xmax(self) -> int:
        """Blocks of the longest sequence (max_seq_len)."""
        return -(-self.max_seq_len // self.block_size)


class CompkvSelectParams(ctypes.Structure):
    _fields_ = [("budget_blocks", ctypes.c_int32), ("n_sink", ctypes.c_int32),
                ("n_recent", ctypes.c_int32), ("scale", ctypes.c_float), ("select_path", ctypes.c_int32),
                ("score_kind", ctypes.c_int32), ("compensation", ctypes.c_int32)]


def make_dims(batch, n_q_heads, n_kv_heads, head_dim, block_size, n_var_groups, capacity_tokens,
              max_seq_len=None, group_layout=COMPKV_GROUPS_ROTATE_HALF, block_table=None, page_tokens=0,
              num_pages=0) -> CompkvDims:
    """Call geometry. For a paged cache pass block_table (int32 [batch][pages_per_seq] on the device;
    the dims keep a reference to it), page_tokens and num_pages; capacity_tokens is then
    pages_per_seq * page_tokens."""
    d = CompkvDims(batch, n_q_heads, n_kv_heads, head_dim, block_size, n_var_groups, group_layout,
                   capacity_tokens, capacity_tokens if max_seq_len is None else max_seq_len)
    if block_table is not None:
        if block_table.dtype != torch.int32 or block_table.dim() != 2 or block_table.shape[0] != batch:
            raise CompkvError("block_table must be int32 [batch][pages_per_seq]")
        if not block_table.is_contiguous():
            raise CompkvError("block_table must be contiguous")
        d.page_tokens, d.num_pages, d.pages_per_seq = int(page_tokens), int(num_pages), int(block_table.shape[1])
        d.block_table = block_table.data_ptr()
        d._table = block_table  # keep the device memory alive as long as the dims
    return d


_lib = None
_vp = ctypes.c_void_p
_i32 = ctypes.c_int32


def library():
    """The loaded libcompkv.so; raises if it has not been built (no fallback exists)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise CompkvError(f"{LIB_PATH} is not built; run __graft_entry__.build() or "
                              "python -m paper_2609_26300_amd.build")
        L = ctypes.CDLL(LIB_PATH)
        dp = ctypes.POINTER(CompkvDims)
        L.compkv_build_stats.argtypes = [dp, _vp, _vp, _vp, _vp, _vp, _vp, _vp]
        L.compkv_append_stats.argtypes = [dp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp]
        L.compkv_score_select.argtypes = [dp, ctypes.POINTER(CompkvSelectParams), _vp, _vp, _vp, _vp, _vp,
                                          _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp]
        L.compkv_sparse_decode.argtypes = [dp, ctypes.c_float, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                           _i32, _vp, _vp, _vp, ctypes.c_size_t, _vp]
        L.compkv_dense_decode.argtypes = [dp, ctypes.c_float, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                          ctypes.c_size_t, _vp]
        L.compkv_decode_step.argtypes = [dp, ctypes.POINTER(CompkvSelectParams), _vp, _vp, _vp, _vp, _vp, _vp,
                                         _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp]
        L.compkv_decode_step_noalloc.argtypes = [dp, ctypes.POINTER(CompkvSelectParams)] + [_vp] * 16
        L.compkv_decode_step_noalloc_limit.argtypes = []
        L.compkv_decode_step_noalloc_limit.restype = ctypes.c_size_t
        L.compkv_decode_step_path.argtypes = [dp, ctypes.POINTER(CompkvSelectParams)]
        L.compkv_phase_trace_set.argtypes = [_vp, _vp]
        L.compkv_phase_trace_set.restype = ctypes.c_int
        L.compkv_host_cache_pointer.argtypes = [_vp, ctypes.POINTER(ctypes.c_void_p)]
        L.compkv_host_cache_pointer.restype = ctypes.c_int
        L.compkv_workspace_bytes.argtypes = [dp, _i32, _i32]
        L.compkv_workspace_bytes.restype = ctypes.c_size_t
        L.compkv_status_string.argtypes = [ctypes.c_int]
        L.compkv_status_string.restype = ctypes.c_char_p
        L.compkv_version.argtypes = []
        for name in ("compkv_build_stats", "compkv_append_stats", "compkv_score_select",
                     "compkv_sparse_decode", "compkv_dense_decode", "compkv_decode_step", "compkv_decode_step_path",
                     "compkv_decode_step_noalloc",
                     "compkv_version"):
            getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def exported_symbols() -> list[str]:
    """Function names declared in include/compkv.h."""
    text = open(HEADER_PATH).read()
    return sorted(set(re.findall(r"^\s*(?:int|size_t|const char\*)\s+(compkv_\w+)\s*\(", text, re.M)))


def compkv_status_string(status: int) -> str:
    return library().compkv_status_string(int(status)).decode()


def compkv_version() -> int:
    return library().compkv_version()


def _check(status: int, what: str):
    if status != 0:
        raise CompkvError(f"{what}: {compkv_status_string(status)}")


def _ptr(t, dtype, shape, name, nullable=False):
    if t is None:
        if nullable:
            return None
        raise CompkvError(f"{name} is required")
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise CompkvError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != dtype:
        raise CompkvError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise CompkvError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise CompkvError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    return t.data_ptr()


def _mem_ptr(t, dtype, shape, name, nullable=False):
    """Device address of a cache or summary array: a CUDA tensor, or a pinned host tensor (the offload
    tier, mapped into the device address space by compkv_host_cache_pointer)."""
    if isinstance(t, torch.Tensor) and t.device.type == "cpu":
        if not t.is_pinned():
            raise CompkvError(f"{name} in host memory must be pinned")
        if t.dtype != dtype or not t.is_contiguous() or tuple(t.shape) != tuple(shape):
            raise CompkvError(f"{name} must be a contiguous {dtype} tensor of shape {tuple(shape)}")
        dev = ctypes.c_void_p()
        _check(library().compkv_host_cache_pointer(ctypes.c_void_p(t.data_ptr()), ctypes.byref(dev)),
               "compkv_host_cache_pointer")
        return dev.value
    return _ptr(t, dtype, shape, name, nullable)


def _kv_ptr(t, shape, name):
    return _mem_ptr(t, torch.bfloat16, shape, name)


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if isinstance(stream, torch.cuda.Stream) else stream


def _ws(workspace):
    if workspace is None or workspace.device.type != "cuda" or not workspace.is_contiguous():
        raise CompkvError("workspace must be a contiguous CUDA tensor")
    return workspace.data_ptr(), workspace.numel() * workspace.element_size()


def compkv_decode_step_path(dims: CompkvDims, params: CompkvSelectParams) -> int:
    """The launch shape compkv_decode_step takes (COMPKV_SELECT_ONE_GROUP / _CHUNKED / _CHUNKED_EXACT)."""
    st = library().compkv_decode_step_path(ctypes.byref(dims), ctypes.byref(params))
    _check(st if st < 0 else 0, "compkv_decode_step_path")
    return int(st)


def compkv_workspace_bytes(dims: CompkvDims, budget_blocks: int, which: int = COMPKV_WS_ALL) -> int:
    return int(library().compkv_workspace_bytes(ctypes.byref(dims), int(budget_blocks), int(which)))


def alloc_workspace(dims: CompkvDims, budget_blocks: int, device="cuda") -> torch.Tensor:
    """Workspace large enough for every call (no initial contents are required)."""
    nbytes = compkv_workspace_bytes(dims, budget_blocks, COMPKV_WS_ALL)
    if nbytes == 0:
        raise CompkvError("invalid dims for workspace sizing")
    return torch.zeros(nbytes, dtype=torch.uint8, device=device)


@dataclass
class Summaries:
    kmean: torch.Tensor  # fp32 [batch][n_kv_heads][Xcap][d]
    dvar: torch.Tensor   # fp32 [batch][n_kv_heads][Xcap][r]
    vmean: torch.Tensor  # fp32 [batch][n_kv_heads][Xcap][d]


def alloc_summaries(dims: CompkvDims, device="cuda") -> Summaries:
    shp = (dims.batch, dims.n_kv_heads, dims.xcap)
    return Summaries(
        kmean=torch.zeros(*shp, dims.head_dim, dtype=torch.float32, device=device),
        dvar=torch.zeros(*shp, dims.n_var_groups, dtype=torch.float32, device=device),
        vmean=torch.zeros(*shp, dims.head_dim, dtype=torch.float32, device=device),
    )


def _shapes(d: CompkvDims):
    cache = ((d.num_pages, d.n_kv_heads, d.page_tokens, d.head_dim) if d.paged
             else (d.batch, d.n_kv_heads, d.capacity_tokens, d.head_dim))
    summ = (d.batch, d.n_kv_heads, d.xcap, d.head_dim)
    dvar = (d.batch, d.n_kv_heads, d.xcap, d.n_var_groups)
    q = (d.batch, d.n_q_heads, d.head_dim)
    return cache, summ, dvar, q


def compkv_build_stats(dims, k_cache, v_cache, seq_lens, kmean, dvar, vmean, stream=None):
    cache, summ, dv, _ = _shapes(dims)
    bf, f32 = torch.bfloat16, torch.float32
    st = library().compkv_build_stats(
        ctypes.byref(dims), _kv_ptr(k_cache, cache, "k_cache"), _kv_ptr(v_cache, cache, "v_cache"),
        _ptr(seq_lens, torch.int32, (dims.batch,), "seq_lens"), _mem_ptr(kmean, f32, summ, "kmean"),
        _mem_ptr(dvar, f32, dv, "dvar"), _mem_ptr(vmean, f32, summ, "vmean"), _stream(stream))
    _check(st, "compkv_build_stats")


def compkv_append_stats(dims, k_cache, v_cache, k_new, v_new, seq_lens, kmean, dvar, vmean, stream=None):
    cache, summ, dv, _ = _shapes(dims)
    bf, f32 = torch.bfloat16, torch.float32
    new = (dims.batch, dims.n_kv_heads, dims.head_dim)
    st = library().compkv_append_stats(
        ctypes.byref(dims), _kv_ptr(k_cache, cache, "k_cache"), _kv_ptr(v_cache, cache, "v_cache"),
        _ptr(k_new, bf, new, "k_new"), _ptr(v_new, bf, new, "v_new"),
        _ptr(seq_lens, torch.int32, (dims.batch,), "seq_lens"), _mem_ptr(kmean, f32, summ, "kmean"),
        _mem_ptr(dvar, f32, dv, "dvar"), _mem_ptr(vmean, f32, summ, "vmean"), _stream(stream))
    _check(st, "compkv_append_stats")


def compkv_score_select(dims, params: CompkvSelectParams, q, kmean, dvar, seq_lens, sel, n_sel, blk_logit,
                        scores, workspace, stream=None):
    _, summ, dv, qs = _shapes(dims)
    f32, i32 = torch.float32, torch.int32
    units = (dims.batch, dims.n_kv_heads)
    ws, ws_bytes = _ws(workspace)
    st = library().compkv_score_select(
        ctypes.byref(dims), ctypes.byref(params), _ptr(q, torch.bfloat16, qs, "q"),
        _mem_ptr(kmean, f32, summ, "kmean"), _mem_ptr(dvar, f32, dv, "dvar"),
        _ptr(seq_lens, i32, (dims.batch,), "seq_lens"), _ptr(sel, i32, (*units, params.budget_blocks), "sel"),
        _ptr(n_sel, i32, units, "n_sel"),
        _ptr(blk_logit, f32, (*units, dims.group, dims.xcap), "blk_logit", nullable=True),
        _ptr(scores, f32, (*units, dims.xcap), "scores", nullable=True), ws, ws_bytes, _stream(stream))
    _check(st, "compkv_score_select")


def compkv_sparse_decode(dims, scale, q, k_cache, v_cache, vmean, blk_logit, seq_lens, sel, n_sel, out,
                         lse=None, workspace=None, stream=None, kmean=None):
    """Compensated sparse decode; vmean = blk_logit = None gives the Drop decode. With blk_logit None
    and vmean given, the block-mean logits are recomputed from kmean."""
    cache, summ, _, qs = _shapes(dims)
    bf, f32, i32 = torch.bfloat16, torch.float32, torch.int32
    units = (dims.batch, dims.n_kv_heads)
    if sel is None or sel.dim() != 3:
        raise CompkvError("sel must be int32 [batch][n_kv_heads][budget]")
    ws, ws_bytes = _ws(workspace)
    st = library().compkv_sparse_decode(
        ctypes.byref(dims), float(scale), _ptr(q, bf, qs, "q"), _kv_ptr(k_cache, cache, "k_cache"),
        _kv_ptr(v_cache, cache, "v_cache"), _mem_ptr(kmean, f32, summ, "kmean", nullable=True),
        _mem_ptr(vmean, f32, summ, "vmean", nullable=True),
        _ptr(blk_logit, f32, (*units, dims.group, dims.xcap), "blk_logit", nullable=True),
        _ptr(seq_lens, i32, (dims.batch,), "seq_lens"), _ptr(sel, i32, (*units, sel.shape[2]), "sel"),
        _ptr(n_sel, i32, units, "n_sel"), int(sel.shape[2]), _ptr(out, f32, qs, "out"),
        _ptr(lse, f32, qs[:2], "lse", nullable=True), ws, ws_bytes, _stream(stream))
    _check(st, "compkv_sparse_decode")


def compkv_dense_decode(dims, scale, q, k_cache, v_cache, seq_lens, out, lse=None, workspace=None, stream=None):
    cache, _, _, qs = _shapes(dims)
    bf, f32 = torch.bfloat16, torch.float32
    ws, ws_bytes = _ws(workspace)
    st = library().compkv_dense_decode(
        ctypes.byref(dims), float(scale), _ptr(q, bf, qs, "q"), _kv_ptr(k_cache, cache, "k_cache"),
        _kv_ptr(v_cache, cache, "v_cache"), _ptr(seq_lens, torch.int32, (dims.batch,), "seq_lens"),
        _ptr(out, f32, qs, "out"), _ptr(lse, f32, qs[:2], "lse", nullable=True), ws, ws_bytes,
        _stream(stream))
    _check(st, "compkv_dense_decode")


def compkv_decode_step(dims, params: CompkvSelectParams, q, k_cache, v_cache, k_new, v_new, seq_lens, kmean,
                       dvar, vmean, sel, n_sel, blk_logit, scores, out, lse=None, workspace=None, stream=None):
    """One fused decode step; seq_lens are the lengths after the new token (k_new/v_new may be None)."""
    cache, summ, dv, qs = _shapes(dims)
    bf, f32, i32 = torch.bfloat16, torch.float32, torch.int32
    units = (dims.batch, dims.n_kv_heads)
    new = (*units, dims.head_dim)
    if (k_new is None) != (v_new is None):
        raise CompkvError("k_new and v_new must be given together")
    ws, ws_bytes = _ws(workspace)
    st = library().compkv_decode_step(
        ctypes.byref(dims), ctypes.byref(params), _ptr(q, bf, qs, "q"), _kv_ptr(k_cache, cache, "k_cache"),
        _kv_ptr(v_cache, cache, "v_cache"), _ptr(k_new, bf, new, "k_new", nullable=True),
        _ptr(v_new, bf, new, "v_new", nullable=True), _ptr(seq_lens, i32, (dims.batch,), "seq_lens"),
        _mem_ptr(kmean, f32, summ, "kmean"), _mem_ptr(dvar, f32, dv, "dvar"), _mem_ptr(vmean, f32, summ, "vmean"),
        _ptr(sel, i32, (*units, params.budget_blocks), "sel"), _ptr(n_sel, i32, units, "n_sel"),
        _ptr(blk_logit, f32, (*units, dims.group, dims.xcap), "blk_logit"),
        _ptr(scores, f32, (*units, dims.xcap), "scores", nullable=True), _ptr(out, f32, qs, "out"),
        _ptr(lse, f32, qs[:2], "lse", nullable=True), ws, ws_bytes, _stream(stream))
    _check(st, "compkv_decode_step")


def compkv_decode_step_noalloc(dims, params: CompkvSelectParams, q, k_cache, v_cache, k_new, v_new, seq_lens,
                               kmean, dvar, vmean, sel, n_sel, blk_logit, scores, out, lse=None, stream=None):
    """compkv_decode_step without a workspace: the library's fixed per-GPU scratch is used instead
    (nothing is allocated; overlapping calls on one GPU race)."""
    cache, summ, dv, qs = _shapes(dims)
    bf, f32, i32 = torch.bfloat16, torch.float32, torch.int32
    units = (dims.batch, dims.n_kv_heads)
    new = (*units, dims.head_dim)
    if (k_new is None) != (v_new is None):
        raise CompkvError("k_new and v_new must be given together")
    st = library().compkv_decode_step_noalloc(
        ctypes.byref(dims), ctypes.byref(params), _ptr(q, bf, qs, "q"), _kv_ptr(k_cache, cache, "k_cache"),
        _kv_ptr(v_cache, cache, "v_cache"), _ptr(k_new, bf, new, "k_new", nullable=True),
        _ptr(v_new, bf, new, "v_new", nullable=True), _ptr(seq_lens, i32, (dims.batch,), "seq_lens"),
        _mem_ptr(kmean, f32, summ, "kmean"), _mem_ptr(dvar, f32, dv, "dvar"), _mem_ptr(vmean, f32, summ, "vmean"),
        _ptr(sel, i32, (*units, params.budget_blocks), "sel"), _ptr(n_sel, i32, units, "n_sel"),
        _ptr(blk_logit, f32, (*units, dims.group, dims.xcap), "blk_logit"),
        _ptr(scores, f32, (*units, dims.xcap), "scores", nullable=True), _ptr(out, f32, qs, "out"),
        _ptr(lse, f32, qs[:2], "lse", nullable=True), _stream(stream))
    _check(st, "compkv_decode_step_noalloc")


def compkv_decode_step_noalloc_limit() -> int:
    return int(library().compkv_decode_step_noalloc_limit())


def compkv_phase_trace_set(chunk_records=None, fused_records=None) -> None:
    """Phase-trace records of the fused step's two launches (int64 device tensors of at least 16 words per
    workgroup), or None for both to stop tracing. Raises on a library built without the trace."""
    ptrs = []
    for t_, name in ((chunk_records, "chunk_records"), (fused_records, "fused_records")):
        if t_ is None:
            ptrs.append(None)
            continue
        if t_.dtype != torch.int64 or not t_.is_cuda or not t_.is_contiguous():
            raise CompkvError(f"{name} must be a contiguous int64 device tensor")
        ptrs.append(ctypes.c_void_p(t_.data_ptr()))
    _check(library().compkv_phase_trace_set(*ptrs), "compkv_phase_trace_set")


def default_scale(head_dim: int) -> float:
    return 1.0 / math.sqrt(head_dim)
