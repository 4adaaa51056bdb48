"""MI355X-native CompKV decode-step attention.

The compute lives in ``libcompkv.so`` (hand-written HIP for gfx950, C ABI in ``include/compkv.h``).
This package is a thin ctypes binding with the same function names: it checks tensor dtypes, shapes
and devices, passes raw device pointers and the current HIP stream, and raises on a non-zero status.
PyTorch only provides device memory and streams. There is no fallback: if the library is not built,
every call raises.
"""
from .binding import (  # noqa: F401
    COMPKV_COMP_DROP,
    COMPKV_COMP_MEAN,
    COMPKV_GROUPS_INTERLEAVED,
    COMPKV_GROUPS_ROTATE_HALF,
    COMPKV_SELECT_AUTO,
    COMPKV_SELECT_CHUNKED,
    COMPKV_SELECT_CHUNKED_EXACT,
    COMPKV_SCORE_COMPKV,
    COMPKV_SCORE_FIRST_ORDER,
    COMPKV_SCORE_MASS,
    COMPKV_SELECT_ONE_GROUP,
    COMPKV_SELECT_STREAM,
    COMPKV_WS_ALL,
    COMPKV_WS_DECODE_STEP,
    COMPKV_WS_DENSE_DECODE,
    COMPKV_WS_SCORE_SELECT,
    COMPKV_WS_SPARSE_DECODE,
    CompkvDims,
    CompkvError,
    CompkvSelectParams,
    Summaries,
    alloc_summaries,
    alloc_workspace,
    compkv_append_stats,
    compkv_build_stats,
    compkv_decode_step,
    compkv_decode_step_noalloc,
    compkv_decode_step_noalloc_limit,
    compkv_phase_trace_set,
    compkv_decode_step_path,
    compkv_dense_decode,
    compkv_score_select,
    compkv_sparse_decode,
    compkv_status_string,
    compkv_version,
    compkv_workspace_bytes,
    exported_symbols,
    library,
    make_dims,
)
