"""Plain fp64 CPU oracle of CompKV's decode-step attention (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and the bench's ``cpu_baseline`` leg may import this
package. It wraps the C library built from ``compkv_oracle.c`` (per-unit functions, fp64) and, in
``diagnostics``, NumPy fp64 quantities that need every key (exact block masses, logit variances,
selection losses), which the method itself never computes on its hot path.

All per-unit inputs are bf16 bit patterns (uint16) as drawn by the ``workloads`` generators.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import build as _build

ROTATE_HALF = 0
INTERLEAVED = 1

_lib = None


def lib():
    """Load (building on first use if nothing is built yet) the C oracle."""
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        L = ctypes.CDLL(_build.LIB)
        u16p = np.ctypeslib.ndpointer(np.uint16, flags="C_CONTIGUOUS")
        f64p = np.ctypeslib.ndpointer(np.float64, flags="C_CONTIGUOUS")
        i32p = np.ctypeslib.ndpointer(np.int32, flags="C_CONTIGUOUS")
        c_int, c_double = ctypes.c_int, ctypes.c_double
        L.orc_num_blocks.argtypes = [c_int, c_int]
        L.orc_block_len.argtypes = [c_int, c_int, c_int]
        L.orc_group_of.argtypes = [c_int, c_int, c_int, c_int]
        L.orc_block_stats.argtypes = [u16p, u16p, c_int, c_int, c_int, c_int, c_int, f64p, f64p, f64p]
        L.orc_block_scores.argtypes = [u16p, c_int, f64p, f64p, c_int, c_int, c_int, c_int, c_int,
                                       c_double, c_int, f64p, f64p, f64p, f64p]
        L.orc_select.argtypes = [f64p, c_int, c_int, c_int, c_int, i32p]
        L.orc_sparse_decode.argtypes = [u16p, c_int, u16p, u16p, f64p, f64p, c_int, c_int, c_int,
                                        c_double, i32p, c_int, c_int, f64p, f64p]
        L.orc_dense_decode.argtypes = [u16p, c_int, u16p, u16p, c_int, c_int, c_double, f64p, f64p]
        _lib = L
    return _lib


class OracleError(ValueError):
    pass


def _u16(a):
    return np.ascontiguousarray(a, dtype=np.uint16)


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def num_blocks(n: int, B: int) -> int:
    return lib().orc_num_blocks(n, B)


def block_len(n: int, B: int, b: int) -> int:
    return lib().orc_block_len(n, B, b)


def group_of(i: int, d: int, r: int, layout: int = ROTATE_HALF) -> int:
    return lib().orc_group_of(i, d, r, layout)


def block_stats(K, V, n: int, B: int, r: int, layout: int = ROTATE_HALF):
    """Per-block (kmean [X][d], dvar [X][r], vmean [X][d]) of the first n rows of one unit."""
    K, V = _u16(K), _u16(V)
    d = K.shape[-1]
    X = num_blocks(n, B)
    kmean = np.zeros((max(X, 1), d))
    vmean = np.zeros((max(X, 1), d))
    dvar = np.zeros((max(X, 1), r))
    if lib().orc_block_stats(K, V, n, d, B, r, layout, kmean, dvar, vmean) != 0:
        raise OracleError(f"invalid (d={d}, r={r}, layout={layout}, B={B})")
    return kmean[:X], dvar[:X], vmean[:X]


# score kinds (Section 5.4 ablations): the CompKV score, the mass-only score sum_g phat, and the
# first-order score whose mass estimate uses the mean-key logits alone
SCORE_COMPKV = 0
SCORE_MASS = 1
SCORE_FIRST_ORDER = 2


def block_scores(q, kmean, dvar, n: int, B: int, r: int, scale: float, layout: int = ROTATE_HALF,
                 kind: int = SCORE_COMPKV):
    """dict(zbar, sig2, phat [G][X], score [X]) for the G query heads q ([G][d] bf16 bits)."""
    q = _u16(q)
    G, d = q.shape
    X = num_blocks(n, B)
    km = np.zeros((max(X, 1), d))
    dv = np.zeros((max(X, 1), r))
    km[:X], dv[:X] = kmean[:X], dvar[:X]
    zbar, sig2, phat = (np.zeros((G, max(X, 1))) for _ in range(3))
    score = np.zeros(max(X, 1))
    rc = lib().orc_block_scores(q, G, km, dv, n, d, B, r, layout, float(scale), int(kind), zbar, sig2, phat,
                                score)
    if rc != 0:
        raise OracleError(f"invalid (d={d}, r={r}, layout={layout}, B={B}, kind={kind})")
    return dict(zbar=zbar[:, :X], sig2=sig2[:, :X], phat=phat[:, :X], score=score[:X])


def select(score, K: int, n_sink: int = 1, n_recent: int = 2) -> np.ndarray:
    """Ascending selected block ids; raises OracleError when K is below the mandatory set."""
    score = _f64(score)
    X = score.shape[0]
    sel = np.zeros(max(min(K, X), 1) + X, dtype=np.int32)
    cnt = lib().orc_select(score if X else np.zeros(1), X, K, n_sink, n_recent, sel)
    if cnt < 0:
        raise OracleError(f"budget {K} is smaller than the mandatory set")
    return sel[:cnt].copy()


def sparse_decode(q, K, V, kmean, vmean, n: int, B: int, scale: float, sel, compensate: bool = True):
    """Compensated output (out [G][d], lse [G]) for the selected ids ``sel``; with compensate=False the
    Drop output (the selected tokens alone, renormalized)."""
    q, K, V = _u16(q), _u16(K), _u16(V)
    G, d = q.shape
    X = num_blocks(n, B)
    km = np.zeros((max(X, 1), d))
    vm = np.zeros((max(X, 1), d))
    km[:X], vm[:X] = kmean[:X], vmean[:X]
    sel = np.ascontiguousarray(sel, dtype=np.int32)
    out = np.zeros((G, d))
    lse = np.zeros(G)
    rc = lib().orc_sparse_decode(q, G, K, V, km, vm, n, d, B, float(scale),
                                 sel if sel.size else np.zeros(1, np.int32), int(sel.size), int(bool(compensate)),
                                 out, lse)
    if rc != 0:
        raise OracleError("selected ids out of range or repeated")
    return out, lse


def dense_decode(q, K, V, n: int, scale: float):
    """Full attention (out [G][d], lse [G]) over the first n rows."""
    q, K, V = _u16(q), _u16(K), _u16(V)
    G, d = q.shape
    out = np.zeros((G, d))
    lse = np.zeros(G)
    lib().orc_dense_decode(q, G, K, V, n, d, float(scale), out, lse)
    return out, lse


def unit_step(q, K, V, n: int, B: int, r: int, budget: int, scale: float, layout: int = ROTATE_HALF,
              n_sink: int = 1, n_recent: int = 2, kind: int = SCORE_COMPKV, compensate: bool = True):
    """Whole decode step of one unit: stats, scores, selection and compensated output."""
    kmean, dvar, vmean = block_stats(K, V, n, B, r, layout)
    sc = block_scores(q, kmean, dvar, n, B, r, scale, layout, kind)
    sel = select(sc["score"], budget, n_sink, n_recent)
    out, lse = sparse_decode(q, K, V, kmean, vmean, n, B, scale, sel, compensate)
    return dict(kmean=kmean, dvar=dvar, vmean=vmean, sel=sel, out=out, lse=lse, **sc)
