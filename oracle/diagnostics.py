"""Exact fp64 quantities that need every key (test infrastructure only).

The method's hot path only sees block summaries. These NumPy diagnostics compute what the paper's
analysis is stated in terms of -- exact logits, block weights Z, masses p, logit variances sigma^2,
residuals rho, the selection loss in its three forms, the Drop comparison and the token-level
compensated distribution -- so that tests can pin the oracle against the paper's identities.
All functions work on one unit: G query heads sharing one KV head.
"""
from __future__ import annotations

import numpy as np

from workloads import bf16_bits_to_f32


def _f(bits) -> np.ndarray:
    return bf16_bits_to_f32(np.asarray(bits, dtype=np.uint16)).astype(np.float64)


def _lse(x: np.ndarray, axis=-1) -> np.ndarray:
    m = np.max(x, axis=axis, keepdims=True)
    return (m + np.log(np.sum(np.exp(x - m), axis=axis, keepdims=True))).squeeze(axis)


def exact_logits(q_bits, K_bits, n: int, scale: float) -> np.ndarray:
    """z[g][j] = s q_g . k_j for the first n tokens (Section 3.1)."""
    return float(scale) * (_f(q_bits) @ _f(K_bits)[:n].T)


def block_ranges(n: int, B: int):
    return [(lo, min(lo + B, n)) for lo in range(0, n, B)]


def block_exact(z: np.ndarray, n: int, B: int) -> dict:
    """Exact per-block quantities of Section 3.2 (Eq. compkv-mass-variance) and Appendix B.1.

    logZ[g][b] = log sum_{j in b} e^{z}, zbar = block-mean logit, sig2 = population variance of the
    block's logits, p = Z / sum_c Z_c, ratio = |b| e^{zbar} / Z, rho = p (1 - ratio).
    """
    G = z.shape[0]
    rng = block_ranges(n, B)
    X = len(rng)
    nb = np.array([hi - lo for lo, hi in rng], dtype=np.float64)
    logZ = np.empty((G, X))
    zbar = np.empty((G, X))
    sig2 = np.empty((G, X))
    for b, (lo, hi) in enumerate(rng):
        zb = z[:, lo:hi]
        logZ[:, b] = _lse(zb, axis=1)
        zbar[:, b] = zb.mean(axis=1)
        sig2[:, b] = ((zb - zbar[:, b:b + 1]) ** 2).mean(axis=1)
    logD = _lse(logZ, axis=1)
    p = np.exp(logZ - logD[:, None])
    ratio = np.exp(np.log(nb)[None, :] + zbar - logZ)
    rho = p * (1.0 - ratio)
    return dict(logZ=logZ, zbar=zbar, sig2=sig2, nb=nb, logD=logD, p=p, ratio=ratio, rho=rho)


def _unselected(X: int, sel) -> np.ndarray:
    mask = np.ones(X, dtype=bool)
    mask[np.asarray(sel, dtype=np.int64)] = False
    return mask


def loss_log_partition(bx: dict, sel) -> float:
    """L(S) = sum_g log(D_g / Dhat_g(S)) (Eq. mean-residual-objective, first form; Appendix A.1)."""
    out = ~_unselected(bx["p"].shape[1], sel)
    log_mean_w = np.log(bx["nb"])[None, :] + bx["zbar"]
    terms = np.where(out[None, :], bx["logZ"], log_mean_w)
    return float(np.sum(bx["logD"] - _lse(terms, axis=1)))


def loss_residual(bx: dict, sel) -> float:
    """L(S) = -sum_g log(1 - R_g(S)), R_g = sum over omitted blocks of rho (second form)."""
    om = _unselected(bx["p"].shape[1], sel)
    R = np.sum(bx["rho"][:, om], axis=1)
    return float(-np.sum(np.log1p(-R)))


def loss_second_order(bx: dict, sel) -> float:
    """Leading term 1/2 sum_g sum_{b not in S} p sigma^2 (Eq. mean-residual-approximation)."""
    om = _unselected(bx["p"].shape[1], sel)
    return float(0.5 * np.sum(bx["p"][:, om] * bx["sig2"][:, om]))


def drop_kl(bx: dict, sel) -> float:
    """sum_g KL(P^Drop_g || P_g) = -sum_g log sum_{b in S} p (Eq. app-drop-kl)."""
    keep = ~_unselected(bx["p"].shape[1], sel)
    return float(-np.sum(np.log(np.sum(bx["p"][:, keep], axis=1))))


def compensated_token_logits(z: np.ndarray, n: int, B: int, sel) -> np.ndarray:
    """zhat[g][j]: exact logit in selected blocks, block-mean logit elsewhere (Section 3.1)."""
    zhat = z[:, :n].copy()
    chosen = set(int(s) for s in np.asarray(sel).ravel())
    for b, (lo, hi) in enumerate(block_ranges(n, B)):
        if b not in chosen:
            zhat[:, lo:hi] = z[:, lo:hi].mean(axis=1, keepdims=True)
    return zhat


def token_kl_compensated(z: np.ndarray, n: int, B: int, sel) -> float:
    """Brute-force sum_g KL(Phat_g(S) || P_g) over individual tokens (objective eq-gqa-exact-kl)."""
    zhat = compensated_token_logits(z, n, B, sel)
    logP = z[:, :n] - _lse(z[:, :n], axis=1)[:, None]
    logPh = zhat - _lse(zhat, axis=1)[:, None]
    return float(np.sum(np.exp(logPh) * (logPh - logP)))


def token_kl_drop(z: np.ndarray, n: int, B: int, sel) -> float:
    """Brute-force sum_g KL(P^Drop_g(S) || P_g): softmax restricted to the selected tokens."""
    keep = np.zeros(n, dtype=bool)
    for b in np.asarray(sel).ravel():
        lo, hi = block_ranges(n, B)[int(b)]
        keep[lo:hi] = True
    logP = z[:, :n] - _lse(z[:, :n], axis=1)[:, None]
    zs = z[:, :n][:, keep]
    logPd = zs - _lse(zs, axis=1)[:, None]
    return float(np.sum(np.exp(logPd) * (logPd - logP[:, keep])))


def compensated_output_tokens(q_bits, K_bits, V_bits, n: int, B: int, scale: float, sel):
    """Phat_g(S) V computed token by token (each omitted token carries its block-mean logit)."""
    z = exact_logits(q_bits, K_bits, n, scale)
    zhat = compensated_token_logits(z, n, B, sel)
    w = np.exp(zhat - zhat.max(axis=1, keepdims=True))
    out = (w @ _f(V_bits)[:n]) / w.sum(axis=1, keepdims=True)
    lse = _lse(zhat, axis=1)
    return out, lse


def rope_pair_groups(d: int, r: int, layout: int = 0) -> list[list[int]]:
    """Coordinate groups of Appendix A.4, built from the list of RoPE frequency pairs.

    layout 0 pairs coordinate f with f + d/2 (rotate-half), layout 1 pairs 2f with 2f + 1; the d/2
    pairs are cut into r equal consecutive groups, and r = d puts each coordinate alone.
    """
    if r == d:
        return [[i] for i in range(d)]
    pairs = [(f, f + d // 2) for f in range(d // 2)] if layout == 0 else [(2 * f, 2 * f + 1) for f in range(d // 2)]
    per = (d // 2) // r
    assert per * r == d // 2, "r must divide d/2 or equal d"
    return [sorted(c for pr in pairs[t * per:(t + 1) * per] for c in pr) for t in range(r)]


def block_key_covariance(K_bits, n: int, B: int) -> np.ndarray:
    """Sigma_k,b [X][d][d]: population covariance of the block's keys (Eq. app-key-covariance)."""
    K = _f(K_bits)[:n]
    out = []
    for lo, hi in block_ranges(n, B):
        dev = K[lo:hi] - K[lo:hi].mean(axis=0, keepdims=True)
        out.append(dev.T @ dev / (hi - lo))
    return np.stack(out)


def sig2_from_covariance(q_bits, cov: np.ndarray, groups, scale: float, diagonal: bool = True):
    """Variance of the logits along the query: s^2 q Sigma q^T, or with Sigma replaced by the
    group-averaged diagonal (Appendix A.4) when ``diagonal``."""
    q = _f(q_bits)
    if not diagonal:
        return float(scale) ** 2 * np.einsum("gi,bij,gj->gb", q, cov, q)
    diag = np.diagonal(cov, axis1=1, axis2=2)  # [X][d]
    approx = np.zeros_like(diag)
    for grp in groups:
        approx[:, grp] = diag[:, grp].mean(axis=1, keepdims=True)
    return float(scale) ** 2 * (q ** 2) @ approx.T


def spearman(a, b) -> float:
    """Spearman rank correlation (average ranks for ties)."""
    def ranks(x):
        x = np.asarray(x, dtype=np.float64)
        order = np.argsort(x, kind="mergesort")
        r = np.empty(len(x))
        r[order] = np.arange(len(x), dtype=np.float64)
        for v in np.unique(x):
            idx = np.where(x == v)[0]
            if len(idx) > 1:
                r[idx] = r[idx].mean()
        return r
    ra, rb = ranks(a), ranks(b)
    ra -= ra.mean()
    rb -= rb.mean()
    den = np.sqrt(np.sum(ra * ra) * np.sum(rb * rb))
    return float(np.sum(ra * rb) / den) if den > 0 else 0.0


def capture(T, chosen, reference) -> float:
    """Residual capture of Appendix B.2: sum of T over the chosen blocks / sum over the reference blocks
    (the exact-residual selection)."""
    T = np.asarray(T, dtype=np.float64)
    den = float(np.sum(T[np.asarray(reference, dtype=np.int64)]))
    return float(np.sum(T[np.asarray(chosen, dtype=np.int64)])) / den if den > 0 else 1.0


def top_blocks(score, k: int, exclude=()) -> np.ndarray:
    """The k blocks of largest score outside `exclude` (ties to the lower id), ascending."""
    score = np.asarray(score, dtype=np.float64)
    skip = set(int(b) for b in exclude)
    cand = [b for b in range(len(score)) if b not in skip]
    cand.sort(key=lambda b: (-score[b], b))
    return np.sort(np.array(cand[:k], dtype=np.int64))


def output_rel_l2(out, ref) -> np.ndarray:
    """Per-head relative L2 error ||out_h - ref_h|| / ||ref_h|| (Eq. residual-diagnostic-errors)."""
    out, ref = np.asarray(out, np.float64), np.asarray(ref, np.float64)
    return np.linalg.norm(out - ref, axis=-1) / np.linalg.norm(ref, axis=-1)

