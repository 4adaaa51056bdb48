"""Pins of the CPU oracle against facts the paper and the mathematics fix (no GPU needed).

Each test names the passage it checks. None of them re-types the oracle's formula: they use
special cases with known answers, closed forms, the paper's identities computed by brute force
over individual tokens, invariances and exhaustive search on tiny inputs.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest

import oracle
from oracle import diagnostics as dg
from workloads import bf16_bits_to_f32, f32_to_bf16_bits

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rand_unit(seed, n, d, G, spread=0.5, qscale=1.0):
    rng = np.random.default_rng(seed)
    B_cent = rng.standard_normal((n, d)).astype(np.float32)
    K = f32_to_bf16_bits(B_cent * spread + rng.standard_normal(d).astype(np.float32))
    V = f32_to_bf16_bits(rng.standard_normal((n, d)).astype(np.float32))
    q = f32_to_bf16_bits(qscale * rng.standard_normal((G, d)).astype(np.float32))
    return q, K, V


def blocky_unit(seed, n, d, G, B, qscale=1.0):
    """Keys with per-block centroids and per-block spreads, as in the synthetic workloads."""
    rng = np.random.default_rng(seed)
    X = -(-n // B)
    cent = rng.standard_normal((X, d)).astype(np.float32)
    sig = np.exp(rng.uniform(np.log(0.05), 0.0, X)).astype(np.float32)
    blk = np.arange(n) // B
    K = f32_to_bf16_bits(cent[blk] + sig[blk, None] * rng.standard_normal((n, d)).astype(np.float32))
    V = f32_to_bf16_bits(rng.standard_normal((n, d)).astype(np.float32))
    q = f32_to_bf16_bits(qscale * rng.standard_normal((G, d)).astype(np.float32))
    return q, K, V


def relerr(x, y):
    x, y = np.asarray(x, np.float64), np.asarray(y, np.float64)
    return float(np.max(np.abs(x - y)) / max(np.max(np.abs(y)), 1e-300))


# ---------------------------------------------------------------- partition and coordinate groups

def test_partition_contiguous_blocks_with_partial_tail():
    """Section 3.1: contiguous fixed-size blocks from the first token; only the last is partial."""
    for n, B in [(1, 16), (16, 16), (17, 16), (4095, 16), (100, 7), (5, 1)]:
        X = oracle.num_blocks(n, B)
        lens = [oracle.block_len(n, B, b) for b in range(X)]
        assert sum(lens) == n and all(L == B for L in lens[:-1]) and 1 <= lens[-1] <= B
    assert oracle.num_blocks(0, 16) == 0


@pytest.mark.parametrize("layout", [oracle.ROTATE_HALF, oracle.INTERLEAVED])
@pytest.mark.parametrize("d", [8, 64, 128])
def test_group_map_follows_rope_pairs(d, layout):
    """Appendix A.4: groups are r equal consecutive runs of RoPE frequency pairs (both coordinates
    of a pair together); r = d puts each coordinate alone; other r are invalid."""
    for r in range(1, d + 1):
        valid = r == d or (d // 2) % r == 0
        got = [oracle.group_of(i, d, r, layout) for i in range(d)]
        if not valid:
            assert got[0] == -1
            continue
        groups = dg.rope_pair_groups(d, r, layout)
        assert len(groups) == r and all(len(gr) == d // r for gr in groups)
        for t, gr in enumerate(groups):
            for i in gr:
                assert got[i] == t


# ---------------------------------------------------------------- statistics and scoring

def test_summary_size_matches_paper():
    """Section 4.2: 2d + r + 1 scalars per block; r = 4 is 1/32 of r = 128's variance metadata."""
    fx = json.load(open(os.path.join(GOLDEN, "summary_size.json")))
    d = fx["head_dim"]
    q, K, V = rand_unit(1, 64, d, 1)
    for case in fx["cases"]:
        km, dv, vm = oracle.block_stats(K, V, 64, 16, case["r"])
        per_block = km.shape[1] + dv.shape[1] + vm.shape[1] + 1  # + |b|
        assert per_block == case["scalars_per_block"]
    assert 4 / 128 == fx["variance_metadata_ratio_r4_over_r128"]


def test_block_size_one_degenerates():
    """B = 1: the mean key is the key, the variance is zero, every score is zero (Section 4.1), so
    the stable Top-K takes the lowest candidate ids, and p-hat is the exact softmax."""
    n, d, G, K_budget = 40, 16, 3, 9
    q, K, V = rand_unit(2, n, d, G)
    km, dv, vm = oracle.block_stats(K, V, n, 1, 4)
    assert np.array_equal(km, bf16_bits_to_f32(K).astype(np.float64))
    assert np.all(dv == 0.0)
    s = 1 / math.sqrt(d)
    sc = oracle.block_scores(q, km, dv, n, 1, 4, s)
    assert np.all(sc["score"] == 0.0)
    z = dg.exact_logits(q, K, n, s)
    p_exact = np.exp(z - z.max(axis=1, keepdims=True))
    p_exact /= p_exact.sum(axis=1, keepdims=True)
    assert relerr(sc["phat"], p_exact) < 1e-12
    sel = oracle.select(sc["score"], K_budget)
    assert list(sel) == list(range(K_budget - 2)) + [n - 2, n - 1]


@pytest.mark.parametrize("budget", [3, 5, 8])
def test_block_size_one_compensation_is_exact(budget):
    """B = 1: a pseudo-token (log 1 + mean logit, mean value) is the token itself, so the
    compensated output equals dense attention for any budget (Eq. compkv-output)."""
    n, d, G = 30, 16, 2
    q, K, V = rand_unit(3, n, d, G)
    s = 1 / math.sqrt(d)
    km, dv, vm = oracle.block_stats(K, V, n, 1, 2)
    sel = oracle.select(oracle.block_scores(q, km, dv, n, 1, 2, s)["score"], budget)
    o_sp, l_sp = oracle.sparse_decode(q, K, V, km, vm, n, 1, s, sel)
    o_de, l_de = oracle.dense_decode(q, K, V, n, s)
    assert relerr(o_sp, o_de) < 1e-12 and relerr(l_sp, l_de) < 1e-12


def test_identical_keys_in_block_make_compensation_exact():
    """Identical keys inside every block: zero variance, Z_b = |b| e^{zbar} exactly, so p-hat is the
    exact mass, the residual is zero and the output equals dense attention although the values
    differ (Eqs. compkv-mass-estimate, compkv-output; Appendix A.2)."""
    n, d, G, B = 77, 16, 4, 8
    rng = np.random.default_rng(4)
    X = -(-n // B)
    cent = rng.standard_normal((X, d)).astype(np.float32)
    K = f32_to_bf16_bits(cent[np.arange(n) // B])
    V = f32_to_bf16_bits(rng.standard_normal((n, d)).astype(np.float32))
    q = f32_to_bf16_bits(rng.standard_normal((G, d)).astype(np.float32))
    s = 1 / math.sqrt(d)
    km, dv, vm = oracle.block_stats(K, V, n, B, 4)
    assert np.all(dv == 0.0)
    sc = oracle.block_scores(q, km, dv, n, B, 4, s)
    bx = dg.block_exact(dg.exact_logits(q, K, n, s), n, B)
    assert relerr(sc["phat"], bx["p"]) < 1e-12
    assert np.allclose(bx["rho"], 0.0, atol=1e-14)
    o_de, l_de = oracle.dense_decode(q, K, V, n, s)
    for budget in (3, 4, 6):
        sel = oracle.select(sc["score"], budget)
        o_sp, l_sp = oracle.sparse_decode(q, K, V, km, vm, n, B, s, sel)
        assert relerr(o_sp, o_de) < 1e-12 and relerr(l_sp, l_de) < 1e-12


@pytest.mark.parametrize("n,B", [(64, 16), (70, 16), (33, 4)])
def test_budget_all_blocks_reproduces_dense(n, B):
    """K >= X: no block is omitted, so Eq. compkv-output is full attention."""
    d, G = 32, 4
    q, K, V = rand_unit(5, n, d, G)
    s = 1 / math.sqrt(d)
    X = oracle.num_blocks(n, B)
    km, dv, vm = oracle.block_stats(K, V, n, B, 4)
    o_de, l_de = oracle.dense_decode(q, K, V, n, s)
    for budget in (X, X + 3):
        sel = oracle.select(oracle.block_scores(q, km, dv, n, B, 4, s)["score"], budget)
        assert list(sel) == list(range(X))
        o_sp, l_sp = oracle.sparse_decode(q, K, V, km, vm, n, B, s, sel)
        assert relerr(o_sp, o_de) < 1e-12 and relerr(l_sp, l_de) < 1e-12


@pytest.mark.parametrize("layout", [oracle.ROTATE_HALF, oracle.INTERLEAVED])
@pytest.mark.parametrize("r", [1, 2, 4, 8, 32])
def test_grouped_variance_is_diagonal_projection(r, layout):
    """Appendix A.4: sigma-hat^2 is s^2 q Sigma' q^T where Sigma' is the block key covariance with
    its diagonal averaged over each coordinate group and its off-diagonal dropped; the stored
    statistic is the group mean of the diagonal (population covariance)."""
    n, d, G, B = 90, 32, 3, 16
    q, K, V = blocky_unit(6, n, d, G, B)
    s = 1 / math.sqrt(d)
    km, dv, vm = oracle.block_stats(K, V, n, B, r, layout)
    cov = dg.block_key_covariance(K, n, B)
    groups = dg.rope_pair_groups(d, r, layout)
    diag = np.diagonal(cov, axis1=1, axis2=2)
    for t, gr in enumerate(groups):
        assert relerr(dv[:, t], diag[:, gr].mean(axis=1)) < 1e-12
    sc = oracle.block_scores(q, km, dv, n, B, r, s, layout)
    assert relerr(sc["sig2"], dg.sig2_from_covariance(q, cov, groups, s)) < 1e-12


def test_per_coordinate_groups_exact_for_one_hot_query():
    """Appendix A.4 at r = d: with a one-hot query the projected variance is the exact logit
    variance of the block (no off-diagonal term survives)."""
    n, d, G, B = 64, 16, 1, 16
    _, K, V = blocky_unit(7, n, d, G, B)
    for i in (0, 5, 15):
        q = np.zeros((1, d), np.float32)
        q[0, i] = 1.5
        qb = f32_to_bf16_bits(q)
        s = 1 / math.sqrt(d)
        km, dv, vm = oracle.block_stats(K, V, n, B, d)
        sc = oracle.block_scores(qb, km, dv, n, B, d, s)
        bx = dg.block_exact(dg.exact_logits(qb, K, n, s), n, B)
        assert relerr(sc["sig2"], bx["sig2"]) < 1e-12


def test_plus_minus_block_closed_form():
    """A block whose keys deviate by +a / -a along one coordinate: logit deviations are +-x with
    x = s q_i a, so sigma^2 = x^2, Z = |b| e^{zbar} cosh x and rho = p (1 - 1/cosh x); at r = d the
    grouped estimate recovers x^2 exactly (Appendices A.2, A.4)."""
    d, B, i, a = 8, 4, 3, 0.5
    base = np.array([1.0, -0.5, 0.25, 2.0, -1.0, 0.75, 0.125, -2.0], np.float32)
    rows = []
    for blk in range(3):
        for j in range(B):
            k = base + blk
            if blk == 1:
                k = k.copy()
                k[i] += a if j % 2 == 0 else -a
            rows.append(k)
    K = f32_to_bf16_bits(np.array(rows))
    V = f32_to_bf16_bits(np.ones((3 * B, d), np.float32))
    q = f32_to_bf16_bits(np.array([[0.5, 1.0, -1.5, 2.0, 0.25, -0.75, 1.25, 0.5]], np.float32))
    n, s = 3 * B, 1 / math.sqrt(d)
    x = s * 2.0 * a  # q_i = 2.0
    km, dv, vm = oracle.block_stats(K, V, n, B, d)
    assert dv[1, i] == pytest.approx(a * a, rel=1e-15) and np.sum(dv) == pytest.approx(a * a, rel=1e-15)
    sc = oracle.block_scores(q, km, dv, n, B, d, s)
    assert sc["sig2"][0, 1] == pytest.approx(x * x, rel=1e-13)
    assert sc["sig2"][0, 0] == 0.0 and sc["sig2"][0, 2] == 0.0
    bx = dg.block_exact(dg.exact_logits(q, K, n, s), n, B)
    assert math.exp(bx["logZ"][0, 1]) == pytest.approx(B * math.exp(bx["zbar"][0, 1]) * math.cosh(x), rel=1e-13)
    assert bx["rho"][0, 1] == pytest.approx(bx["p"][0, 1] * (1 - 1 / math.cosh(x)), rel=1e-11)


def test_mass_estimate_normalized_per_head_over_all_blocks():
    """Eq. compkv-mass-estimate: p-hat sums to one per query head over every block (Appendix A.4)."""
    n, d, G, B = 200, 32, 4, 16
    q, K, V = blocky_unit(8, n, d, G, B, qscale=2.0)
    km, dv, vm = oracle.block_stats(K, V, n, B, 4)
    sc = oracle.block_scores(q, km, dv, n, B, 4, 1 / math.sqrt(d))
    assert np.allclose(sc["phat"].sum(axis=1), 1.0, atol=1e-14)
    assert np.all(sc["score"] >= 0)


def test_mass_estimate_second_order_taylor_regime():
    """Eq. compkv-log-partition: log Z = log|b| + zbar + sigma^2/2 + O(sigma^3). With r = d and a
    one-hot query the oracle's sigma-hat^2 is exact, so its log-mass error must shrink like the cube
    of the key spread (a dropped 1/2 or log|b| would leave a quadratic or constant error)."""
    n, d, B = 96, 16, 16
    rng = np.random.default_rng(9)
    cent = rng.standard_normal((n // B, d))
    u = rng.standard_normal((n, d))
    q = np.zeros((1, d), np.float32)
    q[0, 2] = 4.0
    qb = f32_to_bf16_bits(q)
    s = 1 / math.sqrt(d)
    errs = []
    for eps in (0.08, 0.04, 0.02):
        # keys in float64 exact for bf16 are needed: scale into bf16 and read back
        K = f32_to_bf16_bits((cent[np.arange(n) // B] + eps * u).astype(np.float32))
        km, dv, vm = oracle.block_stats(K, K, n, B, d)
        sc = oracle.block_scores(qb, km, dv, n, B, d, s)
        bx = dg.block_exact(dg.exact_logits(qb, K, n, s), n, B)
        errs.append(np.max(np.abs(np.log(sc["phat"]) - np.log(bx["p"]))))
    assert errs[0] / errs[1] > 5.0 and errs[1] / errs[2] > 5.0, errs


def test_residual_expansion_leading_term():
    """Eq. mean-residual-expansion: rho = p (sigma^2/2 + O(sigma^3)), so rho / (p sigma^2 / 2) -> 1
    with a gap that shrinks linearly in the spread (Appendix A.2)."""
    n, d, G, B = 64, 16, 2, 16
    rng = np.random.default_rng(10)
    cent = rng.standard_normal((n // B, d))
    u = rng.standard_normal((n, d))
    q = f32_to_bf16_bits(2.0 * rng.standard_normal((G, d)).astype(np.float32))
    gaps = []
    for eps in (0.1, 0.05, 0.025):
        K = f32_to_bf16_bits((cent[np.arange(n) // B] + eps * u).astype(np.float32))
        bx = dg.block_exact(dg.exact_logits(q, K, n, 0.25), n, B)
        ratio = bx["rho"] / (bx["p"] * bx["sig2"] / 2)
        gaps.append(np.max(np.abs(ratio - 1)))
    assert gaps[0] > gaps[1] > gaps[2] and gaps[2] < 0.05, gaps


# ---------------------------------------------------------------- selection loss identities

@pytest.mark.parametrize("seed", [11, 12, 13])
def test_kl_log_partition_residual_identity(seed):
    """Appendix A.1: the token-level KL(P-hat || P) summed over heads equals the log-partition gap
    and the residual form, for any selected set."""
    n, d, G, B = 60, 16, 3, 8
    q, K, V = blocky_unit(seed, n, d, G, B, qscale=3.0)
    s = 1 / math.sqrt(d)
    z = dg.exact_logits(q, K, n, s)
    bx = dg.block_exact(z, n, B)
    rng = np.random.default_rng(seed)
    X = bx["p"].shape[1]
    for _ in range(5):
        sel = np.sort(rng.choice(X, size=rng.integers(1, X), replace=False))
        kl = dg.token_kl_compensated(z, n, B, sel)
        assert kl == pytest.approx(dg.loss_log_partition(bx, sel), rel=1e-9, abs=1e-14)
        assert kl == pytest.approx(dg.loss_residual(bx, sel), rel=1e-9, abs=1e-14)


@pytest.mark.parametrize("seed", [14, 15])
def test_oracle_output_is_token_level_compensated_attention(seed):
    """Eq. compkv-output is P-hat(S) V where P-hat is the softmax with each omitted token's logit
    replaced by its block-mean logit (Section 3.1); the oracle's per-block form must match the
    token-by-token computation, and the gap between dense and compensated lse is the KL loss."""
    n, d, G, B = 75, 16, 4, 8
    q, K, V = blocky_unit(seed, n, d, G, B, qscale=3.0)
    s = 1 / math.sqrt(d)
    km, dv, vm = oracle.block_stats(K, V, n, B, 4)
    z = dg.exact_logits(q, K, n, s)
    rng = np.random.default_rng(seed)
    X = oracle.num_blocks(n, B)
    _, l_de = oracle.dense_decode(q, K, V, n, s)
    for _ in range(4):
        sel = np.sort(rng.choice(X, size=rng.integers(1, X), replace=False)).astype(np.int32)
        o_sp, l_sp = oracle.sparse_decode(q, K, V, km, vm, n, B, s, sel)
        o_tk, l_tk = dg.compensated_output_tokens(q, K, V, n, B, s, sel)
        assert relerr(o_sp, o_tk) < 1e-11 and relerr(l_sp, l_tk) < 1e-12
        assert float(np.sum(l_de - l_sp)) == pytest.approx(dg.token_kl_compensated(z, n, B, sel), rel=1e-8, abs=1e-13)


@pytest.mark.parametrize("seed", [16, 17])
def test_mean_compensation_never_worse_than_drop(seed):
    """Eq. app-mean-drop-ordering: 0 <= KL(P-hat) <= KL(Drop) for a nonempty S, and the Jensen bound
    |b| e^{zbar} <= Z_b (Appendix A.5)."""
    n, d, G, B = 64, 16, 2, 8
    q, K, V = blocky_unit(seed, n, d, G, B, qscale=3.0)
    z = dg.exact_logits(q, K, n, 0.3)
    bx = dg.block_exact(z, n, B)
    assert np.all(bx["ratio"] <= 1 + 1e-12)
    rng = np.random.default_rng(seed)
    for _ in range(6):
        sel = np.sort(rng.choice(8, size=rng.integers(1, 8), replace=False))
        kc, kd = dg.token_kl_compensated(z, n, B, sel), dg.token_kl_drop(z, n, B, sel)
        assert -1e-14 <= kc <= kd + 1e-14
        assert kd == pytest.approx(dg.drop_kl(bx, sel), rel=1e-9, abs=1e-14)


def test_exact_residual_topk_is_exact_minimizer_single_head():
    """G = 1: -log(1 - R) is increasing in R and R is additive over omitted blocks (Eq.
    mean-residual-objective), so the blocks with the largest exact residual rho minimize L(S)
    exactly. Checked against every subset of size K (Appendix B.1's exact-residual selector)."""
    n, d, B = 80, 16, 8
    for seed in (18, 19, 20):
        q, K, V = blocky_unit(seed, n, d, 1, B, qscale=4.0)
        bx = dg.block_exact(dg.exact_logits(q, K, n, 0.25), n, B)
        X = bx["p"].shape[1]
        for budget in (2, 4, 6):
            best = min(dg.loss_log_partition(bx, list(c)) for c in itertools.combinations(range(X), budget))
            sel = oracle.select(bx["rho"][0], budget, n_sink=0, n_recent=0)
            assert dg.loss_log_partition(bx, sel) == pytest.approx(best, rel=1e-12, abs=1e-15)


# ---------------------------------------------------------------- selection contract

def test_budget_arithmetic_golden():
    """Appendix B.2: 512-token budget / 16-token blocks with sink + two recent blocks mandatory
    leaves 29 blocks chosen by the score."""
    fx = json.load(open(os.path.join(GOLDEN, "budget_selection.json")))
    K_blocks = fx["budget_tokens"] // fx["block_size"]
    assert K_blocks == fx["budget_blocks"]
    rng = np.random.default_rng(21)
    for X in (35, 64, 2048):
        score = rng.random(X)
        sel = oracle.select(score, K_blocks, fx["n_sink"], fx["n_recent"])
        mand = {b for b in range(X) if b < fx["n_sink"] or b >= X - fx["n_recent"]}
        assert len(sel) == fx["budget_blocks"] and mand <= set(sel.tolist())
        assert len(mand) == fx["mandatory_blocks"]
        assert len(set(sel.tolist()) - mand) == fx["scored_blocks"]


@pytest.mark.parametrize("seed", range(22, 30))
def test_selection_contract_stable_topk(seed):
    """Eq. compkv-selected-set and Appendix E.1: |S| = min(K, X), F inside S, ids ascending and unique;
    every selected candidate outranks every unselected one under (score desc, id asc)."""
    rng = np.random.default_rng(seed)
    X = int(rng.integers(1, 60))
    n_sink, n_recent = int(rng.integers(0, 3)), int(rng.integers(0, 4))
    score = np.round(rng.random(X) * 5) / 5  # many exact ties
    F = {b for b in range(X) if b < n_sink or b >= X - n_recent}
    for K in range(0, X + 3):
        if K < len(F) and K < X:
            with pytest.raises(oracle.OracleError):
                oracle.select(score, K, n_sink, n_recent)
            continue
        sel = oracle.select(score, K, n_sink, n_recent).tolist()
        assert len(sel) == min(K, X) and sel == sorted(set(sel)) and F <= set(sel)
        chosen = set(sel) - F
        rest = set(range(X)) - set(sel)
        for a in chosen:
            for b in rest:
                assert score[a] > score[b] or (score[a] == score[b] and a < b)


def test_mandatory_overlap_counted_once():
    """Section 4.2: sink and recent blocks overlap when X <= 3; the overlap is counted once."""
    for X in (1, 2, 3):
        sel = oracle.select(np.zeros(X), 3)
        assert list(sel) == list(range(X))
    assert list(oracle.select(np.array([0.0, 5.0, 1.0, 0.0]), 3)) == [0, 2, 3]


# ---------------------------------------------------------------- invariances

def test_key_shift_and_token_permutation_invariance():
    """Adding one vector to every key shifts all logits of a head by a constant: variances, scores,
    the selection and the output are unchanged, the mean key shifts (softmax shift invariance,
    Eqs. compkv-mass-estimate, compkv-output). Permuting tokens inside a block changes nothing."""
    n, d, G, B = 64, 16, 4, 8
    rng = np.random.default_rng(31)
    Kq = rng.integers(-60, 60, size=(n, d)) / 16.0  # multiples of 1/16: exact in bf16 after shift
    delta = rng.integers(-40, 40, size=d) / 16.0
    K = f32_to_bf16_bits(Kq.astype(np.float32))
    K2 = f32_to_bf16_bits((Kq + delta).astype(np.float32))
    V = f32_to_bf16_bits(rng.standard_normal((n, d)).astype(np.float32))
    q = f32_to_bf16_bits(rng.standard_normal((G, d)).astype(np.float32))
    s = 1 / math.sqrt(d)
    st1, st2 = oracle.block_stats(K, V, n, B, 4), oracle.block_stats(K2, V, n, B, 4)
    assert relerr(st2[0], st1[0] + delta) < 1e-12 and relerr(st2[1], st1[1]) < 1e-12
    sc1 = oracle.block_scores(q, st1[0], st1[1], n, B, 4, s)
    sc2 = oracle.block_scores(q, st2[0], st2[1], n, B, 4, s)
    assert relerr(sc2["score"], sc1["score"]) < 1e-10
    sel1, sel2 = oracle.select(sc1["score"], 5), oracle.select(sc2["score"], 5)
    assert list(sel1) == list(sel2)
    o1, _ = oracle.sparse_decode(q, K, V, st1[0], st1[2], n, B, s, sel1)
    o2, _ = oracle.sparse_decode(q, K2, V, st2[0], st2[2], n, B, s, sel2)
    assert relerr(o2, o1) < 1e-10
    perm = np.concatenate([lo + rng.permutation(hi - lo) for lo, hi in dg.block_ranges(n, B)])
    st3 = oracle.block_stats(K[perm], V[perm], n, B, 4)
    assert all(relerr(a, b) < 1e-12 for a, b in zip(st3, st1))
    o3, _ = oracle.sparse_decode(q, K[perm], V[perm], st3[0], st3[2], n, B, s, sel1)
    assert relerr(o3, o1) < 1e-12


def test_value_scaling_is_linear():
    """Eq. compkv-output is linear in the values: scaling V by 2 (exact in bf16) doubles the output."""
    n, d, G, B = 48, 16, 2, 8
    q, K, V = blocky_unit(32, n, d, G, B)
    V2 = f32_to_bf16_bits(2 * bf16_bits_to_f32(V))
    s = 1 / math.sqrt(d)
    km, dv, vm = oracle.block_stats(K, V, n, B, 4)
    _, _, vm2 = oracle.block_stats(K, V2, n, B, 4)
    sel = oracle.select(oracle.block_scores(q, km, dv, n, B, 4, s)["score"], 3)
    o1, l1 = oracle.sparse_decode(q, K, V, km, vm, n, B, s, sel)
    o2, l2 = oracle.sparse_decode(q, K, V2, km, vm2, n, B, s, sel)
    assert relerr(o2, 2 * o1) < 1e-14 and relerr(l2, l1) < 1e-14


def test_completed_blocks_unchanged_by_appends():
    """Appendix E.1: appending tokens changes only the active block's summary."""
    n, d, B = 70, 16, 16
    q, K, V = rand_unit(33, n + 20, d, 1)
    base = oracle.block_stats(K, V, n, B, 4)
    for extra in (1, 5, 10, 20):
        grown = oracle.block_stats(K, V, n + extra, B, 4)
        for a, b in zip(base, grown):
            assert np.array_equal(a[: n // B], b[: n // B])


# ---------------------------------------------------------------- ablation variants (Section 5.4, App. A.5)

def test_mass_only_score_block_size_one_is_exact_mass():
    """B = 1: sigma-hat^2 = 0, so the second-order mass estimate is the exact softmax mass of each token
    and the mass-only score is sum_g p_{g,b}; its scores sum to G over the blocks."""
    n, d, G = 40, 16, 3
    q, K, V = rand_unit(31, n, d, G, qscale=2.0)
    s = 1 / math.sqrt(d)
    km, dv, vm = oracle.block_stats(K, V, n, 1, 4)
    sc = oracle.block_scores(q, km, dv, n, 1, 4, s, kind=oracle.SCORE_MASS)
    z = dg.exact_logits(q, K, n, s)
    p = np.exp(z - z.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    assert np.allclose(sc["score"], p.sum(axis=0), rtol=1e-12, atol=1e-15)
    assert sc["score"].sum() == pytest.approx(G, rel=1e-13)


def test_first_order_vs_second_order_mass_on_plus_minus_block():
    """Three blocks with identical keys inside blocks 0 and 2 and a +-a block 1: the first-order
    estimate weighs block 1 by |b| e^{zbar} alone, the second-order one by |b| e^{zbar + x^2/2}, so the
    ratio of their block-1-to-block-0 odds is e^{x^2/2} (Section 5.4; a dropped 1/2 fails). With no
    within-block spread (blocks 0 and 2) both equal the exact mass ratios."""
    d, B, i, a = 8, 4, 3, 0.5
    base = np.array([1.0, -0.5, 0.25, 2.0, -1.0, 0.75, 0.125, -2.0], np.float32)
    rows = []
    for blk in range(3):
        for j in range(B):
            k = (base + blk).copy()
            if blk == 1:
                k[i] += a if j % 2 == 0 else -a
            rows.append(k)
    K = f32_to_bf16_bits(np.array(rows))
    V = f32_to_bf16_bits(np.ones((3 * B, d), np.float32))
    q = f32_to_bf16_bits(np.array([[0.5, 1.0, -1.5, 2.0, 0.25, -0.75, 1.25, 0.5]], np.float32))
    n, s = 3 * B, 1 / math.sqrt(d)
    x = s * 2.0 * a
    km, dv, vm = oracle.block_stats(K, V, n, B, d)
    p2 = oracle.block_scores(q, km, dv, n, B, d, s)["phat"][0]
    f = oracle.block_scores(q, km, dv, n, B, d, s, kind=oracle.SCORE_FIRST_ORDER)
    p1 = f["phat"][0]
    assert (p2[1] / p2[0]) / (p1[1] / p1[0]) == pytest.approx(math.exp(x * x / 2), rel=1e-12)
    bx = dg.block_exact(dg.exact_logits(q, K, n, s), n, B)
    assert p1[2] / p1[0] == pytest.approx(bx["p"][0, 2] / bx["p"][0, 0], rel=1e-12)
    # first-order score = p-hat^(1) sigma-hat^2: only the spread block scores
    assert f["score"][0] == 0.0 and f["score"][2] == 0.0
    assert f["score"][1] == pytest.approx(p1[1] * x * x, rel=1e-12)


def test_first_order_equals_exact_mass_for_identical_keys():
    """Identical keys within every block: Z_b = |b| e^{zbar_b} exactly, so both mass estimates equal the
    exact block masses and every score kind that carries sigma-hat^2 is zero."""
    n, d, G, B = 96, 16, 2, 8
    rng = np.random.default_rng(5)
    X = n // B
    K = f32_to_bf16_bits(np.repeat(rng.standard_normal((X, d)).astype(np.float32), B, axis=0))
    V = f32_to_bf16_bits(rng.standard_normal((n, d)).astype(np.float32))
    q = f32_to_bf16_bits(2 * rng.standard_normal((G, d)).astype(np.float32))
    s = 1 / math.sqrt(d)
    km, dv, vm = oracle.block_stats(K, V, n, B, 4)
    bx = dg.block_exact(dg.exact_logits(q, K, n, s), n, B)
    for kind in (oracle.SCORE_COMPKV, oracle.SCORE_FIRST_ORDER):
        sc = oracle.block_scores(q, km, dv, n, B, 4, s, kind=kind)
        assert np.allclose(sc["phat"], bx["p"], rtol=1e-11)
        assert np.all(sc["score"] == 0.0)
    mass = oracle.block_scores(q, km, dv, n, B, 4, s, kind=oracle.SCORE_MASS)["score"]
    assert np.allclose(mass, bx["p"].sum(axis=0), rtol=1e-11)


def test_drop_decode_is_renormalized_attention_over_selected_tokens():
    """Drop (Appendix A.5): softmax over the selected tokens only, written out with NumPy; every block
    selected gives dense attention; lse_dense - lse_drop = -log sum_{b in S} p_b (Eq. app-drop-kl);
    and lse_drop <= lse_mean <= lse_dense (Eq. app-mean-drop-ordering), strict when a block is omitted."""
    n, d, G, B = 70, 16, 3, 8
    q, K, V = blocky_unit(12, n, d, G, B, qscale=3.0)
    s = 0.3
    X = -(-n // B)
    km, dv, vm = oracle.block_stats(K, V, n, B, 4)
    z = dg.exact_logits(q, K, n, s)
    bx = dg.block_exact(z, n, B)
    Vf = bf16_bits_to_f32(V).astype(np.float64)
    od, ld = oracle.dense_decode(q, K, V, n, s)
    rng = np.random.default_rng(3)
    for _ in range(5):
        sel = np.sort(rng.choice(X, size=rng.integers(1, X), replace=False)).astype(np.int32)
        o, l = oracle.sparse_decode(q, K, V, km, vm, n, B, s, sel, compensate=False)
        keep = np.concatenate([np.arange(b * B, min(b * B + B, n)) for b in sel])
        zs = z[:, keep]
        w = np.exp(zs - zs.max(axis=1, keepdims=True))
        ref = (w @ Vf[keep]) / w.sum(axis=1, keepdims=True)
        assert relerr(o, ref) < 1e-12
        assert np.allclose(ld - l, -np.log(bx["p"][:, sel].sum(axis=1)), rtol=1e-10, atol=1e-13)
        om, lm = oracle.sparse_decode(q, K, V, km, vm, n, B, s, sel)
        assert np.all(l < lm) and np.all(lm < ld + 1e-12)
    o, l = oracle.sparse_decode(q, K, V, km, vm, n, B, s, np.arange(X, dtype=np.int32), compensate=False)
    assert relerr(o, od) < 1e-12 and np.allclose(l, ld, rtol=1e-13)
    # nothing selected: no term at all
    o, l = oracle.sparse_decode(q, K, V, km, vm, n, B, s, np.zeros(0, np.int32), compensate=False)
    assert np.all(o == 0.0) and np.all(np.isinf(l)) and np.all(l < 0)


def test_llama_workload_offset_blocks_mass_vs_compkv():
    """The Llama-shaped 32K layer gives 5% of its blocks a shared key offset along the unit's mean query
    with a small spread: high attention mass, little within-block variation, so Mean compensation
    already reconstructs them well (Sections 3.2 and 4.1). The mass-only score selects every one of
    them; the CompKV score (and its first-order variant) spends no exact read on them."""
    from workloads import WORKLOADS, gen_queries, gen_unit_kv, offset_blocks

    w = WORKLOADS["llama8b_32k"]
    n, B, G = w.context, w.block_size, w.group
    K, V = gen_unit_kv(w, 0, 0, 0)
    q = gen_queries(w, 0, 0, 0)[:G]
    off = set(offset_blocks(w, 0, 0, 0).tolist())
    assert len(off) == 51
    km, dv, vm = oracle.block_stats(K, V, n, B, 4)
    picked = {}
    for kind in (oracle.SCORE_COMPKV, oracle.SCORE_MASS, oracle.SCORE_FIRST_ORDER):
        sc = oracle.block_scores(q, km, dv, n, B, 4, 1 / math.sqrt(w.head_dim), kind=kind)
        picked[kind] = len(off & set(oracle.select(sc["score"], w.budget_blocks).tolist()))
    assert picked[oracle.SCORE_MASS] == 51
    assert picked[oracle.SCORE_COMPKV] == 0 and picked[oracle.SCORE_FIRST_ORDER] == 0


# ---------------------------------------------------------------- fidelity diagnostics (Appendix B)

def test_spearman_matches_library_and_closed_form():
    """Spearman rank correlation: equals scipy's (average ranks for ties) and, without ties, the closed
    form 1 - 6 sum d^2 / (n (n^2 - 1)); monotone maps give 1, reversal -1."""
    from scipy.stats import spearmanr

    rng = np.random.default_rng(4)
    a, b = rng.standard_normal(300), rng.standard_normal(300)
    assert dg.spearman(a, b) == pytest.approx(spearmanr(a, b).statistic, abs=1e-12)
    ra, rb = np.argsort(np.argsort(a)), np.argsort(np.argsort(b))
    n = len(a)
    assert dg.spearman(a, b) == pytest.approx(1 - 6 * np.sum((ra - rb) ** 2) / (n * (n * n - 1)), abs=1e-12)
    t = np.round(a * 3)  # many ties
    assert dg.spearman(t, b) == pytest.approx(spearmanr(t, b).statistic, abs=1e-12)
    assert dg.spearman(a, np.exp(a)) == pytest.approx(1.0) and dg.spearman(a, -a) == pytest.approx(-1.0)


def test_capture_and_top_blocks():
    """Capture (Appendix B.2) is 1 for the exact-residual selection itself and at most 1 for any other
    selection of the same size; the top-k helper skips the excluded (mandatory) blocks and breaks ties
    by the lower id."""
    rng = np.random.default_rng(6)
    T = rng.exponential(size=60)
    ref = dg.top_blocks(T, 10, exclude=[0, 58, 59])
    assert len(ref) == 10 and not {0, 58, 59} & set(ref.tolist())
    assert dg.capture(T, ref, ref) == 1.0
    for _ in range(20):
        other = rng.choice(np.setdiff1d(np.arange(60), [0, 58, 59]), 10, replace=False)
        assert dg.capture(T, other, ref) <= 1.0 + 1e-15
    assert dg.top_blocks([1.0, 2.0, 2.0, 0.5], 2).tolist() == [1, 2]
    assert dg.top_blocks([3.0, 3.0, 3.0], 1, exclude=[0]).tolist() == [1]
