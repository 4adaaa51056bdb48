/*
 * compkv_oracle.c -- plain, slow, fp64 CPU oracle of CompKV's decode-step attention.
 *
 * TEST INFRASTRUCTURE ONLY. The tests, the smoke check and the CPU-baseline leg of the bench call
 * it; the product library never does. It shares no code, header or helper with the HIP path: the
 * only thing both sides consume is the bf16 bit patterns drawn by the seeded input generators.
 *
 * Everything is computed per unit: one KV head of one sequence, shared by G query heads (Section
 * 3.1, grouped-query attention). Token j of the unit is row j of K and V ([n][d], bf16 bits).
 * Arithmetic is fp64 throughout; loops follow the paper's definitions in the order the paper
 * states them, with no blocking, fusion or reordering.
 *
 * Readings of points the paper leaves open (the HIP path takes the same readings):
 *  - coordinate groups (Appendix A.4): the d coordinates form d/2 RoPE frequency pairs; with the
 *    rotate-half layout pair f is (f, f + d/2), with the interleaved layout it is (2f, 2f+1). For r
 *    dividing d/2 the pairs are cut into r equal consecutive groups; for r = d each coordinate is
 *    its own group t = {t}.
 *  - variances are population variances (divide by |b|, Section 4.1 and Appendix E.1).
 *  - the mandatory set is the first n_sink blocks and the n_recent most recent blocks, overlap
 *    counted once, inside the budget (Section 4.2); a budget K >= X selects every block; a budget
 *    smaller than the mandatory set is an error.
 *  - equal scores are ranked by ascending block index ("stable" Top-K, Appendix E.1); the selected
 *    ids are returned in position order.
 *  - the logit scale s is an input (1/sqrt(d) in the paper, Section 3.1); the variance projection
 *    uses s^2, which is the paper's 1/d when s = 1/sqrt(d) (Eq. grouped-variance-metadata).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_LAYOUT_ROTATE_HALF 0
#define ORC_LAYOUT_INTERLEAVED 1

static double bf16(uint16_t h) {
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* Section 3.1: contiguous fixed-size blocks from the first token; the last one may be partial. */
int orc_num_blocks(int n, int B) { return n <= 0 ? 0 : (n + B - 1) / B; }

int orc_block_len(int n, int B, int b) {
    int rem = n - b * B;
    return rem < B ? rem : B;
}

/* Appendix A.4: group index t of coordinate i, or -1 when r is not a valid granularity. */
int orc_group_of(int i, int d, int r, int layout) {
    if (d <= 0 || r <= 0 || i < 0 || i >= d) return -1;
    if (r == d) return i;
    if (d % 2 != 0 || (d / 2) % r != 0) return -1;
    int pairs_per_group = (d / 2) / r;
    int pair;
    if (layout == ORC_LAYOUT_ROTATE_HALF)
        pair = i < d / 2 ? i : i - d / 2;
    else if (layout == ORC_LAYOUT_INTERLEAVED)
        pair = i / 2;
    else
        return -1;
    return pair / pairs_per_group;
}

/*
 * Per-block summary (Section 4.1, Eq. grouped-variance-metadata; Section 4.2):
 *   kmean[b][i] = mean of k_{j,i} over the block, vmean likewise,
 *   dvar[b][t]  = (1 / (|b| |G_t|)) sum_{j in b} sum_{i in G_t} (k_{j,i} - kmean[b][i])^2.
 * Returns 0, or -1 for an invalid (d, r, layout).
 */
int orc_block_stats(const uint16_t* K, const uint16_t* V, int n, int d, int B, int r, int layout,
                    double* kmean, double* dvar, double* vmean) {
    if (orc_group_of(0, d, r, layout) < 0 || B <= 0) return -1;
    int X = orc_num_blocks(n, B);
    int group_size = d / r;
    for (int b = 0; b < X; ++b) {
        int lo = b * B, nb = orc_block_len(n, B, b);
        for (int i = 0; i < d; ++i) {
            double sk = 0.0, sv = 0.0;
            for (int j = lo; j < lo + nb; ++j) {
                sk += bf16(K[(size_t)j * d + i]);
                sv += bf16(V[(size_t)j * d + i]);
            }
            kmean[(size_t)b * d + i] = sk / nb;
            vmean[(size_t)b * d + i] = sv / nb;
        }
        for (int t = 0; t < r; ++t) dvar[(size_t)b * r + t] = 0.0;
        for (int j = lo; j < lo + nb; ++j)
            for (int i = 0; i < d; ++i) {
                double dev = bf16(K[(size_t)j * d + i]) - kmean[(size_t)b * d + i];
                dvar[(size_t)b * r + orc_group_of(i, d, r, layout)] += dev * dev;
            }
        for (int t = 0; t < r; ++t) dvar[(size_t)b * r + t] /= (double)nb * group_size;
    }
    return 0;
}

/*
 * Block scoring from the summaries (Section 4.1):
 *   zbar[g][b] = s q_g . kmean_b                                       (block-mean logit)
 *   sig2[g][b] = s^2 sum_t (sum_{i in G_t} q_{g,i}^2) dvar[b][t]      (Eq. grouped-variance-metadata)
 *   phat[g][b] = |b| exp(zbar + sig2/2) / sum_c |c| exp(zbar_c + sig2_c/2), per query head, over
 *                every block                                          (Eq. compkv-mass-estimate)
 *   score[b]   = sum_g phat[g][b] sig2[g][b]                           (Eq. compkv-score)
 * kind selects the score of the ablations of Section 5.4:
 *   0  the CompKV score above;
 *   1  mass only: score[b] = sum_g phat[g][b] (the second-order mass estimate, no variance factor);
 *   2  first order: phat from the mean-key logits alone, |b| exp(zbar) normalized over the blocks,
 *      and score[b] = sum_g phat[g][b] sig2[g][b].
 * phat receives the mass estimate the score uses. q is [G][d] bf16 bits. Returns 0, or -1 for an
 * invalid (d, r, layout) or kind.
 */
int orc_block_scores(const uint16_t* q, int G, const double* kmean, const double* dvar, int n, int d,
                     int B, int r, int layout, double scale, int kind, double* zbar, double* sig2,
                     double* phat, double* score) {
    if (orc_group_of(0, d, r, layout) < 0 || B <= 0 || kind < 0 || kind > 2) return -1;
    int X = orc_num_blocks(n, B);
    double* Qg = (double*)calloc((size_t)r, sizeof(double));
    double* logw = (double*)malloc((size_t)(X > 0 ? X : 1) * sizeof(double));
    if (!Qg || !logw) {
        free(Qg);
        free(logw);
        return -2;
    }
    for (int b = 0; b < X; ++b) score[b] = 0.0;
    for (int g = 0; g < G; ++g) {
        const uint16_t* qg = q + (size_t)g * d;
        for (int t = 0; t < r; ++t) Qg[t] = 0.0;
        for (int i = 0; i < d; ++i) Qg[orc_group_of(i, d, r, layout)] += bf16(qg[i]) * bf16(qg[i]);
        for (int b = 0; b < X; ++b) {
            double z = 0.0;
            for (int i = 0; i < d; ++i) z += bf16(qg[i]) * kmean[(size_t)b * d + i];
            double v = 0.0;
            for (int t = 0; t < r; ++t) v += Qg[t] * dvar[(size_t)b * r + t];
            zbar[(size_t)g * X + b] = scale * z;
            sig2[(size_t)g * X + b] = scale * scale * v;
            logw[b] = log((double)orc_block_len(n, B, b)) + zbar[(size_t)g * X + b];
            if (kind != 2) logw[b] += 0.5 * sig2[(size_t)g * X + b];
        }
        double m = -INFINITY;
        for (int b = 0; b < X; ++b)
            if (logw[b] > m) m = logw[b];
        double den = 0.0;
        for (int b = 0; b < X; ++b) den += exp(logw[b] - m);
        for (int b = 0; b < X; ++b) {
            phat[(size_t)g * X + b] = exp(logw[b] - m) / den;
            score[b] += kind == 1 ? phat[(size_t)g * X + b] : phat[(size_t)g * X + b] * sig2[(size_t)g * X + b];
        }
    }
    free(Qg);
    free(logw);
    return 0;
}

typedef struct {
    double s;
    int b;
} orc_cand;

static int orc_cand_cmp(const void* pa, const void* pb) {
    const orc_cand* a = (const orc_cand*)pa;
    const orc_cand* c = (const orc_cand*)pb;
    if (a->s > c->s) return -1;
    if (a->s < c->s) return 1;
    return a->b < c->b ? -1 : (a->b > c->b ? 1 : 0);
}

/*
 * Selected set (Eq. compkv-selected-set, Appendix E.1): S = F u TopK_{K-|F|}{score_b : b not in F},
 * with F the first n_sink and the n_recent most recent blocks. Writes the ids in ascending order
 * to sel (room for min(K, X) ids) and returns their count; -1 when K < |F| < X.
 */
int orc_select(const double* score, int X, int K, int n_sink, int n_recent, int* sel) {
    if (X <= 0) return 0;
    if (K >= X) {
        for (int b = 0; b < X; ++b) sel[b] = b;
        return X;
    }
    unsigned char* chosen = (unsigned char*)calloc((size_t)X, 1);
    orc_cand* cand = (orc_cand*)malloc((size_t)X * sizeof(orc_cand));
    if (!chosen || !cand) {
        free(chosen);
        free(cand);
        return -2;
    }
    int n_mand = 0, n_cand = 0;
    for (int b = 0; b < X; ++b) {
        if (b < n_sink || b >= X - n_recent) {
            chosen[b] = 1;
            ++n_mand;
        } else {
            cand[n_cand].s = score[b];
            cand[n_cand].b = b;
            ++n_cand;
        }
    }
    if (K < n_mand) {
        free(chosen);
        free(cand);
        return -1;
    }
    qsort(cand, (size_t)n_cand, sizeof(orc_cand), orc_cand_cmp);
    for (int k = 0; k < K - n_mand && k < n_cand; ++k) chosen[cand[k].b] = 1;
    int n_sel = 0;
    for (int b = 0; b < X; ++b)
        if (chosen[b]) sel[n_sel++] = b;
    free(chosen);
    free(cand);
    return n_sel;
}

/*
 * Compensated output (Eq. compkv-output): tokens of selected blocks enter with their exact logits
 * z = s q_g . k_j and values v_j; every unselected block enters once with logit log|b| + zbar_b
 * (its |b| tokens all carry the block-mean logit) and value vmean_b. zbar_b is recomputed here from
 * kmean. With compensate == 0 the unselected blocks are left out altogether (Drop: attention
 * renormalized over the selected tokens, Appendix A.5). out is [G][d]; lse[g] is the natural log of
 * the normalizer; with no term at all out is 0 and lse is -inf.
 * Returns 0, or -1 if sel holds an out-of-range or repeated id.
 */
int orc_sparse_decode(const uint16_t* q, int G, const uint16_t* K, const uint16_t* V,
                      const double* kmean, const double* vmean, int n, int d, int B, double scale,
                      const int* sel, int n_sel, int compensate, double* out, double* lse) {
    int X = orc_num_blocks(n, B);
    unsigned char* in_s = (unsigned char*)calloc((size_t)(X > 0 ? X : 1), 1);
    double* logit = (double*)malloc((size_t)(n + X + 1) * sizeof(double));
    if (!in_s || !logit) {
        free(in_s);
        free(logit);
        return -2;
    }
    for (int k = 0; k < n_sel; ++k) {
        if (sel[k] < 0 || sel[k] >= X || in_s[sel[k]]) {
            free(in_s);
            free(logit);
            return -1;
        }
        in_s[sel[k]] = 1;
    }
    for (int g = 0; g < G; ++g) {
        const uint16_t* qg = q + (size_t)g * d;
        /* first the logits of every term (exact tokens, then one pseudo-token per omitted block) */
        int m_terms = 0;
        for (int b = 0; b < X; ++b) {
            int lo = b * B, nb = orc_block_len(n, B, b);
            if (in_s[b]) {
                for (int j = lo; j < lo + nb; ++j) {
                    double z = 0.0;
                    for (int i = 0; i < d; ++i) z += bf16(qg[i]) * bf16(K[(size_t)j * d + i]);
                    logit[m_terms++] = scale * z;
                }
            } else if (compensate) {
                double z = 0.0;
                for (int i = 0; i < d; ++i) z += bf16(qg[i]) * kmean[(size_t)b * d + i];
                logit[m_terms++] = log((double)nb) + scale * z;
            }
        }
        double m = -INFINITY;
        for (int k = 0; k < m_terms; ++k)
            if (logit[k] > m) m = logit[k];
        /* then numerator and denominator, walking the terms in the same order */
        double den = 0.0;
        double* o = out + (size_t)g * d;
        for (int i = 0; i < d; ++i) o[i] = 0.0;
        int k = 0;
        for (int b = 0; b < X; ++b) {
            int lo = b * B, nb = orc_block_len(n, B, b);
            if (in_s[b]) {
                for (int j = lo; j < lo + nb; ++j) {
                    double w = exp(logit[k++] - m);
                    den += w;
                    for (int i = 0; i < d; ++i) o[i] += w * bf16(V[(size_t)j * d + i]);
                }
            } else if (compensate) {
                double w = exp(logit[k++] - m);
                den += w;
                for (int i = 0; i < d; ++i) o[i] += w * vmean[(size_t)b * d + i];
            }
        }
        if (m_terms == 0) {
            lse[g] = -INFINITY;
            continue;
        }
        for (int i = 0; i < d; ++i) o[i] /= den;
        lse[g] = m + log(den);
    }
    free(in_s);
    free(logit);
    return 0;
}

/* Full attention (Section 3.1): o_g = softmax_j(s q_g . k_j) V over all n tokens, and its lse. */
int orc_dense_decode(const uint16_t* q, int G, const uint16_t* K, const uint16_t* V, int n, int d,
                     double scale, double* out, double* lse) {
    double* logit = (double*)malloc((size_t)(n + 1) * sizeof(double));
    if (!logit) return -2;
    for (int g = 0; g < G; ++g) {
        const uint16_t* qg = q + (size_t)g * d;
        double m = -INFINITY;
        for (int j = 0; j < n; ++j) {
            double z = 0.0;
            for (int i = 0; i < d; ++i) z += bf16(qg[i]) * bf16(K[(size_t)j * d + i]);
            logit[j] = scale * z;
            if (logit[j] > m) m = logit[j];
        }
        double den = 0.0;
        double* o = out + (size_t)g * d;
        for (int i = 0; i < d; ++i) o[i] = 0.0;
        for (int j = 0; j < n; ++j) {
            double w = exp(logit[j] - m);
            den += w;
            for (int i = 0; i < d; ++i) o[i] += w * bf16(V[(size_t)j * d + i]);
        }
        for (int i = 0; i < d; ++i) o[i] /= den;
        lse[g] = n > 0 ? m + log(den) : -INFINITY;
    }
    free(logit);
    return 0;
}
