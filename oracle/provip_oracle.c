/*
 * provip_oracle.c -- CPU oracle for ProViP's progressive visual-token pruning
 * ("Not All Attention Heads Contribute to Critical Visual Token Selection:
 * Head-Aware Pruning Matters More").
 *
 * TEST INFRASTRUCTURE.  This file is the slow, plain reference that the HIP
 * path is checked against.  Only the test-suite, the smoke check and the
 * benchmark's CPU-baseline leg may load it; the product path never calls it.
 * It shares no code, header, table or helper with the HIP library.
 *
 * Conventions
 *   - fp64 arithmetic from the exact input values, plain loops in index order,
 *     one sample at a time, row-major contiguous arrays.
 *   - Readings of places where the paper is silent are marked "Reading:".
 *   - parity unpinned: orc_merge (the paper defers the aggregation rule to
 *     another work; pinned only to the reading stated at the function).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* --------------------------------------------------------------------------
 * Sec. 4.2, equations for r and T: critical text tokens from the text's own
 * similarity, decoupled from the image.  With E the text embeddings [nt][d],
 *     r[j] = (1/nt) sum_i softmax_j(e_i . e_j)     (no scaling of E E^T),
 *     T    = { j : r[j] > mean(r) }.
 * Reading: when no r[j] lies strictly above the mean (all equal; N(0,1)
 * rows of width >= 256 give that, every softmax row being one-hot on its
 * own token), T is every token.
 * E: [nt][d]; r: [nt] out; mask: [nt] out, 1 for j in T.  Returns |T|, or
 * -3 on no memory.
 * ------------------------------------------------------------------------ */
int orc_critical_text(const double *E, int nt, int d, double *r, int32_t *mask)
{
    double *S = (double *)malloc(sizeof(double) * (size_t)nt * nt);
    if (!S) return -3;
    for (int i = 0; i < nt; ++i) {
        double *row = S + (size_t)i * nt;
        for (int j = 0; j < nt; ++j) {
            double s = 0.0;
            for (int c = 0; c < d; ++c) s += E[(size_t)i * d + c] * E[(size_t)j * d + c];
            row[j] = s;
        }
        double m = row[0];
        for (int j = 1; j < nt; ++j)
            if (row[j] > m) m = row[j];
        double z = 0.0;
        for (int j = 0; j < nt; ++j) {
            row[j] = exp(row[j] - m);
            z += row[j];
        }
        for (int j = 0; j < nt; ++j) row[j] /= z;
    }
    for (int j = 0; j < nt; ++j) {
        double s = 0.0;
        for (int i = 0; i < nt; ++i) s += S[(size_t)i * nt + j];
        r[j] = s / (double)nt;
    }
    double mean = 0.0;
    for (int j = 0; j < nt; ++j) mean += r[j];
    mean /= (double)nt;
    int count = 0;
    for (int j = 0; j < nt; ++j) {
        mask[j] = r[j] > mean ? 1 : 0;
        count += mask[j];
    }
    if (count == 0) {
        for (int j = 0; j < nt; ++j) mask[j] = 1;
        count = nt;
    }
    free(S);
    return count;
}

/* --------------------------------------------------------------------------
 * Sec. 4.3, equation for M: cosine similarity between the i-th critical text
 * token and the j-th visual token,
 *     M[i][j] = (t_i . v_j) / (|t_i| |v_j|).
 * Reading: a zero-norm vector has no direction; M[i][j] := 0 when
 * |t_i| |v_j| == 0.
 * anchors: [nt][d], vis: [nv][d], M: [nt][nv].
 * ------------------------------------------------------------------------ */
void orc_cosine(const double *anchors, int nt, const double *vis, int nv, int d,
                double *M)
{
    for (int i = 0; i < nt; ++i) {
        const double *t = anchors + (size_t)i * d;
        double tt = 0.0;
        for (int c = 0; c < d; ++c) tt += t[c] * t[c];
        double tn = sqrt(tt);
        for (int j = 0; j < nv; ++j) {
            const double *v = vis + (size_t)j * d;
            double vv = 0.0, tv = 0.0;
            for (int c = 0; c < d; ++c) {
                vv += v[c] * v[c];
                tv += t[c] * v[c];
            }
            double den = tn * sqrt(vv);
            M[(size_t)i * nv + j] = (den == 0.0) ? 0.0 : tv / den;
        }
    }
}

/* --------------------------------------------------------------------------
 * Sec. 4.3, equation for M-hat: subtract from each text row its mean over
 * all N_v visual tokens,
 *     Mhat[i][j] = M[i][j] - (1/N_v) sum_k M[i][k].
 * ------------------------------------------------------------------------ */
void orc_center(const double *M, int nt, int nv, double *Mhat)
{
    for (int i = 0; i < nt; ++i) {
        double s = 0.0;
        for (int k = 0; k < nv; ++k) s += M[(size_t)i * nv + k];
        double mean = s / (double)nv;
        for (int j = 0; j < nv; ++j)
            Mhat[(size_t)i * nv + j] = M[(size_t)i * nv + j] - mean;
    }
}

/* --------------------------------------------------------------------------
 * Sec. 4.3, equation for p: max-pooling over the text dimension,
 *     p[j] = max_i Mhat[i][j].
 * ------------------------------------------------------------------------ */
void orc_maxpool(const double *Mhat, int nt, int nv, double *p)
{
    for (int j = 0; j < nv; ++j) {
        double m = Mhat[j];
        for (int i = 1; i < nt; ++i) {
            double x = Mhat[(size_t)i * nv + j];
            if (x > m) m = x;
        }
        p[j] = m;
    }
}

/* --------------------------------------------------------------------------
 * Top-k retention (Sec. 4.3: keep the N_1 highest p; Sec. 4.4: keep the N_2
 * highest v).
 * Reading: token j precedes j' when score[j] > score[j'], or the scores are
 * equal and j < j' (lower index wins a tie; -0 and +0 compare equal).  The k
 * first tokens of that order are kept and written in ascending index order.
 * Written as a rank count so that it reads as the definition.
 * Returns 0, or -1 when k is outside [1, n].
 * ------------------------------------------------------------------------ */
int orc_topk(const double *score, int n, int k, int32_t *kept)
{
    if (k < 1 || k > n) return -1;
    int w = 0;
    for (int j = 0; j < n; ++j) {
        int rank = 0;
        for (int jj = 0; jj < n; ++jj) {
            if (score[jj] > score[j] || (score[jj] == score[j] && jj < j)) ++rank;
        }
        if (rank < k) kept[w++] = j;
    }
    return (w == k) ? 0 : -2;
}

/* --------------------------------------------------------------------------
 * Sec. 4.3, last paragraph: the retained tokens act as cluster centroids and
 * every pruned token goes to its nearest centroid.
 * Reading: "nearest" is the largest cosine similarity (the measure of the
 * equation for M, zero rule included); ties go to the lowest kept index.
 * A kept token is its own centroid.
 *
 * kept: [n1] ascending token indices.  rows: the token indices to assign
 * (NULL = all tokens 0..nv-1, with nrows == nv).  For each listed row r:
 *   assign[r] = slot s in [0, n1) of its centroid kept[s] (a kept token
 *               gets its own slot),
 *   best[r]   = the largest cosine over all slots,
 *   second[r] = the second-largest cosine over all slots (-2 when n1 == 1).
 * best/second may be NULL; they let a caller see how close a decision was.
 * ------------------------------------------------------------------------ */
void orc_assign(const double *vis, int nv, int d, const int32_t *kept, int n1,
                const int32_t *rows, int nrows, int32_t *assign, double *best,
                double *second)
{
    (void)nv;
    for (int r = 0; r < nrows; ++r) {
        int j = rows ? rows[r] : r;
        const double *x = vis + (size_t)j * d;
        int own = -1;
        for (int s = 0; s < n1; ++s)
            if (kept[s] == j) own = s;
        double xx = 0.0;
        for (int c = 0; c < d; ++c) xx += x[c] * x[c];
        double b = -2.0, b2 = -2.0;
        int bs = -1;
        for (int s = 0; s < n1; ++s) {
            const double *y = vis + (size_t)kept[s] * d;
            double yy = 0.0, xy = 0.0;
            for (int c = 0; c < d; ++c) {
                yy += y[c] * y[c];
                xy += x[c] * y[c];
            }
            double den = sqrt(xx) * sqrt(yy);
            double cs = (den == 0.0) ? 0.0 : xy / den;
            if (cs > b) {
                b2 = b;
                b = cs;
                bs = s;
            } else if (cs > b2) {
                b2 = cs;
            }
        }
        if (own >= 0) bs = own;
        assign[r] = bs;
        if (best) best[r] = b;
        if (second) second[r] = b2;
    }
}

/* --------------------------------------------------------------------------
 * Sec. 4.3, last paragraph: pruned embeddings are aggregated into their
 * nearest centroids.  The paper gives no formula (it follows another work).
 * Reading (parity unpinned): each centroid becomes the unweighted mean of its
 * own embedding and the embeddings of the tokens assigned to it,
 *     merged[s] = (vis[kept[s]] + sum_{j pruned, assign[j]==s} vis[j]) / (1 + m_s).
 * assign: [nv] slot per token (kept tokens carry their own slot).
 * merged: [n1][d].
 * ------------------------------------------------------------------------ */
void orc_merge(const double *vis, int nv, int d, const int32_t *kept, int n1,
               const int32_t *assign, double *merged)
{
    for (int s = 0; s < n1; ++s) {
        double *out = merged + (size_t)s * d;
        const double *self = vis + (size_t)kept[s] * d;
        for (int c = 0; c < d; ++c) out[c] = self[c];
        int count = 1;
        for (int j = 0; j < nv; ++j) {
            if (j == kept[s] || assign[j] != s) continue;
            const double *x = vis + (size_t)j * d;
            for (int c = 0; c < d; ++c) out[c] += x[c];
            ++count;
        }
        for (int c = 0; c < d; ++c) out[c] /= (double)count;
    }
}

/* --------------------------------------------------------------------------
 * Sec. 4.3 as a whole for one sample: M, M-hat, p, top-N_1, nearest-centroid
 * assignment and merge.  Outputs may be NULL except kept.
 * Returns 0 or the error of orc_topk.
 * ------------------------------------------------------------------------ */
int orc_dedup(const double *anchors, int nt, const double *vis, int nv, int d,
              int n1, int32_t *kept, double *p_out, int32_t *assign_out,
              double *merged_out)
{
    double *M = (double *)malloc(sizeof(double) * (size_t)nt * nv);
    double *Mh = (double *)malloc(sizeof(double) * (size_t)nt * nv);
    double *p = (double *)malloc(sizeof(double) * (size_t)nv);
    int32_t *as = (int32_t *)malloc(sizeof(int32_t) * (size_t)nv);
    int rc = -3;
    if (!M || !Mh || !p || !as) goto done;
    orc_cosine(anchors, nt, vis, nv, d, M);
    orc_center(M, nt, nv, Mh);
    orc_maxpool(Mh, nt, nv, p);
    rc = orc_topk(p, nv, n1, kept);
    if (rc != 0) goto done;
    if (p_out) memcpy(p_out, p, sizeof(double) * (size_t)nv);
    if (assign_out || merged_out) {
        orc_assign(vis, nv, d, kept, n1, NULL, nv, as, NULL, NULL);
        if (assign_out) memcpy(assign_out, as, sizeof(int32_t) * (size_t)nv);
        if (merged_out) orc_merge(vis, nv, d, kept, n1, as, merged_out);
    }
done:
    free(M);
    free(Mh);
    free(p);
    free(as);
    return rc;
}

/* --------------------------------------------------------------------------
 * Sec. 4.4: the cross-modal attention map of one head, text-query rows over
 * visual keys, A = softmax_j(Q K^T / sqrt(hd)).
 * Reading: the softmax is taken over the visual keys passed in, so each row
 * sums to 1; the scale is the per-head 1/sqrt(hd) of the backbone's attention.
 * The row maximum is subtracted before exponentiation (exact in real
 * arithmetic).
 * q: [nt][hd], k: [n][hd], A: [nt][n].
 * ------------------------------------------------------------------------ */
void orc_attention(const double *q, const double *k, int nt, int n, int hd, double *A)
{
    double scale = 1.0 / sqrt((double)hd);
    for (int i = 0; i < nt; ++i) {
        double *row = A + (size_t)i * n;
        for (int j = 0; j < n; ++j) {
            double s = 0.0;
            for (int c = 0; c < hd; ++c) s += q[(size_t)i * hd + c] * k[(size_t)j * hd + c];
            row[j] = s * scale;
        }
        double m = row[0];
        for (int j = 1; j < n; ++j)
            if (row[j] > m) m = row[j];
        double z = 0.0;
        for (int j = 0; j < n; ++j) {
            row[j] = exp(row[j] - m);
            z += row[j];
        }
        for (int j = 0; j < n; ++j) row[j] /= z;
    }
}

/* --------------------------------------------------------------------------
 * Sec. 4.4, equations for S^vis and v, for one sample:
 *     S[i][j] = (1/|V|) sum_{h in V} A_h[i][j],
 *     v[j]    = (1/N_t) sum_i S[i][j].
 * q: [H][nt][hd], k: [H][n][hd], heads: [nh] head ids (the set V).
 * Returns 0, or -1 on a bad head id.
 * ------------------------------------------------------------------------ */
int orc_head_aware_score(const double *q, const double *k, int H, int nt, int n, int hd,
                         const int32_t *heads, int nh, double *v)
{
    double *A = (double *)malloc(sizeof(double) * (size_t)nt * n);
    double *S = (double *)calloc((size_t)nt * n, sizeof(double));
    int rc = 0;
    if (!A || !S) {
        rc = -3;
        goto done;
    }
    for (int t = 0; t < nh; ++t) {
        int h = heads[t];
        if (h < 0 || h >= H) {
            rc = -1;
            goto done;
        }
        orc_attention(q + (size_t)h * nt * hd, k + (size_t)h * n * hd, nt, n, hd, A);
        for (size_t e = 0; e < (size_t)nt * n; ++e) S[e] += A[e];
    }
    for (size_t e = 0; e < (size_t)nt * n; ++e) S[e] /= (double)nh;
    for (int j = 0; j < n; ++j) {
        double s = 0.0;
        for (int i = 0; i < nt; ++i) s += S[(size_t)i * n + j];
        v[j] = s / (double)nt;
    }
done:
    free(A);
    free(S);
    return rc;
}

/* --------------------------------------------------------------------------
 * Sec. 4.4 for one sample: v, then the top-N_2 tokens (same order rule as
 * orc_topk).  v_out may be NULL.
 * ------------------------------------------------------------------------ */
int orc_head_aware(const double *q, const double *k, int H, int nt, int n, int hd,
                   const int32_t *heads, int nh, int n2, int32_t *kept, double *v_out)
{
    double *v = (double *)malloc(sizeof(double) * (size_t)n);
    if (!v) return -3;
    int rc = orc_head_aware_score(q, k, H, nt, n, hd, heads, nh, v);
    if (rc == 0) rc = orc_topk(v, n, n2, kept);
    if (rc == 0 && v_out) memcpy(v_out, v, sizeof(double) * (size_t)n);
    free(v);
    return rc;
}

/* --------------------------------------------------------------------------
 * Sec. 4.4 with the cross-modal map taken as the model has it: in the
 * backbone, a text row's softmax runs over every key before it (system,
 * visual and earlier text tokens), so A^cross is the visual slice of that
 * row and does not sum to 1.  The non-visual keys enter only through the
 * log-sum-exp of their scaled logits, one number per row:
 *     A[i][j] = exp(s_ij) / (sum_j' exp(s_ij') + exp(lse[i])),
 * with s_ij = q_i . k_j / sqrt(hd).  lse[i] = -inf (no other keys) gives
 * orc_attention.  The largest of the row's logits and lse[i] is
 * subtracted before exponentiation (exact in real arithmetic).
 * q: [nt][hd], k: [n][hd], lse: [nt], A: [nt][n].
 * ------------------------------------------------------------------------ */
void orc_attention_in_model(const double *q, const double *k, const double *lse, int nt, int n,
                            int hd, double *A)
{
    double scale = 1.0 / sqrt((double)hd);
    for (int i = 0; i < nt; ++i) {
        double *row = A + (size_t)i * n;
        for (int j = 0; j < n; ++j) {
            double s = 0.0;
            for (int c = 0; c < hd; ++c) s += q[(size_t)i * hd + c] * k[(size_t)j * hd + c];
            row[j] = s * scale;
        }
        double m = lse[i];
        for (int j = 0; j < n; ++j)
            if (row[j] > m) m = row[j];
        double z = exp(lse[i] - m);
        for (int j = 0; j < n; ++j) {
            row[j] = exp(row[j] - m);
            z += row[j];
        }
        for (int j = 0; j < n; ++j) row[j] /= z;
    }
}

/* --------------------------------------------------------------------------
 * Sec. 4.4, equations for S^vis and v on the in-model map above, for one
 * sample.  lse: [H][nt].  Returns 0, or -1 on a bad head id.
 * ------------------------------------------------------------------------ */
int orc_head_aware_score_in_model(const double *q, const double *k, const double *lse, int H,
                                  int nt, int n, int hd, const int32_t *heads, int nh, double *v)
{
    double *A = (double *)malloc(sizeof(double) * (size_t)nt * n);
    double *S = (double *)calloc((size_t)nt * n, sizeof(double));
    int rc = 0;
    if (!A || !S) {
        rc = -3;
        goto done;
    }
    for (int t = 0; t < nh; ++t) {
        int h = heads[t];
        if (h < 0 || h >= H) {
            rc = -1;
            goto done;
        }
        orc_attention_in_model(q + (size_t)h * nt * hd, k + (size_t)h * n * hd,
                               lse + (size_t)h * nt, nt, n, hd, A);
        for (size_t e = 0; e < (size_t)nt * n; ++e) S[e] += A[e];
    }
    for (size_t e = 0; e < (size_t)nt * n; ++e) S[e] /= (double)nh;
    for (int j = 0; j < n; ++j) {
        double s = 0.0;
        for (int i = 0; i < nt; ++i) s += S[(size_t)i * n + j];
        v[j] = s / (double)nt;
    }
done:
    free(A);
    free(S);
    return rc;
}

/* --------------------------------------------------------------------------
 * Sec. 4.4, equation for C^h: the confidence of head h is the variance of
 * its cross-modal attention scores over the visual keys, taken for each
 * critical text row and summed over those rows,
 *     C[h] = sum_i Var_j(A_h[i][j]).
 * Reading: the population variance (divide by n), written as the mean of
 * the squared deviations from the row mean; the rows passed in are the
 * critical text rows.
 * q: [H][nt][hd], k: [H][n][hd], conf: [H].  Returns 0, or -3 on no memory.
 * ------------------------------------------------------------------------ */
int orc_head_confidence(const double *q, const double *k, int H, int nt, int n, int hd,
                        double *conf)
{
    double *A = (double *)malloc(sizeof(double) * (size_t)nt * n);
    if (!A) return -3;
    for (int h = 0; h < H; ++h) {
        orc_attention(q + (size_t)h * nt * hd, k + (size_t)h * n * hd, nt, n, hd, A);
        double c = 0.0;
        for (int i = 0; i < nt; ++i) {
            const double *row = A + (size_t)i * n;
            double mean = 0.0;
            for (int j = 0; j < n; ++j) mean += row[j];
            mean /= (double)n;
            double var = 0.0;
            for (int j = 0; j < n; ++j) var += (row[j] - mean) * (row[j] - mean);
            c += var / (double)n;
        }
        conf[h] = c;
    }
    free(A);
    return 0;
}

/* --------------------------------------------------------------------------
 * Sec. 4.4, equation for V_l: the visual heads are the N_vis heads of
 * highest confidence (same order rule as orc_topk: a tie goes to the lower
 * head id), listed in ascending order.  conf_out may be NULL.
 * ------------------------------------------------------------------------ */
int orc_visual_heads(const double *q, const double *k, int H, int nt, int n, int hd,
                     int n_vis, int32_t *heads, double *conf_out)
{
    double *c = (double *)malloc(sizeof(double) * (size_t)H);
    if (!c) return -3;
    int rc = orc_head_confidence(q, k, H, nt, n, hd, c);
    if (rc == 0) rc = orc_topk(c, H, n_vis, heads);
    if (rc == 0 && conf_out) memcpy(conf_out, c, sizeof(double) * (size_t)H);
    free(c);
    return rc;
}

/* --------------------------------------------------------------------------
 * Sec. 4.4, equation for C^h, with A^cross taken as the model has it: the
 * visual slice of each text row's softmax over every key before it (the map
 * of orc_attention_in_model, whose non-visual keys enter through one
 * log-sum-exp per row).  The slice of a row sums to less than 1; its
 * variance is the population variance of its n entries about their own
 * mean, and C[h] sums it over the rows passed in.  lse = -inf everywhere
 * gives orc_head_confidence.
 * q: [H][nt][hd], k: [H][n][hd], lse: [H][nt], conf: [H].
 * Returns 0, or -3 on no memory.
 * ------------------------------------------------------------------------ */
int orc_head_confidence_in_model(const double *q, const double *k, const double *lse, int H,
                                 int nt, int n, int hd, double *conf)
{
    double *slice_map = (double *)malloc(sizeof(double) * (size_t)nt * n);
    if (!slice_map) return -3;
    for (int h = 0; h < H; ++h) {
        orc_attention_in_model(q + (size_t)h * nt * hd, k + (size_t)h * n * hd,
                               lse + (size_t)h * nt, nt, n, hd, slice_map);
        double total = 0.0;
        for (int i = 0; i < nt; ++i) {
            const double *slice = slice_map + (size_t)i * n;
            double avg = 0.0;
            for (int j = 0; j < n; ++j) avg += slice[j];
            avg /= (double)n;
            double sq_dev = 0.0;
            for (int j = 0; j < n; ++j) {
                double dev = slice[j] - avg;
                sq_dev += dev * dev;
            }
            total += sq_dev / (double)n;
        }
        conf[h] = total;
    }
    free(slice_map);
    return 0;
}

/* --------------------------------------------------------------------------
 * Sec. 4.4, equation for V_l on the confidence above: the N_vis heads of
 * highest C (orc_topk's order rule), ascending.  conf_out may be NULL.
 * ------------------------------------------------------------------------ */
int orc_visual_heads_in_model(const double *q, const double *k, const double *lse, int H,
                              int nt, int n, int hd, int n_vis, int32_t *heads,
                              double *conf_out)
{
    double *cm = (double *)malloc(sizeof(double) * (size_t)H);
    if (!cm) return -3;
    int rc = orc_head_confidence_in_model(q, k, lse, H, nt, n, hd, cm);
    if (rc == 0) rc = orc_topk(cm, H, n_vis, heads);
    if (rc == 0 && conf_out) memcpy(conf_out, cm, sizeof(double) * (size_t)H);
    free(cm);
    return rc;
}

/* --------------------------------------------------------------------------
 * Sec. 4.1: pruned tokens are excluded from all later computation, so the
 * rows of the kept tokens are compacted, in token order.  Byte copy:
 *     dst[b][g][r] = src[b][g][idx[b][r]]   (rows of row_bytes bytes).
 * Strides in bytes.  Returns 0, or -1 on an index outside [0, n_src).
 * ------------------------------------------------------------------------ */
int orc_gather(const uint8_t *src, uint8_t *dst, const int32_t *idx, int B, int n_src,
               int k, int groups, int64_t row_bytes, int64_t sb, int64_t sg, int64_t sr,
               int64_t db, int64_t dg, int64_t dr)
{
    for (int b = 0; b < B; ++b)
        for (int g = 0; g < groups; ++g)
            for (int r = 0; r < k; ++r) {
                int j = idx[(size_t)b * k + r];
                if (j < 0 || j >= n_src) return -1;
                memcpy(dst + b * db + g * dg + r * dr, src + b * sb + g * sg + j * sr,
                       (size_t)row_bytes);
            }
    return 0;
}
