/*
 * HSA oracle — plain fp64 CPU implementation (test infrastructure only; see hsa_oracle.h).
 *
 * Written from the paper's definitions (arXiv 2504.16795, Sec. 3.1 chunk-selection
 * equation, Sec. 3.1.1 chunk weights and hierarchical attention, Sec. 3.1.2 two-phase
 * backward), with these readings where the paper is silent or ambiguous:
 *   - candidates are the chunks strictly before the token's own chunk;
 *   - the group score uses the concatenated group query against the tiled landmark,
 *     i.e. alpha * (sum_j q_j) . Kbar_c;
 *   - chunk weights are a softmax over the selected scores (the paper's ablation
 *     without stick-breaking), or the stick-breaking weights of the main variant (a dims
 *     flag); intra-chunk attention is the standard softmax, or (a dims flag) the softmax
 *     off by one of the paper's kernels;
 *   - ties in the top-k go to the lower chunk index; slots are ordered by descending
 *     chunk index;
 *   - gradients treat the selected index set as constant.
 * Loops are scalar and unblocked; OpenMP only distributes independent tokens / chunks.
 */
#include "hsa_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
    double s;
    int64_t c;
} cand_t;

/* descending score, ties to the lower chunk index */
static int cmp_score_desc(const void* a, const void* b) {
    const cand_t* x = (const cand_t*)a;
    const cand_t* y = (const cand_t*)b;
    if (x->s > y->s) return -1;
    if (x->s < y->s) return 1;
    if (x->c < y->c) return -1;
    if (x->c > y->c) return 1;
    return 0;
}

/* descending chunk index */
static int cmp_chunk_desc(const void* a, const void* b) {
    const cand_t* x = (const cand_t*)a;
    const cand_t* y = (const cand_t*)b;
    if (x->c > y->c) return -1;
    if (x->c < y->c) return 1;
    return 0;
}

void hsa_oracle_landmarks(const hsa_oracle_dims* dm, const double* K, double* Kbar) {
    const int64_t C = dm->L / dm->S;
    const int d = dm->d, S = dm->S;
#pragma omp parallel for schedule(static)
    for (int64_t c = 0; c < C; ++c) {
        for (int e = 0; e < d; ++e) {
            double acc = 0.0;
            for (int s = 0; s < S; ++s) acc += K[(c * S + s) * d + e];
            Kbar[c * d + e] = acc / (double)S;
        }
    }
}

/* Chunk weights of n selected scores s[0..n) given in slot order (Sec. 3.1.1):
 * a softmax over them (the ablation without stick-breaking), or with dm->stick the
 * stick-breaking weights, b_i = sigmoid(s_i) and slot i takes the share b_i of what the
 * earlier slots left, u_i = prod_{m<i} (1 - b_m). */
static void weight_rule(const hsa_oracle_dims* dm, const double* s, int64_t n, double* w) {
    if (dm->stick) {
        double u = 1.0;
        for (int64_t i = 0; i < n; ++i) {
            const double bi = 1.0 / (1.0 + exp(-s[i]));
            w[i] = bi * u;
            u *= 1.0 - bi;
        }
    } else {
        double m = -INFINITY;
        for (int64_t i = 0; i < n; ++i) m = s[i] > m ? s[i] : m;
        double z = 0.0;
        for (int64_t i = 0; i < n; ++i) z += exp(s[i] - m);
        for (int64_t i = 0; i < n; ++i) w[i] = exp(s[i] - m) / z;
    }
}

/* Group score of one candidate: alpha * (sum_j q_j) . Kbar_c, with the head sum qsum
 * formed first (the same dot product as the concatenated group query against the landmark
 * tiled over the h heads). */
static double group_score(const hsa_oracle_dims* dm, const double* qsum, const double* kb) {
    double acc = 0.0;
    for (int e = 0; e < dm->d; ++e) acc += qsum[e] * kb[e];
    return dm->alpha * acc;
}

static void head_sum(const hsa_oracle_dims* dm, const double* q, double* qsum) {
    for (int e = 0; e < dm->d; ++e) {
        double acc = 0.0;
        for (int j = 0; j < dm->h; ++j) acc += q[j * dm->d + e];
        qsum[e] = acc;
    }
}

/* Selection for one token: q [h, d], candidates c < ncand scored against Kbar. */
static void select_one(const hsa_oracle_dims* dm, const double* q, const double* Kbar,
                       int64_t ncand, int32_t* idx, double* w, double* gap,
                       double* sel_score) {
    const int d = dm->d, k = dm->k;
    for (int i = 0; i < k; ++i) {
        idx[i] = -1;
        w[i] = 0.0;
        if (sel_score) sel_score[i] = 0.0;
    }
    if (gap) *gap = INFINITY;
    if (ncand <= 0) return;

    /* group query: concatenating the h heads and tiling the landmark h times gives the
       same dot product as (sum_j q_j) . Kbar_c */
    double* qsum = (double*)malloc(sizeof(double) * d);
    head_sum(dm, q, qsum);
    cand_t* cand = (cand_t*)malloc(sizeof(cand_t) * ncand);
    for (int64_t c = 0; c < ncand; ++c) {
        cand[c].s = group_score(dm, qsum, Kbar + c * d);
        cand[c].c = c;
    }
    qsort(cand, (size_t)ncand, sizeof(cand_t), cmp_score_desc);
    const int64_t n = ncand < k ? ncand : k;
    if (gap) *gap = (ncand > n) ? (cand[n - 1].s - cand[n].s) : INFINITY;

    /* slots in descending chunk order */
    qsort(cand, (size_t)n, sizeof(cand_t), cmp_chunk_desc);
    double* ssel = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
    for (int64_t i = 0; i < n; ++i) {
        idx[i] = (int32_t)cand[i].c;
        ssel[i] = cand[i].s;
        if (sel_score) sel_score[i] = cand[i].s;
    }
    weight_rule(dm, ssel, n, w);
    free(ssel);
    free(cand);
    free(qsum);
}

void hsa_oracle_select(const hsa_oracle_dims* dm, const double* Q, const double* Kbar,
                       int64_t ntok, const int64_t* rows, int32_t* idx, double* w,
                       double* gap, double* sel_score) {
    const int h = dm->h, d = dm->d, k = dm->k;
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t r = 0; r < ntok; ++r) {
        const int64_t t = rows ? rows[r] : r;
        const int64_t ncand = t / dm->S;
        select_one(dm, Q + t * h * d, Kbar, ncand, idx + r * k, w + r * k,
                   gap ? gap + r : NULL, sel_score ? sel_score + r * k : NULL);
    }
}

void hsa_oracle_scores(const hsa_oracle_dims* dm, const double* q, const double* Kbar,
                       int64_t ncol, int64_t n, const int64_t* pos, double* s) {
    const int h = dm->h, d = dm->d;
#pragma omp parallel for schedule(dynamic, 4)
    for (int64_t r = 0; r < n; ++r) {
        double* qsum = (double*)malloc(sizeof(double) * d);
        head_sum(dm, q + r * h * d, qsum);
        int64_t ncand = pos[r] / dm->S;
        if (ncand > ncol) ncand = ncol;
        for (int64_t c = 0; c < ncol; ++c)
            s[r * ncol + c] = c < ncand ? group_score(dm, qsum, Kbar + c * d) : NAN;
        free(qsum);
    }
}

void hsa_oracle_slot_weights(const hsa_oracle_dims* dm, const double* q, const double* Kbar,
                             int64_t ncol, int64_t n, const int64_t* pos,
                             const int32_t* idx, double* w) {
    const int h = dm->h, d = dm->d, k = dm->k;
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t r = 0; r < n; ++r) {
        double* qsum = (double*)malloc(sizeof(double) * d);
        double* sv = (double*)malloc(sizeof(double) * k);
        double* wv = (double*)malloc(sizeof(double) * k);
        int* slot = (int*)malloc(sizeof(int) * k);
        head_sum(dm, q + r * h * d, qsum);
        int64_t ncand = pos[r] / dm->S;
        if (ncand > ncol) ncand = ncol;
        int64_t nv = 0;
        for (int i = 0; i < k; ++i) {
            const int64_t c = idx[r * k + i];
            w[r * k + i] = 0.0;
            if (c < 0 || c >= ncand) continue;
            sv[nv] = group_score(dm, qsum, Kbar + c * d);
            slot[nv++] = i;
        }
        weight_rule(dm, sv, nv, wv);
        for (int64_t i = 0; i < nv; ++i) w[r * k + slot[i]] = wv[i];
        free(slot);
        free(wv);
        free(sv);
        free(qsum);
    }
}

/* Standard softmax attention of one query row q [d] over the S keys of a chunk:
   P [S] receives the probabilities, o [d] the attended value (P V). */
/* Attention of one query over one chunk's S keys: P = softmax(beta q K_c^T), or with
 * dm->off_by_one P_s = exp(z_s) / (1 + sum_r exp(z_r)) (the "1" is a logit 0 that carries
 * no value; both are evaluated after subtracting the largest logit, the 0 included);
 * o = P V_c. */
static void chunk_attention(const hsa_oracle_dims* dm, const double* q, const double* Kc,
                            const double* Vc, double* P, double* o) {
    const int d = dm->d, S = dm->S;
    double m = dm->off_by_one ? 0.0 : -INFINITY;
    for (int s = 0; s < S; ++s) {
        double acc = 0.0;
        for (int e = 0; e < d; ++e) acc += q[e] * Kc[s * d + e];
        P[s] = dm->beta * acc;
        if (P[s] > m) m = P[s];
    }
    double z = dm->off_by_one ? exp(-m) : 0.0;
    for (int s = 0; s < S; ++s) {
        P[s] = exp(P[s] - m);
        z += P[s];
    }
    for (int s = 0; s < S; ++s) P[s] /= z;
    for (int e = 0; e < d; ++e) {
        double acc = 0.0;
        for (int s = 0; s < S; ++s) acc += P[s] * Vc[s * d + e];
        o[e] = acc;
    }
}

void hsa_oracle_forward(const hsa_oracle_dims* dm, const double* Q, const double* K,
                        const double* V, const int32_t* idx, const double* w,
                        int64_t ntok, const int64_t* rows, double* O) {
    const int h = dm->h, d = dm->d, S = dm->S, k = dm->k;
#pragma omp parallel
    {
        double* P = (double*)malloc(sizeof(double) * S);
        double* o = (double*)malloc(sizeof(double) * d);
#pragma omp for schedule(dynamic, 16)
        for (int64_t r = 0; r < ntok; ++r) {
            const int64_t t = rows ? rows[r] : r;
            double* Ot = O + r * h * d;
            memset(Ot, 0, sizeof(double) * h * d);
            for (int i = 0; i < k; ++i) {
                const int64_t c = idx[t * k + i];
                if (c < 0) continue;
                const double wi = w[t * k + i];
                for (int j = 0; j < h; ++j) {
                    chunk_attention(dm, Q + (t * h + j) * d, K + c * S * d, V + c * S * d, P, o);
                    for (int e = 0; e < d; ++e) Ot[j * d + e] += wi * o[e];
                }
            }
        }
        free(o);
        free(P);
    }
}

/* d loss / d s_i of one token from dw_i = d loss / d w_i, through the weight rule over the
 * valid slots (idx >= 0).  bsb: scratch of k doubles. */
static void score_grad(const hsa_oracle_dims* dm, const int32_t* idx_t, const double* w_t,
                       const double* dw, double* bsb, double* dsl) {
    const int k = dm->k;
    for (int i = 0; i < k; ++i) dsl[i] = 0.0;
    if (dm->stick) {
        /* stick-breaking weights w_i = b_i u_i, u_i = prod_{m<i} (1 - b_m) over the
           valid slots: dw_i reaches s_i through b_i directly and through the (1 - b_i)
           factor of every later slot, ds_i = (1 - b_i) w_i dw_i - b_i sum_{m>i} w_m dw_m */
        double u = 1.0;
        for (int i = 0; i < k; ++i) {
            if (idx_t[i] < 0) continue;
            bsb[i] = u > 0.0 ? w_t[i] / u : 0.0;
            u -= w_t[i];
        }
        double tail = 0.0;
        for (int i = k - 1; i >= 0; --i) {
            if (idx_t[i] < 0) continue;
            const double wd = w_t[i] * dw[i];
            dsl[i] = (1.0 - bsb[i]) * wd - bsb[i] * tail;
            tail += wd;
        }
    } else {
        /* softmax chunk weights: ds_i = w_i (dw_i - sum_m w_m dw_m) */
        double wdw = 0.0;
        for (int i = 0; i < k; ++i) wdw += w_t[i] * dw[i];
        for (int i = 0; i < k; ++i)
            if (idx_t[i] >= 0) dsl[i] = w_t[i] * (dw[i] - wdw);
    }
}

void hsa_oracle_backward_q(const hsa_oracle_dims* dm, const double* Q, const double* K,
                           const double* V, const double* Kbar, const int32_t* idx,
                           const double* w, const double* dO, int64_t ntok,
                           const int64_t* rows, double* dQ, double* ds, double* dw_out) {
    const int h = dm->h, d = dm->d, S = dm->S, k = dm->k;
#pragma omp parallel
    {
        double* P = (double*)malloc(sizeof(double) * S);
        double* dP = (double*)malloc(sizeof(double) * S);
        double* o = (double*)malloc(sizeof(double) * d);
        double* dw = (double*)malloc(sizeof(double) * k);
        double* dsl = (double*)malloc(sizeof(double) * k);
        double* bsb = (double*)malloc(sizeof(double) * k);
#pragma omp for schedule(dynamic, 16)
        for (int64_t r = 0; r < ntok; ++r) {
            const int64_t t = rows ? rows[r] : r;
            double* dQt = dQ + r * h * d;
            memset(dQt, 0, sizeof(double) * h * d);
            for (int i = 0; i < k; ++i) {
                dw[i] = 0.0;
                dsl[i] = 0.0;
            }
            for (int i = 0; i < k; ++i) {
                const int64_t c = idx[t * k + i];
                if (c < 0) continue;
                const double wi = w[t * k + i];
                const double* Kc = K + c * S * d;
                const double* Vc = V + c * S * d;
                for (int j = 0; j < h; ++j) {
                    const double* qj = Q + (t * h + j) * d;
                    const double* gj = dO + (t * h + j) * d;
                    chunk_attention(dm, qj, Kc, Vc, P, o);
                    /* D = dO_j . O_{j,i}  (equivalently sum_s P_s dP_s).  The same holds off
                       by one: its extra logit carries no value, and dP_s/dz_r is still
                       P_s (delta_sr - P_r) */
                    double D = 0.0;
                    for (int e = 0; e < d; ++e) D += gj[e] * o[e];
                    dw[i] += D;
                    for (int s = 0; s < S; ++s) {
                        double acc = 0.0;
                        for (int e = 0; e < d; ++e) acc += gj[e] * Vc[s * d + e];
                        dP[s] = acc;
                    }
                    /* d loss / d logit z_s = w P_s (dP_s - D); z = beta q.k */
                    for (int s = 0; s < S; ++s) {
                        const double dz = wi * P[s] * (dP[s] - D);
                        for (int e = 0; e < d; ++e) dQt[j * d + e] += dm->beta * dz * Kc[s * d + e];
                    }
                }
            }
            if (dw_out)
                for (int i = 0; i < k; ++i) dw_out[r * k + i] = dw[i];
            if (dm->sep) {
                /* the scores do not depend on Q or K: no score term, and no ds for the
                   landmark term of dK */
                if (ds)
                    for (int i = 0; i < k; ++i) ds[r * k + i] = 0.0;
                continue;
            }
            score_grad(dm, idx + t * k, w + t * k, dw, bsb, dsl);
            for (int i = 0; i < k; ++i) {
                const int64_t c = idx[t * k + i];
                if (c < 0) continue;
                /* s_i = alpha (sum_j q_j) . Kbar_c: the same term reaches every head */
                for (int j = 0; j < h; ++j)
                    for (int e = 0; e < d; ++e)
                        dQt[j * d + e] += dm->alpha * dsl[i] * Kbar[c * d + e];
            }
            if (ds)
                for (int i = 0; i < k; ++i) ds[r * k + i] = dsl[i];
        }
        free(bsb);
        free(dsl);
        free(dw);
        free(o);
        free(dP);
        free(P);
    }
}

void hsa_oracle_select_backward(const hsa_oracle_dims* dm, const double* Q,
                                const double* Kbar, const int32_t* idx, const double* w,
                                const double* dw, double* dQ, double* dKbar, double* ds) {
    const int h = dm->h, d = dm->d, k = dm->k;
    const int64_t L = dm->L, C = dm->L / dm->S;
    double* dsl = (double*)malloc(sizeof(double) * k);
    double* bsb = (double*)malloc(sizeof(double) * k);
    double* qs = (double*)malloc(sizeof(double) * d);
    memset(dKbar, 0, sizeof(double) * (size_t)(C > 0 ? C : 0) * d);
    for (int64_t t = 0; t < L; ++t) {
        score_grad(dm, idx + t * k, w + t * k, dw + t * k, bsb, dsl);
        if (ds)
            for (int i = 0; i < k; ++i) ds[t * k + i] = dsl[i];
        /* q~ = sum_j q_j, the query the score was formed with */
        for (int e = 0; e < d; ++e) {
            double a = 0.0;
            for (int j = 0; j < h; ++j) a += Q[(t * h + j) * d + e];
            qs[e] = a;
        }
        double* dQt = dQ + t * h * d;
        memset(dQt, 0, sizeof(double) * h * d);
        for (int i = 0; i < k; ++i) {
            const int64_t c = idx[t * k + i];
            if (c < 0) continue;
            for (int e = 0; e < d; ++e) {
                const double g = dm->alpha * dsl[i] * Kbar[c * d + e];
                for (int j = 0; j < h; ++j) dQt[j * d + e] += g;
                dKbar[c * d + e] += dm->alpha * dsl[i] * qs[e];
            }
        }
    }
    free(qs);
    free(bsb);
    free(dsl);
}

void hsa_oracle_backward_kv(const hsa_oracle_dims* dm, const double* Q, const double* K,
                            const double* V, const int32_t* idx, const double* w,
                            const double* dO, const double* ds, int64_t nch,
                            const int64_t* chunks, double* dK, double* dV) {
    const int h = dm->h, d = dm->d, S = dm->S, k = dm->k;
    const int64_t L = dm->L;
#pragma omp parallel
    {
        double* P = (double*)malloc(sizeof(double) * S);
        double* dP = (double*)malloc(sizeof(double) * S);
        double* o = (double*)malloc(sizeof(double) * d);
        double* dKbar = (double*)malloc(sizeof(double) * d);
        double* qsum = (double*)malloc(sizeof(double) * d);
#pragma omp for schedule(dynamic, 1)
        for (int64_t r = 0; r < nch; ++r) {
            const int64_t c = chunks ? chunks[r] : r;
            double* dKc = dK + r * S * d;
            double* dVc = dV + r * S * d;
            memset(dKc, 0, sizeof(double) * S * d);
            memset(dVc, 0, sizeof(double) * S * d);
            memset(dKbar, 0, sizeof(double) * d);
            const double* Kc = K + c * S * d;
            const double* Vc = V + c * S * d;
            for (int64_t t = (c + 1) * S; t < L; ++t) {
                for (int i = 0; i < k; ++i) {
                    if (idx[t * k + i] != c) continue;
                    const double wi = w[t * k + i];
                    for (int e = 0; e < d; ++e) qsum[e] = 0.0;
                    for (int j = 0; j < h; ++j) {
                        const double* qj = Q + (t * h + j) * d;
                        const double* gj = dO + (t * h + j) * d;
                        for (int e = 0; e < d; ++e) qsum[e] += qj[e];
                        chunk_attention(dm, qj, Kc, Vc, P, o);
                        double D = 0.0;
                        for (int e = 0; e < d; ++e) D += gj[e] * o[e];
                        for (int s = 0; s < S; ++s) {
                            double acc = 0.0;
                            for (int e = 0; e < d; ++e) acc += gj[e] * Vc[s * d + e];
                            dP[s] = acc;
                        }
                        for (int s = 0; s < S; ++s) {
                            const double dz = wi * P[s] * (dP[s] - D);
                            for (int e = 0; e < d; ++e) {
                                dVc[s * d + e] += wi * P[s] * gj[e];
                                dKc[s * d + e] += dm->beta * dz * qj[e];
                            }
                        }
                    }
                    for (int e = 0; e < d; ++e) dKbar[e] += dm->alpha * ds[t * k + i] * qsum[e];
                }
            }
            /* Kbar_c = (1/S) sum_s K[cS+s] */
            for (int s = 0; s < S; ++s)
                for (int e = 0; e < d; ++e) dKc[s * d + e] += dKbar[e] / (double)S;
        }
        free(qsum);
        free(dKbar);
        free(o);
        free(dP);
        free(P);
    }
}

void hsa_oracle_decode(const hsa_oracle_dims* dm, const double* q, const double* Kc,
                       const double* Vc, const double* Kbar_cache, int64_t n_cache,
                       int32_t* idx, double* w, double* o, double* gap) {
    const int h = dm->h, d = dm->d, S = dm->S, k = dm->k;
    select_one(dm, q, Kbar_cache, n_cache / S, idx, w, gap, NULL);
    double* P = (double*)malloc(sizeof(double) * S);
    double* oc = (double*)malloc(sizeof(double) * d);
    memset(o, 0, sizeof(double) * h * d);
    for (int i = 0; i < k; ++i) {
        const int64_t c = idx[i];
        if (c < 0) continue;
        for (int j = 0; j < h; ++j) {
            chunk_attention(dm, q + j * d, Kc + c * S * d, Vc + c * S * d, P, oc);
            for (int e = 0; e < d; ++e) o[j * d + e] += w[i] * oc[e];
        }
    }
    free(oc);
    free(P);
}
