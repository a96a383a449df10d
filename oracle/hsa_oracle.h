/*
 * HSA oracle: a plain, slow, fp64 CPU implementation of Hierarchical Sparse Attention
 * (arXiv 2504.16795).  TEST INFRASTRUCTURE ONLY: it is called by the test-suite, by the
 * smoke check and by the benchmark's CPU-baseline leg, never by the GPU product path,
 * and it shares no code, header or constant with that path.
 *
 * Every function works on ONE (batch, KV-group) slice; the caller splits [B, L, H, d]
 * tensors into such slices.  Within a slice (row-major, last index fastest):
 *     Q, dO, O, dQ : [L, h, d]   (the h query heads of the group)
 *     K, V, dK, dV : [L, d]      (the group's key / value head)
 *     Kbar         : [C, d]      (C = floor(L / S) complete chunks)
 *     idx, w, ds   : [L, k]      (selected chunks, slot order = descending chunk index)
 * A token t (0-indexed) may select only chunks c < floor(t / S): chunks that lie
 * strictly before the token's own chunk.
 *
 * Parity: every function here is pinned by the CPU test-suite (brute force over chunk
 * subsets, closed forms, library-attention reductions, finite differences); none is
 * "parity unpinned".
 */
#ifndef HSA_ORACLE_H
#define HSA_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
    int64_t L;      /* tokens in the slice (for decode: tokens in the cache)          */
    int32_t h;      /* query heads sharing the KV head (GQA ratio)                     */
    int32_t d;      /* head dimension                                                  */
    int32_t S;      /* chunk size                                                      */
    int32_t k;      /* top-k chunks per token                                          */
    double alpha;   /* selection-score scale (paper: 1/sqrt(d_g), d_g = h * d)         */
    double beta;    /* intra-chunk attention scale (1/sqrt(d))                         */
    int32_t stick;  /* chunk weights: 0 softmax over the selected scores; 1 stick-breaking
                       (Sec. 3.1.1): in slot order, b_i = sigmoid(s_i),
                       w_i = b_i prod_{m<i} (1 - b_m)                                     */
    int32_t off_by_one; /* intra-chunk attention: 0 softmax; 1 softmax off by one (Sec. 3.1.2
                       kernel description), P_s = exp(z_s) / (1 + sum_r exp(z_r)), so a
                       token may give a retrieved chunk almost no attention              */
    int32_t sep;    /* 1: the selection scores come from inputs of their own (Sec. 3.1: the
                       selection query and chunk representations), not from Q and K; the
                       attention backward then leaves out the score term (no gradient
                       reaches Q or K through the selection) and reports dw instead       */
} hsa_oracle_dims;

/* Mean-pooled landmark of every complete chunk: Kbar[c] = (1/S) sum_s K[c*S + s]
 * (Fig. 1 caption; Sec. 3.1 "Chunk Selection", mean-pooled chunk representation). */
void hsa_oracle_landmarks(const hsa_oracle_dims* dm, const double* K, double* Kbar);

/* Chunk selection and chunk weights for the tokens listed in rows[0..ntok) (rows == NULL:
 * all L tokens, in order).  Sec. 3.1 chunk-selection equation: group score
 * s_c = alpha * sum_j q_j . Kbar_c over candidates c < floor(t/S); the top-k by score
 * (ties to the lower chunk index) are stored in descending chunk order (the sort of
 * Sec. 3.1.1), padded with idx = -1, w = 0.  Weights are a softmax over the selected
 * scores.  gap (optional) receives s_(n) - s_(n+1) of the descending score order, or
 * +inf when every candidate is selected.  sel_score (optional) receives the selected
 * scores in slot order.  With dm->stick the weights are stick-breaking instead. */
void hsa_oracle_select(const hsa_oracle_dims* dm, const double* Q, const double* Kbar,
                       int64_t ntok, const int64_t* rows, int32_t* idx, double* w,
                       double* gap, double* sel_score);

/* Group scores of every candidate (Sec. 3.1 chunk-selection equation): for n queries
 * q [n, h, d] at sequence positions pos[n], s[r, c] = alpha * (sum_j q_j) . Kbar_c for
 * c < min(floor(pos[r]/S), ncol); the other entries of the row [ncol] are NaN.
 * Kbar has ncol rows [ncol, d]. */
void hsa_oracle_scores(const hsa_oracle_dims* dm, const double* q, const double* Kbar,
                       int64_t ncol, int64_t n, const int64_t* pos, double* s);

/* The chunk-weight rule (Sec. 3.1.1) applied to GIVEN slots: for n queries q [n, h, d]
 * at positions pos[n] and slots idx [n, k], the valid slots (0 <= idx < min(floor(pos/S),
 * ncol)) get the softmax over their scores s_c = alpha (sum_j q_j) . Kbar_c, or with
 * dm->stick the stick-breaking weights in the given slot order; other slots get 0.
 * With the oracle's own selection this is the oracle's w; with another selection of
 * the same scores it is the weight that selection must carry. */
void hsa_oracle_slot_weights(const hsa_oracle_dims* dm, const double* q, const double* Kbar,
                             int64_t ncol, int64_t n, const int64_t* pos,
                             const int32_t* idx, double* w);

/* Forward for the listed tokens (Sec. 3.1.1 "Hierarchical Attention"): for every head j
 * and slot i, O_{j,i} = softmax(beta q_j K_c^T) V_c over the S keys of chunk c = idx[i]
 * (softmax off by one with dm->off_by_one); O_j = sum_i w_i O_{j,i}; O = 0 for a token
 * with no candidate chunk.
 * O has shape [ntok, h, d]. */
void hsa_oracle_forward(const hsa_oracle_dims* dm, const double* Q, const double* K,
                        const double* V, const int32_t* idx, const double* w,
                        int64_t ntok, const int64_t* rows, double* O);

/* Backward phase 1 (query side; the paper's two-phase scheme, Sec. 3.1.2): gradient of
 * sum(dO * O) w.r.t. the queries of the listed tokens, with the selection held fixed and
 * w = softmax(selected scores), or with dm->stick the stick-breaking weights (their
 * b_i recovered from w over the valid slots in slot order: b_i = w_i / (1 - sum_{m<i} w_m)).  Includes the intra-chunk term and the chunk-weight term
 * reaching q through the scores.  dQ: [ntok, h, d]; ds (optional): [ntok, k] gradient
 * w.r.t. the selected scores (0 in padded slots). */
void hsa_oracle_backward_q(const hsa_oracle_dims* dm, const double* Q, const double* K,
                           const double* V, const double* Kbar, const int32_t* idx,
                           const double* w, const double* dO, int64_t ntok,
                           const int64_t* rows, double* dQ, double* ds, double* dw);

/* Gradient through the selection scores alone, for a selection over its own inputs (or
 * the score term of the fused form): given dw [L, k] = d loss / d w (summed over every
 * layer that used the selection), ds_i follows from the weight rule (softmax, or
 * stick-breaking with dm->stick), and with s_i = alpha (sum_j q_j) . Kbar_{c_i}:
 *   dQ[t, j, :]  = alpha sum_i ds_i Kbar_{c_i}       (the same for each of the h rows)
 *   dKbar[c, :]  = alpha sum over (t, i) with c_i = c of ds_i (sum_j q_j)
 * over all L tokens of the slice (dKbar accumulated in increasing token order).  Q [L, h,
 * d], Kbar [C, d]; outputs dQ [L, h, d], dKbar [C, d], ds [L, k] (optional). */
void hsa_oracle_select_backward(const hsa_oracle_dims* dm, const double* Q,
                                const double* Kbar, const int32_t* idx, const double* w,
                                const double* dw, double* dQ, double* dKbar, double* ds);

/* Backward phase 2 (key/value side): gradient w.r.t. K and V of the S tokens of each
 * listed chunk (chunks == NULL: all C complete chunks), accumulated over the tokens that
 * selected it in increasing token order, plus the landmark term dKbar_c / S where
 * dKbar_c = alpha * sum ds * (sum_j q_j).  ds: [L, k] from phase 1 (needed for every
 * token that selected a listed chunk).  dK, dV: [nch, S, d]. */
void hsa_oracle_backward_kv(const hsa_oracle_dims* dm, const double* Q, const double* K,
                            const double* V, const int32_t* idx, const double* w,
                            const double* dO, const double* ds, int64_t nch,
                            const int64_t* chunks, double* dK, double* dV);

/* Single-token decode (Sec. 3.2 "Inference"): the query q [h, d] sits at position
 * t = n_cache and sees the cache chunks c < floor(n_cache / S), scored against the GIVEN
 * landmark cache Kbar_cache [>= floor(n_cache/S), d].  Outputs idx, w [k], o [h, d] and
 * the optional score gap. */
void hsa_oracle_decode(const hsa_oracle_dims* dm, const double* q, const double* Kc,
                       const double* Vc, const double* Kbar_cache, int64_t n_cache,
                       int32_t* idx, double* w, double* o, double* gap);

#ifdef __cplusplus
}
#endif
#endif
