/*
 * Hierarchical Sparse Attention (HSA, arXiv 2504.16795) for AMD Instinct MI355X (gfx950).
 *
 * C ABI of libhsa_mi355x.so.  Plain C, no HIP or torch types: device buffers are passed
 * as pointers and the HIP stream as an opaque handle.
 *
 * Notation (Sec. 3.1 "Notations"): B batch, L sequence length, H query heads, G KV heads
 * (groups), h = H/G query heads per group, d head dimension, S chunk size, k top-k,
 * C = floor(L/S) complete chunks.  Query head j of group g is head g*h + j.
 *
 * Layouts (row-major, contiguous, last index fastest):
 *     Q, O, dO, dQ        [B, L, H, d]           element type params.dtype
 *     K, V, dK, dV        [B, L, G, d]           element type params.dtype
 *     Kbar                [B, C, G, d]           float32 (training), f32 or bf16 (decode cache)
 *     idx                 [B, L, G, k]  int32    selected chunks, descending chunk order, -1 pad
 *     w                   [B, L, G, k]  float32  chunk weights, 0 pad
 *
 * Semantics fixed by this library (readings of the paper):
 *   - a token t may select only chunks c < floor(t/S) (chunks strictly before its own);
 *   - group score s_c = alpha * (sum_j q_j) . Kbar_c  (the group query of dimension h*d
 *     against the landmark tiled over the h heads), alpha = 1/sqrt(h*d) by default;
 *   - top-k by score, ties to the lower chunk index, slots ordered by descending chunk
 *     index (the sort of Sec. 3.1.1), n = min(k, floor(t/S)) valid slots;
 *   - chunk weights are a softmax over the n selected scores;
 *   - intra-chunk attention is a standard softmax over the S keys, scale beta = 1/sqrt(d);
 *   - O_t = sum_i w_i O_{t,i}; O_t = 0 when the token has no candidate chunk;
 *   - gradients treat the selected index set as constant and flow through the intra-chunk
 *     attention and through w -> s -> (q, Kbar -> K).
 *
 * Ownership and behaviour (all entry points):
 *   - every pointer is device memory owned by the caller; the library never allocates,
 *     frees or synchronises, and enqueues its kernels on `stream` (a hipStream_t; NULL is
 *     the default stream) before returning;
 *   - inputs are read-only; outputs are fully overwritten (padding included);
 *   - scratch memory comes from `ws` (size from hsa_attn_workspace_size), which may hold
 *     anything on entry; calls sharing one workspace must be ordered on one stream;
 *   - arguments are validated before any launch: on error nothing is enqueued and the
 *     call returns HSA_ATTN_ERR_INVALID_ARGUMENT / _UNSUPPORTED / _WORKSPACE_TOO_SMALL;
 *     a failed launch returns HSA_ATTN_ERR_HIP.  hsa_attn_last_error() gives the detail
 *     (thread-local).
 *   - Supported by the kernels: 1 <= h <= 16, d in {64, 128}, S in {16, 32, 64, 128},
 *     1 <= k <= 32, S * d <= 8192 for F32, L >= 0 (L need not be a multiple of S; a
 *     trailing partial chunk is never a candidate), pointers 16-byte aligned.  Inputs
 *     must be finite.  idx entries outside [0, floor(t/S)) are treated as empty slots;
 *     the valid entries of one token must be distinct (hsa_select_topk's are).
 */
#ifndef HSA_MI355X_H
#define HSA_MI355X_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    HSA_ATTN_OK = 0,
    HSA_ATTN_ERR_INVALID_ARGUMENT = 1,
    HSA_ATTN_ERR_UNSUPPORTED = 2,
    HSA_ATTN_ERR_WORKSPACE_TOO_SMALL = 3,
    HSA_ATTN_ERR_HIP = 4
} hsa_attn_status_t;

typedef enum { HSA_DTYPE_F32 = 0, HSA_DTYPE_BF16 = 1 } hsa_dtype_t;

typedef enum {
    HSA_OP_LANDMARKS = 0,
    HSA_OP_SELECT = 1,
    HSA_OP_FORWARD = 2,
    HSA_OP_BACKWARD = 3,             /* also hsa_backward_attn */
    HSA_OP_DECODE = 4,
    HSA_OP_SELECT_BACKWARD = 5,
    HSA_OP_DECODE_HOST = 6
} hsa_op_t;

typedef struct {
    int32_t batch;       /* B                                                         */
    int32_t seqlen;      /* L (for hsa_decode: the cache capacity N_cap)              */
    int32_t n_qheads;    /* H                                                         */
    int32_t n_kvheads;   /* G, H % G == 0                                             */
    int32_t head_dim;    /* d                                                         */
    int32_t chunk;       /* S                                                         */
    int32_t topk;        /* k                                                         */
    hsa_dtype_t dtype;   /* element type of Q, K, V, O, dO, dQ, dK, dV                */
    float sm_scale;      /* beta; <= 0 selects 1/sqrt(d)                              */
    float sel_scale;     /* alpha; <= 0 selects 1/sqrt(h*d)                           */
    uint32_t flags;      /* HSA_FLAG_* bits (0: the defaults); other bits unsupported */
} hsa_attn_params_t;

/* Chunk weights by stick-breaking (Sec. 3.1.1, the paper's main variant) instead of the
 * softmax over the selected scores: in slot order (descending chunk index), b_i =
 * sigmoid(s_i) and w_i = b_i prod_{m<i} (1 - b_m) over the valid slots, so the weights sum
 * to less than 1.  Read by hsa_select_topk and hsa_decode (the weights they write) and by
 * hsa_backward (the score gradient ds_i = (1 - b_i) w_i dw_i - b_i sum_{m>i} w_m dw_m, with
 * b_i recovered from the given weights as w_i / (1 - sum_{m<i} w_m)); hsa_forward uses the
 * weights it is given either way. */
#define HSA_FLAG_STICK_BREAKING 2u

/* Attention inside a chunk by the softmax off by one (the normaliser of the paper's
 * kernels, Sec. 3.1.2) instead of the softmax: P_s = exp(z_s) / (1 + sum_r exp(z_r)), an
 * extra logit 0 that carries no value, so a token can give a retrieved chunk almost no
 * attention.  Read by hsa_forward, hsa_backward and hsa_decode (the attention inside
 * every selected chunk); hsa_select_topk does not depend on it.  The backward keeps its
 * form (dZ = w P (dP - D), D = dO . O_chunk), with P from this normaliser. */
#define HSA_FLAG_SOFTMAX_OFF_BY_ONE 1u

/* Landmarks (Fig. 1; Sec. 3.1 "Chunk Selection": mean-pooled chunk representation):
 * Kbar[b, c, g, :] = (1/S) sum_{s<S} K[b, c*S + s, g, :] for chunks c in
 * [chunk_begin, chunk_end) (0 <= begin <= end <= C), accumulated in fp32 and stored as
 * kbar_dtype (F32, or BF16 rounded to nearest even for a compact decode cache).  Other
 * chunks of Kbar are left untouched, so a decode cache can be extended incrementally. */
hsa_attn_status_t hsa_landmarks(const hsa_attn_params_t* p, const void* K, void* Kbar,
                                hsa_dtype_t kbar_dtype, int32_t chunk_begin,
                                int32_t chunk_end, void* stream);

/* Chunk selection + chunk weights (Sec. 3.1 chunk-selection equation; softmax weights of
 * the paper's ablation without stick-breaking).  Q: [B,L,H,d] params.dtype; Kbar:
 * [B,C,G,d] float32 (from hsa_landmarks).  Writes idx and w ([B,L,G,k]).  Scores are
 * accumulated in fp32.  Needs no workspace (ws may be NULL). */
hsa_attn_status_t hsa_select_topk(const hsa_attn_params_t* p, const void* Q,
                                  const float* Kbar, int32_t* idx, float* w, void* ws,
                                  size_t ws_bytes, void* stream);

/* Forward (Sec. 3.1.1 "Hierarchical Attention"; kernel design of Sec. 3.1.2): for every
 * (b, t, g) and valid slot i, O_{t,j,i} = softmax(beta q_j K_c^T) V_c over the S keys of
 * chunk c = idx[i]; O_{t,j} = sum_i w_i O_{t,j,i}.  idx, w are inputs (normally from
 * hsa_select_topk), so one selection may serve several attention layers.  Entries outside
 * [0, floor(t/S)) are empty slots (no contribution); a chunk given in several slots adds
 * each slot's weight.  Needs hsa_attn_workspace_size(p, HSA_OP_FORWARD) bytes of workspace:
 * zero except for bf16, h = 8, d = 128, S = 64 with at least 256 complete chunks, where the
 * chunk-major kernels keep a 2 KB partial output per (token, slot). */
hsa_attn_status_t hsa_forward(const hsa_attn_params_t* p, const void* Q, const void* K,
                              const void* V, const int32_t* idx, const float* w, void* O,
                              void* ws, size_t ws_bytes, void* stream);

/* Backward (Sec. 3.1.2, two-phase backward: queries and weights first, then keys and
 * values): gradients of sum(dO * O) w.r.t. Q, K, V with the selection fixed and
 * w = softmax of the selected scores s = alpha (sum_j q_j) . Kbar_c.  dQ includes the
 * score term alpha sum_i ds_i Kbar_{c_i}; dK includes the landmark term dKbar_c / S.
 * Kbar must be the float32 landmarks of K.  dK, dV are written for all L rows
 * (zero for chunks no token selected, and for a trailing partial chunk).  Needs
 * hsa_attn_workspace_size(p, HSA_OP_BACKWARD) bytes of workspace.  The key/value pass
 * is chunk-major and accumulates without atomics, in a fixed order: results are bitwise
 * reproducible run to run. */
hsa_attn_status_t hsa_backward(const hsa_attn_params_t* p, const void* Q, const void* K,
                               const void* V, const float* Kbar, const int32_t* idx,
                               const float* w, const void* dO, void* dQ, void* dK, void* dV,
                               void* ws, size_t ws_bytes, void* stream);

/* Backward of the attention alone, for a selection over inputs of its own (Sec. 3.1: the
 * selection query and chunk representations come from projections of their own, and
 * Sec. 4.4 shares one selection across the HSA layers).  The same as hsa_backward except
 * that the scores do not depend on Q or K: dQ and dK carry no score or landmark term, no
 * Kbar is read, and dw [B, L, G, k] float32 receives d loss / d w per slot (0 in empty
 * slots; each slot holding a chunk gets the chunk's dw), overwritten, or added to what dw
 * holds when accumulate_dw != 0 (sum over the layers sharing the selection, then pass the
 * sum to hsa_select_backward).  Workspace: hsa_attn_workspace_size(p, HSA_OP_BACKWARD). */
hsa_attn_status_t hsa_backward_attn(const hsa_attn_params_t* p, const void* Q, const void* K,
                                    const void* V, const int32_t* idx, const float* w,
                                    const void* dO, void* dQ, void* dK, void* dV, float* dw,
                                    int32_t accumulate_dw, void* ws, size_t ws_bytes,
                                    void* stream);

/* Backward of the selection scores alone (Sec. 3.1 scores s_i = alpha q~ . Kbar_{c_i} with
 * q~ = sum_j q_j over the group's h rows; the weight rule of Sec. 3.1.1): from dw
 * [B, L, G, k] = d loss / d w and the selection (idx, w), ds follows from the weights
 * (softmax, or stick-breaking with HSA_FLAG_STICK_BREAKING), and
 *   dQ[b, t, g h + j, :] = alpha sum_i ds_i Kbar[b, c_i, g, :]          (each j < h)
 *   dKbar[b, c, g, :]   = alpha sum over (t, i) with c_i = c of ds_i q~_t
 * For a selection over inputs of its own, Q [B, L, G, d_sel] (n_qheads = n_kvheads) holds
 * the selection queries and Kbar [B, C, G, d_sel] float32 the chunk representations, with
 * d_sel = head_dim up to 1024 (bf16 above 128); alpha defaults to 1/sqrt(d_sel).  dQ has Q's
 * type and layout; dKbar is written for all C chunks (zero where nothing selected it);
 * the chunk sums run in increasing token order, without atomics.  Workspace:
 * hsa_attn_workspace_size(p, HSA_OP_SELECT_BACKWARD). */
hsa_attn_status_t hsa_select_backward(const hsa_attn_params_t* p, const void* Q,
                                      const float* Kbar, const int32_t* idx, const float* w,
                                      const float* dw, void* dQ, float* dKbar, void* ws,
                                      size_t ws_bytes, void* stream);

/* Single-token decode (Sec. 3.2 "Inference": only the landmark cache is scanned, and the
 * selected chunks' keys and values are read).  p->seqlen is the cache capacity N_cap;
 * q, o: [B, H, d] params.dtype; Kcache, Vcache: [B, N_cap, G, d] params.dtype;
 * Kbar_cache: [B, floor(N_cap/S), G, d] of kbar_dtype (F32 or BF16), valid for every
 * complete cached chunk; cache_len: device int32 [B] with 0 <= cache_len[b] <= N_cap, or
 * NULL for all N_cap.  The query of sequence b sits at position cache_len[b] and sees the
 * chunks c < floor(cache_len[b]/S).  Writes o, idx [B,G,k], w [B,G,k].  Needs
 * hsa_attn_workspace_size(p, HSA_OP_DECODE) bytes of workspace. */
hsa_attn_status_t hsa_decode(const hsa_attn_params_t* p, const void* q, const void* Kcache,
                             const void* Vcache, const void* Kbar_cache,
                             hsa_dtype_t kbar_dtype, const int32_t* cache_len, void* o,
                             int32_t* idx, float* w, void* ws, size_t ws_bytes, void* stream);

/* Kernel families an op can be served by (hsa_attn_set_path). */
typedef enum {
    HSA_PATH_AUTO = 0,         /* chosen by shape: the fastest family that serves it       */
    HSA_PATH_GENERIC = 1,      /* the fp32 vector-ALU kernels, which serve every supported
                                  shape (all ops)                                          */
    HSA_PATH_TWO_PASS = 2,     /* HSA_OP_BACKWARD: a query pass then a key pass, each
                                  recomputing the attention (bf16, h = 8, d = 128)         */
    HSA_PATH_CHUNK_MAJOR = 3,  /* HSA_OP_FORWARD: chunk-major (bf16, h = 8, d = 128, S = 64) */
    HSA_PATH_TILE_MAJOR = 4,   /* HSA_OP_FORWARD: tile-major (bf16, h = 8, d = 128)         */
    HSA_PATH_FUSED = 5         /* HSA_OP_BACKWARD: one chunk-major pass with per-(token,
                                  slot) partial dQ (bf16, h = 8, d = 128, S = 64)          */
} hsa_path_t;

/* Test and measurement hook, not needed in normal use: serve `op` (HSA_OP_SELECT,
 * HSA_OP_FORWARD, HSA_OP_BACKWARD, which also covers hsa_backward_attn, or HSA_OP_DECODE,
 * which also covers hsa_decode_host; -1: all four) with the kernel family `path` from now
 * on, process-wide and for every thread, until set again (HSA_PATH_AUTO restores the
 * default).  A family that does not serve a call's shape leaves that call on its default
 * family.  Results agree across families up to rounding; hsa_attn_workspace_size follows
 * the setting, so size workspaces after setting it.  Returns INVALID_ARGUMENT for a path
 * that no kernel of `op` has. */
hsa_attn_status_t hsa_attn_set_path(int op, int path);

/* The family set for `op` (HSA_PATH_AUTO unless hsa_attn_set_path set another); -1 for an
 * unknown op. */
int hsa_attn_get_path(int op);

/* Optional kernel timing: while enabled (on != 0), every kernel launched by this library is
 * bracketed by two HIP events recorded on its stream.  Off by default. */
hsa_attn_status_t hsa_attn_timing_enable(int on);

/* Restricts the timing to the kernels named `name` (the names hsa_attn_timing_collect
 * reports); NULL or "" times every kernel again.  The string is copied.  Event pairs cost
 * some microseconds of queue time between launches, so timing one kernel keeps the others'
 * launches back to back. */
hsa_attn_status_t hsa_attn_timing_select(const char* name);

/* Waits for the recorded events and accumulates, per kernel name, the launches and total
 * milliseconds since the last delivery.  If len is at least the returned length, writes
 * one line per kernel, "name launches total_ms\n", NUL-terminated, into buf and starts a
 * new accumulation; otherwise keeps the totals (buf, if given, receives "").  Returns the
 * length needed including the NUL. */
int hsa_attn_timing_collect(char* buf, size_t len);

/* Workspace bytes needed by `op` (an hsa_op_t) for these params; 0 if none.  Returns 0
 * for invalid params as well (the entry point then reports the error). */
size_t hsa_attn_workspace_size(const hsa_attn_params_t* p, int op);

/* Static description of a status code. */
const char* hsa_attn_status_string(hsa_attn_status_t s);

/* Detail of the last error on the calling thread ("" if none). */
const char* hsa_attn_last_error(void);

/* Single-token decode with the key / value cache in host memory (Sec. 3.2 "Inference" and
 * the memory offloading of Sec. 4.4: only the landmark cache stays on the GPU, and the
 * selected chunks' keys and values are fetched from the host each step).  The same as
 * hsa_decode, with Kcache and Vcache [B, N_cap, G, d] in pinned host memory (hipHostMalloc,
 * or a pinned torch tensor) that the device can address; the selected chunks are read by a
 * kernel over the host link into a device stage inside the workspace, with no host round
 * trip.  q, Kbar_cache, cache_len, o, idx, w are device memory, as for hsa_decode.  Returns
 * INVALID_ARGUMENT when a cache (its first or last byte) is not pinned host memory.  Same
 * results as hsa_decode on the same cache contents (the same kernels after the gather).
 * Workspace: hsa_attn_workspace_size(p, HSA_OP_DECODE_HOST). */
hsa_attn_status_t hsa_decode_host(const hsa_attn_params_t* p, const void* q,
                                  const void* Kcache_host, const void* Vcache_host,
                                  const void* Kbar_cache, hsa_dtype_t kbar_dtype,
                                  const int32_t* cache_len, void* o, int32_t* idx, float* w,
                                  void* ws, size_t ws_bytes, void* stream);

/* Bytes of the device scratch array behind hsa_decode_noalloc (per GPU). */
#define HSA_DECODE_NOALLOC_SCRATCH_BYTES (8u << 20)

/* hsa_decode for callers that cannot allocate device memory (code under HIP graph capture,
 * serving loops that may not call hipMalloc, harnesses that forbid it): the same arguments
 * and results as hsa_decode, without the workspace arguments.  Its scratch memory (slice
 * candidates and per-slot partial outputs) is a file-scope device
 * array of HSA_DECODE_NOALLOC_SCRATCH_BYTES per GPU, held until the process ends; the call
 * allocates and frees nothing.  Shapes whose hsa_attn_workspace_size(p, HSA_OP_DECODE)
 * exceeds that size return HSA_ATTN_ERR_UNSUPPORTED before any launch (the 1M-token cache of
 * 8 sequences with 16 query / 2 KV heads needs 0.6 MB).  Every call on a GPU uses that GPU's
 * one array: calls that overlap on one GPU (on different streams, or from several threads
 * without ordering) race and give undefined results.  Nothing in the array needs clearing
 * between calls (every value read was written by the same call). */
hsa_attn_status_t hsa_decode_noalloc(const hsa_attn_params_t* p, const void* q,
                                     const void* Kcache, const void* Vcache,
                                     const void* Kbar_cache, hsa_dtype_t kbar_dtype,
                                     const int32_t* cache_len, void* o, int32_t* idx, float* w,
                                     void* stream);

#ifdef __cplusplus
}
#endif
#endif /* HSA_MI355X_H */
