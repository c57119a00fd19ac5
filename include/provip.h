/*
 * provip.h -- C ABI of the ProViP pruning hot path on AMD Instinct MI355X
 * (gfx950).
 *
 * The method (Ma et al., "Not All Attention Heads Contribute to Critical
 * Visual Token Selection: Head-Aware Pruning Matters More") prunes visual
 * tokens in two places:
 *   - before the LLM (Sec. 4.3): text-guided cosine similarity, row
 *     centring, max-pooling, top-N_1, and aggregation of every pruned token
 *     into its nearest retained token          -> pv_prune_dedup
 *   - inside the LLM at a pruning layer (Sec. 4.4): the softmax attention of
 *     the text-query rows over the visual keys, averaged over a given subset
 *     of heads and over the rows, then top-N_2   -> pv_prune_head_aware
 *   - pruned tokens leave all later computation (Sec. 4.1): order-preserving
 *     compaction of hidden-state and K/V rows     -> pv_prune_gather
 *
 * Conventions shared by every call
 *   - Tensor pointers are DEVICE memory owned by the caller, row-major and
 *     contiguous unless strides are passed.  Device pointers must be 16-byte
 *     aligned.  The library keeps no pointer after a call returns.
 *   - `stream` is a hipStream_t (NULL = the null stream).  Every call checks
 *     its arguments on the host first; on an error nothing is enqueued and a
 *     negative pv_status is returned.  Otherwise all work is enqueued on
 *     `stream` and the call returns PV_OK without synchronising.
 *   - `workspace` is caller-owned device scratch of at least the size the
 *     matching *_workspace_bytes query returns.  Its contents on entry do not
 *     matter; two calls that use one workspace must not overlap in time.
 *   - Scores are float32.  Index outputs are int32 token indices local to the
 *     span passed in, strictly increasing within a sample.
 *   - Ties between equal scores go to the lower token index; -0 and +0 are
 *     equal.  Inputs must be finite (NaN/Inf give unspecified selections).
 *   - Results are deterministic: two calls on the same inputs return the same
 *     bits (no floating-point atomics; every reduction has a fixed order).
 *   - Widths: an embedding width d or head width hd may be any multiple of 8
 *     in range.  The matrix-core kernels stream 128-byte chunks of embedding
 *     rows and a multiple of 32 elements of head rows; a call whose rows
 *     have another width first copies them, zero-padded, into its workspace
 *     (zeros change no dot product and no norm; the attention scale keeps
 *     the true hd).  The workspace queries include those copies.
 */
#ifndef PROVIP_H
#define PROVIP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    PV_OK = 0,
    PV_ERR_NULL = -1,      /* a required pointer is NULL                      */
    PV_ERR_SHAPE = -2,     /* a size is <= 0, too large, or not a multiple the
                              kernels need (see each call)                     */
    PV_ERR_BUDGET = -3,    /* budget < 1 or budget > number of tokens          */
    PV_ERR_HEADS = -4,     /* head list empty, out of range or repeated        */
    PV_ERR_DTYPE = -5,     /* dtype is not PV_F32 or PV_BF16                   */
    PV_ERR_WORKSPACE = -6, /* workspace NULL or smaller than the query         */
    PV_ERR_HIP = -7,       /* a kernel launch failed                            */
    PV_ERR_ALIGN = -8,     /* a pointer, row size or stride is not 16-byte
                              aligned                                          */
    PV_ERR_SCRATCH = -9    /* pv_prune_pipeline_noalloc: the problem needs
                              more than PV_STATIC_SCRATCH_BYTES of scratch     */
} pv_status;

typedef enum { PV_F32 = 0, PV_BF16 = 1 } pv_dtype;

/* Size limits checked by the calls. */
#define PV_MAX_TOKENS 16384   /* visual tokens per sample (Nv, N)            */
#define PV_MAX_TEXT 1024      /* text rows per sample (Nt)                   */
#define PV_MAX_DIM 16384      /* embedding width d                           */
#define PV_MAX_HEAD_DIM 256   /* head width hd                               */
#define PV_MAX_HEADS 512      /* n_heads of one head-aware call              */

/* Static string for a pv_status value (never NULL). */
const char *pv_status_string(int status);

/* ABI version, (major << 16) | minor. */
int pv_version(void);

/* -------------------------------------------------------------------------
 * Critical text tokens (Sec. 4.2, equations for r and T).
 *
 * Per sample b, with e_i the text embeddings text[b][i]:
 *   r[j]  = (1/Nt) sum_i softmax_j( e_i . e_j )   (the unscaled self-similarity)
 *   T     = { j : r[j] > mean(r) }; when no token lies strictly above the
 *           mean (all r equal), T is every token
 *   mask[b][j] = 1 for j in T, else 0;  count[b] = |T|
 * The mask goes to pv_prune_dedup_masked (anchors) and
 * pv_visual_heads_masked (rows of the confidence).
 *
 * text   [B][Nt][d]  dtype        text embeddings
 * mask   [B][Nt]     int32 out    required
 * count  [B]         int32 out    required
 * r      [B][Nt]     float32 out  may be NULL
 * Sizes: 1 <= Nt <= PV_MAX_TEXT, 8 <= d <= PV_MAX_DIM with d % 8 == 0.
 * ---------------------------------------------------------------------- */
size_t pv_critical_text_workspace_bytes(int B, int Nt, int d, int dtype);

int pv_critical_text(const void *text, int B, int Nt, int d, int dtype, int32_t *mask,
                     int32_t *count, float *r, void *workspace, size_t workspace_bytes,
                     void *stream);

/* -------------------------------------------------------------------------
 * Pruning before the LLM (Sec. 4.3).
 *
 * Per sample b (all B samples independent):
 *   M[i][j]  = cos(anchors[b][i], vis[b][j])         (equation for M; a pair
 *              with a zero-norm vector has M = 0)
 *   Mh[i][j] = M[i][j] - mean_k M[i][k]              (equation for M-hat)
 *   p[j]     = max_i Mh[i][j]                        (equation for p)
 *   kept     = the `budget` tokens with the highest p (ties: lower index),
 *              written in ascending index order
 *   assign[j]= slot s in [0, budget) of the kept token nearest to token j by
 *              cosine (ties: lower slot); a kept token gets its own slot
 *   merged[s]= mean of vis[kept[s]] and every pruned token assigned to s
 *              (the paper gives no aggregation formula; this is the unweighted
 *              mean of the centroid and its members)
 *
 * vis      [B][Nv][d]      dtype        visual embeddings (connector output)
 * anchors  [B][Nt][d]      dtype        embeddings of the critical text tokens
 * kept     [B][budget]     int32 out    required
 * score    [B][Nv]         float32 out  p, may be NULL
 * assign   [B][Nv]         int32 out    may be NULL
 * merged   [B][budget][d]  dtype out    may be NULL (then no merge is run)
 * Sizes: 1 <= Nv <= PV_MAX_TOKENS, 1 <= Nt <= PV_MAX_TEXT,
 *        8 <= d <= PV_MAX_DIM with d % 8 == 0, 1 <= budget <= Nv.
 * ---------------------------------------------------------------------- */
size_t pv_dedup_workspace_bytes(int B, int Nv, int Nt, int d, int budget, int dtype);

int pv_prune_dedup(const void *vis, const void *anchors, int B, int Nv, int Nt, int d,
                   int dtype, int budget, int32_t *kept, float *score, int32_t *assign,
                   void *merged, void *workspace, size_t workspace_bytes, void *stream);

/* -------------------------------------------------------------------------
 * pv_prune_dedup on two streams.  In Sec. 4.3 the retained set depends only
 * on the cosine scores; the aggregation of the pruned tokens into their
 * nearest retained token comes after it and nothing else in the step needs
 * it until the kept rows are gathered.  This variant lets that aggregation
 * overlap later work on `stream` (e.g. the layers up to the pruning layer,
 * or pv_prune_head_aware):
 *   - the cosine, centring, max-pool and top-N_1 kernels run on `stream`;
 *     then `selected` is recorded on `stream`;
 *   - `merge_stream` waits for `selected`; the nearest-centroid and merge
 *     kernels run on `merge_stream`; then `merged_done` is recorded there.
 * kept and score are ordered on `stream` as usual; assign and merged are
 * ready only once `merged_done` has completed (make the consumer's stream
 * wait for it).  Until then the call still reads `workspace`, `vis` and
 * `kept`: a later call must not reuse that workspace, nor overwrite vis or
 * kept, before `merged_done`.  selected and merged_done are hipEvent_t
 * handles owned by the caller; merge_stream is a hipStream_t (it may equal
 * stream).  Results are bit-identical to pv_prune_dedup.  Errors as
 * pv_prune_dedup, plus PV_ERR_NULL if merge_stream or an event is NULL.
 * ---------------------------------------------------------------------- */
int pv_prune_dedup_split(const void *vis, const void *anchors, int B, int Nv, int Nt, int d,
                         int dtype, int budget, int32_t *kept, float *score, int32_t *assign,
                         void *merged, void *workspace, size_t workspace_bytes, void *stream,
                         void *merge_stream, void *selected, void *merged_done);

/* -------------------------------------------------------------------------
 * pv_prune_dedup with the anchors restricted to the critical text rows: M
 * has one row per anchor i with anchor_mask[b][i] != 0 (Sec. 4.3 builds M
 * over the critical text tokens only), so the row means and the max-pool
 * run over those rows.  A sample whose mask has no row set uses every row.
 *
 * anchor_mask [B][Nt]  int32  DEVICE memory, 4-byte aligned (e.g. the mask
 *                             of pv_critical_text for the same rows)
 * Everything else, the workspace and the errors are those of pv_prune_dedup
 * (PV_ERR_NULL if anchor_mask is NULL).
 * ---------------------------------------------------------------------- */
int pv_prune_dedup_masked(const void *vis, const void *anchors, const int32_t *anchor_mask,
                          int B, int Nv, int Nt, int d, int dtype, int budget, int32_t *kept,
                          float *score, int32_t *assign, void *merged, void *workspace,
                          size_t workspace_bytes, void *stream);

/* -------------------------------------------------------------------------
 * Head-aware pruning at a pruning layer (Sec. 4.4, equations for S^vis and v).
 *
 * Per sample b, with V_b = heads_host[b*n_heads .. b*n_heads + n_heads):
 *   A_h[i][j] = softmax_j( q[b][h][i] . k[b][h][j] / sqrt(hd) )  over the N
 *               visual keys passed in (each row sums to 1)
 *   v[j]      = (1/|V_b|) sum_{h in V_b} (1/Nt) sum_i A_h[i][j]
 *   kept      = the `budget` tokens with the highest v (ties: lower index),
 *               ascending.
 * Passing every head 0..H-1 gives the all-head aggregation the paper uses at
 * its middle pruning layer.
 *
 * q          [B][H][Nt][hd]  dtype      text-query rows at the pruning layer
 * k          [B][H][N][hd]   dtype      keys of the N visual tokens
 * heads_host [B][n_heads]    int32      HOST memory; distinct ids in [0, H)
 * kept       [B][budget]     int32 out  required
 * score      [B][N]          float32 out  v, may be NULL
 * Sizes: 1 <= N <= PV_MAX_TOKENS, 1 <= Nt <= PV_MAX_TEXT, hd % 8 == 0,
 *        8 <= hd <= PV_MAX_HEAD_DIM, 1 <= n_heads <= min(H, PV_MAX_HEADS),
 *        1 <= budget <= N.
 * ---------------------------------------------------------------------- */
size_t pv_head_aware_workspace_bytes(int B, int H, int Nt, int N, int hd, int n_heads,
                                     int budget, int dtype);

int pv_prune_head_aware(const void *q, const void *k, const int32_t *heads_host, int n_heads,
                        int B, int H, int Nt, int N, int hd, int dtype, int budget,
                        int32_t *kept, float *score, void *workspace, size_t workspace_bytes,
                        void *stream);

/* -------------------------------------------------------------------------
 * The same with the head lists in DEVICE memory, for lists that a kernel
 * produced (pv_visual_heads) and that the caller does not read back.
 *
 * heads_dev  [B][n_heads]    int32      DEVICE memory, 4-byte aligned.  The
 *            library cannot check it before the kernels run: entries outside
 *            [0, H) are clamped into range and a repeated entry is counted as
 *            often as it appears (memory-safe; v is then the mean over the
 *            list as given).  Lists from pv_visual_heads are always valid.
 * Everything else, the workspace and the errors are those of
 * pv_prune_head_aware; results for a valid list are bit-identical to it.
 * ---------------------------------------------------------------------- */
int pv_prune_head_aware_dev(const void *q, const void *k, const int32_t *heads_dev, int n_heads,
                            int B, int H, int Nt, int N, int hd, int dtype, int budget,
                            int32_t *kept, float *score, void *workspace, size_t workspace_bytes,
                            void *stream);

/* -------------------------------------------------------------------------
 * Head-aware pruning on the cross-modal map as the model has it (Sec. 4.4:
 * A^cross is the visual slice of the backbone's attention, whose softmax also
 * runs over the system and text keys before each text row).  The other keys
 * enter through one number per row:
 *   row_lse[b][h][i] = log sum_{other keys j} exp( q . k_j / sqrt(hd) )
 *   A_h[i][j]        = exp(s_ij) / ( sum_{visual j'} exp(s_ij') + exp(row_lse) )
 * so a row's visual mass is below 1; v, the selection and everything else
 * are those of pv_prune_head_aware.  row_lse = NULL, or -INFINITY entries,
 * give the plain call's results.
 *
 * heads_host / heads_dev  exactly one non-NULL: the host list of
 *            pv_prune_head_aware or the device list of
 *            pv_prune_head_aware_dev (PV_ERR_HEADS if both are given)
 * row_lse    [B][H][Nt]  float32  DEVICE memory, 4-byte aligned, finite or
 *            -INFINITY, natural-log units; may be NULL
 * ---------------------------------------------------------------------- */
int pv_prune_head_aware_ex(const void *q, const void *k, const int32_t *heads_host,
                           const int32_t *heads_dev, int n_heads, int B, int H, int Nt, int N,
                           int hd, int dtype, int budget, const float *row_lse, int32_t *kept,
                           float *score, void *workspace, size_t workspace_bytes, void *stream);

/* -------------------------------------------------------------------------
 * Visual-head identification at a shallow pruning layer (Sec. 4.4,
 * equations for C^h and V_l).
 *
 * Per sample b and head h (every head 0..H-1):
 *   A_h[i][j] = softmax_j( q[b][h][i] . k[b][h][j] / sqrt(hd) )  as above
 *   C[b][h]   = sum_i Var_j(A_h[i][j])     population variance over the N
 *               keys, summed over the Nt rows passed in (the critical text
 *               rows)
 *   heads_out = the n_vis heads with the highest C (ties: lower head id),
 *               ascending: the list pv_prune_head_aware_dev takes.
 * One pass over the keys; the attention map is never written out.
 *
 * q          [B][H][Nt][hd]  dtype      text-query rows
 * k          [B][H][N][hd]   dtype      keys of the N visual tokens
 * heads_out  [B][n_vis]      int32 out  required
 * conf       [B][H]          float32 out  C, may be NULL
 * Sizes as pv_prune_head_aware, plus H <= PV_MAX_HEADS, 1 <= n_vis <= H
 * (else PV_ERR_HEADS).  workspace: pv_visual_heads_workspace_bytes_hd(B, H,
 * Nt, N, hd, dtype); pv_visual_heads_workspace_bytes(B, H, Nt) gives the
 * same for hd % 32 == 0.
 * ---------------------------------------------------------------------- */
size_t pv_visual_heads_workspace_bytes(int B, int H, int Nt);
size_t pv_visual_heads_workspace_bytes_hd(int B, int H, int Nt, int N, int hd, int dtype);

/* The same with the confidence summed over the rows i with
 * row_mask[b][i] != 0 only (the critical text rows of Sec. 4.4; a sample
 * whose mask has no row set uses every row).  row_mask: [B][Nt] int32 in
 * DEVICE memory, 4-byte aligned; PV_ERR_NULL if NULL. */
int pv_visual_heads_masked(const void *q, const void *k, const int32_t *row_mask, int B, int H,
                           int Nt, int N, int hd, int dtype, int n_vis, int32_t *heads_out,
                           float *conf, void *workspace, size_t workspace_bytes, void *stream);

int pv_visual_heads(const void *q, const void *k, int B, int H, int Nt, int N, int hd, int dtype,
                    int n_vis, int32_t *heads_out, float *conf, void *workspace,
                    size_t workspace_bytes, void *stream);

/* Visual heads on the cross-modal map as the model has it (Sec. 4.4: the
 * confidence is taken on A^cross, the visual slice of the backbone's
 * attention, whose softmax also runs over the system and text keys before
 * each text row).  With row_lse as in pv_prune_head_aware_ex,
 *   A_h[i][j] = exp(s_ij) / ( sum_{visual j'} exp(s_ij') + exp(row_lse[b][h][i]) )
 *   C[b][h]   = sum_i Var_j(A_h[i][j])    population variance of the row's
 *               visual slice (which sums to less than 1) over the N keys.
 * row_mask  [B][Nt] int32  DEVICE, may be NULL: the rows summed, as in
 *           pv_visual_heads_masked (NULL: every row)
 * row_lse   [B][H][Nt] float32 DEVICE, 4-byte aligned, finite or -INFINITY
 *           (natural-log units), may be NULL: NULL or -INFINITY entries give
 *           pv_visual_heads(_masked)'s results bit for bit.
 * Everything else, the workspace and the errors are those of
 * pv_visual_heads. */
int pv_visual_heads_ex(const void *q, const void *k, const int32_t *row_mask,
                       const float *row_lse, int B, int H, int Nt, int N, int hd, int dtype,
                       int n_vis, int32_t *heads_out, float *conf, void *workspace,
                       size_t workspace_bytes, void *stream);

/* -------------------------------------------------------------------------
 * The retention rule of both stages on its own (Sec. 4.3: keep the N_1
 * tokens with the highest p; Sec. 4.4: keep the N_2 tokens with the highest
 * v), for callers that compute their own scores.  Per sample b: the k
 * highest of scores[b][0..n) (ties: lower index), written ascending; the
 * kernel is the one both pruning calls above run.
 *
 * scores   [B][n]     float32     finite scores
 * kept     [B][k]     int32 out   required
 * rest     [B][n-k]   int32 out   the other indices, ascending; may be NULL
 * slot_of  [B][n]     int32 out   position of j in kept, or -1; may be NULL
 * Sizes: 1 <= B <= 65535, 1 <= n <= PV_MAX_TOKENS, 1 <= k <= n.
 * ---------------------------------------------------------------------- */
int pv_select_topk(const float *scores, int B, int n, int k, int32_t *kept, int32_t *rest,
                   int32_t *slot_of, void *stream);

/* -------------------------------------------------------------------------
 * Order-preserving row compaction (Sec. 4.1: pruned tokens are excluded from
 * all later computation):
 *   dst + b*dst_batch_stride + g*dst_group_stride + r*dst_row_stride
 *     <- row_bytes bytes at
 *   src + b*src_batch_stride + g*src_group_stride + idx[b*k + r]*src_row_stride
 * for b < B, g < groups, r < k.  Use groups = 1 for hidden states [B][N][D]
 * and groups = H for K/V caches [B][H][N][hd].  All strides are in bytes.
 * A pure byte copy: bit-exact.  idx is DEVICE memory [B][k]; an index outside
 * [0, n_src) yields a zero-filled destination row (never an out-of-bounds
 * read).  row_bytes and every stride must be multiples of 16.
 * ---------------------------------------------------------------------- */
int pv_prune_gather(const void *src, void *dst, const int32_t *idx, int B, int n_src, int k,
                    int groups, int64_t row_bytes, int64_t src_batch_stride,
                    int64_t src_group_stride, int64_t src_row_stride, int64_t dst_batch_stride,
                    int64_t dst_group_stride, int64_t dst_row_stride, void *stream);

/* -------------------------------------------------------------------------
 * The same compaction for up to PV_MAX_GATHER tensors that share one index
 * list (typically the hidden states, K and V of one pruning step), in a
 * single kernel launch.  Each descriptor has the meaning of the arguments of
 * pv_prune_gather; idx, B and k are common to all.  Errors as above; nothing
 * is enqueued if any descriptor is invalid.
 * ---------------------------------------------------------------------- */
#define PV_MAX_GATHER 4

typedef struct pv_gather_desc {
    const void *src;
    void *dst;
    int n_src;
    int groups;
    int64_t row_bytes;
    int64_t src_batch_stride, src_group_stride, src_row_stride;
    int64_t dst_batch_stride, dst_group_stride, dst_row_stride;
} pv_gather_desc;

int pv_prune_gather_batch(const pv_gather_desc *descs, int n_desc, const int32_t *idx, int B,
                          int k, void *stream);

/* -------------------------------------------------------------------------
 * Timed variants, for profiling.  Same arguments and results as the calls
 * above, plus an array of hipEvent_t handles: events[i] is recorded on
 * `stream` just before the i-th kernel the call launches and events[n] just
 * after the last one, for n = min(n_events - 1, number of kernels).  With
 * reps > 1 every kernel is launched reps times back to back between its two
 * events (the results are unchanged: no kernel reads what it writes), so
 * that elapsed(events[i], events[i+1]) / reps is the kernel's average
 * duration in a stream of its own launches.  The number of kernels a call
 * launches is returned through *n_kernels and their names (static strings,
 * at most n_events - 1 of them) through names; both may be NULL.  Passing
 * n_events = 0 records nothing.  reps < 1 gives PV_ERR_SHAPE; a NULL handle
 * among events[0 .. n_events) gives PV_ERR_NULL (nothing is enqueued).
 * ---------------------------------------------------------------------- */
int pv_prune_dedup_timed(const void *vis, const void *anchors, int B, int Nv, int Nt, int d,
                         int dtype, int budget, int32_t *kept, float *score, int32_t *assign,
                         void *merged, void *workspace, size_t workspace_bytes, void *stream,
                         void *const *events, int n_events, int reps, int *n_kernels,
                         const char **names);

int pv_prune_head_aware_timed(const void *q, const void *k, const int32_t *heads_host,
                              int n_heads, int B, int H, int Nt, int N, int hd, int dtype,
                              int budget, int32_t *kept, float *score, void *workspace,
                              size_t workspace_bytes, void *stream, void *const *events,
                              int n_events, int reps, int *n_kernels, const char **names);

int pv_prune_head_aware_dev_timed(const void *q, const void *k, const int32_t *heads_dev,
                                  int n_heads, int B, int H, int Nt, int N, int hd, int dtype,
                                  int budget, int32_t *kept, float *score, void *workspace,
                                  size_t workspace_bytes, void *stream, void *const *events,
                                  int n_events, int reps, int *n_kernels, const char **names);

int pv_visual_heads_timed(const void *q, const void *k, int B, int H, int Nt, int N, int hd,
                          int dtype, int n_vis, int32_t *heads_out, float *conf, void *workspace,
                          size_t workspace_bytes, void *stream, void *const *events, int n_events,
                          int reps, int *n_kernels, const char **names);

int pv_prune_head_aware_ex_timed(const void *q, const void *k, const int32_t *heads_host,
                                 const int32_t *heads_dev, int n_heads, int B, int H, int Nt,
                                 int N, int hd, int dtype, int budget, const float *row_lse,
                                 int32_t *kept, float *score, void *workspace,
                                 size_t workspace_bytes, void *stream, void *const *events,
                                 int n_events, int reps, int *n_kernels, const char **names);

int pv_critical_text_timed(const void *text, int B, int Nt, int d, int dtype, int32_t *mask,
                           int32_t *count, float *r, void *workspace, size_t workspace_bytes,
                           void *stream, void *const *events, int n_events, int reps,
                           int *n_kernels, const char **names);

int pv_prune_dedup_masked_timed(const void *vis, const void *anchors, const int32_t *anchor_mask,
                                int B, int Nv, int Nt, int d, int dtype, int budget,
                                int32_t *kept, float *score, int32_t *assign, void *merged,
                                void *workspace, size_t workspace_bytes, void *stream,
                                void *const *events, int n_events, int reps, int *n_kernels,
                                const char **names);

int pv_visual_heads_ex_timed(const void *q, const void *k, const int32_t *row_mask,
                             const float *row_lse, int B, int H, int Nt, int N, int hd,
                             int dtype, int n_vis, int32_t *heads_out, float *conf,
                             void *workspace, size_t workspace_bytes, void *stream,
                             void *const *events, int n_events, int reps, int *n_kernels,
                             const char **names);

int pv_visual_heads_masked_timed(const void *q, const void *k, const int32_t *row_mask, int B,
                                 int H, int Nt, int N, int hd, int dtype, int n_vis,
                                 int32_t *heads_out, float *conf, void *workspace,
                                 size_t workspace_bytes, void *stream, void *const *events,
                                 int n_events, int reps, int *n_kernels, const char **names);

/* -------------------------------------------------------------------------
 * The whole pruning step in one call (Sec. 4.1, 4.3 and 4.4 in sequence):
 *   1. pv_prune_dedup of vis against the text anchors, with the merge
 *      -> kept1 [B][budget1], score1 [B][Nv], assign [B][Nv],
 *         merged [B][budget1][d];
 *   2. the K and V rows of the budget1 kept tokens, compacted as
 *      pv_prune_gather does: k_full, v_full [B][H][Nv][hd] -> k1, v1
 *      [B][H][budget1][hd] (these stand for the keys and values that the
 *      layers up to the pruning layer produce for the retained tokens);
 *   3. pv_prune_head_aware of q [B][H][Nt][hd] over k1 with the host head
 *      list heads_host [B][n_heads] -> kept2 [B][budget2] (indices into the
 *      budget1 retained tokens), score2 [B][budget1];
 *   4. the compaction of merged, k1 and v1 to the budget2 kept tokens
 *      -> hidden2 [B][budget2][d], k2, v2 [B][H][budget2][hd].
 * Every output is the bit-for-bit result of the four calls made one after
 * another.  Where the shapes allow it (the split-k Gram on its square tiles
 * and the plain merge of the dedup, the 16-row score blocks, 256-byte head
 * rows, budget1 <= 256, B * n_heads <= 512), the two independent chains that
 * follow the top-budget1 selection share launches: the score, reading the
 * kept tokens' keys from k_full through kept1, rides in the Gram's launch;
 * the score's top-budget2, the Gram's argmax and the compaction to k1 and v1
 * share the next; and the merge writes the merged rows of the budget2 kept
 * slots to hidden2 itself and carries the compaction to k2 and v2.  The step
 * is then six launches instead of ten.  All pointers are DEVICE memory,
 * contiguous, 16-byte aligned and required (none may be NULL); heads_host is
 * HOST memory.  Errors as for the calls it combines.
 * ---------------------------------------------------------------------- */
size_t pv_pipeline_workspace_bytes(int B, int Nv, int Nt, int d, int H, int hd, int n_heads,
                                   int budget1, int budget2, int dtype);

int pv_prune_pipeline(const void *vis, const void *anchors, const void *q, const void *k_full,
                      const void *v_full, const int32_t *heads_host, int n_heads, int B, int Nv,
                      int Nt, int d, int H, int hd, int dtype, int budget1, int budget2,
                      int32_t *kept1, float *score1, int32_t *assign, void *merged, void *k1,
                      void *v1, int32_t *kept2, float *score2, void *hidden2, void *k2, void *v2,
                      void *workspace, size_t workspace_bytes, void *stream);

/* The step with an event recorded around each of its launches, as the other
 * *_timed calls do (profiling only).  Where the launches are shared, the
 * kernel names are "cos_full" (or "cos_partial", "cos_reduce"), "center",
 * "select", "gram_partial+score_partial",
 * "gram_reduce+score_select+gather_kv1" and "merge+gather_hkv2"; where they
 * are not, the step runs once without events and *n_kernels is 0. */
int pv_prune_pipeline_timed(const void *vis, const void *anchors, const void *q,
                            const void *k_full, const void *v_full, const int32_t *heads_host,
                            int n_heads, int B, int Nv, int Nt, int d, int H, int hd, int dtype,
                            int budget1, int budget2, int32_t *kept1, float *score1,
                            int32_t *assign, void *merged, void *k1, void *v1, int32_t *kept2,
                            float *score2, void *hidden2, void *k2, void *v2, void *workspace,
                            size_t workspace_bytes, void *stream, void *const *events,
                            int n_events, int reps, int *n_kernels, const char **names);

/* The same step with every kernel in its own launch (the reference against
 * which the shared launches are checked; same arguments and results). */
int pv_prune_pipeline_separate(const void *vis, const void *anchors, const void *q,
                               const void *k_full, const void *v_full, const int32_t *heads_host,
                               int n_heads, int B, int Nv, int Nt, int d, int H, int hd, int dtype,
                               int budget1, int budget2, int32_t *kept1, float *score1,
                               int32_t *assign, void *merged, void *k1, void *v1, int32_t *kept2,
                               float *score2, void *hidden2, void *k2, void *v2, void *workspace,
                               size_t workspace_bytes, void *stream);

/* -------------------------------------------------------------------------
 * The progressive schedule of the method in one call (Sec. 4 Overview and
 * Sec. 4.2-4.4): the sequential stages, each the library's call for it, so
 * every output is the bit-for-bit result of those calls made in turn.
 *   1. critical text tokens of `text` (pv_critical_text) -> text_mask;
 *   2. pruning before the LLM on the critical rows (pv_prune_dedup_masked
 *      with the merge) -> kept1 [B][budget1], assign [B][Nv],
 *      merged [B][budget1][d];
 *   3. shallow pruning layer: the keys of the budget1 retained tokens are
 *      gathered from k_s_all; visual heads over the critical rows
 *      (pv_visual_heads_masked, n_vis of them) -> vis_heads [B][n_vis],
 *      conf [B][H]; head-aware pruning on those heads over every text row
 *      (pv_prune_head_aware_dev) -> score2 [B][budget1]; the budget2
 *      survivors' token indices -> kept2 [B][budget2] and their merged rows
 *      -> hidden2 [B][budget2][d];
 *   4. middle pruning layer: the keys of the budget2 survivors are gathered
 *      from k_m_all; head-aware pruning over every head (the all-head
 *      aggregation, no head identification) -> score3 [B][budget2]; the
 *      budget3 survivors' token indices -> kept3 [B][budget3] and rows
 *      -> hidden3 [B][budget3][d].
 * text    [B][Nt][d]      dtype  text embeddings (critical-text selection and
 *                                the anchors of stage 2)
 * vis     [B][Nv][d]      dtype  visual embeddings
 * q_s     [B][H][Nt][hd]  dtype  text-query rows at the shallow layer
 * k_s_all [B][H][Nv][hd]  dtype  shallow-layer keys of every visual token
 * q_m, k_m_all            the same at the middle layer
 * kept1, kept2, kept3     original token indices, ascending
 * conf, score2, score3 may be NULL; every other pointer is required.  All
 * pointers are DEVICE memory, contiguous and 16-byte aligned.
 * Sizes: those of the calls above; 1 <= n_vis <= H,
 * 1 <= budget3 <= budget2 <= budget1 <= Nv (else PV_ERR_HEADS /
 * PV_ERR_BUDGET).  workspace: pv_progressive_workspace_bytes.
 * ---------------------------------------------------------------------- */
size_t pv_progressive_workspace_bytes(int B, int Nv, int Nt, int d, int H, int hd, int budget1,
                                      int n_vis, int budget2, int budget3, int dtype);

int pv_prune_progressive(const void *text, const void *vis, const void *q_s, const void *k_s_all,
                         const void *q_m, const void *k_m_all, int B, int Nv, int Nt, int d,
                         int H, int hd, int dtype, int budget1, int n_vis, int budget2,
                         int budget3, int32_t *text_mask, int32_t *kept1, int32_t *assign,
                         void *merged, int32_t *vis_heads, float *conf, int32_t *kept2,
                         float *score2, void *hidden2, int32_t *kept3, float *score3,
                         void *hidden3, void *workspace, size_t workspace_bytes, void *stream);

/* -------------------------------------------------------------------------
 * pv_prune_pipeline without a workspace argument, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops
 * and harnesses that forbid hipMalloc.  Same arguments (minus workspace and
 * workspace_bytes), same kernels and bit-identical results.
 *
 * The scratch is a static device array inside the library, one copy per
 * GPU, of PV_STATIC_SCRATCH_BYTES; each GPU holds it from the library's
 * first call there until the process ends.  The call allocates nothing: no
 * hipMalloc, hipFree or allocating library routine.  The first call on a GPU
 * looks up that GPU's copy (make the stream's device current, as for every
 * call).  Every call on one GPU uses the same array and leaves its contents
 * behind; nothing in it needs to start at any value.  Two calls that overlap
 * in time on one GPU (two streams, two host threads) race on the array:
 * order them on one stream or with events.
 *
 * Errors: those of pv_prune_pipeline, plus PV_ERR_SCRATCH (nothing is
 * enqueued) when pv_pipeline_workspace_bytes() of the same sizes exceeds
 * PV_STATIC_SCRATCH_BYTES, and PV_ERR_HIP if the array's device address
 * cannot be found.
 * ---------------------------------------------------------------------- */
#define PV_STATIC_SCRATCH_BYTES (64u << 20)

int pv_prune_pipeline_noalloc(const void *vis, const void *anchors, const void *q,
                              const void *k_full, const void *v_full, const int32_t *heads_host,
                              int n_heads, int B, int Nv, int Nt, int d, int H, int hd, int dtype,
                              int budget1, int budget2, int32_t *kept1, float *score1,
                              int32_t *assign, void *merged, void *k1, void *v1, int32_t *kept2,
                              float *score2, void *hidden2, void *k2, void *v2, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* PROVIP_H */
