// Host-side launchers of the ProViP kernels (internal to libprovip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pv {

// Work another launch can carry (pv_jobs.h).
struct GatherJob;
struct ReduceJob;
struct SelectJob;
struct GramJob;
struct MergeCarry;

// Element types of the inputs (values of pv_dtype).
constexpr int kF32 = 0;
constexpr int kBF16 = 1;

constexpr int kMaxHeadArgs = 512;
struct HeadArgs {
    int32_t h[kMaxHeadArgs];
};
// The same list one byte per entry (heads < 256): entry i is byte i % 4 of
// word i / 4.  Four times the entries in the same argument bytes, so a
// large batch of (head, sample) pairs takes few launches.
constexpr int kMaxHeadArgs8 = 2048;
struct HeadArgs8 {
    uint32_t w[kMaxHeadArgs8 / 4];
};


// ---- pruning before the LLM (Sec. 4.3)
constexpr int kSplitTile = 64;  // tile edge of the split-k products
constexpr int kWideTile = 128;  // the cosine's tile edge with more than 64 anchors
// Whether the split-k cosine runs on kWideTile tiles (two workgroups per CU)
// instead of kSplitTile tiles (three per CU).
inline bool cos_uses_wide_tiles(int Nt, int Nv) { return Nt > 64 && Nv >= 512; }
int cos_row_tiles(int Nv);      // token tiles of the row sums written by cos_reduce
int cos_full_row_tiles(int Nv); // token tiles of the row sums written by cos_full
// Whether the cosine runs as one full-k pass over 16 x 16 tiles (small inputs:
// the rows it re-reads, one copy per tile row and column, stay under 48 MB).
inline bool cos_use_full(int B, int Nv, int Nt, int d_bytes) {
    const double reread = (double)B * d_bytes *
                          ((double)((Nt + 15) / 16) * Nv + (double)((Nv + 15) / 16) * Nt);
    return reread <= 48.0 * (1 << 20);
}
hipError_t launch_cos_full(int dt, const void *vis, const void *anchors, int B, int Nv, int Nt,
                           int d, float *M, float *rowsum, float *invn, hipStream_t st);
hipError_t launch_cos_partial(int dt, const void *vis, const void *anchors, int B, int Nv, int Nt,
                              int d, int KS, float *part, float *ssv, float *ssa, hipStream_t st);
hipError_t launch_cos_reduce(const float *part, const float *ssv, const float *ssa, int B, int Nv,
                             int Nt, int KS, float *M, float *rowsum, float *invn, hipStream_t st);
// row_mask [B][Nt] (device, may be NULL): rows with 0 are not anchors; a
// sample whose mask has no row set uses every row.
hipError_t launch_center(const float *M, const float *rowsum, const int32_t *row_mask, int njt,
                         int B, int Nt, int Nv, float *p, hipStream_t st);
hipError_t launch_select(const float *p, int B, int Nv, int budget, int32_t *kept, int32_t *pruned,
                         int32_t *slot_of, hipStream_t st);
// The split-k Gram's partial dot products part[KS][B][Mp][N1], on kSplitTile
// square tiles (three workgroups per CU) or, with `wide`, on kGramWideM x
// kGramWideN tiles (two per CU, each row loaded once for more outputs).
constexpr int kGramWideM = 128, kGramWideN = 96;
hipError_t launch_gram_partial(int dt, const void *vis, int B, int Nv, int d, const int32_t *kept,
                               int N1, const int32_t *pruned, int Mp, int KS, float *part,
                               bool wide, hipStream_t st);
hipError_t launch_gram_reduce(const float *part, int B, int Mp, int N1, int Nv, int KS,
                              const float *invn, const int32_t *pruned, const int32_t *kept,
                              int32_t *assign, hipStream_t st);
// Tile of the full-k Gram (pruned rows x kept rows) used for large inputs:
// kGramTileM x kGramTileN, one workgroup per CU of eight matrix waves and
// kGramProducers producer waves that issue the loads.  The full-k form is
// chosen when the product holds at least 128 such tiles (enough work to keep
// every CU busy without split-k).
constexpr int kGramTileM = 256, kGramTileN = 128, kGramProducers = 4;
hipError_t launch_gram_tile(int dt, const void *vis, int B, int Nv, int d, const int32_t *kept,
                            int N1, const int32_t *pruned, int Mp, const float *invn,
                            float *best_val, int32_t *best_slot, int32_t *assign, hipStream_t st);
hipError_t launch_gram_finish(const float *best_val, const int32_t *best_slot, int B, int ntn,
                              int Mp, int Nv, const int32_t *pruned, int32_t *assign,
                              hipStream_t st);
constexpr int kBucketSlotsPerGroup = 256;  // slots whose member lists one workgroup builds
hipError_t launch_bucket(const int32_t *assign, int B, int Nv, int N1, int32_t *mcount,
                         int32_t *mstart, int32_t *mlist, hipStream_t st);
hipError_t launch_merge_csr(int dt, const void *vis, int B, int Nv, int d, int N1,
                            const int32_t *mcount, const int32_t *mstart, const int32_t *mlist,
                            void *merged, hipStream_t st);
// Whether the merge reads member lists built by the bucket kernel instead of
// scanning the assignment in every workgroup: for batches (one extra launch
// is then cheap next to the work), and whenever the scans would read more
// than the rows they add.
inline bool merge_uses_lists(int B, int N1, int d_bytes) {
    return B > 1 || (long long)((d_bytes / 16 + 63) / 64) * N1 * 4 > d_bytes;
}
// with: the merged rows of the head-aware top-N_2 written to their compacted
// places too, and the compaction of K and V to those slots carried as extra
// workgroups (or NULL).
hipError_t launch_merge(int dt, const void *vis, int B, int Nv, int d, int N1,
                        const int32_t *assign, void *merged, hipStream_t st,
                        const MergeCarry *with = nullptr);

// ---- critical text tokens (Sec. 4.2)
hipError_t launch_text_gram_sum(const float *part, int B, int Nt, int KS, float *G,
                                hipStream_t st);
hipError_t launch_text_rank(const float *G, int B, int Nt, float *r, int32_t *mask, int32_t *count,
                            hipStream_t st);

// ---- head-aware pruning (Sec. 4.4)
// heads_dev == nullptr: the head list is heads_host (host memory); else the
// device list heads_dev (entries clamped into [0, H)).
// Whether the score runs one workgroup per (head, sample) (score_head) and
// writes one row of column sums per (sample, head) instead of one per
// 16-row block.
bool score_uses_head_form(int dt, int B, int H, int n_heads, int Nt, int N, int hd);
// Whether the score runs split over 64-key chunks of every head (two
// launches: row statistics, then column sums; one row of column sums per
// (sample, head)).
bool score_uses_split_form(int dt, int B, int H, int n_heads, int Nt, int N, int hd);
// Rows of column sums the score writes per (sample, selected head): 1 for the
// whole-head and split forms, one per 16-row block otherwise.
int score_parts(int dt, int B, int H, int n_heads, int Nt, int N, int hd);
// Bytes of the split form's row statistics (float2 per row, chunk, head and
// sample).
inline size_t score_split_stats_bytes(int B, int n_heads, int Nt, int N) {
    return (size_t)B * n_heads * ((N + 63) / 64) * Nt * 8;
}
// row_lse [B][H][Nt] (may be NULL): log-sum-exp of each row's scaled logits
// over the non-visual keys, which join the softmax normaliser.
// split_stats: workspace of score_split_stats_bytes (used by the split form).
// hd: the width of the q and k rows (a multiple of 32); hd_scale: the head
// width of the attention scale 1 / sqrt(hd_scale) (the rows may be padded
// with zeros past it).
hipError_t launch_score_partial(int dt, const void *q, const void *k, const int32_t *heads_host,
                                const int32_t *heads_dev, const float *row_lse, int B, int H,
                                int Nt, int N, int hd, int hd_scale, int n_heads, float *partial,
                                float *split_stats, hipStream_t st);
// Head confidence of every head, per 16-row block: partial[b][h][rb].
// row_mask as for launch_center: the rows summed into the confidence.
// row_lse as for launch_score_partial (may be NULL): the variance is then
// taken over the visual slice of the model's softmax.
hipError_t launch_head_conf(int dt, const void *q, const void *k, const int32_t *row_mask,
                            const float *row_lse, int B, int H, int Nt, int N, int hd,
                            int hd_scale, float *partial, hipStream_t st);
hipError_t launch_conf_select(const float *partial, int B, int H, int Nt, float *conf, int n_vis,
                              int32_t *heads, hipStream_t st);
hipError_t launch_score_select(const float *partial, int B, int nparts, int N, float inv_norm,
                               float *v, int budget, int32_t *kept, hipStream_t st);
// The one-call step after the top-N_1 at small batches (see
// head_aware_kernels.hip): the score on the keys of the kept tokens read
// through kidx ([B][N] rows of k_full, [B][H][n_src][hd]) beside the split-k
// Gram's tiles, then the score's top-N_2, the Gram's argmax and the
// compaction of K and V to the N_1 kept in one launch.  The score runs one
// 16-row block per workgroup with every logit in registers.
bool gram_score_supported(int dt, int B, int n_heads, int N, int hd);
hipError_t launch_gram_score(int dt, const void *q, const void *k_full, const int32_t *heads_host,
                             int B, int H, int Nt, int N, int n_src, const int32_t *kidx, int hd,
                             int n_heads, float *partial, const GramJob &gj, hipStream_t st);
hipError_t launch_reduce_select_gather(const ReduceJob &rj, const SelectJob &sj,
                                       const GatherJob &gj, hipStream_t st);

// ---- compaction (Sec. 4.1)
constexpr int kMaxGather = 4;
constexpr int kGatherIT = 4;  // 16-byte pieces per thread
struct GatherDesc {
    const char *src;
    char *dst;
    int n_src, groups, cpr;  // cpr: 16-byte pieces per row
    int bpp;                 // workgroups per plane (sample x head group)
    int64_t sb, sg, sr, db, dg, dr;
};
struct GatherArgs {
    GatherDesc d[kMaxGather];
    int bstart[kMaxGather + 1];  // first workgroup of each tensor; bstart[n] = total
    int n;
};
hipError_t launch_gather(const GatherArgs &ga, const int32_t *idx, int B, int k, hipStream_t st);
// dst row r = src row r (in_bytes) then zeros up to out_bytes (multiples of 16).
hipError_t launch_pad_rows(const void *src, void *dst, long long n_rows, int in_bytes,
                           int out_bytes, hipStream_t st);
// out[b][r] = base[b][idx[b][r]] (b < B, r < k; idx clamped into [0, n_base)).
hipError_t launch_compose_index(const int32_t *base, const int32_t *idx, int B, int n_base, int k,
                                int32_t *out, hipStream_t st);

}  // namespace pv
