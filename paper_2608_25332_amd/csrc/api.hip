// C ABI of libprovip: argument checks, workspace layout, kernel sequence.
// See include/provip.h for the contract of every entry point.
#include "provip.h"

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include <mutex>
#include <vector>

#include "pv_jobs.h"
#include "pv_launch.h"

#define PV_API extern "C" __attribute__((visibility("default")))

namespace {

constexpr size_t kAlign = 256;

// Bump allocator over the caller's workspace; with base == nullptr it only
// measures, so the size query and the call share one layout.
struct Carve {
    char *base;
    size_t off = 0;
    explicit Carve(void *b) : base((char *)b) {}
    template <typename T>
    T *take(size_t n) {
        off = (off + kAlign - 1) / kAlign * kAlign;
        T *p = base ? (T *)(base + off) : nullptr;
        off += n * sizeof(T);
        return p;
    }
};

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

size_t round_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Widths the matrix-core kernels stream: embedding rows in 128-byte k chunks,
// head rows in 64-byte windows with a whole number of 128-byte chunks for
// fp32 (a multiple of 32 elements either way).  A row of another width (any
// multiple of 8 elements) is copied into a zero-padded row of the next such
// width first; zeros change no dot product and no norm.
int padded_d(int d, int esz) { return (d * esz + 127) / 128 * 128 / esz; }
int padded_hd(int hd) { return (hd + 31) / 32 * 32; }

// Launches the kernels of one call.  With events, events[i] is recorded
// before kernel i and events[n] after the last one; with reps > 1 every
// kernel is launched reps times back to back between its two events (the
// kernels are idempotent: none reads what it writes).
struct Trace {
    void *const *ev;
    int n_ev;
    const char **names;
    int reps;
    hipStream_t st;
    int launched = 0;
    // every handle a call may record must exist (checked before any launch)
    bool handles_ok() const {
        for (int i = 0; ev && i < n_ev; ++i)
            if (!ev[i]) return false;
        return true;
    }
    template <typename F>
    bool launch(const char *name, F f) {
        if (ev && launched < n_ev - 1) {
            if (hipEventRecord((hipEvent_t)ev[launched], st) != hipSuccess) return false;
            if (names) names[launched] = name;
        }
        for (int r = 0; r < reps; ++r)
            if (f() != hipSuccess) return false;
        ++launched;
        return true;
    }
    bool after_all() {
        if (ev && launched >= 1 && n_ev >= 1) {
            int i = launched < n_ev - 1 ? launched : n_ev - 1;
            return hipEventRecord((hipEvent_t)ev[i], st) == hipSuccess;
        }
        return true;
    }
};

long long n_tiles(int rows_m, int rows_n, int B, int t) {
    return (long long)((rows_m + t - 1) / t) * ((rows_n + t - 1) / t) * B;
}

// k slices of a split-k product: about `target` workgroups (768: three per CU
// of 256, as three 48 KB LDS rings fit one CU; 512 for the 64 KB rings of the
// wide cosine tiles), at least four 128-byte chunks in every slice.
int pick_slices(long long tiles, int nchunks, int target = 768, bool whole_round = false) {
    // whole_round: no more workgroups than target (a second partial round of
    // workgroups would cost a whole extra round of the ring)
    long long ks = whole_round ? target / tiles : (target + tiles / 2) / tiles;
    const long long max_ks = nchunks / 4 > 1 ? nchunks / 4 : 1;
    if (ks > max_ks) ks = max_ks;
    if (ks < 1) ks = 1;
    return (int)ks;
}

struct DedupPlan {
    int nch;                       // 128-byte k chunks per row
    bool cos_full;                 // cosine in one full-k pass (small inputs)
    int ks_cos, njt;               // cosine: k slices, token tiles of the row sums
    int Mp;
    bool gram_big;                 // full-k 128x128 tiles (operands streamed into LDS)
    int ks_gram, ntn;              // split-k slices (small) / column tiles (big)
    bool gram_wide;                // split-k Gram on the wide tiles
    // workspace
    bool lists;                    // merge reads bucketed member lists
    float *cpart, *ssv, *ssa, *M, *rowsum, *invn, *p, *gpart, *best_val;
    int32_t *pruned, *assign, *best_slot, *mcount, *mstart, *mlist;
    size_t bytes;
};

DedupPlan plan_dedup(void *ws, int B, int Nv, int Nt, int d, int esz, int budget, bool want_p,
                     bool want_assign, bool want_merged) {
    DedupPlan P;
    P.nch = d * esz / 128;
    const int T = pv::kSplitTile;
    // wide cosine tiles: two workgroups per CU (512 for the chip)
    P.ks_cos = pv::cos_uses_wide_tiles(Nt, Nv)
                   ? pick_slices(n_tiles(Nv, Nt, B, pv::kWideTile), P.nch, 512, true)
                   : pick_slices(n_tiles(Nv, Nt, B, T), P.nch);
    P.cos_full = pv::cos_use_full(B, Nv, Nt, d * esz);
    P.njt = P.cos_full ? pv::cos_full_row_tiles(Nv) : pv::cos_row_tiles(Nv);
    P.Mp = Nv - budget;
    const int Mp1 = P.Mp > 0 ? P.Mp : 1;
    P.gram_big = (long long)((Mp1 + pv::kGramTileM - 1) / pv::kGramTileM) *
                     ((budget + pv::kGramTileN - 1) / pv::kGramTileN) * B >= 128;
    P.ks_gram = P.gram_big ? 1 : pick_slices(n_tiles(Mp1, budget, B, T), P.nch);
    {
        // a single round of at most one workgroup per CU when the slice cap
        // leaves between one and two workgroups per CU: the CUs that would
        // hold two set the kernel's time
        const long long t = n_tiles(Mp1, budget, B, T);
        if (t * P.ks_gram > 256 && t * P.ks_gram < 512 && 256 / t >= 1) P.ks_gram = (int)(256 / t);
        else if (t * P.ks_gram > 768 && t * P.ks_gram < 1536 && 768 / t >= 1) P.ks_gram = (int)(768 / t);
    }
    // The wide split-k tiles (two workgroups per CU, a whole round of them)
    // when they load fewer bytes on the busiest CU: a CU streams about the
    // same bytes per second whatever its tiles, so the CU with the most bytes
    // to load sets the kernel's time.
    P.gram_wide = false;
    if (!P.gram_big) {
        const long long tw = (long long)((Mp1 + pv::kGramWideM - 1) / pv::kGramWideM) *
                             ((budget + pv::kGramWideN - 1) / pv::kGramWideN) * B;
        const int ksw = pick_slices(tw, P.nch, 512, true);
        // row chunks the busiest CU loads (workgroups go round-robin to the
        // 256 CUs)
        auto busiest = [&](long long tiles, int ks, int rows) {
            return (double)((tiles * ks + 255) / 256) * rows * ((double)P.nch / ks);
        };
        const double sq = busiest(n_tiles(Mp1, budget, B, T), P.ks_gram, 2 * T);
        const double wd = busiest(tw, ksw, pv::kGramWideM + pv::kGramWideN);
        if (wd < 0.8 * sq) {
            P.gram_wide = true;
            P.ks_gram = ksw;
        }
    }
    P.ntn = P.gram_big ? (budget + pv::kGramTileN - 1) / pv::kGramTileN : 1;
    Carve c(ws);
    if (P.cos_full) {
        P.cpart = P.ssv = P.ssa = nullptr;
    } else {
        P.cpart = c.take<float>((size_t)P.ks_cos * B * Nt * Nv);
        P.ssv = c.take<float>((size_t)P.ks_cos * B * Nv);
        P.ssa = c.take<float>((size_t)P.ks_cos * B * Nt);
    }
    P.M = c.take<float>((size_t)B * Nt * Nv);
    P.rowsum = c.take<float>((size_t)B * P.njt * Nt);
    P.invn = c.take<float>((size_t)B * Nv);
    P.p = want_p ? c.take<float>((size_t)B * Nv) : nullptr;
    P.pruned = c.take<int32_t>((size_t)B * Mp1);
    P.assign = want_assign ? c.take<int32_t>((size_t)B * Nv) : nullptr;
    if (P.gram_big) {
        P.gpart = nullptr;
        P.best_val = c.take<float>((size_t)B * P.ntn * Mp1);
        P.best_slot = c.take<int32_t>((size_t)B * P.ntn * Mp1);
    } else {
        P.gpart = c.take<float>((size_t)P.ks_gram * B * Mp1 * budget);
        P.best_val = nullptr;
        P.best_slot = nullptr;
    }
    P.lists = want_merged && pv::merge_uses_lists(B, budget, d * esz);
    if (P.lists) {
        const int ngroups = (budget + pv::kBucketSlotsPerGroup - 1) / pv::kBucketSlotsPerGroup;
        P.mcount = c.take<int32_t>((size_t)B * budget);
        P.mstart = c.take<int32_t>((size_t)B * budget);
        P.mlist = c.take<int32_t>((size_t)B * ngroups * Nv);
    } else {
        P.mcount = P.mstart = P.mlist = nullptr;
    }
    P.bytes = c.off + kAlign;
    return P;
}

// Workspace of a dedup call: its plan at the streamed width, plus the padded
// copies of the visual tokens and the anchors when d is not that width.
size_t dedup_total_bytes(int B, int Nv, int Nt, int d, int esz, int budget, bool want_p,
                         bool want_assign, bool want_merged) {
    const int dp = padded_d(d, esz);
    size_t b = round_up(plan_dedup(nullptr, B, Nv, Nt, dp, esz, budget, want_p, want_assign,
                                   want_merged).bytes);
    if (dp != d) b += round_up((size_t)B * Nv * dp * esz) + round_up((size_t)B * Nt * dp * esz);
    return b + kAlign;
}

int check_dedup(const void *vis, const void *anchors, int B, int Nv, int Nt, int d, int dtype,
                int budget, const int32_t *kept) {
    if (!vis || !anchors || !kept) return PV_ERR_NULL;
    if (dtype != PV_F32 && dtype != PV_BF16) return PV_ERR_DTYPE;
    if (B < 1 || B > 65535 || Nv < 1 || Nv > PV_MAX_TOKENS || Nt < 1 || Nt > PV_MAX_TEXT ||
        d < 8 || d > PV_MAX_DIM || d % 8 != 0)
        return PV_ERR_SHAPE;
    if (budget < 1 || budget > Nv) return PV_ERR_BUDGET;
    return PV_OK;
}

// Second stream of pv_prune_dedup_split: the assignment and merge kernels run
// there, after `selected` (recorded on the main stream once the kept list
// exists); `merged_done` is recorded there after the last of them.
struct Fork {
    hipStream_t stream;
    hipEvent_t selected;
    hipEvent_t merged_done;
};

// The kernels of the dedup up to the top-N_1: the cosine to the anchors,
// centring and max-pool into p, and the selection (kept, the pruned list
// and, with slot_of, each kept token's own slot).
bool launch_front(Trace &tr, const DedupPlan &P, int dt, const void *vis, const void *anchors,
                  const int32_t *anchor_mask, int B, int Nv, int Nt, int d, int budget, float *p,
                  int32_t *kept, int32_t *slot_of, hipStream_t st) {
    if (P.cos_full) {
        if (!tr.launch("cos_full", [&] {
                return pv::launch_cos_full(dt, vis, anchors, B, Nv, Nt, d, P.M, P.rowsum, P.invn,
                                           st);
            }))
            return false;
    } else {
        if (!tr.launch("cos_partial", [&] {
                return pv::launch_cos_partial(dt, vis, anchors, B, Nv, Nt, d, P.ks_cos, P.cpart,
                                              P.ssv, P.ssa, st);
            }))
            return false;
        if (!tr.launch("cos_reduce", [&] {
                return pv::launch_cos_reduce(P.cpart, P.ssv, P.ssa, B, Nv, Nt, P.ks_cos, P.M,
                                             P.rowsum, P.invn, st);
            }))
            return false;
    }
    return tr.launch("center", [&] {
               return pv::launch_center(P.M, P.rowsum, anchor_mask, P.njt, B, Nt, Nv, p, st);
           }) &&
           tr.launch("select", [&] {
               return pv::launch_select(p, B, Nv, budget, kept, P.pruned, slot_of, st);
           });
}

int dedup_impl(const void *vis, const void *anchors, int B, int Nv, int Nt, int d, int dtype,
               int budget, int32_t *kept, float *score, int32_t *assign, void *merged,
               void *workspace, size_t ws_bytes, void *stream, void *const *events, int n_events,
               int reps, int *n_kernels, const char **names, const Fork *fork = nullptr,
               const int32_t *anchor_mask = nullptr) {
    if (reps < 1) return PV_ERR_SHAPE;
    int rc = check_dedup(vis, anchors, B, Nv, Nt, d, dtype, budget, kept);
    if (rc != PV_OK) return rc;
    if (anchor_mask && (uintptr_t)anchor_mask % 4) return PV_ERR_ALIGN;
    const bool need_assign = assign != nullptr || merged != nullptr;
    const int esz = (dtype == PV_BF16) ? 2 : 4;
    const int dp = padded_d(d, esz);  // the width the products stream
    if (!workspace) return PV_ERR_WORKSPACE;
    if (ws_bytes < dedup_total_bytes(B, Nv, Nt, d, esz, budget, score == nullptr,
                                     need_assign && !assign, merged != nullptr))
        return PV_ERR_WORKSPACE;
    for (const void *p : {vis, anchors, (const void *)kept, (const void *)score,
                          (const void *)assign, (const void *)merged, (const void *)workspace})
        if (p && !aligned16(p)) return PV_ERR_ALIGN;
    // carve from a 256-aligned start
    char *wsa = (char *)(((uintptr_t)workspace + kAlign - 1) / kAlign * kAlign);
    DedupPlan P = plan_dedup(wsa, B, Nv, Nt, dp, esz, budget, score == nullptr,
                             need_assign && !assign, merged != nullptr);
    float *p = score ? score : P.p;
    int32_t *asg = assign ? assign : P.assign;
    const int dt = (dtype == PV_BF16) ? pv::kBF16 : pv::kF32;
    hipStream_t st = (hipStream_t)stream;
    Trace tr{events, n_events, names, reps, st};
    if (!tr.handles_ok()) return PV_ERR_NULL;
    // the rows the products read: the inputs, or their zero-padded copies
    const void *vis_k = vis, *anc_k = anchors;
    if (dp != d) {
        char *vp = wsa + round_up(P.bytes);
        char *ap = vp + round_up((size_t)B * Nv * dp * esz);
        if (!tr.launch("pad", [&] {
                return pv::launch_pad_rows(vis, vp, (long long)B * Nv, d * esz, dp * esz, st);
            }) ||
            !tr.launch("pad", [&] {
                return pv::launch_pad_rows(anchors, ap, (long long)B * Nt, d * esz, dp * esz, st);
            }))
            return PV_ERR_HIP;
        vis_k = vp;
        anc_k = ap;
    }
    if (!launch_front(tr, P, dt, vis_k, anc_k, anchor_mask, B, Nv, Nt, dp, budget, p, kept,
                      need_assign ? asg : nullptr, st))
        return PV_ERR_HIP;
    hipStream_t sm = st;  // stream of the assignment and merge kernels
    if (fork) {
        if (hipEventRecord(fork->selected, st) != hipSuccess ||
            hipStreamWaitEvent(fork->stream, fork->selected, 0) != hipSuccess)
            return PV_ERR_HIP;
        sm = fork->stream;
    }
    if (need_assign && P.Mp > 0) {
        if (P.gram_big) {
            if (!tr.launch("gram_tile", [&] {
                    return pv::launch_gram_tile(dt, vis_k, B, Nv, dp, kept, budget, P.pruned, P.Mp,
                                                P.invn, P.best_val, P.best_slot, asg, sm);
                }))
                return PV_ERR_HIP;
            if (P.ntn > 1) {
                if (!tr.launch("gram_finish", [&] {
                        return pv::launch_gram_finish(P.best_val, P.best_slot, B, P.ntn, P.Mp, Nv,
                                                      P.pruned, asg, sm);
                    }))
                    return PV_ERR_HIP;
            }
        } else {
            if (!tr.launch("gram_partial", [&] {
                    return pv::launch_gram_partial(dt, vis_k, B, Nv, dp, kept, budget, P.pruned,
                                                   P.Mp, P.ks_gram, P.gpart, P.gram_wide, sm);
                }))
                return PV_ERR_HIP;
            if (!tr.launch("gram_reduce", [&] {
                    return pv::launch_gram_reduce(P.gpart, B, P.Mp, budget, Nv, P.ks_gram, P.invn,
                                                  P.pruned, kept, asg, sm);
                }))
                return PV_ERR_HIP;
        }
    }
    if (merged && P.lists) {
        if (!tr.launch("bucket", [&] {
                return pv::launch_bucket(asg, B, Nv, budget, P.mcount, P.mstart, P.mlist, sm);
            }))
            return PV_ERR_HIP;
        if (!tr.launch("merge", [&] {
                return pv::launch_merge_csr(dt, vis, B, Nv, d, budget, P.mcount, P.mstart, P.mlist,
                                            merged, sm);
            }))
            return PV_ERR_HIP;
    } else if (merged) {
        if (!tr.launch("merge", [&] {
                return pv::launch_merge(dt, vis, B, Nv, d, budget, asg, merged, sm);
            }))
            return PV_ERR_HIP;
    }
    if (fork && hipEventRecord(fork->merged_done, sm) != hipSuccess) return PV_ERR_HIP;
    if (!tr.after_all()) return PV_ERR_HIP;
    if (n_kernels) *n_kernels = tr.launched;
    return PV_OK;
}

struct HeadPlan {
    int nrb;
    float *partial;
    float *stats;  // row statistics of the split score form
    float *v;
    size_t bytes;
};

HeadPlan plan_head(void *ws, int B, int Nt, int N, int n_heads, bool want_v) {
    HeadPlan P;
    P.nrb = (Nt + 15) / 16;
    Carve c(ws);
    P.partial = c.take<float>((size_t)B * n_heads * P.nrb * N);
    P.stats = c.take<float>(pv::score_split_stats_bytes(B, n_heads, Nt, N) / sizeof(float));
    P.v = want_v ? c.take<float>((size_t)B * N) : nullptr;
    P.bytes = c.off + kAlign;
    return P;
}

// Workspace of a head-aware call: its plan, plus zero-padded copies of Q and
// K when hd is not a streamed width.
size_t head_total_bytes(int B, int H, int Nt, int N, int hd, int esz, int n_heads, bool want_v) {
    size_t b = round_up(plan_head(nullptr, B, Nt, N, n_heads, want_v).bytes);
    const int hp = padded_hd(hd);
    if (hp != hd) b += round_up((size_t)B * H * Nt * hp * esz) + round_up((size_t)B * H * N * hp * esz);
    return b + kAlign;
}

int check_qk(const void *q, const void *k, int B, int H, int Nt, int N, int hd, int dtype) {
    if (!q || !k) return PV_ERR_NULL;
    if (dtype != PV_F32 && dtype != PV_BF16) return PV_ERR_DTYPE;
    if (B < 1 || B > 65535 || H < 1 || Nt < 1 || Nt > PV_MAX_TEXT || N < 1 || N > PV_MAX_TOKENS ||
        hd < 8 || hd > PV_MAX_HEAD_DIM || hd % 8 != 0)
        return PV_ERR_SHAPE;
    if (!aligned16(q) || !aligned16(k)) return PV_ERR_ALIGN;
    return PV_OK;
}

// heads: the host list (checked here), or NULL when the list is on the device
// (heads_dev, which cannot be checked before the kernels read it).
int check_head(const void *q, const void *k, const int32_t *heads, const int32_t *heads_dev,
               int n_heads, int B, int H, int Nt, int N, int hd, int dtype, int budget,
               const int32_t *kept) {
    if (!kept || (!heads && !heads_dev)) return PV_ERR_NULL;
    int rc = check_qk(q, k, B, H, Nt, N, hd, dtype);
    if (rc != PV_OK) return rc;
    static_assert(PV_MAX_HEADS == pv::kMaxHeadArgs, "one sample's head list fits one launch");
    if (n_heads < 1 || n_heads > H || n_heads > PV_MAX_HEADS) return PV_ERR_HEADS;
    if (!heads) {
        if ((uintptr_t)heads_dev % 4) return PV_ERR_ALIGN;
        return (budget < 1 || budget > N) ? PV_ERR_BUDGET : PV_OK;
    }
    for (int b = 0; b < B; ++b) {
        const int32_t *hb = heads + (size_t)b * n_heads;
        for (int i = 0; i < n_heads; ++i) {
            if (hb[i] < 0 || hb[i] >= H) return PV_ERR_HEADS;
            for (int j = 0; j < i; ++j)
                if (hb[j] == hb[i]) return PV_ERR_HEADS;
        }
    }
    if (budget < 1 || budget > N) return PV_ERR_BUDGET;
    return PV_OK;
}

int head_impl(const void *q, const void *k, const int32_t *heads, const int32_t *heads_dev,
              int n_heads, int B, int H, int Nt, int N, int hd, int dtype, int budget,
              int32_t *kept, float *score, void *workspace, size_t ws_bytes, void *stream,
              void *const *events, int n_events, int reps, int *n_kernels, const char **names,
              const float *row_lse = nullptr) {
    if (reps < 1) return PV_ERR_SHAPE;
    if (heads && heads_dev) return PV_ERR_HEADS;  // one list, on one side
    if (row_lse && (uintptr_t)row_lse % 4) return PV_ERR_ALIGN;
    int rc = check_head(q, k, heads, heads_dev, n_heads, B, H, Nt, N, hd, dtype, budget, kept);
    if (rc != PV_OK) return rc;
    const int esz = (dtype == PV_BF16) ? 2 : 4;
    if (!workspace || ws_bytes < head_total_bytes(B, H, Nt, N, hd, esz, n_heads, score == nullptr))
        return PV_ERR_WORKSPACE;
    for (const void *p : {q, k, (const void *)kept, (const void *)score, (const void *)workspace})
        if (p && !aligned16(p)) return PV_ERR_ALIGN;
    char *wsa = (char *)(((uintptr_t)workspace + kAlign - 1) / kAlign * kAlign);
    HeadPlan P = plan_head(wsa, B, Nt, N, n_heads, score == nullptr);
    float *v = score ? score : P.v;
    const int dt = (dtype == PV_BF16) ? pv::kBF16 : pv::kF32;
    hipStream_t st = (hipStream_t)stream;
    Trace tr{events, n_events, names, reps, st};
    if (!tr.handles_ok()) return PV_ERR_NULL;
    // the rows the products read: the inputs, or their zero-padded copies
    const int hp = padded_hd(hd);
    const void *q_k = q, *k_k = k;
    if (hp != hd) {
        char *qp = wsa + round_up(P.bytes);
        char *kp = qp + round_up((size_t)B * H * Nt * hp * esz);
        if (!tr.launch("pad", [&] {
                return pv::launch_pad_rows(q, qp, (long long)B * H * Nt, hd * esz, hp * esz, st);
            }) ||
            !tr.launch("pad", [&] {
                return pv::launch_pad_rows(k, kp, (long long)B * H * N, hd * esz, hp * esz, st);
            }))
            return PV_ERR_HIP;
        q_k = qp;
        k_k = kp;
    }

    if (!tr.launch("score_partial", [&] {
            return pv::launch_score_partial(dt, q_k, k_k, heads, heads_dev, row_lse, B, H, Nt, N,
                                            hp, hd, n_heads, P.partial, P.stats, st);
        }))
        return PV_ERR_HIP;
    const float inv_norm = (float)(1.0 / ((double)Nt * (double)n_heads));
    if (!tr.launch("score_select", [&] {
            const int parts = pv::score_parts(dt, B, H, n_heads, Nt, N, hp);
            return pv::launch_score_select(P.partial, B, n_heads * parts, N, inv_norm, v, budget,
                                           kept, st);
        }))
        return PV_ERR_HIP;
    if (!tr.after_all()) return PV_ERR_HIP;
    if (n_kernels) *n_kernels = tr.launched;
    return PV_OK;
}

size_t vis_heads_bytes(int B, int H, int Nt) {
    Carve c(nullptr);
    c.take<float>((size_t)B * H * ((Nt + 15) / 16));
    return c.off + kAlign;
}

// The same plus zero-padded copies of Q and K when hd is not a streamed width.
size_t vis_heads_total_bytes(int B, int H, int Nt, int N, int hd, int esz) {
    size_t b = round_up(vis_heads_bytes(B, H, Nt));
    const int hp = padded_hd(hd);
    if (hp != hd) b += round_up((size_t)B * H * Nt * hp * esz) + round_up((size_t)B * H * N * hp * esz);
    return b + kAlign;
}

int vis_heads_impl(const void *q, const void *k, int B, int H, int Nt, int N, int hd, int dtype,
                   int n_vis, int32_t *heads_out, float *conf, void *workspace, size_t ws_bytes,
                   void *stream, void *const *events, int n_events, int reps, int *n_kernels,
                   const char **names, const int32_t *row_mask = nullptr,
                   const float *row_lse = nullptr) {
    if (reps < 1) return PV_ERR_SHAPE;
    if (!heads_out) return PV_ERR_NULL;
    if (row_mask && (uintptr_t)row_mask % 4) return PV_ERR_ALIGN;
    if (row_lse && (uintptr_t)row_lse % 4) return PV_ERR_ALIGN;
    int rc = check_qk(q, k, B, H, Nt, N, hd, dtype);
    if (rc != PV_OK) return rc;
    if (H > PV_MAX_HEADS || n_vis < 1 || n_vis > H) return PV_ERR_HEADS;
    const int esz = (dtype == PV_BF16) ? 2 : 4;
    if (!workspace || ws_bytes < vis_heads_total_bytes(B, H, Nt, N, hd, esz))
        return PV_ERR_WORKSPACE;
    for (const void *p : {(const void *)heads_out, (const void *)conf, (const void *)workspace})
        if (p && !aligned16(p)) return PV_ERR_ALIGN;
    char *wsa = (char *)(((uintptr_t)workspace + kAlign - 1) / kAlign * kAlign);
    float *part = (float *)wsa;
    const int dt = (dtype == PV_BF16) ? pv::kBF16 : pv::kF32;
    hipStream_t st = (hipStream_t)stream;
    Trace tr{events, n_events, names, reps, st};
    if (!tr.handles_ok()) return PV_ERR_NULL;
    // the rows the products read: the inputs, or their zero-padded copies
    const int hp = padded_hd(hd);
    const void *q_k = q, *k_k = k;
    if (hp != hd) {
        char *qp = wsa + round_up(vis_heads_bytes(B, H, Nt));
        char *kp = qp + round_up((size_t)B * H * Nt * hp * esz);
        if (!tr.launch("pad", [&] {
                return pv::launch_pad_rows(q, qp, (long long)B * H * Nt, hd * esz, hp * esz, st);
            }) ||
            !tr.launch("pad", [&] {
                return pv::launch_pad_rows(k, kp, (long long)B * H * N, hd * esz, hp * esz, st);
            }))
            return PV_ERR_HIP;
        q_k = qp;
        k_k = kp;
    }
    if (!tr.launch("head_conf", [&] {
            return pv::launch_head_conf(dt, q_k, k_k, row_mask, row_lse, B, H, Nt, N, hp, hd, part,
                                        st);
        }))
        return PV_ERR_HIP;
    if (!tr.launch("conf_select", [&] {
            return pv::launch_conf_select(part, B, H, Nt, conf, n_vis, heads_out, st);
        }))
        return PV_ERR_HIP;
    if (!tr.after_all()) return PV_ERR_HIP;
    if (n_kernels) *n_kernels = tr.launched;
    return PV_OK;
}

struct TextPlan {
    int ks;
    float *part, *ssv, *ssa, *G;
    size_t bytes;
};

TextPlan plan_text(void *ws, int B, int Nt, int d, int esz);

// Workspace of the critical-text call, with a zero-padded copy of the text
// rows when d is not a streamed width.
size_t text_total_bytes(int B, int Nt, int d, int esz) {
    const int dp = padded_d(d, esz);
    size_t b = round_up(plan_text(nullptr, B, Nt, dp, esz).bytes);
    if (dp != d) b += round_up((size_t)B * Nt * dp * esz);
    return b + kAlign;
}

TextPlan plan_text(void *ws, int B, int Nt, int d, int esz) {
    TextPlan P;
    const int nch = d * esz / 128;
    P.ks = pv::cos_uses_wide_tiles(Nt, Nt) ? pick_slices(n_tiles(Nt, Nt, B, pv::kWideTile), nch, 512, true)
                                            : pick_slices(n_tiles(Nt, Nt, B, pv::kSplitTile), nch);
    Carve c(ws);
    P.part = c.take<float>((size_t)P.ks * B * Nt * Nt);
    P.ssv = c.take<float>((size_t)P.ks * B * Nt);
    P.ssa = c.take<float>((size_t)P.ks * B * Nt);
    P.G = c.take<float>((size_t)B * Nt * Nt);
    P.bytes = c.off + kAlign;
    return P;
}

int text_impl(const void *text, int B, int Nt, int d, int dtype, int32_t *mask, int32_t *count,
              float *r, void *workspace, size_t ws_bytes, void *stream, void *const *events,
              int n_events, int reps, int *n_kernels, const char **names) {
    if (reps < 1) return PV_ERR_SHAPE;
    if (!text || !mask || !count) return PV_ERR_NULL;
    if (dtype != PV_F32 && dtype != PV_BF16) return PV_ERR_DTYPE;
    if (B < 1 || B > 65535 || Nt < 1 || Nt > PV_MAX_TEXT || d < 8 || d > PV_MAX_DIM || d % 8)
        return PV_ERR_SHAPE;
    const int esz = dtype == PV_BF16 ? 2 : 4;
    if (!workspace || ws_bytes < text_total_bytes(B, Nt, d, esz)) return PV_ERR_WORKSPACE;
    for (const void *p : {text, (const void *)mask, (const void *)count, (const void *)r,
                          (const void *)workspace})
        if (p && !aligned16(p)) return PV_ERR_ALIGN;
    char *wsa = (char *)(((uintptr_t)workspace + kAlign - 1) / kAlign * kAlign);
    const int dp = padded_d(d, esz);  // the width the product streams
    TextPlan P = plan_text(wsa, B, Nt, dp, esz);
    const int dt = (dtype == PV_BF16) ? pv::kBF16 : pv::kF32;
    hipStream_t st = (hipStream_t)stream;
    Trace tr{events, n_events, names, reps, st};
    if (!tr.handles_ok()) return PV_ERR_NULL;
    const void *text_k = text;
    if (dp != d) {
        char *tp = wsa + round_up(P.bytes);
        if (!tr.launch("pad", [&] {
                return pv::launch_pad_rows(text, tp, (long long)B * Nt, d * esz, dp * esz, st);
            }))
            return PV_ERR_HIP;
        text_k = tp;
    }
    // E E^T: the text rows are both operands of the split-k product
    if (!tr.launch("text_gram", [&] {
            return pv::launch_cos_partial(dt, text_k, text_k, B, Nt, Nt, dp, P.ks, P.part, P.ssv,
                                          P.ssa, st);
        }))
        return PV_ERR_HIP;
    if (!tr.launch("text_gram_sum", [&] {
            return pv::launch_text_gram_sum(P.part, B, Nt, P.ks, P.G, st);
        }))
        return PV_ERR_HIP;
    if (!tr.launch("text_rank", [&] {
            return pv::launch_text_rank(P.G, B, Nt, r, mask, count, st);
        }))
        return PV_ERR_HIP;
    if (!tr.after_all()) return PV_ERR_HIP;
    if (n_kernels) *n_kernels = tr.launched;
    return PV_OK;
}

}  // namespace

PV_API const char *pv_status_string(int status) {
    switch (status) {
        case PV_OK: return "ok";
        case PV_ERR_NULL: return "a required pointer is NULL";
        case PV_ERR_SHAPE: return "a size is out of range or not a supported multiple";
        case PV_ERR_BUDGET: return "budget must be in [1, number of tokens]";
        case PV_ERR_HEADS: return "head list empty, out of range or repeated";
        case PV_ERR_DTYPE: return "dtype must be PV_F32 or PV_BF16";
        case PV_ERR_WORKSPACE: return "workspace missing or smaller than the query";
        case PV_ERR_HIP: return "kernel launch failed";
        case PV_ERR_ALIGN: return "pointer, row size or stride not 16-byte aligned";
        case PV_ERR_SCRATCH:
            return "the problem needs more scratch than the library's static buffer holds";
    }
    return "unknown status";
}

PV_API int pv_version(void) { return (1 << 16) | 0; }

PV_API size_t pv_dedup_workspace_bytes(int B, int Nv, int Nt, int d, int budget, int dtype) {
    if (B < 1 || Nv < 1 || Nt < 1 || d < 8 || budget < 1 || budget > Nv) return 0;
    if (dtype != PV_F32 && dtype != PV_BF16) return 0;
    // sized for the case that needs the most: no score or assign output
    return dedup_total_bytes(B, Nv, Nt, d, dtype == PV_BF16 ? 2 : 4, budget, true, true, true);
}

PV_API int pv_prune_dedup(const void *vis, const void *anchors, int B, int Nv, int Nt, int d,
                          int dtype, int budget, int32_t *kept, float *score, int32_t *assign,
                          void *merged, void *workspace, size_t workspace_bytes, void *stream) {
    return dedup_impl(vis, anchors, B, Nv, Nt, d, dtype, budget, kept, score, assign, merged,
                      workspace, workspace_bytes, stream, nullptr, 0, 1, nullptr, nullptr);
}

PV_API int pv_prune_dedup_timed(const void *vis, const void *anchors, int B, int Nv, int Nt, int d,
                                int dtype, int budget, int32_t *kept, float *score,
                                int32_t *assign, void *merged, void *workspace,
                                size_t workspace_bytes, void *stream, void *const *events,
                                int n_events, int reps, int *n_kernels, const char **names) {
    return dedup_impl(vis, anchors, B, Nv, Nt, d, dtype, budget, kept, score, assign, merged,
                      workspace, workspace_bytes, stream, events, n_events, reps, n_kernels, names);
}

PV_API int pv_prune_dedup_split(const void *vis, const void *anchors, int B, int Nv, int Nt, int d,
                                int dtype, int budget, int32_t *kept, float *score,
                                int32_t *assign, void *merged, void *workspace,
                                size_t workspace_bytes, void *stream, void *merge_stream,
                                void *selected, void *merged_done) {
    if (!merge_stream || !selected || !merged_done) return PV_ERR_NULL;
    const Fork f{(hipStream_t)merge_stream, (hipEvent_t)selected, (hipEvent_t)merged_done};
    return dedup_impl(vis, anchors, B, Nv, Nt, d, dtype, budget, kept, score, assign, merged,
                      workspace, workspace_bytes, stream, nullptr, 0, 1, nullptr, nullptr, &f);
}

PV_API int pv_prune_dedup_masked(const void *vis, const void *anchors, const int32_t *anchor_mask,
                                 int B, int Nv, int Nt, int d, int dtype, int budget,
                                 int32_t *kept, float *score, int32_t *assign, void *merged,
                                 void *workspace, size_t workspace_bytes, void *stream) {
    if (!anchor_mask) return PV_ERR_NULL;
    return dedup_impl(vis, anchors, B, Nv, Nt, d, dtype, budget, kept, score, assign, merged,
                      workspace, workspace_bytes, stream, nullptr, 0, 1, nullptr, nullptr, nullptr,
                      anchor_mask);
}

PV_API int pv_prune_dedup_masked_timed(const void *vis, const void *anchors,
                                       const int32_t *anchor_mask, int B, int Nv, int Nt, int d,
                                       int dtype, int budget, int32_t *kept, float *score,
                                       int32_t *assign, void *merged, void *workspace,
                                       size_t workspace_bytes, void *stream, void *const *events,
                                       int n_events, int reps, int *n_kernels, const char **names) {
    if (!anchor_mask) return PV_ERR_NULL;
    return dedup_impl(vis, anchors, B, Nv, Nt, d, dtype, budget, kept, score, assign, merged,
                      workspace, workspace_bytes, stream, events, n_events, reps, n_kernels, names,
                      nullptr, anchor_mask);
}

PV_API size_t pv_critical_text_workspace_bytes(int B, int Nt, int d, int dtype) {
    if (B < 1 || Nt < 1 || d < 8 || (dtype != PV_F32 && dtype != PV_BF16)) return 0;
    return text_total_bytes(B, Nt, d, dtype == PV_BF16 ? 2 : 4);
}

PV_API int pv_critical_text(const void *text, int B, int Nt, int d, int dtype, int32_t *mask,
                            int32_t *count, float *r, void *workspace, size_t workspace_bytes,
                            void *stream) {
    return text_impl(text, B, Nt, d, dtype, mask, count, r, workspace, workspace_bytes, stream,
                     nullptr, 0, 1, nullptr, nullptr);
}

PV_API int pv_critical_text_timed(const void *text, int B, int Nt, int d, int dtype, int32_t *mask,
                                  int32_t *count, float *r, void *workspace,
                                  size_t workspace_bytes, void *stream, void *const *events,
                                  int n_events, int reps, int *n_kernels, const char **names) {
    return text_impl(text, B, Nt, d, dtype, mask, count, r, workspace, workspace_bytes, stream,
                     events, n_events, reps, n_kernels, names);
}

PV_API size_t pv_head_aware_workspace_bytes(int B, int H, int Nt, int N, int hd, int n_heads,
                                            int budget, int dtype) {
    (void)budget;
    if (B < 1 || H < 1 || Nt < 1 || N < 1 || hd < 1 || n_heads < 1) return 0;
    if (dtype != PV_F32 && dtype != PV_BF16) return 0;
    return head_total_bytes(B, H, Nt, N, hd, dtype == PV_BF16 ? 2 : 4, n_heads, true);
}

PV_API int pv_prune_head_aware(const void *q, const void *k, const int32_t *heads_host, int n_heads,
                               int B, int H, int Nt, int N, int hd, int dtype, int budget,
                               int32_t *kept, float *score, void *workspace, size_t workspace_bytes,
                               void *stream) {
    if (!heads_host) return PV_ERR_NULL;
    return head_impl(q, k, heads_host, nullptr, n_heads, B, H, Nt, N, hd, dtype, budget, kept,
                     score, workspace, workspace_bytes, stream, nullptr, 0, 1, nullptr, nullptr);
}

PV_API int pv_prune_head_aware_timed(const void *q, const void *k, const int32_t *heads_host,
                                     int n_heads, int B, int H, int Nt, int N, int hd, int dtype,
                                     int budget, int32_t *kept, float *score, void *workspace,
                                     size_t workspace_bytes, void *stream, void *const *events,
                                     int n_events, int reps, int *n_kernels, const char **names) {
    if (!heads_host) return PV_ERR_NULL;
    return head_impl(q, k, heads_host, nullptr, n_heads, B, H, Nt, N, hd, dtype, budget, kept,
                     score, workspace, workspace_bytes, stream, events, n_events, reps, n_kernels,
                     names);
}

PV_API int pv_prune_head_aware_dev(const void *q, const void *k, const int32_t *heads_dev,
                                   int n_heads, int B, int H, int Nt, int N, int hd, int dtype,
                                   int budget, int32_t *kept, float *score, void *workspace,
                                   size_t workspace_bytes, void *stream) {
    if (!heads_dev) return PV_ERR_NULL;
    return head_impl(q, k, nullptr, heads_dev, n_heads, B, H, Nt, N, hd, dtype, budget, kept,
                     score, workspace, workspace_bytes, stream, nullptr, 0, 1, nullptr, nullptr);
}

PV_API int pv_prune_head_aware_dev_timed(const void *q, const void *k, const int32_t *heads_dev,
                                         int n_heads, int B, int H, int Nt, int N, int hd,
                                         int dtype, int budget, int32_t *kept, float *score,
                                         void *workspace, size_t workspace_bytes, void *stream,
                                         void *const *events, int n_events, int reps,
                                         int *n_kernels, const char **names) {
    if (!heads_dev) return PV_ERR_NULL;
    return head_impl(q, k, nullptr, heads_dev, n_heads, B, H, Nt, N, hd, dtype, budget, kept,
                     score, workspace, workspace_bytes, stream, events, n_events, reps, n_kernels,
                     names);
}

PV_API int pv_prune_head_aware_ex(const void *q, const void *k, const int32_t *heads_host,
                                  const int32_t *heads_dev, int n_heads, int B, int H, int Nt,
                                  int N, int hd, int dtype, int budget, const float *row_lse,
                                  int32_t *kept, float *score, void *workspace,
                                  size_t workspace_bytes, void *stream) {
    return head_impl(q, k, heads_host, heads_dev, n_heads, B, H, Nt, N, hd, dtype, budget, kept,
                     score, workspace, workspace_bytes, stream, nullptr, 0, 1, nullptr, nullptr,
                     row_lse);
}

PV_API int pv_prune_head_aware_ex_timed(const void *q, const void *k, const int32_t *heads_host,
                                        const int32_t *heads_dev, int n_heads, int B, int H,
                                        int Nt, int N, int hd, int dtype, int budget,
                                        const float *row_lse, int32_t *kept, float *score,
                                        void *workspace, size_t workspace_bytes, void *stream,
                                        void *const *events, int n_events, int reps,
                                        int *n_kernels, const char **names) {
    return head_impl(q, k, heads_host, heads_dev, n_heads, B, H, Nt, N, hd, dtype, budget, kept,
                     score, workspace, workspace_bytes, stream, events, n_events, reps, n_kernels,
                     names, row_lse);
}

PV_API size_t pv_visual_heads_workspace_bytes(int B, int H, int Nt) {
    if (B < 1 || H < 1 || Nt < 1) return 0;
    return vis_heads_bytes(B, H, Nt);
}

PV_API size_t pv_visual_heads_workspace_bytes_hd(int B, int H, int Nt, int N, int hd, int dtype) {
    if (B < 1 || H < 1 || Nt < 1 || N < 1 || hd < 1) return 0;
    if (dtype != PV_F32 && dtype != PV_BF16) return 0;
    return vis_heads_total_bytes(B, H, Nt, N, hd, dtype == PV_BF16 ? 2 : 4);
}

PV_API int pv_visual_heads(const void *q, const void *k, int B, int H, int Nt, int N, int hd,
                           int dtype, int n_vis, int32_t *heads_out, float *conf, void *workspace,
                           size_t workspace_bytes, void *stream) {
    return vis_heads_impl(q, k, B, H, Nt, N, hd, dtype, n_vis, heads_out, conf, workspace,
                          workspace_bytes, stream, nullptr, 0, 1, nullptr, nullptr);
}

PV_API int pv_visual_heads_masked(const void *q, const void *k, const int32_t *row_mask, int B,
                                  int H, int Nt, int N, int hd, int dtype, int n_vis,
                                  int32_t *heads_out, float *conf, void *workspace,
                                  size_t workspace_bytes, void *stream) {
    if (!row_mask) return PV_ERR_NULL;
    return vis_heads_impl(q, k, B, H, Nt, N, hd, dtype, n_vis, heads_out, conf, workspace,
                          workspace_bytes, stream, nullptr, 0, 1, nullptr, nullptr, row_mask);
}

PV_API int pv_visual_heads_masked_timed(const void *q, const void *k, const int32_t *row_mask,
                                        int B, int H, int Nt, int N, int hd, int dtype, int n_vis,
                                        int32_t *heads_out, float *conf, void *workspace,
                                        size_t workspace_bytes, void *stream, void *const *events,
                                        int n_events, int reps, int *n_kernels,
                                        const char **names) {
    if (!row_mask) return PV_ERR_NULL;
    return vis_heads_impl(q, k, B, H, Nt, N, hd, dtype, n_vis, heads_out, conf, workspace,
                          workspace_bytes, stream, events, n_events, reps, n_kernels, names,
                          row_mask);
}

PV_API int pv_visual_heads_ex(const void *q, const void *k, const int32_t *row_mask,
                              const float *row_lse, int B, int H, int Nt, int N, int hd, int dtype,
                              int n_vis, int32_t *heads_out, float *conf, void *workspace,
                              size_t workspace_bytes, void *stream) {
    return vis_heads_impl(q, k, B, H, Nt, N, hd, dtype, n_vis, heads_out, conf, workspace,
                          workspace_bytes, stream, nullptr, 0, 1, nullptr, nullptr, row_mask,
                          row_lse);
}

PV_API int pv_visual_heads_ex_timed(const void *q, const void *k, const int32_t *row_mask,
                                    const float *row_lse, int B, int H, int Nt, int N, int hd,
                                    int dtype, int n_vis, int32_t *heads_out, float *conf,
                                    void *workspace, size_t workspace_bytes, void *stream,
                                    void *const *events, int n_events, int reps, int *n_kernels,
                                    const char **names) {
    return vis_heads_impl(q, k, B, H, Nt, N, hd, dtype, n_vis, heads_out, conf, workspace,
                          workspace_bytes, stream, events, n_events, reps, n_kernels, names,
                          row_mask, row_lse);
}

PV_API int pv_visual_heads_timed(const void *q, const void *k, int B, int H, int Nt, int N, int hd,
                                 int dtype, int n_vis, int32_t *heads_out, float *conf,
                                 void *workspace, size_t workspace_bytes, void *stream,
                                 void *const *events, int n_events, int reps, int *n_kernels,
                                 const char **names) {
    return vis_heads_impl(q, k, B, H, Nt, N, hd, dtype, n_vis, heads_out, conf, workspace,
                          workspace_bytes, stream, events, n_events, reps, n_kernels, names);
}

namespace {

int fill_desc(const pv_gather_desc &in, int B, int k, pv::GatherDesc &out, int64_t *blocks) {
    if (!in.src || !in.dst) return PV_ERR_NULL;
    if (in.n_src < 1 || in.groups < 1 || in.row_bytes < 16) return PV_ERR_SHAPE;
    if (!aligned16(in.src) || !aligned16(in.dst) || in.row_bytes % 16 || in.src_batch_stride % 16 ||
        in.src_group_stride % 16 || in.src_row_stride % 16 || in.dst_batch_stride % 16 ||
        in.dst_group_stride % 16 || in.dst_row_stride % 16)
        return PV_ERR_ALIGN;
    const int64_t cpr = in.row_bytes / 16;
    const int64_t per_plane = cpr * k;  // 16-byte pieces of one plane
    if (per_plane > 0x3FFFFFFF) return PV_ERR_SHAPE;
    const int64_t span = 256 * pv::kGatherIT;
    const int64_t bpp = (per_plane + span - 1) / span;
    out.src = (const char *)in.src;
    out.dst = (char *)in.dst;
    out.n_src = in.n_src;
    out.groups = in.groups;
    out.cpr = (int)cpr;
    out.bpp = (int)bpp;
    out.sb = in.src_batch_stride;
    out.sg = in.src_group_stride;
    out.sr = in.src_row_stride;
    out.db = in.dst_batch_stride;
    out.dg = in.dst_group_stride;
    out.dr = in.dst_row_stride;
    *blocks = (int64_t)B * in.groups * bpp;
    return PV_OK;
}

}  // namespace

PV_API int pv_select_topk(const float *scores, int B, int n, int k, int32_t *kept, int32_t *rest,
                          int32_t *slot_of, void *stream) {
    if (!scores || !kept) return PV_ERR_NULL;
    if (B < 1 || B > 65535 || n < 1 || n > PV_MAX_TOKENS) return PV_ERR_SHAPE;
    if (k < 1 || k > n) return PV_ERR_BUDGET;
    if (!aligned16(scores) || !aligned16(kept) || (rest && !aligned16(rest)) ||
        (slot_of && !aligned16(slot_of)))
        return PV_ERR_ALIGN;
    if (pv::launch_select(scores, B, n, k, kept, rest, slot_of, (hipStream_t)stream) != hipSuccess)
        return PV_ERR_HIP;
    return PV_OK;
}

namespace {

int make_gather(const pv_gather_desc *descs, int n_desc, const int32_t *idx, int B, int k,
                pv::GatherArgs &ga) {
    if (!descs || !idx) return PV_ERR_NULL;
    if (n_desc < 1 || n_desc > PV_MAX_GATHER || B < 1 || k < 1) return PV_ERR_SHAPE;
    if (!aligned16(idx)) return PV_ERR_ALIGN;
    memset(&ga, 0, sizeof(ga));
    ga.n = n_desc;
    int64_t run = 0;
    for (int t = 0; t < n_desc; ++t) {
        int64_t blocks = 0;
        const int rc = fill_desc(descs[t], B, k, ga.d[t], &blocks);
        if (rc != PV_OK) return rc;
        ga.bstart[t] = (int)run;
        run += blocks;
        if (run > 0x7FFFFFFF) return PV_ERR_SHAPE;
    }
    ga.bstart[n_desc] = (int)run;
    return PV_OK;
}

}  // namespace

PV_API int pv_prune_gather_batch(const pv_gather_desc *descs, int n_desc, const int32_t *idx, int B,
                                 int k, void *stream) {
    pv::GatherArgs ga;
    const int rc = make_gather(descs, n_desc, idx, B, k, ga);
    if (rc != PV_OK) return rc;
    if (pv::launch_gather(ga, idx, B, k, (hipStream_t)stream) != hipSuccess) return PV_ERR_HIP;
    return PV_OK;
}

PV_API int pv_prune_gather(const void *src, void *dst, const int32_t *idx, int B, int n_src, int k,
                           int groups, int64_t row_bytes, int64_t src_batch_stride,
                           int64_t src_group_stride, int64_t src_row_stride,
                           int64_t dst_batch_stride, int64_t dst_group_stride,
                           int64_t dst_row_stride, void *stream) {
    if (!src || !dst || !idx) return PV_ERR_NULL;
    pv_gather_desc d;
    d.src = src;
    d.dst = dst;
    d.n_src = n_src;
    d.groups = groups;
    d.row_bytes = row_bytes;
    d.src_batch_stride = src_batch_stride;
    d.src_group_stride = src_group_stride;
    d.src_row_stride = src_row_stride;
    d.dst_batch_stride = dst_batch_stride;
    d.dst_group_stride = dst_group_stride;
    d.dst_row_stride = dst_row_stride;
    return pv_prune_gather_batch(&d, 1, idx, B, k, stream);
}

// ---------------------------------------------------------------------------
// The whole pruning step in one call: dedup (with the merge), the K/V rows of
// the N_1 kept tokens, the head-aware score and top-N_2, and the compaction of
// the merged hidden rows, K and V to the N_2 kept tokens.
// ---------------------------------------------------------------------------
namespace {

struct PipeSizes {
    size_t dedup, head, slots, total;
};

PipeSizes pipe_sizes(int B, int Nv, int Nt, int d, int H, int hd, int esz, int N1, int n_heads) {
    const size_t D = round_up(dedup_total_bytes(B, Nv, Nt, d, esz, N1, false, false, true));
    const size_t Hh = round_up(head_total_bytes(B, H, Nt, N1, hd, esz, n_heads, false));
    const size_t S = round_up((size_t)B * N1 * sizeof(int32_t));  // each slot's place among the N_2
    return PipeSizes{D, Hh, S, D + Hh + S + kAlign};
}

pv_gather_desc kv_desc(const void *src, void *dst, int H, int n_src, int k, int64_t row) {
    pv_gather_desc g;
    g.src = src;
    g.dst = dst;
    g.n_src = n_src;
    g.groups = H;
    g.row_bytes = row;
    g.src_batch_stride = (int64_t)H * n_src * row;
    g.src_group_stride = (int64_t)n_src * row;
    g.src_row_stride = row;
    g.dst_batch_stride = (int64_t)H * k * row;
    g.dst_group_stride = (int64_t)k * row;
    g.dst_row_stride = row;
    return g;
}

int pipeline_impl(const void *vis, const void *anchors, const void *q, const void *k_full,
                  const void *v_full, const int32_t *heads, int n_heads, int B, int Nv, int Nt,
                  int d, int H, int hd, int dtype, int N1, int N2, int32_t *kept1, float *score1,
                  int32_t *assign, void *merged, void *k1, void *v1, int32_t *kept2, float *score2,
                  void *hidden2, void *k2, void *v2, void *workspace, size_t ws_bytes, void *stream,
                  int force_separate, void *const *events = nullptr, int n_events = 0,
                  int reps = 1, int *n_kernels = nullptr, const char **names = nullptr) {
    if (reps < 1) return PV_ERR_SHAPE;
    if (n_kernels) *n_kernels = 0;
    int rc = check_dedup(vis, anchors, B, Nv, Nt, d, dtype, N1, kept1);
    if (rc != PV_OK) return rc;
    if (!q || !k_full || !v_full || !heads || !score1 || !assign || !merged || !k1 || !v1 ||
        !kept2 || !score2 || !hidden2 || !k2 || !v2)
        return PV_ERR_NULL;
    rc = check_head(q, k1, heads, nullptr, n_heads, B, H, Nt, N1, hd, dtype, N2, kept2);
    if (rc != PV_OK) return rc;
    const int esz = (dtype == PV_BF16) ? 2 : 4;
    const PipeSizes sz = pipe_sizes(B, Nv, Nt, d, H, hd, esz, N1, n_heads);
    if (!workspace || ws_bytes < sz.total) return PV_ERR_WORKSPACE;
    const void *const ptrs[] = {vis,    anchors, q,      k_full, v_full, kept1,   score1, assign, merged,
                                k1,     v1,      kept2,  score2, hidden2, k2,     v2,     workspace};
    for (const void *p : ptrs)
        if (!aligned16(p)) return PV_ERR_ALIGN;
    const int64_t row_kv = (int64_t)hd * esz, row_h = (int64_t)d * esz;
    const pv_gather_desc g1[2] = {kv_desc(k_full, k1, H, Nv, N1, row_kv),
                                  kv_desc(v_full, v1, H, Nv, N1, row_kv)};
    pv_gather_desc g2[3] = {kv_desc(merged, hidden2, 1, N1, N2, row_h),
                            kv_desc(k1, k2, H, N1, N2, row_kv), kv_desc(v1, v2, H, N1, N2, row_kv)};
    pv::GatherArgs ga1, ga2, ga2kv;
    if ((rc = make_gather(g1, 2, kept1, B, N1, ga1)) != PV_OK) return rc;
    if ((rc = make_gather(g2, 3, kept2, B, N2, ga2)) != PV_OK) return rc;
    if ((rc = make_gather(g2 + 1, 2, kept2, B, N2, ga2kv)) != PV_OK) return rc;
    hipStream_t st = (hipStream_t)stream;
    Trace tr{events, n_events, names, reps, st};
    if (!tr.handles_ok()) return PV_ERR_NULL;
    char *wsa = (char *)(((uintptr_t)workspace + kAlign - 1) / kAlign * kAlign);
    char *ws_head = wsa + sz.dedup;
    int32_t *slot_of2 = (int32_t *)(ws_head + sz.head);

    const DedupPlan P = plan_dedup(wsa, B, Nv, Nt, d, esz, N1, false, false, true);
    const int dt = (dtype == PV_BF16) ? pv::kBF16 : pv::kF32;
    // the two chains after the top-N_1 share launches when the dedup takes
    // the split-k Gram and the plain merge, and the score its 16-row blocks
    // with every logit in registers (the same kernels' arithmetic as the
    // separate calls, so the same bits)
    const bool carry = !force_separate && padded_d(d, esz) == d && padded_hd(hd) == hd &&
                       P.Mp > 0 && !P.gram_big && !P.gram_wide && !P.lists && N1 <= 256 &&
                       pv::gram_score_supported(dt, B, n_heads, N1, hd) &&
                       !pv::score_uses_head_form(dt, B, H, n_heads, Nt, N1, hd) &&
                       !pv::score_uses_split_form(dt, B, H, n_heads, Nt, N1, hd);
    if (!carry) {
        rc = dedup_impl(vis, anchors, B, Nv, Nt, d, dtype, N1, kept1, score1, assign, merged, wsa,
                        sz.dedup, stream, nullptr, 0, 1, nullptr, nullptr);
        if (rc != PV_OK) return rc;
        if (pv::launch_gather(ga1, kept1, B, N1, st) != hipSuccess) return PV_ERR_HIP;
        rc = head_impl(q, k1, heads, nullptr, n_heads, B, H, Nt, N1, hd, dtype, N2, kept2, score2,
                       ws_head, sz.head, stream, nullptr, 0, 1, nullptr, nullptr);
        if (rc != PV_OK) return rc;
        if (pv::launch_gather(ga2, kept2, B, N2, st) != hipSuccess) return PV_ERR_HIP;
        return PV_OK;
    }
    const HeadPlan Hh = plan_head(ws_head, B, Nt, N1, n_heads, false);
    // cosine, centring, top-N_1
    if (!launch_front(tr, P, dt, vis, anchors, nullptr, B, Nv, Nt, d, N1, score1, kept1, assign,
                      st))
        return PV_ERR_HIP;
    // score blocks on the keys of the kept tokens + Gram partials
    const int ntm = (P.Mp + pv::kSplitTile - 1) / pv::kSplitTile;
    const int ntn = (N1 + pv::kSplitTile - 1) / pv::kSplitTile;
    const pv::GramJob gram{(const char *)vis, B,      Nv,  d * esz,   kept1,  N1,
                           P.pruned,          P.Mp,   ntm, ntn,       P.ks_gram, P.gpart,
                           B * P.ks_gram * ntm * ntn};
    if (!tr.launch("gram_partial+score_partial", [&] {
            return pv::launch_gram_score(dt, q, k_full, heads, B, H, Nt, N1, Nv, kept1, hd,
                                         n_heads, Hh.partial, gram, st);
        }))
        return PV_ERR_HIP;
    // the score's top-N_2 + the Gram's argmax + the K/V rows of the N_1 kept
    const float inv_norm = (float)(1.0 / ((double)Nt * (double)n_heads));
    const pv::ReduceJob rj{P.gpart, B, P.Mp, N1, Nv, P.ks_gram, P.invn, P.pruned, kept1, assign,
                           B * ((P.Mp + pv::kReduceRowsPerBlock - 1) / pv::kReduceRowsPerBlock)};
    const pv::SelectJob sj{Hh.partial, n_heads * Hh.nrb, N1, inv_norm, score2, N2, kept2, B,
                           slot_of2};
    const pv::GatherJob gj1{ga1, kept1, N1, ga1.bstart[ga1.n]};
    if (!tr.launch("gram_reduce+score_select+gather_kv1", [&] {
            return pv::launch_reduce_select_gather(rj, sj, gj1, st);
        }))
        return PV_ERR_HIP;
    // merge, with the merged rows of the N_2 kept slots written to their
    // compacted places, + K and V of the N_2 kept
    const pv::MergeCarry mc{slot_of2, (char *)hidden2, N2,
                            pv::GatherJob{ga2kv, kept2, N2, ga2kv.bstart[ga2kv.n]}};
    if (!tr.launch("merge+gather_hkv2", [&] {
            return pv::launch_merge(dt, vis, B, Nv, d, N1, assign, merged, st, &mc);
        }))
        return PV_ERR_HIP;
    if (!tr.after_all()) return PV_ERR_HIP;
    if (n_kernels) *n_kernels = tr.launched;
    return PV_OK;
}

}  // namespace

PV_API size_t pv_pipeline_workspace_bytes(int B, int Nv, int Nt, int d, int H, int hd,
                                          int n_heads, int budget1, int budget2, int dtype) {
    (void)H;
    (void)hd;
    (void)budget2;
    if (B < 1 || Nv < 1 || Nt < 1 || d < 1 || n_heads < 1 || budget1 < 1 || budget1 > Nv)
        return 0;
    if (H < 1 || hd < 1) return 0;
    return pipe_sizes(B, Nv, Nt, d, H, hd, (dtype == PV_BF16) ? 2 : 4, budget1, n_heads).total;
}

PV_API int pv_prune_pipeline(const void *vis, const void *anchors, const void *q,
                             const void *k_full, const void *v_full, const int32_t *heads_host,
                             int n_heads, int B, int Nv, int Nt, int d, int H, int hd, int dtype,
                             int budget1, int budget2, int32_t *kept1, float *score1,
                             int32_t *assign, void *merged, void *k1, void *v1, int32_t *kept2,
                             float *score2, void *hidden2, void *k2, void *v2, void *workspace,
                             size_t workspace_bytes, void *stream) {
    return pipeline_impl(vis, anchors, q, k_full, v_full, heads_host, n_heads, B, Nv, Nt, d, H, hd,
                         dtype, budget1, budget2, kept1, score1, assign, merged, k1, v1, kept2,
                         score2, hidden2, k2, v2, workspace, workspace_bytes, stream, 0);
}

PV_API int pv_prune_pipeline_separate(const void *vis, const void *anchors, const void *q,
                                      const void *k_full, const void *v_full,
                                      const int32_t *heads_host, int n_heads, int B, int Nv,
                                      int Nt, int d, int H, int hd, int dtype, int budget1,
                                      int budget2, int32_t *kept1, float *score1, int32_t *assign,
                                      void *merged, void *k1, void *v1, int32_t *kept2,
                                      float *score2, void *hidden2, void *k2, void *v2,
                                      void *workspace, size_t workspace_bytes, void *stream) {
    return pipeline_impl(vis, anchors, q, k_full, v_full, heads_host, n_heads, B, Nv, Nt, d, H, hd,
                         dtype, budget1, budget2, kept1, score1, assign, merged, k1, v1, kept2,
                         score2, hidden2, k2, v2, workspace, workspace_bytes, stream, 1);
}

PV_API int pv_prune_pipeline_timed(const void *vis, const void *anchors, const void *q,
                                   const void *k_full, const void *v_full,
                                   const int32_t *heads_host, int n_heads, int B, int Nv, int Nt,
                                   int d, int H, int hd, int dtype, int budget1, int budget2,
                                   int32_t *kept1, float *score1, int32_t *assign, void *merged,
                                   void *k1, void *v1, int32_t *kept2, float *score2,
                                   void *hidden2, void *k2, void *v2, void *workspace,
                                   size_t workspace_bytes, void *stream, void *const *events,
                                   int n_events, int reps, int *n_kernels, const char **names) {
    return pipeline_impl(vis, anchors, q, k_full, v_full, heads_host, n_heads, B, Nv, Nt, d, H, hd,
                         dtype, budget1, budget2, kept1, score1, assign, merged, k1, v1, kept2,
                         score2, hidden2, k2, v2, workspace, workspace_bytes, stream, 0, events,
                         n_events, reps, n_kernels, names);
}

// ---------------------------------------------------------------------------
// The progressive schedule in one call: critical text, pruning before the
// LLM on the critical rows, visual heads and head-aware pruning at a shallow
// layer, all-head pruning at a middle layer, with the compactions between.
// Every stage is the library's own call for that stage, so every output is
// the bit-for-bit result of those calls made in turn.
// ---------------------------------------------------------------------------
namespace {

struct ProgPlan {
    size_t text, dedup, vh, head_b, head_c;
    int32_t *count, *k2loc, *k3loc;
    char *ks, *km;
    char *ws_text, *ws_dedup, *ws_vh, *ws_head_b, *ws_head_c;
    size_t bytes;
};

ProgPlan plan_prog(void *ws, int B, int Nv, int Nt, int d, int H, int hd, int esz, int N1,
                   int n_vis, int N2, int N3, bool want_s2, bool want_s3) {
    ProgPlan P;
    P.text = text_total_bytes(B, Nt, d, esz);
    P.dedup = dedup_total_bytes(B, Nv, Nt, d, esz, N1, true, false, true);
    P.vh = vis_heads_total_bytes(B, H, Nt, N1, hd, esz);
    P.head_b = head_total_bytes(B, H, Nt, N1, hd, esz, n_vis, !want_s2);
    P.head_c = head_total_bytes(B, H, Nt, N2, hd, esz, H, !want_s3);
    Carve c(ws);
    P.ws_text = c.take<char>(P.text);
    P.ws_dedup = c.take<char>(P.dedup);
    P.ws_vh = c.take<char>(P.vh);
    P.ws_head_b = c.take<char>(P.head_b);
    P.ws_head_c = c.take<char>(P.head_c);
    P.count = c.take<int32_t>((size_t)B);
    P.k2loc = c.take<int32_t>((size_t)B * N2);
    P.k3loc = c.take<int32_t>((size_t)B * N3);
    P.ks = c.take<char>((size_t)B * H * N1 * hd * esz);
    P.km = c.take<char>((size_t)B * H * N2 * hd * esz);
    P.bytes = c.off + kAlign;
    return P;
}

int progressive_impl(const void *text, const void *vis, const void *q_s, const void *k_s_all,
                     const void *q_m, const void *k_m_all, int B, int Nv, int Nt, int d, int H,
                     int hd, int dtype, int N1, int n_vis, int N2, int N3, int32_t *text_mask,
                     int32_t *kept1, int32_t *assign, void *merged, int32_t *vis_heads,
                     float *conf, int32_t *kept2, float *score2, void *hidden2, int32_t *kept3,
                     float *score3, void *hidden3, void *workspace, size_t ws_bytes,
                     void *stream) {
    int rc = check_dedup(vis, text, B, Nv, Nt, d, dtype, N1, kept1);
    if (rc != PV_OK) return rc;
    if ((rc = check_qk(q_s, k_s_all, B, H, Nt, Nv, hd, dtype)) != PV_OK) return rc;
    if ((rc = check_qk(q_m, k_m_all, B, H, Nt, Nv, hd, dtype)) != PV_OK) return rc;
    if (!text_mask || !assign || !merged || !vis_heads || !kept2 || !hidden2 || !kept3 ||
        !hidden3)
        return PV_ERR_NULL;
    if (H > PV_MAX_HEADS || n_vis < 1 || n_vis > H) return PV_ERR_HEADS;
    if (N2 < 1 || N2 > N1 || N3 < 1 || N3 > N2) return PV_ERR_BUDGET;
    const void *const ptrs[] = {text_mask, kept1, assign, merged, vis_heads, conf, kept2,
                                score2, hidden2, kept3, score3, hidden3, workspace};
    for (const void *p : ptrs)
        if (p && !aligned16(p)) return PV_ERR_ALIGN;
    const int esz = (dtype == PV_BF16) ? 2 : 4;
    if (!workspace ||
        ws_bytes < plan_prog(nullptr, B, Nv, Nt, d, H, hd, esz, N1, n_vis, N2, N3, score2 != nullptr,
                             score3 != nullptr).bytes)
        return PV_ERR_WORKSPACE;
    char *wsa = (char *)(((uintptr_t)workspace + kAlign - 1) / kAlign * kAlign);
    const ProgPlan P = plan_prog(wsa, B, Nv, Nt, d, H, hd, esz, N1, n_vis, N2, N3,
                                 score2 != nullptr, score3 != nullptr);
    hipStream_t st = (hipStream_t)stream;
    const int64_t row_kv = (int64_t)hd * esz, row_h = (int64_t)d * esz;
    // critical text tokens (Sec. 4.2)
    rc = text_impl(text, B, Nt, d, dtype, text_mask, P.count, nullptr, P.ws_text, P.text, stream,
                   nullptr, 0, 1, nullptr, nullptr);
    if (rc != PV_OK) return rc;
    // pruning before the LLM on the critical rows (Sec. 4.3), with the merge
    rc = dedup_impl(vis, text, B, Nv, Nt, d, dtype, N1, kept1, nullptr, assign, merged,
                    P.ws_dedup, P.dedup, stream, nullptr, 0, 1, nullptr, nullptr, nullptr,
                    text_mask);
    if (rc != PV_OK) return rc;
    // the shallow layer's keys of the N1 retained tokens
    pv::GatherArgs ga;
    {
        const pv_gather_desc g = kv_desc(k_s_all, P.ks, H, Nv, N1, row_kv);
        if ((rc = make_gather(&g, 1, kept1, B, N1, ga)) != PV_OK) return rc;
        if (pv::launch_gather(ga, kept1, B, N1, st) != hipSuccess) return PV_ERR_HIP;
    }
    // visual heads over the critical rows, then head-aware pruning on them
    // (Sec. 4.4, equations for C^h, V_l, S^vis and v)
    rc = vis_heads_impl(q_s, P.ks, B, H, Nt, N1, hd, dtype, n_vis, vis_heads, conf, P.ws_vh,
                        P.vh, stream, nullptr, 0, 1, nullptr, nullptr, text_mask);
    if (rc != PV_OK) return rc;
    rc = head_impl(q_s, P.ks, nullptr, vis_heads, n_vis, B, H, Nt, N1, hd, dtype, N2, P.k2loc,
                   score2, P.ws_head_b, P.head_b, stream, nullptr, 0, 1, nullptr, nullptr);
    if (rc != PV_OK) return rc;
    // survivors of the shallow layer: token indices, merged rows, and the
    // middle layer's keys of those tokens
    if (pv::launch_compose_index(kept1, P.k2loc, B, N1, N2, kept2, st) != hipSuccess)
        return PV_ERR_HIP;
    {
        const pv_gather_desc g = kv_desc(merged, hidden2, 1, N1, N2, row_h);
        if ((rc = make_gather(&g, 1, P.k2loc, B, N2, ga)) != PV_OK) return rc;
        if (pv::launch_gather(ga, P.k2loc, B, N2, st) != hipSuccess) return PV_ERR_HIP;
        const pv_gather_desc gk = kv_desc(k_m_all, P.km, H, Nv, N2, row_kv);
        if ((rc = make_gather(&gk, 1, kept2, B, N2, ga)) != PV_OK) return rc;
        if (pv::launch_gather(ga, kept2, B, N2, st) != hipSuccess) return PV_ERR_HIP;
    }
    // the middle layer: every head (the all-head aggregation, no head
    // identification)
    std::vector<int32_t> all((size_t)B * H);
    for (int b = 0; b < B; ++b)
        for (int h = 0; h < H; ++h) all[(size_t)b * H + h] = h;
    rc = head_impl(q_m, P.km, all.data(), nullptr, H, B, H, Nt, N2, hd, dtype, N3, P.k3loc,
                   score3, P.ws_head_c, P.head_c, stream, nullptr, 0, 1, nullptr, nullptr);
    if (rc != PV_OK) return rc;
    if (pv::launch_compose_index(kept2, P.k3loc, B, N2, N3, kept3, st) != hipSuccess)
        return PV_ERR_HIP;
    {
        const pv_gather_desc g = kv_desc(hidden2, hidden3, 1, N2, N3, row_h);
        if ((rc = make_gather(&g, 1, P.k3loc, B, N3, ga)) != PV_OK) return rc;
        if (pv::launch_gather(ga, P.k3loc, B, N3, st) != hipSuccess) return PV_ERR_HIP;
    }
    return PV_OK;
}

}  // namespace

PV_API size_t pv_progressive_workspace_bytes(int B, int Nv, int Nt, int d, int H, int hd,
                                             int budget1, int n_vis, int budget2, int budget3,
                                             int dtype) {
    if (B < 1 || Nv < 1 || Nt < 1 || d < 1 || H < 1 || hd < 1 || budget1 < 1 || budget1 > Nv ||
        n_vis < 1 || n_vis > H || budget2 < 1 || budget2 > budget1 || budget3 < 1 ||
        budget3 > budget2 || (dtype != PV_F32 && dtype != PV_BF16))
        return 0;
    return plan_prog(nullptr, B, Nv, Nt, d, H, hd, dtype == PV_BF16 ? 2 : 4, budget1, n_vis,
                     budget2, budget3, false, false)
        .bytes;
}

PV_API int pv_prune_progressive(const void *text, const void *vis, const void *q_s,
                                const void *k_s_all, const void *q_m, const void *k_m_all, int B,
                                int Nv, int Nt, int d, int H, int hd, int dtype, int budget1,
                                int n_vis, int budget2, int budget3, int32_t *text_mask,
                                int32_t *kept1, int32_t *assign, void *merged,
                                int32_t *vis_heads, float *conf, int32_t *kept2, float *score2,
                                void *hidden2, int32_t *kept3, float *score3, void *hidden3,
                                void *workspace, size_t workspace_bytes, void *stream) {
    return progressive_impl(text, vis, q_s, k_s_all, q_m, k_m_all, B, Nv, Nt, d, H, hd, dtype,
                            budget1, n_vis, budget2, budget3, text_mask, kept1, assign, merged,
                            vis_heads, conf, kept2, score2, hidden2, kept3, score3, hidden3,
                            workspace, workspace_bytes, stream);
}

// ---------------------------------------------------------------------------
// The step without a workspace argument, for callers that cannot allocate.
//
// The scratch lives in this file-scope array: one copy per GPU, allocated
// when the library's code object is loaded on that GPU and held until the
// process ends.  Host code never uses the array's name as an address (on the
// host it is only a stand-in for the device symbol): the device address of
// each GPU's copy is looked up once, with that GPU current, and kept.
// ---------------------------------------------------------------------------
static __device__ __align__(256) unsigned char scratch[PV_STATIC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch[kMaxDevices];

// Device address of the current GPU's copy of `scratch` (PV_ERR_HIP if the
// lookup fails or the device id is out of range).
int scratch_of_current_device(void **out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return PV_ERR_HIP;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[dev]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return PV_ERR_HIP;
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return PV_OK;
}

}  // namespace

PV_API int pv_prune_pipeline_noalloc(const void *vis, const void *anchors, const void *q,
                                     const void *k_full, const void *v_full,
                                     const int32_t *heads_host, int n_heads, int B, int Nv,
                                     int Nt, int d, int H, int hd, int dtype, int budget1,
                                     int budget2, int32_t *kept1, float *score1, int32_t *assign,
                                     void *merged, void *k1, void *v1, int32_t *kept2,
                                     float *score2, void *hidden2, void *k2, void *v2,
                                     void *stream) {
    // the checks that need no device first, so that a rejected call touches
    // no GPU state
    int rc = check_dedup(vis, anchors, B, Nv, Nt, d, dtype, budget1, kept1);
    if (rc != PV_OK) return rc;
    if (!heads_host) return PV_ERR_NULL;
    rc = check_head(q, k_full, heads_host, nullptr, n_heads, B, H, Nt, budget1, hd, dtype,
                    budget2, kept2);
    if (rc != PV_OK) return rc;
    const int esz = (dtype == PV_BF16) ? 2 : 4;
    // the step carves its workspace from a 256-byte boundary, which the
    // array's start already is
    if (pipe_sizes(B, Nv, Nt, d, H, hd, esz, budget1, n_heads).total > (size_t)PV_STATIC_SCRATCH_BYTES)
        return PV_ERR_SCRATCH;
    void *ws = nullptr;
    if ((rc = scratch_of_current_device(&ws)) != PV_OK) return rc;
    return pipeline_impl(vis, anchors, q, k_full, v_full, heads_host, n_heads, B, Nv, Nt, d, H,
                         hd, dtype, budget1, budget2, kept1, score1, assign, merged, k1, v1,
                         kept2, score2, hidden2, k2, v2, ws, (size_t)PV_STATIC_SCRATCH_BYTES,
                         stream, 0);
}
