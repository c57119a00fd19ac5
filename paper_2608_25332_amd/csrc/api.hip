// C ABI of libprovip: argument checks, workspace layout, kernel sequence.
// See include/provip.h for the contract of every entry point.
#include "provip.h"

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

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

// Records events[i] before kernel i and events[n] after the last kernel.
struct Trace {
    void *const *ev;
    int n_ev;
    int launched = 0;
    hipStream_t st;
    void before() {
        if (ev && launched < n_ev - 1) (void)hipEventRecord((hipEvent_t)ev[launched], st);
    }
    void after_all() {
        if (ev && launched >= 1 && n_ev >= 1) {
            int i = launched < n_ev - 1 ? launched : n_ev - 1;
            (void)hipEventRecord((hipEvent_t)ev[i], st);
        }
    }
};

// Pick the largest square tile whose grid still gives >= ~1 workgroup per CU
// (256 CUs); fall back to the smallest tile.
int pick_tile(int rows_m, int rows_n, int B) {
    for (int cfg = pv::TILE_128; cfg > pv::TILE_16; --cfg) {
        const int t = pv::tile_size(cfg);
        const long long wgs = (long long)((rows_m + t - 1) / t) * ((rows_n + t - 1) / t) * B;
        if (wgs >= 240) return cfg;
    }
    return pv::TILE_16;
}

struct DedupPlan {
    int cos_cfg, njt;
    int gram_cfg, ntm, ntn, Mp;
    int n_counters;
    // workspace
    float *M, *invn, *rowsum, *p;
    int32_t *pruned, *assign;
    float *best_val;
    int32_t *best_slot;
    unsigned *counters;
    size_t bytes;
};

DedupPlan plan_dedup(void *ws, int B, int Nv, int Nt, int budget, bool want_p, bool want_assign) {
    DedupPlan P;
    P.cos_cfg = pick_tile(Nv, Nt, B);
    const int t1 = pv::tile_size(P.cos_cfg);
    P.njt = (Nv + t1 - 1) / t1;
    P.Mp = Nv - budget;
    P.gram_cfg = pick_tile(P.Mp > 0 ? P.Mp : 1, budget, B);
    const int t4 = pv::tile_size(P.gram_cfg);
    P.ntm = (P.Mp + t4 - 1) / t4;
    P.ntn = (budget + t4 - 1) / t4;
    P.n_counters = B + B * P.ntm;
    Carve c(ws);
    P.M = c.take<float>((size_t)B * Nt * Nv);
    P.invn = c.take<float>((size_t)B * Nv);
    P.rowsum = c.take<float>((size_t)B * P.njt * Nt);
    P.p = want_p ? c.take<float>((size_t)B * Nv) : nullptr;
    P.pruned = c.take<int32_t>((size_t)B * (P.Mp > 0 ? P.Mp : 1));
    P.assign = want_assign ? c.take<int32_t>((size_t)B * Nv) : nullptr;
    P.best_val = c.take<float>((size_t)B * P.ntn * (P.Mp > 0 ? P.Mp : 1));
    P.best_slot = c.take<int32_t>((size_t)B * P.ntn * (P.Mp > 0 ? P.Mp : 1));
    P.counters = c.take<unsigned>((size_t)P.n_counters);
    P.bytes = c.off + kAlign;
    return P;
}

int check_dedup(const void *vis, const void *anchors, int B, int Nv, int Nt, int d, int dtype,
                int budget, const int32_t *kept) {
    if (!vis || !anchors || !kept) return PV_ERR_NULL;
    if (dtype != PV_F32 && dtype != PV_BF16) return PV_ERR_DTYPE;
    if (B < 1 || B > 65535 || Nv < 1 || Nv > PV_MAX_TOKENS || Nt < 1 || Nt > PV_MAX_TEXT ||
        d < 64 || d > PV_MAX_DIM || d % 64 != 0)
        return PV_ERR_SHAPE;
    if (budget < 1 || budget > Nv) return PV_ERR_BUDGET;
    return PV_OK;
}

int dedup_impl(const void *vis, const void *anchors, int B, int Nv, int Nt, int d, int dtype,
               int budget, int32_t *kept, float *score, int32_t *assign, void *merged,
               void *workspace, size_t ws_bytes, void *stream, void *const *events, int n_events,
               int *n_kernels) {
    int rc = check_dedup(vis, anchors, B, Nv, Nt, d, dtype, budget, kept);
    if (rc != PV_OK) return rc;
    const bool need_assign = assign != nullptr || merged != nullptr;
    DedupPlan P0 = plan_dedup(nullptr, B, Nv, Nt, budget, score == nullptr, need_assign && !assign);
    if (!workspace) return PV_ERR_WORKSPACE;
    if (ws_bytes < P0.bytes) return PV_ERR_WORKSPACE;
    for (const void *p : {vis, anchors, (const void *)kept, (const void *)score,
                          (const void *)assign, (const void *)merged, (const void *)workspace})
        if (p && !aligned16(p)) return PV_ERR_ALIGN;
    // carve from a 256-aligned start
    char *wsa = (char *)(((uintptr_t)workspace + kAlign - 1) / kAlign * kAlign);
    DedupPlan P = plan_dedup(wsa, B, Nv, Nt, budget, score == nullptr, need_assign && !assign);
    float *p = score ? score : P.p;
    int32_t *asg = assign ? assign : P.assign;
    const int dt = (dtype == PV_BF16) ? pv::kBF16 : pv::kF32;
    hipStream_t st = (hipStream_t)stream;
    Trace tr{events, n_events, 0, st};
    hipError_t e;

    tr.before();
    e = pv::launch_cos_tile(dt, P.cos_cfg, vis, anchors, B, Nv, Nt, d, P.M, P.invn, P.rowsum,
                            P.counters, P.n_counters, st);
    if (e != hipSuccess) return PV_ERR_HIP;
    ++tr.launched;

    tr.before();
    e = pv::launch_center_select(P.M, P.rowsum, P.njt, B, Nt, Nv, p, budget, kept, P.pruned,
                                 need_assign ? asg : nullptr, P.counters, st);
    if (e != hipSuccess) return PV_ERR_HIP;
    ++tr.launched;

    if (need_assign && P.Mp > 0) {
        tr.before();
        e = pv::launch_gram_assign(dt, P.gram_cfg, vis, B, Nv, d, kept, budget, P.pruned, P.Mp,
                                   P.invn, P.best_val, P.best_slot, asg, P.counters + B, st);
        if (e != hipSuccess) return PV_ERR_HIP;
        ++tr.launched;
    }
    if (merged) {
        tr.before();
        e = pv::launch_merge(dt, vis, B, Nv, d, kept, budget, asg, merged, st);
        if (e != hipSuccess) return PV_ERR_HIP;
        ++tr.launched;
    }
    tr.after_all();
    if (n_kernels) *n_kernels = tr.launched;
    return PV_OK;
}

struct HeadPlan {
    int nrb;
    float *partial;
    float *v;
    size_t bytes;
};

HeadPlan plan_head(void *ws, int B, int Nt, int N, int n_heads, bool want_v) {
    HeadPlan P;
    P.nrb = (Nt + 15) / 16;
    Carve c(ws);
    P.partial = c.take<float>((size_t)B * n_heads * P.nrb * N);
    P.v = want_v ? c.take<float>((size_t)B * N) : nullptr;
    P.bytes = c.off + kAlign;
    return P;
}

int check_head(const void *q, const void *k, const int32_t *heads, int n_heads, int B, int H,
               int Nt, int N, int hd, int dtype, int budget, const int32_t *kept) {
    if (!q || !k || !heads || !kept) return PV_ERR_NULL;
    if (dtype != PV_F32 && dtype != PV_BF16) return PV_ERR_DTYPE;
    if (B < 1 || B > 65535 || H < 1 || Nt < 1 || Nt > PV_MAX_TEXT || N < 1 || N > PV_MAX_TOKENS ||
        hd < 32 || hd > PV_MAX_HEAD_DIM || hd % 32 != 0)
        return PV_ERR_SHAPE;
    if (n_heads < 1 || n_heads > H || n_heads > pv::kMaxHeadArgs) return PV_ERR_HEADS;
    if ((long long)B * n_heads > PV_MAX_HEAD_LIST) return PV_ERR_SHAPE;
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

int head_impl(const void *q, const void *k, const int32_t *heads, int n_heads, int B, int H, int Nt,
              int N, int hd, int dtype, int budget, int32_t *kept, float *score, void *workspace,
              size_t ws_bytes, void *stream, void *const *events, int n_events, int *n_kernels) {
    int rc = check_head(q, k, heads, n_heads, B, H, Nt, N, hd, dtype, budget, kept);
    if (rc != PV_OK) return rc;
    HeadPlan P0 = plan_head(nullptr, B, Nt, N, n_heads, score == nullptr);
    if (!workspace || ws_bytes < P0.bytes) return PV_ERR_WORKSPACE;
    for (const void *p : {q, k, (const void *)kept, (const void *)score, (const void *)workspace})
        if (p && !aligned16(p)) return PV_ERR_ALIGN;
    char *wsa = (char *)(((uintptr_t)workspace + kAlign - 1) / kAlign * kAlign);
    HeadPlan P = plan_head(wsa, B, Nt, N, n_heads, score == nullptr);
    float *v = score ? score : P.v;
    const int dt = (dtype == PV_BF16) ? pv::kBF16 : pv::kF32;
    hipStream_t st = (hipStream_t)stream;
    Trace tr{events, n_events, 0, st};

    pv::HeadArgs ha;
    memset(&ha, 0, sizeof(ha));
    memcpy(ha.h, heads, sizeof(int32_t) * (size_t)B * n_heads);

    tr.before();
    if (pv::launch_score_partial(dt, q, k, ha, B, H, Nt, N, hd, n_heads, P.partial, st) != hipSuccess)
        return PV_ERR_HIP;
    ++tr.launched;
    tr.before();
    const float inv_norm = (float)(1.0 / ((double)Nt * (double)n_heads));
    if (pv::launch_score_select(P.partial, B, n_heads * P.nrb, N, inv_norm, v, budget, kept, st) !=
        hipSuccess)
        return PV_ERR_HIP;
    ++tr.launched;
    tr.after_all();
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
    }
    return "unknown status";
}

PV_API int pv_version(void) { return (1 << 16) | 0; }

PV_API size_t pv_dedup_workspace_bytes(int B, int Nv, int Nt, int d, int budget, int dtype) {
    (void)d;
    (void)dtype;
    if (B < 1 || Nv < 1 || Nt < 1 || budget < 1 || budget > Nv) return 0;
    // sized for the case that needs the most: no score or assign output
    return plan_dedup(nullptr, B, Nv, Nt, budget, true, true).bytes;
}

PV_API int pv_prune_dedup(const void *vis, const void *anchors, int B, int Nv, int Nt, int d,
                          int dtype, int budget, int32_t *kept, float *score, int32_t *assign,
                          void *merged, void *workspace, size_t workspace_bytes, void *stream) {
    return dedup_impl(vis, anchors, B, Nv, Nt, d, dtype, budget, kept, score, assign, merged,
                      workspace, workspace_bytes, stream, nullptr, 0, nullptr);
}

PV_API int pv_prune_dedup_timed(const void *vis, const void *anchors, int B, int Nv, int Nt, int d,
                                int dtype, int budget, int32_t *kept, float *score,
                                int32_t *assign, void *merged, void *workspace,
                                size_t workspace_bytes, void *stream, void *const *events,
                                int n_events, int *n_kernels) {
    return dedup_impl(vis, anchors, B, Nv, Nt, d, dtype, budget, kept, score, assign, merged,
                      workspace, workspace_bytes, stream, events, n_events, n_kernels);
}

PV_API size_t pv_head_aware_workspace_bytes(int B, int H, int Nt, int N, int hd, int n_heads,
                                            int budget, int dtype) {
    (void)H;
    (void)hd;
    (void)budget;
    (void)dtype;
    if (B < 1 || Nt < 1 || N < 1 || n_heads < 1) return 0;
    return plan_head(nullptr, B, Nt, N, n_heads, true).bytes;
}

PV_API int pv_prune_head_aware(const void *q, const void *k, const int32_t *heads_host, int n_heads,
                               int B, int H, int Nt, int N, int hd, int dtype, int budget,
                               int32_t *kept, float *score, void *workspace, size_t workspace_bytes,
                               void *stream) {
    return head_impl(q, k, heads_host, n_heads, B, H, Nt, N, hd, dtype, budget, kept, score,
                     workspace, workspace_bytes, stream, nullptr, 0, nullptr);
}

PV_API int pv_prune_head_aware_timed(const void *q, const void *k, const int32_t *heads_host,
                                     int n_heads, int B, int H, int Nt, int N, int hd, int dtype,
                                     int budget, int32_t *kept, float *score, void *workspace,
                                     size_t workspace_bytes, void *stream, void *const *events,
                                     int n_events, int *n_kernels) {
    return head_impl(q, k, heads_host, n_heads, B, H, Nt, N, hd, dtype, budget, kept, score,
                     workspace, workspace_bytes, stream, events, n_events, n_kernels);
}

PV_API int pv_prune_gather(const void *src, void *dst, const int32_t *idx, int B, int n_src, int k,
                           int groups, int64_t row_bytes, int64_t src_batch_stride,
                           int64_t src_group_stride, int64_t src_row_stride,
                           int64_t dst_batch_stride, int64_t dst_group_stride,
                           int64_t dst_row_stride, void *stream) {
    if (!src || !dst || !idx) return PV_ERR_NULL;
    if (B < 1 || B > 65535 || n_src < 1 || k < 1 || groups < 1 || groups > 65535 || row_bytes < 16)
        return PV_ERR_SHAPE;
    if ((row_bytes / 16) * (long long)k > 0x7FFFFFFFLL) return PV_ERR_SHAPE;
    if (!aligned16(src) || !aligned16(dst) || !aligned16(idx) || row_bytes % 16 ||
        src_batch_stride % 16 || src_group_stride % 16 || src_row_stride % 16 ||
        dst_batch_stride % 16 || dst_group_stride % 16 || dst_row_stride % 16)
        return PV_ERR_ALIGN;
    if (pv::launch_gather(src, dst, idx, B, n_src, k, groups, row_bytes, src_batch_stride,
                          src_group_stride, src_row_stride, dst_batch_stride, dst_group_stride,
                          dst_row_stride, (hipStream_t)stream) != hipSuccess)
        return PV_ERR_HIP;
    return PV_OK;
}
