// Head-aware pruning at a pruning layer (Sec. 4.4, equations for S^vis and v).
//
//   v[j] = (1/(|V| Nt)) sum_{h in V} sum_i softmax_j(q_hi . k_hj / sqrt(hd))
//
// The softmax normalises along a row (over the keys) while the importance
// sums along a column (over the text rows), so there is no single-pass form:
// a row's normaliser is only known once the whole row is seen.
//
// score_partial (grid: 16-row blocks x selected heads x B) keeps the 16 query
// rows of its block in registers as MFMA fragments and streams the head's
// keys from HBM/L2 through LDS, 64 keys per chunk.  When the chunks number at
// most MAXC the logits stay in registers between the row statistics and the
// column sums (one pass over K); otherwise the keys are streamed again in a
// second pass.  Only the selected heads are ever read and the attention map
// is never written out.  score_select (one workgroup per sample) adds the per-(head,
// row-block) column sums in a fixed order and runs the top-N_2.
#include "pv_launch.h"
#include "pv_device.h"

#include <math.h>

namespace pv {

constexpr int kScoreNT = 256;

__device__ __forceinline__ void lse_merge(float &m, float &l, float m2, float l2) {
    const float mn = fmaxf(m, m2);
    if (mn == -INFINITY) return;  // both empty
    l = l * exp2f(m - mn) + l2 * exp2f(m2 - mn);
    m = mn;
}

// Key rows are staged through LDS 64 at a time (one 16-key block per wave)
// with row-major 16-byte loads: 4*NKS consecutive lanes read one key row, the
// access pattern that moves the most bytes per clock into a CU.  The MFMA
// fragments are then read from LDS.
constexpr int kScoreCK = 64;  // keys per staged chunk

template <int NKS>
struct ScoreStage {
    static constexpr int RB = 64 * NKS;     // bytes of one key row
    static constexpr int STRIDE = RB + 16;  // LDS bytes per staged row (16-byte pad)
    static constexpr int PPR = RB / 16;     // 16-byte pieces per row
    static constexpr int PPT = kScoreCK * PPR / kScoreNT;  // pieces per thread per chunk
    static constexpr int LDS = kScoreCK * STRIDE;
    static_assert(kScoreCK * PPR % kScoreNT == 0, "chunk must fill the loaders evenly");
};

template <int DT, int NKS, int MAXC>
__global__ __launch_bounds__(kScoreNT) void score_partial_kernel(
    const char *__restrict__ q, const char *__restrict__ k, HeadArgs heads, int H, int Nt, int N,
    int n_heads, float scale_log2e, float *__restrict__ partial) {
    using S = ScoreStage<NKS>;
    __shared__ __attribute__((aligned(16))) char kst[S::LDS];
    __shared__ float sm_m[4][16], sm_l[4][16];
    __shared__ float row_m[16], row_il[16];
    const int rb = blockIdx.x, hi = blockIdx.y, b = blockIdx.z;
    const int nrb = gridDim.x;
    const int tid = threadIdx.x, lane = tid & 63;
    // uniform wave index: the block guards around the MFMAs become scalar
    // branches (an MFMA does not honour the execution mask)
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int h = heads.h[b * n_heads + hi];
    const char *qb = q + ((size_t)b * H + h) * Nt * S::RB;
    const char *kb = k + ((size_t)b * H + h) * N * S::RB;
    const int koff = (lane >> 4) * 16;

    uint4 qf[NKS];
    {
        const char *qr = qb + (size_t)min(rb * 16 + (lane & 15), Nt - 1) * S::RB + koff;
#pragma unroll
        for (int s = 0; s < NKS; ++s) qf[s] = ld16(qr + s * 64);
    }
    const int nch = (N + kScoreCK - 1) / kScoreCK;

    int srow[S::PPT], scol[S::PPT];
#pragma unroll
    for (int p = 0; p < S::PPT; ++p) {
        const int qq = tid + kScoreNT * p;
        srow[p] = qq / S::PPR;
        scol[p] = (qq % S::PPR) * 16;
    }
    // one pass over the keys: stage chunk ch (the next one is in flight while
    // this one is multiplied) and hand this wave's 16x16 logit block to body
    auto sweep = [&](auto body) {
        uint4 buf[S::PPT];
        auto fetch = [&](int ch) {
#pragma unroll
            for (int p = 0; p < S::PPT; ++p) {
                const int row = min(ch * kScoreCK + srow[p], N - 1);  // past the end: last key
                buf[p] = ld16(kb + (size_t)row * S::RB + scol[p]);
            }
        };
        fetch(0);
        for (int ch = 0; ch < nch; ++ch) {
            __syncthreads();  // the previous chunk's fragment reads are done
#pragma unroll
            for (int p = 0; p < S::PPT; ++p) st16(kst + srow[p] * S::STRIDE + scol[p], buf[p]);
            __syncthreads();
            if (ch + 1 < nch) fetch(ch + 1);
            const char *fr = kst + (wave * 16 + (lane & 15)) * S::STRIDE + koff;
            f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < NKS; ++s) acc = mma16<DT>(qf[s], ld16(fr + s * 64), acc);
            body(ch, acc);
        }
    };

    // pass 1: running (max, sum of exp) of the logits, per lane and row; with
    // MAXC > 0 the logit blocks also stay in registers for pass 2
    float m[4], l[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        m[i] = -INFINITY;
        l[i] = 0.f;
    }
    f32x4_t keep[MAXC > 0 ? MAXC : 1];
    sweep([&](int ch, const f32x4_t &acc) {
        if (MAXC > 0) {
#pragma unroll
            for (int c = 0; c < (MAXC > 0 ? MAXC : 1); ++c) keep[c] = (c == ch) ? acc : keep[c];
        }
        if (ch * kScoreCK + wave * 16 + (lane & 15) < N) {
#pragma unroll
            for (int i = 0; i < 4; ++i) lse_merge(m[i], l[i], acc[i] * scale_log2e, 1.f);
        }
    });
    // combine the 16 lanes that hold the same rows, then the 4 waves
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float m2 = __shfl_xor(m[i], off, 64);
            const float l2 = __shfl_xor(l[i], off, 64);
            lse_merge(m[i], l[i], m2, l2);
        }
    }
    if ((lane & 15) == 0) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            sm_m[wave][(lane >> 4) * 4 + i] = m[i];
            sm_l[wave][(lane >> 4) * 4 + i] = l[i];
        }
    }
    __syncthreads();
    if (tid < 16) {
        float mm = sm_m[0][tid], ll = sm_l[0][tid];
#pragma unroll
        for (int w = 1; w < 4; ++w) lse_merge(mm, ll, sm_m[w][tid], sm_l[w][tid]);
        row_m[tid] = mm;
        row_il[tid] = (rb * 16 + tid < Nt) ? 1.0f / ll : 0.f;  // masked rows add nothing
    }
    __syncthreads();

    float rm[4], ril[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        rm[i] = row_m[(lane >> 4) * 4 + i];
        ril[i] = row_il[(lane >> 4) * 4 + i];
    }
    float *out = partial + (((size_t)b * n_heads + hi) * nrb + rb) * N;
    // pass 2: normalised probabilities, summed over the 16 rows of each column
    auto emit = [&](const f32x4_t &acc, int col) {
        float cs = 0.f;
#pragma unroll
        for (int i = 0; i < 4; ++i) cs += exp2f(acc[i] * scale_log2e - rm[i]) * ril[i];
        cs += __shfl_xor(cs, 16, 64);
        cs += __shfl_xor(cs, 32, 64);
        if (lane < 16 && col < N) out[col] = cs;
    };
    if (MAXC > 0) {
#pragma unroll
        for (int c = 0; c < (MAXC > 0 ? MAXC : 1); ++c)
            if (c < nch) emit(keep[c], c * kScoreCK + wave * 16 + (lane & 15));
    } else {
        sweep([&](int ch, const f32x4_t &acc) {
            emit(acc, ch * kScoreCK + wave * 16 + (lane & 15));
        });
    }
}

constexpr int kSelU = 16;

template <int NT, int EMAX>
__global__ __launch_bounds__(NT) void score_select_kernel(const float *__restrict__ partial,
                                                          int nparts, int N, float inv_norm,
                                                          float *__restrict__ v, int budget,
                                                          int32_t *__restrict__ kept) {
    __shared__ TopkSmem sm;
    const int b = blockIdx.x;
    const float *pb = partial + (size_t)b * nparts * N;
    float *vb = v + (size_t)b * N;
    const int E = topk_per_thread(N, NT), j0 = threadIdx.x * E;
    uint32_t key[EMAX];
#pragma unroll
    for (int e = 0; e < EMAX; ++e) {
        const int j = j0 + e;
        key[e] = 0u;
        if (e < E && j < N) {
            // partials in blocks of kSelU with clamped addresses (all loads of a
            // block in flight), added in part order
            float s = 0.f;
            for (int t0 = 0; t0 < nparts; t0 += kSelU) {
                float v[kSelU];
#pragma unroll
                for (int u = 0; u < kSelU; ++u) v[u] = pb[(size_t)min(t0 + u, nparts - 1) * N + j];
#pragma unroll
                for (int u = 0; u < kSelU; ++u)
                    if (t0 + u < nparts) s += v[u];
            }
            s *= inv_norm;
            vb[j] = s;
            key[e] = order_key(s);
        }
    }
    block_topk<NT, EMAX>(key, N, budget, kept + (size_t)b * budget, nullptr, nullptr, sm);
}

template <int DT, int NKS, int MAXC>
static hipError_t score_go(const void *q, const void *k, const HeadArgs &heads, int B, int H,
                           int Nt, int N, int n_heads, float scale_log2e, float *partial,
                           hipStream_t st) {
    dim3 grid((Nt + 15) / 16, n_heads, B);
    hipLaunchKernelGGL((score_partial_kernel<DT, NKS, MAXC>), grid, dim3(kScoreNT), 0, st,
                       (const char *)q, (const char *)k, heads, H, Nt, N, n_heads, scale_log2e,
                       partial);
    return hipGetLastError();
}

// Logit blocks held in registers between the two passes: the smallest of 1,
// 2, 4, 8, 16 chunks that covers the keys, within a register budget that
// shrinks as the head width grows; otherwise the keys are streamed twice
// (MAXC = 0).
template <int NKS>
constexpr int score_maxc_cap() { return NKS <= 4 ? 16 : (NKS <= 8 ? 8 : 4); }

template <int DT, int NKS>
static hipError_t score_nks(const void *q, const void *k, const HeadArgs &heads, int B, int H,
                            int Nt, int N, int n_heads, float sl2e, float *partial,
                            hipStream_t st) {
    const int nch = (N + kScoreCK - 1) / kScoreCK;
    constexpr int cap = score_maxc_cap<NKS>();
#define PV_MAXC_CASE(mc)                                                                           \
    if (nch <= mc && mc <= cap)                                                                    \
        return score_go<DT, NKS, (mc <= cap ? mc : 0)>(q, k, heads, B, H, Nt, N, n_heads, sl2e,   \
                                                       partial, st);
    PV_MAXC_CASE(1)
    PV_MAXC_CASE(2)
    PV_MAXC_CASE(4)
    PV_MAXC_CASE(8)
    PV_MAXC_CASE(16)
#undef PV_MAXC_CASE
    return score_go<DT, NKS, 0>(q, k, heads, B, H, Nt, N, n_heads, sl2e, partial, st);
}

template <int DT>
static hipError_t score_dt(int nks, const void *q, const void *k, const HeadArgs &heads, int B,
                           int H, int Nt, int N, int n_heads, float sl2e,
                           float *partial, hipStream_t st) {
#define PV_NKS_CASE(n) \
    case n:            \
        return score_nks<DT, n>(q, k, heads, B, H, Nt, N, n_heads, sl2e, partial, st);
    switch (nks) {
        PV_NKS_CASE(1)
        PV_NKS_CASE(2)
        PV_NKS_CASE(3)
        PV_NKS_CASE(4)
        PV_NKS_CASE(5)
        PV_NKS_CASE(6)
        PV_NKS_CASE(7)
        PV_NKS_CASE(8)
        PV_NKS_CASE(10)
        PV_NKS_CASE(12)
        PV_NKS_CASE(14)
        PV_NKS_CASE(16)
    }
#undef PV_NKS_CASE
    return hipErrorInvalidValue;
}

hipError_t launch_score_partial(int dt, const void *q, const void *k, const HeadArgs &heads,
                                int B, int H, int Nt, int N, int hd, int n_heads, float *partial,
                                hipStream_t st) {
    const int esz = (dt == kBF16) ? 2 : 4;
    const int hd_bytes = hd * esz;
    const int nks = hd_bytes / 64;
    const float sl2e = (float)(1.4426950408889634 / sqrt((double)hd));
    if (dt == kBF16) return score_dt<kBF16>(nks, q, k, heads, B, H, Nt, N, n_heads, sl2e, partial, st);
    return score_dt<kF32>(nks, q, k, heads, B, H, Nt, N, n_heads, sl2e, partial, st);
}

hipError_t launch_score_select(const float *partial, int B, int nparts, int N, float inv_norm,
                               float *v, int budget, int32_t *kept, hipStream_t st) {
    if (N <= 256 * 4)
        hipLaunchKernelGGL((score_select_kernel<256, 4>), dim3(B), dim3(256), 0, st, partial,
                           nparts, N, inv_norm, v, budget, kept);
    else if (N <= 512 * 8)
        hipLaunchKernelGGL((score_select_kernel<512, 8>), dim3(B), dim3(512), 0, st, partial,
                           nparts, N, inv_norm, v, budget, kept);
    else if (N <= 1024 * 16)
        hipLaunchKernelGGL((score_select_kernel<1024, 16>), dim3(B), dim3(1024), 0, st, partial,
                           nparts, N, inv_norm, v, budget, kept);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

}  // namespace pv
