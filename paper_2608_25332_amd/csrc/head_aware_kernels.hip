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
// keys from HBM/L2.  When a wave's share of the keys is at most MAXB blocks of
// 16 the logits stay in registers between the row statistics and the column
// sums (one pass over K); otherwise the logits are recomputed in a second
// pass.  Only the selected heads are ever read and the attention map is never
// written out.  score_select (one workgroup per sample) adds the per-(head,
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

template <int DT, int NKS>
__device__ __forceinline__ f32x4_t qk_block(const uint4 (&qf)[NKS], const char *kb, int col, int N,
                                            int hd_bytes, int koff) {
    const char *kr = kb + (size_t)min(col, N - 1) * hd_bytes + koff;
    uint4 kf[NKS];
#pragma unroll
    for (int s = 0; s < NKS; ++s) kf[s] = ld16(kr + s * 64);
    f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < NKS; ++s) acc = mma16<DT>(qf[s], kf[s], acc);
    return acc;
}

template <int DT, int NKS, int MAXB>
__global__ __launch_bounds__(kScoreNT) void score_partial_kernel(
    const char *__restrict__ q, const char *__restrict__ k, HeadArgs heads, int H, int Nt, int N,
    int hd_bytes, int n_heads, float scale_log2e, float *__restrict__ partial) {
    __shared__ float sm_m[4][16], sm_l[4][16];
    __shared__ float row_m[16], row_il[16];
    const int rb = blockIdx.x, hi = blockIdx.y, b = blockIdx.z;
    const int nrb = gridDim.x;
    const int tid = threadIdx.x, lane = tid & 63;
    // uniform wave index: the block guards around the MFMAs become scalar
    // branches (an MFMA does not honour the execution mask)
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int h = heads.h[b * n_heads + hi];
    const char *qb = q + ((size_t)b * H + h) * Nt * hd_bytes;
    const char *kb = k + ((size_t)b * H + h) * N * hd_bytes;
    const int koff = (lane >> 4) * 16;

    uint4 qf[NKS];
    {
        const char *qr = qb + (size_t)min(rb * 16 + (lane & 15), Nt - 1) * hd_bytes + koff;
#pragma unroll
        for (int s = 0; s < NKS; ++s) qf[s] = ld16(qr + s * 64);
    }
    const int nblk = (N + 15) / 16;

    // pass 1: running (max, sum of exp) of the logits, per lane and row
    float m[4], l[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        m[i] = -INFINITY;
        l[i] = 0.f;
    }
    f32x4_t keep[MAXB > 0 ? MAXB : 1];
    if (MAXB > 0) {
        // all key fragments of this wave's blocks in flight at once (rows past
        // the end are clamped to the last key), then the MFMAs
        uint4 kf[MAXB > 0 ? MAXB : 1][NKS];
#pragma unroll
        for (int bi = 0; bi < MAXB; ++bi) {
            const int col = min((wave + 4 * bi) * 16 + (lane & 15), N - 1);
            const char *kr = kb + (size_t)col * hd_bytes + koff;
#pragma unroll
            for (int s2 = 0; s2 < NKS; ++s2) kf[bi][s2] = ld16(kr + s2 * 64);
        }
#pragma unroll
        for (int bi = 0; bi < MAXB; ++bi) {
            if (wave + 4 * bi < nblk) {
                f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int s2 = 0; s2 < NKS; ++s2) acc = mma16<DT>(qf[s2], kf[bi][s2], acc);
                keep[bi] = acc;
            }
        }
#pragma unroll
        for (int bi = 0; bi < MAXB; ++bi) {
            const int blk = wave + 4 * bi;
            if (blk < nblk && blk * 16 + (lane & 15) < N) {
#pragma unroll
                for (int i = 0; i < 4; ++i) lse_merge(m[i], l[i], keep[bi][i] * scale_log2e, 1.f);
            }
        }
    } else {
        for (int blk = wave; blk < nblk; blk += 4) {
            const int col = blk * 16 + (lane & 15);
            const f32x4_t acc = qk_block<DT, NKS>(qf, kb, col, N, hd_bytes, koff);
            if (col < N) {
#pragma unroll
                for (int i = 0; i < 4; ++i) lse_merge(m[i], l[i], acc[i] * scale_log2e, 1.f);
            }
        }
    }
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
    if (MAXB > 0) {
#pragma unroll
        for (int bi = 0; bi < MAXB; ++bi) {
            const int blk = wave + 4 * bi;
            if (blk < nblk) emit(keep[bi], blk * 16 + (lane & 15));
        }
    } else {
        for (int blk = wave; blk < nblk; blk += 4) {
            const int col = blk * 16 + (lane & 15);
            emit(qk_block<DT, NKS>(qf, kb, col, N, hd_bytes, koff), col);
        }
    }
}

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
            float s = 0.f;
            for (int t = 0; t < nparts; ++t) s += pb[(size_t)t * N + j];
            s *= inv_norm;
            vb[j] = s;
            key[e] = order_key(s);
        }
    }
    block_topk<NT, EMAX>(key, N, budget, kept + (size_t)b * budget, nullptr, nullptr, sm);
}

template <int DT, int NKS, int MAXB>
static hipError_t score_go(const void *q, const void *k, const HeadArgs &heads, int B, int H,
                           int Nt, int N, int hd_bytes, int n_heads, float scale_log2e,
                           float *partial, hipStream_t st) {
    dim3 grid((Nt + 15) / 16, n_heads, B);
    hipLaunchKernelGGL((score_partial_kernel<DT, NKS, MAXB>), grid, dim3(kScoreNT), 0, st,
                       (const char *)q, (const char *)k, heads, H, Nt, N, hd_bytes, n_heads,
                       scale_log2e, partial);
    return hipGetLastError();
}

// Key blocks per wave held in registers: the smallest of 1, 2, 4, 8 that
// covers the wave's share, while the fragments stay within 32 x 16 bytes per
// lane; otherwise the two-pass form (MAXB = 0).
template <int DT, int NKS>
static hipError_t score_nks(const void *q, const void *k, const HeadArgs &heads, int B, int H,
                            int Nt, int N, int hd_bytes, int n_heads, float sl2e, float *partial,
                            hipStream_t st) {
    const int bpw = ((N + 15) / 16 + 3) / 4;
#define PV_MAXB_CASE(mb)                                                                           \
    if (bpw <= mb && mb * NKS <= 32)                                                               \
        return score_go<DT, NKS, (mb * NKS <= 32 ? mb : 0)>(q, k, heads, B, H, Nt, N, hd_bytes,    \
                                                            n_heads, sl2e, partial, st);
    PV_MAXB_CASE(1)
    PV_MAXB_CASE(2)
    PV_MAXB_CASE(4)
    PV_MAXB_CASE(8)
#undef PV_MAXB_CASE
    return score_go<DT, NKS, 0>(q, k, heads, B, H, Nt, N, hd_bytes, n_heads, sl2e, partial, st);
}

template <int DT>
static hipError_t score_dt(int nks, const void *q, const void *k, const HeadArgs &heads, int B,
                           int H, int Nt, int N, int hd_bytes, int n_heads, float sl2e,
                           float *partial, hipStream_t st) {
#define PV_NKS_CASE(n) \
    case n:            \
        return score_nks<DT, n>(q, k, heads, B, H, Nt, N, hd_bytes, n_heads, sl2e, partial, st);
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
    if (dt == kBF16) return score_dt<kBF16>(nks, q, k, heads, B, H, Nt, N, hd_bytes, n_heads, sl2e, partial, st);
    return score_dt<kF32>(nks, q, k, heads, B, H, Nt, N, hd_bytes, n_heads, sl2e, partial, st);
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
