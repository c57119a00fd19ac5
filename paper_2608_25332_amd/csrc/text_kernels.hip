// Critical text tokens (Sec. 4.2, equations for r and T).
//
//   r[j] = (1/Nt) sum_i softmax_j(e_i . e_j)      (E E^T without scaling)
//   T    = { j : r[j] > mean(r) }, every token when that is empty
//
// The self-similarity E E^T is a split-k product on the cosine engine (the
// text rows are both operands); text_gram_sum adds its k slices in order
// and text_rank (one workgroup per sample) takes the row softmax
// statistics, the column means and the selection.  All of it is tiny next
// to the pruning stages: Nt is a few hundred rows at most.
#include "provip.h"
#include "pv_launch.h"
#include "pv_device.h"

#include <math.h>

namespace pv {

constexpr int kRankNT = 1024;
constexpr int kRankW = kRankNT / 64;           // waves
constexpr int kRankRows = 4;                   // rows a wave loads at once

// G[b][i][j] = sum over k slices of part[ks][b][i][j], slices in order.
__global__ __launch_bounds__(256) void text_gram_sum_kernel(const float *__restrict__ part, int B,
                                                            int Nt, int KS,
                                                            float *__restrict__ G) {
    const size_t per = (size_t)B * Nt * Nt;
    const size_t e = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (e >= per) return;
    float s = 0.f;
    for (int ks = 0; ks < KS; ++ks) s += part[(size_t)ks * per + e];
    G[e] = s;
}

// Sum of one value per thread over the workgroup, in a fixed order: the
// wave's lanes in the order of a butterfly, then the waves in index order.
__device__ __forceinline__ float block_sum_fixed(float v, float *wsum) {
    v = wave_sum64(v);
    const int wave = threadIdx.x >> 6;
    __syncthreads();
    if ((threadIdx.x & 63) == 0) wsum[wave] = v;
    __syncthreads();
    float t = 0.f;
    for (int w = 0; w < kRankW; ++w) t += wsum[w];
    return t;
}

// One workgroup per sample.  Each wave takes rows w, w + kRankW, ...: a
// row's values stay in registers (PER per lane, PER * 64 >= Nt) for its
// maximum, its sum of exponentials and its normalised probabilities, which
// the wave adds into its own column sums in LDS, row after row; the waves'
// column sums are then added in wave order.  The loads of kRankRows rows are
// issued together.
template <int PER>
__global__ __launch_bounds__(kRankNT) void text_rank_kernel(const float *__restrict__ G, int Nt,
                                                            float *__restrict__ r_out,
                                                            int32_t *__restrict__ mask,
                                                            int32_t *__restrict__ count) {
    __shared__ float csum[kRankW][PV_MAX_TEXT];
    __shared__ float rr[PV_MAX_TEXT];
    __shared__ float wsum[kRankW];
    const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const float *Gb = G + (size_t)b * Nt * Nt;
    for (int j = lane; j < Nt; j += 64) csum[wave][j] = 0.f;
    for (int i0 = wave; i0 < Nt; i0 += kRankRows * kRankW) {
        float g[kRankRows][PER];
#pragma unroll
        for (int q = 0; q < kRankRows; ++q) {
            const int i = i0 + q * kRankW;
#pragma unroll
            for (int t = 0; t < PER; ++t) {
                const int j = lane + 64 * t;
                g[q][t] = (i < Nt && j < Nt) ? Gb[(size_t)i * Nt + j] : -INFINITY;
            }
        }
#pragma unroll
        for (int q = 0; q < kRankRows; ++q) {
            if (i0 + q * kRankW >= Nt) break;  // uniform over the wave
            float m = -INFINITY;
#pragma unroll
            for (int t = 0; t < PER; ++t) m = fmaxf(m, g[q][t]);
            m = wave_max_f32(m);
            float l = 0.f;
#pragma unroll
            for (int t = 0; t < PER; ++t) {
                g[q][t] = expf(g[q][t] - m);  // 0 past the end
                l += g[q][t];
            }
            l = wave_sum64(l);
            const float il = 1.0f / l;
#pragma unroll
            for (int t = 0; t < PER; ++t) {
                const int j = lane + 64 * t;
                if (j < Nt) csum[wave][j] += g[q][t] * il;
            }
        }
    }
    __syncthreads();
    float own = 0.f;
    for (int j = tid; j < Nt; j += kRankNT) {
        float s = 0.f;
        for (int w = 0; w < kRankW; ++w) s += csum[w][j];
        const float r = s / (float)Nt;
        rr[j] = r;
        own += r;
        if (r_out) r_out[(size_t)b * Nt + j] = r;
    }
    const float mean = block_sum_fixed(own, wsum) / (float)Nt;
    int above = 0;
    for (int j = tid; j < Nt; j += kRankNT) above += rr[j] > mean ? 1 : 0;
    const int n_above = (int)block_sum_fixed((float)above, wsum);
    // none strictly above the mean: every token is kept
    for (int j = tid; j < Nt; j += kRankNT)
        mask[(size_t)b * Nt + j] = (n_above == 0 || rr[j] > mean) ? 1 : 0;
    if (tid == 0) count[b] = n_above == 0 ? Nt : n_above;
}

hipError_t launch_text_gram_sum(const float *part, int B, int Nt, int KS, float *G,
                                hipStream_t st) {
    const size_t per = (size_t)B * Nt * Nt;
    hipLaunchKernelGGL(text_gram_sum_kernel, dim3((unsigned)((per + 255) / 256)), dim3(256), 0, st,
                       part, B, Nt, KS, G);
    return hipGetLastError();
}

hipError_t launch_text_rank(const float *G, int B, int Nt, float *r, int32_t *mask, int32_t *count,
                            hipStream_t st) {
    if (Nt > PV_MAX_TEXT) return hipErrorInvalidValue;
#define PV_RANK_CASE(per)                                                                     \
    hipLaunchKernelGGL(text_rank_kernel<per>, dim3(B), dim3(kRankNT), 0, st, G, Nt, r, mask, \
                       count)
    if (Nt <= 64) PV_RANK_CASE(1);
    else if (Nt <= 128) PV_RANK_CASE(2);
    else if (Nt <= 256) PV_RANK_CASE(4);
    else if (Nt <= 512) PV_RANK_CASE(8);
    else PV_RANK_CASE(PV_MAX_TEXT / 64);
#undef PV_RANK_CASE
    return hipGetLastError();
}

}  // namespace pv
