// Pruning before the LLM (Sec. 4.3): cross-modal cosine (equation for M),
// row centring (equation for M-hat), max-pooling (equation for p), top-N_1,
// nearest-centroid assignment of the pruned tokens and their aggregation.
//
// Kernel sequence of one call (all on the caller's stream):
//   cos_tile      anchors x vis on MFMA, norms fused; writes cosines, the
//                 inverse norms of the visual tokens and per-tile row sums
//   center_select p[j] = max_i (M[i][j] - mean_i); the last workgroup of a
//                 sample runs the top-N_1 radix select
//   gram_assign   pruned x kept cosine Gram on MFMA with a fused row argmax;
//                 the last workgroup of a row tile reduces across column tiles
//   merge         centroid <- mean of itself and its members
#include "pv_launch.h"
#include "pv_tile_gemm.h"

#include <math.h>

namespace pv {

int tile_size(int cfg) { return 16 << cfg; }

// ----------------------------------------------------------------------------
// cos_tile: grid (Nv tiles, Nt tiles, B).
// ----------------------------------------------------------------------------
template <int DT, int BM, int BN, int WM, int WN>
__global__ __launch_bounds__(64 * WM * WN) void cos_tile_kernel(
    const char *__restrict__ vis, const char *__restrict__ anchors, int Nv, int Nt, int d_bytes,
    float *__restrict__ M, float *__restrict__ invn_vis, float *__restrict__ rowsum,
    unsigned *__restrict__ counters, int n_counters) {
    using G = TileGemm<DT, BM, BN, WM, WN>;
    __shared__ __attribute__((aligned(16))) char lds[G::LDS_BYTES];
    __shared__ float rowss[G::ROWS];
    __shared__ float rowinv[G::ROWS];
    __shared__ float red[WN][BM];

    const int jt = blockIdx.x, it = blockIdx.y, b = blockIdx.z;
    const int njt = gridDim.x;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;

    // Later kernels of this call count finished workgroups in `counters`.
    if (jt == 0 && it == 0 && b == 0)
        for (int e = tid; e < n_counters; e += G::NT) counters[e] = 0u;

    const int i0 = it * BM, j0 = jt * BN;
    const char *abase = anchors + (size_t)b * Nt * d_bytes;
    const char *vbase = vis + (size_t)b * Nv * d_bytes;
    auto row_ptr = [&](int r) -> const char * {
        if (r < BM) return abase + (size_t)min(i0 + r, Nt - 1) * d_bytes;
        return vbase + (size_t)min(j0 + r - BM, Nv - 1) * d_bytes;
    };

    f32x4_t acc[G::FM][G::FN];
    float ss[G::PPT];
    G::template run<true>(row_ptr, d_bytes / G::CHUNK, lds, acc, ss);
    G::reduce_rows(ss, rowss);
    __syncthreads();
    for (int r = tid; r < G::ROWS; r += G::NT) {
        float s = rowss[r];
        rowinv[r] = (s > 0.f) ? 1.0f / sqrtf(s) : 0.f;
    }
    __syncthreads();

    if (it == 0) {
        for (int c = tid; c < BN; c += G::NT)
            if (j0 + c < Nv) invn_vis[(size_t)b * Nv + j0 + c] = rowinv[BM + c];
    }

#pragma unroll
    for (int fm = 0; fm < G::FM; ++fm) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = wm * G::SUB_M + fm * 16 + (lane >> 4) * 4 + i;
            const int gi = i0 + r;
            const float ia = rowinv[r];
            float rs = 0.f;
#pragma unroll
            for (int fn = 0; fn < G::FN; ++fn) {
                const int c = wn * G::SUB_N + fn * 16 + (lane & 15);
                const int gj = j0 + c;
                const float cs = acc[fm][fn][i] * ia * rowinv[BM + c];
                if (gj < Nv) {
                    rs += cs;
                    if (gi < Nt) M[((size_t)b * Nt + gi) * Nv + gj] = cs;
                }
            }
            rs += __shfl_xor(rs, 1, 64);
            rs += __shfl_xor(rs, 2, 64);
            rs += __shfl_xor(rs, 4, 64);
            rs += __shfl_xor(rs, 8, 64);
            if ((lane & 15) == 0) red[wn][r] = rs;
        }
    }
    __syncthreads();
    for (int r = tid; r < BM; r += G::NT) {
        float s = 0.f;
#pragma unroll
        for (int w = 0; w < WN; ++w) s += red[w][r];
        if (i0 + r < Nt) rowsum[((size_t)b * njt + jt) * Nt + i0 + r] = s;
    }
}

// ----------------------------------------------------------------------------
// center_select: grid (ceil(Nv / 256), B), 256 threads.
// ----------------------------------------------------------------------------
constexpr int kSelNT = 256;

__global__ __launch_bounds__(kSelNT) void center_select_kernel(
    const float *__restrict__ M, const float *__restrict__ rowsum, int njt, int Nt, int Nv,
    float *__restrict__ p, int budget, int32_t *__restrict__ kept, int32_t *__restrict__ pruned,
    int32_t *__restrict__ slot_of, unsigned *__restrict__ counters) {
    extern __shared__ float mu[];  // [Nt]
    __shared__ TopkSmem sm;
    __shared__ int is_last;
    const int b = blockIdx.y, tid = threadIdx.x;
    const int j = blockIdx.x * kSelNT + tid;

    // Row means of M over all Nv tokens, from the per-tile partial sums.
    for (int i = tid; i < Nt; i += kSelNT) {
        float s = 0.f;
        for (int t = 0; t < njt; ++t) s += rowsum[((size_t)b * njt + t) * Nt + i];
        mu[i] = s / (float)Nv;
    }
    __syncthreads();
    if (j < Nv) {
        const float *col = M + (size_t)b * Nt * Nv + j;
        float m = col[0] - mu[0];
        for (int i = 1; i < Nt; ++i) m = fmaxf(m, col[(size_t)i * Nv] - mu[i]);
        p[(size_t)b * Nv + j] = m;
    }

    // The last workgroup of this sample selects the top `budget` tokens.
    __threadfence();
    __syncthreads();
    if (tid == 0) is_last = (atomicAdd(&counters[b], 1u) == gridDim.x - 1);
    __syncthreads();
    if (!is_last) return;
    __threadfence();
    block_topk<kSelNT>(p + (size_t)b * Nv, Nv, budget, kept + (size_t)b * budget,
                       pruned ? pruned + (size_t)b * (Nv - budget) : nullptr,
                       slot_of ? slot_of + (size_t)b * Nv : nullptr, sm);
}

// ----------------------------------------------------------------------------
// gram_assign: grid (N1 tiles, Mp tiles, B).  A rows = pruned tokens, B rows =
// kept tokens.  Each workgroup finds, for each of its pruned rows, the best
// (cosine, slot) within its column tile; ordering (higher cosine, then lower
// slot) is a total order, so the maximum does not depend on reduction order.
// ----------------------------------------------------------------------------
__device__ __forceinline__ bool better(float v, int s, float bv, int bs) {
    return v > bv || (v == bv && s < bs);
}

template <int DT, int BM, int BN, int WM, int WN>
__global__ __launch_bounds__(64 * WM * WN) void gram_assign_kernel(
    const char *__restrict__ vis, int Nv, int d_bytes, const int32_t *__restrict__ kept, int N1,
    const int32_t *__restrict__ pruned, int Mp, const float *__restrict__ invn,
    float *__restrict__ best_val, int32_t *__restrict__ best_slot, int32_t *__restrict__ assign,
    unsigned *__restrict__ counters) {
    using G = TileGemm<DT, BM, BN, WM, WN>;
    __shared__ __attribute__((aligned(16))) char lds[G::LDS_BYTES];
    __shared__ int32_t rowtok[G::ROWS];
    __shared__ float rowinv[G::ROWS];
    __shared__ float red_v[WN][BM];
    __shared__ int red_s[WN][BM];
    __shared__ int is_last;

    const int nt = blockIdx.x, mt = blockIdx.y, b = blockIdx.z;
    const int ntn = gridDim.x, ntm = gridDim.y;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;
    const int m0 = mt * BM, n0 = nt * BN;
    const int32_t *pr = pruned + (size_t)b * Mp;
    const int32_t *kp = kept + (size_t)b * N1;

    for (int r = tid; r < G::ROWS; r += G::NT) {
        int tok = (r < BM) ? pr[min(m0 + r, Mp - 1)] : kp[min(n0 + r - BM, N1 - 1)];
        rowtok[r] = tok;
        rowinv[r] = invn[(size_t)b * Nv + tok];
    }
    __syncthreads();
    const char *vbase = vis + (size_t)b * Nv * d_bytes;
    auto row_ptr = [&](int r) -> const char * { return vbase + (size_t)rowtok[r] * d_bytes; };

    f32x4_t acc[G::FM][G::FN];
    float ss[G::PPT];
    G::template run<false>(row_ptr, d_bytes / G::CHUNK, lds, acc, ss);

#pragma unroll
    for (int fm = 0; fm < G::FM; ++fm) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = wm * G::SUB_M + fm * 16 + (lane >> 4) * 4 + i;
            const float ia = rowinv[r];
            float bv = -INFINITY;
            int bs = 0x7FFFFFFF;
#pragma unroll
            for (int fn = 0; fn < G::FN; ++fn) {
                const int c = wn * G::SUB_N + fn * 16 + (lane & 15);
                const int slot = n0 + c;
                const float cs = acc[fm][fn][i] * ia * rowinv[BM + c];
                if (slot < N1 && better(cs, slot, bv, bs)) {
                    bv = cs;
                    bs = slot;
                }
            }
#pragma unroll
            for (int off = 1; off < 16; off <<= 1) {
                float ov = __shfl_xor(bv, off, 64);
                int os = __shfl_xor(bs, off, 64);
                if (better(ov, os, bv, bs)) {
                    bv = ov;
                    bs = os;
                }
            }
            if ((lane & 15) == 0) {
                red_v[wn][r] = bv;
                red_s[wn][r] = bs;
            }
        }
    }
    __syncthreads();
    for (int r = tid; r < BM; r += G::NT) {
        float bv = red_v[0][r];
        int bs = red_s[0][r];
#pragma unroll
        for (int w = 1; w < WN; ++w)
            if (better(red_v[w][r], red_s[w][r], bv, bs)) {
                bv = red_v[w][r];
                bs = red_s[w][r];
            }
        const int m = m0 + r;
        if (m < Mp) {
            if (ntn == 1) {
                assign[(size_t)b * Nv + rowtok[r]] = bs;
            } else {
                best_val[((size_t)b * ntn + nt) * Mp + m] = bv;
                best_slot[((size_t)b * ntn + nt) * Mp + m] = bs;
            }
        }
    }
    if (ntn == 1) return;

    // The last column tile of this row tile reduces across column tiles.
    __threadfence();
    __syncthreads();
    if (tid == 0) is_last = (atomicAdd(&counters[(size_t)b * ntm + mt], 1u) == (unsigned)ntn - 1);
    __syncthreads();
    if (!is_last) return;
    __threadfence();
    for (int r = tid; r < BM; r += G::NT) {
        const int m = m0 + r;
        if (m >= Mp) continue;
        float bv = -INFINITY;
        int bs = 0x7FFFFFFF;
        for (int t = 0; t < ntn; ++t) {
            float v = best_val[((size_t)b * ntn + t) * Mp + m];
            int s = best_slot[((size_t)b * ntn + t) * Mp + m];
            if (better(v, s, bv, bs)) {
                bv = v;
                bs = s;
            }
        }
        assign[(size_t)b * Nv + rowtok[r]] = bs;
    }
}

// ----------------------------------------------------------------------------
// merge: grid (N1, B), 256 threads.  Members of slot s are found by scanning
// the assignment 64 tokens at a time with a wave ballot, in ascending token
// order, so the fp32 sums have a fixed order.
// ----------------------------------------------------------------------------
constexpr int kMergeNT = 256;
constexpr int kMergeCPT = 4;  // 16-byte chunks per thread per pass

template <int DT>
__global__ __launch_bounds__(kMergeNT) void merge_kernel(const char *__restrict__ vis, int Nv,
                                                         int d_bytes,
                                                         const int32_t *__restrict__ assign,
                                                         int N1, char *__restrict__ merged) {
    constexpr int EPC = (DT == kBF16) ? 8 : 4;  // elements per 16-byte chunk
    const int s = blockIdx.x, b = blockIdx.y;
    const int tid = threadIdx.x, lane = tid & 63;
    const int nchunk = d_bytes / 16;
    const int32_t *as = assign + (size_t)b * Nv;
    const char *vb = vis + (size_t)b * Nv * d_bytes;
    char *out = merged + ((size_t)b * N1 + s) * d_bytes;

    for (int cbase = 0; cbase < nchunk; cbase += kMergeNT * kMergeCPT) {
        float acc[kMergeCPT][EPC];
#pragma unroll
        for (int t = 0; t < kMergeCPT; ++t)
#pragma unroll
            for (int e = 0; e < EPC; ++e) acc[t][e] = 0.f;
        int count = 0;
        for (int base = 0; base < Nv; base += 64) {
            const int jj = base + lane;
            const int a = (jj < Nv) ? as[jj] : -1;
            unsigned long long mask = __ballot(a == s);
            while (mask) {
                const int bit = __ffsll((long long)mask) - 1;
                mask &= mask - 1ull;
                const char *row = vb + (size_t)(base + bit) * d_bytes;
                ++count;
#pragma unroll
                for (int t = 0; t < kMergeCPT; ++t) {
                    const int c = cbase + tid + t * kMergeNT;
                    if (c < nchunk) {
                        uint4 v = ld16(row + (size_t)c * 16);
                        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
                        if (DT == kBF16) {
#pragma unroll
                            for (int q = 0; q < 4; ++q) {
                                acc[t][2 * q] += __uint_as_float(w[q] << 16);
                                acc[t][2 * q + 1] += __uint_as_float(w[q] & 0xFFFF0000u);
                            }
                        } else {
#pragma unroll
                            for (int q = 0; q < 4; ++q) acc[t][q] += __uint_as_float(w[q]);
                        }
                    }
                }
            }
        }
        const float cnt = (float)count;
#pragma unroll
        for (int t = 0; t < kMergeCPT; ++t) {
            const int c = cbase + tid + t * kMergeNT;
            if (c >= nchunk) continue;
            uint4 v;
            uint32_t w[4];
            if (DT == kBF16) {
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    w[q] = f32_to_bf16_rne(acc[t][2 * q] / cnt) |
                           (f32_to_bf16_rne(acc[t][2 * q + 1] / cnt) << 16);
            } else {
#pragma unroll
                for (int q = 0; q < 4; ++q) w[q] = __float_as_uint(acc[t][q] / cnt);
            }
            v.x = w[0];
            v.y = w[1];
            v.z = w[2];
            v.w = w[3];
            st16(out + (size_t)c * 16, v);
        }
    }
}

// ----------------------------------------------------------------------------
// launchers
// ----------------------------------------------------------------------------
template <int DT, int BM, int BN, int WM, int WN>
static hipError_t cos_tile_go(const void *vis, const void *anchors, int B, int Nv, int Nt, int d,
                              float *M, float *invn, float *rowsum, unsigned *counters,
                              int n_counters, hipStream_t st) {
    const int esz = (DT == kBF16) ? 2 : 4;
    dim3 grid((Nv + BN - 1) / BN, (Nt + BM - 1) / BM, B);
    hipLaunchKernelGGL((cos_tile_kernel<DT, BM, BN, WM, WN>), grid, dim3(64 * WM * WN), 0, st,
                       (const char *)vis, (const char *)anchors, Nv, Nt, d * esz, M, invn, rowsum,
                       counters, n_counters);
    return hipGetLastError();
}

template <int DT>
static hipError_t cos_tile_dt(int cfg, const void *vis, const void *anchors, int B, int Nv, int Nt,
                              int d, float *M, float *invn, float *rowsum, unsigned *counters,
                              int n_counters, hipStream_t st) {
    switch (cfg) {
        case TILE_16:
            return cos_tile_go<DT, 16, 16, 1, 1>(vis, anchors, B, Nv, Nt, d, M, invn, rowsum, counters, n_counters, st);
        case TILE_32:
            return cos_tile_go<DT, 32, 32, 2, 2>(vis, anchors, B, Nv, Nt, d, M, invn, rowsum, counters, n_counters, st);
        case TILE_64:
            return cos_tile_go<DT, 64, 64, 2, 2>(vis, anchors, B, Nv, Nt, d, M, invn, rowsum, counters, n_counters, st);
        case TILE_128:
            return cos_tile_go<DT, 128, 128, 2, 2>(vis, anchors, B, Nv, Nt, d, M, invn, rowsum, counters, n_counters, st);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_cos_tile(int dt, int cfg, const void *vis, const void *anchors, int B, int Nv,
                           int Nt, int d, float *M, float *invn, float *rowsum, unsigned *counters,
                           int n_counters, hipStream_t st) {
    if (dt == kBF16)
        return cos_tile_dt<kBF16>(cfg, vis, anchors, B, Nv, Nt, d, M, invn, rowsum, counters, n_counters, st);
    return cos_tile_dt<kF32>(cfg, vis, anchors, B, Nv, Nt, d, M, invn, rowsum, counters, n_counters, st);
}

hipError_t launch_center_select(const float *M, const float *rowsum, int njt, int B, int Nt, int Nv,
                                float *p, int budget, int32_t *kept, int32_t *pruned,
                                int32_t *slot_of, unsigned *counters, hipStream_t st) {
    dim3 grid((Nv + kSelNT - 1) / kSelNT, B);
    hipLaunchKernelGGL(center_select_kernel, grid, dim3(kSelNT), Nt * sizeof(float), st, M, rowsum,
                       njt, Nt, Nv, p, budget, kept, pruned, slot_of, counters);
    return hipGetLastError();
}

template <int DT, int BM, int BN, int WM, int WN>
static hipError_t gram_go(const void *vis, int B, int Nv, int d, const int32_t *kept, int N1,
                          const int32_t *pruned, int Mp, const float *invn, float *best_val,
                          int32_t *best_slot, int32_t *assign, unsigned *counters, hipStream_t st) {
    const int esz = (DT == kBF16) ? 2 : 4;
    dim3 grid((N1 + BN - 1) / BN, (Mp + BM - 1) / BM, B);
    hipLaunchKernelGGL((gram_assign_kernel<DT, BM, BN, WM, WN>), grid, dim3(64 * WM * WN), 0, st,
                       (const char *)vis, Nv, d * esz, kept, N1, pruned, Mp, invn, best_val,
                       best_slot, assign, counters);
    return hipGetLastError();
}

template <int DT>
static hipError_t gram_dt(int cfg, const void *vis, int B, int Nv, int d, const int32_t *kept,
                          int N1, const int32_t *pruned, int Mp, const float *invn,
                          float *best_val, int32_t *best_slot, int32_t *assign,
                          unsigned *counters, hipStream_t st) {
    switch (cfg) {
        case TILE_16:
            return gram_go<DT, 16, 16, 1, 1>(vis, B, Nv, d, kept, N1, pruned, Mp, invn, best_val, best_slot, assign, counters, st);
        case TILE_32:
            return gram_go<DT, 32, 32, 2, 2>(vis, B, Nv, d, kept, N1, pruned, Mp, invn, best_val, best_slot, assign, counters, st);
        case TILE_64:
            return gram_go<DT, 64, 64, 2, 2>(vis, B, Nv, d, kept, N1, pruned, Mp, invn, best_val, best_slot, assign, counters, st);
        case TILE_128:
            return gram_go<DT, 128, 128, 2, 2>(vis, B, Nv, d, kept, N1, pruned, Mp, invn, best_val, best_slot, assign, counters, st);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_gram_assign(int dt, int cfg, const void *vis, int B, int Nv, int d,
                              const int32_t *kept, int N1, const int32_t *pruned, int Mp,
                              const float *invn, float *best_val, int32_t *best_slot,
                              int32_t *assign, unsigned *counters, hipStream_t st) {
    if (dt == kBF16)
        return gram_dt<kBF16>(cfg, vis, B, Nv, d, kept, N1, pruned, Mp, invn, best_val, best_slot, assign, counters, st);
    return gram_dt<kF32>(cfg, vis, B, Nv, d, kept, N1, pruned, Mp, invn, best_val, best_slot, assign, counters, st);
}

hipError_t launch_merge(int dt, const void *vis, int B, int Nv, int d, const int32_t *kept, int N1,
                        const int32_t *assign, void *merged, hipStream_t st) {
    (void)kept;
    dim3 grid(N1, B);
    if (dt == kBF16)
        hipLaunchKernelGGL(merge_kernel<kBF16>, grid, dim3(kMergeNT), 0, st, (const char *)vis, Nv,
                           d * 2, assign, N1, (char *)merged);
    else
        hipLaunchKernelGGL(merge_kernel<kF32>, grid, dim3(kMergeNT), 0, st, (const char *)vis, Nv,
                           d * 4, assign, N1, (char *)merged);
    return hipGetLastError();
}

}  // namespace pv
