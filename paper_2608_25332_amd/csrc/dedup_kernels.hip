// Pruning before the LLM (Sec. 4.3): cross-modal cosine (equation for M),
// row centring (equation for M-hat), max-pooling (equation for p), top-N_1,
// nearest-centroid assignment of the pruned tokens and their aggregation.
//
// Kernel sequence of one call (all on the caller's stream):
//   cos_stream    anchors x vis on MFMA (streaming tiles, norms fused);
//                 writes the cosines, the inverse norms of the visual tokens
//                 and per-tile row sums
//   center        p[j] = max_i (M[i][j] - mean_i)
//   select        top-N_1 radix select, one workgroup per sample
//   gram_*        pruned x kept cosine Gram on MFMA with a fused row argmax
//                 per column tile (streaming tiles at small sizes, LDS-staged
//                 128x128 tiles when the Gram is large enough to be
//                 MFMA-bound)
//   gram_finish   best column tile per pruned row -> assignment
//   merge         centroid <- mean of itself and its members
// Workgroups never wait on or signal each other: every cross-workgroup
// dependency is a kernel boundary, so no kernel needs a device-wide fence
// (on this chip a device-scope fence writes back and invalidates the L2).
#include "pv_launch.h"
#include "pv_stream_tile.h"
#include "pv_tile_gemm.h"

#include <math.h>

namespace pv {

int tile_size(int cfg) { return 16 << cfg; }

// Waves and unroll depth of a streaming tile: enough 16-byte loads in flight
// per workgroup to cover memory latency within ~128 VGPRs of fragments.
template <int T> struct StreamCfg;
template <> struct StreamCfg<16> { static constexpr int NW = 8, U = 8; };
template <> struct StreamCfg<32> { static constexpr int NW = 4, U = 4; };
template <> struct StreamCfg<64> { static constexpr int NW = 4, U = 2; };

// ----------------------------------------------------------------------------
// cos_stream: 1-D grid over (sample, vis tile, anchor tile) in XCD order.
// ----------------------------------------------------------------------------
template <int DT, int T>
__global__ __launch_bounds__(64 * StreamCfg<T>::NW) void cos_stream_kernel(
    const char *__restrict__ vis, const char *__restrict__ anchors, int B, int Nv, int Nt,
    int d_bytes, int njt, int nit, float *__restrict__ M, float *__restrict__ invn_vis,
    float *__restrict__ rowsum) {
    constexpr int NW = StreamCfg<T>::NW, U = StreamCfg<T>::U;
    using S = StreamTile<DT, T, T, NW, U>;
    constexpr int F = T / 16;
    __shared__ float red[S::RED_FLOATS];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int total = B * njt * nit;
    const int tile = xcd_tile(blockIdx.x, total);
    const int it = tile % nit;
    const int jt = (tile / nit) % njt;
    const int b = tile / (nit * njt);

    const int i0 = it * T, j0 = jt * T;
    const int koff = (lane >> 4) * 16;
    const char *abase = anchors + (size_t)b * Nt * d_bytes + koff;
    const char *vbase = vis + (size_t)b * Nv * d_bytes + koff;
    const char *rp[2 * F];
#pragma unroll
    for (int f = 0; f < F; ++f) {
        rp[f] = abase + (size_t)min(i0 + f * 16 + (lane & 15), Nt - 1) * d_bytes;
        rp[F + f] = vbase + (size_t)min(j0 + f * 16 + (lane & 15), Nv - 1) * d_bytes;
    }
    f32x4_t acc[F][F];
    float ss[2 * F];
    S::template run<true>(rp, d_bytes / 64, acc, ss);
    S::template reduce<true>(acc, ss, red);
    if (wave != 0) return;

    float inv[2 * F];
#pragma unroll
    for (int q = 0; q < 2 * F; ++q) inv[q] = (ss[q] > 0.f) ? 1.0f / sqrtf(ss[q]) : 0.f;
    if (it == 0 && lane < 16) {
#pragma unroll
        for (int f = 0; f < F; ++f) {
            const int j = j0 + f * 16 + lane;
            if (j < Nv) invn_vis[(size_t)b * Nv + j] = inv[F + f];
        }
    }
#pragma unroll
    for (int fm = 0; fm < F; ++fm) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int rl = (lane >> 4) * 4 + e;  // row inside the 16-row block
            const int gi = i0 + fm * 16 + rl;
            const float ia = __shfl(inv[fm], rl, 64);
            float rs = 0.f;
#pragma unroll
            for (int fn = 0; fn < F; ++fn) {
                const int gj = j0 + fn * 16 + (lane & 15);
                const float cs = acc[fm][fn][e] * ia * inv[F + fn];
                if (gj < Nv) {
                    rs += cs;
                    if (gi < Nt) M[((size_t)b * Nt + gi) * Nv + gj] = cs;
                }
            }
            rs += __shfl_xor(rs, 1, 64);
            rs += __shfl_xor(rs, 2, 64);
            rs += __shfl_xor(rs, 4, 64);
            rs += __shfl_xor(rs, 8, 64);
            if ((lane & 15) == 0 && gi < Nt) rowsum[((size_t)b * njt + jt) * Nt + gi] = rs;
        }
    }
}

// ----------------------------------------------------------------------------
// center: grid (ceil(Nv / 64), B), 256 threads; 4 threads per token.
// ----------------------------------------------------------------------------
constexpr int kCenNT = 256;
constexpr int kCenTok = 64;

__global__ __launch_bounds__(kCenNT) void center_kernel(const float *__restrict__ M,
                                                        const float *__restrict__ rowsum, int njt,
                                                        int Nt, int Nv, float *__restrict__ p) {
    extern __shared__ float mu[];  // [Nt]
    __shared__ float part[4][kCenTok];
    const int b = blockIdx.y, tid = threadIdx.x;
    // Row means of M over all Nv tokens, from the per-tile partial sums
    // (added in tile order).
    for (int i = tid; i < Nt; i += kCenNT) {
        const float *rs = rowsum + (size_t)b * njt * Nt + i;
        float s = 0.f;
#pragma unroll 8
        for (int t = 0; t < njt; ++t) s += rs[(size_t)t * Nt];
        mu[i] = s / (float)Nv;
    }
    __syncthreads();
    const int jl = tid & (kCenTok - 1), g = tid / kCenTok;
    const int j = blockIdx.x * kCenTok + jl;
    float m = -INFINITY;
    if (j < Nv) {
        const float *col = M + (size_t)b * Nt * Nv + j;
#pragma unroll 4
        for (int i = g; i < Nt; i += 4) m = fmaxf(m, col[(size_t)i * Nv] - mu[i]);
    }
    part[g][jl] = m;
    __syncthreads();
    if (g == 0 && j < Nv)
        p[(size_t)b * Nv + j] = fmaxf(fmaxf(part[0][jl], part[1][jl]), fmaxf(part[2][jl], part[3][jl]));
}

// ----------------------------------------------------------------------------
// select: grid (B), 256 threads; top-`budget` of p with its complement list
// and the slot of every kept token.  Keys are staged in LDS up to kStageKeys.
// ----------------------------------------------------------------------------
constexpr int kSelNT = 256;
constexpr int kStageKeys = 8192;

__global__ __launch_bounds__(kSelNT) void select_kernel(const float *__restrict__ p, int Nv,
                                                        int budget, int32_t *__restrict__ kept,
                                                        int32_t *__restrict__ pruned,
                                                        int32_t *__restrict__ slot_of) {
    extern __shared__ uint32_t keys[];  // [Nv] when staged
    __shared__ TopkSmem sm;
    const int b = blockIdx.x;
    block_topk<kSelNT>(p + (size_t)b * Nv, Nv, budget, kept + (size_t)b * budget,
                       pruned ? pruned + (size_t)b * (Nv - budget) : nullptr,
                       slot_of ? slot_of + (size_t)b * Nv : nullptr, sm,
                       Nv <= kStageKeys ? keys : nullptr);
}

// ----------------------------------------------------------------------------
// Nearest centroid: best (cosine, slot) of every pruned row.  Ordering by
// higher cosine, then lower slot, is a total order, so the maximum does not
// depend on the order in which candidates are combined.
// ----------------------------------------------------------------------------
__device__ __forceinline__ bool better(float v, int s, float bv, int bs) {
    return v > bv || (v == bv && s < bs);
}

// gram_finish: grid (ceil(Mp / 256), B).  Best column tile of every pruned
// row, combined in tile order with the total order above.
constexpr int kFinNT = 256;

__global__ __launch_bounds__(kFinNT) void gram_finish_kernel(const float *__restrict__ best_val,
                                                             const int32_t *__restrict__ best_slot,
                                                             int ntn, int Mp, int Nv,
                                                             const int32_t *__restrict__ pruned,
                                                             int32_t *__restrict__ assign) {
    const int b = blockIdx.y;
    const int m = blockIdx.x * kFinNT + threadIdx.x;
    if (m >= Mp) return;
    float bv = -INFINITY;
    int bs = 0x7FFFFFFF;
    for (int t = 0; t < ntn; ++t) {
        const float v = best_val[((size_t)b * ntn + t) * Mp + m];
        const int s = best_slot[((size_t)b * ntn + t) * Mp + m];
        if (better(v, s, bv, bs)) {
            bv = v;
            bs = s;
        }
    }
    assign[(size_t)b * Nv + pruned[(size_t)b * Mp + m]] = bs;
}

// gram_stream: 1-D grid over (sample, pruned-row tile, kept-column tile).
template <int DT, int T>
__global__ __launch_bounds__(64 * StreamCfg<T>::NW) void gram_stream_kernel(
    const char *__restrict__ vis, int B, int Nv, int d_bytes, const int32_t *__restrict__ kept,
    int N1, const int32_t *__restrict__ pruned, int Mp, int ntm, int ntn,
    const float *__restrict__ invn, float *__restrict__ best_val,
    int32_t *__restrict__ best_slot, int32_t *__restrict__ assign) {
    constexpr int NW = StreamCfg<T>::NW, U = StreamCfg<T>::U;
    using S = StreamTile<DT, T, T, NW, U>;
    constexpr int F = T / 16;
    __shared__ float red[S::RED_FLOATS];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int total = B * ntm * ntn;
    const int tile = xcd_tile(blockIdx.x, total);
    const int nt = tile % ntn;
    const int mt = (tile / ntn) % ntm;
    const int b = tile / (ntn * ntm);
    const int m0 = mt * T, n0 = nt * T;
    const int32_t *pr = pruned + (size_t)b * Mp;
    const int32_t *kp = kept + (size_t)b * N1;
    const int koff = (lane >> 4) * 16;
    const char *vbase = vis + (size_t)b * Nv * d_bytes + koff;

    const char *rp[2 * F];
    float inv[2 * F];
#pragma unroll
    for (int f = 0; f < F; ++f) {
        const int ta = pr[min(m0 + f * 16 + (lane & 15), Mp - 1)];
        const int tb = kp[min(n0 + f * 16 + (lane & 15), N1 - 1)];
        rp[f] = vbase + (size_t)ta * d_bytes;
        rp[F + f] = vbase + (size_t)tb * d_bytes;
        inv[f] = invn[(size_t)b * Nv + ta];
        inv[F + f] = invn[(size_t)b * Nv + tb];
    }
    f32x4_t acc[F][F];
    float ss[2 * F];
    S::template run<false>(rp, d_bytes / 64, acc, ss);
    S::template reduce<false>(acc, ss, red);

    if (wave == 0) {
#pragma unroll
        for (int fm = 0; fm < F; ++fm) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int rl = (lane >> 4) * 4 + e;
                const float ia = __shfl(inv[fm], rl, 64);
                float bv = -INFINITY;
                int bs = 0x7FFFFFFF;
#pragma unroll
                for (int fn = 0; fn < F; ++fn) {
                    const int slot = n0 + fn * 16 + (lane & 15);
                    const float cs = acc[fm][fn][e] * ia * inv[F + fn];
                    if (slot < N1 && better(cs, slot, bv, bs)) {
                        bv = cs;
                        bs = slot;
                    }
                }
#pragma unroll
                for (int off = 1; off < 16; off <<= 1) {
                    const float ov = __shfl_xor(bv, off, 64);
                    const int os = __shfl_xor(bs, off, 64);
                    if (better(ov, os, bv, bs)) {
                        bv = ov;
                        bs = os;
                    }
                }
                const int m = m0 + fm * 16 + rl;
                if ((lane & 15) == 0 && m < Mp) {
                    if (ntn == 1) {
                        assign[(size_t)b * Nv + pr[m]] = bs;
                    } else {
                        best_val[((size_t)b * ntn + nt) * Mp + m] = bv;
                        best_slot[((size_t)b * ntn + nt) * Mp + m] = bs;
                    }
                }
            }
        }
    }
}

// gram_tile: LDS-staged 128 x 128 tiles for the large, MFMA-bound Grams.
// grid (N1 tiles, Mp tiles, B).
template <int DT, int BM, int BN, int WM, int WN>
__global__ __launch_bounds__(64 * WM * WN) void gram_tile_kernel(
    const char *__restrict__ vis, int Nv, int d_bytes, const int32_t *__restrict__ kept, int N1,
    const int32_t *__restrict__ pruned, int Mp, const float *__restrict__ invn,
    float *__restrict__ best_val, int32_t *__restrict__ best_slot, int32_t *__restrict__ assign) {
    using G = TileGemm<DT, BM, BN, WM, WN>;
    __shared__ __attribute__((aligned(16))) char lds[G::LDS_BYTES];
    __shared__ int32_t rowtok[G::ROWS];
    __shared__ float rowinv[G::ROWS];
    __shared__ float red_v[WN][BM];
    __shared__ int red_s[WN][BM];

    const int nt = blockIdx.x, mt = blockIdx.y, b = blockIdx.z;
    const int ntn = gridDim.x;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;
    const int m0 = mt * BM, n0 = nt * BN;
    const int32_t *pr = pruned + (size_t)b * Mp;
    const int32_t *kp = kept + (size_t)b * N1;

    for (int r = tid; r < G::ROWS; r += G::NT) {
        const int tok = (r < BM) ? pr[min(m0 + r, Mp - 1)] : kp[min(n0 + r - BM, N1 - 1)];
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
                const float ov = __shfl_xor(bv, off, 64);
                const int os = __shfl_xor(bs, off, 64);
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
}

// ----------------------------------------------------------------------------
// merge: grid (N1, B), 256 threads.  The members of slot s (the tokens whose
// assignment is s, the kept token itself included) are collected in
// ascending token order by one wave with ballots over the assignment (staged
// in LDS when it fits), then all threads add the member rows in that order
// (fp32), four rows in flight at a time.
// ----------------------------------------------------------------------------
constexpr int kMergeNT = 256;
constexpr int kMergeCPT = 4;      // 16-byte chunks per thread per pass
constexpr int kMergeList = 4096;  // members held in LDS per round; also the
                                  // largest assignment staged in LDS

template <int DT>
__global__ __launch_bounds__(kMergeNT) void merge_kernel(const char *__restrict__ vis, int Nv,
                                                         int d_bytes,
                                                         const int32_t *__restrict__ assign,
                                                         int N1, char *__restrict__ merged) {
    constexpr int EPC = (DT == kBF16) ? 8 : 4;  // elements per 16-byte chunk
    __shared__ int list[kMergeList];
    __shared__ int staged[kMergeList];
    __shared__ int s_count, s_next;
    const int s = blockIdx.x, b = blockIdx.y;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int nchunk = d_bytes / 16;
    const int32_t *as = assign + (size_t)b * Nv;
    const char *vb = vis + (size_t)b * Nv * d_bytes;
    char *out = merged + ((size_t)b * N1 + s) * d_bytes;
    const bool stage = Nv <= kMergeList;
    if (stage) {
        for (int j = tid; j < Nv; j += kMergeNT) staged[j] = as[j];
        __syncthreads();
    }
    const int *src = stage ? (const int *)staged : (const int *)as;

    for (int cbase = 0; cbase < nchunk; cbase += kMergeNT * kMergeCPT) {
        float acc[kMergeCPT][EPC];
#pragma unroll
        for (int t = 0; t < kMergeCPT; ++t)
#pragma unroll
            for (int e = 0; e < EPC; ++e) acc[t][e] = 0.f;
        int scan_from = 0, total = 0;
        while (true) {
            if (wave == 0) {
                // collect up to kMergeList members from token scan_from on
                int cnt = 0, pos = scan_from;
                while (pos < Nv) {
                    const int a0 = (pos + lane < Nv) ? src[pos + lane] : -1;
                    const unsigned long long mk = __ballot(a0 == s);
                    const int nb = __popcll(mk);
                    if (cnt + nb > kMergeList) break;
                    if (a0 == s) list[cnt + __popcll(mk & ((1ull << lane) - 1ull))] = pos + lane;
                    cnt += nb;
                    pos += 64;
                }
                if (lane == 0) {
                    s_count = cnt;
                    s_next = pos;
                }
            }
            __syncthreads();
            const int cnt = s_count;
            scan_from = s_next;
            total += cnt;
            for (int m = 0; m < cnt; m += 4) {
                uint4 v[4][kMergeCPT];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const char *row = vb + (size_t)list[min(m + u, cnt - 1)] * d_bytes;
#pragma unroll
                    for (int t = 0; t < kMergeCPT; ++t) {
                        const int c = min(cbase + tid + t * kMergeNT, nchunk - 1);
                        v[u][t] = ld16(row + (size_t)c * 16);
                    }
                }
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    if (m + u >= cnt) break;
#pragma unroll
                    for (int t = 0; t < kMergeCPT; ++t) {
                        const uint32_t w4[4] = {v[u][t].x, v[u][t].y, v[u][t].z, v[u][t].w};
                        if (DT == kBF16) {
#pragma unroll
                            for (int q = 0; q < 4; ++q) {
                                acc[t][2 * q] += __uint_as_float(w4[q] << 16);
                                acc[t][2 * q + 1] += __uint_as_float(w4[q] & 0xFFFF0000u);
                            }
                        } else {
#pragma unroll
                            for (int q = 0; q < 4; ++q) acc[t][q] += __uint_as_float(w4[q]);
                        }
                    }
                }
            }
            __syncthreads();
            if (scan_from >= Nv) break;
        }
        const float cnt = (float)total;
#pragma unroll
        for (int t = 0; t < kMergeCPT; ++t) {
            const int c = cbase + tid + t * kMergeNT;
            if (c >= nchunk) continue;
            uint32_t w4[4];
            if (DT == kBF16) {
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    w4[q] = f32_to_bf16_rne(acc[t][2 * q] / cnt) |
                            (f32_to_bf16_rne(acc[t][2 * q + 1] / cnt) << 16);
            } else {
#pragma unroll
                for (int q = 0; q < 4; ++q) w4[q] = __float_as_uint(acc[t][q] / cnt);
            }
            st16(out + (size_t)c * 16, uint4{w4[0], w4[1], w4[2], w4[3]});
        }
    }
}

// ----------------------------------------------------------------------------
// launchers
// ----------------------------------------------------------------------------
template <int DT, int T>
static hipError_t cos_go(const void *vis, const void *anchors, int B, int Nv, int Nt, int d,
                         float *M, float *invn, float *rowsum, hipStream_t st) {
    const int esz = (DT == kBF16) ? 2 : 4;
    const int njt = (Nv + T - 1) / T, nit = (Nt + T - 1) / T;
    hipLaunchKernelGGL((cos_stream_kernel<DT, T>), dim3(B * njt * nit),
                       dim3(64 * StreamCfg<T>::NW), 0, st, (const char *)vis, (const char *)anchors,
                       B, Nv, Nt, d * esz, njt, nit, M, invn, rowsum);
    return hipGetLastError();
}

template <int DT>
static hipError_t cos_dt(int cfg, const void *vis, const void *anchors, int B, int Nv, int Nt,
                         int d, float *M, float *invn, float *rowsum, hipStream_t st) {
    switch (cfg) {
        case TILE_16: return cos_go<DT, 16>(vis, anchors, B, Nv, Nt, d, M, invn, rowsum, st);
        case TILE_32: return cos_go<DT, 32>(vis, anchors, B, Nv, Nt, d, M, invn, rowsum, st);
        case TILE_64: return cos_go<DT, 64>(vis, anchors, B, Nv, Nt, d, M, invn, rowsum, st);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_cos_tile(int dt, int cfg, const void *vis, const void *anchors, int B, int Nv,
                           int Nt, int d, float *M, float *invn, float *rowsum, hipStream_t st) {
    if (dt == kBF16) return cos_dt<kBF16>(cfg, vis, anchors, B, Nv, Nt, d, M, invn, rowsum, st);
    return cos_dt<kF32>(cfg, vis, anchors, B, Nv, Nt, d, M, invn, rowsum, st);
}

hipError_t launch_center(const float *M, const float *rowsum, int njt, int B, int Nt, int Nv,
                         float *p, hipStream_t st) {
    dim3 grid((Nv + kCenTok - 1) / kCenTok, B);
    hipLaunchKernelGGL(center_kernel, grid, dim3(kCenNT), (size_t)Nt * sizeof(float), st, M, rowsum,
                       njt, Nt, Nv, p);
    return hipGetLastError();
}

hipError_t launch_select(const float *p, int B, int Nv, int budget, int32_t *kept, int32_t *pruned,
                         int32_t *slot_of, hipStream_t st) {
    const size_t lds = (Nv <= kStageKeys) ? (size_t)Nv * sizeof(uint32_t) : 0;
    hipLaunchKernelGGL(select_kernel, dim3(B), dim3(kSelNT), lds, st, p, Nv, budget, kept, pruned,
                       slot_of);
    return hipGetLastError();
}

template <int DT, int T>
static hipError_t gram_stream_go(const void *vis, int B, int Nv, int d, const int32_t *kept,
                                 int N1, const int32_t *pruned, int Mp, const float *invn,
                                 float *best_val, int32_t *best_slot, int32_t *assign,
                                 hipStream_t st) {
    const int esz = (DT == kBF16) ? 2 : 4;
    const int ntm = (Mp + T - 1) / T, ntn = (N1 + T - 1) / T;
    hipLaunchKernelGGL((gram_stream_kernel<DT, T>), dim3(B * ntm * ntn),
                       dim3(64 * StreamCfg<T>::NW), 0, st, (const char *)vis, B, Nv, d * esz,
                       kept, N1, pruned, Mp, ntm, ntn, invn, best_val, best_slot, assign);
    return hipGetLastError();
}

template <int DT>
static hipError_t gram_tile_go(const void *vis, int B, int Nv, int d, const int32_t *kept, int N1,
                               const int32_t *pruned, int Mp, const float *invn, float *best_val,
                               int32_t *best_slot, int32_t *assign, hipStream_t st) {
    const int esz = (DT == kBF16) ? 2 : 4;
    dim3 grid((N1 + 127) / 128, (Mp + 127) / 128, B);
    hipLaunchKernelGGL((gram_tile_kernel<DT, 128, 128, 2, 2>), grid, dim3(256), 0, st,
                       (const char *)vis, Nv, d * esz, kept, N1, pruned, Mp, invn, best_val,
                       best_slot, assign);
    return hipGetLastError();
}

template <int DT>
static hipError_t gram_dt(int cfg, const void *vis, int B, int Nv, int d, const int32_t *kept,
                          int N1, const int32_t *pruned, int Mp, const float *invn,
                          float *best_val, int32_t *best_slot, int32_t *assign, hipStream_t st) {
    switch (cfg) {
        case TILE_16: return gram_stream_go<DT, 16>(vis, B, Nv, d, kept, N1, pruned, Mp, invn, best_val, best_slot, assign, st);
        case TILE_32: return gram_stream_go<DT, 32>(vis, B, Nv, d, kept, N1, pruned, Mp, invn, best_val, best_slot, assign, st);
        case TILE_64: return gram_stream_go<DT, 64>(vis, B, Nv, d, kept, N1, pruned, Mp, invn, best_val, best_slot, assign, st);
        case TILE_128: return gram_tile_go<DT>(vis, B, Nv, d, kept, N1, pruned, Mp, invn, best_val, best_slot, assign, st);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_gram(int dt, int cfg, const void *vis, int B, int Nv, int d, const int32_t *kept,
                       int N1, const int32_t *pruned, int Mp, const float *invn, float *best_val,
                       int32_t *best_slot, int32_t *assign, hipStream_t st) {
    if (dt == kBF16)
        return gram_dt<kBF16>(cfg, vis, B, Nv, d, kept, N1, pruned, Mp, invn, best_val, best_slot, assign, st);
    return gram_dt<kF32>(cfg, vis, B, Nv, d, kept, N1, pruned, Mp, invn, best_val, best_slot, assign, st);
}

hipError_t launch_gram_finish(const float *best_val, const int32_t *best_slot, int B, int ntn,
                              int Mp, int Nv, const int32_t *pruned, int32_t *assign,
                              hipStream_t st) {
    dim3 grid((Mp + kFinNT - 1) / kFinNT, B);
    hipLaunchKernelGGL(gram_finish_kernel, grid, dim3(kFinNT), 0, st, best_val, best_slot, ntn, Mp,
                       Nv, pruned, assign);
    return hipGetLastError();
}

hipError_t launch_merge(int dt, const void *vis, int B, int Nv, int d, int N1,
                        const int32_t *assign, void *merged, hipStream_t st) {
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
