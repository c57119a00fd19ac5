// Latency-oriented "row x row" tile product on the matrix cores (gfx950).
//
// For the memory-bound products of the pruning path (the text x visual
// cosine, and the pruned x kept Gram at small batch) the limit is how many
// bytes each CU keeps in flight, not MFMA throughput.  Here every wave of the
// workgroup computes the whole BM x BN tile over its own contiguous slice of
// the k dimension and loads its MFMA fragments straight from global memory:
// lane l reads 16 bytes of row (l % 16) at byte (l / 16) * 16 of each 64-byte
// k window, which is the fragment layout, so no LDS staging and no barrier is
// needed in the k loop.  Windows are fetched U at a time and double-buffered
// (the next U windows are in flight while the current U are multiplied).
// At the end the waves' partial tiles are added in LDS in wave order, so the
// result is deterministic and the same for every row position.
#pragma once

#include "pv_device.h"

namespace pv {

template <int DT, int BM, int BN, int NW, int U>
struct StreamTile {
    static constexpr int NT = 64 * NW;
    static constexpr int FM = BM / 16, FN = BN / 16;
    static constexpr int NF = FM + FN;
    // LDS used by reduce(): (NW - 1) partial tiles + (NW - 1) x (BM + BN) sums of squares
    static constexpr int RED_FLOATS = (NW - 1) * (BM * BN + BM + BN);
    static_assert(BM % 16 == 0 && BN % 16 == 0, "16-aligned tiles");

    struct Frag {
        uint4 f[U][NF];
    };

    // Loads are unconditional (windows past the slice are clamped to the
    // slice's last window, or window 0 for an empty slice): the compiler can
    // then count the loads in flight and wait only for the batch it is about
    // to multiply, not for the prefetched one.
    __device__ __forceinline__ static void load(Frag &fr, const char *const (&rp)[NF], int t,
                                                int t_end) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            int tt = t + u;
            tt = tt < t_end ? tt : t_end - 1;
            tt = tt > 0 ? tt : 0;
#pragma unroll
            for (int q = 0; q < NF; ++q) fr.f[u][q] = ld16(rp[q] + (size_t)tt * 64);
        }
    }

    template <bool WANT_SS>
    __device__ __forceinline__ static void compute(const Frag &fr, int t, int t_end,
                                                   f32x4_t (&acc)[FM][FN], float (&ss)[NF]) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (t + u < t_end) {
#pragma unroll
                for (int i = 0; i < FM; ++i)
#pragma unroll
                    for (int j = 0; j < FN; ++j)
                        acc[i][j] = mma16<DT>(fr.f[u][i], fr.f[u][FM + j], acc[i][j]);
                if (WANT_SS) {
#pragma unroll
                    for (int q = 0; q < NF; ++q) ss[q] += sumsq16<DT>(fr.f[u][q]);
                }
            }
        }
    }

    // rp[q]: byte address of this lane's row for fragment q (q < FM: A block
    // rows, q >= FM: B block rows), already offset by the lane's 16-byte slot.
    // nwin: number of 64-byte windows per row (row bytes / 64).
    template <bool WANT_SS>
    __device__ __forceinline__ static void run(const char *const (&rp)[NF], int nwin,
                                               f32x4_t (&acc)[FM][FN], float (&ss)[NF]) {
        // The wave index must be known uniform to the compiler: the window
        // guards below then become scalar branches.  As vector-masked
        // branches, an MFMA in a block whose lanes are all masked off would
        // still run (the matrix core does not honour the execution mask) on
        // fragment registers that were never loaded.
        const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
        const int t0 = (int)(((long long)nwin * wave) / NW);
        const int t1 = (int)(((long long)nwin * (wave + 1)) / NW);
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int q = 0; q < NF; ++q) ss[q] = 0.f;
        Frag a, b;
        load(a, rp, t0, t1);
        for (int t = t0; t < t1; t += 2 * U) {
            load(b, rp, t + U, t1);
            compute<WANT_SS>(a, t, t1, acc, ss);
            load(a, rp, t + 2 * U, t1);
            compute<WANT_SS>(b, t + U, t1, acc, ss);
        }
    }

    // Sum the NW partial tiles (and sums of squares) into wave 0's registers,
    // adding in wave order 0, 1, ..., NW-1.  Per lane the squares are first
    // combined over the four 16-byte slots of a window (xor 16, 32), giving
    // each lane the full partial of its row.  Must be called by all threads.
    template <bool WANT_SS>
    __device__ __forceinline__ static void reduce(f32x4_t (&acc)[FM][FN], float (&ss)[NF],
                                                  float *red) {
        const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
        if (WANT_SS) {
#pragma unroll
            for (int q = 0; q < NF; ++q) {
                ss[q] += __shfl_xor(ss[q], 16, 64);
                ss[q] += __shfl_xor(ss[q], 32, 64);
            }
        }
        if (NW == 1) return;
        if (wave > 0) {
            float *dst = red + (size_t)(wave - 1) * (BM * BN + BM + BN);
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
#pragma unroll
                    for (int e = 0; e < 4; ++e) dst[((i * FN + j) * 4 + e) * 64 + lane] = acc[i][j][e];
            if (WANT_SS && lane < 16) {
#pragma unroll
                for (int q = 0; q < NF; ++q) dst[BM * BN + q * 16 + lane] = ss[q];
            }
        }
        __syncthreads();
        if (wave == 0) {
#pragma unroll
            for (int w = 1; w < NW; ++w) {
                const float *src = red + (size_t)(w - 1) * (BM * BN + BM + BN);
#pragma unroll
                for (int i = 0; i < FM; ++i)
#pragma unroll
                    for (int j = 0; j < FN; ++j)
#pragma unroll
                        for (int e = 0; e < 4; ++e) acc[i][j][e] += src[((i * FN + j) * 4 + e) * 64 + lane];
                if (WANT_SS) {
#pragma unroll
                    for (int q = 0; q < NF; ++q) ss[q] += src[BM * BN + q * 16 + (lane & 15)];
                }
            }
        }
    }
};

}  // namespace pv
