// LDS-staged "row x row" tile product on the matrix cores (gfx950).
//
// Both operands are sets of rows of length d (the embedding width), as stored
// in HBM: C[m][n] = dot(A_row(m), B_row(n)).  That is a GEMM whose two inputs
// are both k-contiguous, which is the layout the MFMA fragments want: every
// lane supplies 16 contiguous bytes of one row.
//
// One workgroup owns a BM x BN output tile and a range of 128-byte k chunks
// (64 bf16 or 32 f32 elements per row); the WM x WN waves each own a
// (BM/WM) x (BN/WN) sub-tile, so no cross-wave reduction is needed.  Rows are
// fetched G chunks at a time with row-major 16-byte loads (8 consecutive
// lanes cover one row's 128 bytes: the pattern that gets the most bytes per
// clock into a CU on this chip), written to LDS with a 16-byte pad per row,
// and the next G chunks are in flight while the current ones are multiplied
// from LDS.  Rows are addressed through a per-row pointer, so gathered
// operands (the pruned and kept token lists) cost nothing extra; rows past the
// valid count are clamped to a valid row by the caller and masked in its
// epilogue.
#pragma once

#include "pv_device.h"

namespace pv {

template <int DT, int BM, int BN, int WM, int WN, int G>
struct TileGemm {
    static constexpr int NT = 64 * WM * WN;
    static constexpr int ROWS = BM + BN;
    static constexpr int CHUNK = 128;   // bytes of one row per k chunk
    static constexpr int STRIDE = 144;  // LDS bytes per staged row (16-byte pad)
    static constexpr int PIECES = ROWS * (CHUNK / 16);
    static constexpr int PPT = PIECES / NT;  // 16-byte pieces per thread per chunk
    static constexpr int SUB_M = BM / WM, SUB_N = BN / WN;
    static constexpr int FM = SUB_M / 16, FN = SUB_N / 16;
    static constexpr int STAGE_BYTES = ROWS * STRIDE;
    static constexpr int LDS_BYTES = G * STAGE_BYTES;
    static_assert(PIECES % NT == 0, "tile rows must fill the loaders evenly");
    static_assert(SUB_M % 16 == 0 && SUB_N % 16 == 0, "wave tile must be 16-aligned");

    // Staged row of piece slot p of this thread (the same for every chunk).
    __device__ __forceinline__ static int row_of_piece(int p) { return (threadIdx.x + p * NT) >> 3; }

    // Multiply the chunks [c_begin, c_end).  row_ptr(r) gives the global byte
    // address of staged row r (r < BM: A rows, r >= BM: B rows).  With WANT_SS,
    // ss[p] is this thread's partial sum of squares of row row_of_piece(p).
    template <bool WANT_SS, typename RowPtr>
    __device__ __forceinline__ static void run(RowPtr row_ptr, int c_begin, int c_end, char *lds,
                                               f32x4_t (&acc)[FM][FN], float (&ss)[PPT]) {
        const int tid = threadIdx.x;
        const int lane = tid & 63;
        const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
        const int wm = wave / WN, wn = wave % WN;
        const char *src[PPT];
        int dst[PPT];
#pragma unroll
        for (int p = 0; p < PPT; ++p) {
            const int q = tid + p * NT;
            const int r = q >> 3, c = q & 7;
            src[p] = row_ptr(r) + c * 16;
            dst[p] = r * STRIDE + c * 16;
            ss[p] = 0.f;
        }
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

        const int a_row = wm * SUB_M + (lane & 15);
        const int b_row = BM + wn * SUB_N + (lane & 15);
        const int koff = (lane >> 4) * 16;

        uint4 buf[G][PPT];
        auto fetch = [&](int c0) {
#pragma unroll
            for (int g = 0; g < G; ++g) {
                int c = c0 + g;
                c = c < c_end ? c : c_end - 1;  // past the range: re-read the last chunk
#pragma unroll
                for (int p = 0; p < PPT; ++p) buf[g][p] = ld16(src[p] + (size_t)c * CHUNK);
            }
        };
        if (c_begin >= c_end) return;
        fetch(c_begin);
        for (int c0 = c_begin; c0 < c_end; c0 += G) {
            __syncthreads();  // the previous group's LDS reads are done
#pragma unroll
            for (int g = 0; g < G; ++g) {
                if (c0 + g < c_end) {
#pragma unroll
                    for (int p = 0; p < PPT; ++p) {
                        st16(lds + g * STAGE_BYTES + dst[p], buf[g][p]);
                        if (WANT_SS) ss[p] += sumsq16<DT>(buf[g][p]);
                    }
                }
            }
            __syncthreads();
            if (c0 + G < c_end) fetch(c0 + G);
#pragma unroll
            for (int g = 0; g < G; ++g) {
                if (c0 + g < c_end) {
                    const char *stage = lds + g * STAGE_BYTES;
#pragma unroll
                    for (int s = 0; s < 2; ++s) {
                        uint4 af[FM], bfr[FN];
#pragma unroll
                        for (int i = 0; i < FM; ++i)
                            af[i] = ld16(stage + (a_row + i * 16) * STRIDE + s * 64 + koff);
#pragma unroll
                        for (int j = 0; j < FN; ++j)
                            bfr[j] = ld16(stage + (b_row + j * 16) * STRIDE + s * 64 + koff);
#pragma unroll
                        for (int i = 0; i < FM; ++i)
#pragma unroll
                            for (int j = 0; j < FN; ++j) acc[i][j] = mma16<DT>(af[i], bfr[j], acc[i][j]);
                    }
                }
            }
        }
    }

    // Reduce the per-piece sums of squares to one value per staged row and
    // store it in rowss[0..ROWS).  The 8 pieces of a row sit in 8 consecutive
    // lanes and are combined by a fixed butterfly, so every row (whatever its
    // position in the tile) is summed in the same order.
    __device__ __forceinline__ static void reduce_rows(const float (&ss)[PPT], float *rowss) {
#pragma unroll
        for (int p = 0; p < PPT; ++p) {
            float v = ss[p];
            v += __shfl_xor(v, 1, 64);
            v += __shfl_xor(v, 2, 64);
            v += __shfl_xor(v, 4, 64);
            if ((threadIdx.x & 7) == 0) rowss[row_of_piece(p)] = v;
        }
    }
};

}  // namespace pv
