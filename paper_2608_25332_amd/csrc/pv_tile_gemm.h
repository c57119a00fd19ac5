// LDS-staged "row x row" tile product on the matrix cores (gfx950).
//
// Both operands are sets of rows of length d (the embedding width), as stored
// in HBM: C[m][n] = dot(A_row(m), B_row(n)).  That is a GEMM whose two inputs
// are both k-contiguous, which is exactly the layout the MFMA fragments want:
// every lane reads 16 contiguous bytes of one row.
//
// One workgroup owns a BM x BN output tile and walks the k dimension in
// 128-byte chunks (64 bf16 or 32 f32 elements per row).  Each chunk of the
// BM + BN rows is fetched with fully coalesced 16-byte loads (8 lanes cover
// one row's 128 bytes), written to LDS with a 16-byte pad per row, and the
// next chunk's loads are in flight while the current chunk is multiplied.
// The WM x WN waves each own a (BM/WM) x (BN/WN) sub-tile of 16x16 blocks.
//
// Rows are addressed through a per-row pointer, so gathered operands (the
// pruned and kept token lists) cost nothing extra.  Rows past the valid count
// are clamped to a valid row and masked by the caller's epilogue.
#pragma once

#include "pv_device.h"

namespace pv {

template <int DT, int BM, int BN, int WM, int WN>
struct TileGemm {
    static constexpr int NT = 64 * WM * WN;
    static constexpr int ROWS = BM + BN;
    static constexpr int CHUNK = 128;   // bytes of one row per k step
    static constexpr int STRIDE = 144;  // LDS bytes per staged row (16-byte pad)
    static constexpr int PIECES = ROWS * (CHUNK / 16);
    static constexpr int PPT = PIECES / NT;  // 16-byte pieces per thread per chunk
    static constexpr int SUB_M = BM / WM, SUB_N = BN / WN;
    static constexpr int FM = SUB_M / 16, FN = SUB_N / 16;
    static constexpr int LDS_BYTES = ROWS * STRIDE;
    static_assert(PIECES % NT == 0, "tile rows must fill the loaders evenly");
    static_assert(SUB_M % 16 == 0 && SUB_N % 16 == 0, "wave tile must be 16-aligned");

    // Run the k loop.  row_ptr(r) gives the global byte address of staged row
    // r (r < BM: A rows, r >= BM: B rows).  When WANT_SS is set, ss[p] returns
    // this thread's partial sum of squares for its p-th piece slot (pieces of
    // one row are spread over 8 consecutive lanes; see row_of_piece).
    template <bool WANT_SS, typename RowPtr>
    __device__ __forceinline__ static void run(RowPtr row_ptr, int nchunks, char *lds,
                                               f32x4_t (&acc)[FM][FN], float (&ss)[PPT]) {
        const int tid = threadIdx.x;
        const int lane = tid & 63, wave = tid >> 6;
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

        uint4 buf[PPT];
#pragma unroll
        for (int p = 0; p < PPT; ++p) buf[p] = ld16(src[p]);

        const int a_row = wm * SUB_M + (lane & 15);
        const int b_row = BM + wn * SUB_N + (lane & 15);
        const int koff = (lane >> 4) * 16;

        for (int kc = 0; kc < nchunks; ++kc) {
            __syncthreads();
#pragma unroll
            for (int p = 0; p < PPT; ++p) {
                st16(lds + dst[p], buf[p]);
                if (WANT_SS) ss[p] += sumsq16<DT>(buf[p]);
            }
            __syncthreads();
            if (kc + 1 < nchunks) {
#pragma unroll
                for (int p = 0; p < PPT; ++p) buf[p] = ld16(src[p] + (size_t)(kc + 1) * CHUNK);
            }
#pragma unroll
            for (int s = 0; s < 2; ++s) {
                uint4 af[FM], bfr[FN];
#pragma unroll
                for (int i = 0; i < FM; ++i)
                    af[i] = ld16(lds + (a_row + i * 16) * STRIDE + s * 64 + koff);
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    bfr[j] = ld16(lds + (b_row + j * 16) * STRIDE + s * 64 + koff);
#pragma unroll
                for (int i = 0; i < FM; ++i)
#pragma unroll
                    for (int j = 0; j < FN; ++j) acc[i][j] = mma16<DT>(af[i], bfr[j], acc[i][j]);
            }
        }
    }

    // Staged row owning piece slot p of this thread.
    __device__ __forceinline__ static int row_of_piece(int p) { return (threadIdx.x + p * NT) >> 3; }

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
