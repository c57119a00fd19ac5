// "Row x row" tile product on the matrix cores with operands streamed straight
// into LDS (gfx950 global_load_lds_dwordx4).
//
// C[m][n] = dot(A_row(m), B_row(n)) over a range of 128-byte k chunks, rows
// addressed through a per-row pointer (gathered row lists cost nothing
// extra).  A direct-to-LDS load writes the 16 bytes of lane i to LDS byte
// 16 * i of the instruction's 1 KB block without passing through registers;
// on this chip one CU then sustains several times the bytes per second that
// register loads reach, and the loads of the next NSTAGE - 1 chunks stay in
// flight while the current one is multiplied.
//
// LDS layout of one stage: row r's 128-byte chunk occupies bytes
// [128 r, 128 r + 128), its eight 16-byte pieces stored at slot
// piece ^ (r & 7).  Because the destination of each lane is fixed, the
// swizzle is applied on the global side: the lane that fills slot s of row r
// loads piece s ^ (r & 7).  The fragment reads (16 rows at one piece) then
// spread over the LDS banks.
//
// The stages form one ring; chunk i of the range goes to stage i % NSTAGE.
//
// Ordering.  Before a stage is read, every wave that loaded part of it waits
// for its own loads of that stage (vmcnt; in run_pc only the producer waves
// load), then all waves meet at a bare barrier: a __syncthreads fence would
// also wait for the younger loads still in flight.  The fragment
// reads are issued as inline assembly: the compiler cannot tell that they do
// not touch the stages still being filled and would otherwise drain every
// load in flight before each read.  Their completion is awaited explicitly
// (lds_wait) and every fragment is tied to that wait before the MFMAs use it.
#pragma once

#include "pv_device.h"

namespace pv {

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding:
// vmcnt in bits 3:0 and 15:14; expcnt and lgkmcnt left at their maximum).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Workgroup barrier without a memory fence (see the ordering note above).
__device__ __forceinline__ void bare_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

typedef __attribute__((address_space(3))) void lds_void_t;

// One direct-to-LDS load: 16 bytes from g per lane into LDS at
// lds + 16 * lane.  A __device__ function: target builtins written inside a
// lambda of a kernel template keep the host compile from emitting the
// kernel's launch stub.
__device__ __forceinline__ void lds_dma16(const void *g, char *lds) {
    __builtin_amdgcn_global_load_lds(g, (lds_void_t *)lds, 16, 0, 0);
}
typedef unsigned lds_u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint4 lds_read16(const char *p) {
    lds_u32x4_t r;
    const unsigned addr = (unsigned)(uintptr_t)p;
    asm volatile("ds_read_b128 %0, %1" : "=v"(r) : "v"(addr) : "memory");
    return uint4{r.x, r.y, r.z, r.w};
}
__device__ __forceinline__ void lds_wait() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
// Wait until at most N LDS reads of this wave are outstanding (they complete
// in issue order; N <= 15).
template <int N>
__device__ __forceinline__ void lds_wait_n() {
    static_assert(N >= 0 && N <= 15, "lgkmcnt is a 4-bit count");
    asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N) : "memory");
}
// Ties a fragment to the preceding lds_wait(): volatile asm statements keep
// their order, so no use of the value can be scheduled before the wait.
__device__ __forceinline__ void lds_after_wait(uint4 &v) {
    lds_u32x4_t r = {v.x, v.y, v.z, v.w};
    asm volatile("" : "+v"(r));
    v = uint4{r.x, r.y, r.z, r.w};
}

template <int DT, int BM, int BN, int WM, int WN, int NSTAGE>
struct TileGemmLds {
    static constexpr int NT = 64 * WM * WN;
    static constexpr int NW = WM * WN;
    static constexpr int ROWS = BM + BN;
    static constexpr int CHUNK = 128;
    static constexpr int STAGE_BYTES = ROWS * CHUNK;
    static constexpr int LDS_BYTES = NSTAGE * STAGE_BYTES;
    static constexpr int IPW = ROWS * 8 / 64 / NW;  // load instructions per wave per stage
    static constexpr int SUB_M = BM / WM, SUB_N = BN / WN;
    static constexpr int FM = SUB_M / 16, FN = SUB_N / 16;
    static_assert(ROWS * 8 % (64 * NW) == 0, "stage rows must split evenly over the waves");
    static_assert(SUB_M % 16 == 0 && SUB_N % 16 == 0, "wave tile must be 16-aligned");
    static_assert(NSTAGE >= 2, "at least double buffering");
    static_assert(IPW * (NSTAGE - 1) < 64, "loads in flight exceed the wait counter");

    // Multiply chunks [c_begin, c_end) into acc.  row_ptr(r) is the global byte
    // address of staged row r (r < BM: A rows, r >= BM: B rows); every row
    // must be valid (clamp past-the-end rows in the caller).  With WANT_SS,
    // ssa[fm] / ssb[fn] receive this lane's partial sums of squares of the A
    // rows (waves with wn == 0) and B rows (waves with wm == 0) it reads; see
    // row_sumsq.  Must be called by every thread of the workgroup.
    template <bool WANT_SS, typename RowPtr>
    __device__ __forceinline__ static void run(RowPtr row_ptr, int c_begin, int c_end,
                                               f32x4_t (&acc)[FM][FN], float (&ssa)[FM],
                                               float (&ssb)[FN]) {
        __shared__ __attribute__((aligned(16))) char ring[LDS_BYTES];
        run_in<WANT_SS>(ring, row_ptr, c_begin, c_end, acc, ssa, ssb);
    }

    // The same on a ring the caller provides (LDS_BYTES of LDS, 16-byte
    // aligned), for kernels whose other workgroups use the same LDS for
    // something else.
    template <bool WANT_SS, typename RowPtr>
    __device__ __forceinline__ static void run_in(char *ring, RowPtr row_ptr, int c_begin,
                                                  int c_end, f32x4_t (&acc)[FM][FN],
                                                  float (&ssa)[FM], float (&ssb)[FN]) {
        const int lane = threadIdx.x & 63;
        const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
        const int wm = wave / WN, wn = wave % WN;
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            ssa[i] = 0.f;
#pragma unroll
            for (int j = 0; j < FN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int j = 0; j < FN; ++j) ssb[j] = 0.f;
        const int nc = c_end - c_begin;
        if (nc <= 0) return;

        // this lane's source row and piece for each of its IPW instructions
        const char *src[IPW];
#pragma unroll
        for (int q = 0; q < IPW; ++q) {
            const int pos = (wave * IPW + q) * 64 + lane;  // 16-byte slot in the stage
            const int r = pos >> 3, slot = pos & 7;
            src[q] = row_ptr(r) + (size_t)c_begin * CHUNK + ((slot ^ (r & 7)) << 4);
        }
        // chunk i (relative to c_begin) goes to stage i % NSTAGE
        auto issue = [&](int i) {
            char *dst = ring + (i % NSTAGE) * STAGE_BYTES + wave * IPW * 1024;
#pragma unroll
            for (int q = 0; q < IPW; ++q)
                lds_dma16(src[q] + (size_t)i * CHUNK, dst + q * 1024);
        };
#pragma unroll
        for (int p = 0; p < NSTAGE - 1; ++p)
            if (p < nc) issue(p);

        const int a_row = wm * SUB_M + (lane & 15);
        const int b_row = BM + wn * SUB_N + (lane & 15);
        const int kq = lane >> 4;  // 16-byte quarter of the 64-byte window
        for (int i = 0; i < nc; ++i) {
            // this wave's loads of chunk i are done once at most the loads of
            // the younger chunks already issued are outstanding
            if (i + NSTAGE - 1 <= nc) wait_vmcnt<IPW * (NSTAGE - 2)>();
            else wait_vmcnt<0>();
            bare_barrier();  // all of chunk i is in LDS; chunk i - 1 has been read
            if (i + NSTAGE - 1 < nc) issue(i + NSTAGE - 1);
            const char *sp = ring + (i % NSTAGE) * STAGE_BYTES;
            // both 64-byte windows of the chunk are read up front: the
            // second window's reads are in flight while the first window's
            // MFMAs run
            uint4 af[2][FM], bfr[2][FN];
#pragma unroll
            for (int s = 0; s < 2; ++s) {
                const int piece = s * 4 + kq;
#pragma unroll
                for (int f = 0; f < FM; ++f) {
                    const int r = a_row + f * 16;
                    af[s][f] = lds_read16(sp + r * CHUNK + ((piece ^ (r & 7)) << 4));
                }
#pragma unroll
                for (int f = 0; f < FN; ++f) {
                    const int r = b_row + f * 16;
                    bfr[s][f] = lds_read16(sp + r * CHUNK + ((piece ^ (r & 7)) << 4));
                }
            }
#pragma unroll
            for (int s = 0; s < 2; ++s) {
                if (s == 0) lds_wait_n<(FM + FN <= 15 ? FM + FN : 0)>();
                else lds_wait();
#pragma unroll
                for (int f = 0; f < FM; ++f) lds_after_wait(af[s][f]);
#pragma unroll
                for (int f = 0; f < FN; ++f) lds_after_wait(bfr[s][f]);
                if (WANT_SS) {
                    if (wn == 0) {
#pragma unroll
                        for (int f = 0; f < FM; ++f) ssa[f] += sumsq16<DT>(af[s][f]);
                    }
                    if (wm == 0) {
#pragma unroll
                        for (int f = 0; f < FN; ++f) ssb[f] += sumsq16<DT>(bfr[s][f]);
                    }
                }
#pragma unroll
                for (int f = 0; f < FM; ++f)
#pragma unroll
                    for (int g = 0; g < FN; ++g)
                        acc[f][g] = mma16<DT>(af[s][f], bfr[s][g], acc[f][g]);
            }
        }
        bare_barrier();  // the stages may be reused by a later call
    }

    // The same product with NP producer waves after the NW matrix waves
    // (blockDim = 64 (NW + NP)) and a three-stage ring.  The producers issue
    // every direct-to-LDS load, so a matrix wave never waits for the CU's load
    // path to take one (about 16 clocks per 1 KB instruction, shared by the
    // CU); the matrix waves read fragments one 64-byte window ahead of their
    // MFMAs: window 1 of chunk i while window 0's MFMAs issue, window 0 of
    // chunk i + 1 while window 1's issue.
    //
    // Barrier j (j = 0 .. nc) closes the reads of chunk j - 1 and opens chunk
    // j: before it the producers wait for their loads of chunk j, and after it
    // they load chunk j + 2 into chunk j - 1's stage (chunks 0 .. 2 are loaded
    // up front).  A matrix wave meets barrier j + 1 after its last read of
    // chunk j and before its first read of chunk j + 1.  Both sides pass
    // nc + 2 barriers.  acc is meaningful in the matrix waves only.
    //
    // m_valid / n_valid: the A / B rows that count (the rest are padding the
    // caller clamps to valid rows); a matrix wave whose A rows or B rows all
    // lie past them keeps only the barriers and returns zero products.
    template <int NP, typename RowPtr>
    __device__ __forceinline__ static void run_pc(char *ring, RowPtr row_ptr, int c_begin, int c_end,
                                                  f32x4_t (&acc)[FM][FN], int m_valid = BM,
                                                  int n_valid = BN) {
        static_assert(NSTAGE == 3, "two chunks in flight and one being read");
        constexpr int IPP = ROWS * 8 / 64 / NP;  // load instructions per producer wave per stage
        static_assert(NP >= 1 && ROWS * 8 % (64 * NP) == 0, "stage rows must split over the producers");
        static_assert(IPP * 2 < 64, "loads in flight exceed the wait counter");
        const int lane = threadIdx.x & 63;
        const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        const int nc = c_end - c_begin;
        if (nc <= 0) return;
        if (wave >= NW) {
            const int pw = wave - NW;
            const char *src[IPP];
#pragma unroll
            for (int q = 0; q < IPP; ++q) {
                const int pos = (pw * IPP + q) * 64 + lane;
                const int r = pos >> 3, slot = pos & 7;
                src[q] = row_ptr(r) + (size_t)c_begin * CHUNK + ((slot ^ (r & 7)) << 4);
            }
            auto issue = [&](int i) {
                char *dst = ring + (i % NSTAGE) * STAGE_BYTES + pw * IPP * 1024;
#pragma unroll
                for (int q = 0; q < IPP; ++q)
                    lds_dma16(src[q] + (size_t)i * CHUNK, dst + q * 1024);
            };
            issue(0);
            if (nc > 1) issue(1);
            if (nc > 2) issue(2);
            // chunk 0 landed (chunks 1 and 2 may still fly)
            if (nc > 2) wait_vmcnt<2 * IPP>();
            else if (nc == 2) wait_vmcnt<IPP>();
            else wait_vmcnt<0>();
            bare_barrier();  // barrier 0
            for (int i = 0; i < nc; ++i) {
                // chunk i + 1 landed (chunk i + 2 may still fly)
                if (i + 2 < nc) wait_vmcnt<IPP>();
                else wait_vmcnt<0>();
                bare_barrier();  // barrier i + 1: chunk i's stage is free
                if (i + 3 < nc) issue(i + 3);
            }
        } else {
            const int wm = wave / WN, wn = wave % WN;
            if (wm * SUB_M >= m_valid || wn * SUB_N >= n_valid) {
                bare_barrier();  // barrier 0
                for (int i = 0; i < nc; ++i) bare_barrier();
                bare_barrier();
                return;
            }
            const int a_row = wm * SUB_M + (lane & 15);
            const int b_row = BM + wn * SUB_N + (lane & 15);
            const int kq = lane >> 4;
            auto read_w = [&](int i, int s, uint4(&a)[FM], uint4(&b)[FN]) {
                const char *sp = ring + (i % NSTAGE) * STAGE_BYTES;
                const int piece = s * 4 + kq;
#pragma unroll
                for (int f = 0; f < FM; ++f) {
                    const int r = a_row + f * 16;
                    a[f] = lds_read16(sp + r * CHUNK + ((piece ^ (r & 7)) << 4));
                }
#pragma unroll
                for (int f = 0; f < FN; ++f) {
                    const int r = b_row + f * 16;
                    b[f] = lds_read16(sp + r * CHUNK + ((piece ^ (r & 7)) << 4));
                }
            };
            auto mma_w = [&](uint4(&a)[FM], uint4(&b)[FN]) {
#pragma unroll
                for (int f = 0; f < FM; ++f)
#pragma unroll
                    for (int g = 0; g < FN; ++g) acc[f][g] = mma16<DT>(a[f], b[g], acc[f][g]);
            };
            uint4 a0[FM], b0[FN], a1[FM], b1[FN];
            bare_barrier();  // barrier 0
            read_w(0, 0, a0, b0);
            for (int i = 0; i < nc; ++i) {
                read_w(i, 1, a1, b1);
                lds_wait_n<(FM + FN <= 15 ? FM + FN : 0)>();  // window 0 of chunk i
#pragma unroll
                for (int f = 0; f < FM; ++f) lds_after_wait(a0[f]);
#pragma unroll
                for (int f = 0; f < FN; ++f) lds_after_wait(b0[f]);
                mma_w(a0, b0);
                lds_wait();  // window 1 of chunk i: every read of chunk i done
#pragma unroll
                for (int f = 0; f < FM; ++f) lds_after_wait(a1[f]);
#pragma unroll
                for (int f = 0; f < FN; ++f) lds_after_wait(b1[f]);
                bare_barrier();  // barrier i + 1
                if (i + 1 < nc) read_w(i + 1, 0, a0, b0);
                mma_w(a1, b1);
            }
        }
        bare_barrier();  // the stages may be reused by a later call
    }

    // Sum of squares of row (lane & 15) of a fragment block: combines the four
    // 16-byte quarters held by lanes l, l+16, l+32, l+48 in a fixed order.
    __device__ __forceinline__ static float row_sumsq(float partial) {
        partial += __shfl_xor(partial, 16, 64);
        partial += __shfl_xor(partial, 32, 64);
        return partial;
    }
};

}  // namespace pv
