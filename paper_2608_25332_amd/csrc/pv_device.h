// Device helpers shared by the ProViP kernels (gfx950 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pv_launch.h"

namespace pv {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_to_f32(uint32_t h16) { return __uint_as_float(h16 << 16); }

// float -> bfloat16 bits, round to nearest even (inputs are finite).
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return u >> 16;
}

// Sum of squares of the elements held in one 16-byte piece, in a fixed order.
template <int DT>
__device__ __forceinline__ float sumsq16(uint4 v);
template <>
__device__ __forceinline__ float sumsq16<kBF16>(uint4 v) {
    float s = 0.f;
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        float lo = __uint_as_float(w[t] << 16);
        float hi = __uint_as_float(w[t] & 0xFFFF0000u);
        s = fmaf(lo, lo, s);
        s = fmaf(hi, hi, s);
    }
    return s;
}
template <>
__device__ __forceinline__ float sumsq16<kF32>(uint4 v) {
    float s = 0.f;
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        float x = __uint_as_float(w[t]);
        s = fmaf(x, x, s);
    }
    return s;
}

// 16x16 fp32 tile += A-fragment x B-fragment, 16 bytes per lane each.
// Lane l supplies row (l % 16) of the A block and row (l % 16) of the B block
// (B rows are the output columns), at byte offset 16 * (l / 16) of a 64-byte
// k window.  A and B use the same element placement, so the window's dot
// product is complete whatever order the matrix core visits the elements in.
//   bf16: the window is 32 elements, one 16x16x32 MFMA;
//   f32 : the window is 16 elements, four 16x16x4 MFMAs.
// The result lives in acc[i] = C[4 * (l / 16) + i][l % 16].
template <int DT>
__device__ __forceinline__ f32x4_t mma16(uint4 a, uint4 b, f32x4_t acc);
template <>
__device__ __forceinline__ f32x4_t mma16<kBF16>(uint4 a, uint4 b, f32x4_t acc) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                   __builtin_bit_cast(bf16x8_t, b), acc, 0, 0, 0);
}
template <>
__device__ __forceinline__ f32x4_t mma16<kF32>(uint4 a, uint4 b, f32x4_t acc) {
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
    return acc;
}

__device__ __forceinline__ uint4 ld16(const void *p) { return *reinterpret_cast<const uint4 *>(p); }
__device__ __forceinline__ void st16(void *p, uint4 v) { *reinterpret_cast<uint4 *>(p) = v; }

// Order-preserving 32-bit key of a float: larger float <=> larger key.
// -0 is mapped to the key of +0 so that the two tie.
__device__ __forceinline__ uint32_t order_key(float f) {
    uint32_t u = __float_as_uint(f);
    if (u == 0x80000000u) u = 0u;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Inclusive prefix sum across the 64 lanes of a wave.
__device__ __forceinline__ int wave_incl_scan(int x) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        int y = __shfl_up(x, off, 64);
        if (lane >= off) x += y;
    }
    return x;
}

// Exclusive prefix sum over a block of NT threads; *total gets the block sum.
// `wsum` is LDS scratch of NT/64 ints.  Contains barriers: every thread of the
// block must call it.
template <int NT>
__device__ __forceinline__ int block_excl_scan(int x, int *wsum, int *total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int inc = wave_incl_scan(x);
    if (lane == 63) wsum[wave] = inc;
    __syncthreads();
    int before = 0, all = 0;
#pragma unroll
    for (int w = 0; w < NT / 64; ++w) {
        int s = wsum[w];
        if (w < wave) before += s;
        all += s;
    }
    __syncthreads();
    *total = all;
    return before + inc - x;
}

// Workgroups are dispatched to the 8 XCDs of the chip round-robin by linear
// id.  Map linear id L to a tile index so that every XCD receives one
// contiguous run of tiles: tiles that share operand rows then share that
// XCD's L2 instead of each fetching the rows from memory.
__device__ __forceinline__ int xcd_tile(int L, int total) {
    const int x = L & 7, q = L >> 3;
    const int base = total >> 3, rem = total & 7;
    return x * base + (x < rem ? x : rem) + q;
}

struct TopkSmem {
    int hist[256];
    int wsum[16];
    uint32_t digit;
    int remaining;
};

// Deterministic top-k of n float scores by one block of NT threads: keeps the
// k highest scores, lower index first among equal scores, and writes
//   kept[0..k)       the kept indices, ascending,
//   rest[0..n-k)     the other indices, ascending (if rest != nullptr),
//   slot_of[j]       position of j in kept, or -1 (if slot_of != nullptr).
// Radix select over the order-preserving keys (four 8-bit digits, most
// significant first) finds the k-th largest key T; the keys above T and the
// first (k - #above) keys equal to T in index order are kept.  When `lds_keys`
// is given (room for n keys) the keys are staged there once; otherwise every
// pass re-reads the scores from global memory (cache resident).
template <int NT>
__device__ void block_topk(const float *score, int n, int k, int32_t *kept, int32_t *rest,
                           int32_t *slot_of, TopkSmem &sm, uint32_t *lds_keys) {
    const int tid = threadIdx.x;
    if (lds_keys) {
        for (int j = tid; j < n; j += NT) lds_keys[j] = order_key(score[j]);
        __syncthreads();
    }
    auto key_of = [&](int j) -> uint32_t { return lds_keys ? lds_keys[j] : order_key(score[j]); };
    uint32_t prefix = 0u, mask = 0u;
    int kr = k;  // rank still to be found inside the current prefix group
    for (int shift = 24; shift >= 0; shift -= 8) {
        for (int e = tid; e < 256; e += NT) sm.hist[e] = 0;
        __syncthreads();
        for (int j = tid; j < n; j += NT) {
            const uint32_t key = key_of(j);
            if ((key & mask) == prefix) atomicAdd(&sm.hist[(key >> shift) & 255u], 1);
        }
        __syncthreads();
        if (tid < 64) {
            // lane owns bins 4*lane .. 4*lane+3
            const int h0 = sm.hist[4 * tid], h1 = sm.hist[4 * tid + 1];
            const int h2 = sm.hist[4 * tid + 2], h3 = sm.hist[4 * tid + 3];
            const int mine = h0 + h1 + h2 + h3;
            // suffix sum over lanes: reverse the lane order, inclusive scan
            const int rev = __shfl(mine, 63 - tid, 64);
            const int inc = wave_incl_scan(rev);
            const int suffix_incl = __shfl(inc, 63 - tid, 64);  // sum over lanes >= tid
            const int above = suffix_incl - mine;                // keys in bins > 4*tid+3
            const int ge3 = above + h3, ge2 = ge3 + h2, ge1 = ge2 + h1, ge0 = ge1 + h0;
            int dsel = -1, gt = 0;
            if (above < kr && kr <= ge3) { dsel = 3; gt = above; }
            else if (ge3 < kr && kr <= ge2) { dsel = 2; gt = ge3; }
            else if (ge2 < kr && kr <= ge1) { dsel = 1; gt = ge2; }
            else if (ge1 < kr && kr <= ge0) { dsel = 0; gt = ge1; }
            if (dsel >= 0) {
                sm.digit = (uint32_t)(4 * tid + dsel);
                sm.remaining = kr - gt;
            }
        }
        __syncthreads();
        prefix |= sm.digit << shift;
        mask |= 0xFFu << shift;
        kr = sm.remaining;
        __syncthreads();
    }
    const uint32_t T = prefix;  // key of the k-th largest score
    int carry_eq = 0, carry_keep = 0;
    for (int base = 0; base < n; base += NT) {
        const int j = base + tid;
        const uint32_t key = (j < n) ? key_of(j) : 0u;
        const int is_gt = (j < n) && key > T;
        const int is_eq = (j < n) && key == T;
        int tot_eq, tot_keep;
        const int eq_before = block_excl_scan<NT>(is_eq, sm.wsum, &tot_eq) + carry_eq;
        const int keep = is_gt || (is_eq && eq_before < kr);
        const int pos = block_excl_scan<NT>(keep, sm.wsum, &tot_keep) + carry_keep;
        if (j < n) {
            if (keep) {
                kept[pos] = j;
            } else if (rest) {
                rest[j - pos] = j;
            }
            if (slot_of) slot_of[j] = keep ? pos : -1;
        }
        carry_eq += tot_eq;
        carry_keep += tot_keep;
    }
}

}  // namespace pv
