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

// 2^x on the transcendental unit, without the library's range reduction for
// results below the smallest normal float (they flush to 0, which no softmax
// sum here can notice next to its maximum term, 1).
__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

// Lane exchange within a row of 16 lanes through DPP (no LDS round trip).
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}
// Maximum and sum over the 16 lanes of a row (lanes 16 r .. 16 r + 15), left
// in every lane of the row.  Partners: lane ^ 1 and lane ^ 2 (quad
// permutations), then the mirror within 8 and within 16 lanes, which after
// the first steps hold the same values as lane ^ 4 and lane ^ 8: the sums
// pair up as an xor butterfly over 1, 2, 4, 8 does, and give its bits.
__device__ __forceinline__ float row16_max(float x) {
    x = fmaxf(x, dpp_f32<0xB1>(x));   // quad_perm [1, 0, 3, 2]
    x = fmaxf(x, dpp_f32<0x4E>(x));   // quad_perm [2, 3, 0, 1]
    x = fmaxf(x, dpp_f32<0x141>(x));  // row_half_mirror
    x = fmaxf(x, dpp_f32<0x140>(x));  // row_mirror
    return x;
}
__device__ __forceinline__ float row16_sum(float x) {
    x += dpp_f32<0xB1>(x);
    x += dpp_f32<0x4E>(x);
    x += dpp_f32<0x141>(x);
    x += dpp_f32<0x140>(x);
    return x;
}

// Order-preserving 32-bit key of a float: larger float <=> larger key.
// -0 is mapped to the key of +0 so that the two tie.
__device__ __forceinline__ uint32_t order_key(float f) {
    uint32_t u = __float_as_uint(f);
    if (u == 0x80000000u) u = 0u;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Sum over the 64 lanes of a wave (every lane active), in every lane: the
// rows by row16_sum, then (row 0 + row 1) + (row 2 + row 3), the order of an
// xor butterfly over 16 and 32, so the bits are that butterfly's.
__device__ __forceinline__ float wave_sum64(float x) {
    x = row16_sum(x);
    const float a = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 0));
    const float b = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 16));
    const float c = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 32));
    const float d = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 48));
    return (a + b) + (c + d);
}

// Maximum over the 64 lanes of a wave (every lane active), in every lane.
__device__ __forceinline__ float wave_max_f32(float x) {
    x = row16_max(x);
    const float a = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 0));
    const float b = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 16));
    const float c = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 32));
    const float d = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 48));
    return fmaxf(fmaxf(a, b), fmaxf(c, d));
}

// Lane exchange within a row of 16 lanes through DPP; a lane whose source
// falls outside the row reads 0.
template <int CTRL>
__device__ __forceinline__ int dpp_i32(int x) {
    return __builtin_amdgcn_update_dpp(0, x, CTRL, 0xF, 0xF, false);
}

// Inclusive prefix sum across the 64 lanes of a wave (every lane active):
// within each row of 16 by DPP row shifts of 1, 2, 4, 8, then the totals of
// the rows below from lanes 15, 31, 47.  Integer sums, so the order of the
// additions does not matter.
__device__ __forceinline__ int wave_incl_scan(int x) {
    const int row = (threadIdx.x & 63) >> 4;
    x += dpp_i32<0x111>(x);  // row_shr:1
    x += dpp_i32<0x112>(x);  // row_shr:2
    x += dpp_i32<0x114>(x);  // row_shr:4
    x += dpp_i32<0x118>(x);  // row_shr:8
    const int t0 = __builtin_amdgcn_readlane(x, 15);
    const int t1 = __builtin_amdgcn_readlane(x, 31);
    const int t2 = __builtin_amdgcn_readlane(x, 47);
    return x + (row >= 1 ? t0 : 0) + (row >= 2 ? t1 : 0) + (row >= 3 ? t2 : 0);
}

// Minimum and maximum over the 64 lanes of a wave, returned to every lane:
// row reductions by DPP (as row16_max), then lanes 0, 16, 32, 48.
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t x) {
    x = min(x, (uint32_t)dpp_i32<0xB1>((int)x));
    x = min(x, (uint32_t)dpp_i32<0x4E>((int)x));
    x = min(x, (uint32_t)dpp_i32<0x141>((int)x));
    x = min(x, (uint32_t)dpp_i32<0x140>((int)x));
    const uint32_t a = __builtin_amdgcn_readlane(x, 0), b = __builtin_amdgcn_readlane(x, 16);
    const uint32_t c = __builtin_amdgcn_readlane(x, 32), d = __builtin_amdgcn_readlane(x, 48);
    return min(min(a, b), min(c, d));
}
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x) {
    x = max(x, (uint32_t)dpp_i32<0xB1>((int)x));
    x = max(x, (uint32_t)dpp_i32<0x4E>((int)x));
    x = max(x, (uint32_t)dpp_i32<0x141>((int)x));
    x = max(x, (uint32_t)dpp_i32<0x140>((int)x));
    const uint32_t a = __builtin_amdgcn_readlane(x, 0), b = __builtin_amdgcn_readlane(x, 16);
    const uint32_t c = __builtin_amdgcn_readlane(x, 32), d = __builtin_amdgcn_readlane(x, 48);
    return max(max(a, b), max(c, d));
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
    int hist[2][256];
    int wsum[16];
    uint32_t wlo[16], whi[16];
    int sel[2][3];  // digit, rank still to find, keys in the digit's bin
};

// Number of keys each thread owns in block_topk: ceil(n / NT).
__host__ __device__ constexpr int topk_per_thread(int n, int NT) { return (n + NT - 1) / NT; }

// Deterministic top-k of n keys by one block of NT threads: keeps the k
// largest keys, lower index first among equal keys, and writes
//   kept[0..k)       the kept indices, ascending,
//   rest[0..n-k)     the other indices, ascending (if rest != nullptr),
//   slot_of[j]       position of j in kept, or -1 (if slot_of != nullptr).
// Thread t owns the E = ceil(n / NT) <= EMAX consecutive indices starting at
// t * E and passes their keys in key[] (entries past n are ignored).  The keys
// are order-preserving images of the scores (order_key), so comparing keys
// compares scores.
//
// Radix select, most significant digit first, but starting just below the
// bits that every key shares (found from the block's min and max key): close
// scores share their sign and exponent bits, and starting there would pile
// every key into one bin.  Each pass histograms the 8-bit digit of the keys
// that still match the prefix found so far and picks the bin that holds the
// rank still sought.  The search stops as soon as that bin is kept whole (its
// count equals the rank sought) or the key is fully resolved; the kept set is
// then every key whose resolved prefix is greater, plus the first `rank`
// keys, in index order, whose prefix is equal.  One packed block scan places
// every index.  k must satisfy 1 <= k <= n.
template <int NT, int EMAX>
__device__ __forceinline__ void block_topk(const uint32_t (&key)[EMAX], int n, int k,
                                           int32_t *kept, int32_t *rest, int32_t *slot_of,
                                           TopkSmem &sm) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    constexpr int NW = NT / 64;
    const int E = topk_per_thread(n, NT);
    const int j0 = tid * E;

    // block min and max key
    uint32_t lo = 0xFFFFFFFFu, hi = 0u;
#pragma unroll
    for (int e = 0; e < EMAX; ++e) {
        if (e < E && j0 + e < n) {
            lo = min(lo, key[e]);
            hi = max(hi, key[e]);
        }
    }
    lo = wave_min_u32(lo);
    hi = wave_max_u32(hi);
    if (lane == 0) {
        sm.wlo[wave] = lo;
        sm.whi[wave] = hi;
    }
    for (int e = tid; e < 256; e += NT) sm.hist[0][e] = 0;
    __syncthreads();
    lo = sm.wlo[0];
    hi = sm.whi[0];
#pragma unroll
    for (int w = 1; w < NW; ++w) {
        lo = min(lo, sm.wlo[w]);
        hi = max(hi, sm.whi[w]);
    }

    // prefix/mask: the bits resolved so far; kr: rank still sought among the
    // keys that match the prefix
    uint32_t prefix = hi, mask = 0xFFFFFFFFu;
    int kr = k;
    const uint32_t diff = lo ^ hi;
    if (diff != 0u) {
        const int top = 31 - __clz(diff);  // highest bit where keys differ
        mask = (top == 31) ? 0u : ~((2u << top) - 1u);
        prefix = hi & mask;
        int shift = top - 7 > 0 ? top - 7 : 0;
        int cur = 0;
        while (true) {
#pragma unroll
            for (int e = 0; e < EMAX; ++e) {
                if (e < E && j0 + e < n && (key[e] & mask) == prefix)
                    atomicAdd(&sm.hist[cur][(key[e] >> shift) & 255u], 1);
            }
            __syncthreads();
            for (int e = tid; e < 256; e += NT) sm.hist[cur ^ 1][e] = 0;
            if (wave == 0) {
                // lane owns bins 4*lane .. 4*lane+3; find the bin holding rank kr
                // counted from the top
                const int h0 = sm.hist[cur][4 * lane], h1 = sm.hist[cur][4 * lane + 1];
                const int h2 = sm.hist[cur][4 * lane + 2], h3 = sm.hist[cur][4 * lane + 3];
                const int mine = h0 + h1 + h2 + h3;
                const int inc = wave_incl_scan(mine);
                const int suffix_incl = __builtin_amdgcn_readlane(inc, 63) - inc + mine;  // lanes >= this one
                const int above = suffix_incl - mine;                 // bins > 4*lane+3
                const int ge3 = above + h3, ge2 = ge3 + h2, ge1 = ge2 + h1, ge0 = ge1 + h0;
                int dsel = -1, gt = 0, cnt = 0;
                if (above < kr && kr <= ge3) { dsel = 3; gt = above; cnt = h3; }
                else if (ge3 < kr && kr <= ge2) { dsel = 2; gt = ge3; cnt = h2; }
                else if (ge2 < kr && kr <= ge1) { dsel = 1; gt = ge2; cnt = h1; }
                else if (ge1 < kr && kr <= ge0) { dsel = 0; gt = ge1; cnt = h0; }
                if (dsel >= 0) {
                    sm.sel[cur][0] = 4 * lane + dsel;
                    sm.sel[cur][1] = kr - gt;
                    sm.sel[cur][2] = cnt;
                }
            }
            __syncthreads();
            const uint32_t digit = (uint32_t)sm.sel[cur][0];
            const int cnt = sm.sel[cur][2];
            kr = sm.sel[cur][1];
            prefix = (prefix & ~(0xFFu << shift)) | (digit << shift);
            mask |= 0xFFu << shift;
            if (cnt == kr || shift == 0) break;
            shift = shift >= 8 ? shift - 8 : 0;
            cur ^= 1;
        }
    }

    // keep: prefix greater, or prefix equal and among the first kr such keys
    int n_gt = 0, n_eq = 0;
#pragma unroll
    for (int e = 0; e < EMAX; ++e) {
        if (e < E && j0 + e < n) {
            const uint32_t m = key[e] & mask;
            n_gt += m > prefix;
            n_eq += m == prefix;
        }
    }
    int total;
    const int before = block_excl_scan<NT>(n_gt | (n_eq << 16), sm.wsum, &total);
    int gt_before = before & 0xFFFF, eq_before = before >> 16;
#pragma unroll
    for (int e = 0; e < EMAX; ++e) {
        const int j = j0 + e;
        if (e < E && j < n) {
            const uint32_t m = key[e] & mask;
            const int pos = gt_before + min(eq_before, kr);
            const bool keep = m > prefix || (m == prefix && eq_before < kr);
            if (keep) kept[pos] = j;
            else if (rest) rest[j - pos] = j;
            if (slot_of) slot_of[j] = keep ? pos : -1;
            gt_before += m > prefix;
            eq_before += m == prefix;
        }
    }
}

}  // namespace pv
