// Steps of the pipeline that can ride along in another stage's launch.
//
// At small batches every kernel of the pipeline is a few microseconds, most
// of it the launch itself, and the two chains that follow the top-N_1
// selection (nearest kept token -> merge, and head-aware score -> top-N_2)
// do not depend on each other.  Their steps then share launches as extra
// workgroups of one grid: the score (reading the kept tokens' keys through
// the kept list) with the Gram tiles; the top-N_2 with the Gram's argmax and
// the compaction of K/V to the N_1 kept; the final compaction with the
// merge.  The bodies below are those steps' workgroup bodies, shared by
// their own kernels and by the kernels that carry them; a job with
// nblocks == 0 adds nothing.
#pragma once

#include "pv_device.h"
#include "pv_launch.h"
#include "pv_tile_lds.h"

namespace pv {

// ---- order-preserving row compaction (Sec. 4.1) ---------------------------
constexpr int kGatherNT = 256;

struct GatherJob {
    GatherArgs ga;
    const int32_t *idx;  // [B][k] kept indices
    int k;
    int nblocks;  // workgroups of the gather (ga.bstart[ga.n]); 0: none
};

// Workgroup blk of the gather: a contiguous span of 16-byte pieces of one
// plane (sample x head group) of one tensor; rows whose index is out of
// range are written as zeros.
__device__ __forceinline__ void gather_block(const GatherArgs &ga, const int32_t *__restrict__ idx,
                                             int k, int blk) {
    int t = 0;
#pragma unroll
    for (int u = 1; u < kMaxGather; ++u)
        if (u < ga.n && blk >= ga.bstart[u]) t = u;
    const GatherDesc &g = ga.d[t];
    const int local = blk - ga.bstart[t];
    const int plane = local / g.bpp, sub = local - plane * g.bpp;
    const int b = plane / g.groups, gr = plane - b * g.groups;
    const int ppp = k * g.cpr;  // pieces in this plane
    const char *s0 = g.src + b * g.sb + gr * g.sg;
    char *d0 = g.dst + b * g.db + gr * g.dg;
    const int32_t *ib = idx + (size_t)b * k;
    uint4 v[kGatherIT];
    int rr[kGatherIT], cc[kGatherIT], jj[kGatherIT];
    // the row indices first, then every piece's load: a piece load issued
    // between two index loads would be waited for with the next index
#pragma unroll
    for (int it = 0; it < kGatherIT; ++it) {
        const int e = (sub * kGatherIT + it) * kGatherNT + threadIdx.x;
        const int ec = e < ppp ? e : ppp - 1;
        const int r = ec / g.cpr, c = ec - r * g.cpr;
        rr[it] = e < ppp ? r : -1;
        cc[it] = c;
        jj[it] = ib[r];
    }
    wait_vmcnt<0>();
#pragma unroll
    for (int it = 0; it < kGatherIT; ++it) {
        const int j = jj[it];
        v[it] = uint4{0u, 0u, 0u, 0u};
        if (j >= 0 && j < g.n_src) v[it] = ld16(s0 + (int64_t)j * g.sr + (int64_t)cc[it] * 16);
    }
#pragma unroll
    for (int it = 0; it < kGatherIT; ++it)
        if (rr[it] >= 0) st16(d0 + (int64_t)rr[it] * g.dr + (int64_t)cc[it] * 16, v[it]);
}

// ---- nearest kept token (Sec. 4.3, assignment of the pruned tokens) -------
// Ordering by higher cosine, then lower slot, is a total order, so the
// maximum does not depend on the order in which candidates are combined.
__device__ __forceinline__ bool better(float v, int s, float bv, int bs) {
    return v > bv || (v == bv && s < bs);
}

// The best (value, slot) of the 16 lanes of each row, left in every lane of
// the row: DPP exchanges pairing lanes as an xor butterfly over 1, 2, 4, 8
// does (the order is total, so any pairing gives the same best).
__device__ __forceinline__ void row16_best(float &bv, int &bs) {
    auto step = [&](float ov, int os) {
        if (better(ov, os, bv, bs)) {
            bv = ov;
            bs = os;
        }
    };
    step(dpp_f32<0xB1>(bv), dpp_i32<0xB1>(bs));
    step(dpp_f32<0x4E>(bv), dpp_i32<0x4E>(bs));
    step(dpp_f32<0x141>(bv), dpp_i32<0x141>(bs));
    step(dpp_f32<0x140>(bv), dpp_i32<0x140>(bs));
}

// The same over the 64 lanes of a wave (every lane active), returned to
// every lane: the rows, then their bests read from lanes 0, 16, 32, 48.
__device__ __forceinline__ void wave_best(float &bv, int &bs) {
    row16_best(bv, bs);
    float v = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(bv), 0));
    int sl = __builtin_amdgcn_readlane(bs, 0);
#pragma unroll
    for (int r = 1; r < 4; ++r) {
        const float rv = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(bv), 16 * r));
        const int rs = __builtin_amdgcn_readlane(bs, 16 * r);
        if (better(rv, rs, v, sl)) {
            v = rv;
            sl = rs;
        }
    }
    bv = v;
    bs = sl;
}

// The split-k Gram's partial dot products part[KS][B][Mp][N1] -> the slot of
// the nearest kept token of every pruned row.
struct ReduceJob {
    const float *part;
    int B, Mp, N1, Nv, KS;
    const float *invn;      // [B][Nv] inverse token norms
    const int32_t *pruned;  // [B][Mp]
    const int32_t *kept;    // [B][N1]
    int32_t *assign;        // [B][Nv]
    int nblocks;            // workgroups of four rows carried by another launch; 0: none
};

// One wave, pruned row m of sample b: adds the k slices in slice order,
// forms the cosine to every kept token and writes the slot of the best one
// (higher cosine, then lower slot).  Slices are loaded in blocks of U with
// clamped addresses, so every load of a block is in flight at once.
template <int U>
__device__ __forceinline__ void gram_reduce_row(const ReduceJob &j, int m, int b, int lane) {
    constexpr int CPL = 4;  // columns per lane per pass
    const int tok = j.pruned[(size_t)b * j.Mp + m];
    const float ia = j.invn[(size_t)b * j.Nv + tok];
    const size_t kstride = (size_t)j.B * j.Mp * j.N1;
    const float *prow = j.part + ((size_t)b * j.Mp + m) * j.N1;
    float bv = -INFINITY;
    int bs = 0x7FFFFFFF;
    for (int n0 = 0; n0 < j.N1; n0 += 64 * CPL) {
        int nc[CPL];
        float kin[CPL], dot[CPL];
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
            nc[c] = min(n0 + c * 64 + lane, j.N1 - 1);
            kin[c] = j.invn[(size_t)b * j.Nv + j.kept[(size_t)b * j.N1 + nc[c]]];
            dot[c] = 0.f;
        }
        for (int ks0 = 0; ks0 < j.KS; ks0 += U) {
            float v[U][CPL];
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int c = 0; c < CPL; ++c)
                    v[u][c] = prow[(size_t)min(ks0 + u, j.KS - 1) * kstride + nc[c]];
#pragma unroll
            for (int u = 0; u < U; ++u)
                if (ks0 + u < j.KS) {
#pragma unroll
                    for (int c = 0; c < CPL; ++c) dot[c] += v[u][c];
                }
        }
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
            const int n = n0 + c * 64 + lane;
            const float cs = dot[c] * ia * kin[c];
            if (n < j.N1 && better(cs, n, bv, bs)) {
                bv = cs;
                bs = n;
            }
        }
    }
    wave_best(bv, bs);
    if (lane == 0) j.assign[(size_t)b * j.Nv + tok] = bs;
}

// Rows of gram_reduce_row per carried workgroup (one per wave of 256).
constexpr int kReduceRowsPerBlock = 4;

// ----------------------------------------------------------------------------
// Split-k products (the cosine, and the Grams that are too small to fill the
// chip with full-k tiles).
//
// A workgroup owns a 64 x 64 output tile and one k slice of its rows (streamed
// into LDS, see pv_tile_lds.h); the k slices are added in slice order by the
// reduce kernels.  Slicing k spreads a B=1 problem over every CU while each
// CU fetches only a few tens of KB; the price is KS fp32 partial tiles, which
// stay in L2.
// ----------------------------------------------------------------------------
constexpr int kPT = 64;  // tile edge of the split-k products
template <int DT, int NS>
using PTile = TileGemmLds<DT, kPT, kPT, 2, 2, NS>;
// Ring depth of the split-k tiles: three 16 KB stages.  Measured: a deeper
// ring costs more (fewer workgroups fit a CU) than the extra loads in flight
// gain.
constexpr int kSplitNS = 3;


// gram_partial: 1-D grid over (sample, k slice, kept tile, pruned tile) in
// XCD order (pruned tiles of one kept tile and slice are adjacent: they share
// the kept rows).  Writes partial dot products part[ks][b][Mp][N1].
// blk: this workgroup's index among the launch's `total` tile workgroups.
// EXT: the LDS ring is `ext_ring` (the tile's LDS_BYTES, shared with the
// other workgroups of a launch that carries another step); else its own.
// Tiles of BM pruned x BN kept rows (four waves of BM/2 x BN/2).
template <int DT, int NS, bool EXT = false, int BM = kPT, int BN = kPT>
__device__ __forceinline__ void gram_partial_tile(const char *__restrict__ vis, int B, int Nv,
                                                  int d_bytes, const int32_t *__restrict__ kept,
                                                  int N1, const int32_t *__restrict__ pruned,
                                                  int Mp, int ntm, int ntn, int KS,
                                                  float *__restrict__ part, int total, int blk,
                                                  char *ext_ring = nullptr) {
    using G = TileGemmLds<DT, BM, BN, 2, 2, NS>;
    __shared__ int32_t rowtok[G::ROWS];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / 2, wn = wave % 2;
    const int tile = xcd_tile(blk, total);
    const int mt = tile % ntm;
    const int nt = (tile / ntm) % ntn;
    const int ks = (tile / (ntm * ntn)) % KS;
    const int b = tile / (ntm * ntn * KS);
    const int m0 = mt * BM, n0 = nt * BN;
    const int32_t *pr = pruned + (size_t)b * Mp;
    const int32_t *kp = kept + (size_t)b * N1;
    for (int r = tid; r < G::ROWS; r += G::NT)
        rowtok[r] = (r < BM) ? pr[min(m0 + r, Mp - 1)] : kp[min(n0 + r - BM, N1 - 1)];
    __syncthreads();
    const char *vbase = vis + (size_t)b * Nv * d_bytes;
    auto row_ptr = [&](int r) -> const char * { return vbase + (size_t)rowtok[r] * d_bytes; };
    const int nch = d_bytes / G::CHUNK;
    const int c0 = (int)(((long long)nch * ks) / KS), c1 = (int)(((long long)nch * (ks + 1)) / KS);
    f32x4_t acc[G::FM][G::FN];
    float sa[G::FM], sb[G::FN];
    if constexpr (EXT) G::template run_in<false>(ext_ring, row_ptr, c0, c1, acc, sa, sb);
    else G::template run<false>(row_ptr, c0, c1, acc, sa, sb);
    float *pb = part + ((size_t)ks * B + b) * Mp * N1;
#pragma unroll
    for (int fm = 0; fm < G::FM; ++fm)
#pragma unroll
        for (int fn = 0; fn < G::FN; ++fn) {
            const int n = n0 + wn * G::SUB_N + fn * 16 + (lane & 15);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int m = m0 + wm * G::SUB_M + fm * 16 + (lane >> 4) * 4 + e;
                if (m < Mp && n < N1) pb[(size_t)m * N1 + n] = acc[fm][fn][e];
            }
        }
}

// The split-k Gram carried by another launch (its tiles after that launch's
// own workgroups).
struct GramJob {
    const char *vis;
    int B, Nv, d_bytes;
    const int32_t *kept;    // [B][N1]
    int N1;
    const int32_t *pruned;  // [B][Mp]
    int Mp, ntm, ntn, KS;
    float *part;            // [KS][B][Mp][N1]
    int nblocks;            // tile workgroups (B * KS * ntm * ntn); 0: none
};

// What the merge launch of the one-call step carries besides the merge: the
// merged rows of the slots the head-aware top-N_2 kept, written straight to
// their compacted places, and the compaction of K and V to those slots.
struct MergeCarry {
    const int32_t *slot_of2;  // [B][N1] position of each slot among the N_2 kept, or -1
    char *hidden2;            // [B][N2] rows of d_bytes
    int N2;
    GatherJob gj;             // K and V of the N_2 kept slots
};


// ---- head-aware score: v and the top-N_2 (Eq. v, Sec. 4.4) ---------------
constexpr int kSelU = 16;

struct SelectJob {
    const float *partial;  // [B][nparts][N] column sums of the score blocks
    int nparts, N;
    float inv_norm;        // 1 / (rows x heads)
    float *v;              // [B][N]
    int budget;
    int32_t *kept;         // [B][budget]
    int nblocks;           // samples carried by another launch; 0: none
    int32_t *slot_of;      // [B][N] position of each column in kept, or -1 (may be NULL)
};

// inv_norm x the partials of column j added in part order, loaded in blocks
// of kSelU with clamped addresses (all loads of a block in flight).
template <int NT, int EMAX>
__device__ __forceinline__ float select_sum(const SelectJob &sj, const float *pb, int j) {
    const int N = sj.N, nparts = sj.nparts;
    float s = 0.f;
    for (int t0 = 0; t0 < nparts; t0 += kSelU) {
        float v[kSelU];
#pragma unroll
        for (int u = 0; u < kSelU; ++u) v[u] = pb[(size_t)min(t0 + u, nparts - 1) * N + j];
#pragma unroll
        for (int u = 0; u < kSelU; ++u)
            if (t0 + u < nparts) s += v[u];
    }
    return s * sj.inv_norm;
}

// Workgroup of NT threads, sample b: v[j] = select_sum for every column, then
// the top-budget of v (lower index first among equal scores), ascending.
template <int NT, int EMAX>
__device__ __forceinline__ void score_select_block(const SelectJob &sj, int b) {
    __shared__ TopkSmem sm;
    const int N = sj.N, nparts = sj.nparts;
    const float *pb = sj.partial + (size_t)b * nparts * N;
    float *vb = sj.v + (size_t)b * N;
    const int E = topk_per_thread(N, NT), t = threadIdx.x;
    uint32_t key[EMAX];
    if constexpr (EMAX == 1) {
        key[0] = 0u;
        if (E == 1 && t < N) {
            const float s = select_sum<NT, EMAX>(sj, pb, t);
            vb[t] = s;
            key[0] = order_key(s);
        }
    } else {
        // the sums with the columns spread over the lanes (each load of a
        // part then covers contiguous columns), handed to block_topk's
        // ownership (E consecutive columns per thread) through LDS
        __shared__ float vs[EMAX * NT];
#pragma unroll
        for (int e = 0; e < EMAX; ++e) {
            const int j = t + e * NT;
            if (e < E && j < N) {
                const float s = select_sum<NT, EMAX>(sj, pb, j);
                vb[j] = s;
                vs[j] = s;
            }
        }
        __syncthreads();
#pragma unroll
        for (int e = 0; e < EMAX; ++e) {
            const int j = t * E + e;
            key[e] = (e < E && j < N) ? order_key(vs[j]) : 0u;
        }
    }
    block_topk<NT, EMAX>(key, N, sj.budget, sj.kept + (size_t)b * sj.budget, nullptr,
                         sj.slot_of ? sj.slot_of + (size_t)b * N : nullptr, sm);
}

}  // namespace pv
