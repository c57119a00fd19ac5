// Pruning before the LLM (Sec. 4.3): cross-modal cosine (equation for M),
// row centring (equation for M-hat), max-pooling (equation for p), top-N_1,
// nearest-centroid assignment of the pruned tokens and their aggregation.
//
// Kernel sequence of one call (all on the caller's stream):
//   cos_partial   anchors x vis on MFMA, split over k: partial dot products
//                 and partial sums of squares
//   cos_reduce    adds the k slices: cosines M, per-tile row sums, inverse
//                 norms of the visual tokens
//   center        p[j] = max_i (M[i][j] - mean_i)
//   select        top-N_1 radix select, one workgroup per sample
//   gram_partial  pruned x kept Gram on MFMA, split over k
//   gram_reduce   adds the k slices, cosine, row argmax -> assignment
//     (large Grams instead: gram_tile, LDS-staged 128x128 full-k tiles with a
//      fused argmax per column tile, then gram_finish across column tiles)
//   merge         centroid <- mean of itself and its members
// In the whole-step call (pv_prune_pipeline) gram_partial also carries the
// K/V compaction of the kept tokens and merge the head-aware top-N_2, as
// extra workgroups (pv_jobs.h); gram_reduce's rows then ride in the score's
// launch.
// Workgroups never wait on or signal each other: every cross-workgroup
// dependency is a kernel boundary, so no kernel needs a device-wide fence
// (on this chip a device-scope fence writes back and invalidates the L2).
#include "pv_jobs.h"
#include "pv_launch.h"
#include "pv_tile_lds.h"

#include <math.h>
#include <string.h>

namespace pv {

// cos_partial: 1-D grid over (sample, k slice, anchor tile, token tile) in XCD
// order (token tiles of one anchor tile and slice are adjacent: they share the
// anchor rows).  Writes partial dot products part[ks][b][Nt][Nv] and partial
// sums of squares of the token rows ssv[ks][b][Nv] and anchor rows
// ssa[ks][b][Nt].
//
// Tiles of BT x BT (four waves of BT/2 x BT/2): 64 with a three-stage ring
// (three workgroups per CU), or 128 with two stages (two per CU) when there
// are more than 64 anchors, which then halves the rows each CU loads per
// output.
template <int DT, int NS, int BT>
__global__ __launch_bounds__(256) void cos_partial_kernel(
    const char *__restrict__ vis, const char *__restrict__ anchors, int B, int Nv, int Nt,
    int d_bytes, int njt, int nit, int KS, float *__restrict__ part, float *__restrict__ ssv,
    float *__restrict__ ssa) {
    using G = TileGemmLds<DT, BT, BT, 2, 2, NS>;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / 2, wn = wave % 2;
    const int total = B * KS * nit * njt;
    const int tile = xcd_tile(blockIdx.x, total);
    const int jt = tile % njt;
    const int it = (tile / njt) % nit;
    const int ks = (tile / (njt * nit)) % KS;
    const int b = tile / (njt * nit * KS);
    const int i0 = it * BT, j0 = jt * BT;
    const char *abase = anchors + (size_t)b * Nt * d_bytes;
    const char *vbase = vis + (size_t)b * Nv * d_bytes;
    auto row_ptr = [&](int r) -> const char * {
        if (r < BT) return abase + (size_t)min(i0 + r, Nt - 1) * d_bytes;
        return vbase + (size_t)min(j0 + r - BT, Nv - 1) * d_bytes;
    };
    const int nch = d_bytes / G::CHUNK;
    const int c0 = (int)(((long long)nch * ks) / KS), c1 = (int)(((long long)nch * (ks + 1)) / KS);
    f32x4_t acc[G::FM][G::FN];
    float sa[G::FM], sb[G::FN];
    G::template run<true>(row_ptr, c0, c1, acc, sa, sb);
    const size_t kb = (size_t)ks * B + b;
    float *pb = part + kb * Nt * Nv;
#pragma unroll
    for (int fm = 0; fm < G::FM; ++fm)
#pragma unroll
        for (int fn = 0; fn < G::FN; ++fn) {
            const int j = j0 + wn * G::SUB_N + fn * 16 + (lane & 15);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int i = i0 + wm * G::SUB_M + fm * 16 + (lane >> 4) * 4 + e;
                if (i < Nt && j < Nv) pb[(size_t)i * Nv + j] = acc[fm][fn][e];
            }
        }
    // sums of squares: anchor rows from the waves of the first column, token
    // rows from the waves of the first row (each row read by exactly one)
    if (wn == 0 && jt == 0) {
#pragma unroll
        for (int f = 0; f < G::FM; ++f) {
            const float v = G::row_sumsq(sa[f]);
            const int i = i0 + wm * G::SUB_M + f * 16 + (lane & 15);
            if (lane < 16 && i < Nt) ssa[kb * Nt + i] = v;
        }
    }
    if (wm == 0 && it == 0) {
#pragma unroll
        for (int f = 0; f < G::FN; ++f) {
            const float v = G::row_sumsq(sb[f]);
            const int j = j0 + wn * G::SUB_N + f * 16 + (lane & 15);
            if (lane < 16 && j < Nv) ssv[kb * Nv + j] = v;
        }
    }
}

// cos_reduce: grid (ceil(Nv / 64), ceil(Nt / 4), B), 256 threads, one output
// per thread (wave = anchor row, lane = token).  Adds the k slices in slice
// order, forms cos = dot / (|a| |v|) (0 for a zero vector), writes
// M[b][Nt][Nv], the row sums of M over this workgroup's 64 tokens
// rowsum[b][Nv/64][Nt] and (first row group) the inverse token norms.
constexpr int kRedTok = 64, kRedRows = 4;

// Slice loads in flight per block of a reduction: the smallest of 1, 2, 4, 8,
// 16 that covers KS (a block of clamped loads past KS would only repeat the
// last slice).
inline int reduce_unroll(int KS) { return KS <= 1 ? 1 : KS <= 2 ? 2 : KS <= 4 ? 4 : KS <= 8 ? 8 : 16; }

template <int kRedU>
__global__ __launch_bounds__(256) void cos_reduce_kernel(
    const float *__restrict__ part, const float *__restrict__ ssv, const float *__restrict__ ssa,
    int B, int Nv, int Nt, int KS, float *__restrict__ M, float *__restrict__ rowsum,
    float *__restrict__ invn_vis) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int jt = blockIdx.x, b = blockIdx.z;
    const int njt = gridDim.x;
    const int i = blockIdx.y * kRedRows + wave;
    const int j = jt * kRedTok + lane;
    const int jc = min(j, Nv - 1), ic = min(i, Nt - 1);
    // slices in blocks of kRedU with clamped (always valid) addresses, so a
    // block's loads are all in flight at once; added in slice order
    float sv = 0.f, sa = 0.f, dot = 0.f;
    for (int ks0 = 0; ks0 < KS; ks0 += kRedU) {
        float v[kRedU], a[kRedU], p[kRedU];
#pragma unroll
        for (int u = 0; u < kRedU; ++u) {
            const size_t kb = (size_t)min(ks0 + u, KS - 1) * B + b;
            v[u] = ssv[kb * Nv + jc];
            a[u] = ssa[kb * Nt + ic];
            p[u] = part[(kb * Nt + ic) * Nv + jc];
        }
#pragma unroll
        for (int u = 0; u < kRedU; ++u) {
            if (ks0 + u < KS) {
                sv += v[u];
                sa += a[u];
                dot += p[u];
            }
        }
    }
    const float inv_v = (sv > 0.f) ? 1.0f / sqrtf(sv) : 0.f;
    const float inv_a = (sa > 0.f) ? 1.0f / sqrtf(sa) : 0.f;
    if (blockIdx.y == 0 && wave == 0 && j < Nv) invn_vis[(size_t)b * Nv + j] = inv_v;
    const float cs = dot * inv_a * inv_v;
    if (i < Nt && j < Nv) M[((size_t)b * Nt + i) * Nv + j] = cs;
    float rs = (j < Nv) ? cs : 0.f;
    rs = wave_sum64(rs);
    if (lane == 0 && i < Nt) rowsum[((size_t)b * njt + jt) * Nt + i] = rs;
}

// ----------------------------------------------------------------------------
// cos_full: the cosine for small inputs (one sample of LLaVA-1.5 size), where
// a split-k pass plus its reduction costs two launches for a few MB.  1-D grid
// over (sample, token tile, anchor tile) of 16 x 16 tiles in XCD order, 512
// threads.  Each workgroup computes its tile of M over the whole k range: the
// eight waves take an eighth of k each and stream their part of the 32 rows
// straight into their own LDS ring, so the k loop needs no barrier.  The wave
// results are added in wave order; the tile then writes M, its per-anchor row
// sums over its 16 tokens (rowsum[b][token tile][Nt]) and, for the first anchor
// tile, the inverse token norms.
// ----------------------------------------------------------------------------
constexpr int kFT = 16;   // tile edge

template <int DT, int NW, int kFNS>
__global__ __launch_bounds__(64 * NW) void cos_full_kernel(
    const char *__restrict__ vis, const char *__restrict__ anchors, int Nv, int Nt, int d_bytes,
    int nit, int njt, float *__restrict__ M, float *__restrict__ rowsum,
    float *__restrict__ invn_vis) {
    constexpr int ROWS = 2 * kFT, STAGE = ROWS * 128, IPW = STAGE / 1024;
    __shared__ __attribute__((aligned(16))) char ring[NW][kFNS][STAGE];
    __shared__ float accb[NW][kFT][kFT];
    __shared__ float ssab[NW][kFT], ssvb[NW][kFT];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    // anchor tiles fastest: the run of tiles an XCD receives covers every
    // anchor tile of a few token tiles, so its L2 holds all the anchor rows
    // and few token rows (token tiles fastest would give it one anchor tile
    // and many token tiles, and every XCD would fetch the token rows again)
    const int L = xcd_tile(blockIdx.x, gridDim.x);
    const int it = L % nit, jt = (L / nit) % njt, b = L / (njt * nit);
    const int i0 = it * kFT, j0 = jt * kFT;
    const char *abase = anchors + (size_t)b * Nt * d_bytes;
    const char *vbase = vis + (size_t)b * Nv * d_bytes;
    const int nch = d_bytes / 128;
    const int c0 = nch * wave / NW, c1 = nch * (wave + 1) / NW;
    const int nc = c1 - c0;

    // this lane's row and piece for each of the IPW loads of a chunk
    const char *src[IPW];
#pragma unroll
    for (int q = 0; q < IPW; ++q) {
        const int pos = q * 64 + lane;
        const int r = pos >> 3, slot = pos & 7;
        const char *row = (r < kFT) ? abase + (size_t)min(i0 + r, Nt - 1) * d_bytes
                                    : vbase + (size_t)min(j0 + r - kFT, Nv - 1) * d_bytes;
        src[q] = row + (size_t)c0 * 128 + ((slot ^ (r & 7)) << 4);
    }
    auto issue = [&](int i) {
        char *dst = ring[wave][i % kFNS];
#pragma unroll
        for (int q = 0; q < IPW; ++q)
            lds_dma16(src[q] + (size_t)i * 128, dst + q * 1024);
    };
#pragma unroll
    for (int pp = 0; pp < kFNS - 1; ++pp)
        if (pp < nc) issue(pp);
    f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
    float sa = 0.f, sv = 0.f;
    const int kq = lane >> 4, ra = lane & 15, rv = kFT + (lane & 15);
    for (int i = 0; i < nc; ++i) {
        if (i + kFNS - 1 <= nc) wait_vmcnt<IPW * (kFNS - 2)>();
        else wait_vmcnt<0>();
        if (i + kFNS - 1 < nc) issue(i + kFNS - 1);
        const char *sp = ring[wave][i % kFNS];
        uint4 a[2], v[2];
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {  // both 64-byte windows of the chunk, one wait
            const int piece = s2 * 4 + kq;
            a[s2] = lds_read16(sp + ra * 128 + ((piece ^ (ra & 7)) << 4));
            v[s2] = lds_read16(sp + rv * 128 + ((piece ^ (rv & 7)) << 4));
        }
        lds_wait();
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
            lds_after_wait(a[s2]);
            lds_after_wait(v[s2]);
            sa += sumsq16<DT>(a[s2]);
            sv += sumsq16<DT>(v[s2]);
            acc = mma16<DT>(a[s2], v[s2], acc);
        }
    }
    // the four quarters of each row's sum of squares, in a fixed order
    sa += __shfl_xor(sa, 16, 64);
    sa += __shfl_xor(sa, 32, 64);
    sv += __shfl_xor(sv, 16, 64);
    sv += __shfl_xor(sv, 32, 64);
#pragma unroll
    for (int e = 0; e < 4; ++e) accb[wave][4 * kq + e][lane & 15] = acc[e];
    if (lane < kFT) {
        ssab[wave][lane] = sa;
        ssvb[wave][lane] = sv;
    }
    __syncthreads();
    if (tid >= kFT * kFT) return;  // no barrier follows
    // one output per thread: anchor ii, token jj; waves added in order
    const int ii = tid >> 4, jj = tid & 15;
    float dot = 0.f, a2 = 0.f, v2 = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
        dot += accb[w][ii][jj];
        a2 += ssab[w][ii];
        v2 += ssvb[w][jj];
    }
    const float inv_a = (a2 > 0.f) ? 1.0f / sqrtf(a2) : 0.f;
    const float inv_v = (v2 > 0.f) ? 1.0f / sqrtf(v2) : 0.f;
    const int i = i0 + ii, j = j0 + jj;
    const float cs = dot * inv_a * inv_v;
    if (i < Nt && j < Nv) M[((size_t)b * Nt + i) * Nv + j] = cs;
    if (it == 0 && ii == 0 && j < Nv) invn_vis[(size_t)b * Nv + j] = inv_v;
    float rs = (j < Nv) ? cs : 0.f;
    rs = row16_sum(rs);
    if (jj == 0 && i < Nt) rowsum[((size_t)b * njt + jt) * Nt + i] = rs;
}

// ----------------------------------------------------------------------------
// center: grid (ceil(Nv / 64), B), 256 threads.  Two phases, each with all of
// its loads in flight before the first is used, so that a phase costs one
// memory latency: the row means from the per-tile partial sums (4 threads per
// row, each adding every fourth tile in tile order, the four partials then
// added in order), and the max over the rows (4 threads per token).
// ----------------------------------------------------------------------------
constexpr int kCenNT = 256;
constexpr int kCenTok = 64;
constexpr int kCenU = 16;  // loads in flight per thread

// base[t * stride] added over t = t0, t0 + step, ... < n, in that order
// (n >= 1; the addresses of a block are clamped, so every load is valid).
__device__ __forceinline__ float strided_sum(const float *__restrict__ base, size_t stride, int t0,
                                             int step, int n) {
    float s = 0.f;
    for (int c = t0; c < n; c += step * kCenU) {
        float v[kCenU];
#pragma unroll
        for (int u = 0; u < kCenU; ++u) v[u] = base[(size_t)min(c + u * step, n - 1) * stride];
#pragma unroll
        for (int u = 0; u < kCenU; ++u)
            if (c + u * step < n) s += v[u];
    }
    return s;
}

__global__ __launch_bounds__(kCenNT) void center_kernel(const float *__restrict__ M,
                                                        const float *__restrict__ rowsum,
                                                        const int32_t *__restrict__ row_mask,
                                                        int njt, int Nt, int Nv,
                                                        float *__restrict__ p) {
    // [0, Nt): row means; [Nt, 2 Nt): the same with +inf for rows that are
    // not anchors (a row at +inf never wins the max)
    extern __shared__ float mu[];
    __shared__ float rpart[4][kCenTok];
    __shared__ int any_row;
    const int b = blockIdx.y, tid = threadIdx.x;
    const int jl = tid & (kCenTok - 1), g = tid / kCenTok;
    const int j = blockIdx.x * kCenTok + jl;
    // the first block of this thread's column of M does not depend on the
    // row means: its loads are in flight during the first phase
    const float *col = M + (size_t)b * Nt * Nv + min(j, Nv - 1);
    float v0[kCenU];
#pragma unroll
    for (int u = 0; u < kCenU; ++u) v0[u] = col[(size_t)min(g + 4 * u, Nt - 1) * Nv];
    if (tid == 0) any_row = row_mask ? 0 : 1;
    for (int r0 = 0; r0 < Nt; r0 += kCenTok) {
        const int i = r0 + (tid >> 2), q = tid & 3;
        float s = 0.f;
        if (i < Nt) s = strided_sum(rowsum + (size_t)b * njt * Nt + i, Nt, q, 4, njt);
        rpart[q][tid >> 2] = s;
        __syncthreads();
        if (tid < kCenTok && r0 + tid < Nt) {
            const int ii = r0 + tid;
            const float m = (((rpart[0][tid] + rpart[1][tid]) + rpart[2][tid]) + rpart[3][tid]) / (float)Nv;
            const bool use = !row_mask || row_mask[(size_t)b * Nt + ii] != 0;
            mu[ii] = m;
            mu[Nt + ii] = use ? m : INFINITY;
            if (use && row_mask) any_row = 1;
        }
        __syncthreads();
    }
    // an empty mask means every row
    const float *mrow = (row_mask && any_row) ? mu + Nt : mu;
    float m = -INFINITY;
    if (j < Nv) {
#pragma unroll
        for (int u = 0; u < kCenU; ++u)
            if (g + 4 * u < Nt) m = fmaxf(m, v0[u] - mrow[g + 4 * u]);
        for (int i0 = g + 4 * kCenU; i0 < Nt; i0 += 4 * kCenU) {
            float v[kCenU];
#pragma unroll
            for (int u = 0; u < kCenU; ++u) v[u] = col[(size_t)min(i0 + 4 * u, Nt - 1) * Nv];
#pragma unroll
            for (int u = 0; u < kCenU; ++u)
                if (i0 + 4 * u < Nt) m = fmaxf(m, v[u] - mrow[i0 + 4 * u]);
        }
    }
    rpart[g][jl] = m;
    __syncthreads();
    if (g == 0 && j < Nv)
        p[(size_t)b * Nv + j] = fmaxf(fmaxf(rpart[0][jl], rpart[1][jl]), fmaxf(rpart[2][jl], rpart[3][jl]));
}

// ----------------------------------------------------------------------------
// select: grid (B), NT threads; top-`budget` of p with its complement list and
// the slot of every kept token.  Each thread holds EMAX keys in registers.
// ----------------------------------------------------------------------------
template <int NT, int EMAX>
__global__ __launch_bounds__(NT) void select_kernel(const float *__restrict__ p, int Nv,
                                                    int budget, int32_t *__restrict__ kept,
                                                    int32_t *__restrict__ pruned,
                                                    int32_t *__restrict__ slot_of) {
    __shared__ TopkSmem sm;
    const int b = blockIdx.x;
    const float *pb = p + (size_t)b * Nv;
    const int E = topk_per_thread(Nv, NT), j0 = threadIdx.x * E;
    uint32_t key[EMAX];
#pragma unroll
    for (int e = 0; e < EMAX; ++e) key[e] = (e < E && j0 + e < Nv) ? order_key(pb[j0 + e]) : 0u;
    block_topk<NT, EMAX>(key, Nv, budget, kept + (size_t)b * budget,
                         pruned ? pruned + (size_t)b * (Nv - budget) : nullptr,
                         slot_of ? slot_of + (size_t)b * Nv : nullptr, sm);
}

// ----------------------------------------------------------------------------
// Nearest centroid: best (cosine, slot) of every pruned row, with the total
// order of `better` (higher cosine, then lower slot).
// ----------------------------------------------------------------------------
// gram_finish: grid (ceil(Mp / 256), B).  Best column tile of every pruned
// row, combined in tile order with the total order above.  The candidates of
// kFinU tiles are loaded at once (a loop that compares each one as it arrives
// waits for every load in turn); past the last tile the last one repeats,
// which cannot change a maximum under a total order.
constexpr int kFinNT = 256;
constexpr int kFinU = 16;

__global__ __launch_bounds__(kFinNT) void gram_finish_kernel(const float *__restrict__ best_val,
                                                             const int32_t *__restrict__ best_slot,
                                                             int ntn, int Mp, int Nv,
                                                             const int32_t *__restrict__ pruned,
                                                             int32_t *__restrict__ assign) {
    const int b = blockIdx.y;
    const int m = blockIdx.x * kFinNT + threadIdx.x;
    if (m >= Mp) return;
    const int tok = pruned[(size_t)b * Mp + m];
    float bv = -INFINITY;
    int bs = 0x7FFFFFFF;
    for (int t0 = 0; t0 < ntn; t0 += kFinU) {
        float v[kFinU];
        int s[kFinU];
#pragma unroll
        for (int u = 0; u < kFinU; ++u) {
            const size_t at = ((size_t)b * ntn + min(t0 + u, ntn - 1)) * Mp + m;
            v[u] = best_val[at];
            s[u] = best_slot[at];
        }
#pragma unroll
        for (int u = 0; u < kFinU; ++u)
            if (better(v[u], s[u], bv, bs)) {
                bv = v[u];
                bs = s[u];
            }
    }
    assign[(size_t)b * Nv + tok] = bs;
}

template <int DT, int NS, int BM, int BN>
__global__ __launch_bounds__(256) void gram_partial_kernel(
    const char *__restrict__ vis, int B, int Nv, int d_bytes, const int32_t *__restrict__ kept,
    int N1, const int32_t *__restrict__ pruned, int Mp, int ntm, int ntn, int KS,
    float *__restrict__ part) {
    gram_partial_tile<DT, NS, false, BM, BN>(vis, B, Nv, d_bytes, kept, N1, pruned, Mp, ntm, ntn,
                                             KS, part, B * KS * ntn * ntm, blockIdx.x);
}

// gram_reduce: grid (ceil(Mp / 2), B), 128 threads, one wave per pruned row
// (gram_reduce_row).
template <int kGramU>
__global__ __launch_bounds__(128) void gram_reduce_kernel(ReduceJob j) {
    const int m = blockIdx.x * 2 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (m >= j.Mp) return;
    gram_reduce_row<kGramU>(j, m, blockIdx.y, threadIdx.x & 63);
}

// gram_tile: the large, MFMA-bound Grams.  1-D grid over (sample, pruned
// tile, kept tile) in XCD order (the kept tiles of one pruned tile are
// adjacent, so they share its rows in one L2); 256 x 128 tiles with the
// operands streamed straight into LDS (TileGemmLds::run_pc): eight matrix
// waves of 64 x 64 that only read fragments and multiply, NP producer waves
// that issue every load, a three-stage ring of 48 KB stages, one workgroup
// per CU.  A matrix wave that issued its own loads waited for the CU's load
// path to take them, between its MFMAs (measured: 29% of its time with
// 128 x 128 tiles); with the producers the Gram also keeps its pace when
// another stream's copies share the CU's load path.
// Writes the best (cosine, slot) of every pruned row within this kept tile,
// or the slot itself when there is only one kept tile.
template <int DT, int BM, int BN, int WM, int WN, int NS, int NP>
__global__ __launch_bounds__(64 * (WM * WN + NP)) void gram_tile_kernel(
    const char *__restrict__ vis, int Nv, int d_bytes, const int32_t *__restrict__ kept, int N1,
    const int32_t *__restrict__ pruned, int Mp, const float *__restrict__ invn, int ntm, int ntn,
    float *__restrict__ best_val, int32_t *__restrict__ best_slot, int32_t *__restrict__ assign) {
    using G = TileGemmLds<DT, BM, BN, WM, WN, NS>;
    constexpr int NTT = G::NT + 64 * NP;  // matrix waves, then producer waves
    __shared__ int32_t rowtok[G::ROWS];
    __shared__ float rowinv[G::ROWS];
    __shared__ float red_v[WN][BM];
    __shared__ int red_s[WN][BM];

    const int L = xcd_tile(blockIdx.x, gridDim.x);
    const int nt = L % ntn, mt = (L / ntn) % ntm, b = L / (ntn * ntm);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;
    const int m0 = mt * BM, n0 = nt * BN;
    const int32_t *pr = pruned + (size_t)b * Mp;
    const int32_t *kp = kept + (size_t)b * N1;

    for (int r = tid; r < G::ROWS; r += NTT) {
        const int tok = (r < BM) ? pr[min(m0 + r, Mp - 1)] : kp[min(n0 + r - BM, N1 - 1)];
        rowtok[r] = tok;
        rowinv[r] = invn[(size_t)b * Nv + tok];
    }
    __syncthreads();
    const char *vbase = vis + (size_t)b * Nv * d_bytes;
    auto row_ptr = [&](int r) -> const char * { return vbase + (size_t)rowtok[r] * d_bytes; };

    f32x4_t acc[G::FM][G::FN];
    __shared__ __attribute__((aligned(16))) char ring[G::LDS_BYTES];
    // matrix waves past the last pruned row or kept slot of an edge tile skip
    // their MFMAs (the epilogue ignores those rows and slots)
    G::template run_pc<NP>(ring, row_ptr, 0, d_bytes / G::CHUNK, acc, Mp - m0, N1 - n0);

    // producer waves hold no products
    if (__builtin_amdgcn_readfirstlane(wave) < WM * WN) {
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
                row16_best(bv, bs);
                if ((lane & 15) == 0) {
                    red_v[wn][r] = bv;
                    red_s[wn][r] = bs;
                }
            }
        }
    }
    __syncthreads();
    for (int r = tid; r < BM; r += NTT) {
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
// merge: grid (ceil(d_bytes / 1024), N1, B), 256 threads.  A workgroup owns
// one slot s and one 1 KB column block (16 bytes per lane).  The members of s
// (the tokens whose assignment is s, the kept token itself included) are
// listed in ascending token order with one block scan per round of 4096
// tokens; the four waves then take every fourth member, each wave one row
// after the other (the slots of the inputs this form serves hold a few
// members each; loading a wave's members together measured slower), and the
// column split spreads one slot's bytes over several CUs.  Each wave adds its
// members in list order (fp32) and the four partial sums are combined in wave
// order, so the result does not depend on timing.
// ----------------------------------------------------------------------------
constexpr int kMergeNT = 256;
constexpr int kMergeRound = 4096;                  // tokens listed per round
constexpr int kMergeTPT = kMergeRound / kMergeNT;  // tokens per thread per round

// Adds the elements of one 16-byte chunk to acc (fp32).
template <int DT>
__device__ __forceinline__ void add16(float (&acc)[DT == kBF16 ? 8 : 4], uint4 v) {
    const uint32_t w4[4] = {v.x, v.y, v.z, v.w};
    if (DT == kBF16) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            acc[2 * q] += __uint_as_float(w4[q] << 16);
            acc[2 * q + 1] += __uint_as_float(w4[q] & 0xFFFF0000u);
        }
    } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[q] += __uint_as_float(w4[q]);
    }
}

// Combines the waves' partial sums in wave order, divides by the member count
// and stores this lane's 16-byte chunk of the output row.
template <int DT, int NW>
__device__ __forceinline__ void merge_finish(float (&acc)[DT == kBF16 ? 8 : 4],
                                             float (&part)[NW][DT == kBF16 ? 8 : 4][64], int wave,
                                             int lane, int c, int nchunk, int total, char *out,
                                             char *out2 = nullptr) {
    constexpr int EPC = (DT == kBF16) ? 8 : 4;
    if (wave > 0) {
#pragma unroll
        for (int e = 0; e < EPC; ++e) part[wave][e][lane] = acc[e];
    }
    __syncthreads();
    if (wave == 0 && c < nchunk) {
#pragma unroll
        for (int w2 = 1; w2 < NW; ++w2)
#pragma unroll
            for (int e = 0; e < EPC; ++e) acc[e] += part[w2][e][lane];
        const float cntf = (float)total;
        uint32_t w4[4];
        if (DT == kBF16) {
#pragma unroll
            for (int q = 0; q < 4; ++q)
                w4[q] = f32_to_bf16_rne(acc[2 * q] / cntf) | (f32_to_bf16_rne(acc[2 * q + 1] / cntf) << 16);
        } else {
#pragma unroll
            for (int q = 0; q < 4; ++q) w4[q] = __float_as_uint(acc[q] / cntf);
        }
        st16(out + (size_t)c * 16, uint4{w4[0], w4[1], w4[2], w4[3]});
        if (out2) st16(out2 + (size_t)c * 16, uint4{w4[0], w4[1], w4[2], w4[3]});
    }
}

template <int DT>
__global__ __launch_bounds__(kMergeNT) void merge_kernel(const char *__restrict__ vis, int Nv,
                                                         int d_bytes,
                                                         const int32_t *__restrict__ assign,
                                                         int N1, char *__restrict__ merged,
                                                         MergeCarry mc) {
    constexpr int EPC = (DT == kBF16) ? 8 : 4;  // elements per 16-byte chunk
    constexpr int NW = kMergeNT / 64;
    __shared__ int list[kMergeRound];
    __shared__ int wsum[NW];
    __shared__ float part[NW][EPC][64];
    const int bx = blockIdx.x, s = blockIdx.y, b = blockIdx.z;
    // a carried compaction takes more rows of slots in sample 0's plane of
    // the grid: workgroup (x, N1 + r, 0) runs its block r * gridDim.x + x
    if (s >= N1) {
        const int g = (s - N1) * (int)gridDim.x + bx;
        if (b == 0 && g < mc.gj.nblocks) gather_block(mc.gj.ga, mc.gj.idx, mc.gj.k, g);
        return;
    }
    // the slot's row among the N_2 kept, when the head-aware top-N_2 kept it
    char *out2 = nullptr;
    if (mc.slot_of2) {
        const int pos = mc.slot_of2[(size_t)b * N1 + s];
        if (pos >= 0) out2 = mc.hidden2 + ((size_t)b * mc.N2 + pos) * d_bytes;
    }
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int nchunk = d_bytes >> 4;
    const int c = bx * 64 + lane;
    const char *col = vis + (size_t)b * Nv * d_bytes + (size_t)min(c, nchunk - 1) * 16;
    const int32_t *as = assign + (size_t)b * Nv;

    float acc[EPC];
#pragma unroll
    for (int e = 0; e < EPC; ++e) acc[e] = 0.f;
    int total = 0;
    for (int r0 = 0; r0 < Nv; r0 += kMergeRound) {
        const int rend = min(r0 + kMergeRound, Nv);
        const int tpt = (rend - r0 + kMergeNT - 1) / kMergeNT;  // uniform
        const int t0 = r0 + tid * tpt;
        int a[kMergeTPT];
#pragma unroll
        for (int e = 0; e < kMergeTPT; ++e)
            if (e < tpt) a[e] = as[min(t0 + e, rend - 1)];
        int mine = 0;
#pragma unroll
        for (int e = 0; e < kMergeTPT; ++e) mine += (e < tpt && t0 + e < rend && a[e] == s);
        int cnt;
        int w = block_excl_scan<kMergeNT>(mine, wsum, &cnt);
#pragma unroll
        for (int e = 0; e < kMergeTPT; ++e)
            if (e < tpt && t0 + e < rend && a[e] == s) list[w++] = t0 + e;
        __syncthreads();
        for (int m = wave; m < cnt; m += NW) add16<DT>(acc, ld16(col + (size_t)list[m] * d_bytes));
        total += cnt;
        __syncthreads();  // the list is rewritten by the next round
    }
    merge_finish<DT, NW>(acc, part, wave, lane, c, nchunk, total,
                         merged + ((size_t)b * N1 + s) * d_bytes, out2);
}

// ----------------------------------------------------------------------------
// Member lists for large inputs, where every merge workgroup scanning the whole
// assignment would cost more than the rows it adds.
//
// bucket: grid (ceil(N1 / 256), B), 512 or 1024 threads.  Lists the members of the
// 256 slots [256 g, 256 g + 256) in ascending token order: mcount[b][s],
// mstart[b][s] (offset in the sample's list region) and the lists themselves
// in mlist[b][g * Nv ...].  The assignment is staged in LDS; the waves take
// consecutive token segments and sweep them twice, 64 tokens per
// step: per-slot counts (integer atomics on the wave's counters in LDS), then
// placement at offsets that keep the segments in order.  In the placement the
// lanes of a step that hold the same slot are found with one ballot per bit
// of the slot offset (the lanes whose offsets agree on every bit), so a step
// costs the same whatever the number of distinct slots in it; each lane takes
// the next places in lane order and the lowest such lane advances the wave's
// counter of that slot.
// ----------------------------------------------------------------------------
constexpr int kBucketBits = 8;
constexpr int kBucketSlots = 1 << kBucketBits;
static_assert(kBucketSlots == kBucketSlotsPerGroup, "slots per bucket group");
// threads: 512, or 1024 from kBucketWideNv tokens (measured: 16 waves sweep
// the longer assignments faster, 8 cost less on short ones)
constexpr int kBucketWideNv = 2048;

// Lanes whose value v agrees with this lane's on the low kBucketBits bits,
// among the lanes in `act`.
__device__ __forceinline__ unsigned long long same_slot_lanes(int v, unsigned long long act) {
    unsigned long long same = act;
#pragma unroll
    for (int bit = 0; bit < kBucketBits; ++bit) {
        const bool on = (v >> bit) & 1;
        const unsigned long long ones = __ballot(on);
        same &= on ? ones : ~ones;
    }
    return same;
}

template <int kBucketNT>
__global__ __launch_bounds__(kBucketNT) void bucket_kernel(const int32_t *__restrict__ assign,
                                                           int Nv, int N1,
                                                           int32_t *__restrict__ mcount,
                                                           int32_t *__restrict__ mstart,
                                                           int32_t *__restrict__ mlist) {
    extern __shared__ int32_t sa[];  // [Nv] the sample's assignment
    constexpr int kBucketW = kBucketNT / 64;
    __shared__ int cur[kBucketW][kBucketSlots];
    __shared__ int wsum[kBucketW];
    const int g = blockIdx.x, b = blockIdx.y, tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int ngroups = gridDim.x;
    const int s0 = g * kBucketSlots;
    const int32_t *as = assign + (size_t)b * Nv;
    int32_t *lst = mlist + ((size_t)b * ngroups + g) * Nv;
    const unsigned long long lt = (1ull << lane) - 1ull;

    for (int e = lane; e < kBucketSlots; e += 64) cur[wave][e] = 0;
    // stage: eight loads per thread in flight per round
    for (int j0 = 0; j0 < Nv; j0 += kBucketNT * 8) {
        int v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = as[min(j0 + u * kBucketNT + tid, Nv - 1)];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            if (j0 + u * kBucketNT + tid < Nv) sa[j0 + u * kBucketNT + tid] = v[u];
    }
    __syncthreads();
    // this wave's token segment [t0, t1), whole 64-token steps
    const int seg = ((Nv + kBucketW - 1) / kBucketW + 63) / 64 * 64;
    const int t0 = min(wave * seg, Nv), t1 = min(t0 + seg, Nv);
    int *wc = cur[wave];

    // pass 1: this wave's count of every slot (integer atomics in LDS: the
    // counts do not depend on their order)
    for (int c0 = t0; c0 < t1; c0 += 64) {
        const int j = c0 + lane;
        const int v = (j < t1) ? sa[j] - s0 : -1;
        if (v >= 0 && v < kBucketSlots) atomicAdd(&wc[v], 1);
    }
    __syncthreads();
    // slot totals and offsets; then each wave's first position per slot
    int tot = 0;
    if (tid < kBucketSlots) {
#pragma unroll
        for (int w = 0; w < kBucketW; ++w) tot += cur[w][tid];
    }
    int all;
    const int base = block_excl_scan<kBucketNT>(tot, wsum, &all);
    if (tid < kBucketSlots) {
        if (s0 + tid < N1) {
            mcount[(size_t)b * N1 + s0 + tid] = tot;
            mstart[(size_t)b * N1 + s0 + tid] = g * Nv + base;
        }
        int run = base;
#pragma unroll
        for (int w = 0; w < kBucketW; ++w) {
            const int c = cur[w][tid];
            cur[w][tid] = run;
            run += c;
        }
    }
    __syncthreads();
    // pass 2: placement in token order
    for (int c0 = t0; c0 < t1; c0 += 64) {
        const int j = c0 + lane;
        const int v = (j < t1) ? sa[j] - s0 : -1;
        const bool rel = v >= 0 && v < kBucketSlots;
        const unsigned long long same = same_slot_lanes(v, __ballot(rel));
        if (rel) {
            lst[wc[v] + __popcll(same & lt)] = j;
            if ((same & lt) == 0ull) wc[v] += __popcll(same);
        }
    }
}

// merge_csr: as merge, with the member list read from the bucket output and
// CPL 16-byte chunks per lane (a column block of 64 * CPL chunks).  The list
// entries are read where they are (they are the same for every lane of a
// wave), so the chain per workgroup is count/offset, list, rows.  Wave w adds
// members w, w + 4, ... in list order.  Most slots hold a few members, one
// or two per wave, and take them one row after the other; a slot with more
// than kMergeFew members keeps kMergeHeavyU rows per wave in flight, so the
// few slots with a hundred members or more do not set the kernel's end.
// (Measured: loading repeats of the last member in place of the missing ones,
// or several rows per wave in every slot, costs the light slots more than it
// saves.)
constexpr int kMergeFew = 8;
constexpr int kMergeHeavyU = 4;
template <int DT, int CPL>
__global__ __launch_bounds__(kMergeNT) void merge_csr_kernel(
    const char *__restrict__ vis, int Nv, int d_bytes, const int32_t *__restrict__ mcount,
    const int32_t *__restrict__ mstart, const int32_t *__restrict__ mlist, int N1, int ngroups,
    char *__restrict__ merged) {
    constexpr int EPC = (DT == kBF16) ? 8 : 4;
    constexpr int NW = kMergeNT / 64;
    __shared__ float part[NW][CPL][EPC][64];
    const int s = blockIdx.y, b = blockIdx.z;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int nchunk = d_bytes >> 4;
    const char *vb = vis + (size_t)b * Nv * d_bytes;
    int cc[CPL];
#pragma unroll
    for (int t = 0; t < CPL; ++t) cc[t] = blockIdx.x * 64 * CPL + t * 64 + lane;
    const int total = mcount[(size_t)b * N1 + s];
    const int32_t *lst = mlist + (size_t)b * ngroups * Nv + mstart[(size_t)b * N1 + s];

    float acc[CPL][EPC];
#pragma unroll
    for (int t = 0; t < CPL; ++t)
#pragma unroll
        for (int e = 0; e < EPC; ++e) acc[t][e] = 0.f;
    if (total > kMergeFew) {
        // kMergeHeavyU rows in flight per wave; a member past the list loads
        // nothing and adds zero (acc starts at +0, so adding +0 changes no bit)
        for (int m0 = wave; m0 < total; m0 += NW * kMergeHeavyU) {
            uint4 v[kMergeHeavyU][CPL];
#pragma unroll
            for (int u = 0; u < kMergeHeavyU; ++u) {
                const char *row = vb + (size_t)lst[min(m0 + u * NW, total - 1)] * d_bytes;
                if (m0 + u * NW < total) {
#pragma unroll
                    for (int t = 0; t < CPL; ++t)
                        v[u][t] = ld16(row + (size_t)min(cc[t], nchunk - 1) * 16);
                } else {
#pragma unroll
                    for (int t = 0; t < CPL; ++t) v[u][t] = uint4{0u, 0u, 0u, 0u};
                }
            }
#pragma unroll
            for (int u = 0; u < kMergeHeavyU; ++u)
#pragma unroll
                for (int t = 0; t < CPL; ++t) add16<DT>(acc[t], v[u][t]);
        }
    } else {
        // at most kMergeFew / NW members per wave, one row after the other
        for (int m = wave; m < total; m += NW) {
            const char *row = vb + (size_t)lst[m] * d_bytes;
#pragma unroll
            for (int t = 0; t < CPL; ++t)
                add16<DT>(acc[t], ld16(row + (size_t)min(cc[t], nchunk - 1) * 16));
        }
    }
    char *out = merged + ((size_t)b * N1 + s) * d_bytes;
    if (wave > 0) {
#pragma unroll
        for (int t = 0; t < CPL; ++t)
#pragma unroll
            for (int e = 0; e < EPC; ++e) part[wave][t][e][lane] = acc[t][e];
    }
    __syncthreads();
    if (wave == 0) {
        const float cntf = (float)total;
#pragma unroll
        for (int t = 0; t < CPL; ++t) {
#pragma unroll
            for (int w2 = 1; w2 < NW; ++w2)
#pragma unroll
                for (int e = 0; e < EPC; ++e) acc[t][e] += part[w2][t][e][lane];
            if (cc[t] >= nchunk) continue;
            uint32_t w4[4];
            if (DT == kBF16) {
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    w4[q] = f32_to_bf16_rne(acc[t][2 * q] / cntf) |
                            (f32_to_bf16_rne(acc[t][2 * q + 1] / cntf) << 16);
            } else {
#pragma unroll
                for (int q = 0; q < 4; ++q) w4[q] = __float_as_uint(acc[t][q] / cntf);
            }
            st16(out + (size_t)cc[t] * 16, uint4{w4[0], w4[1], w4[2], w4[3]});
        }
    }
}

// cos_reduce4: the same for Nv % 4 == 0, four tokens per thread (16-byte
// loads of the slices, a wave covers 256 tokens of one anchor row): grid
// (ceil(Nv / 256), ceil(Nt / 4), B).  The row sums of M over each 64-token
// tile are the thread's four cosines added in order, then the 16 lanes of the
// tile (a DPP row reduction); the layout of rowsum is cos_reduce's.
constexpr int kRed4Tok = 256;

template <int kRedU>
__global__ __launch_bounds__(256) void cos_reduce4_kernel(
    const float *__restrict__ part, const float *__restrict__ ssv, const float *__restrict__ ssa,
    int B, int Nv, int Nt, int KS, float *__restrict__ M, float *__restrict__ rowsum,
    float *__restrict__ invn_vis) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int b = blockIdx.z;
    const int njt = (Nv + kRedTok - 1) / kRedTok;  // 64-token tiles of rowsum
    const int i = blockIdx.y * kRedRows + wave;
    const int j = blockIdx.x * kRed4Tok + lane * 4;
    const int jc = min(j, Nv - 4), ic = min(i, Nt - 1);
    float4 sv = {0.f, 0.f, 0.f, 0.f}, dot = {0.f, 0.f, 0.f, 0.f};
    float sa = 0.f;
    for (int ks0 = 0; ks0 < KS; ks0 += kRedU) {
        float4 v[kRedU], p[kRedU];
        float a[kRedU];
#pragma unroll
        for (int u = 0; u < kRedU; ++u) {
            const size_t kb = (size_t)min(ks0 + u, KS - 1) * B + b;
            v[u] = *reinterpret_cast<const float4 *>(ssv + kb * Nv + jc);
            a[u] = ssa[kb * Nt + ic];
            p[u] = *reinterpret_cast<const float4 *>(part + (kb * Nt + ic) * Nv + jc);
        }
#pragma unroll
        for (int u = 0; u < kRedU; ++u) {
            if (ks0 + u < KS) {
                sv.x += v[u].x; sv.y += v[u].y; sv.z += v[u].z; sv.w += v[u].w;
                sa += a[u];
                dot.x += p[u].x; dot.y += p[u].y; dot.z += p[u].z; dot.w += p[u].w;
            }
        }
    }
    auto inv = [](float q) { return (q > 0.f) ? 1.0f / sqrtf(q) : 0.f; };
    const float4 iv = {inv(sv.x), inv(sv.y), inv(sv.z), inv(sv.w)};
    const float ia = inv(sa);
    const bool live = j < Nv;  // Nv % 4 == 0: all four tokens or none
    if (blockIdx.y == 0 && wave == 0 && live) *reinterpret_cast<float4 *>(invn_vis + (size_t)b * Nv + j) = iv;
    const float4 cs = {dot.x * ia * iv.x, dot.y * ia * iv.y, dot.z * ia * iv.z, dot.w * ia * iv.w};
    if (i < Nt && live) *reinterpret_cast<float4 *>(M + ((size_t)b * Nt + i) * Nv + j) = cs;
    float rs = live ? ((cs.x + cs.y) + cs.z) + cs.w : 0.f;
    rs = row16_sum(rs);
    const int jt = blockIdx.x * (kRed4Tok / kRedTok) + (lane >> 4);
    if ((lane & 15) == 0 && i < Nt && jt < njt) rowsum[((size_t)b * njt + jt) * Nt + i] = rs;
}

// ----------------------------------------------------------------------------
// launchers
// ----------------------------------------------------------------------------
template <int DT, int NS, int BT>
static void cos_partial_go(const void *vis, const void *anchors, int B, int Nv, int Nt,
                           int d_bytes, int KS, float *part, float *ssv, float *ssa,
                           hipStream_t st) {
    const int njt = (Nv + BT - 1) / BT, nit = (Nt + BT - 1) / BT;
    const dim3 grid(B * KS * nit * njt);
    hipLaunchKernelGGL((cos_partial_kernel<DT, NS, BT>), grid, dim3(256), 0, st, (const char *)vis,
                       (const char *)anchors, B, Nv, Nt, d_bytes, njt, nit, KS, part, ssv, ssa);
}

hipError_t launch_cos_partial(int dt, const void *vis, const void *anchors, int B, int Nv, int Nt,
                              int d, int KS, float *part, float *ssv, float *ssa, hipStream_t st) {
    const int d_bytes = d * ((dt == kBF16) ? 2 : 4);
    const bool wide = cos_uses_wide_tiles(Nt, Nv);
    if (dt == kBF16) {
        if (wide) cos_partial_go<kBF16, 2, kWideTile>(vis, anchors, B, Nv, Nt, d_bytes, KS, part, ssv, ssa, st);
        else cos_partial_go<kBF16, kSplitNS, kPT>(vis, anchors, B, Nv, Nt, d_bytes, KS, part, ssv, ssa, st);
    } else {
        if (wide) cos_partial_go<kF32, 2, kWideTile>(vis, anchors, B, Nv, Nt, d_bytes, KS, part, ssv, ssa, st);
        else cos_partial_go<kF32, kSplitNS, kPT>(vis, anchors, B, Nv, Nt, d_bytes, KS, part, ssv, ssa, st);
    }
    return hipGetLastError();
}

hipError_t launch_cos_reduce(const float *part, const float *ssv, const float *ssa, int B, int Nv,
                             int Nt, int KS, float *M, float *rowsum, float *invn, hipStream_t st) {
    if (Nv % 4 == 0) {
        dim3 grid4((Nv + kRed4Tok - 1) / kRed4Tok, (Nt + kRedRows - 1) / kRedRows, B);
#define PV_RED4_CASE(u)                                                                             \
    case u:                                                                                         \
        hipLaunchKernelGGL(cos_reduce4_kernel<u>, grid4, dim3(256), 0, st, part, ssv, ssa, B, Nv,   \
                           Nt, KS, M, rowsum, invn);                                                \
        break;
        switch (reduce_unroll(KS)) {
            PV_RED4_CASE(1)
            PV_RED4_CASE(2)
            PV_RED4_CASE(4)
            PV_RED4_CASE(8)
            PV_RED4_CASE(16)
        }
#undef PV_RED4_CASE
        return hipGetLastError();
    }
    dim3 grid((Nv + kRedTok - 1) / kRedTok, (Nt + kRedRows - 1) / kRedRows, B);
#define PV_RED_CASE(u)                                                                             \
    case u:                                                                                        \
        hipLaunchKernelGGL(cos_reduce_kernel<u>, grid, dim3(256), 0, st, part, ssv, ssa, B, Nv, Nt, \
                           KS, M, rowsum, invn);                                                   \
        break;
    switch (reduce_unroll(KS)) {
        PV_RED_CASE(1)
        PV_RED_CASE(2)
        PV_RED_CASE(4)
        PV_RED_CASE(8)
        PV_RED_CASE(16)
    }
#undef PV_RED_CASE
    return hipGetLastError();
}

int cos_row_tiles(int Nv) { return (Nv + kRedTok - 1) / kRedTok; }
int cos_full_row_tiles(int Nv) { return (Nv + kFT - 1) / kFT; }
constexpr int kFullW = 8, kFullNS = 2;  // waves (k slices) and ring stages of cos_full

hipError_t launch_cos_full(int dt, const void *vis, const void *anchors, int B, int Nv, int Nt,
                           int d, float *M, float *rowsum, float *invn, hipStream_t st) {
    const int d_bytes = d * ((dt == kBF16) ? 2 : 4);
    const int nit = (Nt + kFT - 1) / kFT, njt = (Nv + kFT - 1) / kFT;
    const dim3 grid(B * nit * njt);
    if (dt == kBF16)
        hipLaunchKernelGGL((cos_full_kernel<kBF16, kFullW, kFullNS>), grid, dim3(64 * kFullW), 0, st,
                           (const char *)vis, (const char *)anchors, Nv, Nt, d_bytes, nit, njt, M,
                           rowsum, invn);
    else
        hipLaunchKernelGGL((cos_full_kernel<kF32, kFullW, kFullNS>), grid, dim3(64 * kFullW), 0, st,
                           (const char *)vis, (const char *)anchors, Nv, Nt, d_bytes, nit, njt, M,
                           rowsum, invn);
    return hipGetLastError();
}

hipError_t launch_center(const float *M, const float *rowsum, const int32_t *row_mask, int njt,
                         int B, int Nt, int Nv, float *p, hipStream_t st) {
    dim3 grid((Nv + kCenTok - 1) / kCenTok, B);
    hipLaunchKernelGGL(center_kernel, grid, dim3(kCenNT), 2 * (size_t)Nt * sizeof(float), st, M, rowsum,
                       row_mask, njt, Nt, Nv, p);
    return hipGetLastError();
}

hipError_t launch_select(const float *p, int B, int Nv, int budget, int32_t *kept, int32_t *pruned,
                         int32_t *slot_of, hipStream_t st) {
    if (Nv <= 256 * 4)
        hipLaunchKernelGGL((select_kernel<256, 4>), dim3(B), dim3(256), 0, st, p, Nv, budget, kept,
                           pruned, slot_of);
    else if (Nv <= 512 * 8)
        hipLaunchKernelGGL((select_kernel<512, 8>), dim3(B), dim3(512), 0, st, p, Nv, budget, kept,
                           pruned, slot_of);
    else if (Nv <= 512 * 10)  // (measured at 4608 keys: 7.4 us against 8.1 with 1024 threads)
        hipLaunchKernelGGL((select_kernel<512, 10>), dim3(B), dim3(512), 0, st, p, Nv, budget,
                           kept, pruned, slot_of);
    else if (Nv <= 1024 * 16)
        hipLaunchKernelGGL((select_kernel<1024, 16>), dim3(B), dim3(1024), 0, st, p, Nv, budget,
                           kept, pruned, slot_of);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

template <int DT>
static hipError_t gram_tile_go(const void *vis, int B, int Nv, int d, const int32_t *kept, int N1,
                               const int32_t *pruned, int Mp, const float *invn, float *best_val,
                               int32_t *best_slot, int32_t *assign, hipStream_t st) {
    const int esz = (DT == kBF16) ? 2 : 4;
    const int ntn = (N1 + kGramTileN - 1) / kGramTileN;
    const int ntm = (Mp + kGramTileM - 1) / kGramTileM;
    hipLaunchKernelGGL((gram_tile_kernel<DT, kGramTileM, kGramTileN, 4, 2, 3, kGramProducers>),
                       dim3(B * ntm * ntn), dim3(64 * (8 + kGramProducers)), 0, st,
                       (const char *)vis, Nv, d * esz, kept, N1, pruned, Mp, invn, ntm, ntn,
                       best_val, best_slot, assign);
    return hipGetLastError();
}

template <int DT, int NS, int BM, int BN>
static void gram_partial_go(const void *vis, int B, int Nv, int d_bytes, const int32_t *kept,
                            int N1, const int32_t *pruned, int Mp, int KS, float *part,
                            hipStream_t st) {
    const int ntm = (Mp + BM - 1) / BM, ntn = (N1 + BN - 1) / BN;
    hipLaunchKernelGGL((gram_partial_kernel<DT, NS, BM, BN>), dim3(B * KS * ntm * ntn), dim3(256),
                       0, st, (const char *)vis, B, Nv, d_bytes, kept, N1, pruned, Mp, ntm, ntn,
                       KS, part);
}

hipError_t launch_gram_partial(int dt, const void *vis, int B, int Nv, int d, const int32_t *kept,
                               int N1, const int32_t *pruned, int Mp, int KS, float *part,
                               bool wide, hipStream_t st) {
    const int d_bytes = d * ((dt == kBF16) ? 2 : 4);
    if (wide) {
        if (dt == kBF16)
            gram_partial_go<kBF16, 2, kGramWideM, kGramWideN>(vis, B, Nv, d_bytes, kept, N1, pruned,
                                                              Mp, KS, part, st);
        else
            gram_partial_go<kF32, 2, kGramWideM, kGramWideN>(vis, B, Nv, d_bytes, kept, N1, pruned,
                                                             Mp, KS, part, st);
    } else {
        if (dt == kBF16)
            gram_partial_go<kBF16, kSplitNS, kPT, kPT>(vis, B, Nv, d_bytes, kept, N1, pruned, Mp,
                                                       KS, part, st);
        else
            gram_partial_go<kF32, kSplitNS, kPT, kPT>(vis, B, Nv, d_bytes, kept, N1, pruned, Mp, KS,
                                                      part, st);
    }
    return hipGetLastError();
}

hipError_t launch_gram_reduce(const float *part, int B, int Mp, int N1, int Nv, int KS,
                              const float *invn, const int32_t *pruned, const int32_t *kept,
                              int32_t *assign, hipStream_t st) {
    dim3 grid((Mp + 1) / 2, B);
    const ReduceJob j{part, B, Mp, N1, Nv, KS, invn, pruned, kept, assign, 0};
#define PV_RED_CASE(u)                                                      \
    case u:                                                                 \
        hipLaunchKernelGGL(gram_reduce_kernel<u>, grid, dim3(128), 0, st, j); \
        break;
    switch (reduce_unroll(KS)) {
        PV_RED_CASE(1)
        PV_RED_CASE(2)
        PV_RED_CASE(4)
        PV_RED_CASE(8)
        PV_RED_CASE(16)
    }
#undef PV_RED_CASE
    return hipGetLastError();
}

hipError_t launch_gram_tile(int dt, const void *vis, int B, int Nv, int d, const int32_t *kept,
                            int N1, const int32_t *pruned, int Mp, const float *invn,
                            float *best_val, int32_t *best_slot, int32_t *assign, hipStream_t st) {
    if (dt == kBF16)
        return gram_tile_go<kBF16>(vis, B, Nv, d, kept, N1, pruned, Mp, invn, best_val, best_slot,
                                   assign, st);
    return gram_tile_go<kF32>(vis, B, Nv, d, kept, N1, pruned, Mp, invn, best_val, best_slot,
                              assign, st);
}

hipError_t launch_gram_finish(const float *best_val, const int32_t *best_slot, int B, int ntn,
                              int Mp, int Nv, const int32_t *pruned, int32_t *assign,
                              hipStream_t st) {
    dim3 grid((Mp + kFinNT - 1) / kFinNT, B);
    hipLaunchKernelGGL(gram_finish_kernel, grid, dim3(kFinNT), 0, st, best_val, best_slot, ntn, Mp,
                       Nv, pruned, assign);
    return hipGetLastError();
}

hipError_t launch_bucket(const int32_t *assign, int B, int Nv, int N1, int32_t *mcount,
                         int32_t *mstart, int32_t *mlist, hipStream_t st) {
    const dim3 grid((N1 + kBucketSlots - 1) / kBucketSlots, B);
    if (Nv >= kBucketWideNv)
        hipLaunchKernelGGL(bucket_kernel<1024>, grid, dim3(1024), (size_t)Nv * sizeof(int32_t), st,
                           assign, Nv, N1, mcount, mstart, mlist);
    else
        hipLaunchKernelGGL(bucket_kernel<512>, grid, dim3(512), (size_t)Nv * sizeof(int32_t), st,
                           assign, Nv, N1, mcount, mstart, mlist);
    return hipGetLastError();
}

constexpr int kMergeCPL = 2;  // chunks per lane of merge_csr

hipError_t launch_merge_csr(int dt, const void *vis, int B, int Nv, int d, int N1,
                            const int32_t *mcount, const int32_t *mstart, const int32_t *mlist,
                            void *merged, hipStream_t st) {
    const int d_bytes = d * ((dt == kBF16) ? 2 : 4);
    const int ngroups = (N1 + kBucketSlots - 1) / kBucketSlots;
    const dim3 grid((d_bytes / 16 + 64 * kMergeCPL - 1) / (64 * kMergeCPL), N1, B);
    if (dt == kBF16)
        hipLaunchKernelGGL((merge_csr_kernel<kBF16, kMergeCPL>), grid, dim3(kMergeNT), 0, st,
                           (const char *)vis, Nv, d_bytes, mcount, mstart, mlist, N1, ngroups,
                           (char *)merged);
    else
        hipLaunchKernelGGL((merge_csr_kernel<kF32, kMergeCPL>), grid, dim3(kMergeNT), 0, st,
                           (const char *)vis, Nv, d_bytes, mcount, mstart, mlist, N1, ngroups,
                           (char *)merged);
    return hipGetLastError();
}

hipError_t launch_merge(int dt, const void *vis, int B, int Nv, int d, int N1,
                        const int32_t *assign, void *merged, hipStream_t st,
                        const MergeCarry *with) {
    const int d_bytes = d * ((dt == kBF16) ? 2 : 4);
    MergeCarry mc;
    if (with) {
        mc = *with;
        if (mc.slot_of2 && (!mc.hidden2 || mc.N2 < 1)) return hipErrorInvalidValue;
    } else {
        memset(&mc, 0, sizeof(mc));
    }
    // (measured: the same work on a 1-D grid with the coordinates decoded in
    // the kernel is 15% slower at B = 1)
    const int gx = (d_bytes / 16 + 63) / 64;
    const int extra = (mc.gj.nblocks + gx - 1) / gx;  // rows of slots for the carried blocks
    const dim3 grid(gx, N1 + extra, B);
    if (dt == kBF16)
        hipLaunchKernelGGL(merge_kernel<kBF16>, grid, dim3(kMergeNT), 0, st, (const char *)vis, Nv,
                           d * 2, assign, N1, (char *)merged, mc);
    else
        hipLaunchKernelGGL(merge_kernel<kF32>, grid, dim3(kMergeNT), 0, st, (const char *)vis, Nv,
                           d * 4, assign, N1, (char *)merged, mc);
    return hipGetLastError();
}

}  // namespace pv
