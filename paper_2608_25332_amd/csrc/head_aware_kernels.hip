// Head-aware pruning at a pruning layer (Sec. 4.4, equations for S^vis and v).
//
//   v[j] = (1/(|V| Nt)) sum_{h in V} sum_i softmax_j(q_hi . k_hj / sqrt(hd))
//
// The softmax normalises along a row (over the keys) while the importance
// sums along a column (over the text rows), so there is no single-pass form:
// a row's normaliser is only known once the whole row is seen.
//
// score_partial (grid: 16-row blocks x selected heads x B, XCD ordered) keeps
// the 16 query rows of its block in registers as MFMA fragments and streams
// the head's keys from HBM/L2 straight into LDS, 64 keys per chunk.  When the chunks number at
// most MAXC the logits stay in registers between the row statistics and the
// column sums (one pass over K); otherwise the keys are streamed again in a
// second pass.  Only the selected heads are ever read and the attention map
// is never written out.  score_select (one workgroup per sample) adds the per-(head,
// row-block) column sums in a fixed order and runs the top-N_2.
#include "pv_jobs.h"
#include "pv_launch.h"
#include "pv_tile_lds.h"

#include <math.h>
#include <string.h>

namespace pv {

constexpr int kScoreNT = 256;

__device__ __forceinline__ void lse_merge(float &m, float &l, float m2, float l2) {
    const float mn = fmaxf(m, m2);
    if (mn == -INFINITY) return;  // both empty
    l = l * exp2f(m - mn) + l2 * exp2f(m2 - mn);
    m = mn;
}

// The same merge carrying the sum of squared exponentials, s = sum 2^(2(x - m)),
// which rescales by the square of the factor that rescales l.
__device__ __forceinline__ void lse_merge2(float &m, float &l, float &s, float m2, float l2,
                                           float s2) {
    const float mn = fmaxf(m, m2);
    if (mn == -INFINITY) return;
    const float a = exp2f(m - mn), c = exp2f(m2 - mn);
    l = l * a + l2 * c;
    s = s * (a * a) + s2 * (c * c);
    m = mn;
}

// Key rows are streamed through an LDS ring 64 at a time with direct-to-LDS
// loads (one CU sustains several times the bytes register loads reach), the
// next chunks in flight while the current one is multiplied; each wave takes
// one 16-key block of the chunk.  The row blocks of one head are adjacent in
// the XCD-ordered grid, so they share the head's K in one L2.
constexpr int kScoreCK = 64;     // keys per staged chunk
constexpr int kScoreFlush = 8;   // chunks of column sums held in registers
constexpr int kScoreLdsCap = 160 * 1024;

template <int NKS>
struct ScoreStage {
    static constexpr int RB = 64 * NKS;                 // bytes of one key row
    static constexpr int PPR = RB / 16;                 // 16-byte pieces per row
    static constexpr int SWZ = (NKS % 2 == 0) ? 7 : 3;  // piece swizzle within a row
    static constexpr int STAGE = kScoreCK * RB;         // bytes of one chunk
    static constexpr int IPW = STAGE / 1024 / 4;        // loads per wave per chunk
    static constexpr int NS = NKS <= 8 ? 3 : 2;         // ring stages
    static_assert(STAGE % 4096 == 0, "chunk must split evenly over the waves");
};

// Where the head of list entry hi of sample b comes from.
enum HeadSource { kHeadsArg = 0, kHeadsDevice = 1, kHeadsAll = 2 };

// CONF = false: column sums of the normalised rows (the score).  CONF = true:
// one pass only, also carrying the sum of squared probabilities of each row,
// and one number per workgroup: the sum over its rows of the row variance
// (the head confidence of this row block).

// One score workgroup; n_score: workgroups of the launch that score.
// IDX: key j of the head is row kidx[b][j] of k ([B][H][n_src][hd], the keys
// of every token; kidx[b] holds N indices), so the score needs no compacted
// copy of the kept keys; the ring is then `ext_ring` (S::NS * S::STAGE bytes
// of LDS, shared with the other workgroups of the launch).  N <= 256.
template <int DT, int NKS, int MAXC, bool CONF, bool IDX = false>
__device__ __forceinline__ void score_partial_block(
    const char *__restrict__ q, const char *__restrict__ k, const HeadArgs &heads,
    const int32_t *__restrict__ heads_dev, int head_src, const int32_t *__restrict__ row_mask,
    const float *__restrict__ row_lse, int b0, int H, int Nt, int N, int n_heads,
    float scale_log2e, float *__restrict__ partial, int cols_in_lds, int n_score,
    const int32_t *__restrict__ kidx = nullptr, int n_src = 0, char *ext_ring = nullptr) {
    static_assert(!CONF || MAXC == 0, "the confidence needs no second pass");
    static_assert(!IDX || (!CONF && MAXC > 0 && MAXC * kScoreCK <= 256),
                  "indexed keys: one pass, at most 256 keys");
    using S = ScoreStage<NKS>;
    __shared__ __attribute__((aligned(16))) char own_ring[IDX ? 16 : S::NS * S::STAGE];
    __shared__ int32_t krow[IDX ? 256 : 1];  // IDX: the source row of every key
    char *const ring = IDX ? ext_ring : own_ring;
    __shared__ __attribute__((aligned(16))) char qrows[16 * S::RB];
    __shared__ float sm_m[4][16], sm_l[4][16], sm_s[CONF ? 4 : 1][16];
    __shared__ float row_m[16], row_il[16];
    const int nrb = (Nt + 15) / 16;
    const int L = xcd_tile(blockIdx.x, n_score);
    // heads.h lists the heads of samples b0, b0 + 1, ... of this launch
    const int rb = L % nrb, hi = (L / nrb) % n_heads, bl = L / (nrb * n_heads), b = b0 + bl;
    const int tid = threadIdx.x, lane = tid & 63;
    // uniform wave index: the block guards around the MFMAs become scalar
    // branches (an MFMA does not honour the execution mask)
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    int h;
    if (head_src == kHeadsAll) h = hi;
    else if (head_src == kHeadsDevice) h = min(max(heads_dev[(size_t)b * n_heads + hi], 0), H - 1);
    else h = heads.h[bl * n_heads + hi];
    const char *qb = q + ((size_t)b * H + h) * Nt * S::RB;
    const char *kb = k + ((size_t)b * H + h) * (IDX ? n_src : N) * S::RB;
    if constexpr (IDX) {
        // ordinary loads, all retired at the barrier: the ring's loads below
        // are then the only ones in flight (see the ordering note)
        for (int j = tid; j < N; j += kScoreNT)
            krow[j] = min(max(kidx[(size_t)b * N + j], 0), n_src - 1);
        __syncthreads();
    }

    const int nch = (N + kScoreCK - 1) / kScoreCK;
    uint4 qf[NKS];  // the 16 query rows as MFMA fragments

    // this lane's source key row and piece for each of its loads of a chunk
    int srow[S::IPW], sbyte[S::IPW];
#pragma unroll
    for (int t = 0; t < S::IPW; ++t) {
        const int pos = (wave * S::IPW + t) * 64 + lane;
        const int r = pos / S::PPR, slot = pos % S::PPR;
        srow[t] = r;
        sbyte[t] = (slot ^ (r & S::SWZ)) << 4;
    }
    auto issue = [&](int ch) {
        char *dst = ring + (ch % S::NS) * S::STAGE + wave * S::IPW * 1024;
#pragma unroll
        for (int t = 0; t < S::IPW; ++t) {
            const int key = min(ch * kScoreCK + srow[t], N - 1);  // past the end: last key
            const int row = IDX ? krow[key] : key;
            lds_dma16(kb + (size_t)row * S::RB + sbyte[t], dst + t * 1024);
        }
    };
    // Every global load of the kernel is a direct-to-LDS load, and those
    // retire in the order they were issued, so a partial wait on the load
    // counter names exactly the chunks still in flight.  (With ordinary
    // loads or stores outstanding as well no such guarantee holds: the query
    // rows go through LDS for that reason, and stores wait for a full drain.)
    //
    // The query block (16 rows, NKS KiB) is loaded once, 1 KiB per load,
    // spread over the waves; it is issued before the first key chunk, so
    // waiting for chunk 0 waits for it too.
    auto issue_q = [&]() {
        for (int p = wave; p < NKS; p += 4) {
            const int off = p * 1024 + lane * 16;
            const int r = off / S::RB, slot = (off % S::RB) >> 4;
            // the keys' piece swizzle, so the fragment reads spread over the banks
            lds_dma16(qb + (size_t)min(rb * 16 + r, Nt - 1) * S::RB + ((slot ^ (r & S::SWZ)) << 4),
                      qrows + p * 1024);
        }
    };
    // A pass over the keys: start() fills the whole ring (no buffer is reused
    // before chunk NS); chunk(ch) waits for chunk ch, refills the buffer freed
    // by chunk ch - 1 and returns this wave's 16 x 16 logit block (query rows
    // x keys wave*16 .. wave*16+15 of the chunk); finish() lets the ring be
    // refilled by a later pass.
    auto start = [&]() {
#pragma unroll
        for (int pp = 0; pp < S::NS; ++pp)
            if (pp < nch) issue(pp);
    };
    // the query fragments, once the first wait has covered their loads
    auto read_q = [&]() {
#pragma unroll
        for (int s = 0; s < NKS; ++s)
            qf[s] = lds_read16(qrows + (lane & 15) * S::RB +
                               (((s * 4 + (lane >> 4)) ^ ((lane & 15) & S::SWZ)) << 4));
        lds_wait();
#pragma unroll
        for (int s = 0; s < NKS; ++s) lds_after_wait(qf[s]);
    };
    auto chunk = [&](int ch, bool drain) -> f32x4_t {
        // chunks issued so far, and how many of them are younger than ch
        const int issued = ch == 0 ? min(S::NS, nch) : min(ch + S::NS - 1, nch);
        const int younger = drain ? 0 : issued - 1 - ch;
        static_assert(S::NS <= 3, "at most two chunks younger than the one waited for");
        if (younger >= 2) wait_vmcnt<S::IPW * 2>();
        else if (younger == 1) wait_vmcnt<S::IPW>();
        else wait_vmcnt<0>();
        bare_barrier();  // chunk ch is in LDS; chunk ch - 1 has been read
        if (ch >= 1 && ch + S::NS - 1 < nch) issue(ch + S::NS - 1);
        if (ch == 0) read_q();
        const char *sp = ring + (ch % S::NS) * S::STAGE;
        const int r = wave * 16 + (lane & 15);
        uint4 kf[NKS];
#pragma unroll
        for (int s = 0; s < NKS; ++s) {
            const int piece = s * 4 + (lane >> 4);
            kf[s] = lds_read16(sp + r * S::RB + ((piece ^ (r & S::SWZ)) << 4));
        }
        lds_wait();
        f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < NKS; ++s) {
            lds_after_wait(kf[s]);
            acc = mma16<DT>(qf[s], kf[s], acc);
        }
        return acc;
    };
    auto finish = [&]() { bare_barrier(); };

    // pass 1: running (max, sum of exp) of the logits, per lane and row; with
    // MAXC > 0 the logit blocks also stay in registers for pass 2
    float m[4], l[4], sq[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        m[i] = -INFINITY;
        l[i] = 0.f;
        sq[i] = 0.f;
    }
    auto stats = [&](const f32x4_t &acc, int ch) {
        if (ch * kScoreCK + wave * 16 + (lane & 15) < N) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                if (CONF) lse_merge2(m[i], l[i], sq[i], acc[i] * scale_log2e, 1.f, 1.f);
                else lse_merge(m[i], l[i], acc[i] * scale_log2e, 1.f);
            }
        }
    };
    f32x4_t keep[MAXC > 0 ? MAXC : 1];
    issue_q();
    start();
    if constexpr (MAXC > 0) {
        // unrolled with constant indices (nch is uniform): each block stays
        // in its own registers; the statistics come after the last chunk
#pragma unroll
        for (int ch = 0; ch < MAXC; ++ch)
            if (ch < nch) keep[ch] = chunk(ch, false);
    } else {
        for (int ch = 0; ch < nch; ++ch) stats(chunk(ch, false), ch);
    }
    finish();
    if constexpr (MAXC > 0 && !CONF) {
        // Every logit at hand: the row maximum first (lanes, then waves),
        // then one exponential per logit, kept in place, and the row sums.
        // Keys past N are left out of both.
#pragma unroll
        for (int ch = 0; ch < MAXC; ++ch) {
            if (ch < nch) {
                if ((ch + 1) * kScoreCK > N) {  // the only chunk that can hold keys past N
                    const bool col_ok = ch * kScoreCK + wave * 16 + (lane & 15) < N;
#pragma unroll
                    for (int i = 0; i < 4; ++i) keep[ch][i] = col_ok ? keep[ch][i] : -INFINITY;
                }
#pragma unroll
                for (int i = 0; i < 4; ++i) m[i] = fmaxf(m[i], keep[ch][i]);
            }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) m[i] = row16_max(m[i]);
        if ((lane & 15) == 0)
#pragma unroll
            for (int i = 0; i < 4; ++i) sm_m[wave][(lane >> 4) * 4 + i] = m[i];
        __syncthreads();
        // the row maximum of the scaled logits (scaling by a positive factor
        // and rounding keep the order, so it is the scaled maximum)
        if (tid < 16)
            row_m[tid] = fmaxf(fmaxf(sm_m[0][tid], sm_m[1][tid]), fmaxf(sm_m[2][tid], sm_m[3][tid])) *
                         scale_log2e;
        __syncthreads();
        float rmx[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) rmx[i] = row_m[(lane >> 4) * 4 + i];
#pragma unroll
        for (int ch = 0; ch < MAXC; ++ch) {
            if (ch < nch) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float e = exp2_hw(fmaf(keep[ch][i], scale_log2e, -rmx[i]));  // 0 past N
                    keep[ch][i] = e;
                    l[i] += e;
                }
            }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) l[i] = row16_sum(l[i]);
        if ((lane & 15) == 0)
#pragma unroll
            for (int i = 0; i < 4; ++i) sm_l[wave][(lane >> 4) * 4 + i] = l[i];
        __syncthreads();
        if (tid < 16) {
            float ll = ((sm_l[0][tid] + sm_l[1][tid]) + sm_l[2][tid]) + sm_l[3][tid];
            // the non-visual keys join the normaliser on the scale of the
            // kept exponentials (relative to the row maximum)
            if (row_lse) {
                const float t = row_lse[((size_t)b * H + h) * Nt + min(rb * 16 + tid, Nt - 1)];
                ll += exp2_hw(t * 1.4426950408889634f - row_m[tid]);
            }
            row_il[tid] = (rb * 16 + tid < Nt) ? 1.0f / ll : 0.f;  // masked rows add nothing
        }
        __syncthreads();
        float rl[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) rl[i] = row_il[(lane >> 4) * 4 + i];
        float *outp = partial + (((size_t)b * n_heads + hi) * nrb + rb) * N;
#pragma unroll
        for (int ch = 0; ch < MAXC; ++ch) {
            if (ch < nch) {
                float cs = 0.f;
#pragma unroll
                for (int i = 0; i < 4; ++i) cs += keep[ch][i] * rl[i];
                cs += __shfl_xor(cs, 16, 64);
                cs += __shfl_xor(cs, 32, 64);
                const int col = ch * kScoreCK + wave * 16 + (lane & 15);
                if (lane < 16 && col < N) outp[col] = cs;
            }
        }
        return;
    }
    // combine the 16 lanes that hold the same rows (DPP partners of an xor
    // butterfly over 1, 2, 4, 8; both lanes of a pair compute the same merge,
    // so the pairing gives the butterfly's bits), then the 4 waves
    auto merge_step = [&](auto xch) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float m2 = xch(m[i]), l2 = xch(l[i]);
            if (CONF) {
                const float s2 = xch(sq[i]);
                lse_merge2(m[i], l[i], sq[i], m2, l2, s2);
            } else {
                lse_merge(m[i], l[i], m2, l2);
            }
        }
    };
    merge_step([](float x) { return dpp_f32<0xB1>(x); });
    merge_step([](float x) { return dpp_f32<0x4E>(x); });
    merge_step([](float x) { return dpp_f32<0x141>(x); });
    merge_step([](float x) { return dpp_f32<0x140>(x); });
    if ((lane & 15) == 0) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            sm_m[wave][(lane >> 4) * 4 + i] = m[i];
            sm_l[wave][(lane >> 4) * 4 + i] = l[i];
            if (CONF) sm_s[CONF ? wave : 0][(lane >> 4) * 4 + i] = sq[i];
        }
    }
    __syncthreads();
    if constexpr (CONF) {
        // rows outside row_mask add nothing (an empty mask means every row)
        __shared__ int any_row;
        if (row_mask) {
            if (tid == 0) any_row = 0;
            __syncthreads();
            for (int i = tid; i < Nt; i += kScoreNT)
                if (row_mask[(size_t)b * Nt + i] != 0) any_row = 1;
            __syncthreads();
        }
        // Var_j(A[i][j]) = (sum_j A^2 - S^2 / N) / N over the N visual keys,
        // with D the row's normaliser, S = l / D its visual mass and
        // sum_j A^2 = s / D^2.  Over the visual keys alone D = l and S = 1;
        // on the model's domain the other keys join D through their
        // log-sum-exp (row_lse, natural log of the scaled logits), on the
        // scale of the kept exponentials (relative to the row maximum).  The
        // 16 rows are added in order (rows past Nt add nothing).
        if (tid < 16) {
            float mm = sm_m[0][tid], ll = sm_l[0][tid], ss = sm_s[0][tid];
#pragma unroll
            for (int w = 1; w < 4; ++w) lse_merge2(mm, ll, ss, sm_m[w][tid], sm_l[w][tid], sm_s[w][tid]);
            const float inv_n = 1.0f / (float)N;
            const int i = rb * 16 + tid;
            const bool use = i < Nt && (!row_mask || !any_row || row_mask[(size_t)b * Nt + i] != 0);
            float den = ll;
            if (row_lse) {
                const float t = row_lse[((size_t)b * H + h) * Nt + min(i, Nt - 1)] * 1.4426950408889634f;
                den = ll + exp2_hw(t - mm);  // an overflow means the visual mass is 0 in fp32
            }
            const float mass = ll / den;
            row_m[tid] = use ? (ss / (den * den) - mass * mass * inv_n) * inv_n : 0.f;
        }
        __syncthreads();
        if (tid == 0) {
            float c = 0.f;
            for (int r = 0; r < 16; ++r) c += row_m[r];
            partial[((size_t)b * H + h) * nrb + rb] = c;
        }
        return;
    }
    if (tid < 16) {
        float mm = sm_m[0][tid], ll = sm_l[0][tid];
#pragma unroll
        for (int w = 1; w < 4; ++w) lse_merge(mm, ll, sm_m[w][tid], sm_l[w][tid]);
        // the model's row also runs over the non-visual keys: their
        // log-sum-exp (natural log, scaled logits) joins the normaliser
        if (row_lse) {
            const float t = row_lse[((size_t)b * H + h) * Nt + min(rb * 16 + tid, Nt - 1)];
            lse_merge(mm, ll, t * 1.4426950408889634f, 1.f);
        }
        row_m[tid] = mm;
        row_il[tid] = (rb * 16 + tid < Nt) ? 1.0f / ll : 0.f;  // masked rows add nothing
    }
    __syncthreads();

    float rm[4], ril[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        rm[i] = row_m[(lane >> 4) * 4 + i];
        ril[i] = row_il[(lane >> 4) * 4 + i];
    }
    float *out = partial + (((size_t)b * n_heads + hi) * nrb + rb) * N;
    // pass 2 (keys streamed again): normalised probabilities, summed over the
    // 16 rows of each column
    if constexpr (MAXC == 0) {
        // Stores must not be in flight at a partial wait (see chunk()): the
        // column sums go to LDS while the keys stream and to memory after
        // the pass, or, where N of them do not fit beside the ring, are held
        // in registers kScoreFlush chunks at a time and stored, the next
        // chunk then waiting for everything.
        extern __shared__ float colsum[];  // [N] when cols_in_lds
        float pend[kScoreFlush];
#pragma unroll
        for (int u = 0; u < kScoreFlush; ++u) pend[u] = 0.f;
        start();
        for (int ch = 0; ch < nch; ++ch) {
            const bool after_flush = !cols_in_lds && ch > 0 && ch % kScoreFlush == 0;
            const f32x4_t acc = chunk(ch, after_flush);
            float cs = 0.f;
#pragma unroll
            for (int i = 0; i < 4; ++i) cs += exp2f(acc[i] * scale_log2e - rm[i]) * ril[i];
            cs += __shfl_xor(cs, 16, 64);
            cs += __shfl_xor(cs, 32, 64);
            const int col = ch * kScoreCK + wave * 16 + (lane & 15);
            if (cols_in_lds) {
                if (lane < 16 && col < N) colsum[col] = cs;
            } else {
                const int u0 = ch % kScoreFlush;
#pragma unroll
                for (int u = 0; u < kScoreFlush; ++u) pend[u] = (u == u0) ? cs : pend[u];
                if (u0 == kScoreFlush - 1 || ch == nch - 1) {
                    const int c0 = ch - u0;
#pragma unroll
                    for (int u = 0; u < kScoreFlush; ++u) {
                        const int cu = (c0 + u) * kScoreCK + wave * 16 + (lane & 15);
                        if (u <= u0 && lane < 16 && cu < N) out[cu] = pend[u];
                    }
                }
            }
        }
        finish();
        if (cols_in_lds)
            for (int c = tid; c < N; c += kScoreNT) out[c] = colsum[c];
    }
}

template <int DT, int NKS, int MAXC, bool CONF>
__global__ __launch_bounds__(kScoreNT) void score_partial_kernel(
    const char *__restrict__ q, const char *__restrict__ k, HeadArgs heads,
    const int32_t *__restrict__ heads_dev, int head_src, const int32_t *__restrict__ row_mask,
    const float *__restrict__ row_lse, int b0, int H, int Nt, int N, int n_heads,
    float scale_log2e, float *__restrict__ partial, int cols_in_lds) {
    score_partial_block<DT, NKS, MAXC, CONF>(q, k, heads, heads_dev, head_src, row_mask, row_lse,
                                             b0, H, Nt, N, n_heads, scale_log2e, partial,
                                             cols_in_lds, gridDim.x);
}

// ----------------------------------------------------------------------------
// score_head: one workgroup per (selected head, sample), for up to 64 text
// rows and 256 keys (the shapes of the paper's layers).  Wave w owns text
// rows 16 w .. 16 w + 15 for every key, so its row statistics need no
// exchange with the other waves, and the head's keys are read into LDS once
// for all rows (score_partial reads them once per 16-row block).  The query
// block and the (at most four) key chunks are all issued at the start; the
// logits stay in registers; the four waves' column sums meet in LDS and are
// added in wave order.  Writes one row of column sums per (sample, head).
// ----------------------------------------------------------------------------
constexpr int kHeadMaxRows = 64;
constexpr int kHeadMaxChunks = 4;

// Row statistics of one wave's 16 rows with every raw logit at hand
// (keep[ch][kq][i]: row 4 (lane / 16) + i, key 64 ch + 16 kq + lane % 16):
// keys past N become -inf (only the last chunk can hold them), then m[i] =
// the row maximum, scaled (scaling by a positive factor and rounding keep the
// order, so it is the maximum of the scaled logits).
template <int MAXC>
__device__ __forceinline__ void head_row_max(f32x4_t (&keep)[MAXC][4], int nch, int N, int lane,
                                             float scale_log2e, float (&m)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) m[i] = -INFINITY;
#pragma unroll
    for (int ch = 0; ch < MAXC; ++ch) {
        if (ch < nch) {
            if ((ch + 1) * kScoreCK > N) {
#pragma unroll
                for (int kq = 0; kq < 4; ++kq) {
                    const bool col_ok = ch * kScoreCK + kq * 16 + (lane & 15) < N;
#pragma unroll
                    for (int i = 0; i < 4; ++i) keep[ch][kq][i] = col_ok ? keep[ch][kq][i] : -INFINITY;
                }
            }
#pragma unroll
            for (int kq = 0; kq < 4; ++kq)
#pragma unroll
                for (int i = 0; i < 4; ++i) m[i] = fmaxf(m[i], keep[ch][kq][i]);
        }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) m[i] = row16_max(m[i]) * scale_log2e;
}

// keep <- 2^(scaled logit - m) in place, l[i] += them in (chunk, block) order
// (0 for keys past N); the row sums over the lanes follow.
template <int MAXC>
__device__ __forceinline__ void head_row_exp(f32x4_t (&keep)[MAXC][4], int nch, float scale_log2e,
                                             const float (&m)[4], float (&l)[4]) {
#pragma unroll
    for (int ch = 0; ch < MAXC; ++ch) {
        if (ch < nch) {
#pragma unroll
            for (int kq = 0; kq < 4; ++kq) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float e = exp2_hw(fmaf(keep[ch][kq][i], scale_log2e, -m[i]));
                    keep[ch][kq][i] = e;
                    l[i] += e;
                }
            }
        }
    }
}

// Logits of one wave's 16 query rows (fragments qf) against the 64 keys of a
// staged chunk: out[kq] = rows x keys 16 kq .. 16 kq + 15.  Every fragment of
// the chunk is read before the first MFMA, and the MFMAs go window by window
// across the four key blocks, so that four independent accumulations
// alternate on the matrix core instead of one chain waiting on itself; each
// block's sum still runs over the windows in order.
template <int DT, int NKS>
__device__ __forceinline__ void head_chunk_logits(const char *kb, const uint4 (&qf)[NKS], int lane,
                                                  f32x4_t (&out)[4]) {
    using S = ScoreStage<NKS>;
    uint4 kf[4][NKS];
#pragma unroll
    for (int kq = 0; kq < 4; ++kq) {
        const int r = kq * 16 + (lane & 15);
#pragma unroll
        for (int s = 0; s < NKS; ++s) {
            const int piece = s * 4 + (lane >> 4);
            kf[kq][s] = lds_read16(kb + r * S::RB + ((piece ^ (r & S::SWZ)) << 4));
        }
    }
    lds_wait();
#pragma unroll
    for (int kq = 0; kq < 4; ++kq) {
        out[kq] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < NKS; ++s) lds_after_wait(kf[kq][s]);
    }
#pragma unroll
    for (int s = 0; s < NKS; ++s)
#pragma unroll
        for (int kq = 0; kq < 4; ++kq) out[kq] = mma16<DT>(qf[s], kf[kq][s], out[kq]);
}

template <int DT, int NKS>
__global__ __launch_bounds__(kScoreNT) void score_head_kernel(
    const char *__restrict__ q, const char *__restrict__ k, HeadArgs8 heads,
    const int32_t *__restrict__ heads_dev, int head_src, const float *__restrict__ row_lse, int b0,
    int H, int Nt, int N, int n_heads, float scale_log2e, float *__restrict__ partial) {
    using S = ScoreStage<NKS>;
    constexpr int MAXC = kHeadMaxChunks;
    // the key chunks in dynamic LDS, nch of them (so that three workgroups
    // fit on a CU for 192 keys)
    extern __shared__ __attribute__((aligned(16))) char kdyn[];
    auto kbuf = [&](int ch) { return kdyn + ch * S::STAGE; };
    __shared__ float colpart[4][MAXC * kScoreCK];
    const int L = blockIdx.x;
    const int hi = L % n_heads, bl = L / n_heads, b = b0 + bl;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    int h;
    if (head_src == kHeadsDevice) h = min(max(heads_dev[(size_t)b * n_heads + hi], 0), H - 1);
    else {
        const int e = bl * n_heads + hi;
        h = (int)((heads.w[e >> 2] >> ((e & 3) * 8)) & 0xFFu);
    }
    const char *qb = q + ((size_t)b * H + h) * Nt * S::RB;
    const char *kb = k + ((size_t)b * H + h) * N * S::RB;
    const int nch = (N + kScoreCK - 1) / kScoreCK;  // <= MAXC (host-checked)

    // every load of the kernel is issued up front: this wave's query rows
    // straight into MFMA fragments (rows past Nt repeat the last one; the
    // wave's 16 rows are one contiguous block), then each key chunk
    // direct-to-LDS.  Keeping the query rows out of LDS is what lets a third
    // workgroup onto a CU.
    const bool rows_live = wave * 16 < Nt;  // uniform: this wave has rows to score
    uint4 qf[NKS];
    if (rows_live) {
        const char *qrow = qb + (size_t)min(wave * 16 + (lane & 15), Nt - 1) * S::RB;
#pragma unroll
        for (int s = 0; s < NKS; ++s) qf[s] = ld16(qrow + ((s * 4 + (lane >> 4)) << 4));
    }
#pragma unroll
    for (int ch = 0; ch < MAXC; ++ch) {
        if (ch < nch) {
#pragma unroll
            for (int t = 0; t < S::IPW; ++t) {
                const int pos = (wave * S::IPW + t) * 64 + lane;
                const int r = pos / S::PPR, slot = pos % S::PPR;
                const int row = min(ch * kScoreCK + r, N - 1);  // past the end: last key
                lds_dma16(kb + (size_t)row * S::RB + ((slot ^ (r & S::SWZ)) << 4),
                          kbuf(ch) + (wave * S::IPW + t) * 1024);
            }
        }
    }
    wait_vmcnt<0>();
    bare_barrier();

    // logits of this wave's 16 rows x every key: lane holds rows
    // 4 (lane / 16) + i of column (lane % 16) of each 16-key block
    f32x4_t keep[MAXC][4];
    if (rows_live) {
#pragma unroll
        for (int ch = 0; ch < MAXC; ++ch)
            if (ch < nch) head_chunk_logits<DT, NKS>(kbuf(ch), qf, lane, keep[ch]);
    }
    // Row statistics with every logit at hand: the row maximum first, then
    // one exponential per logit (kept in place of it) and their sum.  Keys
    // past N are left out of both.
    float m[4], il[4];
    if (rows_live) head_row_max<MAXC>(keep, nch, N, lane, scale_log2e, m);
    float l[4] = {0.f, 0.f, 0.f, 0.f};
    if (rows_live) {
        head_row_exp<MAXC>(keep, nch, scale_log2e, m, l);
#pragma unroll
        for (int i = 0; i < 4; ++i) l[i] = row16_sum(l[i]);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int row = wave * 16 + (lane >> 4) * 4 + i;
        float mm = m[i], ll = l[i];
        if (rows_live && row_lse) {
            // the non-visual keys join the normaliser on the scale of the
            // kept exponentials (relative to m; an overflow only means the
            // row's visual mass is 0 in fp32)
            const float t = row_lse[((size_t)b * H + h) * Nt + min(row, Nt - 1)] * 1.4426950408889634f;
            ll += exp2_hw(t - mm);
        }
        il[i] = (rows_live && row < Nt) ? 1.0f / ll : 0.f;  // masked rows add nothing
    }
    // this wave's column sums over its 16 rows, chunk by chunk
#pragma unroll
    for (int ch = 0; ch < MAXC; ++ch) {
        if (ch < nch) {
#pragma unroll
            for (int kq = 0; kq < 4; ++kq) {
                float cs = 0.f;
                if (rows_live) {
#pragma unroll
                    for (int i = 0; i < 4; ++i) cs += keep[ch][kq][i] * il[i];
                }
                cs += __shfl_xor(cs, 16, 64);
                cs += __shfl_xor(cs, 32, 64);
                if (lane < 16) colpart[wave][ch * kScoreCK + kq * 16 + lane] = cs;
            }
        }
    }
    __syncthreads();
    float *out = partial + ((size_t)b * n_heads + hi) * N;
    for (int j = tid; j < N; j += kScoreNT)
        out[j] = ((colpart[0][j] + colpart[1][j]) + colpart[2][j]) + colpart[3][j];
}

// ----------------------------------------------------------------------------
// score_split: long key lists on few (head, sample) pairs (the hi-res and 13B
// shapes), where one workgroup per 16-row block would re-read each head's
// keys once per block and leave most CUs idle.  A workgroup owns one
// (64-key chunk, selected head, sample) and every text row, in XCD order so
// that the chunks of one head share its query rows in one L2.
//   score_split_stats: each row's maximum and sum of exponentials over the
//       chunk's keys -> stats[b][hi][chunk][row] (max in scaled log2 units,
//       sum relative to it);
//   score_split_cols: every row's statistics merged over the chunks in chunk
//       order (with the non-visual keys' log-sum-exp on the model's domain),
//       the chunk's logits formed again, and the normalised probabilities
//       summed over the rows -> partial[b][hi][key], the layout of the
//       whole-head form.
// Each pass reads the keys once; the attention map is never written.  The
// chunk's keys go to LDS once; each wave takes 16 rows of a 64-row block at
// a time, its query fragments loaded straight into registers.
// ----------------------------------------------------------------------------
constexpr int kSplitRowsPerPass = 64;  // rows of one pass of the four waves

// The (chunk, head, sample) of this workgroup and the head it reads.
struct SplitCoord {
    int s, hi, b, h;
};

__device__ __forceinline__ SplitCoord split_coord(const HeadArgs &heads,
                                                  const int32_t *__restrict__ heads_dev,
                                                  int head_src, int b0, int H, int nsplit,
                                                  int n_heads) {
    SplitCoord c;
    const int L = xcd_tile(blockIdx.x, gridDim.x);
    c.s = L % nsplit;
    c.hi = (L / nsplit) % n_heads;
    const int bl = L / (nsplit * n_heads);
    c.b = b0 + bl;
    if (head_src == kHeadsDevice) c.h = min(max(heads_dev[(size_t)c.b * n_heads + c.hi], 0), H - 1);
    else c.h = heads.h[bl * n_heads + c.hi];
    return c;
}

// The chunk's (at most 64) keys into LDS (rows past N repeat the last key).
template <int NKS>
__device__ __forceinline__ void split_load_keys(const char *kb, int key0, int N, char *kbuf,
                                                int wave, int lane) {
    using S = ScoreStage<NKS>;
#pragma unroll
    for (int t = 0; t < S::IPW; ++t) {
        const int pos = (wave * S::IPW + t) * 64 + lane;
        const int r = pos / S::PPR, slot = pos % S::PPR;
        const int row = min(key0 + r, N - 1);
        lds_dma16(kb + (size_t)row * S::RB + ((slot ^ (r & S::SWZ)) << 4),
                  kbuf + (wave * S::IPW + t) * 1024);
    }
    wait_vmcnt<0>();
    bare_barrier();
}

// Logits of this wave's 16 rows starting at r0 against the chunk:
// keep[0][kq] = rows 4 (lane / 16) + i x keys 16 kq + lane % 16.
template <int DT, int NKS>
__device__ __forceinline__ void split_logits(const char *qb, int r0, int Nt, const char *kbuf,
                                             int lane, f32x4_t (&keep)[1][4]) {
    using S = ScoreStage<NKS>;
    uint4 qf[NKS];
    const char *qrow = qb + (size_t)min(r0 + (lane & 15), Nt - 1) * S::RB;
#pragma unroll
    for (int s = 0; s < NKS; ++s) qf[s] = ld16(qrow + ((s * 4 + (lane >> 4)) << 4));
    head_chunk_logits<DT, NKS>(kbuf, qf, lane, keep[0]);
}

template <int DT, int NKS>
__global__ __launch_bounds__(kScoreNT) void score_split_stats_kernel(
    const char *__restrict__ q, const char *__restrict__ k, HeadArgs heads,
    const int32_t *__restrict__ heads_dev, int head_src, int b0, int H, int Nt, int N,
    int n_heads, int nsplit, float scale_log2e, float2 *__restrict__ stats) {
    using S = ScoreStage<NKS>;
    __shared__ __attribute__((aligned(16))) char kbuf[S::STAGE];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const SplitCoord c = split_coord(heads, heads_dev, head_src, b0, H, nsplit, n_heads);
    const char *qb = q + ((size_t)c.b * H + c.h) * Nt * S::RB;
    const char *kb = k + ((size_t)c.b * H + c.h) * N * S::RB;
    const int key0 = c.s * kScoreCK;
    split_load_keys<NKS>(kb, key0, N, kbuf, wave, lane);
    float2 *out = stats + (((size_t)c.b * n_heads + c.hi) * nsplit + c.s) * Nt;
    for (int r0 = wave * 16; r0 < Nt; r0 += kSplitRowsPerPass) {  // uniform per wave
        f32x4_t keep[1][4];
        split_logits<DT, NKS>(qb, r0, Nt, kbuf, lane, keep);
        float m[4], l[4] = {0.f, 0.f, 0.f, 0.f};
        head_row_max<1>(keep, 1, N - key0, lane, scale_log2e, m);  // keys past N left out
        head_row_exp<1>(keep, 1, scale_log2e, m, l);
#pragma unroll
        for (int i = 0; i < 4; ++i) l[i] = row16_sum(l[i]);
        if ((lane & 15) == 0) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int row = r0 + (lane >> 4) * 4 + i;
                if (row < Nt) out[row] = make_float2(m[i], l[i]);
            }
        }
    }
}

constexpr int kSplitStatU = 8;  // chunk statistics in flight per row

template <int DT, int NKS>
__global__ __launch_bounds__(kScoreNT) void score_split_cols_kernel(
    const char *__restrict__ q, const char *__restrict__ k, HeadArgs heads,
    const int32_t *__restrict__ heads_dev, int head_src, const float *__restrict__ row_lse,
    int b0, int H, int Nt, int N, int n_heads, int nsplit, float scale_log2e,
    const float2 *__restrict__ stats, float *__restrict__ partial) {
    using S = ScoreStage<NKS>;
    __shared__ __attribute__((aligned(16))) char kbuf[S::STAGE];
    __shared__ float colpart[4][kScoreCK];
    extern __shared__ float2 rowstat[];  // [Nt]: (row maximum, 1 / normaliser)
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const SplitCoord c = split_coord(heads, heads_dev, head_src, b0, H, nsplit, n_heads);
    const char *qb = q + ((size_t)c.b * H + c.h) * Nt * S::RB;
    const char *kb = k + ((size_t)c.b * H + c.h) * N * S::RB;
    const int key0 = c.s * kScoreCK;
    // the keys' loads first; the rows' statistics are merged while they fly
    {
#pragma unroll
        for (int t = 0; t < S::IPW; ++t) {
            const int pos = (wave * S::IPW + t) * 64 + lane;
            const int r = pos / S::PPR, slot = pos % S::PPR;
            const int row = min(key0 + r, N - 1);
            lds_dma16(kb + (size_t)row * S::RB + ((slot ^ (r & S::SWZ)) << 4),
                      kbuf + (wave * S::IPW + t) * 1024);
        }
    }
    // every row's statistics over all chunks, merged in chunk order
    const float2 *st = stats + ((size_t)c.b * n_heads + c.hi) * nsplit * Nt;
    for (int row = tid; row < Nt; row += kScoreNT) {
        float mm = -INFINITY, ll = 0.f;
        for (int s0 = 0; s0 < nsplit; s0 += kSplitStatU) {
            float2 v[kSplitStatU];
#pragma unroll
            for (int u = 0; u < kSplitStatU; ++u)
                v[u] = st[(size_t)min(s0 + u, nsplit - 1) * Nt + row];
#pragma unroll
            for (int u = 0; u < kSplitStatU; ++u)
                if (s0 + u < nsplit) lse_merge(mm, ll, v[u].x, v[u].y);
        }
        // the model's row also runs over the non-visual keys: their
        // log-sum-exp (natural log, scaled logits) joins the normaliser
        if (row_lse) lse_merge(mm, ll, row_lse[((size_t)c.b * H + c.h) * Nt + row] * 1.4426950408889634f, 1.f);
        rowstat[row] = make_float2(mm, 1.0f / ll);
    }
    wait_vmcnt<0>();
    __syncthreads();  // the keys and every row's statistics are in LDS
    float cs[4] = {0.f, 0.f, 0.f, 0.f};
    const int nkeys = N - key0;
    for (int r0 = wave * 16; r0 < Nt; r0 += kSplitRowsPerPass) {  // uniform per wave
        f32x4_t keep[1][4];
        split_logits<DT, NKS>(qb, r0, Nt, kbuf, lane, keep);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int row = r0 + (lane >> 4) * 4 + i;
            const float2 rs = rowstat[min(row, Nt - 1)];
            const float il = row < Nt ? rs.y : 0.f;  // rows past Nt add nothing
#pragma unroll
            for (int kq = 0; kq < 4; ++kq) {
                const bool col_ok = kq * 16 + (lane & 15) < nkeys;
                const float e = exp2_hw(fmaf(keep[0][kq][i], scale_log2e, -rs.x));
                cs[kq] += col_ok ? e * il : 0.f;
            }
        }
    }
    // this wave's column sums over its rows, then the four waves in order
#pragma unroll
    for (int kq = 0; kq < 4; ++kq) {
        float v = cs[kq];
        v += __shfl_xor(v, 16, 64);
        v += __shfl_xor(v, 32, 64);
        if (lane < 16) colpart[wave][kq * 16 + lane] = v;
    }
    __syncthreads();
    if (tid < kScoreCK && tid < nkeys)
        partial[((size_t)c.b * n_heads + c.hi) * N + key0 + tid] =
            ((colpart[0][tid] + colpart[1][tid]) + colpart[2][tid]) + colpart[3][tid];
}

template <int NT, int EMAX>
__global__ __launch_bounds__(NT) void score_select_kernel(SelectJob sj) {
    score_select_block<NT, EMAX>(sj, blockIdx.x);
}

// The head lists travel as a kernel argument of bounded size: a launch covers
// as many samples as fit, and larger batches take several launches.
struct ScoreLaunch {
    const void *q, *k;
    const int32_t *heads_host;  // kHeadsArg: host list [B][n_heads]
    const int32_t *heads_dev;   // kHeadsDevice: device list [B][n_heads]
    int src;
    const int32_t *row_mask;    // confidence only: rows summed (may be NULL)
    const float *row_lse;       // [B][H][Nt] non-visual log-sum-exp (may be NULL)
    int B, H, Nt, N, n_heads;
    float sl2e;
    float *partial;
    hipStream_t st;
    int hd_scale = 0;  // head width of the attention scale (0: the row width)
};

// A host head list travels as a kernel argument of bounded size: a launch
// covers as many samples as fit, and larger batches take several launches.
// Device lists and the all-heads form need one launch.
template <int DT, int NKS, int MAXC, bool CONF>
static hipError_t score_go(const ScoreLaunch &a) {
    using S = ScoreStage<NKS>;
    // two-pass form: the N column sums in dynamic LDS when they fit beside
    // the ring and the row statistics (at most 64 KiB of it)
    const size_t cols = (size_t)a.N * sizeof(float);
    const bool in_lds = !CONF && MAXC == 0 && cols <= 65536 &&
                        (size_t)S::NS * S::STAGE + 16 * S::RB + 1024 + cols <= (size_t)kScoreLdsCap;
    const int nrb = (a.Nt + 15) / 16;
    const int per_launch = a.src == kHeadsArg ? kMaxHeadArgs / a.n_heads : a.B;
    HeadArgs ha;
    for (int b0 = 0; b0 < a.B; b0 += per_launch) {
        const int nb = a.B - b0 < per_launch ? a.B - b0 : per_launch;
        for (int i = 0; i < kMaxHeadArgs; ++i)
            ha.h[i] = (a.src == kHeadsArg && i < nb * a.n_heads)
                          ? a.heads_host[(size_t)b0 * a.n_heads + i] : 0;
        dim3 grid(nrb * a.n_heads * nb);
        hipLaunchKernelGGL((score_partial_kernel<DT, NKS, MAXC, CONF>), grid, dim3(kScoreNT),
                           in_lds ? cols : 0, a.st, (const char *)a.q, (const char *)a.k, ha,
                           a.heads_dev, a.src, a.row_mask, a.row_lse, b0, a.H, a.Nt, a.N,
                           a.n_heads, a.sl2e, a.partial, in_lds ? 1 : 0);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

// Logit blocks held in registers between the two passes: the smallest of 1,
// 2, 4, 8, 16, 32 chunks that covers the keys, within a register budget that
// shrinks as the head width grows; otherwise the keys are streamed twice
// (MAXC = 0).
template <int NKS>
constexpr int score_maxc_cap() { return NKS <= 4 ? 32 : (NKS <= 8 ? 8 : 4); }

template <int DT, int NKS, bool CONF>
static hipError_t score_nks(const ScoreLaunch &a) {
    if constexpr (CONF) {
        return score_go<DT, NKS, 0, true>(a);
    } else {
        const int nch = (a.N + kScoreCK - 1) / kScoreCK;
        constexpr int cap = score_maxc_cap<NKS>();
#define PV_MAXC_CASE(mc) \
    if (nch <= mc && mc <= cap) return score_go<DT, NKS, (mc <= cap ? mc : 0), false>(a);
        PV_MAXC_CASE(1)
        PV_MAXC_CASE(2)
        PV_MAXC_CASE(4)
        PV_MAXC_CASE(8)
        PV_MAXC_CASE(16)
        PV_MAXC_CASE(32)
#undef PV_MAXC_CASE
        return score_go<DT, NKS, 0, false>(a);
    }
}

template <int DT, bool CONF>
static hipError_t score_dt(int nks, const ScoreLaunch &a) {
#define PV_NKS_CASE(n) \
    case n:            \
        return score_nks<DT, n, CONF>(a);
    switch (nks) {
        PV_NKS_CASE(1)
        PV_NKS_CASE(2)
        PV_NKS_CASE(3)
        PV_NKS_CASE(4)
        PV_NKS_CASE(5)
        PV_NKS_CASE(6)
        PV_NKS_CASE(7)
        PV_NKS_CASE(8)
        PV_NKS_CASE(10)
        PV_NKS_CASE(12)
        PV_NKS_CASE(14)
        PV_NKS_CASE(16)
    }
#undef PV_NKS_CASE
    return hipErrorInvalidValue;
}

template <int DT, int NKS>
static hipError_t score_head_go(const ScoreLaunch &a) {
    const int per_launch = a.src == kHeadsArg ? kMaxHeadArgs8 / a.n_heads : a.B;
    HeadArgs8 ha;
    for (int b0 = 0; b0 < a.B; b0 += per_launch) {
        const int nb = a.B - b0 < per_launch ? a.B - b0 : per_launch;
        for (int i = 0; i < kMaxHeadArgs8 / 4; ++i) ha.w[i] = 0u;
        if (a.src == kHeadsArg)
            for (int i = 0; i < nb * a.n_heads; ++i)
                ha.w[i >> 2] |= (uint32_t)(a.heads_host[(size_t)b0 * a.n_heads + i] & 0xFF)
                                << ((i & 3) * 8);
        const size_t kbytes = (size_t)((a.N + kScoreCK - 1) / kScoreCK) * ScoreStage<NKS>::STAGE;
        hipLaunchKernelGGL((score_head_kernel<DT, NKS>), dim3(a.n_heads * nb), dim3(kScoreNT),
                           kbytes, a.st, (const char *)a.q, (const char *)a.k, ha, a.heads_dev, a.src,
                           a.row_lse, b0, a.H, a.Nt, a.N, a.n_heads, a.sl2e, a.partial);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

// The split form: two launches per bounded head list, statistics then
// column sums.
template <int DT, int NKS>
static hipError_t score_split_go(const ScoreLaunch &a, float2 *stats) {
    const int nsplit = (a.N + kScoreCK - 1) / kScoreCK;
    const int per_launch = a.src == kHeadsArg ? kMaxHeadArgs / a.n_heads : a.B;
    HeadArgs ha;
    for (int b0 = 0; b0 < a.B; b0 += per_launch) {
        const int nb = a.B - b0 < per_launch ? a.B - b0 : per_launch;
        for (int i = 0; i < kMaxHeadArgs; ++i)
            ha.h[i] = (a.src == kHeadsArg && i < nb * a.n_heads)
                          ? a.heads_host[(size_t)b0 * a.n_heads + i] : 0;
        const dim3 grid(nsplit * a.n_heads * nb);
        hipLaunchKernelGGL((score_split_stats_kernel<DT, NKS>), grid, dim3(kScoreNT), 0, a.st,
                           (const char *)a.q, (const char *)a.k, ha, a.heads_dev, a.src, b0, a.H,
                           a.Nt, a.N, a.n_heads, nsplit, a.sl2e, stats);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL((score_split_cols_kernel<DT, NKS>), grid, dim3(kScoreNT),
                           (size_t)a.Nt * sizeof(float2), a.st, (const char *)a.q,
                           (const char *)a.k, ha, a.heads_dev, a.src, a.row_lse, b0, a.H, a.Nt,
                           a.N, a.n_heads, nsplit, a.sl2e, stats, a.partial);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

// log2(e) / sqrt(head width): the attention scale in base-2 units.
static float scale_log2e_of(const ScoreLaunch &a, int hd) {
    return (float)(1.4426950408889634 / sqrt((double)(a.hd_scale > 0 ? a.hd_scale : hd)));
}

template <bool CONF>
static hipError_t score_any(int dt, int hd, ScoreLaunch a) {
    const int esz = (dt == kBF16) ? 2 : 4;
    const int nks = hd * esz / 64;
    a.sl2e = scale_log2e_of(a, hd);
    if (dt == kBF16) return score_dt<kBF16, CONF>(nks, a);
    return score_dt<kF32, CONF>(nks, a);
}

// The whole-head form pays once there are enough (head, sample) pairs to
// fill the chip (measured: from 128 pairs it is faster, below it the
// 16-row blocks spread over more CUs and win by ~0.5 us).
bool score_uses_head_form(int dt, int B, int H, int n_heads, int Nt, int N, int hd) {
    const int nks = hd * ((dt == kBF16) ? 2 : 4) / 64;
    return (nks == 2 || nks == 4) && H <= 256 && Nt <= kHeadMaxRows &&
           N <= kHeadMaxChunks * kScoreCK && (long long)B * n_heads >= 128;
}

// The split form pays for long key lists when the 16-row blocks would not
// give every CU a workgroup (one per 16 rows, selected head and sample).
bool score_uses_split_form(int dt, int B, int H, int n_heads, int Nt, int N, int hd) {
    const int nks = hd * ((dt == kBF16) ? 2 : 4) / 64;
    if (score_uses_head_form(dt, B, H, n_heads, Nt, N, hd)) return false;
    return (nks == 2 || nks == 4) && N > 4 * kScoreCK &&
           (long long)((Nt + 15) / 16) * n_heads * B < 256;
}

int score_parts(int dt, int B, int H, int n_heads, int Nt, int N, int hd) {
    if (score_uses_head_form(dt, B, H, n_heads, Nt, N, hd) ||
        score_uses_split_form(dt, B, H, n_heads, Nt, N, hd))
        return 1;
    return (Nt + 15) / 16;
}

hipError_t launch_score_partial(int dt, const void *q, const void *k, const int32_t *heads_host,
                                const int32_t *heads_dev, const float *row_lse, int B, int H,
                                int Nt, int N, int hd, int hd_scale, int n_heads, float *partial,
                                float *split_stats, hipStream_t st) {
    ScoreLaunch a{q, k, heads_host, heads_dev, heads_dev ? kHeadsDevice : kHeadsArg, nullptr,
                  row_lse, B, H, Nt, N, n_heads, 0.f, partial, st};
    a.hd_scale = hd_scale;
    const int nks = hd * ((dt == kBF16) ? 2 : 4) / 64;
    if (score_uses_split_form(dt, B, H, n_heads, Nt, N, hd)) {
        if (!split_stats) return hipErrorInvalidValue;
        a.sl2e = scale_log2e_of(a, hd);
        float2 *stats = reinterpret_cast<float2 *>(split_stats);
        if (dt == kBF16)
            return nks == 2 ? score_split_go<kBF16, 2>(a, stats) : score_split_go<kBF16, 4>(a, stats);
        return nks == 2 ? score_split_go<kF32, 2>(a, stats) : score_split_go<kF32, 4>(a, stats);
    }
    if (score_uses_head_form(dt, B, H, n_heads, Nt, N, hd)) {
        a.sl2e = scale_log2e_of(a, hd);
        if (dt == kBF16) return nks == 2 ? score_head_go<kBF16, 2>(a) : score_head_go<kBF16, 4>(a);
        return nks == 2 ? score_head_go<kF32, 2>(a) : score_head_go<kF32, 4>(a);
    }
    return score_any<false>(dt, hd, a);
}

hipError_t launch_head_conf(int dt, const void *q, const void *k, const int32_t *row_mask,
                            const float *row_lse, int B, int H, int Nt, int N, int hd,
                            int hd_scale, float *partial, hipStream_t st) {
    ScoreLaunch a{q, k, nullptr, nullptr, kHeadsAll, row_mask, row_lse, B, H, Nt, N, H, 0.f,
                  partial, st};
    a.hd_scale = hd_scale;
    return score_any<true>(dt, hd, a);
}

// ----------------------------------------------------------------------------
// The launches of the one-call step that follow the top-N_1 at small batches.
// The two chains after the selection (nearest kept token -> merge, and
// score -> top-N_2) share launches, so the step is six dependent launches:
//   gram_score: the head-aware score blocks, reading the keys of the kept
//     tokens through the kept list (no compacted copy is needed yet), and the
//     split-k Gram tiles, both on one LDS ring;
//   reduce_select_gather: the score's top-N_2 (with each slot's place among
//     the kept), the Gram's argmax (one pruned row per wave) and the
//     compaction of K and V to the N_1 kept tokens;
//   then the merge, which also writes the merged rows of the N_2 kept slots
//   to their compacted places and carries the compaction of their K and V.
// ----------------------------------------------------------------------------
template <int DT, int NKS, int MAXC>
__global__ __launch_bounds__(kScoreNT) void gram_score_kernel(
    const char *__restrict__ q, const char *__restrict__ k_full, HeadArgs heads, int H, int Nt,
    int N, int n_src, const int32_t *__restrict__ kidx, int n_heads, float scale_log2e,
    float *__restrict__ partial, GramJob gj) {
    using G = PTile<DT, kSplitNS>;
    using S = ScoreStage<NKS>;
    constexpr int RING = G::LDS_BYTES > S::NS * S::STAGE ? G::LDS_BYTES : S::NS * S::STAGE;
    __shared__ __attribute__((aligned(16))) char ring[RING];
    // the score blocks first: they are the longer ones
    const int n_score = (int)gridDim.x - gj.nblocks;
    if ((int)blockIdx.x >= n_score) {
        gram_partial_tile<DT, kSplitNS, true>(gj.vis, gj.B, gj.Nv, gj.d_bytes, gj.kept, gj.N1,
                                              gj.pruned, gj.Mp, gj.ntm, gj.ntn, gj.KS, gj.part,
                                              gj.nblocks, (int)blockIdx.x - n_score, ring);
        return;
    }
    score_partial_block<DT, NKS, MAXC, false, true>(q, k_full, heads, nullptr, kHeadsArg, nullptr,
                                                    nullptr, 0, H, Nt, N, n_heads, scale_log2e,
                                                    partial, 0, n_score, kidx, n_src, ring);
}

__global__ __launch_bounds__(kScoreNT) void reduce_select_gather_kernel(ReduceJob rj, SelectJob sj,
                                                                        GatherJob gj) {
    static_assert(kScoreNT / 64 == kReduceRowsPerBlock, "one Gram row per wave");
    static_assert(kScoreNT == kGatherNT, "the gather's workgroup size");
    int blk = blockIdx.x;
    if (blk < sj.nblocks) {
        score_select_block<kScoreNT, 1>(sj, blk);
        return;
    }
    blk -= sj.nblocks;
    if (blk < rj.nblocks) {
        const int per = (rj.Mp + kReduceRowsPerBlock - 1) / kReduceRowsPerBlock;
        const int m = (blk % per) * kReduceRowsPerBlock + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
        if (m < rj.Mp) gram_reduce_row<16>(rj, m, blk / per, threadIdx.x & 63);
        return;
    }
    blk -= rj.nblocks;
    if (blk < gj.nblocks) gather_block(gj.ga, gj.idx, gj.k, blk);
}

bool gram_score_supported(int dt, int B, int n_heads, int N, int hd) {
    const int nks = hd * ((dt == kBF16) ? 2 : 4) / 64;
    return nks == 4 && N <= 4 * kScoreCK && (long long)B * n_heads <= kMaxHeadArgs;
}

template <int DT, int MAXC>
static void gram_score_go(dim3 grid, const void *q, const void *k_full, const HeadArgs &ha, int H,
                          int Nt, int N, int n_src, const int32_t *kidx, int n_heads, float sl2e,
                          float *partial, const GramJob &gj, hipStream_t st) {
    hipLaunchKernelGGL((gram_score_kernel<DT, 4, MAXC>), grid, dim3(kScoreNT), 0, st,
                       (const char *)q, (const char *)k_full, ha, H, Nt, N, n_src, kidx, n_heads,
                       sl2e, partial, gj);
}

hipError_t launch_gram_score(int dt, const void *q, const void *k_full, const int32_t *heads_host,
                             int B, int H, int Nt, int N, int n_src, const int32_t *kidx, int hd,
                             int n_heads, float *partial, const GramJob &gj, hipStream_t st) {
    if (!gram_score_supported(dt, B, n_heads, N, hd) || N < 1) return hipErrorInvalidValue;
    HeadArgs ha;
    for (int i = 0; i < kMaxHeadArgs; ++i) ha.h[i] = i < B * n_heads ? heads_host[i] : 0;
    const float sl2e = (float)(1.4426950408889634 / sqrt((double)hd));
    const dim3 grid(((Nt + 15) / 16) * n_heads * B + gj.nblocks);
    const int nch = (N + kScoreCK - 1) / kScoreCK;
#define PV_GS_CASE(mc)                                                                            \
    if (nch <= mc) {                                                                              \
        if (dt == kBF16)                                                                          \
            gram_score_go<kBF16, mc>(grid, q, k_full, ha, H, Nt, N, n_src, kidx, n_heads, sl2e,   \
                                     partial, gj, st);                                            \
        else                                                                                      \
            gram_score_go<kF32, mc>(grid, q, k_full, ha, H, Nt, N, n_src, kidx, n_heads, sl2e,    \
                                    partial, gj, st);                                             \
        return hipGetLastError();                                                                 \
    }
    PV_GS_CASE(1)
    PV_GS_CASE(2)
    PV_GS_CASE(4)
#undef PV_GS_CASE
    return hipErrorInvalidValue;
}

hipError_t launch_reduce_select_gather(const ReduceJob &rj, const SelectJob &sj,
                                       const GatherJob &gj, hipStream_t st) {
    if (sj.nblocks > 0 && sj.N > kScoreNT) return hipErrorInvalidValue;
    const int blocks = sj.nblocks + rj.nblocks + gj.nblocks;
    if (blocks < 1) return hipSuccess;
    hipLaunchKernelGGL(reduce_select_gather_kernel, dim3(blocks), dim3(kScoreNT), 0, st, rj, sj, gj);
    return hipGetLastError();
}

// ----------------------------------------------------------------------------
// conf_select: one workgroup per sample.  C[h] = the row-block partials of
// head h added in order; the n_vis heads of largest C (ties to the lower
// head id) are written in ascending order.
// ----------------------------------------------------------------------------
__global__ __launch_bounds__(256) void conf_select_kernel(const float *__restrict__ part, int H,
                                                          int nrb, float *__restrict__ conf,
                                                          int n_vis, int32_t *__restrict__ heads) {
    __shared__ TopkSmem sm;
    const int b = blockIdx.x;
    const int E = topk_per_thread(H, 256), h0 = threadIdx.x * E;
    uint32_t key[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
        const int h = h0 + e;
        key[e] = 0u;
        if (e < E && h < H) {
            const float *ph = part + ((size_t)b * H + h) * nrb;
            float c = 0.f;
            for (int r = 0; r < nrb; ++r) c += ph[r];
            if (conf) conf[(size_t)b * H + h] = c;
            key[e] = order_key(c);
        }
    }
    block_topk<256, 2>(key, H, n_vis, heads + (size_t)b * n_vis, nullptr, nullptr, sm);
}

hipError_t launch_conf_select(const float *partial, int B, int H, int Nt, float *conf, int n_vis,
                              int32_t *heads, hipStream_t st) {
    if (H > 512) return hipErrorInvalidValue;
    hipLaunchKernelGGL(conf_select_kernel, dim3(B), dim3(256), 0, st, partial, H, (Nt + 15) / 16,
                       conf, n_vis, heads);
    return hipGetLastError();
}

hipError_t launch_score_select(const float *partial, int B, int nparts, int N, float inv_norm,
                               float *v, int budget, int32_t *kept, hipStream_t st) {
    // as many threads as keys where possible: each thread's partial sums are
    // then all in flight at once
    const SelectJob sj{partial, nparts, N, inv_norm, v, budget, kept, 0};
#define PV_SEL_CASE(nt, e) \
    hipLaunchKernelGGL((score_select_kernel<nt, e>), dim3(B), dim3(nt), 0, st, sj)
    if (N <= 256)
        PV_SEL_CASE(256, 1);
    else if (N <= 1024)
        PV_SEL_CASE(1024, 1);
    else if (N <= 1024 * 2)
        PV_SEL_CASE(1024, 2);
    else if (N <= 1024 * 4)
        PV_SEL_CASE(1024, 4);
    else if (N <= 1024 * 16)
        PV_SEL_CASE(1024, 16);
    else
        return hipErrorInvalidValue;
#undef PV_SEL_CASE
    return hipGetLastError();
}

}  // namespace pv
