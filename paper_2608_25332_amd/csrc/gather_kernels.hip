// Order-preserving row compaction (Sec. 4.1: pruned tokens are excluded from
// all later computation).  A pure HBM stream.  One launch moves up to
// kMaxGather tensors that share the kept-index list (hidden states, K and V).
// Each tensor is cut into planes (one per sample and head group) of k rows;
// each workgroup copies a contiguous span of 16-byte pieces of one plane, so
// consecutive threads take consecutive pieces of a destination row and both
// the gathered reads (whole source rows) and the writes coalesce.  All index
// arithmetic is 32-bit except the final byte offsets.
#include "pv_launch.h"
#include "pv_device.h"

namespace pv {

constexpr int kGatherNT = 256;

__global__ __launch_bounds__(kGatherNT) void gather_kernel(GatherArgs ga,
                                                           const int32_t *__restrict__ idx, int k) {
    const int blk = blockIdx.x;
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
    int rr[kGatherIT], cc[kGatherIT];
#pragma unroll
    for (int it = 0; it < kGatherIT; ++it) {
        const int e = (sub * kGatherIT + it) * kGatherNT + threadIdx.x;
        const int ec = e < ppp ? e : ppp - 1;
        const int r = ec / g.cpr, c = ec - r * g.cpr;
        rr[it] = e < ppp ? r : -1;
        cc[it] = c;
        const int j = ib[r];
        v[it] = uint4{0u, 0u, 0u, 0u};
        if (j >= 0 && j < g.n_src) v[it] = ld16(s0 + (int64_t)j * g.sr + (int64_t)c * 16);
    }
#pragma unroll
    for (int it = 0; it < kGatherIT; ++it)
        if (rr[it] >= 0) st16(d0 + (int64_t)rr[it] * g.dr + (int64_t)cc[it] * 16, v[it]);
}

hipError_t launch_gather(const GatherArgs &ga, const int32_t *idx, int B, int k, hipStream_t st) {
    (void)B;
    const int blocks = ga.bstart[ga.n];
    hipLaunchKernelGGL(gather_kernel, dim3(blocks), dim3(kGatherNT), 0, st, ga, idx, k);
    return hipGetLastError();
}

}  // namespace pv
