// Order-preserving row compaction (Sec. 4.1: pruned tokens are excluded from
// all later computation).  A pure HBM stream.  One launch moves up to
// kMaxGather tensors that share the kept-index list (hidden states, K and V).
// Each tensor is cut into planes (one per sample and head group) of k rows;
// each workgroup copies a contiguous span of 16-byte pieces of one plane, so
// consecutive threads take consecutive pieces of a destination row and both
// the gathered reads (whole source rows) and the writes coalesce.  All index
// arithmetic is 32-bit except the final byte offsets.
#include "pv_jobs.h"

namespace pv {

__global__ __launch_bounds__(kGatherNT) void gather_kernel(GatherArgs ga,
                                                           const int32_t *__restrict__ idx, int k) {
    gather_block(ga, idx, k, blockIdx.x);
}

hipError_t launch_gather(const GatherArgs &ga, const int32_t *idx, int B, int k, hipStream_t st) {
    (void)B;
    const int blocks = ga.bstart[ga.n];
    hipLaunchKernelGGL(gather_kernel, dim3(blocks), dim3(kGatherNT), 0, st, ga, idx, k);
    return hipGetLastError();
}

// Index composition across two pruning stages: out[b][r] = base[b][idx[b][r]],
// the original token index of each survivor of the later stage (idx indexes
// the earlier stage's kept list, base).  Grid (ceil(k / 256), B); an index
// outside [0, n_base) is clamped into range (memory-safe; the library's own
// selections are always in range).
__global__ __launch_bounds__(256) void compose_index_kernel(const int32_t *__restrict__ base,
                                                            const int32_t *__restrict__ idx,
                                                            int n_base, int k,
                                                            int32_t *__restrict__ out) {
    const int b = blockIdx.y, r = blockIdx.x * 256 + threadIdx.x;
    if (r >= k) return;
    const int j = min(max(idx[(size_t)b * k + r], 0), n_base - 1);
    out[(size_t)b * k + r] = base[(size_t)b * n_base + j];
}

hipError_t launch_compose_index(const int32_t *base, const int32_t *idx, int B, int n_base, int k,
                                int32_t *out, hipStream_t st) {
    hipLaunchKernelGGL(compose_index_kernel, dim3((k + 255) / 256, B), dim3(256), 0, st, base, idx,
                       n_base, k, out);
    return hipGetLastError();
}

}  // namespace pv
