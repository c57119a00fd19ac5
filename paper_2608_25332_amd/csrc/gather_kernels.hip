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

}  // namespace pv
