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

// Rows of a width the matrix-core kernels do not stream (their k chunks are
// 128 bytes of an embedding row and 64 or 128 bytes of a head row) copied
// into rows of the next such width, the tail filled with zeros: a zero
// element changes no dot product and no norm.  dst row r = src row r
// (in_bytes) followed by zeros up to out_bytes; both multiples of 16.
__global__ __launch_bounds__(256) void pad_rows_kernel(const char *__restrict__ src,
                                                       char *__restrict__ dst, long long n_rows,
                                                       int in_pieces, int out_pieces) {
    const long long total = n_rows * out_pieces;
    for (long long i = (long long)blockIdx.x * 256 + threadIdx.x; i < total;
         i += (long long)gridDim.x * 256) {
        const long long r = i / out_pieces;
        const int p = (int)(i - r * out_pieces);
        uint4 v = {0u, 0u, 0u, 0u};
        if (p < in_pieces) v = ld16(src + (r * in_pieces + p) * 16);
        st16(dst + i * 16, v);
    }
}

hipError_t launch_pad_rows(const void *src, void *dst, long long n_rows, int in_bytes,
                           int out_bytes, hipStream_t st) {
    const long long total = n_rows * (out_bytes / 16);
    long long blocks = (total + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(pad_rows_kernel, dim3((unsigned)blocks), dim3(256), 0, st,
                       (const char *)src, (char *)dst, n_rows, in_bytes / 16, out_bytes / 16);
    return hipGetLastError();
}

}  // namespace pv
