// Order-preserving row compaction (Sec. 4.1: pruned tokens are excluded from
// all later computation).  A pure HBM stream: every thread moves 16-byte
// pieces, consecutive threads take consecutive pieces of a destination row,
// so both the gathered reads (whole source rows) and the writes coalesce.
#include "pv_launch.h"
#include "pv_device.h"

namespace pv {

constexpr int kGatherNT = 256;

__global__ __launch_bounds__(kGatherNT) void gather_kernel(
    const char *__restrict__ src, char *__restrict__ dst, const int32_t *__restrict__ idx,
    int n_src, int k, int cpr, int64_t sb, int64_t sg, int64_t sr, int64_t db, int64_t dg,
    int64_t dr) {
    const int g = blockIdx.y, b = blockIdx.z;
    const int total = k * cpr;
    const char *s0 = src + b * sb + g * sg;
    char *d0 = dst + b * db + g * dg;
    const int32_t *ib = idx + (size_t)b * k;
    for (int e = blockIdx.x * kGatherNT + threadIdx.x; e < total; e += gridDim.x * kGatherNT) {
        const int r = e / cpr, c = e - r * cpr;
        const int j = ib[r];
        uint4 v = {0u, 0u, 0u, 0u};
        if (j >= 0 && j < n_src) v = ld16(s0 + j * sr + (int64_t)c * 16);
        st16(d0 + r * dr + (int64_t)c * 16, v);
    }
}

hipError_t launch_gather(const void *src, void *dst, const int32_t *idx, int B, int n_src, int k,
                         int groups, int64_t row_bytes, int64_t sb, int64_t sg, int64_t sr,
                         int64_t db, int64_t dg, int64_t dr, hipStream_t st) {
    const int cpr = (int)(row_bytes / 16);
    const int64_t total = (int64_t)k * cpr;
    int64_t blocks = (total + kGatherNT - 1) / kGatherNT;
    // enough workgroups to cover the chip a few times over, each thread
    // moving a handful of pieces
    int64_t per_plane = (int64_t)groups * B;
    int64_t want = (4096 + per_plane - 1) / per_plane;
    if (blocks > want) blocks = want;
    if (blocks < 1) blocks = 1;
    dim3 grid((unsigned)blocks, groups, B);
    hipLaunchKernelGGL(gather_kernel, grid, dim3(kGatherNT), 0, st, (const char *)src, (char *)dst,
                       idx, n_src, k, cpr, sb, sg, sr, db, dg, dr);
    return hipGetLastError();
}

}  // namespace pv
