// Coalesced row movement: gather of retained rows and restoration of cached
// positions (OmniCache §3.2.1 / §3.2.3 restoration at the original
// positions; App. A gather-scatter).  Each thread moves one 16-byte chunk of
// a row; consecutive threads cover consecutive chunks of a row.
#include "oc_internal.h"
#include "oc_launch.h"
#include "oc_device.h"

namespace oc {

// x_kept[i] = x[kept_idx[i]]
__global__ void k_gather(const uint4 *__restrict__ x, const int32_t *__restrict__ kept_idx, int n_rows, int cpr,
                         long n_src_rows, uint4 *__restrict__ out) {
    const long total = (long)n_rows * cpr;
    for (long c = (long)blockIdx.x * blockDim.x + threadIdx.x; c < total; c += (long)gridDim.x * blockDim.x) {
        const int r = (int)(c / cpr), j = (int)(c - (long)r * cpr);
        const int s = kept_idx[r];
        if (s >= 0 && s < n_src_rows) out[c] = x[(long)s * cpr + j];
    }
}

// y[p] = y_kept[map[p]] (0 <= map < n_rows) or cache_y[p] (map == -1)
__global__ void k_restore(const uint4 *__restrict__ yk, int n_rows, const int32_t *__restrict__ rmap,
                          const uint4 *cache, long n_pos, int cpr, uint4 *y) {
    const long total = n_pos * cpr;
    for (long c = (long)blockIdx.x * blockDim.x + threadIdx.x; c < total; c += (long)gridDim.x * blockDim.x) {
        const long p = c / cpr;
        const int j = (int)(c - p * cpr);
        const int m = rmap[p];
        if (m >= 0 && m < n_rows) y[c] = yk[(long)m * cpr + j];
        else if (m == -1 && cache != nullptr && cache != y) y[c] = cache[c];
    }
}

// y[p] = y[kept_idx[map[p]]] for cached p: the "matched" cold policy after
// the retained rows were written in place.
__global__ void k_copy_matched(const int32_t *__restrict__ cached_idx, int n_cached,
                               const int32_t *__restrict__ rmap, const int32_t *__restrict__ kept_idx, int n_kept,
                               long n_pos, int cpr, uint4 *y) {
    const long total = (long)n_cached * cpr;
    for (long c = (long)blockIdx.x * blockDim.x + threadIdx.x; c < total; c += (long)gridDim.x * blockDim.x) {
        const int i = (int)(c / cpr), j = (int)(c - (long)i * cpr);
        const int p = cached_idx[i];
        if (p < 0 || p >= n_pos) continue;
        const int m = rmap[p];
        if (m < 0 || m >= n_kept) continue;
        const int src = kept_idx[m];
        if (src < 0 || src >= n_pos) continue;
        y[(long)p * cpr + j] = y[(long)src * cpr + j];
    }
}

__global__ void k_fill_i32(int32_t *__restrict__ dst, long n, int32_t value) {
    for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x) dst[i] = value;
}

static unsigned grid_for(long chunks) {
    const long b = (chunks + 255) / 256;
    return (unsigned)(b < 1 ? 1 : (b > 8192 ? 8192 : b));
}

hipError_t launch_gather(const Plan &p, const void *x, const int32_t *kept_idx, int n_rows, void *x_kept,
                         hipStream_t st) {
    const int cpr = p.C * p.esz / 16;
    {
        StageScope _stage(st, "gather");
        launch_k(k_gather, grid_for((long)n_rows * cpr), 256, 0, st, (const uint4 *)x, kept_idx, n_rows, cpr,
                                                               (long)p.F * p.N, (uint4 *)x_kept);
    }
    return hipGetLastError();
}

hipError_t launch_restore(const Plan &p, const void *y_kept, int n_rows, const int32_t *rmap, const void *cache_y,
                          void *y, hipStream_t st) {
    const int cpr = p.C * p.esz / 16;
    const long n_pos = (long)p.F * p.N;
    {
        StageScope _stage(st, "restore");
        launch_k(k_restore, grid_for(n_pos * cpr), 256, 0, st, (const uint4 *)y_kept, n_rows, rmap, (const uint4 *)cache_y,
                                                         n_pos, cpr, (uint4 *)y);
    }
    return hipGetLastError();
}

hipError_t launch_copy_matched(const Plan &p, const int32_t *cached_idx, int n_cached, const int32_t *rmap,
                               const int32_t *kept_idx, void *y, hipStream_t st) {
    if (n_cached == 0) return hipSuccess;
    const int cpr = p.C * p.esz / 16;
    {
        StageScope _stage(st, "copy_matched");
        launch_k(k_copy_matched, grid_for((long)n_cached * cpr), 256, 0, st, cached_idx, n_cached, rmap, kept_idx, p.n_kept,
                                                                       (long)p.F * p.N, cpr, (uint4 *)y);
    }
    return hipGetLastError();
}

}  // namespace oc

namespace oc {
hipError_t launch_fill_i32(int32_t *dst, long n, int32_t value, hipStream_t st) {
    if (n <= 0) return hipSuccess;
    {
        StageScope _stage(st, "fill");
        launch_k(k_fill_i32, grid_for(n), 256, 0, st, dst, n, value);
    }
    return hipGetLastError();
}
}  // namespace oc
