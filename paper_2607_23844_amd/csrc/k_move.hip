// Coalesced row movement: gather of retained rows and restoration of cached
// positions (OmniCache §3.2.1 / §3.2.3 restoration at the original
// positions; App. A gather-scatter).  Rows move in 16-byte chunks,
// consecutive threads on consecutive chunks of a row.
#include "oc_internal.h"
#include "oc_launch.h"
#include "oc_device.h"

namespace oc {

// A thread moves CPT 16-byte chunks of one row: with upr = cpr / CPT
// threads per row, thread l of a row takes chunks l, l + upr, ... so that
// each load and store instruction of a wave covers consecutive chunks.  All
// loads are issued before the stores.  Index math is 32-bit unless the
// chunk count reaches 2^31 (WIDE).
template <int CPT, bool WIDE>
__device__ __forceinline__ void unit_of(long u, int upr, long &row, int &lane) {
    if constexpr (WIDE) {
        row = u / upr;
        lane = (int)(u - row * upr);
    } else {
        const int r = (int)u / upr;
        row = r;
        lane = (int)u - r * upr;
    }
}

// CPT chunks at stride upr: every load before any store, in named registers
// (a private array here was placed in LDS by the compiler)
template <int CPT>
__device__ __forceinline__ void copy_chunks(const uint4 *src, uint4 *dst, int upr) {
    if constexpr (CPT == 4) {
        const uint4 a = src[0], b = src[upr], c = src[2 * upr], d = src[3 * upr];
        dst[0] = a;
        dst[upr] = b;
        dst[2 * upr] = c;
        dst[3 * upr] = d;
    } else {
        static_assert(CPT == 1, "one or four chunks per thread");
        dst[0] = src[0];
    }
}

// x_kept[i] = x[kept_idx[i]]
template <int CPT, bool WIDE>
__global__ void k_gather(const uint4 *__restrict__ x, const int32_t *__restrict__ kept_idx, int n_rows, int cpr,
                         long n_src_rows, uint4 *__restrict__ out) {
    const int upr = cpr / CPT;
    const long total = (long)n_rows * upr;
    for (long u = (long)blockIdx.x * blockDim.x + threadIdx.x; u < total; u += (long)gridDim.x * blockDim.x) {
        long r;
        int l;
        unit_of<CPT, WIDE>(u, upr, r, l);
        const int s = kept_idx[r];
        if (s < 0 || s >= n_src_rows) continue;
        const uint4 *src = x + (long)s * cpr + l;
        uint4 *dst = out + r * cpr + l;
        copy_chunks<CPT>(src, dst, upr);
    }
}

// y[p] = y_kept[map[p]] (0 <= map < n_rows) or cache_y[p] (map == -1)
template <int CPT, bool WIDE>
__global__ void k_restore(const uint4 *__restrict__ yk, int n_rows, const int32_t *__restrict__ rmap,
                          const uint4 *cache, long n_pos, int cpr, uint4 *y) {
    const int upr = cpr / CPT;
    const long total = n_pos * upr;
    for (long u = (long)blockIdx.x * blockDim.x + threadIdx.x; u < total; u += (long)gridDim.x * blockDim.x) {
        long p;
        int l;
        unit_of<CPT, WIDE>(u, upr, p, l);
        const int m = rmap[p];
        const uint4 *src;
        if (m >= 0 && m < n_rows) src = yk + (long)m * cpr + l;
        else if (m == -1 && cache != nullptr && cache != y) src = cache + p * cpr + l;
        else continue;
        uint4 *dst = y + p * cpr + l;
        copy_chunks<CPT>(src, dst, upr);
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

template <typename G4, typename G1>
static void launch_rows(long rows, int cpr, G4 four, G1 one) {
    const bool by4 = cpr % 4 == 0;
    const long units = rows * (by4 ? cpr / 4 : cpr);
    const bool wide = units >= (1L << 31);
    if (by4) four(units, wide);
    else one(units, wide);
}

// Residual connection between the spatial and the temporal layer of a
// block: h = x + y elementwise, added in fp32 and rounded once (bf16: RNE),
// 16 bytes per operand and thread.
__global__ void k_add_bf16(const uint4 *__restrict__ x, const uint4 *__restrict__ y, uint4 *__restrict__ h, long n8) {
    for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n8; i += (long)gridDim.x * blockDim.x) {
        const uint4 a = x[i], b = y[i];
        const uint32_t *pa = reinterpret_cast<const uint32_t *>(&a), *pb = reinterpret_cast<const uint32_t *>(&b);
        uint4 o;
        uint32_t *po = reinterpret_cast<uint32_t *>(&o);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const float lo = __uint_as_float(pa[j] << 16) + __uint_as_float(pb[j] << 16);
            const float hi = __uint_as_float(pa[j] & 0xFFFF0000u) + __uint_as_float(pb[j] & 0xFFFF0000u);
            po[j] = (uint32_t)f2bf(lo) | ((uint32_t)f2bf(hi) << 16);
        }
        h[i] = o;
    }
}

__global__ void k_add_f32(const float4 *__restrict__ x, const float4 *__restrict__ y, float4 *__restrict__ h, long n4) {
    for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += (long)gridDim.x * blockDim.x) {
        const float4 a = x[i], b = y[i];
        h[i] = make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w);
    }
}

hipError_t launch_add(const Plan &p, const void *x, const void *y, void *h, hipStream_t st) {
    StageScope _stage(st, "residual");
    const long n = (long)p.F * p.N * p.C;
    if (p.bf16) {
        const long n8 = n / 8;
        const long blocks = std::min<long>((n8 + 255) / 256, 4L * 1024);
        launch_k(k_add_bf16, (unsigned)blocks, 256, 0, st, (const uint4 *)x, (const uint4 *)y, (uint4 *)h, n8);
    } else {
        const long n4 = n / 4;
        const long blocks = std::min<long>((n4 + 255) / 256, 4L * 1024);
        launch_k(k_add_f32, (unsigned)blocks, 256, 0, st, (const float4 *)x, (const float4 *)y, (float4 *)h, n4);
    }
    return hipGetLastError();
}

hipError_t launch_gather(const Plan &p, const void *x, const int32_t *kept_idx, int n_rows, void *x_kept,
                         hipStream_t st) {
    const int cpr = p.C * p.esz / 16;
    const long n_src = (long)p.F * p.N;
    StageScope _stage(st, "gather");
    auto go = [&](auto kern, long units) {
        launch_k(kern, grid_for(units), 256, 0, st, (const uint4 *)x, kept_idx, n_rows, cpr, n_src, (uint4 *)x_kept);
    };
    launch_rows(n_rows, cpr,
                [&](long u, bool wide) { wide ? go(k_gather<4, true>, u) : go(k_gather<4, false>, u); },
                [&](long u, bool wide) { wide ? go(k_gather<1, true>, u) : go(k_gather<1, false>, u); });
    return hipGetLastError();
}

hipError_t launch_restore(const Plan &p, const void *y_kept, int n_rows, const int32_t *rmap, const void *cache_y,
                          void *y, hipStream_t st) {
    const int cpr = p.C * p.esz / 16;
    const long n_pos = (long)p.F * p.N;
    StageScope _stage(st, "restore");
    auto go = [&](auto kern, long units) {
        launch_k(kern, grid_for(units), 256, 0, st, (const uint4 *)y_kept, n_rows, rmap, (const uint4 *)cache_y, n_pos,
                 cpr, (uint4 *)y);
    };
    launch_rows(n_pos, cpr,
                [&](long u, bool wide) { wide ? go(k_restore<4, true>, u) : go(k_restore<4, false>, u); },
                [&](long u, bool wide) { wide ? go(k_restore<1, true>, u) : go(k_restore<1, false>, u); });
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
