// Selection of the most redundant candidates and the bookkeeping that turns
// it into the reduced attention batch (OmniCache §3.2.1-§3.2.3: "the r most
// redundant" items are cached, the retained ones are computed, cached
// positions are later restored at their original positions).
//
// Selection per group is an exact radix select on order-preserving 32-bit
// keys of node_max: the R largest keys are cached, ties at the threshold go
// to the smallest candidate positions (ascending global id), so exactly R
// are cached.  No floating-point atomics; integer LDS histograms only.
#include "oc_internal.h"
#include "oc_device.h"
#include "oc_block.h"
#include <algorithm>

namespace oc {

constexpr int SEL_THREADS = 1024;
constexpr int SEL_IPT = 16;            // candidates per thread: groups up to 16384
constexpr int CMP_THREADS = 1024;

__global__ __launch_bounds__(SEL_THREADS) void k_select(const float *__restrict__ node_max,
                                                        const int32_t *__restrict__ node_idx,
                                                        const int32_t *__restrict__ src_ids,
                                                        const int32_t *__restrict__ dst_ids,
                                                        const int32_t *__restrict__ grp_R, int S, int D,
                                                        int32_t *__restrict__ flag, int32_t *__restrict__ mtok) {
    __shared__ int hist[256];
    __shared__ int sh[17];
    __shared__ uint32_t shu[16];
    __shared__ int sel_info[2];
    const int g = blockIdx.x;
    const int t = threadIdx.x;
    const int ipt = cdiv(S, SEL_THREADS);
    const float *nm = node_max + (long)g * S;
    const int32_t *src = src_ids + (long)g * S;
    const int R = grp_R[g];

    uint32_t key[SEL_IPT];
    uint32_t vmask = 0;
    int nvalid_local = 0;
    uint32_t lo = 0xFFFFFFFFu, hi = 0u;
#pragma unroll
    for (int j = 0; j < SEL_IPT; ++j) {
        key[j] = 0;
        const int i = t * ipt + j;
        if (j < ipt && i < S && src[i] >= 0) {
            key[j] = float_key(nm[i]);
            vmask |= 1u << j;
            ++nvalid_local;
            lo = min(lo, key[j]);
            hi = max(hi, key[j]);
        }
    }
    int n_valid;
    (void)block_exclusive_scan(nvalid_local, sh, n_valid);
    const uint32_t kmin = block_reduce_u32(lo, false, shu);
    const uint32_t kmax = block_reduce_u32(hi, true, shu);

    // threshold key tau (the R-th largest) and how many keys equal to tau are taken
    uint32_t tau = 0;
    int need = 0;
    const bool none = R <= 0;
    const bool all = R >= n_valid;
    if (!none && !all) {
        const uint32_t diff = kmin ^ kmax;
        int remaining = R;
        uint32_t prefix, mask;
        int bit_hi;
        if (diff == 0) {
            prefix = kmax;
            mask = 0xFFFFFFFFu;
            bit_hi = -1;
        } else {
            const int top = 31 - __clz(diff);
            mask = top == 31 ? 0u : ~((2u << top) - 1u);
            prefix = kmax & mask;
            bit_hi = top;
        }
        while (bit_hi >= 0) {
            const int bit_lo = max(bit_hi - 7, 0);
            const int nbits = bit_hi - bit_lo + 1;
            const uint32_t dmask = (1u << nbits) - 1u;
            if (t < 256) hist[t] = 0;
            __syncthreads();
#pragma unroll
            for (int j = 0; j < SEL_IPT; ++j)
                if (((vmask >> j) & 1u) && (key[j] & mask) == prefix) atomicAdd(&hist[(key[j] >> bit_lo) & dmask], 1);
            __syncthreads();
            if (t < 64) {
                // lane covers bins [4*t, 4*t+4); suffix sums from the top bin down
                int c[4], s = 0;
#pragma unroll
                for (int q = 0; q < 4; ++q) { c[q] = hist[4 * t + q]; s += c[q]; }
                int incl = s;   // inclusive suffix over lanes >= t
#pragma unroll
                for (int o = 1; o < 64; o <<= 1) {
                    const int y = __shfl_down(incl, o, 64);
                    if (t + o < 64) incl += y;
                }
                int above = incl - s;   // count in bins above this lane's bins
#pragma unroll
                for (int q = 3; q >= 0; --q) {
                    if (above < remaining && remaining <= above + c[q]) {
                        sel_info[0] = 4 * t + q;
                        sel_info[1] = above;
                    }
                    above += c[q];
                }
            }
            __syncthreads();
            const int sel = sel_info[0];
            remaining -= sel_info[1];
            prefix |= (uint32_t)sel << bit_lo;
            mask |= dmask << bit_lo;
            bit_hi = bit_lo - 1;
            __syncthreads();
        }
        tau = prefix;
        need = remaining;
    }

    // exact selection: key > tau, or key == tau among the first `need` in index order
    int eq_local = 0;
#pragma unroll
    for (int j = 0; j < SEL_IPT; ++j)
        if (((vmask >> j) & 1u) && key[j] == tau) ++eq_local;
    int eq_total;
    int eq_rank = block_exclusive_scan((!none && !all) ? eq_local : 0, sh, eq_total);
#pragma unroll
    for (int j = 0; j < SEL_IPT; ++j) {
        if (!((vmask >> j) & 1u)) continue;
        const int i = t * ipt + j;
        bool c;
        if (none) c = false;
        else if (all) c = true;
        else if (key[j] > tau) c = true;
        else if (key[j] == tau) { c = eq_rank < need; ++eq_rank; }
        else c = false;
        const int id = src[i];
        flag[id] = c ? 1 : 0;
        mtok[id] = c ? node_idx[(long)g * S + i] : -1;
    }
    const int32_t *dst = dst_ids + (long)g * D;
    for (int i = t; i < D; i += SEL_THREADS) {
        const int id = dst[i];
        if (id >= 0) { flag[id] = 0; mtok[id] = -1; }
    }
}

hipError_t launch_select(const Plan &p, const float *node_max, const int32_t *node_idx, const int32_t *src_ids,
                         const int32_t *dst_ids, const int32_t *grp_R, int32_t *flag, int32_t *mtok,
                         hipStream_t st) {
    {
        StageScope _stage(st, "select");
        k_select<<<p.n_groups, SEL_THREADS, 0, st>>>(node_max, node_idx, src_ids, dst_ids, grp_R, p.n_src_max,
                                                     p.n_dst_max, flag, mtok);
    }
    return hipGetLastError();
}

}  // namespace oc
