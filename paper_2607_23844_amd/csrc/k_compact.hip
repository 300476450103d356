// Bookkeeping that turns the per-item cache flags into the reduced attention
// batch and the restore map (OmniCache §3.2.1-§3.2.3: retained items are
// computed, cached positions keep their original place).  Sequences are
// ordered by the smallest item they cover; rows inside a sequence follow
// ascending token id (block sequences: frames 0..F-1 of one position).
// Every write is bounded by the plan's static counts, so inconsistent flags
// can produce wrong indices but never an out-of-range access.
#include "oc_internal.h"
#include "oc_launch.h"
#include "oc_device.h"
#include "oc_block.h"
#include <algorithm>

namespace oc {

constexpr int CMP_THREADS = 1024;

// cached tokens per frame (token-kind flags)
__global__ void k_frame_counts(const int32_t *__restrict__ flag, int N, int32_t *__restrict__ fcnt) {
    __shared__ int sh[17];
    const int f = blockIdx.x;
    int c = 0;
    for (int n = threadIdx.x; n < N; n += blockDim.x) c += flag[(long)f * N + n] ? 1 : 0;
    int total;
    (void)block_exclusive_scan(c, sh, total);
    if (threadIdx.x == 0) fcnt[f] = total;
}

// One block per attention unit (a frame, or a frame pair s, d): retained
// tokens of the unit's frames in ascending id become rows [u*L, u*L+L).
// fcnt == nullptr: every frame caches static_cnt tokens (token groups of
// plain frames, a fixed budget per group).
__global__ __launch_bounds__(CMP_THREADS) void k_compact_units(const int32_t *__restrict__ units, int F,
                                                               const int32_t *__restrict__ flag,
                                                               const int32_t *__restrict__ fcnt, int static_cnt,
                                                               int N, int L, int n_cached,
                                                               int32_t *__restrict__ kept_idx,
                                                               int32_t *__restrict__ cached_idx,
                                                               int32_t *__restrict__ rmap) {
    __shared__ int sh[17];
    __shared__ int base[3];
    const int u = blockIdx.x;
    int fa = u, fb = -1;
    if (units != nullptr) {
        const int s = units[2 * u], d = units[2 * u + 1];
        fa = d >= 0 ? min(s, d) : s;
        fb = d >= 0 ? max(s, d) : -1;
    }
    if (fa < 0 || fa >= F || fb >= F) return;   // malformed unit table
    if (threadIdx.x == 0) {
        if (fcnt == nullptr) {
            base[0] = fa * static_cnt;
            base[1] = fb >= 0 ? fb * static_cnt : 0;
            base[2] = static_cnt;
        } else {
            int ca = 0, cb = 0;
            for (int f = 0; f < fa; ++f) ca += fcnt[f];
            if (fb >= 0) for (int f = 0; f < fb; ++f) cb += fcnt[f];
            base[0] = ca;          // cached tokens before frame fa
            base[1] = cb;          // cached tokens before frame fb
            base[2] = fcnt[fa];    // cached tokens in frame fa
        }
    }
    __syncthreads();
    const int n_u = fb >= 0 ? 2 * N : N;
    const int ipt = cdiv(n_u, CMP_THREADS);
    const int i0 = threadIdx.x * ipt;
    int kept_local = 0, cached_local = 0;
    for (int j = 0; j < ipt; ++j) {
        const int i = i0 + j;
        if (i >= n_u) break;
        const int p = i < N ? fa * N + i : fb * N + (i - N);
        if (flag[p]) ++cached_local; else ++kept_local;
    }
    int tot;
    int krank = block_exclusive_scan(kept_local, sh, tot);
    int crank = block_exclusive_scan(cached_local, sh, tot);
    for (int j = 0; j < ipt; ++j) {
        const int i = i0 + j;
        if (i >= n_u) break;
        const bool second = i >= N;
        const int p = second ? fb * N + (i - N) : fa * N + i;
        if (flag[p]) {
            const int pos = second ? base[1] + (crank - base[2]) : base[0] + crank;
            if (pos >= 0 && pos < n_cached) cached_idx[pos] = p;
            rmap[p] = -1;
            ++crank;
        } else {
            const int row = u * L + krank;
            if (krank < L) kept_idx[row] = p;
            rmap[p] = krank < L ? row : -2;
            ++krank;
        }
    }
}

// Block kind: the b-th retained position (ascending) becomes sequence b with
// rows b*F + f; cached tokens ascend frame-major.
__global__ __launch_bounds__(CMP_THREADS) void k_compact_blocks(const int32_t *__restrict__ flag, int F, int N,
                                                                int n_seq, int32_t *__restrict__ kept_idx,
                                                                int32_t *__restrict__ cached_idx,
                                                                int32_t *__restrict__ rmap) {
    __shared__ int sh[17];
    const int n_cb = N - n_seq;
    const int ipt = cdiv(N, CMP_THREADS);
    const int n0 = threadIdx.x * ipt;
    int kl = 0, cl = 0;
    for (int j = 0; j < ipt; ++j) {
        const int n = n0 + j;
        if (n >= N) break;
        if (flag[n]) ++cl; else ++kl;
    }
    int tot;
    int kr = block_exclusive_scan(kl, sh, tot);
    int cr = block_exclusive_scan(cl, sh, tot);
    for (int j = 0; j < ipt; ++j) {
        const int n = n0 + j;
        if (n >= N) break;
        if (flag[n]) {
            for (int f = 0; f < F; ++f) {
                if (cr < n_cb) cached_idx[f * n_cb + cr] = f * N + n;
                rmap[f * N + n] = -1;
            }
            ++cr;
        } else {
            for (int f = 0; f < F; ++f) {
                if (kr < n_seq) kept_idx[kr * F + f] = f * N + n;
                rmap[f * N + n] = kr < n_seq ? kr * F + f : -2;
            }
            ++kr;
        }
    }
}

// Frame kind: retained frames in ascending order, N rows each.
__global__ void k_compact_frames(const int32_t *__restrict__ flag, int F, int N, int n_seq,
                                 int32_t *__restrict__ kept_idx, int32_t *__restrict__ cached_idx,
                                 int32_t *__restrict__ rmap) {
    __shared__ int krank[64], crank[64];
    if (threadIdx.x == 0) {
        int k = 0, c = 0;
        for (int f = 0; f < F; ++f) {
            krank[f] = k;
            crank[f] = c;
            if (flag[f]) ++c; else ++k;
        }
    }
    __syncthreads();
    const int n_cf = F - n_seq;
    const long total = (long)F * N;
    for (long p = (long)blockIdx.x * blockDim.x + threadIdx.x; p < total; p += (long)gridDim.x * blockDim.x) {
        const int f = (int)(p / N), n = (int)(p - (long)f * N);
        if (flag[f]) {
            if (crank[f] < n_cf) cached_idx[(long)crank[f] * N + n] = (int)p;
            rmap[p] = -1;
        } else {
            const bool ok = krank[f] < n_seq;
            if (ok) kept_idx[(long)krank[f] * N + n] = (int)p;
            rmap[p] = ok ? krank[f] * N + n : -2;
        }
    }
}

// "matched" restore map: a cached position points at the row of the token
// whose fresh output replaces it (its matched representative; same position
// in the matched frame; same frame at the matched block position).
__global__ void k_map_matched(int kind, const int32_t *__restrict__ flag, const int32_t *__restrict__ mtok, int F,
                              int N, int32_t *__restrict__ rmap) {
    const long total = (long)F * N;
    for (long p = (long)blockIdx.x * blockDim.x + threadIdx.x; p < total; p += (long)gridDim.x * blockDim.x) {
        const int f = (int)(p / N), n = (int)(p - (long)f * N);
        long src = -1;
        if (kind == KIND_TOKEN) {
            if (flag[p]) { const int m = mtok[p]; src = (m >= 0 && m < total) ? m : -1; }
        } else if (kind == KIND_BLOCK) {
            if (flag[n]) { const int m = mtok[n]; src = (m >= 0 && m < N) ? (long)f * N + m : -1; }
        } else {
            if (flag[f]) { const int m = mtok[f]; src = (m >= 0 && m < F) ? (long)m * N + n : -1; }
        }
        if (src >= 0) rmap[p] = rmap[src];
    }
}

hipError_t launch_compact(const Plan &p, const int32_t *units, const int32_t *flag, const int32_t *mtok,
                          int32_t *fcnt, int32_t *kept_idx, int32_t *cached_idx, int32_t *rmap, int map_matched,
                          hipStream_t st) {
    const long total = (long)p.F * p.N;
    const unsigned grid = (unsigned)std::min<long>((total + 255) / 256, 4096);
    if (p.kind == KIND_TOKEN) {
        // frame pairs split their budget between two frames in a data-dependent
        // way: count per frame; plain frames cache k*k*R_tok tokens each
        const bool pairs = p.gran == 3;
        if (pairs) {
            StageScope _stage(st, "frame_counts");
            launch_k(k_frame_counts, p.F, 1024, 0, st, flag, p.N, fcnt);
        }
        {
            StageScope _stage(st, "compact");
            launch_k(k_compact_units, p.n_units, CMP_THREADS, 0, st, pairs ? units : nullptr, p.F, flag,
                                                                pairs ? fcnt : nullptr, p.k * p.k * p.R_tok, p.N,
                                                                p.seq_len, p.n_cached, kept_idx, cached_idx, rmap);
        }
    } else if (p.kind == KIND_BLOCK) {
        {
            StageScope _stage(st, "compact");
            launch_k(k_compact_blocks, 1, CMP_THREADS, 0, st, flag, p.F, p.N, p.n_seq, kept_idx, cached_idx, rmap);
        }
    } else {
        {
            StageScope _stage(st, "compact");
            launch_k(k_compact_frames, grid, 256, 0, st, flag, p.F, p.N, p.n_seq, kept_idx, cached_idx, rmap);
        }
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !map_matched) return e;
    return launch_map_matched(p, flag, mtok, rmap, st);
}

hipError_t launch_map_matched(const Plan &p, const int32_t *flag, const int32_t *mtok, int32_t *rmap,
                              hipStream_t st) {
    const long total = (long)p.F * p.N;
    const unsigned grid = (unsigned)std::min<long>((total + 255) / 256, 4096);
    {
        StageScope _stage(st, "map_matched");
        launch_k(k_map_matched, grid, 256, 0, st, p.kind, flag, mtok, p.F, p.N, rmap);
    }
    return hipGetLastError();
}

}  // namespace oc
