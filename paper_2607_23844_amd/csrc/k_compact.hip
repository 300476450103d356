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

// Token kinds, chunked: a frame's tokens in chunks of CMP_THREADS (one per
// thread).  k_chunk_counts counts each chunk's cached tokens; block (unit u,
// chunk q) of k_compact_chunks then takes its bases from those counts (kept
// rows before it in its unit, cached tokens before it in id order) and its
// in-chunk ranks from per-wave ballots.  A unit's chunks are those of frame
// fa, then those of frame fb (pairs).
__global__ __launch_bounds__(CMP_THREADS) void k_chunk_counts(const int32_t *__restrict__ flag, int N, int nch,
                                                              int32_t *__restrict__ ccnt) {
    __shared__ int wsum[CMP_THREADS / 64];
    const int f = blockIdx.x / nch, c = blockIdx.x - f * nch;
    const int i = c * CMP_THREADS + threadIdx.x;
    const bool cached = i < N && flag[(long)f * N + i] != 0;
    const unsigned long long b = __builtin_amdgcn_ballot_w64(cached);
    if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = __builtin_popcountll(b);
    __syncthreads();
    if (threadIdx.x == 0) {
        int tot = 0;
        for (int w = 0; w < CMP_THREADS / 64; ++w) tot += wsum[w];
        ccnt[blockIdx.x] = tot;
    }
}

__global__ __launch_bounds__(CMP_THREADS) void k_compact_chunks(const int32_t *__restrict__ units, int F, int N,
                                                                int nch, const int32_t *__restrict__ flag,
                                                                const int32_t *__restrict__ ccnt, int L,
                                                                int n_cached, int32_t *__restrict__ kept_idx,
                                                                int32_t *__restrict__ cached_idx,
                                                                int32_t *__restrict__ rmap) {
    __shared__ int sh[17];
    __shared__ int wpre[CMP_THREADS / 64];
    const int u = blockIdx.x / (2 * nch), q = blockIdx.x - u * 2 * nch;
    int fa = u, fb = -1;
    if (units != nullptr) {
        const int s = units[2 * u], d = units[2 * u + 1];
        fa = d >= 0 ? min(s, d) : s;
        fb = d >= 0 ? max(s, d) : -1;
    }
    if (fa < 0 || fa >= F || fb >= F) return;   // malformed unit table
    if (q >= (fb >= 0 ? 2 : 1) * nch) return;
    const int f = q < nch ? fa : fb, c = q < nch ? q : q - nch;
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    // bases: kept rows of the unit's earlier chunks, cached tokens of earlier
    // chunks in id order (earlier frames, then earlier chunks of this frame)
    int kb = 0, cb = 0;
    for (int e = t; e < F * nch; e += CMP_THREADS) {
        const int fe = e / nch, ce = e - fe * nch;
        const int n = ccnt[e];
        const int len = min(CMP_THREADS, N - ce * CMP_THREADS);
        if (fe < f || (fe == f && ce < c)) cb += n;
        const bool in_unit_before = (fe == fa && (f == fb || ce < c)) || (fe == fb && f == fb && ce < c);
        if (in_unit_before) kb += len - n;
    }
    int tot;
    (void)block_exclusive_scan(kb, sh, tot);
    kb = tot;
    (void)block_exclusive_scan(cb, sh, tot);
    cb = tot;
    const int i = c * CMP_THREADS + t;
    const long p = (long)f * N + i;
    const bool cached = i < N && flag[p] != 0;
    const unsigned long long b = __builtin_amdgcn_ballot_w64(cached);
    if (lane == 0) wpre[wave] = __builtin_popcountll(b);
    __syncthreads();
    if (t == 0) {
        int run = 0;
        for (int w = 0; w < CMP_THREADS / 64; ++w) { const int x = wpre[w]; wpre[w] = run; run += x; }
    }
    __syncthreads();
    if (i >= N) return;
    const int crank = wpre[wave] + __builtin_popcountll(b & ((1ull << lane) - 1ull));
    const int krank = t - crank;
    if (cached) {
        const int pos = cb + crank;
        if (pos < n_cached) cached_idx[pos] = (int)p;
        rmap[p] = -1;
    } else {
        const int k = kb + krank;
        const int row = u * L + k;
        if (k < L) kept_idx[row] = (int)p;
        rmap[p] = k < L ? row : -2;
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

// Frame Cache on k x k patches: a token is skipped when its (frame, patch)
// tile is cached (flag at the tile's top-left token).  Every block stages
// the F*k*k tile flags in LDS and derives the per-frame retained counts (the
// sequence offsets, frames in order) and the cached totals before each
// frame; a token's rank inside its frame is its position minus the cached
// tokens of its frame with a smaller id, counted tile by tile (tiles are
// rectangles: whole tile rows above it plus, in its own tile row, the part
// of each tile to its left).  Rows and ranks are checked against the plan's
// static counts before any write.
constexpr int FP_MAX_TILES = 8192;   // F * k * k (frames <= 32, k*k <= 256)

__device__ __forceinline__ int fp_cached_before(const uint8_t *fl, int f, int kk, int k, int ph, int pw, int y,
                                                int x) {
    int c = 0;
    for (int t = 0; t < kk; ++t) {
        if (!fl[f * kk + t]) continue;
        const int ty = (t / k) * ph, tx = (t % k) * pw;
        c += pw * min(max(y - ty, 0), ph);                       // whole rows of the tile above row y
        if (y >= ty && y < ty + ph) c += min(max(x - tx, 0), pw);   // its part of row y left of x
    }
    return c;
}

__global__ __launch_bounds__(256) void k_compact_fpatch(const int32_t *__restrict__ flag,
                                                        const int32_t *__restrict__ mtok, int F, int N, int W, int k,
                                                        int ph, int pw, int n_kept, int n_cached, int map_matched,
                                                        int32_t *__restrict__ kept_idx,
                                                        int32_t *__restrict__ cached_idx, int32_t *__restrict__ rmap,
                                                        int32_t *__restrict__ seq_off) {
    __shared__ uint8_t fl[FP_MAX_TILES];
    __shared__ int off[33], cpre[33];
    const int kk = k * k, tile = ph * pw;
    for (int i = threadIdx.x; i < F * kk; i += blockDim.x) {
        const int f = i / kk, t = i - f * kk;
        const long tl = (long)f * N + (long)(t / k) * ph * W + (t % k) * pw;
        fl[i] = flag[tl] != 0 ? 1 : 0;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        int o = 0, c = 0;
        for (int f = 0; f < F; ++f) {
            int cf = 0;
            for (int t = 0; t < kk; ++t) cf += fl[f * kk + t];
            off[f] = o;
            cpre[f] = c;
            o += N - cf * tile;
            c += cf * tile;
        }
        off[F] = o;
        cpre[F] = c;
    }
    __syncthreads();
    if (blockIdx.x == 0)
        for (int f = threadIdx.x; f <= F; f += blockDim.x) seq_off[f] = min(off[f], n_kept);
    const long total = (long)F * N;
    for (long p = (long)blockIdx.x * blockDim.x + threadIdx.x; p < total; p += (long)gridDim.x * blockDim.x) {
        const int f = (int)(p / N), n = (int)(p - (long)f * N), y = n / W, x = n - y * W;
        const int t = (y / ph) * k + x / pw;
        const int cb = fp_cached_before(fl, f, kk, k, ph, pw, y, x);
        if (!fl[f * kk + t]) {
            const int row = off[f] + n - cb;
            const bool ok = row >= 0 && row < n_kept;
            if (ok) kept_idx[row] = (int)p;
            rmap[p] = ok ? row : -2;
        } else {
            const int cr = cpre[f] + cb;
            if (cr >= 0 && cr < n_cached) cached_idx[cr] = (int)p;
            int m = -1;
            if (map_matched) {
                // token n of the tile reads token n of the matched frame
                const long tl = (long)f * N + (long)(y / ph) * ph * W + (x / pw) * pw;
                const int d = mtok[tl] / N;
                m = -2;
                if (d >= 0 && d < F && !fl[d * kk + t]) {
                    const int row = off[d] + n - fp_cached_before(fl, d, kk, k, ph, pw, y, x);
                    if (row >= 0 && row < n_kept) m = row;
                }
            }
            rmap[p] = m;
        }
    }
}

hipError_t launch_compact_fpatch(const Plan &p, const int32_t *flag, const int32_t *mtok, int32_t *kept_idx,
                                 int32_t *cached_idx, int32_t *rmap, int32_t *seq_off, int map_matched,
                                 hipStream_t st) {
    if (p.F * p.k * p.k > FP_MAX_TILES || p.F > 32) return hipErrorInvalidValue;
    const long total = (long)p.F * p.N;
    const unsigned grid = (unsigned)std::min<long>((total + 255) / 256, 1024);
    {
        StageScope _stage(st, "compact");
        launch_k(k_compact_fpatch, grid, 256, 0, st, flag, mtok, p.F, p.N, p.W, p.k, p.ph, p.pw, p.n_kept, p.n_cached,
                 map_matched, kept_idx, cached_idx, rmap, seq_off);
    }
    return hipGetLastError();
}

hipError_t launch_compact(const Plan &p, const int32_t *units, const int32_t *flag, const int32_t *mtok,
                          int32_t *fcnt, int32_t *kept_idx, int32_t *cached_idx, int32_t *rmap, int map_matched,
                          hipStream_t st) {
    const long total = (long)p.F * p.N;
    const unsigned grid = (unsigned)std::min<long>((total + 255) / 256, 4096);
    if (p.kind == KIND_TOKEN) {
        // chunk counts, then every (unit, chunk) block from them
        const int nch = cdiv(p.N, CMP_THREADS);
        const bool pairs = p.gran == 3;
        {
            StageScope _stage(st, "compact");
            launch_k(k_chunk_counts, (unsigned)(p.F * nch), CMP_THREADS, 0, st, flag, p.N, nch, fcnt);
            launch_k(k_compact_chunks, (unsigned)(p.n_units * 2 * nch), CMP_THREADS, 0, st, pairs ? units : nullptr,
                     p.F, p.N, nch, flag, (const int32_t *)fcnt, p.seq_len, p.n_cached, kept_idx, cached_idx, rmap);
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
