// Frame stage (OmniCache §3.2.2 Frame Cache; §3.2.3 frame-pair metadata):
// the F x F Gram matrix of whole-frame descriptors (N*C values each) on
// MFMA with a deterministic split-K reduction (per-block partials, then one
// wave per Gram entry summing them in fp64 in a fixed order), then frame
// similarities, best matches, the selection of the most redundant odd frames
// and their one-to-one pairing with even frames.
#include "oc_internal.h"
#include "oc_launch.h"
#include "oc_device.h"
#include "oc_mfma_tile.h"
#include <algorithm>

namespace oc {

constexpr int GRAM_WAVES = 4;
constexpr int GRAM_TARGET_BLOCKS = 1024;
constexpr int FMAX = 32;   // frames supported by the frame stage

// K range of one wave: a multiple of 64, and of C when the Gram launch also
// computes the token norms (each wave then covers whole tokens)
inline int gram_kw(const Plan &p) {
    const long D = (long)p.N * p.C;
    const long unit = gram_norms(p) ? p.C : 64;
    long kw = (D + (long)GRAM_WAVES * GRAM_TARGET_BLOCKS - 1) / ((long)GRAM_WAVES * GRAM_TARGET_BLOCKS);
    kw = ((kw + unit - 1) / unit) * unit;
    return (int)(kw < unit ? unit : kw);
}
int gram_blocks(const Plan &p) {
    const long D = (long)p.N * p.C;
    const long per_block = (long)gram_kw(p) * GRAM_WAVES;
    return (int)((D + per_block - 1) / per_block);
}

// Partial Gram of frames over k in this block's range; lane l of a wave feeds
// frame (l % 16) (+16 for the second tile) and k chunks [g*16, g*16+8) and
// [g*16+8, g*16+16) of each 64-wide step (g = l / 16); the same fragment is
// both MFMA operands, so the result is X X^T.  Entry (m, n) of block b goes
// to part[(m*F + n) * n_blocks + b]: one entry's partials are contiguous.
// The launch also does the token-level preparation that would otherwise
// read x again (inv non-null: every wave covers whole tokens of C elements,
// C a multiple of 64, and writes inv[f*N + n] = 1/||token||, the sum of
// squares of the 16 lanes' fp32 partials in a fixed order), clears pack[0,
// n_pack) for the arg-max atomics, and converts wo to fp16 in the blocks
// past the Gram's (blockIdx.x >= gram_blocks).
template <bool TWO>
__global__ __launch_bounds__(256) void k_frame_gram(const uint16_t *__restrict__ x, int F, long D, int kw,
                                                     float *__restrict__ part, int gram_blocks, float *__restrict__ inv,
                                                     int C, unsigned long long *__restrict__ pack, long n_pack,
                                                     const uint4 *__restrict__ wo, long n8, uint4 *__restrict__ wo16) {
    __shared__ float red[GRAM_WAVES][FMAX * FMAX];
    if ((int)blockIdx.x >= gram_blocks) {
        const long nb = gridDim.x - gram_blocks;
        for (long i = (long)(blockIdx.x - gram_blocks) * blockDim.x + threadIdx.x; i < n8; i += nb * blockDim.x)
            wo16[i] = bf16x8_to_f16x8(wo[i]);
        return;
    }
    for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n_pack; i += (long)gram_blocks * blockDim.x)
        pack[i] = 0ull;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const long k_begin = ((long)blockIdx.x * GRAM_WAVES + wave) * kw;
    const long k_end = min(k_begin + kw, D);
    const int fr = lane & 15, g = lane >> 4;
    const uint16_t *row0 = fr < F ? x + (long)fr * D : nullptr;
    const uint16_t *row1 = (TWO && fr + 16 < F) ? x + (long)(fr + 16) * D : nullptr;
    f32x4 acc00 = {0, 0, 0, 0}, acc01 = {0, 0, 0, 0}, acc10 = {0, 0, 0, 0}, acc11 = {0, 0, 0, 0};
    const int csteps = C / 64;   // steps per token (norms)
    int left = csteps;
    float ss0 = 0.f, ss1 = 0.f;
    // this lane's 16-byte chunks of one 64-wide step (zero past the range)
    auto load = [&](long k, uint4 *v0, uint4 *v1) {
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            const long kk = k + g * 16 + t * 8;
            v0[t] = make_uint4(0, 0, 0, 0);
            v1[t] = make_uint4(0, 0, 0, 0);
            if (kk < k_end) {
                if (row0) v0[t] = *reinterpret_cast<const uint4 *>(row0 + kk);
                if (TWO && row1) v1[t] = *reinterpret_cast<const uint4 *>(row1 + kk);
            }
        }
    };
    // one step of loads ahead: step k+64 is in flight while step k is used
    uint4 nx0[2], nx1[2];
    if (k_begin < k_end) load(k_begin, nx0, nx1);
    for (long k = k_begin; k < k_end; k += 64) {
        bf16x8 a0[2], a1[2];
        uint4 r0[2], r1[2];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            r0[t] = nx0[t];
            r1[t] = nx1[t];
        }
        if (k + 64 < k_end) load(k + 64, nx0, nx1);
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            a0[t] = *reinterpret_cast<bf16x8 *>(&r0[t]);
            a1[t] = *reinterpret_cast<bf16x8 *>(&r1[t]);
        }
        if (inv != nullptr) {
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                const uint16_t *e0 = reinterpret_cast<const uint16_t *>(&r0[t]);
                const uint16_t *e1 = reinterpret_cast<const uint16_t *>(&r1[t]);
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const float f0 = bf2f(e0[j]);
                    ss0 = fmaf(f0, f0, ss0);
                    if (TWO) {
                        const float f1 = bf2f(e1[j]);
                        ss1 = fmaf(f1, f1, ss1);
                    }
                }
            }
            if (--left == 0) {
                // token k / C complete: lanes fr, fr+16, fr+32, fr+48 hold its partials
                left = csteps;
                float s0 = ss0 + __shfl_xor(ss0, 16, 64);
                s0 += __shfl_xor(s0, 32, 64);
                float s1 = 0.f;
                if (TWO) {
                    s1 = ss1 + __shfl_xor(ss1, 16, 64);
                    s1 += __shfl_xor(s1, 32, 64);
                }
                ss0 = ss1 = 0.f;
                const long n = k / C, N = D / C;
                if (g == 0) {
                    if (fr < F) inv[fr * N + n] = s0 > 0.f ? (float)(1.0 / sqrt((double)s0)) : 0.f;
                    if (TWO && fr + 16 < F) inv[(fr + 16) * N + n] = s1 > 0.f ? (float)(1.0 / sqrt((double)s1)) : 0.f;
                }
            }
        }
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            acc00 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0[t], a0[t], acc00, 0, 0, 0);
            if (TWO) {
                acc01 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0[t], a1[t], acc01, 0, 0, 0);
                acc10 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1[t], a0[t], acc10, 0, 0, 0);
                acc11 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1[t], a1[t], acc11, 0, 0, 0);
            }
        }
    }
    // lane holds rows m = 4*g + e, column n = lane % 16 of each 16x16 tile
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int m = 4 * g + e, n = fr;
        red[wave][m * FMAX + n] = acc00[e];
        if (TWO) {
            red[wave][m * FMAX + n + 16] = acc01[e];
            red[wave][(m + 16) * FMAX + n] = acc10[e];
            red[wave][(m + 16) * FMAX + n + 16] = acc11[e];
        } else {
            red[wave][m * FMAX + n + 16] = 0.f;
            red[wave][(m + 16) * FMAX + n] = 0.f;
            red[wave][(m + 16) * FMAX + n + 16] = 0.f;
        }
    }
    __syncthreads();
    for (int e = threadIdx.x; e < F * F; e += blockDim.x) {
        const int src = (e / F) * FMAX + e % F;
        float s = red[0][src];
#pragma unroll
        for (int w = 1; w < GRAM_WAVES; ++w) s += red[w][src];
        part[(long)e * gram_blocks + blockIdx.x] = s;
    }
}

// fp32 frames (small layers): one block per frame pair, fp64 accumulation,
// a single partial.
__global__ void k_frame_gram_f32(const float *__restrict__ x, int F, long D, float *__restrict__ part) {
    __shared__ double red[256];
    const int i = blockIdx.x / F, j = blockIdx.x % F;
    double s = 0.0;
    for (long k = threadIdx.x; k < D; k += blockDim.x) s += (double)x[(long)i * D + k] * (double)x[(long)j * D + k];
    red[threadIdx.x] = s;
    __syncthreads();
    for (int o = 128; o > 0; o >>= 1) {
        if ((int)threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
        __syncthreads();
    }
    if (threadIdx.x == 0) part[i * F + j] = (float)red[0];
}

// Gram entry e = sum of its n_part partials, in fp64, one wave per entry:
// lane l adds partials l, l+64, ... in order, then a fixed butterfly.
__global__ __launch_bounds__(256) void k_frame_reduce(const float *__restrict__ part, int n_part, int n_entries,
                                                      double *__restrict__ gram) {
    const int lane = threadIdx.x & 63;
    const int e = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (e >= n_entries) return;
    const float *pe = part + (long)e * n_part;
    double s = 0.0;
    for (int b = lane; b < n_part; b += 64) s += (double)pe[b];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
    if (lane == 0) gram[e] = s;
}

// Frame cosines from the Gram matrix, best matches of odd frames (one
// thread each), the R_f most redundant odd frames by rank (largest
// similarity first, smallest frame on ties), and then either the Frame Cache
// flags (flag / mtok per frame, when given) or, in pairing mode, the greedy
// one-to-one pairing in selection order (a wave arg-max over the free even
// frames per step) and the attention-unit table.  One block, F <= 32.  With
// kept_idx given (Frame Cache) the block also compacts: retained frames in
// ascending order become rows [k*N, k*N+N) (k = the frame's rank among the
// retained ones, at most n_seq), cached frames fill cached_idx in ascending
// order, and rmap maps every token to its row (-1 cached, -2 past n_seq).
__global__ __launch_bounds__(1024) void k_frame_final(const double *__restrict__ gram, int F, int R_f,
                                                      int pairing, double *__restrict__ fsim,
                                                      float *__restrict__ node_max, int32_t *__restrict__ node_idx,
                                                      int32_t *__restrict__ forder, int32_t *__restrict__ pairs,
                                                      int32_t *__restrict__ units, int32_t *__restrict__ flag,
                                                      int32_t *__restrict__ mtok, int N, int n_seq,
                                                      int32_t *__restrict__ kept_idx, int32_t *__restrict__ cached_idx,
                                                      int32_t *__restrict__ rmap) {
    __shared__ int fcached[FMAX], frank[FMAX];
    __shared__ double G[FMAX * FMAX];
    __shared__ double cs[FMAX * FMAX];
    __shared__ double bm[FMAX / 2];
    __shared__ int bidx[FMAX / 2];
    __shared__ int order[FMAX / 2];
    const int t = threadIdx.x;
    const int n_src = F / 2, n_dst = (F + 1) / 2;
    if (t < FMAX * FMAX) {
        const int i = t / FMAX, j = t % FMAX;
        G[t] = (i < F && j < F) ? gram[i * F + j] : 0.0;
    }
    __syncthreads();
    if (t < FMAX * FMAX) {
        const int i = t / FMAX, j = t % FMAX;
        double c = 0.0;
        if (i < F && j < F) {
            const double d = sqrt(G[i * FMAX + i]) * sqrt(G[j * FMAX + j]);
            c = d > 0.0 ? G[t] / d : 0.0;
        }
        cs[t] = c;
        fsim[t] = c;
    }
    __syncthreads();
    if (t < n_src) {
        const int s = 2 * t + 1;
        double best = -INFINITY;
        int bi = -1;
        for (int j = 0; j < n_dst; ++j) {
            const double c = cs[s * FMAX + 2 * j];
            if (c > best) { best = c; bi = 2 * j; }
        }
        bm[t] = best;
        bidx[t] = bi;
        node_max[t] = (float)best;
        node_idx[t] = bi;
    }
    __syncthreads();
    bool sel = false;
    if (t < n_src) {
        int rank = 0;
        for (int j = 0; j < n_src; ++j) rank += (bm[j] > bm[t] || (bm[j] == bm[t] && j < t)) ? 1 : 0;
        sel = rank < R_f;
        if (sel) {
            order[rank] = 2 * t + 1;
            forder[rank] = 2 * t + 1;
        }
    }
    if (flag != nullptr && t < F) {
        // Frame Cache: odd frame 2i+1 cached when selected, matched to its best even frame
        const bool odd = t & 1;
        bool c = false;
        int m = -1;
        if (odd) {
            const int i = t >> 1;
            int rank = 0;
            for (int j = 0; j < n_src; ++j) rank += (bm[j] > bm[i] || (bm[j] == bm[i] && j < i)) ? 1 : 0;
            c = rank < R_f;
            m = c ? bidx[i] : -1;
        }
        flag[t] = c ? 1 : 0;
        mtok[t] = m;
        fcached[t] = c ? 1 : 0;
    }
    if (flag != nullptr && kept_idx != nullptr) {
        __syncthreads();
        if (t == 0) {
            // rank of each frame among the retained, or among the cached, frames
            int k = 0, c = 0;
            for (int f = 0; f < F; ++f) frank[f] = fcached[f] ? c++ : k++;
        }
        __syncthreads();
        const int n_cf = F - n_seq;
        const long total = (long)F * N;
        for (long q = t; q < total; q += blockDim.x) {
            const int f = (int)(q / N), n = (int)(q - (long)f * N);
            const int r = frank[f];
            if (fcached[f]) {
                if (r < n_cf) cached_idx[(long)r * N + n] = (int)q;
                rmap[q] = -1;
            } else {
                const bool ok = r < n_seq;
                if (ok) kept_idx[(long)r * N + n] = (int)q;
                rmap[q] = ok ? r * N + n : -2;
            }
        }
    }
    if (!pairing) return;
    __syncthreads();
    if (t >= 64) return;
    // wave 0: lane j stands for even frame 2j
    const int lane = t;
    bool taken = false;
    int my_s = -1, my_d = -1;   // lane f < F: the pair whose smaller frame is f
    unsigned long long in_pair = 0ull;
    for (int r = 0; r < R_f; ++r) {
        const int s = order[r];
        double v = (lane < n_dst && !taken) ? cs[s * FMAX + 2 * lane] : -INFINITY;
        int ix = (lane < n_dst && !taken) ? lane : 64;
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
            const double v2 = __shfl_xor(v, o, 64);
            const int i2 = __shfl_xor(ix, o, 64);
            if (v2 > v || (v2 == v && i2 < ix)) { v = v2; ix = i2; }
        }
        const int d = 2 * ix;
        if (lane == ix) taken = true;
        if (lane == 0) {
            pairs[2 * r] = s;
            pairs[2 * r + 1] = d;
        }
        in_pair |= (1ull << s) | (1ull << d);
        if (lane == min(s, d)) {
            my_s = s;
            my_d = d;
        }
    }
    // attention units ordered by their smallest frame: frame f starts a unit
    // when it is in no pair or is the smaller frame of its pair
    const bool starts = lane < F && (!((in_pair >> lane) & 1ull) || my_s >= 0);
    const unsigned long long ballot = __builtin_amdgcn_ballot_w64(starts);
    const int u = __builtin_popcountll(ballot & ((1ull << lane) - 1ull));
    if (starts) {
        units[2 * u] = my_s >= 0 ? my_s : lane;
        units[2 * u + 1] = my_s >= 0 ? my_d : -1;
    }
}

hipError_t launch_frame_stage(const Plan &p, const Layout &L, const void *x, char *ws, float *node_max,
                              int32_t *node_idx, int32_t *flag, int32_t *mtok, float *inv,
                              unsigned long long *pack, long n_pack, const void *wo, void *wo16, int32_t *kept_idx,
                              int32_t *cached_idx, int32_t *rmap, hipStream_t st) {
    if (kept_idx != nullptr && (flag == nullptr || cached_idx == nullptr || rmap == nullptr)) return hipErrorInvalidValue;
    const long D = (long)p.N * p.C;
    int nb = gram_blocks(p);
    float *part = (float *)(ws + L.gram_part);
    if (!p.bf16) {
        nb = 1;
        {
            StageScope _stage(st, "frame_gram");
            launch_k(k_frame_gram_f32, p.F * p.F, 256, 0, st, (const float *)x, p.F, D, part);
        }
    } else {
        if (inv != nullptr && !gram_norms(p)) return hipErrorInvalidValue;
        const long n8 = (wo != nullptr && wo16 != nullptr) ? (long)p.C * p.hd / 8 : 0;
        const int cvt_blocks = n8 > 0 ? (int)std::min<long>((n8 + 255) / 256, 1024) : 0;
        StageScope _stage(st, "frame_gram");
        if (p.F > 16)
            launch_k(k_frame_gram<true>, nb + cvt_blocks, 256, 0, st, (const uint16_t *)x, p.F, D, gram_kw(p), part,
                     nb, inv, p.C, pack, pack ? n_pack : 0, (const uint4 *)wo, n8, (uint4 *)wo16);
        else
            launch_k(k_frame_gram<false>, nb + cvt_blocks, 256, 0, st, (const uint16_t *)x, p.F, D, gram_kw(p), part,
                     nb, inv, p.C, pack, pack ? n_pack : 0, (const uint4 *)wo, n8, (uint4 *)wo16);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    double *gram = (double *)(ws + L.fgram);
    {
        StageScope _stage(st, "frame_reduce");
        launch_k(k_frame_reduce, (unsigned)cdiv(p.F * p.F, 4), 256, 0, st, (const float *)part, nb, p.F * p.F, gram);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    {
        StageScope _stage(st, "frame_final");
        launch_k(k_frame_final, 1, 1024, 0, st, (const double *)gram, p.F, p.R_f, p.gran == 3 ? 1 : 0,
                 (double *)(ws + L.fsim), node_max, node_idx, (int32_t *)(ws + L.forder), (int32_t *)(ws + L.pairs),
                 (int32_t *)(ws + L.units), flag, mtok, p.N, p.n_seq, kept_idx, cached_idx, rmap);
    }
    return hipGetLastError();
}

}  // namespace oc
