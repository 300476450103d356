// Matching kernels: descriptor inverse norms and the similarity tile GEMM
// with a fused row arg-max (OmniCache §3.2.1-§3.2.3 cosine-similarity
// matching, patch-local per §3.3).  Group members come from GroupMap.
#include "oc_internal.h"
#include "oc_launch.h"
#include "oc_groups.h"
#include "oc_device.h"
#include "oc_mfma_tile.h"
#include "oc_dma_tile.h"
#include "oc_attn_common.h"
#include <algorithm>

namespace oc {

// ----------------------------------------------------------------------------
// inverse L2 norms of item descriptors: one wave per item, or one block per
// item for descriptors made of several segments (blocks: a position over all
// frames); blocks past the norm blocks convert the output-projection weights
// bf16 -> fp16 (exact in the fp16 normal range, saturating outside), 8
// elements per thread
// ----------------------------------------------------------------------------
// lanes per item for rows of `chunks` 16-byte chunks: the largest power of
// two not above chunks, between 8 and 64
__host__ __device__ inline int lanes_per_item(int chunks) {
    int l = 8;
    while (l < 64 && 2 * l <= chunks) l *= 2;
    return l;
}

template <typename T>
__global__ void k_inv_norm(const T *__restrict__ x, float *__restrict__ inv, int n_items, int n_sub,
                           long sub_stride, int C, int norm_blocks, unsigned long long *__restrict__ pack,
                           long n_pack, const uint4 *__restrict__ wo, long n8, uint4 *__restrict__ wo16) {
    if ((int)blockIdx.x >= norm_blocks) {
        const long nb = gridDim.x - norm_blocks;
        for (long i = (long)(blockIdx.x - norm_blocks) * blockDim.x + threadIdx.x; i < n8; i += nb * blockDim.x)
            wo16[i] = bf16x8_to_f16x8(wo[i]);
        return;
    }
    for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n_pack; i += (long)norm_blocks * blockDim.x)
        pack[i] = 0ull;
    constexpr int VEC = 16 / sizeof(T);
    const int lane = threadIdx.x & (WAVE - 1);
    if (n_sub > 1) {
        // block per item: the segments' 16-byte chunks spread over the block,
        // partial sums reduced in a fixed order
        __shared__ float wsum[4];
        const int item = blockIdx.x;
        const int cpr = C / VEC;
        float ss = 0.f;
        const int nq = n_sub * cpr;
        // four chunks' loads in flight before their sums (same order of
        // accumulation as one chunk at a time)
        for (int q0 = threadIdx.x; q0 < nq; q0 += 4 * blockDim.x) {
            // (a chunk past the end re-reads the last one, unbranched, and
            // its sum is dropped)
            uint4 v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int q = min(q0 + u * (int)blockDim.x, nq - 1);
                const int sg = q / cpr, c = (q - sg * cpr) * VEC;
                v[u] = *reinterpret_cast<const uint4 *>(x + sg * sub_stride + (long)item * C + c);
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const T *e = reinterpret_cast<const T *>(&v[u]);
                float part = ss;
#pragma unroll
                for (int j = 0; j < VEC; ++j) {
                    const float f = Elem<T>::ld(e + j);
                    part = fmaf(f, f, part);
                }
                ss = q0 + u * (int)blockDim.x < nq ? part : ss;
            }
        }
        ss = wave_sum(ss);
        if (lane == 0) wsum[threadIdx.x / WAVE] = ss;
        __syncthreads();
        if (threadIdx.x == 0) {
            const float t = (wsum[0] + wsum[1]) + (wsum[2] + wsum[3]);
            inv[item] = t > 0.f ? (float)(1.0 / sqrt((double)t)) : 0.f;
        }
        return;
    }
    // LPI lanes per item (a power of two up to 64, about one 16-byte chunk
    // per lane for short rows): 256 / LPI items per block
    const int lpi = lanes_per_item(C / VEC);
    const int sub = threadIdx.x & (lpi - 1);
    const int item = blockIdx.x * (blockDim.x / lpi) + threadIdx.x / lpi;
    if (item >= n_items) return;   // (whole lane groups: the reduction below stays inside one)
    const T *row = x + (long)item * C;
    float ss = 0.f;
    // up to four chunks' loads in flight before their sums (same order of
    // accumulation as one chunk at a time)
    const int step = lpi * VEC;
    for (int c0 = sub * VEC; c0 < C; c0 += 4 * step) {
        // (a chunk past the end re-reads the last one, unbranched, and its
        // sum is dropped)
        uint4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u)
            v[u] = *reinterpret_cast<const uint4 *>(row + min(c0 + u * step, C - VEC));
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const T *e = reinterpret_cast<const T *>(&v[u]);
            float part = ss;
#pragma unroll
            for (int j = 0; j < VEC; ++j) {
                const float f = Elem<T>::ld(e + j);
                part = fmaf(f, f, part);
            }
            ss = c0 + u * step < C ? part : ss;
        }
    }
    for (int o = lpi >> 1; o > 0; o >>= 1) ss += __shfl_xor(ss, o, WAVE);
    if (sub == 0) inv[item] = ss > 0.f ? (float)(1.0 / sqrt((double)ss)) : 0.f;
}

hipError_t launch_inv_norm(const Plan &p, const void *x, float *inv, unsigned long long *node_pack, long n_pack,
                           const void *wo, void *wo16, long n_wo, hipStream_t st) {
    StageScope _stage(st, "inv_norm");
    const int n_items = p.kind == KIND_BLOCK ? p.N : p.F * p.N;
    const int n_sub = p.kind == KIND_BLOCK ? p.F : 1;
    const long sub = (long)p.N * p.C;
    const int chunks = p.C / (p.bf16 ? 8 : 4);
    const int blocks = n_sub > 1 ? n_items : cdiv(n_items, 256 / lanes_per_item(chunks));
    const long n8 = (wo && wo16 && p.bf16) ? n_wo / 8 : 0;
    const int cvt_blocks = n8 > 0 ? (int)std::min<long>((n8 + 255) / 256, 1024) : 0;
    if (p.bf16)
        launch_k(k_inv_norm<uint16_t>, blocks + cvt_blocks, 256, 0, st, (const uint16_t *)x, inv, n_items, n_sub, sub, p.C,
                                                                 blocks, node_pack, n_pack, (const uint4 *)wo, n8,
                                                                 (uint4 *)wo16);
    else
        launch_k(k_inv_norm<float>, blocks, 256, 0, st, (const float *)x, inv, n_items, n_sub, sub, p.C, blocks, node_pack,
                                                  n_pack, nullptr, 0, nullptr);
    return hipGetLastError();
}

// Frame Cache on patches: one block per (frame, patch) tile, the sum of
// squares of its ph rows of pw*C elements (16-byte chunks spread over the
// block, wave partials added in a fixed order), stored at the tile's
// top-left token; the blocks past the tiles clear pack and convert wo.
template <typename T>
__global__ void k_tile_norm(const T *__restrict__ x, float *__restrict__ inv, int F, int N, int W, int k, int ph,
                            int pw, int C, int norm_blocks, unsigned long long *__restrict__ pack, long n_pack,
                            const uint4 *__restrict__ wo, long n8, uint4 *__restrict__ wo16) {
    if ((int)blockIdx.x >= norm_blocks) {
        const long nb = gridDim.x - norm_blocks;
        for (long i = (long)(blockIdx.x - norm_blocks) * blockDim.x + threadIdx.x; i < n8; i += nb * blockDim.x)
            wo16[i] = bf16x8_to_f16x8(wo[i]);
        return;
    }
    for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n_pack; i += (long)norm_blocks * blockDim.x)
        pack[i] = 0ull;
    constexpr int VEC = 16 / sizeof(T);
    __shared__ float wsum[4];
    const int kk = k * k, f = blockIdx.x / kk, g = blockIdx.x - f * kk;
    const long tl = (long)f * N + (long)(g / k) * ph * W + (g % k) * pw;
    const int cpr = pw * C / VEC;                  // chunks per tile row
    float ss = 0.f;
    for (int q = threadIdx.x; q < ph * cpr; q += blockDim.x) {
        const int row = q / cpr, c = (q - row * cpr) * VEC;
        const uint4 v = *reinterpret_cast<const uint4 *>(x + (tl + (long)row * W) * C + c);
        const T *e = reinterpret_cast<const T *>(&v);
#pragma unroll
        for (int j = 0; j < VEC; ++j) {
            const float fv = Elem<T>::ld(e + j);
            ss = fmaf(fv, fv, ss);
        }
    }
    ss = wave_sum(ss);
    if ((threadIdx.x & (WAVE - 1)) == 0) wsum[threadIdx.x / WAVE] = ss;
    __syncthreads();
    if (threadIdx.x == 0) {
        const float t = (wsum[0] + wsum[1]) + (wsum[2] + wsum[3]);
        inv[tl] = t > 0.f ? (float)(1.0 / sqrt((double)t)) : 0.f;
    }
}

hipError_t launch_tile_norm(const Plan &p, const void *x, float *inv, unsigned long long *node_pack, long n_pack,
                            const void *wo, void *wo16, long n_wo, hipStream_t st) {
    StageScope _stage(st, "inv_norm");
    const int blocks = p.F * p.k * p.k;
    const long n8 = (wo && wo16 && p.bf16) ? n_wo / 8 : 0;
    const int cvt_blocks = n8 > 0 ? (int)std::min<long>((n8 + 255) / 256, 1024) : 0;
    if (p.bf16)
        launch_k(k_tile_norm<uint16_t>, blocks + cvt_blocks, 256, 0, st, (const uint16_t *)x, inv, p.F, p.N, p.W, p.k,
                 p.ph, p.pw, p.C, blocks, node_pack, n_pack, (const uint4 *)wo, n8, (uint4 *)wo16);
    else
        launch_k(k_tile_norm<float>, blocks, 256, 0, st, (const float *)x, inv, p.F, p.N, p.W, p.k, p.ph, p.pw, p.C,
                 blocks, node_pack, n_pack, nullptr, 0, nullptr);
    return hipGetLastError();
}

// ----------------------------------------------------------------------------
// similarity + arg-max, bf16 MFMA
// ----------------------------------------------------------------------------
// Block (candidate tile bt, representative tile at, group g), in an
// XCD-aware order: t = dot(src_b, dst_a) * inv(dst_a); per candidate the
// largest t over this block's representatives (smallest position on ties)
// is merged into node_pack[g][b] with one 64-bit atomic maximum of the
// packed pair, so the representative tiles need no second pass.  The
// representative norm is applied before the arg-max, the candidate's own
// norm (a positive constant per row) when unpacking.
template <int BA, int BB, int WA, int WB, bool DMA>
using MatchTile = typename std::conditional<DMA, DmaTile<BA, BB, WA, WB, false, 2>, MfmaTile<BA, BB, WA, WB>>::type;

template <int BA, int BB, int WA, int WB, bool DMA>
__global__ __launch_bounds__(256) void k_match_mfma(const uint16_t *__restrict__ x, const float *__restrict__ inv,
                                                     GroupMap gm, int G, int S, int D,
                                                     int K, int seg_len, long sub_stride, long item_stride,
                                                     int n_bt, int n_at,
                                                     unsigned long long *__restrict__ node_pack) {
    using T = MatchTile<BA, BB, WA, WB, DMA>;
    extern __shared__ __align__(16) uint16_t lds[];
    const int total = n_bt * n_at * G;
    const int lid = xcd_remap(blockIdx.x, total);
    // consecutive logical blocks: the representative tiles of one candidate tile
    const int at = lid % n_at, bt = (lid / n_at) % n_bt, g = lid / (n_at * n_bt);
    const GroupMap::Grp gr = gm.group(g);
    if (bt * BB >= gr.nsrc) return;   // past this group's candidates (groups of one call differ in size)
    const uint16_t *rowsA[T::CA], *rowsB[T::CB];
#pragma unroll
    for (int i = 0; i < T::CA; ++i) {
        const int a = at * BA + T::chunk_row(i);
        const int id = a < D ? gm.dst_id(gr, a) : -1;
        rowsA[i] = id >= 0 ? x + (long)id * item_stride : nullptr;
    }
#pragma unroll
    for (int i = 0; i < T::CB; ++i) {
        const int b = bt * BB + T::chunk_row(i);
        const int id = b < S ? gm.src_id(gr, b) : -1;
        rowsB[i] = id >= 0 ? x + (long)id * item_stride : nullptr;
    }
    T tile;
    // rows without an item read x's first row (DMA) or zeros; either way
    // their results are discarded below
    if constexpr (DMA) tile.run(lds, rowsA, rowsB, x, x, K, seg_len, sub_stride);
    else tile.run(lds, rowsA, rowsB, K, seg_len, sub_stride);

    // representative norms of this tile (0 for padding, which never wins)
    float *sinv = reinterpret_cast<float *>(lds);
    float *sv = sinv + BA;
    int *si = reinterpret_cast<int *>(sv + WA * BB);
    for (int a = threadIdx.x; a < BA; a += 256) {
        const int ga = at * BA + a;
        const int id = ga < D ? gm.dst_id(gr, ga) : -1;
        sinv[a] = id >= 0 ? inv[id] : -1.f;
    }
    __syncthreads();
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wa = wave / WB;
#pragma unroll
    for (int j = 0; j < T::TB; ++j) {
        float bv = -INFINITY;
        int bi = -1;
#pragma unroll
        for (int i = 0; i < T::TA; ++i)
#pragma unroll
            for (int g4 = 0; g4 < 4; ++g4)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int al = T::a_of(i, g4) + e;
                    const float w = sinv[al];
                    if (w >= 0.f) argmax_merge(bv, bi, tile.acc[i][j][4 * g4 + e] * w, at * BA + al);
                }
        const float v2 = __shfl_xor(bv, 32, WAVE);
        const int i2 = __shfl_xor(bi, 32, WAVE);
        argmax_merge(bv, bi, v2, i2);
        if (lane < 32) {
            const int bl = T::b_of(j);
            sv[wa * BB + bl] = bv;
            si[wa * BB + bl] = bi;
        }
    }
    __syncthreads();
    // merge the WA waves that share a candidate range, in ascending a order
    for (int bl = threadIdx.x; bl < BB; bl += 256) {
        float v = sv[bl];
        int ix = si[bl];
        for (int w = 1; w < WA; ++w) argmax_merge(v, ix, sv[w * BB + bl], si[w * BB + bl]);
        const int b = bt * BB + bl;
        if (b < S && ix >= 0) atomicMax(&node_pack[(long)g * S + b], pack_argmax(v, ix));
    }
}

// Sweep variant for many candidate tiles and several representative tiles:
// block (candidate tile bt, group g) streams every representative tile (and
// its candidates again, from L2) through one continuous double-buffered
// LDS-DMA pipeline (small enough for two blocks per CU), keeps each
// candidate's best (value, position) in registers and publishes it once (one
// 64-bit atomic maximum per candidate).  The representative tiles of one
// candidate tile are split over n_part consecutive blocks (adjacent logical
// blocks run on one XCD at the same time, so they share the candidate rows
// in its L2 instead of each block re-reading its own tile from memory for
// every representative tile); their atomics merge the parts.  The group's
// representative norms are staged in LDS first (D <= SWEEP_MAX_D).
template <int BA, int BB, int WA, int WB>
__global__ __launch_bounds__(256) void k_match_sweep(const uint16_t *__restrict__ x, const float *__restrict__ inv,
                                                      GroupMap gm, int G, int S, int D, int K, int seg_len,
                                                      long sub_stride, long item_stride, int n_bt, int n_at,
                                                      int n_part, unsigned long long *__restrict__ node_pack) {
    using T = DmaTile<BA, BB, WA, WB, false, 2>;
    extern __shared__ __align__(16) uint16_t lds[];
    float *const snorm = reinterpret_cast<float *>(lds + T::LDS_BYTES / 2);   // n_at * BA norms after the ring
    __shared__ float sv[WA * BB];
    __shared__ int si[WA * BB];
    const int lid = xcd_remap(blockIdx.x, n_bt * G * n_part);
    const int part = lid % n_part, tl = lid / n_part;
    const int bt = tl % n_bt, g = tl / n_bt;
    const int u0 = part * n_at / n_part, u1 = (part + 1) * n_at / n_part;   // this block's representative tiles
    const GroupMap::Grp gr = gm.group(g);
    if (bt * BB >= gr.nsrc || u0 >= u1) return;
    for (int a = threadIdx.x; a < n_at * BA; a += 256) {
        const int id = a < D ? gm.dst_id(gr, a) : -1;
        snorm[a] = id >= 0 ? inv[id] : -1.f;
    }
    __syncthreads();
    const uint16_t *rowsB[T::CB];
#pragma unroll
    for (int i = 0; i < T::CB; ++i) {
        const int b = bt * BB + T::chunk_row(i);
        const int id = b < S ? gm.src_id(gr, b) : -1;
        rowsB[i] = id >= 0 ? x + (long)id * item_stride : nullptr;
    }
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wa = wave / WB;
    float bv[T::TB];
    int bi[T::TB];
#pragma unroll
    for (int j = 0; j < T::TB; ++j) {
        bv[j] = -INFINITY;
        bi[j] = -1;
    }
    T tile;
    auto rows_a = [&](int u, int i) -> const uint16_t * {
        const int a = (u0 + u) * BA + T::chunk_row(i);
        const int id = a < D ? gm.dst_id(gr, a) : -1;
        return id >= 0 ? x + (long)id * item_stride : nullptr;
    };
    // per tile: scale by the representative norms, take the tile maximum per
    // candidate and lane half, and only when it beats the running best find
    // its smallest position (tiles come in ascending position, so a later
    // equal value never replaces an earlier one); the lane halves are merged
    // once at the end
    const int d_full = D - BA;   // tiles starting at or below this have only valid representatives
    auto epi = [&](int ul) {
        const int u = u0 + ul;
        const bool full = u * BA <= d_full && gm.dst_id(gr, u * BA + BA - 1) >= 0;
#pragma unroll
        for (int j = 0; j < T::TB; ++j)
#pragma unroll
            for (int i = 0; i < T::TA; ++i) {
                float t[16];
#pragma unroll
                for (int g4 = 0; g4 < 4; ++g4) {
                    const int al = u * BA + T::a_of(i, g4);
                    const float4 w = *reinterpret_cast<const float4 *>(&snorm[al]);
                    const float wv[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        float v = tile.acc[i][j][4 * g4 + e] * wv[e];
                        if (!full && wv[e] < 0.f) v = -INFINITY;
                        t[4 * g4 + e] = v;
                    }
                }
                float m = t[0];
#pragma unroll
                for (int k = 1; k < 16; ++k) m = fmaxf(m, t[k]);
                if (m > bv[j]) {
                    int ix = -1;
#pragma unroll
                    for (int k = 15; k >= 0; --k)
                        if (t[k] == m) ix = u * BA + T::a_of(i, k >> 2) + (k & 3);
                    bv[j] = m;
                    bi[j] = ix;
                }
            }
    };
    tile.run_tiles(lds, rows_a, rowsB, x, x, K, seg_len, sub_stride, u1 - u0, epi);
#pragma unroll
    for (int j = 0; j < T::TB; ++j) argmax_merge(bv[j], bi[j], __shfl_xor(bv[j], 32, WAVE), __shfl_xor(bi[j], 32, WAVE));
    if (lane < 32) {
#pragma unroll
        for (int j = 0; j < T::TB; ++j) {
            const int bl = T::b_of(j);
            sv[wa * BB + bl] = bv[j];
            si[wa * BB + bl] = bi[j];
        }
    }
    __syncthreads();
    for (int bl = threadIdx.x; bl < BB; bl += 256) {
        float v = sv[bl];
        int ix = si[bl];
        for (int w = 1; w < WA; ++w) argmax_merge(v, ix, sv[w * BB + bl], si[w * BB + bl]);
        const int b = bt * BB + bl;
        if (b < S && ix >= 0) atomicMax(&node_pack[(long)g * S + b], pack_argmax(v, ix));
    }
}

// Split-K variant for long descriptors and few tiles (Block Cache: a
// position's descriptor spans all frames): block (tile, split) computes the
// raw dot products over its K range (whole 64-steps inside one segment) and
// stores them to part[split][g][b][a]; k_match_part_reduce sums the splits in
// order, applies the representative norms and takes the arg-max.
template <int BA, int BB, int WA, int WB, bool DMA>
__global__ __launch_bounds__(256) void k_match_part(const uint16_t *__restrict__ x, GroupMap gm, int G, int S, int D,
                                                     int kc, int seg_len, long sub_stride, long item_stride,
                                                     int n_bt, int n_at, int n_split, float *__restrict__ part) {
    using T = MatchTile<BA, BB, WA, WB, DMA>;
    extern __shared__ __align__(16) uint16_t lds[];
    const int total = n_bt * n_at * G * n_split;
    const int lid = xcd_remap(blockIdx.x, total);
    const int sp = lid % n_split, tl = lid / n_split;
    const int at = tl % n_at, bt = (tl / n_at) % n_bt, g = tl / (n_at * n_bt);
    const GroupMap::Grp gr = gm.group(g);
    if (bt * BB >= gr.nsrc) return;
    // K range of this split: inside one segment
    const long k0 = (long)sp * kc;
    const long off = seg_len > 0 ? (k0 / seg_len) * sub_stride + (k0 % seg_len) : k0;
    const uint16_t *rowsA[T::CA], *rowsB[T::CB];
#pragma unroll
    for (int i = 0; i < T::CA; ++i) {
        const int a = at * BA + T::chunk_row(i);
        const int id = a < D ? gm.dst_id(gr, a) : -1;
        rowsA[i] = id >= 0 ? x + (long)id * item_stride + off : nullptr;
    }
#pragma unroll
    for (int i = 0; i < T::CB; ++i) {
        const int b = bt * BB + T::chunk_row(i);
        const int id = b < S ? gm.src_id(gr, b) : -1;
        rowsB[i] = id >= 0 ? x + (long)id * item_stride + off : nullptr;
    }
    T tile;
    if constexpr (DMA) tile.run(lds, rowsA, rowsB, x, x, kc, 0, 0);
    else tile.run(lds, rowsA, rowsB, kc, 0, 0);
    float *pp = part + ((long)sp * G + g) * S * D;
#pragma unroll
    for (int j = 0; j < T::TB; ++j) {
        const int b = bt * BB + T::b_of(j);
        if (b >= S) continue;
#pragma unroll
        for (int i = 0; i < T::TA; ++i)
#pragma unroll
            for (int g4 = 0; g4 < 4; ++g4)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int a = at * BA + T::a_of(i, g4) + e;
                    if (a < D) pp[(long)b * D + a] = tile.acc[i][j][4 * g4 + e];
                }
    }
}

// One block per (group, candidate): wave q sums the splits q, q+4, ... of
// representatives a = lane + 64c, wave 0 adds the four partial sums in order,
// applies the representative norm and keeps the arg-max.
__global__ __launch_bounds__(256) void k_match_part_reduce(const float *__restrict__ part, int n_split, int G, int S,
                                                            int D, const float *__restrict__ inv, GroupMap gm,
                                                            unsigned long long *__restrict__ node_pack) {
    __shared__ float red[4][64];
    const int lane = threadIdx.x & 63, q = threadIdx.x >> 6;
    const int g = blockIdx.x / S, b = blockIdx.x - g * S;
    const GroupMap::Grp gr = gm.group(g);
    if (gm.src_id(gr, b) < 0) return;
    float bv = -INFINITY;
    int bi = -1;
    for (int a0 = 0; a0 < D; a0 += 64) {
        const int a = a0 + lane;
        float sum = 0.f;
        if (a < D) {
            // splits q, q+4, ... added in ascending order; the loads of eight
            // of them are issued before the first is added
            const long stride = 4L * G * S * D;
            const float *pp = part + (((long)q * G + g) * S + b) * D + a;
            for (int sp0 = q; sp0 < n_split; sp0 += 32, pp += 8 * stride) {
                float v[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) v[u] = sp0 + 4 * u < n_split ? pp[u * stride] : 0.f;
#pragma unroll
                for (int u = 0; u < 8; ++u)
                    if (sp0 + 4 * u < n_split) sum += v[u];
            }
        }
        red[q][lane] = sum;
        __syncthreads();
        if (q == 0 && a < D) {
            const int id = gm.dst_id(gr, a);
            const float dot = ((red[0][lane] + red[1][lane]) + red[2][lane]) + red[3][lane];
            if (id >= 0) argmax_merge(bv, bi, dot * inv[id], a);
        }
        __syncthreads();
    }
    if (q != 0) return;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) argmax_merge(bv, bi, __shfl_xor(bv, o, WAVE), __shfl_xor(bi, o, WAVE));
    if (lane == 0 && bi >= 0) node_pack[(long)g * S + b] = pack_argmax(bv, bi);
}

// fp32 similarity + arg-max (small fp32 layers): one thread per candidate.
__global__ void k_match_f32(const float *__restrict__ x, const float *__restrict__ inv, GroupMap gm, int /*G*/, int S,
                            int D, int K, int seg_len, long sub_stride, long item_stride,
                            unsigned long long *__restrict__ node_pack) {
    const int g = blockIdx.y;
    const int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= S) return;
    const GroupMap::Grp gr = gm.group(g);
    const int sid = gm.src_id(gr, b);
    float bv = -INFINITY;
    int bi = -1;
    if (sid >= 0) {
        const float *u = x + (long)sid * item_stride;
        for (int a = 0; a < D; ++a) {
            const int did = gm.dst_id(gr, a);
            if (did < 0) continue;
            const float *v = x + (long)did * item_stride;
            float dot = 0.f;
            for (int kk = 0; kk < K; ++kk) {
                long off = kk;
                if (seg_len > 0) { const int s = kk / seg_len; off = (long)s * sub_stride + (kk - s * seg_len); }
                dot = fmaf(u[off], v[off], dot);
            }
            argmax_merge(bv, bi, dot * inv[did], a);
        }
    }
    node_pack[(long)g * S + b] = bi >= 0 ? pack_argmax(bv, bi) : 0ull;
}

// Unpack the best pair, convert the winning position to a global id and
// apply the candidate's norm.
__global__ void k_match_unpack(const unsigned long long *__restrict__ node_pack, int G, int S,
                               const float *__restrict__ inv, GroupMap gm, float *__restrict__ node_max,
                               int32_t *__restrict__ node_idx) {
    const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (long)G * S) return;
    const int g = (int)(i / S);
    const GroupMap::Grp gr = gm.group(g);
    const int sid = gm.src_id(gr, (int)(i - (long)g * S));
    if (sid < 0) {
        node_max[i] = -INFINITY;
        node_idx[i] = -1;
        return;
    }
    float v;
    int ix;
    unpack_argmax(node_pack[i], v, ix);
    node_max[i] = v * inv[sid];
    node_idx[i] = ix >= 0 ? gm.dst_id(gr, ix) : -1;
}

template <typename KernelPtr>
static hipError_t allow_lds(KernelPtr k, size_t lds) {
    return raise_lds_limit((const void *)k, lds);
}

template <int BA, int BB, int WA, int WB, bool DMA>
static hipError_t go_match(const Plan &p, const uint16_t *x, const float *inv, const GroupMap &gm, int K,
                           int seg_len, long sub_stride, long item_stride, unsigned long long *node_pack,
                           hipStream_t st) {
    using T = MatchTile<BA, BB, WA, WB, DMA>;
    const int G = p.n_groups, S = p.n_src_max, D = p.n_dst_max;
    const int n_bt = cdiv(S, BB), n_at = cdiv(D, BA);
    const size_t lds = T::LDS_BYTES;
    hipError_t e = allow_lds(k_match_mfma<BA, BB, WA, WB, DMA>, lds);
    if (e != hipSuccess) return e;
    launch_k(k_match_mfma<BA, BB, WA, WB, DMA>, n_bt * n_at * G, 256, lds, st, x, inv, gm, G, S, D, K, seg_len,
             sub_stride, item_stride, n_bt, n_at, node_pack);
    return hipGetLastError();
}

template <int BA, int BB, int WA, int WB>
static hipError_t go_sweep(const Plan &p, const uint16_t *x, const float *inv, const GroupMap &gm, int K,
                           int seg_len, long sub_stride, long item_stride, unsigned long long *node_pack,
                           hipStream_t st) {
    using T = DmaTile<BA, BB, WA, WB, false, 2>;
    const int G = p.n_groups, S = p.n_src_max, D = p.n_dst_max;
    const int n_bt = cdiv(S, BB), n_at = cdiv(D, BA);
    if (n_at * BA > SWEEP_MAX_D) return hipErrorInvalidValue;
    const size_t lds = T::LDS_BYTES + (size_t)n_at * BA * 4;
    hipError_t e = allow_lds(k_match_sweep<BA, BB, WA, WB>, lds);
    if (e != hipSuccess) return e;
    // two blocks per candidate tile once each keeps three or more
    // representative tiles (SVD-XT-like frames: 8x less memory traffic than
    // one block, 203 against 1627 MiB per launch, at the same time; three or
    // six parts measured no faster)
    const int n_part = n_at >= 6 ? 2 : 1;
    launch_k(k_match_sweep<BA, BB, WA, WB>, n_bt * G * n_part, 256, lds, st, x, inv, gm, G, S, D, K, seg_len,
             sub_stride, item_stride, n_bt, n_at, n_part, node_pack);
    return hipGetLastError();
}

template <int BA, int BB, int WA, int WB, bool DMA>
static hipError_t go_split(const Plan &p, const MatchSplit &ms, const uint16_t *x, const float *inv,
                           const GroupMap &gm, int seg_len, long sub_stride, long item_stride, float *part,
                           unsigned long long *node_pack, hipStream_t st) {
    using T = MatchTile<BA, BB, WA, WB, DMA>;
    const int G = p.n_groups, S = p.n_src_max, D = p.n_dst_max;
    const int n_bt = cdiv(S, BB), n_at = cdiv(D, BA);
    const size_t lds = T::LDS_BYTES;
    hipError_t e = allow_lds(k_match_part<BA, BB, WA, WB, DMA>, lds);
    if (e != hipSuccess) return e;
    launch_k(k_match_part<BA, BB, WA, WB, DMA>, n_bt * n_at * G * ms.n_split, 256, lds, st, x, gm, G, S, D, ms.kc,
             seg_len, sub_stride, item_stride, n_bt, n_at, ms.n_split, part);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    launch_k(k_match_part_reduce, (unsigned)((long)G * S), 256, 0, st, (const float *)part, ms.n_split, G, S, D, inv,
             gm, node_pack);
    return hipGetLastError();
}

hipError_t launch_match(const Plan &p, const void *x, const float *inv, const int32_t *units,
                        unsigned long long *node_pack, float *part, float *node_max, int32_t *node_idx,
                        hipStream_t st) {
    const GroupMap gm = group_map(p, units);
    const int G = p.n_groups, S = p.n_src_max, D = p.n_dst_max;
    const MatchGeom mg = match_geom(p);
    const int K = mg.K;
    const int seg_len = mg.seg_len;
    const long sub_stride = mg.sub_stride;
    const long item_stride = mg.item_stride;
    {
        StageScope _stage(st, "match");
        if (p.bf16) {
            const uint16_t *xb = (const uint16_t *)x;
            const MatchSplit ms = match_split(p);
            const bool dma = K % 64 == 0 && (seg_len == 0 || seg_len % 64 == 0);
            hipError_t e;
            if (ms.n_split > 1) {
                // long descriptors, few tiles: split K (64-row tiles)
                e = go_split<64, 64, 2, 2, true>(p, ms, xb, inv, gm, seg_len, sub_stride, item_stride, part,
                                                 node_pack, st);
            } else if (D > 64 && dma && match_sweeps(p)) {
                // many candidate tiles: each block sweeps all representative tiles
                e = go_sweep<128, 128, 2, 2>(p, xb, inv, gm, K, seg_len, sub_stride, item_stride, node_pack,
                                                   st);
            } else if (D > 64 && dma && (long)cdiv(D, 128) * cdiv(S, 64) * G < 2L * N_CUS) {
                // a 128 x 64 grid under two blocks per CU: 64 x 64 tiles, three
                // to five per CU (the SD3-like layer: 768 blocks, 20 against 23 us)
                e = go_match<64, 64, 2, 2, true>(p, xb, inv, gm, K, seg_len, sub_stride, item_stride, node_pack,
                                                 st);
            } else if (D > 64) {
                // representative tile height by group size: 128, 64 or 32; large
                // groups stream by LDS DMA when the K steps allow it
                e = dma ? go_match<128, 64, 2, 2, true>(p, xb, inv, gm, K, seg_len, sub_stride, item_stride,
                                                        node_pack, st)
                        : go_match<128, 64, 2, 2, false>(p, xb, inv, gm, K, seg_len, sub_stride, item_stride,
                                                         node_pack, st);
            } else if (D > 32) {
                e = go_match<64, 64, 2, 2, false>(p, xb, inv, gm, K, seg_len, sub_stride, item_stride, node_pack,
                                                  st);
            } else {
                e = go_match<32, 128, 1, 4, false>(p, xb, inv, gm, K, seg_len, sub_stride, item_stride, node_pack,
                                                   st);
            }
            if (e != hipSuccess) return e;
        } else {
            dim3 grid(cdiv(S, 64), G);
            launch_k(k_match_f32, grid, 64, 0, st, (const float *)x, inv, gm, G, S, D, K, seg_len, sub_stride,
                     item_stride, node_pack);
        }
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || node_max == nullptr) return e;   // no outputs: the selection unpacks node_pack
    const long n = (long)G * S;
    {
        StageScope _stage(st, "match_unpack");
        launch_k(k_match_unpack, (unsigned)cdiv((int)n, 256), 256, 0, st, node_pack, G, S, inv, gm, node_max, node_idx);
    }
    return hipGetLastError();
}

}  // namespace oc
