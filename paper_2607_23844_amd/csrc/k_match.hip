// Matching kernels: group id lists, descriptor inverse norms, and the
// similarity tile GEMM with a fused row arg-max (OmniCache §3.2.1-§3.2.3
// cosine-similarity matching, patch-local per §3.3).
#include "oc_internal.h"
#include "oc_device.h"
#include "oc_mfma_tile.h"
#include "oc_attn_common.h"

namespace oc {

// ----------------------------------------------------------------------------
// group id lists
// ----------------------------------------------------------------------------
// Unit u covers frame s (and frame d for a frame pair, d = -1 otherwise);
// group g = u * k*k + patch.  Candidates are listed in ascending global id,
// representatives (top-left token of each 2x2 window, in frame d for a pair)
// likewise.  BLOCK groups use spatial positions as ids (frame term 0).

__device__ __forceinline__ void patch_tok(int i, int pw, int &y, int &x) { y = i / pw; x = i - y * pw; }
__device__ __forceinline__ void patch_nonrep(int i, int pw, int &y, int &x) {
    const int per2 = 3 * pw / 2, q = i / per2, rem = i - q * per2;
    if (rem < pw / 2) { y = 2 * q; x = 2 * rem + 1; }
    else { y = 2 * q + 1; x = rem - pw / 2; }
}
__device__ __forceinline__ void patch_rep(int i, int pw, int &y, int &x) {
    const int h = pw / 2, q = i / h;
    y = 2 * q; x = 2 * (i - q * h);
}

__global__ void k_group_ids(int kind, int F, int N, int W, int k, int ph, int pw, int np, int np_src, int np_dst,
                            int S, int D, int R_tok, int R_pair, const int32_t *__restrict__ units,
                            int32_t *__restrict__ src_ids, int32_t *__restrict__ dst_ids,
                            int32_t *__restrict__ grp_R) {
    const int g = blockIdx.x;
    const int kk = k * k;
    const int u = g / kk, patch = g - u * kk;
    const int oy = (patch / k) * ph, ox = (patch % k) * pw;
    int s = u, d = -1;
    if (units != nullptr) { s = units[2 * u]; d = units[2 * u + 1]; }
    const long fbase = (kind == KIND_BLOCK) ? 0 : (long)N;
    const bool bad = units != nullptr && (s < 0 || s >= F || d >= F || s == d);   // malformed unit table
    if (bad) { s = 0; d = -1; }
    const bool pair = d >= 0;
    const int a = pair ? min(s, d) : s, b = pair ? max(s, d) : -1;
    const int n_a = (pair && a == d) ? np_src : np;   // tokens of frame a in the list
    const int nsrc = pair ? np + np_src : np_src;
    for (int i = threadIdx.x; i < S; i += blockDim.x) {
        int id = -1;
        if (i < nsrc) {
            int f, y, x;
            if (!pair) { f = s; patch_nonrep(i, pw, y, x); }
            else if (i < n_a) { f = a; if (a == d) patch_nonrep(i, pw, y, x); else patch_tok(i, pw, y, x); }
            else { f = b; const int j = i - n_a; if (b == d) patch_nonrep(j, pw, y, x); else patch_tok(j, pw, y, x); }
            id = (int)(f * fbase + (long)(oy + y) * W + (ox + x));
        }
        src_ids[(long)g * S + i] = id;
    }
    const int rf = pair ? d : s;
    for (int i = threadIdx.x; i < D; i += blockDim.x) {
        int id = -1;
        if (i < np_dst) {
            int y, x;
            patch_rep(i, pw, y, x);
            id = (int)(rf * fbase + (long)(oy + y) * W + (ox + x));
        }
        dst_ids[(long)g * D + i] = id;
    }
    if (threadIdx.x == 0) grp_R[g] = pair ? R_pair : R_tok;
}

__global__ void k_frame_ids(int F, int S, int D, int R, int32_t *src_ids, int32_t *dst_ids, int32_t *grp_R) {
    for (int i = threadIdx.x; i < S; i += blockDim.x) src_ids[i] = 2 * i + 1 < F ? 2 * i + 1 : -1;
    for (int i = threadIdx.x; i < D; i += blockDim.x) dst_ids[i] = 2 * i < F ? 2 * i : -1;
    if (threadIdx.x == 0) grp_R[0] = R;
}

hipError_t launch_group_ids(const Plan &p, const int32_t *units, int32_t *src_ids, int32_t *dst_ids,
                            int32_t *grp_R, hipStream_t st) {
    StageScope _stage(st, "group_ids");
    if (p.kind == KIND_FRAME) {
        k_frame_ids<<<1, 64, 0, st>>>(p.F, p.n_src_max, p.n_dst_max, p.R_f, src_ids, dst_ids, grp_R);
    } else {
        k_group_ids<<<p.n_groups, 256, 0, st>>>(p.kind, p.F, p.N, p.W, p.k, p.ph, p.pw, p.np, p.np_src, p.np_dst,
                                                p.n_src_max, p.n_dst_max, p.R_tok, p.R_pair, units, src_ids,
                                                dst_ids, grp_R);
    }
    return hipGetLastError();
}

// ----------------------------------------------------------------------------
// inverse L2 norms of item descriptors (one wave per item)
// ----------------------------------------------------------------------------
template <typename T>
__global__ void k_inv_norm(const T *__restrict__ x, float *__restrict__ inv, int n_items, int n_sub,
                           long sub_stride, int C) {
    constexpr int VEC = 16 / sizeof(T);
    const int item = blockIdx.x * (blockDim.x / WAVE) + (threadIdx.x / WAVE);
    const int lane = threadIdx.x & (WAVE - 1);
    if (item >= n_items) return;
    float ss = 0.f;
    for (int s = 0; s < n_sub; ++s) {
        const T *row = x + s * sub_stride + (long)item * C;
        for (int c = lane * VEC; c < C; c += WAVE * VEC) {
            const uint4 v = *reinterpret_cast<const uint4 *>(row + c);
            const T *e = reinterpret_cast<const T *>(&v);
#pragma unroll
            for (int j = 0; j < VEC; ++j) {
                const float f = Elem<T>::ld(e + j);
                ss = fmaf(f, f, ss);
            }
        }
    }
    ss = wave_sum(ss);
    if (lane == 0) inv[item] = ss > 0.f ? (float)(1.0 / sqrt((double)ss)) : 0.f;
}

hipError_t launch_inv_norm(const Plan &p, const void *x, float *inv, hipStream_t st) {
    StageScope _stage(st, "inv_norm");
    const int n_items = p.kind == KIND_BLOCK ? p.N : p.F * p.N;
    const int n_sub = p.kind == KIND_BLOCK ? p.F : 1;
    const long sub = (long)p.N * p.C;
    const int blocks = cdiv(n_items, 4);
    if (p.bf16)
        k_inv_norm<uint16_t><<<blocks, 256, 0, st>>>((const uint16_t *)x, inv, n_items, n_sub, sub, p.C);
    else
        k_inv_norm<float><<<blocks, 256, 0, st>>>((const float *)x, inv, n_items, n_sub, sub, p.C);
    return hipGetLastError();
}

// ----------------------------------------------------------------------------
// similarity + arg-max, bf16 MFMA
// ----------------------------------------------------------------------------
// Block (candidate tile bt, representative tile at, group g), in an
// XCD-aware order: t = dot(src_b, dst_a) * inv(dst_a); per candidate the
// largest t over this block's representatives (smallest position on ties)
// goes to part[at][g][b].  The representative norm is applied before the
// arg-max, the candidate's own norm (a positive constant per row) after.
template <int BA, int BB, int WA, int WB>
__global__ __launch_bounds__(256) void k_match_mfma(const uint16_t *__restrict__ x, const float *__restrict__ inv,
                                                     const int32_t *__restrict__ src_ids,
                                                     const int32_t *__restrict__ dst_ids, int G, int S, int D,
                                                     int K, int seg_len, long sub_stride, long item_stride,
                                                     int n_bt, int n_at, float *__restrict__ part_max,
                                                     int32_t *__restrict__ part_idx) {
    using T = MfmaTile<BA, BB, WA, WB>;
    extern __shared__ __align__(16) uint16_t lds[];
    const int total = n_bt * n_at * G;
    const int lid = xcd_remap(blockIdx.x, total);
    // consecutive logical blocks: the representative tiles of one candidate tile
    const int at = lid % n_at, bt = (lid / n_at) % n_bt, g = lid / (n_at * n_bt);
    const int32_t *src = src_ids + (long)g * S;
    const int32_t *dst = dst_ids + (long)g * D;
    const uint16_t *rowsA[T::CA], *rowsB[T::CB];
#pragma unroll
    for (int i = 0; i < T::CA; ++i) {
        const int a = at * BA + T::chunk_row(i);
        const int id = a < D ? dst[a] : -1;
        rowsA[i] = id >= 0 ? x + (long)id * item_stride : nullptr;
    }
#pragma unroll
    for (int i = 0; i < T::CB; ++i) {
        const int b = bt * BB + T::chunk_row(i);
        const int id = b < S ? src[b] : -1;
        rowsB[i] = id >= 0 ? x + (long)id * item_stride : nullptr;
    }
    T tile;
    tile.run(lds, rowsA, rowsB, K, seg_len, sub_stride);

    // representative norms of this tile (0 for padding, which never wins)
    float *sinv = reinterpret_cast<float *>(lds);
    float *sv = sinv + BA;
    int *si = reinterpret_cast<int *>(sv + WA * BB);
    for (int a = threadIdx.x; a < BA; a += 256) {
        const int ga = at * BA + a;
        const int id = ga < D ? dst[ga] : -1;
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
        if (b < S) {
            const long o = ((long)at * G + g) * S + b;
            part_max[o] = v;
            part_idx[o] = ix;
        }
    }
}

// fp32 similarity + arg-max (small fp32 layers): one thread per candidate.
__global__ void k_match_f32(const float *__restrict__ x, const float *__restrict__ inv,
                            const int32_t *__restrict__ src_ids, const int32_t *__restrict__ dst_ids, int G, int S,
                            int D, int K, int seg_len, long sub_stride, long item_stride,
                            float *__restrict__ part_max, int32_t *__restrict__ part_idx) {
    const int g = blockIdx.y;
    const int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= S) return;
    const int sid = src_ids[(long)g * S + b];
    float bv = -INFINITY;
    int bi = -1;
    if (sid >= 0) {
        const float *u = x + (long)sid * item_stride;
        for (int a = 0; a < D; ++a) {
            const int did = dst_ids[(long)g * D + a];
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
    part_max[(long)g * S + b] = bv;
    part_idx[(long)g * S + b] = bi;
}

// Merge the rep-range partials in ascending order, convert the winning
// position to a global id and apply the candidate's norm.
__global__ void k_match_reduce(const float *__restrict__ part_max, const int32_t *__restrict__ part_idx,
                               int n_split, int G, int S, int D, const float *__restrict__ inv,
                               const int32_t *__restrict__ src_ids, const int32_t *__restrict__ dst_ids,
                               float *__restrict__ node_max, int32_t *__restrict__ node_idx) {
    const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (long)G * S) return;
    const int g = (int)(i / S);
    const int sid = src_ids[i];
    if (sid < 0) {
        node_max[i] = -INFINITY;
        node_idx[i] = -1;
        return;
    }
    float v = part_max[i];
    int ix = part_idx[i];
    for (int s = 1; s < n_split; ++s) argmax_merge(v, ix, part_max[(long)s * G * S + i], part_idx[(long)s * G * S + i]);
    node_max[i] = v * inv[sid];
    node_idx[i] = ix >= 0 ? dst_ids[(long)g * D + ix] : -1;
}

template <int BA, int BB, int WA, int WB>
static void go_match(const Plan &p, const uint16_t *x, const float *inv, const int32_t *src_ids,
                     const int32_t *dst_ids, int K, int seg_len, long sub_stride, long item_stride, float *part_max,
                     int32_t *part_idx, hipStream_t st) {
    using T = MfmaTile<BA, BB, WA, WB>;
    const int G = p.n_groups, S = p.n_src_max, D = p.n_dst_max;
    const int n_bt = cdiv(S, BB), n_at = cdiv(D, BA);
    const size_t lds = T::LDS_BYTES;
    k_match_mfma<BA, BB, WA, WB><<<n_bt * n_at * G, 256, lds, st>>>(x, inv, src_ids, dst_ids, G, S, D, K, seg_len,
                                                                     sub_stride, item_stride, n_bt, n_at, part_max,
                                                                     part_idx);
}

hipError_t launch_match(const Plan &p, const Layout &L, const void *x, const float *inv, const int32_t *src_ids,
                        const int32_t *dst_ids, float *part_max, int32_t *part_idx, float *node_max,
                        int32_t *node_idx, hipStream_t st) {
    const int G = p.n_groups, S = p.n_src_max, D = p.n_dst_max;
    const bool block = p.kind == KIND_BLOCK;
    const int K = block ? p.F * p.C : p.C;
    const int seg_len = block ? p.C : 0;
    const long sub_stride = (long)p.N * p.C;
    const long item_stride = p.C;
    const int n_split = match_split(p);
    {
        StageScope _stage(st, "match");
        if (p.bf16) {
            const uint16_t *xb = (const uint16_t *)x;
            // representative tile height as in match_split(): 128, 64 or 32
            if (D > 64)
                go_match<128, 64, 2, 2>(p, xb, inv, src_ids, dst_ids, K, seg_len, sub_stride, item_stride, part_max,
                                        part_idx, st);
            else if (D > 32)
                go_match<64, 64, 2, 2>(p, xb, inv, src_ids, dst_ids, K, seg_len, sub_stride, item_stride, part_max,
                                       part_idx, st);
            else
                go_match<32, 128, 1, 4>(p, xb, inv, src_ids, dst_ids, K, seg_len, sub_stride, item_stride, part_max,
                                        part_idx, st);
        } else {
            dim3 grid(cdiv(S, 64), G);
            k_match_f32<<<grid, 64, 0, st>>>((const float *)x, inv, src_ids, dst_ids, G, S, D, K, seg_len, sub_stride,
                                             item_stride, part_max, part_idx);
        }
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const long n = (long)G * S;
    {
        StageScope _stage(st, "match_reduce");
        k_match_reduce<<<(unsigned)cdiv((int)n, 256), 256, 0, st>>>(part_max, part_idx, n_split, G, S, D, inv,
                                                                     src_ids, dst_ids, node_max, node_idx);
    }
    return hipGetLastError();
}

}  // namespace oc
