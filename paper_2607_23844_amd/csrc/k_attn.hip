// Reduced-token attention (OmniCache §3.2.3: the layer runs on the retained
// tokens only; cached tokens are neither queries nor keys/values).
//
// bf16 path (x, weights and the output y are bf16; products of bf16 inputs
// are exact and accumulate in fp32; the intermediates Q, K, V, P and O are
// held in fp16, whose three extra mantissa bits keep the score error below
// the bf16 output rounding):
//   QK projection  [rows, C] x [2*H*dh, C]^T -> Q, K [rows, H*dh]     (MFMA)
//   V projection   -> Vt [H][seq][dh][Lpad] (keys contiguous per d)    (MFMA)
//   flash attention per (query tile, head, sequence): S^T = K Q^T and
//     O^T = Vt P^T on MFMA, K / Vt tiles staged in LDS, online softmax in
//     the log2 domain; each lane owns one query, so row statistics need
//     only a 4-lane-group reduction for the running maximum.
//   output projection [rows, H*dh] x [C, H*dh]^T -> y rows, optionally
//     scattered straight to their positions (row -> out_idx[row]).
// Rows r < n_main come from x (through row_idx when given), rows after
// them are the uncached context tokens of a single sequence.
// fp32 path: the same dataflow with plain VALU kernels (small layers).
#include "oc_internal.h"
#include "oc_device.h"
#include "oc_mfma_tile.h"

namespace oc {

struct RowMap {
    const uint16_t *x; const int32_t *row_idx; int n_main;
    const uint16_t *ctx; int n_rows; int C;
    __device__ __forceinline__ const uint16_t *row(int r) const {
        if (r >= n_rows) return nullptr;
        if (r < n_main) return x + (long)(row_idx ? row_idx[r] : r) * C;
        return ctx + (long)(r - n_main) * C;
    }
};

// sequence and position of batch row r
__device__ __forceinline__ void seq_pos(int r, int n_seq, int L, int &s, int &j) {
    if (n_seq == 1) { s = 0; j = r; }
    else { s = r / L; j = r - s * L; }
}

// ---------------------------------------------------------------------------
// projections (bf16 MFMA)
// ---------------------------------------------------------------------------
constexpr int PBA = 128, PBB = 128;
using PTile = MfmaTile<PBA, PBB, 2, 2>;
// output projection: O rows are fp16, wo (bf16) is converted to fp16 as it is staged
using OTile = MfmaTile<PBA, PBB, 2, 2, true, true>;

// a in [0, 2*hd): rows of wq then wk; b = batch rows.  Q/K[b][a % hd].
__global__ __launch_bounds__(256) void k_proj_qk(RowMap rm, const uint16_t *__restrict__ wq,
                                                 const uint16_t *__restrict__ wk, int hd,
                                                 uint16_t *__restrict__ Q, uint16_t *__restrict__ K) {
    extern __shared__ __align__(16) uint16_t lds[];
    const int at = blockIdx.y, bt = blockIdx.x;
    const uint16_t *rowsA[PTile::CA], *rowsB[PTile::CB];
#pragma unroll
    for (int i = 0; i < PTile::CA; ++i) {
        const int a = at * PBA + PTile::chunk_row(i);
        rowsA[i] = a < hd ? wq + (long)a * rm.C : (a < 2 * hd ? wk + (long)(a - hd) * rm.C : nullptr);
    }
#pragma unroll
    for (int i = 0; i < PTile::CB; ++i) rowsB[i] = rm.row(bt * PBB + PTile::chunk_row(i));
    PTile t;
    t.run(lds, rowsA, rowsB, rm.C, 0, 0);
#pragma unroll
    for (int j = 0; j < PTile::TB; ++j) {
        const int b = bt * PBB + PTile::b_of(j);
        if (b >= rm.n_rows) continue;
#pragma unroll
        for (int i = 0; i < PTile::TA; ++i) {
            const int a = at * PBA + PTile::a_of(i, 0);
            if (a >= 2 * hd) continue;
            uint16_t *dst = a < hd ? Q + (long)b * hd + a : K + (long)b * hd + (a - hd);
            u16x4 v;
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = f2h_bits(t.acc[i][j][e]);
            *reinterpret_cast<u16x4 *>(dst) = v;
        }
    }
}

// a = batch rows, b in [0, hd): rows of wv.  Vt[h][s][d][j].
__global__ __launch_bounds__(256) void k_proj_v(RowMap rm, const uint16_t *__restrict__ wv, int hd, int dh,
                                                int n_seq, int L, int lpad, uint16_t *__restrict__ Vt) {
    extern __shared__ __align__(16) uint16_t lds[];
    const int at = blockIdx.y, bt = blockIdx.x;
    const uint16_t *rowsA[PTile::CA], *rowsB[PTile::CB];
#pragma unroll
    for (int i = 0; i < PTile::CA; ++i) rowsA[i] = rm.row(at * PBA + PTile::chunk_row(i));
#pragma unroll
    for (int i = 0; i < PTile::CB; ++i) {
        const int b = bt * PBB + PTile::chunk_row(i);
        rowsB[i] = b < hd ? wv + (long)b * rm.C : nullptr;
    }
    PTile t;
    t.run(lds, rowsA, rowsB, rm.C, 0, 0);
#pragma unroll
    for (int j = 0; j < PTile::TB; ++j) {
        const int f = bt * PBB + PTile::b_of(j);
        if (f >= hd) continue;
        const int h = f / dh, d = f - h * dh;
#pragma unroll
        for (int i = 0; i < PTile::TA; ++i)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int r = at * PBA + PTile::a_of(i, e);
                if (r >= rm.n_rows) continue;
                int s, jj;
                seq_pos(r, n_seq, L, s, jj);
                Vt[(((long)h * n_seq + s) * dh + d) * lpad + jj] = f2h_bits(t.acc[i][j][e]);
            }
    }
}

// a in [0, C): rows of wo; b = batch rows of O.  y[out row][a].
__global__ __launch_bounds__(256) void k_proj_out(const uint16_t *__restrict__ O, int n_rows, int hd,
                                                  const uint16_t *__restrict__ wo, int C, int n_main,
                                                  const int32_t *__restrict__ out_idx, uint16_t *__restrict__ y,
                                                  uint16_t *__restrict__ y_ctx) {
    extern __shared__ __align__(16) uint16_t lds[];
    const int at = blockIdx.y, bt = blockIdx.x;
    const uint16_t *rowsA[OTile::CA], *rowsB[OTile::CB];
#pragma unroll
    for (int i = 0; i < OTile::CA; ++i) {
        const int a = at * PBA + OTile::chunk_row(i);
        rowsA[i] = a < C ? wo + (long)a * hd : nullptr;
    }
#pragma unroll
    for (int i = 0; i < OTile::CB; ++i) {
        const int b = bt * PBB + OTile::chunk_row(i);
        rowsB[i] = b < n_rows ? O + (long)b * hd : nullptr;
    }
    OTile t;
    t.run(lds, rowsA, rowsB, hd, 0, 0);
#pragma unroll
    for (int j = 0; j < OTile::TB; ++j) {
        const int b = bt * PBB + OTile::b_of(j);
        if (b >= n_rows) continue;
        uint16_t *yrow = b < n_main ? y + (long)(out_idx ? out_idx[b] : b) * C : y_ctx + (long)(b - n_main) * C;
#pragma unroll
        for (int i = 0; i < OTile::TA; ++i) {
            const int a = at * PBA + OTile::a_of(i, 0);
            if (a >= C) continue;
            u16x4 v;
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = f2bf(t.acc[i][j][e]);
            *reinterpret_cast<u16x4 *>(yrow + a) = v;
        }
    }
}

// ---------------------------------------------------------------------------
// flash attention (bf16 MFMA)
// ---------------------------------------------------------------------------
// Grid (query tiles of 64*QB, heads, sequences); 4 waves, wave w owns
// queries [tile*64*QB + w*16*QB, +16*QB) as QB blocks of 16.
template <int DH, int QB>
__global__ __launch_bounds__(256) void k_flash(const uint16_t *__restrict__ Q, const uint16_t *__restrict__ K,
                                               const uint16_t *__restrict__ Vt, uint16_t *__restrict__ O, int hd,
                                               int n_seq, int L, int Lk, int lpad, float scale_log2) {
    constexpr int DK = (DH + 31) / 32 * 32;   // head dim padded for the S^T k-loop
    constexpr int DV = (DH + 15) / 16 * 16;   // head dim padded for O^T tiles
    constexpr int KT = 64;                    // keys per tile
    constexpr int LDK = DK + 8;
    constexpr int LDV = KT + 8;
    __shared__ __align__(16) uint16_t Ks[KT * LDK];
    __shared__ __align__(16) uint16_t Vs[DV * LDV];
    const int qt = blockIdx.x, h = blockIdx.y, s = blockIdx.z;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int lr = lane & 15, lg = lane >> 4;
    const long row0 = (long)s * L;
    const int q_base = qt * 64 * QB + wave * 16 * QB;

    f16x8 qf[QB][DK / 32];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        const int q = q_base + qb * 16 + lr;
#pragma unroll
        for (int ks = 0; ks < DK / 32; ++ks) {
            const int d0 = ks * 32 + lg * 8;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (q < Lk && d0 < DH) v = *reinterpret_cast<const uint4 *>(Q + (row0 + q) * hd + h * DH + d0);
            qf[qb][ks] = *reinterpret_cast<f16x8 *>(&v);
        }
    }
    float m[QB], l[QB];
    f32x4 o[QB][DV / 16];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        m[qb] = -INFINITY;
        l[qb] = 0.f;
#pragma unroll
        for (int dt = 0; dt < DV / 16; ++dt) o[qb][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    const uint16_t *vbase = Vt + ((long)h * n_seq + s) * DH * lpad;
    const int n_kt = cdiv(Lk, KT);
    for (int kt = 0; kt < n_kt; ++kt) {
        const int k0 = kt * KT;
        __syncthreads();
        // K tile [key][d], zero outside the sequence and beyond DH
        for (int c = threadIdx.x; c < KT * (DK / 8); c += 256) {
            const int key = c / (DK / 8), d0 = (c % (DK / 8)) * 8;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (k0 + key < Lk && d0 < DH) v = *reinterpret_cast<const uint4 *>(K + (row0 + k0 + key) * hd + h * DH + d0);
            *reinterpret_cast<uint4 *>(Ks + key * LDK + d0) = v;
        }
        // Vt tile [d][key], keys permuted inside each 32-key block so that the
        // 8 keys one lane feeds to the PV MFMA are contiguous
        for (int c = threadIdx.x; c < DV * (KT / 8); c += 256) {
            const int d = c / (KT / 8), kc = c % (KT / 8);
            uint4 v = make_uint4(0, 0, 0, 0);
            if (d < DH) {
                v = *reinterpret_cast<const uint4 *>(vbase + (long)d * lpad + k0 + kc * 8);
                const int valid = Lk - (k0 + kc * 8);
                if (valid < 8) {
                    uint16_t *e = reinterpret_cast<uint16_t *>(&v);
#pragma unroll
                    for (int q = 0; q < 8; ++q)
                        if (q >= valid) e[q] = 0;
                }
            }
            const int kk0 = (kc & 3) * 8;                 // first key inside the 32-key block
            const int g0 = (kk0 & 15) >> 2, e0 = kk0 >= 16 ? 4 : 0;
            uint16_t *dst = Vs + d * LDV + (kc >> 2) * 32;
            *reinterpret_cast<uint2 *>(dst + g0 * 8 + e0) = make_uint2(v.x, v.y);
            *reinterpret_cast<uint2 *>(dst + (g0 + 1) * 8 + e0) = make_uint2(v.z, v.w);
        }
        __syncthreads();

        // scores S^T[key][query]: lane holds query lr, keys kt16*16 + 4*lg + e
        f32x4 sc[QB][4];
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
#pragma unroll
            for (int t4 = 0; t4 < 4; ++t4) sc[qb][t4] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int t4 = 0; t4 < 4; ++t4)
#pragma unroll
            for (int ks = 0; ks < DK / 32; ++ks) {
                const f16x8 kf = *reinterpret_cast<const f16x8 *>(Ks + (t4 * 16 + lr) * LDK + ks * 32 + lg * 8);
#pragma unroll
                for (int qb = 0; qb < QB; ++qb)
                    sc[qb][t4] = __builtin_amdgcn_mfma_f32_16x16x32_f16(kf, qf[qb][ks], sc[qb][t4], 0, 0, 0);
            }
        // online softmax (log2 domain)
        f16x8 pf[QB][2];
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
            float mt = -INFINITY;
#pragma unroll
            for (int t4 = 0; t4 < 4; ++t4)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int key = k0 + t4 * 16 + lg * 4 + e;
                    const float v = key < Lk ? sc[qb][t4][e] * scale_log2 : -INFINITY;
                    sc[qb][t4][e] = v;
                    mt = fmaxf(mt, v);
                }
            mt = fmaxf(mt, __shfl_xor(mt, 16, 64));
            mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
            const float mn = fmaxf(m[qb], mt);
            const float alpha = exp2f(m[qb] - mn);
            m[qb] = mn;
            float ls = 0.f;
            float pv[4][4];
#pragma unroll
            for (int t4 = 0; t4 < 4; ++t4)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    pv[t4][e] = exp2f(sc[qb][t4][e] - mn);
                    ls += pv[t4][e];
                }
            l[qb] = l[qb] * alpha + ls;
#pragma unroll
            for (int dt = 0; dt < DV / 16; ++dt) o[qb][dt] *= alpha;
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                f16x8 f;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    f[e] = (_Float16)pv[2 * j][e];
                    f[4 + e] = (_Float16)pv[2 * j + 1][e];
                }
                pf[qb][j] = f;
            }
        }
        // O^T[d][query] += Vt[d][keys] P^T[keys][query]
#pragma unroll
        for (int dt = 0; dt < DV / 16; ++dt)
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const f16x8 vf = *reinterpret_cast<const f16x8 *>(Vs + (dt * 16 + lr) * LDV + j * 32 + lg * 8);
#pragma unroll
                for (int qb = 0; qb < QB; ++qb)
                    o[qb][dt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(vf, pf[qb][j], o[qb][dt], 0, 0, 0);
            }
    }
    // normalise and store: lane holds query lr, d = dt*16 + 4*lg + e
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        float lt = l[qb];
        lt += __shfl_xor(lt, 16, 64);
        lt += __shfl_xor(lt, 32, 64);
        const float inv = 1.f / lt;
        const int q = q_base + qb * 16 + lr;
        if (q >= Lk) continue;
        uint16_t *orow = O + (row0 + q) * hd + h * DH;
#pragma unroll
        for (int dt = 0; dt < DV / 16; ++dt) {
            const int d = dt * 16 + lg * 4;
            if (d >= DH) continue;
            u16x4 v;
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = f2h_bits(o[qb][dt][e] * inv);
            *reinterpret_cast<u16x4 *>(orow + d) = v;
        }
    }
}

// ---------------------------------------------------------------------------
// fp32 path (small layers): projections, attention, output projection
// ---------------------------------------------------------------------------
struct RowMapF {
    const float *x; const int32_t *row_idx; int n_main;
    const float *ctx; int n_rows; int C;
    __device__ __forceinline__ const float *row(int r) const {
        if (r < n_main) return x + (long)(row_idx ? row_idx[r] : r) * C;
        return ctx + (long)(r - n_main) * C;
    }
};

// QKV[r][f] for f in [0, 3*hd): one thread per output
__global__ void k_proj_f32(RowMapF rm, const float *__restrict__ wq, const float *__restrict__ wk,
                           const float *__restrict__ wv, int hd, float *__restrict__ Q, float *__restrict__ K,
                           float *__restrict__ V) {
    const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (long)rm.n_rows * 3 * hd) return;
    const int r = (int)(i / (3 * hd)), f = (int)(i - (long)r * 3 * hd);
    const int which = f / hd, c = f - which * hd;
    const float *w = (which == 0 ? wq : which == 1 ? wk : wv) + (long)c * rm.C;
    const float *x = rm.row(r);
    float acc = 0.f;
    for (int k = 0; k < rm.C; ++k) acc = fmaf(x[k], w[k], acc);
    (which == 0 ? Q : which == 1 ? K : V)[(long)r * hd + c] = acc;
}

// one thread per (query row, head): online softmax over the sequence's keys
__global__ void k_attn_f32(const float *__restrict__ Q, const float *__restrict__ K, const float *__restrict__ V,
                           float *__restrict__ O, int n_rows, int heads, int dh, int n_seq, int L, int Lk,
                           float scale) {
    const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (long)n_rows * heads) return;
    const int r = (int)(i / heads), h = (int)(i - (long)r * heads);
    const int hd = heads * dh;
    int s, j;
    seq_pos(r, n_seq, L, s, j);
    const long row0 = (long)s * L;
    const float *q = Q + (long)r * hd + h * dh;
    float acc[128];
    for (int d = 0; d < dh; ++d) acc[d] = 0.f;
    float m = -INFINITY, l = 0.f;
    for (int kk = 0; kk < Lk; ++kk) {
        const float *k = K + (row0 + kk) * hd + h * dh;
        float sc = 0.f;
        for (int d = 0; d < dh; ++d) sc = fmaf(q[d], k[d], sc);
        sc *= scale;
        const float mn = fmaxf(m, sc);
        const float a = expf(m - mn), p = expf(sc - mn);
        l = l * a + p;
        const float *v = V + (row0 + kk) * hd + h * dh;
        for (int d = 0; d < dh; ++d) acc[d] = acc[d] * a + p * v[d];
        m = mn;
    }
    float *o = O + (long)r * hd + h * dh;
    for (int d = 0; d < dh; ++d) o[d] = acc[d] / l;
}

__global__ void k_out_f32(const float *__restrict__ O, int n_rows, int hd, const float *__restrict__ wo, int C,
                          int n_main, const int32_t *__restrict__ out_idx, float *__restrict__ y,
                          float *__restrict__ y_ctx) {
    const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (long)n_rows * C) return;
    const int r = (int)(i / C), c = (int)(i - (long)r * C);
    const float *o = O + (long)r * hd;
    const float *w = wo + (long)c * hd;
    float acc = 0.f;
    for (int k = 0; k < hd; ++k) acc = fmaf(o[k], w[k], acc);
    if (r < n_main) y[(long)(out_idx ? out_idx[r] : r) * C + c] = acc;
    else y_ctx[(long)(r - n_main) * C + c] = acc;
}

// ---------------------------------------------------------------------------
AttnWs attn_ws(const Plan &p, int n_seq, int L, size_t base) {
    AttnWs w;
    const long rows = (long)n_seq * L + p.n_ctx;
    const int Lk = L + (n_seq == 1 ? p.n_ctx : 0);
    w.lpad = cdiv(Lk > 0 ? Lk : 1, 64) * 64;
    auto al = [](size_t b) { return (b + 255) & ~(size_t)255; };
    const size_t e = p.esz;
    const size_t m = al((size_t)rows * p.hd * e);
    w.q = base;
    w.k = w.q + m;
    w.o = w.k + m;
    w.v = w.o + m;
    const size_t vb = p.bf16 ? al((size_t)p.heads * n_seq * p.dh * w.lpad * e) : m;
    w.bytes = w.v + vb - base;
    return w;
}

bool attn_head_dim_supported(int dh) {
    switch (dh) {
        case 16: case 32: case 48: case 64: case 72: case 80: case 96: case 128: return true;
        default: return false;
    }
}

template <int DH>
static void go_flash(const Plan &p, const AttnArgs &a, int Lk, hipStream_t st) {
    const float scale_log2 = (float)(1.4426950408889634 / sqrt((double)DH));
    if (Lk >= 4096) {
        dim3 grid(cdiv(Lk, 128), p.heads, a.n_seq);
        {
            StageScope _stage(st, "flash");
            k_flash<DH, 2><<<grid, 256, 0, st>>>((const uint16_t *)a.q, (const uint16_t *)a.k, (const uint16_t *)a.vt,
                                                (uint16_t *)a.o, p.hd, a.n_seq, a.L, Lk, a.lpad, scale_log2);
        }
    } else {
        dim3 grid(cdiv(Lk, 64), p.heads, a.n_seq);
        {
            StageScope _stage(st, "flash");
            k_flash<DH, 1><<<grid, 256, 0, st>>>((const uint16_t *)a.q, (const uint16_t *)a.k, (const uint16_t *)a.vt,
                                                (uint16_t *)a.o, p.hd, a.n_seq, a.L, Lk, a.lpad, scale_log2);
        }
    }
}

hipError_t launch_attention(const Plan &p, const AttnArgs &a, hipStream_t st) {
    const int n_rows = a.n_seq * a.L + a.n_ctx;
    const int Lk = a.L + (a.n_seq == 1 ? a.n_ctx : 0);
    if (n_rows == 0) return hipSuccess;
    if (p.bf16) {
        RowMap rm{(const uint16_t *)a.x, a.row_idx, a.n_main, (const uint16_t *)a.ctx, n_rows, p.C};
        const size_t lds = PTile::LDS_BYTES;
        {
            StageScope _stage(st, "proj_qk");
            k_proj_qk<<<dim3(cdiv(n_rows, PBB), cdiv(2 * p.hd, PBA)), 256, lds, st>>>(
                rm, (const uint16_t *)a.wq, (const uint16_t *)a.wk, p.hd, (uint16_t *)a.q, (uint16_t *)a.k);
        }
        {
            StageScope _stage(st, "proj_v");
            k_proj_v<<<dim3(cdiv(p.hd, PBB), cdiv(n_rows, PBA)), 256, lds, st>>>(
                rm, (const uint16_t *)a.wv, p.hd, p.dh, a.n_seq, a.L, a.lpad, (uint16_t *)a.vt);
        }
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        switch (p.dh) {
            case 16: go_flash<16>(p, a, Lk, st); break;
            case 32: go_flash<32>(p, a, Lk, st); break;
            case 48: go_flash<48>(p, a, Lk, st); break;
            case 64: go_flash<64>(p, a, Lk, st); break;
            case 72: go_flash<72>(p, a, Lk, st); break;
            case 80: go_flash<80>(p, a, Lk, st); break;
            case 96: go_flash<96>(p, a, Lk, st); break;
            case 128: go_flash<128>(p, a, Lk, st); break;
            default: return hipErrorInvalidValue;
        }
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        {
            StageScope _stage(st, "proj_out");
            k_proj_out<<<dim3(cdiv(n_rows, PBB), cdiv(p.C, PBA)), 256, lds, st>>>(
                (const uint16_t *)a.o, n_rows, p.hd, (const uint16_t *)a.wo, p.C, a.n_main, a.out_idx, (uint16_t *)a.y,
                (uint16_t *)a.y_ctx);
        }
        return hipGetLastError();
    }
    RowMapF rm{(const float *)a.x, a.row_idx, a.n_main, (const float *)a.ctx, n_rows, p.C};
    const long nq = (long)n_rows * 3 * p.hd;
    {
        StageScope _stage(st, "proj_f32");
        k_proj_f32<<<(unsigned)((nq + 255) / 256), 256, 0, st>>>(rm, (const float *)a.wq, (const float *)a.wk,
                                                                  (const float *)a.wv, p.hd, (float *)a.q, (float *)a.k,
                                                                  (float *)a.vt);
    }
    const long na = (long)n_rows * p.heads;
    {
        StageScope _stage(st, "attn_f32");
        k_attn_f32<<<(unsigned)((na + 127) / 128), 128, 0, st>>>((const float *)a.q, (const float *)a.k,
                                                                  (const float *)a.vt, (float *)a.o, n_rows, p.heads, p.dh,
                                                                  a.n_seq, a.L, Lk, (float)(1.0 / sqrt((double)p.dh)));
    }
    const long no = (long)n_rows * p.C;
    {
        StageScope _stage(st, "out_f32");
        k_out_f32<<<(unsigned)((no + 255) / 256), 256, 0, st>>>((const float *)a.o, n_rows, p.hd, (const float *)a.wo,
                                                                 p.C, a.n_main, a.out_idx, (float *)a.y, (float *)a.y_ctx);
    }
    return hipGetLastError();
}

}  // namespace oc
