// Projections of the reduced attention layer on the MFMA tile engine.
//
// x, weights and y are bf16; products of bf16 inputs are exact and
// accumulate in fp32.  The attention intermediates Q, K, V and O are stored
// in fp16 (three more mantissa bits than bf16, same MFMA rate): Q is stored
// pre-multiplied by log2(e)/sqrt(head_dim) so that the attention kernel's
// scores are already in the log2 domain.
//   k_proj_qk : [rows, C] x [2*H*dh, C]^T -> Q, K [rows, H*dh]
//   k_proj_v  : -> Vt [H][seq][dh][Lpad], keys contiguous per (head, d),
//               quads 1 and 2 of every 16-key block swapped (vt_key_of_pos)
//   k_proj_out: O [rows, H*dh] (fp16) x wo [C, H*dh] -> y rows, written
//               straight to their positions (row -> out_idx[row]) or to the
//               context output
// Rows r < n_main come from x (through row_idx when given); rows after them
// are the uncached context tokens of a single sequence.
//
// Tile order: blocks are remapped so that each XCD runs a contiguous range
// of logical tiles, and logical tiles are grouped GA weight tiles wide, so
// one XCD's L2 sees a few weight tiles and a few token tiles instead of all.
#include "oc_internal.h"
#include "oc_device.h"
#include "oc_mfma_tile.h"
#include "oc_attn_common.h"

namespace oc {

constexpr int PBA = 128, PBB = 128;
using PTile = MfmaTile<PBA, PBB, 2, 2>;
// output projection: O rows and wo (converted once per call) are fp16
using OTile = MfmaTile<PBA, PBB, 2, 2, true, false>;
constexpr int GA = 6;

// logical tile lid -> (a tile, b tile), GA a-tiles per group, b fastest inside
__device__ __forceinline__ void tile_order(int lid, int n_at, int n_bt, int &at, int &bt) {
    const int per = GA * n_bt;
    const int grp = lid / per, idx = lid - grp * per;
    const int ga = min(GA, n_at - grp * GA);
    at = grp * GA + idx % ga;
    bt = idx / ga;
}

// a in [0, 2*hd): rows of wq then wk; b = batch rows.  Q/K[b][a % hd].
__global__ __launch_bounds__(256) void k_proj_qk(RowMap rm, const uint16_t *__restrict__ wq,
                                                 const uint16_t *__restrict__ wk, int hd, float qscale, int n_at,
                                                 int n_bt, uint16_t *__restrict__ Q, uint16_t *__restrict__ K) {
    extern __shared__ __align__(16) uint16_t lds[];
    int at, bt;
    tile_order(xcd_remap(blockIdx.x, n_at * n_bt), n_at, n_bt, at, bt);
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
        for (int i = 0; i < PTile::TA; ++i)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int a = at * PBA + PTile::a_of(i, g);
                if (a >= 2 * hd) continue;
                const bool isq = a < hd;
                uint16_t *dst = isq ? Q + (long)b * hd + a : K + (long)b * hd + (a - hd);
                const float sc = isq ? qscale : 1.f;
                u16x4 v;
#pragma unroll
                for (int e = 0; e < 4; ++e) v[e] = f2h_bits(t.acc[i][j][4 * g + e] * sc);
                *reinterpret_cast<u16x4 *>(dst) = v;
            }
    }
}

// a = batch rows, b in [0, hd): rows of wv.  Vt[h][s][d][j].  A lane holds
// four consecutive rows of one feature: one 8-byte store when they are
// consecutive positions of one sequence.
__global__ __launch_bounds__(256) void k_proj_v(RowMap rm, const uint16_t *__restrict__ wv, int hd, int dh,
                                                int n_seq, int L, int lpad, int n_at, int n_bt, int zero_pad,
                                                uint16_t *__restrict__ Vt) {
    extern __shared__ __align__(16) uint16_t lds[];
    int at, bt;
    tile_order(xcd_remap(blockIdx.x, n_at * n_bt), n_at, n_bt, at, bt);
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
            for (int g = 0; g < 4; ++g) {
                const int r0 = at * PBA + PTile::a_of(i, g);
                if (r0 >= rm.n_rows) continue;
                int s0, j0, s3, j3;
                seq_pos(r0, n_seq, L, s0, j0);
                seq_pos(r0 + 3, n_seq, L, s3, j3);
                if (r0 + 3 < rm.n_rows && s0 == s3 && (j0 & 3) == 0) {
                    u16x4 v;
#pragma unroll
                    for (int e = 0; e < 4; ++e) v[e] = f2h_bits(t.acc[i][j][4 * g + e]);
                    *reinterpret_cast<u16x4 *>(Vt + (((long)h * n_seq + s0) * dh + d) * lpad + vt_key_of_pos(j0)) = v;
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int r = r0 + e;
                        if (r >= rm.n_rows) continue;
                        int s, jj;
                        seq_pos(r, n_seq, L, s, jj);
                        Vt[(((long)h * n_seq + s) * dh + d) * lpad + vt_key_of_pos(jj)] = f2h_bits(t.acc[i][j][4 * g + e]);
                    }
                }
            }
    }
    // zero the padded key positions [Lk, lpad) of this block's features, for
    // the sequences s = at, at + n_at, ... (the DMA-staged attention reads them)
    const int Lk = n_seq == 1 ? rm.n_rows : L, npad = lpad - Lk;
    if (zero_pad && npad > 0) {
        for (int sq = at; sq < n_seq; sq += n_at)
            for (int idx = threadIdx.x; idx < PBB * npad; idx += blockDim.x) {
                const int f = bt * PBB + idx / npad, jj = Lk + idx % npad;
                if (f >= hd) continue;
                const int h = f / dh, d = f - h * dh;
                Vt[(((long)h * n_seq + sq) * dh + d) * lpad + vt_key_of_pos(jj)] = 0;
            }
    }
}

// a in [0, C): rows of wo; b = batch rows of O.  y[out row][a].
__global__ __launch_bounds__(256) void k_proj_out(const uint16_t *__restrict__ O, int n_rows, int hd,
                                                  const uint16_t *__restrict__ wo, int C, int n_main,
                                                  const int32_t *__restrict__ out_idx, int n_at, int n_bt,
                                                  uint16_t *__restrict__ y, uint16_t *__restrict__ y_ctx) {
    extern __shared__ __align__(16) uint16_t lds[];
    int at, bt;
    tile_order(xcd_remap(blockIdx.x, n_at * n_bt), n_at, n_bt, at, bt);
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
        for (int i = 0; i < OTile::TA; ++i)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int a = at * PBA + OTile::a_of(i, g);
                if (a >= C) continue;
                u16x4 v;
#pragma unroll
                for (int e = 0; e < 4; ++e) v[e] = f2bf(t.acc[i][j][4 * g + e]);
                *reinterpret_cast<u16x4 *>(yrow + a) = v;
            }
    }
}

hipError_t launch_proj_qkv(const Plan &p, const RowMap &rm, const AttnArgs &a, hipStream_t st) {
    const size_t lds = PTile::LDS_BYTES;
    const float qscale = (float)(1.4426950408889634 / sqrt((double)p.dh));
    {
        StageScope _stage(st, "proj_qk");
        const int n_at = cdiv(2 * p.hd, PBA), n_bt = cdiv(rm.n_rows, PBB);
        k_proj_qk<<<n_at * n_bt, 256, lds, st>>>(rm, (const uint16_t *)a.wq, (const uint16_t *)a.wk, p.hd, qscale,
                                                 n_at, n_bt, (uint16_t *)a.q, (uint16_t *)a.k);
    }
    {
        StageScope _stage(st, "proj_v");
        const int n_at = cdiv(rm.n_rows, PBA), n_bt = cdiv(p.hd, PBB);
        const int Lk = a.n_seq == 1 ? rm.n_rows : a.L;
        k_proj_v<<<n_at * n_bt, 256, lds, st>>>(rm, (const uint16_t *)a.wv, p.hd, p.dh, a.n_seq, a.L, a.lpad, n_at,
                                                n_bt, flash_uses_dma(p.dh, Lk) ? 1 : 0, (uint16_t *)a.vt);
    }
    return hipGetLastError();
}

// bf16 -> fp16 (exact in the fp16 normal range, saturating outside), 8 per thread
__global__ void k_to_f16(const uint4 *__restrict__ src, long n8, uint4 *__restrict__ dst) {
    for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n8; i += (long)gridDim.x * blockDim.x)
        dst[i] = bf16x8_to_f16x8(src[i]);
}

hipError_t launch_proj_out(const Plan &p, int n_rows, const AttnArgs &a, hipStream_t st) {
    const long n8 = (long)p.C * p.hd / 8;
    if (!a.wo16_ready) {
        StageScope _stage(st, "wo_f16");
        const long blocks = (n8 + 255) / 256;
        k_to_f16<<<(unsigned)(blocks < 2048 ? blocks : 2048), 256, 0, st>>>((const uint4 *)a.wo, n8,
                                                                            (uint4 *)a.wo16);
    }
    StageScope _stage(st, "proj_out");
    const int n_at = cdiv(p.C, PBA), n_bt = cdiv(n_rows, PBB);
    k_proj_out<<<n_at * n_bt, 256, OTile::LDS_BYTES, st>>>((const uint16_t *)a.o, n_rows, p.hd,
                                                           (const uint16_t *)a.wo16, p.C, a.n_main, a.out_idx, n_at,
                                                           n_bt, (uint16_t *)a.y, (uint16_t *)a.y_ctx);
    return hipGetLastError();
}

}  // namespace oc
