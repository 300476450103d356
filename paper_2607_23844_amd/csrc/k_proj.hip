// Projections of the reduced attention layer on the MFMA tile engines.
//
// x, weights and y are bf16; products of bf16 inputs are exact and
// accumulate in fp32.  The attention intermediates Q, K, V and O are stored
// in fp16 (three more mantissa bits than bf16, same MFMA rate): Q is stored
// pre-multiplied by log2(e)/sqrt(head_dim) so that the attention kernel's
// scores are already in the log2 domain.
//   k_proj_qkv: [rows, C] x [3*H*dh, C]^T -> Q, K [rows, H*dh] and
//               Vt [H][seq][dh][Lpad], keys contiguous per (head, d),
//               quads 1 and 2 of every 16-key block swapped (vt_key_of_pos)
//   k_proj_out: O [rows, H*dh] (fp16) x wo [C, H*dh] -> y rows, written
//               straight to their positions (row -> out_idx[row]) or to the
//               context output
// Rows r < n_main come from x (through row_idx when given); rows after them
// are the uncached context tokens of a single sequence.
//
// Engines: with K a multiple of 64 the LDS-DMA tile, double buffered (Q/K/V:
// 128 x 128; output: 128 x 64, or 160 x 128 when C = 160 k), the
// register-staged tile (128 x 128) otherwise.  Epilogues go through LDS: the tile is staged as
// whole output rows and written in 16-byte chunks, so every store is a
// contiguous run of a row (Vt rows included).
//
// Tile order: blocks are remapped so that each XCD runs a contiguous range
// of logical tiles, and logical tiles are grouped GA weight tiles wide, so
// one XCD's L2 sees a few weight tiles and a few token tiles instead of all.
#include "oc_internal.h"
#include "oc_launch.h"
#include "oc_device.h"
#include "oc_mfma_tile.h"
#include "oc_dma_tile.h"
#include "oc_attn_common.h"
#include "oc_gemm_epi.h"

namespace oc {

// ---------------------------------------------------------------------------
// Q, K and V in one launch of 128 x 128 tiles.  The first n_qk tiles are
// row tiles: a in [0, nw*hd) are rows of wq, wk (and wv when nw = 3), b =
// batch rows, staged as rows of Q, K (and of V, row-major [rows, H*dh], for
// short sequences, whose attention reads V by rows).  With nw = 2 the rest
// are V tiles with the roles swapped: a = batch
// rows, b in [0, hd) = rows of wv, so that a staged row is a row of
// Vt[h][s][d][pos].  V tiles whose rows are a 16-aligned run of one
// sequence (a single sequence, or L % 128 == 0) are written as Vt rows:
// the positions of the tile's tokens, zero for positions past the end (the
// key padding up to lpad), in whole chunks.  Otherwise elements are stored
// one by one and, when the attention kernel needs it, the key padding is
// zeroed separately.  The DMA engine runs double-buffered (two blocks per
// CU).
// ---------------------------------------------------------------------------
// Tile shapes (SH): 0 = 128 x 128; 1 = 192 x 128 (192 rows of the A side:
// weight rows in the row tiles, batch rows in the V tiles); 2 = 128 x 192
// (192 of the B side: batch rows in the row tiles, rows of wv in the V
// tiles).  The wide ones take 80 KB of LDS, still two blocks per CU, and run
// where they need fewer block rounds for the work.
template <bool DMA, int SH>
struct QKVShape {
    static constexpr int BA = 128, BB = 128;
    using Tile = MfmaTile<128, 128, 2, 2>;
};
template <int SH>
struct QKVShape<true, SH> {
    static constexpr int BA = SH == 1 ? 192 : 128, BB = SH == 2 ? 192 : 128;
    using Tile = DmaTile<BA, BB, 2, 2, false, 2>;
};
template <bool DMA, int SH = 0>
using QKVTile = typename QKVShape<DMA, SH>::Tile;

template <bool DMA, int SH, bool VARLEN>
__global__ __launch_bounds__(256) void k_proj_qkv(RowMap rm, const uint16_t *__restrict__ wq,
                                                  const uint16_t *__restrict__ wk, const uint16_t *__restrict__ wv,
                                                  int hd, int dh, float qscale, int nw, int n_qk_at, int n_bt,
                                                  int n_v_at, int n_v_bt, int n_seq, int L, int lpad, int zero_pad,
                                                  const int32_t *__restrict__ seq_off, uint16_t *__restrict__ Q,
                                                  uint16_t *__restrict__ K, uint16_t *__restrict__ Vt) {
    using T = QKVTile<DMA, SH>;
    using Rows = typename std::conditional<DMA, DmaRows, RegRows>::type;
    constexpr int BA = QKVShape<DMA, SH>::BA, BB = QKVShape<DMA, SH>::BB;
    static_assert((size_t)BB * (BA + 8) * 2 <= T::LDS_BYTES, "staged rows fit in the ring");
    extern __shared__ __align__(16) uint16_t lds[];
    const int n_qk = n_qk_at * n_bt;
    const int total = n_qk + n_v_at * n_v_bt;
    const int lid = xcd_remap(blockIdx.x, total);
    const uint16_t *rowsA[T::CA], *rowsB[T::CB];
    T t;
    if (lid < n_qk) {
        int at, bt;
        tile_order(lid, n_qk_at, n_bt, at, bt);
#pragma unroll
        for (int i = 0; i < T::CA; ++i) {
            const int a = at * BA + T::chunk_row(i);
            const uint16_t *w = a < hd ? wq + (long)a * rm.C
                              : a < 2 * hd ? wk + (long)(a - hd) * rm.C
                                           : wv + (long)(a - 2 * hd) * rm.C;
            rowsA[i] = a < nw * hd ? w : nullptr;
        }
#pragma unroll
        for (int i = 0; i < T::CB; ++i) rowsB[i] = rm.row(bt * BB + T::chunk_row(i));
        run_tile(t, lds, rowsA, rowsB, wq, rm.row(0), rm.C, Rows{});
        const int a0 = at * BA, b0 = bt * BB;
        stage_rows<BA>(t, lds, [&](float v, int a) { return f2h_bits(a0 + a < hd ? v * qscale : v); },
                       [](int a) { return a; });
        __syncthreads();
        write_rows<BA, BB>(lds, min(BA, nw * hd - a0), [&](int b, int c0) -> uint16_t * {
            const int r = b0 + b, a = a0 + c0;
            if (r >= rm.n_rows) return nullptr;
            return a < hd ? Q + (long)r * hd + a
                 : a < 2 * hd ? K + (long)r * hd + (a - hd)
                              : Vt + (long)r * hd + (a - 2 * hd);
        });
        return;
    }
    // V tile: at over batch rows, bt over features
    int at, bt;
    tile_order(lid - n_qk, n_v_at, n_v_bt, at, bt);
#pragma unroll
    for (int i = 0; i < T::CA; ++i) rowsA[i] = rm.row(at * BA + T::chunk_row(i));
#pragma unroll
    for (int i = 0; i < T::CB; ++i) {
        const int b = bt * BB + T::chunk_row(i);
        rowsB[i] = b < hd ? wv + (long)b * rm.C : nullptr;
    }
    run_tile(t, lds, rowsA, rowsB, rm.row(0), wv, rm.C, Rows{});
    const int Lk = n_seq == 1 ? rm.n_rows : L;
    const int r0 = at * BA, f0 = bt * BB;
    if (!VARLEN && (n_seq == 1 || L % BA == 0)) {
        const int s = n_seq == 1 ? 0 : r0 / L, j0 = r0 - s * L;   // j0 is a multiple of BA
        stage_rows<BA>(t, lds, [&](float v, int a) { return (uint16_t)(j0 + a < Lk ? f2h_bits(v) : 0); },
                       [](int a) { return vt_key_of_pos(a); });
        __syncthreads();
        write_rows<BA, BB>(lds, min(BA, lpad - j0), [&](int b, int c0) -> uint16_t * {
            const int f = f0 + b;
            if (f >= hd) return nullptr;
            const int h = f / dh, d = f - h * dh;
            return Vt + (((long)h * n_seq + s) * dh + d) * lpad + j0 + c0;
        });
        return;
    }
#pragma unroll
    for (int j = 0; j < T::TB; ++j) {
        const int f = f0 + T::b_of(j);
        if (f >= hd) continue;
        const int h = f / dh, d = f - h * dh;
#pragma unroll
        for (int i = 0; i < T::TA; ++i)
#pragma unroll
            for (int g = 0; g < 4; ++g)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int r = r0 + T::a_of(i, g) + e;
                    if (r >= rm.n_rows) continue;
                    int s, jj;
                    seq_pos(r, n_seq, L, s, jj, VARLEN ? seq_off : nullptr);
                    Vt[(((long)h * n_seq + s) * dh + d) * lpad + vt_key_of_pos(jj)] = f2h_bits(t.acc[i][j][4 * g + e]);
                }
    }
    // zero the padded key positions [Lk, lpad) of this block's features, for
    // the sequences s = at, at + n_v_at, ... (the DMA-staged attention reads them)
    const int npad = lpad - Lk;
    if (!VARLEN && zero_pad && npad > 0) {
        for (int sq = at; sq < n_seq; sq += n_v_at)
            for (int idx = threadIdx.x; idx < BB * npad; idx += blockDim.x) {
                const int f = f0 + idx / npad, jj = Lk + idx % npad;
                if (f >= hd) continue;
                const int h = f / dh, d = f - h * dh;
                Vt[(((long)h * n_seq + sq) * dh + d) * lpad + vt_key_of_pos(jj)] = 0;
            }
    }
}

// tiles of a BA x BB launch over rows
static long qkv_tiles(const Plan &p, int rows, int nw, int BA, int BB) {
    return (long)cdiv(nw * p.hd, BA) * cdiv(rows, BB) + (nw == 3 ? 0L : (long)cdiv(rows, BA) * cdiv(p.hd, BB));
}

template <bool DMA, int SH, bool VARLEN>
static hipError_t launch_qkv(const Plan &p, const RowMap &rm, const AttnArgs &a, float qscale, int nw, int zero_pad,
                             hipStream_t st) {
    constexpr int BA = QKVShape<DMA, SH>::BA, BB = QKVShape<DMA, SH>::BB;
    const hipError_t e = allow_lds(k_proj_qkv<DMA, SH, VARLEN>, QKVTile<DMA, SH>::LDS_BYTES);
    if (e != hipSuccess) return e;
    const int n_qk_at = cdiv(nw * p.hd, BA), n_bt = cdiv(rm.n_rows, BB);
    const int n_v_at = nw == 3 ? 0 : cdiv(rm.n_rows, BA), n_v_bt = nw == 3 ? 0 : cdiv(p.hd, BB);
    const int total = n_qk_at * n_bt + n_v_at * n_v_bt;
    launch_k(k_proj_qkv<DMA, SH, VARLEN>, total, 256, QKVTile<DMA, SH>::LDS_BYTES, st, rm, (const uint16_t *)a.wq,
             (const uint16_t *)a.wk, (const uint16_t *)a.wv, p.hd, p.dh, qscale, nw, n_qk_at, n_bt, n_v_at, n_v_bt,
             a.n_seq, a.L, a.lpad, zero_pad, a.seq_off, (uint16_t *)a.q, (uint16_t *)a.k, (uint16_t *)a.vt);
    return hipGetLastError();
}

// Tile shape by block rounds; V: sequences of varying length (a separate
// instance, so that the uniform kernels carry none of its code)
template <bool V>
static hipError_t launch_shape(const Plan &p, const RowMap &rm, const AttnArgs &a, float qscale, int nw,
                               int zero_pad, hipStream_t st) {
    if (p.C % 64 != 0) return launch_qkv<false, 0, V>(p, rm, a, qscale, nw, zero_pad, st);
    // block rounds (two blocks per CU) times the work of one tile, a wide
    // tile being 1.5 units (the SD3-like layer at r = 0.5: 460 tiles of 192 x
    // 128 in one round, 44 us, against 684 of 128 x 128 in two, 51 us; one
    // round either way, or two either way, keeps the smaller tiles).  192-row
    // V tiles must stay whole runs of one sequence (else Vt is stored element
    // by element: 58 against 42 us on the Latte-like spatial layer, 256-token
    // sequences), which 128 x 192 keeps at 128 rows.
    const long slots = 2L * N_CUS;
    const long c128 = 2 * ((qkv_tiles(p, rm.n_rows, nw, 128, 128) + slots - 1) / slots);
    const long c192a = 3 * ((qkv_tiles(p, rm.n_rows, nw, 192, 128) + slots - 1) / slots);
    const long c192b = 3 * ((qkv_tiles(p, rm.n_rows, nw, 128, 192) + slots - 1) / slots);
    const bool rows192 = nw == 3 || a.n_seq == 1 || a.L % 192 == 0;
    if (rows192 && c192a < c128 && c192a <= c192b) return launch_qkv<true, 1, V>(p, rm, a, qscale, nw, zero_pad, st);
    if (c192b < c128) return launch_qkv<true, 2, V>(p, rm, a, qscale, nw, zero_pad, st);
    return launch_qkv<true, 0, V>(p, rm, a, qscale, nw, zero_pad, st);
}

hipError_t launch_proj_qkv(const Plan &p, const RowMap &rm, const AttnArgs &a, hipStream_t st) {
    const float qscale = (float)(1.4426950408889634 / sqrt((double)p.dh));
    StageScope _stage(st, "proj_qkv");
    const int Lk = a.n_seq == 1 ? rm.n_rows : a.L;
    // sequences of varying length: Vt slots per sequence, filled element by
    // element; the attention masks their ends itself (no padding to zero)
    const bool varlen = a.seq_off != nullptr;
    const int zero_pad = !varlen && flash_uses_dma(p.dh, Lk, p.hd) ? 1 : 0;
    // short sequences: V rows from the Q/K tiles (nw = 3), no V tiles
    const int nw = !varlen && attn_short(Lk) ? 3 : 2;
    return varlen ? launch_shape<true>(p, rm, a, qscale, nw, zero_pad, st)
                  : launch_shape<false>(p, rm, a, qscale, nw, zero_pad, st);
}

// ---------------------------------------------------------------------------
// Output projection: a in [0, C) = rows of wo (fp16); b = batch rows of O.
// y[out row][a].
// ---------------------------------------------------------------------------
// Tiles (double-buffered DMA): 128 output features x 64 rows, or 64 x 64
// where the 128 x 64 grid would give fewer than 1.5 blocks per CU (the
// SD3-like layer at r = 0.75, 1357 rows: 528 small blocks instead of 264,
// 2.4 us less per step; at r = 0.5 and 0.25 the 128-wide tiles are faster);
// for C a multiple of 160 but not of 128 (e.g. 320) 160 features x 128 rows
// (one wave row of four), so that no feature column is computed in vain.
template <bool DMA, int BA = 128>
using OTile = typename std::conditional<
    DMA,
    typename std::conditional<
        BA == 160, DmaTile<160, 128, 1, 4, true, 2>,
        typename std::conditional<BA == 64, DmaTile<64, 64, 2, 2, true, 2>, DmaTile<128, 64, 2, 2, true, 2>>::type>::type,
    MfmaTile<128, 128, 2, 2, true, false>>::type;

template <bool DMA, int BA>
__global__ __launch_bounds__(256) void k_proj_out(const uint16_t *__restrict__ O, int n_rows, int hd,
                                                  const uint16_t *__restrict__ wo, int C, int n_main,
                                                  const int32_t *__restrict__ out_idx, int tF, int tN, int n_at,
                                                  int n_bt,
                                                  uint16_t *__restrict__ y, uint16_t *__restrict__ y_ctx) {
    using T = OTile<DMA, BA>;
    constexpr int BB = DMA ? (BA == 160 ? 128 : 64) : 128;
    extern __shared__ __align__(16) uint16_t lds[];
    int at, bt;
    tile_order(xcd_remap(blockIdx.x, n_at * n_bt), n_at, n_bt, at, bt);
    const uint16_t *rowsA[T::CA], *rowsB[T::CB];
#pragma unroll
    for (int i = 0; i < T::CA; ++i) {
        const int a = at * BA + T::chunk_row(i);
        rowsA[i] = a < C ? wo + (long)a * hd : nullptr;
    }
#pragma unroll
    for (int i = 0; i < T::CB; ++i) {
        const int b = bt * BB + T::chunk_row(i);
        rowsB[i] = b < n_rows ? O + (long)b * hd : nullptr;
    }
    T t;
    run_tile(t, lds, rowsA, rowsB, wo, O, hd, typename std::conditional<DMA, DmaRows, RegRows>::type{});
    const int a0 = at * BA, b0 = bt * BB;
    stage_rows<BA>(t, lds, [](float v, int) { return f2bf(v); }, [](int a) { return a; });
    __syncthreads();
    write_rows<BA, BB>(lds, min(BA, C - a0), [&](int b, int c0) -> uint16_t * {
        const int r = b0 + b;
        if (r >= n_rows) return nullptr;
        uint16_t *yrow = r < n_main ? y + batch_token(r, out_idx, tF, tN) * C : y_ctx + (long)(r - n_main) * C;
        return yrow + a0 + c0;
    });
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
        launch_k(k_to_f16, (unsigned)(blocks < 2048 ? blocks : 2048), 256, 0, st, (const uint4 *)a.wo, n8,
                                                                            (uint4 *)a.wo16);
    }
    StageScope _stage(st, "proj_out");
    auto go = [&](auto kern, size_t lds, int BA, int BB) -> hipError_t {
        const int n_at = cdiv(p.C, BA), n_bt = cdiv(n_rows, BB);
        launch_k(kern, n_at * n_bt, 256, lds, st, (const uint16_t *)a.o, n_rows, p.hd, (const uint16_t *)a.wo16, p.C,
                 a.n_main, a.out_idx, a.tF, a.tN, n_at, n_bt, (uint16_t *)a.y, (uint16_t *)a.y_ctx);
        return hipSuccess;
    };
    if (p.hd % 64 == 0) {
        if (p.C % 160 == 0 && p.C % 128 != 0) {
            hipError_t e = allow_lds(k_proj_out<true, 160>, OTile<true, 160>::LDS_BYTES);
            if (e != hipSuccess) return e;
            go(k_proj_out<true, 160>, OTile<true, 160>::LDS_BYTES, 160, 128);
        } else if (2L * cdiv(p.C, 128) * cdiv(n_rows, 64) < 3L * N_CUS) {
            go(k_proj_out<true, 64>, OTile<true, 64>::LDS_BYTES, 64, 64);
        } else {
            hipError_t e = allow_lds(k_proj_out<true, 128>, OTile<true, 128>::LDS_BYTES);
            if (e != hipSuccess) return e;
            go(k_proj_out<true, 128>, OTile<true, 128>::LDS_BYTES, 128, 64);
        }
    } else {
        go(k_proj_out<false, 128>, OTile<false, 128>::LDS_BYTES, 128, 128);
    }
    return hipGetLastError();
}

}  // namespace oc
