// Short sequences (at most 64 keys, head dim 64, e.g. a temporal layer over
// 25 frames): the Q, K and V projections of one head and the attention over
// the sequences of a tile in one kernel (OmniCache §3.2.1: the temporal
// attention runs per spatial position over the frames), so Q, K and V never
// reach HBM; only O is written, for the output projection.
//
// Block (row tile t, head h).  A row tile holds S_t = floor(128 / L) whole
// sequences: slot b (0..127) is token j = b mod L of sequence t*S_t + b / L
// (slots past S_t*L, or past the last sequence, carry no token).  The MFMA
// tile computes [192 features x 128 slots] over K = C: features 0..63 are
// rows of wq for head h, 64..127 of wk, 128..191 of wv (bf16 products,
// fp32 accumulation; Q scaled by log2(e)/sqrt(dh)).  The epilogue stages Q
// and K by slot rows and V transposed (d rows, slot positions permuted inside
// 16-slot blocks as the Vt layout of the long-sequence kernels), all fp16 in
// LDS.  Each wave then takes 32 query slots: S^T = K Q^T over the 32-slot key
// blocks that hold its queries' sequences, keys of other sequences masked,
// the exact maximum, P = exp2(s - max) in fp16, the running sum of that
// fp16 P, O^T = Vt P^T, and O = O^T / sum written by rows [rows, H*dh].
#include "oc_internal.h"
#include "oc_launch.h"
#include "oc_device.h"
#include "oc_mfma_tile.h"
#include "oc_dma_tile.h"
#include "oc_attn_common.h"

namespace oc {

namespace {
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
using ShortTile = DmaTile<192, 128, 2, 2, false, 2>;
constexpr int SH_DH = 64;
constexpr int QKS = 128 + 8;   // LDS row of a slot: Q (64) | K (64) | pad, halves
constexpr int VTS = 128 + 8;   // LDS row of one V dim over the 128 slots, halves
constexpr size_t SH_STAGE_BYTES = (size_t)(128 * QKS + SH_DH * VTS) * 2;
static_assert(SH_STAGE_BYTES <= ShortTile::LDS_BYTES, "staging fits in the ring");
}  // namespace

__global__ __launch_bounds__(256) void k_qkv_attn_short(RowMap rm, const uint16_t *__restrict__ wq,
                                                        const uint16_t *__restrict__ wk,
                                                        const uint16_t *__restrict__ wv, int hd, int heads,
                                                        int n_seq, int L, int s_t, int n_tiles, float qscale,
                                                        uint16_t *__restrict__ O) {
    using T = ShortTile;
    extern __shared__ __align__(16) uint16_t lds[];
    const int lid = xcd_remap(blockIdx.x, n_tiles * heads);
    const int h = lid % heads, tile = lid / heads;
    const int seq0 = tile * s_t;
    const int n_valid_seq = min(s_t, n_seq - seq0);
    const int n_slots = n_valid_seq * L;
    const int C = rm.C;

    // ---- projection: [192 features x 128 slots] ----
    const uint16_t *rowsA[T::CA], *rowsB[T::CB];
#pragma unroll
    for (int i = 0; i < T::CA; ++i) {
        const int a = T::chunk_row(i);
        const uint16_t *w = a < SH_DH ? wq : (a < 2 * SH_DH ? wk : wv);
        rowsA[i] = w + (long)(h * SH_DH + (a & (SH_DH - 1))) * C;
    }
#pragma unroll
    for (int i = 0; i < T::CB; ++i) {
        const int b = T::chunk_row(i);
        rowsB[i] = b < n_slots ? rm.row(seq0 * L + b) : nullptr;
    }
    T t;
    t.run(lds, rowsA, rowsB, wq, rm.row(seq0 * L), C, 0, 0);

    // ---- stage Q, K by slot rows and V transposed, fp16 ----
    uint16_t *const QK = lds;
    uint16_t *const VT = lds + 128 * QKS;
#pragma unroll
    for (int j = 0; j < T::TB; ++j) {
        const int b = T::b_of(j);
#pragma unroll
        for (int i = 0; i < T::TA; ++i)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int a = T::a_of(i, g);   // 4 consecutive features a .. a+3 (never straddling Q/K/V)
                if (a < 2 * SH_DH) {
                    const float sc = a < SH_DH ? qscale : 1.f;
                    u16x4 v;
#pragma unroll
                    for (int e = 0; e < 4; ++e) v[e] = f2h_bits(t.acc[i][j][4 * g + e] * sc);
                    *reinterpret_cast<u16x4 *>(QK + b * QKS + a) = v;
                } else {
                    const int pos = vt_key_of_pos(b);
#pragma unroll
                    for (int e = 0; e < 4; ++e) VT[(a - 2 * SH_DH + e) * VTS + pos] = f2h_bits(t.acc[i][j][4 * g + e]);
                }
            }
    }
    __syncthreads();

    // ---- attention: wave w takes query slots 32w .. 32w+31 ----
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, ln = lane & 31, lg = lane >> 5;
    const int qs = wave * 32 + ln;
    const int sq = qs / L;
    const int lo = sq * L, hi = lo + L;
    const bool qvalid = qs < n_slots;
    // key blocks holding the sequences of this wave's valid queries
    const int q_first = wave * 32, q_last = min(wave * 32 + 31, n_slots - 1);
    if (q_first >= n_slots) return;   // no valid query in this wave (no barrier follows)
    const int kb_lo = (q_first / L) * L / 32, kb_hi = ((q_last / L) * L + L - 1) / 32;
    f16x8 qf[4];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) qf[ks] = *reinterpret_cast<const f16x8 *>(QK + qs * QKS + ks * 16 + lg * 8);
    f32x16 sc[4];
    float m = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
        if (kb < kb_lo || kb > kb_hi) {
#pragma unroll
            for (int i = 0; i < 16; ++i) sc[kb][i] = -INFINITY;   // no key of these queries: P = 0
            continue;
        }
        sc[kb] = f32x16{};
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            const f16x8 kf = *reinterpret_cast<const f16x8 *>(QK + (kb * 32 + ln) * QKS + SH_DH + ks * 16 + lg * 8);
            sc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(kf, qf[ks], sc[kb], 0, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int key = kb * 32 + 8 * (i >> 2) + 4 * lg + (i & 3);
            if (key < lo || key >= hi) sc[kb][i] = -INFINITY;
            m = fmaxf(m, sc[kb][i]);
        }
    }
    m = fmaxf(m, __shfl_xor(m, 32, 64));
    if (!(m > -INFINITY)) m = 0.f;   // a query with no key (not stored)
    const f16x2 ones = {(_Float16)1.f, (_Float16)1.f};
    f16x8 pf[8];
    float l0 = 0.f, l1 = 0.f;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
            f16x8 f;
#pragma unroll
            for (int e = 0; e < 8; ++e) f[e] = (_Float16)__builtin_amdgcn_exp2f(sc[kb][8 * hf + e] - m);
            pf[kb * 2 + hf] = f;
            l0 = __builtin_amdgcn_fdot2(f.s01, ones, l0, false);
            l1 = __builtin_amdgcn_fdot2(f.s23, ones, l1, false);
            l0 = __builtin_amdgcn_fdot2(f.s45, ones, l0, false);
            l1 = __builtin_amdgcn_fdot2(f.s67, ones, l1, false);
        }
    float lt = l0 + l1;
    lt += __shfl_xor(lt, 32, 64);
    f32x16 o[2];
#pragma unroll
    for (int db = 0; db < 2; ++db) {
        o[db] = f32x16{};
#pragma unroll
        for (int k4 = 0; k4 < 8; ++k4) {
            if (k4 / 2 < kb_lo || k4 / 2 > kb_hi) continue;
            const f16x8 vf = *reinterpret_cast<const f16x8 *>(VT + (db * 32 + ln) * VTS + k4 * 16 + lg * 8);
            o[db] = __builtin_amdgcn_mfma_f32_32x32x16_f16(vf, pf[k4], o[db], 0, 0, 0);
        }
    }
    if (!qvalid) return;
    const float inv = 1.f / lt;
    const long row = (long)(seq0 + sq) * L + (qs - lo);
    uint16_t *orow = O + row * hd + h * SH_DH;
#pragma unroll
    for (int db = 0; db < 2; ++db)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
            const int d = db * 32 + 8 * g4 + 4 * lg;
            u16x4 v;
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = f2h_bits(o[db][4 * g4 + e] * inv);
            *reinterpret_cast<u16x4 *>(orow + d) = v;
        }
}

bool qkv_attn_short_applies(const Plan &p, const AttnArgs &a) {
    return p.bf16 && p.dh == SH_DH && p.C % 64 == 0 && a.n_ctx == 0 && a.seq_off == nullptr && a.n_seq >= 1 &&
           a.L >= 1 &&
           attn_short(a.L) && (long)a.n_seq * a.L < (1L << 31);
}

hipError_t launch_qkv_attn_short(const Plan &p, const RowMap &rm, const AttnArgs &a, hipStream_t st) {
    if (!qkv_attn_short_applies(p, a)) return hipErrorInvalidValue;
    StageScope _stage(st, "qkv_attn_short");
    const int s_t = 128 / a.L;
    const int n_tiles = cdiv(a.n_seq, s_t);
    const float qscale = (float)(1.4426950408889634 / sqrt((double)p.dh));
    const hipError_t e = raise_lds_limit((const void *)k_qkv_attn_short, ShortTile::LDS_BYTES);
    if (e != hipSuccess) return e;
    launch_k(k_qkv_attn_short, (unsigned)(n_tiles * p.heads), 256, ShortTile::LDS_BYTES, st, rm,
             (const uint16_t *)a.wq, (const uint16_t *)a.wk, (const uint16_t *)a.wv, p.hd, p.heads, a.n_seq, a.L,
             s_t, n_tiles, qscale, (uint16_t *)a.o);
    return hipGetLastError();
}

}  // namespace oc
