// Flash-style attention over the retained tokens (OmniCache §3.2.3: the
// layer runs on the retained tokens only), fp16 MFMA with fp32 accumulation.
//
// One block = NW waves of one (sequence, head); a wave owns QB blocks of 32
// queries.  Per 64-key tile:
//   S^T = K Q^T  on v_mfma_f32_32x32x16_f16: K rows from LDS are the A
//                operand, the wave's Q fragments (registers) the B operand,
//                so the result lane l holds query l%32 and 16 of the 32 keys
//                of each key block (rows 8*(i/4) + 4*(l/32) + i%4);
//   softmax in the log2 domain (Q is pre-scaled by log2(e)/sqrt(dh)) with a
//                lazily rebased reference maximum m: the S accumulator starts
//                at -m, so the MFMA itself yields s - m; only when a score
//                exceeds m by more than REBASE (or on the first tile) is m
//                raised and O and the running sum rescaled.  P = exp2(s - m)
//                <= 2^REBASE stays well inside fp16.  One lane owns one query:
//                the tile maximum needs a single exchange with lane l^32, the
//                running sum none until the end;
//   O^T += Vt P^T on the same MFMA: P leaves the score registers as the B
//                operand directly (8 consecutive accumulator slots = 8 keys),
//                and Vt rows are staged in LDS with the keys of each 16-key
//                block permuted so that the matching A operand is one
//                contiguous 16-byte read.
// K and Vt tiles are double-buffered in LDS with a register prefetch of the
// next tile and one barrier per tile; only the last tile is masked.  Blocks
// of one head are kept on one XCD (xcd_remap) so its K/V stay in its L2.
#include "oc_attn_common.h"
#include "oc_mfma_tile.h"

namespace oc {

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr float REBASE = 8.f;

template <int DH, int QB, int NW>
__global__ __launch_bounds__(NW * 64) void k_flash(const uint16_t *__restrict__ Q, const uint16_t *__restrict__ K,
                                                    const uint16_t *__restrict__ Vt, uint16_t *__restrict__ O,
                                                    int hd, int heads, int n_seq, int L, int Lk, int lpad,
                                                    int n_qt) {
    constexpr int DK = (DH + 15) / 16 * 16;     // S^T k-loop (16 per MFMA)
    constexpr int DV = (DH + 31) / 32 * 32;     // O^T row blocks of 32
    constexpr int KT = 64;                      // keys per tile
    constexpr int LDK = DK + 8, LDV = KT + 8;   // padded LDS rows (halves)
    constexpr int NT = NW * 64, QW = 32 * QB, QT = QW * NW;
    constexpr int KCH = KT * (DK / 8), VCH = DV * (KT / 8);
    constexpr int KPT = (KCH + NT - 1) / NT, VPT = (VCH + NT - 1) / NT;
    __shared__ __align__(16) uint16_t Ks[2][KT * LDK];
    __shared__ __align__(16) uint16_t Vs[2][DV * LDV];

    const int total = n_qt * heads * n_seq;
    const int lid = xcd_remap(blockIdx.x, total);
    const int qt = lid % n_qt, hs = lid / n_qt, h = hs % heads, s = hs / heads;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, ln = lane & 31, lg = lane >> 5;
    const long row0 = (long)s * L;
    const int q_base = qt * QT + wave * QW;
    const uint16_t *kbase = K + row0 * hd + h * DH;
    const uint16_t *vbase = Vt + ((long)h * n_seq + s) * DH * lpad;

    f16x8 qf[QB][DK / 16];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        const int q = q_base + qb * 32 + ln;
#pragma unroll
        for (int ks = 0; ks < DK / 16; ++ks) {
            const int d0 = ks * 16 + lg * 8;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (q < Lk && d0 < DH) v = *reinterpret_cast<const uint4 *>(Q + (row0 + q) * hd + h * DH + d0);
            qf[qb][ks] = *reinterpret_cast<f16x8 *>(&v);
        }
    }

    // this thread's staging slots (fixed across tiles)
    const uint16_t *kp[KPT];
    int kkey[KPT], klds[KPT];
    bool kok[KPT];
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
        const int c = threadIdx.x + i * NT;
        const int key = c / (DK / 8), d0 = (c % (DK / 8)) * 8;
        kok[i] = c < KCH && d0 < DH;
        kkey[i] = key;
        kp[i] = kbase + (long)key * hd + d0;
        klds[i] = key * LDK + d0;
    }
    const uint16_t *vp[VPT];
    int vkey[VPT], vlds[VPT];
    bool vok[VPT];
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
        const int c = threadIdx.x + i * NT;
        const int d = c >> 3, kc = c & 7;
        vok[i] = c < VCH && d < DH;
        vkey[i] = kc * 8;
        vp[i] = vbase + (long)d * lpad + kc * 8;
        // keys 8kc..8kc+3 -> position off, keys 8kc+4..8kc+7 -> 8+off of their 16-key block
        vlds[i] = d * LDV + (kc >> 1) * 16 + (kc & 1) * 4;
    }
    uint4 kr0[KPT], vr0[VPT], kr1[KPT], vr1[VPT];
    const long kstep = (long)KT * hd;
    auto load = [&](int k0, bool tail, uint4 *kr, uint4 *vr) {
#pragma unroll
        for (int i = 0; i < KPT; ++i) {
            uint4 v = make_uint4(0, 0, 0, 0);
            if (kok[i] && (!tail || k0 + kkey[i] < Lk)) v = *reinterpret_cast<const uint4 *>(kp[i] + (k0 / KT) * kstep);
            kr[i] = v;
        }
#pragma unroll
        for (int i = 0; i < VPT; ++i) {
            uint4 v = make_uint4(0, 0, 0, 0);
            if (vok[i]) {
                v = *reinterpret_cast<const uint4 *>(vp[i] + k0);
                if (tail) {
                    const int valid = Lk - (k0 + vkey[i]);
                    uint16_t *e = reinterpret_cast<uint16_t *>(&v);
#pragma unroll
                    for (int t = 0; t < 8; ++t)
                        if (t >= valid) e[t] = 0;
                }
            }
            vr[i] = v;
        }
    };
    auto store = [&](int buf, const uint4 *kr, const uint4 *vr) {
#pragma unroll
        for (int i = 0; i < KPT; ++i)
            if (threadIdx.x + i * NT < KCH) *reinterpret_cast<uint4 *>(&Ks[buf][klds[i]]) = kr[i];
#pragma unroll
        for (int i = 0; i < VPT; ++i)
            if (threadIdx.x + i * NT < VCH) {
                uint16_t *dst = &Vs[buf][vlds[i]];
                *reinterpret_cast<uint2 *>(dst) = make_uint2(vr[i].x, vr[i].y);
                *reinterpret_cast<uint2 *>(dst + 8) = make_uint2(vr[i].z, vr[i].w);
            }
    };

    f32x16 o[QB][DV / 32];
    float m[QB], l[QB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        m[qb] = 0.f;
        l[qb] = 0.f;
#pragma unroll
        for (int db = 0; db < DV / 32; ++db) o[qb][db] = f32x16{};
    }

    // tile kt lives in LDS buffer kt&1; global loads run two tiles ahead of
    // the buffer they fill, through two register sets
    const int n_kt = cdiv(Lk, KT);
    load(0, KT > Lk, kr0, vr0);
    store(0, kr0, vr0);
    if (n_kt > 1) load(KT, 2 * KT > Lk, kr1, vr1);
    if (n_kt > 2) load(2 * KT, 3 * KT > Lk, kr0, vr0);
    __syncthreads();
    auto tile = [&](int kt, int buf) {
        const int k0 = kt * KT;
        f32x16 sc[QB][2];
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
            f32x16 init;
#pragma unroll
            for (int i = 0; i < 16; ++i) init[i] = -m[qb];
            sc[qb][0] = sc[qb][1] = init;
        }
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int ks = 0; ks < DK / 16; ++ks) {
                const f16x8 kf = *reinterpret_cast<const f16x8 *>(&Ks[buf][(kb * 32 + ln) * LDK + ks * 16 + lg * 8]);
#pragma unroll
                for (int qb = 0; qb < QB; ++qb)
                    sc[qb][kb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(kf, qf[qb][ks], sc[qb][kb], 0, 0, 0);
            }
        if (k0 + KT > Lk) {
#pragma unroll
            for (int qb = 0; qb < QB; ++qb)
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int i = 0; i < 16; ++i)
                        if (k0 + kb * 32 + 8 * (i >> 2) + 4 * lg + (i & 3) >= Lk) sc[qb][kb][i] = -INFINITY;
        }
        f16x8 pf[QB][4];
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
            float t = -INFINITY;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 16; ++i) t = fmaxf(t, sc[qb][kb][i]);
            t = fmaxf(t, __shfl_xor(t, 32, 64));
            if (kt == 0 || t > REBASE) {
                // raise the reference maximum by t: rescale what was accumulated
                // (nothing yet on the first tile, where t may be of any sign)
                if (kt > 0) {
                    const float alpha = __builtin_amdgcn_exp2f(-t);
                    l[qb] *= alpha;
#pragma unroll
                    for (int db = 0; db < DV / 32; ++db) o[qb][db] *= alpha;
                }
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int i = 0; i < 16; ++i) sc[qb][kb][i] -= t;
                m[qb] += t;
            }
            float ls = 0.f;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int hf = 0; hf < 2; ++hf) {
                    f16x8 f;
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const float p = __builtin_amdgcn_exp2f(sc[qb][kb][8 * hf + e]);
                        ls += p;
                        f[e] = (_Float16)p;
                    }
                    pf[qb][kb * 2 + hf] = f;
                }
            l[qb] += ls;
        }
#pragma unroll
        for (int db = 0; db < DV / 32; ++db)
#pragma unroll
            for (int kstep4 = 0; kstep4 < 4; ++kstep4) {
                const f16x8 vf =
                    *reinterpret_cast<const f16x8 *>(&Vs[buf][(db * 32 + ln) * LDV + kstep4 * 16 + lg * 8]);
#pragma unroll
                for (int qb = 0; qb < QB; ++qb)
                    o[qb][db] = __builtin_amdgcn_mfma_f32_32x32x16_f16(vf, pf[qb][kstep4], o[qb][db], 0, 0, 0);
            }
    };
    for (int kt = 0; kt < n_kt; kt += 2) {
        tile(kt, 0);
        if (kt + 1 < n_kt) store(1, kr1, vr1);
        if (kt + 3 < n_kt) load((kt + 3) * KT, (kt + 4) * KT > Lk, kr1, vr1);
        __syncthreads();
        if (kt + 1 >= n_kt) break;
        tile(kt + 1, 1);
        if (kt + 2 < n_kt) store(0, kr0, vr0);
        if (kt + 4 < n_kt) load((kt + 4) * KT, (kt + 5) * KT > Lk, kr0, vr0);
        __syncthreads();
    }
    // normalise and store: lane holds query ln, d = db*32 + 8*g4 + 4*lg + e
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        const float lt = l[qb] + __shfl_xor(l[qb], 32, 64);
        const float inv = 1.f / lt;
        const int q = q_base + qb * 32 + ln;
        if (q >= Lk) continue;
        uint16_t *orow = O + (row0 + q) * hd + h * DH;
#pragma unroll
        for (int db = 0; db < DV / 32; ++db)
#pragma unroll
            for (int g4 = 0; g4 < 4; ++g4) {
                const int d = db * 32 + 8 * g4 + 4 * lg;
                if (d >= DH) continue;
                u16x4 v;
#pragma unroll
                for (int e = 0; e < 4; ++e) v[e] = f2h_bits(o[qb][db][4 * g4 + e] * inv);
                *reinterpret_cast<u16x4 *>(orow + d) = v;
            }
    }
}

template <int DH, int QB, int NW>
static hipError_t go(const Plan &p, const AttnArgs &a, int Lk, hipStream_t st) {
    const int n_qt = cdiv(Lk, 32 * QB * NW);
    const int total = n_qt * p.heads * a.n_seq;
    k_flash<DH, QB, NW><<<total, NW * 64, 0, st>>>((const uint16_t *)a.q, (const uint16_t *)a.k,
                                                    (const uint16_t *)a.vt, (uint16_t *)a.o, p.hd, p.heads, a.n_seq,
                                                    a.L, Lk, a.lpad, n_qt);
    return hipGetLastError();
}

// Query-tile shape by sequence length (measured on MI355X: 4 waves of 32
// queries beat 2 and beat two 32-query blocks per wave at every length of
// the SD3-like layer): a short sequence gets one or two waves per block.
template <int DH>
static hipError_t go_dh(const Plan &p, const AttnArgs &a, int Lk, hipStream_t st) {
    if (Lk <= 32) return go<DH, 1, 1>(p, a, Lk, st);
    if (Lk <= 64) return go<DH, 1, 2>(p, a, Lk, st);
    return go<DH, 1, 4>(p, a, Lk, st);
}

hipError_t launch_flash(const Plan &p, const AttnArgs &a, int Lk, hipStream_t st) {
    StageScope _stage(st, "flash");
    switch (p.dh) {
        case 16: return go_dh<16>(p, a, Lk, st);
        case 32: return go_dh<32>(p, a, Lk, st);
        case 48: return go_dh<48>(p, a, Lk, st);
        case 64: return go_dh<64>(p, a, Lk, st);
        case 72: return go_dh<72>(p, a, Lk, st);
        case 80: return go_dh<80>(p, a, Lk, st);
        case 96: return go_dh<96>(p, a, Lk, st);
        case 128: return go_dh<128>(p, a, Lk, st);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace oc
