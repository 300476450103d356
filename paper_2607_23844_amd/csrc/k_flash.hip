// Flash-style attention over the retained tokens (OmniCache §3.2.3: the
// layer runs on the retained tokens only), fp16 MFMA with fp32 accumulation.
//
// One block = NW waves of one (sequence, head); a wave owns 32 queries.  Per
// 64-key tile:
//   S^T = K Q^T  on v_mfma_f32_32x32x16_f16: K rows from LDS are the A
//                operand, the wave's Q fragments (registers) the B operand,
//                so lane l holds query l%32 and 16 of the 32 keys of each key
//                block (rows 8*(i/4) + 4*(l/32) + i%4);
//   softmax in the log2 domain (Q is pre-scaled by log2(e)/sqrt(dh)) against
//                a lazily raised reference maximum m: the S accumulator starts
//                at -m, so the MFMA itself yields s - m.  P = exp2(s - m) is
//                rounded to fp16 for the PV product; the packed fp16 maximum
//                of P tells whether any score exceeds m by more than REBASE
//                (or overflowed fp16).  Only then (and on the first tile) does
//                the wave take the slow path: the fp32 maximum t of both
//                lane halves, m += t, O and the running sum scaled by
//                exp2(-t), P recomputed.  The running sum adds the fp16 P that
//                the PV product uses (v_dot2 with ones, fp32 accumulation);
//   O^T += Vt P^T on the same MFMA: P leaves the score registers as the B
//                operand directly (8 consecutive accumulator slots = 8 keys).
//                Vt is stored with the keys of each 16-key block permuted
//                (quads 1 and 2 swapped, written so by the V projection), so
//                the matching A operand is one contiguous 16-byte read.
// K and Vt tiles go through a ring of LDS buffers with one barrier per tile;
// the K fragments of tile kt+1 are read into registers while tile kt
// finishes.  Two ways to fill the ring:
//   DMA (long sequences): global_load_lds moves 16 bytes per lane straight
//     into LDS, three tiles ahead, into a ring of four buffers.  Rows of 64
//     or 128 features (K of a head dim that is a multiple of 64, and every
//     Vt row of 64 keys) are unpadded with their 16-byte chunks XOR-swizzled
//     by row (chunk c of row r at slot c ^ ((r >> sh) & 7), sh = 1 for
//     128-byte rows, two of which fill the 64 LDS banks, 0 for 256-byte
//     rows); K rows of other head dims (72, 80, 96, ...) are padded to an odd
//     number of 16-byte chunks, whose feature padding the DMA fills with
//     zeros.  Either way the fragment reads of 16 consecutive rows hit
//     distinct banks.  Key rows past the end read as zeros (their scores
//     are masked) and the V projection zeroes the padded key
//     positions of Vt, so nothing needs masking in LDS; the Vt rows past the
//     head dim are never loaded and only feed output rows that are not
//     stored;
//   registers (short sequences, large grids of padded head dims): global
//     loads one tile ahead, masked, written to a ring of three padded
//     buffers.
// Only the last tile's scores are masked.  Blocks of one head are kept on one
// XCD (xcd_remap) so its K/V stay in that XCD's L2.
#include "oc_attn_common.h"
#include "oc_launch.h"
#include "oc_mfma_tile.h"

namespace oc {

typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

constexpr float REBASE = 8.f;   // P = exp2(s - m) stays below 2^REBASE on the fast path

template <int DH, bool DMA, int NW = 4>
struct FlashCfg {
    static constexpr int DK = (DH + 15) / 16 * 16;   // S^T k-loop (16 per MFMA)
    static constexpr int NKS = DK / 16;
    static constexpr int DV = (DH + 31) / 32 * 32;   // O^T row blocks of 32
    static constexpr int NDB = DV / 32;
    static constexpr int KT = 64;                    // keys per tile
    static constexpr int NBUF = DMA ? 4 : 3;
    // K rows: unpadded and swizzled for DMA of a head dim that is a multiple
    // of 64, else padded by 16 bytes (an odd number of 16-byte chunks per
    // row, so 16 consecutive rows start in distinct bank groups).  V rows
    // (64 keys): swizzled for DMA, padded otherwise.
    static constexpr bool KSW = DMA && DK % 64 == 0;
    static constexpr int LDK = KSW ? DK : DK + 8, LDV = DMA ? KT : KT + 8;
    static constexpr int KBUF = KT * LDK, VBUF = DV * LDV;
    // DMA: 64-lane instructions per tile (K: every slot of the padded rows;
    // V: the DH real rows), spread over the NW waves; the surplus
    // instructions of a wave load zeros into a spare 1 KB, so that every
    // wave issues the same count (its vmcnt waits stay uniform)
    static constexpr int NIK = KT * (LDK / 8) / 64, NIV = DH * (KT / 8) / 64;
    static constexpr int IK = (NIK + NW - 1) / NW, IV = (NIV + NW - 1) / NW;
    static constexpr bool SPARE = DMA && (IK * NW != NIK || IV * NW != NIV);
    static constexpr size_t LDS_BYTES = (size_t)NBUF * (KBUF + VBUF) * 2 + (SPARE ? 1024 : 0);
    static_assert(!DMA || (DH % 8 == 0 && (KT * (LDK / 8)) % 64 == 0), "DMA staging needs head_dim % 8 == 0");
};

// XOR swizzle of the DMA layout: slot of chunk c in row r (rows of LD halves)
template <int LD>
__device__ __forceinline__ int dma_slot(int r, int c) { return c ^ ((r >> (LD * 2 >= 256 ? 0 : 1)) & 7); }

// LDS offset (halves) of the 8-element chunk c of row r in a buffer of rows
// of LD halves, swizzled (SW) or plain
template <bool SW, int LD>
__device__ __forceinline__ int lds_chunk(int r, int c) {
    return SW ? r * LD + (dma_slot<LD>(r, c) << 3) : r * LD + (c << 3);
}

template <int DH, int NW, bool DMA, bool VARLEN = false>
__global__ __launch_bounds__(NW * 64) void k_flash(const uint16_t *__restrict__ Q, const uint16_t *__restrict__ K,
                                                    const uint16_t *__restrict__ Vt, uint16_t *__restrict__ O,
                                                    int hd, int heads, int n_seq, int L, int Lk, int lpad,
                                                    int n_qt, const int32_t *__restrict__ seq_off) {
    using C = FlashCfg<DH, DMA, NW>;
    constexpr int DK = C::DK, NKS = C::NKS, DV = C::DV, NDB = C::NDB, KT = C::KT, LDK = C::LDK, LDV = C::LDV;
    constexpr bool KSW = C::KSW;
    constexpr int NT = NW * 64, QT = 32 * NW;
    constexpr int KCH = KT * (DK / 8), VCH = DV * (KT / 8);
    constexpr int KPT = (KCH + NT - 1) / NT, VPT = (VCH + NT - 1) / NT;
    extern __shared__ __align__(16) uint16_t lds[];
    uint16_t *const Ks = lds;                       // [NBUF][KT][LDK]
    uint16_t *const Vs = lds + C::NBUF * C::KBUF;   // [NBUF][DV][LDV]

    const int total = n_qt * heads * n_seq;
    const int lid = xcd_remap(blockIdx.x, total);
    const int qt = lid % n_qt, hs = lid / n_qt, h = hs % heads, s = hs / heads;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, ln = lane & 31, lg = lane >> 5;
    long row0 = (long)s * L;
    if constexpr (VARLEN) {
        // sequences of varying length: this sequence's rows and key count;
        // query tiles past its end leave at once (the whole block)
        row0 = seq_off[s];
        Lk = seq_off[s + 1] - seq_off[s];
        if (qt * QT >= Lk) return;
    }
    const int q_base = qt * QT + wave * 32;
    const uint16_t *kbase = K + row0 * hd + h * DH;
    const uint16_t *vbase = Vt + ((long)h * n_seq + s) * DH * lpad;

    f16x8 qf[NKS];
    {
        const int q = q_base + ln;
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
            const int d0 = ks * 16 + lg * 8;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (q < Lk && d0 < DH) v = *reinterpret_cast<const uint4 *>(Q + (row0 + q) * hd + h * DH + d0);
            qf[ks] = __builtin_bit_cast(f16x8, v);
        }
    }

    // DMA: instruction j of this wave fills LDS chunks q = (wave*I + j)*64 + lane
    // of a buffer (row q / chunks-per-row, slot q % chunks-per-row); the lane
    // fetches the chunk that the swizzle puts in that slot.  Buffer loads
    // with a fixed per-lane offset and the tile's offset in a scalar: K rows
    // past the end read as zeros (their scores are masked), and no address
    // arithmetic is left per tile.
    // instruction j of wave w covers the 64 slots of index j*NW + w; a slot
    // past the tile's (a surplus instruction) or in a K row's padding
    // (head-dim chunks >= DH/8 and the row's spare chunk) gets an offset past
    // the end of the buffer by itself, which the hardware reads as zero
    constexpr int IK = DMA ? C::IK : 1, IV = DMA ? C::IV : 1;
    constexpr int KCPR = LDK / 8;   // 16-byte slots per K row in LDS
    constexpr int OOB = 0x40000000;
    const int wv = __builtin_amdgcn_readfirstlane(wave);
    i32x4 krs = {0, 0, 0, 0}, vrs = {0, 0, 0, 0};
    int kvo[IK], vvo[IV];
    if constexpr (DMA) {
        krs = buffer_rsrc(kbase, (int)((long)(Lk - 1) * hd * 2 + DH * 2));
        vrs = buffer_rsrc(vbase, DH * lpad * 2);
#pragma unroll
        for (int j = 0; j < IK; ++j) {
            const int q = (j * NW + wave) * 64 + lane;
            const int r = q / KCPR, slot = q % KCPR, c = KSW ? dma_slot<LDK>(r, slot) : slot;
            kvo[j] = (j * NW + wave < C::NIK && c < DH / 8) ? (r * hd + c * 8) * 2 : OOB;
        }
#pragma unroll
        for (int j = 0; j < IV; ++j) {
            const int q = (j * NW + wave) * 64 + lane;
            const int d = q / (KT / 8), c = dma_slot<LDV>(d, q % (KT / 8));
            vvo[j] = j * NW + wave < C::NIV ? (d * lpad + c * 8) * 2 : OOB;
        }
    }
    uint16_t *const spare = lds + C::NBUF * (C::KBUF + C::VBUF);
    auto issue = [&](int kt) {
        const int k0 = kt * KT, buf = kt & 3;
        uint16_t *kb = Ks + buf * C::KBUF;
        uint16_t *vb = Vs + buf * C::VBUF;
#pragma unroll
        for (int j = 0; j < IK; ++j) {
            const int ix = j * NW + wv;
            buffer_load_lds(krs, (lds_vp)(C::SPARE && ix >= C::NIK ? spare : kb + ix * 512), 16, kvo[j],
                            k0 * hd * 2, 0, 0);
        }
#pragma unroll
        for (int j = 0; j < IV; ++j) {
            const int ix = j * NW + wv;
            buffer_load_lds(vrs, (lds_vp)(C::SPARE && ix >= C::NIV ? spare : vb + ix * 512), 16, vvo[j], k0 * 2,
                            0, 0);
        }
    };

    // this thread's staging chunks (fixed across tiles)
    const uint16_t *kp[KPT];
    int kkey[KPT], klds[KPT];
    bool kok[KPT];
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
        const int c = threadIdx.x + i * NT;
        const int key = c / (DK / 8), d0 = (c % (DK / 8)) * 8;
        kok[i] = (KCH % NT == 0 || c < KCH) && (DK == DH || d0 < DH);
        kkey[i] = key;
        kp[i] = kbase + (long)key * hd + d0;
        klds[i] = key * LDK + d0;
    }
    const uint16_t *vp[VPT];
    int vpos[VPT], vlds[VPT];
    bool vok[VPT];
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
        const int c = threadIdx.x + i * NT;
        const int d = c >> 3, kc = c & 7;
        vok[i] = (VCH % NT == 0 || c < VCH) && (DV == DH || d < DH);
        vpos[i] = kc * 8;
        vp[i] = vbase + (long)d * lpad + kc * 8;
        vlds[i] = d * LDV + kc * 8;
    }
    uint4 kr[KPT], vr[VPT];
    const long kstep = (long)KT * hd;
    auto load = [&](int kt) {
        const int k0 = kt * KT;
        const bool tail = k0 + KT > Lk;
#pragma unroll
        for (int i = 0; i < KPT; ++i) {
            uint4 v = make_uint4(0, 0, 0, 0);
            if (kok[i] && (!tail || k0 + kkey[i] < Lk)) v = *reinterpret_cast<const uint4 *>(kp[i] + kt * kstep);
            kr[i] = v;
        }
#pragma unroll
        for (int i = 0; i < VPT; ++i) {
            uint4 v = make_uint4(0, 0, 0, 0);
            if (vok[i]) {
                v = *reinterpret_cast<const uint4 *>(vp[i] + k0);
                if (tail) {
                    // zero the stored positions whose key is past the end
                    uint16_t *e = reinterpret_cast<uint16_t *>(&v);
                    const int blk = vpos[i] & ~15, p0 = vpos[i] & 15;
#pragma unroll
                    for (int t = 0; t < 8; ++t)
                        if (k0 + blk + vt_key_of_pos(p0 + t) >= Lk) e[t] = 0;
                }
            }
            vr[i] = v;
        }
    };
    auto store = [&](int buf) {
        uint16_t *kb = Ks + buf * C::KBUF;
        uint16_t *vb = Vs + buf * C::VBUF;
#pragma unroll
        for (int i = 0; i < KPT; ++i)
            if (KCH % NT == 0 || threadIdx.x + i * NT < KCH) *reinterpret_cast<uint4 *>(kb + klds[i]) = kr[i];
#pragma unroll
        for (int i = 0; i < VPT; ++i)
            if (VCH % NT == 0 || threadIdx.x + i * NT < VCH) *reinterpret_cast<uint4 *>(vb + vlds[i]) = vr[i];
    };

    f16x8 kf[2][NKS];
    auto read_k = [&](int buf) {
        const uint16_t *kb = Ks + buf * C::KBUF;
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
            for (int kb2 = 0; kb2 < 2; ++kb2)
                kf[kb2][ks] = *reinterpret_cast<const f16x8 *>(kb + lds_chunk<KSW, LDK>(kb2 * 32 + ln, ks * 2 + lg));
    };

    // output accumulator o (MFMA) and the part saved at the last rebase osv;
    // the attention output is (osv + o) / l
    // wide heads (three or more row blocks of O) rescale o in place instead:
    // the saved sum would cost 16 registers per row block
    constexpr bool SAVE = NDB <= 2;
    f32x16 o[NDB], osv[SAVE ? NDB : 1];
#pragma unroll
    for (int db = 0; db < NDB; ++db) o[db] = f32x16{};
#pragma unroll
    for (int db = 0; db < (SAVE ? NDB : 1); ++db) osv[db] = f32x16{};
    float m = 0.f, l0 = 0.f, l1 = 0.f;
    // -m in every slot: the first S MFMA of a tile adds it (changes only on the slow path)
    f32x16 negm = f32x16{};

    const int n_kt = cdiv(Lk, KT);
    constexpr int IPT = IK + IV;   // DMA instructions per wave and tile
    if constexpr (DMA) {
        issue(0);
        if (n_kt > 1) issue(1);
        if (n_kt > 2) {
            issue(2);
            OC_WAIT_VMCNT(IPT);   // Q and tiles 0, 1 landed; tile 2 may be in flight
        } else {
            OC_WAIT_VMCNT(0);
        }
    } else {
        load(0);
        store(0);
        if (n_kt > 1) {
            load(1);
            store(1);
        }
        if (n_kt > 2) load(2);
        // the Q fragments and tile 2 must have landed before the loop: its
        // first MFMA then never waits on the loads a previous tile left in flight
        OC_WAIT_VMCNT(0);
    }
    if constexpr (DMA) barrier_lds(); else __syncthreads();
    // K fragments one tile ahead, except for the widest heads, which read
    // them at the top of each tile (the prefetch would cost a wave per SIMD)
    constexpr bool KPRE = NKS <= 6;
    if constexpr (KPRE) read_k(0);

    const f16x2 ones = {(_Float16)1.f, (_Float16)1.f};
    const _Float16 big = (_Float16)(float)(1 << (int)REBASE);
    int b0 = 0;
    for (int kt = 0; kt < n_kt; ++kt) {
        const int b1 = DMA ? (kt + 1) & 3 : (b0 == 2 ? 0 : b0 + 1), b2 = b1 == 2 ? 0 : b1 + 1;
        const int k0 = kt * KT;
        // DMA: tile kt+3 into the buffer that tile kt-1 left (free since the last barrier)
        if (DMA && kt + 3 < n_kt) issue(kt + 3);
        if constexpr (!KPRE) read_k(b0);
        // S^T - m
        f32x16 sc[2];
#pragma unroll
        for (int kb2 = 0; kb2 < 2; ++kb2) sc[kb2] = __builtin_amdgcn_mfma_f32_32x32x16_f16(kf[kb2][0], qf[0], negm, 0, 0, 0);
#pragma unroll
        for (int ks = 1; ks < NKS; ++ks)
#pragma unroll
            for (int kb2 = 0; kb2 < 2; ++kb2)
                sc[kb2] = __builtin_amdgcn_mfma_f32_32x32x16_f16(kf[kb2][ks], qf[ks], sc[kb2], 0, 0, 0);
        // V fragments of this tile (wide heads: read per key block just before use)
        constexpr int VK = SAVE ? 4 : 1;
        f16x8 vf[NDB][VK];
        const uint16_t *vbt = Vs + b0 * C::VBUF;
        if constexpr (SAVE) {
#pragma unroll
            for (int k4 = 0; k4 < 4; ++k4)
#pragma unroll
                for (int db = 0; db < NDB; ++db)
                    vf[db][k4] = *reinterpret_cast<const f16x8 *>(vbt + lds_chunk<DMA, LDV>(db * 32 + ln, k4 * 2 + lg));
        }
        // registers: tile kt+2 into the free buffer, then the global loads of tile kt+3
        if (!DMA && kt + 2 < n_kt) {
            store(b2);
            if (kt + 3 < n_kt) load(kt + 3);
        }
        if (k0 + KT > Lk) {
#pragma unroll
            for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
                for (int i = 0; i < 16; ++i)
                    if (k0 + kb2 * 32 + 8 * (i >> 2) + 4 * lg + (i & 3) >= Lk) sc[kb2][i] = -INFINITY;
        }
        f16x8 pf[4];
        auto exps = [&]() {
#pragma unroll
            for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
                for (int hf = 0; hf < 2; ++hf) {
                    f16x8 f;
#pragma unroll
                    for (int e = 0; e < 8; ++e) f[e] = (_Float16)__builtin_amdgcn_exp2f(sc[kb2][8 * hf + e]);
                    pf[kb2 * 2 + hf] = f;
                }
        };
        exps();
        // largest P of this lane (packed fp16; overflow gives +inf)
        f16x2 mx = __builtin_elementwise_maximum(pf[0].s01, pf[0].s23);
        mx = __builtin_elementwise_maximum(__builtin_elementwise_maximum(mx, pf[0].s45), pf[0].s67);
#pragma unroll
        for (int j = 1; j < 4; ++j) {
            mx = __builtin_elementwise_maximum(__builtin_elementwise_maximum(mx, pf[j].s01), pf[j].s23);
            mx = __builtin_elementwise_maximum(__builtin_elementwise_maximum(mx, pf[j].s45), pf[j].s67);
        }
        const bool over = mx[0] > big || mx[1] > big;
        if (kt == 0 || __builtin_amdgcn_ballot_w64(over) != 0) {
            // raise the reference maximum of the queries that need it by the
            // tile maximum t of both lane halves (any sign on the first tile)
            float t = -INFINITY;
#pragma unroll
            for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
                for (int i = 0; i < 16; ++i) t = fmaxf(t, sc[kb2][i]);
            t = fmaxf(t, __shfl_xor(t, 32, 64));
            const float tt = (kt == 0 || t > REBASE) ? t : 0.f;
            float alpha = 1.f;
            if (kt > 0) alpha = __builtin_amdgcn_exp2f(-tt);
            l0 *= alpha;
            l1 *= alpha;
            // fold the MFMA accumulator into the rescaled saved sum and
            // restart it at zero: O itself is never scaled element-wise,
            // which keeps it in the same registers on both paths (wide
            // heads scale O in place)
            if constexpr (SAVE) {
#pragma unroll
                for (int db = 0; db < NDB; ++db) {
#pragma unroll
                    for (int i = 0; i < 16; ++i) osv[db][i] = (osv[db][i] + o[db][i]) * alpha;
                    o[db] = f32x16{};
                }
            } else {
#pragma unroll
                for (int db = 0; db < NDB; ++db)
#pragma unroll
                    for (int i = 0; i < 16; ++i) o[db][i] *= alpha;
            }
#pragma unroll
            for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
                for (int i = 0; i < 16; ++i) sc[kb2][i] -= tt;
            m += tt;
#pragma unroll
            for (int i = 0; i < 16; ++i) negm[i] = -m;
            exps();
        }
        // running sum of the fp16 P, fp32 accumulation
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            l0 = __builtin_amdgcn_fdot2(pf[j].s01, ones, l0, false);
            l1 = __builtin_amdgcn_fdot2(pf[j].s23, ones, l1, false);
            l0 = __builtin_amdgcn_fdot2(pf[j].s45, ones, l0, false);
            l1 = __builtin_amdgcn_fdot2(pf[j].s67, ones, l1, false);
        }
        // K fragments of the next tile (its buffer was filled before the last barrier)
        if (KPRE && kt + 1 < n_kt) read_k(b1);
#pragma unroll
        for (int k4 = 0; k4 < 4; ++k4) {
            if constexpr (!SAVE) {
#pragma unroll
                for (int db = 0; db < NDB; ++db)
                    vf[db][0] = *reinterpret_cast<const f16x8 *>(vbt + lds_chunk<DMA, LDV>(db * 32 + ln, k4 * 2 + lg));
            }
#pragma unroll
            for (int db = 0; db < NDB; ++db)
                o[db] = __builtin_amdgcn_mfma_f32_32x32x16_f16(vf[db][SAVE ? k4 : 0], pf[k4], o[db], 0, 0, 0);
        }
        // DMA: this wave's part of tile kt+2 must have landed before the
        // barrier that publishes it (only tile kt+3 may still be in flight)
        if constexpr (DMA) {
            if (kt + 2 < n_kt) {
                if (kt + 3 < n_kt) {
                    OC_WAIT_VMCNT(IPT);
                } else {
                    OC_WAIT_VMCNT(0);
                }
            }
            barrier_lds();
        } else {
            __syncthreads();
        }
        b0 = b1;
    }
    // normalise and store: lane holds query ln, d = db*32 + 8*g4 + 4*lg + e
    float lt = l0 + l1;
    lt += __shfl_xor(lt, 32, 64);
    const float inv = 1.f / lt;
    const int q = q_base + ln;
    if (q >= Lk) return;
    uint16_t *orow = O + (row0 + q) * hd + h * DH;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
            const int d = db * 32 + 8 * g4 + 4 * lg;
            if (d >= DH) continue;
            u16x4 v;
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = f2h_bits(((SAVE ? osv[SAVE ? db : 0][4 * g4 + e] : 0.f) + o[db][4 * g4 + e]) * inv);
            *reinterpret_cast<u16x4 *>(orow + d) = v;
        }
}

// Short sequences (at most 64 keys, e.g. temporal attention over frames):
// one wave per (sequence, head), no LDS and no barriers.  V comes by rows
// here (the projection writes it like Q and K).  The wave holds K and the
// Vt fragments of the whole sequence in registers (KB blocks of 32 keys) and, per
// block of 32 queries, computes S^T = K Q^T, the exact row maximum, P =
// exp2(s - max) in fp16, the running sum of that fp16 P, and O^T = Vt P^T on
// the same MFMA layouts as the long-sequence kernel.
template <int DH, int KB>
__global__ __launch_bounds__(256) void k_attn_short(const uint16_t *__restrict__ Q, const uint16_t *__restrict__ K,
                                                     const uint16_t *__restrict__ V, uint16_t *__restrict__ O, int hd,
                                                     int heads, int n_seq, int L, int Lk) {
    constexpr int DK = (DH + 15) / 16 * 16, NKS = DK / 16;
    constexpr int DV = (DH + 31) / 32 * 32, NDB = DV / 32;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, ln = lane & 31, lg = lane >> 5;
    const long unit = (long)blockIdx.x * 4 + wave;
    if (unit >= (long)n_seq * heads) return;   // whole waves only; the kernel has no block barrier
    const int h = (int)(unit % heads), s = (int)(unit / heads);
    const long row0 = (long)s * L;
    auto ld = [](const uint16_t *p, bool ok) {
        uint4 v = make_uint4(0, 0, 0, 0);
        if (ok) v = *reinterpret_cast<const uint4 *>(p);
        return __builtin_bit_cast(f16x8, v);
    };
    f16x8 kf[KB][NKS], vf[NDB][2 * KB];
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
        const int key = kb * 32 + ln;
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
            const int d0 = ks * 16 + lg * 8;
            kf[kb][ks] = ld(K + (row0 + key) * hd + h * DH + d0, key < Lk && d0 < DH);
        }
    }
    // V is stored by rows here: the A operand of O^T = Vt P^T (lane: d, 8
    // keys) is gathered from 8 rows, in the key order of the score slots
    // (vt_key_of_pos); keys past the end are zero
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int k4 = 0; k4 < 2 * KB; ++k4) {
            const int d = db * 32 + ln;
            f16x8 v;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int key = k4 * 16 + vt_key_of_pos(lg * 8 + e);
                uint16_t b = 0;
                if (key < Lk && d < DH) b = V[(row0 + key) * hd + h * DH + d];
                v[e] = __builtin_bit_cast(_Float16, b);
            }
            vf[db][k4] = v;
        }
    const f16x2 ones = {(_Float16)1.f, (_Float16)1.f};
    const int n_qb = (Lk + 31) / 32;
    for (int qb = 0; qb < n_qb; ++qb) {
        const int q = qb * 32 + ln;
        f16x8 qf[NKS];
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
            const int d0 = ks * 16 + lg * 8;
            qf[ks] = ld(Q + (row0 + q) * hd + h * DH + d0, q < Lk && d0 < DH);
        }
        f32x16 sc[KB];
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
            sc[kb] = f32x16{};
#pragma unroll
            for (int ks = 0; ks < NKS; ++ks)
                sc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(kf[kb][ks], qf[ks], sc[kb], 0, 0, 0);
        }
        float m = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                if (kb * 32 + 8 * (i >> 2) + 4 * lg + (i & 3) >= Lk) sc[kb][i] = -INFINITY;
                m = fmaxf(m, sc[kb][i]);
            }
        m = fmaxf(m, __shfl_xor(m, 32, 64));
        f16x8 pf[2 * KB];
        float l0 = 0.f, l1 = 0.f;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
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
        f32x16 o[NDB];
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
            o[db] = f32x16{};
#pragma unroll
            for (int k4 = 0; k4 < 2 * KB; ++k4)
                o[db] = __builtin_amdgcn_mfma_f32_32x32x16_f16(vf[db][k4], pf[k4], o[db], 0, 0, 0);
        }
        if (q >= Lk) continue;
        const float inv = 1.f / lt;
        uint16_t *orow = O + (row0 + q) * hd + h * DH;
#pragma unroll
        for (int db = 0; db < NDB; ++db)
#pragma unroll
            for (int g4 = 0; g4 < 4; ++g4) {
                const int d = db * 32 + 8 * g4 + 4 * lg;
                if (d >= DH) continue;
                u16x4 v;
#pragma unroll
                for (int e = 0; e < 4; ++e) v[e] = f2h_bits(o[db][4 * g4 + e] * inv);
                *reinterpret_cast<u16x4 *>(orow + d) = v;
            }
    }
}

template <int DH, int KB>
static hipError_t go_short(const Plan &p, const AttnArgs &a, int Lk, hipStream_t st) {
    const long waves = (long)a.n_seq * p.heads;
    launch_k(k_attn_short<DH, KB>, (unsigned)((waves + 3) / 4), 256, 0, st, (const uint16_t *)a.q,
             (const uint16_t *)a.k, (const uint16_t *)a.vt, (uint16_t *)a.o, p.hd, p.heads, a.n_seq, a.L, Lk);
    return hipGetLastError();
}

template <int DH, int NW, bool DMA, bool VARLEN = false>
static hipError_t go(const Plan &p, const AttnArgs &a, int Lk, hipStream_t st) {
    const int n_qt = cdiv(Lk, 32 * NW);
    const int total = n_qt * p.heads * a.n_seq;
    const size_t lds = FlashCfg<DH, DMA, NW>::LDS_BYTES;
    const hipError_t e = raise_lds_limit((const void *)k_flash<DH, NW, DMA, VARLEN>, lds);
    if (e != hipSuccess) return e;
    launch_k(k_flash<DH, NW, DMA, VARLEN>, total, NW * 64, lds, st, (const uint16_t *)a.q, (const uint16_t *)a.k,
                                                      (const uint16_t *)a.vt, (uint16_t *)a.o, p.hd, p.heads,
                                                      a.n_seq, a.L, Lk, a.lpad, n_qt, a.seq_off);
    return hipGetLastError();
}

// By sequence length: up to 64 keys the register-only short kernel, else
// four waves (32 queries each) per block (eight when the grid is small),
// DMA-staged when the head dim allows it.
template <int DH>
static hipError_t go_dh(const Plan &p, const AttnArgs &a, int Lk, hipStream_t st) {
    // sequences of varying length: the register-staged kernel, which masks
    // every sequence's end itself (Lk is the longest)
    if (a.seq_off != nullptr) return go<DH, 4, false, true>(p, a, Lk, st);
    if (attn_short(Lk)) return Lk <= 32 ? go_short<DH, 1>(p, a, Lk, st) : go_short<DH, 2>(p, a, Lk, st);
    // a grid of four-wave blocks that would not fill two per CU: eight-wave
    // blocks (256 queries share each K/V tile)
    const bool eight = (long)cdiv(Lk, 128) * p.heads * a.n_seq <= 2L * N_CUS;
    if (flash_uses_dma(DH, Lk, p.hd)) {
        if (eight) return go<DH, 8, true>(p, a, Lk, st);
        // padded head dims: the four-buffer ring with padded K rows would
        // leave one four-wave block per CU
        if constexpr (DH % 64 == 0) return go<DH, 4, true>(p, a, Lk, st);
    }
    if constexpr (DH <= 96) {
        if (eight) return go<DH, 8, false>(p, a, Lk, st);
    }
    return go<DH, 4, false>(p, a, Lk, st);
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
