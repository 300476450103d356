// LDS-DMA MFMA tile engine for gfx950: the same block tile as MfmaTile
// (C[b][a] = sum_k A[a][k] * B[b][k], 256 threads = 4 wave64s arranged
// WA x WB, 32x32 accumulators of v_mfma_f32_32x32x16_{bf16,f16}), but the
// operands travel global -> LDS with global_load_lds (16 bytes per lane, no
// staging registers).
//
// K is walked in steps of 64 through a ring of NST LDS stages.  With NST = 2
// (double buffer, small enough for two blocks per CU) step kt+1 is loaded
// while step kt's MFMAs run.  With NST >= 3, iteration kt
// issues the loads of step kt+NST-1 into the stage that step kt-1 left, waits
// for this wave's loads of step kt+1, passes one barrier (which publishes
// step kt+1 from every wave), reads step kt+1's MFMA fragments into the
// spare register set and then runs step kt's MFMAs from the fragments read
// one iteration earlier: LDS latency hides behind the MFMAs and global
// latency behind NST-1 steps.  An LDS row is the 128 bytes of one operand
// row's step, unpadded; its 16-byte chunk c sits in slot c ^ ((row >> 1) & 7):
// two rows fill the 64 LDS banks, so the fragment reads of 16 consecutive
// rows hit distinct banks.  DMA
// instruction i of a wave fills the 64 slots (wave + 4i)*64 .. +63 of the
// operand's stage, that is rows chunk_row(i) of MfmaTile: callers pass the
// same per-thread row bases.  Rows without data (nullptr) read the fallback
// row instead; their accumulators are garbage and must be discarded.
// Requirements: K % 64 == 0, 16-byte aligned row bases; with segments
// (seg_len > 0) seg_len % 64 == 0.
#pragma once
#include "oc_mfma_tile.h"
#include <type_traits>

namespace oc {

template <int BA, int BB, int WA, int WB, bool F16 = false, int NST = 3>
struct DmaTile {
    static constexpr int BK = 64;
    static constexpr int WTA = BA / WA, WTB = BB / WB;
    static constexpr int TA = WTA / 32, TB = WTB / 32;
    static constexpr int CA = BA / 32, CB = BB / 32;   // DMA instructions per wave and step
    static constexpr int IPT = CA + CB;
    static constexpr int STAGE = (BA + BB) * BK;       // halves per stage
    static constexpr size_t LDS_BYTES = (size_t)NST * STAGE * 2;
    static_assert(WA * WB == 4, "4 waves");
    static_assert(TA >= 1 && TB >= 1 && WTA % 32 == 0 && WTB % 32 == 0, "wave tile must be a multiple of 32");
    static_assert(BA % 32 == 0 && BB % 32 == 0, "tile rows per DMA instruction");
    static_assert(NST >= 2 && NST <= 4, "ring of 2 to 4 stages");
    typedef typename std::conditional<F16, f16x8, bf16x8>::type frag;

    f32x16 acc[TA][TB];

    __device__ __forceinline__ static int slot(int r, int c) { return r * BK + ((c ^ ((r >> 1) & 7)) << 3); }

    // MFMA fragments of one step: [ks][i] for A, [ks][j] for B
    struct Frags {
        frag a[4][TA], b[4][TB];
    };

    __device__ __forceinline__ static void read_frags(const uint16_t *st, Frags &f) {
        const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
        const int wa = wave / WB, wb = wave % WB;
        const int lr = lane & 31, lh = lane >> 5;
        const uint16_t *As = st, *Bs = st + BA * BK;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            const int c = ks * 2 + lh;
#pragma unroll
            for (int i = 0; i < TA; ++i) f.a[ks][i] = *reinterpret_cast<const frag *>(As + slot(wa * WTA + i * 32 + lr, c));
#pragma unroll
            for (int j = 0; j < TB; ++j) f.b[ks][j] = *reinterpret_cast<const frag *>(Bs + slot(wb * WTB + j * 32 + lr, c));
        }
    }

    __device__ __forceinline__ void mfmas(const Frags &f) {
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
#pragma unroll
            for (int i = 0; i < TA; ++i)
#pragma unroll
                for (int j = 0; j < TB; ++j) {
                    if constexpr (F16)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(f.a[ks][i], f.b[ks][j], acc[i][j], 0, 0, 0);
                    else
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[ks][i], f.b[ks][j], acc[i][j], 0, 0, 0);
                }
    }

    // Full K loop.  rowsA[i] / rowsB[i]: this thread's row bases for
    // chunk_row(i) (nullptr: use the fallback row).
    __device__ __forceinline__ void run(uint16_t *lds, const uint16_t *const *rowsA, const uint16_t *const *rowsB,
                                        const uint16_t *fallbackA, const uint16_t *fallbackB, int K, int seg_len,
                                        long sub_stride) {
        const int t = threadIdx.x, wave = t >> 6;
#pragma unroll
        for (int i = 0; i < TA; ++i)
#pragma unroll
            for (int j = 0; j < TB; ++j) acc[i][j] = f32x16{};
        // this lane's source chunk of each instruction: slot t&7 of its row
        const uint16_t *pa[CA], *pb[CB];
#pragma unroll
        for (int i = 0; i < CA; ++i) {
            const int r = chunk_row(i);
            pa[i] = (rowsA[i] ? rowsA[i] : fallbackA) + (((t & 7) ^ ((r >> 1) & 7)) << 3);
        }
#pragma unroll
        for (int i = 0; i < CB; ++i) {
            const int r = chunk_row(i);
            pb[i] = (rowsB[i] ? rowsB[i] : fallbackB) + (((t & 7) ^ ((r >> 1) & 7)) << 3);
        }
        const int nk = K / BK;
        constexpr int D = NST - 1;   // issue distance in steps
        auto issue = [&](int kt) {
            const int k0 = kt * BK;
            long off = k0;
            if (seg_len > 0) {
                const int s = k0 / seg_len;
                off = (long)s * sub_stride + (k0 - s * seg_len);
            }
            uint16_t *st = lds + (kt % NST) * STAGE;
#pragma unroll
            for (int i = 0; i < CA; ++i)
                __builtin_amdgcn_global_load_lds((glb_vp)(pa[i] + off), (lds_vp)(st + (wave + 4 * i) * 512), 16, 0, 0);
#pragma unroll
            for (int i = 0; i < CB; ++i)
                __builtin_amdgcn_global_load_lds((glb_vp)(pb[i] + off), (lds_vp)(st + BA * BK + (wave + 4 * i) * 512),
                                                 16, 0, 0);
        };
        // wait until this wave's loads of step s landed, knowing that the
        // loads of steps s+1 .. last_issued may still be in flight
        auto wait_for = [&](int s, int last_issued) {
            const int later = last_issued - s;
            if (NST == 4 && later >= 2) {
                OC_WAIT_VMCNT(2 * IPT);
            } else if (later >= 1) {
                OC_WAIT_VMCNT(IPT);
            } else {
                OC_WAIT_VMCNT(0);
            }
        };
        if constexpr (NST == 2) {
            // double buffer: the MFMAs of step kt overlap the DMA of step
            // kt+1; the fragments of kt+1 are read after the barrier that
            // publishes it (two blocks per CU hide that latency)
            issue(0);
            OC_WAIT_VMCNT(0);
            barrier_lds();
            Frags f;
            read_frags(lds, f);
            for (int kt = 0; kt < nk; ++kt) {
                if (kt + 1 < nk) issue(kt + 1);   // its stage was last read before the previous barrier
                mfmas(f);
                if (kt + 1 < nk) {
                    OC_WAIT_VMCNT(0);
                    barrier_lds();
                    read_frags(lds + ((kt + 1) & 1) * STAGE, f);
                }
            }
            OC_WAIT_VMCNT(0);
            __syncthreads();
            return;
        }
#pragma unroll
        for (int s = 0; s < D; ++s)
            if (s < nk) issue(s);
        wait_for(0, (nk < D ? nk : D) - 1);
        barrier_lds();
        Frags f0, f1;
        read_frags(lds, f0);
        for (int kt = 0; kt < nk; kt += 2) {
            // even step kt: fragments in f0
            if (kt + D < nk) issue(kt + D);
            if (kt + 1 < nk) {
                wait_for(kt + 1, kt + D < nk ? kt + D : nk - 1);
                barrier_lds();
                read_frags(lds + ((kt + 1) % NST) * STAGE, f1);
            }
            mfmas(f0);
            if (kt + 1 >= nk) break;
            // odd step kt+1: fragments in f1
            if (kt + 1 + D < nk) issue(kt + 1 + D);
            if (kt + 2 < nk) {
                wait_for(kt + 2, kt + 1 + D < nk ? kt + 1 + D : nk - 1);
                barrier_lds();
                read_frags(lds + ((kt + 2) % NST) * STAGE, f0);
            }
            mfmas(f1);
        }
        OC_WAIT_VMCNT(0);
        __syncthreads();   // the epilogue may reuse the LDS
    }

    // Several output tiles along A back to back in one continuous pipeline
    // (no refill between tiles): tile u reads A rows rows_a(u, i) (nullptr:
    // the fallback row) and the same B rows; steps are s = u*nk + kt.  After
    // the last K step of tile u, epi(u) consumes acc, which is then cleared.
    // epi must not touch this ring's LDS.
    template <typename RowsA, typename Epi>
    __device__ __forceinline__ void run_tiles(uint16_t *lds, RowsA rows_a, const uint16_t *const *rowsB,
                                              const uint16_t *fallbackA, const uint16_t *fallbackB, int K,
                                              int seg_len, long sub_stride, int n_tiles, Epi epi) {
        const int t = threadIdx.x, wave = t >> 6;
        auto clear = [&]() {
#pragma unroll
            for (int i = 0; i < TA; ++i)
#pragma unroll
                for (int j = 0; j < TB; ++j) acc[i][j] = f32x16{};
        };
        clear();
        int ca[CA];
        const uint16_t *pb[CB];
#pragma unroll
        for (int i = 0; i < CA; ++i) {
            const int r = chunk_row(i);
            ca[i] = ((t & 7) ^ ((r >> 1) & 7)) << 3;
        }
#pragma unroll
        for (int i = 0; i < CB; ++i) {
            const int r = chunk_row(i);
            pb[i] = (rowsB[i] ? rowsB[i] : fallbackB) + (((t & 7) ^ ((r >> 1) & 7)) << 3);
        }
        const int nk = K / BK, ns = nk * n_tiles;
        // A rows of the tile being issued (issue() is called with rising s)
        int cur_u = -1;
        const uint16_t *pa[CA];
        auto issue = [&](int s) {
            const int u = s / nk, kt = s - u * nk;
            if (u != cur_u) {
                cur_u = u;
#pragma unroll
                for (int i = 0; i < CA; ++i) {
                    const uint16_t *r = rows_a(u, i);
                    pa[i] = (r ? r : fallbackA) + ca[i];
                }
            }
            const int k0 = kt * BK;
            long off = k0;
            if (seg_len > 0) {
                const int sg = k0 / seg_len;
                off = (long)sg * sub_stride + (k0 - sg * seg_len);
            }
            uint16_t *st = lds + (s % NST) * STAGE;
#pragma unroll
            for (int i = 0; i < CA; ++i)
                __builtin_amdgcn_global_load_lds((glb_vp)(pa[i] + off), (lds_vp)(st + (wave + 4 * i) * 512), 16, 0, 0);
#pragma unroll
            for (int i = 0; i < CB; ++i)
                __builtin_amdgcn_global_load_lds((glb_vp)(pb[i] + off), (lds_vp)(st + BA * BK + (wave + 4 * i) * 512),
                                                 16, 0, 0);
        };
        auto wait_for = [&](int s, int last_issued) {
            const int later = last_issued - s;
            if (NST == 4 && later >= 2) {
                OC_WAIT_VMCNT(2 * IPT);
            } else if (later >= 1) {
                OC_WAIT_VMCNT(IPT);
            } else {
                OC_WAIT_VMCNT(0);
            }
        };
        constexpr int D = NST - 1;
        auto finish = [&](int s) {
            if (s % nk == nk - 1) {
                epi(s / nk);
                clear();
            }
        };
        if constexpr (NST == 2) {
            // double buffer: the MFMAs of step s overlap the DMA of step s+1
            issue(0);
            OC_WAIT_VMCNT(0);
            barrier_lds();
            Frags f;
            read_frags(lds, f);
            for (int s = 0; s < ns; ++s) {
                if (s + 1 < ns) issue(s + 1);   // its stage was last read before the previous barrier
                mfmas(f);
                finish(s);
                if (s + 1 < ns) {
                    OC_WAIT_VMCNT(0);
                    barrier_lds();
                    read_frags(lds + ((s + 1) & 1) * STAGE, f);
                }
            }
            OC_WAIT_VMCNT(0);
            __syncthreads();
            return;
        }
#pragma unroll
        for (int s = 0; s < D; ++s)
            if (s < ns) issue(s);
        wait_for(0, (ns < D ? ns : D) - 1);
        barrier_lds();
        Frags f0, f1;
        read_frags(lds, f0);
        for (int s = 0; s < ns; s += 2) {
            if (s + D < ns) issue(s + D);
            if (s + 1 < ns) {
                wait_for(s + 1, s + D < ns ? s + D : ns - 1);
                barrier_lds();
                read_frags(lds + ((s + 1) % NST) * STAGE, f1);
            }
            mfmas(f0);
            finish(s);
            if (s + 1 >= ns) break;
            if (s + 1 + D < ns) issue(s + 1 + D);
            if (s + 2 < ns) {
                wait_for(s + 2, s + 1 + D < ns ? s + 1 + D : ns - 1);
                barrier_lds();
                read_frags(lds + ((s + 2) % NST) * STAGE, f0);
            }
            mfmas(f1);
            finish(s + 1);
        }
        OC_WAIT_VMCNT(0);
        __syncthreads();
    }

    __device__ __forceinline__ static int a_of(int i, int g) {
        const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
        return (wave / WB) * WTA + i * 32 + 8 * g + 4 * (lane >> 5);
    }
    __device__ __forceinline__ static int b_of(int j) {
        const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
        return (wave % WB) * WTB + j * 32 + (lane & 31);
    }
    // Row of the tile that DMA instruction i of this thread loads (as MfmaTile).
    __device__ __forceinline__ static int chunk_row(int i) { return (threadIdx.x + 256 * i) >> 3; }
};

}  // namespace oc
