// LDS-staged MFMA tile engine for gfx950 (bf16 or fp16 operands, fp32
// accumulation in VGPRs).
//
// Computes a BA x BB block of  C[b][a] = sum_k A[a][k] * B[b][k]  where both
// operands are K-contiguous rows (the "NT" form: token rows times
// linear-layer weight rows, or candidate rows times representative rows).
// 256 threads = 4 wave64s arranged WA x WB; each wave owns a
// (BA/WA) x (BB/WB) sub-block of 32x32 accumulators of
// v_mfma_f32_32x32x16_{bf16,f16}.
//
// MFMA operand layout (32x32x16): lane l feeds row/column (l % 32) and the 8
// consecutive k of chunk (l / 32).  The result lane l holds column
// b = l % 32 and, for accumulator slot 4g+e, row a = 8g + 4(l/32) + e: one b
// and groups of four consecutive a per lane, which the epilogues use for
// 8-byte stores.
//
// K is walked in steps of BK = 64 through two LDS buffers: the next step is
// loaded from global memory into registers while the current one feeds the
// MFMAs, then written to the other buffer; one barrier per step.  LDS rows
// are padded by 16 bytes so the 16-byte fragment reads of 32 consecutive
// rows spread over the banks.  With F16 set, operand A may be stored as bf16
// in memory and converted to fp16 as it is staged (CVT_A); bf16 values
// convert exactly inside the fp16 normal range and saturate at +-65504.
#pragma once
#include "oc_device.h"

namespace oc {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ uint16_t f2h_bits(float f) {
    f = fminf(fmaxf(f, -65504.f), 65504.f);
    const _Float16 h = (_Float16)f;
    return *reinterpret_cast<const uint16_t *>(&h);
}

__device__ __forceinline__ uint4 bf16x8_to_f16x8(uint4 v) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    uint32_t o[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t lo = f2h_bits(__uint_as_float(w[i] << 16));
        const uint32_t hi = f2h_bits(__uint_as_float(w[i] & 0xFFFF0000u));
        o[i] = lo | (hi << 16);
    }
    return make_uint4(o[0], o[1], o[2], o[3]);
}

template <int BA, int BB, int WA, int WB, bool F16 = false, bool CVT_A = false>
struct MfmaTile {
    static constexpr int BK = 64;
    static constexpr int LDK = BK + 8;                 // padded LDS row (elements)
    static constexpr int WTA = BA / WA, WTB = BB / WB; // wave sub-block
    static constexpr int TA = WTA / 32, TB = WTB / 32;
    static constexpr int CA = BA * (BK / 8) / 256;     // A chunks per thread
    static constexpr int CB = BB * (BK / 8) / 256;
    static_assert(WA * WB == 4, "4 waves");
    static_assert(TA >= 1 && TB >= 1 && WTA % 32 == 0 && WTB % 32 == 0, "wave tile must be a multiple of 32");
    static_assert(CA >= 1 && CB >= 1, "tile too small for 256 threads");
    static_assert(!CVT_A || F16, "conversion only towards fp16");
    static constexpr int BUF = (BA + BB) * LDK;        // elements per LDS buffer
    static constexpr size_t LDS_BYTES = (size_t)2 * BUF * 2;

    f32x16 acc[TA][TB];

    // Load one BK step of this thread's chunks into registers.  rows[i] is
    // the row base of chunk slot i (nullptr: zero row); rows are descriptors
    // of segments of seg_len elements, segment s at base + s * sub_stride
    // (seg_len == 0: one plain row).
    template <bool CVT, int NC>
    __device__ __forceinline__ static void load_step(const uint16_t *const *rows, int k0, int K, int seg_len,
                                                      long sub_stride, uint4 *regs) {
        const int kc = (threadIdx.x & 7) * 8;
#pragma unroll
        for (int i = 0; i < NC; ++i) {
            const int k = k0 + kc;
            const uint16_t *p = rows[i];
            uint4 v = make_uint4(0, 0, 0, 0);
            if (p != nullptr && k < K) {
                if (seg_len > 0) {
                    const int s = k / seg_len;
                    p += (long)s * sub_stride + (k - s * seg_len);
                } else {
                    p += k;
                }
                v = *reinterpret_cast<const uint4 *>(p);
                if (CVT) v = bf16x8_to_f16x8(v);
            }
            regs[i] = v;
        }
    }

    template <int NC>
    __device__ __forceinline__ static void store_step(uint16_t *lds, const uint4 *regs) {
        const int t = threadIdx.x;
#pragma unroll
        for (int i = 0; i < NC; ++i) {
            const int c = t + 256 * i;
            *reinterpret_cast<uint4 *>(lds + (c >> 3) * LDK + (c & 7) * 8) = regs[i];
        }
    }

    // One BK step of MFMAs from LDS.
    __device__ __forceinline__ void compute(const uint16_t *As, const uint16_t *Bs) {
        const int lane = threadIdx.x & 63;
        const int wave = threadIdx.x >> 6;
        const int wa = wave / WB, wb = wave % WB;
        const int lr = lane & 31, lk = (lane >> 5) * 8;
#pragma unroll
        for (int ks = 0; ks < BK; ks += 16) {
            if constexpr (F16) {
                f16x8 fa[TA], fb[TB];
#pragma unroll
                for (int i = 0; i < TA; ++i)
                    fa[i] = *reinterpret_cast<const f16x8 *>(As + (wa * WTA + i * 32 + lr) * LDK + ks + lk);
#pragma unroll
                for (int j = 0; j < TB; ++j)
                    fb[j] = *reinterpret_cast<const f16x8 *>(Bs + (wb * WTB + j * 32 + lr) * LDK + ks + lk);
#pragma unroll
                for (int i = 0; i < TA; ++i)
#pragma unroll
                    for (int j = 0; j < TB; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(fa[i], fb[j], acc[i][j], 0, 0, 0);
            } else {
                bf16x8 fa[TA], fb[TB];
#pragma unroll
                for (int i = 0; i < TA; ++i)
                    fa[i] = *reinterpret_cast<const bf16x8 *>(As + (wa * WTA + i * 32 + lr) * LDK + ks + lk);
#pragma unroll
                for (int j = 0; j < TB; ++j)
                    fb[j] = *reinterpret_cast<const bf16x8 *>(Bs + (wb * WTB + j * 32 + lr) * LDK + ks + lk);
#pragma unroll
                for (int i = 0; i < TA; ++i)
#pragma unroll
                    for (int j = 0; j < TB; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
            }
        }
    }

    // Full K loop.  rowsA[i] / rowsB[i] are this thread's chunk-slot row bases.
    // Global loads run two steps ahead of the LDS buffer they fill (two
    // register sets), so each load has two compute phases to arrive.
    __device__ __forceinline__ void run(uint16_t *lds, const uint16_t *const *rowsA, const uint16_t *const *rowsB,
                                        int K, int seg_len, long sub_stride) {
        uint4 ra0[CA], rb0[CB], ra1[CA], rb1[CB];
#pragma unroll
        for (int i = 0; i < TA; ++i)
#pragma unroll
            for (int j = 0; j < TB; ++j) acc[i][j] = f32x16{};
        const int nk = cdiv(K, BK);
        uint16_t *L0 = lds, *L1 = lds + BUF;
        load_step<CVT_A, CA>(rowsA, 0, K, seg_len, sub_stride, ra0);
        load_step<false, CB>(rowsB, 0, K, seg_len, sub_stride, rb0);
        store_step<CA>(L0, ra0);
        store_step<CB>(L0 + BA * LDK, rb0);
        if (nk > 1) {
            load_step<CVT_A, CA>(rowsA, BK, K, seg_len, sub_stride, ra1);
            load_step<false, CB>(rowsB, BK, K, seg_len, sub_stride, rb1);
        }
        if (nk > 2) {
            load_step<CVT_A, CA>(rowsA, 2 * BK, K, seg_len, sub_stride, ra0);
            load_step<false, CB>(rowsB, 2 * BK, K, seg_len, sub_stride, rb0);
        }
        __syncthreads();
        for (int kt = 0; kt < nk; kt += 2) {
            // even step kt: buffer L0; step kt+1 (regs 1) -> L1; regs 1 <- step kt+3
            compute(L0, L0 + BA * LDK);
            if (kt + 1 < nk) {
                store_step<CA>(L1, ra1);
                store_step<CB>(L1 + BA * LDK, rb1);
            }
            if (kt + 3 < nk) {
                load_step<CVT_A, CA>(rowsA, (kt + 3) * BK, K, seg_len, sub_stride, ra1);
                load_step<false, CB>(rowsB, (kt + 3) * BK, K, seg_len, sub_stride, rb1);
            }
            __syncthreads();
            if (kt + 1 >= nk) break;
            // odd step kt+1: buffer L1; step kt+2 (regs 0) -> L0; regs 0 <- step kt+4
            compute(L1, L1 + BA * LDK);
            if (kt + 2 < nk) {
                store_step<CA>(L0, ra0);
                store_step<CB>(L0 + BA * LDK, rb0);
            }
            if (kt + 4 < nk) {
                load_step<CVT_A, CA>(rowsA, (kt + 4) * BK, K, seg_len, sub_stride, ra0);
                load_step<false, CB>(rowsB, (kt + 4) * BK, K, seg_len, sub_stride, rb0);
            }
            __syncthreads();
        }
    }

    // Coordinates of accumulator (i, j) slot 4g+e for this lane, relative to
    // the block: a_of(i, g) + e and b_of(j).
    __device__ __forceinline__ static int a_of(int i, int g) {
        const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
        return (wave / WB) * WTA + i * 32 + 8 * g + 4 * (lane >> 5);
    }
    __device__ __forceinline__ static int b_of(int j) {
        const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
        return (wave % WB) * WTB + j * 32 + (lane & 31);
    }
    // Row of the tile that chunk slot i of this thread loads.
    __device__ __forceinline__ static int chunk_row(int i) { return (threadIdx.x + 256 * i) >> 3; }
};

}  // namespace oc
