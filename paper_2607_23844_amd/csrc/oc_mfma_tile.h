// LDS-staged MFMA tile engine for gfx950 (bf16 or fp16 operands, fp32
// accumulation).
//
// Computes a BA x BB block of  C[b][a] = sum_k A[a][k] * B[b][k]  where both
// operands are K-contiguous rows (the "NT" form: token rows times
// linear-layer weight rows, or candidate rows times representative rows).
// 256 threads = 4 wave64s arranged WA x WB; each wave owns a
// (BA/WA) x (BB/WB) sub-block built from 16x16 accumulators of
// v_mfma_f32_16x16x32_{bf16,f16}.
//
// MFMA operand layout (16x16x32): lane l feeds row/column (l % 16) and the
// 8 consecutive k of chunk (l / 16).  The result lane l holds column
// b = l % 16 and rows a = 4*(l/16) .. 4*(l/16)+3: one b and four consecutive
// a per lane, which the epilogues exploit for 8-byte stores.
//
// K is walked in steps of BK = 64 with a register prefetch of the next
// step; LDS rows are padded by 16 bytes so that the 16-byte fragment reads
// of 16 consecutive rows fall on distinct banks.  With F16 set, operand A
// may be stored as bf16 in memory and converted to fp16 while it is staged
// (CVT_A); bf16 values convert exactly inside the fp16 normal range and are
// saturated at +-65504 outside it.
#pragma once
#include "oc_device.h"

namespace oc {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

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
    static constexpr int TA = BA / WA / 16;
    static constexpr int TB = BB / WB / 16;
    static constexpr int CA = BA * (BK / 8) / 256;     // A chunks per thread
    static constexpr int CB = BB * (BK / 8) / 256;
    static_assert(WA * WB == 4, "4 waves");
    static_assert(TA >= 1 && TB >= 1, "tile too small");
    static_assert(CA >= 1 && CB >= 1, "tile too small for 256 threads");
    static_assert(!CVT_A || F16, "conversion only towards fp16");
    static constexpr size_t LDS_BYTES = (size_t)(BA + BB) * LDK * 2;

    f32x4 acc[TA][TB];

    __device__ __forceinline__ void zero() {
#pragma unroll
        for (int i = 0; i < TA; ++i)
#pragma unroll
            for (int j = 0; j < TB; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    // Load one BK step of this thread's chunks into registers.  rows[i] is
    // the row base of chunk slot i (nullptr: zero row); rows are descriptors
    // of segments of seg_len elements, segment s at base + s * sub_stride
    // (seg_len == 0: one plain row).
    template <bool CVT>
    __device__ __forceinline__ static void load_step(const uint16_t *const *rows, int nchunk, int k0, int K,
                                                      int seg_len, long sub_stride, uint4 *regs) {
        const int t = threadIdx.x;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            if (i >= nchunk) break;
            const int c = t + 256 * i;
            const int k = k0 + (c & 7) * 8;
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

    __device__ __forceinline__ static void store_step(uint16_t *lds, int nchunk, const uint4 *regs) {
        const int t = threadIdx.x;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            if (i >= nchunk) break;
            const int c = t + 256 * i;
            const int r = c >> 3;
            *reinterpret_cast<uint4 *>(lds + r * LDK + (c & 7) * 8) = regs[i];
        }
    }

    // One BK step of MFMAs from LDS.
    __device__ __forceinline__ void compute(const uint16_t *As, const uint16_t *Bs) {
        const int lane = threadIdx.x & 63;
        const int wave = threadIdx.x >> 6;
        const int wa = wave / WB, wb = wave % WB;
        const int lr = lane & 15, lk = (lane >> 4) * 8;
#pragma unroll
        for (int ks = 0; ks < BK; ks += 32) {
            if constexpr (F16) {
                f16x8 fa[TA], fb[TB];
#pragma unroll
                for (int i = 0; i < TA; ++i)
                    fa[i] = *reinterpret_cast<const f16x8 *>(As + (wa * (BA / WA) + i * 16 + lr) * LDK + ks + lk);
#pragma unroll
                for (int j = 0; j < TB; ++j)
                    fb[j] = *reinterpret_cast<const f16x8 *>(Bs + (wb * (BB / WB) + j * 16 + lr) * LDK + ks + lk);
#pragma unroll
                for (int i = 0; i < TA; ++i)
#pragma unroll
                    for (int j = 0; j < TB; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(fa[i], fb[j], acc[i][j], 0, 0, 0);
            } else {
                bf16x8 fa[TA], fb[TB];
#pragma unroll
                for (int i = 0; i < TA; ++i)
                    fa[i] = *reinterpret_cast<const bf16x8 *>(As + (wa * (BA / WA) + i * 16 + lr) * LDK + ks + lk);
#pragma unroll
                for (int j = 0; j < TB; ++j)
                    fb[j] = *reinterpret_cast<const bf16x8 *>(Bs + (wb * (BB / WB) + j * 16 + lr) * LDK + ks + lk);
#pragma unroll
                for (int i = 0; i < TA; ++i)
#pragma unroll
                    for (int j = 0; j < TB; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
            }
        }
    }

    // Full K loop.  rowsA[i] / rowsB[i] are this thread's chunk-slot row bases.
    __device__ __forceinline__ void run(uint16_t *lds, const uint16_t *const *rowsA, const uint16_t *const *rowsB,
                                        int K, int seg_len, long sub_stride) {
        uint16_t *As = lds;
        uint16_t *Bs = lds + BA * LDK;
        uint4 ra[CA], rb[CB];
        zero();
        const int nk = cdiv(K, BK);
        load_step<CVT_A>(rowsA, CA, 0, K, seg_len, sub_stride, ra);
        load_step<false>(rowsB, CB, 0, K, seg_len, sub_stride, rb);
        store_step(As, CA, ra);
        store_step(Bs, CB, rb);
        __syncthreads();
        for (int kt = 0; kt < nk; ++kt) {
            const bool more = kt + 1 < nk;
            if (more) {
                load_step<CVT_A>(rowsA, CA, (kt + 1) * BK, K, seg_len, sub_stride, ra);
                load_step<false>(rowsB, CB, (kt + 1) * BK, K, seg_len, sub_stride, rb);
            }
            compute(As, Bs);
            __syncthreads();
            if (more) {
                store_step(As, CA, ra);
                store_step(Bs, CB, rb);
            }
            __syncthreads();
        }
    }

    // Coordinates of accumulator (i, j, e) for this lane, relative to the block.
    __device__ __forceinline__ static int a_of(int i, int e) {
        const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
        return (wave / WB) * (BA / WA) + i * 16 + (lane >> 4) * 4 + e;
    }
    __device__ __forceinline__ static int b_of(int j) {
        const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
        return (wave % WB) * (BB / WB) + j * 16 + (lane & 15);
    }
    // Row of the tile that chunk slot i of this thread loads.
    __device__ __forceinline__ static int chunk_row(int i) { return (threadIdx.x + 256 * i) >> 3; }
};

}  // namespace oc
