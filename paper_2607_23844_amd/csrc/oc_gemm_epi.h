// Pieces shared by the GEMM-shaped kernels (projections, feed-forward):
// XCD-grouped tile order, the LDS-staged row epilogue and the engine switch.
#pragma once
#include "oc_internal.h"
#include "oc_launch.h"
#include "oc_device.h"
#include "oc_mfma_tile.h"
#include "oc_dma_tile.h"

namespace oc {

constexpr int GA = 6;

// logical tile lid -> (a tile, b tile), GA a-tiles per group, b fastest inside
__device__ __forceinline__ void tile_order(int lid, int n_at, int n_bt, int &at, int &bt) {
    const int per = GA * n_bt;
    const int grp = lid / per, idx = lid - grp * per;
    const int ga = min(GA, n_at - grp * GA);
    at = grp * GA + idx % ga;
    bt = idx / ga;
}

// Stage the block's results as rows of b with the a values contiguous:
// S[b][col(a)], row stride BA + 8 halves.  cvt(value, a) gives the 16-bit
// pattern of element (a, b); col maps an aligned quad of a to an aligned
// quad of columns.
template <int BA, typename T, typename Cvt, typename Col>
__device__ __forceinline__ void stage_rows(const T &t, uint16_t *S, Cvt cvt, Col col) {
    constexpr int SROW = BA + 8;
#pragma unroll
    for (int j = 0; j < T::TB; ++j) {
        const int b = T::b_of(j);
#pragma unroll
        for (int i = 0; i < T::TA; ++i)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int a = T::a_of(i, g);
                u16x4 v;
#pragma unroll
                for (int e = 0; e < 4; ++e) v[e] = cvt(t.acc[i][j][4 * g + e], a + e);
                *reinterpret_cast<u16x4 *>(S + b * SROW + col(a)) = v;
            }
    }
}

// Write the staged rows in 16-byte chunks: chunk (b, c0) (columns c0..c0+7,
// c0 < ncol) goes to dst(b, c0); nullptr skips it.
template <int BA, int BB, typename Dst>
__device__ __forceinline__ void write_rows(const uint16_t *S, int ncol, Dst dst) {
    constexpr int SROW = BA + 8, CPR = BA / 8;
    for (int c = threadIdx.x; c < BB * CPR; c += 256) {
        const int b = c / CPR, c0 = (c - b * CPR) * 8;
        if (c0 >= ncol) continue;
        uint16_t *d = dst(b, c0);
        if (d != nullptr) *reinterpret_cast<uint4 *>(d) = *reinterpret_cast<const uint4 *>(S + b * SROW + c0);
    }
}

struct RegRows { static constexpr bool dma = false; };
struct DmaRows { static constexpr bool dma = true; };
template <typename T, typename Rows>
__device__ __forceinline__ void run_tile(T &t, uint16_t *lds, const uint16_t *const *rowsA,
                                         const uint16_t *const *rowsB, const uint16_t *fbA, const uint16_t *fbB, int K,
                                         Rows) {
    if constexpr (Rows::dma) t.run(lds, rowsA, rowsB, fbA, fbB, K, 0, 0);
    else t.run(lds, rowsA, rowsB, K, 0, 0);
}

template <typename KernelPtr>
static hipError_t allow_lds(KernelPtr k, size_t bytes) {
    return raise_lds_limit((const void *)k, bytes);
}

}  // namespace oc
