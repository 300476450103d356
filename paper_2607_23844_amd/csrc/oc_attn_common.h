// Shared pieces of the reduced-attention kernels.
#pragma once
#include "oc_internal.h"
#include "oc_device.h"

namespace oc {

// Batch row r of the reduced attention: x rows (through row_idx) then the
// context rows.  nullptr past the end (a zero row for the tile loaders).
// Batch row r (< n_main) -> token: through idx when given, else, for the
// uncached temporal layer (tF > 0), the sequence-per-position order
// r = n*tF + f -> token f*tN + n, else r itself.
__device__ __forceinline__ long batch_token(int r, const int32_t *idx, int tF, int tN) {
    if (idx != nullptr) return idx[r];
    if (tF > 0) {
        const int n = r / tF;
        return (long)(r - n * tF) * tN + n;
    }
    return r;
}

struct RowMap {
    const uint16_t *x; const int32_t *row_idx; int n_main;
    const uint16_t *ctx; int n_rows; int C;
    int tF, tN;
    __device__ __forceinline__ const uint16_t *row(int r) const {
        if (r >= n_rows) return nullptr;
        if (r < n_main) return x + batch_token(r, row_idx, tF, tN) * C;
        return ctx + (long)(r - n_main) * C;
    }
};

// sequence and position of batch row r (a single sequence also owns the
// context rows appended after its L retained tokens); with seq_off,
// sequence s owns rows [seq_off[s], seq_off[s+1]) (binary search; empty
// sequences are skipped over)
__device__ __forceinline__ void seq_pos(int r, int n_seq, int L, int &s, int &j,
                                        const int32_t *seq_off = nullptr) {
    if (seq_off != nullptr) {
        int lo = 0, hi = n_seq - 1;          // last s with seq_off[s] <= r
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (seq_off[mid] <= r) lo = mid; else hi = mid - 1;
        }
        s = lo;
        j = r - seq_off[lo];
        return;
    }
    if (n_seq == 1) { s = 0; j = r; }
    else { s = r / L; j = r - s * L; }
}

// Work-groups are dispatched round-robin over the 8 XCDs (id % 8).  This
// maps a dispatch id to a logical id such that logical ids
// [start_x, start_x + count_x) all run on XCD x: consecutive logical blocks
// share an XCD and its L2.  A bijection on [0, total).
__device__ __forceinline__ int xcd_remap(int id, int total) {
    const int x = id & 7, k = id >> 3;
    int start = 0;
#pragma unroll
    for (int j = 0; j < 7; ++j)
        if (j < x) start += (total - j + 7) >> 3;
    return start + k;
}

// Vt rows store the keys of each 16-key block with quads 1 and 2 swapped:
// the key held at position p (and the position of key p; the map is its own
// inverse).  The attention kernel's PV operand is then one 16-byte read.
__device__ __forceinline__ int vt_key_of_pos(int p) { return (p & ~12) | ((p & 4) << 1) | ((p & 8) >> 1); }

// Whether the attention kernel may stage K/V by DMA for this head dim and
// key count (head dims that are not a multiple of 64 take it only for grids
// of eight-wave blocks).  The DMA path relies on the V projection having
// zeroed the padded key positions [Lk, lpad) of every Vt row.
// (buffer offsets of K are 32-bit: Lk * hd * 2 bytes must stay below 2^31)
inline bool flash_uses_dma(int dh, int Lk, int hd) {
    return dh % 8 == 0 && dh <= 128 && Lk >= 256 && (long)Lk * hd * 2 < (1L << 31);
}

// Whether the attention runs the register-only kernel for short sequences
// (at most 64 keys).  V is then stored row-major like Q and K ([rows, H*dh],
// fp16) instead of as Vt.
inline bool attn_short(int Lk) { return Lk <= 64; }

// Compute units of the MI355X (launch shapes that count block rounds).
constexpr int N_CUS = 256;

// Q/K/V projection and attention fused for short sequences of head dim 64
// (k_short.hip); O is then projected by launch_proj_out.
bool qkv_attn_short_applies(const Plan &p, const AttnArgs &a);
hipError_t launch_qkv_attn_short(const Plan &p, const RowMap &rm, const AttnArgs &a, hipStream_t st);

hipError_t launch_proj_qkv(const Plan &p, const RowMap &rm, const AttnArgs &a, hipStream_t st);
hipError_t launch_proj_out(const Plan &p, int n_rows, const AttnArgs &a, hipStream_t st);
hipError_t launch_flash(const Plan &p, const AttnArgs &a, int Lk, hipStream_t st);

}  // namespace oc
