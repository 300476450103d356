// Feed-forward sublayer under the attention's selection (the SD3 experiments
// cache attention and FFN layers alike): y[row] = GELU(x[row] W1^T) W2^T for
// the retained rows only, on the LDS-DMA MFMA tile engine (bf16 operands,
// fp32 accumulation).
//   k_ffn_up:   [rows, C] x [hidden, C]^T -> H [rows, hidden] fp16, the
//               batch rows gathered from x through kept_idx in the operand
//               load (no separate gather), GELU applied in the epilogue;
//               the launch's extra blocks convert W2 to fp16 meanwhile;
//   k_ffn_down: H x [C, hidden]^T (fp16 MFMA) -> y rows (bf16), written
//               straight to their token positions (restoration in place:
//               cached rows are never touched) or to a compact [rows, C]
//               buffer.
// H is fp16 rather than bf16: three more significant bits for the one
// intermediate that every output sums 'hidden' terms of (bf16 measured
// 0.93% of the output RMS at the SD3 shape beyond the output's own rounding).
// GELU is the tanh form, evaluated as v / (1 + exp(-2 z)) with
// z = sqrt(2/pi) (v + 0.044715 v^3), which equals 0.5 v (1 + tanh z).
#include "oc_gemm_epi.h"
#include "oc_attn_common.h"

namespace oc {

namespace {

__device__ __forceinline__ float gelu_tanh_f(float v) {
    const float z = 0.7978845608028654f * fmaf(0.044715f * v, v * v, v);
    return v / (1.0f + __expf(-2.0f * z));
}

// Batch row r -> token row of x (nullptr past the batch or for an index
// outside [0, FN): such a row computes garbage that is never stored)
__device__ __forceinline__ const uint16_t *ffn_row(const uint16_t *x, const int32_t *idx, int n_rows, int FN, int C,
                                                   int r) {
    if (r >= n_rows) return nullptr;
    const long t = idx != nullptr ? (long)idx[r] : (long)r;
    return (t >= 0 && t < FN) ? x + t * C : nullptr;
}

template <int BA, int BB, bool F16 = false>
using FfnTile = DmaTile<BA, BB, 2, 2, F16, 2>;

// up: a = rows of w1 (hidden), b = batch rows
template <int BA, int BB>
__global__ __launch_bounds__(256) void k_ffn_up(const uint16_t *__restrict__ x, const int32_t *__restrict__ idx,
                                                int n_rows, int FN, int C, const uint16_t *__restrict__ w1,
                                                int hidden, int n_at, int n_bt, uint16_t *__restrict__ H,
                                                const uint4 *__restrict__ w2, long n8, uint4 *__restrict__ w2h) {
    using T = FfnTile<BA, BB>;
    static_assert((size_t)BB * (BA + 8) * 2 <= T::LDS_BYTES, "staged rows fit in the ring");
    extern __shared__ __align__(16) uint16_t lds[];
    const int n_tiles = n_at * n_bt;
    if ((int)blockIdx.x >= n_tiles) {
        // W2 -> fp16 for the down-projection, 8 elements per thread
        const long nb = gridDim.x - n_tiles;
        for (long i = (long)(blockIdx.x - n_tiles) * blockDim.x + threadIdx.x; i < n8; i += nb * blockDim.x)
            w2h[i] = bf16x8_to_f16x8(w2[i]);
        return;
    }
    int at, bt;
    tile_order(xcd_remap(blockIdx.x, n_tiles), n_at, n_bt, at, bt);
    const uint16_t *rowsA[T::CA], *rowsB[T::CB];
#pragma unroll
    for (int i = 0; i < T::CA; ++i) {
        const int a = at * BA + T::chunk_row(i);
        rowsA[i] = a < hidden ? w1 + (long)a * C : nullptr;
    }
#pragma unroll
    for (int i = 0; i < T::CB; ++i) rowsB[i] = ffn_row(x, idx, n_rows, FN, C, bt * BB + T::chunk_row(i));
    T t;
    t.run(lds, rowsA, rowsB, w1, x, C, 0, 0);
    const int a0 = at * BA, b0 = bt * BB;
    stage_rows<BA>(t, lds, [](float v, int) { return f2h_bits(gelu_tanh_f(v)); }, [](int a) { return a; });
    __syncthreads();
    write_rows<BA, BB>(lds, min(BA, hidden - a0), [&](int b, int c0) -> uint16_t * {
        const int r = b0 + b;
        return r < n_rows ? H + (long)r * hidden + a0 + c0 : nullptr;
    });
}

// down: a = rows of w2 (fp16, C), b = rows of H; row r goes to y row idx[r]
// (scatter) or r, and nowhere when its token index was outside [0, FN)
template <int BA, int BB>
__global__ __launch_bounds__(256) void k_ffn_down(const uint16_t *__restrict__ H, int n_rows, int hidden,
                                                  const uint16_t *__restrict__ w2, int C,
                                                  const int32_t *__restrict__ idx, int scatter, int FN, int n_at,
                                                  int n_bt, uint16_t *__restrict__ y) {
    using T = FfnTile<BA, BB, true>;
    static_assert((size_t)BB * (BA + 8) * 2 <= T::LDS_BYTES, "staged rows fit in the ring");
    extern __shared__ __align__(16) uint16_t lds[];
    int at, bt;
    tile_order(xcd_remap(blockIdx.x, n_at * n_bt), n_at, n_bt, at, bt);
    const uint16_t *rowsA[T::CA], *rowsB[T::CB];
#pragma unroll
    for (int i = 0; i < T::CA; ++i) {
        const int a = at * BA + T::chunk_row(i);
        rowsA[i] = a < C ? w2 + (long)a * hidden : nullptr;
    }
#pragma unroll
    for (int i = 0; i < T::CB; ++i) {
        const int b = bt * BB + T::chunk_row(i);
        rowsB[i] = b < n_rows ? H + (long)b * hidden : nullptr;
    }
    T t;
    t.run(lds, rowsA, rowsB, w2, H, hidden, 0, 0);
    const int a0 = at * BA, b0 = bt * BB;
    stage_rows<BA>(t, lds, [](float v, int) { return f2bf(v); }, [](int a) { return a; });
    __syncthreads();
    write_rows<BA, BB>(lds, min(BA, C - a0), [&](int b, int c0) -> uint16_t * {
        const int r = b0 + b;
        if (r >= n_rows) return nullptr;
        const long tok = idx != nullptr ? (long)idx[r] : (long)r;
        if (tok < 0 || tok >= FN) return nullptr;          // the row was never read
        return y + (scatter ? tok : (long)r) * C + a0 + c0;
    });
}

template <typename K, typename... A>
hipError_t go(K kern, size_t lds, unsigned blocks, hipStream_t st, A... args) {
    const hipError_t e = raise_lds_limit((const void *)kern, lds);
    if (e != hipSuccess) return e;
    launch_k(kern, blocks, 256, lds, st, args...);
    return hipGetLastError();
}

}  // namespace

size_t ffn_h_bytes(int n_rows, int hidden) { return ((size_t)n_rows * hidden * 2 + 255) & ~(size_t)255; }
size_t ffn_workspace_bytes(int n_rows, int hidden, int C) {
    if (n_rows == 0) return 0;   // nothing is launched
    return ffn_h_bytes(n_rows, hidden) + (((size_t)C * hidden * 2 + 255) & ~(size_t)255);
}

hipError_t launch_ffn(const FfnArgs &a, hipStream_t st) {
    if (a.n_rows == 0) return hipSuccess;
    if (a.C % 64 || a.hidden % 64) return hipErrorInvalidValue;
    uint16_t *h = (uint16_t *)a.h;
    uint16_t *w2h = (uint16_t *)((char *)a.h + ffn_h_bytes(a.n_rows, a.hidden));
    const long n8 = (long)a.C * a.hidden / 8;
    const unsigned cvt_blocks = (unsigned)std::min<long>((n8 + 255) / 256, 256);
    // up-projection: 192 x 128 tiles where they need fewer block rounds
    // (two blocks per CU) times tile work than 128 x 128 (a wide tile is 1.5)
    {
        StageScope _stage(st, "ffn_up");
        const long slots = 2L * N_CUS;
        const long t128 = (long)cdiv(a.hidden, 128) * cdiv(a.n_rows, 128);
        const long t192 = (long)cdiv(a.hidden, 192) * cdiv(a.n_rows, 128);
        const long c128 = 2 * ((t128 + slots - 1) / slots), c192 = 3 * ((t192 + slots - 1) / slots);
        hipError_t e;
        if (c192 < c128) {
            const int n_at = cdiv(a.hidden, 192), n_bt = cdiv(a.n_rows, 128);
            e = go(k_ffn_up<192, 128>, FfnTile<192, 128>::LDS_BYTES, (unsigned)(n_at * n_bt) + cvt_blocks, st,
                   (const uint16_t *)a.x, a.idx, a.n_rows, a.FN, a.C, (const uint16_t *)a.w1, a.hidden, n_at, n_bt, h,
                   (const uint4 *)a.w2, n8, (uint4 *)w2h);
        } else {
            const int n_at = cdiv(a.hidden, 128), n_bt = cdiv(a.n_rows, 128);
            e = go(k_ffn_up<128, 128>, FfnTile<128, 128>::LDS_BYTES, (unsigned)(n_at * n_bt) + cvt_blocks, st,
                   (const uint16_t *)a.x, a.idx, a.n_rows, a.FN, a.C, (const uint16_t *)a.w1, a.hidden, n_at, n_bt, h,
                   (const uint4 *)a.w2, n8, (uint4 *)w2h);
        }
        if (e != hipSuccess) return e;
    }
    // down-projection: 128 x 64 tiles (K = hidden is long; three blocks per CU)
    StageScope _stage(st, "ffn_down");
    const int n_at = cdiv(a.C, 128), n_bt = cdiv(a.n_rows, 64);
    return go(k_ffn_down<128, 64>, FfnTile<128, 64, true>::LDS_BYTES, (unsigned)(n_at * n_bt), st, h, a.n_rows,
              a.hidden, w2h, a.C, a.idx, a.scatter, a.FN, n_at, n_bt, (uint16_t *)a.y);
}

}  // namespace oc
