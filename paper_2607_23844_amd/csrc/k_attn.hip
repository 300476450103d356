// Reduced-token attention dispatcher (OmniCache §3.2.3: the layer runs on
// the retained tokens only; cached tokens are neither queries nor
// keys/values), its workspace layout, and the fp32 path for small layers.
//
// bf16 layers: QKV projection (k_proj.hip) -> flash attention (k_flash.hip)
// -> output projection written straight to the output positions.
// fp32 layers: the same dataflow with plain VALU kernels (below).
#include "oc_attn_common.h"
#include "oc_launch.h"

namespace oc {

struct RowMapF {
    const float *x; const int32_t *row_idx; int n_main;
    const float *ctx; int n_rows; int C;
    int tF, tN;
    __device__ __forceinline__ const float *row(int r) const {
        if (r < n_main) return x + batch_token(r, row_idx, tF, tN) * C;
        return ctx + (long)(r - n_main) * C;
    }
};

// Q/K/V[r][f] for f in [0, 3*hd): one thread per output
__global__ void k_proj_f32(RowMapF rm, const float *__restrict__ wq, const float *__restrict__ wk,
                           const float *__restrict__ wv, int hd, float *__restrict__ Q, float *__restrict__ K,
                           float *__restrict__ V) {
    const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (long)rm.n_rows * 3 * hd) return;
    const int r = (int)(i / (3 * hd)), f = (int)(i - (long)r * 3 * hd);
    const int which = f / hd, c = f - which * hd;
    const float *w = (which == 0 ? wq : which == 1 ? wk : wv) + (long)c * rm.C;
    const float *x = rm.row(r);
    float acc = 0.f;
    for (int k = 0; k < rm.C; ++k) acc = fmaf(x[k], w[k], acc);
    (which == 0 ? Q : which == 1 ? K : V)[(long)r * hd + c] = acc;
}

// one thread per (query row, head): online softmax over the sequence's keys
__global__ void k_attn_f32(const float *__restrict__ Q, const float *__restrict__ K, const float *__restrict__ V,
                           float *__restrict__ O, int n_rows, int heads, int dh, int n_seq, int L, int Lk,
                           float scale, const int32_t *__restrict__ seq_off) {
    const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (long)n_rows * heads) return;
    const int r = (int)(i / heads), h = (int)(i - (long)r * heads);
    const int hd = heads * dh;
    int s, j;
    seq_pos(r, n_seq, L, s, j, seq_off);
    long row0 = (long)s * L;
    if (seq_off != nullptr) {
        row0 = seq_off[s];
        Lk = seq_off[s + 1] - seq_off[s];
    }
    const float *q = Q + (long)r * hd + h * dh;
    float acc[128];
    for (int d = 0; d < dh; ++d) acc[d] = 0.f;
    float m = -INFINITY, l = 0.f;
    for (int kk = 0; kk < Lk; ++kk) {
        const float *k = K + (row0 + kk) * hd + h * dh;
        float sc = 0.f;
        for (int d = 0; d < dh; ++d) sc = fmaf(q[d], k[d], sc);
        sc *= scale;
        const float mn = fmaxf(m, sc);
        const float a = expf(m - mn), p = expf(sc - mn);
        l = l * a + p;
        const float *v = V + (row0 + kk) * hd + h * dh;
        for (int d = 0; d < dh; ++d) acc[d] = acc[d] * a + p * v[d];
        m = mn;
    }
    float *o = O + (long)r * hd + h * dh;
    for (int d = 0; d < dh; ++d) o[d] = acc[d] / l;
}

__global__ void k_out_f32(const float *__restrict__ O, int n_rows, int hd, const float *__restrict__ wo, int C,
                          int n_main, const int32_t *__restrict__ out_idx, int tF, int tN, float *__restrict__ y,
                          float *__restrict__ y_ctx) {
    const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (long)n_rows * C) return;
    const int r = (int)(i / C), c = (int)(i - (long)r * C);
    const float *o = O + (long)r * hd;
    const float *w = wo + (long)c * hd;
    float acc = 0.f;
    for (int k = 0; k < hd; ++k) acc = fmaf(o[k], w[k], acc);
    if (r < n_main) y[batch_token(r, out_idx, tF, tN) * C + c] = acc;
    else y_ctx[(long)(r - n_main) * C + c] = acc;
}

AttnWs attn_ws(const Plan &p, int n_seq, int L, size_t base) {
    AttnWs w;
    const long rows = (long)n_seq * L + p.n_ctx;
    const int Lk = L + (n_seq == 1 ? p.n_ctx : 0);
    w.lpad = cdiv(Lk > 0 ? Lk : 1, 64) * 64;
    auto al = [](size_t b) { return (b + 255) & ~(size_t)255; };
    const size_t e = p.esz == 2 ? 2 : 4;   // fp16 intermediates for bf16 layers
    const size_t m = al((size_t)rows * p.hd * e);
    w.q = base;
    w.k = w.q + m;
    w.o = w.k + m;
    w.v = w.o + m;
    // Vt (or, for short sequences, V rows: never more than m)
    const size_t vt = al((size_t)p.heads * n_seq * p.dh * w.lpad * e);
    const size_t vb = p.bf16 ? (vt > m ? vt : m) : m;
    w.wo16 = w.v + vb;
    const size_t wb = p.bf16 ? al((size_t)p.C * p.hd * 2) : 0;
    w.bytes = w.wo16 + wb - base;
    return w;
}

bool attn_head_dim_supported(int dh) {
    switch (dh) {
        case 16: case 32: case 48: case 64: case 72: case 80: case 96: case 128: return true;
        default: return false;
    }
}

hipError_t launch_attention(const Plan &p, const AttnArgs &a, hipStream_t st) {
    const int n_rows = a.seq_off != nullptr ? a.n_main : a.n_seq * a.L + a.n_ctx;
    const int Lk = a.L + (a.n_seq == 1 ? a.n_ctx : 0);
    if (n_rows == 0) return hipSuccess;
    if (p.bf16) {
        const RowMap rm{(const uint16_t *)a.x, a.row_idx, a.n_main, (const uint16_t *)a.ctx, n_rows, p.C, a.tF, a.tN};
        hipError_t e;
        if (qkv_attn_short_applies(p, a)) {
            if ((e = launch_qkv_attn_short(p, rm, a, st)) != hipSuccess) return e;
            return launch_proj_out(p, n_rows, a, st);
        }
        e = launch_proj_qkv(p, rm, a, st);
        if (e != hipSuccess) return e;
        if ((e = launch_flash(p, a, Lk, st)) != hipSuccess) return e;
        return launch_proj_out(p, n_rows, a, st);
    }
    const RowMapF rm{(const float *)a.x, a.row_idx, a.n_main, (const float *)a.ctx, n_rows, p.C, a.tF, a.tN};
    const long nq = (long)n_rows * 3 * p.hd;
    {
        StageScope _stage(st, "proj_f32");
        launch_k(k_proj_f32, (unsigned)((nq + 255) / 256), 256, 0, st, rm, (const float *)a.wq, (const float *)a.wk,
                                                                  (const float *)a.wv, p.hd, (float *)a.q,
                                                                  (float *)a.k, (float *)a.vt);
    }
    const long na = (long)n_rows * p.heads;
    {
        StageScope _stage(st, "attn_f32");
        launch_k(k_attn_f32, (unsigned)((na + 127) / 128), 128, 0, st, (const float *)a.q, (const float *)a.k,
                                                                  (const float *)a.vt, (float *)a.o, n_rows, p.heads,
                                                                  p.dh, a.n_seq, a.L, Lk,
                                                                  (float)(1.0 / sqrt((double)p.dh)), a.seq_off);
    }
    const long no = (long)n_rows * p.C;
    {
        StageScope _stage(st, "out_f32");
        launch_k(k_out_f32, (unsigned)((no + 255) / 256), 256, 0, st, (const float *)a.o, n_rows, p.hd,
                                                                 (const float *)a.wo, p.C, a.n_main, a.out_idx, a.tF,
                                                                 a.tN, (float *)a.y, (float *)a.y_ctx);
    }
    return hipGetLastError();
}

}  // namespace oc
