/*
 * A chain of cached layer steps driven through the C ABI alone (include/oc.h
 * and liboc.so, no Python): the caller owns every device buffer, plans the
 * call, allocates the workspace the plan asks for, and carries the layer
 * cache from step to step (OmniCache §3.2: each cached step restores the
 * skipped positions from the previous step's layer output).
 *
 *   layer_chain <in.bin> <out.bin>
 *
 * in.bin (little endian): 14 int32 (F, H, W, C, heads, head_dim, n_ctx,
 * dtype, gran, patch_k, cold, n_steps, element size, coarse_k), 3 float64
 * (r, r_frame, r_coarse), then the raw elements of wq, wk, wv, wo, ctx
 * (n_ctx rows, if any) and the n_steps inputs x.  out.bin: per step, the layer output y
 * [F, N, C] followed by the context rows' output [n_ctx, C].
 * Exit status 0 on success; on any error the status, oc_last_error() and
 * the failing call are printed and the status is 1.
 */
#include <stdio.h>
#include <stdlib.h>
#include <string.h>
#include <hip/hip_runtime_api.h>
#include "oc.h"

static int fail_hip(hipError_t e, const char *what) {
    fprintf(stderr, "%s: %s\n", what, hipGetErrorString(e));
    return 1;
}

static int fail_oc(oc_status s, const char *what) {
    fprintf(stderr, "%s: %s: %s\n", what, oc_status_string(s), oc_last_error());
    return 1;
}

/* read n bytes into a new device buffer */
static int upload(FILE *f, size_t n, void **dev) {
    void *h = malloc(n ? n : 1);
    if (!h || fread(h, 1, n, f) != n) {
        fprintf(stderr, "short input file\n");
        free(h);
        return 1;
    }
    hipError_t e = hipMalloc(dev, n ? n : 16);
    if (e == hipSuccess) e = hipMemcpy(*dev, h, n, hipMemcpyHostToDevice);
    free(h);
    return e == hipSuccess ? 0 : fail_hip(e, "upload");
}

int main(int argc, char **argv) {
    if (argc != 3) {
        fprintf(stderr, "usage: %s <in.bin> <out.bin>\n", argv[0]);
        return 2;
    }
    FILE *in = fopen(argv[1], "rb");
    if (!in) {
        perror(argv[1]);
        return 1;
    }
    int32_t hd[14];
    double ratios[3];
    if (fread(hd, sizeof(int32_t), 14, in) != 14 || fread(ratios, sizeof(double), 3, in) != 3) {
        fprintf(stderr, "bad header\n");
        return 1;
    }
    oc_shape sh = {hd[0], hd[1], hd[2], hd[3], hd[4], hd[5], hd[6], hd[7]};
    oc_cfg cfg = {hd[8], hd[9], ratios[0], ratios[1], hd[10], hd[13], ratios[2]};
    const int n_steps = hd[11];
    const size_t esz = (size_t)hd[12];
    const size_t FN = (size_t)sh.F * sh.H * sh.W, hdim = (size_t)sh.heads * sh.head_dim;
    const size_t w_bytes = hdim * sh.C * esz, x_bytes = FN * sh.C * esz, ctx_bytes = (size_t)sh.n_ctx * sh.C * esz;

    oc_plan_info info;
    oc_status s = oc_plan(&sh, &cfg, &info);
    if (s != OC_OK) return fail_oc(s, "oc_plan");

    void *wq, *wk, *wv, *wo, *ctx = NULL, *y, *y_ctx = NULL, *ws;
    if (upload(in, w_bytes, &wq) || upload(in, w_bytes, &wk) || upload(in, w_bytes, &wv) ||
        upload(in, w_bytes, &wo))
        return 1;
    if (sh.n_ctx > 0 && upload(in, ctx_bytes, &ctx)) return 1;
    void **xs = (void **)calloc((size_t)n_steps, sizeof(void *));
    for (int i = 0; i < n_steps; ++i)
        if (upload(in, x_bytes, &xs[i])) return 1;
    fclose(in);

    hipError_t e = hipMalloc(&y, x_bytes);
    if (e == hipSuccess && sh.n_ctx > 0) e = hipMalloc(&y_ctx, ctx_bytes);
    if (e == hipSuccess) e = hipMalloc(&ws, info.workspace_bytes ? info.workspace_bytes : 16);
    if (e != hipSuccess) return fail_hip(e, "hipMalloc");
    hipStream_t st;
    if ((e = hipStreamCreate(&st)) != hipSuccess) return fail_hip(e, "hipStreamCreate");

    oc_attn_weights w = {wq, wk, wv, wo};
    oc_cache cache = {y, 0, 0};
    FILE *out = fopen(argv[2], "wb");
    if (!out) {
        perror(argv[2]);
        return 1;
    }
    unsigned char *hy = (unsigned char *)malloc(x_bytes + ctx_bytes + 1);
    for (int i = 0; i < n_steps; ++i) {
        s = oc_layer_cached(&sh, &cfg, xs[i], ctx, &w, &cache, y_ctx, NULL, ws, info.workspace_bytes, st);
        if (s != OC_OK) return fail_oc(s, "oc_layer_cached");
        if ((e = hipStreamSynchronize(st)) != hipSuccess) return fail_hip(e, "hipStreamSynchronize");
        if ((e = hipMemcpy(hy, y, x_bytes, hipMemcpyDeviceToHost)) != hipSuccess) return fail_hip(e, "copy y");
        if (sh.n_ctx > 0 && (e = hipMemcpy(hy + x_bytes, y_ctx, ctx_bytes, hipMemcpyDeviceToHost)) != hipSuccess)
            return fail_hip(e, "copy y_ctx");
        if (fwrite(hy, 1, x_bytes + ctx_bytes, out) != x_bytes + ctx_bytes) {
            fprintf(stderr, "write failed\n");
            return 1;
        }
    }
    fclose(out);
    if (cache.valid != 1 || cache.step != n_steps) {
        fprintf(stderr, "cache state after %d steps: valid %d, step %d\n", n_steps, cache.valid, cache.step);
        return 1;
    }
    printf("layer_chain: %d steps, %d of %zu tokens retained per warm step\n", n_steps, info.n_kept, FN);
    free(hy);
    for (int i = 0; i < n_steps; ++i) hipFree(xs[i]);
    free(xs);
    hipFree(wq); hipFree(wk); hipFree(wv); hipFree(wo); hipFree(y); hipFree(ws);
    if (ctx) hipFree(ctx);
    if (y_ctx) hipFree(y_ctx);
    hipStreamDestroy(st);
    return 0;
}
