// Host side of the OmniCache C ABI: validation, static planning, workspace
// carving and launch sequencing.  No device memory is allocated here; all
// work goes on the caller's stream.
#include "../../include/oc.h"
#include "oc_internal.h"

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>

using namespace oc;

namespace {

thread_local std::string g_err;

oc_status fail(oc_status s, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_err = buf;
    return s;
}

oc_status ok() {
    g_err.clear();
    return OC_OK;
}

// floor(ratio * n) with a guard against binary representation error
int floor_ratio(double r, int n) { return (int)std::floor(r * (double)n + 1e-9); }

size_t al(size_t b) { return (b + 255) & ~(size_t)255; }

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

oc_status check_shape(const oc_shape *sh) {
    if (!sh) return fail(OC_ERR_INVALID_ARG, "shape is NULL");
    if (sh->dtype != OC_F32 && sh->dtype != OC_BF16) return fail(OC_ERR_DTYPE, "unknown dtype %d", sh->dtype);
    if (sh->F < 1 || sh->H < 1 || sh->W < 1 || sh->C < 1 || sh->heads < 1 || sh->head_dim < 1 || sh->n_ctx < 0)
        return fail(OC_ERR_SHAPE, "shape fields must be positive (n_ctx >= 0)");
    if (sh->C % 8) return fail(OC_ERR_SHAPE, "C=%d must be a multiple of 8", sh->C);
    if (sh->head_dim % 8 || sh->head_dim > 128)
        return fail(OC_ERR_SHAPE, "head_dim=%d must be a multiple of 8 and <= 128", sh->head_dim);
    if (sh->dtype == OC_BF16 && !attn_head_dim_supported(sh->head_dim))
        return fail(OC_ERR_SHAPE, "bf16 head_dim=%d not one of 16,32,48,64,72,80,96,128", sh->head_dim);
    const long long fn = (long long)sh->F * sh->H * sh->W;
    if (fn * sh->C >= (1LL << 31) || fn + sh->n_ctx >= (1LL << 30))
        return fail(OC_ERR_SHAPE, "tensor too large for 32-bit token indices");
    return OC_OK;
}

oc_status check_cfg(const oc_cfg *cfg) {
    if (!cfg) return fail(OC_ERR_INVALID_ARG, "cfg is NULL");
    if (cfg->gran < 0 || cfg->gran > 3) return fail(OC_ERR_INVALID_ARG, "unknown granularity %d", cfg->gran);
    if (cfg->cold != OC_COLD_MATCHED && cfg->cold != OC_COLD_FULL)
        return fail(OC_ERR_INVALID_ARG, "unknown cold policy %d", cfg->cold);
    if (cfg->coarse_k != 0) {
        if (cfg->gran != OC_GRAN_TOKEN && cfg->gran != OC_GRAN_BLOCK)
            return fail(OC_ERR_INVALID_ARG, "a coarser level (coarse_k) is defined for Token and Block Cache only");
        if (cfg->coarse_k < 1 || cfg->coarse_k >= cfg->patch_k || cfg->patch_k % cfg->coarse_k != 0)
            return fail(OC_ERR_SHAPE, "coarse_k=%d must divide patch_k=%d and be smaller", cfg->coarse_k,
                        cfg->patch_k);
        if (!(cfg->r_coarse >= 0.0 && cfg->r_coarse < 1.0))
            return fail(OC_ERR_INVALID_ARG, "r_coarse=%g outside [0,1)", cfg->r_coarse);
    }
    if (!(cfg->r >= 0.0 && cfg->r < 1.0)) return fail(OC_ERR_INVALID_ARG, "r=%g outside [0,1)", cfg->r);
    if (!(cfg->r_frame >= 0.0 && cfg->r_frame < 1.0))
        return fail(OC_ERR_INVALID_ARG, "r_frame=%g outside [0,1)", cfg->r_frame);
    if (cfg->patch_k < 1) return fail(OC_ERR_SHAPE, "patch_k=%d must be >= 1", cfg->patch_k);
    return OC_OK;
}

// Static plan of one call.  no_skip sets every budget to 0.
oc_status make_plan(const oc_shape *sh, const oc_cfg *cfg, bool no_skip, Plan &p) {
    oc_status s = check_shape(sh);
    if (s != OC_OK) return s;
    if ((s = check_cfg(cfg)) != OC_OK) return s;
    std::memset(&p, 0, sizeof(p));
    p.F = sh->F; p.H = sh->H; p.W = sh->W; p.C = sh->C; p.N = sh->H * sh->W;
    p.heads = sh->heads; p.dh = sh->head_dim; p.hd = sh->heads * sh->head_dim; p.n_ctx = sh->n_ctx;
    p.bf16 = sh->dtype == OC_BF16;
    p.esz = p.bf16 ? 2 : 4;
    p.gran = cfg->gran;
    p.k = cfg->patch_k;
    p.r = no_skip ? 0.0 : cfg->r;
    p.r_frame = no_skip ? 0.0 : cfg->r_frame;
    if (sh->H % (2 * p.k) || sh->W % (2 * p.k))
        return fail(OC_ERR_SHAPE, "H=%d and W=%d must be divisible by 2*patch_k=%d", sh->H, sh->W, 2 * p.k);
    if (sh->n_ctx > 0 && (sh->F != 1 || cfg->gran != OC_GRAN_TOKEN))
        return fail(OC_ERR_SHAPE, "context tokens need F == 1 and OC_GRAN_TOKEN");
    if ((cfg->gran == OC_GRAN_FRAME || cfg->gran == OC_GRAN_FRAME_TOKEN) && (sh->F < 2 || sh->F > 32))
        return fail(OC_ERR_SHAPE, "frame caching needs 2 <= F <= 32 (F=%d)", sh->F);
    if (cfg->gran == OC_GRAN_FRAME && p.k > 1 && p.k * p.k > 256)
        return fail(OC_ERR_SHAPE, "Frame Cache on patches needs patch_k <= 16 (patch_k=%d)", p.k);
    p.ph = p.H / p.k;
    p.pw = p.W / p.k;
    p.np = p.ph * p.pw;
    p.np_dst = p.np / 4;
    p.np_src = p.np - p.np_dst;
    const int kk = p.k * p.k;
    auto clampi = [](int a, int b) { return a < b ? a : b; };
    p.R_tok = clampi(floor_ratio(p.r, p.np), p.np_src);
    switch (cfg->gran) {
        case OC_GRAN_TOKEN:
            p.kind = KIND_TOKEN;
            p.n_groups = p.F * kk; p.n_src_max = p.np_src; p.n_dst_max = p.np_dst;
            p.n_units = p.F;
            p.n_seq = p.F; p.seq_len = p.N - kk * p.R_tok;
            p.n_items = p.F * p.N;
            break;
        case OC_GRAN_BLOCK:
            p.kind = KIND_BLOCK;
            p.n_groups = kk; p.n_src_max = p.np_src; p.n_dst_max = p.np_dst;
            p.n_seq = p.N - kk * p.R_tok; p.seq_len = p.F;
            p.n_items = p.N;
            break;
        case OC_GRAN_FRAME:
            p.n_fsrc = p.F / 2; p.n_fdst = (p.F + 1) / 2;
            p.R_f = clampi(floor_ratio(p.r_frame, p.F), p.n_fsrc);
            p.n_src_max = p.n_fsrc; p.n_dst_max = p.n_fdst;
            if (p.k == 1) {
                p.kind = KIND_FRAME;
                p.n_groups = 1;
                p.n_seq = p.F - p.R_f; p.seq_len = p.N;
                p.n_items = p.F;
            } else {
                // per patch: R_f of the odd frames' tiles; every frame keeps a
                // varying number of tokens, R_f * N in all are cached
                p.kind = KIND_FPATCH;
                p.n_groups = kk;
                p.n_seq = p.F; p.seq_len = p.N;
                p.n_items = p.F * p.N;
            }
            break;
        default: {  // OC_GRAN_FRAME_TOKEN
            p.kind = KIND_TOKEN;
            p.n_fsrc = p.F / 2; p.n_fdst = (p.F + 1) / 2;
            p.R_f = clampi(floor_ratio(p.r_frame, p.F), p.n_fsrc);
            p.n_units = p.F - p.R_f;
            p.n_groups = p.n_units * kk;
            p.n_src_max = p.R_f > 0 ? p.np + p.np_src : p.np_src;
            p.n_dst_max = p.np_dst;
            p.R_pair = clampi(p.np + floor_ratio(p.r, p.np), p.np + p.np_src);
            p.n_seq = p.n_units; p.seq_len = kk * (p.np - p.R_tok);
            if (p.R_f > 0 && kk * (2 * p.np - p.R_pair) != p.seq_len)
                return fail(OC_ERR_SHAPE, "internal: pair and frame sequence lengths differ");
            p.n_items = p.F * p.N;
            break;
        }
    }
    if (p.n_src_max > 16384) return fail(OC_ERR_SHAPE, "group of %d candidates exceeds 16384", p.n_src_max);
    if (cfg->coarse_k > 0) {
        // second level: each coarse patch holds (k/k2)^2 first-level patches,
        // every one of which cached exactly R_tok, so its remaining
        // candidates and its budget are static
        p.k2 = cfg->coarse_k;
        p.r2 = no_skip ? 0.0 : cfg->r_coarse;
        p.np2 = (p.H / p.k2) * (p.W / p.k2);
        p.np2_dst = p.np2 / 4;
        p.np2_src = p.np2 - p.np2_dst;
        const int sub = (p.k / p.k2) * (p.k / p.k2);
        p.R2 = clampi(floor_ratio(p.r2, p.np2), p.np2_src - sub * p.R_tok);
        if (p.np2_src > 16384) return fail(OC_ERR_SHAPE, "coarse group of %d candidates exceeds 16384", p.np2_src);
        const int more = p.k2 * p.k2 * p.R2;   // per frame (Token) or in all (Block)
        if (p.kind == KIND_TOKEN) p.seq_len -= more;
        else p.n_seq -= more;
    }
    p.n_kept = p.kind == KIND_FPATCH ? (p.F - p.R_f) * p.N : p.n_seq * p.seq_len;
    p.n_cached = p.F * p.N - p.n_kept;
    return OC_OK;
}

// The matching problem of the second level: the same plan with its patches
// and budget (the reduced batch and the counts stay those of the whole call).
Plan coarse_plan(const Plan &p) {
    Plan q = p;
    q.k = p.k2;
    q.ph = p.H / p.k2;
    q.pw = p.W / p.k2;
    q.np = p.np2;
    q.np_src = p.np2_src;
    q.np_dst = p.np2_dst;
    q.R_tok = p.R2;
    q.r = p.r2;
    q.n_groups = (p.kind == KIND_TOKEN ? p.F : 1) * p.k2 * p.k2;
    q.n_src_max = p.np2_src;
    q.n_dst_max = p.np2_dst;
    q.k2 = 0;
    return q;
}

// The plan of the uncached layer: spatial (per frame) or temporal (per position).
Plan full_plan(const Plan &p) {
    Plan q = p;
    q.r = q.r_frame = 0.0;
    q.R_tok = q.R_pair = q.R_f = 0;
    if (p.kind == KIND_BLOCK) {
        q.n_seq = p.N; q.seq_len = p.F;
    } else {
        q.kind = KIND_TOKEN; q.gran = OC_GRAN_TOKEN;
        q.n_units = p.F; q.n_seq = p.F; q.seq_len = p.N;
    }
    q.n_kept = p.F * p.N;
    q.n_cached = 0;
    return q;
}

Layout make_layout(const Plan &p) {
    Layout L;
    std::memset(&L, 0, sizeof(L));
    size_t o = 0;
    auto take = [&o](size_t bytes) { const size_t at = o; o += al(bytes); return at; };
    const size_t FN = (size_t)p.F * p.N;
    const size_t GS = (size_t)p.n_groups * p.n_src_max;
    L.inv = take(FN * 4);
    // (the second level's arg-max uses the same buffer: as many candidates in all)
    const size_t GS2 = p.k2 > 0 ? (size_t)coarse_plan(p).n_groups * p.np2_src : 0;
    L.node_pack = take((GS > GS2 ? GS : GS2) * 8);
    L.node_max = take(GS * 4);
    L.node_idx = take(GS * 4);
    {
        const MatchSplit ms = match_split(p);
        size_t mp = ms.n_split > 1 ? (size_t)ms.n_split * GS * p.n_dst_max * 4 : 0;
        if (p.k2 > 0) {
            // the second level reuses the arg-max and partial-sum buffers
            const Plan q = coarse_plan(p);
            const MatchSplit m2 = match_split(q);
            const size_t GS2 = (size_t)q.n_groups * q.n_src_max;
            if (m2.n_split > 1 && (size_t)m2.n_split * GS2 * q.n_dst_max * 4 > mp)
                mp = (size_t)m2.n_split * GS2 * q.n_dst_max * 4;
        }
        L.mpart = take(mp);
    }
    const bool frames = p.kind == KIND_FRAME || p.gran == OC_GRAN_FRAME_TOKEN;
    L.gram_part = take(frames ? (size_t)gram_blocks(p) * 1024 * 4 : 0);
    L.fgram = take(frames ? 1024 * 8 : 0);
    L.fsim = take(frames ? 1024 * 8 : 0);
    L.fmax = take(64 * 4);
    L.fidx = take(64 * 4);
    L.forder = take(64 * 4);
    L.pairs = take(64 * 4);
    L.units = take(64 * 4);
    L.flag = take(FN * 4);
    L.mtok = take(FN * 4);
    L.fcnt = take((size_t)p.F * ((p.N + 1023) / 1024) * 4);   // cached tokens per 1024-token chunk
    L.kept = take(FN * 4);
    L.cached = take(FN * 4);
    L.rmap = take(FN * 4);
    L.seqoff = take((size_t)(p.F + 1) * 4);
    L.attn = o;
    const Plan fp = full_plan(p);
    const AttnWs a1 = attn_ws(p, p.n_seq, p.seq_len, o);
    const AttnWs a2 = attn_ws(fp, fp.n_seq, fp.seq_len, o);
    L.total = o + (a1.bytes > a2.bytes ? a1.bytes : a2.bytes);
    return L;
}

// Group-size-independent workspace: the layout of the plan with the largest
// groups (cold "full" steps need none larger; the frame-token plan with
// pairs has the widest groups).
size_t workspace_for(const oc_shape *sh, const oc_cfg *cfg) {
    Plan p;
    if (make_plan(sh, cfg, false, p) != OC_OK) return 0;
    size_t t = make_layout(p).total;
    Plan q;
    if (make_plan(sh, cfg, true, q) == OC_OK) {
        const size_t t2 = make_layout(q).total;
        if (t2 > t) t = t2;
    }
    return t;
}

oc_status hip_fail(hipError_t e, const char *what) {
    return fail(OC_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

#define HIP_TRY(call, what)                    \
    do {                                       \
        hipError_t e_ = (call);                \
        if (e_ != hipSuccess) return hip_fail(e_, what); \
    } while (0)

oc_status check_ws(void *ws, size_t ws_bytes, size_t need) {
    if (ws_bytes < need) return fail(OC_ERR_WORKSPACE, "workspace %zu bytes < required %zu", ws_bytes, need);
    if (need > 0 && (!ws || ((uintptr_t)ws & 255u)))
        return fail(OC_ERR_INVALID_ARG, "workspace must be non-NULL and 256-byte aligned");
    return OC_OK;
}

template <typename T> T *at(void *ws, size_t off) { return reinterpret_cast<T *>((char *)ws + off); }

const int32_t *units_of(const Plan &p, const Layout &L, void *ws) {
    return p.gran == OC_GRAN_FRAME_TOKEN ? at<int32_t>(ws, L.units) : nullptr;
}

// Match stage.  With reduce, (node_max, node_idx) are produced; without,
// only the packed arg-max is left in ws for launch_select_packed (frame
// granularity always produces node_max / node_idx).  Leaves the frame stage
// and norms in ws; wo / wo16, when given (bf16), are converted in the first
// launch that reads x (the frame Gram, else the norms).
oc_status run_match(const Plan &p, const Layout &L, const void *x, float *node_max, int32_t *node_idx, bool reduce,
                    void *ws, hipStream_t st, const void *wo = nullptr, void *wo16 = nullptr,
                    bool frame_compact = false) {
    char *w = (char *)ws;
    const bool frames = p.kind == KIND_FRAME || p.gran == OC_GRAN_FRAME_TOKEN;
    unsigned long long *pack = at<unsigned long long>(ws, L.node_pack);
    const long n_pack = (long)p.n_groups * p.n_src_max;
    // Frame+Token Cache: the Gram launch also writes the token norms and clears pack
    const bool gram_prep = frames && gram_norms(p);
    if (frames) {
        float *fm = p.gran == OC_GRAN_FRAME ? node_max : at<float>(ws, L.fmax);
        int32_t *fi = p.gran == OC_GRAN_FRAME ? node_idx : at<int32_t>(ws, L.fidx);
        // Frame Cache: the frame stage also writes the per-frame selection
        const bool fsel = p.gran == OC_GRAN_FRAME;
        const bool cvt = p.bf16 && (fsel || gram_prep);
        // (a layer call's Frame Cache: the compaction as well)
        const bool fcomp = fsel && frame_compact;
        HIP_TRY(launch_frame_stage(p, L, x, w, fm, fi, fsel ? at<int32_t>(ws, L.flag) : nullptr,
                                   fsel ? at<int32_t>(ws, L.mtok) : nullptr,
                                   gram_prep ? at<float>(ws, L.inv) : nullptr, gram_prep ? pack : nullptr, n_pack,
                                   cvt ? wo : nullptr, cvt ? wo16 : nullptr,
                                   fcomp ? at<int32_t>(ws, L.kept) : nullptr,
                                   fcomp ? at<int32_t>(ws, L.cached) : nullptr,
                                   fcomp ? at<int32_t>(ws, L.rmap) : nullptr, st),
                "frame stage");
    }
    if (p.kind == KIND_FRAME) return OC_OK;
    if (p.kind == KIND_FPATCH)
        HIP_TRY(launch_tile_norm(p, x, at<float>(ws, L.inv), pack, n_pack, wo, wo16, (long)p.C * p.hd, st),
                "tile norms");
    else if (!gram_prep)
        HIP_TRY(launch_inv_norm(p, x, at<float>(ws, L.inv), pack, n_pack, wo, wo16, (long)p.C * p.hd, st),
                "inv_norm");
    HIP_TRY(launch_match(p, x, at<float>(ws, L.inv), units_of(p, L, ws), pack, at<float>(ws, L.mpart),
                         reduce ? node_max : nullptr,
                         reduce ? node_idx : nullptr, st),
            "match");
    return OC_OK;
}

// Selection and compaction.  from_pack: unpack the similarity arg-max in
// the selection kernel (writing node_max / node_idx too), and compact there
// as well when every frame is one group.
// Whether a layer call's selection launch converts wo (the packed selection
// runs on one CU per group, the rest of the chip is idle); otherwise the
// first launch of the match stage does.
bool select_converts_wo(const Plan &p) {
    return p.bf16 && p.kind != KIND_FRAME && !(p.gran == OC_GRAN_FRAME_TOKEN && gram_norms(p));
}

oc_status run_select(const Plan &p, const Layout &L, float *node_max, int32_t *node_idx, bool from_pack,
                     int32_t *kept, int32_t *cached, int32_t *rmap, int map_matched, void *ws, hipStream_t st,
                     const void *x = nullptr, const void *wo = nullptr, void *wo16 = nullptr) {
    const int32_t *units = units_of(p, L, ws);
    if (from_pack && p.kind != KIND_FRAME) {
        const bool fused = select_compacts(p);
        // the per-token flags and matches stay in the workspace only where
        // something reads them: the separate compaction, or the cold
        // "matched" mapping after the fused one
        const bool flags = !fused || map_matched;
        HIP_TRY(launch_select_packed(p, units, at<unsigned long long>(ws, L.node_pack), at<float>(ws, L.inv),
                                     node_max, node_idx, flags ? at<int32_t>(ws, L.flag) : nullptr,
                                     flags ? at<int32_t>(ws, L.mtok) : nullptr, fused ? kept : nullptr,
                                     fused ? cached : nullptr, fused ? rmap : nullptr, st, nullptr, p.k2 > 0 ? 1 : 0,
                                     wo, wo16, (long)p.C * p.hd),
                "select");
        if (fused) {
            if (map_matched)
                HIP_TRY(launch_map_matched(p, at<int32_t>(ws, L.flag), at<int32_t>(ws, L.mtok), rmap, st),
                        "map matched");
            return OC_OK;
        }
        if (p.k2 > 0) {
            // second, coarser level (§3.3): similarity over the coarse
            // patches, then the selection among the candidates the first
            // level left (its flags exclude the rest and stay as they are)
            if (!x) return fail(OC_ERR_INVALID_ARG, "internal: the coarse level needs x");
            const Plan q = coarse_plan(p);
            // (the first level's selection left the packed arg-max zeroed:
            // both levels cover the same number of candidate slots)
            unsigned long long *pack = at<unsigned long long>(ws, L.node_pack);
            int32_t *flag = at<int32_t>(ws, L.flag);
            HIP_TRY(launch_match(q, x, at<float>(ws, L.inv), units, pack, at<float>(ws, L.mpart), nullptr, nullptr,
                                 st),
                    "coarse match");
            HIP_TRY(launch_select_packed(q, units, pack, at<float>(ws, L.inv), nullptr, nullptr, flag,
                                         at<int32_t>(ws, L.mtok), nullptr, nullptr, nullptr, st, flag),
                    "coarse select");
        }
    } else if (!(from_pack && p.kind == KIND_FRAME)) {
        HIP_TRY(launch_select(p, units, node_max, node_idx, at<int32_t>(ws, L.flag), at<int32_t>(ws, L.mtok), st),
                "select");
    } else {
        // Frame Cache in a layer call: the frame stage wrote the selection
        // and the compaction
        if (map_matched)
            HIP_TRY(launch_map_matched(p, at<int32_t>(ws, L.flag), at<int32_t>(ws, L.mtok), rmap, st),
                    "map matched");
        return OC_OK;
    }
    if (p.kind == KIND_FPATCH) {
        HIP_TRY(launch_compact_fpatch(p, at<int32_t>(ws, L.flag), at<int32_t>(ws, L.mtok), kept, cached, rmap,
                                      at<int32_t>(ws, L.seqoff), map_matched, st),
                "compact");
        return OC_OK;
    }
    HIP_TRY(launch_compact(p, at<int32_t>(ws, L.units), at<int32_t>(ws, L.flag), at<int32_t>(ws, L.mtok),
                           at<int32_t>(ws, L.fcnt), kept, cached, rmap, map_matched, st),
            "compact");
    return OC_OK;
}

oc_status check_weights(const oc_attn_weights *w) {
    if (!w || !w->wq || !w->wk || !w->wv || !w->wo) return fail(OC_ERR_INVALID_ARG, "weights NULL");
    if (!aligned16(w->wq) || !aligned16(w->wk) || !aligned16(w->wv) || !aligned16(w->wo))
        return fail(OC_ERR_INVALID_ARG, "weights must be 16-byte aligned");
    return OC_OK;
}

oc_status copy_d2d(void *dst, const void *src, size_t bytes, hipStream_t st) {
    if (!dst || bytes == 0) return OC_OK;
    HIP_TRY(hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToDevice, st), "trace copy");
    return OC_OK;
}

}  // namespace

namespace oc {
// Status and message for the host-only entry points in other sources.
oc_status record_error(oc_status s, const char *msg) {
    if (s == OC_OK) return ok();
    return fail(s, "%s", msg);
}
}  // namespace oc

extern "C" {

const char *oc_status_string(oc_status s) {
    switch (s) {
        case OC_OK: return "OC_OK";
        case OC_ERR_INVALID_ARG: return "OC_ERR_INVALID_ARG";
        case OC_ERR_SHAPE: return "OC_ERR_SHAPE";
        case OC_ERR_DTYPE: return "OC_ERR_DTYPE";
        case OC_ERR_WORKSPACE: return "OC_ERR_WORKSPACE";
        case OC_ERR_CACHE_STATE: return "OC_ERR_CACHE_STATE";
        case OC_ERR_HIP: return "OC_ERR_HIP";
    }
    return "unknown oc_status";
}

const char *oc_last_error(void) { return g_err.c_str(); }

oc_status oc_plan(const oc_shape *shape, const oc_cfg *cfg, oc_plan_info *out) {
    if (!out) return fail(OC_ERR_INVALID_ARG, "out is NULL");
    Plan p;
    oc_status s = make_plan(shape, cfg, false, p);
    if (s != OC_OK) return s;
    out->n_groups = p.n_groups;
    out->n_src_max = p.n_src_max;
    out->n_dst_max = p.n_dst_max;
    out->n_frame_src = p.n_fsrc;
    out->n_frame_dst = p.n_fdst;
    out->n_frame_cached = p.R_f;
    out->n_kept = p.n_kept;
    out->n_cached = p.n_cached;
    out->n_seq = p.n_seq;
    out->seq_len = p.seq_len;
    out->workspace_bytes = workspace_for(shape, cfg);
    return ok();
}

size_t oc_attn_workspace_bytes(const oc_shape *shape, int32_t n_seq, int32_t seq_len) {
    if (check_shape(shape) != OC_OK || n_seq < 0 || seq_len < 0) return 0;
    Plan p;
    std::memset(&p, 0, sizeof(p));
    p.C = shape->C; p.heads = shape->heads; p.dh = shape->head_dim; p.hd = p.heads * p.dh;
    p.n_ctx = shape->n_ctx; p.bf16 = shape->dtype == OC_BF16; p.esz = p.bf16 ? 2 : 4;
    return attn_ws(p, n_seq, seq_len, 0).bytes;
}

oc_status oc_match(const oc_shape *shape, const oc_cfg *cfg, const void *x, float *node_max, int32_t *node_idx,
                   oc_frame_info *frames, void *ws, size_t ws_bytes, hipStream_t stream) {
    Plan p;
    oc_status s = make_plan(shape, cfg, false, p);
    if (s != OC_OK) return s;
    if (p.k2 > 0)
        return fail(OC_ERR_INVALID_ARG, "the two-level hierarchy (coarse_k > 0) runs in oc_layer_cached only");
    if (!x || !node_max || !node_idx) return fail(OC_ERR_INVALID_ARG, "NULL pointer");
    if (!aligned16(x)) return fail(OC_ERR_INVALID_ARG, "x must be 16-byte aligned");
    const Layout L = make_layout(p);
    if ((s = check_ws(ws, ws_bytes, workspace_for(shape, cfg))) != OC_OK) return s;
    if ((s = run_match(p, L, x, node_max, node_idx, true, ws, stream)) != OC_OK) return s;
    if (frames && p.gran == OC_GRAN_FRAME_TOKEN) {
        if ((s = copy_d2d(frames->frame_max, at<float>(ws, L.fmax), (size_t)p.n_fsrc * 4, stream)) != OC_OK) return s;
        if ((s = copy_d2d(frames->frame_idx, at<int32_t>(ws, L.fidx), (size_t)p.n_fsrc * 4, stream)) != OC_OK) return s;
        if ((s = copy_d2d(frames->pairs, at<int32_t>(ws, L.pairs), (size_t)p.R_f * 8, stream)) != OC_OK) return s;
    }
    return ok();
}

oc_status oc_select(const oc_shape *shape, const oc_cfg *cfg, const float *node_max, const int32_t *node_idx,
                    int32_t *kept_idx, int32_t *cached_idx, int32_t *restore_map, int32_t map_matched, void *ws,
                    size_t ws_bytes, hipStream_t stream) {
    Plan p;
    oc_status s = make_plan(shape, cfg, false, p);
    if (s != OC_OK) return s;
    if (p.k2 > 0)
        return fail(OC_ERR_INVALID_ARG, "the two-level hierarchy (coarse_k > 0) runs in oc_layer_cached only");
    if (!node_max || !node_idx || !kept_idx || !cached_idx || !restore_map)
        return fail(OC_ERR_INVALID_ARG, "NULL pointer");
    if (map_matched != 0 && map_matched != 1) return fail(OC_ERR_INVALID_ARG, "map_matched must be 0 or 1");
    const Layout L = make_layout(p);
    if ((s = check_ws(ws, ws_bytes, workspace_for(shape, cfg))) != OC_OK) return s;
    // FRAME_TOKEN groups follow the unit table oc_match left in ws
    if ((s = run_select(p, L, const_cast<float *>(node_max), const_cast<int32_t *>(node_idx), false, kept_idx,
                        cached_idx, restore_map, map_matched, ws, stream)) != OC_OK)
        return s;
    return ok();
}

oc_status oc_gather(const oc_shape *shape, const oc_cfg *cfg, const void *x, const int32_t *kept_idx, void *x_kept,
                    hipStream_t stream) {
    Plan p;
    oc_status s = make_plan(shape, cfg, false, p);
    if (s != OC_OK) return s;
    if (!x || !kept_idx || !x_kept) return fail(OC_ERR_INVALID_ARG, "NULL pointer");
    if (!aligned16(x) || !aligned16(x_kept)) return fail(OC_ERR_INVALID_ARG, "x / x_kept must be 16-byte aligned");
    if (x == x_kept) return fail(OC_ERR_INVALID_ARG, "x_kept must not alias x");
    HIP_TRY(launch_gather(p, x, kept_idx, p.n_kept, x_kept, stream), "gather");
    return ok();
}

oc_status oc_attn_reduced(const oc_shape *shape, const void *x_kept, int32_t n_seq, int32_t seq_len, const void *ctx,
                          const oc_attn_weights *w, void *y_kept, void *y_ctx, void *ws, size_t ws_bytes,
                          hipStream_t stream) {
    oc_status s = check_shape(shape);
    if (s != OC_OK) return s;
    if (n_seq < 0 || seq_len < 0) return fail(OC_ERR_SHAPE, "n_seq and seq_len must be >= 0");
    if ((long long)n_seq * seq_len + shape->n_ctx >= (1LL << 30)) return fail(OC_ERR_SHAPE, "batch too large");
    if (shape->n_ctx > 0 && n_seq != 1) return fail(OC_ERR_SHAPE, "context tokens need exactly one sequence");
    if ((s = check_weights(w)) != OC_OK) return s;
    const long rows = (long)n_seq * seq_len;
    if (rows > 0 && (!x_kept || !y_kept)) return fail(OC_ERR_INVALID_ARG, "NULL x_kept / y_kept");
    if (shape->n_ctx > 0 && (!ctx || !y_ctx)) return fail(OC_ERR_INVALID_ARG, "NULL ctx / y_ctx");
    if ((x_kept && !aligned16(x_kept)) || (y_kept && !aligned16(y_kept)) || (ctx && !aligned16(ctx)) ||
        (y_ctx && !aligned16(y_ctx)))
        return fail(OC_ERR_INVALID_ARG, "buffers must be 16-byte aligned");
    Plan p;
    std::memset(&p, 0, sizeof(p));
    p.F = shape->F; p.H = shape->H; p.W = shape->W; p.N = p.H * p.W;
    p.C = shape->C; p.heads = shape->heads; p.dh = shape->head_dim; p.hd = p.heads * p.dh;
    p.n_ctx = shape->n_ctx; p.bf16 = shape->dtype == OC_BF16; p.esz = p.bf16 ? 2 : 4;
    const AttnWs aw = attn_ws(p, n_seq, seq_len, 0);
    if ((s = check_ws(ws, ws_bytes, aw.bytes)) != OC_OK) return s;
    if (rows + shape->n_ctx == 0) return ok();
    AttnArgs a;
    std::memset(&a, 0, sizeof(a));
    a.x = x_kept; a.row_idx = nullptr; a.n_main = (int)rows;
    a.ctx = shape->n_ctx > 0 ? ctx : nullptr; a.n_ctx = shape->n_ctx;
    a.n_seq = n_seq; a.L = seq_len;
    a.wq = w->wq; a.wk = w->wk; a.wv = w->wv; a.wo = w->wo;
    a.y = y_kept; a.out_idx = nullptr; a.y_ctx = y_ctx;
    a.q = at<char>(ws, aw.q); a.k = at<char>(ws, aw.k); a.o = at<char>(ws, aw.o); a.vt = at<char>(ws, aw.v);
    a.lpad = aw.lpad;
    a.wo16 = at<char>(ws, aw.wo16);
    HIP_TRY(launch_attention(p, a, stream), "attention");
    return ok();
}

oc_status oc_restore(const oc_shape *shape, const void *y_kept, int32_t n_rows, const int32_t *restore_map,
                     const void *cache_y, void *y, hipStream_t stream) {
    oc_status s = check_shape(shape);
    if (s != OC_OK) return s;
    if (!restore_map || !y || (n_rows > 0 && !y_kept)) return fail(OC_ERR_INVALID_ARG, "NULL pointer");
    if (n_rows < 0) return fail(OC_ERR_INVALID_ARG, "n_rows < 0");
    if (!aligned16(y) || (y_kept && !aligned16(y_kept)) || (cache_y && !aligned16(cache_y)))
        return fail(OC_ERR_INVALID_ARG, "buffers must be 16-byte aligned");
    Plan p;
    std::memset(&p, 0, sizeof(p));
    p.F = shape->F; p.N = shape->H * shape->W; p.C = shape->C; p.esz = shape->dtype == OC_BF16 ? 2 : 4;
    HIP_TRY(launch_restore(p, y_kept, n_rows, restore_map, cache_y, y, stream), "restore");
    return ok();
}

oc_status oc_layer_cached(const oc_shape *shape, const oc_cfg *cfg, const void *x, const void *ctx,
                          const oc_attn_weights *w, oc_cache *cache, void *y_ctx, oc_trace *trace, void *ws,
                          size_t ws_bytes, hipStream_t stream) {
    oc_status s = check_shape(shape);
    if (s != OC_OK) return s;
    if ((s = check_cfg(cfg)) != OC_OK) return s;
    if (!cache || !cache->y) return fail(OC_ERR_CACHE_STATE, "cache or cache->y is NULL");
    if (cache->valid != 0 && cache->valid != 1) return fail(OC_ERR_CACHE_STATE, "cache->valid must be 0 or 1");
    const bool cold = cache->valid == 0;
    Plan p;
    if ((s = make_plan(shape, cfg, cold && cfg->cold == OC_COLD_FULL, p)) != OC_OK) return s;
    if (!x) return fail(OC_ERR_INVALID_ARG, "x is NULL");
    if ((s = check_weights(w)) != OC_OK) return s;
    if (shape->n_ctx > 0 && (!ctx || !y_ctx)) return fail(OC_ERR_INVALID_ARG, "NULL ctx / y_ctx");
    if (!aligned16(x) || !aligned16(cache->y) || (ctx && !aligned16(ctx)) || (y_ctx && !aligned16(y_ctx)))
        return fail(OC_ERR_INVALID_ARG, "buffers must be 16-byte aligned");
    if (x == cache->y) return fail(OC_ERR_INVALID_ARG, "x must not alias cache->y");
    const Layout L = make_layout(p);
    if ((s = check_ws(ws, ws_bytes, workspace_for(shape, cfg))) != OC_OK) return s;
    const int map_matched = cold ? 1 : 0;

    float *nm = at<float>(ws, L.node_max);
    int32_t *ni = at<int32_t>(ws, L.node_idx);
    const AttnWs aw = attn_ws(p, p.n_seq, p.seq_len, L.attn);
    // bf16 layers: the fp16 copy of wo is made beside the selection, or by
    // the first launch of the match stage
    const bool wo_early = p.bf16;
    const bool wo_sel = select_converts_wo(p);
    if ((s = run_match(p, L, x, nm, ni, false, ws, stream, wo_early && !wo_sel ? w->wo : nullptr,
                       wo_early && !wo_sel ? at<char>(ws, aw.wo16) : nullptr, true)) != OC_OK)
        return s;
    int32_t *kept = at<int32_t>(ws, L.kept), *cached = at<int32_t>(ws, L.cached), *rmap = at<int32_t>(ws, L.rmap);
    if ((s = run_select(p, L, nm, ni, true, kept, cached, rmap, map_matched, ws, stream, x, wo_sel ? w->wo : nullptr,
                        wo_sel ? at<char>(ws, aw.wo16) : nullptr)) != OC_OK)
        return s;

    AttnArgs a;
    std::memset(&a, 0, sizeof(a));
    a.x = x; a.row_idx = kept; a.n_main = p.n_kept;
    a.ctx = shape->n_ctx > 0 ? ctx : nullptr; a.n_ctx = shape->n_ctx;
    a.n_seq = p.n_seq; a.L = p.seq_len;
    a.wq = w->wq; a.wk = w->wk; a.wv = w->wv; a.wo = w->wo;
    a.y = cache->y; a.out_idx = kept; a.y_ctx = y_ctx;
    a.q = at<char>(ws, aw.q); a.k = at<char>(ws, aw.k); a.o = at<char>(ws, aw.o); a.vt = at<char>(ws, aw.v);
    a.lpad = aw.lpad;
    a.wo16 = at<char>(ws, aw.wo16);
    a.wo16_ready = wo_early ? 1 : 0;
    a.seq_off = p.kind == KIND_FPATCH ? at<int32_t>(ws, L.seqoff) : nullptr;
    HIP_TRY(launch_attention(p, a, stream), "attention");
    if (map_matched) HIP_TRY(launch_copy_matched(p, cached, p.n_cached, rmap, kept, cache->y, stream), "copy matched");

    if (trace) {
        const size_t GS = (size_t)p.n_groups * p.n_src_max * 4;
        if ((s = copy_d2d(trace->node_max, nm, GS, stream)) != OC_OK) return s;
        if ((s = copy_d2d(trace->node_idx, ni, GS, stream)) != OC_OK) return s;
        if ((s = copy_d2d(trace->kept_idx, kept, (size_t)p.n_kept * 4, stream)) != OC_OK) return s;
        if ((s = copy_d2d(trace->cached_idx, cached, (size_t)p.n_cached * 4, stream)) != OC_OK) return s;
        if ((s = copy_d2d(trace->restore_map, rmap, (size_t)p.F * p.N * 4, stream)) != OC_OK) return s;
        if (p.gran == OC_GRAN_FRAME_TOKEN) {
            if ((s = copy_d2d(trace->frames.frame_max, at<float>(ws, L.fmax), (size_t)p.n_fsrc * 4, stream)) != OC_OK) return s;
            if ((s = copy_d2d(trace->frames.frame_idx, at<int32_t>(ws, L.fidx), (size_t)p.n_fsrc * 4, stream)) != OC_OK) return s;
            if ((s = copy_d2d(trace->frames.pairs, at<int32_t>(ws, L.pairs), (size_t)p.R_f * 8, stream)) != OC_OK) return s;
        }
    }
    cache->valid = 1;
    cache->step += 1;
    return ok();
}

size_t oc_ffn_workspace_bytes(const oc_shape *shape, int32_t hidden, int32_t n_rows) {
    if (check_shape(shape) != OC_OK || hidden < 0 || n_rows < 0) return 0;
    return ffn_workspace_bytes(n_rows, hidden, shape->C);
}

oc_status oc_ffn_reduced(const oc_shape *shape, const void *x, const int32_t *kept_idx, int32_t n_rows,
                         const oc_ffn_weights *w, void *y, int32_t scatter, void *ws, size_t ws_bytes,
                         hipStream_t stream) {
    oc_status s = check_shape(shape);
    if (s != OC_OK) return s;
    if (shape->dtype != OC_BF16) return fail(OC_ERR_DTYPE, "the feed-forward path takes bf16 tensors only");
    if (!w || !w->w1 || !w->w2) return fail(OC_ERR_INVALID_ARG, "weights NULL");
    if (w->reserved != 0) return fail(OC_ERR_INVALID_ARG, "oc_ffn_weights.reserved must be 0");
    if (w->hidden < 64 || w->hidden % 64 || shape->C % 64)
        return fail(OC_ERR_SHAPE, "feed-forward needs C=%d and hidden=%d to be positive multiples of 64", shape->C,
                    w->hidden);
    const long long FN = (long long)shape->F * shape->H * shape->W;
    if (n_rows < 0 || n_rows > FN) return fail(OC_ERR_SHAPE, "n_rows=%d outside [0, F*N=%lld]", n_rows, FN);
    if ((long long)w->hidden * shape->C >= (1LL << 31) || (long long)n_rows * w->hidden >= (1LL << 31))
        return fail(OC_ERR_SHAPE, "feed-forward too large for 32-bit element offsets");
    if (scatter != 0 && scatter != 1) return fail(OC_ERR_INVALID_ARG, "scatter must be 0 or 1");
    if (!x || !y) return fail(OC_ERR_INVALID_ARG, "NULL x / y");
    if (!aligned16(x) || !aligned16(y) || !aligned16(w->w1) || !aligned16(w->w2))
        return fail(OC_ERR_INVALID_ARG, "x, y and the weights must be 16-byte aligned");
    if (x == y) return fail(OC_ERR_INVALID_ARG, "y must not alias x");
    if ((s = check_ws(ws, ws_bytes, ffn_workspace_bytes(n_rows, w->hidden, shape->C))) != OC_OK) return s;
    if (n_rows == 0) return ok();
    FfnArgs a;
    std::memset(&a, 0, sizeof(a));
    a.x = x; a.idx = kept_idx; a.n_rows = n_rows; a.FN = (int)FN; a.C = shape->C; a.hidden = w->hidden;
    a.w1 = w->w1; a.w2 = w->w2; a.h = ws;
    a.scatter = scatter;
    a.y = y;
    HIP_TRY(launch_ffn(a, stream), "feed-forward");
    return ok();
}

oc_status oc_residual_add(const oc_shape *shape, const void *x, const void *y, void *h, hipStream_t stream) {
    oc_status s = check_shape(shape);
    if (s != OC_OK) return s;
    if (!x || !y || !h) return fail(OC_ERR_INVALID_ARG, "NULL pointer");
    if (!aligned16(x) || !aligned16(y) || !aligned16(h)) return fail(OC_ERR_INVALID_ARG, "buffers must be 16-byte aligned");
    Plan p;
    std::memset(&p, 0, sizeof(p));
    p.F = shape->F; p.N = shape->H * shape->W; p.C = shape->C; p.bf16 = shape->dtype == OC_BF16;
    HIP_TRY(launch_add(p, x, y, h, stream), "residual add");
    return ok();
}

oc_status oc_block_cached(const oc_shape *shape, const oc_cfg *spatial, const oc_cfg *temporal, const void *x,
                          const oc_attn_weights *w_spatial, const oc_attn_weights *w_temporal, oc_cache *cache_spatial,
                          oc_cache *cache_temporal, void *h, oc_trace *trace_spatial, oc_trace *trace_temporal,
                          void *ws, size_t ws_bytes, hipStream_t stream) {
    // everything is validated before the first launch
    Plan ps, pt;
    oc_status s;
    if ((s = make_plan(shape, spatial, false, ps)) != OC_OK) return s;
    if ((s = make_plan(shape, temporal, false, pt)) != OC_OK) return s;
    if (spatial->gran == OC_GRAN_BLOCK) return fail(OC_ERR_INVALID_ARG, "the spatial layer's cache cannot be BLOCK");
    if (temporal->gran != OC_GRAN_BLOCK) return fail(OC_ERR_INVALID_ARG, "the temporal layer's cache must be BLOCK");
    if (shape->n_ctx != 0) return fail(OC_ERR_SHAPE, "a spatial+temporal block takes no context tokens");
    if (!x || !h) return fail(OC_ERR_INVALID_ARG, "NULL x / h");
    if ((s = check_weights(w_spatial)) != OC_OK || (s = check_weights(w_temporal)) != OC_OK) return s;
    for (const oc_cache *c : {cache_spatial, cache_temporal}) {
        if (!c || !c->y) return fail(OC_ERR_CACHE_STATE, "cache or cache->y is NULL");
        if (c->valid != 0 && c->valid != 1) return fail(OC_ERR_CACHE_STATE, "cache->valid must be 0 or 1");
    }
    if (!aligned16(x) || !aligned16(h) || !aligned16(cache_spatial->y) || !aligned16(cache_temporal->y))
        return fail(OC_ERR_INVALID_ARG, "buffers must be 16-byte aligned");
    const void *bufs[4] = {x, h, cache_spatial->y, cache_temporal->y};
    for (int i = 0; i < 4; ++i)
        for (int j = i + 1; j < 4; ++j)
            if (bufs[i] == bufs[j]) return fail(OC_ERR_INVALID_ARG, "x, h and the two caches must be distinct buffers");
    const size_t need_s = workspace_for(shape, spatial), need_t = workspace_for(shape, temporal);
    if ((s = check_ws(ws, ws_bytes, need_s > need_t ? need_s : need_t)) != OC_OK) return s;
    if ((s = oc_layer_cached(shape, spatial, x, nullptr, w_spatial, cache_spatial, nullptr, trace_spatial, ws, ws_bytes,
                             stream)) != OC_OK)
        return s;
    if ((s = oc_residual_add(shape, x, cache_spatial->y, h, stream)) != OC_OK) return s;
    return oc_layer_cached(shape, temporal, h, nullptr, w_temporal, cache_temporal, nullptr, trace_temporal, ws,
                           ws_bytes, stream);
}

size_t oc_block_workspace_bytes(const oc_shape *shape, const oc_cfg *spatial, const oc_cfg *temporal) {
    const size_t a = workspace_for(shape, spatial), b = workspace_for(shape, temporal);
    return a > b ? a : b;
}

oc_status oc_layer_cached_static(const oc_shape *shape, const oc_cfg *cfg, const void *x, const void *ctx,
                                 const oc_attn_weights *w, oc_cache *cache, void *y_ctx, oc_trace *trace,
                                 hipStream_t stream) {
    Plan p;
    oc_status s = make_plan(shape, cfg, false, p);
    if (s != OC_OK) return s;
    const size_t need = workspace_for(shape, cfg);
    if (need > OC_STATIC_SCRATCH_BYTES)
        return fail(OC_ERR_WORKSPACE,
                    "this layer needs %zu bytes of scratch, more than the library's static scratch of %zu bytes: "
                    "call oc_layer_cached with a workspace instead",
                    need, (size_t)OC_STATIC_SCRATCH_BYTES);
    void *ws = nullptr;
    HIP_TRY(static_scratch(&ws), "static scratch address");
    return oc_layer_cached(shape, cfg, x, ctx, w, cache, y_ctx, trace, ws, OC_STATIC_SCRATCH_BYTES, stream);
}

size_t oc_static_scratch_bytes(void) { return OC_STATIC_SCRATCH_BYTES; }

oc_status oc_attn_full(const oc_shape *shape, const oc_cfg *cfg, const void *x, const void *ctx,
                       const oc_attn_weights *w, void *y, void *y_ctx, void *ws, size_t ws_bytes,
                       hipStream_t stream) {
    Plan p0;
    oc_status s = make_plan(shape, cfg, true, p0);
    if (s != OC_OK) return s;
    if (!x || !y) return fail(OC_ERR_INVALID_ARG, "NULL pointer");
    if ((s = check_weights(w)) != OC_OK) return s;
    if (shape->n_ctx > 0 && (!ctx || !y_ctx)) return fail(OC_ERR_INVALID_ARG, "NULL ctx / y_ctx");
    if (!aligned16(x) || !aligned16(y) || (ctx && !aligned16(ctx)) || (y_ctx && !aligned16(y_ctx)))
        return fail(OC_ERR_INVALID_ARG, "buffers must be 16-byte aligned");
    if (x == y) return fail(OC_ERR_INVALID_ARG, "y must not alias x");
    const Plan p = full_plan(p0);
    const Layout L = make_layout(p0);
    if ((s = check_ws(ws, ws_bytes, workspace_for(shape, cfg))) != OC_OK) return s;
    // no index lists: spatial layers keep every token in place, temporal
    // layers take one sequence per position (row n*F + f is token f*N + n)
    const bool temporal = p.kind == KIND_BLOCK;
    const AttnWs aw = attn_ws(p, p.n_seq, p.seq_len, L.attn);
    AttnArgs a;
    std::memset(&a, 0, sizeof(a));
    a.tF = temporal ? p.F : 0;
    a.tN = p.N;
    a.x = x; a.row_idx = nullptr; a.n_main = p.n_kept;
    a.ctx = shape->n_ctx > 0 ? ctx : nullptr; a.n_ctx = shape->n_ctx;
    a.n_seq = p.n_seq; a.L = p.seq_len;
    a.wq = w->wq; a.wk = w->wk; a.wv = w->wv; a.wo = w->wo;
    a.y = y; a.out_idx = nullptr; a.y_ctx = y_ctx;
    a.q = at<char>(ws, aw.q); a.k = at<char>(ws, aw.k); a.o = at<char>(ws, aw.o); a.vt = at<char>(ws, aw.v);
    a.lpad = aw.lpad;
    a.wo16 = at<char>(ws, aw.wo16);
    HIP_TRY(launch_attention(p, a, stream), "attention");
    return ok();
}

}  // extern "C"
