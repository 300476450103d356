// Matching groups as a pure function of the plan (and, for the frame-token
// granularity, the unit table the frame stage wrote): the global ids of a
// group's candidates and representatives (OmniCache §3.2.1-§3.2.3, patch-local
// groups per §3.3).  Computed where they are used instead of materialised.
//
// Unit u covers frame s (and frame d for a frame pair, d = -1 otherwise);
// group g = u * k*k + patch.  Candidates are listed in ascending global id:
// the non-representative tokens of the unit's frame, or for a pair all
// tokens of both frames except the representatives of frame d.
// Representatives are the top-left tokens of the 2x2 windows (of frame d for
// a pair), ascending.  Block groups use spatial positions as ids (no frame
// term).  Frame groups: odd frames are candidates, even frames
// representatives.  Frame-patch groups (one per patch): the odd frames'
// tiles of the patch are candidates, the even frames' tiles representatives,
// each tile named by its top-left token id.
#pragma once
#include "oc_internal.h"

namespace oc {

struct GroupMap {
    int kind, F, N, W, k, ph, pw, np, np_src, np_dst, R_tok, R_pair, R_f;
    const int32_t *units;   // frame-token unit table (s, d) per unit, or nullptr

    struct Grp {
        int s, d, a, b, n_a, nsrc, oy, ox, rf, R;
        bool pair;
        long fbase;
    };

    __device__ __forceinline__ Grp group(int g) const {
        Grp r;
        if (kind == KIND_FPATCH) {
            // patch g: its frames' tiles, named by their top-left tokens
            r.s = r.d = r.a = r.b = r.rf = 0;
            r.n_a = 0;
            r.oy = (g / k) * ph;
            r.ox = (g % k) * pw;
            r.nsrc = F / 2;
            r.pair = false;
            r.fbase = N;
            r.R = R_f;
            return r;
        }
        if (kind == KIND_FRAME) {
            r.s = r.d = r.a = r.b = r.rf = r.oy = r.ox = 0;
            r.n_a = 0;
            r.nsrc = F / 2;
            r.pair = false;
            r.fbase = 0;
            r.R = R_f;
            return r;
        }
        const int kk = k * k;
        const int u = g / kk, patch = g - u * kk;
        r.oy = (patch / k) * ph;
        r.ox = (patch % k) * pw;
        int s = u, d = -1;
        if (units != nullptr) {
            s = units[2 * u];
            d = units[2 * u + 1];
            if (s < 0 || s >= F || d >= F || s == d) { s = 0; d = -1; }   // malformed unit table
        }
        r.s = s;
        r.d = d;
        r.pair = d >= 0;
        r.fbase = kind == KIND_BLOCK ? 0 : (long)N;
        r.a = r.pair ? min(s, d) : s;
        r.b = r.pair ? max(s, d) : -1;
        r.n_a = (r.pair && r.a == d) ? np_src : np;
        r.nsrc = r.pair ? np + np_src : np_src;
        r.rf = r.pair ? d : s;
        r.R = r.pair ? R_pair : R_tok;
        return r;
    }

    // i-th token of a patch, row-major
    __device__ __forceinline__ void patch_tok(int i, int &y, int &x) const { y = i / pw; x = i - y * pw; }
    // i-th non-representative token of a patch (ascending id)
    __device__ __forceinline__ void patch_nonrep(int i, int &y, int &x) const {
        const int per2 = 3 * pw / 2, q = i / per2, rem = i - q * per2;
        if (rem < pw / 2) { y = 2 * q; x = 2 * rem + 1; }
        else { y = 2 * q + 1; x = rem - pw / 2; }
    }
    // i-th representative of a patch
    __device__ __forceinline__ void patch_rep(int i, int &y, int &x) const {
        const int h = pw / 2, q = i / h;
        y = 2 * q;
        x = 2 * (i - q * h);
    }

    // global id of candidate i of the group, -1 past its end
    __device__ __forceinline__ int src_id(const Grp &r, int i) const {
        if (i < 0 || i >= r.nsrc) return -1;
        if (kind == KIND_FRAME) return 2 * i + 1;
        if (kind == KIND_FPATCH) return (int)((2 * i + 1) * r.fbase + (long)r.oy * W + r.ox);
        int f, y, x;
        if (!r.pair) { f = r.s; patch_nonrep(i, y, x); }
        else if (i < r.n_a) {
            f = r.a;
            if (r.a == r.d) patch_nonrep(i, y, x); else patch_tok(i, y, x);
        } else {
            f = r.b;
            const int j = i - r.n_a;
            if (r.b == r.d) patch_nonrep(j, y, x); else patch_tok(j, y, x);
        }
        return (int)(f * r.fbase + (long)(r.oy + y) * W + (r.ox + x));
    }

    // global id of representative i of the group, -1 past its end
    __device__ __forceinline__ int dst_id(const Grp &r, int i) const {
        if (kind == KIND_FRAME) return (i >= 0 && 2 * i < F) ? 2 * i : -1;
        if (kind == KIND_FPATCH) return (i >= 0 && 2 * i < F) ? (int)(2 * i * r.fbase + (long)r.oy * W + r.ox) : -1;
        if (i < 0 || i >= np_dst) return -1;
        int y, x;
        patch_rep(i, y, x);
        return (int)(r.rf * r.fbase + (long)(r.oy + y) * W + (r.ox + x));
    }
};

inline GroupMap group_map(const Plan &p, const int32_t *units) {
    GroupMap m;
    m.kind = p.kind; m.F = p.F; m.N = p.N; m.W = p.W; m.k = p.k; m.ph = p.ph; m.pw = p.pw; m.np = p.np;
    m.np_src = p.np_src; m.np_dst = p.np_dst; m.R_tok = p.R_tok; m.R_pair = p.R_pair; m.R_f = p.R_f;
    m.units = units;
    return m;
}

}  // namespace oc
