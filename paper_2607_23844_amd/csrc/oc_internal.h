// Internal plan and kernel-launcher declarations of the OmniCache library.
// Host code (oc_api.cpp) validates, plans and carves the workspace; the
// launchers below enqueue gfx950 kernels on the caller's stream.
#pragma once
#include <cstddef>
#include <cstdint>
#include <hip/hip_runtime_api.h>

namespace oc {

// KIND_FPATCH: Frame Cache on k x k patches (k > 1): one group per patch, its
// items the frames' tiles of that patch, named by their top-left token id.
enum Kind { KIND_TOKEN = 0, KIND_BLOCK = 1, KIND_FRAME = 2, KIND_FPATCH = 3 };

// Static sizes of one call; everything depends only on shape and cfg.
struct Plan {
    int F, H, W, C, N, heads, dh, hd, n_ctx;
    bool bf16;
    int esz;                 // bytes per element of x / weights
    int gran, k;             // granularity, patch_k
    int ph, pw, np;          // patch height, width, tokens per patch
    int np_src, np_dst;      // candidates / representatives per frame-patch (3/4, 1/4)
    double r, r_frame;
    // matching stage reported by oc_match
    int kind;                // KIND_TOKEN (token / pair groups), KIND_BLOCK, KIND_FRAME, KIND_FPATCH
    int n_groups, n_src_max, n_dst_max;
    int R_tok;               // budget of a token / block group (unmatched frame-patch)
    int R_pair;              // budget of a frame-pair patch group
    // frame stage (FRAME and FRAME_TOKEN)
    int n_fsrc, n_fdst, R_f;
    int n_units;             // attention units: frames (TOKEN), pairs + unmatched (FRAME_TOKEN)
    // reduced batch
    int n_kept, n_cached, n_seq, seq_len;   // KIND_FPATCH: n_seq = F sequences of at most seq_len = N
                                            // tokens each, of varying length (seq_off in the workspace)
    int n_items;             // matched items: F*N tokens, N blocks, F frames
    // second, coarser level of the hierarchy (§3.3), Token and Block Cache:
    // k2 = 0 none; else patches of k2 x k2 (k2 divides k), np2 items each,
    // R2 more of the candidates the first level left cached per patch
    int k2, np2, np2_src, np2_dst, R2;
    double r2;
};


// Workspace carve-up (byte offsets from the caller's ws base).
struct Layout {
    size_t inv, node_pack, node_max, node_idx, mpart;
    size_t gram_part, fgram, fsim, fmax, fidx, forder, pairs, units;
    size_t flag, mtok, fcnt, kept, cached, rmap;
    size_t seqoff;           // KIND_FPATCH: sequence offsets [F + 1]
    size_t attn;             // start of the attention workspace (Q, K, O, V)
    size_t total;
};

// Attention workspace carved at `base`: Q, K, O [rows, H*dh] and V
// (bf16: Vt [H][seq][dh][lpad]; fp32: [rows, H*dh]).
struct AttnWs { size_t q, k, o, v, wo16, bytes; int lpad; };
AttnWs attn_ws(const Plan &p, int n_seq, int L, size_t base);
int gram_blocks(const Plan &p);
// Whether the frame Gram launch also computes the token norms that token
// matching needs (Frame+Token Cache, bf16, C a multiple of 64), so that x is
// read once for both.
inline bool gram_norms(const Plan &p) { return p.bf16 && p.gran == 3 && p.C % 64 == 0; }

// Stage timing: while a timer is attached to the calling thread, the
// kernels launched (launch_k, oc_launch.h) inside a StageScope are timed
// under its name (oc_timer.cpp).
struct StageScope {
    StageScope(hipStream_t st, const char *name);
    ~StageScope();
    int prev;
};

// ---- launchers (k_*.hip) ---------------------------------------------------
// Group members are computed from the plan (GroupMap, oc_groups.h); units is
// the frame-token unit table in the workspace (nullptr for other kinds).
// node_pack [G, S] holds each candidate's best (similarity, representative
// position) packed for a 64-bit atomic maximum (pack_argmax).
// launch_inv_norm also clears node_pack (n_pack entries) and, with wo / wo16
// given, converts the output-projection weights wo (bf16, n_wo elements) to
// fp16 into wo16, all in one launch.
hipError_t launch_inv_norm(const Plan &p, const void *x, float *inv, unsigned long long *node_pack, long n_pack,
                           const void *wo, void *wo16, long n_wo, hipStream_t st);
// Similarity kernel choice (bf16): long descriptors over few 64x64 tiles
// (Block Cache) split K into n_split ranges of kc elements, each inside one
// segment of the descriptor, with fp32 partials [n_split][G][S][D] in the
// workspace; many candidate tiles with several representative tiles sweep
// the representatives per candidate tile; otherwise one block per tile pair.
struct MatchSplit { int n_split, kc; };
// Descriptor geometry of the matched items: item id i starts at element
// i * item_stride of x and is K elements long, read as segments of seg_len
// contiguous elements sub_stride apart (seg_len == 0: one contiguous run).
// Tokens: a C-vector; blocks: F segments of C, a frame apart; frame-patch
// tiles: ph segments of pw*C, an image row apart.
struct MatchGeom { int K, seg_len; long sub_stride, item_stride; };
inline MatchGeom match_geom(const Plan &p) {
    if (p.kind == KIND_BLOCK) return MatchGeom{p.F * p.C, p.C, (long)p.N * p.C, p.C};
    if (p.kind == KIND_FPATCH) return MatchGeom{p.ph * p.pw * p.C, p.pw * p.C, (long)p.W * p.C, p.C};
    return MatchGeom{p.C, 0, (long)p.N * p.C, p.C};
}
inline MatchSplit match_split(const Plan &p) {
    MatchSplit m{1, 0};
    if (!p.bf16 || p.kind == KIND_FRAME) return m;
    const MatchGeom mg = match_geom(p);
    const int K = mg.K;
    const int seg = mg.seg_len;
    if (K % 64 != 0 || (seg > 0 && seg % 64 != 0)) return m;
    const int nk = K / 64;
    const long tiles = (long)((p.n_src_max + 63) / 64) * ((p.n_dst_max + 63) / 64) * p.n_groups;
    if (tiles >= 128 || nk < 16) return m;
    const long target = 256 / tiles;
    int sps = (int)((nk + target - 1) / target);   // 64-steps per split
    const int per_seg = seg > 0 ? seg / 64 : nk;
    while (per_seg % sps != 0 || nk % sps != 0) ++sps;
    if (nk / sps < 2) return m;
    m.n_split = nk / sps;
    m.kc = sps * 64;
    return m;
}
constexpr int SWEEP_MAX_D = 4096;   // representatives per group for the sweep variant (norms in LDS)
inline bool match_sweeps(const Plan &p) {
    const int n_bt = (p.n_src_max + 127) / 128, n_at = (p.n_dst_max + 127) / 128;
    return p.bf16 && p.kind == KIND_TOKEN && p.C % 64 == 0 && n_at >= 2 && n_at * 128 <= SWEEP_MAX_D &&
           (long)n_bt * p.n_groups >= 512;
}
// node_max == nullptr: node_pack only (the selection unpacks it); part: the
// split-K partials (match_split), unused otherwise
hipError_t launch_match(const Plan &p, const void *x, const float *inv, const int32_t *units,
                        unsigned long long *node_pack, float *part, float *node_max, int32_t *node_idx,
                        hipStream_t st);
// flag / mtok given (Frame Cache): the frame stage also writes the per-frame
// selection, so no selection launch is needed, and with kept_idx /
// cached_idx / rmap given also the compaction.  bf16 layers: inv given
// (gram_norms), the Gram launch writes the token norms; pack given, it clears
// pack[0, n_pack); wo / wo16 given, it converts wo to fp16.
hipError_t launch_frame_stage(const Plan &p, const Layout &L, const void *x, char *ws, float *node_max,
                              int32_t *node_idx, int32_t *flag, int32_t *mtok, float *inv,
                              unsigned long long *pack, long n_pack, const void *wo, void *wo16, int32_t *kept_idx,
                              int32_t *cached_idx, int32_t *rmap, hipStream_t st);
hipError_t launch_select(const Plan &p, const int32_t *units, const float *node_max, const int32_t *node_idx,
                         int32_t *flag, int32_t *mtok, hipStream_t st);
// selection straight from node_pack; node_max / node_idx are written as
// well when non-null.  With kept_idx given (plain frames or Block Cache,
// patch_k == 1: one group per frame, or one group of all positions) the same
// launch also compacts into kept_idx, cached_idx and rmap, as
// launch_compact would.
// excl (optional, per item): candidates with a nonzero entry are not
// candidates of this selection and their flag / mtok entries stay as they
// are (the second level of the hierarchy after the first).  clear_pack:
// leave the packed arg-max zeroed (a second level's similarity follows).
// wo / wo16 given (bf16): extra blocks of the same launch convert the
// output-projection weights (n_wo elements) to fp16 beside the selection.
hipError_t launch_select_packed(const Plan &p, const int32_t *units, unsigned long long *node_pack,
                                const float *inv, float *node_max, int32_t *node_idx, int32_t *flag, int32_t *mtok,
                                int32_t *kept_idx, int32_t *cached_idx, int32_t *rmap, hipStream_t st,
                                const int32_t *excl = nullptr, int clear_pack = 0, const void *wo = nullptr,
                                void *wo16 = nullptr, long n_wo = 0);
// whether launch_select_packed can compact in the same launch (the frame's
// flags are staged in LDS: N below SEL_COMPACT_MAX_N)
constexpr int SEL_COMPACT_MAX_N = 24576;
inline bool select_compacts(const Plan &p) {
    return (p.kind == KIND_TOKEN || p.kind == KIND_BLOCK) && p.gran != 3 && p.k == 1 && p.N < SEL_COMPACT_MAX_N;
}
hipError_t launch_compact(const Plan &p, const int32_t *units, const int32_t *flag, const int32_t *mtok,
                          int32_t *fcnt, int32_t *kept_idx, int32_t *cached_idx, int32_t *rmap,
                          int map_matched, hipStream_t st);
// Frame Cache on patches: from the tiles' flags / matched tiles (at their
// top-left ids), the frame-major kept list, the cached list, the restore map
// (cold "matched": token n of a skipped tile reads token n of the matched
// frame) and the sequence offsets seq_off[F + 1].
hipError_t launch_compact_fpatch(const Plan &p, const int32_t *flag, const int32_t *mtok, int32_t *kept_idx,
                                 int32_t *cached_idx, int32_t *rmap, int32_t *seq_off, int map_matched,
                                 hipStream_t st);
// Frame Cache on patches: the tiles' inverse norms (at their top-left ids),
// with the same pack clearing and wo conversion as launch_inv_norm.
hipError_t launch_tile_norm(const Plan &p, const void *x, float *inv, unsigned long long *node_pack, long n_pack,
                            const void *wo, void *wo16, long n_wo, hipStream_t st);
// cold "matched" restore map: cached positions point at their matched row
hipError_t launch_map_matched(const Plan &p, const int32_t *flag, const int32_t *mtok, int32_t *rmap,
                              hipStream_t st);
hipError_t launch_gather(const Plan &p, const void *x, const int32_t *kept_idx, int n_rows, void *x_kept,
                         hipStream_t st);
hipError_t launch_restore(const Plan &p, const void *y_kept, int n_rows, const int32_t *rmap,
                          const void *cache_y, void *y, hipStream_t st);
hipError_t launch_copy_matched(const Plan &p, const int32_t *cached_idx, int n_cached,
                               const int32_t *rmap, const int32_t *kept_idx, void *y, hipStream_t st);
hipError_t launch_fill_i32(int32_t *dst, long n, int32_t value, hipStream_t st);
hipError_t launch_add(const Plan &p, const void *x, const void *y, void *h, hipStream_t st);

// Reduced attention: rows r < n_main come from x rows (row_idx[r] if row_idx,
// else r), rows n_main..n_main+n_ctx from ctx.  Sequence s owns rows
// [s*L, s*L+L) plus, for a single sequence, the context rows.  Output rows
// r < n_main go to y[out_idx[r]] (or y[r]); context rows go to y_ctx.
struct AttnArgs {
    const void *x; const int32_t *row_idx; int n_main;
    const void *ctx; int n_ctx;
    int n_seq, L;                     // sequences and retained tokens per sequence
    const void *wq, *wk, *wv, *wo;
    void *y; const int32_t *out_idx;  // main outputs
    void *y_ctx;
    void *q, *k, *vt, *o;             // workspace
    void *wo16;                       // workspace: wo converted to fp16 (bf16 layers)
    int wo16_ready;                   // wo16 already converted by an earlier launch of this call
    int lpad;                         // padded keys per sequence in vt
    int tF, tN;                       // no index lists: row r = n*tF + f is token f*tN + n (tF > 0)
    const int32_t *seq_off;           // sequences of varying length: sequence s owns rows
                                      // [seq_off[s], seq_off[s+1]) (n_main rows in all, no context,
                                      // L the longest); nullptr: every sequence has L rows
};
hipError_t launch_attention(const Plan &p, const AttnArgs &a, hipStream_t st);

// Feed-forward sublayer over retained rows (k_ffn.hip).
struct FfnArgs {
    const void *x; const int32_t *idx;   // batch row r -> token idx[r] (idx == nullptr: r)
    int n_rows, FN, C, hidden;
    const void *w1, *w2;                 // [hidden, C], [C, hidden]
    void *h;                             // scratch: H [n_rows, hidden] fp16, then W2 as fp16
    int scatter;                         // 1: row r -> y row idx[r] (or r); 0: y row r
    void *y;
};
size_t ffn_workspace_bytes(int n_rows, int hidden, int C);
hipError_t launch_ffn(const FfnArgs &a, hipStream_t st);

// Library-owned device scratch of oc_layer_cached_static: size, and the
// current device's address (looked up once per device).
constexpr size_t OC_STATIC_SCRATCH_BYTES = (size_t)96 << 20;
hipError_t static_scratch(void **out);
bool attn_head_dim_supported(int dh);

}  // namespace oc
