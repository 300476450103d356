/*
 * oc.h — C ABI of the OmniCache cached attention layer for MI355X (gfx950).
 *
 * One attention layer of a diffusion denoiser with OmniCache's per-layer
 * feature caches (OmniCache §3.2 "OmniCache", §3.3 "Hierarchical Caching"):
 *   Token Cache  (§3.2.3): 2x2 token neighbourhoods inside a frame,
 *   Frame Cache  (§3.2.2): odd frames matched against even frames,
 *   Block Cache  (§3.2.1): per-position temporal blocks in 2x2 groups,
 *   Frame+Token  (§3.2.3, second paragraph): token caching inside matched
 *                frame pairs (2x2x2 cubes) and unmatched frames.
 * Every call: cosine-similarity matching against fixed representatives ->
 * the r most redundant candidates are cached -> the retained tokens are
 * gathered and run through multi-head attention -> cached positions are
 * restored from the layer cache at their original positions.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Token tensor x is [F, N = H*W, C] row-major (C contiguous); token
 *    (f, y, x) has global id f*N + y*W + x.  Element type per oc_shape.dtype:
 *    float (OC_F32) or bfloat16 bit patterns (OC_BF16).
 *  - Weights use the out-features x in-features layout of a linear layer:
 *    wq, wk, wv are [heads*head_dim, C] and wo is [C, heads*head_dim];
 *    q = x wq^T etc.  Same element type as x.
 *  - All device pointers are caller-owned device memory, 16-byte aligned.
 *    The library allocates no device memory and keeps no device state
 *    between calls; scratch space is the caller's workspace of at least
 *    oc_plan_info.workspace_bytes.  The one exception is
 *    oc_layer_cached_static, whose scratch is a static device array of the
 *    library (see there).  Its only shared host state is a
 *    mutex-guarded record of the kernels whose dynamic-LDS limit it has
 *    raised on each device (plus the thread-local error message and stage
 *    timer), so concurrent calls from several threads are safe.
 *  - Numeric range: inside the attention the projections q, k, v, the
 *    probabilities and the per-head outputs are held in fp16 (11
 *    significant bits, fp32 accumulation everywhere).  Two limits follow,
 *    and neither is reported (the call returns OC_OK):
 *      precision: a logit q.k/sqrt(head_dim) carries a relative error of
 *      about 2^-11, so outputs stay within 1% of their RMS while the largest
 *      |logit| of a sequence is below about 100; larger logits (e.g. input
 *      channels 50x or more above the rest, with no normalisation before
 *      the layer) make the softmax ill-conditioned at 16-bit q and k, and
 *      the error grows with the logits (measured 1.7% of RMS at 2e2, 12-19%
 *      at 8e4 for 256-token sequences);
 *      range: q, k, v or per-head outputs beyond 65504 in magnitude are
 *      saturated to +-65504.
 *  - All work is enqueued on the caller's stream; calls are asynchronous.
 *    Results are deterministic: the same inputs give bit-identical outputs.
 *  - Every function validates its arguments on the host first.  On any
 *    error nothing is enqueued and no output is touched; the status says
 *    why and oc_last_error() holds a message (thread-local).  Asynchronous
 *    device faults surface at the caller's next synchronisation.
 *  - Calls on different streams with different workspaces may overlap.
 *
 * Readings of the paper that fix details it leaves open (ratios are
 * fractions of all items of a group, floored and clamped to the candidates;
 * representatives are the top-left token of each 2x2 window; odd frames are
 * frame candidates; ties go to the smallest id; ...) are listed with the
 * design notes of this library.
 */
#ifndef OMNICACHE_OC_H
#define OMNICACHE_OC_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    OC_OK = 0,
    OC_ERR_INVALID_ARG = 1,   /* NULL or misaligned pointer, ratio outside [0,1) or NaN, bad enum */
    OC_ERR_SHAPE = 2,         /* shape not supported (see oc_plan) */
    OC_ERR_DTYPE = 3,         /* unknown element type */
    OC_ERR_WORKSPACE = 4,     /* ws_bytes smaller than oc_plan_info.workspace_bytes */
    OC_ERR_CACHE_STATE = 5,   /* cache->y NULL or cache->valid not 0/1 */
    OC_ERR_HIP = 6            /* a HIP launch or copy failed */
} oc_status;

typedef enum { OC_F32 = 0, OC_BF16 = 1 } oc_dtype;

typedef enum {
    OC_GRAN_TOKEN = 0,        /* Token Cache (spatial layer), ratio r       */
    OC_GRAN_FRAME = 1,        /* Frame Cache (spatial layer), ratio r_frame */
    OC_GRAN_BLOCK = 2,        /* Block Cache (temporal layer), ratio r      */
    OC_GRAN_FRAME_TOKEN = 3   /* Frame + Token Cache (spatial layer)        */
} oc_gran;

typedef enum {
    OC_COLD_MATCHED = 0,      /* no valid cache: a cached position takes its matched
                                 representative's fresh output (a copy, never an average) */
    OC_COLD_FULL = 1          /* no valid cache: nothing is cached in that call */
} oc_cold;

typedef struct {
    int32_t F, H, W, C;       /* frames, grid height/width (N = H*W), channels */
    int32_t heads, head_dim;  /* attention heads and head dimension */
    int32_t n_ctx;            /* uncached context tokens appended to the image
                                 sequence (text tokens of a joint-attention layer);
                                 >0 only with F == 1 and OC_GRAN_TOKEN */
    int32_t dtype;            /* oc_dtype */
} oc_shape;

typedef struct {
    int32_t gran;             /* oc_gran */
    int32_t patch_k;          /* k x k patch-local matching (§3.3), >= 1; 1 for FRAME */
    double  r;                /* token / block ratio in [0,1) */
    double  r_frame;          /* frame ratio in [0,1) (FRAME, FRAME_TOKEN) */
    int32_t cold;             /* oc_cold */
    int32_t coarse_k;         /* 0: one level.  Otherwise a second, coarser level of
                                 the hierarchy (§3.3: reuse first inside k x k
                                 patches, then in coarser patches or the whole
                                 frame), TOKEN and BLOCK only: 1 <= coarse_k <
                                 patch_k, patch_k % coarse_k == 0 */
    double  r_coarse;         /* the second level's ratio in [0,1) */
} oc_cfg;

typedef struct {
    void   *y;                /* [F, N, C] device buffer: the layer cache, which is
                                 also the layer output (updated in place) */
    int32_t valid;            /* 0: no previous step; 1: y holds the previous step */
    int32_t step;             /* incremented by every oc_layer_cached call */
} oc_cache;

typedef struct {
    const void *wq, *wk, *wv; /* [heads*head_dim, C] */
    const void *wo;           /* [C, heads*head_dim] */
} oc_attn_weights;

typedef struct {
    /* matching problem of the (token / block / frame) stage returned by oc_match */
    int32_t n_groups;         /* groups                                          */
    int32_t n_src_max;        /* candidates per group (padded maximum)           */
    int32_t n_dst_max;        /* representatives per group (padded maximum)      */
    /* frame stage of OC_GRAN_FRAME_TOKEN */
    int32_t n_frame_src, n_frame_dst, n_frame_cached;
    /* reduced attention batch */
    int32_t n_kept;           /* retained tokens = n_seq * seq_len               */
    int32_t n_cached;         /* cached tokens = F*N - n_kept                    */
    int32_t n_seq, seq_len;   /* sequences of the reduced batch, tokens each     */
    size_t  workspace_bytes;  /* enough for every entry point with this shape/cfg */
} oc_plan_info;

typedef struct {
    float   *frame_max;       /* [n_frame_src] best frame similarity per odd frame */
    int32_t *frame_idx;       /* [n_frame_src] matched even frame                  */
    int32_t *pairs;           /* [n_frame_cached * 2] (s, d) in pairing order      */
} oc_frame_info;

typedef struct {
    float   *node_max;        /* [n_groups * n_src_max]        */
    int32_t *node_idx;        /* [n_groups * n_src_max]        */
    int32_t *kept_idx;        /* [n_kept]                      */
    int32_t *cached_idx;      /* [n_cached]                    */
    int32_t *restore_map;     /* [F*N]                         */
    oc_frame_info frames;     /* OC_GRAN_FRAME_TOKEN only      */
} oc_trace;                   /* every pointer may be NULL: that output is not copied */

/*
 * oc_plan — host only, no device work.  Validates shape and cfg and returns
 * the static sizes of one call (they depend only on shape and cfg): the
 * matching groups of each cache (§3.2.1 2x2 block groups, §3.2.2 the
 * alternating odd / even frame sets, §3.2.3 2x2 token neighbourhoods and
 * 2x2x2 cubes of frame pairs, all inside k x k patches per §3.3), the
 * skip budgets that the ratios r_b, r_f and r_t of §3.2 give each group,
 * and the reduced attention batch.
 * Requirements (OC_ERR_SHAPE otherwise): F, H, W, C, heads, head_dim >= 1;
 * H and W divisible by 2*patch_k; C % 8 == 0; head_dim % 8 == 0 and
 * head_dim <= 128; 2 <= F <= 32 for FRAME and FRAME_TOKEN; patch_k <= 16
 * for FRAME; n_ctx == 0 unless F == 1 and gran == TOKEN.
 * FRAME with patch_k > 1 is Frame Cache on k x k patches (§3.3: every
 * patch's frame set is matched on its own): n_groups = k*k, the items of a
 * group are the frames' tiles of that patch, named by their top-left token
 * id; each patch caches R = min(floor(r_frame*F), F/2) odd-frame tiles.  Its
 * n_seq = F sequences (one per frame, in frame order) have varying lengths
 * of at most seq_len = N tokens (a frame may keep none), n_kept = (F - R)*N
 * in all; x_kept is then the packed [n_kept, C] batch, which only
 * oc_layer_cached runs (oc_attn_reduced takes equal-length sequences).
 * Skip counts: a group of n items caches min(floor(r*n), candidates); frame
 * pairs cache min(n_f + floor(r*n_f), candidates) of their 2*n_f tokens.
 * With coarse_k > 0 the first level's groups are those of patch_k; then
 * every coarse_k x coarse_k patch (a union of (patch_k/coarse_k)^2 of them)
 * of n2 items caches min(floor(r_coarse*n2), the candidates the first level
 * left) more, by the same rule among those candidates against the same
 * representatives.  The reduced batch holds the tokens neither level
 * cached; n_groups, n_src_max and n_dst_max describe the first level, and
 * only oc_layer_cached (and the calls built on it) runs two levels
 * (oc_match and oc_select return OC_ERR_INVALID_ARG).
 */
oc_status oc_plan(const oc_shape *shape, const oc_cfg *cfg, oc_plan_info *out);

/*
 * oc_match — cosine-similarity matching (§3.2.1-§3.2.3, patch-local per
 * §3.3).  For every candidate of every group: the largest cosine similarity
 * to a representative of its group (node_max, fp32) and that
 * representative's id (node_idx; smallest id on ties).  Ids are global token
 * ids (TOKEN, FRAME_TOKEN), spatial positions n (BLOCK), frame indices
 * (FRAME) or, for FRAME on patches, the tiles' top-left token ids.  Layout [n_groups, n_src_max], candidates of a group in ascending
 * id; padding entries hold -inf / -1.  Group order: TOKEN frame-major then
 * patches row-major; BLOCK patches; FRAME one group; FRAME_TOKEN attention
 * units (frame pairs and unmatched frames, by smallest frame) then patches.
 * FRAME_TOKEN first matches, selects and pairs frames; that frame stage is
 * kept in ws (which oc_select must then receive unchanged) and optionally
 * copied to *frames.  frames may be NULL.
 */
oc_status oc_match(const oc_shape *shape, const oc_cfg *cfg, const void *x,
                   float *node_max, int32_t *node_idx, oc_frame_info *frames,
                   void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * oc_select — the R most redundant candidates of each group are cached
 * (§3.2.1 "the r_b most redundant blocks", §3.2.2, §3.2.3): largest
 * node_max first, smallest id on ties, exactly R per group.  Emits
 *   kept_idx    [n_kept]  retained global token ids in row order of the
 *                         reduced batch: sequences ordered by the smallest
 *                         item they cover, ascending token id inside (block
 *                         sequences list frames 0..F-1 of one position);
 *   cached_idx  [n_cached] cached token ids, ascending;
 *   restore_map [F*N]     row of kept_idx holding p's output, or, for a
 *                         cached p: -1 (take the layer cache) when
 *                         map_matched == 0, else the row of p's matched
 *                         representative token.
 * node_max/node_idx are oc_match's outputs (same layout).
 */
oc_status oc_select(const oc_shape *shape, const oc_cfg *cfg,
                    const float *node_max, const int32_t *node_idx,
                    int32_t *kept_idx, int32_t *cached_idx, int32_t *restore_map,
                    int32_t map_matched, void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * oc_gather — x_kept[i] = x[kept_idx[i]] for the plan's n_kept rows
 * (§3.2.3 reduced token set; App. A gather).  x_kept is [n_seq, seq_len, C].
 * kept_idx entries outside [0, F*N) leave their row untouched.
 */
oc_status oc_gather(const oc_shape *shape, const oc_cfg *cfg, const void *x,
                    const int32_t *kept_idx, void *x_kept, hipStream_t stream);

/*
 * oc_attn_reduced — multi-head self-attention over each of n_seq sequences
 * of seq_len retained tokens (x_kept [n_seq, seq_len, C]); cached tokens
 * take no part (§3.2.3).  With n_ctx > 0 (n_seq must be 1) the context rows
 * ctx [n_ctx, C] are appended to the sequence and their outputs written to
 * y_ctx [n_ctx, C].  y_kept is [n_seq*seq_len, C].  softmax(q k^T /
 * sqrt(head_dim)) v per head, heads concatenated, then wo; no bias.
 * ws_bytes must be >= oc_attn_workspace_bytes(shape, n_seq, seq_len).
 */
oc_status oc_attn_reduced(const oc_shape *shape, const void *x_kept, int32_t n_seq, int32_t seq_len,
                          const void *ctx, const oc_attn_weights *w, void *y_kept, void *y_ctx,
                          void *ws, size_t ws_bytes, hipStream_t stream);

size_t oc_attn_workspace_bytes(const oc_shape *shape, int32_t n_seq, int32_t seq_len);

/*
 * oc_restore — cached positions restored at their original positions
 * (§3.2.1 "restores cached blocks to their original spatial positions",
 * §3.2.3 "scattered back to the original frame layout"): for every p in
 * [0, F*N): y[p] = y_kept[restore_map[p]] if 0 <= restore_map[p] < n_rows,
 * y[p] = cache_y[p] if restore_map[p] == -1 (cache_y may be NULL when the
 * map has no -1; y may alias cache_y, then those rows are left as they are);
 * other values leave y[p] untouched.
 */
oc_status oc_restore(const oc_shape *shape, const void *y_kept, int32_t n_rows,
                     const int32_t *restore_map, const void *cache_y, void *y, hipStream_t stream);

/*
 * oc_layer_cached — one cached layer call (match, select, reduced attention,
 * restore) writing the layer output in place into cache->y: retained
 * positions get fresh outputs, cached positions keep cache->y from the
 * previous step (§3.2.3 "restored from cached activations associated with
 * the same positions at the previous denoising step").  If cache->valid is 0
 * the cold policy applies.  Afterwards cache->valid = 1 and cache->step is
 * incremented (host-side fields).  x must not alias cache->y.  trace may be
 * NULL; non-NULL fields receive copies of this call's decisions.
 */
oc_status oc_layer_cached(const oc_shape *shape, const oc_cfg *cfg, const void *x, const void *ctx,
                          const oc_attn_weights *w, oc_cache *cache, void *y_ctx,
                          oc_trace *trace, void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * oc_residual_add — h = x + y elementwise over [F, N, C] (added in fp32,
 * rounded once to the tensor's type, bf16: round to nearest even): the
 * residual connection that feeds a block's spatial-layer output to its
 * temporal layer.  h may alias x or y.
 */
oc_status oc_residual_add(const oc_shape *shape, const void *x, const void *y, void *h, hipStream_t stream);

/*
 * oc_block_cached — one spatial + temporal block of a video denoiser with all
 * three caches at once (§3.2: Frame and Token Cache on the spatial layer,
 * Block Cache on the temporal layer; §4.2 runs them together at ratios
 * r_f / r_b / r_t such as 50/40/50 for SVD-XT and 30/40/20 for Latte):
 *   spatial layer:  oc_layer_cached(shape, spatial, x) -> cache_spatial->y;
 *   residual:       h = x + cache_spatial->y (oc_residual_add);
 *   temporal layer: oc_layer_cached(shape, temporal, h) -> cache_temporal->y,
 * each layer with its own weights and its own layer cache (the temporal
 * layer's cached blocks are matched on h).  spatial->gran is TOKEN, FRAME or
 * FRAME_TOKEN, temporal->gran is BLOCK; n_ctx must be 0.  x, h and the two
 * caches are distinct [F, N, C] buffers; the traces may be NULL.  Every
 * argument of both layers is validated before anything is enqueued.
 * ws_bytes >= oc_block_workspace_bytes(shape, spatial, temporal) (the two
 * layers run one after the other on the stream and share it).
 */
oc_status oc_block_cached(const oc_shape *shape, const oc_cfg *spatial, const oc_cfg *temporal, const void *x,
                          const oc_attn_weights *w_spatial, const oc_attn_weights *w_temporal,
                          oc_cache *cache_spatial, oc_cache *cache_temporal, void *h, oc_trace *trace_spatial,
                          oc_trace *trace_temporal, void *ws, size_t ws_bytes, hipStream_t stream);

size_t oc_block_workspace_bytes(const oc_shape *shape, const oc_cfg *spatial, const oc_cfg *temporal);

/*
 * Feed-forward sublayer under the same selection.  The SD3 experiments cache
 * attention and feed-forward layers alike (§4.2 "Design choices"): the
 * tokens the attention sublayer retained also go through the FFN, and the
 * rest are restored at their positions.  The FFN is two linear maps with a
 * tanh-approximated GELU between them and no bias.
 */
typedef struct {
    const void *w1;           /* [hidden, C]: first linear map, out x in      */
    const void *w2;           /* [C, hidden]: second linear map, out x in     */
    int32_t hidden;           /* inner width (SD3: 4 C)                       */
    int32_t reserved;         /* must be 0                                     */
} oc_ffn_weights;

/*
 * oc_ffn_reduced — for the n_rows retained tokens t_i = kept_idx[i] (or
 * t_i = i when kept_idx is NULL):
 *   z_i = GELU(x[t_i] W1^T) W2^T,  GELU(v) = 0.5 v (1 + tanh(sqrt(2/pi)(v + 0.044715 v^3)));
 * x is [F, N, C] bf16 (the FFN input of every position; only retained rows
 * are read).  scatter = 1: y is [F, N, C] and z_i is written to y[t_i],
 * every other row of y is left untouched (y holding the previous step's FFN
 * output, that is restoration in place, as oc_layer_cached does for the
 * attention); scatter = 0: y is [n_rows, C] and z_i goes to row i (then
 * oc_restore with the attention call's restore map covers the cold step).
 * bf16 only (OC_ERR_DTYPE otherwise); C and hidden multiples of 64
 * (OC_ERR_SHAPE); kept_idx entries outside [0, F*N) are not read and their
 * rows not written.  ws_bytes >= oc_ffn_workspace_bytes(shape, hidden,
 * n_rows): the [n_rows, hidden] activations between the two maps, held in
 * fp16 (range and precision as stated for the attention intermediates),
 * and an fp16 copy of W2 made by the same call.
 * y must not alias x.
 */
oc_status oc_ffn_reduced(const oc_shape *shape, const void *x, const int32_t *kept_idx, int32_t n_rows,
                         const oc_ffn_weights *w, void *y, int32_t scatter, void *ws, size_t ws_bytes,
                         hipStream_t stream);

size_t oc_ffn_workspace_bytes(const oc_shape *shape, int32_t hidden, int32_t n_rows);

/*
 * oc_layer_cached_static — oc_layer_cached without a workspace argument, for
 * callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc).  Same arguments,
 * results and errors as oc_layer_cached; the scratch is a library-owned
 * device array of oc_static_scratch_bytes() (96 MiB) per device, which every
 * device the library runs on holds until the process ends.  Allocates
 * nothing.  A layer whose oc_plan_info.workspace_bytes exceeds that size is
 * rejected with OC_ERR_WORKSPACE before anything is enqueued (the SD3-1024
 * and Latte-sized layers fit; the SVD-XT-sized level, 576 MiB, does not).
 * The stream must belong to the current device.  All calls on one device
 * share that device's array, and each call rewrites what it reads of it:
 * calls that overlap on one device (different streams or threads without
 * ordering between them) race on it and must be serialised by the caller.
 */
oc_status oc_layer_cached_static(const oc_shape *shape, const oc_cfg *cfg, const void *x, const void *ctx,
                                 const oc_attn_weights *w, oc_cache *cache, void *y_ctx, oc_trace *trace,
                                 hipStream_t stream);

/* Size in bytes of the static scratch oc_layer_cached_static uses. */
size_t oc_static_scratch_bytes(void);

/*
 * oc_attn_full — the uncached baseline: the layer as it runs without any
 * cache, i.e. the computation every cache of §3.2 skips part of (the
 * denominator of a cached layer's speed-up).  Spatial attention per frame
 * over all N tokens (+ context) for TOKEN/FRAME/FRAME_TOKEN, or temporal
 * attention per position over all F frames for BLOCK (§3.2.1: the temporal
 * layer's H*W sequences of length T).  Same kernels and numerics as the
 * reduced attention.  y is [F, N, C]; ws_bytes >=
 * oc_plan_info.workspace_bytes.  Errors as for oc_layer_cached.
 */
oc_status oc_attn_full(const oc_shape *shape, const oc_cfg *cfg, const void *x, const void *ctx,
                       const oc_attn_weights *w, void *y, void *y_ctx,
                       void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * Layered Cache schedule proposal (§3.4, Alg. 1), host only.  For each
 * candidate layer-timestep pair (l, t) the caller gives the latency L[l,t]
 * that reusing the cache there saves and the quality loss Q[l,t] it costs
 * (row-major [n_layers, n_steps] tables); mask (may be NULL: every pair)
 * marks the candidates.  Pairs are scored w = Q/L, taken from the lowest
 * score up and written to out as (l, t, interval) until the saved latency
 * is at least (1 - 1/target_speedup) times the summed latency of all
 * candidates (or no candidate is left).  Candidates are enumerated
 * layer-major; equal scores keep that order and sums run in that order.
 * Requirements (OC_ERR_INVALID_ARG otherwise): target_speedup >= 1,
 * interval >= 1, every candidate's L finite and > 0 and Q finite, and
 * capacity at least the number of pairs chosen (n_layers * n_steps always
 * suffices).  *n_out receives the count; saved / budget (may be NULL) the
 * saved latency and the budget.
 */
typedef struct { int32_t layer, step, interval; } oc_cache_entry;

oc_status oc_layered_schedule(int32_t n_layers, int32_t n_steps, const double *latency, const double *quality,
                              const uint8_t *mask, double target_speedup, int32_t interval, oc_cache_entry *out,
                              int32_t capacity, int32_t *n_out, double *saved, double *budget);

const char *oc_status_string(oc_status s);
const char *oc_last_error(void);

/*
 * Stage timing (a profiling aid, not part of the method).  A caller-owned
 * timer holds HIP events; while it is attached to a thread with
 * oc_timer_use, every kernel the library enqueues from that thread is
 * launched with a pair of the timer's events that the runtime stamps at the
 * kernel's start and end (so a stage's time is its kernels' durations), tagged
 * with its stage name ("match", "select", "flash", ...).  oc_timer_collect
 * waits for the events and adds each kernel's duration to its stage's total
 * and 1 to its stage's launch count.  oc_timer_use(NULL) detaches.
 */
typedef struct oc_timer oc_timer;
oc_status oc_timer_create(oc_timer **out);
void oc_timer_destroy(oc_timer *t);
oc_status oc_timer_use(oc_timer *t);
oc_status oc_timer_collect(oc_timer *t);
oc_status oc_timer_reset(oc_timer *t);
int32_t oc_timer_stage_count(const oc_timer *t);
oc_status oc_timer_stage(const oc_timer *t, int32_t i, const char **name, double *total_ms, int64_t *launches);

/*
 * oc_clock_sample — shader clock sampler (a measurement aid, not part of the
 * method).  Enqueues on `stream` a one-wave kernel that writes n pairs
 * samples[2i] = shader clock count (s_memtime), samples[2i+1] = 100 MHz
 * real-time count (s_memrealtime), one pair every gap_ticks real-time ticks
 * (gap_ticks / 100 µs).  samples is a device buffer of 2n int64 owned by the
 * caller.  Launched on a second stream beside a workload, the ratio of the
 * differences gives the clock that workload runs at (GHz = d_clock /
 * (10 d_realtime)).  The kernel occupies one wave slot of one CU and ends
 * after n samples.  OC_ERR_INVALID_ARG for a null buffer, n <= 0 or gap_ticks
 * outside [0, 1e8]; OC_ERR_HIP if the launch fails.
 */
oc_status oc_clock_sample(int64_t *samples, int32_t n, int32_t gap_ticks, hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* OMNICACHE_OC_H */
