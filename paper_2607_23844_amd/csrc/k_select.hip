// Selection of the most redundant candidates and the bookkeeping that turns
// it into the reduced attention batch (OmniCache §3.2.1-§3.2.3: "the r most
// redundant" items are cached, the retained ones are computed, cached
// positions are later restored at their original positions).
//
// Selection per group is an exact radix select on order-preserving 32-bit
// keys of node_max: the R largest keys are cached, ties at the threshold go
// to the smallest candidate positions (ascending global id), so exactly R
// are cached.  No floating-point atomics; integer LDS histograms only.
#include "oc_internal.h"
#include "oc_launch.h"
#include "oc_device.h"
#include "oc_block.h"
#include "oc_groups.h"
#include "oc_mfma_tile.h"
#include "oc_attn_common.h"
#include <algorithm>

namespace oc {

constexpr int SEL_IPT = 16;            // candidates per thread: groups up to 16 x the block size
constexpr int SEL_HISTS = 4;           // radix histograms (one per SIMD)
// Block size: eight waves for small groups (up to 4 candidates per thread:
// fewer waves per barrier), sixteen otherwise (up to 16384 candidates; four
// waves with 12 candidates each measured 50% slower than sixteen at 3072)
constexpr int SEL_SMALL = 512, SEL_LARGE = 1024;


// One block per group.  PACKED: node_max / node_idx are unpacked from the
// similarity kernel's packed arg-max (the candidate's inverse norm applied
// last) and written out when node_max_out is given; otherwise they are read.
// With kept_idx (one group per plain frame) the block then compacts its
// frame: retained tokens in ascending id become rows [g*L, g*L+L), cached
// ones go to cached_idx[g*Rc...] (Rc = the frame's static budget).  Block
// Cache (tF = F > 0, one group of all N positions): the b-th retained
// position becomes sequence b (rows b*F + f, token f*N + n), cached
// positions ascend frame-major in cached_idx[f*Rc + rank].  The per-token
// flag / mtok arrays are written only when given: a compacting warm step
// passes none, since only the cold "matched" mapping reads them then.
template <bool PACKED, int SEL_THREADS, int IPT>
__global__ __launch_bounds__(SEL_THREADS) void k_select(const float *__restrict__ node_max_in,
                                                        const int32_t *__restrict__ node_idx_in,
                                                        unsigned long long *__restrict__ node_pack,
                                                        const float *__restrict__ inv,
                                                        float *__restrict__ node_max_out,
                                                        int32_t *__restrict__ node_idx_out, GroupMap gm, int G,
                                                        int S, int D, int32_t *flag,
                                                        int32_t *__restrict__ mtok, int32_t *__restrict__ kept_idx,
                                                        int32_t *__restrict__ cached_idx,
                                                        int32_t *__restrict__ rmap, int N, int L, int tF,
                                                        const int32_t *excl,   // may alias flag (read first, per block)
                                                        int clear_pack, const uint4 *__restrict__ wo, long n8,
                                                        uint4 *__restrict__ wo16) {
    // blocks past the groups: convert wo to fp16 for the output projection
    // (independent work on the CUs the selection leaves idle)
    if ((int)blockIdx.x >= G) {
        const long nb = gridDim.x - G;
        for (long i = (long)(blockIdx.x - G) * SEL_THREADS + threadIdx.x; i < n8; i += nb * SEL_THREADS)
            wo16[i] = bf16x8_to_f16x8(wo[i]);
        return;
    }
    constexpr int SEL_WAVES = SEL_THREADS / 64;
    // digit histograms, one per SIMD (waves w, w+4, ... share one),
    // double-buffered across radix passes
    __shared__ int hist[2][SEL_HISTS][256];
    __shared__ uint32_t red[3][SEL_WAVES];
    __shared__ int sh[17];
    __shared__ int sel_info[3];
    // candidate keys, staged through LDS (klds, S words): read from global
    // memory in slabs (thread t: i = j*SEL_THREADS + t, coalesced), then held
    // by thread t as the contiguous run i = t*ipt + j for the radix passes, so
    // that one wave's histogram updates mix distant (less correlated)
    // candidates; candidates i >= the group's count are not valid
    extern __shared__ uint32_t klds[];
    const int g = blockIdx.x;
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int ipt = cdiv(S, SEL_THREADS);
    const GroupMap::Grp gr = gm.group(g);
    const int R = gr.R;
    const int n_src = min(gr.nsrc, S);

    // slab layout: every load of the thread's candidates is issued first
    // (one round trip), then they are unpacked
    int32_t nid[IPT], sids[IPT], exv[IPT];
    unsigned long long pk[IPT];
    float iv[IPT];
#pragma unroll
    for (int j = 0; j < IPT; ++j) {
        nid[j] = -1;
        sids[j] = -1;
        exv[j] = 0;
        if (j >= ipt) continue;
        const int i = j * SEL_THREADS + t;
        const long gi = (long)g * S + i;
        const int sid = i < S ? gm.src_id(gr, i) : -1;
        sids[j] = sid;
        pk[j] = 0;
        iv[j] = 0.f;
        if (sid >= 0) {
            if constexpr (PACKED) {
                pk[j] = node_pack[gi];
                iv[j] = inv[sid];
            } else {
                iv[j] = node_max_in[gi];
                nid[j] = node_idx_in[gi];
            }
            if (excl != nullptr) exv[j] = excl[sid];
        }
    }
    // a second level follows: leave the packed arg-max zeroed for its
    // similarity kernel (every slot g*S + i of this launch, read above)
    if (PACKED && clear_pack) {
        // (the thread that read a slot clears it, after its load in program order)
#pragma unroll
        for (int j = 0; j < IPT; ++j) {
            const int i = j * SEL_THREADS + t;
            if (j < ipt && i < S) node_pack[(long)g * S + i] = 0ull;
        }
    }
    // excluded candidates (slab layout bits): key 0 in LDS, which no value
    // maps to (float_key gives 0 only for one NaN pattern), marks them for
    // the run layout
    uint32_t exm = 0;
#pragma unroll
    for (int j = 0; j < IPT; ++j) {
        const int i = j * SEL_THREADS + t;
        if (j >= ipt || i >= S) continue;
        const long gi = (long)g * S + i;
        if (sids[j] < 0 || exv[j] != 0) {
            if (PACKED && node_max_out != nullptr) {
                node_max_out[gi] = -INFINITY;
                node_idx_out[gi] = -1;
            }
            if (sids[j] >= 0) {
                exm |= 1u << j;
                klds[i] = 0u;
            }
            continue;
        }
        float v = iv[j];
        if constexpr (PACKED) {
            int ix;
            unpack_argmax(pk[j], v, ix);
            v *= iv[j];
            nid[j] = ix >= 0 ? gm.dst_id(gr, ix) : -1;
            if (node_max_out != nullptr) {
                node_max_out[gi] = v;
                node_idx_out[gi] = nid[j];
            }
        }
        klds[i] = float_key(v);
    }
    __syncthreads();
    uint32_t key[IPT];   // run layout
    uint32_t vmask = 0;
    int nvalid_local = 0;
    uint32_t lo = 0xFFFFFFFFu, hi = 0u;
#pragma unroll
    for (int j = 0; j < IPT; ++j) {
        key[j] = 0;
        const int i = t * ipt + j;
        if (j >= ipt || i >= n_src) continue;
        key[j] = klds[i];
        if (key[j] == 0u) continue;   // excluded
        vmask |= 1u << j;
        ++nvalid_local;
        lo = min(lo, key[j]);
        hi = max(hi, key[j]);
    }
    // valid count, smallest and largest key: one combined block reduction
    uint32_t cnt = (uint32_t)nvalid_local;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        cnt += __shfl_xor(cnt, o, 64);
        lo = min(lo, (uint32_t)__shfl_xor(lo, o, 64));
        hi = max(hi, (uint32_t)__shfl_xor(hi, o, 64));
    }
    if (lane == 0) {
        red[0][wave] = cnt;
        red[1][wave] = lo;
        red[2][wave] = hi;
    }
    // clear both histogram buffers meanwhile
    for (int e = t; e < 2 * SEL_HISTS * 256; e += SEL_THREADS) (&hist[0][0][0])[e] = 0;
    __syncthreads();
    int n_valid = 0;
    uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
#pragma unroll
    for (int w = 0; w < SEL_WAVES; ++w) {
        n_valid += (int)red[0][w];
        kmin = min(kmin, red[1][w]);
        kmax = max(kmax, red[2][w]);
    }

    // threshold key tau (the R-th largest), how many keys equal to tau are
    // taken (need) and how many there are (n_eq: the count of the last
    // selected bin, which holds exactly the keys equal to tau)
    uint32_t tau = 0;
    int need = 0, n_eq = n_valid;
    const bool none = R <= 0;
    const bool all = R >= n_valid;
    if (!none && !all) {
        // keys share every bit above the highest bit where kmin and kmax
        // differ (bit_hi = -1: all keys equal).  The mask is one 64-bit shift:
        // a nested select here was compiled with the wrong condition.
        const uint32_t diff = kmin ^ kmax;
        int bit_hi = diff == 0 ? -1 : 31 - __clz((int)diff);
        uint32_t mask = (uint32_t)(0xFFFFFFFFull << (bit_hi + 1));
        uint32_t prefix = kmax & mask;
        int remaining = R;
        int buf = 0;
        while (bit_hi >= 0) {
            const int bit_lo = max(bit_hi - 7, 0);
            const int nbits = bit_hi - bit_lo + 1;
            const uint32_t dmask = (1u << nbits) - 1u;
            int *hw = hist[buf][wave % SEL_HISTS];
#pragma unroll
            for (int j = 0; j < IPT; ++j)
                if (((vmask >> j) & 1u) && (key[j] & mask) == prefix) atomicAdd(&hw[(key[j] >> bit_lo) & dmask], 1);
            __syncthreads();
            if (t < 64) {
                // lane covers bins [4*t, 4*t+4); suffix sums from the top bin down
                int c[4], sum = 0;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    int cq = 0;
#pragma unroll
                    for (int w = 0; w < SEL_HISTS; ++w) cq += hist[buf][w][4 * t + q];
                    c[q] = cq;
                    sum += cq;
                }
                int incl = sum;   // inclusive suffix over lanes >= t
#pragma unroll
                for (int o = 1; o < 64; o <<= 1) {
                    const int y = __shfl_down(incl, o, 64);
                    if (t + o < 64) incl += y;
                }
                int above = incl - sum;   // count in bins above this lane's bins
#pragma unroll
                for (int q = 3; q >= 0; --q) {
                    if (above < remaining && remaining <= above + c[q]) {
                        sel_info[0] = 4 * t + q;
                        sel_info[1] = above;
                        sel_info[2] = c[q];
                    }
                    above += c[q];
                }
            }
            // the other buffer, used by the next pass, was last read a pass ago
            for (int e = t; e < SEL_HISTS * 256; e += SEL_THREADS) (&hist[buf ^ 1][0][0])[e] = 0;
            __syncthreads();
            const int sel = sel_info[0];
            remaining -= sel_info[1];
            n_eq = sel_info[2];
            prefix |= (uint32_t)sel << bit_lo;
            mask |= dmask << bit_lo;
            bit_hi = bit_lo - 1;
            buf ^= 1;
            // the whole selected bin is taken: every key of it is >= prefix
            // (lower bits zero) and every key below it is < prefix, so prefix
            // is an exact threshold with no tie to break
            if (remaining == n_eq) break;
        }
        tau = prefix;
        need = remaining;
    }

    // exact selection: key > tau, or key == tau among the first `need` in
    // index order; without a tie to break (every key equal to tau taken, or
    // the passes stopped at a bin taken whole) no rank is needed
    const bool tie = !none && !all && need < n_eq;
    int eq_rank = 0;
    if (tie) {
        int eq_local = 0;
#pragma unroll
        for (int j = 0; j < IPT; ++j)
            if (((vmask >> j) & 1u) && key[j] == tau) ++eq_local;
        int eq_total;
        eq_rank = block_exclusive_scan(eq_local, sh, eq_total);
    }
    // decisions in the run layout, published as bytes in klds (every thread
    // read its keys from klds before the barriers above)
    uint8_t *cbyte = reinterpret_cast<uint8_t *>(klds);
    if (!none && !all) {
#pragma unroll
        for (int j = 0; j < IPT; ++j) {
            if (!((vmask >> j) & 1u)) continue;
            bool c;
            if (key[j] > tau) c = true;
            else if (key[j] == tau) { c = !tie || eq_rank < need; ++eq_rank; }
            else c = false;
            cbyte[t * ipt + j] = c ? 1 : 0;
        }
    }
    __syncthreads();
    // frame compaction (kept_idx given): flags of the frame's N tokens in LDS
    __shared__ uint8_t fl[SEL_COMPACT_MAX_N];
    const bool compact = kept_idx != nullptr;
    const long fbase = (long)g * N;
#pragma unroll
    for (int j = 0; j < IPT; ++j) {
        const int i = j * SEL_THREADS + t;
        if (j >= ipt || i >= n_src || ((exm >> j) & 1u)) continue;
        const bool c = all || (!none && cbyte[i] != 0);
        const int id = sids[j];
        if (flag != nullptr) {
            flag[id] = c ? 1 : 0;
            mtok[id] = c ? nid[j] : -1;
        }
        if (compact) fl[id - fbase] = c ? 1 : 0;
    }
    for (int i = t; i < D; i += SEL_THREADS) {
        const int id = gm.dst_id(gr, i);
        if (id >= 0) {
            if (flag != nullptr) {
                flag[id] = 0;
                mtok[id] = -1;
            }
            if (compact) fl[id - fbase] = 0;
        }
    }
    if (!compact) return;
    __syncthreads();
    // ranks over the frame's tokens in id order: position n = j*SEL_THREADS
    // + t (slab j, wave, lane); a slab's cached tokens counted per wave by a
    // ballot, one scan over the (slab, wave) counts, then a lane's cached
    // rank is its wave's prefix plus the cached lanes below it; the kept rank
    // is the position minus the cached rank
    __shared__ int wcnt[SEL_COMPACT_MAX_N / 64];
    const int nslab = cdiv(N, SEL_THREADS);
    for (int j = 0; j < nslab; ++j) {
        const int n = j * SEL_THREADS + t;
        const unsigned long long b = __builtin_amdgcn_ballot_w64(n < N && fl[n] != 0);
        if (lane == 0) wcnt[j * SEL_WAVES + wave] = __builtin_popcountll(b);
    }
    __syncthreads();
    const int n_cnt = nslab * SEL_WAVES;   // <= SEL_COMPACT_MAX_N / 64 = 384 <= SEL_THREADS
    int tot;
    const int pre = block_exclusive_scan(t < n_cnt ? wcnt[t] : 0, sh, tot);
    if (t < n_cnt) wcnt[t] = pre;
    __syncthreads();
    const int n_c = gr.R;   // every frame caches exactly its budget
    const unsigned long long below = (1ull << lane) - 1ull;
    for (int j = 0; j < nslab; ++j) {
        const int n = j * SEL_THREADS + t;
        const bool c = n < N && fl[n] != 0;
        const unsigned long long b = __builtin_amdgcn_ballot_w64(c);
        if (n >= N) continue;
        const int crank = wcnt[j * SEL_WAVES + wave] + __builtin_popcountll(b & below);
        const int krank = n - crank;
        const int pid = (int)(fbase + n);
        if (tF > 0) {
            // Block Cache: the position's F tokens
            for (int f = 0; f < tF; ++f) {
                const int tok = f * N + n;
                if (c) {
                    if (crank < n_c) cached_idx[(long)f * n_c + crank] = tok;
                    rmap[tok] = -1;
                } else {
                    const int row = krank * tF + f;
                    if (krank < L) kept_idx[row] = tok;
                    rmap[tok] = krank < L ? row : -2;
                }
            }
        } else if (c) {
            if (crank < n_c) cached_idx[(long)g * n_c + crank] = pid;
            rmap[pid] = -1;
        } else {
            const int row = g * L + krank;
            if (krank < L) kept_idx[row] = pid;
            rmap[pid] = krank < L ? row : -2;
        }
    }
}

// The kernel instance whose unrolled per-thread loops fit ipt = candidates
// per thread (1, 2, 3, 4, 8 or 16): a selection runs once per group from a
// cold instruction cache, so its code is kept to the loops it needs (the
// SD3-like group, 3 candidates per thread: 16.4 us with 16-wide loops,
// 12.7 with 4-wide, 0.5 less again with 3-wide).
template <bool PACKED, int T, typename... A>
static void go_sel(int ipt, unsigned grid, size_t lds, hipStream_t st, A... args) {
    if (ipt <= 1) launch_k(k_select<PACKED, T, 1>, grid, T, lds, st, args...);
    else if (ipt <= 2) launch_k(k_select<PACKED, T, 2>, grid, T, lds, st, args...);
    else if (ipt == 3) launch_k(k_select<PACKED, T, 3>, grid, T, lds, st, args...);
    else if (ipt <= 4 || T == SEL_SMALL) launch_k(k_select<PACKED, T, 4>, grid, T, lds, st, args...);
    else if (ipt <= 8) launch_k(k_select<PACKED, T, 8>, grid, T, lds, st, args...);
    else launch_k(k_select<PACKED, T, SEL_IPT>, grid, T, lds, st, args...);
}

// the small block while the candidates fit 4 per thread and the
// compaction's (slab, wave) counts fit one per thread
static bool select_small(const Plan &p, bool compact) {
    return p.n_src_max <= SEL_SMALL * 4 && (!compact || p.N <= SEL_SMALL * 64);
}

hipError_t launch_select(const Plan &p, const int32_t *units, const float *node_max, const int32_t *node_idx,
                         int32_t *flag, int32_t *mtok, hipStream_t st) {
    {
        StageScope _stage(st, "select");
        const size_t lds = (size_t)p.n_src_max * 4;
        if (select_small(p, false))
            go_sel<false, SEL_SMALL>(cdiv(p.n_src_max, SEL_SMALL), p.n_groups, lds, st, node_max, node_idx,
                                     (unsigned long long *)nullptr, (const float *)nullptr, (float *)nullptr,
                                     (int32_t *)nullptr, group_map(p, units), p.n_groups, p.n_src_max, p.n_dst_max,
                                     flag, mtok, (int32_t *)nullptr, (int32_t *)nullptr, (int32_t *)nullptr, p.N,
                                     p.seq_len, 0, (const int32_t *)nullptr, 0, (const uint4 *)nullptr, 0L,
                                     (uint4 *)nullptr);
        else
            go_sel<false, SEL_LARGE>(cdiv(p.n_src_max, SEL_LARGE), p.n_groups, lds, st, node_max, node_idx,
                                     (unsigned long long *)nullptr, (const float *)nullptr, (float *)nullptr,
                                     (int32_t *)nullptr, group_map(p, units), p.n_groups, p.n_src_max, p.n_dst_max,
                                     flag, mtok, (int32_t *)nullptr, (int32_t *)nullptr, (int32_t *)nullptr, p.N,
                                     p.seq_len, 0, (const int32_t *)nullptr, 0, (const uint4 *)nullptr, 0L,
                                     (uint4 *)nullptr);
    }
    return hipGetLastError();
}

hipError_t launch_select_packed(const Plan &p, const int32_t *units, unsigned long long *node_pack,
                                const float *inv, float *node_max, int32_t *node_idx, int32_t *flag, int32_t *mtok,
                                int32_t *kept_idx, int32_t *cached_idx, int32_t *rmap, hipStream_t st,
                                const int32_t *excl, int clear_pack, const void *wo, void *wo16, long n_wo) {
    const bool compact = kept_idx != nullptr;
    if (compact && !select_compacts(p)) return hipErrorInvalidValue;
    if (compact && excl != nullptr) return hipErrorInvalidValue;   // an excluding selection never compacts
    // Block Cache: sequences of F tokens, n_seq of them
    const int tF = compact && p.kind == KIND_BLOCK ? p.F : 0;
    const int L = tF > 0 ? p.n_seq : p.seq_len;
    {
        StageScope _stage(st, "select");
        const size_t lds = (size_t)p.n_src_max * 4;
        const long n8 = (wo && wo16 && p.bf16) ? n_wo / 8 : 0;
        const bool small = select_small(p, compact);
        const int threads = small ? SEL_SMALL : SEL_LARGE;
        const int cvt_blocks = n8 > 0 ? (int)std::min<long>((n8 + threads - 1) / threads, 2 * N_CUS) : 0;
        const unsigned grid = p.n_groups + cvt_blocks;
        if (small)
            go_sel<true, SEL_SMALL>(cdiv(p.n_src_max, SEL_SMALL), grid, lds, st, (const float *)nullptr,
                                    (const int32_t *)nullptr, node_pack, inv, node_max, node_idx, group_map(p, units),
                                    p.n_groups, p.n_src_max, p.n_dst_max, flag, mtok, kept_idx, cached_idx, rmap, p.N,
                                    L, tF, excl, clear_pack, (const uint4 *)wo, n8, (uint4 *)wo16);
        else
            go_sel<true, SEL_LARGE>(cdiv(p.n_src_max, SEL_LARGE), grid, lds, st, (const float *)nullptr,
                                    (const int32_t *)nullptr, node_pack, inv, node_max, node_idx, group_map(p, units),
                                    p.n_groups, p.n_src_max, p.n_dst_max, flag, mtok, kept_idx, cached_idx, rmap, p.N,
                                    L, tF, excl, clear_pack, (const uint4 *)wo, n8, (uint4 *)wo16);
    }
    return hipGetLastError();
}

}  // namespace oc
