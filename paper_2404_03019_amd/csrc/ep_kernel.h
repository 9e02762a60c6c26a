// Element-parallel segment reduction for gfx950.
//
// The rows are cut into chunks of equal size, one chunk per block and column
// tile, regardless of where segments begin, so the work per block is the same
// for any length distribution (the heavy tails of power-law graphs included).
// Inside a block, each row group (L lanes sharing one row; lane j holds
// columns j*V .. j*V+V-1 of the tile, NT times) takes K consecutive rows and
// reduces them serially in registers, storing every segment that starts and
// ends inside its run with one plain store (the paper's sequential reduction,
// Section III-B, with the N-loop held in registers). The first and last
// segment of each run are then combined across the row groups of the block
// by a segmented scan (the paper's parallel reduction, Algorithm 1, recast):
// inside each wave, DPP row shifts scan the groups of every 16-lane row and
// DPP row broadcasts (or lane shuffles, when a group spans several lanes)
// carry the rows into each other; across the four waves the scan goes
// through LDS. A segment that crosses the block's
// first or last row leaves one partial per block side ("lo" and "hi"); these
// partials are themselves a sorted list of rows with counts, and the same
// kernel reduces them at the next level until one block remains. No atomics,
// no output memset, and the result does not depend on timing.
//
// src / X may be stored as fp32, bf16 or fp16 and the index (and col) as int64
// or int32: the first pass widens on load and reduces in fp32; later passes
// read the fp32 partials. Max may also record, beside every value, its
// recipient: the lowest row (edge) whose term equals it (RED_MAXARG; pairs
// combine by max_arg in common.h through the walk, the scan and the levels).
// Each (storage, index) pair is instantiated in a translation unit of its own
// (ep_<storage>_<index>.hip), which this header is included into.
#pragma once

#include <type_traits>

#include "common.h"

namespace geot {

namespace {

// Rows mode may load the streamed rows non-temporally (NTS). That pays when a
// row group's load covers whole 128-byte lines (measured on MI355X: 9 % on
// 128-byte rows, 10 % on 1 KiB rows, a loss on narrower rows, whose other half
// line the next load wants); it is instantiated only for such tiles. Ids, edge
// metadata and gathered X rows use ordinary loads (non-temporal ones measured
// slower: the ids are reread at block edges, X rows are reused).
template <int MODE, int V, int NT, int L, int E>
constexpr bool nts_eligible() {
    return MODE == SRC_ROWS && (int64_t)L * V * NT * (int64_t)sizeof(typename ElemT<E>::T) >= 128;
}

// One block's work of an element-parallel pass: block `bid` of `nblk`.
template <int RED, int MODE, int V, int NT, int L, int E, typename I, bool NTS>
__device__ __forceinline__ void ep_body(const EpArgs &a, const int64_t bid, const int64_t nblk) {
    constexpr int NV = V * NT;        // floats per lane
    constexpr int GW = 64 / L;        // row groups per wave
    constexpr int NW = kBlock / 64;   // waves per block
    constexpr int G = kBlock / L;     // row groups per block
    constexpr int TW = NT * L * V;    // columns per tile
    // rows loaded ahead per row group: 8 for 4-float lanes with at least 8 lanes a row and for
    // 8-element lanes (16-bit storage), without recipients (the point cloud's mean 0.807 ->
    // 0.786 ms, the power-law graph's sum 2.368 -> 2.353 ms, its bf16 sum 1.42 -> 1.38 ms; 118
    // VGPRs and 4 waves per SIMD instead of 92 and 5), else 4 (8 for narrower lanes)
    constexpr int U = (NV == 4 && L >= 8 || NV == 8) && RED != RED_MAXARG ? 8 : (NV >= 4 ? 4 : 8);
    // edges per batch of the gather pipeline: 8 for 4-float lanes whose group shares the
    // metadata loads (L >= 8) and carries no recipients (the SpMM graph: fp32 sum 5.18 ->
    // 5.14 ms, its gradient w.r.t. X 4.13 -> 4.06 ms), else 4 (8 for narrower lanes; bf16 lanes
    // of 8 elements took 2.80 -> 2.92 ms with 8)
    constexpr int UG = NV == 4 && L >= 8 && RED != RED_MAXARG ? 8 : (NV >= 4 ? 4 : 8);
    // Segment ids fit 32 bits (the host rejects num_segments >= 2^31). Row counts
    // of one block fit 32 bits; partial levels add counts of many blocks: 64 bits.
    using Cnt = typename std::conditional<MODE == SRC_PIECES, int64_t, int32_t>::type;
    static_assert(MODE != SRC_PIECES || (E == ELEM_F32 && std::is_same<I, int64_t>::value),
                  "partials are fp32 with int64 segment ids");
    using T = typename ElemT<E>::T;
    // max with recipients (RED_MAXARG): beside every value, the lowest row (edge; for a
    // partial, the row it carries) whose term equals it
    constexpr bool ARG = RED == RED_MAXARG;
    constexpr int NX = ARG ? NV : 1;   // recipient registers per lane (one unused otherwise)
    const T *src = static_cast<const T *>(a.src);
    const I *idx = static_cast<const I *>(a.idx);
    const I *col = static_cast<const I *>(a.col);
    // gather mode: edge e's id, column and weight sit at [e * ms] (records of ms words), else ms = 1
    const int64_t ms = MODE == SRC_GATHER && a.meta_stride > 1 ? (int64_t)a.meta_stride : 1;

    __shared__ float s_v[NW][TW];
    __shared__ Cnt s_n[NW];
    __shared__ int s_f[NW];
    __shared__ uint32_t s_x[NW][ARG ? TW : 1];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int gw = lane / L;          // row group within the wave
    const int gl = lane - gw * L;     // lane within the row group
    const int g = wave * GW + gw;     // row group within the block

    if constexpr (MODE == SRC_PIECES) {
        // the final level's extra blocks write the runs of empty segments level 0 listed
        const int64_t main_blocks = nblk - a.gap_blocks;
        if (a.gap_blocks > 0 && bid >= main_blocks) {
            gap_fill_rows_body<V>(a.out, a.F, a.ld_out, (int64_t)TW, a.S, a.gaps, bid - main_blocks,
                                  a.gap_blocks, a.arg_out);
            return;
        }
    }
    // tile-major: the blocks in flight share one column tile, so a gather reads one
    // slab of X at a time (the metadata is read once per tile)
    int64_t chunk;
    int tile;
    if (a.tile_major) {
        const int64_t nch = (nblk - (MODE == SRC_PIECES ? (int64_t)a.gap_blocks : 0)) / a.ntiles;
        tile = (int)(bid / nch);
        chunk = bid - (int64_t)tile * nch;
    } else {
        chunk = bid / a.ntiles;
        tile = (int)(bid - chunk * a.ntiles);
    }
    const int64_t bsize = (int64_t)G * a.K;
    const int64_t bstart = chunk * bsize;
    const int64_t bend = min(bstart + bsize, a.n);
    const int64_t r0 = min(bstart + (int64_t)g * a.K, bend);
    const int64_t r1 = min(r0 + (int64_t)a.K, bend);
    const bool has_rows = r0 < r1;

    // Columns of this lane's vectors. Where F is not a multiple of V (fp32 only), the vector
    // that would cross the row's end takes the row's last V columns instead: its loads stay
    // inside the row, and the columns it shares with the previous vector are reduced in the
    // same order by both lanes, so both store the same values.
    int64_t cb[NT];
    bool cv[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        cb[j] = (int64_t)tile * TW + (int64_t)(j * L + gl) * V;
        cv[j] = cb[j] < a.F;
        if (cv[j]) cb[j] = min(cb[j], a.F - V);
    }
    const float neutral = red_neutral<RED>();

    // ---- helpers -------------------------------------------------------
    auto store_seg = [&](int32_t seg, const float *v, Cnt n, const uint32_t *vx) {
        if (MODE == SRC_PIECES && n == 0) return;     // only empty partials: stored elsewhere
        if (seg < 0 || (int64_t)seg >= a.S) return;   // out-of-range id: skip the store
        float *o = a.out + (int64_t)seg * a.ld_out;
        if constexpr (ARG) {
            float *ao = reinterpret_cast<float *>(a.arg_out + (int64_t)seg * a.ld_out);
#pragma unroll
            for (int j = 0; j < NT; ++j) {
                if (!cv[j]) continue;
                float t[V];
#pragma unroll
                for (int k = 0; k < V; ++k) {   // a NaN maximum has none
                    const float m = v[j * V + k];
                    t[k] = __uint_as_float(m != m ? kNoRecipient : vx[j * V + k]);
                }
                store_vec_nt<V>(ao + cb[j], t);
            }
        }
        if (a.mean) {  // uniform across the grid: a scalar branch, no division on the sum path
            const float fn = (float)n;
#pragma unroll
            for (int j = 0; j < NT; ++j) {
                if (!cv[j]) continue;
                float t[V];
#pragma unroll
                for (int k = 0; k < V; ++k) t[k] = v[j * V + k] / fn;
                store_vec_nt<V>(o + cb[j], t);
            }
        } else {
#pragma unroll
            for (int j = 0; j < NT; ++j)
                if (cv[j]) store_vec_nt<V>(o + cb[j], v + j * V);
        }
    };
    // Segments [s_lo, s_hi) have no rows. Short runs are written here by the row
    // group; a longer run goes to the gap list (written afterwards by a grid-wide
    // pass). All lanes of a row group take the same path.
    const int gbase_fill = gw * L;
    auto fill_empty = [&](int64_t s_lo, int64_t s_hi) {
        s_lo = max(s_lo, (int64_t)0);
        s_hi = min(s_hi, a.S);
        if (s_hi - s_lo > kGapRun && gap_push(a.gaps, s_lo, s_hi, tile, gbase_fill, gl, L)) return;
        float z[V], none[V];
#pragma unroll
        for (int k = 0; k < V; ++k) {
            z[k] = 0.0f;
            none[k] = __uint_as_float(kNoRecipient);
        }
        for (int64_t s = s_lo; s < s_hi; ++s) {
            float *o = a.out + s * a.ld_out;
#pragma unroll
            for (int j = 0; j < NT; ++j)
                if (cv[j]) store_vec_nt<V>(o + cb[j], z);
            if constexpr (ARG) {
                float *ao = reinterpret_cast<float *>(a.arg_out + s * a.ld_out);
#pragma unroll
                for (int j = 0; j < NT; ++j)
                    if (cv[j]) store_vec_nt<V>(ao + cb[j], none);
            }
        }
    };
    auto write_partial = [&](int slot, int32_t seg, const float *v, Cnt n, const uint32_t *vx) {
        if (a.pv == nullptr) return;
        const int64_t row = 2 * chunk + slot;
        if (n > 0) {
            float *p = a.pv + row * a.ld_p;
#pragma unroll
            for (int j = 0; j < NT; ++j)
                if (cv[j]) store_vec<V>(p + cb[j], v + j * V);
            if constexpr (ARG) {
                float *px = reinterpret_cast<float *>(a.pix + row * a.ld_p);
#pragma unroll
                for (int j = 0; j < NT; ++j) {
                    if (!cv[j]) continue;
                    float t[V];
#pragma unroll
                    for (int k = 0; k < V; ++k) t[k] = __uint_as_float(vx[j * V + k]);
                    store_vec<V>(px + cb[j], t);
                }
            }
        }
        if (tile == 0 && gl == 0) {
            a.pseg[row] = (int64_t)seg;
            a.pcnt[row] = (int64_t)n;
        }
    };
    // Loads of one row's columns in this tile, as loaded (see Raw); columns
    // outside the tile are not loaded, and widen_term makes them neutral.
    using RV = Raw<E, V>;
    auto load_term = [&](int64_t r, RV *xr, Cnt &c) {
        const T *p = src + r * a.ld_src;
        if constexpr (MODE == SRC_PIECES) {
            // the values load beside the count, not after it: an empty partial's row (never
            // written) is loaded too and made neutral where it is reduced (see `piece`)
            c = (Cnt)a.cnt[r];
#pragma unroll
            for (int j = 0; j < NT; ++j) {
                if (cv[j]) load_raw<E, V>(p + cb[j], xr[j]);
                else for (int k = 0; k < V; ++k) xr[j].v[k] = neutral;  // partials are fp32
            }
        } else {
            c = 1;
#pragma unroll
            for (int j = 0; j < NT; ++j)
                if (cv[j]) load_raw<E, V, NTS>(p + cb[j], xr[j]);
        }
    };
    auto widen_term = [&](const RV *xr, float *x) {
#pragma unroll
        for (int j = 0; j < NT; ++j) {
            if (cv[j]) widen<E, V>(xr[j], x + j * V);
            else for (int k = 0; k < V; ++k) x[j * V + k] = neutral;
        }
    };
    // a partial's terms: neutral when it is empty (count 0), with no recipient
    auto piece = [&](float *x, Cnt c, uint32_t *xi) {
        if constexpr (MODE == SRC_PIECES) {
            if (c == 0) {
#pragma unroll
                for (int k = 0; k < NV; ++k) x[k] = neutral;
#pragma unroll
                for (int k = 0; k < NX; ++k) xi[k] = kNoRecipient;
            }
        }
    };
    // the recipients a partial carries (max with recipients, partial levels): beside its values
    auto load_six = [&](int64_t r, uint32_t *xi) {
        if constexpr (ARG && MODE == SRC_PIECES) {
            const float *p = reinterpret_cast<const float *>(a.six + r * a.ld_src);
#pragma unroll
            for (int j = 0; j < NT; ++j) {
                float t[V];
                if (cv[j]) load_vec<V>(p + cb[j], t);
#pragma unroll
                for (int k = 0; k < V; ++k) xi[j * V + k] = cv[j] ? __float_as_uint(t[k]) : kNoRecipient;
            }
        }
    };

    // ---- serial reduction of this row group's run [r0, r1) --------------
    int32_t first_seg = -1, cur = -1;
    Cnt accn = 0, headn = 0;
    float acc[NV], head[NV];
    uint32_t aix[NX], hix[NX];   // their recipients (max with recipients)
    bool head_done = false;
#pragma unroll
    for (int k = 0; k < NV; ++k) { acc[k] = neutral; head[k] = neutral; }
#pragma unroll
    for (int k = 0; k < NX; ++k) { aix[k] = kNoRecipient; hix[k] = kNoRecipient; }

    // xi: the terms' recipients (the row or edge itself; for a partial, the ones it carries)
    auto step = [&](int32_t s, const float *x, Cnt c, const uint32_t *xi) {
        if (s != cur) {
            if (!head_done) {
#pragma unroll
                for (int k = 0; k < NV; ++k) head[k] = acc[k];
#pragma unroll
                for (int k = 0; k < NX; ++k) hix[k] = aix[k];
                headn = accn;
                head_done = true;
            } else {
                store_seg(cur, acc, accn, aix);  // started and ended inside this run
            }
            if (a.fill_gaps) fill_empty((int64_t)cur + 1, (int64_t)s);
            cur = s;
#pragma unroll
            for (int k = 0; k < NV; ++k) acc[k] = x[k];
            if constexpr (ARG) {
#pragma unroll
                for (int k = 0; k < NV; ++k) aix[k] = xi[k];
            }
            accn = c;
        } else {
            if constexpr (ARG) {
#pragma unroll
                for (int k = 0; k < NV; ++k) max_arg<MODE != SRC_ROWS>(acc[k], aix[k], x[k], xi[k]);
            } else {
#pragma unroll
                for (int k = 0; k < NV; ++k) acc[k] = red_apply<RED>(acc[k], x[k]);
            }
            accn += c;
        }
    };
    // the recipient of a row's (edge's) own terms: the row itself
    auto self_ix = [&](int64_t r, uint32_t *xi) {
#pragma unroll
        for (int k = 0; k < NX; ++k) xi[k] = (uint32_t)r;
    };

    int32_t prev = -1, next = -1;
    if (has_rows) {
        first_seg = (int32_t)idx[r0 * ms];
        cur = first_seg;
        if constexpr (ARG && MODE != SRC_PIECES) {
            // The run's first segment starts from the neutral value: its recipient starts at the
            // run's first row, which the walk reduces first, so a first term equal to the
            // neutral value (-inf) keeps it (the rows walk takes the later side only where it is
            // strictly larger). Partials carry their own recipients and start from none.
#pragma unroll
            for (int k = 0; k < NX; ++k) aix[k] = (uint32_t)r0;
        }
        prev = r0 > 0 ? (int32_t)idx[(r0 - 1) * ms] : -1;
        next = r1 < a.n ? (int32_t)idx[r1 * ms] : -1;

        if constexpr (MODE == SRC_GATHER) {
            // Edge metadata (segment id, source row, weight) of the next UG edges is
            // loaded while the X rows of the current UG edges are in flight, so the
            // dependent gathers never wait behind their own column loads. Rows past
            // r1 are clamped to r1 - 1 (valid addresses) and not reduced.
            // With at least UG lanes per row group, lane u of the group loads the
            // metadata of edge r + u (one coalesced load per array) and every lane
            // reads it back with a lane shuffle; otherwise each lane loads all UG.
            constexpr bool kShared = L >= UG;
            constexpr int UM = kShared ? 1 : UG;
            const int gbase = gw * L;
            int32_t ns[UM];
            I nc[UM];
            float nw[UM];
            auto load_meta = [&](int64_t rb) {
#pragma unroll
                for (int m = 0; m < UM; ++m) {
                    const int64_t rr = min(rb + (kShared ? (int64_t)min(gl, UG - 1) : (int64_t)m), r1 - 1);
                    ns[m] = (int32_t)idx[rr * ms];
                    nc[m] = col[rr * ms];
                    nw[m] = a.w ? a.w[rr * ms] : 1.0f;
                }
            };
            load_meta(r0);
            for (int64_t r = r0; r < r1; r += UG) {
                int32_t s[UG];
                float wt[UG];
                bool okv[UG];
                RV xr[UG][NT];
#pragma unroll
                for (int u = 0; u < UG; ++u) {
                    int64_t c;
                    if constexpr (kShared) {
                        s[u] = __shfl(ns[0], gbase + u, 64);
                        wt[u] = __shfl(nw[0], gbase + u, 64);
                        if constexpr (sizeof(I) == 8) {
                            const int lo = __shfl((int)(uint32_t)(uint64_t)nc[0], gbase + u, 64);
                            const int hi = __shfl((int)(uint32_t)((uint64_t)nc[0] >> 32), gbase + u, 64);
                            c = (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint64_t)(uint32_t)lo);
                        } else {
                            c = (int64_t)__shfl((int)nc[0], gbase + u, 64);
                        }
                    } else {
                        s[u] = ns[u];
                        wt[u] = nw[u];
                        c = (int64_t)nc[u];
                    }
                    // an out-of-range column reads row 0 and contributes the neutral value
                    okv[u] = (uint64_t)c < (uint64_t)a.num_x_rows;
                    const T *p = src + (okv[u] ? c : 0) * a.ld_src;
#pragma unroll
                    for (int j = 0; j < NT; ++j)
                        if (cv[j]) load_raw<E, V>(p + cb[j], xr[u][j]);
                }
                if (r + UG < r1) load_meta(r + UG);
#pragma unroll
                for (int u = 0; u < UG; ++u) {
                    if (r + u < r1) {
                        float x[NV];
                        widen_term(xr[u], x);
#pragma unroll
                        for (int k = 0; k < NV; ++k) x[k] = okv[u] ? wt[u] * x[k] : neutral;
                        uint32_t xi[NX];
                        self_ix(okv[u] ? r + u : (int64_t)kNoRecipient, xi);
                        step(s[u], x, 1, xi);
                    }
                }
            }
        } else if constexpr (MODE == SRC_ROWS && L >= U) {
            // Lane u of the row group loads the segment id of row r + u (one
            // coalesced load per batch, one batch ahead); the group reads the ids
            // back with lane shuffles. Rows past r1 are clamped and not reduced.
            const int gbase = gw * L;
            const int lu = min(gl, U - 1);
            int32_t nid = (int32_t)idx[min(r0 + lu, r1 - 1)];
            for (int64_t r = r0; r < r1; r += U) {
                const int32_t id = nid;
                RV xr[U][NT];
                Cnt c;
#pragma unroll
                for (int u = 0; u < U; ++u) load_term(min(r + u, r1 - 1), xr[u], c);
                if (r + U < r1) nid = (int32_t)idx[min(r + U + lu, r1 - 1)];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int32_t su = __shfl(id, gbase + u, 64);
                    if (r + u < r1) {
                        float x[NV];
                        widen_term(xr[u], x);
                        uint32_t xi[NX];
                        self_ix(r + u, xi);
                        step(su, x, 1, xi);
                    }
                }
            }
        } else {
            int64_t r = r0;
            for (; r + U <= r1; r += U) {
                int32_t s[U];
                Cnt c[U];
                RV xr[U][NT];
                uint32_t xi[U][NX];
#pragma unroll
                for (int u = 0; u < U; ++u) s[u] = (int32_t)idx[r + u];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    load_term(r + u, xr[u], c[u]);
                    if constexpr (MODE == SRC_PIECES) load_six(r + u, xi[u]);
                    else self_ix(r + u, xi[u]);
                }
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    float x[NV];
                    widen_term(xr[u], x);
                    piece(x, c[u], xi[u]);
                    step(s[u], x, c[u], xi[u]);
                }
            }
            for (; r < r1; ++r) {
                RV xr[NT];
                float x[NV];
                uint32_t xi[NX];
                Cnt c;
                const int32_t s = (int32_t)idx[r];
                load_term(r, xr, c);
                if constexpr (MODE == SRC_PIECES) load_six(r, xi);
                else self_ix(r, xi);
                widen_term(xr, x);
                piece(x, c, xi);
                step(s, x, c, xi);
            }
        }
        // empty segments before this run (written after the row loop, so the first loads of
        // the loop do not wait for the neighbour's id) and, for the last run, after it
        if (a.fill_gaps) fill_empty((int64_t)prev + 1, (int64_t)first_seg);
        if (a.fill_gaps && r1 == a.n) fill_empty((int64_t)cur + 1, a.S);
    }
    const bool single_run = !head_done;  // the run holds one segment only: head == tail
    if (single_run) {
#pragma unroll
        for (int k = 0; k < NV; ++k) head[k] = acc[k];
#pragma unroll
        for (int k = 0; k < NX; ++k) hix[k] = aix[k];
        headn = accn;
    }
    const int32_t last_seg = cur;
    const bool starts = has_rows && prev != first_seg;     // first segment begins at r0
    const bool ends_tail = has_rows && next != last_seg;   // last segment ends at r1 - 1

    // ---- segmented scan of the run tails across row groups --------------
    // Element of group g: (flag = a segment begins inside the run, tail partial, tail count).
    // (f1, v1, n1) (+) (f2, v2, n2) = (f1 | f2, f2 ? v2 : v1 (+) v2, f2 ? n2 : n1 + n2).
    bool f = has_rows && (starts || !single_run);
    float v[NV];
    uint32_t vx[NX];   // recipients of v (max with recipients)
    Cnt n = has_rows ? accn : 0;
#pragma unroll
    for (int k = 0; k < NV; ++k) v[k] = acc[k];
#pragma unroll
    for (int k = 0; k < NX; ++k) vx[k] = aix[k];
    // (f, v, n) absorbs the element (fo, vo, no) of an earlier group when `take`
    auto absorb = [&](bool take, int fo, const float *vo, Cnt no, const uint32_t *vxo) {
        if (take) {
            if (!f) {
                if constexpr (ARG) {
#pragma unroll
                    for (int k = 0; k < NV; ++k) {
                        float t = vo[k];
                        uint32_t ti = vxo[k];
                        max_arg<true>(t, ti, v[k], vx[k]);
                        v[k] = t;
                        vx[k] = ti;
                    }
                } else {
#pragma unroll
                    for (int k = 0; k < NV; ++k) v[k] = red_apply<RED>(vo[k], v[k]);
                }
                n += no;
            }
            f = f || (fo != 0);
        }
    };
    // DPP step inside 16-lane rows: take the group S lanes below, if it is in this row
    auto dpp_row_step = [&](auto shift_tag) {
        constexpr int S = decltype(shift_tag)::value;
        float vo[NV];
        uint32_t vxo[NX];
#pragma unroll
        for (int k = 0; k < NV; ++k) vo[k] = dpp_f<kDppRowShr + S, 0xf>(v[k]);
        if constexpr (ARG) {
#pragma unroll
            for (int k = 0; k < NX; ++k) vxo[k] = (uint32_t)dpp_i<kDppRowShr + S, 0xf>((int)vx[k]);
        }
        const int fo = dpp_i<kDppRowShr + S, 0xf>((int)f);
        const Cnt no = dpp_cnt<kDppRowShr + S, 0xf>(n);
        absorb((lane & 15) >= S, fo, vo, no, vxo);
    };
    if constexpr (L < 16) {
        // 1. segmented scan of the groups of each 16-lane row with DPP row shifts
        if constexpr (1 * L < 16) dpp_row_step(std::integral_constant<int, 1 * L>{});
        if constexpr (2 * L < 16) dpp_row_step(std::integral_constant<int, 2 * L>{});
        if constexpr (4 * L < 16) dpp_row_step(std::integral_constant<int, 4 * L>{});
        if constexpr (8 * L < 16) dpp_row_step(std::integral_constant<int, 8 * L>{});
        // 2. rows absorb the last group of earlier rows
        const int row = lane >> 4;
        if constexpr (L == 1) {
            {   // lane 15 -> row 1, lane 47 -> row 3
                float vo[NV];
                uint32_t vxo[NX];
#pragma unroll
                for (int k = 0; k < NV; ++k) vo[k] = dpp_f<kDppRowBcast15, 0xa>(v[k]);
                if constexpr (ARG) {
#pragma unroll
                    for (int k = 0; k < NX; ++k) vxo[k] = (uint32_t)dpp_i<kDppRowBcast15, 0xa>((int)vx[k]);
                }
                const int fo = dpp_i<kDppRowBcast15, 0xa>((int)f);
                const Cnt no = dpp_cnt<kDppRowBcast15, 0xa>(n);
                absorb((row & 1) != 0, fo, vo, no, vxo);
            }
            {   // lane 31 -> rows 2 and 3
                float vo[NV];
                uint32_t vxo[NX];
#pragma unroll
                for (int k = 0; k < NV; ++k) vo[k] = dpp_f<kDppRowBcast31, 0xc>(v[k]);
                if constexpr (ARG) {
#pragma unroll
                    for (int k = 0; k < NX; ++k) vxo[k] = (uint32_t)dpp_i<kDppRowBcast31, 0xc>((int)vx[k]);
                }
                const int fo = dpp_i<kDppRowBcast31, 0xc>((int)f);
                const Cnt no = dpp_cnt<kDppRowBcast31, 0xc>(n);
                absorb(row >= 2, fo, vo, no, vxo);
            }
        } else {
#pragma unroll
            for (int dr = 1; dr <= 2; dr <<= 1) {   // previous row, then two rows back
                const int src = max(row - dr, 0) * 16 + 16 - L + gl;
                float vo[NV];
                uint32_t vxo[NX];
#pragma unroll
                for (int k = 0; k < NV; ++k) vo[k] = shfl_f(v[k], src);
                if constexpr (ARG) {
#pragma unroll
                    for (int k = 0; k < NX; ++k) vxo[k] = (uint32_t)shfl_i((int)vx[k], src);
                }
                const int fo = shfl_i((int)f, src);
                const Cnt no = shfl_cnt(n, src);
                absorb(row >= dr, fo, vo, no, vxo);
            }
        }
    } else {
        // groups of 16 or more lanes: Hillis-Steele over groups with lane shuffles
#pragma unroll
        for (int d = 1; d < GW; d <<= 1) {
            const int fo = shfl_up_i((int)f, d * L);
            const Cnt no = shfl_up_cnt(n, d * L);
            float vo[NV];
            uint32_t vxo[NX];
#pragma unroll
            for (int k = 0; k < NV; ++k) vo[k] = shfl_up_f(v[k], d * L);
            if constexpr (ARG) {
#pragma unroll
                for (int k = 0; k < NX; ++k) vxo[k] = (uint32_t)shfl_up_i((int)vx[k], d * L);
            }
            absorb(gw >= d, fo, vo, no, vxo);
        }
    }
    if (gw == GW - 1) {
#pragma unroll
        for (int j = 0; j < NT; ++j)
#pragma unroll
            for (int k = 0; k < V; ++k) s_v[wave][(j * L + gl) * V + k] = v[j * V + k];
        if constexpr (ARG) {
#pragma unroll
            for (int j = 0; j < NT; ++j)
#pragma unroll
                for (int k = 0; k < V; ++k) s_x[wave][(j * L + gl) * V + k] = vx[j * V + k];
        }
        if (gl == 0) {
            s_n[wave] = n;
            s_f[wave] = (int)f;
        }
    }
    __syncthreads();

    // exclusive prefix of this group: waves before this one, then groups before it in the wave
    bool ef = false;
    float ev[NV];
    uint32_t ex[NX];
    Cnt en = 0;
#pragma unroll
    for (int k = 0; k < NV; ++k) ev[k] = neutral;
#pragma unroll
    for (int k = 0; k < NX; ++k) ex[k] = kNoRecipient;
    for (int w2 = 0; w2 < wave; ++w2) {
        const bool f2 = s_f[w2] != 0;
        const Cnt n2 = s_n[w2];
#pragma unroll
        for (int j = 0; j < NT; ++j)
#pragma unroll
            for (int k = 0; k < V; ++k) {
                const float x2 = s_v[w2][(j * L + gl) * V + k];
                if constexpr (ARG) {
                    const uint32_t i2 = s_x[w2][(j * L + gl) * V + k];
                    if (f2) {
                        ev[j * V + k] = x2;
                        ex[j * V + k] = i2;
                    } else {
                        max_arg<true>(ev[j * V + k], ex[j * V + k], x2, i2);
                    }
                } else {
                    ev[j * V + k] = f2 ? x2 : red_apply<RED>(ev[j * V + k], x2);
                }
            }
        en = f2 ? n2 : en + n2;
        ef = ef || f2;
    }
    {
        const int fo = shfl_up_i((int)f, L);
        const Cnt no = shfl_up_cnt(n, L);
        float vo[NV];
        uint32_t vxo[NX];
#pragma unroll
        for (int k = 0; k < NV; ++k) vo[k] = shfl_up_f(v[k], L);
        if constexpr (ARG) {
#pragma unroll
            for (int k = 0; k < NX; ++k) vxo[k] = (uint32_t)shfl_up_i((int)vx[k], L);
        }
        if (gw > 0) {
            if constexpr (ARG) {
#pragma unroll
                for (int k = 0; k < NV; ++k) {
                    if (fo) {
                        ev[k] = vo[k];
                        ex[k] = vxo[k];
                    } else {
                        max_arg<true>(ev[k], ex[k], vo[k], vxo[k]);
                    }
                }
            } else {
#pragma unroll
                for (int k = 0; k < NV; ++k) ev[k] = fo ? vo[k] : red_apply<RED>(ev[k], vo[k]);
            }
            en = fo ? no : en + no;
            ef = ef || (fo != 0);
        }
    }

    // ---- finish the head and tail segments of the run -------------------
    if (has_rows) {
        const bool last_group = (r1 == bend);
        bool hi_written = false;
        // value of the run's first segment including what precedes it in the block
        float hv[NV];
        uint32_t hx[NX];
        Cnt hn;
        bool h_in_block;
        if (starts) {
#pragma unroll
            for (int k = 0; k < NV; ++k) hv[k] = head[k];
#pragma unroll
            for (int k = 0; k < NX; ++k) hx[k] = hix[k];
            hn = headn;
            h_in_block = true;
        } else {
            if constexpr (ARG) {
#pragma unroll
                for (int k = 0; k < NV; ++k) {
                    hv[k] = ev[k];
                    hx[k] = ex[k];
                    max_arg<true>(hv[k], hx[k], head[k], hix[k]);
                }
            } else {
#pragma unroll
                for (int k = 0; k < NV; ++k) hv[k] = red_apply<RED>(ev[k], head[k]);
            }
            hn = en + headn;
            h_in_block = ef;
        }
        if (!single_run) {
            // the first segment ends inside the run
            if (h_in_block) store_seg(first_seg, hv, hn, hx);
            else write_partial(0, first_seg, hv, hn, hx);
            // the last segment began inside the run
            if (ends_tail) {
                store_seg(last_seg, acc, accn, aix);
            } else if (last_group) {
                write_partial(1, last_seg, acc, accn, aix);
                hi_written = true;
            }
        } else if (ends_tail) {
            if (h_in_block) store_seg(first_seg, hv, hn, hx);
            else write_partial(0, first_seg, hv, hn, hx);
        } else if (last_group) {
            write_partial(h_in_block ? 1 : 0, first_seg, hv, hn, hx);
            hi_written = h_in_block;
        }
        // empty partials keep the list of partials sorted and complete
        if (g == 0 && starts && a.pv != nullptr && tile == 0 && gl == 0) {
            a.pseg[2 * chunk] = (int64_t)first_seg;
            a.pcnt[2 * chunk] = 0;
        }
        if (last_group && !hi_written && a.pv != nullptr && tile == 0 && gl == 0) {
            a.pseg[2 * chunk + 1] = (int64_t)last_seg;
            a.pcnt[2 * chunk + 1] = 0;
        }
    }
}

template <int RED, int MODE, int V, int NT, int L, int E, typename I, bool NTS>
__global__ __launch_bounds__(kBlock) void ep_kernel(const EpArgs a) {
    ep_body<RED, MODE, V, NT, L, E, I, NTS>(a, blockIdx.x, gridDim.x);
}

template <int RED, int MODE, int V, int NT, int L, int E, typename I>
hipError_t launch_one(const EpArgs &a, int64_t nchunks, hipStream_t stream) {
    const int64_t blocks = nchunks * a.ntiles + (MODE == SRC_PIECES ? (int64_t)a.gap_blocks : 0);
    if (blocks <= 0) return hipSuccess;
    if (blocks > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    if (a.nt_rows) {
        if constexpr (nts_eligible<MODE, V, NT, L, E>())
            hipLaunchKernelGGL((ep_kernel<RED, MODE, V, NT, L, E, I, true>), dim3((unsigned)blocks), dim3(kBlock),
                               0, stream, a);
        else
            return hipErrorInvalidValue;
    } else {
        hipLaunchKernelGGL((ep_kernel<RED, MODE, V, NT, L, E, I, false>), dim3((unsigned)blocks), dim3(kBlock), 0,
                           stream, a);
    }
    return hipGetLastError();
}

template <int RED, int MODE, int V, int NT, int E, typename I>
hipError_t by_lanes(const EpArgs &a, int L, int64_t nchunks, hipStream_t st) {
    if constexpr (NT > 1) {
        if (L != 64) return hipErrorInvalidValue;
        return launch_one<RED, MODE, V, NT, 64, E, I>(a, nchunks, st);
    } else {
        switch (L) {
            case 1: return launch_one<RED, MODE, V, 1, 1, E, I>(a, nchunks, st);
            case 2: return launch_one<RED, MODE, V, 1, 2, E, I>(a, nchunks, st);
            case 4: return launch_one<RED, MODE, V, 1, 4, E, I>(a, nchunks, st);
            case 8: return launch_one<RED, MODE, V, 1, 8, E, I>(a, nchunks, st);
            case 16: return launch_one<RED, MODE, V, 1, 16, E, I>(a, nchunks, st);
            case 32: return launch_one<RED, MODE, V, 1, 32, E, I>(a, nchunks, st);
            case 64:
                if constexpr (V == 8) return hipErrorInvalidValue;
                else return launch_one<RED, MODE, V, 1, 64, E, I>(a, nchunks, st);
            default: return hipErrorInvalidValue;
        }
    }
}

template <int RED, int MODE, int E, typename I>
hipError_t by_shape(const EpArgs &a, int V, int NT, int L, int64_t nchunks, hipStream_t st) {
    if constexpr (E != ELEM_F32) {  // 16-byte loads of 16-bit storage, at most 32 lanes
        if (V == 8 && NT == 1) {
            if (L > 32) return hipErrorInvalidValue;
            return by_lanes<RED, MODE, 8, 1, E, I>(a, L, nchunks, st);
        }
    }
    if (V == 4 && NT == 1) return by_lanes<RED, MODE, 4, 1, E, I>(a, L, nchunks, st);
    if constexpr (E == ELEM_F32) {  // three-float rows (F = 3), one lane a row
        if (V == 3 && NT == 1) {
            if (L != 1) return hipErrorInvalidValue;
            return launch_one<RED, MODE, 3, 1, 1, E, I>(a, nchunks, st);
        }
    }
    if (V == 2 && NT == 1) return by_lanes<RED, MODE, 2, 1, E, I>(a, L, nchunks, st);
    if (V == 2 && NT == 2) return by_lanes<RED, MODE, 2, 2, E, I>(a, L, nchunks, st);
    if (V == 1 && NT == 1) return by_lanes<RED, MODE, 1, 1, E, I>(a, L, nchunks, st);
    if (V == 1 && NT == 2) return by_lanes<RED, MODE, 1, 2, E, I>(a, L, nchunks, st);
    if (V == 1 && NT == 4) return by_lanes<RED, MODE, 1, 4, E, I>(a, L, nchunks, st);
    return hipErrorInvalidValue;
}

// The first-pass modes (rows, gather) for storage E and index I; the partial
// levels (fp32 partials, int64 ids) only where PIECES is set.
template <int E, typename I, bool PIECES>
hipError_t ep_dispatch(const EpArgs &a, int red, int mode, int V, int NT, int L, int64_t nchunks,
                       hipStream_t st) {
    if (red == RED_SUM) {
        if (mode == SRC_ROWS) return by_shape<RED_SUM, SRC_ROWS, E, I>(a, V, NT, L, nchunks, st);
        if (mode == SRC_GATHER) return by_shape<RED_SUM, SRC_GATHER, E, I>(a, V, NT, L, nchunks, st);
        if constexpr (PIECES)
            if (mode == SRC_PIECES) return by_shape<RED_SUM, SRC_PIECES, E, I>(a, V, NT, L, nchunks, st);
    } else if (red == RED_MAX) {
        if (mode == SRC_ROWS) return by_shape<RED_MAX, SRC_ROWS, E, I>(a, V, NT, L, nchunks, st);
        if (mode == SRC_GATHER) return by_shape<RED_MAX, SRC_GATHER, E, I>(a, V, NT, L, nchunks, st);
        if constexpr (PIECES)
            if (mode == SRC_PIECES) return by_shape<RED_MAX, SRC_PIECES, E, I>(a, V, NT, L, nchunks, st);
    } else if (red == RED_MAXARG) {
        if (mode == SRC_ROWS) return by_shape<RED_MAXARG, SRC_ROWS, E, I>(a, V, NT, L, nchunks, st);
        if (mode == SRC_GATHER) return by_shape<RED_MAXARG, SRC_GATHER, E, I>(a, V, NT, L, nchunks, st);
        if constexpr (PIECES)
            if (mode == SRC_PIECES) return by_shape<RED_MAXARG, SRC_PIECES, E, I>(a, V, NT, L, nchunks, st);
    }
    return hipErrorInvalidValue;
}

}  // namespace
}  // namespace geot
