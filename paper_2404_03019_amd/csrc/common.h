// Device helpers shared by the reduction kernels: vector loads/stores of 1, 2
// or 4 floats, the reduction operator and lane shuffles.
#pragma once

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "internal.h"

namespace geot {

template <int RED>
__device__ __forceinline__ float red_neutral() {
    return RED == RED_SUM ? 0.0f : -INFINITY;
}

// Max is the IEEE 754-2019 maximum operation: a NaN operand gives NaN, and +0 ranks
// above -0. It is commutative and associative, so the result of a segment does not
// depend on the order in which its rows are combined (v_maximum3_f32 on gfx950, one
// instruction, where fmaxf drops NaN and leaves the sign of a zero to the order).
template <int RED>
__device__ __forceinline__ float red_apply(float a, float b) {
    if constexpr (RED == RED_SUM) {
        return a + b;
    } else {
        return __builtin_elementwise_maximum(a, b);
    }
}

// Max with recipients: (v, i), the maximum of some terms and the lowest row among them whose
// term equals it, takes in (b, ib) from LATER rows (every combine does: the walk goes up the
// rows, the scan and the levels take earlier groups and partials into later ones). The later
// side's row counts only where its value is larger: equal values (+0 and -0 compare equal)
// keep the earlier, lower row. A side with no recipient (an empty partial: the neutral value)
// yields to the other, which is checked only where one can occur (NONE_OK). NaN maxima are
// not tracked here: NaN propagates in the value, and the store writes no recipient for it.
// The result is the recipient rule of the max gradients, whatever the schedule.
template <bool NONE_OK>
__device__ __forceinline__ void max_arg(float &v, uint32_t &i, float b, uint32_t ib) {
    const bool later = b > v || (NONE_OK && i == kNoRecipient);
    i = later ? ib : i;
    v = __builtin_elementwise_maximum(v, b);
}

// fp32 vectors of 2, 3 and 4 elements that need only 4-byte alignment. gfx950 loads and
// stores them with one dwordx2 / x3 / x4 instruction at any 4-byte aligned address, so a
// row of odd width (rows at F * 4 bytes) still moves in whole vectors: a lane whose
// vector would cross the end of the row takes the last V columns instead (overlapping
// its neighbour's, which it computes identically).
typedef float f32x2_t __attribute__((ext_vector_type(2), aligned(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4), aligned(4)));
struct f32x3_t {
    float x, y, z;
};
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

template <int V>
__device__ __forceinline__ void load_vec(const float *p, float *x) {
    if constexpr (V == 4) {
        const f32x4_t t = *reinterpret_cast<const f32x4_t *>(p);
        x[0] = t.x; x[1] = t.y; x[2] = t.z; x[3] = t.w;
    } else if constexpr (V == 3) {
        const f32x3_t t = *reinterpret_cast<const f32x3_t *>(p);
        x[0] = t.x; x[1] = t.y; x[2] = t.z;
    } else if constexpr (V == 2) {
        const f32x2_t t = *reinterpret_cast<const f32x2_t *>(p);
        x[0] = t.x; x[1] = t.y;
    } else {
        x[0] = *p;
    }
}

// Non-temporal loads (the `nt` cache policy): for data read exactly once, such
// as streamed rows and ids, which then does not displace data that is reused.

template <bool NT, typename T>
__device__ __forceinline__ T ld(const T *p) {
    if constexpr (NT) return __builtin_nontemporal_load(p);
    else return *p;
}

template <int V, bool NT>
__device__ __forceinline__ void load_vec_p(const float *p, float *x) {
    if constexpr (!NT) {
        load_vec<V>(p, x);
    } else if constexpr (V == 4) {
        const f32x4_t t = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t *>(p));
        x[0] = t.x; x[1] = t.y; x[2] = t.z; x[3] = t.w;
    } else if constexpr (V == 3) {
        x[0] = __builtin_nontemporal_load(p);
        x[1] = __builtin_nontemporal_load(p + 1);
        x[2] = __builtin_nontemporal_load(p + 2);
    } else if constexpr (V == 2) {
        const f32x2_t t = __builtin_nontemporal_load(reinterpret_cast<const f32x2_t *>(p));
        x[0] = t.x; x[1] = t.y;
    } else {
        x[0] = __builtin_nontemporal_load(p);
    }
}

template <int V>
__device__ __forceinline__ void store_vec(float *p, const float *x) {
    if constexpr (V == 8) {  // 16-bit storage loads 8 elements per lane; fp32 results go out as 2 x 16 B
        *reinterpret_cast<float4 *>(p) = make_float4(x[0], x[1], x[2], x[3]);
        *reinterpret_cast<float4 *>(p + 4) = make_float4(x[4], x[5], x[6], x[7]);
    } else if constexpr (V == 4) {
        *reinterpret_cast<f32x4_t *>(p) = f32x4_t{x[0], x[1], x[2], x[3]};
    } else if constexpr (V == 3) {
        *reinterpret_cast<f32x3_t *>(p) = f32x3_t{x[0], x[1], x[2]};
    } else if constexpr (V == 2) {
        *reinterpret_cast<f32x2_t *>(p) = f32x2_t{x[0], x[1]};
    } else {
        *p = x[0];
    }
}

// Non-temporal stores (the `nt` cache policy) of the output rows, which are written once
// and not read again by the kernel that writes them: on MI355X they cost the streaming
// reads around them less than ordinary stores (the point-cloud workload, 16-row segments of
// 64 floats, 268 MB written beside 4.4 GB read: 859 -> 803 us; the SpMM workload 5.26 ->
// 5.18 ms).
template <int V>
__device__ __forceinline__ void store_vec_nt(float *p, const float *x) {
    if constexpr (V == 8) {
        __builtin_nontemporal_store(f32x4_t{x[0], x[1], x[2], x[3]}, reinterpret_cast<f32x4_t *>(p));
        __builtin_nontemporal_store(f32x4_t{x[4], x[5], x[6], x[7]}, reinterpret_cast<f32x4_t *>(p + 4));
    } else if constexpr (V == 4) {
        __builtin_nontemporal_store(f32x4_t{x[0], x[1], x[2], x[3]}, reinterpret_cast<f32x4_t *>(p));
    } else if constexpr (V == 2) {
        __builtin_nontemporal_store(f32x2_t{x[0], x[1]}, reinterpret_cast<f32x2_t *>(p));
    } else {
#pragma unroll
        for (int k = 0; k < V; ++k) __builtin_nontemporal_store(x[k], p + k);
    }
}

// Storage types: src / X elements are widened to fp32 when loaded. A bf16 value
// is the upper half of the fp32 with the same value; fp16 converts exactly.
template <int E> struct ElemT;
template <> struct ElemT<ELEM_F32> { using T = float; };
template <> struct ElemT<ELEM_BF16> { using T = uint16_t; };
template <> struct ElemT<ELEM_F16> { using T = _Float16; };

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// V consecutive elements as loaded: the fp32 values themselves, or the 32-bit
// words that hold 16-bit elements. Loads fill these; rows are widened where
// they are reduced, so only the loaded words occupy registers while loads are
// in flight.
template <int E, int V> struct Raw { float v[V]; };
template <int V> struct Raw<ELEM_BF16, V> { uint32_t w[(V + 1) / 2]; };
template <int V> struct Raw<ELEM_F16, V> { uint32_t w[(V + 1) / 2]; };

// V consecutive elements at p (aligned to V elements); NT: non-temporal load
template <int E, int V, bool NT = false>
__device__ __forceinline__ void load_raw(const typename ElemT<E>::T *p, Raw<E, V> &r) {
    if constexpr (E == ELEM_F32) {
        load_vec_p<V, NT>(p, r.v);
    } else if constexpr (V == 8) {
        const u32x4_t t = ld<NT>(reinterpret_cast<const u32x4_t *>(p));
        r.w[0] = t.x; r.w[1] = t.y; r.w[2] = t.z; r.w[3] = t.w;
    } else if constexpr (V == 4) {
        const u32x2_t t = ld<NT>(reinterpret_cast<const u32x2_t *>(p));
        r.w[0] = t.x; r.w[1] = t.y;
    } else if constexpr (V == 2) {
        r.w[0] = ld<NT>(reinterpret_cast<const uint32_t *>(p));
    } else {
        r.w[0] = (uint32_t)ld<NT>(reinterpret_cast<const uint16_t *>(p));
    }
}

// element k of a word pair: the low half comes first in memory
template <int E, int V>
__device__ __forceinline__ void widen(const Raw<E, V> &r, float *x) {
#pragma unroll
    for (int k = 0; k < V; ++k) {
        if constexpr (E == ELEM_F32) {
            x[k] = r.v[k];
        } else if constexpr (E == ELEM_BF16) {
            x[k] = (k & 1) ? bf16_hi(r.w[k / 2]) : bf16_lo(r.w[k / 2]);
        } else {
            const uint16_t h = (uint16_t)((k & 1) ? (r.w[k / 2] >> 16) : (r.w[k / 2] & 0xffffu));
            x[k] = (float)__builtin_bit_cast(_Float16, h);
        }
    }
}

// Value of `v` held by lane (lane - delta) of the wave; lanes below `delta`
// get their own value back (callers mask them). ds_bpermute underneath.
__device__ __forceinline__ float shfl_up_f(float v, int delta) {
    return __shfl_up(v, (unsigned)delta, 64);
}

__device__ __forceinline__ int shfl_up_i(int v, int delta) {
    return __shfl_up(v, (unsigned)delta, 64);
}

__device__ __forceinline__ int64_t shfl_up_i64(int64_t v, int delta) {
    const int lo = __shfl_up((int)(uint32_t)(uint64_t)v, (unsigned)delta, 64);
    const int hi = __shfl_up((int)(uint32_t)((uint64_t)v >> 32), (unsigned)delta, 64);
    return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint64_t)(uint32_t)lo);
}

__device__ __forceinline__ int32_t shfl_up_cnt(int32_t v, int delta) { return shfl_up_i(v, delta); }
__device__ __forceinline__ int64_t shfl_up_cnt(int64_t v, int delta) { return shfl_up_i64(v, delta); }

// Appends the run of segments [lo, hi) (value carried along) to a gap list,
// cut into records of 2^kGapChunkLog2 segments, or of the least power of two
// that cuts it into at most 2^kGapMaxRecsLog2 records (so no run needs more
// slots than that). Runs are shorter than 2^31 (num_segments < 2^31) and longer
// than kGapRun, so the cut takes 32-bit shifts, no division (which would hold
// registers in the loops this is inlined into). `lanes` lanes starting at lane
// `lead` (all in the same state) call it together; the lead lane takes the
// slots and the lanes share the writes. Returns false when the list is full:
// the caller then writes the run itself (the slots it took hold empty records).
__device__ __forceinline__ bool gap_push(const GapList &g, int64_t lo, int64_t hi, int64_t value,
                                         int lead, int lane_in, int lanes) {
    const unsigned len = (unsigned)(hi - lo);
    const int sh = max(kGapChunkLog2, (32 - __clz((int)(len - 1u))) - kGapMaxRecsLog2);  // ceil(log2 len) - 6
    const unsigned nrec = (unsigned)(((uint64_t)len + ((uint64_t)1 << sh) - 1u) >> sh);
    unsigned base = 0;
    if (lane_in == 0) base = atomicAdd(g.count, nrec);
    if (lanes > 1) base = (unsigned)__shfl((int)base, lead, 64);
    const bool fits = (uint64_t)base + nrec <= (uint64_t)kGapCap;
    const unsigned end = fits ? nrec : (kGapCap > base ? kGapCap - base : 0u);
    for (unsigned q = (unsigned)lane_in; q < end; q += (unsigned)lanes) {
        int64_t *r = g.rec + 3 * ((int64_t)base + q);
        const int64_t a = fits ? lo + ((int64_t)q << sh) : 0;
        r[0] = a;
        r[1] = fits ? min(hi, a + ((int64_t)1 << sh)) : 0;
        r[2] = value;
    }
    return fits;
}

// A fill block's record count: read once per block, before the block takes
// its ticket (so before the list can be reset).
__device__ __forceinline__ unsigned gap_count(const GapList &g) {
    __shared__ unsigned s_cnt;
    if (threadIdx.x == 0) s_cnt = min(*g.count, kGapCap);
    __syncthreads();
    return s_cnt;
}

// A fill block is done. Only the blocks that read records (blk < cnt: the
// first min(cnt, nblk) of the pass) take a ticket, and the last of them empties
// the list; each read the count before taking its ticket, so before the reset.
// A block that reads the count after the reset sees 0, and is one with no
// record under the true count either. An empty list costs no atomic.
__device__ __forceinline__ void gap_done(const GapList &g, int64_t blk, int64_t nblk, unsigned cnt) {
    if (blk >= (int64_t)cnt) return;
    const int64_t parts = min((int64_t)cnt, nblk);
    __syncthreads();
    if (threadIdx.x == 0) {
        __threadfence();
        const unsigned t = atomicAdd(g.ticket, 1u);
        if ((int64_t)t == parts - 1) {
            atomicExch(g.count, 0u);
            atomicExch(g.ticket, 0u);
        }
    }
}

// One block's share of the gap-list fill: records q = blk, blk + nblk, ...;
// rows [first, end) of record q's column tile (tiles of `tw` columns) = 0,
// clamped to `rows`. The pass's last block empties the list.
template <int V>
__device__ __forceinline__ void gap_fill_rows_body(float *out, int64_t F, int64_t ld, int64_t tw, int64_t rows,
                                                   const GapList &g, int64_t blk, int64_t nblk,
                                                   uint32_t *arg = nullptr) {
    const unsigned cnt = gap_count(g);
    float z[V], none[V];   // arg (max with recipients): empty rows have none
#pragma unroll
    for (int k = 0; k < V; ++k) {
        z[k] = 0.0f;
        none[k] = __uint_as_float(kNoRecipient);
    }
    for (int64_t q = blk; q < (int64_t)cnt; q += nblk) {
        const int64_t *r = g.rec + 3 * q;
        const int64_t lo = max(r[0], (int64_t)0), hi = min(r[1], rows);
        const int64_t c0 = r[2] * tw;
        const int64_t ncol = min(tw, F - c0);
        if (hi <= lo || c0 < 0 || ncol <= 0) continue;
        const int nvec = (int)((ncol + V - 1) / V);
        int tpr = 1;  // threads per row (power of two)
        while (tpr < nvec && tpr < 256) tpr <<= 1;
        const int rows_per_pass = 256 / tpr;
        const int j0 = threadIdx.x % tpr;
        for (int64_t row = lo + threadIdx.x / tpr; row < hi; row += rows_per_pass) {
            float *o = out + row * ld;
            // a vector that would pass the row's end takes its last V columns (all zero)
            for (int j = j0; j < nvec; j += tpr) {
                const int64_t c = min(c0 + (int64_t)j * V, F - V);
                store_vec<V>(o + c, z);
                if (arg) store_vec<V>(reinterpret_cast<float *>(arg + row * ld + c), none);
            }
        }
    }
    gap_done(g, blk, nblk, cnt);
}

// DPP lane moves (GFX9 encodings): row_shr:S shifts within each 16-lane row;
// row_bcast:15 / row_bcast:31 broadcast lane 15 of a row (lane 31) to the
// next row (rows 2 and 3). Lanes whose source does not exist keep their own
// value; callers decide by lane position which lanes use the result.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ int dpp_i(int v) {
    return __builtin_amdgcn_update_dpp(v, v, CTRL, ROW_MASK, 0xf, false);
}

template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_f(float v) {
    return __int_as_float(dpp_i<CTRL, ROW_MASK>(__float_as_int(v)));
}

template <int CTRL, int ROW_MASK>
__device__ __forceinline__ int32_t dpp_cnt(int32_t v) {
    return dpp_i<CTRL, ROW_MASK>(v);
}

template <int CTRL, int ROW_MASK>
__device__ __forceinline__ int64_t dpp_cnt(int64_t v) {
    const int lo = dpp_i<CTRL, ROW_MASK>((int)(uint32_t)(uint64_t)v);
    const int hi = dpp_i<CTRL, ROW_MASK>((int)(uint32_t)((uint64_t)v >> 32));
    return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint64_t)(uint32_t)lo);
}

constexpr int kDppRowShr = 0x110;     // + shift (1..15)
constexpr int kDppRowBcast15 = 0x142;
constexpr int kDppRowBcast31 = 0x143;

__device__ __forceinline__ float shfl_f(float v, int src) { return __shfl(v, src, 64); }
__device__ __forceinline__ int shfl_i(int v, int src) { return __shfl(v, src, 64); }
__device__ __forceinline__ int32_t shfl_cnt(int32_t v, int src) { return __shfl(v, src, 64); }
__device__ __forceinline__ int64_t shfl_cnt(int64_t v, int src) {
    const int lo = __shfl((int)(uint32_t)(uint64_t)v, src, 64);
    const int hi = __shfl((int)(uint32_t)((uint64_t)v >> 32), src, 64);
    return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint64_t)(uint32_t)lo);
}

__device__ __forceinline__ float shfl_down_f(float v, int delta) {
    return __shfl_down(v, (unsigned)delta, 64);
}

}  // namespace geot
