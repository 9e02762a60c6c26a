// Gradients of segment reduction and of the fused gather-weight form.
//
// Every kernel here is a row- (or edge-) parallel stream. A thread owns one
// V-float vector of one row: `tpr` threads (a power of two) cover a row, and a
// block covers kPasses passes of 256 / tpr consecutive rows: one contiguous
// range, with as many blocks as the rows need and no grid-stride loop. The
// resident blocks then read and write one compact window of addresses (on
// MI355X a one-shot 16 GiB store reaches 6.9 TB/s, a grid-stride loop 5.5).
// Consecutive rows share their segment, so the per-segment operands
// (grad_out, out, the max recipients) stay in cache.
//
// Max routes each (segment, feature) gradient to the first member attaining
// the forward maximum: one pass takes the minimum row index of the attaining
// members with 64-bit atomicMin (order-independent, so deterministic), the
// next pass writes the gradients.
#include <algorithm>
#include <type_traits>

#include "common.h"

namespace geot {

namespace {

constexpr int kPasses = 4;  // passes of one block over its rows
constexpr int kWPasses8 = 2;   // the same for the weight gradient with 8-element vectors
constexpr int kArgPasses = 2;  // the same for the fused max recipients

struct RowMap {
    int tpr;      // threads per row
    int rsub;     // this thread's row within a pass
    int j0;       // this thread's first vector
    int rows;     // rows per pass of one block
    int passes;   // passes of one block
    __device__ int64_t row(int q) const {  // this thread's row in pass q
        return ((int64_t)blockIdx.x * passes + q) * rows + rsub;
    }
};

__device__ __forceinline__ RowMap row_map(int nvec, int passes = kPasses) {
    RowMap m;
    m.passes = passes;
    int t = 1;
    while (t < nvec && t < 64) t <<= 1;
    m.tpr = t;
    m.rsub = threadIdx.x / t;
    m.j0 = threadIdx.x % t;
    m.rows = 256 / t;
    return m;
}

// V fp32 gradient values (8 as two 16-byte loads)
template <int V>
__device__ __forceinline__ void load_f32(const float *p, float *x) {
    if constexpr (V == 8) {
        load_vec<4>(p, x);
        load_vec<4>(p + 4, x + 4);
    } else {
        load_vec<V>(p, x);
    }
}

// Two fp32 values narrowed to storage type E, rounded to nearest even (a NaN stays a NaN),
// packed low first. gfx950 converts the pair in one instruction (v_cvt_pk_bf16_f32,
// v_cvt_pk_f16_f32); a rounding written out in integer operations compiled to a branch per
// element around its NaN case, and held bf16 gradient stores of the power-law graph at 4.7 TB/s.
template <int E>
__device__ __forceinline__ uint32_t narrow_pair(float a, float b) {
    const f32x2_t v = {a, b};
    if constexpr (E == ELEM_BF16) {
        typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
        return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
    } else {
        typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
        return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, f16x2_t));
    }
}

// one value stored with the non-temporal cache policy (NT) or an ordinary store
template <bool NT, typename T>
__device__ __forceinline__ void put(T *p, T v) {
    if constexpr (NT) __builtin_nontemporal_store(v, p);
    else *p = v;
}

// V fp32 values stored as V elements of storage type E at p (aligned to V elements), with
// non-temporal stores when NT
template <int E, int V, bool NT = false>
__device__ __forceinline__ void store_elems(typename ElemT<E>::T *p, const float *x) {
    if constexpr (E == ELEM_F32) {
        if constexpr (NT) store_vec_nt<V>(p, x);
        else store_vec<V>(p, x);
    } else if constexpr (V == 1) {
        put<NT>(reinterpret_cast<uint16_t *>(p), (uint16_t)narrow_pair<E>(x[0], 0.0f));
    } else {
        uint32_t w[V / 2];
#pragma unroll
        for (int k = 0; k < V / 2; ++k) w[k] = narrow_pair<E>(x[2 * k], x[2 * k + 1]);
        if constexpr (V == 8) {
            put<NT>(reinterpret_cast<u32x4_t *>(p), u32x4_t{w[0], w[1], w[2], w[3]});
        } else if constexpr (V == 4) {
            put<NT>(reinterpret_cast<u32x2_t *>(p), u32x2_t{w[0], w[1]});
        } else {
            put<NT>(reinterpret_cast<uint32_t *>(p), w[0]);
        }
    }
}

// grad_src[i] = grad_out[idx[i]] (times 1 / len for mean), stored in the source's type E.
// The ids of all the block's passes load first, so their latency overlaps; then the rows.
template <int E, typename I, int V, bool MEAN>
__global__ __launch_bounds__(256) void seg_bwd_bcast_kernel(const float *__restrict__ gout,
                                                            const I *__restrict__ idx,
                                                            const int64_t *__restrict__ off, int64_t n,
                                                            int64_t S, int64_t F,
                                                            typename ElemT<E>::T *__restrict__ gsrc) {
    const int nvec = (int)(F / V);
    const RowMap m = row_map(nvec);
    int64_t seg[kPasses];
#pragma unroll
    for (int q = 0; q < kPasses; ++q) {
        const int64_t i = m.row(q);
        seg[q] = i < n ? (int64_t)idx[i] : -1;
    }
    // mean: every pass's segment starts load together, branchless (a segment out of range
    // reads segment 0's), before the first gradient row
    int64_t o0[kPasses], o1[kPasses];
    if (MEAN) {
#pragma unroll
        for (int q = 0; q < kPasses; ++q) {
            const int64_t s = (uint64_t)seg[q] < (uint64_t)S ? seg[q] : 0;
            o0[q] = off[s];
            o1[q] = off[s + 1];
        }
    }
    if (nvec <= m.tpr) {
        // one vector per thread and row: every pass's gradient row loads before the first store
        // (one memory latency per block instead of one per pass)
        if (m.j0 >= nvec) return;
        float x[kPasses][V];
#pragma unroll
        for (int q = 0; q < kPasses; ++q) {
            const bool ok = m.row(q) < n && (uint64_t)seg[q] < (uint64_t)S;
            if (ok) {
                load_f32<V>(gout + seg[q] * F + (int64_t)m.j0 * V, x[q]);
            } else {
#pragma unroll
                for (int k = 0; k < V; ++k) x[q][k] = 0.0f;
            }
        }
#pragma unroll
        for (int q = 0; q < kPasses; ++q) {
            const int64_t i = m.row(q);
            if (i >= n) break;
            if (MEAN && (uint64_t)seg[q] < (uint64_t)S) {
                const float inv = 1.0f / (float)(o1[q] - o0[q]);
#pragma unroll
                for (int k = 0; k < V; ++k) x[q][k] = x[q][k] * inv;
            }
            store_elems<E, V>(gsrc + i * F + (int64_t)m.j0 * V, x[q]);
        }
        return;
    }
#pragma unroll
    for (int q = 0; q < kPasses; ++q) {
        const int64_t i = m.row(q);
        if (i < n) {
            const int64_t s = seg[q];
            const bool ok = (uint64_t)s < (uint64_t)S;
            float inv = 1.0f;
            if (MEAN && ok) inv = 1.0f / (float)(o1[q] - o0[q]);
            for (int j = m.j0; j < nvec; j += m.tpr) {
                float x[V];
                if (ok) {
                    load_f32<V>(gout + s * F + (int64_t)j * V, x);
                    if (MEAN) {
#pragma unroll
                        for (int k = 0; k < V; ++k) x[k] = x[k] * inv;
                    }
                } else {
#pragma unroll
                    for (int k = 0; k < V; ++k) x[k] = 0.0f;
                }
                store_elems<E, V>(gsrc + i * F + (int64_t)j * V, x);
            }
        }
    }
}

// Segments of a thread's rows taken from the offsets instead of the ids. The offsets pass
// stores the ids of every block's first and last rows (first[2b], first[2b + 1]). A block that
// lies in one segment needs nothing more; another stages off[first[2b] .. first[2b] + 255] in
// LDS (s_off, 256 entries) and each row finds its segment there by binary search. A row past
// the staged starts (a block with more than 255 segment ends) or in a block whose first id is
// out of range reads its id. seg[q] is the segment of m.row(q) (-1 past the last row); with
// MEAN, inv[q] is 1 / its length. Returns whether the block lies in one segment (then every
// seg[q] of a row before n is the same). Holds a barrier where the block spans several segments
// (a condition uniform over the block).
template <typename I, bool MEAN>
__device__ __forceinline__ bool segments_from_offsets(const RowMap &m, const I *__restrict__ idx,
                                                      const int64_t *__restrict__ off,
                                                      const int64_t *__restrict__ first, int64_t n, int64_t S,
                                                      int64_t *s_off, int64_t (&seg)[kPasses],
                                                      float (&inv)[kPasses]) {
    constexpr int K = 256;
    const longlong2 ends = *reinterpret_cast<const longlong2 *>(first + 2 * (int64_t)blockIdx.x);
    const int64_t seg0 = ends.x;
    const bool valid = (uint64_t)seg0 < (uint64_t)S;
    const bool one = valid && ends.y == seg0;
    if (one) {
        float in = 1.0f;
        if (MEAN) in = 1.0f / (float)(off[seg0 + 1] - off[seg0]);
#pragma unroll
        for (int q = 0; q < kPasses; ++q) {
            seg[q] = m.row(q) < n ? seg0 : -1;
            inv[q] = in;
        }
        return true;
    }
    if (valid) {
        s_off[threadIdx.x] = off[min(seg0 + (int64_t)threadIdx.x, S)];
        __syncthreads();
    }
    // the block's rows lie in segments seg0 .. ends.y, so the first staged start above a row
    // is one of the first ends.y - seg0 + 1 (a search over all 256 took the bf16 gradient of
    // the power-law graph 1.61 ms instead of 1.47)
    const int span = (int)min((int64_t)K, max((int64_t)1, ends.y - seg0 + 1));
#pragma unroll
    for (int q = 0; q < kPasses; ++q) {
        const int64_t i = m.row(q);
        seg[q] = -1;
        inv[q] = 1.0f;
        if (i >= n) continue;
        int p = K;   // first staged start above row i
        if (valid) {
            int lo = 1, hi = span;
            while (lo < hi) {
                const int mid = (lo + hi) >> 1;
                if (s_off[mid] > i) hi = mid;
                else lo = mid + 1;
            }
            p = lo;
        }
        if (p < K) {
            seg[q] = seg0 + p - 1;
            if (MEAN) inv[q] = 1.0f / (float)(s_off[p] - s_off[p - 1]);
        } else {
            seg[q] = (int64_t)idx[i];
            if (MEAN && (uint64_t)seg[q] < (uint64_t)S) inv[q] = 1.0f / (float)(off[seg[q] + 1] - off[seg[q]]);
        }
    }
    return false;
}

// The broadcast gradient with the segments from the offsets. The offsets and the gradient rows
// stay in cache, so the kernel's HBM traffic is its stores alone: the ids, 6 % of the bytes at
// F = 32, read in among the stores, slowed the stream by a third.
template <int E, typename I, int V, bool MEAN>
__global__ __launch_bounds__(256) void seg_bwd_bcast_off_kernel(const float *__restrict__ gout,
                                                                const I *__restrict__ idx,
                                                                const int64_t *__restrict__ off,
                                                                const int64_t *__restrict__ first, int64_t n,
                                                                int64_t S, int64_t F,
                                                                typename ElemT<E>::T *__restrict__ gsrc) {
    __shared__ int64_t s_off[256];
    // non-temporal stores, except for the fp32 sum: on the power-law graph they take the
    // bf16 sum 1.47 -> 1.24 ms and the fp32 mean 2.54 -> 2.50 ms, but the fp32 sum
    // 2.46 -> 2.63 ms
    constexpr bool kNt = E != ELEM_F32 || MEAN;
    const int nvec = (int)(F / V);
    const RowMap m = row_map(nvec);
    int64_t seg[kPasses];
    float inv[kPasses];
    if (segments_from_offsets<I, MEAN>(m, idx, off, first, n, S, s_off, seg, inv)) {
        // one segment: each vector of its gradient row loads once for all the thread's rows
        if (m.row(0) >= n) return;   // no row here (seg[0] is -1)
        for (int j = m.j0; j < nvec; j += m.tpr) {
            float x[V];
            load_f32<V>(gout + seg[0] * F + (int64_t)j * V, x);
            if (MEAN) {
#pragma unroll
                for (int k = 0; k < V; ++k) x[k] = x[k] * inv[0];
            }
#pragma unroll
            for (int q = 0; q < kPasses; ++q) {
                const int64_t i = m.row(q);
                if (i >= n) break;
                store_elems<E, V, kNt>(gsrc + i * F + (int64_t)j * V, x);
            }
        }
        return;
    }
    for (int j = m.j0; j < nvec; j += m.tpr) {
        float x[kPasses][V];
#pragma unroll
        for (int q = 0; q < kPasses; ++q) {
            if ((uint64_t)seg[q] < (uint64_t)S) {
                load_f32<V>(gout + seg[q] * F + (int64_t)j * V, x[q]);
            } else {
#pragma unroll
                for (int k = 0; k < V; ++k) x[q][k] = 0.0f;
            }
        }
#pragma unroll
        for (int q = 0; q < kPasses; ++q) {
            const int64_t i = m.row(q);
            if (i >= n) break;
            if (MEAN) {
#pragma unroll
                for (int k = 0; k < V; ++k) x[q][k] = x[q][k] * inv[q];
            }
            store_elems<E, V, kNt>(gsrc + i * F + (int64_t)j * V, x[q]);
        }
    }
}

// Recipient vectors: V consecutive entries of a recipient table of 32- or 64-bit row numbers
// (16-byte loads where V entries fill them; entries at a multiple of V)
template <typename A, int V>
__device__ __forceinline__ void load_arg(const A *a, A (&w)[V]) {
    if constexpr (sizeof(A) == 8 && V >= 2) {
#pragma unroll
        for (int k = 0; k < V; k += 2) {
            const ulonglong2 t = *reinterpret_cast<const ulonglong2 *>(a + k);
            w[k] = t.x;
            w[k + 1] = t.y;
        }
    } else if constexpr (sizeof(A) == 4 && V >= 4) {
#pragma unroll
        for (int k = 0; k < V; k += 4) {
            const uint4 t = *reinterpret_cast<const uint4 *>(a + k);
            w[k] = t.x;
            w[k + 1] = t.y;
            w[k + 2] = t.z;
            w[k + 3] = t.w;
        }
    } else if constexpr (sizeof(A) == 4 && V == 2) {
        const uint2 t = *reinterpret_cast<const uint2 *>(a);
        w[0] = t.x;
        w[1] = t.y;
    } else {
#pragma unroll
        for (int k = 0; k < V; ++k) w[k] = a[k];
    }
}

// arg[s, f] = min row i of segment s with src[i, f] == out[s, f]. The ids of all passes
// load first, then every pass's row and output vector, then the compares (one memory
// latency per step, not per pass).
template <int E, typename I, int V, typename A>
__global__ __launch_bounds__(256) void seg_bwd_max_arg_kernel(const typename ElemT<E>::T *__restrict__ src,
                                                              const I *__restrict__ idx,
                                                              const float *__restrict__ out, int64_t n, int64_t S,
                                                              int64_t F, A *arg) {
    const int nvec = (int)(F / V);
    const RowMap m = row_map(nvec);
    int64_t seg[kPasses];
#pragma unroll
    for (int q = 0; q < kPasses; ++q) {
        const int64_t i = m.row(q);
        seg[q] = i < n ? (int64_t)idx[i] : -1;
    }
    if (nvec <= m.tpr) {  // one vector per thread and row
        float x[kPasses][V], o[kPasses][V];
        bool ok[kPasses];
#pragma unroll
        for (int q = 0; q < kPasses; ++q) {
            ok[q] = m.row(q) < n && (uint64_t)seg[q] < (uint64_t)S && m.j0 < nvec;
            if (ok[q]) {
                Raw<E, V> r;
                load_raw<E, V>(src + m.row(q) * F + (int64_t)m.j0 * V, r);
                widen<E, V>(r, x[q]);
                load_f32<V>(out + seg[q] * F + (int64_t)m.j0 * V, o[q]);
            }
        }
#pragma unroll
        for (int q = 0; q < kPasses; ++q) {
            if (!ok[q]) continue;
#pragma unroll
            for (int k = 0; k < V; ++k)
                if (x[q][k] == o[q][k])
                    atomicMin(arg + seg[q] * F + (int64_t)m.j0 * V + k, (A)m.row(q));
        }
        return;
    }
    for (int q = 0; q < kPasses; ++q) {
        const int64_t i = m.row(q);
        const int64_t s = seg[q];
        if (i >= n || (uint64_t)s >= (uint64_t)S) continue;
        for (int j = m.j0; j < nvec; j += m.tpr) {
            float x[V], o[V];
            Raw<E, V> r;
            load_raw<E, V>(src + i * F + (int64_t)j * V, r);
            widen<E, V>(r, x);
            load_f32<V>(out + s * F + (int64_t)j * V, o);
#pragma unroll
            for (int k = 0; k < V; ++k)
                if (x[k] == o[k]) atomicMin(arg + s * F + (int64_t)j * V + k, (A)i);
        }
    }
}

// The recipients with the segments from the offsets (as the broadcast above). The rows of src
// load first (non-temporal: each is read once), before the segments are known, so that the
// stream does not wait for the segment lookup; the outputs they are compared with follow (once
// per thread where the block lies in one segment).
template <int E, typename I, int V, typename A>
__global__ __launch_bounds__(256) void seg_bwd_max_arg_off_kernel(const typename ElemT<E>::T *__restrict__ src,
                                                                  const I *__restrict__ idx,
                                                                  const int64_t *__restrict__ off,
                                                                  const int64_t *__restrict__ first,
                                                                  const float *__restrict__ out, int64_t n,
                                                                  int64_t S, int64_t F, A *arg) {
    __shared__ int64_t s_off[256];
    const int nvec = (int)(F / V);
    const RowMap m = row_map(nvec);
    int64_t seg[kPasses];
    float inv[kPasses];
    if (nvec <= m.tpr) {  // one vector per thread and row
        const bool lane = m.j0 < nvec;
        Raw<E, V> r[kPasses];
#pragma unroll
        for (int q = 0; q < kPasses; ++q)
            if (lane && m.row(q) < n) load_raw<E, V, true>(src + m.row(q) * F + (int64_t)m.j0 * V, r[q]);
        const bool one = segments_from_offsets<I, false>(m, idx, off, first, n, S, s_off, seg, inv);
        if (!lane) return;
        float o[kPasses][V];
        if (one) {
            if (m.row(0) >= n) return;   // no row here (seg[0] is -1)
            load_f32<V>(out + seg[0] * F + (int64_t)m.j0 * V, o[0]);
#pragma unroll
            for (int q = 1; q < kPasses; ++q)
#pragma unroll
                for (int k = 0; k < V; ++k) o[q][k] = o[0][k];
        } else {
#pragma unroll
            for (int q = 0; q < kPasses; ++q)
                if ((uint64_t)seg[q] < (uint64_t)S) load_f32<V>(out + seg[q] * F + (int64_t)m.j0 * V, o[q]);
        }
#pragma unroll
        for (int q = 0; q < kPasses; ++q) {
            if ((uint64_t)seg[q] >= (uint64_t)S) continue;   // past the last row, or an id out of range
            float x[V];
            widen<E, V>(r[q], x);
            // the matching features as a bit mask, then one atomic per set bit: a branch per
            // row, not per feature (bf16 / int32 on the power-law graph 3.14 -> 3.08 ms)
            unsigned hit = 0u;
#pragma unroll
            for (int k = 0; k < V; ++k) hit |= (x[k] == o[q][k] ? 1u : 0u) << k;
            while (hit) {
                const int k = __builtin_ctz(hit);
                hit &= hit - 1u;
                atomicMin(arg + seg[q] * F + (int64_t)m.j0 * V + k, (A)m.row(q));
            }
        }
        return;
    }
    segments_from_offsets<I, false>(m, idx, off, first, n, S, s_off, seg, inv);
    for (int q = 0; q < kPasses; ++q) {
        const int64_t i = m.row(q);
        const int64_t s = seg[q];
        if (i >= n || (uint64_t)s >= (uint64_t)S) continue;
        for (int j = m.j0; j < nvec; j += m.tpr) {
            float x[V], o[V];
            Raw<E, V> r;
            load_raw<E, V, true>(src + i * F + (int64_t)j * V, r);
            widen<E, V>(r, x);
            load_f32<V>(out + s * F + (int64_t)j * V, o);
#pragma unroll
            for (int k = 0; k < V; ++k)
                if (x[k] == o[k]) atomicMin(arg + s * F + (int64_t)j * V + k, (A)i);
        }
    }
}

// grad_src[i, f] = grad_out[s, f] where i is the recipient of (s, f), else 0; ids first,
// then every pass's gradient and recipient vectors, then the stores
template <int E, typename I, int V, typename A>
__global__ __launch_bounds__(256) void seg_bwd_max_write_kernel(const float *__restrict__ gout,
                                                                const I *__restrict__ idx,
                                                                const A *__restrict__ arg,
                                                                int64_t n, int64_t S, int64_t F,
                                                                typename ElemT<E>::T *__restrict__ gsrc) {
    const int nvec = (int)(F / V);
    const RowMap m = row_map(nvec);
    int64_t seg[kPasses];
#pragma unroll
    for (int q = 0; q < kPasses; ++q) {
        const int64_t i = m.row(q);
        seg[q] = i < n ? (int64_t)idx[i] : -1;
    }
    if (nvec <= m.tpr) {
        float x[kPasses][V];
        A w[kPasses][V];
#pragma unroll
        for (int q = 0; q < kPasses; ++q) {
            const bool ok = (uint64_t)seg[q] < (uint64_t)S && m.j0 < nvec;
            if (ok) {
                load_f32<V>(gout + seg[q] * F + (int64_t)m.j0 * V, x[q]);
                load_arg<A, V>(arg + seg[q] * F + (int64_t)m.j0 * V, w[q]);
            } else {
#pragma unroll
                for (int k = 0; k < V; ++k) {
                    x[q][k] = 0.0f;
                    w[q][k] = (A)~(A)0;
                }
            }
        }
#pragma unroll
        for (int q = 0; q < kPasses; ++q) {
            const int64_t i = m.row(q);
            if (i >= n || m.j0 >= nvec) continue;
#pragma unroll
            for (int k = 0; k < V; ++k)
                if (w[q][k] != (A)i) x[q][k] = 0.0f;
            store_elems<E, V>(gsrc + i * F + (int64_t)m.j0 * V, x[q]);
        }
        return;
    }
    for (int q = 0; q < kPasses; ++q) {
        const int64_t i = m.row(q);
        if (i >= n) break;
        const int64_t s = seg[q];
        const bool ok = (uint64_t)s < (uint64_t)S;
        for (int j = m.j0; j < nvec; j += m.tpr) {
            float x[V];
            if (ok) {
                load_f32<V>(gout + s * F + (int64_t)j * V, x);
#pragma unroll
                for (int k = 0; k < V; ++k)
                    if (arg[s * F + (int64_t)j * V + k] != (A)i) x[k] = 0.0f;
            } else {
#pragma unroll
                for (int k = 0; k < V; ++k) x[k] = 0.0f;
            }
            store_elems<E, V>(gsrc + i * F + (int64_t)j * V, x);
        }
    }
}

// The max gradient's stores with the segments from the offsets (as the broadcast above): the
// recipients and gradient rows stay in cache, so the stores are the kernel's HBM stream, and
// they are non-temporal (the power-law graph: fp32 4.87 -> 4.80 ms, bf16 3.33 -> 3.13 ms).
template <int E, typename I, int V, typename A>
__global__ __launch_bounds__(256) void seg_bwd_max_write_off_kernel(const float *__restrict__ gout,
                                                                    const I *__restrict__ idx,
                                                                    const int64_t *__restrict__ off,
                                                                    const int64_t *__restrict__ first,
                                                                    const A *__restrict__ arg,
                                                                    int64_t n, int64_t S, int64_t F,
                                                                    typename ElemT<E>::T *__restrict__ gsrc) {
    __shared__ int64_t s_off[256];
    const int nvec = (int)(F / V);
    const RowMap m = row_map(nvec);
    int64_t seg[kPasses];
    float inv[kPasses];
    if (segments_from_offsets<I, false>(m, idx, off, first, n, S, s_off, seg, inv)) {
        // one segment: its gradient and recipient vectors load once for all the thread's rows
        if (m.row(0) >= n) return;   // no row here (seg[0] is -1)
        for (int j = m.j0; j < nvec; j += m.tpr) {
            float x[V];
            A w[V];
            load_f32<V>(gout + seg[0] * F + (int64_t)j * V, x);
            load_arg<A, V>(arg + seg[0] * F + (int64_t)j * V, w);
#pragma unroll
            for (int q = 0; q < kPasses; ++q) {
                const int64_t i = m.row(q);
                if (i >= n) break;
                float y[V];
#pragma unroll
                for (int k = 0; k < V; ++k) y[k] = w[k] == (A)i ? x[k] : 0.0f;
                store_elems<E, V, true>(gsrc + i * F + (int64_t)j * V, y);
            }
        }
        return;
    }
    // several segments: two passes' vectors in flight at a time (all four held the 16-bit kernel
    // at 108 VGPRs, 4 waves per SIMD, for the single-segment path as well)
    constexpr int QB = 2;
    for (int j = m.j0; j < nvec; j += m.tpr) {
#pragma unroll
        for (int q0 = 0; q0 < kPasses; q0 += QB) {
            float x[QB][V];
            A w[QB][V];
#pragma unroll
            for (int u = 0; u < QB; ++u) {
                const int q = q0 + u;
                if ((uint64_t)seg[q] < (uint64_t)S) {
                    load_f32<V>(gout + seg[q] * F + (int64_t)j * V, x[u]);
                    load_arg<A, V>(arg + seg[q] * F + (int64_t)j * V, w[u]);
                } else {
#pragma unroll
                    for (int k = 0; k < V; ++k) {
                        x[u][k] = 0.0f;
                        w[u][k] = (A)~(A)0;
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < QB; ++u) {
                const int64_t i = m.row(q0 + u);
                if (i >= n) break;
#pragma unroll
                for (int k = 0; k < V; ++k)
                    if (w[u][k] != (A)i) x[u][k] = 0.0f;
                store_elems<E, V, true>(gsrc + i * F + (int64_t)j * V, x[u]);
            }
        }
    }
}

// fused form, max: arg[r, f] = min edge e of row r whose rounded product equals out[r, f].
// Ids of all passes first, then every pass's X and output vectors, then the compares.
template <int E, typename I, int V, typename A, int P>
__global__ __launch_bounds__(256) void gs_bwd_max_arg_kernel(const typename ElemT<E>::T *__restrict__ X, int64_t nx,
                                                             const I *__restrict__ col,
                                                             const float *__restrict__ w,
                                                             const I *__restrict__ row,
                                                             const float *__restrict__ out, int64_t n, int64_t R,
                                                             int64_t F, A *arg) {
    const int nvec = (int)(F / V);
    const RowMap m = row_map(nvec, P);
    // Slot of this thread's edge q among the block's P * rows consecutive edges: a row group
    // takes P consecutive edges, which mostly share their output row, loaded once per run (SpMM
    // graph, the three max passes: bf16 / int32 26.9 -> 25.6 ms; fp32 27.0 -> 27.3 ms, which
    // edges rows apart measured the same with this code)
    auto slot_of = [&](int q) { return m.rsub * P + q; };
    auto edge = [&](int q) { return (int64_t)blockIdx.x * P * m.rows + slot_of(q); };
    int64_t rr[P], cc[P];
    float wt[P];
#pragma unroll
    for (int q = 0; q < P; ++q) {
        const int64_t e = edge(q);
        rr[q] = e < n ? (int64_t)row[e] : -1;
        cc[q] = e < n ? (int64_t)col[e] : -1;
        wt[q] = e < n && w ? w[e] : 1.0f;
    }
    if (nvec <= m.tpr) {
        // The block's edges are the consecutive slots (slot_of). For each (row, column) the
        // block's lowest matching slot is found with LDS atomics (the slot where the row starts in
        // the block keys the table); only that slot stores. A row that lies wholly in this block
        // stores its recipient plainly; a row that continues into the previous or next block takes
        // the lowest edge over the blocks with a global atomicMin. With sorted rows this equals the
        // plain rule (the lowest attaining edge); the global atomics are about one per row end.
        __shared__ unsigned s_min[P * 256 * V];   // slots * columns <= P * 256 * V
        __shared__ int64_t s_row[P * 256];
        const int slots = P * m.rows, ncol = nvec * V;
        const int64_t e0 = (int64_t)blockIdx.x * slots;   // edge of slot 0
        for (int t = threadIdx.x; t < slots * ncol; t += 256) s_min[t] = 0xffffffffu;
        if (m.j0 == 0) {
#pragma unroll
            for (int q = 0; q < P; ++q)   // slots past the last edge sort after every row
                s_row[slot_of(q)] = edge(q) < n ? rr[q] : INT64_MAX;
        }
        const bool has_prev = e0 > 0, has_next = e0 + slots < n;
        const int64_t prev_row = has_prev ? (int64_t)row[e0 - 1] : 0;
        const int64_t next_row = has_next ? (int64_t)row[e0 + slots] : 0;
        // X rows of every edge, and the output row once per run of edges with the same row
        Raw<E, V> rx[P];
        float o[P][V];
        bool ok[P], lead[P];
#pragma unroll
        for (int q = 0; q < P; ++q) {
            ok[q] = (uint64_t)rr[q] < (uint64_t)R && (uint64_t)cc[q] < (uint64_t)nx && m.j0 < nvec;
            lead[q] = !(q > 0 && ok[q - 1] && rr[q] == rr[q - 1]);
            if (ok[q]) load_raw<E, V>(X + cc[q] * F + (int64_t)m.j0 * V, rx[q]);
            if (ok[q] && lead[q]) load_f32<V>(out + rr[q] * F + (int64_t)m.j0 * V, o[q]);
        }
        __syncthreads();
        float cur[V];
        unsigned hit[P];   // bit k: column j0 * V + k of this pass's edge attains the maximum
        int rs[P];         // slot where this pass's row starts in the block
#pragma unroll
        for (int q = 0; q < P; ++q) {
            hit[q] = 0;
            rs[q] = 0;
            if (!ok[q]) continue;
            if (lead[q]) {
#pragma unroll
                for (int k = 0; k < V; ++k) cur[k] = o[q][k];
            }
            float x[V];
            widen<E, V>(rx[q], x);
            const int slot = slot_of(q);
            int lo = 0, hi = slot;   // lowest slot holding this row (s_row[slot] is it)
            while (lo < hi) {
                const int mid = (lo + hi) >> 1;
                if (s_row[mid] < rr[q]) lo = mid + 1;
                else hi = mid;
            }
            rs[q] = lo;
#pragma unroll
            for (int k = 0; k < V; ++k) {
                const float t = w ? wt[q] * x[k] : x[k];  // the forward's term: one rounded product
                if (t == cur[k]) {
                    hit[q] |= 1u << k;
                    atomicMin(&s_min[lo * ncol + m.j0 * V + k], (unsigned)slot);
                }
            }
        }
        __syncthreads();
#pragma unroll
        for (int q = 0; q < P; ++q) {
            if (!hit[q]) continue;
            const int slot = slot_of(q);
            const bool shared_row = (has_prev && prev_row == rr[q]) || (has_next && next_row == rr[q]);
#pragma unroll
            for (int k = 0; k < V; ++k) {
                if (!(hit[q] >> k & 1u) || s_min[rs[q] * ncol + m.j0 * V + k] != (unsigned)slot) continue;
                A *a = arg + rr[q] * F + (int64_t)m.j0 * V + k;
                if (shared_row) atomicMin(a, (A)edge(q));
                else *a = (A)edge(q);
            }
        }
        return;
    }
    for (int q = 0; q < P; ++q) {
        const int64_t e = edge(q);
        const int64_t r = rr[q], c = cc[q];
        if (e >= n || (uint64_t)r >= (uint64_t)R || (uint64_t)c >= (uint64_t)nx) continue;
        for (int j = m.j0; j < nvec; j += m.tpr) {
            float x[V], o[V];
            Raw<E, V> rx;
            load_raw<E, V>(X + c * F + (int64_t)j * V, rx);
            widen<E, V>(rx, x);
            load_f32<V>(out + r * F + (int64_t)j * V, o);
#pragma unroll
            for (int k = 0; k < V; ++k) {
                const float t = w ? wt[q] * x[k] : x[k];
                if (t == o[k]) atomicMin(arg + r * F + (int64_t)j * V + k, (A)e);
            }
        }
    }
}

// fused form, max, w.r.t. X: one thread per V-vector of a row r of the recipients; for each
// (r, f) with a recipient edge e, grad_X[col[e], f] += coef(e) * grad_out[r, f]. Walks the
// R * F recipients once (arg and grad_out stream) instead of every edge's row of them.
template <typename I, int V, typename A>
__global__ __launch_bounds__(256) void gs_bwd_x_max_kernel(const A *__restrict__ arg,
                                                           const I *__restrict__ col, int64_t nx,
                                                           const float *__restrict__ w,
                                                           const float *__restrict__ gout, int64_t n,
                                                           int64_t R, int64_t F, float *gX) {
    const int nvec = (int)(F / V);
    const RowMap m = row_map(nvec);
    for (int q = 0; q < kPasses; ++q) {
        const int64_t r = m.row(q);
        if (r >= R) break;
        for (int j = m.j0; j < nvec; j += m.tpr) {
            float g[V];
            A a[V];
            load_f32<V>(gout + r * F + (int64_t)j * V, g);
            load_arg<A, V>(arg + r * F + (int64_t)j * V, a);
#pragma unroll
            for (int k = 0; k < V; ++k) {
                if ((uint64_t)a[k] >= (uint64_t)n) continue;  // no recipient (empty row)
                const int64_t c = (int64_t)col[a[k]];
                if ((uint64_t)c >= (uint64_t)nx) continue;
                const float coef = w ? w[a[k]] : 1.0f;
                unsafeAtomicAdd(gX + c * F + (int64_t)j * V + k, coef * g[k]);
            }
        }
    }
}

// fused form, max: the recipients by runs of consecutive edges. A row group takes kArgRun
// consecutive edges and walks them in order, keeping in registers, per feature, the first edge
// whose rounded term equals out; at each change of row it stores that row's recipients: plainly
// for a row wholly inside the run, with atomicMin for the run's first and last rows, which may
// continue into the neighbouring runs (the lowest over the runs is then the lowest attaining
// edge). No LDS table and no barrier: the slot-table kernel above ran 3.9 M blocks of 16 edges
// on the SpMM graph. For one vector per thread (nvec <= 64); X rows of kArgBatch edges load
// together. (Loading the next batch's ids beside them held 83 VGPRs instead of 67, 5 waves per
// SIMD instead of 7, and measured the same on the SpMM graph: 6.65 ms; the run's ids loaded by
// the group together and handed out by shuffles took the whole max gradient 15.0 -> 14.65 ms.)
constexpr int kArgRun = 32;
constexpr int kArgBatch = 4;
template <int E, typename I, int V, typename A>
__global__ __launch_bounds__(256) void gs_bwd_max_arg_run_kernel(const typename ElemT<E>::T *__restrict__ X,
                                                                 int64_t nx, const I *__restrict__ col,
                                                                 const float *__restrict__ w,
                                                                 const I *__restrict__ row,
                                                                 const float *__restrict__ out, int64_t n, int64_t R,
                                                                 int64_t F, A *arg) {
    const int nvec = (int)(F / V);
    const RowMap m = row_map(nvec, 1);
    // a group of at least kArgRun threads loads its run's ids together (below)
    const bool coop = m.tpr >= kArgRun;
    if (!coop && m.j0 >= nvec) return;   // no barrier or shuffle below
    const bool lane = m.j0 < nvec;
    const int64_t e0 = ((int64_t)blockIdx.x * m.rows + m.rsub) * kArgRun;
    if (e0 >= n) return;   // the same for the whole group
    const int64_t e1 = min(e0 + (int64_t)kArgRun, n);
    const int64_t row_before = e0 > 0 ? (int64_t)row[e0 - 1] : -1;
    const int64_t row_after = e1 < n ? (int64_t)row[e1] : -1;
    const A none = (A)~(A)0;
    int64_t cur = -1;   // row of the edges walked so far
    A best[V];
    float o[V];
#pragma unroll
    for (int k = 0; k < V; ++k) {
        best[k] = none;
        o[k] = 0.0f;
    }
    auto flush = [&]() {
        if ((uint64_t)cur >= (uint64_t)R || !lane) return;
        const bool shared = cur == row_before || cur == row_after;
        A *a = arg + cur * F + (int64_t)m.j0 * V;
#pragma unroll
        for (int k = 0; k < V; ++k) {
            if (best[k] == none) continue;
            if (shared) atomicMin(a + k, best[k]);
            else a[k] = best[k];
        }
    };
    // coop: lane i of the group loads edge e0 + i's ids (one coalesced load each, instead of a
    // broadcast load per edge and id), handed out by lane shuffles, so that a batch waits only
    // for its X rows; row ids fit 31 bits (the host rejects num_rows >= 2^31)
    int my_r = -1, my_clo = -1, my_chi = -1;
    float my_w = 1.0f;
    const int gb = (int)(threadIdx.x & 63) - m.j0;   // the group's first lane in the wave
    if (coop && m.j0 < kArgRun && e0 + m.j0 < e1) {
        const int64_t e = e0 + m.j0;
        const int64_t c = (int64_t)col[e];
        my_r = (int)row[e];
        my_clo = (int)(uint32_t)(uint64_t)c;
        my_chi = (int)(uint32_t)((uint64_t)c >> 32);
        my_w = w ? w[e] : 1.0f;
    }
    for (int64_t b = e0; b < e1; b += kArgBatch) {
        int64_t rr[kArgBatch], cc[kArgBatch];
        float wt[kArgBatch];
        Raw<E, V> rx[kArgBatch];
        if (coop) {
#pragma unroll
            for (int u = 0; u < kArgBatch; ++u) {   // b - e0 + u < kArgRun: past e1, the sentinels
                const int src = gb + (int)(b - e0) + u;
                rr[u] = __shfl(my_r, src, 64);
                cc[u] = (int64_t)(((uint64_t)(uint32_t)__shfl(my_chi, src, 64) << 32) |
                                  (uint64_t)(uint32_t)__shfl(my_clo, src, 64));
                wt[u] = __shfl(my_w, src, 64);
            }
        } else {
#pragma unroll
            for (int u = 0; u < kArgBatch; ++u) {
                const int64_t e = b + u;
                rr[u] = e < e1 ? (int64_t)row[e] : -1;
                cc[u] = e < e1 ? (int64_t)col[e] : -1;
                wt[u] = e < e1 && w ? w[e] : 1.0f;
            }
        }
#pragma unroll
        for (int u = 0; u < kArgBatch; ++u)
            if (lane && (uint64_t)rr[u] < (uint64_t)R && (uint64_t)cc[u] < (uint64_t)nx)
                load_raw<E, V>(X + cc[u] * F + (int64_t)m.j0 * V, rx[u]);
#pragma unroll
        for (int u = 0; u < kArgBatch; ++u) {
            const int64_t e = b + u;
            if (e >= e1) break;
            if (rr[u] != cur) {   // a new row: store the last one's recipients, load this one's output
                flush();
                cur = rr[u];
#pragma unroll
                for (int k = 0; k < V; ++k) best[k] = none;
                if (lane && (uint64_t)cur < (uint64_t)R) load_f32<V>(out + cur * F + (int64_t)m.j0 * V, o);
            }
            if ((uint64_t)rr[u] >= (uint64_t)R || (uint64_t)cc[u] >= (uint64_t)nx) continue;
            float x[V];
            widen<E, V>(rx[u], x);
#pragma unroll
            for (int k = 0; k < V; ++k) {
                const float t = w ? wt[u] * x[k] : x[k];  // the forward's term: one rounded product
                if (t == o[k] && best[k] == none) best[k] = (A)e;
            }
        }
    }
    flush();
}

// fused form, max, w.r.t. X, pulled over the transposed list: a row group per X row c walks the
// records of column c (16-byte records {column, row, coefficient, edge}, sorted by column;
// column starts in off) and sums coefficient * grad_out[row, f] over the features f whose
// recipient is that edge. Every row of grad_X is written once: no fill and no float atomics
// (on the SpMM graph 313 M of them, about 10 ms). Records load kU at a time.
template <int V>
__global__ __launch_bounds__(256) void gs_bwd_x_max_pull_kernel(const int32_t *__restrict__ rec,
                                                                const int64_t *__restrict__ off,
                                                                const unsigned *__restrict__ arg,
                                                                const float *__restrict__ gout, int64_t nx, int64_t R,
                                                                int64_t F, float *__restrict__ gX) {
    constexpr int kU = 4;
    // the column's terms add into `run`, which joins acc every kPullRun records, so a hub
    // column's long chain rounds like short runs (the fp32 bound holds)
    constexpr int kPullRun = 256;
    const int nvec = (int)(F / V);
    const RowMap m = row_map(nvec);
    if (nvec <= m.tpr && m.tpr >= kU) {
        // One vector per thread: the group loads up to tpr records of its column at once (lane i
        // the i-th: one coalesced load instead of one broadcast load per record) and hands them
        // out by lane shuffles, so a batch waits only for its recipients and grad_out rows. The
        // batches are the same runs of kU records as below, so the sums are the same.
        const int4 *rec4 = reinterpret_cast<const int4 *>(rec);
        const int gb = (int)(threadIdx.x & 63) - m.j0;   // the group's first lane in the wave
        const bool lane = m.j0 < nvec;
        for (int q = 0; q < kPasses; ++q) {
            const int64_t c = m.row(q);
            if (c >= nx) break;   // the same for the whole group
            const int64_t lo = off[c], hi = off[c + 1];
            float acc[V], run[V];
#pragma unroll
            for (int k = 0; k < V; ++k) acc[k] = run[k] = 0.0f;
            int steps = 0;
            for (int64_t k0 = lo; k0 < hi; k0 += m.tpr) {
                const int4 mine = k0 + m.j0 < hi ? rec4[k0 + m.j0] : make_int4(0, -1, 0, 0);
                const int cnt = (int)min((int64_t)m.tpr, hi - k0);
                for (int u0 = 0; u0 < cnt; u0 += kU) {
                    int r[kU];
                    unsigned ed[kU];
                    float coef[kU];
#pragma unroll
                    for (int u = 0; u < kU; ++u) {   // u0 + u < tpr: past the column, the sentinel
                        const int src = gb + u0 + u;
                        r[u] = __shfl(mine.y, src, 64);
                        coef[u] = __int_as_float(__shfl(mine.z, src, 64));
                        ed[u] = (unsigned)__shfl(mine.w, src, 64);
                    }
                    unsigned a[kU][V];
                    float g[kU][V];
#pragma unroll
                    for (int u = 0; u < kU; ++u) {
                        if (lane && (uint64_t)(int64_t)r[u] < (uint64_t)R) {
                            load_arg<unsigned, V>(arg + (int64_t)r[u] * F + (int64_t)m.j0 * V, a[u]);
                        } else {
#pragma unroll
                            for (int k = 0; k < V; ++k) a[u][k] = ~0u;
                        }
                    }
#pragma unroll
                    for (int u = 0; u < kU; ++u) {
                        bool any = false;
#pragma unroll
                        for (int k = 0; k < V; ++k) any |= a[u][k] == ed[u];
                        if (any) {
                            load_f32<V>(gout + (int64_t)r[u] * F + (int64_t)m.j0 * V, g[u]);
                        } else {
#pragma unroll
                            for (int k = 0; k < V; ++k) g[u][k] = 0.0f;
                        }
                    }
#pragma unroll
                    for (int u = 0; u < kU; ++u)
#pragma unroll
                        for (int k = 0; k < V; ++k)
                            if (a[u][k] == ed[u]) run[k] += coef[u] * g[u][k];
                    if (++steps == kPullRun / kU) {
#pragma unroll
                        for (int k = 0; k < V; ++k) {
                            acc[k] += run[k];
                            run[k] = 0.0f;
                        }
                        steps = 0;
                    }
                }
            }
#pragma unroll
            for (int k = 0; k < V; ++k) acc[k] += run[k];
            if (lane) store_vec<V>(gX + c * F + (int64_t)m.j0 * V, acc);
        }
        return;
    }
    for (int q = 0; q < kPasses; ++q) {
        const int64_t c = m.row(q);
        if (c >= nx) break;
        const int64_t lo = off[c], hi = off[c + 1];
        for (int j = m.j0; j < nvec; j += m.tpr) {
            float acc[V], run[V];
#pragma unroll
            for (int k = 0; k < V; ++k) acc[k] = run[k] = 0.0f;
            int steps = 0;
            for (int64_t k0 = lo; k0 < hi; k0 += kU) {
                int4 t[kU];
#pragma unroll
                for (int u = 0; u < kU; ++u)
                    t[u] = k0 + u < hi ? *reinterpret_cast<const int4 *>(rec + 4 * (k0 + u)) : make_int4(0, -1, 0, 0);
                float g[kU][V];
                unsigned a[kU][V];
#pragma unroll
                for (int u = 0; u < kU; ++u) {
                    const int64_t r = (int64_t)t[u].y;
                    if ((uint64_t)r < (uint64_t)R) {
                        load_arg<unsigned, V>(arg + r * F + (int64_t)j * V, a[u]);
                    } else {
#pragma unroll
                        for (int k = 0; k < V; ++k) a[u][k] = ~0u;
                    }
                }
                // grad_out only where the record's edge receives one of this thread's features
                // (the SpMM graph: 5.34 -> 4.53 ms; most records receive none)
#pragma unroll
                for (int u = 0; u < kU; ++u) {
                    bool any = false;
#pragma unroll
                    for (int k = 0; k < V; ++k) any |= a[u][k] == (unsigned)t[u].w;
                    if (any) {
                        load_f32<V>(gout + (int64_t)t[u].y * F + (int64_t)j * V, g[u]);
                    } else {
#pragma unroll
                        for (int k = 0; k < V; ++k) g[u][k] = 0.0f;
                    }
                }
#pragma unroll
                for (int u = 0; u < kU; ++u) {
                    const float coef = __int_as_float(t[u].z);
#pragma unroll
                    for (int k = 0; k < V; ++k)
                        if (a[u][k] == (unsigned)t[u].w) run[k] += coef * g[u][k];
                }
                if (++steps == kPullRun / kU) {
#pragma unroll
                    for (int k = 0; k < V; ++k) {
                        acc[k] += run[k];
                        run[k] = 0.0f;
                    }
                    steps = 0;
                }
            }
#pragma unroll
            for (int k = 0; k < V; ++k) acc[k] += run[k];
            store_vec<V>(gX + c * F + (int64_t)j * V, acc);
        }
    }
}

// fused form, w.r.t. the weights: grad_w[e] = dot(grad_out[row[e]], X[col[e]]) (restricted for max;
// mean divides afterwards, in scale_by_count_kernel). This kernel serves the rows that take
// fewer than 4 threads or more than 64 vectors (gs_bwd_w_run_kernel below takes the others,
// max included). A row group takes P consecutive edges
// (rows are sorted, so they mostly share their grad_out row); every thread runs all of them (the
// group reduction is uniform). The edges' ids load first, then every edge's X row and, once per
// run of edges with the same row, the grad_out row (and for max its recipients), then the
// products. Loading grad_out for every edge cost the SpMM graph 0.9 of 6.6 ms: the rows come
// from cache, but about 25 times each.
template <int E, typename I, int V, int OP, int P, typename A>
__global__ __launch_bounds__(256) void gs_bwd_w_kernel(const typename ElemT<E>::T *__restrict__ X, int64_t nx,
                                                       const I *__restrict__ col,
                                                       const I *__restrict__ row,
                                                       const A *__restrict__ arg,
                                                       const float *__restrict__ gout, int64_t n, int64_t R,
                                                       int64_t F, float *__restrict__ gw) {
    const int nvec = (int)(F / V);
    const RowMap m = row_map(nvec, P);
    const int64_t e0 = ((int64_t)blockIdx.x * m.rows + m.rsub) * P;   // this group's first edge
    int64_t rr[P], cc[P];
    bool ok[P];
#pragma unroll
    for (int q = 0; q < P; ++q) {
        const int64_t e = e0 + q;
        rr[q] = e < n ? (int64_t)row[e] : -1;
        cc[q] = e < n ? (int64_t)col[e] : -1;
    }
#pragma unroll
    for (int q = 0; q < P; ++q)
        ok[q] = (uint64_t)rr[q] < (uint64_t)R && (uint64_t)cc[q] < (uint64_t)nx;
    static_assert(OP != GEOT_BWD_MEAN, "mean: the sum kernel, then scale_by_count_kernel");
    float acc[P];
    if (OP == GEOT_BWD_MAX && nvec <= m.tpr) {
        // max: each (row, feature) has one recipient, so on a power-law graph most edges of a
        // long row receive none (on the SpMM graph a third of the edges receive any). The
        // recipients therefore decide which X vectors are read at all: the grad_out row and its
        // recipients load first (once per run of equal rows), and a thread loads its X vector of
        // an edge only where that edge receives one of the thread's features. On the SpMM graph
        // this pass took 7.28 -> 4.94 ms (fp32 X) and 7.20 -> 5.23 ms (bf16 X, int32 ids).
        const bool lane = m.j0 < nvec;
        bool lead[P];
        float g[P][V];
        A a[P][V];
        Raw<E, V> rx[P];
#pragma unroll
        for (int q = 0; q < P; ++q) {
            lead[q] = !(q > 0 && ok[q - 1] && rr[q] == rr[q - 1]);
            if (ok[q] && lane && lead[q]) {
                load_f32<V>(gout + rr[q] * F + (int64_t)m.j0 * V, g[q]);
                load_arg<A, V>(arg + rr[q] * F + (int64_t)m.j0 * V, a[q]);
            } else {
#pragma unroll
                for (int k = 0; k < V; ++k) {
                    g[q][k] = 0.0f;
                    a[q][k] = (A)~(A)0;
                }
            }
        }
        float cur[V];
        A ca[V];
        unsigned mine[P];   // bit k: this edge is feature k's recipient
#pragma unroll
        for (int q = 0; q < P; ++q) {
            if (lead[q]) {
#pragma unroll
                for (int k = 0; k < V; ++k) {
                    cur[k] = g[q][k];
                    ca[k] = a[q][k];
                }
            }
            const A e = (A)(e0 + q);
            mine[q] = 0u;
#pragma unroll
            for (int k = 0; k < V; ++k) {
                if (ca[k] == e) mine[q] |= 1u << k;
                g[q][k] = cur[k];   // this edge's grad_out values (its run's lead row)
            }
            if (ok[q] && mine[q]) load_raw<E, V>(X + cc[q] * F + (int64_t)m.j0 * V, rx[q]);
            else rx[q] = Raw<E, V>{};
        }
#pragma unroll
        for (int q = 0; q < P; ++q) {
            float x[V];
            widen<E, V>(rx[q], x);
            acc[q] = 0.0f;
#pragma unroll
            for (int k = 0; k < V; ++k) {
                // a selected product, not a product by 0: the other features' values may be inf or NaN
                const float t = g[q][k] * x[k];
                acc[q] += (mine[q] >> k) & 1u ? t : 0.0f;
            }
        }
    } else if (nvec <= m.tpr) {  // sum, one vector per thread and edge: all loads of the group's edges in flight together
        // X rows stay in their loaded words until the products (16-bit X: half the registers of
        // widened rows; bf16 / int32 on the SpMM graph held 92 VGPRs, 5 waves per SIMD, widened)
        const bool lane = m.j0 < nvec;
        bool lead[P];   // the first edge of a run with the same (valid) row: loads the row
        float g[P][V];
        Raw<E, V> rx[P];
#pragma unroll
        for (int q = 0; q < P; ++q) {
            lead[q] = !(q > 0 && ok[q - 1] && rr[q] == rr[q - 1]);
            if (ok[q] && lane) {
                load_raw<E, V>(X + cc[q] * F + (int64_t)m.j0 * V, rx[q]);
            } else {
                rx[q] = Raw<E, V>{};
            }
            if (ok[q] && lane && lead[q]) {
                load_f32<V>(gout + rr[q] * F + (int64_t)m.j0 * V, g[q]);
            } else {
#pragma unroll
                for (int k = 0; k < V; ++k) g[q][k] = 0.0f;
            }
        }
        float cur[V];
#pragma unroll
        for (int q = 0; q < P; ++q) {
            if (lead[q]) {
#pragma unroll
                for (int k = 0; k < V; ++k) cur[k] = g[q][k];
            }
            float x[V];
            widen<E, V>(rx[q], x);
            acc[q] = 0.0f;
#pragma unroll
            for (int k = 0; k < V; ++k) acc[q] += cur[k] * x[k];
        }
    } else {
#pragma unroll
        for (int q = 0; q < P; ++q) {
            acc[q] = 0.0f;
            if (!ok[q]) continue;
            const int64_t e = e0 + q;
            for (int j = m.j0; j < nvec; j += m.tpr) {
                float g[V], x[V];
                load_f32<V>(gout + rr[q] * F + (int64_t)j * V, g);
                Raw<E, V> rx;
                load_raw<E, V>(X + cc[q] * F + (int64_t)j * V, rx);
                widen<E, V>(rx, x);
#pragma unroll
                for (int k = 0; k < V; ++k) {
                    if (OP == GEOT_BWD_MAX && arg[rr[q] * F + (int64_t)j * V + k] != (A)e) continue;
                    acc[q] += g[k] * x[k];
                }
            }
        }
    }
#pragma unroll
    for (int q = 0; q < P; ++q) {
        float a = acc[q];
        for (int d = m.tpr / 2; d >= 1; d >>= 1) a += __shfl_xor(a, d, 64);
        const int64_t e = e0 + q;
        if (e < n && m.j0 == 0) {
            gw[e] = ok[q] ? a : 0.0f;
        }
    }
}

// fused form, sum, mean and max, w.r.t. the weights, where a row's vectors take 4 to 64 threads
// (one vector each): a block takes 256 consecutive edges and stages their ids in LDS with one coalesced
// load, and each row group (tpr threads) walks tpr of them in batches of kB = 4, loading the
// grad_out row once per run of edges with the same row. A batch's four dot products are
// reduced together: across the group's highest lane bit each lane keeps two of the four sums
// and trades the other two, across the next bit one, and a butterfly over the remaining bits
// completes it, so that 6 shuffles at tpr = 32 (instead of 4 x 5) leave edge q's sum in the
// lanes whose two highest group bits read q, one of which stores it (at tpr = 4 the two
// exchanges finish it and every lane stores its own edge's). Max loads the recipient
// vectors with the grad_out rows and an edge's X vector only where the edge receives one of the
// thread's features.
template <int E, typename I, int V, int OP, typename A>
__global__ __launch_bounds__(256) void gs_bwd_w_run_kernel(const typename ElemT<E>::T *__restrict__ X, int64_t nx,
                                                           const I *__restrict__ col, const I *__restrict__ row,
                                                           const A *__restrict__ arg, const int64_t *__restrict__ off,
                                                           const float *__restrict__ gout, int64_t n, int64_t R,
                                                           int64_t F, float *__restrict__ gw) {
    constexpr int kB = 4;
    constexpr bool MX = OP == GEOT_BWD_MAX;
    // mean: the row's edge count loads with its grad_out row (once per run) and the dot product
    // is divided by it before the store, as scale_by_count_kernel divides it (the same rounding)
    constexpr bool MEAN = OP == GEOT_BWD_MEAN;
    __shared__ int64_t s_c[256], s_r[256];
    const int nvec = (int)(F / V);
    int tpr = 1;
    while (tpr < nvec && tpr < 64) tpr <<= 1;   // 4 .. 64: the launch checks
    const int gl = threadIdx.x & (tpr - 1);     // lane within the row group
    const int base = threadIdx.x - gl;          // the group's first edge within the block
    const int64_t b0 = (int64_t)blockIdx.x * 256;
    {
        const int64_t e = b0 + threadIdx.x;
        s_c[threadIdx.x] = e < n ? (int64_t)col[e] : -1;
        s_r[threadIdx.x] = e < n ? (int64_t)row[e] : -1;
    }
    __syncthreads();
    const bool lane = gl < nvec;
    const int hi = tpr >> 1, q2 = tpr >> 2;     // the two highest lane bits of the group
    const bool bh = (gl & hi) != 0, bq = (gl & q2) != 0;
    int64_t prev = -1;                           // the row whose vectors `cur` (and `ca`) hold
    float cnt = 1.0f;                            // mean: that row's edge count
    float cur[V];
    A ca[V];   // max: the recipient edges of the row's features (none: all ones)
#pragma unroll
    for (int k = 0; k < V; ++k) {
        cur[k] = 0.0f;
        ca[k] = (A)~(A)0;
    }
    for (int j0 = 0; j0 < tpr; j0 += kB) {
        int64_t rr[kB], cc[MX ? kB : 1];
        bool ok[kB], lead[kB];
        float g[kB][V];
        float cn[MEAN ? kB : 1];   // mean: the counts of the rows that start here
        A ga[MX ? kB : 1][V];
        Raw<E, V> rx[kB];
#pragma unroll
        for (int q = 0; q < kB; ++q) {
            const int64_t c = s_c[base + j0 + q];
            rr[q] = s_r[base + j0 + q];
            ok[q] = (uint64_t)rr[q] < (uint64_t)R && (uint64_t)c < (uint64_t)nx;
            lead[q] = rr[q] != (q > 0 ? rr[q - 1] : prev);
            if constexpr (MX) {
                cc[q] = c;
            } else {   // sum: every edge's X vector loads at once
                if (ok[q] && lane) load_raw<E, V>(X + c * F + (int64_t)gl * V, rx[q]);
                else rx[q] = Raw<E, V>{};
            }
            // a new row loads its vectors whether or not this edge's column is valid, since the
            // next edges of the run use them
            if constexpr (MEAN)
                cn[q] = lead[q] && (uint64_t)rr[q] < (uint64_t)R ? (float)(off[rr[q] + 1] - off[rr[q]]) : 1.0f;
            if (lead[q] && lane && (uint64_t)rr[q] < (uint64_t)R) {
                load_f32<V>(gout + rr[q] * F + (int64_t)gl * V, g[q]);
                if constexpr (MX) load_arg<A, V>(arg + rr[q] * F + (int64_t)gl * V, ga[q]);
            } else {
#pragma unroll
                for (int k = 0; k < V; ++k) {
                    g[q][k] = 0.0f;
                    if constexpr (MX) ga[q][k] = (A)~(A)0;
                }
            }
        }
        float a[kB];
        float cq[MEAN ? kB : 1];   // mean: each edge's row count
        if constexpr (!MX) {
            // sum and mean: the products with each edge's run's row
#pragma unroll
            for (int q = 0; q < kB; ++q) {
                if (lead[q]) {
#pragma unroll
                    for (int k = 0; k < V; ++k) cur[k] = g[q][k];
                    if constexpr (MEAN) cnt = cn[q];
                }
                if constexpr (MEAN) cq[q] = cnt;
                float x[V];
                widen<E, V>(rx[q], x);
                a[q] = 0.0f;
#pragma unroll
                for (int k = 0; k < V; ++k) a[q] += cur[k] * x[k];
            }
        } else {
            // max: an edge's X vector loads only where the edge receives one of this thread's
            // features (bit k of mine), so the recipients come first
            unsigned mine[kB];
#pragma unroll
            for (int q = 0; q < kB; ++q) {
                if (lead[q]) {
#pragma unroll
                    for (int k = 0; k < V; ++k) {
                        cur[k] = g[q][k];
                        ca[k] = ga[q][k];
                    }
                }
                mine[q] = 0u;
#pragma unroll
                for (int k = 0; k < V; ++k) {
                    g[q][k] = cur[k];   // from here on: this edge's grad_out values
                    mine[q] |= (ca[k] == (A)(b0 + base + j0 + q) ? 1u : 0u) << k;
                }
                if (ok[q] && lane && mine[q]) load_raw<E, V>(X + cc[q] * F + (int64_t)gl * V, rx[q]);
                else rx[q] = Raw<E, V>{};
            }
#pragma unroll
            for (int q = 0; q < kB; ++q) {
                float x[V];
                widen<E, V>(rx[q], x);
                a[q] = 0.0f;
                // a selected product, not a product by 0 (another feature's value may be inf or NaN)
#pragma unroll
                for (int k = 0; k < V; ++k) a[q] += (mine[q] >> k) & 1u ? g[q][k] * x[k] : 0.0f;
            }
        }
        prev = rr[kB - 1];
        // keep sums {0, 1} (highest bit clear) or {2, 3}, trade the others
        const float s0 = __shfl_xor(bh ? a[0] : a[2], hi, 64);
        const float s1 = __shfl_xor(bh ? a[1] : a[3], hi, 64);
        const float k0 = (bh ? a[2] : a[0]) + s0;
        const float k1 = (bh ? a[3] : a[1]) + s1;
        // keep one of the two by the next bit
        float v = (bq ? k1 : k0) + __shfl_xor(bq ? k0 : k1, q2, 64);
        for (int d = q2 >> 1; d >= 1; d >>= 1) v += __shfl_xor(v, d, 64);
        const int q = (bh ? 2 : 0) + (bq ? 1 : 0);
        const int64_t e = b0 + base + j0 + q;
        if constexpr (MEAN) {
            const float c = q == 0 ? cq[0] : q == 1 ? cq[1] : q == 2 ? cq[2] : cq[3];
            v = v / c;
        }
        if ((gl & (q2 - 1)) == 0 && e < n) gw[e] = ok[q] ? v : 0.0f;
    }
}

// mean, for the rows gs_bwd_w_kernel serves: grad_w[e] /= the edge count of row[e]. A pass of
// its own: inside that dot-product
// kernel the row starts either waited after the reduction (one more memory latency per
// block) or held registers through it (5 waves per SIMD instead of 7); both cost C4 1.5 ms,
// this pass about 0.2. Rows of all passes load first, then their starts and the values.
template <typename I>
__global__ __launch_bounds__(256) void scale_by_count_kernel(float *__restrict__ gw, const I *__restrict__ row,
                                                             const int64_t *__restrict__ off, int64_t n, int64_t R) {
    int64_t r[kPasses];
#pragma unroll
    for (int q = 0; q < kPasses; ++q) {
        const int64_t e = ((int64_t)blockIdx.x * kPasses + q) * 256 + threadIdx.x;
        r[q] = e < n ? (int64_t)row[e] : -1;
    }
    float v[kPasses], c[kPasses];
#pragma unroll
    for (int q = 0; q < kPasses; ++q) {
        const int64_t e = ((int64_t)blockIdx.x * kPasses + q) * 256 + threadIdx.x;
        const bool ok = (uint64_t)r[q] < (uint64_t)R;
        const int64_t rs = ok ? r[q] : 0;
        c[q] = (float)(off[rs + 1] - off[rs]);
        v[q] = e < n ? gw[e] : 0.0f;
    }
#pragma unroll
    for (int q = 0; q < kPasses; ++q) {
        const int64_t e = ((int64_t)blockIdx.x * kPasses + q) * 256 + threadIdx.x;
        if (e < n && (uint64_t)r[q] < (uint64_t)R) gw[e] = v[q] / c[q];
    }
}

// ---- counting sort of the edges by source row (the transposed problem) ----
// both edge passes: block b takes edges [b, b + 1) * 256 * kPasses, one pass of 256 at a time
template <typename I>
__global__ __launch_bounds__(256) void hist_kernel(const I *col, int64_t n, int64_t nx,
                                                   unsigned *counts) {
    for (int q = 0; q < kPasses; ++q) {
        const int64_t e = ((int64_t)blockIdx.x * kPasses + q) * 256 + threadIdx.x;
        if (e >= n) break;
        const int64_t c = (int64_t)col[e];
        if ((uint64_t)c < (uint64_t)nx) atomicAdd(counts + c, 1u);
    }
}

constexpr int kScanItems = 16;                       // per thread
constexpr int kScanTile = 256 * kScanItems;          // per block

// exclusive scan of counts within each tile; tile totals to sums[]
__global__ __launch_bounds__(256) void scan_tiles_kernel(const unsigned *counts, int64_t n, int64_t *off,
                                                         int64_t *sums) {
    __shared__ int64_t s_t[256];
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
    int64_t v[kScanItems];
    int64_t t = 0;
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) {
        v[k] = base + k < n ? (int64_t)counts[base + k] : 0;
        t += v[k];
    }
    s_t[threadIdx.x] = t;
    __syncthreads();
    for (int d = 1; d < 256; d <<= 1) {          // inclusive Hillis-Steele over thread totals
        const int64_t o = threadIdx.x >= (unsigned)d ? s_t[threadIdx.x - d] : 0;
        __syncthreads();
        s_t[threadIdx.x] += o;
        __syncthreads();
    }
    int64_t run = s_t[threadIdx.x] - t;
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) {
        if (base + k < n) off[base + k] = run;
        run += v[k];
    }
    if (threadIdx.x == 255) sums[blockIdx.x] = s_t[255];
}

// exclusive scan of the tile totals by one block (serial chunks per thread)
__global__ __launch_bounds__(256) void scan_sums_kernel(int64_t *sums, int64_t ntiles) {
    __shared__ int64_t s_t[256];
    const int64_t per = (ntiles + 255) / 256;
    const int64_t b0 = (int64_t)threadIdx.x * per;
    int64_t t = 0;
    for (int64_t i = b0; i < min(b0 + per, ntiles); ++i) t += sums[i];
    s_t[threadIdx.x] = t;
    __syncthreads();
    for (int d = 1; d < 256; d <<= 1) {
        const int64_t o = threadIdx.x >= (unsigned)d ? s_t[threadIdx.x - d] : 0;
        __syncthreads();
        s_t[threadIdx.x] += o;
        __syncthreads();
    }
    int64_t run = s_t[threadIdx.x] - t;
    for (int64_t i = b0; i < min(b0 + per, ntiles); ++i) {
        const int64_t x = sums[i];
        sums[i] = run;
        run += x;
    }
}

__global__ __launch_bounds__(256) void scan_add_kernel(int64_t *off, int64_t n, const int64_t *sums,
                                                       int64_t total_slot) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) off[i] += sums[i / kScanTile];
    if (i == 0) off[n] = total_slot;
}

// edge e goes to slot off[col[e]] + (a decrementing per-row cursor): the
// transposed problem's segment id (col), gather row (row) and coefficient,
// as three arrays or as one 16-byte record (one store per edge: the slots are
// random, and every store touches its own cache line)
template <bool PACKED, typename I>
__global__ __launch_bounds__(256) void place_kernel(const I *col, int64_t nx, const I *row,
                                                    const float *w, const int64_t *roff, int64_t nrows, int mean,
                                                    int64_t n, const int64_t *off, unsigned *cursor,
                                                    int64_t *key_t, int64_t *row_t, float *w_t, int32_t *rec) {
    for (int q = 0; q < kPasses; ++q) {
        const int64_t e = ((int64_t)blockIdx.x * kPasses + q) * 256 + threadIdx.x;
        if (e >= n) break;
        const int64_t c = (int64_t)col[e];
        if ((uint64_t)c >= (uint64_t)nx) continue;
        const int64_t pos = off[c] + (int64_t)atomicSub(cursor + c, 1u) - 1;
        const int64_t r = (int64_t)row[e];
        float coef = w ? w[e] : 1.0f;
        if (mean && (uint64_t)r < (uint64_t)nrows) coef = coef / (float)(roff[r + 1] - roff[r]);
        if constexpr (PACKED) {
            *reinterpret_cast<int4 *>(rec + 4 * pos) = make_int4((int)c, (int)r, __float_as_int(coef), (int)(uint32_t)e);
        } else {
            key_t[pos] = c;
            row_t[pos] = r;
            w_t[pos] = coef;
        }
    }
}

// ---- the transposition as a radix partition by columns (from 2^20 edges) ----
// Columns fall into bins of 2^shift consecutive columns, bins into coarse buckets of 2^b2 bins.
// One pass counts the edges per bin (LDS counts per block, then summed and scanned), a grouping
// pass moves the edges as records {column, row, coefficient[, edge]} into coarse-bucket order, a
// splitting pass moves each coarse bucket's records into bin order, and a final pass sorts each
// bin by column in LDS. The grouping and splitting passes stage a tile of kRxTile records in
// LDS, ordered by destination, and take one global atomic per (tile, destination) for the run's
// place, so every record store is part of a run of consecutive addresses. The final pass writes
// each bin's records in column order from LDS, as whole runs. Nothing here takes a global atomic
// per edge (on MI355X those run at about 33 G/s, local or not). The order of the edges within a
// column depends on timing (the runs of different tiles take their places in arrival order).
// Records are 12 bytes where the edge numbers are not needed, else 16.
constexpr int64_t kRxMinEdges = 1 << 20;  // below this the direct transposition is as fast
constexpr int kRxTile = 8192;      // edges per tile of the grouping pass (and chunks of the counting pass)
// records per tile of the splitting pass: 12-byte records split fastest in tiles of 4,096 (two
// blocks per CU: 329 against 430 us on the SpMM graph), 16-byte ones in tiles of 8,192 (399
// against 424 us)
template <int W> constexpr int kRxSplitTile = W == 3 ? 4096 : 8192;
constexpr int kRxMaxBins = 32768;  // bins counted in LDS by the counting pass
constexpr int kRxBinColsLog = 11;  // at most 2^11 columns per bin (the final pass's LDS counts)
constexpr int kRxAim = 4096;       // records per bin aimed at
constexpr int kRxPer = 6;          // records per thread of the final pass
constexpr int kRxStage = 4096;     // records per round of the final pass's LDS staging
constexpr int kRxCap = 1024 * kRxPer;  // records per bin sorted from registers; larger bins walk twice
constexpr int kRxSpan = 1024;      // bins one splitting tile counts in LDS

// a record of W words: {column, row, coefficient bits} and for W = 4 the edge number
template <int W> struct RxRec;
template <> struct RxRec<3> {
    using T = int3;
    static __device__ __forceinline__ T make(int c, int r, int coef, int e) { return make_int3(c, r, coef); }
};
template <> struct RxRec<4> {
    using T = int4;
    static __device__ __forceinline__ T make(int c, int r, int coef, int e) { return make_int4(c, r, coef, e); }
};

// Ids per lane load in the radix passes: a 16-byte load (4 int32 or 2 int64 ids) where the
// arrays are 16-byte aligned (VEC), else 1. One 4-byte id per lane and load held the int32
// passes below the int64 ones on the SpMM graph (count 140 against 105 us, grouping 540
// against 425 us) although they read half the bytes.
template <typename I, bool VEC>
constexpr int rx_ids_per_load() {
    return VEC ? 16 / (int)sizeof(I) : 1;
}

// VL consecutive ids p[e .. e + VL) widened to int64, -1 at and past `end`
template <typename I, int VL>
__device__ __forceinline__ void rx_load_ids(const I *p, int64_t e, int64_t end, int64_t *c) {
    if constexpr (VL == 4) {
        if (e + 4 <= end) {
            const int4 t = *reinterpret_cast<const int4 *>(p + e);
            c[0] = t.x;
            c[1] = t.y;
            c[2] = t.z;
            c[3] = t.w;
            return;
        }
    } else if constexpr (VL == 2) {
        if (e + 2 <= end) {
            const longlong2 t = *reinterpret_cast<const longlong2 *>(p + e);
            c[0] = t.x;
            c[1] = t.y;
            return;
        }
    }
#pragma unroll
    for (int k = 0; k < VL; ++k) c[k] = e + k < end ? (int64_t)p[e + k] : -1;
}

// VL consecutive weights w[e ..] (1 where w is NULL or at and past `end`)
template <int VL>
__device__ __forceinline__ void rx_load_w(const float *w, int64_t e, int64_t end, float *x) {
    if (w && e + VL <= end) {
        if constexpr (VL == 4) {
            const float4 t = *reinterpret_cast<const float4 *>(w + e);
            x[0] = t.x;
            x[1] = t.y;
            x[2] = t.z;
            x[3] = t.w;
            return;
        } else if constexpr (VL == 2) {
            const float2 t = *reinterpret_cast<const float2 *>(w + e);
            x[0] = t.x;
            x[1] = t.y;
            return;
        }
    }
#pragma unroll
    for (int k = 0; k < VL; ++k) x[k] = w && e + k < end ? w[e + k] : 1.0f;
}

// exclusive scan of one value per thread over a block of 1024 threads; *total gets the sum.
// Every thread of the block must call it (two barriers).
__device__ __forceinline__ unsigned block_excl_scan(unsigned v, unsigned *s_wave, unsigned *total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    unsigned x = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const unsigned y = (unsigned)__shfl_up((int)x, d, 64);
        if (lane >= d) x += y;
    }
    if (lane == 63) s_wave[wave] = x;
    __syncthreads();
    unsigned before = 0, all = 0;
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        const unsigned t = s_wave[k];
        before += k < wave ? t : 0u;
        all += t;
    }
    __syncthreads();
    *total = all;
    return before + x - v;
}

// slot of this lane's record among its key's in the LDS counters h: a wave whose lanes share
// lane 0's key takes their slots with one LDS atomic (so one hub column does not serialise)
__device__ __forceinline__ unsigned lds_claim(unsigned *h, unsigned key, bool valid) {
    const int lane = threadIdx.x & 63;
    const unsigned k0 = (unsigned)__shfl((int)key, 0, 64);
    const bool same = valid && key == k0;
    const unsigned long long m = __ballot(same);
    const int leader = m ? __ffsll((long long)m) - 1 : 0;
    unsigned base = 0;
    if (same && lane == leader) base = atomicAdd(&h[k0], (unsigned)__popcll(m));
    base = (unsigned)__shfl((int)base, leader, 64);
    unsigned r = 0;
    if (same) r = base + (unsigned)__popcll(m & ((1ull << lane) - 1ull));
    else if (valid) r = atomicAdd(&h[key], 1u);
    return r;
}

// per block, the edges of its chunk per bin, cnt[block * nbins + bin], and per coarse bucket,
// cc[block * 256 + k]
template <typename I, bool VEC>
__global__ __launch_bounds__(1024) void rx_count_kernel(const I *col, int64_t n, int64_t nx, int shift, int nbins,
                                                        int b2, int64_t chunk, unsigned *cnt, unsigned *cc) {
    constexpr int kU = 16;  // ids in flight per thread
    constexpr int VL = rx_ids_per_load<I, VEC>();
    __shared__ unsigned h[kRxMaxBins];
    for (int b = threadIdx.x; b < nbins; b += 1024) h[b] = 0;
    __syncthreads();
    const int64_t e0 = (int64_t)blockIdx.x * chunk;
    const int64_t e1 = min(e0 + chunk, n);
    for (int64_t b0 = e0; b0 < e1; b0 += kU * 1024) {
        int64_t c[kU];
#pragma unroll
        for (int u = 0; u < kU / VL; ++u)
            rx_load_ids<I, VL>(col, b0 + ((int64_t)u * 1024 + threadIdx.x) * VL, e1, c + u * VL);
#pragma unroll
        for (int u = 0; u < kU; ++u)
            if ((uint64_t)c[u] < (uint64_t)nx) atomicAdd(&h[(int)(c[u] >> shift)], 1u);
    }
    __syncthreads();
    for (int b = threadIdx.x; b < nbins; b += 1024) cnt[(int64_t)blockIdx.x * nbins + b] = h[b];
    if (threadIdx.x < 256) {
        const int k = threadIdx.x;
        unsigned t = 0;
        for (int b = k << b2; b < min((k + 1) << b2, nbins); ++b) t += h[b];
        cc[(int64_t)blockIdx.x * 256 + k] = t;
    }
}

// tot[bin] = the bin's edges over all counting blocks: a block takes 64 bins, 4 threads per bin
// each sum every 4th block's counts with 16 loads in flight, and the four sums meet in LDS
__global__ __launch_bounds__(256) void rx_reduce_kernel(const unsigned *cnt, int64_t nblk, int nbins, unsigned *tot) {
    __shared__ unsigned s_part[4][64];
    const int j = threadIdx.x & 63, q = threadIdx.x >> 6;
    const int b = blockIdx.x * 64 + j;
    unsigned s = 0;
    if (b < nbins) {
        for (int64_t k0 = q; k0 < nblk; k0 += 4 * 16) {
            unsigned v[16];
#pragma unroll
            for (int u = 0; u < 16; ++u) {
                const int64_t k = k0 + 4 * u;
                v[u] = k < nblk ? cnt[k * nbins + b] : 0u;
            }
#pragma unroll
            for (int u = 0; u < 16; ++u) s += v[u];
        }
    }
    s_part[q][j] = s;
    __syncthreads();
    if (q == 0 && b < nbins) tot[b] = s_part[0][j] + s_part[1][j] + s_part[2][j] + s_part[3][j];
}

// one block: start[bin] (exclusive scan of tot, start[nbins] = all records) and the cursors of
// the splitting pass (fcur[bin] = start[bin]). The totals pass through LDS so that the global
// loads and stores are coalesced while each thread scans a contiguous range.
__global__ __launch_bounds__(1024) void rx_scan_kernel(const unsigned *tot, int nbins, int64_t *start,
                                                       unsigned *fcur) {
    __shared__ unsigned s_v[kRxMaxBins];
    __shared__ unsigned s_wave[16];
    for (int i = threadIdx.x; i < nbins; i += 1024) s_v[i] = tot[i];
    __syncthreads();
    const int per = (nbins + 1023) / 1024;
    const int i0 = threadIdx.x * per, i1 = min(i0 + per, nbins);
    unsigned t = 0;
    for (int i = i0; i < i1; ++i) t += s_v[i];
    unsigned all;
    unsigned run = block_excl_scan(t, s_wave, &all);
    for (int i = i0; i < i1; ++i) {
        const unsigned x = s_v[i];
        s_v[i] = run;
        run += x;
    }
    __syncthreads();
    for (int i = threadIdx.x; i < nbins; i += 1024) {
        start[i] = s_v[i];
        fcur[i] = s_v[i];
    }
    if (threadIdx.x == 0) start[nbins] = all;
}

// the grouping pass's cursors, one per (counting block, coarse bucket): ccur[blk * 256 + k] =
// the start of bucket k's first bin plus the bucket's edges in the chunks of the blocks before
// blk. Block k of this kernel scans over the counting blocks (at most 256). The grouping tiles of
// one chunk then share its cursors: a few dozen atomics per cursor, not one per tile of the input
// (with shared cursors the grouping pass took 523 against 481 us on the SpMM graph).
__global__ __launch_bounds__(256) void rx_cursor_kernel(const unsigned *cc, int64_t nblk, const int64_t *start,
                                                        int b2, unsigned *ccur) {
    __shared__ unsigned s_t[256];
    const int k = blockIdx.x;
    const unsigned v = (int64_t)threadIdx.x < nblk ? cc[(int64_t)threadIdx.x * 256 + k] : 0u;
    s_t[threadIdx.x] = v;
    __syncthreads();
    for (int d = 1; d < 256; d <<= 1) {
        const unsigned o = threadIdx.x >= (unsigned)d ? s_t[threadIdx.x - d] : 0u;
        __syncthreads();
        s_t[threadIdx.x] += o;
        __syncthreads();
    }
    if ((int64_t)threadIdx.x < nblk)
        ccur[(int64_t)threadIdx.x * 256 + k] = (unsigned)start[(int64_t)k << b2] + s_t[threadIdx.x] - v;
}

// grouping pass: tile t's edges [t * kRxTile, ..) as W-word records into coarse-bucket order
// (bucket = (col >> shift) >> b2): counted and ordered in LDS, then written as one run per bucket
// at a place taken from the cursors of the tile's chunk (tpc tiles per chunk): neighbouring
// tiles, which run at the same time, write neighbouring runs (blocks of different chunks side
// by side measured slower: 538 against 481 us). The cursor atomics are issued before the
// records are staged and waited for after.
template <typename I, int W, bool VEC>
__global__ __launch_bounds__(1024) void rx_group_kernel(const I *col, int64_t nx, const I *row, const float *w,
                                                        const int64_t *roff, int64_t nrows, int mean, int64_t n,
                                                        int shift, int b2, int64_t tpc, unsigned *ccur,
                                                        typename RxRec<W>::T *dst) {
    using R = typename RxRec<W>::T;
    constexpr int kRxU = kRxTile / 1024;  // edges per thread
    __shared__ R s_rec[kRxTile];
    __shared__ unsigned s_cnt[256];
    __shared__ unsigned s_base[256];
    __shared__ unsigned s_wave[16];
    const int64_t chunk = (int64_t)blockIdx.x / tpc;
    const int64_t t0 = (int64_t)blockIdx.x * kRxTile;
    if (threadIdx.x < 256) s_cnt[threadIdx.x] = 0;
    __syncthreads();
    constexpr int VL = rx_ids_per_load<I, VEC>();
    // this thread's edges: VL consecutive ones per load, u-th load at t0 + (u * 1024 + tid) * VL
    auto edge = [&](int u) { return t0 + ((int64_t)(u / VL) * 1024 + threadIdx.x) * VL + u % VL; };
    int64_t c[kRxU], r[kRxU];
    float wt[kRxU];
#pragma unroll
    for (int u = 0; u < kRxU; u += VL) {
        const int64_t e = edge(u);
        rx_load_ids<I, VL>(col, e, n, c + u);
        rx_load_ids<I, VL>(row, e, n, r + u);
        rx_load_w<VL>(w, e, n, wt + u);
    }
    unsigned rank[kRxU];
    int kb[kRxU];
#pragma unroll
    for (int u = 0; u < kRxU; ++u) {
        kb[u] = (uint64_t)c[u] < (uint64_t)nx ? (int)((c[u] >> shift) >> b2) : -1;
        rank[u] = kb[u] >= 0 ? atomicAdd(&s_cnt[kb[u]], 1u) : 0u;
        if (mean && kb[u] >= 0 && (uint64_t)r[u] < (uint64_t)nrows) wt[u] = wt[u] / (float)(roff[r[u] + 1] - roff[r[u]]);
    }
    __syncthreads();
    const unsigned v = threadIdx.x < 256 ? s_cnt[threadIdx.x] : 0u;
    unsigned m;
    const unsigned ex = block_excl_scan(v, s_wave, &m);
    if (threadIdx.x < 256) s_cnt[threadIdx.x] = ex;
    __syncthreads();
    unsigned gb = 0;
    if (threadIdx.x < 256 && v) gb = atomicAdd(&ccur[chunk * 256 + threadIdx.x], v);
#pragma unroll
    for (int u = 0; u < kRxU; ++u)
        if (kb[u] >= 0)
            s_rec[s_cnt[kb[u]] + rank[u]] = RxRec<W>::make((int)c[u], (int)r[u], __float_as_int(wt[u]),
                                                           (int)(uint32_t)edge(u));
    if (threadIdx.x < 256) s_base[threadIdx.x] = gb;
    __syncthreads();
    for (unsigned i = threadIdx.x; i < m; i += 1024) {
        const R x = s_rec[i];
        const int k = (int)(((unsigned)x.x >> shift) >> b2);
        const int64_t pos = (int64_t)s_base[k] + (int64_t)(i - s_cnt[k]);
        if (pos < n) dst[pos] = x;
    }
}

// splitting pass: tile t's records src[t * kRxSplitTile, ..) (grouped by coarse bucket) into bin
// order, one run per bin at a place taken from fcur. A tile counts the bins of the coarse buckets
// it spans in LDS; one that spans more than kRxSpan bins places each record with an atomic.
template <int W>
__global__ __launch_bounds__(1024) void rx_split_kernel(const typename RxRec<W>::T *src, const int64_t *start,
                                                        int nbins, int shift, int b2, unsigned *fcur,
                                                        typename RxRec<W>::T *dst) {
    using R = typename RxRec<W>::T;
    constexpr int kT = kRxSplitTile<W>;
    constexpr int kRxU = kT / 1024;  // records per thread
    __shared__ R s_rec[kT];
    __shared__ unsigned s_cnt[kRxSpan];
    __shared__ unsigned s_base[kRxSpan];
    __shared__ unsigned s_wave[16];
    const int64_t total = start[nbins];
    const int64_t t0 = (int64_t)blockIdx.x * kT;
    if (t0 >= total) return;
    const int64_t t1 = min(t0 + (int64_t)kT, total);
    const unsigned f0 = (((unsigned)src[t0].x >> shift) >> b2) << b2;
    const unsigned f1 = ((((unsigned)src[t1 - 1].x >> shift) >> b2) + 1u) << b2;
    const unsigned span = f1 > f0 ? f1 - f0 : 0u;
    R x[kRxU];
#pragma unroll
    for (int u = 0; u < kRxU; ++u) {
        const int64_t i = t0 + u * 1024 + threadIdx.x;
        if (i < t1) x[u] = src[i];
        else x[u].x = -1;
    }
    if (span == 0 || span > (unsigned)kRxSpan) {
#pragma unroll
        for (int u = 0; u < kRxU; ++u) {
            const unsigned f = (unsigned)x[u].x >> shift;
            if (t0 + u * 1024 + threadIdx.x < t1 && f < (unsigned)nbins) {
                const int64_t pos = (int64_t)atomicAdd(&fcur[f], 1u);
                if (pos < total) dst[pos] = x[u];
            }
        }
        return;
    }
    for (unsigned b = threadIdx.x; b < span; b += 1024) s_cnt[b] = 0;
    __syncthreads();
    unsigned lf[kRxU], rank[kRxU];
#pragma unroll
    for (int u = 0; u < kRxU; ++u) {
        lf[u] = ((unsigned)x[u].x >> shift) - f0;
        const bool ok = t0 + u * 1024 + threadIdx.x < t1 && lf[u] < span;
        if (!ok) lf[u] = 0xffffffffu;
        rank[u] = ok ? atomicAdd(&s_cnt[lf[u]], 1u) : 0u;
    }
    __syncthreads();
    const unsigned v = threadIdx.x < span ? s_cnt[threadIdx.x] : 0u;
    unsigned m;
    const unsigned ex = block_excl_scan(v, s_wave, &m);
    if (threadIdx.x < span) s_cnt[threadIdx.x] = ex;
    __syncthreads();
    unsigned gb = 0;
    if (threadIdx.x < span && v) gb = atomicAdd(&fcur[f0 + threadIdx.x], v);
#pragma unroll
    for (int u = 0; u < kRxU; ++u)
        if (lf[u] != 0xffffffffu) s_rec[s_cnt[lf[u]] + rank[u]] = x[u];
    if (threadIdx.x < span) s_base[threadIdx.x] = gb;
    __syncthreads();
    for (unsigned i = threadIdx.x; i < m; i += 1024) {
        const R y = s_rec[i];
        const unsigned l = ((unsigned)y.x >> shift) - f0;
        const int64_t pos = (int64_t)s_base[l] + (int64_t)(i - s_cnt[l]);
        if (pos < total) dst[pos] = y;
    }
}

// record slot p of the output: one record, or the three arrays
template <bool ARRAYS, typename R>
__device__ __forceinline__ void rx_put(int64_t p, R x, R *rec, int64_t *key_t, int64_t *row_t, float *w_t) {
    if constexpr (ARRAYS) {
        key_t[p] = (int64_t)x.x;
        row_t[p] = (int64_t)x.y;
        w_t[p] = __int_as_float(x.z);
    } else {
        rec[p] = x;
    }
}

// final pass, one block per bin: the bin's records src[start[b], start[b + 1]) ordered by
// column and written from LDS as runs, kRxStage records at a time (up to kRxCap records, held in
// registers); a bin of one column is copied; a larger bin is walked twice and its records
// placed one by one within the bin's range. Writes the column starts col_off[c] (col_off[nx]
// by the last bin).
template <bool ARRAYS, int W>
__global__ __launch_bounds__(1024) __attribute__((amdgpu_waves_per_eu(8))) void rx_final_kernel(
    const typename RxRec<W>::T *src, const int64_t *start, int nbins, int shift, int64_t nx,
    typename RxRec<W>::T *rec, int64_t *key_t, int64_t *row_t, float *w_t, int64_t *col_off) {
    using R = typename RxRec<W>::T;
    __shared__ R s_rec[kRxStage];
    __shared__ unsigned h[1 << kRxBinColsLog];
    __shared__ unsigned s_wave[16];
    const int b = blockIdx.x;
    const int64_t lo = start[b], hi = start[b + 1];
    const int64_t c0 = (int64_t)b << shift;
    const int ncols = (int)min((int64_t)1 << shift, nx - c0);
    const unsigned mask = (1u << shift) - 1u;
    if (b == nbins - 1 && threadIdx.x == 0 && col_off) col_off[nx] = hi;
    if (hi <= lo || ncols == 1) {
        if (col_off)
            for (int c = threadIdx.x; c < ncols; c += 1024) col_off[c0 + c] = lo;
        for (int64_t i = lo + threadIdx.x; i < hi; i += 1024) rx_put<ARRAYS>(i, src[i], rec, key_t, row_t, w_t);
        return;
    }
    const int64_t m = hi - lo;
    for (int c = threadIdx.x; c < ncols; c += 1024) h[c] = 0;
    __syncthreads();
    // exclusive scan of h[0, ncols) in place (two columns per thread), and the column starts
    auto scan_cols = [&]() {
        const int c = 2 * threadIdx.x;
        const unsigned a = c < ncols ? h[c] : 0u, d = c + 1 < ncols ? h[c + 1] : 0u;
        unsigned all;
        const unsigned ex = block_excl_scan(a + d, s_wave, &all);
        if (c < ncols) h[c] = ex;
        if (c + 1 < ncols) h[c + 1] = ex + a;
        if (col_off && c < ncols) col_off[c0 + c] = lo + ex;
        if (col_off && c + 1 < ncols) col_off[c0 + c + 1] = lo + ex + a;
        __syncthreads();
    };
    if (m <= kRxCap) {
        R x[kRxPer];
        unsigned rank[kRxPer];
#pragma unroll
        for (int u = 0; u < kRxPer; ++u) {
            const int64_t i = lo + u * 1024 + threadIdx.x;
            if (i < hi) x[u] = src[i];
            else x[u].x = 0;
        }
#pragma unroll
        for (int u = 0; u < kRxPer; ++u) rank[u] = lds_claim(h, (unsigned)x[u].x & mask, u * 1024 + threadIdx.x < m);
        __syncthreads();
        scan_cols();
#pragma unroll
        for (int u = 0; u < kRxPer; ++u) rank[u] += h[(unsigned)x[u].x & mask];
        for (int64_t s0 = 0; s0 < m; s0 += kRxStage) {
#pragma unroll
            for (int u = 0; u < kRxPer; ++u) {
                const int64_t p = (int64_t)rank[u] - s0;
                if (u * 1024 + threadIdx.x < m && p >= 0 && p < kRxStage) s_rec[p] = x[u];
            }
            __syncthreads();
            const int64_t len = min((int64_t)kRxStage, m - s0);
            for (int i = threadIdx.x; i < len; i += 1024) rx_put<ARRAYS>(lo + s0 + i, s_rec[i], rec, key_t, row_t, w_t);
            __syncthreads();
        }
        return;
    }
    for (int64_t i0 = lo; i0 < hi; i0 += 1024 * kRxPer) {
        unsigned key[kRxPer];
#pragma unroll
        for (int u = 0; u < kRxPer; ++u) {
            const int64_t i = i0 + u * 1024 + threadIdx.x;
            key[u] = i < hi ? ((unsigned)src[i].x & mask) : 0u;
        }
#pragma unroll
        for (int u = 0; u < kRxPer; ++u) (void)lds_claim(h, key[u], i0 + u * 1024 + threadIdx.x < hi);
    }
    __syncthreads();
    scan_cols();
    for (int64_t i0 = lo; i0 < hi; i0 += 1024 * kRxPer) {
        R x[kRxPer];
#pragma unroll
        for (int u = 0; u < kRxPer; ++u) {
            const int64_t i = i0 + u * 1024 + threadIdx.x;
            if (i < hi) x[u] = src[i];
            else x[u].x = 0;
        }
#pragma unroll
        for (int u = 0; u < kRxPer; ++u) {
            const bool valid = i0 + u * 1024 + threadIdx.x < hi;
            const unsigned r = lds_claim(h, (unsigned)x[u].x & mask, valid);
            if (valid && (int64_t)r < m) rx_put<ARRAYS>(lo + (int64_t)r, x[u], rec, key_t, row_t, w_t);
        }
    }
}

// the 16-byte records {col, row, coefficient, 0} as three arrays (one streaming pass)
__global__ __launch_bounds__(256) void unpack_kernel(const int32_t *rec, int64_t n, int64_t *key_t,
                                                     int64_t *row_t, float *w_t) {
    for (int q = 0; q < kPasses; ++q) {
        const int64_t e = ((int64_t)blockIdx.x * kPasses + q) * 256 + threadIdx.x;
        if (e >= n) break;
        const int4 v = *reinterpret_cast<const int4 *>(rec + 4 * e);
        key_t[e] = (int64_t)v.x;
        row_t[e] = (int64_t)v.y;
        w_t[e] = __int_as_float(v.z);
    }
}

__global__ __launch_bounds__(256) void fill_u64_kernel(unsigned long long *p, int64_t n,
                                                       unsigned long long v) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

// blocks of kPasses * (256 / tpr) rows; the callers check the count fits a grid
// threads per row of the row-parallel kernels (row_map's tpr)
int row_threads(int nvec) {
    int t = 1;
    while (t < nvec && t < 64) t <<= 1;
    return t;
}

int64_t grid_rows(int64_t rows, int nvec, int passes = kPasses) {
    const int t = row_threads(nvec);
    const int64_t per_block = (int64_t)passes * (256 / t);
    const int64_t b = (rows + per_block - 1) / per_block;
    return b < 1 ? 1 : b;
}

// exclusive scan of len unsigned counts into off (sums: ceil(len / kScanTile) scratch); off[len] = last
hipError_t scan_counts(const unsigned *counts, int64_t len, int64_t *off, int64_t *sums, int64_t last,
                       hipStream_t st) {
    const int64_t ntiles = (len + kScanTile - 1) / kScanTile;
    if (ntiles > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(scan_tiles_kernel, dim3((unsigned)ntiles), dim3(256), 0, st, counts, len, off, sums);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(scan_sums_kernel, dim3(1), dim3(256), 0, st, sums, ntiles);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(scan_add_kernel, dim3((unsigned)((len + 255) / 256)), dim3(256), 0, st, off, len, sums, last);
    return hipGetLastError();
}

// radix layout: bins of 2^shift columns, coarse buckets of 2^b2 bins (b2 = 0: the grouping pass
// places bins directly), and the counting pass's blocks of chunk edges
struct RxPlan {
    int shift, b2, nbins;
    int64_t chunk, nblk;
};

// Whether the radix partition takes (n, nx), and its layout: at most kRxMaxBins bins of at most
// 2^kRxBinColsLog columns, the widest bins that keep about kRxAim records per bin on average
// where that many bins allow it (bins of one column take any number; beyond that the final pass
// walks the larger bins twice), at most 256 coarse buckets, and 256 counting blocks. Record
// positions and counts are 32-bit (n < 2^32), columns fit the records' 32-bit word.
bool rx_plan(int64_t n, int64_t nx, RxPlan *p) {
    if (n < kRxMinEdges || n > (int64_t)UINT32_MAX || nx < 1 || nx > ((int64_t)1 << 23)) return false;
    int nb = 0;
    while (((int64_t)1 << nb) < nx) ++nb;
    auto bins = [&](int sh) { return ((nx - 1) >> sh) + 1; };
    int shift = std::max(0, nb - 15);
    while (shift < kRxBinColsLog && n <= (int64_t)kRxAim * bins(shift + 1)) ++shift;
    p->shift = shift;
    p->nbins = (int)bins(shift);
    int fb = 0;
    while ((1 << fb) < p->nbins) ++fb;
    p->b2 = std::max(0, fb - 8);
    const int64_t per = (n + 255) / 256;
    p->chunk = (per + kRxTile - 1) / kRxTile * kRxTile;
    p->nblk = (n + p->chunk - 1) / p->chunk;
    return true;
}

// radix scratch: per-block bin counts, per-block coarse-bucket counts, bin totals, bin starts,
// the splitting and grouping cursors, and a second buffer of n records of `words` words
// (offsets into one allocation in o[0..6])
size_t rx_scratch(const RxPlan &p, int64_t n, int words, size_t o[7]) {
    auto a256 = [](size_t x) { return (x + 255) & ~(size_t)255; };
    size_t at = 0;
    const size_t sz[7] = {(size_t)(p.nblk * p.nbins) * 4, (size_t)p.nblk * 256 * 4, (size_t)p.nbins * 4,
                          (size_t)(p.nbins + 1) * 8, (size_t)p.nbins * 4, (size_t)p.nblk * 256 * 4,
                          (size_t)n * 4 * words};
    for (int i = 0; i < 7; ++i) {
        o[i] = at;
        at += a256(sz[i]);
    }
    return at;
}

}  // namespace

size_t transpose_scratch_bytes(int64_t n, int64_t nx, bool edges) {
    RxPlan rp;
    size_t o[7];
    return rx_plan(n, nx, &rp) ? rx_scratch(rp, n, edges ? 4 : 3, o) : 0;
}

namespace {

// The radix partition with W-word records: counts, their sum over blocks and scan, the grouping
// cursors, then the grouping pass (into rec when a splitting pass follows, else into the scratch
// records), the splitting pass (rec into the scratch records) and the final pass (into rec, or
// into the three arrays when `arrays`).
template <typename I, int W>
hipError_t launch_transpose_radix(const RxPlan &p, const I *col, int64_t nx, const I *row, const float *w,
                                  const int64_t *roff, int64_t nrows, bool mean, int64_t n, int64_t *key_t,
                                  int64_t *row_t, float *w_t, int32_t *rec, char *scratch, int64_t *col_off,
                                  bool arrays, hipStream_t st) {
    using R = typename RxRec<W>::T;
    size_t o[7];
    (void)rx_scratch(p, n, W, o);
    unsigned *cnt = (unsigned *)(scratch + o[0]);
    unsigned *cc = (unsigned *)(scratch + o[1]);
    unsigned *tot = (unsigned *)(scratch + o[2]);
    int64_t *start = (int64_t *)(scratch + o[3]);
    unsigned *fcur = (unsigned *)(scratch + o[4]);
    unsigned *ccur = (unsigned *)(scratch + o[5]);
    R *tmp = (R *)(scratch + o[6]);
    R *r4 = (R *)rec;
    const int64_t tiles = (n + kRxTile - 1) / kRxTile;
    const int64_t stiles = (n + kRxSplitTile<W> - 1) / kRxSplitTile<W>;
    const int ncoarse = ((p.nbins - 1) >> p.b2) + 1;
    if (p.nblk > 256 || p.chunk % kRxTile != 0 || stiles > 0x7fffffffLL || p.nbins > kRxMaxBins || ncoarse > 256)
        return hipErrorInvalidConfiguration;
    // 16-byte id (and weight) loads where every array is 16-byte aligned
    const bool vec = (((uintptr_t)col | (uintptr_t)row | (uintptr_t)w) & 15) == 0;
    if (vec)
        hipLaunchKernelGGL((rx_count_kernel<I, true>), dim3((unsigned)p.nblk), dim3(1024), 0, st, col, n, nx, p.shift,
                           p.nbins, p.b2, p.chunk, cnt, cc);
    else
        hipLaunchKernelGGL((rx_count_kernel<I, false>), dim3((unsigned)p.nblk), dim3(1024), 0, st, col, n, nx, p.shift,
                           p.nbins, p.b2, p.chunk, cnt, cc);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(rx_reduce_kernel, dim3((unsigned)((p.nbins + 63) / 64)), dim3(256), 0, st, cnt, p.nblk,
                       p.nbins, tot);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(rx_scan_kernel, dim3(1), dim3(1024), 0, st, tot, p.nbins, start, fcur);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(rx_cursor_kernel, dim3((unsigned)ncoarse), dim3(256), 0, st, cc, p.nblk, start, p.b2, ccur);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (vec)
        hipLaunchKernelGGL((rx_group_kernel<I, W, true>), dim3((unsigned)tiles), dim3(1024), 0, st, col, nx, row, w,
                           roff, nrows, mean ? 1 : 0, n, p.shift, p.b2, p.chunk / kRxTile, ccur, p.b2 > 0 ? r4 : tmp);
    else
        hipLaunchKernelGGL((rx_group_kernel<I, W, false>), dim3((unsigned)tiles), dim3(1024), 0, st, col, nx, row, w,
                           roff, nrows, mean ? 1 : 0, n, p.shift, p.b2, p.chunk / kRxTile, ccur, p.b2 > 0 ? r4 : tmp);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (p.b2 > 0) {
        hipLaunchKernelGGL(rx_split_kernel<W>, dim3((unsigned)stiles), dim3(1024), 0, st, r4, start, p.nbins,
                           p.shift, p.b2, fcur, tmp);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (arrays)
        hipLaunchKernelGGL((rx_final_kernel<true, W>), dim3((unsigned)p.nbins), dim3(1024), 0, st, tmp, start,
                           p.nbins, p.shift, nx, nullptr, key_t, row_t, w_t, col_off);
    else
        hipLaunchKernelGGL((rx_final_kernel<false, W>), dim3((unsigned)p.nbins), dim3(1024), 0, st, tmp, start,
                           p.nbins, p.shift, nx, r4, nullptr, nullptr, nullptr, col_off);
    return hipGetLastError();
}

template <typename I>
hipError_t launch_transpose_t(const I *col, int64_t nx, const I *row, const float *w,
                              const int64_t *roff, int64_t nrows, bool mean, int64_t n, unsigned *counts, int64_t *off,
                              int64_t *sums, int64_t *key_t, int64_t *row_t, float *w_t, int32_t *rec,
                              char *rx_scratch_p, bool edges, int *rec_words, bool *arrays_written, hipStream_t st) {
    RxPlan rp;
    if (rx_scratch_p && rec && rx_plan(n, nx, &rp)) {
        const bool arrays = key_t && row_t && w_t;
        if (arrays_written) *arrays_written = arrays;
        if (rec_words) *rec_words = edges ? 4 : 3;
        if (edges)
            return launch_transpose_radix<I, 4>(rp, col, nx, row, w, roff, nrows, mean, n, key_t, row_t, w_t, rec,
                                                rx_scratch_p, off, arrays, st);
        return launch_transpose_radix<I, 3>(rp, col, nx, row, w, roff, nrows, mean, n, key_t, row_t, w_t, rec,
                                            rx_scratch_p, off, arrays, st);
    }
    hipError_t e = launch_zero_u64((unsigned long long *)counts, (nx + 1) / 2, st);
    if (e != hipSuccess) return e;
    const int64_t geb = (n + 256 * kPasses - 1) / (256 * kPasses);
    if (geb > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    const unsigned ge = (unsigned)geb;
    hipLaunchKernelGGL(hist_kernel<I>, dim3(ge), dim3(256), 0, st, col, n, nx, counts);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = scan_counts(counts, nx, off, sums, n, st)) != hipSuccess) return e;
    if (rec)
        hipLaunchKernelGGL((place_kernel<true, I>), dim3(ge), dim3(256), 0, st, col, nx, row, w, roff, nrows,
                           mean ? 1 : 0, n,
                           off, counts, key_t, row_t, w_t, rec);
    else
        hipLaunchKernelGGL((place_kernel<false, I>), dim3(ge), dim3(256), 0, st, col, nx, row, w, roff, nrows,
                           mean ? 1 : 0,
                           n, off, counts, key_t, row_t, w_t, rec);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_transpose(const void *col, int64_t nx, const void *row, int idx32, const float *w,
                            const int64_t *roff, int64_t nrows, bool mean, int64_t n, unsigned *counts, int64_t *off,
                            int64_t *sums, int64_t *key_t, int64_t *row_t, float *w_t, int32_t *rec,
                            char *rx_scratch_p, bool edges, int *rec_words, bool *arrays_written, hipStream_t st) {
    if (arrays_written) *arrays_written = false;
    if (rec_words) *rec_words = 4;
    if (n <= 0 || nx <= 0) return hipSuccess;
    if (idx32)
        return launch_transpose_t(static_cast<const int32_t *>(col), nx, static_cast<const int32_t *>(row), w, roff,
                                  nrows, mean, n, counts, off, sums, key_t, row_t, w_t, rec, rx_scratch_p, edges,
                                  rec_words, arrays_written, st);
    return launch_transpose_t(static_cast<const int64_t *>(col), nx, static_cast<const int64_t *>(row), w, roff, nrows,
                              mean, n, counts, off, sums, key_t, row_t, w_t, rec, rx_scratch_p, edges, rec_words,
                              arrays_written, st);
}

hipError_t launch_gs_bwd_x_max_pull(const int32_t *rec, const int64_t *off, const void *arg, const float *gout,
                                    int64_t nx, int64_t R, int64_t F, int V, float *gX, hipStream_t st) {
    if (nx <= 0 || F <= 0) return hipSuccess;
    if (!(V == 1 || V == 2 || V == 4 || V == 8) || F % V != 0) return hipErrorInvalidValue;
    const int64_t gb = grid_rows(nx, (int)(F / V));
    if (gb > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    const unsigned g = (unsigned)gb;
    const unsigned *a = static_cast<const unsigned *>(arg);
    if (V == 8)
        hipLaunchKernelGGL(gs_bwd_x_max_pull_kernel<8>, dim3(g), dim3(256), 0, st, rec, off, a, gout, nx, R, F, gX);
    else if (V == 4)
        hipLaunchKernelGGL(gs_bwd_x_max_pull_kernel<4>, dim3(g), dim3(256), 0, st, rec, off, a, gout, nx, R, F, gX);
    else if (V == 2)
        hipLaunchKernelGGL(gs_bwd_x_max_pull_kernel<2>, dim3(g), dim3(256), 0, st, rec, off, a, gout, nx, R, F, gX);
    else
        hipLaunchKernelGGL(gs_bwd_x_max_pull_kernel<1>, dim3(g), dim3(256), 0, st, rec, off, a, gout, nx, R, F, gX);
    return hipGetLastError();
}

hipError_t launch_unpack(const int32_t *rec, int64_t n, int64_t *key_t, int64_t *row_t, float *w_t,
                         hipStream_t st) {
    if (n <= 0) return hipSuccess;
    const int64_t b = (n + 256 * kPasses - 1) / (256 * kPasses);
    if (b > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(unpack_kernel, dim3((unsigned)b), dim3(256), 0, st, rec, n, key_t, row_t, w_t);
    return hipGetLastError();
}

hipError_t launch_fill_u64(unsigned long long *p, int64_t n, unsigned long long v, hipStream_t st) {
    if (n <= 0) return hipSuccess;
    int64_t b = (n + 2047) / 2048;
    b = b < 1 ? 1 : (b > 65536 ? 65536 : b);
    hipLaunchKernelGGL(fill_u64_kernel, dim3((unsigned)b), dim3(256), 0, st, p, n, v);
    return hipGetLastError();
}


namespace {

template <typename T> struct TypeTag { using type = T; };

// f(E, I) with the storage type and id type as compile-time tags
template <typename Fn>
hipError_t by_types(int elem, int idx32, Fn &&f) {
    auto by_idx = [&](auto e) -> hipError_t {
        return idx32 ? f(e, TypeTag<int32_t>{}) : f(e, TypeTag<int64_t>{});
    };
    if (elem == ELEM_BF16) return by_idx(std::integral_constant<int, ELEM_BF16>{});
    if (elem == ELEM_F16) return by_idx(std::integral_constant<int, ELEM_F16>{});
    if (elem == ELEM_F32) return by_idx(std::integral_constant<int, ELEM_F32>{});
    return hipErrorInvalidValue;
}

// f(V) with the vector width as a compile-time value (8 for 16-bit storage only)
template <int E, typename Fn>
hipError_t by_width(int V, Fn &&f) {
    if (V == 8) {
        if constexpr (E != ELEM_F32) return f(std::integral_constant<int, 8>{});
        else return hipErrorInvalidValue;
    }
    if (V == 4) return f(std::integral_constant<int, 4>{});
    if (V == 2) return f(std::integral_constant<int, 2>{});
    return f(std::integral_constant<int, 1>{});
}

}  // namespace

int seg_bwd_rows_log2(int64_t F, int V) {
    const int nvec = (int)(F / V);
    int t = 1, lt = 0;
    while (t < nvec && t < 64) t <<= 1, ++lt;
    return 10 - lt;   // kPasses * 256 / t rows
}

int64_t seg_bwd_blocks(int64_t n, int64_t F, int V) { return grid_rows(n, (int)(F / V)); }

hipError_t launch_seg_bwd_bcast(const float *gout, const void *idx, int idx32, const int64_t *off,
                                const int64_t *first, int64_t n, int64_t S, int64_t F, int V, int elem, bool mean,
                                void *gsrc, hipStream_t st) {
    static_assert(kPasses * 256 == 1 << 10, "seg_bwd_rows_log2 assumes 1024 thread-rows per block");
    if (n <= 0) return hipSuccess;
    if (first && !off) return hipErrorInvalidValue;
    const int64_t gb = grid_rows(n, (int)(F / V));
    if (gb > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    const unsigned g = (unsigned)gb;
    return by_types(elem, idx32, [&](auto et, auto it) -> hipError_t {
        constexpr int E = decltype(et)::value;
        using I = typename decltype(it)::type;
        using T = typename ElemT<E>::T;
        return by_width<E>(V, [&](auto vt) -> hipError_t {
            constexpr int VV = decltype(vt)::value;
            if (first && mean)
                hipLaunchKernelGGL((seg_bwd_bcast_off_kernel<E, I, VV, true>), dim3(g), dim3(256), 0, st, gout,
                                   static_cast<const I *>(idx), off, first, n, S, F, static_cast<T *>(gsrc));
            else if (first)
                hipLaunchKernelGGL((seg_bwd_bcast_off_kernel<E, I, VV, false>), dim3(g), dim3(256), 0, st, gout,
                                   static_cast<const I *>(idx), off, first, n, S, F, static_cast<T *>(gsrc));
            else if (mean)
                hipLaunchKernelGGL((seg_bwd_bcast_kernel<E, I, VV, true>), dim3(g), dim3(256), 0, st, gout,
                                   static_cast<const I *>(idx), off, n, S, F, static_cast<T *>(gsrc));
            else
                hipLaunchKernelGGL((seg_bwd_bcast_kernel<E, I, VV, false>), dim3(g), dim3(256), 0, st, gout,
                                   static_cast<const I *>(idx), off, n, S, F, static_cast<T *>(gsrc));
            return hipGetLastError();
        });
    });
}

bool seg_bwd_arg32(int64_t n) { return n < (int64_t)0xffffffffLL; }

hipError_t launch_seg_bwd_max(const float *gout, const void *idx, int idx32, const void *src, const float *out,
                              const int64_t *off, const int64_t *first, int64_t n, int64_t S, int64_t F, int V,
                              int elem, void *arg, bool given, void *gsrc, hipStream_t st) {
    if (n <= 0) return hipSuccess;
    if (first && !off) return hipErrorInvalidValue;
    const bool a32 = seg_bwd_arg32(n);
    if (given && !a32) return hipErrorInvalidValue;   // recorded recipients are 32-bit
    // all ones ("no recipient") in either width: S * F entries, rounded up to 8 bytes (the
    // table's allocation is a multiple of 256 bytes)
    if (!given) {
        hipError_t e = launch_fill_u64(static_cast<unsigned long long *>(arg), a32 ? (S * F + 1) / 2 : S * F, ~0ull, st);
        if (e != hipSuccess) return e;
    }
    const int64_t gb = grid_rows(n, (int)(F / V));
    if (gb > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    const unsigned g = (unsigned)gb;
    auto run = [&](auto at) -> hipError_t {
        using A = typename decltype(at)::type;
        A *ap = static_cast<A *>(arg);
        return by_types(elem, idx32, [&](auto et, auto it) -> hipError_t {
            constexpr int E = decltype(et)::value;
            using I = typename decltype(it)::type;
            using T = typename ElemT<E>::T;
            return by_width<E>(V, [&](auto vt) -> hipError_t {
                constexpr int VV = decltype(vt)::value;
                if (!given) {   // the recipients: the lowest attaining row of each (segment, feature)
                    if (first)
                        hipLaunchKernelGGL((seg_bwd_max_arg_off_kernel<E, I, VV, A>), dim3(g), dim3(256), 0, st,
                                           static_cast<const T *>(src), static_cast<const I *>(idx), off, first, out,
                                           n, S, F, ap);
                    else
                        hipLaunchKernelGGL((seg_bwd_max_arg_kernel<E, I, VV, A>), dim3(g), dim3(256), 0, st,
                                           static_cast<const T *>(src), static_cast<const I *>(idx), out, n, S, F, ap);
                    hipError_t e2 = hipGetLastError();
                    if (e2 != hipSuccess) return e2;
                }
                if (first)
                    hipLaunchKernelGGL((seg_bwd_max_write_off_kernel<E, I, VV, A>), dim3(g), dim3(256), 0, st, gout,
                                       static_cast<const I *>(idx), off, first, ap, n, S, F, static_cast<T *>(gsrc));
                else
                    hipLaunchKernelGGL((seg_bwd_max_write_kernel<E, I, VV, A>), dim3(g), dim3(256), 0, st, gout,
                                       static_cast<const I *>(idx), ap, n, S, F, static_cast<T *>(gsrc));
                return hipGetLastError();
            });
        });
    };
    return a32 ? run(TypeTag<unsigned>{}) : run(TypeTag<unsigned long long>{});
}

hipError_t launch_gs_bwd(const void *X, int elem, int64_t nx, const void *col, int idx32, const float *w,
                         const void *row, const int64_t *off, const float *out, const float *gout, int64_t n, int64_t R,
                         int64_t F, int V, int op, void *arg, bool given, float *gX, float *gw, hipStream_t st) {
    if (n <= 0) return hipSuccess;
    if (op == GEOT_BWD_MAX && !arg) return hipErrorInvalidValue;
    if (op == GEOT_BWD_MEAN && gw && !off) return hipErrorInvalidValue;   // mean divides by the row counts
    if (given && !seg_bwd_arg32(n)) return hipErrorInvalidValue;   // recorded recipients are 32-bit
    if (grid_rows(n, (int)(F / V)) > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    // recipients as 32-bit edge numbers below 2^32 - 1 edges, else 64-bit
    const bool a32 = seg_bwd_arg32(n);
    auto run = [&](auto at) -> hipError_t {
    using A = typename decltype(at)::type;
    A *ap = static_cast<A *>(arg);
    return by_types(elem, idx32, [&](auto et, auto it) -> hipError_t {
        constexpr int E = decltype(et)::value;
        using I = typename decltype(it)::type;
        using T = typename ElemT<E>::T;
        const T *Xt = static_cast<const T *>(X);
        const I *ct = static_cast<const I *>(col), *rt = static_cast<const I *>(row);
        return by_width<E>(V, [&](auto vt) -> hipError_t {
            constexpr int VV = decltype(vt)::value;
            hipError_t e;
            if (op == GEOT_BWD_MAX && !given) {
                e = launch_fill_u64(static_cast<unsigned long long *>(arg), a32 ? (R * F + 1) / 2 : R * F, ~0ull, st);
                if (e != hipSuccess) return e;
                if (F / VV <= 64) {   // one vector per thread: runs of consecutive edges
                    const int64_t groups = 256 / (int64_t)row_threads((int)(F / VV));
                    const int64_t gab = (n + groups * kArgRun - 1) / (groups * kArgRun);
                    if (gab > 0x7fffffffLL) return hipErrorInvalidConfiguration;
                    hipLaunchKernelGGL((gs_bwd_max_arg_run_kernel<E, I, VV, A>), dim3((unsigned)gab), dim3(256), 0, st,
                                       Xt, nx, ct, w, rt, out, n, R, F, ap);
                } else {
                    const int64_t gab = grid_rows(n, (int)(F / VV), kArgPasses);
                    if (gab > 0x7fffffffLL) return hipErrorInvalidConfiguration;
                    hipLaunchKernelGGL((gs_bwd_max_arg_kernel<E, I, VV, A, kArgPasses>), dim3((unsigned)gab), dim3(256),
                                       0, st, Xt, nx, ct, w, rt, out, n, R, F, ap);
                }
                if ((e = hipGetLastError()) != hipSuccess) return e;
            }
            if (gX) {  // max only (sum and mean gather over the transposed list)
                if (op != GEOT_BWD_MAX) return hipErrorInvalidValue;
                e = launch_fill(gX, nx, F, F, 0.0f, st);
                if (e != hipSuccess) return e;
                const int64_t gr = grid_rows(R, (int)(F / VV));
                if (gr > 0x7fffffffLL) return hipErrorInvalidConfiguration;
                hipLaunchKernelGGL((gs_bwd_x_max_kernel<I, VV, A>), dim3((unsigned)gr), dim3(256), 0, st, ap, ct, nx,
                                   w, gout, n, R, F, gX);
                if ((e = hipGetLastError()) != hipSuccess) return e;
            }
            if (gw) {
                // 8-element vectors: 2 passes per block (their fp32 operand vectors fill half the
                // registers that 4 passes' do)
                constexpr int WP = VV == 8 ? kWPasses8 : kPasses;
                const int64_t gwb = grid_rows(n, (int)(F / VV), WP);
                if (gwb > 0x7fffffffLL) return hipErrorInvalidConfiguration;
                const int tpr = row_threads((int)(F / VV));
                const bool runs = tpr >= 4 && F / VV <= 64;
                if (op == GEOT_BWD_MAX && runs)
                    hipLaunchKernelGGL((gs_bwd_w_run_kernel<E, I, VV, GEOT_BWD_MAX, A>), dim3((unsigned)((n + 255) / 256)),
                                       dim3(256), 0, st, Xt, nx, ct, rt, ap, off, gout, n, R, F, gw);
                else if (op == GEOT_BWD_MAX)
                    hipLaunchKernelGGL((gs_bwd_w_kernel<E, I, VV, GEOT_BWD_MAX, WP, A>), dim3((unsigned)gwb), dim3(256), 0,
                                       st, Xt, nx, ct, rt, ap, gout, n, R, F, gw);
                else if (runs && op == GEOT_BWD_MEAN)
                    hipLaunchKernelGGL((gs_bwd_w_run_kernel<E, I, VV, GEOT_BWD_MEAN, A>), dim3((unsigned)((n + 255) / 256)),
                                       dim3(256), 0, st, Xt, nx, ct, rt, ap, off, gout, n, R, F, gw);
                else if (runs)
                    hipLaunchKernelGGL((gs_bwd_w_run_kernel<E, I, VV, GEOT_BWD_SUM, A>), dim3((unsigned)((n + 255) / 256)),
                                       dim3(256), 0, st, Xt, nx, ct, rt, ap, off, gout, n, R, F, gw);
                else
                    hipLaunchKernelGGL((gs_bwd_w_kernel<E, I, VV, GEOT_BWD_SUM, WP, A>), dim3((unsigned)gwb), dim3(256), 0,
                                       st, Xt, nx, ct, rt, ap, gout, n, R, F, gw);
                if ((e = hipGetLastError()) != hipSuccess) return e;
                if (op == GEOT_BWD_MEAN && !runs) {
                    const int64_t sb = (n + 256 * kPasses - 1) / (256 * kPasses);
                    if (sb > 0x7fffffffLL) return hipErrorInvalidConfiguration;
                    hipLaunchKernelGGL(scale_by_count_kernel<I>, dim3((unsigned)sb), dim3(256), 0, st, gw, rt, off,
                                       n, R);
                    if ((e = hipGetLastError()) != hipSuccess) return e;
                }
            }
            return hipSuccess;
        });
    });
    };
    // sum and mean read no recipients: their kernels take the 32-bit instance
    return a32 || op != GEOT_BWD_MAX ? run(TypeTag<unsigned>{}) : run(TypeTag<unsigned long long>{});
}

}  // namespace geot
