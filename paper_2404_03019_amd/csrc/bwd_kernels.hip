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

#include "common.h"

namespace geot {

namespace {

constexpr int kPasses = 4;  // passes of one block over its rows

struct RowMap {
    int tpr;    // threads per row
    int rsub;   // this thread's row within a pass
    int j0;     // this thread's first vector
    int rows;   // rows per pass of one block
    __device__ int64_t row(int q) const {  // this thread's row in pass q
        return ((int64_t)blockIdx.x * kPasses + q) * rows + rsub;
    }
};

__device__ __forceinline__ RowMap row_map(int nvec) {
    RowMap m;
    int t = 1;
    while (t < nvec && t < 64) t <<= 1;
    m.tpr = t;
    m.rsub = threadIdx.x / t;
    m.j0 = threadIdx.x % t;
    m.rows = 256 / t;
    return m;
}

// grad_src[i] = grad_out[idx[i]] (times 1 / len for mean). The ids of all the
// block's passes load first, so their latency overlaps; then the rows.
template <int V, bool MEAN>
__global__ __launch_bounds__(256) void seg_bwd_bcast_kernel(const float *__restrict__ gout,
                                                            const int64_t *__restrict__ idx,
                                                            const int64_t *__restrict__ off, int64_t n,
                                                            int64_t S, int64_t F, float *__restrict__ gsrc) {
    const int nvec = (int)(F / V);
    const RowMap m = row_map(nvec);
    int64_t seg[kPasses];
#pragma unroll
    for (int q = 0; q < kPasses; ++q) {
        const int64_t i = m.row(q);
        seg[q] = i < n ? idx[i] : -1;
    }
#pragma unroll
    for (int q = 0; q < kPasses; ++q) {
        const int64_t i = m.row(q);
        if (i < n) {
            const int64_t s = seg[q];
            const bool ok = (uint64_t)s < (uint64_t)S;
            float inv = 1.0f;
            if (MEAN && ok) inv = 1.0f / (float)(off[s + 1] - off[s]);
            for (int j = m.j0; j < nvec; j += m.tpr) {
                float x[V];
                if (ok) {
                    load_vec<V>(gout + s * F + (int64_t)j * V, x);
                    if (MEAN) {
#pragma unroll
                        for (int k = 0; k < V; ++k) x[k] = x[k] * inv;
                    }
                } else {
#pragma unroll
                    for (int k = 0; k < V; ++k) x[k] = 0.0f;
                }
                store_vec<V>(gsrc + i * F + (int64_t)j * V, x);
            }
        }
    }
}

// arg[s, f] = min row i of segment s with src[i, f] == out[s, f]
template <int V>
__global__ __launch_bounds__(256) void seg_bwd_max_arg_kernel(const float *src, const int64_t *idx,
                                                              const float *out, int64_t n, int64_t S,
                                                              int64_t F, unsigned long long *arg) {
    const int nvec = (int)(F / V);
    const RowMap m = row_map(nvec);
    for (int q = 0; q < kPasses; ++q) {
        const int64_t i = m.row(q);
        if (i >= n) break;
        const int64_t s = idx[i];
        if ((uint64_t)s >= (uint64_t)S) continue;
        for (int j = m.j0; j < nvec; j += m.tpr) {
            float x[V], o[V];
            load_vec<V>(src + i * F + (int64_t)j * V, x);
            load_vec<V>(out + s * F + (int64_t)j * V, o);
#pragma unroll
            for (int k = 0; k < V; ++k)
                if (x[k] == o[k]) atomicMin(arg + s * F + (int64_t)j * V + k, (unsigned long long)i);
        }
    }
}

// grad_src[i, f] = grad_out[s, f] where i is the recipient of (s, f), else 0
template <int V>
__global__ __launch_bounds__(256) void seg_bwd_max_write_kernel(const float *gout, const int64_t *idx,
                                                                const unsigned long long *arg, int64_t n,
                                                                int64_t S, int64_t F, float *gsrc) {
    const int nvec = (int)(F / V);
    const RowMap m = row_map(nvec);
    for (int q = 0; q < kPasses; ++q) {
        const int64_t i = m.row(q);
        if (i >= n) break;
        const int64_t s = idx[i];
        const bool ok = (uint64_t)s < (uint64_t)S;
        for (int j = m.j0; j < nvec; j += m.tpr) {
            float x[V];
            if (ok) {
                load_vec<V>(gout + s * F + (int64_t)j * V, x);
#pragma unroll
                for (int k = 0; k < V; ++k)
                    if (arg[s * F + (int64_t)j * V + k] != (unsigned long long)i) x[k] = 0.0f;
            } else {
#pragma unroll
                for (int k = 0; k < V; ++k) x[k] = 0.0f;
            }
            store_vec<V>(gsrc + i * F + (int64_t)j * V, x);
        }
    }
}

// fused form, max: arg[r, f] = min edge e of row r whose rounded product equals out[r, f]
template <int V>
__global__ __launch_bounds__(256) void gs_bwd_max_arg_kernel(const float *X, int64_t nx, const int64_t *col,
                                                             const float *w, const int64_t *row,
                                                             const float *out, int64_t n, int64_t R,
                                                             int64_t F, unsigned long long *arg) {
    const int nvec = (int)(F / V);
    const RowMap m = row_map(nvec);
    for (int q = 0; q < kPasses; ++q) {
        const int64_t e = m.row(q);
        if (e >= n) break;
        const int64_t r = row[e];
        const int64_t c = col[e];
        if ((uint64_t)r >= (uint64_t)R || (uint64_t)c >= (uint64_t)nx) continue;
        const float wt = w ? w[e] : 1.0f;
        for (int j = m.j0; j < nvec; j += m.tpr) {
            float x[V], o[V];
            load_vec<V>(X + c * F + (int64_t)j * V, x);
            load_vec<V>(out + r * F + (int64_t)j * V, o);
#pragma unroll
            for (int k = 0; k < V; ++k) {
                const float t = w ? wt * x[k] : x[k];  // the forward's term: one rounded product
                if (t == o[k]) atomicMin(arg + r * F + (int64_t)j * V + k, (unsigned long long)e);
            }
        }
    }
}

// fused form, w.r.t. X: grad_X[col[e]] += coef(e) * grad_out[row[e]] (atomic adds)
template <int V, int OP>
__global__ __launch_bounds__(256) void gs_bwd_x_kernel(const int64_t *col, int64_t nx, const float *w,
                                                       const int64_t *row, const int64_t *off,
                                                       const unsigned long long *arg, const float *gout,
                                                       int64_t n, int64_t R, int64_t F, float *gX) {
    const int nvec = (int)(F / V);
    const RowMap m = row_map(nvec);
    for (int q = 0; q < kPasses; ++q) {
        const int64_t e = m.row(q);
        if (e >= n) break;
        const int64_t r = row[e];
        const int64_t c = col[e];
        if ((uint64_t)r >= (uint64_t)R || (uint64_t)c >= (uint64_t)nx) continue;
        float coef = w ? w[e] : 1.0f;
        if (OP == GEOT_BWD_MEAN) coef = coef / (float)(off[r + 1] - off[r]);
        for (int j = m.j0; j < nvec; j += m.tpr) {
            float g[V];
            load_vec<V>(gout + r * F + (int64_t)j * V, g);
#pragma unroll
            for (int k = 0; k < V; ++k) {
                if (OP == GEOT_BWD_MAX && arg[r * F + (int64_t)j * V + k] != (unsigned long long)e) continue;
                unsafeAtomicAdd(gX + c * F + (int64_t)j * V + k, coef * g[k]);
            }
        }
    }
}

// fused form, w.r.t. the weights: grad_w[e] = dot(grad_out[row[e]], X[col[e]]) (restricted for max).
// Every thread runs all passes (the group reduction is uniform); the edges'
// ids load first, then both operand rows of every pass, then the products.
template <int V, int OP>
__global__ __launch_bounds__(256) void gs_bwd_w_kernel(const float *__restrict__ X, int64_t nx,
                                                       const int64_t *__restrict__ col,
                                                       const int64_t *__restrict__ row,
                                                       const int64_t *__restrict__ off,
                                                       const unsigned long long *__restrict__ arg,
                                                       const float *__restrict__ gout, int64_t n, int64_t R,
                                                       int64_t F, float *__restrict__ gw) {
    const int nvec = (int)(F / V);
    const RowMap m = row_map(nvec);
    int64_t rr[kPasses], cc[kPasses];
    bool ok[kPasses];
#pragma unroll
    for (int q = 0; q < kPasses; ++q) {
        const int64_t e = m.row(q);
        rr[q] = e < n ? row[e] : -1;
        cc[q] = e < n ? col[e] : -1;
    }
#pragma unroll
    for (int q = 0; q < kPasses; ++q)
        ok[q] = (uint64_t)rr[q] < (uint64_t)R && (uint64_t)cc[q] < (uint64_t)nx;
    float acc[kPasses];
    if (nvec <= m.tpr) {  // one vector per thread and row: all loads of the block's passes in flight together
        float g[kPasses][V], x[kPasses][V];
#pragma unroll
        for (int q = 0; q < kPasses; ++q) {
            if (ok[q] && m.j0 < nvec) {
                load_vec<V>(gout + rr[q] * F + (int64_t)m.j0 * V, g[q]);
                load_vec<V>(X + cc[q] * F + (int64_t)m.j0 * V, x[q]);
            } else {
#pragma unroll
                for (int k = 0; k < V; ++k) g[q][k] = x[q][k] = 0.0f;
            }
        }
#pragma unroll
        for (int q = 0; q < kPasses; ++q) {
            acc[q] = 0.0f;
            const int64_t e = m.row(q);
#pragma unroll
            for (int k = 0; k < V; ++k) {
                if (OP == GEOT_BWD_MAX && ok[q] && m.j0 < nvec &&
                    arg[rr[q] * F + (int64_t)m.j0 * V + k] != (unsigned long long)e)
                    continue;
                acc[q] += g[q][k] * x[q][k];
            }
        }
    } else {
#pragma unroll
        for (int q = 0; q < kPasses; ++q) {
            acc[q] = 0.0f;
            if (!ok[q]) continue;
            const int64_t e = m.row(q);
            for (int j = m.j0; j < nvec; j += m.tpr) {
                float g[V], x[V];
                load_vec<V>(gout + rr[q] * F + (int64_t)j * V, g);
                load_vec<V>(X + cc[q] * F + (int64_t)j * V, x);
#pragma unroll
                for (int k = 0; k < V; ++k) {
                    if (OP == GEOT_BWD_MAX && arg[rr[q] * F + (int64_t)j * V + k] != (unsigned long long)e) continue;
                    acc[q] += g[k] * x[k];
                }
            }
        }
    }
#pragma unroll
    for (int q = 0; q < kPasses; ++q) {
        float a = acc[q];
        for (int d = m.tpr / 2; d >= 1; d >>= 1) a += __shfl_xor(a, d, 64);
        const int64_t e = m.row(q);
        if (e < n && m.j0 == 0) {
            float v = ok[q] ? a : 0.0f;
            if (ok[q] && OP == GEOT_BWD_MEAN) v = v / (float)(off[rr[q] + 1] - off[rr[q]]);
            gw[e] = v;
        }
    }
}

// ---- counting sort of the edges by source row (the transposed problem) ----
// both edge passes: block b takes edges [b, b + 1) * 256 * kPasses, one pass of 256 at a time
__global__ __launch_bounds__(256) void hist_kernel(const int64_t *col, int64_t n, int64_t nx,
                                                   unsigned *counts) {
    for (int q = 0; q < kPasses; ++q) {
        const int64_t e = ((int64_t)blockIdx.x * kPasses + q) * 256 + threadIdx.x;
        if (e >= n) break;
        const int64_t c = col[e];
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
template <bool PACKED>
__global__ __launch_bounds__(256) void place_kernel(const int64_t *col, int64_t nx, const int64_t *row,
                                                    const float *w, const int64_t *roff, int mean,
                                                    int64_t n, const int64_t *off, unsigned *cursor,
                                                    int64_t *key_t, int64_t *row_t, float *w_t, int32_t *rec) {
    for (int q = 0; q < kPasses; ++q) {
        const int64_t e = ((int64_t)blockIdx.x * kPasses + q) * 256 + threadIdx.x;
        if (e >= n) break;
        const int64_t c = col[e];
        if ((uint64_t)c >= (uint64_t)nx) continue;
        const int64_t pos = off[c] + (int64_t)atomicSub(cursor + c, 1u) - 1;
        const int64_t r = row[e];
        float coef = w ? w[e] : 1.0f;
        if (mean) coef = coef / (float)(roff[r + 1] - roff[r]);
        if constexpr (PACKED) {
            *reinterpret_cast<int4 *>(rec + 4 * pos) = make_int4((int)c, (int)r, __float_as_int(coef), 0);
        } else {
            key_t[pos] = c;
            row_t[pos] = r;
            w_t[pos] = coef;
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
int64_t grid_rows(int64_t rows, int nvec) {
    int t = 1;
    while (t < nvec && t < 64) t <<= 1;
    const int64_t per_block = (int64_t)kPasses * (256 / t);
    const int64_t b = (rows + per_block - 1) / per_block;
    return b < 1 ? 1 : b;
}

}  // namespace

hipError_t launch_transpose(const int64_t *col, int64_t nx, const int64_t *row, const float *w,
                            const int64_t *roff, bool mean, int64_t n, unsigned *counts, int64_t *off,
                            int64_t *sums, int64_t *key_t, int64_t *row_t, float *w_t, int32_t *rec,
                            hipStream_t st) {
    if (n <= 0 || nx <= 0) return hipSuccess;
    hipError_t e = launch_zero_u64((unsigned long long *)counts, (nx + 1) / 2, st);
    if (e != hipSuccess) return e;
    const int64_t geb = (n + 256 * kPasses - 1) / (256 * kPasses);
    if (geb > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    const unsigned ge = (unsigned)geb;
    hipLaunchKernelGGL(hist_kernel, dim3(ge), dim3(256), 0, st, col, n, nx, counts);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const int64_t ntiles = (nx + kScanTile - 1) / kScanTile;
    hipLaunchKernelGGL(scan_tiles_kernel, dim3((unsigned)ntiles), dim3(256), 0, st, counts, nx, off, sums);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(scan_sums_kernel, dim3(1), dim3(256), 0, st, sums, ntiles);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(scan_add_kernel, dim3((unsigned)((nx + 255) / 256)), dim3(256), 0, st, off, nx, sums, n);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (rec)
        hipLaunchKernelGGL(place_kernel<true>, dim3(ge), dim3(256), 0, st, col, nx, row, w, roff, mean ? 1 : 0, n,
                           off, counts, key_t, row_t, w_t, rec);
    else
        hipLaunchKernelGGL(place_kernel<false>, dim3(ge), dim3(256), 0, st, col, nx, row, w, roff, mean ? 1 : 0,
                           n, off, counts, key_t, row_t, w_t, rec);
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

#define GEOT_BY_V(V, CALL)                   \
    do {                                     \
        if ((V) == 4) { constexpr int VV = 4; CALL; } \
        else if ((V) == 2) { constexpr int VV = 2; CALL; } \
        else { constexpr int VV = 1; CALL; } \
    } while (0)

hipError_t launch_seg_bwd_bcast(const float *gout, const int64_t *idx, const int64_t *off, int64_t n,
                                int64_t S, int64_t F, int V, bool mean, float *gsrc, hipStream_t st) {
    if (n <= 0) return hipSuccess;
    const int64_t gb = grid_rows(n, (int)(F / V));
    if (gb > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    const unsigned g = (unsigned)gb;
    if (mean)
        GEOT_BY_V(V, hipLaunchKernelGGL((seg_bwd_bcast_kernel<VV, true>), dim3(g), dim3(256), 0, st,
                                        gout, idx, off, n, S, F, gsrc));
    else
        GEOT_BY_V(V, hipLaunchKernelGGL((seg_bwd_bcast_kernel<VV, false>), dim3(g), dim3(256), 0, st,
                                        gout, idx, off, n, S, F, gsrc));
    return hipGetLastError();
}

hipError_t launch_seg_bwd_max(const float *gout, const int64_t *idx, const float *src, const float *out,
                              int64_t n, int64_t S, int64_t F, int V, unsigned long long *arg, float *gsrc,
                              hipStream_t st) {
    if (n <= 0) return hipSuccess;
    hipError_t e = launch_fill_u64(arg, S * F, ~0ull, st);
    if (e != hipSuccess) return e;
    const int64_t gb = grid_rows(n, (int)(F / V));
    if (gb > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    const unsigned g = (unsigned)gb;
    GEOT_BY_V(V, hipLaunchKernelGGL((seg_bwd_max_arg_kernel<VV>), dim3(g), dim3(256), 0, st, src, idx,
                                    out, n, S, F, arg));
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    GEOT_BY_V(V, hipLaunchKernelGGL((seg_bwd_max_write_kernel<VV>), dim3(g), dim3(256), 0, st, gout,
                                    idx, arg, n, S, F, gsrc));
    return hipGetLastError();
}

hipError_t launch_gs_bwd(const float *X, int64_t nx, const int64_t *col, const float *w, const int64_t *row,
                         const int64_t *off, const float *out, const float *gout, int64_t n, int64_t R,
                         int64_t F, int V, int op, unsigned long long *arg, float *gX, float *gw,
                         hipStream_t st) {
    if (n <= 0) return hipSuccess;
    const int64_t gb = grid_rows(n, (int)(F / V));
    if (gb > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    const unsigned g = (unsigned)gb;
    hipError_t e;
    if (op == GEOT_BWD_MAX) {
        e = launch_fill_u64(arg, R * F, ~0ull, st);
        if (e != hipSuccess) return e;
        GEOT_BY_V(V, hipLaunchKernelGGL((gs_bwd_max_arg_kernel<VV>), dim3(g), dim3(256), 0, st, X, nx,
                                        col, w, row, out, n, R, F, arg));
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (gX) {
        e = launch_fill(gX, nx, F, F, 0.0f, st);
        if (e != hipSuccess) return e;
        if (op == GEOT_BWD_SUM)
            GEOT_BY_V(V, hipLaunchKernelGGL((gs_bwd_x_kernel<VV, GEOT_BWD_SUM>), dim3(g), dim3(256), 0, st,
                                            col, nx, w, row, off, arg, gout, n, R, F, gX));
        else if (op == GEOT_BWD_MEAN)
            GEOT_BY_V(V, hipLaunchKernelGGL((gs_bwd_x_kernel<VV, GEOT_BWD_MEAN>), dim3(g), dim3(256), 0,
                                            st, col, nx, w, row, off, arg, gout, n, R, F, gX));
        else
            GEOT_BY_V(V, hipLaunchKernelGGL((gs_bwd_x_kernel<VV, GEOT_BWD_MAX>), dim3(g), dim3(256), 0, st,
                                            col, nx, w, row, off, arg, gout, n, R, F, gX));
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (gw) {
        if (op == GEOT_BWD_SUM)
            GEOT_BY_V(V, hipLaunchKernelGGL((gs_bwd_w_kernel<VV, GEOT_BWD_SUM>), dim3(g), dim3(256), 0, st,
                                            X, nx, col, row, off, arg, gout, n, R, F, gw));
        else if (op == GEOT_BWD_MEAN)
            GEOT_BY_V(V, hipLaunchKernelGGL((gs_bwd_w_kernel<VV, GEOT_BWD_MEAN>), dim3(g), dim3(256), 0,
                                            st, X, nx, col, row, off, arg, gout, n, R, F, gw));
        else
            GEOT_BY_V(V, hipLaunchKernelGGL((gs_bwd_w_kernel<VV, GEOT_BWD_MAX>), dim3(g), dim3(256), 0, st,
                                            X, nx, col, row, off, arg, gout, n, R, F, gw));
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace geot
