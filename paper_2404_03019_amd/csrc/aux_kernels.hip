// Small helper kernels: output fill, segment starts from a sorted index,
// segment-length statistics and the precondition check.
#include "common.h"

namespace geot {

namespace {

__global__ __launch_bounds__(256) void fill_kernel(float *out, int64_t rows, int64_t F, int64_t ld,
                                                   float value) {
    const int64_t total = rows * F;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t r = i / F;
        out[r * ld + (i - r * F)] = value;
    }
}

// off[s] = first row i with idx[i] >= s. Row i writes the starts of every
// segment in (idx[i-1], idx[i]] (so empty segments get the next start), and
// the last row also writes (idx[n-1], S] = n. Runs longer than kGapRun go to
// the gap list instead (value = the row they start at). With `first`, the
// ids of the first and the last row of every block of 2^shift rows go to
// first[2b] and first[2b + 1] (the segments a block of the gradient kernels
// starts and ends in).
template <typename I>
constexpr int kOffsetsRowsPerThread = 64 / (int)sizeof(I);

template <typename I>
__global__ __launch_bounds__(256) void offsets_kernel(const I *idx, int64_t n, int64_t S,
                                                      int64_t *off, GapList gaps, int64_t *first, int shift) {
    auto put = [&](int64_t lo, int64_t hi, int64_t row) {  // off[lo, hi) = row
        lo = max(lo, (int64_t)0);
        hi = min(hi, S + 1);
        if (hi - lo > kGapRun && gap_push(gaps, lo, hi, row, 0, 0, 1)) return;
        for (int64_t t = lo; t < hi; ++t) off[t] = row;
    };
    auto row_done = [&](int64_t i, int64_t s, int64_t sp) {
        if (s != sp) put(sp + 1, s + 1, i);
        if (i == n - 1) put(s + 1, S + 1, n);
        if (first) {   // ids of the first and the last row of each block of 2^shift rows
            const int64_t mask = ((int64_t)1 << shift) - 1;
            if ((i & mask) == 0) first[2 * (i >> shift)] = s;
            if ((i & mask) == mask || i == n - 1) first[2 * (i >> shift) + 1] = s;
        }
    };
    // kOffsetsRowsPerThread<I> consecutive ids (64 bytes) per thread in 16-byte loads (idx
    // 16-byte aligned; the launcher checks); the id before them comes from the next lower lane,
    // lane 0 loads its own
    constexpr int kR = kOffsetsRowsPerThread<I>;
    const int lane = threadIdx.x & 63;
    for (int64_t b0 = (int64_t)blockIdx.x * (256 * kR); b0 < n; b0 += (int64_t)gridDim.x * (256 * kR)) {
        const int64_t base = b0 + (int64_t)threadIdx.x * kR;
        int64_t cur[kR];
        if (base + kR <= n) {
#pragma unroll
            for (int v = 0; v < kR * (int)sizeof(I) / 16; ++v) {
                if constexpr (sizeof(I) == 8) {
                    const longlong2 a = *reinterpret_cast<const longlong2 *>(idx + base + 2 * v);
                    cur[2 * v] = a.x; cur[2 * v + 1] = a.y;
                } else {
                    const int4 a = *reinterpret_cast<const int4 *>(idx + base + 4 * v);
                    cur[4 * v] = a.x; cur[4 * v + 1] = a.y; cur[4 * v + 2] = a.z; cur[4 * v + 3] = a.w;
                }
            }
        } else {
#pragma unroll
            for (int k = 0; k < kR; ++k) cur[k] = base + k < n ? (int64_t)idx[base + k] : 0;
        }
        int64_t prev = __shfl_up((long long)cur[kR - 1], 1u, 64);
        if (lane == 0) prev = base > 0 && base - 1 < n ? (int64_t)idx[base - 1] : -1;
#pragma unroll
        for (int k = 0; k < kR; ++k) {
            const int64_t i = base + k;
            if (i >= n) break;
            row_done(i, cur[k], k == 0 ? prev : cur[k - 1]);
        }
    }
}

// The same with one id per thread and step, for an index that is not 16-byte aligned.
template <typename I>
__global__ __launch_bounds__(256) void offsets_unaligned_kernel(const I *idx, int64_t n, int64_t S,
                                                                int64_t *off, GapList gaps, int64_t *first,
                                                                int shift) {
    auto put = [&](int64_t lo, int64_t hi, int64_t row) {  // off[lo, hi) = row
        lo = max(lo, (int64_t)0);
        hi = min(hi, S + 1);
        if (hi - lo > kGapRun && gap_push(gaps, lo, hi, row, 0, 0, 1)) return;
        for (int64_t t = lo; t < hi; ++t) off[t] = row;
    };
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t s = (int64_t)idx[i];
        const int64_t sp = i > 0 ? (int64_t)idx[i - 1] : -1;
        if (s != sp) put(sp + 1, s + 1, i);
        if (i == n - 1) put(s + 1, S + 1, n);
        if (first) {
            const int64_t mask = ((int64_t)1 << shift) - 1;
            if ((i & mask) == 0) first[2 * (i >> shift)] = s;
            if ((i & mask) == mask || i == n - 1) first[2 * (i >> shift) + 1] = s;
        }
    }
}

// One block per record at a time: rows [first, end) of the record's column tile = 0.
template <int V>
__global__ __launch_bounds__(256) void gap_fill_rows_kernel(float *out, int64_t F, int64_t ld,
                                                            int64_t tw, int64_t rows, GapList g, uint32_t *arg) {
    gap_fill_rows_body<V>(out, F, ld, tw, rows, g, blockIdx.x, gridDim.x, arg);
}

__global__ __launch_bounds__(256) void gap_fill_i64_kernel(int64_t *arr, int64_t len, GapList g) {
    const unsigned cnt = gap_count(g);
    for (unsigned q = blockIdx.x; q < cnt; q += gridDim.x) {
        const int64_t *r = g.rec + 3 * (int64_t)q;
        const int64_t lo = max(r[0], (int64_t)0), hi = min(r[1], len), v = r[2];
        for (int64_t t = lo + threadIdx.x; t < hi; t += 256) arr[t] = v;
    }
    gap_done(g, blockIdx.x, gridDim.x, cnt);
}

__global__ __launch_bounds__(256) void len_stats_kernel(const int64_t *off, int64_t S,
                                                        unsigned long long *acc) {
    unsigned long long sq = 0, mx = 0, ne = 0;
    for (int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; s < S;
         s += (int64_t)gridDim.x * blockDim.x) {
        const int64_t len = off[s + 1] - off[s];
        const unsigned long long l = len > 0 ? (unsigned long long)len : 0ull;
        sq += l * l;
        mx = l > mx ? l : mx;
        ne += len == 0 ? 1ull : 0ull;
    }
    __shared__ unsigned long long s_sq[256], s_mx[256], s_ne[256];
    s_sq[threadIdx.x] = sq;
    s_mx[threadIdx.x] = mx;
    s_ne[threadIdx.x] = ne;
    __syncthreads();
    for (int h = 128; h > 0; h >>= 1) {
        if ((int)threadIdx.x < h) {
            s_sq[threadIdx.x] += s_sq[threadIdx.x + h];
            s_mx[threadIdx.x] = max(s_mx[threadIdx.x], s_mx[threadIdx.x + h]);
            s_ne[threadIdx.x] += s_ne[threadIdx.x + h];
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        atomicAdd(&acc[0], s_sq[0]);
        atomicMax(&acc[1], s_mx[0]);
        atomicAdd(&acc[2], s_ne[0]);
    }
}

__global__ __launch_bounds__(256) void check_kernel(const int64_t *idx, int64_t n, int64_t S,
                                                    const int64_t *col, int64_t nx,
                                                    unsigned int *flags) {
    unsigned int bad = 0;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t s = idx[i];
        if (s < 0 || s >= S) bad |= 1u;
        if (i > 0 && s < idx[i - 1]) bad |= 2u;
        if (col != nullptr) {
            const int64_t c = col[i];
            if (c < 0 || c >= nx) bad |= 1u;
        }
    }
    __shared__ unsigned int s_bad[256];
    s_bad[threadIdx.x] = bad;
    __syncthreads();
    for (int h = 128; h > 0; h >>= 1) {
        if ((int)threadIdx.x < h) s_bad[threadIdx.x] |= s_bad[threadIdx.x + h];
        __syncthreads();
    }
    if (threadIdx.x == 0 && s_bad[0] != 0) atomicOr(flags, s_bad[0]);
}

__global__ void zero_u64_kernel(unsigned long long *p, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = 0ull;
}

unsigned grid_for(int64_t work, int64_t per_block, int64_t cap) {
    int64_t b = (work + per_block - 1) / per_block;
    if (b < 1) b = 1;
    if (b > cap) b = cap;
    return (unsigned)b;
}

}  // namespace

hipError_t launch_fill(float *out, int64_t rows, int64_t F, int64_t ld, float value,
                       hipStream_t stream) {
    if (rows <= 0 || F <= 0) return hipSuccess;
    hipLaunchKernelGGL(fill_kernel, dim3(grid_for(rows * F, 256 * 8, 65536)), dim3(256), 0, stream,
                       out, rows, F, ld, value);
    return hipGetLastError();
}

hipError_t launch_offsets(const int64_t *idx, int64_t n, int64_t S, int64_t *off, GapList gaps,
                          hipStream_t stream, int64_t *first, int shift) {
    if (n <= 0 || shift < 0 || shift > 40) return hipErrorInvalidValue;
    if (((uintptr_t)idx & 15) == 0)
        hipLaunchKernelGGL(offsets_kernel<int64_t>, dim3(grid_for(n, 256 * kOffsetsRowsPerThread<int64_t>, 1 << 20)),
                           dim3(256), 0, stream,
                           idx, n, S, off, gaps, first, shift);
    else
        hipLaunchKernelGGL(offsets_unaligned_kernel<int64_t>, dim3(grid_for(n, 256 * 4, 1 << 20)), dim3(256), 0,
                           stream, idx, n, S, off, gaps, first, shift);
    return hipGetLastError();
}

hipError_t launch_offsets_i32(const int32_t *idx, int64_t n, int64_t S, int64_t *off, GapList gaps,
                              hipStream_t stream, int64_t *first, int shift) {
    if (n <= 0 || shift < 0 || shift > 40) return hipErrorInvalidValue;
    if (((uintptr_t)idx & 15) == 0)
        hipLaunchKernelGGL(offsets_kernel<int32_t>, dim3(grid_for(n, 256 * kOffsetsRowsPerThread<int32_t>, 1 << 20)),
                           dim3(256), 0, stream,
                           idx, n, S, off, gaps, first, shift);
    else
        hipLaunchKernelGGL(offsets_unaligned_kernel<int32_t>, dim3(grid_for(n, 256 * 4, 1 << 20)), dim3(256), 0,
                           stream, idx, n, S, off, gaps, first, shift);
    return hipGetLastError();
}

// 1024 blocks: a list with many records keeps the chip busy, an empty list
// costs one counter read per block.
hipError_t launch_gap_fill_rows(float *out, int64_t F, int64_t ld, int V, int64_t tw, int64_t rows,
                                GapList gaps, uint32_t *arg, hipStream_t stream) {
    if (V == 4)
        hipLaunchKernelGGL(gap_fill_rows_kernel<4>, dim3(1024), dim3(256), 0, stream, out, F, ld, tw, rows, gaps, arg);
    else if (V == 2)
        hipLaunchKernelGGL(gap_fill_rows_kernel<2>, dim3(1024), dim3(256), 0, stream, out, F, ld, tw, rows, gaps, arg);
    else
        hipLaunchKernelGGL(gap_fill_rows_kernel<1>, dim3(1024), dim3(256), 0, stream, out, F, ld, tw, rows, gaps, arg);
    return hipGetLastError();
}

hipError_t launch_gap_fill_i64(int64_t *arr, int64_t len, GapList gaps, hipStream_t stream) {
    hipLaunchKernelGGL(gap_fill_i64_kernel, dim3(1024), dim3(256), 0, stream, arr, len, gaps);
    return hipGetLastError();
}

hipError_t launch_len_stats(const int64_t *off, int64_t S, unsigned long long *acc,
                            hipStream_t stream) {
    hipLaunchKernelGGL(len_stats_kernel, dim3(grid_for(S, 256 * 16, 4096)), dim3(256), 0, stream,
                       off, S, acc);
    return hipGetLastError();
}

hipError_t launch_check(const int64_t *idx, int64_t n, int64_t S, const int64_t *col, int64_t nx,
                        unsigned int *flags, hipStream_t stream) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(check_kernel, dim3(grid_for(n, 256 * 16, 8192)), dim3(256), 0, stream, idx,
                       n, S, col, nx, flags);
    return hipGetLastError();
}

hipError_t launch_zero_u64(unsigned long long *p, int64_t n, hipStream_t stream) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(zero_u64_kernel, dim3(grid_for(n, 256, 1024)), dim3(256), 0, stream, p, n);
    return hipGetLastError();
}

}  // namespace geot
