// Segment-parallel segment reduction for gfx950.
//
// Segment s covers rows off[s] .. off[s+1]-1 (segment starts come from one
// pass over the sorted index). A team of `groups` row groups of one wave
// (each row group: L lanes over the columns of one row, V floats per lane,
// NT times) owns one segment: group j of the team reduces rows off[s] + j,
// off[s] + j + groups, ... serially in registers, the team combines its
// groups with lane shuffles, and the team's first group stores the row once.
// groups == 1 is one sub-wave group per segment; groups == 64 / L is one
// whole wave per segment. No atomics and no partials, but the time of a team
// grows with its segment, so the selector keeps this family to short, even
// segments.
#include "common.h"

namespace geot {

namespace {

template <int RED, int MODE, int V, int NT, int L>
__global__ __launch_bounds__(kBlock) void sp_kernel(const SpArgs a) {
    constexpr int NV = V * NT;
    constexpr int GW = 64 / L;
    constexpr int TW = NT * L * V;
    constexpr int U = NV >= 4 ? 4 : 8;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int gw = lane / L;
    const int gl = lane - gw * L;
    const int team_size = a.groups;            // row groups per team (power of two <= GW)
    const int teams_per_wave = GW / team_size;
    const int team = gw / team_size;           // team within the wave
    const int tj = gw - team * team_size;      // group within the team

    const int64_t bidx = blockIdx.x / a.ntiles;
    const int tile = (int)(blockIdx.x - bidx * a.ntiles);
    const int64_t segs_per_block = (int64_t)(kBlock / 64) * teams_per_wave;
    const int64_t s = bidx * segs_per_block + (int64_t)wave * teams_per_wave + team;

    int64_t cb[NT];
    bool cv[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        cb[j] = (int64_t)tile * TW + (int64_t)(j * L + gl) * V;
        cv[j] = cb[j] < a.F;
        // F no multiple of V: the vector that would cross the row's end takes the last V
        // columns (4-byte aligned loads and stores; shared columns reduce identically)
        if (cv[j]) cb[j] = min(cb[j], a.F - V);
    }
    const float neutral = red_neutral<RED>();
    const bool live = s < a.S;

    int64_t beg = 0, end = 0;
    if (live) {
        beg = a.off[s];
        end = a.off[s + 1];
        const int64_t nrows = a.off[a.S];  // total rows: keeps garbage starts in bounds
        beg = min(max(beg, (int64_t)0), nrows);
        end = min(max(end, beg), nrows);
    }
    float acc[NV];
#pragma unroll
    for (int k = 0; k < NV; ++k) acc[k] = neutral;

    auto load_term = [&](int64_t r, float *x) {
        const float *p;
        float wt = 1.0f;
        bool ok = true;
        if constexpr (MODE == SRC_GATHER) {
            const int64_t c = a.col[r];
            if (a.w) wt = a.w[r];
            ok = (uint64_t)c < (uint64_t)a.num_x_rows;
            p = a.src + c * a.ld_src;
        } else {
            p = a.src + r * a.ld_src;
        }
#pragma unroll
        for (int j = 0; j < NT; ++j) {
            if (cv[j] && ok) {
                load_vec<V>(p + cb[j], x + j * V);
                if constexpr (MODE == SRC_GATHER) {
#pragma unroll
                    for (int k = 0; k < V; ++k) x[j * V + k] = wt * x[j * V + k];
                }
            } else {
#pragma unroll
                for (int k = 0; k < V; ++k) x[j * V + k] = neutral;
            }
        }
    };

    if (live) {
        // A group's rows of one segment form one chain, as long as the segment. For sum the
        // rows add into `run`, which joins acc every kSpRun of the group's rows: a chain of n
        // rows then rounds like runs of kSpRun terms and n / kSpRun run sums, so the fp32
        // error stays within the bound on long segments of same-signed values too (one
        // serial chain of 600,000 such terms is off by about 2.6e-5 of their absolute sum).
        constexpr int kSpRun = 256;
        float run[NV];
#pragma unroll
        for (int k = 0; k < NV; ++k) run[k] = neutral;
        int steps = 0;
        int64_t r = beg + tj;
        const int64_t stride = team_size;
        for (; r + (U - 1) * stride < end; r += U * stride) {
            float x[U][NV];
#pragma unroll
            for (int u = 0; u < U; ++u) load_term(r + u * stride, x[u]);
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int k = 0; k < NV; ++k) run[k] = red_apply<RED>(run[k], x[u][k]);
            if (RED == RED_SUM && ++steps == kSpRun / U) {
#pragma unroll
                for (int k = 0; k < NV; ++k) {
                    acc[k] += run[k];
                    run[k] = 0.0f;
                }
                steps = 0;
            }
        }
        for (; r < end; r += stride) {
            float x[NV];
            load_term(r, x);
#pragma unroll
            for (int k = 0; k < NV; ++k) run[k] = red_apply<RED>(run[k], x[k]);
        }
#pragma unroll
        for (int k = 0; k < NV; ++k) acc[k] = red_apply<RED>(acc[k], run[k]);
    }
    // combine the groups of a team (groups are L lanes apart, teams are aligned)
    for (int d = team_size / 2; d >= 1; d >>= 1) {
#pragma unroll
        for (int k = 0; k < NV; ++k) {
            const float o = shfl_down_f(acc[k], d * L);
            acc[k] = red_apply<RED>(acc[k], o);
        }
    }
    if (live && tj == 0) {
        const int64_t n = end - beg;
        float *o = a.out + s * a.ld_out;
        const float fn = (float)n;
#pragma unroll
        for (int j = 0; j < NT; ++j) {
            if (!cv[j]) continue;
            float t[V];
#pragma unroll
            for (int k = 0; k < V; ++k) {
                const float x = acc[j * V + k];
                t[k] = n == 0 ? 0.0f : (a.mean ? x / fn : x);
            }
            store_vec_nt<V>(o + cb[j], t);
        }
    }
}

template <int RED, int MODE, int V, int NT, int L>
hipError_t launch_one(const SpArgs &a, hipStream_t stream) {
    constexpr int GW = 64 / L;
    if (a.groups < 1 || a.groups > GW || (a.groups & (a.groups - 1)) != 0) return hipErrorInvalidValue;
    const int64_t segs_per_block = (int64_t)(kBlock / 64) * (GW / a.groups);
    const int64_t nb = (a.S + segs_per_block - 1) / segs_per_block;
    const int64_t blocks = nb * a.ntiles;
    if (blocks <= 0) return hipSuccess;
    if (blocks > 0x7fffffffLL) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL((sp_kernel<RED, MODE, V, NT, L>), dim3((unsigned)blocks), dim3(kBlock), 0,
                       stream, a);
    return hipGetLastError();
}

template <int RED, int MODE, int V, int NT>
hipError_t by_lanes(const SpArgs &a, int L, hipStream_t st) {
    if constexpr (NT > 1) {
        if (L != 64) return hipErrorInvalidValue;
        return launch_one<RED, MODE, V, NT, 64>(a, st);
    } else {
        switch (L) {
            case 1: return launch_one<RED, MODE, V, 1, 1>(a, st);
            case 2: return launch_one<RED, MODE, V, 1, 2>(a, st);
            case 4: return launch_one<RED, MODE, V, 1, 4>(a, st);
            case 8: return launch_one<RED, MODE, V, 1, 8>(a, st);
            case 16: return launch_one<RED, MODE, V, 1, 16>(a, st);
            case 32: return launch_one<RED, MODE, V, 1, 32>(a, st);
            case 64: return launch_one<RED, MODE, V, 1, 64>(a, st);
            default: return hipErrorInvalidValue;
        }
    }
}

template <int RED, int MODE>
hipError_t by_shape(const SpArgs &a, int V, int NT, int L, hipStream_t st) {
    if (V == 4 && NT == 1) return by_lanes<RED, MODE, 4, 1>(a, L, st);
    if (V == 3 && NT == 1) {  // rows of 3 floats, one lane a row
        if (L != 1) return hipErrorInvalidValue;
        return launch_one<RED, MODE, 3, 1, 1>(a, st);
    }
    if (V == 2 && NT == 1) return by_lanes<RED, MODE, 2, 1>(a, L, st);
    if (V == 2 && NT == 2) return by_lanes<RED, MODE, 2, 2>(a, L, st);
    if (V == 1 && NT == 1) return by_lanes<RED, MODE, 1, 1>(a, L, st);
    if (V == 1 && NT == 2) return by_lanes<RED, MODE, 1, 2>(a, L, st);
    if (V == 1 && NT == 4) return by_lanes<RED, MODE, 1, 4>(a, L, st);
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_sp(const SpArgs &a, int red, int mode, int V, int NT, int L, hipStream_t stream) {
    if (red == RED_SUM) {
        if (mode == SRC_ROWS) return by_shape<RED_SUM, SRC_ROWS>(a, V, NT, L, stream);
        if (mode == SRC_GATHER) return by_shape<RED_SUM, SRC_GATHER>(a, V, NT, L, stream);
    } else if (red == RED_MAX) {
        if (mode == SRC_ROWS) return by_shape<RED_MAX, SRC_ROWS>(a, V, NT, L, stream);
        if (mode == SRC_GATHER) return by_shape<RED_MAX, SRC_GATHER>(a, V, NT, L, stream);
    }
    return hipErrorInvalidValue;
}

}  // namespace geot
