// Host side of libgeot_hip: argument checks, kernel selection, temporary
// memory, launch sequencing and the extern "C" entry points of geot.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/geot.h"
#include "internal.h"
#include "selector_generated.h"

// Temporary memory of geot_segment_reduce_noalloc, for callers that cannot allocate:
// one array per GPU, held from the library's load until the process ends. In host code
// `scratch` names a host-side stand-in, not device memory: kernels and copies take the
// per-device address that hipGetSymbolAddress returns for it (noalloc_scratch below).
static constexpr size_t kNoAllocBytes = (size_t)128 << 20;
static __device__ __align__(256) char scratch[kNoAllocBytes];

namespace geot {
namespace {

thread_local std::string t_detail;
thread_local geot_kernel_choice_t t_last_choice = {0, 0, 0, 0, 0, 0};

geot_status_t fail(geot_status_t st, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    t_detail = buf;
    return st;
}

geot_status_t hip_fail(hipError_t e, const char *what) {
    return fail(GEOT_ERROR_HIP, "%s: %s (%d)", what, hipGetErrorString(e), (int)e);
}

#define GEOT_HIP(expr, what)                        \
    do {                                            \
        hipError_t e_ = (expr);                     \
        if (e_ != hipSuccess) return hip_fail(e_, what); \
    } while (0)

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

int pow2ceil(int64_t x) {
    int p = 1;
    while (p < x && p < (1 << 30)) p <<= 1;
    return p;
}

bool is_pow2(int64_t x) { return x > 0 && (x & (x - 1)) == 0; }

// ---------------------------------------------------------------------------
// temporary device memory: one stream-ordered pool per device
// ---------------------------------------------------------------------------
std::mutex g_pool_mu;
std::map<int, hipMemPool_t> g_pools;

geot_status_t scratch_alloc(void **p, size_t bytes, hipStream_t st) {
    *p = nullptr;
    if (bytes == 0) return GEOT_SUCCESS;
    int dev = 0;
    GEOT_HIP(hipGetDevice(&dev), "hipGetDevice");
    hipMemPool_t pool = nullptr;
    {
        std::lock_guard<std::mutex> lk(g_pool_mu);
        auto it = g_pools.find(dev);
        if (it == g_pools.end()) {
            hipMemPoolProps props;
            memset(&props, 0, sizeof(props));
            props.allocType = hipMemAllocationTypePinned;
            props.location.type = hipMemLocationTypeDevice;
            props.location.id = dev;
            GEOT_HIP(hipMemPoolCreate(&pool, &props), "hipMemPoolCreate");
            uint64_t keep = UINT64_MAX;  // keep freed blocks for reuse
            GEOT_HIP(hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &keep),
                     "hipMemPoolSetAttribute");
            g_pools[dev] = pool;
        } else {
            pool = it->second;
        }
    }
    GEOT_HIP(hipMallocFromPoolAsync(p, bytes, pool, st), "hipMallocFromPoolAsync");
    return GEOT_SUCCESS;
}

geot_status_t scratch_free(void *p, hipStream_t st) {
    if (p) GEOT_HIP(hipFreeAsync(p, st), "hipFreeAsync");
    return GEOT_SUCCESS;
}

struct ScratchGuard {
    void *p = nullptr;
    hipStream_t st = nullptr;
    ~ScratchGuard() {
        if (p) (void)hipFreeAsync(p, st);
    }
};

// Reduction calls keep their temporary buffer per (device, stream) and reuse it
// in stream order, growing it (stream-ordered free of the old block, then a new
// allocation) when a call needs more. Kernels of one stream run in order, so
// consecutive calls never overlap on the buffer. The buffer starts with the
// gap list (two counters and kGapCap records); the counters are zeroed when
// the buffer is allocated and, after that, by the fill passes themselves.
struct StreamKey {
    int dev;
    hipStream_t st;
    bool operator<(const StreamKey &o) const { return dev != o.dev ? dev < o.dev : st < o.st; }
};
struct StreamCtx {
    void *p = nullptr;
    size_t bytes = 0;
    bool dirty = false;     // a launch failed after the gap list was handed out
    bool captured = false;  // a call on this buffer was captured into a graph, which keeps its address
};
std::mutex g_cache_mu;
std::map<StreamKey, StreamCtx> g_cache;
// Buffers replaced by a larger one after a graph captured them: a replay of that graph
// still reads and writes them, so they are freed only by geot_release_scratch.
std::vector<std::pair<int, void *>> g_retired;

constexpr size_t kGapHeader = 256;
constexpr size_t kGapArea = kGapHeader + (size_t)kGapCap * 3 * sizeof(int64_t);

// `user` gets `bytes` of scratch after the gap list; `g` the list of this call
// (NULL when the call runs no gap-fill pass: only a call that runs one may take
// the list, since its fill pass is what empties it again).
geot_status_t stream_scratch(size_t bytes, hipStream_t st, void **user, GapList *g,
                             StreamCtx **ctx_out) {
    *user = nullptr;
    int dev = 0;
    GEOT_HIP(hipGetDevice(&dev), "hipGetDevice");
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    GEOT_HIP(hipStreamIsCapturing(st, &cap), "hipStreamIsCapturing");
    const bool capturing = cap != hipStreamCaptureStatusNone;
    std::lock_guard<std::mutex> lk(g_cache_mu);
    StreamCtx &e = g_cache[StreamKey{dev, st}];
    const size_t need = kGapArea + ((bytes + 255) & ~(size_t)255);
    bool fresh = false;
    if (e.bytes < need) {
        // Growing inside a capture would record the free and the allocation into the graph.
        if (capturing)
            return fail(GEOT_ERROR_INVALID_VALUE,
                        "stream capture: the stream's temporary buffer holds %zu bytes and this call needs %zu; "
                        "make one call of these shapes on the stream before capturing",
                        e.bytes, need);
        const size_t grown = std::max(need, e.bytes + e.bytes / 2);  // grow by half at least
        if (e.p) {
            if (e.captured) g_retired.emplace_back(dev, e.p);  // a captured graph still uses it
            else GEOT_HIP(hipFreeAsync(e.p, st), "hipFreeAsync");
            e.p = nullptr;
            e.bytes = 0;
            e.captured = false;
        }
        void *q = nullptr;
        geot_status_t s = scratch_alloc(&q, grown, st);
        if (s != GEOT_SUCCESS) return s;
        e.p = q;
        e.bytes = grown;
        fresh = true;
    }
    if (capturing) e.captured = true;
    if (fresh || e.dirty) {
        GEOT_HIP(launch_zero_u64((unsigned long long *)e.p, kGapHeader / 8, st), "launch zero kernel");
        e.dirty = false;
    }
    if (g) {
        unsigned *ctrl = (unsigned *)e.p;
        g->count = ctrl;
        g->ticket = ctrl + 1;
        g->rec = (int64_t *)((char *)e.p + kGapHeader);
    }
    *user = bytes ? (char *)e.p + kGapArea : nullptr;
    *ctx_out = &e;
    return GEOT_SUCCESS;
}

// Device memory of one reduction call given by the caller (the *_ws calls): its first
// kGapArea bytes hold the gap list, zeroed by the call itself, then the partials.
struct Workspace {
    char *p;
    size_t bytes;
};

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// The temporary memory of one call: `bytes` after the gap list, from the caller's workspace
// when `ws` is given, else from the stream's cached buffer.
geot_status_t call_scratch(size_t bytes, hipStream_t st, const Workspace *ws, void **user, GapList *g,
                           StreamCtx **ctx_out) {
    if (!ws) return stream_scratch(bytes, st, user, g, ctx_out);
    *ctx_out = nullptr;
    const size_t need = kGapArea + align256(bytes);
    if (ws->bytes < need)
        return fail(GEOT_ERROR_INVALID_VALUE, "workspace of %zu bytes, this call needs %zu", ws->bytes, need);
    GEOT_HIP(launch_zero_u64((unsigned long long *)ws->p, kGapHeader / 8, st), "launch zero kernel");
    unsigned *ctrl = (unsigned *)ws->p;
    g->count = ctrl;
    g->ticket = ctrl + 1;
    g->rec = (int64_t *)(ws->p + kGapHeader);
    *user = bytes ? ws->p + kGapArea : nullptr;
    return GEOT_SUCCESS;
}

// Marks the context so the next call re-zeroes the gap counters.
geot_status_t poison(StreamCtx *ctx, geot_status_t s) {
    if (s != GEOT_SUCCESS && ctx) {
        std::lock_guard<std::mutex> lk(g_cache_mu);
        ctx->dirty = true;
    }
    return s;
}

// ---------------------------------------------------------------------------
// measurement hooks (geot_profile_begin / _end)
// ---------------------------------------------------------------------------
struct Profile {
    bool armed = false;
    int cap = 0;
    std::vector<std::pair<hipEvent_t, hipEvent_t>> ev;
} g_prof;

// Set while geot_segment_reduce_noalloc runs: it records no profiling events (creating
// them is a runtime allocation).
thread_local bool t_no_events = false;

bool prof_take(hipEvent_t *a, hipEvent_t *b) {
    if (t_no_events || !g_prof.armed || (int)g_prof.ev.size() >= g_prof.cap) return false;
    hipEvent_t e0, e1;
    if (hipEventCreate(&e0) != hipSuccess) return false;
    if (hipEventCreate(&e1) != hipSuccess) {
        (void)hipEventDestroy(e0);
        return false;
    }
    g_prof.ev.emplace_back(e0, e1);
    *a = e0;
    *b = e1;
    return true;
}

// ---------------------------------------------------------------------------
// problem description and choice resolution
// ---------------------------------------------------------------------------
struct Problem {
    bool gather;
    const void *src;       // rows or X, of type elem
    int64_t num_x_rows;
    const void *col;       // int32 when idx32, else int64 (as idx)
    const float *w;
    const void *idx;
    int64_t nnz, S, F;
    geot_op_t op;
    float *out;
    int elem = ELEM_F32;   // storage type of src / X
    int idx32 = 0;         // idx and col hold int32
    int meta_stride = 1;   // gather: idx, col and w of edge e at [e * meta_stride] (internal records)
    uint32_t *arg = nullptr;   // max only: each output element's recipient row (edge), [S x F]
    size_t esize() const { return elem == ELEM_F32 ? 4 : 2; }
    size_t isize() const { return idx32 ? 4 : 8; }
    bool typed() const { return elem != ELEM_F32 || idx32 != 0; }
};

struct Resolved {
    int family, V, NT, L, K, groups, ntiles;
    int nt_rows;     // EP rows mode: non-temporal row loads
    int tile_major;  // EP level 0: column tiles in sequence (blocks of one tile together)
};

int max_nt(int V) { return V == 4 ? 1 : (V == 2 ? 2 : 4); }

bool valid_shape(int V, int NT, int L) {
    if (!(V == 1 || V == 2 || V == 4 || V == 8)) return false;
    if (!is_pow2(L) || L > 64) return false;
    if (V == 8) return NT == 1 && L <= 32;
    if (NT == 1) return true;
    return L == 64 && NT <= max_nt(V) && is_pow2(NT);
}

void auto_lanes(int64_t F, int V, int *L, int *NT) {
    const int64_t vecs = ceil_div(F, V);
    if (V == 8) {  // 16-bit storage: at most 32 lanes, more column tiles beyond 256 columns
        *L = (int)std::min<int64_t>(32, pow2ceil(vecs));
        *NT = 1;
    } else if (vecs <= 64) {
        *L = pow2ceil(vecs);
        *NT = 1;
    } else {
        *L = 64;
        *NT = std::min<int>(max_nt(V), pow2ceil(ceil_div(vecs, 64)));
    }
}

int auto_rows(int64_t nnz, int L, int V, int NT, int ntiles, int64_t esize) {
    const int64_t G = kBlock / L;
    const int64_t row_bytes = (int64_t)L * V * NT * esize;
    const int64_t target_rows = std::max<int64_t>(512, (256 * 1024) / row_bytes);
    int64_t K = ceil_div(target_rows, G);
    // keep at least ~1024 blocks in flight when the input allows it
    const int64_t k_fill = ceil_div(nnz, G * std::max<int64_t>(1, 1024 / ntiles));
    K = std::min(K, std::max<int64_t>(k_fill, 1));
    return (int)std::max<int64_t>(1, std::min<int64_t>(K, 512));
}

int widest_vec(const Problem &p) {
    // src loads of V elements; fp32 stores of at most 4 floats (V = 8 stores 2 x 4)
    auto aligned = [&](int V) {
        const uintptr_t ms = (uintptr_t)(p.esize() * V - 1), mo = (uintptr_t)(4 * std::min(V, 4) - 1);
        if (p.F % V != 0) return false;
        if (((uintptr_t)p.src & ms) != 0 || (((uintptr_t)p.out | (uintptr_t)p.arg) & mo) != 0) return false;
        return true;
    };
    if (p.esize() == 2 && aligned(8)) return 8;
    if (aligned(4)) return 4;
    if (aligned(2)) return 2;
    return 1;
}

// fp32 rows whose width is no multiple of 4 still move in 4-float vectors: gfx950 loads
// and stores them at any 4-byte aligned address, and the vector that would cross a row's
// end takes the row's last 4 columns (overlapping its neighbour). Rows of 3 floats take
// one 3-float vector a lane. 0: neither applies.
int ragged_vec(const Problem &p) {
    if (p.elem != ELEM_F32 || p.F < 3 || p.F % 4 == 0) return 0;
    if (((uintptr_t)p.src & 3) != 0 || (((uintptr_t)p.out | (uintptr_t)p.arg) & 3) != 0) return 0;
    return p.F == 3 ? 3 : 4;
}

geot_status_t resolve(const Problem &p, const geot_kernel_choice_t &c, Resolved *r,
                      bool from_selector = false) {
    const int loads = GEOT_FLAG_NT_LOADS | GEOT_FLAG_CACHED_LOADS;
    const int known = loads | GEOT_FLAG_TILE_MAJOR;
    if ((c.flags & ~known) != 0 || (c.flags & loads) == loads)
        return fail(GEOT_ERROR_UNSUPPORTED, "choice.flags: unknown bit, or both load policies");
    r->family = c.family == GEOT_FAMILY_AUTO ? GEOT_FAMILY_EP : c.family;
    if (r->family != GEOT_FAMILY_EP && r->family != GEOT_FAMILY_SP)
        return fail(GEOT_ERROR_UNSUPPORTED, "unknown kernel family %d", c.family);
    if (r->family == GEOT_FAMILY_SP && p.typed())
        return fail(GEOT_ERROR_UNSUPPORTED, "the segment-parallel family takes fp32 data with int64 ids only");
    if (r->family == GEOT_FAMILY_SP && p.arg)
        return fail(GEOT_ERROR_UNSUPPORTED, "recipients come from the element-parallel family only");
    const int vmax = widest_vec(p);
    // ragged rows: 4-float vectors (3 for F = 3) where the width allows no exact one (3-float
    // vectors: one lane a row)
    const int vrag = ragged_vec(p);
    int V = c.vec == 0 ? (vrag ? vrag : vmax) : c.vec;
    int lanes = c.lanes, rows = c.rows;
    if (V == 3 && lanes > 1) V = vmax;   // a 3-float vector covers the row alone
    if (from_selector && p.esize() == 2 && vmax == 8) {
        // tree leaves are fit on fp32 shapes, which load 4 floats here (F % 8 == 0): load 8
        // 16-bit elements instead, keeping the columns of one row group and the bytes it
        // reads (half the lanes, twice the rows)
        const int v32 = c.vec != 0 ? std::min(c.vec, 4) : 4;
        V = 8;
        if (lanes != 0) lanes = std::max(1, lanes * v32 / V);
        if (rows != 0) rows = std::min(4096, rows * V / v32);
    }
    if (from_selector && p.arg && rows != 0) {
        // Carrying the recipients doubles what the block scan moves and holds registers (the
        // SpMM gather: 94 -> 114 VGPRs, 4 waves per SIMD); longer row runs amortise the scan
        // over more rows. Twice the tree's run, measured against 1x, 2x, 4x and 8x: the
        // power-law graph 2.70 -> 2.54 ms (plain max 2.36), the SpMM gather 5.86 -> 5.59 ms
        // (plain 5.19), in bf16 / int32 4.06 -> 3.91 ms; 4x was within 2 % on the gathers and
        // 9 % slower on the power-law graph.
        rows = std::min(4096, rows * 2);
    }
    if (!(V == 1 || V == 2 || V == 3 || V == 4 || V == 8))
        return fail(GEOT_ERROR_UNSUPPORTED, "vec must be 1, 2, 4 or (16-bit storage) 8");
    if (V == 8 && p.esize() != 2) return fail(GEOT_ERROR_UNSUPPORTED, "vec 8 needs 16-bit storage");
    if (V == 3 && c.vec == 3 && vrag != 3)
        return fail(GEOT_ERROR_UNSUPPORTED, "vec 3 needs fp32 rows of 3 floats");
    if (V != vrag || V == 0) {
        if (V == 3) V = vmax;
        while (V > vmax) V >>= 1;  // clamp to what F and the pointers allow
    }
    int L, NT;
    auto_lanes(p.F, V, &L, &NT);
    if (lanes != 0) {
        if (!is_pow2(lanes) || lanes > 64)
            return fail(GEOT_ERROR_UNSUPPORTED, "lanes must be a power of two <= 64");
        L = V == 8 ? std::min(lanes, 32) : lanes;
        if (L != 64) NT = 1;
    }
    if (!valid_shape(V, NT, L)) NT = 1;
    r->V = V;
    r->NT = NT;
    r->L = L;
    const int64_t TW = (int64_t)L * V * NT;
    const int64_t ntiles = ceil_div(p.F, TW);
    if (ntiles > 4096) return fail(GEOT_ERROR_UNSUPPORTED, "F too large for lanes*vec");
    r->ntiles = (int)ntiles;
    if (rows < 0 || rows > 4096) return fail(GEOT_ERROR_UNSUPPORTED, "rows must be in 0..4096");
    // Non-temporal row loads where a row group's load covers whole 128-byte lines: the
    // element-parallel rows mode, a tile and a row of at least 128 bytes.
    const bool nt_ok = r->family == GEOT_FAMILY_EP && !p.gather && TW * (int64_t)p.esize() >= 128;
    if ((c.flags & GEOT_FLAG_NT_LOADS) && !nt_ok)
        return fail(GEOT_ERROR_UNSUPPORTED, "non-temporal loads need the element-parallel rows mode and a "
                                            "tile of at least 128 bytes");
    r->nt_rows = (c.flags & GEOT_FLAG_NT_LOADS) ? 1
                 : (c.flags & GEOT_FLAG_CACHED_LOADS) ? 0
                 : (nt_ok && p.F * (int64_t)p.esize() >= 128 ? 1 : 0);
    r->tile_major = (c.flags & GEOT_FLAG_TILE_MAJOR) != 0 && r->family == GEOT_FAMILY_EP && ntiles > 1;
    r->K = rows == 0 ? auto_rows(p.nnz, L, V, NT, r->ntiles, (int64_t)p.esize()) : rows;
    const int GW = 64 / L;
    geot_kernel_choice_t cc = c;
    if (from_selector && cc.groups > GW) cc.groups = GW;  // tree leaves are shape-independent
    if (cc.groups < 0 || (cc.groups != 0 && (!is_pow2(cc.groups) || cc.groups > GW)))
        return fail(GEOT_ERROR_UNSUPPORTED, "groups must be a power of two <= 64/lanes");
    if (cc.groups != 0) {
        r->groups = cc.groups;
    } else {
        const double mean = p.S > 0 ? (double)p.nnz / (double)p.S : 0.0;
        int gsz = 1;
        while (gsz < GW && mean >= 16.0 * gsz) gsz <<= 1;
        r->groups = gsz;
    }
    return GEOT_SUCCESS;
}

geot_kernel_choice_t to_choice(const Resolved &r) {
    geot_kernel_choice_t c;
    c.family = r.family;
    c.vec = r.V;
    c.lanes = r.L;
    c.rows = r.K;
    c.groups = r.groups;
    c.flags = (r.nt_rows ? GEOT_FLAG_NT_LOADS : 0) | (r.tile_major ? GEOT_FLAG_TILE_MAJOR : 0);
    return c;
}

// A leaf's column tiles in sequence, undone: the lanes come from the shape again.
void untile(geot_kernel_choice_t *c) {
    if (c->flags & GEOT_FLAG_TILE_MAJOR) {
        c->flags &= ~GEOT_FLAG_TILE_MAJOR;
        c->lanes = 0;
    }
}

void select_raw(int64_t nnz, int64_t S, int64_t F, geot_op_t op, int gather,
                const geot_index_stats_t *stats, geot_kernel_choice_t *c) {
    double cv = 0.0, max_rel = 0.0;
    const double mean = S > 0 ? (double)nnz / (double)S : 0.0;
    if (stats && mean > 0) {
        cv = stats->var_len > 0 ? std::sqrt(stats->var_len) / mean : 0.0;
        max_rel = (double)stats->max_len / mean;
    }
    int32_t o[6];
    tree_select((double)nnz, (double)S, (double)F, (int)op, gather, stats != nullptr, cv, max_rel, o);
    // One segment-parallel team owns a whole segment: never used where the longest segment
    // exceeds 256x the mean (the range the trees were fitted on leaves it unmeasured there)
    if (o[0] == GEOT_FAMILY_SP && max_rel > 256.0)
        tree_select((double)nnz, (double)S, (double)F, (int)op, gather, 0, cv, max_rel, o);
    c->family = o[0];
    c->vec = o[1];
    c->lanes = o[2];
    c->rows = o[3];
    c->groups = o[4];
    c->flags = 0;
    if (o[0] == GEOT_FAMILY_EP && o[5] > 1 && F % 4 == 0) {
        // o[5] column tiles run one after another: the lanes of the 4-wide shape of F, divided
        // (leaves are fit on fp32 shapes; 16-bit storage halves them again in resolve)
        const int64_t vecs = F / 4;
        int L = 1;
        while (L < vecs && L < 64) L <<= 1;
        c->lanes = std::max(1, L / o[5]);
        c->flags = GEOT_FLAG_TILE_MAJOR;
    }
}

// ---------------------------------------------------------------------------
// argument checks (host only, before any device work)
// ---------------------------------------------------------------------------
bool overlaps(const void *a, size_t na, const void *b, size_t nb) {
    if (!a || !b || na == 0 || nb == 0) return false;
    const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
    return a0 < b0 + nb && b0 < a0 + na;
}

geot_status_t check_args(const Problem &p) {
    if (p.op != GEOT_OP_SUM && p.op != GEOT_OP_MEAN && p.op != GEOT_OP_MAX)
        return fail(GEOT_ERROR_INVALID_VALUE, "unknown op %d", (int)p.op);
    if (p.elem != ELEM_F32 && p.elem != ELEM_BF16 && p.elem != ELEM_F16)
        return fail(GEOT_ERROR_INVALID_VALUE, "unknown data type %d", p.elem);
    if (p.idx32 != 0 && p.idx32 != 1)
        return fail(GEOT_ERROR_INVALID_VALUE, "unknown index type %d", p.idx32);
    if (p.nnz < 0 || p.S < 0 || p.F < 0 || (p.gather && p.num_x_rows < 0))
        return fail(GEOT_ERROR_INVALID_VALUE, "negative size");
    if (p.S == 0 || p.F == 0) return GEOT_SUCCESS;
    if (p.S > (int64_t)INT32_MAX) return fail(GEOT_ERROR_INVALID_VALUE, "num_segments must be < 2^31");
    const int64_t kMax = (int64_t)1 << 62;
    if (p.F > ((int64_t)1 << 31) || p.S > kMax / p.F || p.nnz > kMax / p.F ||
        (p.gather && p.num_x_rows > kMax / p.F))
        return fail(GEOT_ERROR_INVALID_VALUE, "size overflow");
    if (!p.out) return fail(GEOT_ERROR_INVALID_VALUE, "out is NULL");
    const size_t out_bytes = (size_t)(p.S * p.F) * 4;
    if (p.nnz > 0) {
        if (!p.idx) return fail(GEOT_ERROR_INVALID_VALUE, "index is NULL");
        if (!p.src) return fail(GEOT_ERROR_INVALID_VALUE, p.gather ? "X is NULL" : "src is NULL");
        if (p.gather) {
            if (!p.col) return fail(GEOT_ERROR_INVALID_VALUE, "col is NULL");
            if (p.num_x_rows == 0) return fail(GEOT_ERROR_INVALID_VALUE, "X has no rows but nnz > 0");
        }
        const size_t src_rows = (size_t)(p.gather ? p.num_x_rows : p.nnz);
        if (overlaps(p.out, out_bytes, p.src, src_rows * (size_t)p.F * p.esize()) ||
            overlaps(p.out, out_bytes, p.idx, (size_t)p.nnz * p.isize()) ||
            overlaps(p.out, out_bytes, p.col, p.gather ? (size_t)p.nnz * p.isize() : 0) ||
            overlaps(p.out, out_bytes, p.w, p.gather ? (size_t)p.nnz * 4 : 0))
            return fail(GEOT_ERROR_INVALID_VALUE, "out overlaps an input");
    }
    if (p.arg) {   // the recipients of a max, 32-bit row (edge) numbers beside out
        if (p.op != GEOT_OP_MAX) return fail(GEOT_ERROR_INVALID_VALUE, "recipients are those of a max");
        if (p.nnz >= (int64_t)kNoRecipient)
            return fail(GEOT_ERROR_UNSUPPORTED, "recipients are 32-bit row numbers: fewer than 2^32 - 1 rows");
        const size_t src_rows = (size_t)(p.gather ? p.num_x_rows : p.nnz);
        if (overlaps(p.arg, out_bytes, p.out, out_bytes) ||
            overlaps(p.arg, out_bytes, p.src, p.nnz > 0 ? src_rows * (size_t)p.F * p.esize() : 0) ||
            overlaps(p.arg, out_bytes, p.idx, (size_t)p.nnz * p.isize()) ||
            overlaps(p.arg, out_bytes, p.col, p.gather ? (size_t)p.nnz * p.isize() : 0) ||
            overlaps(p.arg, out_bytes, p.w, p.gather ? (size_t)p.nnz * 4 : 0))
            return fail(GEOT_ERROR_INVALID_VALUE, "arg overlaps out or an input");
    }
    return GEOT_SUCCESS;
}

// ---------------------------------------------------------------------------
// launch sequences
// ---------------------------------------------------------------------------
struct Level {
    int64_t n, K, nchunks;
};

// Partial levels are small and latency-bound: short serial runs (at most 8
// partials per row group) and one more level rather than one long block.
int64_t piece_rows_k(int64_t n, int64_t G) {
    return std::max<int64_t>(1, std::min<int64_t>(8, ceil_div(n, G)));
}

// blocks that write the gap list, as a pass of their own or riding on the final partial level
constexpr int kFoldedGapBlocks = 1024;
// segment sum and max gradients from this many bytes of grad_src take the offsets pass first
// (below, the kernels read the ids, which saves two launches)
constexpr size_t kBcastOffsetsMinBytes = (size_t)64 << 20;

geot_status_t run_ep_levels(const Problem &p, const Resolved &r, const std::vector<Level> &lv,
                            char *base, const std::vector<size_t> &off_v,
                            const std::vector<size_t> &off_s, const std::vector<size_t> &off_c,
                            const std::vector<size_t> &off_x, int64_t ld_p, GapList gaps, hipStream_t st);

// Shape of the passes over fp32 partials: 8-element vectors (16-bit storage)
// become 4-element vectors over twice the lanes, so the column tiles match.
void piece_shape(const Resolved &r, int *V, int *L) {
    *V = r.V == 8 ? 4 : r.V;
    *L = r.V == 8 ? 2 * r.L : r.L;
}

// The passes of an element-parallel call: level 0 over the input, then levels over the
// partials of block-crossing segments until one block remains, and where each level's
// partials live in the temporary memory.
struct EpPlan {
    std::vector<Level> lv;
    std::vector<size_t> off_v, off_s, off_c, off_x;  // per level: values, segment ids, counts, recipients
    size_t bytes = 0;
    int64_t ld_p = 0;
};

geot_status_t plan_ep(const Problem &p, const Resolved &r, EpPlan *pl) {
    const int64_t G = kBlock / r.L;
    int Vp, Lp;
    piece_shape(r, &Vp, &Lp);
    const int64_t Gp = kBlock / Lp;
    pl->ld_p = ceil_div(p.F, 4) * 4;
    std::vector<Level> &lv = pl->lv;
    lv.clear();
    lv.push_back({p.nnz, r.K, ceil_div(p.nnz, G * r.K)});
    while (lv.back().nchunks > 1) {
        const int64_t n = 2 * lv.back().nchunks;
        const int64_t K = piece_rows_k(n, Gp);
        lv.push_back({n, K, ceil_div(n, Gp * K)});
        if (lv.size() > 64) return fail(GEOT_ERROR_HIP, "internal: level count");
    }
    pl->off_v.assign(lv.size(), 0);
    pl->off_s.assign(lv.size(), 0);
    pl->off_c.assign(lv.size(), 0);
    pl->off_x.assign(lv.size(), 0);
    size_t bytes = 0;
    for (size_t l = 1; l < lv.size(); ++l) {
        pl->off_v[l] = bytes;
        bytes = align256(bytes + (size_t)lv[l].n * (size_t)pl->ld_p * 4);
        pl->off_s[l] = bytes;
        bytes = align256(bytes + (size_t)lv[l].n * 8);
        pl->off_c[l] = bytes;
        bytes = align256(bytes + (size_t)lv[l].n * 8);
        if (p.arg) {
            pl->off_x[l] = bytes;
            bytes = align256(bytes + (size_t)lv[l].n * (size_t)pl->ld_p * 4);
        }
    }
    pl->bytes = bytes;
    return GEOT_SUCCESS;
}

geot_status_t run_ep(const Problem &p, const Resolved &r, hipStream_t st, const Workspace *ws = nullptr) {
    EpPlan pl;
    geot_status_t s = plan_ep(p, r, &pl);
    if (s != GEOT_SUCCESS) return s;
    void *scratch = nullptr;
    GapList gaps;
    StreamCtx *ctx = nullptr;
    s = call_scratch(pl.bytes, st, ws, &scratch, &gaps, &ctx);
    if (s != GEOT_SUCCESS) return s;
    return poison(ctx, run_ep_levels(p, r, pl.lv, (char *)scratch, pl.off_v, pl.off_s, pl.off_c, pl.off_x, pl.ld_p,
                                     gaps, st));
}

geot_status_t run_ep_levels(const Problem &p, const Resolved &r, const std::vector<Level> &lv,
                            char *base, const std::vector<size_t> &off_v,
                            const std::vector<size_t> &off_s, const std::vector<size_t> &off_c,
                            const std::vector<size_t> &off_x, int64_t ld_p, GapList gaps, hipStream_t st) {
    const int red = p.op == GEOT_OP_MAX ? (p.arg ? RED_MAXARG : RED_MAX) : RED_SUM;
    for (size_t l = 0; l < lv.size(); ++l) {
        EpArgs a;
        memset(&a, 0, sizeof(a));
        if (l == 0) {
            a.src = p.src;
            a.ld_src = p.F;
            a.idx = p.idx;
            a.col = p.col;
            a.w = p.w;
            a.num_x_rows = p.num_x_rows;
            a.fill_gaps = 1;
            a.gaps = gaps;
            a.elem = p.elem;
            a.idx32 = p.idx32;
            a.nt_rows = r.nt_rows;
            a.meta_stride = p.meta_stride;
            a.tile_major = r.tile_major;
        } else {
            a.src = (const float *)(base + off_v[l]);
            a.ld_src = ld_p;
            a.idx = (const int64_t *)(base + off_s[l]);
            a.cnt = (const int64_t *)(base + off_c[l]);
            if (p.arg) a.six = (const uint32_t *)(base + off_x[l]);
            a.fill_gaps = 0;
        }
        a.arg_out = p.arg;
        a.n = lv[l].n;
        a.S = p.S;
        a.F = p.F;
        a.out = p.out;
        a.ld_out = p.F;
        if (l + 1 < lv.size()) {
            a.pv = (float *)(base + off_v[l + 1]);
            a.pseg = (int64_t *)(base + off_s[l + 1]);
            a.pcnt = (int64_t *)(base + off_c[l + 1]);
            if (p.arg) a.pix = (uint32_t *)(base + off_x[l + 1]);
            a.ld_p = ld_p;
        }
        if (l + 1 == lv.size() && l > 0) {  // the final level also fills the gap list of level 0
            a.gaps = gaps;
            a.gap_blocks = kFoldedGapBlocks;
        }
        a.K = (int32_t)lv[l].K;
        a.ntiles = r.ntiles;
        a.mean = p.op == GEOT_OP_MEAN ? 1 : 0;
        const int mode = l == 0 ? (p.gather ? SRC_GATHER : SRC_ROWS) : SRC_PIECES;
        hipEvent_t e0 = nullptr, e1 = nullptr;
        const bool prof = l == 0 && prof_take(&e0, &e1);
        if (prof) GEOT_HIP(hipEventRecord(e0, st), "hipEventRecord");
        int V = r.V, L = r.L;
        if (l > 0) piece_shape(r, &V, &L);
        GEOT_HIP(launch_ep(a, red, mode, V, r.NT, L, lv[l].nchunks, st), "launch element-parallel kernel");
        if (prof) GEOT_HIP(hipEventRecord(e1, st), "hipEventRecord");
        if (l == 0 && lv.size() == 1)  // one level: a pass of its own (else the final level's extra blocks)
            GEOT_HIP(launch_gap_fill_rows(p.out, p.F, p.F, std::min(r.V, 4), (int64_t)r.L * r.V * r.NT, p.S,
                                          gaps, p.arg, st),
                     "launch gap fill kernel");
    }
    return GEOT_SUCCESS;
}

geot_status_t run_sp_kernels(const Problem &p, const Resolved &r, int64_t *off, GapList gaps,
                             hipStream_t st);

geot_status_t run_sp(const Problem &p, const Resolved &r, hipStream_t st, const Workspace *ws = nullptr) {
    void *scratch = nullptr;
    GapList gaps;
    StreamCtx *ctx = nullptr;
    geot_status_t s = call_scratch((size_t)(p.S + 1) * 8, st, ws, &scratch, &gaps, &ctx);
    if (s != GEOT_SUCCESS) return s;
    return poison(ctx, run_sp_kernels(p, r, (int64_t *)scratch, gaps, st));
}

geot_status_t run_sp_kernels(const Problem &p, const Resolved &r, int64_t *off, GapList gaps,
                             hipStream_t st) {
    if (p.typed()) return fail(GEOT_ERROR_UNSUPPORTED, "internal: typed problem in the segment-parallel path");
    GEOT_HIP(launch_offsets(static_cast<const int64_t *>(p.idx), p.nnz, p.S, off, gaps, st), "launch offsets kernel");
    GEOT_HIP(launch_gap_fill_i64(off, p.S + 1, gaps, st), "launch gap fill kernel");
    SpArgs a;
    memset(&a, 0, sizeof(a));
    a.src = static_cast<const float *>(p.src);
    a.ld_src = p.F;
    a.off = off;
    a.col = static_cast<const int64_t *>(p.col);
    a.w = p.w;
    a.num_x_rows = p.num_x_rows;
    a.S = p.S;
    a.F = p.F;
    a.out = p.out;
    a.ld_out = p.F;
    a.groups = r.groups;
    a.ntiles = r.ntiles;
    a.mean = p.op == GEOT_OP_MEAN ? 1 : 0;
    const int red = p.op == GEOT_OP_MAX ? RED_MAX : RED_SUM;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    const bool prof = prof_take(&e0, &e1);
    if (prof) GEOT_HIP(hipEventRecord(e0, st), "hipEventRecord");
    GEOT_HIP(launch_sp(a, red, p.gather ? SRC_GATHER : SRC_ROWS, r.V, r.NT, r.L, st),
             "launch segment-parallel kernel");
    if (prof) GEOT_HIP(hipEventRecord(e1, st), "hipEventRecord");
    return GEOT_SUCCESS;
}

// The kernel choice of a call: the forced one, else the selector's for the problem.
geot_kernel_choice_t choose(const Problem &p, const geot_kernel_choice_t *forced) {
    if (forced) return *forced;
    geot_kernel_choice_t c;
    select_raw(p.nnz, p.S, p.F, p.op, p.gather ? (p.w ? 1 : 2) : 0, nullptr, &c);
    if ((p.typed() || p.arg) && c.family == GEOT_FAMILY_SP) c = geot_kernel_choice_t{GEOT_FAMILY_EP, 0, 0, 0, 0, 0};
    // The leaves are fit on fp32 timings. A 16-bit X is half the bytes, and there the
    // ids read once per tile cost more than the smaller slab saves (SpMM shape, bf16:
    // 2.92 ms with two tiles in sequence, 2.83 ms without).
    if (p.esize() == 2) untile(&c);
    return c;
}

// Temporary bytes (gap list included) that a resolved call takes.
geot_status_t scratch_need(const Problem &p, const Resolved &r, size_t *need) {
    if (r.family == GEOT_FAMILY_SP) {
        *need = kGapArea + align256((size_t)(p.S + 1) * 8);
        return GEOT_SUCCESS;
    }
    EpPlan pl;
    geot_status_t s = plan_ep(p, r, &pl);
    if (s == GEOT_SUCCESS) *need = kGapArea + align256(pl.bytes);
    return s;
}

geot_status_t reduce(const Problem &p, hipStream_t st, const geot_kernel_choice_t *forced,
                     const Workspace *ws = nullptr) {
    t_detail.clear();
    geot_status_t s = check_args(p);
    if (s != GEOT_SUCCESS) return s;
    if (p.S == 0 || p.F == 0) return GEOT_SUCCESS;
    if (p.nnz == 0) {
        GEOT_HIP(launch_fill(p.out, p.S, p.F, p.F, GEOT_EMPTY_FILL, st), "launch fill kernel");
        if (p.arg) {   // no recipients: all ones
            float none;
            const uint32_t bits = kNoRecipient;
            memcpy(&none, &bits, 4);
            GEOT_HIP(launch_fill(reinterpret_cast<float *>(p.arg), p.S, p.F, p.F, none, st), "launch fill kernel");
        }
        t_last_choice = geot_kernel_choice_t{0, 0, 0, 0, 0, 0};
        return GEOT_SUCCESS;
    }
    const geot_kernel_choice_t c = choose(p, forced);
    Resolved r;
    s = resolve(p, c, &r, forced == nullptr);
    if (s != GEOT_SUCCESS) return s;
    s = r.family == GEOT_FAMILY_SP ? run_sp(p, r, st, ws) : run_ep(p, r, st, ws);
    if (s == GEOT_SUCCESS) t_last_choice = to_choice(r);
    return s;
}

// Workspace a call of this shape needs, whatever the alignment of its arrays: the largest
// need over the vector widths that F and the pointers may allow (the pointers decide the
// width, and the width the partials' count).
geot_status_t workspace_size(Problem p, const geot_kernel_choice_t *forced, size_t *bytes) {
    t_detail.clear();
    if (!bytes) return fail(GEOT_ERROR_INVALID_VALUE, "bytes is NULL");
    *bytes = 0;
    if (p.op != GEOT_OP_SUM && p.op != GEOT_OP_MEAN && p.op != GEOT_OP_MAX)
        return fail(GEOT_ERROR_INVALID_VALUE, "unknown op %d", (int)p.op);
    if (p.nnz < 0 || p.S < 0 || p.F < 0) return fail(GEOT_ERROR_INVALID_VALUE, "negative size");
    if (p.S > (int64_t)INT32_MAX) return fail(GEOT_ERROR_INVALID_VALUE, "num_segments must be < 2^31");
    const int64_t kMax = (int64_t)1 << 62;
    if (p.F > ((int64_t)1 << 31) || (p.F > 0 && (p.S > kMax / p.F || p.nnz > kMax / p.F)))
        return fail(GEOT_ERROR_INVALID_VALUE, "size overflow");
    if (p.nnz == 0 || p.S == 0 || p.F == 0) return GEOT_SUCCESS;  // no temporary memory
    size_t most = 0;
    for (uintptr_t align : {(uintptr_t)256, (uintptr_t)8, (uintptr_t)4}) {
        p.src = (const void *)align;
        p.out = (float *)align;
        Resolved r;
        geot_status_t s = resolve(p, choose(p, forced), &r, forced == nullptr);
        if (s != GEOT_SUCCESS) return s;
        size_t need = 0;
        s = scratch_need(p, r, &need);
        if (s != GEOT_SUCCESS) return s;
        most = std::max(most, need);
    }
    *bytes = most;
    return GEOT_SUCCESS;
}

// A caller's workspace: NULL only with 0 bytes (enough for calls that need none), else
// 256-byte aligned (hipMalloc's alignment; the gap list's records are 8-byte words).
geot_status_t check_workspace(const void *workspace, size_t bytes) {
    if (!workspace && bytes > 0) return fail(GEOT_ERROR_INVALID_VALUE, "workspace is NULL with %zu bytes", bytes);
    if (((uintptr_t)workspace & 255) != 0) return fail(GEOT_ERROR_INVALID_VALUE, "workspace must be 256-byte aligned");
    return GEOT_SUCCESS;
}

// ---------------------------------------------------------------------------
// temporary memory for callers that cannot allocate (geot_segment_reduce_noalloc)
// ---------------------------------------------------------------------------
std::mutex g_noalloc_mu;
std::map<int, char *> g_noalloc_ptr;  // device -> address of that device's `scratch`

// The current device's copy of `scratch`, looked up once per device (with it current).
geot_status_t noalloc_scratch(char **ptr) {
    int dev = 0;
    GEOT_HIP(hipGetDevice(&dev), "hipGetDevice");
    std::lock_guard<std::mutex> lk(g_noalloc_mu);
    auto it = g_noalloc_ptr.find(dev);
    if (it != g_noalloc_ptr.end()) {
        *ptr = it->second;
        return GEOT_SUCCESS;
    }
    void *q = nullptr;
    GEOT_HIP(hipGetSymbolAddress(&q, HIP_SYMBOL(::scratch)), "hipGetSymbolAddress(scratch)");
    if (!q || ((uintptr_t)q & 255) != 0) return fail(GEOT_ERROR_HIP, "scratch array has no aligned device address");
    g_noalloc_ptr[dev] = (char *)q;
    *ptr = (char *)q;
    return GEOT_SUCCESS;
}

}  // namespace
}  // namespace geot

using namespace geot;

extern "C" {

geot_status_t geot_segment_reduce_noalloc(const float *src, const int64_t *sorted_index, int64_t nnz,
                                          int64_t num_segments, int64_t F, geot_op_t op, float *out,
                                          void *stream) {
    t_detail.clear();
    char *ptr = nullptr;
    geot_status_t s = noalloc_scratch(&ptr);
    if (s != GEOT_SUCCESS) return s;
    Problem p{false, src, 0, nullptr, nullptr, sorted_index, nnz, num_segments, F, op, out};
    Workspace ws{ptr, kNoAllocBytes};
    t_no_events = true;
    s = reduce(p, (hipStream_t)stream, nullptr, &ws);
    t_no_events = false;
    return s;
}

size_t geot_noalloc_scratch_bytes(void) { return kNoAllocBytes; }

geot_status_t geot_segment_reduce_with(const float *src, const int64_t *sorted_index, int64_t nnz,
                                       int64_t num_segments, int64_t F, geot_op_t op, float *out,
                                       void *stream, const geot_kernel_choice_t *choice) {
    Problem p{false, src, 0, nullptr, nullptr, sorted_index, nnz, num_segments, F, op, out};
    return reduce(p, (hipStream_t)stream, choice);
}

geot_status_t geot_segment_reduce(const float *src, const int64_t *sorted_index, int64_t nnz,
                                  int64_t num_segments, int64_t F, geot_op_t op, float *out,
                                  void *stream) {
    return geot_segment_reduce_with(src, sorted_index, nnz, num_segments, F, op, out, stream, nullptr);
}

geot_status_t geot_segment_reduce_workspace_size(int64_t nnz, int64_t num_segments, int64_t F, geot_op_t op,
                                                 const geot_kernel_choice_t *choice, size_t *bytes) {
    Problem p{false, nullptr, 0, nullptr, nullptr, nullptr, nnz, num_segments, F, op, nullptr};
    return workspace_size(p, choice, bytes);
}

geot_status_t geot_segment_reduce_ws(const float *src, const int64_t *sorted_index, int64_t nnz,
                                     int64_t num_segments, int64_t F, geot_op_t op, float *out,
                                     void *workspace, size_t workspace_bytes, void *stream,
                                     const geot_kernel_choice_t *choice) {
    t_detail.clear();
    geot_status_t s = check_workspace(workspace, workspace_bytes);
    if (s != GEOT_SUCCESS) return s;
    Problem p{false, src, 0, nullptr, nullptr, sorted_index, nnz, num_segments, F, op, out};
    const size_t out_bytes = (size_t)std::max<int64_t>(num_segments, 0) * (size_t)std::max<int64_t>(F, 0) * 4;
    if (overlaps(workspace, workspace_bytes, out, out_bytes) ||
        overlaps(workspace, workspace_bytes, src, (size_t)std::max<int64_t>(nnz, 0) * (size_t)std::max<int64_t>(F, 0) * 4) ||
        overlaps(workspace, workspace_bytes, sorted_index, (size_t)std::max<int64_t>(nnz, 0) * 8))
        return fail(GEOT_ERROR_INVALID_VALUE, "workspace overlaps an argument");
    Workspace ws{(char *)workspace, workspace_bytes};
    return reduce(p, (hipStream_t)stream, choice, &ws);
}

geot_status_t geot_gather_scatter_workspace_size(int64_t nnz, int64_t num_rows, int64_t F, geot_op_t op,
                                                 int32_t weighted, const geot_kernel_choice_t *choice,
                                                 size_t *bytes) {
    // only the presence of weights matters to the selector: any non-null stand-in
    Problem p{true, nullptr, 1, nullptr, weighted ? (const float *)(uintptr_t)256 : nullptr, nullptr,
              nnz, num_rows, F, op, nullptr};
    return workspace_size(p, choice, bytes);
}

geot_status_t geot_gather_scatter_ws(const float *X, int64_t num_x_rows, const int64_t *col,
                                     const float *weight, const int64_t *sorted_row, int64_t nnz,
                                     int64_t num_rows, int64_t F, geot_op_t op, float *out,
                                     void *workspace, size_t workspace_bytes, void *stream,
                                     const geot_kernel_choice_t *choice) {
    t_detail.clear();
    geot_status_t s = check_workspace(workspace, workspace_bytes);
    if (s != GEOT_SUCCESS) return s;
    Problem p{true, X, num_x_rows, col, weight, sorted_row, nnz, num_rows, F, op, out};
    const size_t n = (size_t)std::max<int64_t>(nnz, 0);
    const size_t out_bytes = (size_t)std::max<int64_t>(num_rows, 0) * (size_t)std::max<int64_t>(F, 0) * 4;
    if (overlaps(workspace, workspace_bytes, out, out_bytes) ||
        overlaps(workspace, workspace_bytes, X,
                 (size_t)std::max<int64_t>(num_x_rows, 0) * (size_t)std::max<int64_t>(F, 0) * 4) ||
        overlaps(workspace, workspace_bytes, col, n * 8) || overlaps(workspace, workspace_bytes, sorted_row, n * 8) ||
        overlaps(workspace, workspace_bytes, weight, weight ? n * 4 : 0))
        return fail(GEOT_ERROR_INVALID_VALUE, "workspace overlaps an argument");
    Workspace ws{(char *)workspace, workspace_bytes};
    return reduce(p, (hipStream_t)stream, choice, &ws);
}

geot_status_t geot_gather_scatter_with(const float *X, int64_t num_x_rows, const int64_t *col,
                                       const float *weight, const int64_t *sorted_row, int64_t nnz,
                                       int64_t num_rows, int64_t F, geot_op_t op, float *out,
                                       void *stream, const geot_kernel_choice_t *choice) {
    Problem p{true, X, num_x_rows, col, weight, sorted_row, nnz, num_rows, F, op, out};
    return reduce(p, (hipStream_t)stream, choice);
}

geot_status_t geot_gather_scatter(const float *X, int64_t num_x_rows, const int64_t *col,
                                  const float *weight, const int64_t *sorted_row, int64_t nnz,
                                  int64_t num_rows, int64_t F, geot_op_t op, float *out,
                                  void *stream) {
    return geot_gather_scatter_with(X, num_x_rows, col, weight, sorted_row, nnz, num_rows, F, op,
                                    out, stream, nullptr);
}

// The segment gradient; for max, `given` (may be NULL) holds the recipients a forward
// geot_segment_reduce_max_arg recorded, and then src and out are not read.
static geot_status_t seg_backward(const float *grad_out, const void *sorted_index, geot_index_type_t index_type,
                                  int64_t nnz, int64_t num_segments, int64_t F, geot_op_t op, const void *src,
                                  geot_dtype_t src_type, const float *out, const uint32_t *given, void *grad_src,
                                  void *stream) {
    t_detail.clear();
    if (op != GEOT_OP_SUM && op != GEOT_OP_MEAN && op != GEOT_OP_MAX)
        return fail(GEOT_ERROR_INVALID_VALUE, "unknown op %d", (int)op);
    if (src_type != GEOT_DTYPE_F32 && src_type != GEOT_DTYPE_BF16 && src_type != GEOT_DTYPE_F16)
        return fail(GEOT_ERROR_INVALID_VALUE, "unknown storage type %d", (int)src_type);
    if (index_type != GEOT_INDEX_I64 && index_type != GEOT_INDEX_I32)
        return fail(GEOT_ERROR_INVALID_VALUE, "unknown index type %d", (int)index_type);
    if (nnz < 0 || num_segments < 0 || F < 0) return fail(GEOT_ERROR_INVALID_VALUE, "negative size");
    if (nnz == 0 || F == 0) return GEOT_SUCCESS;
    if (num_segments == 0) return fail(GEOT_ERROR_INVALID_VALUE, "num_segments is 0 but nnz > 0");
    if (num_segments > (int64_t)INT32_MAX) return fail(GEOT_ERROR_INVALID_VALUE, "num_segments must be < 2^31");
    const int64_t kMax = (int64_t)1 << 62;
    if (F > ((int64_t)1 << 31) || num_segments > kMax / F || nnz > kMax / F)
        return fail(GEOT_ERROR_INVALID_VALUE, "size overflow");
    if (!grad_out || !sorted_index || !grad_src) return fail(GEOT_ERROR_INVALID_VALUE, "NULL array");
    if (given && op != GEOT_OP_MAX) return fail(GEOT_ERROR_INVALID_VALUE, "recipients are those of a max");
    if (given && nnz >= (int64_t)kNoRecipient)
        return fail(GEOT_ERROR_UNSUPPORTED, "recipients are 32-bit row numbers: fewer than 2^32 - 1 rows");
    if (op == GEOT_OP_MAX && !given && (!src || !out)) return fail(GEOT_ERROR_INVALID_VALUE, "max needs src and out");
    const size_t es = src_type == GEOT_DTYPE_F32 ? 4 : 2, is = index_type == GEOT_INDEX_I32 ? 4 : 8;
    const size_t gb = (size_t)(nnz * F) * es;
    const bool reads = op == GEOT_OP_MAX && !given;   // src and out
    if (overlaps(grad_src, gb, grad_out, (size_t)(num_segments * F) * 4) ||
        overlaps(grad_src, gb, sorted_index, (size_t)nnz * is) ||
        overlaps(grad_src, gb, src, reads ? gb : 0) ||
        overlaps(grad_src, gb, out, reads ? (size_t)(num_segments * F) * 4 : 0) ||
        overlaps(grad_src, gb, given, given ? (size_t)(num_segments * F) * 4 : 0))
        return fail(GEOT_ERROR_INVALID_VALUE, "grad_src overlaps an input");
    // widest vector that F and every pointer allow (fp32 operands: 16-byte loads of 4; 16-bit
    // storage also 8 elements, loaded and stored as 16 bytes)
    const uintptr_t ptrs = (uintptr_t)grad_out | (uintptr_t)grad_src | (uintptr_t)given |
                           (reads ? ((uintptr_t)src | (uintptr_t)out) : 0);
    int V = 1;
    if (es == 2 && F % 8 == 0 && (ptrs & 15) == 0) V = 8;
    else if (F % 4 == 0 && (ptrs & 15) == 0) V = 4;
    else if (F % 2 == 0 && (ptrs & 7) == 0) V = 2;
    const int elem = (int)src_type, idx32 = index_type == GEOT_INDEX_I32 ? 1 : 0;
    hipStream_t st = (hipStream_t)stream;
    void *scratch = nullptr;
    StreamCtx *ctx = nullptr;
    const bool mean = op == GEOT_OP_MEAN, mx = op == GEOT_OP_MAX;
    // From kBcastOffsetsMinBytes, where the segments average at least a block's rows (so most
    // blocks lie in one segment), an offsets pass reads the ids once and keeps each block's first
    // and last ids; the kernels that write grad_src then take every row's segment from the
    // offsets, so that their only HBM stream is their stores. Otherwise the ids are read where
    // they are needed (two launches fewer; mean still takes the offsets pass for the lengths).
    // 2,000,000 rows in 100,000 segments, sum: 34 against 44 us at F = 16, 460 against 468 at
    // F = 256 with the ids read; the power-law graph (114,615,892 rows, 232,965 segments, F =
    // 32): 2.63 against 3.40 ms from the offsets.
    const int rows_log2 = seg_bwd_rows_log2(F, V);
    const bool use_first = gb >= kBcastOffsetsMinBytes && (nnz >> rows_log2) >= num_segments;
    const bool from_off = mean || use_first;
    const size_t o_arg = 0,
                 arg_b = mx && !given ? align256((size_t)(num_segments * F) * (seg_bwd_arg32(nnz) ? 4 : 8)) : 0;
    const size_t o_off = o_arg + arg_b, o_first = o_off + (from_off ? align256((size_t)(num_segments + 1) * 8) : 0);
    const int64_t blocks = seg_bwd_blocks(nnz, F, V);
    GapList gaps;
    if ((mx && !given) || from_off) {
        geot_status_t s = stream_scratch(o_first + (use_first ? (size_t)blocks * 16 : 0), st, &scratch,
                                         from_off ? &gaps : nullptr, &ctx);
        if (s != GEOT_SUCCESS) return s;
    }
    void *arg = mx ? (given ? (void *)given : scratch) : nullptr;
    int64_t *off = from_off ? (int64_t *)((char *)scratch + o_off) : nullptr;
    int64_t *first = use_first ? (int64_t *)((char *)scratch + o_first) : nullptr;
    if (!from_off) {
        if (mx)
            GEOT_HIP(launch_seg_bwd_max(grad_out, sorted_index, idx32, src, out, nullptr, nullptr, nnz, num_segments,
                                        F, V, elem, arg, given != nullptr, grad_src, st),
                     "launch max backward kernels");
        else
            GEOT_HIP(launch_seg_bwd_bcast(grad_out, sorted_index, idx32, nullptr, nullptr, nnz, num_segments, F, V,
                                          elem, false, grad_src, st),
                     "launch backward kernel");
        return GEOT_SUCCESS;
    }
    const int shift = rows_log2;
    return poison(ctx, [&]() -> geot_status_t {
        if (idx32)
            GEOT_HIP(launch_offsets_i32(static_cast<const int32_t *>(sorted_index), nnz, num_segments, off, gaps, st,
                                        first, shift),
                     "launch offsets kernel");
        else
            GEOT_HIP(launch_offsets(static_cast<const int64_t *>(sorted_index), nnz, num_segments, off, gaps, st,
                                    first, shift),
                     "launch offsets kernel");
        GEOT_HIP(launch_gap_fill_i64(off, num_segments + 1, gaps, st), "launch gap fill kernel");
        if (mx)
            GEOT_HIP(launch_seg_bwd_max(grad_out, sorted_index, idx32, src, out, off, first, nnz, num_segments, F, V,
                                        elem, arg, given != nullptr, grad_src, st),
                     "launch max backward kernels");
        else
            GEOT_HIP(launch_seg_bwd_bcast(grad_out, sorted_index, idx32, off, first, nnz, num_segments, F, V, elem,
                                          mean, grad_src, st),
                     "launch backward kernel");
        return GEOT_SUCCESS;
    }());
}

geot_status_t geot_segment_reduce_backward_typed(const float *grad_out, const void *sorted_index,
                                                 geot_index_type_t index_type, int64_t nnz, int64_t num_segments,
                                                 int64_t F, geot_op_t op, const void *src, geot_dtype_t src_type,
                                                 const float *out, void *grad_src, void *stream) {
    return seg_backward(grad_out, sorted_index, index_type, nnz, num_segments, F, op, src, src_type, out, nullptr,
                        grad_src, stream);
}

geot_status_t geot_segment_reduce_backward_max_arg(const float *grad_out, const void *sorted_index,
                                                   geot_index_type_t index_type, int64_t nnz, int64_t num_segments,
                                                   int64_t F, const uint32_t *arg, void *grad_src,
                                                   geot_dtype_t src_type, void *stream) {
    if (!arg) {
        t_detail.clear();
        return fail(GEOT_ERROR_INVALID_VALUE, "arg is NULL");
    }
    return seg_backward(grad_out, sorted_index, index_type, nnz, num_segments, F, GEOT_OP_MAX, nullptr, src_type,
                        nullptr, arg, grad_src, stream);
}

geot_status_t geot_segment_reduce_backward(const float *grad_out, const int64_t *sorted_index,
                                           int64_t nnz, int64_t num_segments, int64_t F, geot_op_t op,
                                           const float *src, const float *out, float *grad_src,
                                           void *stream) {
    return geot_segment_reduce_backward_typed(grad_out, sorted_index, GEOT_INDEX_I64, nnz, num_segments, F, op,
                                              src, GEOT_DTYPE_F32, out, grad_src, stream);
}

geot_status_t geot_segment_reduce_typed(const void *src, geot_dtype_t src_type, const void *sorted_index,
                                        geot_index_type_t index_type, int64_t nnz, int64_t num_segments,
                                        int64_t F, geot_op_t op, float *out, void *stream,
                                        const geot_kernel_choice_t *choice) {
    Problem p{false, src, 0, nullptr, nullptr, sorted_index, nnz, num_segments, F, op, out};
    p.elem = (int)src_type;
    p.idx32 = (int)index_type;
    return reduce(p, (hipStream_t)stream, choice);
}

geot_status_t geot_gather_scatter_typed(const void *X, geot_dtype_t x_type, int64_t num_x_rows, const void *col,
                                        const float *weight, const void *sorted_row,
                                        geot_index_type_t index_type, int64_t nnz, int64_t num_rows, int64_t F,
                                        geot_op_t op, float *out, void *stream,
                                        const geot_kernel_choice_t *choice) {
    Problem p{true, X, num_x_rows, col, weight, sorted_row, nnz, num_rows, F, op, out};
    p.elem = (int)x_type;
    p.idx32 = (int)index_type;
    return reduce(p, (hipStream_t)stream, choice);
}

geot_status_t geot_segment_reduce_max_arg(const void *src, geot_dtype_t src_type, const void *sorted_index,
                                          geot_index_type_t index_type, int64_t nnz, int64_t num_segments,
                                          int64_t F, float *out, uint32_t *arg, void *stream,
                                          const geot_kernel_choice_t *choice) {
    t_detail.clear();
    if (!arg) return fail(GEOT_ERROR_INVALID_VALUE, "arg is NULL");
    Problem p{false, src, 0, nullptr, nullptr, sorted_index, nnz, num_segments, F, GEOT_OP_MAX, out};
    p.elem = (int)src_type;
    p.idx32 = (int)index_type;
    p.arg = arg;
    return reduce(p, (hipStream_t)stream, choice);
}

geot_status_t geot_gather_scatter_max_arg(const void *X, geot_dtype_t x_type, int64_t num_x_rows, const void *col,
                                          const float *weight, const void *sorted_row,
                                          geot_index_type_t index_type, int64_t nnz, int64_t num_rows, int64_t F,
                                          float *out, uint32_t *arg, void *stream,
                                          const geot_kernel_choice_t *choice) {
    t_detail.clear();
    if (!arg) return fail(GEOT_ERROR_INVALID_VALUE, "arg is NULL");
    Problem p{true, X, num_x_rows, col, weight, sorted_row, nnz, num_rows, F, GEOT_OP_MAX, out};
    p.elem = (int)x_type;
    p.idx32 = (int)index_type;
    p.arg = arg;
    return reduce(p, (hipStream_t)stream, choice);
}

// The fused-form gradients; for max, `given` (may be NULL) holds the recipients a forward
// geot_gather_scatter_max_arg recorded, and then out is not read and no recipient pass runs.
static geot_status_t gs_backward(const void *X, geot_dtype_t x_type, int64_t num_x_rows, const void *col,
                                 const float *weight, const void *sorted_row, geot_index_type_t index_type,
                                 int64_t nnz, int64_t num_rows, int64_t F, geot_op_t op, const float *grad_out,
                                 const float *out, const uint32_t *given, float *grad_X, float *grad_weight,
                                 void *stream) {
    t_detail.clear();
    if (op != GEOT_OP_SUM && op != GEOT_OP_MEAN && op != GEOT_OP_MAX)
        return fail(GEOT_ERROR_INVALID_VALUE, "unknown op %d", (int)op);
    if (x_type != GEOT_DTYPE_F32 && x_type != GEOT_DTYPE_BF16 && x_type != GEOT_DTYPE_F16)
        return fail(GEOT_ERROR_INVALID_VALUE, "unknown storage type %d", (int)x_type);
    if (index_type != GEOT_INDEX_I64 && index_type != GEOT_INDEX_I32)
        return fail(GEOT_ERROR_INVALID_VALUE, "unknown index type %d", (int)index_type);
    const int elem = (int)x_type, idx32 = index_type == GEOT_INDEX_I32 ? 1 : 0;
    const size_t es = x_type == GEOT_DTYPE_F32 ? 4 : 2, is = idx32 ? 4 : 8;
    if (nnz < 0 || num_rows < 0 || F < 0 || num_x_rows < 0)
        return fail(GEOT_ERROR_INVALID_VALUE, "negative size");
    if (grad_weight && !weight) return fail(GEOT_ERROR_INVALID_VALUE, "grad_weight needs weight");
    if (num_rows > (int64_t)INT32_MAX) return fail(GEOT_ERROR_INVALID_VALUE, "num_rows must be < 2^31");
    const int64_t kMax = (int64_t)1 << 62;
    if (F > ((int64_t)1 << 31) || num_rows > kMax / F || nnz > kMax / F || num_x_rows > kMax / (F ? F : 1))
        return fail(GEOT_ERROR_INVALID_VALUE, "size overflow");
    hipStream_t st = (hipStream_t)stream;
    if (F == 0) return GEOT_SUCCESS;
    if (nnz == 0) {  // no edge: every gradient is zero
        if (grad_X) GEOT_HIP(launch_fill(grad_X, num_x_rows, F, F, 0.0f, st), "launch fill kernel");
        return GEOT_SUCCESS;
    }
    if (num_rows == 0 || num_x_rows == 0) return fail(GEOT_ERROR_INVALID_VALUE, "empty row or X range with nnz > 0");
    if (!col || !sorted_row || !grad_out) return fail(GEOT_ERROR_INVALID_VALUE, "NULL array");
    if (given && op != GEOT_OP_MAX) return fail(GEOT_ERROR_INVALID_VALUE, "recipients are those of a max");
    if (given && nnz >= (int64_t)kNoRecipient)
        return fail(GEOT_ERROR_UNSUPPORTED, "recipients are 32-bit edge numbers: fewer than 2^32 - 1 edges");
    if ((grad_weight || (op == GEOT_OP_MAX && !given)) && !X) return fail(GEOT_ERROR_INVALID_VALUE, "X is NULL");
    if (op == GEOT_OP_MAX && !given && !out) return fail(GEOT_ERROR_INVALID_VALUE, "max needs out");
    const size_t xb = (size_t)(num_x_rows * F) * 4;
    if (grad_X && (overlaps(grad_X, xb, X, X ? (size_t)(num_x_rows * F) * es : 0) ||
                   overlaps(grad_X, xb, grad_out, (size_t)(num_rows * F) * 4) ||
                   overlaps(grad_X, xb, col, (size_t)nnz * is) || overlaps(grad_X, xb, sorted_row, (size_t)nnz * is) ||
                   overlaps(grad_X, xb, weight, weight ? (size_t)nnz * 4 : 0) ||
                   overlaps(grad_X, xb, grad_weight, grad_weight ? (size_t)nnz * 4 : 0)))
        return fail(GEOT_ERROR_INVALID_VALUE, "grad_X overlaps another array");
    if (grad_weight && (overlaps(grad_weight, (size_t)nnz * 4, weight, (size_t)nnz * 4) ||
                        overlaps(grad_weight, (size_t)nnz * 4, col, (size_t)nnz * is) ||
                        overlaps(grad_weight, (size_t)nnz * 4, sorted_row, (size_t)nnz * is) ||
                        overlaps(grad_weight, (size_t)nnz * 4, X, X ? (size_t)(num_x_rows * F) * es : 0)))
        return fail(GEOT_ERROR_INVALID_VALUE, "grad_weight overlaps an input");
    if (!grad_X && !grad_weight) return GEOT_SUCCESS;
    // widest vector that F and every pointer allow (fp32 operands: 16-byte loads of 4; 16-bit X
    // also 8 elements, loaded as 16 bytes, except for max: its three passes ran faster with 4 on
    // the SpMM graph, bf16 / int32: 30.7 against 32.8 ms)
    const uintptr_t ptrs = (uintptr_t)grad_out | (uintptr_t)X | (uintptr_t)grad_X | (uintptr_t)out | (uintptr_t)given;
    int V = 1;
    if (es == 2 && op != GEOT_OP_MAX && F % 8 == 0 && (ptrs & 15) == 0) V = 8;
    else if (F % 4 == 0 && (ptrs & 15) == 0) V = 4;
    else if (F % 2 == 0 && (ptrs & 7) == 0) V = 2;
    // temporaries from the stream-ordered pool (the forward call below uses the per-stream buffer):
    // row starts (mean), max recipients (max), the transposed edge list (grad_X for sum and mean)
    const bool mean = op == GEOT_OP_MEAN, mx = op == GEOT_OP_MAX;
    // max: grad_X pulled over the transposed list where its records are packed (X below 2^31
    // rows) and the recipients 32-bit; otherwise one atomic add per recipient
    const bool pull = mx && grad_X && num_x_rows <= (int64_t)INT32_MAX && seg_bwd_arg32(nnz);
    const bool transpose = grad_X && (!mx || pull);
    size_t at = 0;
    auto take = [&](size_t b) { const size_t o = at; at = align256(at + b); return o; };
    const size_t o_roff = mean ? take((size_t)(num_rows + 1) * 8) : 0;
    const size_t o_arg = mx && !given ? take((size_t)(num_rows * F) * (seg_bwd_arg32(nnz) ? 4 : 8)) : 0;
    const int64_t nx = num_x_rows;
    const size_t o_cnt = transpose ? take((size_t)((nx + 1) & ~(int64_t)1) * 4) : 0;
    const size_t o_off = transpose ? take((size_t)(nx + 1) * 8) : 0;
    const size_t o_sums = transpose ? take((size_t)((nx + 4095) / 4096 + 1) * 8) : 0;
    // the transposed list: records {col, row, coefficient, edge} with int32 ids (12 bytes, no
    // edge, from the radix partition where the edge numbers are not needed), or (X with 2^31
    // rows or more) three arrays
    const bool packed = nx <= (int64_t)INT32_MAX;
    const size_t bucket_b = transpose ? transpose_scratch_bytes(nnz, nx, pull) : 0;
    const size_t o_rec = transpose && packed ? take((size_t)nnz * (bucket_b && !pull ? 12 : 16)) : 0;
    const size_t o_bucket = bucket_b ? take(bucket_b) : 0;
    const size_t o_key = transpose && !packed ? take((size_t)nnz * 8) : 0;
    const size_t o_row = transpose && !packed ? take((size_t)nnz * 8) : 0;
    const size_t o_w = transpose && !packed ? take((size_t)nnz * 4) : 0;
    ScratchGuard sg;
    sg.st = st;
    geot_status_t s = scratch_alloc(&sg.p, at, st);
    if (s != GEOT_SUCCESS) return s;
    char *base = (char *)sg.p;
    int64_t *roff = mean ? (int64_t *)(base + o_roff) : nullptr;
    void *arg = mx ? (given ? (void *)given : (void *)(base + o_arg)) : nullptr;
    if (mean) {
        void *unused = nullptr;
        GapList gaps;
        StreamCtx *ctx = nullptr;
        s = stream_scratch(0, st, &unused, &gaps, &ctx);
        if (s != GEOT_SUCCESS) return s;
        s = poison(ctx, [&]() -> geot_status_t {
            if (idx32)
                GEOT_HIP(launch_offsets_i32(static_cast<const int32_t *>(sorted_row), nnz, num_rows, roff, gaps, st),
                         "launch offsets kernel");
            else
                GEOT_HIP(launch_offsets(static_cast<const int64_t *>(sorted_row), nnz, num_rows, roff, gaps, st),
                         "launch offsets kernel");
            GEOT_HIP(launch_gap_fill_i64(roff, num_rows + 1, gaps, st), "launch gap fill kernel");
            return GEOT_SUCCESS;
        }());
        if (s != GEOT_SUCCESS) return s;
    }
    const int bop = op == GEOT_OP_SUM ? GEOT_BWD_SUM : (mean ? GEOT_BWD_MEAN : GEOT_BWD_MAX);
    // weights (and, for max where it is not pulled, X through atomic adds of the recipients only)
    GEOT_HIP(launch_gs_bwd(X, elem, num_x_rows, col, idx32, weight, sorted_row, roff, out, grad_out, nnz, num_rows,
                           F, V, bop, arg, given != nullptr, mx && !pull ? grad_X : nullptr, grad_weight, st),
             "launch fused backward kernels");
    if (transpose) {
        // grad_X = gather_scatter of grad_out over the edges sorted by col (sum of coef * grad_out rows)
        int64_t *key_t = packed ? nullptr : (int64_t *)(base + o_key);
        int64_t *row_t = packed ? nullptr : (int64_t *)(base + o_row);
        float *w_t = packed ? nullptr : (float *)(base + o_w);
        int32_t *rec = packed ? (int32_t *)(base + o_rec) : nullptr;
        int rec_words = 4;
        GEOT_HIP(launch_transpose(col, nx, sorted_row, idx32, weight, roff, num_rows, mean, nnz, (unsigned *)(base + o_cnt),
                                  (int64_t *)(base + o_off), (int64_t *)(base + o_sums), key_t, row_t, w_t, rec,
                                  bucket_b ? base + o_bucket : nullptr, pull, &rec_words, nullptr, st),
                 "launch transpose kernels");
        if (pull) {
            GEOT_HIP(launch_gs_bwd_x_max_pull(rec, (const int64_t *)(base + o_off), arg, grad_out, nx, num_rows, F, V,
                                              grad_X, st),
                     "launch max pull kernel");
            void *p_pull = sg.p;
            sg.p = nullptr;
            return scratch_free(p_pull, st);
        }
        Problem tp{true, grad_out, num_rows, row_t, w_t, key_t, nnz, nx, F, GEOT_OP_SUM, grad_X};
        if (packed) {
            tp.idx = rec;
            tp.col = rec + 1;
            tp.w = (const float *)(rec + 2);
            tp.idx32 = 1;
            tp.meta_stride = rec_words;
        }
        geot_kernel_choice_t c;
        select_raw(nnz, nx, F, GEOT_OP_SUM, 1, nullptr, &c);
        if (tp.typed() && c.family == GEOT_FAMILY_SP) c = geot_kernel_choice_t{GEOT_FAMILY_EP, 0, 0, 0, 0, 0};
        // The transposed list gathers the destination rows, which repeat as often as the rows'
        // edge counts and stay in cache: no column tiles in sequence (on the SpMM graph, 3.41 ms
        // over the kept list without them, 3.55 ms with two), and longer row runs per group
        // (there, one 128-column tile: 64 rows 3.16 ms, 128 rows 3.05-3.12, 256 rows 3.01, 512
        // rows 3.00, 1,024 rows 3.06).
        untile(&c);
        if (nnz >= ((int64_t)1 << 20) && c.family == GEOT_FAMILY_EP && c.rows != 0 && c.rows < 256) c.rows = 256;
        Resolved r;
        s = resolve(tp, c, &r, true);
        if (s != GEOT_SUCCESS) return s;
        s = run_ep(tp, r, st);
        if (s != GEOT_SUCCESS) return s;
    }
    void *p_free = sg.p;
    sg.p = nullptr;
    return scratch_free(p_free, st);
}

geot_status_t geot_gather_scatter_backward_typed(const void *X, geot_dtype_t x_type, int64_t num_x_rows,
                                                 const void *col, const float *weight, const void *sorted_row,
                                                 geot_index_type_t index_type, int64_t nnz, int64_t num_rows, int64_t F,
                                                 geot_op_t op, const float *grad_out, const float *out, float *grad_X,
                                                 float *grad_weight, void *stream) {
    return gs_backward(X, x_type, num_x_rows, col, weight, sorted_row, index_type, nnz, num_rows, F, op, grad_out,
                       out, nullptr, grad_X, grad_weight, stream);
}

geot_status_t geot_gather_scatter_backward_max_arg(const void *X, geot_dtype_t x_type, int64_t num_x_rows,
                                                   const void *col, const float *weight, const void *sorted_row,
                                                   geot_index_type_t index_type, int64_t nnz, int64_t num_rows,
                                                   int64_t F, const float *grad_out, const uint32_t *arg,
                                                   float *grad_X, float *grad_weight, void *stream) {
    if (!arg) {
        t_detail.clear();
        return fail(GEOT_ERROR_INVALID_VALUE, "arg is NULL");
    }
    return gs_backward(X, x_type, num_x_rows, col, weight, sorted_row, index_type, nnz, num_rows, F, GEOT_OP_MAX,
                       grad_out, nullptr, arg, grad_X, grad_weight, stream);
}

geot_status_t geot_gather_scatter_backward(const float *X, int64_t num_x_rows, const int64_t *col,
                                           const float *weight, const int64_t *sorted_row, int64_t nnz,
                                           int64_t num_rows, int64_t F, geot_op_t op,
                                           const float *grad_out, const float *out, float *grad_X,
                                           float *grad_weight, void *stream) {
    return geot_gather_scatter_backward_typed(X, GEOT_DTYPE_F32, num_x_rows, col, weight, sorted_row, GEOT_INDEX_I64,
                                              nnz, num_rows, F, op, grad_out, out, grad_X, grad_weight, stream);
}

geot_status_t geot_transpose_edges(const int64_t *col, int64_t num_x_rows, const float *weight,
                                   const int64_t *sorted_row, int64_t nnz, int64_t num_rows, geot_op_t op,
                                   int64_t *sorted_col_out, int64_t *row_out, float *coef_out, void *stream) {
    t_detail.clear();
    if (op != GEOT_OP_SUM && op != GEOT_OP_MEAN)
        return fail(GEOT_ERROR_INVALID_VALUE, "a transposed list serves sum and mean only");
    if (nnz < 0 || num_rows < 0 || num_x_rows < 0) return fail(GEOT_ERROR_INVALID_VALUE, "negative size");
    if (nnz == 0) return GEOT_SUCCESS;
    if (num_rows == 0 || num_x_rows == 0) return fail(GEOT_ERROR_INVALID_VALUE, "empty row or X range with nnz > 0");
    if (num_rows > (int64_t)INT32_MAX) return fail(GEOT_ERROR_INVALID_VALUE, "num_rows must be < 2^31");
    if (nnz > ((int64_t)1 << 60)) return fail(GEOT_ERROR_INVALID_VALUE, "size overflow");
    if (!col || !sorted_row || !sorted_col_out || !row_out || !coef_out)
        return fail(GEOT_ERROR_INVALID_VALUE, "NULL array");
    const size_t n8 = (size_t)nnz * 8, n4 = (size_t)nnz * 4;
    const void *outs[3] = {sorted_col_out, row_out, coef_out};
    const size_t out_b[3] = {n8, n8, n4};
    for (int i = 0; i < 3; ++i) {
        if (overlaps(outs[i], out_b[i], col, n8) || overlaps(outs[i], out_b[i], sorted_row, n8) ||
            overlaps(outs[i], out_b[i], weight, weight ? n4 : 0))
            return fail(GEOT_ERROR_INVALID_VALUE, "an output overlaps an input");
        for (int j = i + 1; j < 3; ++j)
            if (overlaps(outs[i], out_b[i], outs[j], out_b[j]))
                return fail(GEOT_ERROR_INVALID_VALUE, "the outputs overlap");
    }
    hipStream_t st = (hipStream_t)stream;
    const bool mean = op == GEOT_OP_MEAN;
    const int64_t nx = num_x_rows;
    size_t at = 0;
    auto take = [&](size_t b) { const size_t o = at; at = align256(at + b); return o; };
    const size_t o_roff = mean ? take((size_t)(num_rows + 1) * 8) : 0;
    const size_t o_cnt = take((size_t)((nx + 1) & ~(int64_t)1) * 4);
    const size_t o_off = take((size_t)(nx + 1) * 8);
    const size_t o_sums = take((size_t)((nx + 4095) / 4096 + 1) * 8);
    // the radix partition (from 2^20 edges where its bins stay small) writes the outputs from
    // its final pass; otherwise the edges are placed as 16-byte records (one store per edge)
    // and split into the outputs by one streaming pass
    const size_t bucket_b = transpose_scratch_bytes(nnz, nx, false);
    const size_t o_bucket = bucket_b ? take(bucket_b) : 0;
    const bool packed = nx <= (int64_t)INT32_MAX;
    const size_t o_rec = packed ? take((size_t)nnz * (bucket_b ? 12 : 16)) : 0;
    ScratchGuard sg;
    sg.st = st;
    geot_status_t s = scratch_alloc(&sg.p, at, st);
    if (s != GEOT_SUCCESS) return s;
    char *base = (char *)sg.p;
    int64_t *roff = mean ? (int64_t *)(base + o_roff) : nullptr;
    int32_t *rec = packed ? (int32_t *)(base + o_rec) : nullptr;
    if (mean) {
        void *unused = nullptr;
        GapList gaps;
        StreamCtx *ctx = nullptr;
        s = stream_scratch(0, st, &unused, &gaps, &ctx);
        if (s != GEOT_SUCCESS) return s;
        s = poison(ctx, [&]() -> geot_status_t {
            GEOT_HIP(launch_offsets(sorted_row, nnz, num_rows, roff, gaps, st), "launch offsets kernel");
            GEOT_HIP(launch_gap_fill_i64(roff, num_rows + 1, gaps, st), "launch gap fill kernel");
            return GEOT_SUCCESS;
        }());
        if (s != GEOT_SUCCESS) return s;
    }
    bool written = false;
    GEOT_HIP(launch_transpose(col, nx, sorted_row, 0, weight, roff, num_rows, mean, nnz, (unsigned *)(base + o_cnt),
                              (int64_t *)(base + o_off), (int64_t *)(base + o_sums), sorted_col_out, row_out,
                              coef_out, rec, bucket_b ? base + o_bucket : nullptr, false, nullptr, &written, st),
             "launch transpose kernels");
    if (packed && !written)
        GEOT_HIP(launch_unpack(rec, nnz, sorted_col_out, row_out, coef_out, st), "launch unpack kernel");
    void *p_free = sg.p;
    sg.p = nullptr;
    return scratch_free(p_free, st);
}

geot_status_t geot_select(int64_t nnz, int64_t num_segments, int64_t F, geot_op_t op, int32_t gather,
                          const geot_index_stats_t *stats, geot_kernel_choice_t *out) {
    t_detail.clear();
    if (!out) return fail(GEOT_ERROR_INVALID_VALUE, "out is NULL");
    if (op != GEOT_OP_SUM && op != GEOT_OP_MEAN && op != GEOT_OP_MAX)
        return fail(GEOT_ERROR_INVALID_VALUE, "unknown op %d", (int)op);
    if (nnz < 0 || num_segments < 0 || F < 0) return fail(GEOT_ERROR_INVALID_VALUE, "negative size");
    geot_kernel_choice_t c;
    select_raw(nnz, num_segments, F, op, gather == 0 ? 0 : (gather == 2 ? 2 : 1), stats, &c);
    if (F == 0) {
        *out = c;
        return GEOT_SUCCESS;
    }
    // resolve against 256-byte aligned pointers (what device allocators return)
    Problem p{gather != 0, (const float *)(uintptr_t)256, 0, nullptr, nullptr, nullptr,
              nnz, num_segments, F, op, (float *)(uintptr_t)256};
    Resolved r;
    geot_status_t s = resolve(p, c, &r, true);
    if (s != GEOT_SUCCESS) return s;
    *out = to_choice(r);
    return GEOT_SUCCESS;
}

geot_status_t geot_index_stats(const int64_t *sorted_index, int64_t nnz, int64_t num_segments,
                               geot_index_stats_t *host_out, void *stream) {
    t_detail.clear();
    if (!host_out) return fail(GEOT_ERROR_INVALID_VALUE, "host_out is NULL");
    if (nnz < 0 || num_segments <= 0) return fail(GEOT_ERROR_INVALID_VALUE, "need nnz >= 0 and num_segments > 0");
    if (num_segments > (int64_t)INT32_MAX) return fail(GEOT_ERROR_INVALID_VALUE, "num_segments must be < 2^31");
    if (nnz > 0 && !sorted_index) return fail(GEOT_ERROR_INVALID_VALUE, "index is NULL");
    geot_index_stats_t o;
    memset(&o, 0, sizeof(o));
    o.nnz = nnz;
    o.num_segments = num_segments;
    o.mean_len = (double)nnz / (double)num_segments;
    if (nnz == 0) {
        o.num_empty = num_segments;
        *host_out = o;
        return GEOT_SUCCESS;
    }
    hipStream_t st = (hipStream_t)stream;
    const size_t off_bytes = align256((size_t)(num_segments + 1) * 8);
    void *scratch = nullptr;
    GapList gaps;
    StreamCtx *ctx = nullptr;
    geot_status_t s = stream_scratch(off_bytes + 64, st, &scratch, &gaps, &ctx);
    if (s != GEOT_SUCCESS) return s;
    int64_t *off = (int64_t *)scratch;
    unsigned long long *acc = (unsigned long long *)((char *)scratch + off_bytes);
    unsigned long long h[3] = {0, 0, 0};
    s = poison(ctx, [&]() -> geot_status_t {
        GEOT_HIP(launch_offsets(sorted_index, nnz, num_segments, off, gaps, st), "launch offsets kernel");
        GEOT_HIP(launch_gap_fill_i64(off, num_segments + 1, gaps, st), "launch gap fill kernel");
        GEOT_HIP(launch_zero_u64(acc, 3, st), "launch zero kernel");
        GEOT_HIP(launch_len_stats(off, num_segments, acc, st), "launch length statistics kernel");
        GEOT_HIP(hipMemcpyAsync(h, acc, sizeof(h), hipMemcpyDeviceToHost, st), "hipMemcpyAsync");
        GEOT_HIP(hipStreamSynchronize(st), "hipStreamSynchronize");
        return GEOT_SUCCESS;
    }());
    if (s != GEOT_SUCCESS) return s;
    o.sum_len_sq = (int64_t)h[0];
    o.max_len = (int64_t)h[1];
    o.num_empty = (int64_t)h[2];
    const double ex2 = (double)o.sum_len_sq / (double)num_segments;
    o.var_len = std::max(0.0, ex2 - o.mean_len * o.mean_len);
    *host_out = o;
    return GEOT_SUCCESS;
}

geot_status_t geot_check_index(const int64_t *sorted_index, int64_t nnz, int64_t num_segments,
                               const int64_t *col, int64_t num_x_rows, void *stream) {
    t_detail.clear();
    if (nnz < 0 || num_segments < 0 || num_x_rows < 0)
        return fail(GEOT_ERROR_INVALID_VALUE, "negative size");
    if (nnz == 0) return GEOT_SUCCESS;
    if (!sorted_index) return fail(GEOT_ERROR_INVALID_VALUE, "index is NULL");
    hipStream_t st = (hipStream_t)stream;
    ScratchGuard sg;
    sg.st = st;
    geot_status_t s = scratch_alloc(&sg.p, 64, st);
    if (s != GEOT_SUCCESS) return s;
    unsigned int *flags = (unsigned int *)sg.p;
    GEOT_HIP(launch_zero_u64((unsigned long long *)sg.p, 1, st), "launch zero kernel");
    GEOT_HIP(launch_check(sorted_index, nnz, num_segments, col, num_x_rows, flags, st),
             "launch check kernel");
    unsigned int h = 0;
    GEOT_HIP(hipMemcpyAsync(&h, flags, sizeof(h), hipMemcpyDeviceToHost, st), "hipMemcpyAsync");
    void *p_free = sg.p;
    sg.p = nullptr;
    s = scratch_free(p_free, st);
    if (s != GEOT_SUCCESS) return s;
    GEOT_HIP(hipStreamSynchronize(st), "hipStreamSynchronize");
    if (h & 1u) return fail(GEOT_ERROR_OUT_OF_RANGE, "index or column out of range");
    if (h & 2u) return fail(GEOT_ERROR_NOT_SORTED, "index is not non-decreasing");
    return GEOT_SUCCESS;
}

geot_status_t geot_release_scratch(void) {
    t_detail.clear();
    std::lock_guard<std::mutex> lk(g_cache_mu);
    geot_status_t st = GEOT_SUCCESS;
    for (auto &kv : g_cache) {
        if (!kv.second.p) continue;
        int cur = 0;
        hipError_t e = hipGetDevice(&cur);
        if (e == hipSuccess) e = hipSetDevice(kv.first.dev);
        if (e == hipSuccess) e = hipFreeAsync(kv.second.p, kv.first.st);
        if (e == hipSuccess) e = hipStreamSynchronize(kv.first.st);
        (void)hipSetDevice(cur);
        if (e != hipSuccess && st == GEOT_SUCCESS) st = hip_fail(e, "release scratch");
    }
    g_cache.clear();
    for (auto &r : g_retired) {  // buffers captured graphs held (the graphs are invalid from here on)
        int cur = 0;
        hipError_t e = hipGetDevice(&cur);
        if (e == hipSuccess) e = hipSetDevice(r.first);
        if (e == hipSuccess) e = hipDeviceSynchronize();
        if (e == hipSuccess) e = hipFreeAsync(r.second, nullptr);
        if (e == hipSuccess) e = hipDeviceSynchronize();
        (void)hipSetDevice(cur);
        if (e != hipSuccess && st == GEOT_SUCCESS) st = hip_fail(e, "release retired scratch");
    }
    g_retired.clear();
    return st;
}

geot_status_t geot_last_choice(geot_kernel_choice_t *out) {
    if (!out) return fail(GEOT_ERROR_INVALID_VALUE, "out is NULL");
    *out = t_last_choice;
    return GEOT_SUCCESS;
}

geot_status_t geot_profile_begin(int32_t max_records) {
    if (max_records < 0 || max_records > (1 << 20)) return fail(GEOT_ERROR_INVALID_VALUE, "bad max_records");
    for (auto &e : g_prof.ev) {
        (void)hipEventDestroy(e.first);
        (void)hipEventDestroy(e.second);
    }
    g_prof.ev.clear();
    g_prof.ev.reserve((size_t)max_records);
    g_prof.cap = max_records;
    g_prof.armed = max_records > 0;
    return GEOT_SUCCESS;
}

geot_status_t geot_profile_end(float *durations_ms, int32_t capacity, int32_t *count) {
    geot_status_t st = GEOT_SUCCESS;
    int32_t n = 0;
    for (auto &e : g_prof.ev) {
        float ms = 0.0f;
        hipError_t r = hipEventSynchronize(e.second);
        if (r == hipSuccess) r = hipEventElapsedTime(&ms, e.first, e.second);
        if (r != hipSuccess && st == GEOT_SUCCESS) st = hip_fail(r, "profile events");
        if (durations_ms && n < capacity) durations_ms[n] = ms;
        ++n;
        (void)hipEventDestroy(e.first);
        (void)hipEventDestroy(e.second);
    }
    g_prof.ev.clear();
    g_prof.armed = false;
    g_prof.cap = 0;
    if (count) *count = n;
    return st;
}

const char *geot_status_string(geot_status_t status) {
    switch (status) {
        case GEOT_SUCCESS: return "success";
        case GEOT_ERROR_INVALID_VALUE: return "invalid value";
        case GEOT_ERROR_NOT_SORTED: return "index not sorted";
        case GEOT_ERROR_OUT_OF_RANGE: return "index out of range";
        case GEOT_ERROR_HIP: return "HIP runtime error";
        case GEOT_ERROR_UNSUPPORTED: return "unsupported kernel choice";
    }
    return "unknown status";
}

const char *geot_last_error_detail(void) { return t_detail.c_str(); }

int32_t geot_version(void) { return GEOT_VERSION; }

}  // extern "C"
