// Internal declarations shared by the kernel files and the host dispatch of
// libgeot_hip. Not part of the public ABI (include/geot.h is).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace geot {

constexpr int kBlock = 256;  // threads per block for every reduction kernel (4 waves of 64)

enum SrcMode : int {
    SRC_ROWS = 0,    // term = src[row, :]
    SRC_GATHER = 1,  // term = w[row] * X[col[row], :] (w == nullptr: X[col[row], :])
    SRC_PIECES = 2,  // term = partial[row, :] carrying a row count (cnt[row] == 0: no term)
};

// mean = sum, divided by the count on store; RED_MAXARG = max that also records, for every
// output element, its recipient: the lowest row (edge) whose term equals the maximum
enum RedOp : int { RED_SUM = 0, RED_MAX = 1, RED_MAXARG = 2 };
// a recorded recipient where there is none (an empty segment, a NaN maximum)
constexpr uint32_t kNoRecipient = 0xffffffffu;

// Storage type of src / X at level 0 (partials are always fp32 with int64 ids).
// Elements are widened to fp32 on load, which is exact for all three types.
enum ElemType : int { ELEM_F32 = 0, ELEM_BF16 = 1, ELEM_F16 = 2 };

// Runs of empty segments longer than kGapRun segments are not written by the
// kernel that finds them: it appends them to a device list, cut into records
// of kGapChunk segments (at most kGapMaxRecs records per run), and a grid-wide
// pass writes them afterwards.
// The fill pass resets the list itself: each of its blocks reads the count
// once and then takes a ticket, and the block that takes the last ticket
// zeroes the count and the ticket. The list is therefore empty whenever no
// call is running (no memset, no host-side state: calls captured in a HIP
// graph replay correctly).
constexpr int kGapRun = 32;
constexpr int kGapChunkLog2 = 13;       // records of 2^13 = 8192 segments, or of the least power of two
constexpr int kGapMaxRecsLog2 = 6;      // that cuts the run into at most 2^6 = 64 records
constexpr unsigned kGapCap = 65536;     // records in the list (24 bytes each)

struct GapList {
    unsigned int *count;   // records appended in this call
    unsigned int *ticket;  // fill blocks done (the last one resets count and ticket)
    int64_t *rec;          // [kGapCap][3]: first segment, end segment, value
};

// Arguments of one element-parallel pass (level 0 over the input rows, or a
// later level over the partials of segments that crossed block boundaries).
struct EpArgs {
    const void *src;        // rows (SRC_ROWS / SRC_PIECES) or X (SRC_GATHER), of type `elem`
    int64_t ld_src;         // row stride of src in elements
    const void *idx;        // sorted segment id of each row (int32 when idx32, else int64)
    const int64_t *cnt;     // SRC_PIECES: rows represented by each partial
    const void *col;        // SRC_GATHER: source row of each edge (same type as idx)
    const float *w;         // SRC_GATHER: edge weight or nullptr
    int64_t num_x_rows;     // SRC_GATHER: rows of X
    int64_t n;              // rows (edges, partials) of this pass
    int64_t S;              // output rows
    int64_t F;              // columns
    float *out;             // [S x ld_out]
    int64_t ld_out;
    float *pv;              // partials of this pass: [2 * chunks x ld_p], nullptr when one chunk
    int64_t *pseg;          // segment id of each partial
    int64_t *pcnt;          // row count of each partial
    int64_t ld_p;
    int32_t K;              // rows per row group
    int32_t ntiles;         // column tiles (blocks per chunk)
    int32_t mean;           // divide by the count when a segment is stored
    int32_t fill_gaps;      // write empty segments (level 0 only)
    GapList gaps;           // long runs of empty segments (level 0 only)
    int32_t elem;           // ElemType of src (SRC_PIECES: ELEM_F32)
    int32_t idx32;          // idx and col hold int32 (SRC_PIECES: 0)
    int32_t nt_rows;        // rows mode: non-temporal row loads (tiles of >= 128 bytes only)
    int32_t meta_stride;    // gather mode: idx, col and w of edge e at [e * meta_stride] (0 or 1: arrays)
    int32_t gap_blocks;     // SRC_PIECES, final level: this many extra blocks fill the gap list `gaps`
                            // (written by level 0, which has finished), in tiles of the level's width
    int32_t tile_major;     // block b takes column tile b / chunks and chunk b % chunks (else the
                            // ntiles tiles of a chunk are adjacent blocks)
    // RED_MAXARG only: recipients [S x ld_out] written beside out (kNoRecipient where none),
    // the recipients of this pass's partials [2 * chunks x ld_p], and (SRC_PIECES) those of
    // the partials it reads [n x ld_src]
    uint32_t *arg_out;
    uint32_t *pix;
    const uint32_t *six;
};

// Dispatches on (elem, idx32) to the translation unit holding those instantiations.
hipError_t launch_ep(const EpArgs &a, int red, int mode, int V, int NT, int L, int64_t nchunks,
                     hipStream_t stream);
#define GEOT_EP_LAUNCHER(NAME)                                                                  \
    hipError_t NAME(const EpArgs &a, int red, int mode, int V, int NT, int L, int64_t nchunks, \
                    hipStream_t stream)
GEOT_EP_LAUNCHER(launch_ep_f32_i64);
GEOT_EP_LAUNCHER(launch_ep_f32_i32);
GEOT_EP_LAUNCHER(launch_ep_bf16_i64);
GEOT_EP_LAUNCHER(launch_ep_bf16_i32);
GEOT_EP_LAUNCHER(launch_ep_f16_i64);
GEOT_EP_LAUNCHER(launch_ep_f16_i32);

// Segment-parallel pass: segment s covers rows off[s] .. off[s+1]-1.
struct SpArgs {
    const float *src;
    int64_t ld_src;
    const int64_t *off;     // [S + 1] segment starts
    const int64_t *col;
    const float *w;
    int64_t num_x_rows;
    int64_t S;
    int64_t F;
    float *out;
    int64_t ld_out;
    int32_t groups;         // row groups cooperating on one segment (power of two, <= 64 / L)
    int32_t ntiles;
    int32_t mean;
};

hipError_t launch_sp(const SpArgs &a, int red, int mode, int V, int NT, int L, hipStream_t stream);

// off[s] = first row with idx >= s for s in [0, S]; one pass over the index.
// Long runs go to `gaps` (value = the row they start at): run launch_gap_fill_i64 after.
// With `first` (optional, 2 * ceil(n / 2^shift) entries): first[2b] and first[2b + 1] = the ids
// of the first and the last row of block b of 2^shift rows.
hipError_t launch_offsets(const int64_t *idx, int64_t n, int64_t S, int64_t *off, GapList gaps,
                          hipStream_t stream, int64_t *first = nullptr, int shift = 0);
// the same over int32 ids
hipError_t launch_offsets_i32(const int32_t *idx, int64_t n, int64_t S, int64_t *off, GapList gaps,
                              hipStream_t stream, int64_t *first = nullptr, int shift = 0);

// Grid-wide passes over a gap list: out rows [first, end) = 0 in the columns of
// tile `value` (tiles of `tw` columns), or arr[first, end) = value. Both leave
// the list empty.
// Records are clamped to the `rows` (or `len`) of the current call.
hipError_t launch_gap_fill_rows(float *out, int64_t F, int64_t ld, int V, int64_t tw, int64_t rows,
                                 GapList gaps, uint32_t *arg, hipStream_t stream);
hipError_t launch_gap_fill_i64(int64_t *arr, int64_t len, GapList gaps, hipStream_t stream);

// out[0 .. rows*ld) = value for the first F columns of each row.
hipError_t launch_fill(float *out, int64_t rows, int64_t F, int64_t ld, float value, hipStream_t stream);

// Index statistics from segment starts: acc[0] += sum len^2, acc[1] = max len,
// acc[2] += empty count. acc must be zeroed first (launch_zero_i64).
hipError_t launch_len_stats(const int64_t *off, int64_t S, unsigned long long *acc, hipStream_t stream);

// Precondition check: flags |= 1 (out of range), 2 (not sorted).
hipError_t launch_check(const int64_t *idx, int64_t n, int64_t S, const int64_t *col, int64_t nx,
                        unsigned int *flags, hipStream_t stream);

hipError_t launch_zero_u64(unsigned long long *p, int64_t n, hipStream_t stream);

// ---- gradients (bwd_kernels.hip) ------------------------------------------
enum BwdOp : int { GEOT_BWD_SUM = 0, GEOT_BWD_MEAN = 1, GEOT_BWD_MAX = 2 };

hipError_t launch_fill_u64(unsigned long long *p, int64_t n, unsigned long long v, hipStream_t st);

// records {int32 key, int32 row, float coefficient, 0} -> key_t, row_t, w_t
hipError_t launch_unpack(const int32_t *rec, int64_t n, int64_t *key_t, int64_t *row_t, float *w_t,
                         hipStream_t st);

// Counting sort of the edges by col: key_t (sorted col), row_t and w_t (weight, divided by
// the row's edge count for mean; roff = row starts) of the transposed problem.
// counts [nx] (rounded up to even) and off [nx + 1] / sums [ceil(nx / 4096)] are scratch.
// With rec != nullptr (needs nx and the rows < 2^31) each edge is one 16-byte record
// {int32 key, int32 row, float coefficient, uint32 edge number (its low 32 bits)} at
// rec[4 * slot] and key_t, row_t, w_t are unused. rx_scratch (transpose_scratch_bytes(n, nx,
// edges) bytes, or nullptr) lets inputs from 2^20 edges take a radix partition by bins of
// columns in LDS-staged runs, with no global atomic per edge; counts and sums are then unused,
// and its records have 3 words {key, row, coefficient} unless `edges` asks for the edge numbers.
// *rec_words (nullable) gets the words per record written to rec (3 or 4). Either way off[c]
// (nx + 1 entries) ends as the start of column c's records. When rec and all three arrays are
// given and the radix partition runs, it writes the three arrays directly (rec is then scratch)
// and sets *arrays_written (nullable); otherwise the records are in rec.
// col and row are int32 when idx32, else int64.
hipError_t launch_transpose(const void *col, int64_t nx, const void *row, int idx32, const float *w,
                            const int64_t *roff, int64_t nrows, bool mean, int64_t n, unsigned *counts, int64_t *off,
                            int64_t *sums, int64_t *key_t, int64_t *row_t, float *w_t, int32_t *rec,
                            char *rx_scratch, bool edges, int *rec_words, bool *arrays_written, hipStream_t st);
// scratch of the radix transposition (0: the input takes the direct one); `edges`: 16-byte
// records that keep the edge numbers, else 12-byte ones
size_t transpose_scratch_bytes(int64_t n, int64_t nx, bool edges);
// fused form, max, w.r.t. X from the packed transposed list (rec, column starts off, both from
// launch_transpose) and the 32-bit recipients arg [R x F]: grad_X written whole, no atomics
hipError_t launch_gs_bwd_x_max_pull(const int32_t *rec, const int64_t *off, const void *arg, const float *gout,
                                    int64_t nx, int64_t R, int64_t F, int V, float *gX, hipStream_t st);

// grad_src[i] = grad_out[idx[i]] (divided by the segment length from off when mean), stored in
// the source's ElemType `elem` (16-bit: rounded to nearest even); idx int32 when idx32. V is 1,
// 2, 4 or (16-bit) 8. With `first` (the ids of each block's first and last rows, from
// launch_offsets with shift = seg_bwd_rows_log2(F, V)) and complete offsets, rows take their
// segments from off and the ids are read only where a block spans more than 255 segment ends.
hipError_t launch_seg_bwd_bcast(const float *gout, const void *idx, int idx32, const int64_t *off,
                                const int64_t *first, int64_t n, int64_t S, int64_t F, int V, int elem, bool mean,
                                void *gsrc, hipStream_t st);
// log2 of the rows one block of the segment gradient kernels covers, and their block count
int seg_bwd_rows_log2(int64_t F, int V);
int64_t seg_bwd_blocks(int64_t n, int64_t F, int V);

// max: arg [S x F] scratch of row numbers, 32-bit where seg_bwd_arg32(n), else 64-bit (a
// multiple of 8 bytes); grad_src gets grad_out at the first attaining row of each (s, f); src
// and grad_src of ElemType `elem`. off and first (optional) as for launch_seg_bwd_bcast: the
// stores then take their segments from the offsets.
bool seg_bwd_arg32(int64_t n);
// `given`: arg already holds the (32-bit) recipients, recorded by the forward; no recipient pass.
hipError_t launch_seg_bwd_max(const float *gout, const void *idx, int idx32, const void *src, const float *out,
                              const int64_t *off, const int64_t *first, int64_t n, int64_t S, int64_t F, int V,
                              int elem, void *arg, bool given, void *gsrc, hipStream_t st);

// fused form: grad_w, and for max grad_X (zero-filled here, then one atomic add per recipient;
// sum and mean take grad_X from the transposed gather, and passing grad_X for them is an error);
// off = row starts (mean), arg [R x F] scratch of edge numbers for max (32-bit where
// seg_bwd_arg32(n), else 64-bit; a multiple of 8 bytes). X of ElemType elem, col and row int32
// when idx32.
// `given`: arg already holds the (32-bit) recipients, recorded by the forward; no recipient pass.
hipError_t launch_gs_bwd(const void *X, int elem, int64_t nx, const void *col, int idx32, const float *w,
                         const void *row, const int64_t *off, const float *out, const float *gout, int64_t n, int64_t R,
                         int64_t F, int V, int op, void *arg, bool given, float *gX, float *gw, hipStream_t st);

}  // namespace geot
