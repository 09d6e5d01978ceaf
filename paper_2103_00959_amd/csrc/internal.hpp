// Host-side internals shared by the translation units of the library: the
// plan object, the device primitives (scan, stable radix sort) and argument
// validation helpers.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "cogdl.h"

namespace cogdl {

// Work unit: edges [beg, end) of one row, reduced either straight into the
// output (part < 0) or into partial-sum slot `part`.
// Layout int4 {row, beg, end, part}.

// Column slices of a sliced plan: one per XCD of the MI355X.
constexpr int kSlices = 8;

struct Plan {
    int32_t n_rows = 0;
    int64_t nnz = 0;
    int32_t group_size = 0;
    int32_t max_feat = 0;
    int32_t max_heads = 0;
    cogdl_balance mode_req = COGDL_BALANCE_AUTO;
    int device = 0;

    int64_t cap_units = 0;     // >= sum_i max(1, ceil(d_i / G))
    int64_t cap_split = 0;     // >= number of rows with d_i > G
    int64_t cap_partials = 0;  // >= sum over split rows of ceil(d_i / G)

    void *base = nullptr;
    size_t bytes = 0;

    int4 *units = nullptr;        // [cap_units] execution order
    int4 *units_tmp = nullptr;    // [cap_units] row order (build scratch)
    int4 *split_rows = nullptr;   // [cap_split] {row, first partial slot, #slots, degree}
    int4 *part_units = nullptr;   // [cap_partials] {row, beg, end, split index}
    int32_t *row_units = nullptr; // [n_rows + 1] exclusive scan; [n_rows] = #units
    int32_t *row_parts = nullptr; // [n_rows + 1]; [n_rows] = #partial slots
    int32_t *row_split = nullptr; // [n_rows + 1]; [n_rows] = #split rows
    int32_t *counters = nullptr;  // [8]: 0 close-degree rows, 1 chosen mode,
                                  //      2 units longer than kTinyUnit, 3 zero,
                                  //      4 sliced plan: 1 when its rows were sliced,
                                  //      5 1 when the last build's totals exceeded the
                                  //        capacities (the plan was left empty)
    uint32_t *sort_keys = nullptr;   // [4 * cap_units]: keys, 2 ping buffers, sorted keys
    uint32_t *sort_vals = nullptr;   // [3 * cap_units]: order, then 2 ping buffers
    void *sort_ws = nullptr;
    size_t sort_ws_bytes = 0;
    void *scan_ws = nullptr;
    size_t scan_ws_bytes = 0;
    float *partials = nullptr;    // [cap_partials * max_feat]
    int32_t *parg = nullptr;      // [cap_partials * max_feat] edge ids of partial maxima
    float *gstats = nullptr;      // [cap_partials * max_heads * 2] per-group (m, z)
    float *rstats = nullptr;      // [cap_split * max_heads * 2] per-split-row (m, z)

    // Sliced plans (cogdl_plan_create_sliced): in neighbour-group mode a row
    // with more than slice_min edges is cut at the boundaries of kSlices equal
    // column ranges (then into groups of at most group_size edges), and the
    // units form kSlices lists, slice s in list s and every other unit in list
    // row % kSlices, so that each list's gathers stay inside one column range.
    int32_t sliced = 0;
    int32_t n_cols = 0;
    int32_t slice_min = 0;
    int32_t key_bits = 0;         // bits of the in-list sort key (group_size - size)
    void *base2 = nullptr;        // second allocation (sliced plans)
    int32_t *lists_tbl = nullptr; // [3 * kSlices]: list starts, ends of the long units, list ends
    int32_t *alt_units = nullptr; // [n_rows + 1] x 3: the unsliced counts, used when the
    int32_t *alt_parts = nullptr; //   sliced ones exceed the capacities
    int32_t *alt_split = nullptr;
    int32_t *row_cuts = nullptr;  // [n_rows][kSlices - 1]: the inner cuts of each sliced row
    unsigned long long *totals = nullptr;  // [3]: sliced units, partial slots, split rows
    unsigned long long *block_totals = nullptr;  // [3 per workgroup of the count pass]

    const int32_t *n_units_dev() const { return row_units + n_rows; }
    const int32_t *n_big_dev() const { return counters + 2; }
    const int32_t *zero_dev() const { return counters + 3; }
    const int32_t *n_split_dev() const { return row_split + n_rows; }
    const int32_t *n_parts_dev() const { return row_parts + n_rows; }
};

// Units of at most this many edges run in the narrow-sub-group path.
constexpr int kTinyUnit = 8;

// The unit ranges a launch walks (see unit_walk): the long units, the tiny
// units or all of them; one range, or one per list for a sliced plan.
struct UnitRange {
    const int32_t *lo;
    const int32_t *hi;
    int lists;
};

inline UnitRange long_units(const Plan &P)
{
    if (P.sliced) return {P.lists_tbl, P.lists_tbl + kSlices, kSlices};
    return {P.zero_dev(), P.n_big_dev(), 1};
}

inline UnitRange tiny_units(const Plan &P)
{
    if (P.sliced) return {P.lists_tbl + kSlices, P.lists_tbl + 2 * kSlices, kSlices};
    return {P.n_big_dev(), P.n_units_dev(), 1};
}

inline UnitRange all_units(const Plan &P)
{
    if (P.sliced) return {P.lists_tbl, P.lists_tbl + 2 * kSlices, kSlices};
    return {P.zero_dev(), P.n_units_dev(), 1};
}

template <typename Args>
inline void set_units(Args &a, const UnitRange &r)
{
    a.u_lo = r.lo;
    a.u_hi = r.hi;
    a.lists = r.lists;
}

// A grid of `blocks` workgroups adjusted for `lists` lists: a multiple of it.
inline int64_t list_grid(int64_t blocks, int lists)
{
    if (lists <= 1) return blocks > 0 ? blocks : 1;
    const int64_t b = blocks / lists * lists;
    return b < lists ? lists : b;
}

const Plan *plan_of(const cogdl_plan *h);

// Workgroups of `block` threads of `kernel` that fit on the device at once
// (all compute units), cached per kernel.
int resident_blocks(const void *kernel, int block);

// Y[row] = sum of the partial rows of every split row of the plan (F columns),
// divided by the row's degree when `mean`, then act(. + bias) when given.
cogdl_status sum_reduce_launch(const char *name, const Plan &P, int64_t F, void *Y, int ydt,
                               bool mean, const float *bias, int act, hipStream_t s);

// Kernel tracing hooks (no-ops unless cogdl_trace_enable was called).
int trace_begin(const char *name, hipStream_t s);
void trace_end(int slot, hipStream_t s);

// ---------------------------------------------------------- primitives

// Exclusive prefix sum of n int32 values; out has n + 1 entries and out[n]
// receives the total.  in and out may alias.  Workspace size from
// scan_workspace_bytes(n, 1).  exclusive_scan3 scans three arrays of n + 1
// entries in place with the launches of one (workspace scan_workspace_bytes(n, 3)).
size_t scan_workspace_bytes(int64_t n, int arrays = 1);
hipError_t exclusive_scan(const int32_t *in, int32_t *out, int64_t n, void *ws, hipStream_t s);
hipError_t exclusive_scan3(int32_t *a0, int32_t *a1, int32_t *a2, int64_t n, void *ws, hipStream_t s);

// An extra 32-bit array carried through a radix sort: read from `in`,
// written in sorted order to `out`; `ping` is 2 * n elements of scratch.
// For the first payload only, `in` may be nullptr with `rowptr` set: the
// values are then the CSR rows of the elements (element e = edge e of the
// rowptr of n_rows rows), found by the sort itself instead of read.
struct RadixPayload {
    const uint32_t *in = nullptr;
    uint32_t *out = nullptr;
    uint32_t *ping = nullptr;
    const int32_t *rowptr = nullptr;
    int64_t n_rows = 0;
};

// Stable LSD radix sort of (key, value) pairs on the low `bits` bits of the
// keys.  vals_in == nullptr means values 0..n-1.  Results land in keys_out /
// vals_out (keys_out may be nullptr when the sorted keys are not needed); up
// to two payload arrays move with the keys.  ping: 2 * n keys and 2 * n
// values of scratch.  Digits are at most 8 bits wide, the key bits spread
// evenly over the fewest passes that allows.
size_t radix_workspace_bytes(int64_t n);
hipError_t radix_sort_pairs(const uint32_t *keys_in, const uint32_t *vals_in, uint32_t *keys_out,
                            uint32_t *vals_out, int64_t n, int bits, uint32_t *ping_keys,
                            uint32_t *ping_vals, void *ws, hipStream_t s,
                            RadixPayload pay0 = RadixPayload(), RadixPayload pay1 = RadixPayload());

// Fill n int32 with a value (a kernel, so it is safe inside graph capture).
hipError_t fill_i32(int32_t *p, int64_t n, int32_t v, hipStream_t s);

// ---------------------------------------------------------- validation

inline bool dtype_ok(int d) { return d == COGDL_F32 || d == COGDL_BF16 || d == COGDL_F16; }
inline int dtype_bytes(int d) { return d == COGDL_F32 ? 4 : 2; }

inline int bits_for(uint64_t max_value)
{
    int b = 0;
    while (b < 32 && (max_value >> b) != 0) ++b;
    return b;
}

inline int next_pow2(int v)
{
    int p = 1;
    while (p < v) p <<= 1;
    return p;
}

inline int log2i(int v)
{
    int l = 0;
    while ((1 << l) < v) ++l;
    return l;
}

// Launch geometry of the gather kernels for one row of `width` elements of a
// `bytes`-wide format: VEC elements per lane, S lanes per edge row, CH chunks
// per lane and the number of feature slabs.
struct RowMap {
    int vec = 1;
    int S = 64;
    int log2S = 6;
    int ch = 1;
    int slab = 0;      // elements per slab
    int n_slabs = 1;
};

RowMap row_map(int64_t width, int elem_bytes, int unit_elems /* vec must divide it */,
               bool aligned16);

}  // namespace cogdl

// Launch a kernel between the tracing events; return COGDL_ERR_LAUNCH from the
// enclosing function if the launch fails.
#define COGDL_LAUNCH(name, kern, grid, block, stream, ...)            \
    do {                                                             \
        const int _slot = ::cogdl::trace_begin(name, stream);        \
        kern<<<(grid), (block), 0, (stream)>>>(__VA_ARGS__);         \
        const hipError_t _e = hipGetLastError();                     \
        ::cogdl::trace_end(_slot, stream);                           \
        if (_e != hipSuccess) return COGDL_ERR_LAUNCH;               \
    } while (0)

// The same with `shm` bytes of dynamic LDS per workgroup.
#define COGDL_LAUNCH_SHM(name, kern, grid, block, shm, stream, ...)   \
    do {                                                             \
        const int _slot = ::cogdl::trace_begin(name, stream);        \
        kern<<<(grid), (block), (shm), (stream)>>>(__VA_ARGS__);     \
        const hipError_t _e = hipGetLastError();                     \
        ::cogdl::trace_end(_slot, stream);                           \
        if (_e != hipSuccess) return COGDL_ERR_LAUNCH;               \
    } while (0)

// Same for functions returning hipError_t.
#define COGDL_LAUNCH_HIP(name, kern, grid, block, stream, ...)        \
    do {                                                             \
        const int _slot = ::cogdl::trace_begin(name, stream);        \
        kern<<<(grid), (block), 0, (stream)>>>(__VA_ARGS__);         \
        const hipError_t _e = hipGetLastError();                     \
        ::cogdl::trace_end(_slot, stream);                           \
        if (_e != hipSuccess) return _e;                             \
    } while (0)

#define COGDL_HIP_TRY(expr)                                  \
    do {                                                     \
        hipError_t _e = (expr);                              \
        if (_e != hipSuccess) return COGDL_ERR_LAUNCH;       \
    } while (0)
