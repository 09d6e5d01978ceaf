// The data-aware workload balancer of section 2.2 (the "workload balance
// abstraction" listing): a preprocessing pass, run on the device, that
//   1. counts the rows whose degree is close to the average degree and picks
//      the row-split backend when at least 90% of them are, the neighbour-group
//      backend otherwise;
//   2. cuts each row into work units (one per row for row split; slices of at
//      most group_size edges for neighbour groups) and numbers the partial-sum
//      slots of rows cut into several units;
//   3. orders the units longest first (a stable sort, so equal lengths keep
//      row order) so that wavefronts sharing a workgroup get equal work and
//      the heaviest units start first.
// Every count stays on the device: no host synchronization, nothing read back
// (a column-sliced plan reads its unit totals back once, at creation, to size
// itself).
//
// Column-sliced plans (an MI355X addition, cogdl_plan_create_sliced): in
// neighbour-group mode a row with more than slice_min edges is also cut at the
// boundaries of kSlices equal column ranges, and the units form kSlices lists
// (range s in list s, every other unit in list row % kSlices), sorted by
// (list, length), each walked by the workgroups of one XCD.
#include <new>

#include "common.hpp"
#include "internal.hpp"

struct cogdl_plan {
    cogdl::Plan p;
};

namespace cogdl {
namespace {

// Rows whose degree is close to the average; one atomic per workgroup (a
// grid-stride loop over a bounded grid keeps same-address atomics few).
__global__ __launch_bounds__(256) void k_plan_close(const int32_t *__restrict__ rowptr, int32_t n_rows,
                                                    int64_t nnz, int32_t *__restrict__ counters)
{
    __shared__ int wsum[4];
    int close = 0;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_rows;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t d = (int64_t)rowptr[i + 1] - rowptr[i];
        close += (2 * d * n_rows >= nnz && d * n_rows <= 2 * nnz) ? 1 : 0;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) close += __shfl_xor(close, off);
    if (lane_id() == 0) wsum[threadIdx.x / kWave] = close;
    __syncthreads();
    if (threadIdx.x == 0) {
        const int t = wsum[0] + wsum[1] + wsum[2] + wsum[3];
        if (t) atomicAdd(&counters[0], t);
    }
}

__device__ __forceinline__ int plan_mode(const int32_t *counters, int32_t n_rows, int req)
{
    if (req != COGDL_BALANCE_AUTO) return req;
    return (10LL * counters[0] >= 9LL * n_rows) ? COGDL_BALANCE_ROW_SPLIT : COGDL_BALANCE_NEIGHBOR_GROUP;
}

__global__ void k_plan_counts(const int32_t *__restrict__ rowptr, int32_t n_rows, int32_t G, int req,
                              int32_t *__restrict__ counters, int32_t *__restrict__ row_units,
                              int32_t *__restrict__ row_parts, int32_t *__restrict__ row_split)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    const int mode = plan_mode(counters, n_rows, req);
    if (i == 0) counters[1] = mode;
    if (i >= n_rows) return;
    const int d = rowptr[i + 1] - rowptr[i];
    int u = 1;
    if (mode == COGDL_BALANCE_NEIGHBOR_GROUP && d > G) u = (d + G - 1) / G;
    row_units[i] = u;
    row_parts[i] = u > 1 ? u : 0;
    row_split[i] = u > 1 ? 1 : 0;
}

// After the count scan: the totals (units, partial slots, split rows) of this
// rowptr must fit the capacities the plan was allocated with.  They do
// whenever rowptr[n_rows] is the nnz given at creation; a rowptr with more
// edges would make the emit pass write past the plan's arrays, so instead the
// totals are set to zero (an empty plan, no unit runs) and counters[5] = 1,
// which cogdl_plan_query reports as COGDL_ERR_PLAN.
__global__ void k_plan_check(int32_t *__restrict__ n_units, int32_t *__restrict__ n_parts,
                             int32_t *__restrict__ n_split, int64_t cap_units, int64_t cap_partials,
                             int64_t cap_split, int32_t *__restrict__ counters)
{
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    const bool fits = *n_units <= cap_units && *n_parts <= cap_partials && *n_split <= cap_split &&
                      *n_units >= 0 && *n_parts >= 0 && *n_split >= 0;
    if (!fits) {
        *n_units = 0;
        *n_parts = 0;
        *n_split = 0;
    }
    counters[5] = fits ? 0 : 1;
}

// Emit the units of each row in row order, with their sort keys.
__global__ void k_plan_emit(const int32_t *__restrict__ rowptr, int32_t n_rows, int32_t G,
                            const int32_t *__restrict__ counters,
                            const int32_t *__restrict__ row_units,
                            const int32_t *__restrict__ row_parts,
                            const int32_t *__restrict__ row_split, int4 *__restrict__ units_tmp,
                            uint32_t *__restrict__ keys, int4 *__restrict__ split_rows,
                            int4 *__restrict__ part_units)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n_rows || counters[5] != 0) return;
    const bool ng = counters[1] == COGDL_BALANCE_NEIGHBOR_GROUP;
    const int beg = rowptr[i], end = rowptr[i + 1];
    const int u0 = row_units[i];
    const int nu = row_units[i + 1] - u0;
    if (nu == 1) {
        units_tmp[u0] = make_int4(i, beg, end, -1);
        const int size = end - beg;
        keys[u0] = ng ? (uint32_t)(G - (size < G ? size : G)) : 0u;
        return;
    }
    const int p0 = row_parts[i];
    const int s = row_split[i];
    split_rows[s] = make_int4(i, p0, nu, end - beg);
    for (int g = 0; g < nu; ++g) {
        const int b = beg + g * G;
        const int e = (end - b > G) ? b + G : end;
        units_tmp[u0 + g] = make_int4(i, b, e, p0 + g);
        part_units[p0 + g] = make_int4(i, b, e, s);
        keys[u0 + g] = (uint32_t)(G - (e - b));
    }
}

// Units are sorted by key G - size (ascending): the tiny units (size <= T)
// form the tail.  counters[2] = number of units longer than T (all of them
// in row-split mode, whose keys are all 0), counters[3] = 0.
__global__ void k_plan_split(const uint32_t *__restrict__ sorted_keys,
                             const int32_t *__restrict__ n_units, int32_t G, int32_t T,
                             int32_t *__restrict__ counters)
{
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    const uint32_t bound = G > T ? (uint32_t)(G - T) : 0u;
    int32_t lo = 0, hi = *n_units;
    while (lo < hi) {
        const int32_t mid = lo + (hi - lo) / 2;
        if (sorted_keys[mid] < bound) lo = mid + 1; else hi = mid;
    }
    counters[2] = (G > T) ? lo : *n_units;
    counters[3] = 0;
}

// ----------------------------------------------------------- sliced plans

// Cuts of row [beg, end) (end > beg) at the column-range boundaries: cut[s]
// is the lower bound of column s * width in the row (a binary search over
// the whole row), and a running maximum keeps the cuts ordered for any column
// order: on sorted rows they are the exact boundaries, and any ordered cuts
// partition the row.  The seven searches advance in lockstep, so their loads
// are independent and a long row waits out one memory latency per halving
// instead of one per probe of each search in turn.
__device__ __forceinline__ void slice_cuts(const int32_t *__restrict__ col, int beg, int end, int64_t width,
                                           int (&cut)[kSlices + 1])
{
    int lo[kSlices - 1], hi[kSlices - 1];
#pragma unroll
    for (int s = 0; s < kSlices - 1; ++s) {
        lo[s] = beg;
        hi[s] = end;
    }
    int steps = 0;
    for (int n = end - beg; n > 0; n >>= 1) ++steps;
    for (int t = 0; t < steps; ++t) {
#pragma unroll
        for (int s = 0; s < kSlices - 1; ++s) {
            const int mid = lo[s] + ((hi[s] - lo[s]) >> 1);
            const int32_t v = col[mid < end ? mid : end - 1];
            const bool open = lo[s] < hi[s];
            const bool below = (int64_t)v < (int64_t)(s + 1) * width;
            lo[s] = (open && below) ? mid + 1 : lo[s];
            hi[s] = (open && !below) ? mid : hi[s];
        }
    }
    cut[0] = beg;
#pragma unroll
    for (int s = 0; s < kSlices - 1; ++s) cut[s + 1] = lo[s] > cut[s] ? lo[s] : cut[s];
    cut[kSlices] = end;
}

// The sliced unit count of row i (its cuts stored in row_cuts) after writing
// its unsliced counts to the alt arrays.
__device__ __forceinline__ int row_counts_sliced(const int32_t *__restrict__ rowptr,
                                                      const int32_t *__restrict__ col, int i, int32_t G,
                                                      int mode, int64_t width, int32_t slice_min,
                                                      int32_t *__restrict__ alt_units,
                                                      int32_t *__restrict__ alt_parts,
                                                      int32_t *__restrict__ alt_split,
                                                      int32_t *__restrict__ row_cuts)
{
    const int beg = rowptr[i], end = rowptr[i + 1];
    const int d = end - beg;
    const bool ng = mode == COGDL_BALANCE_NEIGHBOR_GROUP;
    int u = (ng && d > G) ? ceil_div(d, G) : 1;
    alt_units[i] = u;
    alt_parts[i] = u > 1 ? u : 0;
    alt_split[i] = u > 1 ? 1 : 0;
    if (ng && d > slice_min) {
        int cut[kSlices + 1];
        slice_cuts(col, beg, end, width, cut);
        u = 0;
        for (int s = 0; s < kSlices; ++s) u += ceil_div(cut[s + 1] - cut[s], G);
#pragma unroll
        for (int s = 1; s < kSlices; ++s) row_cuts[(int64_t)i * (kSlices - 1) + s - 1] = cut[s];
    }
    return u;
}

// Per-row counts of a sliced plan: the sliced ones (a row with more than
// slice_min edges gives ceil(len / G) units per nonempty slice), summed per
// workgroup into block_totals, and, in the alt arrays, the
// unsliced ones the build falls back to when the sliced totals exceed the
// plan's capacities.
__global__ void k_plan_counts_sliced(const int32_t *__restrict__ rowptr, const int32_t *__restrict__ col,
                                     int32_t n_rows, int32_t G, int req, int64_t width, int32_t slice_min,
                                     int32_t *__restrict__ counters, int32_t *__restrict__ row_units,
                                     int32_t *__restrict__ row_parts, int32_t *__restrict__ row_split,
                                     int32_t *__restrict__ alt_units, int32_t *__restrict__ alt_parts,
                                     int32_t *__restrict__ alt_split, int32_t *__restrict__ row_cuts,
                                     unsigned long long *__restrict__ block_totals)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    const int mode = plan_mode(counters, n_rows, req);
    if (i == 0) counters[1] = mode;
    uint32_t su = 0, sp = 0, ss = 0;
    if (i < n_rows) {
        const int u = row_counts_sliced(rowptr, col, i, G, mode, width, slice_min, alt_units, alt_parts,
                                        alt_split, row_cuts);
        row_units[i] = u;
        row_parts[i] = u > 1 ? u : 0;
        row_split[i] = u > 1 ? 1 : 0;
        su = (uint32_t)u;
        sp = u > 1 ? (uint32_t)u : 0u;
        ss = u > 1 ? 1u : 0u;
    }
    // workgroup sums, one slot per workgroup (k_plan_fit adds them up: atomics
    // from every wavefront on three addresses serialize)
    __shared__ uint32_t wsum[3][256 / kWave];
    const auto add = [](uint32_t a, uint32_t b) { return a + b; };
    su = group_reduce(su, kWave, add);
    sp = group_reduce(sp, kWave, add);
    ss = group_reduce(ss, kWave, add);
    const int w = threadIdx.x / kWave;
    if (lane_id() == 0) {
        wsum[0][w] = su;
        wsum[1][w] = sp;
        wsum[2][w] = ss;
    }
    __syncthreads();
    if (threadIdx.x < 3) {
        unsigned long long t = 0;
        for (int j = 0; j < (int)(blockDim.x / kWave); ++j) t += wsum[threadIdx.x][j];
        block_totals[(int64_t)blockIdx.x * 3 + threadIdx.x] = t;
    }
}

// counters[4] = 1 when the sliced totals fit the capacities (else the
// unsliced counts replace them and no row is sliced).
// The sliced totals (units, partial slots, split rows) from the workgroup sums
// of k_plan_counts_sliced, in a fixed order (one workgroup of 256 threads).
__global__ __launch_bounds__(256) void k_plan_fit(const unsigned long long *__restrict__ block_totals,
                                                  int64_t n_blocks, int64_t cap_units, int64_t cap_partials,
                                                  int64_t cap_split, unsigned long long *__restrict__ totals,
                                                  int32_t *__restrict__ counters)
{
    __shared__ unsigned long long part[3][256];
    unsigned long long t[3] = {0, 0, 0};
    for (int64_t b = threadIdx.x; b < n_blocks; b += blockDim.x)
#pragma unroll
        for (int c = 0; c < 3; ++c) t[c] += block_totals[b * 3 + c];
#pragma unroll
    for (int c = 0; c < 3; ++c) part[c][threadIdx.x] = t[c];
    __syncthreads();
    if (threadIdx.x < 3) {
        unsigned long long sum = 0;
        for (int j = 0; j < (int)blockDim.x; ++j) sum += part[threadIdx.x][j];
        totals[threadIdx.x] = sum;
        part[threadIdx.x][0] = sum;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        const bool fits = part[0][0] <= (unsigned long long)cap_units &&
                          part[1][0] <= (unsigned long long)cap_partials &&
                          part[2][0] <= (unsigned long long)cap_split;
        counters[4] = fits ? 1 : 0;
    }
}

__global__ void k_plan_fallback(int32_t n_rows, const int32_t *__restrict__ counters,
                                int32_t *__restrict__ row_units, int32_t *__restrict__ row_parts,
                                int32_t *__restrict__ row_split, const int32_t *__restrict__ alt_units,
                                const int32_t *__restrict__ alt_parts, const int32_t *__restrict__ alt_split)
{
    if (counters[4] != 0) return;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_rows;
         i += (int64_t)gridDim.x * blockDim.x) {
        row_units[i] = alt_units[i];
        row_parts[i] = alt_parts[i];
        row_split[i] = alt_split[i];
    }
}

// Units of a sliced plan with their sort keys (list << kb) | (G - size)
// (neighbour groups; row split: list << kb).  Slice s of a sliced row is in
// list s, every other unit in list row % kSlices.
__global__ void k_plan_emit_sliced(const int32_t *__restrict__ rowptr, int32_t n_rows, int32_t G,
                                   int kb, int32_t slice_min, const int32_t *__restrict__ row_cuts,
                                   const int32_t *__restrict__ counters,
                                   const int32_t *__restrict__ row_units,
                                   const int32_t *__restrict__ row_parts,
                                   const int32_t *__restrict__ row_split, int4 *__restrict__ units_tmp,
                                   uint32_t *__restrict__ keys, int4 *__restrict__ split_rows,
                                   int4 *__restrict__ part_units)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n_rows || counters[5] != 0) return;
    const bool ng = counters[1] == COGDL_BALANCE_NEIGHBOR_GROUP;
    const bool slice = ng && counters[4] != 0;
    const int beg = rowptr[i], end = rowptr[i + 1];
    const int d = end - beg;
    const int u0 = row_units[i];
    const int nu = row_units[i + 1] - u0;
    int cut[kSlices + 1];
    const bool sliced_row = slice && d > slice_min;
    if (sliced_row) {
        // the cuts the count pass found (the same for the same columns)
        cut[0] = beg;
#pragma unroll
        for (int s = 1; s < kSlices; ++s) cut[s] = row_cuts[(int64_t)i * (kSlices - 1) + s - 1];
        cut[kSlices] = end;
    }
    if (nu == 1) {
        uint32_t list = (uint32_t)(i % kSlices);
        if (sliced_row)
            for (int s = 0; s < kSlices; ++s)
                if (cut[s + 1] > cut[s]) list = (uint32_t)s;
        units_tmp[u0] = make_int4(i, beg, end, -1);
        keys[u0] = (list << kb) | (ng ? (uint32_t)(G - (d < G ? d : G)) : 0u);
        return;
    }
    const int p0 = row_parts[i];
    const int sidx = row_split[i];
    split_rows[sidx] = make_int4(i, p0, nu, d);
    if (sliced_row) {
        int g = 0;
        for (int s = 0; s < kSlices; ++s) {
            for (int b = cut[s]; b < cut[s + 1]; b += G) {
                const int e = (cut[s + 1] - b > G) ? b + G : cut[s + 1];
                if (g < nu) {
                    units_tmp[u0 + g] = make_int4(i, b, e, p0 + g);
                    part_units[p0 + g] = make_int4(i, b, e, sidx);
                    keys[u0 + g] = ((uint32_t)s << kb) | (uint32_t)(G - (e - b));
                }
                ++g;
            }
        }
        return;
    }
    const uint32_t home = (uint32_t)(i % kSlices) << kb;
    for (int g = 0; g < nu; ++g) {
        const int b = beg + g * G;
        const int e = (end - b > G) ? b + G : end;
        units_tmp[u0 + g] = make_int4(i, b, e, p0 + g);
        part_units[p0 + g] = make_int4(i, b, e, sidx);
        keys[u0 + g] = home | (uint32_t)(G - (e - b));
    }
}

// The list table of a sliced plan from the sorted keys: for list x its first
// unit, the end of its long units (keys below (x << kb) | (G - T)) and its
// end; counters[2] = the long units of all lists, counters[3] = 0.
__global__ void k_plan_lists(const uint32_t *__restrict__ sorted, const int32_t *__restrict__ n_units,
                             int32_t G, int32_t T, int kb, int32_t *__restrict__ tbl,
                             int32_t *__restrict__ counters)
{
    __shared__ int32_t longs[kSlices];
    const int x = threadIdx.x;
    if (x < kSlices) {
        const int32_t n = *n_units;
        const auto lb = [&](uint32_t key) {
            int32_t lo = 0, hi = n;
            while (lo < hi) {
                const int32_t mid = lo + (hi - lo) / 2;
                if (sorted[mid] < key) lo = mid + 1;
                else hi = mid;
            }
            return lo;
        };
        const uint32_t base = (uint32_t)x << kb;
        const int32_t lo = lb(base);
        const int32_t hi = x + 1 < kSlices ? lb((uint32_t)(x + 1) << kb) : n;
        const int32_t big = G > T ? lb(base | (uint32_t)(G - T)) : hi;
        tbl[x] = lo;
        tbl[kSlices + x] = big;
        tbl[2 * kSlices + x] = hi;
        longs[x] = big - lo;
    }
    __syncthreads();
    if (x == 0) {
        int32_t t = 0;
        for (int i = 0; i < kSlices; ++i) t += longs[i];
        counters[2] = t;
        counters[3] = 0;
    }
}

__global__ void k_plan_gather(const int4 *__restrict__ units_tmp, const uint32_t *__restrict__ order,
                              const int32_t *__restrict__ n_units, int64_t cap,
                              int4 *__restrict__ units)
{
    const int64_t n = *n_units;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n && i < cap;
         i += (int64_t)gridDim.x * blockDim.x)
        units[i] = units_tmp[order[i]];
}

__global__ void k_plan_export(const int4 *__restrict__ units, const int32_t *__restrict__ n_units,
                              int64_t capacity, int4 *__restrict__ out)
{
    const int64_t n = *n_units < capacity ? *n_units : capacity;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        out[i] = units[i];
}

size_t align256(size_t b) { return (b + 255) & ~size_t(255); }

// Rows per unit-count pass; the sliced counts and their fallback.
cogdl_status plan_counts_sliced(Plan &P, const int32_t *rowptr, const int32_t *col, hipStream_t s)
{
    const int n = P.n_rows;
    const unsigned blocks = (unsigned)((n + 255) / 256);
    const int64_t width = ((int64_t)P.n_cols + kSlices - 1) / kSlices;
    COGDL_LAUNCH("plan_counts", k_plan_counts_sliced, blocks, 256, s, rowptr, col, n, P.group_size,
                 (int)P.mode_req, width > 0 ? width : 1, P.slice_min, P.counters, P.row_units,
                 P.row_parts, P.row_split, P.alt_units, P.alt_parts, P.alt_split, P.row_cuts,
                 P.block_totals);
    COGDL_LAUNCH("plan_fit", k_plan_fit, 1, 256, s, P.block_totals, (int64_t)blocks, P.cap_units,
                 P.cap_partials, P.cap_split, P.totals, P.counters);
    return COGDL_OK;
}

cogdl_status plan_build(Plan &P, const int32_t *rowptr, const int32_t *col, hipStream_t s)
{
    const int n = P.n_rows;
    COGDL_HIP_TRY(fill_i32(P.counters, 8, 0, s));
    const int32_t G = P.group_size;
    const int kb = P.sliced ? P.key_bits : 0;
    // Pad keys sort after every real unit; the sort covers the capacity.
    const uint32_t pad = P.sliced ? (((uint32_t)(kSlices - 1) << kb) | (uint32_t)(G + 1))
                                  : (uint32_t)G + 1u;
    COGDL_HIP_TRY(fill_i32(reinterpret_cast<int32_t *>(P.sort_keys), P.cap_units, (int32_t)pad, s));
    if (n == 0) {
        COGDL_HIP_TRY(fill_i32(P.row_units, 1, 0, s));
        COGDL_HIP_TRY(fill_i32(P.row_parts, 1, 0, s));
        COGDL_HIP_TRY(fill_i32(P.row_split, 1, 0, s));
        if (P.sliced) COGDL_HIP_TRY(fill_i32(P.lists_tbl, 3 * kSlices, 0, s));
        return COGDL_OK;
    }
    const unsigned blocks = (unsigned)((n + 255) / 256);
    COGDL_LAUNCH("plan_close", k_plan_close, blocks < 512 ? blocks : 512, 256, s, rowptr, n, P.nnz,
                 P.counters);
    if (P.sliced) {
        const cogdl_status st = plan_counts_sliced(P, rowptr, col, s);
        if (st != COGDL_OK) return st;
        COGDL_LAUNCH("plan_fallback", k_plan_fallback, blocks < 1024 ? blocks : 1024, 256, s, n,
                     P.counters, P.row_units, P.row_parts, P.row_split, P.alt_units, P.alt_parts,
                     P.alt_split);
        COGDL_HIP_TRY(exclusive_scan3(P.row_units, P.row_parts, P.row_split, n, P.scan_ws, s));
        COGDL_LAUNCH("plan_check", k_plan_check, 1, 64, s, P.row_units + n, P.row_parts + n,
                     P.row_split + n, P.cap_units, P.cap_partials, P.cap_split, P.counters);
        COGDL_LAUNCH("plan_emit", k_plan_emit_sliced, blocks, 256, s, rowptr, n, G, kb, P.slice_min,
                     P.row_cuts, P.counters, P.row_units, P.row_parts, P.row_split, P.units_tmp,
                     P.sort_keys, P.split_rows, P.part_units);
    } else {
        COGDL_LAUNCH("plan_counts", k_plan_counts, blocks, 256, s, rowptr, n, G, (int)P.mode_req,
                     P.counters, P.row_units, P.row_parts, P.row_split);
        COGDL_HIP_TRY(exclusive_scan3(P.row_units, P.row_parts, P.row_split, n, P.scan_ws, s));
        COGDL_LAUNCH("plan_check", k_plan_check, 1, 64, s, P.row_units + n, P.row_parts + n,
                     P.row_split + n, P.cap_units, P.cap_partials, P.cap_split, P.counters);
        COGDL_LAUNCH("plan_emit", k_plan_emit, blocks, 256, s, rowptr, n, G, P.counters,
                     P.row_units, P.row_parts, P.row_split, P.units_tmp, P.sort_keys, P.split_rows,
                     P.part_units);
    }
    uint32_t *order = P.sort_vals;                    // [cap]: final order
    uint32_t *ping_k = P.sort_keys + P.cap_units;     // [2 * cap] ping buffers
    uint32_t *ping_v = P.sort_vals + P.cap_units;
    uint32_t *sorted = P.sort_keys + 3 * P.cap_units; // [cap] keys in execution order
    const int bits = bits_for(pad);
    COGDL_HIP_TRY(radix_sort_pairs(P.sort_keys, nullptr, sorted, order, P.cap_units, bits, ping_k,
                                   ping_v, P.sort_ws, s));
    if (P.sliced)
        COGDL_LAUNCH("plan_lists", k_plan_lists, 1, 64, s, sorted, P.n_units_dev(), G, kTinyUnit, kb,
                     P.lists_tbl, P.counters);
    else
        COGDL_LAUNCH("plan_split", k_plan_split, 1, 64, s, sorted, P.n_units_dev(), G, kTinyUnit,
                     P.counters);
    const int64_t gb = (P.cap_units + 255) / 256;
    COGDL_LAUNCH("plan_gather", k_plan_gather, (unsigned)(gb < 8192 ? gb : 8192), 256, s,
                 P.units_tmp, order, P.n_units_dev(), P.cap_units, P.units);
    return COGDL_OK;
}

}  // namespace
}  // namespace cogdl

using cogdl::Plan;

extern "C" {

const char *cogdl_status_string(cogdl_status s)
{
    switch (s) {
    case COGDL_OK: return "ok";
    case COGDL_ERR_INVALID: return "invalid argument";
    case COGDL_ERR_DTYPE: return "unsupported dtype";
    case COGDL_ERR_PLAN: return "plan does not match the call";
    case COGDL_ERR_NOMEM: return "device allocation failed";
    case COGDL_ERR_LAUNCH: return "kernel launch or HIP call failed";
    case COGDL_ERR_TOO_LARGE: return "size exceeds a limit of the call (int32 indices, or the static scratch of the allocation-free transpose)";
    }
    return "unknown status";
}

int32_t cogdl_version(void) { return 100; }

}  // extern "C"

namespace cogdl {
namespace {

cogdl_status plan_args(int32_t n_rows, int64_t nnz, const int32_t *rowptr, int32_t max_feat,
                       int32_t max_heads, cogdl_balance mode, int32_t group_size)
{
    if (n_rows < 0 || nnz < 0 || max_feat < 1 || max_heads < 0 || max_heads > COGDL_MAX_HEADS ||
        group_size < 0 || (n_rows > 0 && !rowptr) ||
        (mode != COGDL_BALANCE_AUTO && mode != COGDL_BALANCE_ROW_SPLIT &&
         mode != COGDL_BALANCE_NEIGHBOR_GROUP))
        return COGDL_ERR_INVALID;
    if (nnz > COGDL_MAX_NNZ || n_rows == INT32_MAX) return COGDL_ERR_TOO_LARGE;
    if (n_rows == 0 && nnz != 0) return COGDL_ERR_INVALID;
    return COGDL_OK;
}

int32_t default_group(int32_t group_size, int64_t nnz)
{
    int32_t G = group_size;
    if (G == 0) {
        G = 256;
        while (G < 4096 && (int64_t)G * 2 * 16384 <= nnz) G *= 2;
    }
    return G;
}

// The per-row arrays, counters and scan workspace: in the main allocation of
// a plain plan, in base2 of a sliced one (which also holds the unsliced
// counts and the list table), allocated first so that the creation can size
// the rest from the sliced totals.
size_t row_layout(Plan &P, char *b, bool assign)
{
    size_t off = 0;
    auto take = [&](size_t bytes) { size_t o = off; off += align256(bytes); return o; };
    const size_t rows = 4 * ((size_t)P.n_rows + 1);
    const size_t o_row_units = take(rows), o_row_parts = take(rows), o_row_split = take(rows);
    const size_t o_counters = take(4 * 8);
    P.scan_ws_bytes = scan_workspace_bytes(P.n_rows, 3);
    const size_t o_scan_ws = take(P.scan_ws_bytes);
    size_t o_alt = 0, o_tbl = 0, o_cuts = 0, o_tot = 0, o_btot = 0;
    if (P.sliced) {
        o_alt = take(3 * rows);
        o_tbl = take(4 * 3 * kSlices);
        o_cuts = take(4 * (kSlices - 1) * (size_t)P.n_rows);
        o_tot = take(8 * 3);
        o_btot = take(8 * 3 * (((size_t)P.n_rows + 255) / 256 + 1));
    }
    if (assign) {
        P.row_units = reinterpret_cast<int32_t *>(b + o_row_units);
        P.row_parts = reinterpret_cast<int32_t *>(b + o_row_parts);
        P.row_split = reinterpret_cast<int32_t *>(b + o_row_split);
        P.counters = reinterpret_cast<int32_t *>(b + o_counters);
        P.scan_ws = b + o_scan_ws;
        if (P.sliced) {
            P.alt_units = reinterpret_cast<int32_t *>(b + o_alt);
            P.alt_parts = P.alt_units + (P.n_rows + 1);
            P.alt_split = P.alt_parts + (P.n_rows + 1);
            P.lists_tbl = reinterpret_cast<int32_t *>(b + o_tbl);
            P.row_cuts = reinterpret_cast<int32_t *>(b + o_cuts);
            P.totals = reinterpret_cast<unsigned long long *>(b + o_tot);
            P.block_totals = reinterpret_cast<unsigned long long *>(b + o_btot);
        }
    }
    return off;
}

// The main allocation, sized by the capacities (with the row arrays unless the
// plan is sliced).
cogdl_status plan_alloc(Plan &P)
{
    const int64_t pstride = (P.max_feat + 7) / 8 * 8;
    size_t off = P.sliced ? 0 : row_layout(P, nullptr, false);
    auto take = [&](size_t bytes) { size_t o = off; off += align256(bytes); return o; };
    const size_t o_units = take(sizeof(int4) * P.cap_units);
    const size_t o_units_tmp = take(sizeof(int4) * P.cap_units);
    const size_t o_split = take(sizeof(int4) * P.cap_split);
    const size_t o_part_units = take(sizeof(int4) * P.cap_partials);
    const size_t o_keys = take(4 * 4 * (size_t)P.cap_units);
    const size_t o_vals = take(4 * 3 * (size_t)P.cap_units);
    P.sort_ws_bytes = radix_workspace_bytes(P.cap_units);
    const size_t o_sort_ws = take(P.sort_ws_bytes);
    const size_t o_partials = take(sizeof(float) * (size_t)P.cap_partials * pstride);
    const size_t o_parg = take(sizeof(int32_t) * (size_t)P.cap_partials * pstride);
    const size_t o_gstats = take(sizeof(float) * 2 * (size_t)P.cap_partials * P.max_heads);
    const size_t o_rstats = take(sizeof(float) * 2 * (size_t)P.cap_split * P.max_heads);
    P.bytes = off;
    if (hipMalloc(&P.base, P.bytes) != hipSuccess) {
        (void)hipGetLastError();
        P.base = nullptr;
        return COGDL_ERR_NOMEM;
    }
    char *b = static_cast<char *>(P.base);
    if (!P.sliced) row_layout(P, b, true);
    P.units = reinterpret_cast<int4 *>(b + o_units);
    P.units_tmp = reinterpret_cast<int4 *>(b + o_units_tmp);
    P.split_rows = reinterpret_cast<int4 *>(b + o_split);
    P.part_units = reinterpret_cast<int4 *>(b + o_part_units);
    P.sort_keys = reinterpret_cast<uint32_t *>(b + o_keys);
    P.sort_vals = reinterpret_cast<uint32_t *>(b + o_vals);
    P.sort_ws = b + o_sort_ws;
    P.partials = reinterpret_cast<float *>(b + o_partials);
    P.parg = reinterpret_cast<int32_t *>(b + o_parg);
    P.gstats = reinterpret_cast<float *>(b + o_gstats);
    P.rstats = reinterpret_cast<float *>(b + o_rstats);
    return COGDL_OK;
}

void plan_free(cogdl_plan *h)
{
    (void)hipDeviceSynchronize();
    if (h->p.base) (void)hipFree(h->p.base);
    if (h->p.base2) (void)hipFree(h->p.base2);
    delete h;
}

}  // namespace
}  // namespace cogdl

extern "C" {

cogdl_status cogdl_plan_create(int32_t n_rows, int64_t nnz, const int32_t *rowptr, int32_t max_feat,
                               int32_t max_heads, cogdl_balance mode, int32_t group_size,
                               hipStream_t stream, cogdl_plan **out)
{
    if (!out) return COGDL_ERR_INVALID;
    const cogdl_status va = cogdl::plan_args(n_rows, nnz, rowptr, max_feat, max_heads, mode, group_size);
    if (va != COGDL_OK) return va;
    const int32_t G = cogdl::default_group(group_size, nnz);

    cogdl_plan *h = new (std::nothrow) cogdl_plan;
    if (!h) return COGDL_ERR_NOMEM;
    Plan &P = h->p;
    P.n_rows = n_rows;
    P.nnz = nnz;
    P.group_size = G;
    P.max_feat = max_feat;
    P.max_heads = max_heads;
    P.mode_req = mode;
    if (hipGetDevice(&P.device) != hipSuccess) { delete h; return COGDL_ERR_LAUNCH; }
    P.cap_units = (int64_t)n_rows + nnz / G + 1;
    P.cap_split = nnz / G + 1;
    P.cap_partials = 2 * (nnz / G) + 2;
    if (cogdl::plan_alloc(P) != COGDL_OK) { delete h; return COGDL_ERR_NOMEM; }

    cogdl_status st = cogdl::plan_build(P, rowptr, nullptr, stream);
    if (st != COGDL_OK) {
        cogdl::plan_free(h);
        return st;
    }
    *out = h;
    return COGDL_OK;
}

cogdl_status cogdl_plan_create_sliced(int32_t n_rows, int64_t nnz, const int32_t *rowptr,
                                      const int32_t *col, int32_t n_cols, int32_t max_feat,
                                      int32_t max_heads, cogdl_balance mode, int32_t group_size,
                                      int32_t slice_min, hipStream_t stream, cogdl_plan **out)
{
    if (!out) return COGDL_ERR_INVALID;
    const cogdl_status va = cogdl::plan_args(n_rows, nnz, rowptr, max_feat, max_heads, mode, group_size);
    if (va != COGDL_OK) return va;
    if (n_cols < 0 || slice_min < 0 || (nnz > 0 && (!col || n_cols < 1)) || group_size > (1 << 24))
        return COGDL_ERR_INVALID;
    const int32_t G = cogdl::default_group(group_size, nnz);

    cogdl_plan *h = new (std::nothrow) cogdl_plan;
    if (!h) return COGDL_ERR_NOMEM;
    Plan &P = h->p;
    P.n_rows = n_rows;
    P.nnz = nnz;
    P.group_size = G;
    P.max_feat = max_feat;
    P.max_heads = max_heads;
    P.mode_req = mode;
    P.sliced = 1;
    P.n_cols = n_cols;
    P.slice_min = slice_min > 0 ? slice_min : COGDL_DEFAULT_SLICE_MIN;
    P.key_bits = cogdl::bits_for((uint64_t)G + 1);
    if (hipGetDevice(&P.device) != hipSuccess) { delete h; return COGDL_ERR_LAUNCH; }
    const size_t rows_bytes = cogdl::row_layout(P, nullptr, false);
    if (hipMalloc(&P.base2, rows_bytes) != hipSuccess) {
        (void)hipGetLastError();
        delete h;
        return COGDL_ERR_NOMEM;
    }
    cogdl::row_layout(P, static_cast<char *>(P.base2), true);
    // Capacities: the unsliced bounds, raised to the sliced totals of this
    // graph (counted here, the one host read-back of the plan); a rebuild on
    // a graph whose sliced totals exceed them falls back to unsliced units.
    P.cap_units = (int64_t)n_rows + nnz / G + 1;
    P.cap_split = nnz / G + 1;
    P.cap_partials = 2 * (nnz / G) + 2;
    if (n_rows > 0) {
        unsigned long long tot[3] = {0, 0, 0};
        const unsigned blocks = (unsigned)((n_rows + 255) / 256);
        cogdl_status st = COGDL_OK;
        if (cogdl::fill_i32(P.counters, 8, 0, stream) != hipSuccess) st = COGDL_ERR_LAUNCH;
        if (st == COGDL_OK) {
            cogdl::k_plan_close<<<blocks < 512 ? blocks : 512, 256, 0, stream>>>(rowptr, n_rows, nnz,
                                                                                  P.counters);
            if (hipGetLastError() != hipSuccess) st = COGDL_ERR_LAUNCH;
        }
        if (st == COGDL_OK) st = cogdl::plan_counts_sliced(P, rowptr, col, stream);
        if (st == COGDL_OK &&
            (hipMemcpyAsync(&tot[0], P.totals, sizeof(tot), hipMemcpyDeviceToHost, stream) != hipSuccess ||
             hipStreamSynchronize(stream) != hipSuccess))
            st = COGDL_ERR_LAUNCH;
        if (st != COGDL_OK) {
            cogdl::plan_free(h);
            return st;
        }
        if ((int64_t)tot[0] + 1 > P.cap_units) P.cap_units = (int64_t)tot[0] + 1;
        if ((int64_t)tot[1] + 2 > P.cap_partials) P.cap_partials = (int64_t)tot[1] + 2;
        if ((int64_t)tot[2] + 1 > P.cap_split) P.cap_split = (int64_t)tot[2] + 1;
    }
    if (cogdl::plan_alloc(P) != COGDL_OK) {
        cogdl::plan_free(h);
        return COGDL_ERR_NOMEM;
    }
    P.bytes += rows_bytes;                 // both allocations, as cogdl_plan_query reports them
    cogdl_status st = cogdl::plan_build(P, rowptr, col, stream);
    if (st != COGDL_OK) {
        cogdl::plan_free(h);
        return st;
    }
    *out = h;
    return COGDL_OK;
}

cogdl_status cogdl_plan_rebuild(cogdl_plan *plan, const int32_t *rowptr, hipStream_t stream)
{
    if (!plan || plan->p.sliced || (plan->p.n_rows > 0 && !rowptr)) return COGDL_ERR_INVALID;
    return cogdl::plan_build(plan->p, rowptr, nullptr, stream);
}

cogdl_status cogdl_plan_rebuild_sliced(cogdl_plan *plan, const int32_t *rowptr, const int32_t *col,
                                       hipStream_t stream)
{
    if (!plan || !plan->p.sliced || (plan->p.n_rows > 0 && !rowptr) || (plan->p.nnz > 0 && !col))
        return COGDL_ERR_INVALID;
    return cogdl::plan_build(plan->p, rowptr, col, stream);
}

cogdl_status cogdl_plan_destroy(cogdl_plan *plan)
{
    if (!plan) return COGDL_OK;
    cogdl_status st = COGDL_OK;
    if (hipDeviceSynchronize() != hipSuccess) st = COGDL_ERR_LAUNCH;
    if (hipFree(plan->p.base) != hipSuccess) st = COGDL_ERR_LAUNCH;
    if (plan->p.base2 && hipFree(plan->p.base2) != hipSuccess) st = COGDL_ERR_LAUNCH;
    delete plan;
    return st;
}

cogdl_status cogdl_plan_query(const cogdl_plan *plan, hipStream_t stream, cogdl_plan_info *info)
{
    if (!plan || !info) return COGDL_ERR_INVALID;
    const Plan &P = plan->p;
    int32_t v[6] = {0, 0, 0, 0, 0, 0};
    COGDL_HIP_TRY(hipMemcpyAsync(&v[0], P.n_units_dev(), 4, hipMemcpyDeviceToHost, stream));
    COGDL_HIP_TRY(hipMemcpyAsync(&v[1], P.n_split_dev(), 4, hipMemcpyDeviceToHost, stream));
    COGDL_HIP_TRY(hipMemcpyAsync(&v[2], P.n_parts_dev(), 4, hipMemcpyDeviceToHost, stream));
    COGDL_HIP_TRY(hipMemcpyAsync(&v[3], P.counters + 1, 4, hipMemcpyDeviceToHost, stream));
    COGDL_HIP_TRY(hipMemcpyAsync(&v[4], P.counters + 2, 4, hipMemcpyDeviceToHost, stream));
    COGDL_HIP_TRY(hipMemcpyAsync(&v[5], P.counters + 5, 4, hipMemcpyDeviceToHost, stream));
    COGDL_HIP_TRY(hipStreamSynchronize(stream));
    info->n_rows = P.n_rows;
    info->nnz = P.nnz;
    info->group_size = P.group_size;
    info->max_feat = P.max_feat;
    info->max_heads = P.max_heads;
    info->n_units = v[0];
    info->n_long_units = v[4];
    info->n_split_rows = v[1];
    info->n_partials = v[2];
    info->mode = P.n_rows == 0 ? (P.mode_req == COGDL_BALANCE_AUTO ? COGDL_BALANCE_ROW_SPLIT
                                                                     : (int32_t)P.mode_req)
                               : v[3];
    info->device_bytes = (int64_t)P.bytes;
    // the last build's rowptr held more edges than the plan was created for:
    // the plan was left empty (see k_plan_check)
    return (P.n_rows > 0 && v[5] != 0) ? COGDL_ERR_PLAN : COGDL_OK;
}

cogdl_status cogdl_plan_units(const cogdl_plan *plan, int32_t *units, int64_t capacity,
                              hipStream_t stream)
{
    if (!plan || capacity < 0 || (capacity > 0 && !units)) return COGDL_ERR_INVALID;
    if (capacity == 0) return COGDL_OK;
    const Plan &P = plan->p;
    const int64_t cap = capacity < P.cap_units ? capacity : P.cap_units;
    const int64_t gb = (cap + 255) / 256;
    COGDL_LAUNCH("plan_export", cogdl::k_plan_export, (unsigned)(gb < 4096 ? gb : 4096), 256,
                 stream, P.units, P.n_units_dev(), cap, reinterpret_cast<int4 *>(units));
    return COGDL_OK;
}

}  // extern "C"

namespace cogdl {
const Plan *plan_of(const cogdl_plan *h) { return h ? &h->p : nullptr; }
}  // namespace cogdl
