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
// Every count stays on the device: no host synchronization, nothing read back.
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
    if (i >= n_rows) return;
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

cogdl_status plan_build(Plan &P, const int32_t *rowptr, hipStream_t s)
{
    const int n = P.n_rows;
    COGDL_HIP_TRY(fill_i32(P.counters, 4, 0, s));
    // Pad keys sort after every real unit; the sort covers the capacity.
    const uint32_t pad = (uint32_t)P.group_size + 1u;
    COGDL_HIP_TRY(fill_i32(reinterpret_cast<int32_t *>(P.sort_keys), P.cap_units, (int32_t)pad, s));
    if (n == 0) {
        COGDL_HIP_TRY(fill_i32(P.counters, 4, 0, s));
        COGDL_HIP_TRY(fill_i32(P.row_units, 1, 0, s));
        COGDL_HIP_TRY(fill_i32(P.row_parts, 1, 0, s));
        COGDL_HIP_TRY(fill_i32(P.row_split, 1, 0, s));
        return COGDL_OK;
    }
    const unsigned blocks = (unsigned)((n + 255) / 256);
    COGDL_LAUNCH("plan_close", k_plan_close, blocks < 512 ? blocks : 512, 256, s, rowptr, n, P.nnz,
                 P.counters);
    COGDL_LAUNCH("plan_counts", k_plan_counts, blocks, 256, s, rowptr, n, P.group_size,
                 (int)P.mode_req, P.counters, P.row_units, P.row_parts, P.row_split);
    COGDL_HIP_TRY(exclusive_scan3(P.row_units, P.row_parts, P.row_split, n, P.scan_ws, s));
    COGDL_LAUNCH("plan_emit", k_plan_emit, blocks, 256, s, rowptr, n, P.group_size, P.counters,
                 P.row_units, P.row_parts, P.row_split, P.units_tmp, P.sort_keys, P.split_rows,
                 P.part_units);
    uint32_t *order = P.sort_vals;                    // [cap]: final order
    uint32_t *ping_k = P.sort_keys + P.cap_units;     // [2 * cap] ping buffers
    uint32_t *ping_v = P.sort_vals + P.cap_units;
    uint32_t *sorted = P.sort_keys + 3 * P.cap_units; // [cap] keys in execution order
    const int bits = bits_for(pad);
    COGDL_HIP_TRY(radix_sort_pairs(P.sort_keys, nullptr, sorted, order, P.cap_units, bits, ping_k,
                                   ping_v, P.sort_ws, s));
    COGDL_LAUNCH("plan_split", k_plan_split, 1, 64, s, sorted, P.n_units_dev(), P.group_size,
                 kTinyUnit, P.counters);
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
    case COGDL_ERR_TOO_LARGE: return "size exceeds the int32 index format";
    }
    return "unknown status";
}

int32_t cogdl_version(void) { return 100; }

cogdl_status cogdl_plan_create(int32_t n_rows, int64_t nnz, const int32_t *rowptr, int32_t max_feat,
                               int32_t max_heads, cogdl_balance mode, int32_t group_size,
                               hipStream_t stream, cogdl_plan **out)
{
    if (!out) return COGDL_ERR_INVALID;
    if (n_rows < 0 || nnz < 0 || max_feat < 1 || max_heads < 0 || max_heads > COGDL_MAX_HEADS ||
        group_size < 0 || (n_rows > 0 && !rowptr) ||
        (mode != COGDL_BALANCE_AUTO && mode != COGDL_BALANCE_ROW_SPLIT &&
         mode != COGDL_BALANCE_NEIGHBOR_GROUP))
        return COGDL_ERR_INVALID;
    if (nnz > COGDL_MAX_NNZ || n_rows == INT32_MAX) return COGDL_ERR_TOO_LARGE;
    if (n_rows == 0 && nnz != 0) return COGDL_ERR_INVALID;
    int32_t G = group_size;
    if (G == 0) {
        G = 256;
        while (G < 4096 && (int64_t)G * 2 * 16384 <= nnz) G *= 2;
    }

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
    const int64_t pstride = (max_feat + 7) / 8 * 8;

    size_t off = 0;
    auto take = [&](size_t bytes) { size_t o = off; off += cogdl::align256(bytes); return o; };
    const size_t o_units = take(sizeof(int4) * P.cap_units);
    const size_t o_units_tmp = take(sizeof(int4) * P.cap_units);
    const size_t o_split = take(sizeof(int4) * P.cap_split);
    const size_t o_part_units = take(sizeof(int4) * P.cap_partials);
    const size_t o_row_units = take(4 * ((size_t)n_rows + 1));
    const size_t o_row_parts = take(4 * ((size_t)n_rows + 1));
    const size_t o_row_split = take(4 * ((size_t)n_rows + 1));
    const size_t o_counters = take(4 * 4);
    const size_t o_keys = take(4 * 4 * (size_t)P.cap_units);
    const size_t o_vals = take(4 * 3 * (size_t)P.cap_units);
    P.sort_ws_bytes = cogdl::radix_workspace_bytes(P.cap_units);
    const size_t o_sort_ws = take(P.sort_ws_bytes);
    P.scan_ws_bytes = cogdl::scan_workspace_bytes(n_rows, 3);
    const size_t o_scan_ws = take(P.scan_ws_bytes);
    const size_t o_partials = take(sizeof(float) * (size_t)P.cap_partials * pstride);
    const size_t o_parg = take(sizeof(int32_t) * (size_t)P.cap_partials * pstride);
    const size_t o_gstats = take(sizeof(float) * 2 * (size_t)P.cap_partials * max_heads);
    const size_t o_rstats = take(sizeof(float) * 2 * (size_t)P.cap_split * max_heads);
    P.bytes = off;
    if (hipMalloc(&P.base, P.bytes) != hipSuccess) {
        (void)hipGetLastError();
        delete h;
        return COGDL_ERR_NOMEM;
    }
    char *b = static_cast<char *>(P.base);
    P.units = reinterpret_cast<int4 *>(b + o_units);
    P.units_tmp = reinterpret_cast<int4 *>(b + o_units_tmp);
    P.split_rows = reinterpret_cast<int4 *>(b + o_split);
    P.part_units = reinterpret_cast<int4 *>(b + o_part_units);
    P.row_units = reinterpret_cast<int32_t *>(b + o_row_units);
    P.row_parts = reinterpret_cast<int32_t *>(b + o_row_parts);
    P.row_split = reinterpret_cast<int32_t *>(b + o_row_split);
    P.counters = reinterpret_cast<int32_t *>(b + o_counters);
    P.sort_keys = reinterpret_cast<uint32_t *>(b + o_keys);
    P.sort_vals = reinterpret_cast<uint32_t *>(b + o_vals);
    P.sort_ws = b + o_sort_ws;
    P.scan_ws = b + o_scan_ws;
    P.partials = reinterpret_cast<float *>(b + o_partials);
    P.parg = reinterpret_cast<int32_t *>(b + o_parg);
    P.gstats = reinterpret_cast<float *>(b + o_gstats);
    P.rstats = reinterpret_cast<float *>(b + o_rstats);

    cogdl_status st = cogdl::plan_build(P, rowptr, stream);
    if (st != COGDL_OK) {
        (void)hipDeviceSynchronize();
        (void)hipFree(P.base);
        delete h;
        return st;
    }
    *out = h;
    return COGDL_OK;
}

cogdl_status cogdl_plan_rebuild(cogdl_plan *plan, const int32_t *rowptr, hipStream_t stream)
{
    if (!plan || (plan->p.n_rows > 0 && !rowptr)) return COGDL_ERR_INVALID;
    return cogdl::plan_build(plan->p, rowptr, stream);
}

cogdl_status cogdl_plan_destroy(cogdl_plan *plan)
{
    if (!plan) return COGDL_OK;
    cogdl_status st = COGDL_OK;
    if (hipDeviceSynchronize() != hipSuccess) st = COGDL_ERR_LAUNCH;
    if (hipFree(plan->p.base) != hipSuccess) st = COGDL_ERR_LAUNCH;
    delete plan;
    return st;
}

cogdl_status cogdl_plan_query(const cogdl_plan *plan, hipStream_t stream, cogdl_plan_info *info)
{
    if (!plan || !info) return COGDL_ERR_INVALID;
    const Plan &P = plan->p;
    int32_t v[5] = {0, 0, 0, 0, 0};
    COGDL_HIP_TRY(hipMemcpyAsync(&v[0], P.n_units_dev(), 4, hipMemcpyDeviceToHost, stream));
    COGDL_HIP_TRY(hipMemcpyAsync(&v[1], P.n_split_dev(), 4, hipMemcpyDeviceToHost, stream));
    COGDL_HIP_TRY(hipMemcpyAsync(&v[2], P.n_parts_dev(), 4, hipMemcpyDeviceToHost, stream));
    COGDL_HIP_TRY(hipMemcpyAsync(&v[3], P.counters + 1, 4, hipMemcpyDeviceToHost, stream));
    COGDL_HIP_TRY(hipMemcpyAsync(&v[4], P.counters + 2, 4, hipMemcpyDeviceToHost, stream));
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
    return COGDL_OK;
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
