// CSR -> CSC transpose of the graph structure, the setup of the backward
// pass of Eq. 1 (the gradient with respect to the node features is A^T G).
//
// A stable LSD radix sort of the edge ids keyed by column (digits of at most
// 8 bits, as many passes as the column count needs) gives perm directly, with
// each edge's row and value bits carried along as payloads (so nothing is
// gathered at random afterwards); colptr is read off the sorted keys.  Every step is
// integer work in a fixed order, so the result is bit-for-bit unique: inside
// a column the edges keep increasing CSR edge id.
#include <mutex>

#include "common.hpp"
#include "internal.hpp"

namespace cogdl {
namespace {

constexpr int kBlock = 256;

// Row of every edge (the transpose without edge ids): wavefront w covers the
// edges [w * kExpandSpan, ...) with a RowCursor, 4 x 64 edges per round.
constexpr int kExpandSpan = 2048;
constexpr int kExpandEdges = 4;

__global__ __launch_bounds__(kBlock) void k_expand_rows(const int32_t *__restrict__ rowptr,
                                                        int32_t n_rows, int64_t nnz,
                                                        uint32_t *__restrict__ row_of)
{
    const int lane = lane_id();
    const int64_t e0 = ((int64_t)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave) * kExpandSpan;
    if (e0 >= nnz) return;
    const int64_t e1 = e0 + kExpandSpan < nnz ? e0 + kExpandSpan : nnz;
    RowCursor rc;
    rc.start(rowptr, n_rows, e0);
    for (int64_t c = e0; c < e1; c += (int64_t)kWave * kExpandEdges) {
        int64_t e[kExpandEdges], row[kExpandEdges];
        bool want[kExpandEdges];
#pragma unroll
        for (int j = 0; j < kExpandEdges; ++j) {
            e[j] = c + (int64_t)j * kWave + lane;
            want[j] = e[j] < e1;
        }
        rc.resolve<kExpandEdges>(e, want, row);
#pragma unroll
        for (int j = 0; j < kExpandEdges; ++j)
            if (want[j]) row_of[e[j]] = (uint32_t)row[j];
    }
}

// colptr[c] = first slot whose key is >= c, from the sorted keys; each thread
// reads four consecutive keys with one 16-byte load.
__global__ __launch_bounds__(kBlock) void k_colptr(const uint32_t *__restrict__ skeys, int64_t nnz,
                                                   int32_t n_cols, int32_t *__restrict__ colptr)
{
    const int64_t q = ((int64_t)blockIdx.x * kBlock + threadIdx.x) * 4;
    if (q >= nnz) return;
    uint32_t k[4];
    if (q + 4 <= nnz) {
        const uint4 v = *reinterpret_cast<const uint4 *>(skeys + q);
        k[0] = v.x; k[1] = v.y; k[2] = v.z; k[3] = v.w;
    } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) k[i] = q + i < nnz ? skeys[q + i] : 0u;
    }
    int64_t prev = q > 0 ? (int64_t)skeys[q - 1] : -1;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int64_t p = q + i;
        if (p >= nnz) break;
        const int64_t key = k[i];
        for (int64_t c = prev + 1; c <= key; ++c) colptr[c] = (int32_t)p;
        prev = key;
        if (p == nnz - 1)
            for (int64_t c = key + 1; c <= n_cols; ++c) colptr[c] = (int32_t)nnz;
    }
}

struct CscLayout {
    size_t row_of, ping_k, ping_v, ping_r, ping_w, skeys, radix, total;
};

size_t al(size_t b) { return (b + 255) & ~size_t(255); }

CscLayout csc_layout(int64_t nnz)
{
    CscLayout L;
    size_t off = 0;
    L.row_of = off; off += al(4 * (size_t)nnz);
    L.ping_k = off; off += al(8 * (size_t)nnz);
    L.ping_v = off; off += al(8 * (size_t)nnz);
    L.ping_r = off; off += al(8 * (size_t)nnz);
    L.ping_w = off; off += al(8 * (size_t)nnz);
    L.skeys = off;  off += al(4 * (size_t)nnz);
    L.radix = off;  off += al(radix_workspace_bytes(nnz));
    L.total = off;
    return L;
}


// Scratch of cogdl_csr_to_csc_noalloc: one copy per GPU, placed by the code
// object loader and held until the process ends.  Host code never passes the
// array's name to a kernel (on the host it is only a stand-in symbol): it
// uses the device address hipGetSymbolAddress returns, looked up once per
// device on the first call with that device current.
__device__ __align__(256) unsigned char scratch[COGDL_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex scratch_mu;
void *scratch_ptr[kMaxDevices] = {};

cogdl_status device_scratch(void **out)
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return COGDL_ERR_LAUNCH;
    std::lock_guard<std::mutex> lock(scratch_mu);
    if (!scratch_ptr[dev]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
            (void)hipGetLastError();
            return COGDL_ERR_LAUNCH;
        }
        scratch_ptr[dev] = p;
    }
    *out = scratch_ptr[dev];
    return COGDL_OK;
}

cogdl_status csc_check(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *rowptr,
                       const int32_t *col, const float *val, const int32_t *colptr,
                       const int32_t *row_t, const float *val_t)
{
    if (n_rows < 0 || n_cols < 0 || nnz < 0) return COGDL_ERR_INVALID;
    if (nnz > COGDL_MAX_NNZ) return COGDL_ERR_TOO_LARGE;
    if (!colptr) return COGDL_ERR_INVALID;
    if (n_rows > 0 && !rowptr) return COGDL_ERR_INVALID;
    if (nnz > 0 && (!col || !row_t || n_rows == 0 || n_cols == 0)) return COGDL_ERR_INVALID;
    if ((val == nullptr) != (val_t == nullptr)) return COGDL_ERR_INVALID;
    return COGDL_OK;
}

// The transpose on a validated call, with `ws` holding at least
// csc_layout(nnz).total bytes (256-byte aligned).
cogdl_status csc_run(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *rowptr,
                     const int32_t *col, const float *val, int32_t *colptr, int32_t *row_t,
                     float *val_t, int32_t *perm, char *ws, hipStream_t stream)
{
    const CscLayout L = csc_layout(nnz);
    if (nnz == 0) {
        COGDL_HIP_TRY(fill_i32(colptr, (int64_t)n_cols + 1, 0, stream));
        return COGDL_OK;
    }
    uint32_t *row_of = reinterpret_cast<uint32_t *>(ws + L.row_of);
    uint32_t *ping_k = reinterpret_cast<uint32_t *>(ws + L.ping_k);
    uint32_t *ping_v = reinterpret_cast<uint32_t *>(ws + L.ping_v);
    uint32_t *skeys = reinterpret_cast<uint32_t *>(ws + L.skeys);

    const int64_t waves = (nnz + kExpandSpan - 1) / kExpandSpan;
    if (!perm)
        COGDL_LAUNCH("csc_expand_rows", k_expand_rows,
                     (unsigned)((waves + kBlock / kWave - 1) / (kBlock / kWave)), kBlock, stream,
                     rowptr, n_rows, nnz, row_of);
    const int bits = bits_for((uint64_t)(n_cols - 1));
    RadixPayload vals;
    if (val) {
        vals.in = reinterpret_cast<const uint32_t *>(val);
        vals.out = reinterpret_cast<uint32_t *>(val_t);
        vals.ping = reinterpret_cast<uint32_t *>(ws + L.ping_w);
    }
    if (perm) {
        // edge ids as the sorted values, rows (found from rowptr by the first
        // pass) and edge values as payloads
        RadixPayload rows{nullptr, reinterpret_cast<uint32_t *>(row_t),
                          reinterpret_cast<uint32_t *>(ws + L.ping_r), rowptr, n_rows};
        COGDL_HIP_TRY(radix_sort_pairs(reinterpret_cast<const uint32_t *>(col), nullptr, skeys,
                                       reinterpret_cast<uint32_t *>(perm), nnz, bits, ping_k, ping_v,
                                       ws + L.radix, stream, rows, vals));
    } else {
        // no edge ids wanted: the rows are the sorted values, one array less per pass
        COGDL_HIP_TRY(radix_sort_pairs(reinterpret_cast<const uint32_t *>(col), row_of, skeys,
                                       reinterpret_cast<uint32_t *>(row_t), nnz, bits, ping_k, ping_v,
                                       ws + L.radix, stream, vals, RadixPayload{}));
    }
    COGDL_LAUNCH("csc_colptr", k_colptr, (unsigned)((nnz + 4 * kBlock - 1) / (4 * kBlock)), kBlock,
                 stream, skeys, nnz, n_cols, colptr);
    return COGDL_OK;
}

}  // namespace
}  // namespace cogdl

using namespace cogdl;

extern "C" {

cogdl_status cogdl_csr_to_csc_workspace(int32_t n_rows, int32_t n_cols, int64_t nnz, size_t *bytes)
{
    if (!bytes || n_rows < 0 || n_cols < 0 || nnz < 0) return COGDL_ERR_INVALID;
    if (nnz > COGDL_MAX_NNZ) return COGDL_ERR_TOO_LARGE;
    *bytes = csc_layout(nnz).total;
    return COGDL_OK;
}

cogdl_status cogdl_csr_to_csc(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *rowptr,
                              const int32_t *col, const float *val, int32_t *colptr,
                              int32_t *row_t, float *val_t, int32_t *perm, void *workspace,
                              size_t workspace_bytes, hipStream_t stream)
{
    const cogdl_status st = csc_check(n_rows, n_cols, nnz, rowptr, col, val, colptr, row_t, val_t);
    if (st != COGDL_OK) return st;
    if (nnz > 0 && (!workspace || workspace_bytes < csc_layout(nnz).total ||
                    (uintptr_t)workspace % 256 != 0))
        return COGDL_ERR_INVALID;
    return csc_run(n_rows, n_cols, nnz, rowptr, col, val, colptr, row_t, val_t, perm,
                   static_cast<char *>(workspace), stream);
}

cogdl_status cogdl_csr_to_csc_noalloc(int32_t n_rows, int32_t n_cols, int64_t nnz,
                                      const int32_t *rowptr, const int32_t *col, const float *val,
                                      int32_t *colptr, int32_t *row_t, float *val_t, int32_t *perm,
                                      hipStream_t stream)
{
    const cogdl_status st = csc_check(n_rows, n_cols, nnz, rowptr, col, val, colptr, row_t, val_t);
    if (st != COGDL_OK) return st;
    if (csc_layout(nnz).total > (size_t)COGDL_NOALLOC_SCRATCH_BYTES) return COGDL_ERR_TOO_LARGE;
    void *ws = nullptr;
    if (nnz > 0) {
        const cogdl_status sp = device_scratch(&ws);
        if (sp != COGDL_OK) return sp;
    }
    return csc_run(n_rows, n_cols, nnz, rowptr, col, val, colptr, row_t, val_t, perm,
                   static_cast<char *>(ws), stream);
}

}  // extern "C"
