// CSR -> CSC transpose of the graph structure, the setup of the backward
// pass of Eq. 1 (the gradient with respect to the node features is A^T G).
//
// A stable LSD radix sort of the edge ids keyed by column (digits of at most
// 8 bits, as many passes as the column count needs) gives perm directly, with
// each edge's row and value bits carried along as payloads (so nothing is
// gathered at random afterwards); colptr is read off the sorted keys.  Every step is
// integer work in a fixed order, so the result is bit-for-bit unique: inside
// a column the edges keep increasing CSR edge id.
#include "common.hpp"
#include "internal.hpp"

namespace cogdl {
namespace {

constexpr int kBlock = 256;

__global__ __launch_bounds__(kBlock) void k_expand_rows(const int32_t *__restrict__ rowptr,
                                                        int32_t n_rows,
                                                        uint32_t *__restrict__ row_of)
{
    const int lane = lane_id();
    const int64_t waves = (int64_t)gridDim.x * (kBlock / kWave);
    for (int64_t i = (int64_t)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave; i < n_rows;
         i += waves) {
        const int beg = rowptr[i], end = rowptr[i + 1];
        for (int k = beg + lane; k < end; k += kWave) row_of[k] = (uint32_t)i;
    }
}

// colptr[c] = first slot whose key is >= c, from the sorted keys.
__global__ __launch_bounds__(kBlock) void k_colptr(const uint32_t *__restrict__ skeys, int64_t nnz,
                                                   int32_t n_cols, int32_t *__restrict__ colptr)
{
    for (int64_t p = (int64_t)blockIdx.x * kBlock + threadIdx.x; p < nnz;
         p += (int64_t)gridDim.x * kBlock) {
        const int64_t key = skeys[p];
        const int64_t prev = p > 0 ? (int64_t)skeys[p - 1] : -1;
        for (int64_t c = prev + 1; c <= key; ++c) colptr[c] = (int32_t)p;
        if (p == nnz - 1)
            for (int64_t c = key + 1; c <= n_cols; ++c) colptr[c] = (int32_t)nnz;
    }
}

struct CscLayout {
    size_t row_of, ping_k, ping_v, ping_r, ping_w, skeys, vtmp, radix, total;
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
    L.vtmp = off;   off += al(4 * (size_t)nnz);
    L.radix = off;  off += al(radix_workspace_bytes(nnz));
    L.total = off;
    return L;
}

unsigned grid_for(int64_t n, int per_block)
{
    int64_t b = (n + per_block - 1) / per_block;
    if (b > 16384) b = 16384;
    if (b < 1) b = 1;
    return (unsigned)b;
}

}  // namespace
}  // namespace cogdl

using namespace cogdl;

extern "C" {

cogdl_status cogdl_csr_to_csc_workspace(int32_t n_rows, int32_t n_cols, int64_t nnz, size_t *bytes)
{
    if (!bytes || n_rows < 0 || n_cols < 0 || nnz < 0) return COGDL_ERR_INVALID;
    if (nnz > INT32_MAX) return COGDL_ERR_TOO_LARGE;
    *bytes = csc_layout(nnz).total;
    return COGDL_OK;
}

cogdl_status cogdl_csr_to_csc(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *rowptr,
                              const int32_t *col, const float *val, int32_t *colptr,
                              int32_t *row_t, float *val_t, int32_t *perm, void *workspace,
                              size_t workspace_bytes, hipStream_t stream)
{
    if (n_rows < 0 || n_cols < 0 || nnz < 0) return COGDL_ERR_INVALID;
    if (nnz > INT32_MAX) return COGDL_ERR_TOO_LARGE;
    if (!colptr) return COGDL_ERR_INVALID;
    if (n_rows > 0 && !rowptr) return COGDL_ERR_INVALID;
    if (nnz > 0 && (!col || !row_t || n_rows == 0 || n_cols == 0)) return COGDL_ERR_INVALID;
    if ((val == nullptr) != (val_t == nullptr)) return COGDL_ERR_INVALID;
    const CscLayout L = csc_layout(nnz);
    if (nnz > 0 && (!workspace || workspace_bytes < L.total || (uintptr_t)workspace % 256 != 0))
        return COGDL_ERR_INVALID;
    if (nnz == 0) {
        COGDL_HIP_TRY(fill_i32(colptr, (int64_t)n_cols + 1, 0, stream));
        return COGDL_OK;
    }
    char *ws = static_cast<char *>(workspace);
    uint32_t *row_of = reinterpret_cast<uint32_t *>(ws + L.row_of);
    uint32_t *ping_k = reinterpret_cast<uint32_t *>(ws + L.ping_k);
    uint32_t *ping_v = reinterpret_cast<uint32_t *>(ws + L.ping_v);
    uint32_t *skeys = reinterpret_cast<uint32_t *>(ws + L.skeys);

    COGDL_LAUNCH("csc_expand_rows", k_expand_rows, grid_for(n_rows, kBlock / kWave), kBlock, stream,
                 rowptr, n_rows, row_of);
    const int bits = bits_for((uint64_t)(n_cols - 1));
    RadixPayload vals;
    if (val) {
        vals.in = reinterpret_cast<const uint32_t *>(val);
        vals.out = reinterpret_cast<uint32_t *>(val_t);
        vals.ping = reinterpret_cast<uint32_t *>(ws + L.ping_w);
    }
    if (perm) {
        // edge ids as the sorted values, rows and edge values as payloads
        RadixPayload rows{row_of, reinterpret_cast<uint32_t *>(row_t),
                          reinterpret_cast<uint32_t *>(ws + L.ping_r)};
        COGDL_HIP_TRY(radix_sort_pairs(reinterpret_cast<const uint32_t *>(col), nullptr, skeys,
                                       reinterpret_cast<uint32_t *>(perm), nnz, bits, ping_k, ping_v,
                                       ws + L.radix, stream, rows, vals));
    } else {
        // no edge ids wanted: the rows are the sorted values, one array less per pass
        COGDL_HIP_TRY(radix_sort_pairs(reinterpret_cast<const uint32_t *>(col), row_of, skeys,
                                       reinterpret_cast<uint32_t *>(row_t), nnz, bits, ping_k, ping_v,
                                       ws + L.radix, stream, vals, RadixPayload{}));
    }
    COGDL_LAUNCH("csc_colptr", k_colptr, grid_for(nnz, kBlock), kBlock, stream, skeys, nnz, n_cols,
                 colptr);
    return COGDL_OK;
}

}  // extern "C"
