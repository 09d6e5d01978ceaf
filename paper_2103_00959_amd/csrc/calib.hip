// Kernels of known memory traffic (see cogdl_calib.h): the yardsticks that
// turn the L2-to-fabric byte counters into calibrated HBM bytes.  Each kernel
// touches exactly the bytes its arguments name, with 16-byte accesses, and
// writes almost nothing it does not have to.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "cogdl_calib.h"

namespace {

constexpr int kBlock = 256;
constexpr int kSinkBlocks = 4096;

__device__ __forceinline__ uint32_t fold(uint4 v) { return v.x ^ v.y ^ v.z ^ v.w; }

__global__ __launch_bounds__(kBlock) void k_calib_read(const uint4 *__restrict__ src, int64_t n16,
                                                       uint32_t *__restrict__ sink)
{
    uint32_t acc = 0;
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n16; i += (int64_t)gridDim.x * kBlock)
        acc ^= fold(src[i]);
    __shared__ uint32_t part[kBlock];
    part[threadIdx.x] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t t = 0;
        for (int j = 0; j < kBlock; ++j) t ^= part[j];
        sink[blockIdx.x] = t;
    }
}

__global__ __launch_bounds__(kBlock) void k_calib_copy(const uint4 *__restrict__ src, uint4 *__restrict__ dst,
                                                       int64_t n16)
{
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n16; i += (int64_t)gridDim.x * kBlock)
        dst[i] = src[i];
}

// L lanes per row (L = row_bytes / 16): each lane loads one 16-byte piece, the
// row's pieces are folded across its L adjacent lanes, and the row's first
// lane writes the checksum.
template <int L>
__global__ __launch_bounds__(kBlock) void k_calib_gather(const unsigned char *__restrict__ table,
                                                         int64_t stride, const int32_t *__restrict__ idx,
                                                         int64_t n, uint32_t *__restrict__ out)
{
    const int sub = threadIdx.x % L;
    const int64_t rows_per_step = (int64_t)gridDim.x * (kBlock / L);
    for (int64_t i = (int64_t)blockIdx.x * (kBlock / L) + threadIdx.x / L; i < n; i += rows_per_step) {
        const int64_t r = idx[i];
        uint32_t v = fold(*reinterpret_cast<const uint4 *>(table + r * stride + 16 * sub));
        for (int off = 1; off < L; off <<= 1) v ^= __shfl_xor(v, off);
        if (sub == 0) out[i] = v;
    }
}

unsigned grid_for(int64_t items, int per_block)
{
    int64_t b = (items + per_block - 1) / per_block;
    if (b > kSinkBlocks) b = kSinkBlocks;
    return (unsigned)(b < 1 ? 1 : b);
}

}  // namespace

extern "C" {

int cogdl_calib_read(const void *src, int64_t bytes, uint32_t *sink, hipStream_t stream)
{
    if (!src || !sink || bytes <= 0 || bytes % 16 != 0 || (uintptr_t)src % 16 != 0) return 1;
    const int64_t n16 = bytes / 16;
    k_calib_read<<<grid_for(n16, kBlock * 16), kBlock, 0, stream>>>(static_cast<const uint4 *>(src), n16,
                                                                     sink);
    return hipGetLastError() == hipSuccess ? 0 : 5;
}

int cogdl_calib_copy(const void *src, void *dst, int64_t bytes, hipStream_t stream)
{
    if (!src || !dst || bytes <= 0 || bytes % 16 != 0 || (uintptr_t)src % 16 != 0 ||
        (uintptr_t)dst % 16 != 0)
        return 1;
    const int64_t n16 = bytes / 16;
    k_calib_copy<<<grid_for(n16, kBlock * 16), kBlock, 0, stream>>>(static_cast<const uint4 *>(src),
                                                                     static_cast<uint4 *>(dst), n16);
    return hipGetLastError() == hipSuccess ? 0 : 5;
}

int cogdl_calib_gather(const void *table, int64_t stride, int32_t row_bytes, const int32_t *idx,
                       int64_t n, uint32_t *out, hipStream_t stream)
{
    if (!table || !idx || !out || n <= 0 ||
        (row_bytes != 16 && row_bytes != 32 && row_bytes != 64 && row_bytes != 128) || stride < row_bytes ||
        stride % 128 != 0 || (uintptr_t)table % 128 != 0)
        return 1;
    const unsigned char *t = static_cast<const unsigned char *>(table);
    const int L = row_bytes / 16;
    const unsigned g = grid_for(n, (kBlock / L) * 8);
    if (L == 1) k_calib_gather<1><<<g, kBlock, 0, stream>>>(t, stride, idx, n, out);
    else if (L == 2) k_calib_gather<2><<<g, kBlock, 0, stream>>>(t, stride, idx, n, out);
    else if (L == 4) k_calib_gather<4><<<g, kBlock, 0, stream>>>(t, stride, idx, n, out);
    else k_calib_gather<8><<<g, kBlock, 0, stream>>>(t, stride, idx, n, out);
    return hipGetLastError() == hipSuccess ? 0 : 5;
}

}  // extern "C"
