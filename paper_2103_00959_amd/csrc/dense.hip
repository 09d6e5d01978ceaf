// Dense parts of the 2-layer GCN and GAT models around the sparse operators:
// the feature transform Y = act(X W^T + b) of every layer, on the matrix
// cores, and the per-head attention scores of a GAT layer.
//
// cogdl_linear: a workgroup of four wavefronts owns 128 rows of X and
// 32 * NT output columns; each wavefront accumulates a 32-row block with
// v_mfma_f32_32x32x16_{bf16,f16} (A = 32 rows x 16 k of X, B = 16 k x 32
// columns of W^T), fp32 accumulators in registers, and the bias and the
// activation are applied before the single store.  The layers are tall and
// skinny (k, m at most a few hundred, n in the millions): X is streamed once
// per column block through LDS in 64-k chunks, W comes from the caches.
//
// cogdl_head_scores: lanes over the features of a node's heads, a butterfly
// for each head's two dot products (several nodes per wavefront when the
// heads split into whole 16-byte vectors, else a wavefront per node).
#include "common.hpp"
#include "internal.hpp"

namespace cogdl {
namespace {

constexpr int kBlock = 256;
constexpr int kRowsPerBlock = 128;

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

// D = A B + C for a 32 x 16 A fragment and a 16 x 32 B fragment, each lane
// holding 8 consecutive k of one row of A / one column of B.
template <typename T>
__device__ __forceinline__ f32x16 mfma_32x32x16(uint4 a, uint4 b, f32x16 c)
{
    if constexpr (Fmt<T>::code == COGDL_BF16)
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                       __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a),
                                                      __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}

typedef uint32_t u32x4_a4 __attribute__((ext_vector_type(4), aligned(4)));

// Elements [i, i + 8) of a row, all inside the row, as one 16-byte load (zeros
// when !ok).  ALIGN16: the address is 16-byte aligned; else only 4-byte
// aligned (gfx950 serves unaligned vector loads).
template <typename T, bool ALIGN16>
__device__ __forceinline__ uint4 load8_full(const T *__restrict__ p, int64_t i, bool ok)
{
    if (!ok) return make_uint4(0u, 0u, 0u, 0u);
    if constexpr (ALIGN16) return *reinterpret_cast<const uint4 *>(p + i);
    else {
        const u32x4_a4 v = *reinterpret_cast<const u32x4_a4 *>(p + i);
        return make_uint4(v.x, v.y, v.z, v.w);
    }
}

// Elements [kk, kk + 8) of the row at row_base, zero past its width k or when
// !ok (element loads: the last, partial k-step of a row).
template <typename T>
__device__ __forceinline__ uint4 load8_tail(const T *__restrict__ p, int64_t row_base, int kk, int k,
                                            bool ok)
{
    uint32_t w[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const uint32_t lo = (ok && kk + 2 * j < k) ? p[row_base + kk + 2 * j].bits : 0u;
        const uint32_t hi = (ok && kk + 2 * j + 1 < k) ? p[row_base + kk + 2 * j + 1].bits : 0u;
        w[j] = lo | (hi << 16);
    }
    return make_uint4(w[0], w[1], w[2], w[3]);
}

struct LinearArgs {
    int64_t n;
    int32_t k;
    int32_t m;
    const void *X;      // n x k
    const void *W;      // m x k (a layer's out x in weights)
    const float *bias;  // m, nullable
    int32_t act;
    void *Y;            // n x m
};

// The k dimension runs in chunks of kKChunk.  For each chunk the workgroup
// stages its 128 rows of X and its 32 * NT rows of W in LDS (8 lanes per row
// read 128 contiguous bytes, so a load instruction touches 8 rows instead of
// the 32 a fragment spans), then every wavefront reads its MFMA fragments
// from LDS.  The next chunk's global loads are issued before the current
// chunk's matrix-core work, into registers, so one chunk of loads is always
// in flight.  LDS rows are padded to 144 bytes: the 16 lanes of a 16-byte LDS
// read phase then cover all 64 banks once.
// MODE 0: rows 16-byte aligned (k % 8 == 0); 1: rows 4-byte aligned (k even):
// every 8-element piece inside the row is one 16-byte load; 2: element loads.
// Pieces past the row's end (or past n rows / m columns) are zeros.
constexpr int kKChunk = 64;
constexpr int kLdsRow = kKChunk + 8;     // elements per LDS row
constexpr int kPiecesPerRow = kKChunk / 8;

template <typename T, int MODE>
__device__ __forceinline__ uint4 load_piece(const T *__restrict__ row, int kk, int k, bool ok)
{
    if (!ok || kk >= k) return make_uint4(0u, 0u, 0u, 0u);
    if (MODE != 2 && kk + 8 <= k) return load8_full<T, MODE == 0>(row, kk, true);
    return load8_tail<T>(row, 0, kk, k, true);
}

template <typename T, typename TY, int NT, int MODE>
__global__ __launch_bounds__(kBlock) void k_linear(LinearArgs a)
{
    constexpr int kBRows = 32 * NT;
    constexpr int kAPieces = kRowsPerBlock * kPiecesPerRow / kBlock;   // 4 per thread
    constexpr int kBPieces = kBRows * kPiecesPerRow / kBlock;          // NT per thread
    __shared__ uint4 sA[kRowsPerBlock][kLdsRow / 8];
    __shared__ uint4 sB[kBRows][kLdsRow / 8];
    const int tid = threadIdx.x;
    const int lane = lane_id();
    const int wave = tid / kWave;
    const int i = lane & 31;          // row of the A fragment, column of the B fragment
    const int kq = lane >> 5;         // this lane's 8-k half of a 16-k step
    const int64_t rb = (int64_t)blockIdx.x * kRowsPerBlock;
    const int c0 = blockIdx.y * kBRows;
    const T *__restrict__ X = static_cast<const T *>(a.X);
    const T *__restrict__ W = static_cast<const T *>(a.W);
    const int seg = tid % kPiecesPerRow;      // piece of its row this thread stages
    const T *__restrict__ arow[kAPieces];
    bool a_ok[kAPieces];
#pragma unroll
    for (int q = 0; q < kAPieces; ++q) {
        const int64_t r = rb + (tid + q * kBlock) / kPiecesPerRow;
        a_ok[q] = r < a.n;
        arow[q] = X + (a_ok[q] ? r : 0) * a.k;
    }
    const T *__restrict__ brow[kBPieces];
    bool b_ok[kBPieces];
#pragma unroll
    for (int q = 0; q < kBPieces; ++q) {
        const int c = c0 + (tid + q * kBlock) / kPiecesPerRow;
        b_ok[q] = c < a.m;
        brow[q] = W + (int64_t)(b_ok[q] ? c : 0) * a.k;
    }
    f32x16 acc[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[t][r] = 0.f;

    uint4 pa[kAPieces], pb[kBPieces];
    auto fetch = [&](int k0) {
        const int kk = k0 + seg * 8;
#pragma unroll
        for (int q = 0; q < kAPieces; ++q) pa[q] = load_piece<T, MODE>(arow[q], kk, a.k, a_ok[q]);
#pragma unroll
        for (int q = 0; q < kBPieces; ++q) pb[q] = load_piece<T, MODE>(brow[q], kk, a.k, b_ok[q]);
    };
    fetch(0);
    for (int k0 = 0; k0 < a.k; k0 += kKChunk) {
        __syncthreads();                       // the previous chunk's fragments are read
#pragma unroll
        for (int q = 0; q < kAPieces; ++q) sA[(tid + q * kBlock) / kPiecesPerRow][seg] = pa[q];
#pragma unroll
        for (int q = 0; q < kBPieces; ++q) sB[(tid + q * kBlock) / kPiecesPerRow][seg] = pb[q];
        __syncthreads();
        if (k0 + kKChunk < a.k) fetch(k0 + kKChunk);
        const int steps = (a.k - k0 >= kKChunk) ? kKChunk / 16 : (a.k - k0 + 15) / 16;
#pragma unroll
        for (int s = 0; s < kKChunk / 16; ++s) {
            if (s < steps) {
                const uint4 af = sA[32 * wave + i][2 * s + kq];
#pragma unroll
                for (int t = 0; t < NT; ++t)
                    acc[t] = mfma_32x32x16<T>(af, sB[32 * t + i][2 * s + kq], acc[t]);
            }
        }
    }
    // C fragment: register r of lane l holds row 8 (r / 4) + 4 (l / 32) + r % 4,
    // column l % 32 of the wavefront's 32 x 32 block.
    TY *__restrict__ Y = static_cast<TY *>(a.Y);
    const int64_t r0 = rb + 32 * wave;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int c = c0 + 32 * t + i;
        if (c >= a.m) continue;
        const float b = a.bias ? a.bias[c] : 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int64_t row = r0 + 8 * (r / 4) + 4 * (lane >> 5) + (r % 4);
            if (row >= a.n) continue;
            const float v[1] = {apply_act(acc[t][r] + b, a.act)};
            store_out<TY, 1>(Y, row * a.m + c, v);
        }
    }
}

// s_src[i, h] = sum_d Z[i, h, d] a_src[h, d] and s_dst likewise; a wavefront
// per node (grid-stride), lanes over d.
template <typename T>
__global__ __launch_bounds__(kBlock) void k_head_scores(int64_t n, int H, int D,
                                                        const T *__restrict__ Z,
                                                        const float *__restrict__ a_src,
                                                        const float *__restrict__ a_dst,
                                                        float *__restrict__ s_src,
                                                        float *__restrict__ s_dst)
{
    const int lane = lane_id();
    const int64_t waves = (int64_t)gridDim.x * (kBlock / kWave);
    const int64_t W = (int64_t)H * D;
    for (int64_t node = (int64_t)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave; node < n;
         node += waves) {
        for (int h = 0; h < H; ++h) {
            float ps = 0.f, pd = 0.f;
            for (int d = lane; d < D; d += kWave) {
                float z[1];
                load_vec<T, 1>(Z, node * W + (int64_t)h * D + d, z);
                ps = fmaf(z[0], a_src[(int64_t)h * D + d], ps);
                pd = fmaf(z[0], a_dst[(int64_t)h * D + d], pd);
            }
            ps = group_sum(ps, kWave);
            pd = group_sum(pd, kWave);
            if (lane == 0) {
                if (s_src) s_src[node * H + h] = ps;
                if (s_dst) s_dst[node * H + h] = pd;
            }
        }
    }
}

// Vector form of the same sums when every head's features split into whole
// 16-byte vectors: VEC features per lane, the L = D / VEC lanes of a head
// adjacent, the H * L lanes of a node a power-of-two group, so a wavefront
// holds 64 / (H * L) nodes; each lane keeps its VEC weights of a_src and a_dst
// in registers, and a butterfly over the head's L lanes finishes each sum.
template <typename T, int VEC>
__global__ __launch_bounds__(kBlock) void k_head_scores_vec(int64_t n, int H, int D, int log2L, int log2G,
                                                            const T *__restrict__ Z,
                                                            const float *__restrict__ a_src,
                                                            const float *__restrict__ a_dst,
                                                            float *__restrict__ s_src,
                                                            float *__restrict__ s_dst)
{
    const int lane = lane_id();
    const int p = lane & ((1 << log2G) - 1);     // vector of the node's row held by this lane
    const int h = p >> log2L;
    const int L = 1 << log2L;
    const int64_t W = (int64_t)H * D;
    const int64_t e0 = (int64_t)p * VEC;          // feature h * D + d of the row (and of a_src)
    float as[VEC], ad[VEC];
#pragma unroll
    for (int j = 0; j < VEC; ++j) {
        as[j] = s_src ? a_src[e0 + j] : 0.f;
        ad[j] = s_dst ? a_dst[e0 + j] : 0.f;
    }
    const int per_wave = kWave >> log2G;
    const int64_t step = (int64_t)gridDim.x * (kBlock / kWave) * per_wave;
    for (int64_t base = ((int64_t)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave) * per_wave; base < n;
         base += step) {
        const int64_t node = base + (lane >> log2G);
        const bool ok = node < n;
        float z[VEC];
        if (ok) load_vec<T, VEC>(Z, node * W + e0, z);
        else
#pragma unroll
            for (int j = 0; j < VEC; ++j) z[j] = 0.f;
        float ps = 0.f, pd = 0.f;
#pragma unroll
        for (int j = 0; j < VEC; ++j) {
            ps = fmaf(z[j], as[j], ps);
            pd = fmaf(z[j], ad[j], pd);
        }
        ps = group_sum(ps, L);
        pd = group_sum(pd, L);
        if (ok && (p & (L - 1)) == 0) {
            if (s_src) s_src[node * H + h] = ps;
            if (s_dst) s_dst[node * H + h] = pd;
        }
    }
}

// Grid of the head-score kernels: enough workgroups for n nodes at per_block
// nodes each, at most half as many as fit on the device at once.  Each
// wavefront loads its weights once and then strides over the nodes; on a
// 233k-node layer this ran 3x faster than one short-lived workgroup per 16
// nodes (the weight loads and wavefront start-up dominated).
unsigned score_blocks(int64_t n, int64_t per_block, const void *kernel)
{
    int64_t blocks = (n + per_block - 1) / per_block;
    const int64_t cap = resident_blocks(kernel, kBlock) / 2;
    if (blocks > cap) blocks = cap > 0 ? cap : 1;
    return (unsigned)blocks;
}

using LinearKernel = void (*)(LinearArgs);

// NT: 32-column tiles per workgroup, the fewest that cover m up to 128.
template <typename T, typename TY, int MODE>
LinearKernel pick_linear_nt(int m)
{
    if (m <= 32) return k_linear<T, TY, 1, MODE>;
    if (m <= 64) return k_linear<T, TY, 2, MODE>;
    return k_linear<T, TY, 4, MODE>;
}

template <typename T, typename TY>
LinearKernel pick_linear_v(int mode, int m)
{
    if (mode == 0) return pick_linear_nt<T, TY, 0>(m);
    if (mode == 1) return pick_linear_nt<T, TY, 1>(m);
    return pick_linear_nt<T, TY, 2>(m);
}

template <typename T>
LinearKernel pick_linear_y(int ydt, int mode, int m)
{
    if (ydt == COGDL_F32) return pick_linear_v<T, float>(mode, m);
    if (ydt == COGDL_BF16) return pick_linear_v<T, bf16_t>(mode, m);
    return pick_linear_v<T, f16_t>(mode, m);
}

}  // namespace
}  // namespace cogdl

using namespace cogdl;

extern "C" {

cogdl_status cogdl_linear(int64_t n, int32_t k, int32_t m, const void *X, const void *W,
                          cogdl_dtype dtype, const float *bias, cogdl_act act, void *Y,
                          cogdl_dtype y_dtype, hipStream_t stream)
{
    if (n < 0 || k < 0 || m < 0) return COGDL_ERR_INVALID;
    if (act < COGDL_ACT_NONE || act > COGDL_ACT_ELU) return COGDL_ERR_INVALID;
    if (dtype != COGDL_BF16 && dtype != COGDL_F16) return COGDL_ERR_DTYPE;
    if (!dtype_ok(y_dtype)) return COGDL_ERR_DTYPE;
    if (n > 0 && m > 0 && !Y) return COGDL_ERR_INVALID;
    if (n > 0 && k > 0 && !X) return COGDL_ERR_INVALID;
    if (m > 0 && k > 0 && !W) return COGDL_ERR_INVALID;
    if (n == 0 || m == 0) return COGDL_OK;
    const int64_t row_blocks = (n + kRowsPerBlock - 1) / kRowsPerBlock;
    if (row_blocks > INT32_MAX) return COGDL_ERR_TOO_LARGE;
    LinearArgs a{n, k, m, X, W, bias, (int32_t)act, Y};
    const int mode = (k % 8 == 0 && (uintptr_t)X % 16 == 0 && (uintptr_t)W % 16 == 0) ? 0
                     : (k % 2 == 0 && (uintptr_t)X % 4 == 0 && (uintptr_t)W % 4 == 0) ? 1 : 2;
    LinearKernel kern = dtype == COGDL_BF16 ? pick_linear_y<bf16_t>((int)y_dtype, mode, m)
                                            : pick_linear_y<f16_t>((int)y_dtype, mode, m);
    const int cols = m <= 32 ? 32 : m <= 64 ? 64 : 128;
    const dim3 grid((unsigned)row_blocks, (unsigned)((m + cols - 1) / cols));
    COGDL_LAUNCH("linear", kern, grid, kBlock, stream, a);
    return COGDL_OK;
}

cogdl_status cogdl_head_scores(int64_t n, int32_t H, int32_t D, const void *Z,
                               cogdl_dtype z_dtype, const float *a_src, const float *a_dst,
                               float *s_src, float *s_dst, hipStream_t stream)
{
    if (n < 0 || H < 1 || H > COGDL_MAX_HEADS || D < 1) return COGDL_ERR_INVALID;
    if (!dtype_ok(z_dtype)) return COGDL_ERR_DTYPE;
    if ((s_src && !a_src) || (s_dst && !a_dst)) return COGDL_ERR_INVALID;
    if (n > 0 && !Z) return COGDL_ERR_INVALID;
    if (n == 0 || (!s_src && !s_dst)) return COGDL_OK;
    const int vec = z_dtype == COGDL_F32 ? 4 : 8;
    const int64_t L = D / vec;
    if (D % vec == 0 && (uintptr_t)Z % 16 == 0 && (L & (L - 1)) == 0 && (H & (H - 1)) == 0 &&
        (int64_t)H * L <= kWave) {
        const int log2L = log2i((int)L), log2G = log2i((int)(H * L));
        const int64_t per_block = (kBlock / kWave) * (kWave >> log2G);
        const void *kern = z_dtype == COGDL_F32 ? (const void *)k_head_scores_vec<float, 4>
                           : z_dtype == COGDL_BF16 ? (const void *)k_head_scores_vec<bf16_t, 8>
                                                   : (const void *)k_head_scores_vec<f16_t, 8>;
        const unsigned b = score_blocks(n, per_block, kern);
        if (z_dtype == COGDL_F32)
            COGDL_LAUNCH("head_scores", (k_head_scores_vec<float, 4>), b, kBlock, stream, n, H, D, log2L,
                         log2G, static_cast<const float *>(Z), a_src, a_dst, s_src, s_dst);
        else if (z_dtype == COGDL_BF16)
            COGDL_LAUNCH("head_scores", (k_head_scores_vec<bf16_t, 8>), b, kBlock, stream, n, H, D, log2L,
                         log2G, static_cast<const bf16_t *>(Z), a_src, a_dst, s_src, s_dst);
        else
            COGDL_LAUNCH("head_scores", (k_head_scores_vec<f16_t, 8>), b, kBlock, stream, n, H, D, log2L,
                         log2G, static_cast<const f16_t *>(Z), a_src, a_dst, s_src, s_dst);
        return COGDL_OK;
    }
    const void *kern = z_dtype == COGDL_F32 ? (const void *)k_head_scores<float>
                       : z_dtype == COGDL_BF16 ? (const void *)k_head_scores<bf16_t>
                                               : (const void *)k_head_scores<f16_t>;
    const unsigned b = score_blocks(n, kBlock / kWave, kern);
    if (z_dtype == COGDL_F32)
        COGDL_LAUNCH("head_scores", k_head_scores<float>, b, kBlock, stream, n, H, D,
                     static_cast<const float *>(Z), a_src, a_dst, s_src, s_dst);
    else if (z_dtype == COGDL_BF16)
        COGDL_LAUNCH("head_scores", k_head_scores<bf16_t>, b, kBlock, stream, n, H, D,
                     static_cast<const bf16_t *>(Z), a_src, a_dst, s_src, s_dst);
    else
        COGDL_LAUNCH("head_scores", k_head_scores<f16_t>, b, kBlock, stream, n, H, D,
                     static_cast<const f16_t *>(Z), a_src, a_dst, s_src, s_dst);
    return COGDL_OK;
}

}  // extern "C"
