// Dense parts of the 2-layer GCN and GAT models around the sparse operators:
// the feature transform Y = act(X W^T + b) of every layer, on the matrix
// cores, and the per-head attention scores of a GAT layer.
//
// cogdl_linear: a workgroup of four wavefronts owns 128 rows of X and
// 32 * NT output columns; each wavefront accumulates a 32-row block with
// v_mfma_f32_32x32x16_{bf16,f16} (A = 32 rows x 16 k of X, B = 16 k x 32
// columns of W^T), fp32 accumulators in registers, and the bias and the
// activation are applied before the single store.  Operand fragments are read
// straight from memory (8 consecutive 16-bit values per lane, one 16-byte load,
// unaligned when the width k is even but not a multiple of 8, element loads
// for the partial last k-step): the layers are tall and skinny (k, m at most a
// few hundred, n in the millions), so X is streamed once per column block and
// W stays in the caches.
//
// cogdl_head_scores: a wavefront per node, lanes over the features of one
// head, a butterfly for each head's two dot products.
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

// MODE 0: rows 16-byte aligned (k % 8 == 0); 1: rows 4-byte aligned (k even);
// 2: element loads only.  Full 16-k steps use one 16-byte load per operand
// fragment in modes 0 and 1; the partial last step (and mode 2) load elements.
template <typename T, typename TY, int NT, int MODE>
__global__ __launch_bounds__(kBlock) void k_linear(LinearArgs a)
{
    const int lane = lane_id();
    const int wave = threadIdx.x / kWave;
    const int i = lane & 31;          // row of the A fragment, column of the B fragment
    const int kq = (lane >> 5) * 8;   // this lane's first k within a 16-k step
    const int64_t r0 = (int64_t)blockIdx.x * kRowsPerBlock + 32 * wave;
    const int c0 = blockIdx.y * 32 * NT;
    const T *__restrict__ X = static_cast<const T *>(a.X);
    const T *__restrict__ W = static_cast<const T *>(a.W);
    const int64_t xr = r0 + i;
    const bool x_ok = xr < a.n;
    f32x16 acc[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[t][r] = 0.f;
    const int k_full = MODE == 2 ? 0 : a.k / 16 * 16;
    for (int k0 = 0; k0 < k_full; k0 += 16) {
        const int kk = k0 + kq;
        const uint4 af = load8_full<T, MODE == 0>(X, xr * a.k + kk, x_ok);
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const int c = c0 + 32 * t + i;
            const uint4 bf = load8_full<T, MODE == 0>(W, (int64_t)c * a.k + kk, c < a.m);
            acc[t] = mfma_32x32x16<T>(af, bf, acc[t]);
        }
    }
    for (int k0 = k_full; k0 < a.k; k0 += 16) {
        const int kk = k0 + kq;
        const uint4 af = load8_tail<T>(X, xr * a.k, kk, a.k, x_ok);
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const int c = c0 + 32 * t + i;
            const uint4 bf = load8_tail<T>(W, (int64_t)c * a.k, kk, a.k, c < a.m);
            acc[t] = mfma_32x32x16<T>(af, bf, acc[t]);
        }
    }
    // C fragment: register r of lane l holds row 8 (r / 4) + 4 (l / 32) + r % 4,
    // column l % 32 of the wavefront's 32 x 32 block.
    TY *__restrict__ Y = static_cast<TY *>(a.Y);
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

using LinearKernel = void (*)(LinearArgs);

template <typename T, typename TY>
LinearKernel pick_linear_v(int mode)
{
    if (mode == 0) return k_linear<T, TY, 4, 0>;
    if (mode == 1) return k_linear<T, TY, 4, 1>;
    return k_linear<T, TY, 4, 2>;
}

template <typename T>
LinearKernel pick_linear_y(int ydt, int mode)
{
    if (ydt == COGDL_F32) return pick_linear_v<T, float>(mode);
    if (ydt == COGDL_BF16) return pick_linear_v<T, bf16_t>(mode);
    return pick_linear_v<T, f16_t>(mode);
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
    LinearKernel kern = dtype == COGDL_BF16 ? pick_linear_y<bf16_t>((int)y_dtype, mode)
                                            : pick_linear_y<f16_t>((int)y_dtype, mode);
    const dim3 grid((unsigned)row_blocks, (unsigned)((m + 127) / 128));
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
    int64_t blocks = (n + (kBlock / kWave) - 1) / (kBlock / kWave);
    if (blocks > 8192) blocks = 8192;
    const unsigned b = (unsigned)blocks;
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
