// Device helpers shared by the gfx950 kernels: feature formats, vector loads
// and stores, wave64 lane exchange.  Every kernel runs with 64-lane
// wavefronts; sub-groups of S lanes (S a power of two <= 64) are aligned
// inside a wavefront.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "cogdl.h"

namespace cogdl {

constexpr int kWave = 64;

// ----------------------------------------------------------------- formats

struct bf16_t { uint16_t bits; };
struct f16_t { uint16_t bits; };

template <typename T> struct Fmt;
template <> struct Fmt<float> { static constexpr int bytes = 4; static constexpr cogdl_dtype code = COGDL_F32; };
template <> struct Fmt<bf16_t> { static constexpr int bytes = 2; static constexpr cogdl_dtype code = COGDL_BF16; };
template <> struct Fmt<f16_t> { static constexpr int bytes = 2; static constexpr cogdl_dtype code = COGDL_F16; };

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 -> bf16, round to nearest even; NaN stays a quiet NaN.
__device__ __forceinline__ uint32_t f32_to_bf16(float f)
{
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
}

__device__ __forceinline__ float f16_bits_to_f32(uint32_t h)
{
    _Float16 v;
    uint16_t b = (uint16_t)h;
    __builtin_memcpy(&v, &b, 2);
    return (float)v;
}

// fp32 -> fp16 with the hardware conversion (round to nearest even).
__device__ __forceinline__ uint32_t f32_to_f16(float f)
{
    _Float16 v = (_Float16)f;
    uint16_t b;
    __builtin_memcpy(&b, &v, 2);
    return b;
}

// Load VEC consecutive elements (VEC * bytes is 4, 8 or 16, or VEC == 1)
// starting at element index `idx` and widen them to fp32.
template <typename T, int VEC>
__device__ __forceinline__ void load_vec(const T *__restrict__ base, int64_t idx, float (&out)[VEC]);

template <>
__device__ __forceinline__ void load_vec<float, 4>(const float *__restrict__ p, int64_t i, float (&o)[4])
{
    float4 v = *reinterpret_cast<const float4 *>(p + i);
    o[0] = v.x; o[1] = v.y; o[2] = v.z; o[3] = v.w;
}
template <>
__device__ __forceinline__ void load_vec<float, 1>(const float *__restrict__ p, int64_t i, float (&o)[1])
{
    o[0] = p[i];
}
template <>
__device__ __forceinline__ void load_vec<bf16_t, 8>(const bf16_t *__restrict__ p, int64_t i, float (&o)[8])
{
    uint4 v = *reinterpret_cast<const uint4 *>(p + i);
    o[0] = bf16_lo(v.x); o[1] = bf16_hi(v.x); o[2] = bf16_lo(v.y); o[3] = bf16_hi(v.y);
    o[4] = bf16_lo(v.z); o[5] = bf16_hi(v.z); o[6] = bf16_lo(v.w); o[7] = bf16_hi(v.w);
}
template <>
__device__ __forceinline__ void load_vec<bf16_t, 1>(const bf16_t *__restrict__ p, int64_t i, float (&o)[1])
{
    o[0] = __uint_as_float((uint32_t)p[i].bits << 16);
}
template <>
__device__ __forceinline__ void load_vec<f16_t, 8>(const f16_t *__restrict__ p, int64_t i, float (&o)[8])
{
    uint4 v = *reinterpret_cast<const uint4 *>(p + i);
    uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        o[2 * j] = f16_bits_to_f32(w[j] & 0xffffu);
        o[2 * j + 1] = f16_bits_to_f32(w[j] >> 16);
    }
}
template <>
__device__ __forceinline__ void load_vec<f16_t, 1>(const f16_t *__restrict__ p, int64_t i, float (&o)[1])
{
    o[0] = f16_bits_to_f32(p[i].bits);
}

// Store VEC fp32 values as T (rounded to nearest even for narrow T).
template <typename T, int N>
__device__ __forceinline__ void store_vec(T *__restrict__ base, int64_t idx, const float (&v)[N]);

template <>
__device__ __forceinline__ void store_vec<float, 4>(float *__restrict__ p, int64_t i, const float (&v)[4])
{
    *reinterpret_cast<float4 *>(p + i) = make_float4(v[0], v[1], v[2], v[3]);
}
template <>
__device__ __forceinline__ void store_vec<float, 8>(float *__restrict__ p, int64_t i, const float (&v)[8])
{
    *reinterpret_cast<float4 *>(p + i) = make_float4(v[0], v[1], v[2], v[3]);
    *reinterpret_cast<float4 *>(p + i + 4) = make_float4(v[4], v[5], v[6], v[7]);
}
template <>
__device__ __forceinline__ void store_vec<float, 1>(float *__restrict__ p, int64_t i, const float (&v)[1])
{
    p[i] = v[0];
}
template <>
__device__ __forceinline__ void store_vec<bf16_t, 8>(bf16_t *__restrict__ p, int64_t i, const float (&v)[8])
{
    uint4 w;
    w.x = f32_to_bf16(v[0]) | (f32_to_bf16(v[1]) << 16);
    w.y = f32_to_bf16(v[2]) | (f32_to_bf16(v[3]) << 16);
    w.z = f32_to_bf16(v[4]) | (f32_to_bf16(v[5]) << 16);
    w.w = f32_to_bf16(v[6]) | (f32_to_bf16(v[7]) << 16);
    *reinterpret_cast<uint4 *>(p + i) = w;
}
template <>
__device__ __forceinline__ void store_vec<bf16_t, 4>(bf16_t *__restrict__ p, int64_t i, const float (&v)[4])
{
    uint2 w;
    w.x = f32_to_bf16(v[0]) | (f32_to_bf16(v[1]) << 16);
    w.y = f32_to_bf16(v[2]) | (f32_to_bf16(v[3]) << 16);
    *reinterpret_cast<uint2 *>(p + i) = w;
}
template <>
__device__ __forceinline__ void store_vec<bf16_t, 1>(bf16_t *__restrict__ p, int64_t i, const float (&v)[1])
{
    p[i].bits = (uint16_t)f32_to_bf16(v[0]);
}
template <>
__device__ __forceinline__ void store_vec<f16_t, 8>(f16_t *__restrict__ p, int64_t i, const float (&v)[8])
{
    uint4 w;
    w.x = f32_to_f16(v[0]) | (f32_to_f16(v[1]) << 16);
    w.y = f32_to_f16(v[2]) | (f32_to_f16(v[3]) << 16);
    w.z = f32_to_f16(v[4]) | (f32_to_f16(v[5]) << 16);
    w.w = f32_to_f16(v[6]) | (f32_to_f16(v[7]) << 16);
    *reinterpret_cast<uint4 *>(p + i) = w;
}
template <>
__device__ __forceinline__ void store_vec<f16_t, 4>(f16_t *__restrict__ p, int64_t i, const float (&v)[4])
{
    uint2 w;
    w.x = f32_to_f16(v[0]) | (f32_to_f16(v[1]) << 16);
    w.y = f32_to_f16(v[2]) | (f32_to_f16(v[3]) << 16);
    *reinterpret_cast<uint2 *>(p + i) = w;
}
template <>
__device__ __forceinline__ void store_vec<f16_t, 1>(f16_t *__restrict__ p, int64_t i, const float (&v)[1])
{
    p[i].bits = (uint16_t)f32_to_f16(v[0]);
}

// Store VEC values where the output may be wider than the input vector
// (fp32 output of a 16-bit input uses two 16-byte stores per 8 values).
template <typename T, int VEC>
__device__ __forceinline__ void store_out(T *__restrict__ p, int64_t i, const float (&v)[VEC])
{
    store_vec<T, VEC>(p, i, v);
}

// ------------------------------------------------------------ row gathers

// Raw buffer descriptor word 3 for gfx9-family (CDNA) buffers: 32-bit data,
// no swizzle, raw (stride 0) addressing.
constexpr int kBufferWord3 = 0x00020000;
// Largest buffer the 32-bit offsets of the buffer gathers address.
constexpr uint64_t kBufferMaxBytes = 0xffffff00ull;

template <typename T, int VEC> struct VecBytes { static constexpr int value = (int)sizeof(T) * VEC; };

// Gathers VEC consecutive feature elements of one row of X.
//   BUF = true : raw buffer loads with 32-bit byte offsets (X smaller than
//                4 GiB); a masked lane passes an offset past the end of the
//                buffer and reads zeros without touching memory, so no branch.
//   BUF = false: 64-bit addresses; a masked lane reads element 0 and discards.
template <typename TX, int VEC, bool BUF>
struct RowGather {
    __amdgpu_buffer_rsrc_t rsrc;
    const TX *base;
    uint32_t oob;

    __device__ __forceinline__ RowGather(const void *x, uint64_t bytes)
    {
        base = static_cast<const TX *>(x);
        oob = (uint32_t)(bytes > 0xffffffffull ? 0xffffffffull : bytes);
        if constexpr (BUF)
            rsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(x), (short)0, (int)oob,
                                                     kBufferWord3);
    }

    // Elements [idx, idx + VEC) widened to fp32; zeros when !ok.
    __device__ __forceinline__ void load(int64_t idx, bool ok, float (&o)[VEC]) const
    {
        if constexpr (BUF) {
            const uint32_t off = ok ? (uint32_t)idx * (uint32_t)sizeof(TX) : oob;
            if constexpr (VecBytes<TX, VEC>::value == 16) {
                const auto w = __builtin_amdgcn_raw_buffer_load_b128(rsrc, (int)off, 0, 0);
                unpack16(w[0], w[1], w[2], w[3], o);
            } else if constexpr (sizeof(TX) == 4) {
                o[0] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rsrc, (int)off, 0, 0));
            } else {
                const uint32_t h = __builtin_amdgcn_raw_buffer_load_b16(rsrc, (int)off, 0, 0);
                o[0] = widen1(h);
            }
        } else {
            const int64_t i = ok ? idx : 0;
            load_vec<TX, VEC>(base, i, o);
            if (!ok) {
#pragma unroll
                for (int e = 0; e < VEC; ++e) o[e] = 0.f;
            }
        }
    }

    // The 16 raw bytes of elements [idx, idx + VEC) of a 16-byte vector
    // (packed pairs for 16-bit formats); zeros when !ok.
    __device__ __forceinline__ uint4 load_raw16(int64_t idx, bool ok) const
    {
        static_assert(VecBytes<TX, VEC>::value == 16, "16-byte vectors only");
        if constexpr (BUF) {
            const uint32_t off = ok ? (uint32_t)idx * (uint32_t)sizeof(TX) : oob;
            const auto w = __builtin_amdgcn_raw_buffer_load_b128(rsrc, (int)off, 0, 0);
            return make_uint4(w[0], w[1], w[2], w[3]);
        } else {
            const uint4 v = *reinterpret_cast<const uint4 *>(base + (ok ? idx : 0));
            return ok ? v : make_uint4(0u, 0u, 0u, 0u);
        }
    }

    // widening of raw words, for callers that keep rows packed
    __device__ __forceinline__ static float widen1(uint32_t h)
    {
        if constexpr (Fmt<TX>::code == COGDL_BF16) return __uint_as_float(h << 16);
        else return f16_bits_to_f32(h & 0xffffu);
    }
    __device__ __forceinline__ static void unpack16(uint32_t a, uint32_t b, uint32_t c, uint32_t d,
                                                    float (&o)[VEC])
    {
        const uint32_t w[4] = {a, b, c, d};
        if constexpr (sizeof(TX) == 4) {
#pragma unroll
            for (int j = 0; j < 4; ++j) o[j] = __uint_as_float(w[j]);
        } else if constexpr (Fmt<TX>::code == COGDL_BF16) {
#pragma unroll
            for (int j = 0; j < 4; ++j) { o[2 * j] = bf16_lo(w[j]); o[2 * j + 1] = bf16_hi(w[j]); }
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                o[2 * j] = f16_bits_to_f32(w[j] & 0xffffu);
                o[2 * j + 1] = f16_bits_to_f32(w[j] >> 16);
            }
        }
    }
};

// c + a.lo * b.lo + a.hi * b.hi for two packed 16-bit pairs (the gfx950 dot2
// instructions, fp32 accumulation).
template <typename T>
__device__ __forceinline__ float dot2_acc(uint32_t a, uint32_t b, float c)
{
    if constexpr (Fmt<T>::code == COGDL_BF16) {
        typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
        return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                               __builtin_bit_cast(bf16x2_t, b), c, false);
    } else {
        typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
        return __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2_t, a), __builtin_bit_cast(f16x2_t, b),
                                      c, false);
    }
}

// ------------------------------------------------------------ lane exchange

__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & (kWave - 1)); }

// Value of `v` held by lane `src` (0..63) of the calling wavefront.
__device__ __forceinline__ int lane_bcast(int v, int src)
{
    return __builtin_amdgcn_ds_bpermute(src << 2, v);
}
__device__ __forceinline__ float lane_bcast(float v, int src)
{
    return __int_as_float(__builtin_amdgcn_ds_bpermute(src << 2, __float_as_int(v)));
}

__device__ __forceinline__ float lane_xor(float v, int mask)
{
    return __int_as_float(__builtin_amdgcn_ds_bpermute((lane_id() ^ mask) << 2, __float_as_int(v)));
}

// Butterfly reductions over the G adjacent lanes of a group (G a power of two
// up to 64, groups aligned to G): every lane ends with its group's reduction,
// and partners pair up exactly as in a lane ^ 1, ^ 2, ..., ^ G/2 butterfly.
// Levels 1 and 2 are DPP quad permutes (lane ^ 1, lane ^ 2); levels 4 and 8 the
// DPP mirrors within 8 and 16 lanes (lane 7 - i, 15 - i), which once the lower
// levels have made each half of the span uniform hold the same value as lane
// ^ 4 / lane ^ 8; level 16 a swizzle (lane ^ 16 inside 32 lanes); level 32
// ds_bpermute.  DPP moves do not go through the LDS crossbar, so a reduction
// costs a few cycles per level instead of an LDS round trip.  Every lane of a
// group must be active.
template <int OFF>
__device__ __forceinline__ int bfly_partner(int v)
{
    if constexpr (OFF == 1) return __builtin_amdgcn_update_dpp(v, v, 0xB1, 0xF, 0xF, false);
    else if constexpr (OFF == 2) return __builtin_amdgcn_update_dpp(v, v, 0x4E, 0xF, 0xF, false);
    else if constexpr (OFF == 4) return __builtin_amdgcn_update_dpp(v, v, 0x141, 0xF, 0xF, false);
    else if constexpr (OFF == 8) return __builtin_amdgcn_update_dpp(v, v, 0x140, 0xF, 0xF, false);
    else if constexpr (OFF == 16) return __builtin_amdgcn_ds_swizzle(v, 0x401F);
    else return __builtin_amdgcn_ds_bpermute((lane_id() ^ OFF) << 2, v);
}

template <int OFF>
__device__ __forceinline__ float bfly_partner(float v)
{
    return __int_as_float(bfly_partner<OFF>(__float_as_int(v)));
}

template <int OFF>
__device__ __forceinline__ uint32_t bfly_partner(uint32_t v)
{
    return (uint32_t)bfly_partner<OFF>((int)v);
}

// Reduce v over groups of G lanes (G uniform across the wavefront) with op.
template <typename T, typename Op>
__device__ __forceinline__ T group_reduce(T v, int G, Op op)
{
    if (G > 1) v = op(v, bfly_partner<1>(v));
    if (G > 2) v = op(v, bfly_partner<2>(v));
    if (G > 4) v = op(v, bfly_partner<4>(v));
    if (G > 8) v = op(v, bfly_partner<8>(v));
    if (G > 16) v = op(v, bfly_partner<16>(v));
    if (G > 32) v = op(v, bfly_partner<32>(v));
    return v;
}

__device__ __forceinline__ float group_sum(float v, int G)
{
    return group_reduce(v, G, [](float a, float b) { return a + b; });
}

__device__ __forceinline__ int ceil_div(int a, int b) { return (a + b - 1) / b; }

// Rows of CSR edges, resolved by one wavefront (all 64 lanes, uniform control
// flow) for edges handed over in increasing order.  start(e0) finds the row
// holding edge e0 by a 64-way search of rowptr (each round narrows the
// candidate rows 64-fold); the cursor then keeps a window of 64 consecutive
// row ends, one per lane, and the row of edge e is the window's first row plus
// the number of window rows ending at or before e (a binary search across the
// lanes).  Empty rows need no care: the search keeps the last row starting at
// or before the edge, and the window just moves on.
struct RowCursor {
    const int32_t *rowptr;
    int64_t n_rows;
    int64_t r0;   // first row of the window
    int rend;     // end of row r0 + lane (INT32_MAX past the last row)

    // The row holding edge e0: the largest r < n with rp[r] <= e0.
    __device__ __forceinline__ static int64_t find(const int32_t *rp, int64_t n, int64_t e0)
    {
        const int lane = lane_id();
        int64_t lo = 0, hi = n;   // rp[lo] <= e0, answer in [lo, hi)
        while (hi - lo > 1) {
            const int64_t step = (hi - lo + kWave - 1) / kWave;
            const int64_t p = lo + (int64_t)lane * step;
            const uint64_t b = __ballot(p < hi && rp[p] <= e0);   // a prefix of the lanes
            const int top = 63 - __clzll(b);                       // lane 0 always holds
            lo += (int64_t)top * step;
            hi = lo + step < hi ? lo + step : hi;
        }
        return lo;
    }

    // Window at row r (which must hold the first edge handed over).
    __device__ __forceinline__ void start_at(const int32_t *rp, int64_t n, int64_t r)
    {
        rowptr = rp;
        n_rows = n;
        r0 = r;
        const int lane = lane_id();
        rend = r0 + lane < n ? rp[r0 + lane + 1] : INT32_MAX;
    }

    __device__ __forceinline__ void start(const int32_t *rp, int64_t n, int64_t e0)
    {
        start_at(rp, n, find(rp, n, e0));
    }

    // row[j] of edge e[j] for the lanes with want[j]; every e[j] must be at or
    // after the edges of earlier calls (the window only moves forward).  The NE
    // lane searches are independent and interleave.
    template <int NE>
    __device__ __forceinline__ void resolve(const int64_t (&e)[NE], const bool (&want)[NE],
                                            int64_t (&row)[NE])
    {
        const int lane = lane_id();
        bool done[NE];
#pragma unroll
        for (int j = 0; j < NE; ++j) {
            done[j] = !want[j];
            row[j] = 0;
        }
        for (;;) {
            int k[NE];
#pragma unroll
            for (int j = 0; j < NE; ++j) k[j] = 0;
#pragma unroll
            for (int b = kWave / 2; b > 0; b >>= 1)
#pragma unroll
                for (int j = 0; j < NE; ++j) {
                    const int probe = __shfl(rend, k[j] + b - 1);
                    if ((int64_t)probe <= e[j]) k[j] += b;
                }
            const int last_end = __shfl(rend, kWave - 1);
            bool left = false;
#pragma unroll
            for (int j = 0; j < NE; ++j) {
                if (!done[j] && e[j] < (int64_t)last_end) {
                    row[j] = r0 + k[j];
                    done[j] = true;
                }
                left = left || !done[j];
            }
            if (__ballot(left) == 0) break;
            r0 += kWave;
            rend = r0 + lane < n_rows ? rowptr[r0 + lane + 1] : INT32_MAX;
        }
    }
};

// Merge two online-softmax states (m, z): the pair describing
// z * exp(m) = sum exp(e).  An empty state is (-inf, 0).
__device__ __forceinline__ void softmax_merge(float &m, float &z, float m2, float z2)
{
    float mn = fmaxf(m, m2);
    if (mn == -INFINITY) return;
    z = z * __expf(m - mn) + z2 * __expf(m2 - mn);
    m = mn;
}

__device__ __forceinline__ float leaky_relu(float t, float slope) { return t > 0.f ? t : slope * t; }

// An attention weight for storing, alpha = exp(e - m) * rz, with e the fp32
// score of the edge (as the softmax loops compute it), m the row's maximum of
// those scores and rz = 1 / z its normalizer.  The fast exponential of the
// loops evaluates exp on the rounded product (e - m) * log2(e), whose rounding
// error grows with |e - m|; here e - m and the product are carried as
// unevaluated pairs (hi, lo) of fp32 values (the two-sum and fma error terms,
// Knuth / Dekker), so only the hardware exp2 of the high part (v_exp_f32) and
// the final roundings err:
//     exp(x_hi + x_lo) = 2^y_hi * (1 + y_lo ln 2 + x_lo),  y = x_hi log2(e).
// A row's maximal score gives exactly exp(0) = 1 (so a degree-1 row's weight
// is exactly 1).
__device__ __forceinline__ float alpha_value(float e, float m, float rz)
{
    constexpr float kLog2e = 1.44269502f;        // log2(e) rounded to fp32
    constexpr float kLog2eLo = 1.92596299e-8f;   // log2(e) - kLog2e
    constexpr float kLn2 = 0.693147182f;
    const float x = e - m;
    const float c = x - e;
    const float x_lo = (e - (x - c)) + (-m - c);
    const float y = x * kLog2e;
    const float y_lo = fmaf(x, kLog2e, -y) + x * kLog2eLo;
    const float r = __builtin_amdgcn_exp2f(y);
    const float corr = fmaf(y_lo, kLn2, x_lo);
    return fmaf(r, corr, r) * rz;
}

// The epilogue activations of the layer entry points (cogdl_act codes).
__device__ __forceinline__ float apply_act(float v, int act)
{
    if (act == COGDL_ACT_RELU) return v > 0.f ? v : 0.f;
    if (act == COGDL_ACT_ELU) return v > 0.f ? v : expm1f(v);
    return v;
}

// v[e] = act(v[e] + bias[f + e]) over VEC features starting at f; nothing to
// do for a plain aggregation (no bias, no activation).
template <int VEC>
__device__ __forceinline__ void epilogue(float (&v)[VEC], const float *__restrict__ bias, int act,
                                         int64_t f)
{
    if (bias) {
#pragma unroll
        for (int e = 0; e < VEC; ++e) v[e] += bias[f + e];
    }
    if (act != COGDL_ACT_NONE) {
#pragma unroll
        for (int e = 0; e < VEC; ++e) v[e] = apply_act(v[e], act);
    }
}

// Work-unit walk of a resident grid.  Sub-group `sub` (of `per_block` in each
// workgroup) starts at unit `first` and steps by `step` while below `end`.
// Without a unit list the walk covers rows [0, n_rows).  With `lists` == 1 it
// covers units [*lo, *hi).  With `lists` > 1 the units form that many
// consecutive lists, list x being [lo[x], hi[x]), and workgroup b walks list
// b % lists together with the other workgroups of that list (the grid is a
// multiple of `lists`): workgroups are dealt to the XCDs round-robin, so every
// list runs on one XCD and its gathers share that XCD's L2.
struct UnitWalk {
    int64_t first, end, step;
};

__device__ __forceinline__ UnitWalk unit_walk(bool has_units, const int32_t *lo, const int32_t *hi,
                                              int lists, int64_t n_rows, int per_block, int sub)
{
    if (!has_units)
        return {(int64_t)blockIdx.x * per_block + sub, n_rows, (int64_t)gridDim.x * per_block};
    if (lists <= 1)
        return {(int64_t)*lo + (int64_t)blockIdx.x * per_block + sub, (int64_t)*hi,
                (int64_t)gridDim.x * per_block};
    const int x = blockIdx.x % lists;
    return {(int64_t)lo[x] + (int64_t)(blockIdx.x / lists) * per_block + sub, (int64_t)hi[x],
            (int64_t)(gridDim.x / lists) * per_block};
}

}  // namespace cogdl
