// Activation compression: per-group b-bit quantization with stochastic
// rounding, the technique the paper extends to GNN training to shrink the
// activations kept for the backward pass (2, 3 and 4 bits in its evaluation).
//
// Format (n x F activations, groups of G consecutive features of a row, G a
// multiple of 64, the last group of a row possibly shorter):
//   stats[2g], stats[2g + 1] = (m, r): the group minimum and its step
//     r = (M - m) / (2^b - 1)  (0 for a constant group);
//   codes: per group, G / 64 blocks of b uint64 bit planes; plane p of a
//     block holds bit p of the codes of its 64 consecutive features.
// Encoding of x (flat index e = i * F + f), all in fp32:
//   q = clamp(floor(fma(x - m, s, u)), 0, 2^b - 1),  s = (2^b - 1) / (M - m),
// u the uniform of e from Philox4x32-10 (Salmon et al., SC 2011) at counter
// (e / 4, 0, 0) and key = seed, word e mod 4, top 24 bits times 2^-24.
// Decoding: x' = fma(q, r, m), an unbiased estimate of x within one step.
//
// Mapping on gfx950.  Rows of whole groups with 16-byte aligned rows (the
// usual case, e.g. one group per 256-wide row): 8 consecutive features per
// lane in 16-byte vectors, a group on G / 8 adjacent lanes (several groups per
// wavefront), min/max by a butterfly within the group, each 64-feature block
// of codes assembled from its 8 lanes' bytes by lane exchanges.  Otherwise
// (ragged rows): a wavefront per group, one feature per lane, each block's b
// bit planes as b wavefront ballots.  Either way a group of bf16 features
// reads 2G bytes and writes G b / 8 + 8.
#include "common.hpp"
#include "internal.hpp"

namespace cogdl {
namespace {

constexpr int kBlock = 256;

// The four words of Philox4x32-10 at counter (c, 0, 0) (c = e / 4 as 64 bits)
// with key = seed.
__device__ __forceinline__ uint4 philox4(uint64_t seed, uint64_t c)
{
    uint32_t c0 = (uint32_t)c, c1 = (uint32_t)(c >> 32), c2 = 0u, c3 = 0u;
    uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
#pragma unroll
    for (int round = 0; round < 10; ++round) {
        // each 32 x 32 -> 64-bit product in one instruction (v_mad_u64_u32)
        // instead of separate high and low multiplies
        const uint64_t p0 = (uint64_t)0xD2511F53u * c0, p1 = (uint64_t)0xCD9E8D57u * c2;
        const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        const uint32_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
        c0 = n0;
        c1 = lo1;
        c2 = n2;
        c3 = lo0;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    return make_uint4(c0, c1, c2, c3);
}

__device__ __forceinline__ uint32_t philox_word(uint64_t seed, int64_t e)
{
    const uint4 r = philox4(seed, (uint64_t)e >> 2);
    const int w = (int)(e & 3);
    return w == 0 ? r.x : w == 1 ? r.y : w == 2 ? r.z : r.w;
}

__device__ __forceinline__ float uniform24(uint32_t r) { return (float)(r >> 8) * (1.0f / 16777216.0f); }

__device__ __forceinline__ float wave_min(float v)
{
    return group_reduce(v, kWave, [](float a, float b) { return fminf(a, b); });
}

__device__ __forceinline__ float wave_max(float v)
{
    return group_reduce(v, kWave, [](float a, float b) { return fmaxf(a, b); });
}

struct CodecArgs {
    int64_t n;
    int32_t F;
    int32_t bits;
    int32_t G;
    int32_t ng;       // groups per row
    uint64_t seed;
    const void *A;
    uint64_t *codes;
    float *stats;
};

template <typename TA>
__global__ __launch_bounds__(kBlock) void k_compress(CodecArgs a)
{
    const int lane = lane_id();
    const int64_t groups = a.n * a.ng;
    const int64_t waves = (int64_t)gridDim.x * (kBlock / kWave);
    const int nb = a.G / kWave;
    const float qmax = (float)((1 << a.bits) - 1);
    const TA *__restrict__ A = static_cast<const TA *>(a.A);
    for (int64_t g = (int64_t)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave; g < groups;
         g += waves) {
        const int64_t i = g / a.ng;
        const int f0 = (int)(g % a.ng) * a.G;
        const int len = a.F - f0 < a.G ? a.F - f0 : a.G;
        const int64_t base = i * a.F + f0;
        float lo = INFINITY, hi = -INFINITY;
        for (int j = lane; j < len; j += kWave) {
            float x[1];
            load_vec<TA, 1>(A, base + j, x);
            lo = fminf(lo, x[0]);
            hi = fmaxf(hi, x[0]);
        }
        const float m = wave_min(lo), M = wave_max(hi);
        const float range = M - m;
        const float s = range > 0.f ? qmax / range : 0.f;
        const float r = range > 0.f ? range / qmax : 0.f;
        if (lane == 0) {
            a.stats[2 * g] = m;
            a.stats[2 * g + 1] = r;
        }
        uint64_t *__restrict__ w = a.codes + g * (int64_t)nb * a.bits;
        for (int t = 0; t < nb; ++t) {
            const int j = t * kWave + lane;
            uint32_t q = 0;
            if (j < len) {
                float x[1];
                load_vec<TA, 1>(A, base + j, x);
                const float u = uniform24(philox_word(a.seed, base + j));
                float v = floorf(fmaf(x[0] - m, s, u));
                v = v < 0.f ? 0.f : (v > qmax ? qmax : v);
                q = (uint32_t)v;
            }
            for (int p = 0; p < a.bits; ++p) {
                const uint64_t plane = __ballot((q >> p) & 1u);
                if (lane == p) w[(int64_t)t * a.bits + p] = plane;
            }
        }
    }
}

template <typename TO>
__global__ __launch_bounds__(kBlock) void k_decompress(int64_t n, int F, int bits, int G, int ng,
                                                       const uint64_t *__restrict__ codes,
                                                       const float *__restrict__ stats,
                                                       TO *__restrict__ out)
{
    const int lane = lane_id();
    const int64_t groups = n * ng;
    const int64_t waves = (int64_t)gridDim.x * (kBlock / kWave);
    const int nb = G / kWave;
    for (int64_t g = (int64_t)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave; g < groups;
         g += waves) {
        const int64_t i = g / ng;
        const int f0 = (int)(g % ng) * G;
        const int len = F - f0 < G ? F - f0 : G;
        const float m = stats[2 * g], r = stats[2 * g + 1];
        const uint64_t *__restrict__ w = codes + g * (int64_t)nb * bits;
        for (int t = 0; t < nb; ++t) {
            const int j = t * kWave + lane;
            uint32_t q = 0;
            for (int p = 0; p < bits; ++p)
                q |= (uint32_t)((w[(int64_t)t * bits + p] >> lane) & 1u) << p;
            if (j < len) {
                const float v[1] = {fmaf((float)q, r, m)};
                store_out<TO, 1>(out, i * F + f0 + j, v);
            }
        }
    }
}

cogdl_status check_codec(int64_t n, int32_t F, int32_t bits, int32_t group)
{
    if (n < 0 || F < 1 || bits < 1 || bits > 8 || group < kWave || group % kWave != 0)
        return COGDL_ERR_INVALID;
    return COGDL_OK;
}

// Workgroups for `waves` wavefronts of work, at most what fits on the chip at once.
unsigned resident_grid(const void *kernel, int64_t waves)
{
    int64_t b = (waves + (kBlock / kWave) - 1) / (kBlock / kWave);
    const int64_t res = resident_blocks(kernel, kBlock);
    if (b > res) b = res;
    if (b < 1) b = 1;
    return (unsigned)b;
}

unsigned codec_grid(int64_t groups)
{
    int64_t b = (groups + (kBlock / kWave) - 1) / (kBlock / kWave);
    if (b > 65536) b = 65536;
    if (b < 1) b = 1;
    return (unsigned)b;
}

// ------------------------------------------------ vectorized path
// Rows made of whole groups (F a multiple of G) with 16-byte aligned rows:
// each lane holds 8 consecutive features, a group is LG = G / (8 NV) adjacent
// lanes (8 to 64) holding NV vectors each, so a wavefront reads and writes
// full 16-byte vectors and covers 64 / LG groups at a time.  A 64-feature
// block of codes is 8 lanes: each contributes one byte per bit plane (its 8
// codes), and the bytes are combined by a three-level butterfly sum.

template <typename T> struct Vec8;
template <> struct Vec8<bf16_t> {
    __device__ static void load(const bf16_t *p, int64_t i, float (&o)[8]) { load_vec<bf16_t, 8>(p, i, o); }
    __device__ static void store(bf16_t *p, int64_t i, const float (&v)[8]) { store_vec<bf16_t, 8>(p, i, v); }
};
template <> struct Vec8<f16_t> {
    __device__ static void load(const f16_t *p, int64_t i, float (&o)[8]) { load_vec<f16_t, 8>(p, i, o); }
    __device__ static void store(f16_t *p, int64_t i, const float (&v)[8]) { store_vec<f16_t, 8>(p, i, v); }
};
template <> struct Vec8<float> {
    __device__ static void load(const float *p, int64_t i, float (&o)[8])
    {
        float lo[4], hi[4];
        load_vec<float, 4>(p, i, lo);
        load_vec<float, 4>(p, i + 4, hi);
#pragma unroll
        for (int e = 0; e < 4; ++e) { o[e] = lo[e]; o[4 + e] = hi[e]; }
    }
    __device__ static void store(float *p, int64_t i, const float (&v)[8]) { store_vec<float, 8>(p, i, v); }
};

template <typename TA, int NV>
__global__ __launch_bounds__(kBlock) void k_compress_v(CodecArgs a)
{
    const int lane = lane_id();
    const int LG = a.G / (8 * NV);
    const int sl = lane & (LG - 1);
    const int per_wave = kWave / LG;
    const int64_t groups = a.n * a.ng;
    const int64_t wave = (int64_t)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave;
    const int64_t stride = (int64_t)gridDim.x * (kBlock / kWave) * per_wave;
    const float qmax = (float)((1 << a.bits) - 1);
    const int nb = a.G / kWave;
    const TA *__restrict__ A = static_cast<const TA *>(a.A);
    for (int64_t g = wave * per_wave + lane / LG; g - lane / LG < groups; g += stride) {
        const bool gok = g < groups;
        const int64_t base = g * a.G;          // whole groups: the flat index of feature j is base + j
        float x[NV][8];
        float lo = INFINITY, hi = -INFINITY;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
            if (gok) {
                Vec8<TA>::load(A, base + (int64_t)(v * LG + sl) * 8, x[v]);
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e) x[v][e] = 0.f;
            }
#pragma unroll
            for (int e = 0; e < 8; ++e) {         // (a group past the end writes nothing)
                lo = fminf(lo, x[v][e]);
                hi = fmaxf(hi, x[v][e]);
            }
        }
        lo = group_reduce(lo, LG, [](float u, float v) { return fminf(u, v); });
        hi = group_reduce(hi, LG, [](float u, float v) { return fmaxf(u, v); });
        const float range = hi - lo;
        const float s = range > 0.f ? qmax / range : 0.f;
        const float r = range > 0.f ? range / qmax : 0.f;
        if (gok && sl == 0) {
            a.stats[2 * g] = lo;
            a.stats[2 * g + 1] = r;
        }
        uint64_t *__restrict__ w = a.codes + g * (int64_t)nb * a.bits;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
            const int64_t e0 = base + (int64_t)(v * LG + sl) * 8;   // a multiple of 8
            // the 8 uniforms of these features: two Philox blocks of 4
            const uint4 r0 = philox4(a.seed, (uint64_t)e0 >> 2);
            const uint4 r1 = philox4(a.seed, ((uint64_t)e0 >> 2) + 1);
            const uint32_t rw[8] = {r0.x, r0.y, r0.z, r0.w, r1.x, r1.y, r1.z, r1.w};
            uint32_t q[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float u = uniform24(rw[e]);
                // the clamp to [0, qmax] as one median of three (t is finite)
                const float t = __builtin_amdgcn_fmed3f(floorf(fmaf(x[v][e] - lo, s, u)), 0.f, qmax);
                q[e] = (uint32_t)t;
            }
            const int blk = (v * LG + sl) / 8;     // 64-feature block of these 8 features
            const int byte = sl & 7;               // their byte within the block's planes
            for (int p = 0; p < a.bits; ++p) {
                uint32_t frag = 0;
#pragma unroll
                for (int e = 0; e < 8; ++e) frag |= ((q[e] >> p) & 1u) << e;
                // bytes 0-3 of the plane in the low word, 4-7 in the high word
                uint32_t wlo = byte < 4 ? frag << (8 * byte) : 0u;
                uint32_t whi = byte >= 4 ? frag << (8 * (byte - 4)) : 0u;
                const auto add = [](uint32_t u, uint32_t v) { return u + v; };
                wlo = group_reduce(wlo, 8, add);
                whi = group_reduce(whi, 8, add);
                if (gok && byte == 0) w[(int64_t)blk * a.bits + p] = ((uint64_t)whi << 32) | wlo;
            }
        }
    }
}

template <typename TO, int NV>
__global__ __launch_bounds__(kBlock) void k_decompress_v(int64_t n, int bits, int G, int ng,
                                                         const uint64_t *__restrict__ codes,
                                                         const float *__restrict__ stats,
                                                         TO *__restrict__ out)
{
    const int lane = lane_id();
    const int LG = G / (8 * NV);
    const int sl = lane & (LG - 1);
    const int per_wave = kWave / LG;
    const int64_t groups = n * ng;
    const int64_t wave = (int64_t)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave;
    const int64_t stride = (int64_t)gridDim.x * (kBlock / kWave) * per_wave;
    const int nb = G / kWave;
    const int byte = sl & 7;   // this lane's byte of each plane word of its block
    const uint32_t *__restrict__ c32 = reinterpret_cast<const uint32_t *>(codes);
    // a group's stats and, per vector and plane, the 32-bit half of the plane
    // word that holds this lane's byte; fetched one group ahead
    const auto fetch = [&](int64_t g, float &m, float &r, uint32_t (&h)[NV][8]) {
        m = stats[2 * g];
        r = stats[2 * g + 1];
        const int64_t w0 = g * (int64_t)nb * bits;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
            const int blk = (v * LG + sl) / 8;
#pragma unroll
            for (int p = 0; p < 8; ++p)
                h[v][p] = p < bits ? c32[2 * (w0 + (int64_t)blk * bits + p) + (byte >> 2)] : 0u;
        }
    };
    int64_t g = wave * per_wave + lane / LG;
    float mn = 0.f, rn = 0.f;
    uint32_t hn[NV][8] = {};
    if (g < groups) fetch(g, mn, rn, hn);
    for (; g - lane / LG < groups; g += stride) {
        const bool gok = g < groups;
        const float m = mn, r = rn;
        uint32_t h[NV][8];
#pragma unroll
        for (int v = 0; v < NV; ++v)
#pragma unroll
            for (int p = 0; p < 8; ++p) h[v][p] = hn[v][p];
        if (g + stride < groups) fetch(g + stride, mn, rn, hn);
        if (!gok) continue;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
            uint32_t q[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};
#pragma unroll
            for (int p = 0; p < 8; ++p) {
                const uint32_t b8 = (h[v][p] >> (8 * (byte & 3))) & 0xffu;
#pragma unroll
                for (int e = 0; e < 8; ++e) q[e] |= ((b8 >> e) & 1u) << p;
            }
            float y[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) y[e] = fmaf((float)q[e], r, m);
            Vec8<TO>::store(out, g * G + (int64_t)(v * LG + sl) * 8, y);
        }
    }
}

using CompressKernel = void (*)(CodecArgs);

template <typename TA>
CompressKernel pick_compress_v(int nv)
{
    if (nv == 1) return k_compress_v<TA, 1>;
    if (nv == 2) return k_compress_v<TA, 2>;
    if (nv == 4) return k_compress_v<TA, 4>;
    return k_compress_v<TA, 8>;
}

// NV for the vectorized path (0: not applicable)
int vector_nv(int32_t F, int32_t group, const void *p)
{
    if (F % group != 0 || group > 4096 || (uintptr_t)p % 16 != 0) return 0;
    return group >= 512 ? group / 512 : 1;
}

}  // namespace
}  // namespace cogdl

using namespace cogdl;

extern "C" {

cogdl_status cogdl_act_codec_size(int64_t n, int32_t F, int32_t bits, int32_t group,
                                  int64_t *code_words, int64_t *stat_floats)
{
    cogdl_status st = check_codec(n, F, bits, group);
    if (st != COGDL_OK) return st;
    if (!code_words || !stat_floats) return COGDL_ERR_INVALID;
    const int64_t ng = (F + group - 1) / group;
    *code_words = n * ng * (group / kWave) * bits;
    *stat_floats = n * ng * 2;
    return COGDL_OK;
}

cogdl_status cogdl_act_compress(int64_t n, int32_t F, const void *A, cogdl_dtype a_dtype,
                                int32_t bits, int32_t group, uint64_t seed, uint64_t *codes,
                                float *stats, hipStream_t stream)
{
    cogdl_status st = check_codec(n, F, bits, group);
    if (st != COGDL_OK) return st;
    if (!dtype_ok(a_dtype)) return COGDL_ERR_DTYPE;
    if (n > 0 && (!A || !codes || !stats)) return COGDL_ERR_INVALID;
    if (n == 0) return COGDL_OK;
    CodecArgs a{n, F, bits, group, (F + group - 1) / group, seed, A, codes, stats};
    const unsigned b = codec_grid(n * a.ng);
    const int nv = vector_nv(F, group, A);
    if (nv > 0) {
        const int per_wave = kWave / (group / (8 * nv));
        CompressKernel k = a_dtype == COGDL_F32    ? pick_compress_v<float>(nv)
                           : a_dtype == COGDL_BF16 ? pick_compress_v<bf16_t>(nv)
                                                   : pick_compress_v<f16_t>(nv);
        // a grid past the resident size, no prefetch: a resident grid walking the
        // groups with the next one fetched ahead measured 10-15% slower here
        const unsigned bv = codec_grid((n * a.ng + per_wave - 1) / per_wave);
        COGDL_LAUNCH("act_compress", k, bv, kBlock, stream, a);
        return COGDL_OK;
    }
    if (a_dtype == COGDL_F32)
        COGDL_LAUNCH("act_compress", k_compress<float>, b, kBlock, stream, a);
    else if (a_dtype == COGDL_BF16)
        COGDL_LAUNCH("act_compress", k_compress<bf16_t>, b, kBlock, stream, a);
    else
        COGDL_LAUNCH("act_compress", k_compress<f16_t>, b, kBlock, stream, a);
    return COGDL_OK;
}

cogdl_status cogdl_act_decompress(int64_t n, int32_t F, int32_t bits, int32_t group,
                                  const uint64_t *codes, const float *stats, void *out,
                                  cogdl_dtype out_dtype, hipStream_t stream)
{
    cogdl_status st = check_codec(n, F, bits, group);
    if (st != COGDL_OK) return st;
    if (!dtype_ok(out_dtype)) return COGDL_ERR_DTYPE;
    if (n > 0 && (!out || !codes || !stats)) return COGDL_ERR_INVALID;
    if (n == 0) return COGDL_OK;
    const int ng = (F + group - 1) / group;
    const unsigned b = codec_grid(n * ng);
    const int nv = vector_nv(F, group, out);
    if (nv > 0) {
        const int per_wave = kWave / (group / (8 * nv));
        const int64_t wv = (n * ng + per_wave - 1) / per_wave;
#define COGDL_DECOMP_V(TO)                                                                       \
    do {                                                                                         \
        auto k = nv == 1 ? k_decompress_v<TO, 1> : nv == 2 ? k_decompress_v<TO, 2>              \
                 : nv == 4 ? k_decompress_v<TO, 4> : k_decompress_v<TO, 8>;                     \
        const unsigned bv = codec_grid(wv);    /* past the resident size: 2-4% faster */      \
        COGDL_LAUNCH("act_decompress", k, bv, kBlock, stream, n, bits, group, ng, codes, stats,  \
                     static_cast<TO *>(out));                                                    \
    } while (0)
        if (out_dtype == COGDL_F32) COGDL_DECOMP_V(float);
        else if (out_dtype == COGDL_BF16) COGDL_DECOMP_V(bf16_t);
        else COGDL_DECOMP_V(f16_t);
#undef COGDL_DECOMP_V
        return COGDL_OK;
    }
    if (out_dtype == COGDL_F32)
        COGDL_LAUNCH("act_decompress", k_decompress<float>, b, kBlock, stream, n, F, bits, group,
                     ng, codes, stats, static_cast<float *>(out));
    else if (out_dtype == COGDL_BF16)
        COGDL_LAUNCH("act_decompress", k_decompress<bf16_t>, b, kBlock, stream, n, F, bits, group,
                     ng, codes, stats, static_cast<bf16_t *>(out));
    else
        COGDL_LAUNCH("act_decompress", k_decompress<f16_t>, b, kBlock, stream, n, F, bits, group,
                     ng, codes, stats, static_cast<f16_t *>(out));
    return COGDL_OK;
}

}  // extern "C"
