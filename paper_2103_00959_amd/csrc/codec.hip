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
// Mapping on gfx950: a wavefront per group.  The min/max is a butterfly over
// the 64 lanes; each lane quantizes one feature of a block, and a block's b
// bit planes are b wavefront ballots (one 64-bit mask each), written by lanes
// 0..b-1, so a group of bf16 features reads 2G bytes and writes G b / 8.
#include "common.hpp"
#include "internal.hpp"

namespace cogdl {
namespace {

constexpr int kBlock = 256;

__device__ __forceinline__ uint32_t philox_word(uint64_t seed, int64_t e)
{
    uint32_t c0 = (uint32_t)((uint64_t)e >> 2), c1 = (uint32_t)((uint64_t)e >> 34), c2 = 0u, c3 = 0u;
    uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
#pragma unroll
    for (int round = 0; round < 10; ++round) {
        const uint32_t hi0 = __umulhi(0xD2511F53u, c0), lo0 = 0xD2511F53u * c0;
        const uint32_t hi1 = __umulhi(0xCD9E8D57u, c2), lo1 = 0xCD9E8D57u * c2;
        const uint32_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
        c0 = n0;
        c1 = lo1;
        c2 = n2;
        c3 = lo0;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    const int w = (int)(e & 3);
    return w == 0 ? c0 : w == 1 ? c1 : w == 2 ? c2 : c3;
}

__device__ __forceinline__ float wave_min(float v)
{
    for (int off = 1; off < kWave; off <<= 1) v = fminf(v, lane_xor(v, off));
    return v;
}

__device__ __forceinline__ float wave_max(float v)
{
    for (int off = 1; off < kWave; off <<= 1) v = fmaxf(v, lane_xor(v, off));
    return v;
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
                const float u = (float)(philox_word(a.seed, base + j) >> 8) * (1.0f / 16777216.0f);
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

unsigned codec_grid(int64_t groups)
{
    int64_t b = (groups + (kBlock / kWave) - 1) / (kBlock / kWave);
    if (b > 65536) b = 65536;
    if (b < 1) b = 1;
    return (unsigned)b;
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
