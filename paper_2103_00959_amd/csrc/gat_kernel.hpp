// The gather kernel of the attention path (section 2.2: SDDMM of the scores,
// LeakyReLU, edge softmax and multi-head SpMM, fused), shared by gat.hip (the
// forward variants) and gat_bwd.hip (the backward variant on the CSC).  See
// gat.hip for the mapping onto gfx950.
#pragma once

#include "common.hpp"
#include "internal.hpp"

namespace cogdl {

constexpr int kGatBlock = 256;

struct GatArgs {
    const int4 *units;
    const int32_t *u_lo;        // with units: this launch runs units [*u_lo, *u_hi)
    const int32_t *u_hi;        // (lists > 1: list x is [u_lo[x], u_hi[x]), see unit_walk)
    int32_t lists = 1;
    int32_t n_rows;
    const int32_t *rowptr;
    const int32_t *col;
    int32_t H;
    int32_t D;
    int64_t W;                  // H * D
    const float *s_dst;
    const float *s_src;
    float slope;
    const float *alpha_in;      // weights given: skip the attention steps
    const void *X;
    uint64_t x_bytes;           // size of X, bounds the buffer gathers
    void *Y;
    float *alpha_out;
    float *row_stats;           // softmax: per row the final (m, 1/z) of each head, 2H floats (nullable)
    float *partials;
    int64_t pstride;
    float *gstats;              // per partial slot: m[max_heads], z[max_heads]
    const int32_t *perm;        // BWD: edge k of this CSC is edge perm[k] of the CSR
    const float2 *rec;          // BWD: per CSR edge and head (weight, value summed per row)
    float *ds_out;              // BWD: those sums, n_rows x H (split rows: gstats)
    const float *bias;          // epilogue: Y = act(aggregate + bias), bias nullable
    int32_t act;
    const float *a_src;         // PROJ: the source score is X[j, h, :] . a_src[h, :] (H x D fp32)
    int32_t park_cap;           // alpha wanted: LDS floats per sub-group for parked scores (0: none)
    int32_t sstride;            // 2 * max_heads
    int32_t slab;
    int32_t log2S;
};

// Descriptor {row, first edge, end edge, partial slot} of unit u (an empty
// unit past the end, so prefetching one unit ahead needs no branch around it).
__device__ __forceinline__ int4 fetch_gat_unit(const GatArgs &a, int64_t u, int64_t hi)
{
    if (u >= hi) return make_int4(0, 0, 0, -1);
    if (a.units) return a.units[u];
    const int r = (int)u;
    return make_int4(r, a.rowptr[r], a.rowptr[r + 1], -1);
}

// alpha[k, h] = alpha_value(e_kh, m, rz) for the edges k = beg + slot + j * slots
// of one head h, R loads in flight per lane; the raw scores e_kh are read from
// `parked` at index (k - base) * H + h, where the aggregation or the softmax
// parked them: alpha itself (base 0; a contiguous re-read instead of a second
// random gather of s_src) or a row buffer in LDS (base = beg).
template <int R>
__device__ __forceinline__ void alpha_from_parked(const float *parked, int64_t base,
                                                  float *__restrict__ alpha, int H, int h, float m,
                                                  float rz, int beg, int end, int slot, int slots)
{
    for (int k0 = beg + slot; k0 < end; k0 += R * slots) {
        float e[R];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int k = k0 + r * slots;
            e[r] = k < end ? parked[(k - base) * H + h] : 0.f;
        }
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int k = k0 + r * slots;
            if (k < end) alpha[(int64_t)k * H + h] = alpha_value(e[r], m, rz);
        }
    }
}

// Scores of a whole-row unit parked in LDS when alpha is wanted: each sub-group
// of a k_gat workgroup owns kParkFloats / (sub-groups per workgroup) floats of
// the dynamic LDS, enough for rows of that many / H edges; longer rows and
// neighbour groups of split rows park in alpha.
constexpr int kParkFloats = 8192;   // 32 KB per workgroup

// Sum over the 8 lanes of an aligned group of each lane's v[t], scattered:
// lane hp (its position in the group) ends with the full sum of v[hp].  Three
// exchange levels (lane ^ 1, ^ 2 by DPP, ^ 4 by a swizzle), each lane keeping
// the half of its values whose index bit matches its own position bit.
__device__ __forceinline__ float reduce_scatter8(const float (&v)[8], int hp)
{
    const bool b0 = hp & 1, b1 = hp & 2, b2 = hp & 4;
    float k4[4], k2[2];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float keep = b0 ? v[2 * i + 1] : v[2 * i];
        const float send = b0 ? v[2 * i] : v[2 * i + 1];
        k4[i] = keep + bfly_partner<1>(send);
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const float keep = b1 ? k4[2 * i + 1] : k4[2 * i];
        const float send = b1 ? k4[2 * i] : k4[2 * i + 1];
        k2[i] = keep + bfly_partner<2>(send);
    }
    const float keep = b2 ? k2[1] : k2[0];
    const float send = b2 ? k2[0] : k2[1];
    // lane ^ 4 inside each 32-lane half: swizzle bit mode, and 0x1f, or 0, xor 4
    return keep + __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(send), 0x101F));
}

// The value of lane T of this lane's aligned group of 8 (swizzle bit mode:
// and 0x18 keeps the group, or T picks the lane).
template <int T>
__device__ __forceinline__ float from_group8(float v)
{
    return __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v), 0x18 | (T << 5)));
}

// PM (source-score mode): 0 and 3 read s_src (or, BWD / alpha_in, the given
// weights); 1 and 2 form it from the gathered row.
// PM = 1: the source score of each edge is formed from the gathered
// feature row itself, s = X[j, h, :] . a_src[h, :] (each lane's VEC products,
// then a butterfly over the L = D / VEC adjacent lanes of the head, which
// leaves every lane of the head with the same bits), instead of being gathered
// from s_src: a GAT layer's source score is that projection, and the random
// 4H-byte score row of each edge costs a whole cache line.  Needs 16-byte
// vectors, L a power of two and each head inside one chunk (the host checks).
// PM = 2 (one chunk, L equal to the U edges of a batch): the partial products
// are reduce-scattered over the head's lanes instead, so each lane ends with
// the score of one edge of the batch and does that edge's softmax arithmetic
// alone (LeakyReLU, exp, its share of z; the batch maximum by a butterfly),
// and the weights are handed back to the head's lanes by swizzles: the
// per-edge scalar work of the softmax is done once per head instead of once
// per lane of the head.  PM = 3 is the same distribution with the scores read
// from s_src: each lane reads the score of its own edge only.  BWD with PM = 3:
// each lane reads the (weight, value) record of its own edge of the batch, the
// weights reach the head's lanes by swizzles and each lane sums the values of
// its own edges, added over the head at the unit's end.
// The forward's four-chunk kernel with given scores and packed 16-bit rows runs
// three wavefronts per SIMD (a few registers spilled, still faster than two).
template <int VEC, int CH, bool BUF, bool BWD, int PM, int XB>
constexpr bool gat_given_packed = BUF && !BWD && PM == 0 && CH == 4 && VEC == 8 && XB == 2;

template <typename TX, typename TY, int VEC, int CH, bool BUF, bool BWD, int PM = 0>
__global__ __launch_bounds__(kGatBlock, ((CH == 1 && BUF && !BWD)                                   ? 4
                                         : (gat_given_packed<VEC, CH, BUF, BWD, PM, (int)sizeof(TX)>) ? 3
                                                                                                      : 1))
void k_gat(GatArgs a)
{
    constexpr bool PROJ = PM == 1 || PM == 2;
    constexpr bool DIST = PM == 2 || PM == 3;
    static_assert(!BWD || PM == 0 || PM == 3, "the backward reads its weights");
    constexpr int U = (VEC == 1 ? 16 : 8) / CH;
    const int log2S = a.log2S;
    const int S = 1 << log2S;
    const int lane = lane_id();
    const int lig = lane & (S - 1);
    const int gbase = lane & ~(S - 1);
    const int H = a.H;
    const bool soft = !BWD && a.alpha_in == nullptr;   // the backward reads its weights
    const UnitWalk walk = unit_walk(a.units != nullptr, a.u_lo, a.u_hi, a.lists, a.n_rows,
                                    kGatBlock >> log2S, threadIdx.x >> log2S);
    const int64_t stride = walk.step;
    const int64_t hi = walk.end;

    const int64_t f0 = (int64_t)blockIdx.y * a.slab;
    const int64_t f_end = (f0 + a.slab < a.W) ? f0 + a.slab : a.W;
    int64_t fe[CH];
    bool act[CH];
    int hd[CH];
#pragma unroll
    for (int c = 0; c < CH; ++c) {
        fe[c] = f0 + (int64_t)(c * S + lig) * VEC;
        act[c] = fe[c] < f_end;
        hd[c] = act[c] ? (int)(fe[c] / a.D) : 0;
    }
    const RowGather<TX, VEC, BUF> X(a.X, a.x_bytes);
    const int32_t *__restrict__ col = a.col;
    const float *__restrict__ wsrc = soft ? a.s_src : a.alpha_in;
    constexpr float kLog2eF = 1.44269504f;
    // PROJ: this lane's VEC entries of a_src, and the lanes per head.  With
    // several chunks per lane (the tiny-unit kernels) the slab's a_src sits in
    // LDS instead and is read per batch, which keeps CH * VEC registers free.
    constexpr bool ASRC_LDS = PM == 1 && CH > 1;
    constexpr int kAsrcMax = kWave * CH * VEC;          // a slab's width at most
    __shared__ float asrc_lds[ASRC_LDS ? kAsrcMax : 1];
    float asrc[PROJ && !ASRC_LDS ? CH : 1][PROJ && !ASRC_LDS ? VEC : 1];
    const int hl = PROJ ? a.D / VEC : 1;
    if constexpr (ASRC_LDS) {
        for (int64_t f = threadIdx.x; f < f_end - f0; f += kGatBlock) asrc_lds[f] = a.a_src[f0 + f];
        __syncthreads();
    } else if constexpr (PROJ) {
#pragma unroll
        for (int c = 0; c < CH; ++c)
#pragma unroll
            for (int e = 0; e < VEC; ++e) asrc[c][e] = act[c] ? a.a_src[fe[c] + e] : 0.f;
    }
    // (edge slot, head) lane layout of the alpha sweep: eps edges per step
    const int eps = S / H;
    extern __shared__ float park_buf[];
    // whole-row units whose scores fit this sub-group's LDS buffer park there
    // (computed where used: both stay out of the registers of the main loop)
#define COGDL_PARK_LDS (a.park_cap > 0 && part < 0 && (end - beg) * H <= a.park_cap)
#define COGDL_LDS_PARK (park_buf + (threadIdx.x >> log2S) * a.park_cap)
    const int q_slot = lig / H, q_head = lig % H;

    // Resident grid, software-pipelined over units as in the SpMM kernel.
    int64_t u = walk.first;
    if (u >= hi) return;
    int4 d = fetch_gat_unit(a, u, hi);
    int c_cur = 0, p_cur = 0;
    if (d.z > d.y) {
        const int k = d.y + lig < d.z - 1 ? d.y + lig : d.z - 1;
        c_cur = col[k];
        if constexpr (BWD) p_cur = a.perm[k];
    }
    for (;;) {
        const int64_t un = u + stride;
        const int4 dn = fetch_gat_unit(a, un, hi);
        const int row = d.x, beg = d.y, end = d.z, part = d.w;
        float sd[CH], m[CH], z[CH], dsum[CH];
        float acc[CH][VEC];
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            dsum[c] = 0.f;
            sd[c] = soft ? a.s_dst[(int64_t)row * H + hd[c]] : 0.f;
            m[c] = -INFINITY;
            z[c] = 0.f;
#pragma unroll
            for (int e = 0; e < VEC; ++e) acc[c][e] = 0.f;
        }

        // Branch-free batches: index loads are clamped to the unit's last
        // edge, masked gathers read zeros, masked weights are -inf (softmax)
        // or 0.
        const int last = end - 1;
        for (int k0 = beg; k0 < end; k0 += S) {
            const int n = (end - k0 < S) ? end - k0 : S;
            const int kn = k0 + S + lig < last ? k0 + S + lig : last;
            const int c_nxt = col[kn];
            const int p_nxt = BWD ? a.perm[kn] : 0;
            for (int j = 0; j < n; j += U) {
                int cc[U], pk[U];
                bool ok[U];
#pragma unroll
                for (int t = 0; t < U; ++t) {
                    ok[t] = j + t < n;
                    cc[t] = lane_bcast(c_cur, gbase + (ok[t] ? j + t : j));
                    if constexpr (BWD && !DIST) pk[t] = lane_bcast(p_cur, gbase + (ok[t] ? j + t : j));
                }
                float w[U][CH];
                // the multi-chunk (tiny-unit) kernels keep 16-bit rows packed, one
                // 16-byte word per chunk, and widen them where used: the projected ones
                // with a_src in LDS and the given-score four-chunk one gain a wavefront
                // per SIMD (the other kernels gain none)
                constexpr bool XPACK = (ASRC_LDS && sizeof(TX) == 2 && VEC == 8) ||
                                       gat_given_packed<VEC, CH, BUF, BWD, PM, (int)sizeof(TX)>;
                float xv[XPACK ? 1 : U][XPACK ? 1 : CH][XPACK ? 1 : VEC];
                uint4 xw[XPACK ? U : 1][XPACK ? CH : 1];
#pragma unroll
                for (int t = 0; t < U; ++t)
#pragma unroll
                    for (int c = 0; c < CH; ++c) {
                        const bool on = ok[t] && act[c];
                        const int64_t wi = BWD ? (int64_t)pk[t] * H + hd[c]
                                         : soft ? (int64_t)cc[t] * H + hd[c]
                                                : (int64_t)(k0 + j + t) * H + hd[c];
                        if constexpr (BWD && !DIST) {
                            const float2 r = a.rec[on ? wi : 0];
                            w[t][c] = r.x;
                            dsum[c] += on ? r.y : 0.f;
                        } else if constexpr (!PROJ && !DIST) {
                            w[t][c] = wsrc[on ? wi : 0];
                        }
                        if constexpr (XPACK) xw[t][c] = X.load_raw16((int64_t)cc[t] * a.W + fe[c], on);
                        else X.load((int64_t)cc[t] * a.W + fe[c], on, xv[t][c]);
                    }
                if constexpr (DIST && BWD) {
                    static_assert(CH == 1 && U == 8, "one chunk, batches of 8 edges");
                    const int hp = lig & (U - 1);
                    const bool mine = j + hp < n && act[0];
                    const int pme = lane_bcast(p_cur, gbase + j + hp);
                    const float2 r = a.rec[mine ? (int64_t)pme * H + hd[0] : 0];
                    dsum[0] += mine ? r.y : 0.f;
                    const float wv = mine ? r.x : 0.f;
                    float wt[U];
                    wt[0] = from_group8<0>(wv); wt[1] = from_group8<1>(wv);
                    wt[2] = from_group8<2>(wv); wt[3] = from_group8<3>(wv);
                    wt[4] = from_group8<4>(wv); wt[5] = from_group8<5>(wv);
                    wt[6] = from_group8<6>(wv); wt[7] = from_group8<7>(wv);
#pragma unroll
                    for (int t = 0; t < U; ++t)
#pragma unroll
                        for (int e = 0; e < VEC; ++e) acc[0][e] = fmaf(wt[t], xv[t][0][e], acc[0][e]);
                    continue;
                } else if constexpr (DIST) {
                    static_assert(CH == 1 && U == 8, "one chunk, batches of 8 edges");
                    const int hp = lig & (U - 1);
                    const bool mine = j + hp < n && act[0];       // this lane's edge of the batch
                    float sc;
                    if constexpr (PROJ) {
                        float pp[U];
#pragma unroll
                        for (int t = 0; t < U; ++t) {
                            float p = 0.f;
#pragma unroll
                            for (int e = 0; e < VEC; ++e) p = fmaf(xv[t][0][e], asrc[0][e], p);
                            pp[t] = p;
                        }
                        sc = reduce_scatter8(pp, hp);
                    } else {
                        const int cme = lane_bcast(c_cur, gbase + j + hp);
                        sc = wsrc[mine ? (int64_t)cme * H + hd[0] : 0];
                    }
                    const float e1 = mine ? leaky_relu(sd[0] + sc, a.slope) : -INFINITY;
                    if constexpr (!PROJ) {
                        // alpha wanted: each lane parks the score of its own edge
                        if (a.alpha_out != nullptr && mine) {
                            const int k = k0 + j + hp;
                            if (COGDL_PARK_LDS) COGDL_LDS_PARK[(k - beg) * H + hd[0]] = e1;
                            else a.alpha_out[(int64_t)k * H + hd[0]] = e1;
                        }
                    }
                    const float mb = fmaxf(m[0], group_reduce(e1, U, [](float x, float y) { return fmaxf(x, y); }));
                    if (mb > m[0]) {
                        const float r = __expf(m[0] - mb);
                        z[0] *= r;
#pragma unroll
                        for (int e = 0; e < VEC; ++e) acc[0][e] *= r;
                        m[0] = mb;
                    }
                    const float pl = __builtin_amdgcn_exp2f(fmaf(e1, kLog2eF, -m[0] * kLog2eF));
                    z[0] += pl;            // this lane's share of z, summed over the head at the unit's end
                    float wt[U];
                    wt[0] = from_group8<0>(pl); wt[1] = from_group8<1>(pl);
                    wt[2] = from_group8<2>(pl); wt[3] = from_group8<3>(pl);
                    wt[4] = from_group8<4>(pl); wt[5] = from_group8<5>(pl);
                    wt[6] = from_group8<6>(pl); wt[7] = from_group8<7>(pl);
#pragma unroll
                    for (int t = 0; t < U; ++t)
#pragma unroll
                        for (int e = 0; e < VEC; ++e) acc[0][e] = fmaf(wt[t], xv[t][0][e], acc[0][e]);
                    continue;
                }
                if constexpr (ASRC_LDS) {
                    // (no instruction: keeps the a_src reads in the loop, out of registers)
                    asm volatile("" ::: "memory");
#pragma unroll
                    for (int c = 0; c < CH; ++c) {
                        float as[VEC];
#pragma unroll
                        for (int e = 0; e < VEC; ++e) as[e] = asrc_lds[fe[c] - f0 + e];
#pragma unroll
                        for (int t = 0; t < U; ++t) {
                            float xe[VEC];
                            if constexpr (XPACK) {
                                RowGather<TX, VEC, BUF>::unpack16(xw[t][c].x, xw[t][c].y, xw[t][c].z,
                                                                  xw[t][c].w, xe);
                            } else {
#pragma unroll
                                for (int e = 0; e < VEC; ++e) xe[e] = xv[t][c][e];
                            }
                            float p = 0.f;
#pragma unroll
                            for (int e = 0; e < VEC; ++e) p = fmaf(xe[e], as[e], p);
                            w[t][c] = group_sum(p, hl);
                        }
                    }
                } else if constexpr (PROJ) {
#pragma unroll
                    for (int t = 0; t < U; ++t)
#pragma unroll
                        for (int c = 0; c < CH; ++c) {
                            float p = 0.f;
#pragma unroll
                            for (int e = 0; e < VEC; ++e) p = fmaf(xv[t][c][e], asrc[c][e], p);
                            w[t][c] = group_sum(p, hl);
                        }
                }
                if (soft) {
#pragma unroll
                    for (int c = 0; c < CH; ++c) {
                        float mb = m[c];
#pragma unroll
                        for (int t = 0; t < U; ++t) {
                            w[t][c] = (ok[t] && act[c]) ? leaky_relu(sd[c] + w[t][c], a.slope) : -INFINITY;
                            mb = fmaxf(mb, w[t][c]);
                        }
                        // alpha wanted: park the raw scores, one lane per head and edge
                        // (the lane of the head's first feature in this slab)
                        if constexpr (!PROJ) {
                            if (a.alpha_out != nullptr && act[c] && fe[c] % a.D == 0) {
#pragma unroll
                                for (int t = 0; t < U; ++t) {
                                    if (!ok[t]) continue;
                                    const int k = k0 + j + t;
                                    if (COGDL_PARK_LDS) COGDL_LDS_PARK[(k - beg) * H + hd[c]] = w[t][c];
                                    else a.alpha_out[(int64_t)k * H + hd[c]] = w[t][c];
                                }
                            }
                        }
                        if (mb > m[c]) {
                            const float r = __expf(m[c] - mb);
                            z[c] *= r;
#pragma unroll
                            for (int e = 0; e < VEC; ++e) acc[c][e] *= r;
                            m[c] = mb;
                        }
                        // exp(w - m) = 2^(w log2 e - m log2 e): one fma per edge; a masked
                        // edge (-inf) gives 2^-inf = 0.  m is finite here on every lane that
                        // stores (its first batch holds a valid edge); a lane past the row's
                        // width (no store) may compute NaN, which no other lane reads.
                        const float ml = m[c] * kLog2eF;
                        float zb = 0.f;
#pragma unroll
                        for (int t = 0; t < U; ++t) {
                            w[t][c] = __builtin_amdgcn_exp2f(fmaf(w[t][c], kLog2eF, -ml));
                            zb += w[t][c];
                        }
                        z[c] += zb;
                    }
                } else {
#pragma unroll
                    for (int t = 0; t < U; ++t)
#pragma unroll
                        for (int c = 0; c < CH; ++c)
                            if (!(ok[t] && act[c])) w[t][c] = 0.f;
                }
#pragma unroll
                for (int t = 0; t < U; ++t)
#pragma unroll
                    for (int c = 0; c < CH; ++c)
                        if constexpr (XPACK) {
                            // widened again here (the asm keeps the first widening from
                            // being carried in registers across the softmax step)
                            uint4 q = xw[t][c];
                            asm volatile("" : "+v"(q.x), "+v"(q.y), "+v"(q.z), "+v"(q.w));
                            float xe[VEC];
                            RowGather<TX, VEC, BUF>::unpack16(q.x, q.y, q.z, q.w, xe);
#pragma unroll
                            for (int e = 0; e < VEC; ++e) acc[c][e] = fmaf(w[t][c], xe[e], acc[c][e]);
                        } else {
#pragma unroll
                            for (int e = 0; e < VEC; ++e) acc[c][e] = fmaf(w[t][c], xv[t][c][e], acc[c][e]);
                        }
            }
            c_cur = c_nxt;
            if constexpr (BWD) p_cur = p_nxt;
        }
        if constexpr (DIST && BWD) dsum[0] = group_sum(dsum[0], U);   // the head's shares
        else if constexpr (DIST) z[0] = group_sum(z[0], U);          // the head's shares of z
        int c_first_next = 0, p_first_next = 0;
        if (dn.z > dn.y) {
            const int k = dn.y + lig < dn.z - 1 ? dn.y + lig : dn.z - 1;
            c_first_next = col[k];
            if constexpr (BWD) p_first_next = a.perm[k];
        }
        if constexpr (BWD) {
            // the per-head sum, written once by the lane holding the head's first feature
#pragma unroll
            for (int c = 0; c < CH; ++c) {
                if (!act[c] || fe[c] % a.D != 0) continue;
                if (part >= 0) a.gstats[(int64_t)part * a.sstride + hd[c]] = dsum[c];
                else a.ds_out[(int64_t)row * H + hd[c]] = dsum[c];
            }
        }

        if (part >= 0) {
            // neighbour group of a split row: unnormalized partial + (m, z) per head
#pragma unroll
            for (int c = 0; c < CH; ++c) {
                if (!act[c]) continue;
                store_vec<float, VEC>(a.partials, (int64_t)part * a.pstride + fe[c], acc[c]);
                if (soft && fe[c] % a.D == 0) {
                    a.gstats[(int64_t)part * a.sstride + hd[c]] = m[c];
                    a.gstats[(int64_t)part * a.sstride + (a.sstride >> 1) + hd[c]] = z[c];
                }
            }
        } else {
            float rz[CH];
#pragma unroll
            for (int c = 0; c < CH; ++c) {
                rz[c] = (soft && z[c] > 0.f) ? 1.f / z[c] : 1.f;
                // the row's softmax state, from which alpha = alpha_value(e, m, 1/z) can be
                // rebuilt (every lane of the head holds it; the lane of its first feature writes)
                if (soft && a.row_stats != nullptr && act[c] && fe[c] % a.D == 0) {
                    a.row_stats[(int64_t)row * 2 * H + hd[c]] = m[c];
                    a.row_stats[(int64_t)row * 2 * H + H + hd[c]] = rz[c];
                }
            }
#pragma unroll
            for (int c = 0; c < CH; ++c) {
                float v[VEC];
#pragma unroll
                for (int e = 0; e < VEC; ++e) v[e] = acc[c][e] * rz[c];
                if (act[c]) {
                    epilogue<VEC>(v, a.bias, a.act, fe[c]);
                    store_out<TY, VEC>(static_cast<TY *>(a.Y), (int64_t)row * a.W + fe[c], v);
                }
            }
            if (!PROJ && soft && a.alpha_out != nullptr) {   // (the PROJ entry writes no alpha)
                // alpha of this whole-row unit: lanes as (edge slot, head); the
                // (m, z) of head h comes from the lane holding the first feature
                // of h in this slab.
                const int h1 = q_head;
                const int slot = q_slot;
                const int64_t hf = (int64_t)h1 * a.D;
                const bool mine_head = hf >= f0 && hf < f_end;
                const int idx = mine_head ? (int)((hf - f0) / VEC) : 0;
                const int src_c = idx / S, src_l = idx % S;
                float m1 = 0.f, r1 = 0.f;
#pragma unroll
                for (int c = 0; c < CH; ++c) {
                    const float mm = lane_bcast(m[c], gbase + src_l);
                    const float rr = lane_bcast(rz[c], gbase + src_l);
                    if (c == src_c) { m1 = mm; r1 = rr; }
                }
                // the scores were parked by other lanes of this wavefront: wait for
                // those stores before reading them back
                __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
                __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
                if (mine_head && slot < eps) {
                    if (COGDL_PARK_LDS)
                        alpha_from_parked<4>(COGDL_LDS_PARK, beg, a.alpha_out, H, h1, m1, r1, beg, end, slot, eps);
                    else alpha_from_parked<4>(a.alpha_out, 0, a.alpha_out, H, h1, m1, r1, beg, end, slot, eps);
                }
            }
        }
        if (un >= hi) break;
        u = un;
        d = dn;
        c_cur = c_first_next;
        p_cur = p_first_next;
    }
}

#undef COGDL_PARK_LDS
#undef COGDL_LDS_PARK

using GatKernel = void (*)(GatArgs);

template <typename TX, typename TY, bool BUF, bool BWD>
GatKernel gat_pick_vec(int vec, int ch, bool dist)
{
    constexpr int V = (int)(16 / sizeof(TX));
    if (vec == 1) {
        if (ch == 1) return k_gat<TX, TY, 1, 1, BUF, BWD>;
        if (ch == 2) return k_gat<TX, TY, 1, 2, BUF, BWD>;
        return k_gat<TX, TY, 1, 4, BUF, BWD>;
    }
    if (ch == 1) {
        if (dist) return k_gat<TX, TY, V, 1, BUF, BWD, 3>;
        return k_gat<TX, TY, V, 1, BUF, BWD>;
    }
    if (ch == 2) return k_gat<TX, TY, V, 2, BUF, BWD>;
    return k_gat<TX, TY, V, 4, BUF, BWD>;
}

template <typename TX, bool BUF, bool BWD>
GatKernel gat_pick_y(int ydt, int vec, int ch, bool dist)
{
    if (ydt == COGDL_F32) return gat_pick_vec<TX, float, BUF, BWD>(vec, ch, dist);
    if (ydt == COGDL_BF16) return gat_pick_vec<TX, bf16_t, BUF, BWD>(vec, ch, dist);
    return gat_pick_vec<TX, f16_t, BUF, BWD>(vec, ch, dist);
}

// dist: the distributed kernel (PM = 3: scores read from s_src, or BWD's
// records, one edge per lane; one chunk of 16-byte vectors, 8 lanes per head).
template <bool BWD>
GatKernel gat_pick(int xdt, int ydt, int vec, int ch, bool buf, bool dist = false)
{
    if (buf) {
        if (xdt == COGDL_F32) return gat_pick_y<float, true, BWD>(ydt, vec, ch, dist);
        if (xdt == COGDL_BF16) return gat_pick_y<bf16_t, true, BWD>(ydt, vec, ch, dist);
        return gat_pick_y<f16_t, true, BWD>(ydt, vec, ch, dist);
    }
    if (xdt == COGDL_F32) return gat_pick_y<float, false, BWD>(ydt, vec, ch, dist);
    if (xdt == COGDL_BF16) return gat_pick_y<bf16_t, false, BWD>(ydt, vec, ch, dist);
    return gat_pick_y<f16_t, false, BWD>(ydt, vec, ch, dist);
}

// The forward kernels with projected source scores (16-byte vectors only),
// instantiated in gat_proj.hip; dist: the distributed-softmax mode (one chunk,
// 8 lanes per head).
GatKernel gat_pick_proj(int xdt, int ydt, int ch, bool buf, bool dist);

}  // namespace cogdl
