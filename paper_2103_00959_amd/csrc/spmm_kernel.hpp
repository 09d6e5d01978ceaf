// The gather kernel of the generalized SpMM (section 2.2, Eq. 1), shared by
// the translation units that instantiate its variants: spmm.hip (sum of
// products, the hot path) and gspmm.hip (max, and the add / subtract
// messages).  See spmm.hip for the mapping onto gfx950.
#pragma once

#include "common.hpp"
#include "internal.hpp"

namespace cogdl {

constexpr int kSpmmBlock = 256;

struct SpmmArgs {
    const int4 *units;          // nullptr: one unit per row in row order
    const int32_t *u_lo;        // with units: this launch runs units [*u_lo, *u_hi)
    const int32_t *u_hi;        // (lists > 1: list x is [u_lo[x], u_hi[x]), see unit_walk)
    int32_t lists = 1;
    int32_t n_rows;
    const int32_t *rowptr;
    const int32_t *col;
    const float *val;           // nullptr: all ones
    const void *X;
    void *Y;
    int32_t *arg;               // max: edge id of each output maximum (nullable)
    float *partials;
    int32_t *parg;              // max: edge id of each partial maximum
    int64_t pstride;
    int64_t F;
    uint64_t x_bytes;           // size of X, bounds the buffer gathers
    int32_t slab;
    int32_t log2S;
    int32_t mean;               // sum / mean: divide whole rows by their degree
    float bsign;                // ADDOP: message x + bsign * val (+1 add, -1 subtract)
    const float *bias;          // epilogue: Y = act(reduced + bias), bias nullable
    int32_t act;
};

// Descriptor {row, first edge, end edge, partial slot} of unit u (an empty
// unit past the end, so prefetching one unit ahead needs no branch around it).
__device__ __forceinline__ int4 fetch_unit(const SpmmArgs &a, int64_t u, int64_t hi)
{
    if (u >= hi) return make_int4(0, 0, 0, -1);
    if (a.units) return a.units[u];
    const int r = (int)u;
    return make_int4(r, a.rowptr[r], a.rowptr[r + 1], -1);
}

// Stores N edge ids (16-byte stores when N is a multiple of four; the offsets
// and the base are then 16-byte aligned).
template <int N>
__device__ __forceinline__ void store_ids(int32_t *__restrict__ p, int64_t i, const int32_t (&v)[N])
{
    if constexpr (N % 4 == 0) {
#pragma unroll
        for (int e = 0; e < N; e += 4)
            *reinterpret_cast<int4 *>(p + i + e) = make_int4(v[e], v[e + 1], v[e + 2], v[e + 3]);
    } else {
#pragma unroll
        for (int e = 0; e < N; ++e) p[i + e] = v[e];
    }
}

// The message of edge k is val[k] * x (ADDOP = false; copy is val = 1) or
// x + bsign * val[k] (ADDOP = true: add, subtract).
// MAXR = false: sum of the messages (mean scales whole rows by 1 / degree);
// MAXR = true: maximum of the messages, each rounded once to fp32, edges
// taken in CSR order, the first edge kept unconditionally and a later one
// only if strictly greater, so the recorded edge is the first that attains
// the maximum.
template <typename TX, typename TY, int VEC, int CH, bool BUF, bool MAXR, bool ADDOP>
__global__ __launch_bounds__(kSpmmBlock) void k_spmm(SpmmArgs a)
{
    constexpr int U = (VEC == 1 ? 16 : 8) / CH;
    constexpr int AC = MAXR ? CH : 1;
    constexpr int AV = MAXR ? VEC : 1;
    const int log2S = a.log2S;
    const int S = 1 << log2S;
    const int lane = lane_id();
    const int lig = lane & (S - 1);
    const int gbase = lane & ~(S - 1);
    const UnitWalk walk = unit_walk(a.units != nullptr, a.u_lo, a.u_hi, a.lists, a.n_rows,
                                    kSpmmBlock >> log2S, threadIdx.x >> log2S);
    const int64_t stride = walk.step;
    const int64_t hi = walk.end;

    const int64_t f0 = (int64_t)blockIdx.y * a.slab;
    const int64_t f_end = (f0 + a.slab < a.F) ? f0 + a.slab : a.F;
    int64_t fe[CH];
    bool act[CH];
#pragma unroll
    for (int c = 0; c < CH; ++c) {
        fe[c] = f0 + (int64_t)(c * S + lig) * VEC;
        act[c] = fe[c] < f_end;
    }
    const RowGather<TX, VEC, BUF> X(a.X, a.x_bytes);
    const int32_t *__restrict__ col = a.col;
    const float *__restrict__ val = a.val;

    // Resident grid: sub-group i of a list runs its units i, i + stride, ...;
    // the units are sorted by length, so neighbouring sub-groups get equal work.
    // The loop is software-pipelined: the next unit's descriptor is fetched
    // when a unit starts and its first index chunk before the current output
    // is stored, so short units do not pay three dependent memory trips each.
    int64_t u = walk.first;
    if (u >= hi) return;
    int4 d = fetch_unit(a, u, hi);
    int c_cur = 0;
    float v_cur = 0.f;
    if (d.z > d.y) {
        // index loads are clamped to the unit's last edge instead of masked:
        // no branch, and lanes past the end are never read back
        const int k = d.y + lig < d.z - 1 ? d.y + lig : d.z - 1;
        c_cur = col[k];
        v_cur = val ? val[k] : 1.f;
    }
    for (;;) {
        const int64_t un = u + stride;
        const int4 dn = fetch_unit(a, un, hi);
        const int row = d.x, beg = d.y, end = d.z, part = d.w;
        float acc[CH][VEC];
        int32_t am[AC][AV];
#pragma unroll
        for (int c = 0; c < CH; ++c)
#pragma unroll
            for (int e = 0; e < VEC; ++e) acc[c][e] = 0.f;
#pragma unroll
        for (int c = 0; c < AC; ++c)
#pragma unroll
            for (int e = 0; e < AV; ++e) am[c][e] = -1;

        const int last = end - 1;
        for (int k0 = beg; k0 < end; k0 += S) {
            const int n = (end - k0 < S) ? end - k0 : S;
            const int k = k0 + S + lig < last ? k0 + S + lig : last;
            const int c_nxt = col[k];
            const float v_nxt = val ? val[k] : 1.f;
            for (int j = 0; j < n; j += U) {
                int cc[U];
                float vv[U];
                bool ok[U];
#pragma unroll
                for (int t = 0; t < U; ++t) {
                    ok[t] = j + t < n;
                    const int src = gbase + (ok[t] ? j + t : j);
                    cc[t] = lane_bcast(c_cur, src);
                    vv[t] = lane_bcast(v_cur, src);
                    // a masked slot must add nothing: its gathered x is 0, so its w is too
                    if constexpr (ADDOP) vv[t] = ok[t] ? vv[t] * a.bsign : 0.f;
                }
                float xv[U][CH][VEC];
#pragma unroll
                for (int t = 0; t < U; ++t)
#pragma unroll
                    for (int c = 0; c < CH; ++c)
                        X.load((int64_t)cc[t] * a.F + fe[c], ok[t] && act[c], xv[t][c]);
                if constexpr (MAXR) {
#pragma unroll
                    for (int t = 0; t < U; ++t)
#pragma unroll
                        for (int c = 0; c < CH; ++c)
#pragma unroll
                            for (int e = 0; e < VEC; ++e) {
                                const float p = ADDOP ? xv[t][c][e] + vv[t] : vv[t] * xv[t][c][e];
                                const bool take = ok[t] && (am[c][e] < 0 || p > acc[c][e]);
                                acc[c][e] = take ? p : acc[c][e];
                                am[c][e] = take ? k0 + j + t : am[c][e];
                            }
                } else {
#pragma unroll
                    for (int t = 0; t < U; ++t)
#pragma unroll
                        for (int c = 0; c < CH; ++c)
#pragma unroll
                            for (int e = 0; e < VEC; ++e) {
                                if constexpr (ADDOP) acc[c][e] += xv[t][c][e] + vv[t];
                                else acc[c][e] = fmaf(vv[t], xv[t][c][e], acc[c][e]);
                            }
                }
            }
            c_cur = c_nxt;
            v_cur = v_nxt;
        }

        // first index chunk of the next unit, issued before this unit's stores
        if (dn.z > dn.y) {
            const int k = dn.y + lig < dn.z - 1 ? dn.y + lig : dn.z - 1;
            c_cur = col[k];
            v_cur = val ? val[k] : 1.f;
        }
        if (part < 0) {
            TY *__restrict__ Y = static_cast<TY *>(a.Y);
            if (!MAXR && a.mean && end > beg) {
                const float r = 1.f / (float)(end - beg);
#pragma unroll
                for (int c = 0; c < CH; ++c)
#pragma unroll
                    for (int e = 0; e < VEC; ++e) acc[c][e] *= r;
            }
#pragma unroll
            for (int c = 0; c < CH; ++c) {
                if (!act[c]) continue;
                epilogue<VEC>(acc[c], a.bias, a.act, fe[c]);
                store_out<TY, VEC>(Y, (int64_t)row * a.F + fe[c], acc[c]);
                if constexpr (MAXR) {
                    if (a.arg) store_ids<VEC>(a.arg, (int64_t)row * a.F + fe[c], am[c]);
                }
            }
        } else {
#pragma unroll
            for (int c = 0; c < CH; ++c) {
                if (!act[c]) continue;
                store_vec<float, VEC>(a.partials, (int64_t)part * a.pstride + fe[c], acc[c]);
                if constexpr (MAXR)
                    store_ids<VEC>(a.parg, (int64_t)part * a.pstride + fe[c], am[c]);
            }
        }
        if (un >= hi) break;
        u = un;
        d = dn;
    }
}

using SpmmKernel = void (*)(SpmmArgs);

// Kernel for (VEC, CH) of one variant.  Max outputs keep the input format or
// widen it to fp32 (each output is one fp32 message rounded once); the caller
// rejects other pairs.
template <typename TX, typename TY, bool BUF, bool MAXR, bool ADDOP>
SpmmKernel spmm_pick_vec(int vec, int ch)
{
    constexpr int V = (int)(16 / sizeof(TX));
    if (vec == 1) {
        if (ch == 1) return k_spmm<TX, TY, 1, 1, BUF, MAXR, ADDOP>;
        if (ch == 2) return k_spmm<TX, TY, 1, 2, BUF, MAXR, ADDOP>;
        return k_spmm<TX, TY, 1, 4, BUF, MAXR, ADDOP>;
    }
    if (ch == 1) return k_spmm<TX, TY, V, 1, BUF, MAXR, ADDOP>;
    if (ch == 2) return k_spmm<TX, TY, V, 2, BUF, MAXR, ADDOP>;
    return k_spmm<TX, TY, V, 4, BUF, MAXR, ADDOP>;
}

template <typename TX, bool BUF, bool MAXR, bool ADDOP>
SpmmKernel spmm_pick_y(int ydt, int vec, int ch)
{
    if (ydt == COGDL_F32) return spmm_pick_vec<TX, float, BUF, MAXR, ADDOP>(vec, ch);
    if constexpr (MAXR) {
        return spmm_pick_vec<TX, TX, BUF, MAXR, ADDOP>(vec, ch);
    } else {
        if (ydt == COGDL_BF16) return spmm_pick_vec<TX, bf16_t, BUF, MAXR, ADDOP>(vec, ch);
        return spmm_pick_vec<TX, f16_t, BUF, MAXR, ADDOP>(vec, ch);
    }
}

template <bool MAXR, bool ADDOP>
SpmmKernel spmm_pick(int xdt, int ydt, int vec, int ch, bool buf)
{
    if (buf) {
        if (xdt == COGDL_F32) return spmm_pick_y<float, true, MAXR, ADDOP>(ydt, vec, ch);
        if (xdt == COGDL_BF16) return spmm_pick_y<bf16_t, true, MAXR, ADDOP>(ydt, vec, ch);
        return spmm_pick_y<f16_t, true, MAXR, ADDOP>(ydt, vec, ch);
    }
    if (xdt == COGDL_F32) return spmm_pick_y<float, false, MAXR, ADDOP>(ydt, vec, ch);
    if (xdt == COGDL_BF16) return spmm_pick_y<bf16_t, false, MAXR, ADDOP>(ydt, vec, ch);
    return spmm_pick_y<f16_t, false, MAXR, ADDOP>(ydt, vec, ch);
}

// The variants instantiated in gspmm.hip (max of products, sum and max of
// x + bsign * val); the sum of products is instantiated in spmm.hip.
SpmmKernel gspmm_pick(bool maxr, bool addop, int xdt, int ydt, int vec, int ch, bool buf);

}  // namespace cogdl
