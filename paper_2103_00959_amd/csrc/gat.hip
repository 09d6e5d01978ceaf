// Attention path of section 2.2: the SDDMM of per-head scores (additive GAT
// form), LeakyReLU, the edge-wise softmax over the edges of each destination
// row, and the multi-head SpMM that aggregates neighbour features with one
// weight per edge and head.
//
// cogdl_sddmm_edge_softmax (alpha only): a wavefront per long unit, laid out
// as (edge slot, head) so that 64/H edges are scored per step with as many
// steps in flight as the unit needs (2 to 16); each lane keeps an online
// softmax state (m, z), the states of one head are merged across slots with
// lane exchanges (a butterfly when H is a power of two), and alpha =
// exp(e - m) / z is written with coalesced stores, from registers when the
// unit fitted in one pass.  The tiny tail runs a quad of lanes per unit (each
// edge's H scores gathered as whole words) or, for other head counts, 4H
// lanes in the (edge slot, head) layout.
//
// cogdl_gat_aggregate (fused): the gather mapping of the SpMM (S lanes x VEC
// features per edge row).  Every lane computes the weight of its own head for
// each gathered edge and folds it into an online softmax: when a batch of U
// edges raises the running maximum, the accumulators and the running sum are
// rescaled once.  The unnormalized sum is divided by z at the end, so alpha
// never has to reach memory.  Neighbour groups of split rows leave (acc, m, z)
// per group; a fixed-order merge combines them (the log-sum-exp rule).
#include "gat_kernel.hpp"

namespace cogdl {
namespace {

constexpr int kBlock = kGatBlock;

// --------------------------------------------------- softmax-only kernels

struct SoftArgs {
    const int4 *units;
    const int32_t *u_lo;        // with units: this launch runs units [*u_lo, *u_hi)
    const int32_t *u_hi;        // (lists > 1: list x is [u_lo[x], u_hi[x]), see unit_walk)
    int32_t lists = 1;
    int32_t n_rows;
    const int32_t *rowptr;
    const int32_t *col;
    int32_t H;
    const float *s_dst;
    const float *s_src;
    float slope;
    float *alpha;
    float *gstats;
    int32_t sstride;
    int32_t log2S;              // k_softmax: lanes per unit
    const int4 *part_units;     // k_alpha_split: {row, beg, end, split}
    const int32_t *n_parts;
    const float *rstats;        // per split row: m[max_heads], z[max_heads]
};

// Merge the (m, z) states of the lanes of one S-lane sub-group (base gbase)
// that hold the same head h = lane % H: slots are (lane - gbase) / H, S / H of
// them.  Result in every lane of head h.
__device__ __forceinline__ void merge_slots(float &m, float &z, int H, int S, int gbase)
{
    if ((H & (H - 1)) == 0) {
        for (int off = H; off < S; off <<= 1) {
            const float m2 = lane_xor(m, off);
            const float z2 = lane_xor(z, off);
            softmax_merge(m, z, m2, z2);
        }
        return;
    }
    const int slots = S / H;
    const int h = (lane_id() - gbase) % H;
    float mm = -INFINITY, zz = 0.f;
    for (int s = 0; s < slots; ++s) {
        const float m2 = lane_bcast(m, gbase + s * H + h);
        const float z2 = lane_bcast(z, gbase + s * H + h);
        softmax_merge(mm, zz, m2, z2);
    }
    m = mm;
    z = zz;
}

__device__ __forceinline__ int4 fetch_soft_unit(const SoftArgs &a, int64_t u, int64_t hi)
{
    if (u >= hi) return make_int4(0, 0, 0, -1);
    if (a.units) return a.units[u];
    const int r = (int)u;
    return make_int4(r, a.rowptr[r], a.rowptr[r + 1], -1);
}

// One work unit of k_softmax with RR steps per pass: S lanes laid out as
// (edge slot, head), slots = S / H edges per step.  Whole rows: alpha written
// (from the scores kept in registers when the row fits in one pass of RR
// steps, else by a second, batched sweep over the scores parked in alpha);
// neighbour groups: (m, z) per head into gstats, scores parked.  Stored
// weights go through alpha_value.  A lane's weight indices advance by a fixed
// step per edge slot step, formed once per pass.
template <int RR>
__device__ __forceinline__ void soft_unit(const SoftArgs &a, int4 d, int H, int S, int slots, int h, int slot,
                                          bool live, int gbase)
{
    const int32_t *__restrict__ col = a.col;
    const int row = d.x, beg = d.y, end = d.z, part = d.w;
    const float sd = a.s_dst[(int64_t)row * H + h];
    const int64_t hstep = slots * H;    // index step from one edge slot step to the next
    // A unit longer than one pass parks its raw scores in alpha and the
    // second sweep reads them back (each lane only its own elements):
    // a contiguous re-read instead of a second random gather of s_src.
    const bool park = end - beg > RR * slots || part >= 0;
    float m = -INFINITY, z = 0.f;
    float ev[RR];
    for (int k0 = beg + slot; k0 < end + slot; k0 += RR * slots) {
        const int64_t i0 = (int64_t)k0 * H + h;    // alpha index of this lane's first edge of the pass
        int cc[RR];
#pragma unroll
        for (int r = 0; r < RR; ++r) {
            const int k = k0 + r * slots;
            cc[r] = col[k < end ? k : end - 1];
        }
        float mb = m;
#pragma unroll
        for (int r = 0; r < RR; ++r) {
            const float sv = a.s_src[(int64_t)cc[r] * H + h];
            ev[r] = (live && k0 + r * slots < end) ? leaky_relu(sd + sv, a.slope) : -INFINITY;
            mb = fmaxf(mb, ev[r]);
        }
        if (park && live) {
#pragma unroll
            for (int r = 0; r < RR; ++r) {
                const int k = k0 + r * slots;
                if (k < end) a.alpha[i0 + r * hstep] = ev[r];
            }
        }
        if (mb > m) {
            z *= __expf(m - mb);
            m = mb;
        }
        // masked steps (score -inf) add nothing, also while m is still -inf
        float zb = 0.f;
#pragma unroll
        for (int r = 0; r < RR; ++r) zb += ev[r] == -INFINITY ? 0.f : __expf(ev[r] - m);
        z += zb;
    }
    if (!live) { m = -INFINITY; z = 0.f; }
    merge_slots(m, z, H, S, gbase);
    if (part >= 0) {
        if (slot == 0) {
            a.gstats[(int64_t)part * a.sstride + h] = m;
            a.gstats[(int64_t)part * a.sstride + (a.sstride >> 1) + h] = z;
        }
    } else if (live && end > beg) {
        const float rz = 1.f / z;
        if (!park) {
            // one pass: this lane's scores are still in ev
            const int64_t i0 = (int64_t)(beg + slot) * H + h;
#pragma unroll
            for (int r = 0; r < RR; ++r) {
                const int k = beg + slot + r * slots;
                if (k < end) a.alpha[i0 + r * hstep] = alpha_value(ev[r], m, rz);
            }
        } else {
            // the parked scores, same lane-to-element map as when they were written
            for (int k0 = beg + slot; k0 < end; k0 += RR * slots) {
                const int64_t i0 = (int64_t)k0 * H + h;
                float e[RR];
#pragma unroll
                for (int r = 0; r < RR; ++r) {
                    const int k = k0 + r * slots;
                    e[r] = k < end ? a.alpha[i0 + r * hstep] : 0.f;
                }
#pragma unroll
                for (int r = 0; r < RR; ++r) {
                    const int k = k0 + r * slots;
                    if (k < end) a.alpha[i0 + r * hstep] = alpha_value(e[r], m, rz);
                }
            }
        }
    }
}

// A unit with the fewest steps per pass out of RR, 2 RR, ..., R that holds it
// in one pass (R for longer ones).
template <int RR, int R>
__device__ __forceinline__ void soft_class(const SoftArgs &a, int4 d, int H, int S, int slots, int h, int slot,
                                           bool live, int gbase)
{
    if constexpr (RR >= R) {
        soft_unit<R>(a, d, H, S, slots, h, slot, live, gbase);
    } else {
        if (d.z - d.y <= RR * slots) soft_unit<RR>(a, d, H, S, slots, h, slot, live, gbase);
        else soft_class<2 * RR, R>(a, d, H, S, slots, h, slot, live, gbase);
    }
}

// S lanes per work unit, resident grid, each sub-group striding over the
// units with the next descriptor prefetched.  Each unit runs with the fewest
// steps per pass out of R0, 2 R0, ..., R that hold it in one pass: a short
// unit issues fewer gathers for steps past its end, a longer one is kept out
// of parking.
template <int R, int R0>
__global__ __launch_bounds__(kBlock) void k_softmax(SoftArgs a)
{
    const int log2S = a.log2S;
    const int S = 1 << log2S;
    const int lane = lane_id();
    const int lig = lane & (S - 1);
    const int gbase = lane & ~(S - 1);
    const int H = a.H;
    const int slots = S / H;
    const int h = lig % H;
    const int slot = lig / H;
    const bool live = slot < slots;
    const UnitWalk walk = unit_walk(a.units != nullptr, a.u_lo, a.u_hi, a.lists, a.n_rows,
                                    kBlock >> log2S, threadIdx.x >> log2S);
    const int64_t stride = walk.step;
    const int64_t hi = walk.end;

    int64_t u = walk.first;
    if (u >= hi) return;
    int4 d = fetch_soft_unit(a, u, hi);
    for (;;) {
        const int64_t un = u + stride;
        const int4 dn = fetch_soft_unit(a, un, hi);
        soft_class<R0, R>(a, d, H, S, slots, h, slot, live, gbase);
        if (un >= hi) break;
        u = un;
        d = dn;
    }
}

// The H scores of one node or edge as whole 8- and 16-byte words (H = 1, 2, 4
// or 8, p aligned to min(4 H, 16) bytes).
template <int H>
__device__ __forceinline__ void load_heads(const float *__restrict__ p, float (&v)[H])
{
    if constexpr (H == 1) {
        v[0] = p[0];
    } else if constexpr (H == 2) {
        const float2 t = *reinterpret_cast<const float2 *>(p);
        v[0] = t.x;
        v[1] = t.y;
    } else {
#pragma unroll
        for (int q = 0; q < H / 4; ++q) {
            const float4 t = reinterpret_cast<const float4 *>(p)[q];
            v[4 * q] = t.x;
            v[4 * q + 1] = t.y;
            v[4 * q + 2] = t.z;
            v[4 * q + 3] = t.w;
        }
    }
}

template <int H>
__device__ __forceinline__ void store_heads(float *__restrict__ p, const float (&v)[H])
{
    if constexpr (H == 1) {
        p[0] = v[0];
    } else if constexpr (H == 2) {
        *reinterpret_cast<float2 *>(p) = make_float2(v[0], v[1]);
    } else {
#pragma unroll
        for (int q = 0; q < H / 4; ++q)
            reinterpret_cast<float4 *>(p)[q] = make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
    }
}

// Tiny units (at most kTinyUnit = 8 edges) for H = 1, 2, 4 or 8 heads: a quad
// of lanes per unit (16 units per wavefront), each lane two edges (beg + lane
// + 4 r) with all H source scores gathered as whole words.  The unit is one
// pass: its maximum per head over the quad first (two DPP butterfly levels),
// then the sum of exp(e - m), then the weights; a neighbour group of a split
// row parks its raw scores and writes its (m, z) instead, as in k_softmax.
template <int H>
__global__ __launch_bounds__(kBlock) void k_softmax_quads(SoftArgs a)
{
    constexpr int L = 4, R = 2;
    static_assert(L * R >= kTinyUnit, "one pass covers a tiny unit");
    const int sub = lane_id() & (L - 1);
    const UnitWalk walk = unit_walk(a.units != nullptr, a.u_lo, a.u_hi, a.lists, a.n_rows, kBlock / L,
                                    threadIdx.x / L);
    const int64_t stride = walk.step;
    const int64_t hi = walk.end;
    const int32_t *__restrict__ col = a.col;
    const float *__restrict__ s_src = a.s_src;
    float *__restrict__ alpha = a.alpha;

    int64_t u = walk.first;
    if (u >= hi) return;
    int4 d = fetch_soft_unit(a, u, hi);
    for (;;) {
        const int64_t un = u + stride;
        const int4 dn = fetch_soft_unit(a, un, hi);
        const int row = d.x, beg = d.y, end = d.z, part = d.w;
        if (end > beg) {
            float sd[H];
            load_heads<H>(a.s_dst + (int64_t)row * H, sd);
            int cc[R];
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const int k = beg + sub + L * r;
                cc[r] = col[k < end ? k : end - 1];
            }
            float e[R][H];
#pragma unroll
            for (int r = 0; r < R; ++r) {
                float sv[H];
                load_heads<H>(s_src + (int64_t)cc[r] * H, sv);
                const bool in = beg + sub + L * r < end;
#pragma unroll
                for (int h = 0; h < H; ++h) e[r][h] = in ? leaky_relu(sd[h] + sv[h], a.slope) : -INFINITY;
            }
            float m[H], z[H];
#pragma unroll
            for (int h = 0; h < H; ++h) {
                float mh = e[0][h];
#pragma unroll
                for (int r = 1; r < R; ++r) mh = fmaxf(mh, e[r][h]);
                mh = group_reduce(mh, L, [](float x, float y) { return fmaxf(x, y); });
                float zh = 0.f;
#pragma unroll
                for (int r = 0; r < R; ++r) zh += e[r][h] == -INFINITY ? 0.f : __expf(e[r][h] - mh);
                m[h] = mh;
                z[h] = group_reduce(zh, L, [](float x, float y) { return x + y; });
            }
            if (part >= 0) {
                if (sub == 0) {
#pragma unroll
                    for (int h = 0; h < H; ++h) {
                        a.gstats[(int64_t)part * a.sstride + h] = m[h];
                        a.gstats[(int64_t)part * a.sstride + (a.sstride >> 1) + h] = z[h];
                    }
                }
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    const int k = beg + sub + L * r;
                    if (k < end) store_heads<H>(alpha + (int64_t)k * H, e[r]);
                }
            } else {
                float rz[H];
#pragma unroll
                for (int h = 0; h < H; ++h) rz[h] = 1.f / z[h];
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    const int k = beg + sub + L * r;
                    if (k < end) {
                        float o[H];
#pragma unroll
                        for (int h = 0; h < H; ++h) o[h] = alpha_value(e[r][h], m[h], rz[h]);
                        store_heads<H>(alpha + (int64_t)k * H, o);
                    }
                }
            }
        }
        if (un >= hi) break;
        u = un;
        d = dn;
    }
}

// Per split row: merge the (m, z) of its groups in slot order (64/H chains,
// then the chains in order) into rstats.
__device__ __forceinline__ void merge_groups(const float *gstats, int sstride, int p0, int np,
                                             int H, float &m, float &z)
{
    const int lane = lane_id();
    const int chains = kWave / H;
    const int h = lane % H;
    const int chain = lane / H;
    m = -INFINITY;
    z = 0.f;
    if (chain < chains) {
        for (int g = chain; g < np; g += chains) {
            const float *st = gstats + (int64_t)(p0 + g) * sstride;
            softmax_merge(m, z, st[h], st[(sstride >> 1) + h]);
        }
    }
    float mm = -INFINITY, zz = 0.f;
    for (int s = 0; s < chains; ++s) {
        const int src = s * H + h;
        const float m2 = lane_bcast(m, src < kWave ? src : h);
        const float z2 = lane_bcast(z, src < kWave ? src : h);
        softmax_merge(mm, zz, m2, z2);
    }
    m = mm;
    z = zz;
}

__global__ __launch_bounds__(kBlock) void k_softmax_merge(const int4 *__restrict__ split_rows,
                                                          const int32_t *__restrict__ n_split,
                                                          const float *__restrict__ gstats,
                                                          int sstride, int H,
                                                          float *__restrict__ rstats)
{
    const int lane = lane_id();
    const int64_t waves = (int64_t)gridDim.x * (kBlock / kWave);
    const int32_t ns = *n_split;
    for (int64_t s = (int64_t)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave; s < ns; s += waves) {
        const int4 d = split_rows[s];
        float m, z;
        merge_groups(gstats, sstride, d.y, d.z, H, m, z);
        if (lane < H) {
            rstats[s * sstride + lane] = m;
            rstats[s * sstride + (sstride >> 1) + lane] = z;
        }
    }
}

// alpha for the edges of split rows, one wavefront per neighbour group, from
// the raw scores that k_softmax or k_gat parked in alpha.
__global__ __launch_bounds__(kBlock) void k_alpha_split(SoftArgs a)
{
    const int lane = lane_id();
    const int H = a.H;
    const int eps = kWave / H;
    const int h = lane % H;
    const int slot = lane / H;
    if (slot >= eps) return;
    const int64_t waves = (int64_t)gridDim.x * (kBlock / kWave);
    const int32_t np = *a.n_parts;
    for (int64_t p = (int64_t)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave; p < np; p += waves) {
        const int4 d = a.part_units[p];
        const float m = a.rstats[(int64_t)d.w * a.sstride + h];
        const float rz = 1.f / a.rstats[(int64_t)d.w * a.sstride + (a.sstride >> 1) + h];
        alpha_from_parked<8>(a.alpha, 0, a.alpha, H, h, m, rz, d.y, d.z, slot, eps);
    }
}

// GAT split rows: combine the groups' unnormalized sums with the log-sum-exp
// rule, write Y and the row's (m, z) for the alpha pass.  A wavefront per
// split row: it merges the groups' (m, z) states, then group g, scaled by
// exp(m_g - m), goes to chain g mod 4; the chains add their groups in
// increasing order and are combined as (c0 + c1) + (c2 + c3).
template <typename TY, int VEC>
__global__ __launch_bounds__(kBlock) void k_gat_reduce(const int4 *__restrict__ split_rows,
                                                       const int32_t *__restrict__ n_split,
                                                       const float *__restrict__ partials,
                                                       int64_t pstride,
                                                       const float *__restrict__ gstats,
                                                       int sstride, int H, int D,
                                                       float *__restrict__ rstats,
                                                       float *__restrict__ row_stats,
                                                       const float *__restrict__ bias, int act_code,
                                                       TY *__restrict__ Y)
{
    const int lane = lane_id();
    const int64_t W = (int64_t)H * D;
    const int32_t ns = *n_split;
    const int64_t waves = (int64_t)gridDim.x * (kBlock / kWave);
    for (int64_t s = (int64_t)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave; s < ns;
         s += waves) {
        const int4 d = split_rows[s];
        const int64_t row = d.x;
        const int p0 = d.y, np = d.z;
        float m, z;
        merge_groups(gstats, sstride, p0, np, H, m, z);   // lane h holds head h
        if (lane < H) {
            rstats[s * sstride + lane] = m;
            rstats[s * sstride + (sstride >> 1) + lane] = z;
            if (row_stats) {                  // (m, 1/z), as the split-row alpha pass forms them
                row_stats[row * 2 * H + lane] = m;
                row_stats[row * 2 * H + H + lane] = 1.f / z;
            }
        }
        for (int64_t fb = 0; fb < W; fb += kWave * VEC) {
            const int64_t f = fb + (int64_t)lane * VEC;
            const bool act = f < W;
            const int h = act ? (int)(f / D) : 0;
            const float M = lane_bcast(m, h);
            const float rZ = 1.f / lane_bcast(z, h);
            if (!act) continue;
            float c[4][VEC];
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int e = 0; e < VEC; ++e) c[j][e] = 0.f;
            int g = 0;
            for (; g + 4 <= np; g += 4) {
                float x[4][VEC], sc[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int64_t q = p0 + g + j;
                    sc[j] = __expf(gstats[q * sstride + h] - M);
                    load_vec<float, VEC>(partials, q * pstride + f, x[j]);
                }
#pragma unroll
                for (int j = 0; j < 4; ++j)
#pragma unroll
                    for (int e = 0; e < VEC; ++e) c[j][e] = fmaf(x[j][e], sc[j], c[j][e]);
            }
#pragma unroll
            for (int j = 0; j < 3; ++j) {
                if (g + j < np) {
                    const int64_t q = p0 + g + j;
                    const float sc = __expf(gstats[q * sstride + h] - M);
                    float x[VEC];
                    load_vec<float, VEC>(partials, q * pstride + f, x);
#pragma unroll
                    for (int e = 0; e < VEC; ++e) c[j][e] = fmaf(x[e], sc, c[j][e]);
                }
            }
            float v[VEC];
#pragma unroll
            for (int e = 0; e < VEC; ++e) v[e] = ((c[0][e] + c[1][e]) + (c[2][e] + c[3][e])) * rZ;
            epilogue<VEC>(v, bias, act_code, f);
            store_out<TY, VEC>(Y, row * W + f, v);
        }
    }
}

unsigned grid_waves(int64_t work)
{
    int64_t b = (work + (kBlock / kWave) - 1) / (kBlock / kWave);
    if (b > 2048) b = 2048;
    if (b < 1) b = 1;
    return (unsigned)b;
}

cogdl_status check_graph(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *rowptr,
                         const int32_t *col, int32_t H)
{
    if (n_rows < 0 || n_cols < 0 || nnz < 0) return COGDL_ERR_INVALID;
    if (H < 1 || H > COGDL_MAX_HEADS) return COGDL_ERR_INVALID;
    if (nnz > COGDL_MAX_NNZ) return COGDL_ERR_TOO_LARGE;
    if (n_rows > 0 && !rowptr) return COGDL_ERR_INVALID;
    if (nnz > 0 && (!col || n_rows == 0 || n_cols == 0)) return COGDL_ERR_INVALID;
    return COGDL_OK;
}

cogdl_status gat_aggregate_impl(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *rowptr,
                                const int32_t *col, int32_t H, int32_t D, const float *s_dst,
                                const float *s_src, const float *a_src, float negative_slope,
                                const float *alpha_in, const void *X, cogdl_dtype x_dtype, void *Y,
                                cogdl_dtype y_dtype, float *alpha_out, float *row_stats,
                                const float *bias, cogdl_act act, const cogdl_plan *plan,
                                hipStream_t stream);

}  // namespace
}  // namespace cogdl

using namespace cogdl;

extern "C" {

cogdl_status cogdl_sddmm_edge_softmax(int32_t n_rows, int32_t n_cols, int64_t nnz,
                                      const int32_t *rowptr, const int32_t *col, int32_t H,
                                      const float *s_dst, const float *s_src, float negative_slope,
                                      float *alpha, const cogdl_plan *plan, hipStream_t stream)
{
    cogdl_status st = check_graph(n_rows, n_cols, nnz, rowptr, col, H);
    if (st != COGDL_OK) return st;
    if (n_rows > 0 && !s_dst) return COGDL_ERR_INVALID;
    if (nnz > 0 && (!s_src || !alpha)) return COGDL_ERR_INVALID;
    const Plan *P = plan_of(plan);
    if (P && (P->n_rows != n_rows || P->nnz != nnz || P->max_heads < H)) return COGDL_ERR_PLAN;
    if (nnz == 0) return COGDL_OK;

    SoftArgs a{};
    a.units = P ? P->units : nullptr;
    if (P) set_units(a, long_units(*P));
    a.n_rows = n_rows;
    a.rowptr = rowptr;
    a.col = col;
    a.H = H;
    a.s_dst = s_dst;
    a.s_src = s_src;
    a.slope = negative_slope;
    a.alpha = alpha;
    a.gstats = P ? P->gstats : nullptr;
    a.sstride = P ? 2 * P->max_heads : 0;
    a.part_units = P ? P->part_units : nullptr;
    a.n_parts = P ? P->n_parts_dev() : nullptr;
    a.rstats = P ? P->rstats : nullptr;
    // Units with more than kTinyUnit edges: a wavefront each, up to 16 steps of
    // 64 / H edges in flight.  The sorted tail of tiny units: a quad of lanes
    // each (or 4H lanes, at most 64, two steps), so that one pass covers a unit
    // of kTinyUnit edges.
    const int64_t units = P ? P->cap_units : n_rows;
    auto launch = [&](const char *name, void (*k)(SoftArgs), const SoftArgs &args) {
        const int64_t upb = kBlock >> args.log2S;
        int64_t blocks = (units + upb - 1) / upb;
        const int64_t res = resident_blocks(reinterpret_cast<const void *>(k), kBlock);
        if (blocks > res) blocks = res;
        blocks = list_grid(blocks, args.lists);
        COGDL_LAUNCH(name, k, (unsigned)blocks, kBlock, stream, args);
        return COGDL_OK;
    };
    a.log2S = 6;
    st = launch("softmax", k_softmax<16, 2>, a);
    if (st != COGDL_OK) return st;
    if (P) {
        SoftArgs b = a;
        set_units(b, tiny_units(*P));
        // a quad per unit where the heads fill whole words, else 4H lanes as
        // (edge slot, head), two steps
        void (*k_tiny)(SoftArgs) = nullptr;
        const uintptr_t words = (uintptr_t)s_dst | (uintptr_t)s_src | (uintptr_t)alpha;
        if (words % (4 * (H < 4 ? H : 4)) == 0) {
            if (H == 1) k_tiny = k_softmax_quads<1>;
            else if (H == 2) k_tiny = k_softmax_quads<2>;
            else if (H == 4) k_tiny = k_softmax_quads<4>;
            else if (H == 8) k_tiny = k_softmax_quads<8>;
        }
        b.log2S = k_tiny ? 2 : log2i(next_pow2(4 * H) < kWave ? next_pow2(4 * H) : kWave);
        if (!k_tiny) k_tiny = k_softmax<2, 2>;
        st = launch("softmax_tiny", k_tiny, b);
        if (st != COGDL_OK) return st;
        COGDL_LAUNCH("softmax_merge", k_softmax_merge, grid_waves(P->cap_split), kBlock, stream,
                     P->split_rows, P->n_split_dev(), P->gstats, a.sstride, H, P->rstats);
        COGDL_LAUNCH("softmax_alpha_split", k_alpha_split, grid_waves(P->cap_partials), kBlock,
                     stream, a);
    }
    return COGDL_OK;
}

cogdl_status cogdl_gat_aggregate(int32_t n_rows, int32_t n_cols, int64_t nnz,
                                 const int32_t *rowptr, const int32_t *col, int32_t H, int32_t D,
                                 const float *s_dst, const float *s_src, float negative_slope,
                                 const float *alpha_in, const void *X, cogdl_dtype x_dtype,
                                 void *Y, cogdl_dtype y_dtype, float *alpha_out,
                                 const cogdl_plan *plan, hipStream_t stream)
{
    return cogdl_gat_aggregate_act(n_rows, n_cols, nnz, rowptr, col, H, D, s_dst, s_src,
                                   negative_slope, alpha_in, X, x_dtype, Y, y_dtype, alpha_out,
                                   nullptr, COGDL_ACT_NONE, plan, stream);
}

cogdl_status cogdl_gat_aggregate_act(int32_t n_rows, int32_t n_cols, int64_t nnz,
                                     const int32_t *rowptr, const int32_t *col, int32_t H,
                                     int32_t D, const float *s_dst, const float *s_src,
                                     float negative_slope, const float *alpha_in, const void *X,
                                     cogdl_dtype x_dtype, void *Y, cogdl_dtype y_dtype,
                                     float *alpha_out, const float *bias, cogdl_act act,
                                     const cogdl_plan *plan, hipStream_t stream)
{
    return gat_aggregate_impl(n_rows, n_cols, nnz, rowptr, col, H, D, s_dst, s_src, nullptr,
                              negative_slope, alpha_in, X, x_dtype, Y, y_dtype, alpha_out, nullptr, bias,
                              act, plan, stream);
}

cogdl_status cogdl_gat_aggregate_proj(int32_t n_rows, int32_t n_cols, int64_t nnz,
                                      const int32_t *rowptr, const int32_t *col, int32_t H,
                                      int32_t D, const float *s_dst, const float *a_src,
                                      float negative_slope, const void *X, cogdl_dtype x_dtype,
                                      void *Y, cogdl_dtype y_dtype, const float *bias,
                                      cogdl_act act, const cogdl_plan *plan, hipStream_t stream)
{
    if (!a_src) return COGDL_ERR_INVALID;
    return gat_aggregate_impl(n_rows, n_cols, nnz, rowptr, col, H, D, s_dst, nullptr, a_src,
                              negative_slope, nullptr, X, x_dtype, Y, y_dtype, nullptr, nullptr, bias,
                              act, plan, stream);
}

cogdl_status cogdl_gat_aggregate_stats(int32_t n_rows, int32_t n_cols, int64_t nnz,
                                       const int32_t *rowptr, const int32_t *col, int32_t H,
                                       int32_t D, const float *s_dst, const float *s_src,
                                       const float *a_src, float negative_slope, const void *X,
                                       cogdl_dtype x_dtype, void *Y, cogdl_dtype y_dtype,
                                       float *row_stats, const float *bias, cogdl_act act,
                                       const cogdl_plan *plan, hipStream_t stream)
{
    // exactly one of s_src (scores given) and a_src (scores projected)
    if ((s_src == nullptr) == (a_src == nullptr)) return COGDL_ERR_INVALID;
    if (n_rows > 0 && !row_stats) return COGDL_ERR_INVALID;
    return gat_aggregate_impl(n_rows, n_cols, nnz, rowptr, col, H, D, s_dst, s_src, a_src,
                              negative_slope, nullptr, X, x_dtype, Y, y_dtype, nullptr, row_stats, bias,
                              act, plan, stream);
}

}  // extern "C"

namespace cogdl {
namespace {

cogdl_status gat_aggregate_impl(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *rowptr,
                                const int32_t *col, int32_t H, int32_t D, const float *s_dst,
                                const float *s_src, const float *a_src, float negative_slope,
                                const float *alpha_in, const void *X, cogdl_dtype x_dtype, void *Y,
                                cogdl_dtype y_dtype, float *alpha_out, float *row_stats,
                                const float *bias, cogdl_act act, const cogdl_plan *plan,
                                hipStream_t stream)
{
    if (act < COGDL_ACT_NONE || act > COGDL_ACT_ELU) return COGDL_ERR_INVALID;
    cogdl_status st = check_graph(n_rows, n_cols, nnz, rowptr, col, H);
    if (st != COGDL_OK) return st;
    if (D < 1) return COGDL_ERR_INVALID;
    if (!dtype_ok(x_dtype) || !dtype_ok(y_dtype)) return COGDL_ERR_DTYPE;
    const int64_t W = (int64_t)H * D;
    if (W > INT32_MAX) return COGDL_ERR_TOO_LARGE;
    const bool proj = a_src != nullptr;
    const bool soft = alpha_in == nullptr;
    if (soft && n_rows > 0 && !s_dst) return COGDL_ERR_INVALID;
    if (soft && !proj && nnz > 0 && !s_src) return COGDL_ERR_INVALID;
    if (proj && (!soft || alpha_out)) return COGDL_ERR_INVALID;
    if (row_stats && !soft) return COGDL_ERR_INVALID;
    if (n_rows > 0 && !Y) return COGDL_ERR_INVALID;
    if (nnz > 0 && !X) return COGDL_ERR_INVALID;
    const Plan *P = plan_of(plan);
    if (P && (P->n_rows != n_rows || P->nnz != nnz || P->max_feat < W || (soft && P->max_heads < H)))
        return COGDL_ERR_PLAN;
    if (n_rows == 0) return COGDL_OK;

    const bool aligned = ((uintptr_t)X % 16 == 0) && ((uintptr_t)Y % 16 == 0);
    RowMap m = row_map(W, dtype_bytes(x_dtype), D, aligned);
    if (m.S < H) {
        m.S = next_pow2(H);
        m.log2S = log2i(m.S);
        m.slab = m.S * m.ch * m.vec;
        m.n_slabs = (int)((W + m.slab - 1) / m.slab);
    }
    // projected source scores: each head on L = D / VEC adjacent lanes of one chunk
    const int hl = D / m.vec;
    if (proj && (m.vec * dtype_bytes(x_dtype) != 16 || D % m.vec != 0 || (hl & (hl - 1)) != 0 ||
                 hl > m.S))
        return COGDL_ERR_INVALID;
    GatArgs a{};
    a.units = P ? P->units : nullptr;
    a.n_rows = n_rows;
    a.rowptr = rowptr;
    a.col = col;
    a.H = H;
    a.D = D;
    a.W = W;
    a.s_dst = s_dst;
    a.s_src = s_src;
    a.slope = negative_slope;
    a.alpha_in = alpha_in;
    a.X = X;
    a.x_bytes = (uint64_t)n_cols * (uint64_t)W * (uint64_t)dtype_bytes(x_dtype);
    a.Y = Y;
    a.alpha_out = soft ? alpha_out : nullptr;
    a.row_stats = row_stats;
    a.bias = bias;
    a.act = act;
    a.a_src = a_src;
    a.park_cap = 0;
    a.partials = P ? P->partials : nullptr;
    a.pstride = P ? (P->max_feat + 7) / 8 * 8 : 0;
    a.gstats = P ? P->gstats : nullptr;
    a.sstride = P ? 2 * P->max_heads : 0;
    a.slab = m.slab;
    a.log2S = m.log2S;
    const bool buf = a.x_bytes <= kBufferMaxBytes;
    const int64_t units = P ? P->cap_units : n_rows;
    // tiny units (the sorted tail): S/4 lanes and four chunks per lane
    const bool tiny = P && m.ch == 1 && m.S >= 8 && m.S / 4 >= H && (!proj || hl <= m.S / 4);
    if (P) set_units(a, tiny ? long_units(*P) : all_units(*P));
    {
        const int64_t upb = kBlock >> m.log2S;
        // one chunk of 16-byte vectors with 8 lanes per head: the distributed-softmax
        // kernel (batches of 8 edges, one edge's score per lane)
        const bool dist = soft && m.ch == 1 && m.vec * dtype_bytes(x_dtype) == 16 && D % m.vec == 0 && hl == 8;
        GatKernel k = proj ? gat_pick_proj(x_dtype, y_dtype, m.ch, buf, dist)
                           : gat_pick<false>(x_dtype, y_dtype, m.vec, m.ch, buf, dist);
        int64_t blocks = (units + upb - 1) / upb;
        const int64_t res = resident_blocks(reinterpret_cast<const void *>(k), kBlock);
        if (blocks > res) blocks = res;
        blocks = list_grid(blocks, a.lists);
        // alpha wanted: each sub-group parks whole rows' scores in its share of kParkFloats of LDS
        const size_t shm = a.alpha_out ? sizeof(float) * kParkFloats : 0;
        a.park_cap = a.alpha_out ? kParkFloats / (kBlock >> m.log2S) : 0;
        COGDL_LAUNCH_SHM(proj ? "gat_proj" : "gat", k, dim3((unsigned)blocks, (unsigned)m.n_slabs), kBlock,
                         shm, stream, a);
    }
    if (tiny) {
        GatArgs b = a;
        set_units(b, tiny_units(*P));
        b.log2S = m.log2S - 2;
        const int64_t upb = kBlock >> b.log2S;
        GatKernel k = proj ? gat_pick_proj(x_dtype, y_dtype, 4, buf, false)
                           : gat_pick<false>(x_dtype, y_dtype, m.vec, 4, buf);
        int64_t blocks = (units + upb - 1) / upb;
        const int64_t res = resident_blocks(reinterpret_cast<const void *>(k), kBlock);
        if (blocks > res) blocks = res;
        blocks = list_grid(blocks, b.lists);
        const size_t shm = b.alpha_out ? sizeof(float) * kParkFloats : 0;
        b.park_cap = b.alpha_out ? kParkFloats / (kBlock >> b.log2S) : 0;
        COGDL_LAUNCH_SHM(proj ? "gat_proj_tiny" : "gat_tiny", k, dim3((unsigned)blocks, (unsigned)m.n_slabs),
                         kBlock, shm, stream, b);
    }
    if (!P) return COGDL_OK;

    if (!soft) return sum_reduce_launch("gat_sum_reduce", *P, W, Y, y_dtype, false, bias, act, stream);
    const unsigned rb = grid_waves(P->cap_split);
    const bool v4 = D % 4 == 0 && (uintptr_t)Y % (4 * dtype_bytes(y_dtype)) == 0;
#define COGDL_GAT_REDUCE(TY, V)                                                                  \
    COGDL_LAUNCH("gat_reduce", (k_gat_reduce<TY, V>), rb, kBlock, stream, P->split_rows,         \
                 P->n_split_dev(), P->partials, a.pstride, P->gstats, a.sstride, H, D, P->rstats, \
                 row_stats, bias, act, static_cast<TY *>(Y))
    if (y_dtype == COGDL_F32) {
        if (v4) COGDL_GAT_REDUCE(float, 4); else COGDL_GAT_REDUCE(float, 1);
    } else if (y_dtype == COGDL_BF16) {
        if (v4) COGDL_GAT_REDUCE(bf16_t, 4); else COGDL_GAT_REDUCE(bf16_t, 1);
    } else {
        if (v4) COGDL_GAT_REDUCE(f16_t, 4); else COGDL_GAT_REDUCE(f16_t, 1);
    }
#undef COGDL_GAT_REDUCE
    if (alpha_out) {
        SoftArgs sa{};
        sa.col = col;
        sa.H = H;
        sa.s_dst = s_dst;
        sa.s_src = s_src;
        sa.slope = negative_slope;
        sa.alpha = alpha_out;
        sa.sstride = a.sstride;
        sa.part_units = P->part_units;
        sa.n_parts = P->n_parts_dev();
        sa.rstats = P->rstats;
        COGDL_LAUNCH("gat_alpha_split", k_alpha_split, grid_waves(P->cap_partials), kBlock, stream,
                     sa);
    }
    return COGDL_OK;
}

}  // namespace
}  // namespace cogdl

