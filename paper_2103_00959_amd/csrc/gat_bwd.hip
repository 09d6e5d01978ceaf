// Backward pass of the attention path of section 2.2, and the dot-product
// SDDMM that carries the gradient to the attention matrix.
//
// For the loss gradient dY of Y[i,h,:] = sum_k alpha[k,h] X[col[k],h,:]:
//   dalpha[k,h] = <dY[i,h,:], X[j,h,:]>          SDDMM  A (.) (dY_h X_h^T)
//   c[i,h]      = sum_{k in row i} alpha[k,h] dalpha[k,h]
//   dscore[k,h] = f * alpha[k,h] * (dalpha[k,h] - c[i,h]),  f = 1 if the
//                 pre-activation s_dst[i,h] + s_src[j,h] > 0 else the slope
//   ds_dst[i,h] = sum_{k in row i} dscore[k,h]
//   ds_src[j,h] = sum_{k: col[k] = j} dscore[k,h]
//   dX[j,h,:]   = sum_{k: col[k] = j} alpha[k,h] dY[i,h,:]
//
// Pass 1 runs on the CSR units.  With the SpMM lane map (S lanes x VEC
// features of a row, the L = D / VEC lanes of a head side by side) each lane
// multiplies its dY elements into every gathered neighbour row and a
// reduction over the head's lanes completes the dot product, so the gathered
// rows are read once, as in the forward aggregation.  The lanes fold the row
// sum c as they go and park dalpha and u = f alpha of every edge (each value
// by a fixed lane: in LDS for a whole row that fits, else in memory); once c
// is complete, the same lanes read their own parked values back and write
// dscore and ds_dst.  A neighbour group of a split row leaves its share of c
// in the plan, and two small kernels finish those rows once every group is
// done.  dalpha and dscore are optional outputs: a layer's backward needs
// only ds_dst, ds_src and dX, and its kernels then park in LDS and the
// records alone.
//
// The pairs (alpha, dscore) of an edge's heads end side by side in the
// caller's edge workspace, 8 H bytes per edge in CSR order.  Pass 2 is the
// aggregation kernel run on the CSC (rows = source nodes), reaching each
// edge's pair through perm: one random 8H-byte record per edge instead of
// two 4H-byte rows in two arrays, each of which costs a cache line.  It sums
// dscore per head along the way: dX and ds_src in one sweep over dY.
#include "gat_kernel.hpp"

namespace cogdl {
namespace {

constexpr int kBlock = kGatBlock;

struct BwdArgs {
    const int4 *units;          // nullptr: one unit per row in row order
    const int32_t *u_lo;        // units [*u_lo, *u_hi), or per list (see unit_walk)
    const int32_t *u_hi;
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
    const float *alpha;         // forward weights [nnz][H]; nullptr: rebuilt from row_stats, or the SDDMM alone
    const float *row_stats;     // per row the forward's (m, 1/z) of each head, 2H floats (or nullptr)
    const void *X;              // gathered operand, n_cols x W
    uint64_t x_bytes;
    const void *P;              // row operand (dY), n_rows x W
    float *dalpha;              // [nnz][H], or nullptr (not written)
    float *dscore;              // [nnz][H], or nullptr (not written)
    float2 *rec;                // [nnz][H] parked pairs (see park_edge), then (alpha, dscore)
    int32_t park_cap;           // LDS floats per sub-group for whole rows' parked values (0: none)
    float *ds_dst;              // [n_rows][H]
    float *gstats;              // split rows: per partial slot c[max_heads], sum[max_heads]
    int32_t sstride;            // 2 * max_heads
    const int4 *part_units;     // {row, beg, end, split index} per partial slot
    const int32_t *n_parts;
    const int4 *split_rows;     // {row, first slot, #slots, degree}
    const int32_t *n_split;
    int32_t log2S;
    int32_t log2L;              // lanes per head (fast kernel)
};

__device__ __forceinline__ int4 fetch_bwd_unit(const BwdArgs &a, int64_t u, int64_t hi)
{
    if (u >= hi) return make_int4(0, 0, 0, -1);
    if (a.units) return a.units[u];
    const int r = (int)u;
    return make_int4(r, a.rowptr[r], a.rowptr[r + 1], -1);
}

// The score gradient of edge k and head h is f * alpha * (dalpha - c), with f
// the LeakyReLU slope at the pre-activation t and c the row's sum of alpha *
// dalpha.  Pass 1 parks u = f * alpha and dalpha, as ParkMode below lays
// out (c is not known yet); once c is known, dscore = u (dalpha - c), and the
// edge's record ends as (alpha, dscore).
__device__ __forceinline__ float park_value(float t, float slope, float al)
{
    return (t > 0.f ? 1.f : slope) * al;
}

__device__ __forceinline__ float parked_grad(float u, float da, float c) { return u * (da - c); }

// a + b rounded on its own: a sum of stored values is not fused with the
// multiply that produced b (so every kernel variant forms ds_dst from exactly
// the dscore values it writes).
__device__ __forceinline__ float add_stored(float a, float b)
{
#pragma clang fp contract(off)
    return a + b;
}

// How pass 1 parks what the fix-up needs (c is not known yet):
//   kParkSep:   alpha given, dalpha and dscore both written.  dalpha is in its
//               output, so u alone parks: in dscore for a split row, in the LDS
//               slot li for a whole row that fits its sub-group's share, else
//               beside alpha in the record (alpha, u).
//   kParkPair:  alpha given, an output left out: the pair (dalpha, u) parks in
//               LDS (slots 2 li, 2 li + 1) or in the record.
//   kParkStats: alpha rebuilt from the row's softmax state: the pair
//               (dalpha, v) parks, v = alpha on the LeakyReLU's positive branch
//               and -alpha on the other (alpha >= 0 here), so alpha = |v| and u
//               = f alpha come back with the same bits.
enum ParkMode { kParkSep, kParkPair, kParkStats };

// Fix-up of one parked edge-head: dscore from alpha, the parked u and
// dalpha, into the record and the dscore output (when there is one).
template <int PK>
__device__ __forceinline__ float finish_edge(const BwdArgs &a, int64_t i, float al, float u, float da, float c)
{
    const float g = parked_grad(u, da, c);
    if (PK == kParkSep || a.dscore) a.dscore[i] = g;
    a.rec[i] = make_float2(al, g);
    return g;
}

template <int PK>
__device__ __forceinline__ void park_edge(const BwdArgs &a, int64_t i, bool split, float al, float da, float u,
                                          float *lds, int li)
{
    if constexpr (PK == kParkSep) {
        if (split) a.dscore[i] = u;
        else if (lds) lds[li] = u;
        else a.rec[i] = make_float2(al, u);
    } else {
        const float v = PK == kParkStats ? (u == al ? al : -al) : u;
        if (lds) {
            lds[2 * li] = da;
            lds[2 * li + 1] = v;
        } else {
            a.rec[i] = make_float2(da, v);
        }
    }
}

// (alpha, u) from a kParkStats value v.
__device__ __forceinline__ float2 unpark_stats(float v, float slope)
{
    const float al = fabsf(v);
    return make_float2(al, signbit(v) ? slope * al : al);
}

// LDS floats of a rows workgroup for whole rows' parked values, shared by its sub-groups.
constexpr int kRowParkFloats = 4096;

// Pass 1, feature-parallel: one S-lane sub-group per unit, lane = VEC
// consecutive features, head h on lanes [h L, (h + 1) L).  Requires one
// chunk per lane (H * D <= S * VEC) and L a power of two.  Every edge k of a
// unit is owned by lane q = (k - beg) mod M of its head, M = min(L, U): that
// lane alone loads the edge's alpha and source score, adds its term of c, and
// parks its dalpha and u; the head's lanes then add up their shares of c.
// RS (batches of U = 8 edges, L >= 8): the head's partial dot products are
// reduce-scattered over aligned groups of 8 lanes, so lane q ends with the
// group's sum for its own edge q mod 8 (7 exchanges for the batch instead of
// 8 butterflies of log2 L), and L > 8 adds the groups by a butterfly.
template <typename TX, int VEC, bool BUF, bool DOT, bool RS = false, int PK = kParkSep>
__global__ __launch_bounds__(kBlock) void k_bwd_rows(BwdArgs a)
{
    constexpr int U = VEC == 1 ? 16 : 8;
    static_assert(!RS || U == 8, "reduce-scatter over batches of 8 edges");
    // 16-bit features stay packed: four dot2 instructions per 16-byte vector
    // instead of widening both operands to fp32 (half the registers).
    constexpr bool PACKED = sizeof(TX) == 2 && VEC == 8;
    const int log2S = a.log2S;
    const int S = 1 << log2S;
    const int lane = lane_id();
    const int lig = lane & (S - 1);
    const int gbase = lane & ~(S - 1);
    const int L = 1 << a.log2L;
    const int q = lig & (L - 1);
    const int h = lig >> a.log2L;
    const int M = L < U ? L : U;
    const int64_t fe = (int64_t)lig * VEC;
    const bool act = fe < a.W;
    const bool writer = act && q < M;
    const int H = a.H;
    const UnitWalk walk = unit_walk(a.units != nullptr, a.u_lo, a.u_hi, a.lists, a.n_rows,
                                    kBlock >> log2S, threadIdx.x >> log2S);
    const int64_t stride = walk.step;
    const int64_t hi = walk.end;
    const RowGather<TX, VEC, BUF> X(a.X, a.x_bytes);
    const TX *__restrict__ P = static_cast<const TX *>(a.P);
    const int32_t *__restrict__ col = a.col;
    extern __shared__ float row_park[];
    float *const park_mine = row_park + (threadIdx.x >> log2S) * a.park_cap;

    int64_t u = walk.first;
    if (u >= hi) return;
    int4 d = fetch_bwd_unit(a, u, hi);
    int c_cur = 0;
    if (d.z > d.y) c_cur = col[d.y + lig < d.z - 1 ? d.y + lig : d.z - 1];
    for (;;) {
        const int64_t un = u + stride;
        const int4 dn = fetch_bwd_unit(a, un, hi);
        const int row = d.x, beg = d.y, end = d.z, part = d.w;
        // a whole row whose parked values fit this sub-group's LDS share parks them
        // there (reduce-scatter kernels; the others keep their registers for the batch)
        float *const lds =
            (RS && !DOT && part < 0 && (end - beg) * H * (PK == kParkSep ? 1 : 2) <= a.park_cap) ? park_mine
                                                                                                 : nullptr;
        float p[PACKED ? 1 : VEC];
        uint4 pw = make_uint4(0u, 0u, 0u, 0u);
        if constexpr (PACKED) {
            if (act) pw = *reinterpret_cast<const uint4 *>(P + (int64_t)row * a.W + fe);
        } else if (act) {
            load_vec<TX, VEC>(P, (int64_t)row * a.W + fe, p);
        } else {
#pragma unroll
            for (int e = 0; e < VEC; ++e) p[e] = 0.f;
        }
        const float sd = (!DOT && act) ? a.s_dst[(int64_t)row * H + h] : 0.f;
        // kParkStats: the row's softmax state for this lane's head
        const float rm = (PK == kParkStats && act) ? a.row_stats[(int64_t)row * 2 * H + h] : 0.f;
        const float rrz = (PK == kParkStats && act) ? a.row_stats[(int64_t)row * 2 * H + H + h] : 0.f;
        float c = 0.f;

        const int last = end - 1;
        for (int k0 = beg; k0 < end; k0 += S) {
            const int n = (end - k0 < S) ? end - k0 : S;
            const int c_nxt = col[k0 + S + lig < last ? k0 + S + lig : last];
            for (int j = 0; j < n; j += U) {
                int cc[U];
                bool ok[U];
#pragma unroll
                for (int t = 0; t < U; ++t) {
                    ok[t] = j + t < n;
                    cc[t] = lane_bcast(c_cur, gbase + (ok[t] ? j + t : j));
                }
                float xv[PACKED ? 1 : U][VEC];
                uint4 xw[PACKED ? U : 1];
                float al[U], ss[U];
                bool mine[U];
#pragma unroll
                for (int t = 0; t < U; ++t) {
                    const bool on = ok[t] && act;
                    mine[t] = on && writer && (t & (M - 1)) == q;
                    if constexpr (PACKED) xw[t] = X.load_raw16((int64_t)cc[t] * a.W + fe, on);
                    else X.load((int64_t)cc[t] * a.W + fe, on, xv[t]);
                    al[t] = 0.f;
                    ss[t] = 0.f;
                    if constexpr (!DOT && !RS) {
                        if (mine[t]) {
                            ss[t] = a.s_src[(int64_t)cc[t] * H + h];
                            if constexpr (PK == kParkStats)
                                al[t] = alpha_value(leaky_relu(sd + ss[t], a.slope), rm, rrz);
                            else
                                al[t] = a.alpha[(int64_t)(k0 + j + t) * H + h];
                        }
                    }
                }
                float pd[U];
#pragma unroll
                for (int t = 0; t < U; ++t) {
                    float s = 0.f;
                    if constexpr (PACKED) {
                        s = dot2_acc<TX>(xw[t].x, pw.x, s);
                        s = dot2_acc<TX>(xw[t].y, pw.y, s);
                        s = dot2_acc<TX>(xw[t].z, pw.z, s);
                        s = dot2_acc<TX>(xw[t].w, pw.w, s);
                    } else {
#pragma unroll
                        for (int e = 0; e < VEC; ++e) s = fmaf(p[e], xv[t][e], s);
                    }
                    pd[t] = s;
                }
                if constexpr (RS) {
                    // lane q completes the dot product of edge j + (q mod 8)
                    const int t = q & 7;
                    float s = reduce_scatter8(pd, t);
                    for (int off = 8; off < L; off <<= 1) s += lane_xor(s, off);
                    const bool own = j + t < n && writer;
                    const int64_t k = k0 + j + t;
                    // (a cross-lane read: every lane takes part)
                    const int cme = DOT ? 0 : lane_bcast(c_cur, gbase + j + t);
                    if (own) {
                        if (DOT || PK == kParkSep || a.dalpha) a.dalpha[k * H + h] = s;
                        if constexpr (!DOT) {
                            const float ss1 = a.s_src[(int64_t)cme * H + h];
                            const float al1 = PK == kParkStats ? alpha_value(leaky_relu(sd + ss1, a.slope), rm, rrz)
                                                               : a.alpha[k * H + h];
                            c = fmaf(al1, s, c);
                            park_edge<PK>(a, k * H + h, part >= 0, al1, s, park_value(sd + ss1, a.slope, al1),
                                          lds, (int)(k - beg) * H + h);
                        }
                    }
                    continue;
                }
                // complete the dot products over the head's lanes (every lane of
                // the head ends with the same bits: each level adds the same pair)
#pragma unroll
                for (int t = 0; t < U; ++t) pd[t] = group_sum(pd[t], L);
#pragma unroll
                for (int t = 0; t < U; ++t) {
                    const int64_t k = k0 + j + t;
                    if (mine[t]) {
                        if (DOT || PK == kParkSep || a.dalpha) a.dalpha[k * H + h] = pd[t];
                        if constexpr (!DOT) {
                            c = fmaf(al[t], pd[t], c);
                            park_edge<PK>(a, k * H + h, part >= 0, al[t], pd[t],
                                          park_value(sd + ss[t], a.slope, al[t]), lds, (int)(k - beg) * H + h);
                        }
                    }
                }
            }
            c_cur = c_nxt;
        }
        const int c_first_next =
            (dn.z > dn.y) ? col[dn.y + lig < dn.z - 1 ? dn.y + lig : dn.z - 1] : 0;

        if constexpr (!DOT) {
            // the head's lanes hold shares of c (owners only, the others 0)
            c = group_sum(c, L);
            if (part >= 0) {
                if (act && q == 0) a.gstats[(int64_t)part * a.sstride + h] = c;
            } else {
                // this lane's parked edges: offsets q, q + M, ... of the row
                constexpr int R = 4;
                float sdt = 0.f;
                if (writer) {
                    for (int o0 = q; o0 < end - beg; o0 += R * M) {
                        float al[R], da[R], uv[R];
#pragma unroll
                        for (int r = 0; r < R; ++r) {
                            const int o = o0 + r * M;
                            const int oc = o < end - beg ? o : o0;
                            const int64_t i = ((int64_t)beg + oc) * H + h;
                            const int li = oc * H + h;
                            if constexpr (PK == kParkSep) {
                                // dalpha from its output; u from LDS (alpha from the input)
                                // or the record (alpha, u)
                                da[r] = a.dalpha[i];
                                const float2 p = lds ? make_float2(a.alpha[i], lds[li]) : a.rec[i];
                                al[r] = p.x;
                                uv[r] = p.y;
                            } else {
                                // the pair from LDS or the record: (dalpha, u) with alpha from
                                // the input, or (dalpha, v) holding alpha and u
                                const float2 p = lds ? make_float2(lds[2 * li], lds[2 * li + 1]) : a.rec[i];
                                da[r] = p.x;
                                if constexpr (PK == kParkStats) {
                                    const float2 q = unpark_stats(p.y, a.slope);
                                    al[r] = q.x;
                                    uv[r] = q.y;
                                } else {
                                    al[r] = a.alpha[i];
                                    uv[r] = p.y;
                                }
                            }
                        }
#pragma unroll
                        for (int r = 0; r < R; ++r) {
                            const int o = o0 + r * M;
                            if (o < end - beg)
                                sdt = add_stored(sdt, finish_edge<PK>(a, ((int64_t)beg + o) * H + h, al[r], uv[r],
                                                                       da[r], c));
                        }
                    }
                }
                sdt = group_sum(sdt, L);
                if (act && q == 0) a.ds_dst[(int64_t)row * H + h] = sdt;
            }
        }
        if (un >= hi) break;
        u = un;
        d = dn;
        c_cur = c_first_next;
    }
}

// Sum over the slots of one head in a wavefront laid out as (slot, head):
// lanes s * H + h, s < 64 / H.  The same fixed order in every lane of h.
__device__ __forceinline__ float slot_sum(float v, int H)
{
    if ((H & (H - 1)) == 0) {
        for (int off = H; off < kWave; off <<= 1) v += lane_xor(v, off);
        return v;
    }
    const int slots = kWave / H;
    const int h = lane_id() % H;
    float s = 0.f;
    for (int i = 0; i < slots; ++i) s += lane_bcast(v, i * H + h);
    return s;
}

// Pass 1 for any shape: a wavefront per unit, lanes as (edge slot, head),
// each lane forming whole dot products element by element.  Every edge is
// parked by the lane of its slot.
template <typename TX, typename TP, bool DOT, int PK = kParkSep>
__global__ __launch_bounds__(kBlock) void k_bwd_rows_any(BwdArgs a)
{
    const int lane = lane_id();
    const int H = a.H;
    const int eps = kWave / H;
    const int h = lane % H;
    const int slot = lane / H;
    const bool live = slot < eps;
    const UnitWalk walk = unit_walk(a.units != nullptr, a.u_lo, a.u_hi, a.lists, a.n_rows,
                                    kBlock / kWave, threadIdx.x / kWave);
    const int64_t hi = walk.end;
    const TX *__restrict__ X = static_cast<const TX *>(a.X);
    const TP *__restrict__ P = static_cast<const TP *>(a.P);
    for (int64_t u = walk.first; u < hi; u += walk.step) {
        const int4 d = fetch_bwd_unit(a, u, hi);
        const int row = d.x, beg = d.y, end = d.z, part = d.w;
        const float sd = DOT ? 0.f : a.s_dst[(int64_t)row * H + h];
        const float rm = PK == kParkStats ? a.row_stats[(int64_t)row * 2 * H + h] : 0.f;
        const float rrz = PK == kParkStats ? a.row_stats[(int64_t)row * 2 * H + H + h] : 0.f;
        float c = 0.f;
        if (live) {
            for (int k = beg + slot; k < end; k += eps) {
                const int j = a.col[k];
                float s = 0.f;
                for (int e = 0; e < a.D; ++e) {
                    float pv[1], xv[1];
                    load_vec<TP, 1>(P, (int64_t)row * a.W + (int64_t)h * a.D + e, pv);
                    load_vec<TX, 1>(X, (int64_t)j * a.W + (int64_t)h * a.D + e, xv);
                    s = fmaf(pv[0], xv[0], s);
                }
                if (DOT || PK == kParkSep || a.dalpha) a.dalpha[(int64_t)k * H + h] = s;
                if constexpr (!DOT) {
                    const float ss1 = a.s_src[(int64_t)j * H + h];
                    const float al = PK == kParkStats ? alpha_value(leaky_relu(sd + ss1, a.slope), rm, rrz)
                                                      : a.alpha[(int64_t)k * H + h];
                    c = fmaf(al, s, c);
                    park_edge<PK>(a, (int64_t)k * H + h, part >= 0, al, s, park_value(sd + ss1, a.slope, al),
                                  nullptr, 0);
                }
            }
        }
        if constexpr (DOT) continue;
        c = slot_sum(live ? c : 0.f, H);
        if (part >= 0) {
            if (slot == 0) a.gstats[(int64_t)part * a.sstride + h] = c;
            continue;
        }
        float sdt = 0.f;
        if (live) {
            for (int k = beg + slot; k < end; k += eps) {
                const int64_t i = (int64_t)k * H + h;
                const float2 r = a.rec[i];
                float g;
                if constexpr (PK == kParkSep) {
                    g = finish_edge<PK>(a, i, r.x, r.y, a.dalpha[i], c);           // (alpha, u)
                } else if constexpr (PK == kParkPair) {
                    g = finish_edge<PK>(a, i, a.alpha[i], r.y, r.x, c);            // (dalpha, u)
                } else {
                    const float2 q = unpark_stats(r.y, a.slope);                   // (dalpha, v)
                    g = finish_edge<PK>(a, i, q.x, q.y, r.x, c);
                }
                sdt = add_stored(sdt, g);
            }
        }
        sdt = slot_sum(live ? sdt : 0.f, H);
        if (slot == 0) a.ds_dst[(int64_t)row * H + h] = sdt;
    }
}

// Split rows, after pass 1: every neighbour group adds up the shares of c of
// all groups of its row, turns its parked edges into dscore and leaves its
// share of ds_dst.  One wavefront per group, lanes (slot, head); the shares
// are loaded by the slots side by side and summed over the slots in a fixed
// order (every group of a row forms the same c), and the next group's
// descriptors are fetched while this one is processed.
template <int PK>
__global__ __launch_bounds__(kBlock) void k_bwd_split_edges(BwdArgs a)
{
    const int lane = lane_id();
    const int H = a.H;
    const int eps = kWave / H;
    const int h = lane % H;
    const int slot = lane / H;
    const bool live = slot < eps;
    const int half = a.sstride >> 1;
    const int64_t waves = (int64_t)gridDim.x * (kBlock / kWave);
    const int32_t np = *a.n_parts;
    int64_t p = (int64_t)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave;
    if (p >= np) return;
    int4 d = a.part_units[p];
    int4 sr = a.split_rows[d.w];
    for (;;) {
        const int64_t pn = p + waves;
        const int4 dn = pn < np ? a.part_units[pn] : make_int4(0, 0, 0, 0);
        float cs = 0.f;
        if (live)
            for (int g = slot; g < sr.z; g += eps) cs += a.gstats[(int64_t)(sr.y + g) * a.sstride + h];
        const float c = slot_sum(live ? cs : 0.f, H);
        const int4 srn = pn < np ? a.split_rows[dn.w] : make_int4(0, 0, 0, 0);
        constexpr int R = 8;
        float sdt = 0.f;
        if (live) {
            for (int k0 = d.y + slot; k0 < d.z; k0 += R * eps) {
                float da[R], uv[R], al[R];
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    const int k = k0 + r * eps;
                    const int64_t i = (int64_t)(k < d.z ? k : k0) * H + h;
                    if constexpr (PK == kParkSep) {         // dalpha and the u parked in dscore
                        da[r] = a.dalpha[i];
                        uv[r] = a.dscore[i];
                        al[r] = a.alpha[i];
                    } else if constexpr (PK == kParkPair) { // the parked pair (dalpha, u)
                        const float2 q = a.rec[i];
                        da[r] = q.x;
                        uv[r] = q.y;
                        al[r] = a.alpha[i];
                    } else {                                // (dalpha, v): alpha and u from v
                        const float2 q = a.rec[i];
                        const float2 w = unpark_stats(q.y, a.slope);
                        da[r] = q.x;
                        al[r] = w.x;
                        uv[r] = w.y;
                    }
                }
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    const int k = k0 + r * eps;
                    if (k < d.z) sdt = add_stored(sdt, finish_edge<PK>(a, (int64_t)k * H + h, al[r], uv[r], da[r], c));
                }
            }
        }
        sdt = slot_sum(live ? sdt : 0.f, H);
        if (slot == 0) a.gstats[p * a.sstride + half + h] = sdt;
        if (pn >= np) break;
        p = pn;
        d = dn;
        sr = srn;
    }
}

// ds[row, h] = sum of the groups' shares (slot order), one wavefront per split
// row; the shares sit at offset `base` of each partial slot's stats.
__global__ __launch_bounds__(kBlock) void k_split_head_sums(const int4 *__restrict__ split_rows,
                                                            const int32_t *__restrict__ n_split,
                                                            const float *__restrict__ gstats,
                                                            int sstride, int base, int H,
                                                            float *__restrict__ out)
{
    const int lane = lane_id();
    const int64_t waves = (int64_t)gridDim.x * (kBlock / kWave);
    const int32_t ns = *n_split;
    for (int64_t s = (int64_t)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave; s < ns;
         s += waves) {
        const int4 d = split_rows[s];
        if (lane < H) {
            float v = 0.f;
            for (int g = 0; g < d.z; ++g) v += gstats[(int64_t)(d.y + g) * sstride + base + lane];
            out[(int64_t)d.x * H + lane] = v;
        }
    }
}

using BwdKernel = void (*)(BwdArgs);

template <typename TX, int VEC, bool DOT, int PK>
BwdKernel pick_rows_rs(bool buf, bool rs)
{
    if constexpr (VEC == 1) {
        return buf ? k_bwd_rows<TX, 1, true, DOT, false, PK> : k_bwd_rows<TX, 1, false, DOT, false, PK>;
    } else {
        if (rs)
            return buf ? k_bwd_rows<TX, VEC, true, DOT, true, PK> : k_bwd_rows<TX, VEC, false, DOT, true, PK>;
        return buf ? k_bwd_rows<TX, VEC, true, DOT, false, PK> : k_bwd_rows<TX, VEC, false, DOT, false, PK>;
    }
}

template <bool DOT, int PK>
BwdKernel pick_rows_t(int dt, bool buf, int vec, bool rs)
{
    if (dt == COGDL_F32) {
        if (vec == 4) return pick_rows_rs<float, 4, DOT, PK>(buf, rs);
        return pick_rows_rs<float, 1, DOT, PK>(buf, rs);
    }
    if (dt == COGDL_BF16) {
        if (vec == 8) return pick_rows_rs<bf16_t, 8, DOT, PK>(buf, rs);
        return pick_rows_rs<bf16_t, 1, DOT, PK>(buf, rs);
    }
    if (vec == 8) return pick_rows_rs<f16_t, 8, DOT, PK>(buf, rs);
    return pick_rows_rs<f16_t, 1, DOT, PK>(buf, rs);
}

// rs: the head spans 8 or more lanes (reduce-scatter; vector kernels only);
// pk: the parking mode (the dot-product kernels have one)
template <bool DOT>
BwdKernel pick_rows(int dt, bool buf, int vec, bool rs, int pk)
{
    if (DOT || pk == kParkSep) return pick_rows_t<DOT, kParkSep>(dt, buf, vec, rs);
    if (pk == kParkPair) return pick_rows_t<DOT, kParkPair>(dt, buf, vec, rs);
    return pick_rows_t<DOT, kParkStats>(dt, buf, vec, rs);
}

template <typename TX, bool DOT, int PK>
BwdKernel pick_any_p(int pdt)
{
    if (pdt == COGDL_F32) return k_bwd_rows_any<TX, float, DOT, PK>;
    if (pdt == COGDL_BF16) return k_bwd_rows_any<TX, bf16_t, DOT, PK>;
    return k_bwd_rows_any<TX, f16_t, DOT, PK>;
}

template <bool DOT, int PK>
BwdKernel pick_any_t(int xdt, int pdt)
{
    if (xdt == COGDL_F32) return pick_any_p<float, DOT, PK>(pdt);
    if (xdt == COGDL_BF16) return pick_any_p<bf16_t, DOT, PK>(pdt);
    return pick_any_p<f16_t, DOT, PK>(pdt);
}

template <bool DOT>
BwdKernel pick_any(int xdt, int pdt, int pk)
{
    if (DOT || pk == kParkSep) return pick_any_t<DOT, kParkSep>(xdt, pdt);
    if (pk == kParkPair) return pick_any_t<DOT, kParkPair>(xdt, pdt);
    return pick_any_t<DOT, kParkStats>(xdt, pdt);
}

unsigned wave_grid(int64_t work)
{
    int64_t b = (work + (kBlock / kWave) - 1) / (kBlock / kWave);
    if (b > 2048) b = 2048;
    if (b < 1) b = 1;
    return (unsigned)b;
}

// Pass 1 over the units of `plan` (or the rows in order): the fast kernel
// when the shape allows it, else the general one.
template <bool DOT>
cogdl_status rows_pass(BwdArgs a, const Plan *P, int xdt, int pdt, const char *name,
                       hipStream_t stream)
{
    const int64_t units = P ? P->cap_units : a.n_rows;
    const int xb = dtype_bytes(xdt);
    const int pk = a.row_stats ? kParkStats : (a.dalpha && a.dscore) ? kParkSep : kParkPair;
    const bool aligned = ((uintptr_t)a.X % 16 == 0) && ((uintptr_t)a.P % 16 == 0);
    const RowMap m = row_map(a.W, xb, a.D, aligned);
    const int L = a.D / m.vec;
    const bool fast = xdt == pdt && m.ch == 1 && m.n_slabs == 1 && (L & (L - 1)) == 0;
    if (fast) {
        a.log2S = m.log2S;
        a.log2L = log2i(L);
        const bool rs = m.vec > 1 && L >= 8;
        BwdKernel k = pick_rows<DOT>(xdt, a.x_bytes <= kBufferMaxBytes, m.vec, rs, pk);
        const int64_t upb = kBlock >> m.log2S;
        const bool park_lds = !DOT && rs;
        a.park_cap = park_lds ? kRowParkFloats / (int)upb : 0;
        const size_t shm = park_lds ? sizeof(float) * kRowParkFloats : 0;
        int64_t blocks = (units + upb - 1) / upb;
        const int64_t res = resident_blocks(reinterpret_cast<const void *>(k), kBlock);
        if (blocks > res) blocks = res;
        blocks = list_grid(blocks, a.lists);
        COGDL_LAUNCH_SHM(name, k, (unsigned)blocks, kBlock, shm, stream, a);
    } else {
        BwdKernel k = pick_any<DOT>(xdt, pdt, pk);
        a.park_cap = 0;
        int64_t blocks = (units + (kBlock / kWave) - 1) / (kBlock / kWave);
        const int64_t res = resident_blocks(reinterpret_cast<const void *>(k), kBlock);
        if (blocks > res) blocks = res;
        blocks = list_grid(blocks, a.lists);
        COGDL_LAUNCH(name, k, (unsigned)blocks, kBlock, stream, a);
    }
    return COGDL_OK;
}

cogdl_status check_heads(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *rowptr,
                         const int32_t *col, int32_t H, int32_t D)
{
    if (n_rows < 0 || n_cols < 0 || nnz < 0) return COGDL_ERR_INVALID;
    if (H < 1 || H > COGDL_MAX_HEADS || D < 1) return COGDL_ERR_INVALID;
    if (nnz > COGDL_MAX_NNZ || (int64_t)H * D > INT32_MAX) return COGDL_ERR_TOO_LARGE;
    if (n_rows > 0 && !rowptr) return COGDL_ERR_INVALID;
    if (nnz > 0 && (!col || n_rows == 0 || n_cols == 0)) return COGDL_ERR_INVALID;
    return COGDL_OK;
}

}  // namespace
}  // namespace cogdl

using namespace cogdl;

extern "C" {

cogdl_status cogdl_sddmm_dot(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *rowptr,
                             const int32_t *col, int32_t H, int32_t D, const void *P,
                             cogdl_dtype p_dtype, const void *Q, cogdl_dtype q_dtype, float *out,
                             const cogdl_plan *plan, hipStream_t stream)
{
    cogdl_status st = check_heads(n_rows, n_cols, nnz, rowptr, col, H, D);
    if (st != COGDL_OK) return st;
    if (!dtype_ok(p_dtype) || !dtype_ok(q_dtype)) return COGDL_ERR_DTYPE;
    if (nnz > 0 && (!P || !Q || !out)) return COGDL_ERR_INVALID;
    const Plan *Pl = plan_of(plan);
    if (Pl && (Pl->n_rows != n_rows || Pl->nnz != nnz)) return COGDL_ERR_PLAN;
    if (nnz == 0) return COGDL_OK;
    BwdArgs a{};
    a.units = Pl ? Pl->units : nullptr;
    if (Pl) set_units(a, all_units(*Pl));
    a.n_rows = n_rows;
    a.rowptr = rowptr;
    a.col = col;
    a.H = H;
    a.D = D;
    a.W = (int64_t)H * D;
    a.X = Q;
    a.x_bytes = (uint64_t)n_cols * (uint64_t)a.W * (uint64_t)dtype_bytes(q_dtype);
    a.P = P;
    a.dalpha = out;
    return rows_pass<true>(a, Pl, (int)q_dtype, (int)p_dtype, "sddmm_dot", stream);
}

}  // extern "C"

namespace cogdl {
namespace {

// The backward with the forward weights given (alpha) or rebuilt from the
// forward's row softmax states (row_stats): exactly one of them.
cogdl_status gat_backward_impl(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *rowptr,
                               const int32_t *col, const int32_t *colptr, const int32_t *row_t,
                               const int32_t *perm, int32_t H, int32_t D, const float *s_dst,
                               const float *s_src, float negative_slope, const float *alpha,
                               const float *row_stats, const void *X, cogdl_dtype x_dtype,
                               const void *dY, cogdl_dtype dy_dtype, void *dX, cogdl_dtype dx_dtype,
                               float *dalpha, float *dscore, float *ds_dst, float *ds_src,
                               float *edge_work, const cogdl_plan *plan, const cogdl_plan *plan_t,
                               hipStream_t stream)
{
    cogdl_status st = check_heads(n_rows, n_cols, nnz, rowptr, col, H, D);
    if (st != COGDL_OK) return st;
    if (!dtype_ok(x_dtype) || !dtype_ok(dy_dtype) || !dtype_ok(dx_dtype)) return COGDL_ERR_DTYPE;
    if (n_cols > 0 && (!colptr || !dX || !ds_src)) return COGDL_ERR_INVALID;
    if (n_rows > 0 && (!ds_dst || !s_dst || !dY)) return COGDL_ERR_INVALID;
    if (nnz > 0 && (!row_t || !perm || !s_src || (alpha == nullptr) == (row_stats == nullptr) || !X ||
                    !edge_work || (uintptr_t)edge_work % alignof(float2) != 0))
        return COGDL_ERR_INVALID;
    float2 *rec = reinterpret_cast<float2 *>(edge_work);
    const int64_t W = (int64_t)H * D;
    const Plan *Pr = plan_of(plan);
    const Plan *Pc = plan_of(plan_t);
    if (Pr && (Pr->n_rows != n_rows || Pr->nnz != nnz || Pr->max_heads < H)) return COGDL_ERR_PLAN;
    if (Pc && (Pc->n_rows != n_cols || Pc->nnz != nnz || Pc->max_feat < W || Pc->max_heads < H))
        return COGDL_ERR_PLAN;

    // pass 1 on the CSR: dalpha, dscore, ds_dst
    if (n_rows > 0) {
        BwdArgs a{};
        a.units = Pr ? Pr->units : nullptr;
        if (Pr) set_units(a, all_units(*Pr));
        a.n_rows = n_rows;
        a.rowptr = rowptr;
        a.col = col;
        a.H = H;
        a.D = D;
        a.W = W;
        a.s_dst = s_dst;
        a.s_src = s_src;
        a.slope = negative_slope;
        a.alpha = alpha;
        a.row_stats = row_stats;
        a.X = X;
        a.x_bytes = (uint64_t)n_cols * (uint64_t)W * (uint64_t)dtype_bytes(x_dtype);
        a.P = dY;
        a.dalpha = dalpha;
        a.dscore = dscore;
        a.rec = rec;
        a.ds_dst = ds_dst;
        a.gstats = Pr ? Pr->gstats : nullptr;
        a.sstride = Pr ? 2 * Pr->max_heads : 0;
        a.part_units = Pr ? Pr->part_units : nullptr;
        a.n_parts = Pr ? Pr->n_parts_dev() : nullptr;
        a.split_rows = Pr ? Pr->split_rows : nullptr;
        a.n_split = Pr ? Pr->n_split_dev() : nullptr;
        st = rows_pass<false>(a, Pr, (int)x_dtype, (int)dy_dtype, "gat_bwd_rows", stream);
        if (st != COGDL_OK) return st;
        if (Pr) {
            if (row_stats)
                COGDL_LAUNCH("gat_bwd_split_edges", k_bwd_split_edges<kParkStats>, wave_grid(Pr->cap_partials),
                             kBlock, stream, a);
            else if (dalpha && dscore)
                COGDL_LAUNCH("gat_bwd_split_edges", k_bwd_split_edges<kParkSep>, wave_grid(Pr->cap_partials),
                             kBlock, stream, a);
            else
                COGDL_LAUNCH("gat_bwd_split_edges", k_bwd_split_edges<kParkPair>, wave_grid(Pr->cap_partials),
                             kBlock, stream, a);
            COGDL_LAUNCH("gat_bwd_split_dst", k_split_head_sums, wave_grid(Pr->cap_split), kBlock,
                         stream, Pr->split_rows, Pr->n_split_dev(), Pr->gstats, a.sstride,
                         Pr->max_heads, H, ds_dst);
        }
    }
    if (n_cols == 0) return COGDL_OK;

    // pass 2 on the CSC: dX and ds_src
    const bool aligned = ((uintptr_t)dY % 16 == 0) && ((uintptr_t)dX % 16 == 0);
    RowMap m = row_map(W, dtype_bytes(dy_dtype), D, aligned);
    if (m.S < H) {
        m.S = next_pow2(H);
        m.log2S = log2i(m.S);
        m.slab = m.S * m.ch * m.vec;
        m.n_slabs = (int)((W + m.slab - 1) / m.slab);
    }
    GatArgs g{};
    g.units = Pc ? Pc->units : nullptr;
    g.n_rows = n_cols;
    g.rowptr = colptr;
    g.col = row_t;
    g.H = H;
    g.D = D;
    g.W = W;
    g.alpha_in = alpha;
    g.X = dY;
    g.x_bytes = (uint64_t)n_rows * (uint64_t)W * (uint64_t)dtype_bytes(dy_dtype);
    g.Y = dX;
    g.partials = Pc ? Pc->partials : nullptr;
    g.pstride = Pc ? (Pc->max_feat + 7) / 8 * 8 : 0;
    g.gstats = Pc ? Pc->gstats : nullptr;
    g.sstride = Pc ? 2 * Pc->max_heads : 0;
    g.perm = perm;
    g.rec = rec;
    g.ds_out = ds_src;
    g.slab = m.slab;
    g.log2S = m.log2S;
    const bool buf = g.x_bytes <= kBufferMaxBytes;
    const int64_t units = Pc ? Pc->cap_units : n_cols;
    const bool tiny = Pc && m.ch == 1 && m.S >= 8 && m.S / 4 >= H;
    if (Pc) set_units(g, tiny ? long_units(*Pc) : all_units(*Pc));
    {
        const int64_t upb = kBlock >> m.log2S;
        // one edge's record per lane when a head is exactly eight 16-byte vectors
        const bool dist = m.ch == 1 && m.vec * dtype_bytes(dy_dtype) == 16 && D == 8 * m.vec;
        GatKernel k = gat_pick<true>((int)dy_dtype, (int)dx_dtype, m.vec, m.ch, buf, dist);
        int64_t blocks = (units + upb - 1) / upb;
        const int64_t res = resident_blocks(reinterpret_cast<const void *>(k), kBlock);
        if (blocks > res) blocks = res;
        blocks = list_grid(blocks, g.lists);
        COGDL_LAUNCH("gat_bwd_cols", k, dim3((unsigned)blocks, (unsigned)m.n_slabs), kBlock, stream, g);
    }
    if (tiny) {
        GatArgs b = g;
        set_units(b, tiny_units(*Pc));
        b.log2S = m.log2S - 2;
        const int64_t upb = kBlock >> b.log2S;
        GatKernel k = gat_pick<true>((int)dy_dtype, (int)dx_dtype, m.vec, 4, buf);
        int64_t blocks = (units + upb - 1) / upb;
        const int64_t res = resident_blocks(reinterpret_cast<const void *>(k), kBlock);
        if (blocks > res) blocks = res;
        blocks = list_grid(blocks, b.lists);
        COGDL_LAUNCH("gat_bwd_cols_tiny", k, dim3((unsigned)blocks, (unsigned)m.n_slabs), kBlock, stream, b);
    }
    if (!Pc) return COGDL_OK;
    st = sum_reduce_launch("gat_bwd_dx_reduce", *Pc, W, dX, (int)dx_dtype, false, nullptr,
                           COGDL_ACT_NONE, stream);
    if (st != COGDL_OK) return st;
    COGDL_LAUNCH("gat_bwd_split_src", k_split_head_sums, wave_grid(Pc->cap_split), kBlock, stream,
                 Pc->split_rows, Pc->n_split_dev(), Pc->gstats, g.sstride, 0, H, ds_src);
    return COGDL_OK;
}

}  // namespace
}  // namespace cogdl

extern "C" {

cogdl_status cogdl_gat_backward(int32_t n_rows, int32_t n_cols, int64_t nnz,
                                const int32_t *rowptr, const int32_t *col, const int32_t *colptr,
                                const int32_t *row_t, const int32_t *perm, int32_t H, int32_t D,
                                const float *s_dst, const float *s_src, float negative_slope,
                                const float *alpha, const void *X, cogdl_dtype x_dtype,
                                const void *dY, cogdl_dtype dy_dtype, void *dX,
                                cogdl_dtype dx_dtype, float *dalpha, float *dscore, float *ds_dst,
                                float *ds_src, float *edge_work, const cogdl_plan *plan,
                                const cogdl_plan *plan_t, hipStream_t stream)
{
    if (nnz > 0 && !alpha) return COGDL_ERR_INVALID;
    return gat_backward_impl(n_rows, n_cols, nnz, rowptr, col, colptr, row_t, perm, H, D, s_dst, s_src,
                             negative_slope, alpha, nullptr, X, x_dtype, dY, dy_dtype, dX, dx_dtype,
                             dalpha, dscore, ds_dst, ds_src, edge_work, plan, plan_t, stream);
}

cogdl_status cogdl_gat_backward_stats(int32_t n_rows, int32_t n_cols, int64_t nnz,
                                      const int32_t *rowptr, const int32_t *col,
                                      const int32_t *colptr, const int32_t *row_t,
                                      const int32_t *perm, int32_t H, int32_t D,
                                      const float *s_dst, const float *s_src,
                                      float negative_slope, const float *row_stats, const void *X,
                                      cogdl_dtype x_dtype, const void *dY, cogdl_dtype dy_dtype,
                                      void *dX, cogdl_dtype dx_dtype, float *dalpha,
                                      float *dscore, float *ds_dst, float *ds_src,
                                      float *edge_work, const cogdl_plan *plan,
                                      const cogdl_plan *plan_t, hipStream_t stream)
{
    if (nnz > 0 && !row_stats) return COGDL_ERR_INVALID;
    return gat_backward_impl(n_rows, n_cols, nnz, rowptr, col, colptr, row_t, perm, H, D, s_dst, s_src,
                             negative_slope, nullptr, row_stats, X, x_dtype, dY, dy_dtype, dX, dx_dtype,
                             dalpha, dscore, ds_dst, ds_src, edge_work, plan, plan_t, stream);
}

}  // extern "C"
