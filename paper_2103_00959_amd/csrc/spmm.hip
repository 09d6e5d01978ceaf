// Generalized SpMM of section 2.2, Eq. 1: H' = A H (reduce = sum, compute =
// multiply by the edge value), its reduce (mean, max) and compute (add,
// subtract, copy) variants, and the transposed product A^T G of its backward
// pass.  The gather kernel itself is in spmm_kernel.hpp.
//
// Mapping on gfx950 (64-lane wavefronts):
//   - A work unit (a whole row, or a neighbour group of a long row) belongs to
//     a sub-group of S lanes; S lanes times VEC elements cover one feature row
//     (S = 32 for a 512-byte row read as 16-byte vectors), CH chunks when the
//     row is wider than 64 vectors, feature slabs beyond that.
//   - The sub-group reads the unit's column indices and edge values S at a
//     time with one coalesced load, prefetching the next S while it works, and
//     hands them to every lane with ds_bpermute.
//   - For every edge each lane gathers its VEC contiguous features of the
//     neighbour row (one 16-byte load) and accumulates in fp32 registers; U
//     edges are unrolled so that U row gathers are in flight per lane.
//   - A unit that covers a whole row writes the output row once; a neighbour
//     group writes an fp32 partial row (for max also the edge id of each
//     partial maximum), and a second kernel combines the partials of each
//     split row in a fixed order (no floating-point atomics).
#include "spmm_kernel.hpp"

namespace cogdl {
namespace {

constexpr int kBlock = kSpmmBlock;

// Y[row, :] = sum of the row's partial rows (times 1 / degree for mean).  A
// wavefront per split row (grid-stride over the device-side count, uniform
// per wavefront), VEC features per lane: slot g goes to chain g mod 4, the
// four chains add their slots in increasing order and are combined as
// (c0 + c1) + (c2 + c3), so the result does not depend on timing.  Four
// slots' loads are in flight per step, and a workgroup's four wavefronts work
// on four different rows (column-sliced plans make a hundred thousand short
// split rows, where a workgroup per row waited on its own barrier).
template <typename TY, int VEC>
__global__ __launch_bounds__(kBlock) void k_spmm_reduce(const int4 *__restrict__ split_rows,
                                                        const int32_t *__restrict__ n_split,
                                                        const float *__restrict__ partials,
                                                        int64_t pstride, int64_t F, int mean,
                                                        const float *__restrict__ bias, int act_code,
                                                        TY *__restrict__ Y)
{
    const int lane = lane_id();
    const int64_t waves = (int64_t)gridDim.x * (kBlock / kWave);
    const int32_t ns = *n_split;
    for (int64_t s = (int64_t)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave; s < ns;
         s += waves) {
        const int4 d = split_rows[s];
        const int64_t row = d.x, p0 = d.y;
        const int np = d.z;
        const float scale = (mean && d.w > 0) ? 1.f / (float)d.w : 1.f;
        for (int64_t fb = 0; fb < F; fb += kWave * VEC) {
            const int64_t f = fb + (int64_t)lane * VEC;
            if (f >= F) continue;
            float c[4][VEC];
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int e = 0; e < VEC; ++e) c[j][e] = 0.f;
            const float *p = partials + p0 * pstride + f;
            int g = 0;
            for (; g + 4 <= np; g += 4) {
                float x[4][VEC];
#pragma unroll
                for (int j = 0; j < 4; ++j) load_vec<float, VEC>(p, (int64_t)(g + j) * pstride, x[j]);
#pragma unroll
                for (int j = 0; j < 4; ++j)
#pragma unroll
                    for (int e = 0; e < VEC; ++e) c[j][e] += x[j][e];
            }
#pragma unroll
            for (int j = 0; j < 3; ++j) {
                if (g + j < np) {
                    float x[VEC];
                    load_vec<float, VEC>(p, (int64_t)(g + j) * pstride, x);
#pragma unroll
                    for (int e = 0; e < VEC; ++e) c[j][e] += x[e];
                }
            }
            float v[VEC];
#pragma unroll
            for (int e = 0; e < VEC; ++e) {
                v[e] = (c[0][e] + c[1][e]) + (c[2][e] + c[3][e]);
                if (mean) v[e] *= scale;
            }
            epilogue<VEC>(v, bias, act_code, f);
            store_out<TY, VEC>(Y, row * F + f, v);
        }
    }
}

// Max over a split row's partial maxima, slots in edge order: the first slot
// is kept and a later one only if strictly greater, which keeps the first
// edge attaining the row maximum.  One wavefront per split row, one feature
// per lane (split rows are few; the slots of a row are contiguous, so each
// wavefront reads whole 256-byte lines).
template <typename TY>
__global__ __launch_bounds__(kBlock) void k_spmm_reduce_max(const int4 *__restrict__ split_rows,
                                                            const int32_t *__restrict__ n_split,
                                                            const float *__restrict__ partials,
                                                            const int32_t *__restrict__ parg,
                                                            int64_t pstride, int64_t F,
                                                            const float *__restrict__ bias, int act_code,
                                                            TY *__restrict__ Y,
                                                            int32_t *__restrict__ arg)
{
    const int lane = lane_id();
    const int64_t waves = (int64_t)gridDim.x * (kBlock / kWave);
    const int32_t ns = *n_split;
    for (int64_t s = (int64_t)blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave; s < ns;
         s += waves) {
        const int4 d = split_rows[s];
        for (int64_t f = lane; f < F; f += kWave) {
            float best = 0.f;
            int32_t bk = -1;
            for (int g = 0; g < d.z; ++g) {
                const int64_t q = (int64_t)(d.y + g) * pstride + f;
                const float v = partials[q];
                if (bk < 0 || v > best) { best = v; bk = parg[q]; }
            }
            float out[1] = {best};
            epilogue<1>(out, bias, act_code, f);
            store_out<TY, 1>(Y, (int64_t)d.x * F + f, out);
            if (arg) arg[(int64_t)d.x * F + f] = bk;
        }
    }
}

template <int VEC>
cogdl_status reduce_launch_v(const char *name, const Plan &P, int64_t F, void *Y, int ydt,
                             bool mean, const float *bias, int act, hipStream_t s)
{
    const int64_t pstride = (P.max_feat + 7) / 8 * 8;
    constexpr int wpb = kBlock / kWave;
    int64_t blocks = (P.cap_split + wpb - 1) / wpb;
    if (blocks > 2048) blocks = 2048;
    if (blocks < 1) blocks = 1;
    const unsigned b = (unsigned)blocks;
    const int mn = mean ? 1 : 0;
    if (ydt == COGDL_F32)
        COGDL_LAUNCH(name, (k_spmm_reduce<float, VEC>), b, kBlock, s, P.split_rows, P.n_split_dev(),
                     P.partials, pstride, F, mn, bias, act, static_cast<float *>(Y));
    else if (ydt == COGDL_BF16)
        COGDL_LAUNCH(name, (k_spmm_reduce<bf16_t, VEC>), b, kBlock, s, P.split_rows, P.n_split_dev(),
                     P.partials, pstride, F, mn, bias, act, static_cast<bf16_t *>(Y));
    else
        COGDL_LAUNCH(name, (k_spmm_reduce<f16_t, VEC>), b, kBlock, s, P.split_rows, P.n_split_dev(),
                     P.partials, pstride, F, mn, bias, act, static_cast<f16_t *>(Y));
    return COGDL_OK;
}

cogdl_status max_reduce_launch(const char *name, const Plan &P, int64_t F, void *Y, int ydt,
                               const float *bias, int act, int32_t *arg, hipStream_t s)
{
    const int64_t pstride = (P.max_feat + 7) / 8 * 8;
    constexpr int wpb = kBlock / kWave;
    int64_t blocks = (P.cap_split + wpb - 1) / wpb;
    if (blocks > 2048) blocks = 2048;
    if (blocks < 1) blocks = 1;
    const unsigned b = (unsigned)blocks;
    if (ydt == COGDL_F32)
        COGDL_LAUNCH(name, k_spmm_reduce_max<float>, b, kBlock, s, P.split_rows, P.n_split_dev(),
                     P.partials, P.parg, pstride, F, bias, act, static_cast<float *>(Y), arg);
    else if (ydt == COGDL_BF16)
        COGDL_LAUNCH(name, k_spmm_reduce_max<bf16_t>, b, kBlock, s, P.split_rows, P.n_split_dev(),
                     P.partials, P.parg, pstride, F, bias, act, static_cast<bf16_t *>(Y), arg);
    else
        COGDL_LAUNCH(name, k_spmm_reduce_max<f16_t>, b, kBlock, s, P.split_rows, P.n_split_dev(),
                     P.partials, P.parg, pstride, F, bias, act, static_cast<f16_t *>(Y), arg);
    return COGDL_OK;
}

}  // namespace

// Four features per lane when the rows allow 16-byte partial loads and
// aligned output stores, one otherwise.
cogdl_status sum_reduce_launch(const char *name, const Plan &P, int64_t F, void *Y, int ydt,
                               bool mean, const float *bias, int act, hipStream_t s)
{
    const int ybytes = dtype_bytes(ydt);
    if (F % 4 == 0 && (uintptr_t)Y % (4 * ybytes) == 0)
        return reduce_launch_v<4>(name, P, F, Y, ydt, mean, bias, act, s);
    return reduce_launch_v<1>(name, P, F, Y, ydt, mean, bias, act, s);
}

namespace {

struct LaunchNames {
    const char *main, *tiny, *reduce;
};

// Shared body of the SpMM entry points: out_rows x F output, gathering rows of
// an in_rows x F input through (ptr, idx, w), combined by `reduce`.
cogdl_status spmm_common(int32_t out_rows, int32_t in_rows, int64_t nnz, const int32_t *ptr,
                         const int32_t *idx, const float *w, int32_t F, const void *X, int xdt,
                         void *Y, int ydt, int reduce, int compute, const float *bias, int act,
                         int32_t *arg, const cogdl_plan *plan_h, hipStream_t s, LaunchNames names)
{
    if (out_rows < 0 || in_rows < 0 || nnz < 0 || F < 0) return COGDL_ERR_INVALID;
    if (reduce != COGDL_REDUCE_SUM && reduce != COGDL_REDUCE_MEAN && reduce != COGDL_REDUCE_MAX)
        return COGDL_ERR_INVALID;
    if (compute < COGDL_COMPUTE_MUL || compute > COGDL_COMPUTE_COPY) return COGDL_ERR_INVALID;
    if (act < COGDL_ACT_NONE || act > COGDL_ACT_ELU) return COGDL_ERR_INVALID;
    if (!dtype_ok(xdt) || !dtype_ok(ydt)) return COGDL_ERR_DTYPE;
    const bool maxr = reduce == COGDL_REDUCE_MAX;
    if (maxr && ydt != COGDL_F32 && ydt != xdt) return COGDL_ERR_DTYPE;
    if (nnz > COGDL_MAX_NNZ) return COGDL_ERR_TOO_LARGE;
    if (out_rows > 0 && !ptr) return COGDL_ERR_INVALID;
    if (nnz > 0 && (!idx || out_rows == 0 || in_rows == 0)) return COGDL_ERR_INVALID;
    if (out_rows > 0 && F > 0 && !Y) return COGDL_ERR_INVALID;
    if (nnz > 0 && F > 0 && !X) return COGDL_ERR_INVALID;
    const Plan *P = plan_of(plan_h);
    if (P && (P->n_rows != out_rows || P->nnz != nnz || P->max_feat < F)) return COGDL_ERR_PLAN;
    if (out_rows == 0 || F == 0) return COGDL_OK;

    const bool aligned = ((uintptr_t)X % 16 == 0) && ((uintptr_t)Y % 16 == 0) &&
                         (!maxr || !arg || (uintptr_t)arg % 16 == 0);
    const RowMap m = row_map(F, dtype_bytes(xdt), F, aligned);
    SpmmArgs a;
    a.units = P ? P->units : nullptr;
    a.u_lo = nullptr;
    a.u_hi = nullptr;
    a.n_rows = out_rows;
    a.rowptr = ptr;
    a.col = idx;
    a.val = compute == COGDL_COMPUTE_COPY ? nullptr : w;
    a.X = X;
    a.Y = Y;
    a.arg = maxr ? arg : nullptr;
    a.partials = P ? P->partials : nullptr;
    a.parg = P ? P->parg : nullptr;
    a.pstride = P ? (P->max_feat + 7) / 8 * 8 : 0;
    a.F = F;
    a.x_bytes = (uint64_t)in_rows * (uint64_t)F * (uint64_t)dtype_bytes(xdt);
    a.slab = m.slab;
    a.log2S = m.log2S;
    a.mean = reduce == COGDL_REDUCE_MEAN ? 1 : 0;
    a.bsign = compute == COGDL_COMPUTE_SUB ? -1.f : 1.f;
    a.bias = bias;
    a.act = act;
    const bool addop = compute == COGDL_COMPUTE_ADD || compute == COGDL_COMPUTE_SUB;
    const bool buf = a.x_bytes <= kBufferMaxBytes;
    auto pick = [&](int ch) {
        return (maxr || addop) ? gspmm_pick(maxr, addop, xdt, ydt, m.vec, ch, buf)
                               : spmm_pick<false, false>(xdt, ydt, m.vec, ch, buf);
    };
    const int64_t units = P ? P->cap_units : out_rows;
    // Units of at most kTinyUnit edges (the sorted tail) run with S/4 lanes and
    // four chunks per lane: four times as many rows in flight per wavefront.
    const bool tiny = P && m.ch == 1 && m.S >= 8;
    if (P) set_units(a, tiny ? long_units(*P) : all_units(*P));
    {
        const int64_t upb = kBlock >> m.log2S;
        SpmmKernel k = pick(m.ch);
        if (!k) return COGDL_ERR_DTYPE;
        int64_t blocks = (units + upb - 1) / upb;
        const int64_t res = resident_blocks(reinterpret_cast<const void *>(k), kBlock);
        if (blocks > res) blocks = res;
        blocks = list_grid(blocks, a.lists);
        COGDL_LAUNCH(names.main, k, dim3((unsigned)blocks, (unsigned)m.n_slabs), kBlock, s, a);
    }
    if (tiny) {
        SpmmArgs b = a;
        set_units(b, tiny_units(*P));
        b.log2S = m.log2S - 2;
        const int64_t upb = kBlock >> b.log2S;
        SpmmKernel k = pick(4);
        if (!k) return COGDL_ERR_DTYPE;
        int64_t blocks = (units + upb - 1) / upb;
        const int64_t res = resident_blocks(reinterpret_cast<const void *>(k), kBlock);
        if (blocks > res) blocks = res;
        blocks = list_grid(blocks, b.lists);
        COGDL_LAUNCH(names.tiny, k, dim3((unsigned)blocks, (unsigned)m.n_slabs), kBlock, s, b);
    }
    if (!P) return COGDL_OK;
    if (maxr) return max_reduce_launch(names.reduce, *P, F, Y, ydt, bias, act, a.arg, s);
    return sum_reduce_launch(names.reduce, *P, F, Y, ydt, a.mean != 0, bias, act, s);
}

}  // namespace
}  // namespace cogdl

extern "C" {

cogdl_status cogdl_spmm(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *rowptr,
                        const int32_t *col, const float *val, int32_t F, const void *X,
                        cogdl_dtype x_dtype, void *Y, cogdl_dtype y_dtype, const cogdl_plan *plan,
                        hipStream_t stream)
{
    return cogdl::spmm_common(n_rows, n_cols, nnz, rowptr, col, val, F, X, (int)x_dtype, Y,
                              (int)y_dtype, COGDL_REDUCE_SUM, COGDL_COMPUTE_MUL, nullptr,
                              COGDL_ACT_NONE, nullptr, plan, stream,
                              {"spmm", "spmm_tiny", "spmm_reduce"});
}

cogdl_status cogdl_gspmm(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *rowptr,
                         const int32_t *col, const float *val, int32_t F, const void *X,
                         cogdl_dtype x_dtype, void *Y, cogdl_dtype y_dtype, cogdl_reduce reduce,
                         cogdl_compute compute, const float *bias, cogdl_act act, int32_t *arg,
                         const cogdl_plan *plan, hipStream_t stream)
{
    return cogdl::spmm_common(n_rows, n_cols, nnz, rowptr, col, val, F, X, (int)x_dtype, Y,
                              (int)y_dtype, (int)reduce, (int)compute, bias, (int)act, arg, plan,
                              stream, {"gspmm", "gspmm_tiny", "gspmm_reduce"});
}

cogdl_status cogdl_spmm_t(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *colptr,
                          const int32_t *row_t, const float *val_t, int32_t F, const void *G,
                          cogdl_dtype g_dtype, void *dX, cogdl_dtype dx_dtype,
                          const cogdl_plan *plan_t, hipStream_t stream)
{
    // A^T has n_cols rows, each gathering rows of the n_rows x F input G.
    return cogdl::spmm_common(n_cols, n_rows, nnz, colptr, row_t, val_t, F, G, (int)g_dtype, dX,
                              (int)dx_dtype, COGDL_REDUCE_SUM, COGDL_COMPUTE_MUL, nullptr,
                              COGDL_ACT_NONE, nullptr, plan_t, stream,
                              {"spmm_t", "spmm_t_tiny", "spmm_t_reduce"});
}

}  // extern "C"
