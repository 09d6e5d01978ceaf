/*
 * oracle.c -- plain, slow, obviously correct CPU reference for the GNN
 * message-passing operators of the CogDL paper (arxiv 2103.00959), section 2.2
 * "Efficient Sparse Operators".
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library calls, links or
 * loads this file; only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg do.  It shares no code, header or constant with the HIP
 * library: it decodes its own input formats, rounds with its own routine and
 * implements each operator straight from its definition.
 *
 * Conventions (readings of the paper, each listed in the design notes):
 *  - CSR row i is the aggregating node u of Eq. 1, column j the message
 *    source v; edge k = (i, col[k]) carries the value val[k].
 *  - All floating-point work is in double precision, visiting the edges of a
 *    row in CSR order; callers round once to the output format with
 *    oracle_round().
 *  - Duplicate (i, j) pairs are separate terms; empty rows produce zero.
 *
 * Functions that take (n_sel, sel) compute only the listed rows (or columns
 * for the transposed product) and pack results in list order; sel == NULL
 * means every row.  All array arguments are host pointers.  Every function
 * returns 0 on success and a negative value on a bad argument.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { ORACLE_F32 = 0, ORACLE_BF16 = 1, ORACLE_F16 = 2 };

/* ---------------------------------------------------------------- formats */

/* bfloat16: the upper 16 bits of an IEEE binary32. Exact widening. */
static double decode_bf16(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* IEEE binary16: 1 sign, 5 exponent (bias 15), 10 fraction bits. */
static double decode_f16(uint16_t h)
{
    int sign = h >> 15;
    int ex = (h >> 10) & 31;
    int fr = h & 1023;
    double v;
    if (ex == 0)
        v = ldexp((double)fr, -24);              /* subnormal: fr * 2^-24 */
    else if (ex == 31)
        v = fr ? NAN : INFINITY;
    else
        v = ldexp((double)(1024 + fr), ex - 25); /* (1 + fr/1024) * 2^(ex-15) */
    return sign ? -v : v;
}

static double load_elem(const void *x, int dtype, int64_t i)
{
    if (dtype == ORACLE_F32) return (double)((const float *)x)[i];
    if (dtype == ORACLE_BF16) return decode_bf16(((const uint16_t *)x)[i]);
    return decode_f16(((const uint16_t *)x)[i]);
}

/* Round v to the nearest value (ties to even) of a binary format with p
 * significand bits, minimum normal exponent emin and maximum exponent emax,
 * directly from double (no intermediate rounding). */
static double round_to_format(double v, int p, int emin, int emax)
{
    if (isnan(v) || isinf(v) || v == 0.0) return v;
    int e;
    frexp(fabs(v), &e);
    int lead = e - 1;                   /* exponent of the leading bit */
    if (lead < emin) lead = emin;       /* subnormals share one quantum */
    double quantum = ldexp(1.0, lead - (p - 1));
    double r = rint(v / quantum) * quantum;   /* rint: ties to even */
    double max_finite = ldexp(2.0 - ldexp(1.0, 1 - p), emax);
    if (fabs(r) > max_finite) r = copysign(INFINITY, v);
    return r;
}

static uint16_t encode_f16(double r)
{
    /* r is already a binary16 value (or inf/nan). */
    uint16_t sign = signbit(r) ? 0x8000 : 0;
    double a = fabs(r);
    if (isnan(r)) return 0x7e00;
    if (isinf(a)) return sign | 0x7c00;
    if (a == 0.0) return sign;
    int e;
    frexp(a, &e);
    int lead = e - 1;
    if (lead < -14) /* subnormal: a = fr * 2^-24 */
        return sign | (uint16_t)(a / ldexp(1.0, -24));
    uint16_t fr = (uint16_t)(a / ldexp(1.0, lead - 10) - 1024.0);
    return sign | (uint16_t)((lead + 15) << 10) | fr;
}

/* Round n doubles to dtype (RNE) and store the encoded values in out. */
int oracle_round(const double *in, int64_t n, int32_t dtype, void *out)
{
    if (n < 0 || (n > 0 && (!in || !out))) return -1;
    for (int64_t i = 0; i < n; ++i) {
        if (dtype == ORACLE_F32) {
            ((float *)out)[i] = (float)round_to_format(in[i], 24, -126, 127);
        } else if (dtype == ORACLE_BF16) {
            float f = (float)round_to_format(in[i], 8, -126, 127);
            uint32_t u;
            memcpy(&u, &f, sizeof u);
            if (isnan(f)) u = 0x7fc00000u;
            ((uint16_t *)out)[i] = (uint16_t)(u >> 16);
        } else if (dtype == ORACLE_F16) {
            ((uint16_t *)out)[i] = encode_f16(round_to_format(in[i], 11, -14, 15));
        } else {
            return -2;
        }
    }
    return 0;
}

/* Decode n stored values of dtype to double. */
int oracle_decode(const void *in, int64_t n, int32_t dtype, double *out)
{
    if (n < 0 || (n > 0 && (!in || !out))) return -1;
    if (dtype < 0 || dtype > 2) return -2;
    for (int64_t i = 0; i < n; ++i) out[i] = load_elem(in, dtype, i);
    return 0;
}

/* ------------------------------------------------------ the balancer (a1) */

/* Section 2.2 and its workload-balance listing: a data-aware balancer picks
 * the row-split backend when the degrees of most (90%) of the nodes are close
 * to the average degree, otherwise the neighbor-group backend.  "Close" is
 * read as avg/2 <= d <= 2*avg, evaluated exactly in integers:
 *   d >= avg/2  <=>  2*d*n_rows >= nnz,   d <= 2*avg  <=>  d*n_rows <= 2*nnz.
 * Returns 1 (row split) or 2 (neighbor group). */
int oracle_balance_mode(int32_t n_rows, int64_t nnz, const int32_t *rowptr)
{
    if (n_rows < 0 || nnz < 0 || (n_rows > 0 && !rowptr)) return -1;
    if (n_rows == 0) return 1;
    int64_t close = 0;
    for (int32_t i = 0; i < n_rows; ++i) {
        int64_t d = (int64_t)rowptr[i + 1] - rowptr[i];
        if (2 * d * n_rows >= nnz && d * n_rows <= 2 * nnz) ++close;
    }
    return (10 * close >= 9 * (int64_t)n_rows) ? 1 : 2;
}

/* Neighbor groups: every row is cut into consecutive slices of at most
 * group_size edges (an empty row is one empty slice).  With mode 1 (row
 * split) each row is one slice.  Writes (row, begin, end) triples in row
 * order when out != NULL; returns the number of slices. */
int64_t oracle_neighbor_groups(int32_t n_rows, const int32_t *rowptr, int32_t group_size,
                               int32_t mode, int32_t *out)
{
    if (n_rows < 0 || group_size < 1 || (n_rows > 0 && !rowptr)) return -1;
    int64_t n = 0;
    for (int32_t i = 0; i < n_rows; ++i) {
        int32_t beg = rowptr[i], end = rowptr[i + 1];
        if (mode == 1 || end - beg <= group_size) {
            if (out) { out[3 * n] = i; out[3 * n + 1] = beg; out[3 * n + 2] = end; }
            ++n;
            continue;
        }
        for (int32_t s = beg; s < end; s += group_size) {
            int32_t e = (end - s > group_size) ? s + group_size : end;
            if (out) { out[3 * n] = i; out[3 * n + 1] = s; out[3 * n + 2] = e; }
            ++n;
        }
    }
    return n;
}

/* ------------------------------------------------------------- SpMM (a2) */

/* Eq. 1 with reduce = sum and compute = multiply, i.e. H' = A H:
 *   Y[i,f] = sum_{k in row i} val[k] * X[col[k], f]
 * Abs[i,f] = sum |val[k]| * |X[col[k], f]| is the forward-error scale.
 * val == NULL means every edge value is 1. */
int oracle_spmm(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *rowptr,
                const int32_t *col, const float *val, int32_t F, const void *X,
                int32_t x_dtype, int32_t n_sel, const int32_t *sel, double *Y, double *Abs)
{
    if (n_rows < 0 || n_cols < 0 || nnz < 0 || F < 0) return -1;
    int32_t n_out = sel ? n_sel : n_rows;
    #pragma omp parallel for schedule(dynamic, 64)
    for (int32_t r = 0; r < n_out; ++r) {
        int32_t i = sel ? sel[r] : r;
        double *y = Y + (int64_t)r * F;
        double *a = Abs ? Abs + (int64_t)r * F : NULL;
        for (int32_t f = 0; f < F; ++f) { y[f] = 0.0; if (a) a[f] = 0.0; }
        for (int32_t k = rowptr[i]; k < rowptr[i + 1]; ++k) {
            double w = val ? (double)val[k] : 1.0;
            int64_t base = (int64_t)col[k] * F;
            for (int32_t f = 0; f < F; ++f) {
                double x = load_elem(X, x_dtype, base + f);
                y[f] += w * x;
                if (a) a[f] += fabs(w) * fabs(x);
            }
        }
    }
    return 0;
}

/* ------------------------------------------------ GSpMM reduce / compute */

/* The message of edge k for feature f under the compute operator psi of
 * Eq. 1, with w = val[k] (1 when val is NULL): multiply (0) w * x, add (1)
 * x + w, subtract (2) x - w, copy (3) x.  Evaluated in double. */
static double gspmm_message(int32_t compute, double w, double x)
{
    switch (compute) {
    case 0: return w * x;
    case 1: return x + w;
    case 2: return x - w;
    default: return x;
    }
}

/* Eq. 1 with compute psi (above) and reduce phi = sum (0), mean (1) or
 * max (2) over the edges of row i:
 *   sum : Y[i,f] = sum_k m_kf                    Abs[i,f] = sum_k |m_kf|
 *   mean: Y[i,f] = (1/d_i) sum_k m_kf            Abs scaled the same way
 *         (d_i = number of edges of row i, duplicates included)
 *   max : Y[i,f] = max_k fl32(m_kf), arg[i,f] = the first k (CSR order)
 *         attaining it; Abs = 0
 * An empty row gives 0 (and arg -1).  The max compares the messages as the
 * fp32 values a GPU multiply / add produces (the exact result rounded once to
 * float), so the chosen edge is decided in the kernel's precision; its value
 * is then exact.  With compute = multiply, sum is oracle_spmm. */
int oracle_gspmm(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *rowptr,
                 const int32_t *col, const float *val, int32_t F, const void *X, int32_t x_dtype,
                 int32_t reduce, int32_t compute, int32_t n_sel, const int32_t *sel, double *Y,
                 double *Abs, int32_t *arg)
{
    if (n_rows < 0 || n_cols < 0 || nnz < 0 || F < 0 || reduce < 0 || reduce > 2 ||
        compute < 0 || compute > 3)
        return -1;
    int32_t n_out = sel ? n_sel : n_rows;
    #pragma omp parallel for schedule(dynamic, 64)
    for (int32_t r = 0; r < n_out; ++r) {
        int32_t i = sel ? sel[r] : r;
        int32_t d = rowptr[i + 1] - rowptr[i];
        for (int32_t f = 0; f < F; ++f) {
            int64_t t = (int64_t)r * F + f;
            double sum = 0.0, abs_sum = 0.0;
            float best = 0.0f;
            int32_t best_k = -1;
            for (int32_t k = rowptr[i]; k < rowptr[i + 1]; ++k) {
                double w = val ? (double)val[k] : 1.0;
                double x = load_elem(X, x_dtype, (int64_t)col[k] * F + f);
                double m = gspmm_message(compute, w, x);
                if (reduce == 2) {
                    float p = (float)m;
                    if (best_k < 0 || p > best) { best = p; best_k = k; }
                } else {
                    sum += m;
                    abs_sum += fabs(m);
                }
            }
            if (reduce == 2) {
                Y[t] = best_k < 0 ? 0.0 : (double)best;
                if (Abs) Abs[t] = 0.0;
                if (arg) arg[t] = best_k;
            } else {
                if (reduce == 1 && d > 0) { sum /= d; abs_sum /= d; }
                Y[t] = sum;
                if (Abs) Abs[t] = abs_sum;
            }
        }
    }
    return 0;
}

/* ------------------------------------------------------- CSR -> CSC (a3) */

/* Transpose of the sparsity structure by a stable counting sort of the edge
 * ids on their column: colptr is the exclusive prefix sum of the column
 * counts, and inside a column the edges keep increasing CSR edge id.
 * perm[p] = CSR edge id placed at CSC slot p, row_t[p] its row, val_t[p] a
 * bit copy of val[perm[p]] (val / val_t may be NULL together). */
int oracle_csr_to_csc(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *rowptr,
                      const int32_t *col, const float *val, int32_t *colptr, int32_t *row_t,
                      float *val_t, int32_t *perm)
{
    if (n_rows < 0 || n_cols < 0 || nnz < 0) return -1;
    int64_t *next = (int64_t *)calloc((size_t)n_cols + 1, sizeof(int64_t));
    if (!next) return -3;
    for (int64_t k = 0; k < nnz; ++k) next[col[k] + 1]++;
    for (int32_t j = 0; j < n_cols; ++j) next[j + 1] += next[j];
    for (int32_t j = 0; j <= n_cols; ++j) colptr[j] = (int32_t)next[j];
    for (int32_t i = 0; i < n_rows; ++i) {
        for (int32_t k = rowptr[i]; k < rowptr[i + 1]; ++k) {
            int64_t p = next[col[k]]++;
            perm[p] = k;
            row_t[p] = i;
            if (val && val_t) memcpy(&val_t[p], &val[k], sizeof(float));
        }
    }
    free(next);
    return 0;
}

/* ---------------------------------------------- transposed SpMM (a4) */

/* Backward of H' = A H with respect to H:  dX = A^T G, i.e.
 *   dX[j,f] = sum_{k : col[k] = j} val[k] * G[row(k), f]
 * computed by scattering straight from the CSR (not from a CSC), adding the
 * terms of a column in increasing edge id.  With sel != NULL only the listed
 * columns are produced (one pass over all edges). */
int oracle_spmm_t(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *rowptr,
                  const int32_t *col, const float *val, int32_t F, const void *G,
                  int32_t g_dtype, int32_t n_sel, const int32_t *sel, double *dX, double *Abs)
{
    if (n_rows < 0 || n_cols < 0 || nnz < 0 || F < 0) return -1;
    int32_t n_out = sel ? n_sel : n_cols;
    int32_t *slot = (int32_t *)malloc(sizeof(int32_t) * ((size_t)n_cols + 1));
    if (!slot) return -3;
    for (int32_t j = 0; j < n_cols; ++j) slot[j] = sel ? -1 : j;
    if (sel)
        for (int32_t r = 0; r < n_sel; ++r) slot[sel[r]] = r;
    for (int64_t t = 0; t < (int64_t)n_out * F; ++t) { dX[t] = 0.0; if (Abs) Abs[t] = 0.0; }
    for (int32_t i = 0; i < n_rows; ++i) {
        for (int32_t k = rowptr[i]; k < rowptr[i + 1]; ++k) {
            int32_t r = slot[col[k]];
            if (r < 0) continue;
            double w = val ? (double)val[k] : 1.0;
            for (int32_t f = 0; f < F; ++f) {
                double g = load_elem(G, g_dtype, (int64_t)i * F + f);
                dX[(int64_t)r * F + f] += w * g;
                if (Abs) Abs[(int64_t)r * F + f] += fabs(w) * fabs(g);
            }
        }
    }
    free(slot);
    return 0;
}

/* ------------------------------------ SDDMM + LeakyReLU + edge softmax */

/* Additive per-head attention score of edge k = (i, j) for head h:
 *   t = s_dst[i,h] + s_src[j,h],  e = t if t > 0 else slope * t,
 * i.e. the SDDMM A (.) (P Q^T) with P = [s_dst, 1], Q = [1, s_src] per head,
 * followed by LeakyReLU. */
static double edge_score(const float *s_dst, const float *s_src, int32_t H, int32_t i,
                         int32_t j, int32_t h, double slope)
{
    double t = (double)s_dst[(int64_t)i * H + h] + (double)s_src[(int64_t)j * H + h];
    return t > 0.0 ? t : slope * t;
}

/* Edge-wise softmax over the edges of each destination row, per head:
 *   alpha[k,h] = exp(e[k,h] - m) / sum_{k' in row} exp(e[k',h] - m)
 * where m is the row maximum (subtracting it changes nothing mathematically
 * and keeps exp from overflowing).  Output layout alpha[k*H + h]; with sel,
 * the listed rows' edges are packed in list order. */
int oracle_edge_softmax(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *rowptr,
                        const int32_t *col, int32_t H, const float *s_dst, const float *s_src,
                        double slope, int32_t n_sel, const int32_t *sel, double *alpha)
{
    if (n_rows < 0 || n_cols < 0 || nnz < 0 || H < 1) return -1;
    int32_t n_out = sel ? n_sel : n_rows;
    int64_t *off = (int64_t *)malloc(sizeof(int64_t) * ((size_t)n_out + 1));
    if (!off) return -3;
    off[0] = 0;
    for (int32_t r = 0; r < n_out; ++r) {
        int32_t i = sel ? sel[r] : r;
        off[r + 1] = off[r] + (rowptr[i + 1] - rowptr[i]);
    }
    #pragma omp parallel for schedule(dynamic, 64)
    for (int32_t r = 0; r < n_out; ++r) {
        int32_t i = sel ? sel[r] : r;
        int32_t beg = rowptr[i], end = rowptr[i + 1];
        for (int32_t h = 0; h < H; ++h) {
            double m = -INFINITY;
            for (int32_t k = beg; k < end; ++k) {
                double e = edge_score(s_dst, s_src, H, i, col[k], h, slope);
                if (e > m) m = e;
            }
            double z = 0.0;
            for (int32_t k = beg; k < end; ++k)
                z += exp(edge_score(s_dst, s_src, H, i, col[k], h, slope) - m);
            for (int32_t k = beg; k < end; ++k) {
                double e = edge_score(s_dst, s_src, H, i, col[k], h, slope);
                alpha[(off[r] + (k - beg)) * H + h] = exp(e - m) / z;
            }
        }
    }
    free(off);
    return 0;
}

/* ------------------------------------------------- multi-head SpMM (a7) */

/* GAT aggregation with one weight per edge and head:
 *   Y[i,h,d] = sum_{k in row i} alpha[k,h] * X[col[k], h, d]
 * X and Y are [node][head][d] row-major.  With alpha_in == NULL the weights
 * are the edge softmax above, kept in double; otherwise alpha_in[k*H+h] (fp32)
 * is used exactly. */
int oracle_gat(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *rowptr,
               const int32_t *col, int32_t H, int32_t D, const float *s_dst, const float *s_src,
               double slope, const float *alpha_in, const void *X, int32_t x_dtype,
               int32_t n_sel, const int32_t *sel, double *Y, double *Abs)
{
    if (n_rows < 0 || n_cols < 0 || nnz < 0 || H < 1 || D < 0) return -1;
    int32_t n_out = sel ? n_sel : n_rows;
    int64_t HD = (int64_t)H * D;
    int rc = 0;
    #pragma omp parallel for schedule(dynamic, 16)
    for (int32_t r = 0; r < n_out; ++r) {
        int32_t i = sel ? sel[r] : r;
        int32_t beg = rowptr[i], end = rowptr[i + 1];
        int32_t deg = end - beg;
        double *y = Y + (int64_t)r * HD;
        double *a = Abs ? Abs + (int64_t)r * HD : NULL;
        for (int64_t t = 0; t < HD; ++t) { y[t] = 0.0; if (a) a[t] = 0.0; }
        if (deg == 0) continue;
        double *w = (double *)malloc(sizeof(double) * (size_t)deg * H);
        if (!w) { rc = -3; continue; }
        if (alpha_in) {
            for (int32_t k = beg; k < end; ++k)
                for (int32_t h = 0; h < H; ++h)
                    w[(int64_t)(k - beg) * H + h] = (double)alpha_in[(int64_t)k * H + h];
        } else {
            oracle_edge_softmax(n_rows, n_cols, nnz, rowptr, col, H, s_dst, s_src, slope, 1, &i, w);
        }
        for (int32_t k = beg; k < end; ++k) {
            int64_t base = (int64_t)col[k] * HD;
            for (int32_t h = 0; h < H; ++h) {
                double wk = w[(int64_t)(k - beg) * H + h];
                for (int32_t d = 0; d < D; ++d) {
                    double x = load_elem(X, x_dtype, base + (int64_t)h * D + d);
                    y[(int64_t)h * D + d] += wk * x;
                    if (a) a[(int64_t)h * D + d] += fabs(wk) * fabs(x);
                }
            }
        }
        free(w);
    }
    return rc;
}

/* ---------------------------------------------------- GAT backward (next) */

/* Gradients of the GAT layer of section 2.2 for a loss L with dY = dL/dY,
 * derived by the chain rule through the forward operators (score SDDMM,
 * LeakyReLU, edge softmax per row, weighted multi-head SpMM).  For edge
 * k = (i, j) and head h, with alpha the forward weights (given, used exactly):
 *   dalpha[k,h] = sum_d dY[i,h,d] * X[j,h,d]
 *                 (the dot-product SDDMM A (.) (dY_h X_h^T) of section 2.2,
 *                  which carries the gradient to the attention matrix)
 *   c[i,h]      = sum_{k in row i} alpha[k,h] * dalpha[k,h]
 *   dscore[k,h] = f_kh * alpha[k,h] * (dalpha[k,h] - c[i,h])
 *                 (softmax backward times the LeakyReLU slope: f = 1 when the
 *                  pre-activation t = s_dst[i,h] + s_src[j,h] is > 0, else slope)
 *   ds_dst[i,h] = sum_{k in row i} dscore[k,h]
 *   ds_src[j,h] = sum_{k: col[k] = j} dscore[k,h]
 *   dX[j,h,d]   = sum_{k: col[k] = j} alpha[k,h] * dY[i,h,d]
 * Each value comes with its error scale (_abs): the same expression with
 * every term replaced by its absolute value and every difference by a sum.
 * Row outputs (dalpha, dscore: packed edges of the selected rows in list and
 * CSR order; ds_dst) are for rows sel[0..n_sel) (all when sel is NULL);
 * column outputs (ds_src, dX) for columns csel[0..n_csel) (all when NULL).
 * Any output may be NULL.  Sums run over edges in CSR order. */
static void gat_bwd_row(int32_t i, const int32_t *rowptr, const int32_t *col, int32_t H,
                        int32_t D, const float *s_dst, const float *s_src, double slope,
                        const float *alpha, const void *X, int32_t x_dtype, const void *dY,
                        int32_t dy_dtype, double *da, double *da_abs, double *dt, double *dt_abs)
{
    int32_t beg = rowptr[i], end = rowptr[i + 1];
    int64_t HD = (int64_t)H * D;
    for (int32_t h = 0; h < H; ++h) {
        double c = 0.0, c_abs = 0.0;
        for (int32_t k = beg; k < end; ++k) {
            double s = 0.0, s_abs = 0.0;
            for (int32_t d = 0; d < D; ++d) {
                double g = load_elem(dY, dy_dtype, (int64_t)i * HD + (int64_t)h * D + d);
                double x = load_elem(X, x_dtype, (int64_t)col[k] * HD + (int64_t)h * D + d);
                s += g * x;
                s_abs += fabs(g) * fabs(x);
            }
            int64_t e = (int64_t)(k - beg) * H + h;
            da[e] = s;
            da_abs[e] = s_abs;
            double a = (double)alpha[(int64_t)k * H + h];
            c += a * s;
            c_abs += fabs(a) * s_abs;
        }
        for (int32_t k = beg; k < end; ++k) {
            int64_t e = (int64_t)(k - beg) * H + h;
            double t = (double)s_dst[(int64_t)i * H + h] + (double)s_src[(int64_t)col[k] * H + h];
            double f = t > 0.0 ? 1.0 : slope;
            double a = (double)alpha[(int64_t)k * H + h];
            dt[e] = f * a * (da[e] - c);
            dt_abs[e] = fabs(f) * fabs(a) * (da_abs[e] + c_abs);
        }
    }
}

int oracle_gat_backward(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *rowptr,
                        const int32_t *col, int32_t H, int32_t D, const float *s_dst,
                        const float *s_src, double slope, const float *alpha, const void *X,
                        int32_t x_dtype, const void *dY, int32_t dy_dtype, int32_t n_sel,
                        const int32_t *sel, double *dalpha, double *dalpha_abs, double *dscore,
                        double *dscore_abs, double *ds_dst, double *ds_dst_abs, int32_t n_csel,
                        const int32_t *csel, double *ds_src, double *ds_src_abs, double *dX,
                        double *dX_abs)
{
    if (n_rows < 0 || n_cols < 0 || nnz < 0 || H < 1 || D < 0) return -1;
    int64_t HD = (int64_t)H * D;
    int rc = 0;

    /* row outputs */
    int32_t n_out = sel ? n_sel : n_rows;
    int64_t *off = (int64_t *)malloc(sizeof(int64_t) * ((size_t)n_out + 1));
    if (!off) return -3;
    off[0] = 0;
    for (int32_t r = 0; r < n_out; ++r) {
        int32_t i = sel ? sel[r] : r;
        off[r + 1] = off[r] + (rowptr[i + 1] - rowptr[i]);
    }
    #pragma omp parallel for schedule(dynamic, 16)
    for (int32_t r = 0; r < n_out; ++r) {
        int32_t i = sel ? sel[r] : r;
        int32_t deg = rowptr[i + 1] - rowptr[i];
        size_t n = (size_t)deg * H + 1;
        double *da = (double *)malloc(sizeof(double) * n), *dab = (double *)malloc(sizeof(double) * n);
        double *dt = (double *)malloc(sizeof(double) * n), *dtb = (double *)malloc(sizeof(double) * n);
        if (!da || !dab || !dt || !dtb) {
            rc = -3;
        } else {
            gat_bwd_row(i, rowptr, col, H, D, s_dst, s_src, slope, alpha, X, x_dtype, dY, dy_dtype,
                        da, dab, dt, dtb);
            for (int32_t h = 0; h < H; ++h) {
                double s = 0.0, sb = 0.0;
                for (int32_t e = 0; e < deg; ++e) {
                    int64_t q = (off[r] + e) * H + h, p = (int64_t)e * H + h;
                    if (dalpha) dalpha[q] = da[p];
                    if (dalpha_abs) dalpha_abs[q] = dab[p];
                    if (dscore) dscore[q] = dt[p];
                    if (dscore_abs) dscore_abs[q] = dtb[p];
                    s += dt[p];
                    sb += dtb[p];
                }
                if (ds_dst) ds_dst[(int64_t)r * H + h] = s;
                if (ds_dst_abs) ds_dst_abs[(int64_t)r * H + h] = sb;
            }
        }
        free(da); free(dab); free(dt); free(dtb);
    }
    free(off);
    if (rc != 0 || (!ds_src && !ds_src_abs && !dX && !dX_abs)) return rc;

    /* column outputs: the edges into the selected columns, from the rows holding them */
    int32_t n_cout = csel ? n_csel : n_cols;
    int32_t *slot = (int32_t *)malloc(sizeof(int32_t) * ((size_t)n_cols + 1));
    char *need = (char *)calloc((size_t)n_rows + 1, 1);
    int64_t *roff = (int64_t *)malloc(sizeof(int64_t) * ((size_t)n_rows + 1));
    if (!slot || !need || !roff) { free(slot); free(need); free(roff); return -3; }
    for (int32_t j = 0; j < n_cols; ++j) slot[j] = csel ? -1 : j;
    if (csel)
        for (int32_t c = 0; c < n_csel; ++c) slot[csel[c]] = c;
    for (int32_t i = 0; i < n_rows; ++i)
        for (int32_t k = rowptr[i]; k < rowptr[i + 1] && !need[i]; ++k)
            if (slot[col[k]] >= 0) need[i] = 1;
    roff[0] = 0;
    for (int32_t i = 0; i < n_rows; ++i)
        roff[i + 1] = roff[i] + (need[i] ? (int64_t)(rowptr[i + 1] - rowptr[i]) * H : 0);
    double *dt = (double *)malloc(sizeof(double) * ((size_t)roff[n_rows] + 1));
    double *dtb = (double *)malloc(sizeof(double) * ((size_t)roff[n_rows] + 1));
    if (!dt || !dtb) { free(slot); free(need); free(roff); free(dt); free(dtb); return -3; }
    #pragma omp parallel for schedule(dynamic, 16)
    for (int32_t i = 0; i < n_rows; ++i) {
        if (!need[i]) continue;
        size_t n = (size_t)(rowptr[i + 1] - rowptr[i]) * H + 1;
        double *da = (double *)malloc(sizeof(double) * n), *dab = (double *)malloc(sizeof(double) * n);
        if (!da || !dab) { rc = -3; free(da); free(dab); continue; }
        gat_bwd_row(i, rowptr, col, H, D, s_dst, s_src, slope, alpha, X, x_dtype, dY, dy_dtype,
                    da, dab, dt + roff[i], dtb + roff[i]);
        free(da); free(dab);
    }
    if (rc == 0) {
        for (int32_t c = 0; c < n_cout; ++c) {
            for (int32_t h = 0; h < H; ++h) {
                if (ds_src) ds_src[(int64_t)c * H + h] = 0.0;
                if (ds_src_abs) ds_src_abs[(int64_t)c * H + h] = 0.0;
            }
            for (int64_t t = 0; t < HD; ++t) {
                if (dX) dX[(int64_t)c * HD + t] = 0.0;
                if (dX_abs) dX_abs[(int64_t)c * HD + t] = 0.0;
            }
        }
        for (int32_t i = 0; i < n_rows; ++i) {
            if (!need[i]) continue;
            for (int32_t k = rowptr[i]; k < rowptr[i + 1]; ++k) {
                int32_t c = slot[col[k]];
                if (c < 0) continue;
                for (int32_t h = 0; h < H; ++h) {
                    int64_t p = roff[i] + (int64_t)(k - rowptr[i]) * H + h;
                    if (ds_src) ds_src[(int64_t)c * H + h] += dt[p];
                    if (ds_src_abs) ds_src_abs[(int64_t)c * H + h] += dtb[p];
                    double a = (double)alpha[(int64_t)k * H + h];
                    for (int32_t d = 0; d < D; ++d) {
                        double g = load_elem(dY, dy_dtype, (int64_t)i * HD + (int64_t)h * D + d);
                        if (dX) dX[(int64_t)c * HD + (int64_t)h * D + d] += a * g;
                        if (dX_abs) dX_abs[(int64_t)c * HD + (int64_t)h * D + d] += fabs(a) * fabs(g);
                    }
                }
            }
        }
    }
    free(slot); free(need); free(roff); free(dt); free(dtb);
    return rc;
}

/* The dot-product SDDMM of section 2.2, T = A (.) (P Q^T), per head:
 *   out[k,h] = sum_d P[i,h,d] * Q[col[k],h,d]   for edge k = (i, col[k])
 * (structure only: the edge values of A are not applied), with its error
 * scale; rows sel[0..n_sel) (all when NULL), edges packed as above. */
int oracle_sddmm_dot(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *rowptr,
                     const int32_t *col, int32_t H, int32_t D, const void *P, int32_t p_dtype,
                     const void *Q, int32_t q_dtype, int32_t n_sel, const int32_t *sel, double *out,
                     double *out_abs)
{
    if (n_rows < 0 || n_cols < 0 || nnz < 0 || H < 1 || D < 0) return -1;
    int64_t HD = (int64_t)H * D;
    int32_t n_out = sel ? n_sel : n_rows;
    int64_t *off = (int64_t *)malloc(sizeof(int64_t) * ((size_t)n_out + 1));
    if (!off) return -3;
    off[0] = 0;
    for (int32_t r = 0; r < n_out; ++r) {
        int32_t i = sel ? sel[r] : r;
        off[r + 1] = off[r] + (rowptr[i + 1] - rowptr[i]);
    }
    #pragma omp parallel for schedule(dynamic, 64)
    for (int32_t r = 0; r < n_out; ++r) {
        int32_t i = sel ? sel[r] : r;
        for (int32_t k = rowptr[i]; k < rowptr[i + 1]; ++k)
            for (int32_t h = 0; h < H; ++h) {
                double s = 0.0, sb = 0.0;
                for (int32_t d = 0; d < D; ++d) {
                    double p = load_elem(P, p_dtype, (int64_t)i * HD + (int64_t)h * D + d);
                    double q = load_elem(Q, q_dtype, (int64_t)col[k] * HD + (int64_t)h * D + d);
                    s += p * q;
                    sb += fabs(p) * fabs(q);
                }
                int64_t e = (off[r] + (k - rowptr[i])) * H + h;
                out[e] = s;
                if (out_abs) out_abs[e] = sb;
            }
    }
    free(off);
    return 0;
}

/* ------------------------------------------------ dense layers (next row 3) */

/* The activations of the layer epilogues: 0 identity, 1 ReLU max(v, 0),
 * 2 ELU (v > 0 ? v : exp(v) - 1). */
static double act_apply(int32_t act, double v)
{
    if (act == 1) return v > 0.0 ? v : 0.0;
    if (act == 2) return v > 0.0 ? v : expm1(v);
    return v;
}

/* In-place act(v + bias[f]) over an n x F array (bias may be NULL). */
int oracle_epilogue(int64_t n, int32_t F, const float *bias, int32_t act, double *v)
{
    if (n < 0 || F < 0 || act < 0 || act > 2) return -1;
    for (int64_t i = 0; i < n; ++i)
        for (int32_t f = 0; f < F; ++f) {
            double x = v[i * F + f] + (bias ? (double)bias[f] : 0.0);
            v[i * F + f] = act_apply(act, x);
        }
    return 0;
}

/* Dense layer: Y[i,c] = act(sum_j X[i,j] W[c,j] + bias[c]) with X n x k and W
 * m x k (the layer's out x in weights), in double; Abs[i,c] = sum_j |X||W| +
 * |bias[c]| (the activations are 1-Lipschitz, so it bounds the error of the
 * activated value too). */
int oracle_linear(int64_t n, int32_t k, int32_t m, const void *X, int32_t x_dtype, const void *W,
                  int32_t w_dtype, const float *bias, int32_t act, double *Y, double *Abs)
{
    if (n < 0 || k < 0 || m < 0 || act < 0 || act > 2) return -1;
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        for (int32_t c = 0; c < m; ++c) {
            double s = 0.0, sa = 0.0;
            for (int32_t j = 0; j < k; ++j) {
                double x = load_elem(X, x_dtype, i * k + j);
                double w = load_elem(W, w_dtype, (int64_t)c * k + j);
                s += x * w;
                sa += fabs(x) * fabs(w);
            }
            double b = bias ? (double)bias[c] : 0.0;
            Y[i * m + c] = act_apply(act, s + b);
            if (Abs) Abs[i * m + c] = sa + fabs(b);
        }
    return 0;
}

/* Per-head attention scores: s_src[i,h] = sum_d Z[i,h,d] a_src[h,d], s_dst
 * likewise with a_dst, in double, with their error scales (sums of |terms|). */
int oracle_head_scores(int64_t n, int32_t H, int32_t D, const void *Z, int32_t z_dtype,
                       const float *a_src, const float *a_dst, double *s_src, double *s_dst,
                       double *src_abs, double *dst_abs)
{
    if (n < 0 || H < 1 || D < 1) return -1;
    int64_t HD = (int64_t)H * D;
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        for (int32_t h = 0; h < H; ++h) {
            double ps = 0.0, pd = 0.0, as = 0.0, ad = 0.0;
            for (int32_t d = 0; d < D; ++d) {
                double z = load_elem(Z, z_dtype, i * HD + (int64_t)h * D + d);
                ps += z * (double)a_src[(int64_t)h * D + d];
                pd += z * (double)a_dst[(int64_t)h * D + d];
                as += fabs(z) * fabs((double)a_src[(int64_t)h * D + d]);
                ad += fabs(z) * fabs((double)a_dst[(int64_t)h * D + d]);
            }
            s_src[i * H + h] = ps;
            s_dst[i * H + h] = pd;
            if (src_abs) src_abs[i * H + h] = as;
            if (dst_abs) dst_abs[i * H + h] = ad;
        }
    return 0;
}

/* ------------------------------------- activation compression (next row 4) */

/* Philox4x32-10, the counter-based generator of Salmon, Moraes, Dror and Shaw
 * ("Parallel random numbers: as easy as 1, 2, 3", SC 2011): ten rounds of two
 * 32x32 -> 64-bit multiplications (multipliers 0xD2511F53 and 0xCD9E8D57)
 * whose high halves are xored with the other counter words and the key, the
 * key advanced by the Weyl constants 0x9E3779B9 and 0xBB67AE85 between
 * rounds. */
void oracle_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
    uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) { k0 += 0x9E3779B9u; k1 += 0xBB67AE85u; }
        uint64_t p0 = (uint64_t)0xD2511F53u * c0;
        uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        uint32_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
        c0 = n0; c1 = lo1; c2 = n2; c3 = lo0;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* Uniform in [0, 1) for element e of an activation array: word e mod 4 of
 * Philox4x32-10 at counter (e / 4 low, e / 4 high, 0, 0) with key (seed low,
 * seed high), its top 24 bits scaled by 2^-24 (exact in fp32). */
static float codec_uniform(uint64_t seed, int64_t e)
{
    uint32_t ctr[4] = {(uint32_t)((uint64_t)e >> 2), (uint32_t)((uint64_t)e >> 34), 0u, 0u};
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    uint32_t r[4];
    oracle_philox4x32_10(ctr, key, r);
    return (float)(r[e & 3] >> 8) * (1.0f / 16777216.0f);
}

/* Per-group b-bit quantization with stochastic rounding (activation
 * compression, section 2 and the activation-memory table of the evaluation;
 * the scheme follows the ActNN line of work the paper builds on):
 * each row of the n x F array A is cut into groups of G consecutive features
 * (G a multiple of 64, the last group of a row may be shorter).  For a group
 * with minimum m and maximum M (fp32), range = M - m, s = (2^b - 1) / range and
 * r = range / (2^b - 1) (both 0 when range is 0), every element x gets the
 * code  q = clamp(floor(fma(x - m, s, u)), 0, 2^b - 1)  with u the uniform of
 * its flat index e = i * F + f, all in fp32 (so the integer decision is taken
 * in the kernel's precision).  Codes are stored as bit planes: each block of 64
 * consecutive codes of a group is b uint64 words, word p holding bit p of
 * code j at bit j (codes past the end of the row are 0).  stats[2g], stats[2g+1]
 * = (m, r).  Decoding: x' = fma(q, r, m). */
int oracle_act_compress(int64_t n, int32_t F, const void *A, int32_t a_dtype, int32_t bits,
                        int32_t G, uint64_t seed, uint64_t *codes, float *stats)
{
    if (n < 0 || F < 1 || bits < 1 || bits > 8 || G < 64 || G % 64 != 0) return -1;
    int32_t ng = (F + G - 1) / G, nb = G / 64;
    float qmax = (float)((1 << bits) - 1);
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        for (int32_t gi = 0; gi < ng; ++gi) {
            int64_t g = i * ng + gi;
            int32_t f0 = gi * G, f1 = f0 + G < F ? f0 + G : F;
            float m = (float)load_elem(A, a_dtype, i * F + f0), M = m;
            for (int32_t f = f0; f < f1; ++f) {
                float x = (float)load_elem(A, a_dtype, i * F + f);
                if (x < m) m = x;
                if (x > M) M = x;
            }
            float range = M - m;
            float s = range > 0.0f ? qmax / range : 0.0f;
            float r = range > 0.0f ? range / qmax : 0.0f;
            stats[2 * g] = m;
            stats[2 * g + 1] = r;
            uint64_t *w = codes + g * (int64_t)nb * bits;
            for (int64_t t = 0; t < (int64_t)nb * bits; ++t) w[t] = 0;
            for (int32_t f = f0; f < f1; ++f) {
                float x = (float)load_elem(A, a_dtype, i * F + f);
                float u = codec_uniform(seed, i * F + f);
                float v = floorf(fmaf(x - m, s, u));
                if (v < 0.0f) v = 0.0f;
                if (v > qmax) v = qmax;
                uint32_t q = (uint32_t)v;
                int32_t j = f - f0, blk = j / 64, bit = j % 64;
                for (int32_t p = 0; p < bits; ++p)
                    if ((q >> p) & 1u) w[(int64_t)blk * bits + p] |= (uint64_t)1 << bit;
            }
        }
    return 0;
}

/* The decoded n x F array (fp32 values; callers round to the output format). */
int oracle_act_decompress(int64_t n, int32_t F, int32_t bits, int32_t G, const uint64_t *codes,
                          const float *stats, float *out)
{
    if (n < 0 || F < 1 || bits < 1 || bits > 8 || G < 64 || G % 64 != 0) return -1;
    int32_t ng = (F + G - 1) / G, nb = G / 64;
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        for (int32_t f = 0; f < F; ++f) {
            int64_t g = i * ng + f / G;
            int32_t j = f % G, blk = j / 64, bit = j % 64;
            const uint64_t *w = codes + g * (int64_t)nb * bits + (int64_t)blk * bits;
            uint32_t q = 0;
            for (int32_t p = 0; p < bits; ++p) q |= (uint32_t)((w[p] >> bit) & 1u) << p;
            out[i * F + f] = fmaf((float)q, stats[2 * g + 1], stats[2 * g]);
        }
    return 0;
}
