/*
 * rt3d_oracle.c -- plain CPU oracle for kernel-group-structured (KGS) sparse
 * 3-D convolution.  TEST INFRASTRUCTURE ONLY: the test-suite, the smoke check
 * and the CPU-baseline leg of the benchmark call it; the product library never
 * links, loads or calls it, and it shares no code, header or table with the
 * GPU path.
 *
 * Everything here is written straight from the definitions in the paper
 * (RT3D, arXiv 2007.09835):
 *   - Section 3: a CONV layer's weight tensor is 5-D, M filters x N input
 *     channels x a 3-D kernel; it is partitioned into kernel groups of
 *     g_M x g_N kernels.
 *   - Section 3, Fig. 1(b): under KGS sparsity all kernels of one group are
 *     pruned at the same kernel locations; a vanilla-pruned group is the
 *     special case where every location of the group is pruned.
 *   - Section 3 (reshaping paragraph): each group, reshaped to a
 *     g_M x (g_N * K_s) matrix, loses whole columns, so the KGS layer is the
 *     dense layer with the pruned weights removed.
 *   - Section 4: P = ceil(M / g_M), Q = ceil(N / g_N); trailing groups are
 *     partial.
 *   - Section 4 (regularization-based and reweighted pruning): the l1 / l2
 *     norm of a group's weights at one kernel position (KGS) or over the
 *     whole group (vanilla), the penalty term of eq. (3) and the update of
 *     its penalty factors.
 *
 * Conventions (the paper is silent on them; readings recorded in the design
 * notes):
 *   x        [n][c_in][t][h][w]                 (input, NCDHW)
 *   w        [c_out][c_in][kt][kh][kw]          (kt = kernel depth K_d)
 *   mask     [P][Q][kt*kh*kw], 1 = keep, 0 = pruned; the kernel position
 *            index is pos = (it*kh + ih)*kw + iw
 *   y        [n][c_out][to][ho][wo], to = (t + 2*pt - kt)/st + 1 etc.
 *   The operation is cross-correlation (no kernel flip), zero padding.
 *   y = act(sum + bias[m] + residual), act = max(.,0) when relu != 0.
 *
 * Arithmetic: inputs arrive as float64 (exact images of the bf16 / fp16 /
 * fp32 values the GPU path consumes); every product and sum is float64.
 * Parallelism: OpenMP over (batch, filter); each output is one sequential
 * sum, so results do not depend on the thread count.
 */
#include <stdint.h>
#include <stddef.h>
#include <string.h>
#include <math.h>

#define ORACLE_OK 0
#define ORACLE_BAD_ARG 1

/* Output length of a zero-padded, strided correlation along one axis
 * (floor division; returns <= 0 when the kernel does not fit). */
static long out_len(long in, long k, long s, long p)
{
    long span = in + 2 * p - k;
    if (span < 0) return 0;
    return span / s + 1;
}

static int check_geometry(int n, int c_in, int c_out, int t, int h, int w,
                          int kt, int kh, int kw, int st, int sh, int sw,
                          int pt, int ph, int pw)
{
    if (n < 0 || c_in <= 0 || c_out <= 0 || t <= 0 || h <= 0 || w <= 0) return ORACLE_BAD_ARG;
    if (kt <= 0 || kh <= 0 || kw <= 0 || st <= 0 || sh <= 0 || sw <= 0) return ORACLE_BAD_ARG;
    if (pt < 0 || ph < 0 || pw < 0) return ORACLE_BAD_ARG;
    if (out_len(t, kt, st, pt) <= 0 || out_len(h, kh, sh, ph) <= 0 || out_len(w, kw, sw, pw) <= 0)
        return ORACLE_BAD_ARG;
    return ORACLE_OK;
}

/* Geometry of one layer, gathered so the per-output sum reads cleanly. */
typedef struct {
    long n, c_in, c_out, t, h, w, kt, kh, kw, st, sh, sw, pt, ph, pw, g_m, g_n;
    long to, ho, wo, ks, q_groups;
} geom;

static geom make_geom(int n, int c_in, int c_out, int t, int h, int w,
                      int kt, int kh, int kw, int st, int sh, int sw,
                      int pt, int ph, int pw, int g_m, int g_n)
{
    geom g = {n, c_in, c_out, t, h, w, kt, kh, kw, st, sh, sw, pt, ph, pw, g_m, g_n,
              0, 0, 0, 0, 0};
    g.to = out_len(t, kt, st, pt);
    g.ho = out_len(h, kh, sh, ph);
    g.wo = out_len(w, kw, sw, pw);
    g.ks = (long)kt * kh * kw;
    g.q_groups = g_n > 0 ? (c_in + g_n - 1) / g_n : 0;
    return g;
}

/*
 * One output value y[b][m][ot][oh][ow].  When mask is NULL every weight takes
 * part (the dense 3-D CONV of Section 3); otherwise a weight W[m][c][pos]
 * takes part only when mask[m / g_m][c / g_n][pos] == 1 (KGS, Section 3).
 * A pruned weight is never read, so its stored value cannot reach y.
 */
static double one_output(const geom *g, long b, long m, long ot, long oh, long ow,
                         const double *x, const double *wt, const uint8_t *mask,
                         const double *bias, const double *residual, int relu)
{
    const long in_vol = g->t * g->h * g->w;
    double acc = 0.0;
    for (long c = 0; c < g->c_in; ++c)
    for (long it = 0; it < g->kt; ++it)
    for (long ih = 0; ih < g->kh; ++ih)
    for (long iw = 0; iw < g->kw; ++iw) {
        const long pos = (it * g->kh + ih) * g->kw + iw;
        if (mask) {
            const long p = m / g->g_m, q = c / g->g_n;
            if (mask[(p * g->q_groups + q) * g->ks + pos] != 1) continue;
        }
        const long zt = ot * g->st + it - g->pt;
        const long zh = oh * g->sh + ih - g->ph;
        const long zw = ow * g->sw + iw - g->pw;
        if (zt < 0 || zt >= g->t || zh < 0 || zh >= g->h || zw < 0 || zw >= g->w) continue;
        const double xv = x[(b * g->c_in + c) * in_vol + (zt * g->h + zh) * g->w + zw];
        const double wv = wt[(m * g->c_in + c) * g->ks + pos];
        acc += wv * xv;
    }
    if (bias) acc += bias[m];
    if (residual) acc += residual[(b * g->c_out + m) * (g->to * g->ho * g->wo)
                                  + (ot * g->ho + oh) * g->wo + ow];
    if (relu && !(acc > 0.0)) acc = 0.0;
    return acc;
}

static int conv3d_direct(int n, int c_in, int c_out, int t, int h, int w,
                         int kt, int kh, int kw, int st, int sh, int sw,
                         int pt, int ph, int pw, int g_m, int g_n,
                         const double *x, const double *wt, const uint8_t *mask,
                         const double *bias, const double *residual, int relu,
                         double *y)
{
    if (check_geometry(n, c_in, c_out, t, h, w, kt, kh, kw, st, sh, sw, pt, ph, pw))
        return ORACLE_BAD_ARG;
    if (!x || !wt || !y) return ORACLE_BAD_ARG;
    if (mask && (g_m <= 0 || g_n <= 0)) return ORACLE_BAD_ARG;
    const geom g = make_geom(n, c_in, c_out, t, h, w, kt, kh, kw, st, sh, sw, pt, ph, pw,
                             g_m, g_n);
    const long out_vol = g.to * g.ho * g.wo;
    long nm;
#pragma omp parallel for schedule(dynamic, 1)
    for (nm = 0; nm < (long)n * c_out; ++nm) {
        const long b = nm / c_out, m = nm % c_out;
        for (long ot = 0; ot < g.to; ++ot)
        for (long oh = 0; oh < g.ho; ++oh)
        for (long ow = 0; ow < g.wo; ++ow)
            y[nm * out_vol + (ot * g.ho + oh) * g.wo + ow] =
                one_output(&g, b, m, ot, oh, ow, x, wt, mask, bias, residual, relu);
    }
    return ORACLE_OK;
}

static int mask_is_binary(int c_out, int c_in, int kt, int kh, int kw, int g_m, int g_n,
                          const uint8_t *mask)
{
    const long p_groups = (c_out + g_m - 1) / g_m;
    const long q_groups = (c_in + g_n - 1) / g_n;
    const long cells = p_groups * q_groups * (long)kt * kh * kw;
    for (long i = 0; i < cells; ++i)
        if (mask[i] > 1) return 0;
    return 1;
}

/* Dense 3-D CONV layer (Section 3: 5-D weight tensor, M x N x 3-D kernel). */
int oracle_conv3d_dense(int n, int c_in, int c_out, int t, int h, int w,
                        int kt, int kh, int kw, int st, int sh, int sw,
                        int pt, int ph, int pw,
                        const double *x, const double *wt, const double *bias,
                        const double *residual, int relu, double *y)
{
    return conv3d_direct(n, c_in, c_out, t, h, w, kt, kh, kw, st, sh, sw, pt, ph, pw,
                         0, 0, x, wt, NULL, bias, residual, relu, y);
}

/* KGS-sparse 3-D CONV layer (Section 3, Fig. 1(b); vanilla is the special
 * case of all-0 / all-1 mask rows).  Every mask byte must be 0 or 1. */
int oracle_conv3d_kgs(int n, int c_in, int c_out, int t, int h, int w,
                      int kt, int kh, int kw, int st, int sh, int sw,
                      int pt, int ph, int pw, int g_m, int g_n,
                      const double *x, const double *wt, const uint8_t *mask,
                      const double *bias, const double *residual, int relu,
                      double *y)
{
    if (!mask || g_m <= 0 || g_n <= 0 || kt <= 0 || kh <= 0 || kw <= 0) return ORACLE_BAD_ARG;
    if (!mask_is_binary(c_out, c_in, kt, kh, kw, g_m, g_n, mask)) return ORACLE_BAD_ARG;
    return conv3d_direct(n, c_in, c_out, t, h, w, kt, kh, kw, st, sh, sw, pt, ph, pw,
                         g_m, g_n, x, wt, mask, bias, residual, relu, y);
}

/* The KGS layer evaluated only at selected outputs: idx[i] is the flat index
 * of y[b][m][ot][oh][ow] in the [n][c_out][to][ho][wo] array; out[i] receives
 * that value.  Same per-output sum as the full layer, so a sampled check of a
 * layer too large for the full oracle compares against identical arithmetic.
 * mask == NULL evaluates the dense layer. */
int oracle_conv3d_points(int n, int c_in, int c_out, int t, int h, int w,
                         int kt, int kh, int kw, int st, int sh, int sw,
                         int pt, int ph, int pw, int g_m, int g_n,
                         const double *x, const double *wt, const uint8_t *mask,
                         const double *bias, const double *residual, int relu,
                         long npoints, const int64_t *idx, double *out)
{
    if (check_geometry(n, c_in, c_out, t, h, w, kt, kh, kw, st, sh, sw, pt, ph, pw))
        return ORACLE_BAD_ARG;
    if (!x || !wt || (npoints > 0 && (!idx || !out))) return ORACLE_BAD_ARG;
    if (mask && (g_m <= 0 || g_n <= 0 || !mask_is_binary(c_out, c_in, kt, kh, kw, g_m, g_n, mask)))
        return ORACLE_BAD_ARG;
    const geom g = make_geom(n, c_in, c_out, t, h, w, kt, kh, kw, st, sh, sw, pt, ph, pw,
                             g_m, g_n);
    const long out_vol = g.to * g.ho * g.wo;
    const long total = (long)n * c_out * out_vol;
    for (long i = 0; i < npoints; ++i)
        if (idx[i] < 0 || idx[i] >= total) return ORACLE_BAD_ARG;
    long i;
#pragma omp parallel for schedule(dynamic, 16)
    for (i = 0; i < npoints; ++i) {
        long r = idx[i];
        const long ow = r % g.wo; r /= g.wo;
        const long oh = r % g.ho; r /= g.ho;
        const long ot = r % g.to; r /= g.to;
        const long m = r % c_out;
        const long b = r / c_out;
        out[i] = one_output(&g, b, m, ot, oh, ow, x, wt, mask, bias, residual, relu);
    }
    return ORACLE_OK;
}

/*
 * Compact per-group weight format (Section 3, reshaping paragraph: each
 * kernel group is a g_M x (g_N * K_s) matrix, and KGS pruning removes whole
 * columns of it).  Groups are visited p-major, q-minor.  For group g = p*Q+q
 * with kept positions pos_0 < pos_1 < ... < pos_{k-1}:
 *   group_ptr[g] .. group_ptr[g+1]   its slice of pos[] (k entries, ascending)
 *   val_ptr[g]   .. val_ptr[g+1]     its slice of vals[] (gm * gn * k entries)
 *   vals[val_ptr[g] + (i * gn + j) * k + r] = W[p*g_m + i][q*g_n + j][pos_r]
 * where gm = min(g_m, M - p*g_m), gn = min(g_n, N - q*g_n) (partial edge
 * groups of Section 4).  That is the group matrix, row i = filter, column
 * (j, r) = (channel in group, kept position), with pruned columns dropped.
 * Element bytes are copied verbatim (esize bytes each).
 *
 * Passing NULL for every output array only counts: *total_pos receives the
 * number of kept positions summed over groups, *total_vals the number of
 * weights kept.
 */
int oracle_kgs_pack(int c_out, int c_in, int kt, int kh, int kw, int g_m, int g_n,
                    int esize, const void *w, const uint8_t *mask,
                    uint32_t *group_ptr, uint16_t *pos, uint64_t *val_ptr, void *vals,
                    uint64_t *total_pos, uint64_t *total_vals)
{
    if (c_out <= 0 || c_in <= 0 || kt <= 0 || kh <= 0 || kw <= 0 || g_m <= 0 || g_n <= 0)
        return ORACLE_BAD_ARG;
    if (!mask || esize <= 0) return ORACLE_BAD_ARG;
    const long ks = (long)kt * kh * kw;
    const long p_groups = (c_out + g_m - 1) / g_m;
    const long q_groups = (c_in + g_n - 1) / g_n;
    const int writing = (group_ptr || pos || val_ptr || vals);
    if (writing && !(group_ptr && pos && val_ptr && vals && w)) return ORACLE_BAD_ARG;

    uint64_t npos = 0, nval = 0;
    for (long p = 0; p < p_groups; ++p) {
        const long gm = (c_out - p * g_m < g_m) ? c_out - p * g_m : g_m;
        for (long q = 0; q < q_groups; ++q) {
            const long gn = (c_in - q * g_n < g_n) ? c_in - q * g_n : g_n;
            const long g = p * q_groups + q;
            const uint8_t *row = mask + g * ks;
            long k = 0;
            for (long s = 0; s < ks; ++s) {
                if (row[s] > 1) return ORACLE_BAD_ARG;
                k += row[s];
            }
            if (writing) {
                group_ptr[g] = (uint32_t)npos;
                val_ptr[g] = nval;
                long r = 0;
                for (long s = 0; s < ks; ++s)
                    if (row[s]) pos[npos + r++] = (uint16_t)s;
                for (long i = 0; i < gm; ++i)
                    for (long j = 0; j < gn; ++j)
                        for (r = 0; r < k; ++r) {
                            const long m = p * g_m + i, c = q * g_n + j;
                            const long s = pos[npos + r];
                            const char *src = (const char *)w + ((m * c_in + c) * ks + s) * esize;
                            char *dst = (char *)vals + (nval + (i * gn + j) * k + r) * esize;
                            memcpy(dst, src, (size_t)esize);
                        }
            }
            npos += (uint64_t)k;
            nval += (uint64_t)(gm * gn * k);
        }
    }
    if (writing) {
        group_ptr[p_groups * q_groups] = (uint32_t)npos;
        val_ptr[p_groups * q_groups] = nval;
    }
    if (total_pos) *total_pos = npos;
    if (total_vals) *total_vals = nval;
    return ORACLE_OK;
}

/* 3-D max pooling (the pooling layers between the convolutions): window
 * kt x kh x kw, strides st, sh, sw, padding pt, ph, pw on each side; padded
 * positions take no part in the max (every window must hold an input voxel:
 * padding at most half the window), floor output size.
 * x [n][c][t][h][w] -> y [n][c][to][ho][wo]. */
int oracle_maxpool3d(int n, int c, int t, int h, int w, int kt, int kh, int kw,
                     int st, int sh, int sw, int pt, int ph, int pw, const double *x, double *y)
{
    if (n < 0 || c <= 0 || t <= 0 || h <= 0 || w <= 0 || kt <= 0 || kh <= 0 || kw <= 0 ||
        st <= 0 || sh <= 0 || sw <= 0) return ORACLE_BAD_ARG;
    if (pt < 0 || ph < 0 || pw < 0 || 2 * pt > kt || 2 * ph > kh || 2 * pw > kw) return ORACLE_BAD_ARG;
    if (!x || !y) return ORACLE_BAD_ARG;
    const long to = out_len(t, kt, st, pt), ho = out_len(h, kh, sh, ph), wo = out_len(w, kw, sw, pw);
    if (to <= 0 || ho <= 0 || wo <= 0) return ORACLE_BAD_ARG;
    long bc;
#pragma omp parallel for
    for (bc = 0; bc < (long)n * c; ++bc) {
        const double *xs = x + bc * (long)t * h * w;
        double *ys = y + bc * to * ho * wo;
        for (long ot = 0; ot < to; ++ot)
        for (long oh = 0; oh < ho; ++oh)
        for (long ow = 0; ow < wo; ++ow) {
            int seen = 0;
            double best = 0.0;
            for (long it = 0; it < kt; ++it)
            for (long ih = 0; ih < kh; ++ih)
            for (long iw = 0; iw < kw; ++iw) {
                const long zt = ot * st - pt + it, zh = oh * sh - ph + ih, zw = ow * sw - pw + iw;
                if (zt < 0 || zt >= t || zh < 0 || zh >= h || zw < 0 || zw >= w) continue;
                const double v = xs[(zt * h + zh) * w + zw];
                if (!seen || v > best) best = v;
                seen = 1;
            }
            ys[(ot * ho + oh) * wo + ow] = best;
        }
    }
    return ORACLE_OK;
}

/*
 * Group norms and the reweighted group-lasso penalty (Section 4).
 *
 * Weights w [c_out][c_in][ks] (ks = kt*kh*kw kernel positions), kernel
 * groups of g_m x g_n kernels, P = ceil(c_out/g_m) by Q = ceil(c_in/g_n)
 * (trailing groups partial).  A "unit" u is what one norm covers:
 *   scope 0 (KGS):     one kernel position of one group, u = (p*Q + q)*ks + pos
 *                      (the norm in the caption of Fig. 2 / eq. (2));
 *   scope 1 (vanilla): a whole group, u = p*Q + q (the group norm of eq. (1)).
 * norm = 1 or 2 selects the l1 or l2 norm of the unit's weights:
 *   n_u = (sum over the unit of |w|^norm)^(1/norm).
 * With P_u the current penalty factors (pen; NULL means all ones) the call
 * evaluates
 *   reg        = lambda * sum_u P_u * n_u        (penalty term of eq. (3))
 *   pen_next_u = 1 / (n_u^2 + eps)               (reweighting update, Section 4)
 *   mask       = n_u > tau for every kernel position of the unit (pruning the
 *                units whose norm has converged to zero), layout [P][Q][ks]
 *   grad      += lambda * P_u * d n_u / d w      (the penalty's contribution to
 *                the weight gradient: w / n_u for l2, 0 when n_u = 0; sign(w)
 *                for l1, 0 at w = 0)
 *   w_prox     = argmin_z 1/2 |z - w|^2 + step * lambda * sum_u P_u * n_u(z):
 *                l2: w * max(0, 1 - theta / n_u), 0 when n_u = 0;
 *                l1: the unit's norm is a sum of |w|, so the map is the
 *                elementwise sign(w) * max(0, |w| - theta);
 *                theta = step * lambda * P_u.
 * Any output may be NULL.  norms and pen_next have one entry per unit.
 * Sums run in a fixed order (filters, then channels, then positions), float64.
 */
static double unit_weight_sum(const double *w, long c_in, long ks, long m0, long m1,
                              long c0, long c1, long s0, long s1, int norm)
{
    double acc = 0.0;
    for (long m = m0; m < m1; ++m)
        for (long c = c0; c < c1; ++c)
            for (long s = s0; s < s1; ++s) {
                const double v = w[(m * c_in + c) * ks + s];
                acc += norm == 2 ? v * v : fabs(v);
            }
    return acc;
}

int oracle_group_reweight(int c_out, int c_in, int ks, int g_m, int g_n, int norm, int scope,
                          const double *w, const double *pen, double lambda, double eps,
                          double tau, double step, double *norms, double *pen_next,
                          double *reg, unsigned char *mask, double *grad, double *w_prox)
{
    if (c_out <= 0 || c_in <= 0 || ks <= 0 || g_m <= 0 || g_n <= 0) return ORACLE_BAD_ARG;
    if ((norm != 1 && norm != 2) || (scope != 0 && scope != 1) || !w) return ORACLE_BAD_ARG;
    if (!(eps > 0.0)) return ORACLE_BAD_ARG;
    const long P = (c_out + g_m - 1) / g_m, Q = (c_in + g_n - 1) / g_n;
    const long per_group = scope == 0 ? ks : 1;
    double total = 0.0;
    for (long p = 0; p < P; ++p)
    for (long q = 0; q < Q; ++q)
    for (long r = 0; r < per_group; ++r) {
        const long m0 = p * g_m, m1 = m0 + g_m < c_out ? m0 + g_m : c_out;
        const long c0 = q * g_n, c1 = c0 + g_n < c_in ? c0 + g_n : c_in;
        const long s0 = scope == 0 ? r : 0, s1 = scope == 0 ? r + 1 : ks;
        const long u = (p * Q + q) * per_group + r;
        const double sum = unit_weight_sum(w, c_in, ks, m0, m1, c0, c1, s0, s1, norm);
        const double n = norm == 2 ? sqrt(sum) : sum;
        const double pu = pen ? pen[u] : 1.0;
        total += pu * n;
        if (norms) norms[u] = n;
        if (pen_next) pen_next[u] = 1.0 / (n * n + eps);
        if (mask)
            for (long s = s0; s < s1; ++s) mask[(p * Q + q) * ks + s] = n > tau ? 1 : 0;
        const double theta = step * lambda * pu;
        for (long m = m0; m < m1; ++m)
        for (long c = c0; c < c1; ++c)
        for (long s = s0; s < s1; ++s) {
            const long e = (m * c_in + c) * ks + s;
            const double v = w[e];
            const double sgn = v > 0.0 ? 1.0 : (v < 0.0 ? -1.0 : 0.0);
            if (grad) {
                if (norm == 2) grad[e] += n > 0.0 ? lambda * pu * v / n : 0.0;
                else grad[e] += lambda * pu * sgn;
            }
            if (w_prox) {
                if (norm == 2) {
                    const double f = n > 0.0 ? 1.0 - theta / n : 0.0;
                    w_prox[e] = f > 0.0 ? v * f : 0.0;
                } else {
                    const double a = fabs(v) - theta;
                    w_prox[e] = a > 0.0 ? sgn * a : 0.0;
                }
            }
        }
    }
    if (reg) *reg = lambda * total;
    return ORACLE_OK;
}

/* Number of threads the OpenMP loops above use (reported with timings). */
#ifdef _OPENMP
#include <omp.h>
#endif
int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Thread count for the loops above (timing runs on one core); n < 1 is ignored. */
void oracle_set_threads(int n)
{
#ifdef _OPENMP
    if (n >= 1) omp_set_num_threads(n);
#else
    (void)n;
#endif
}
