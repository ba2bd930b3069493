/*
 * CPU oracle for the prefix-masked MoE layer forward of FlexMoE.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the checker: the parity tests, the
 * smoke check and the CPU-baseline leg of the benchmark call it; the product
 * library never links it, includes it or calls it.  It shares no code with the
 * GPU path.  Everything is plain, slow and written to be checked by eye
 * against the paper: fp64 accumulation, one loop per sum, no blocking.
 *
 * What is computed (paper, Sec. 3 and App. C):
 *   - the expert FFN  FFN(h) = W_down (phi(W_gate h) * W_up h), phi = SiLU (Eq. 1);
 *   - the prefix-sliced expert of Eq. 4: only the first k_e ranked channels
 *     take part, channels c >= k_e are never touched;
 *   - the routed layer in the per-expert loop form of the naive online
 *     clipped FFN (App. C.1, Algorithm 1): for each active expert gather its
 *     tokens, run the sliced FFN, weight by the router score and add into Y;
 *   - the channel reorder of Eq. 3 (Sec. 3.1): a descending sort of the
 *     saliency scores gives pi; gate/up rows and down columns are permuted
 *     consistently;
 *   - k = ceil(r * d_ff) for a retention ratio r (Sec. 3.1, after Eq. 3);
 *   - the first-order Taylor channel saliency of Eq. 2 (Sec. 3.1): the
 *     gradient of a loss with respect to every routed expert weight, then
 *     per hidden channel j the sum over its group (gate row j, up row j,
 *     down column j) of (theta * dL/dtheta)^2.  The paper's loss is the
 *     language-model loss; here it is the layer-level
 *     L = 1/2 sum_t ||y_t - y_target_t||^2, with the gradients written out
 *     by the chain rule (router weights and logits are inputs, not trained);
 *   - action learning (Sec. 3.2, Eqs. 5-8): the straight-through Gumbel-softmax
 *     sample of one discrete width per expert, the backward of the masked
 *     layer (input, router-logit and mask gradients), and the gradient of the
 *     action logits through the straight-through estimator plus the
 *     load-weighted cost and the entropy regulariser.
 *
 * Readings where the paper is silent (each listed with its reason in the
 * design notes):
 *   - router: softmax over all E fp32 logits, top-k selected on the raw
 *     logits ordered by (logit descending, expert id ascending); NaN logits
 *     order after every number; with norm_topk the k selected probabilities
 *     are divided by their sum;
 *   - dispatch order inside one expert: ascending assignment id a = t*k + j;
 *   - k_e = 0: the expert keeps its routing slot and weight, contributes
 *     exactly 0 and is left out of the permutation;
 *   - the router weight multiplies the expert output after the down
 *     projection (Algorithm 1 and Algorithm 2 both do this);
 *   - one optional shared expert, unpruned, added with weight 1;
 *   - reorder ties keep the lower original channel index first; NaN scores
 *     order after every number.
 *
 * Layouts (row-major):  x [T][d]; logits [T][E] fp32;
 *   w_gate, w_up [E][I][d];  w_down [E][d][I]  (row = hidden unit, column =
 *   channel);  shared ws_gate, ws_up [I_s][d], ws_down [d][I_s].
 * Element type of x and weights: dtype 0 = fp32, 1 = bf16 (raw bits).
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_F32 0
#define ORACLE_BF16 1

/* Accumulator of the forward's dot products.  The parity build accumulates
 * in fp64 (acc_t = double); defining ORACLE_ACC_F32 builds the same source
 * with fp32 accumulators, a build used only to time the CPU baseline.  Its
 * outputs are never compared with anything. */
#ifdef ORACLE_ACC_F32
typedef float acc_t;
#else
typedef double acc_t;
#endif

/* Exact decode of one stored element to double (bf16 -> fp32 is a shift). */
static double elem(const void *base, int dtype, size_t i)
{
    if (dtype == ORACLE_F32)
        return (double)((const float *)base)[i];
    uint32_t bits = ((uint32_t)((const uint16_t *)base)[i]) << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

static void store(void *base, int dtype, size_t i, const void *src, size_t j)
{
    if (dtype == ORACLE_F32)
        ((float *)base)[i] = ((const float *)src)[j];
    else
        ((uint16_t *)base)[i] = ((const uint16_t *)src)[j];
}

/* Routing order: does (va, ia) come before (vb, ib)?  Larger logit first,
 * equal logits -> lower expert id first, NaN after every number. */
static int route_before(float va, int ia, float vb, int ib)
{
    int na = isnan(va), nb = isnan(vb);
    if (na != nb)
        return nb;
    if (!na && va != vb)
        return va > vb;
    return ia < ib;
}

/* Per token: top-k experts by logit and their router weights.
 * idx [T][k], w [T][k] (fp64). */
int oracle_route(int T, int E, int k, const float *logits, int norm_topk,
                 int32_t *idx, double *w)
{
    if (T < 0 || E < 1 || k < 1 || k > E || !logits || !idx || !w)
        return -1;
    char *taken = (char *)malloc((size_t)E);
    if (!taken)
        return -1;
    for (int t = 0; t < T; ++t) {
        const float *l = logits + (size_t)t * E;
        memset(taken, 0, (size_t)E);
        /* selection: k rounds, each picks the first not-yet-taken expert in
         * routing order */
        for (int j = 0; j < k; ++j) {
            int best = -1;
            for (int e = 0; e < E; ++e) {
                if (taken[e])
                    continue;
                if (best < 0 || route_before(l[e], e, l[best], best))
                    best = e;
            }
            taken[best] = 1;
            idx[(size_t)t * k + j] = best;
        }
        /* softmax over all E experts, shifted by the largest logit */
        double m = -INFINITY;
        for (int e = 0; e < E; ++e)
            if ((double)l[e] > m)
                m = (double)l[e];
        double z = 0.0;
        for (int e = 0; e < E; ++e)
            z += exp((double)l[e] - m);
        double s = 0.0;
        for (int j = 0; j < k; ++j) {
            int e = idx[(size_t)t * k + j];
            w[(size_t)t * k + j] = exp((double)l[e] - m) / z;
            s += w[(size_t)t * k + j];
        }
        if (norm_topk)
            for (int j = 0; j < k; ++j)
                w[(size_t)t * k + j] /= s;
    }
    free(taken);
    return 0;
}

/* Stable counting sort of the T*k assignments by expert id, active experts
 * only (k_e > 0).  counts [E] = raw n_e of every expert; offsets [E+1] over
 * active experts; perm [P] = assignment ids; pos [T*k] = slot in perm or -1.
 * Returns P (number of active assignments) or -1. */
int oracle_dispatch(int T, int E, int k, const int32_t *idx, const int32_t *keep,
                    int32_t *counts, int32_t *offsets, int32_t *perm, int32_t *pos)
{
    if (T < 0 || E < 1 || k < 1 || !idx || !keep || !counts || !offsets)
        return -1;
    size_t A = (size_t)T * k;
    for (int e = 0; e < E; ++e)
        counts[e] = 0;
    for (size_t a = 0; a < A; ++a) {
        if (idx[a] < 0 || idx[a] >= E)
            return -1;
        counts[idx[a]]++;
    }
    offsets[0] = 0;
    for (int e = 0; e < E; ++e)
        offsets[e + 1] = offsets[e] + (keep[e] > 0 ? counts[e] : 0);
    int32_t *fill = (int32_t *)calloc((size_t)E, sizeof(int32_t));
    if (!fill)
        return -1;
    for (size_t a = 0; a < A; ++a) {
        int e = idx[a];
        if (keep[e] > 0) {
            int32_t p = offsets[e] + fill[e]++;
            if (perm)
                perm[p] = (int32_t)a;
            if (pos)
                pos[a] = p;
        } else if (pos) {
            pos[a] = -1;
        }
    }
    free(fill);
    return offsets[E];
}

/* One prefix-sliced SwiGLU expert applied to one token (Eq. 4):
 *   g_c = <W_gate[c], x>, u_c = <W_up[c], x>, h_c = silu(g_c) * u_c  (c < kk)
 *   out[n] = sum_{c < kk} h_c * W_down[n][c]
 * wg/wu point at the expert's [I][d] blocks, wd at its [d][ld_down] block. */
static void sliced_ffn(int d, int kk, int ld_down, int dtype, const void *x, size_t x_off,
                       const void *wg, const void *wu, const void *wd, size_t w_off,
                       size_t wd_off, double *h, double *out)
{
    for (int c = 0; c < kk; ++c) {
        acc_t g = 0, u = 0;
        for (int i = 0; i < d; ++i) {
            acc_t xi = (acc_t)elem(x, dtype, x_off + i);
            g += (acc_t)elem(wg, dtype, w_off + (size_t)c * d + i) * xi;
            u += (acc_t)elem(wu, dtype, w_off + (size_t)c * d + i) * xi;
        }
        h[c] = g / (1.0 + exp(-(double)g)) * u;
    }
    for (int n = 0; n < d; ++n) {
        acc_t acc = 0;
        for (int c = 0; c < kk; ++c)
            acc += (acc_t)h[c] * (acc_t)elem(wd, dtype, wd_off + (size_t)n * ld_down + c);
        out[n] = acc;
    }
}

/* Masked MoE layer forward.  y [T][d] fp64, unrounded.  The routing and
 * dispatch results are returned through the optional pointers (NULL = skip):
 * idx/w [T][k], counts [E], offsets [E+1], perm [T*k], pos [T*k].
 * Returns 0, or -1 on bad arguments, -3 on a keep count outside [0, I]. */
int oracle_layer_forward(int T, int d, int E, int I, int k, int I_s, int dtype,
                         int norm_topk, const void *x, const float *logits,
                         const void *w_gate, const void *w_up, const void *w_down,
                         const int32_t *keep, const void *ws_gate, const void *ws_up,
                         const void *ws_down, double *y, int32_t *idx_out, double *w_out,
                         int32_t *counts_out, int32_t *offsets_out, int32_t *perm_out,
                         int32_t *pos_out)
{
    if (T < 0 || d < 1 || E < 1 || I < 1 || k < 1 || k > E || I_s < 0 || !y || !keep)
        return -1;
    if (dtype != ORACLE_F32 && dtype != ORACLE_BF16)
        return -1;
    for (int e = 0; e < E; ++e)
        if (keep[e] < 0 || keep[e] > I)
            return -3;
    if (T == 0)
        return 0;
    size_t A = (size_t)T * k;
    int32_t *idx = (int32_t *)malloc(A * sizeof(int32_t));
    double *w = (double *)malloc(A * sizeof(double));
    int32_t *counts = (int32_t *)malloc((size_t)E * sizeof(int32_t));
    int32_t *offsets = (int32_t *)malloc((size_t)(E + 1) * sizeof(int32_t));
    int32_t *perm = (int32_t *)malloc(A * sizeof(int32_t));
    int32_t *pos = (int32_t *)malloc(A * sizeof(int32_t));
    double *O = (double *)malloc(A * (size_t)d * sizeof(double));
    int rc = -1;
    if (!idx || !w || !counts || !offsets || !perm || !pos || !O)
        goto done;

    /* step 1: routing (the router is an input of Algorithm 1) */
    if (oracle_route(T, E, k, logits, norm_topk, idx, w) != 0)
        goto done;
    /* step 2: group the routed assignments by expert, skipping k_e = 0 */
    int P = oracle_dispatch(T, E, k, idx, keep, counts, offsets, perm, pos);
    if (P < 0)
        goto done;

    /* step 3: for each active expert, its sliced FFN on each routed token */
    for (int e = 0; e < E; ++e) {
        int kk = keep[e];
        if (kk == 0)
            continue;
#pragma omp parallel for schedule(dynamic, 1)
        for (int p = offsets[e]; p < offsets[e + 1]; ++p) {
            double *h = (double *)malloc((size_t)kk * sizeof(double));
            int t = perm[p] / k;
            sliced_ffn(d, kk, I, dtype, x, (size_t)t * d, w_gate, w_up, w_down,
                       (size_t)e * I * d, (size_t)e * d * I, h, O + (size_t)p * d);
            free(h);
        }
    }

    /* step 4: weight by router score after the down projection and add into
     * Y in ascending slot order; then the shared expert with weight 1 */
#pragma omp parallel for schedule(static)
    for (int t = 0; t < T; ++t) {
        double *yt = y + (size_t)t * d;
        for (int n = 0; n < d; ++n)
            yt[n] = 0.0;
        for (int j = 0; j < k; ++j) {
            int32_t p = pos[(size_t)t * k + j];
            if (p < 0)
                continue;
            double wt = w[(size_t)t * k + j];
            for (int n = 0; n < d; ++n)
                yt[n] += wt * O[(size_t)p * d + n];
        }
        if (I_s > 0) {
            double *h = (double *)malloc((size_t)I_s * sizeof(double));
            double *s = (double *)malloc((size_t)d * sizeof(double));
            sliced_ffn(d, I_s, I_s, dtype, x, (size_t)t * d, ws_gate, ws_up, ws_down, 0, 0, h, s);
            for (int n = 0; n < d; ++n)
                yt[n] += s[n];
            free(h);
            free(s);
        }
    }

    if (idx_out)
        memcpy(idx_out, idx, A * sizeof(int32_t));
    if (w_out)
        memcpy(w_out, w, A * sizeof(double));
    if (counts_out)
        memcpy(counts_out, counts, (size_t)E * sizeof(int32_t));
    if (offsets_out)
        memcpy(offsets_out, offsets, (size_t)(E + 1) * sizeof(int32_t));
    if (perm_out)
        memcpy(perm_out, perm, (size_t)P * sizeof(int32_t));
    if (pos_out)
        memcpy(pos_out, pos, A * sizeof(int32_t));
    rc = 0;
done:
    free(idx);
    free(w);
    free(counts);
    free(offsets);
    free(perm);
    free(pos);
    free(O);
    return rc;
}

/* Gradients of L = 1/2 sum_t sum_n (y[t][n] - y_target[t][n])^2 for the
 * masked layer above, with respect to the routed experts' weights (Sec. 3.1,
 * the g of Eq. 2).  With dY_t = y_t - y_target_t, for every active
 * assignment a = (t, j) of expert e with router weight w_a and every kept
 * channel c < k_e:
 *   g_c = <W_gate[c], x_t>, u_c = <W_up[c], x_t>, h_c = silu(g_c) u_c
 *   dO_a[n]  = w_a dY_t[n]                      (y_t = sum_a w_a O_a + S_t)
 *   dL/dW_down[n][c] += dO_a[n] h_c             (O_a[n] = sum_c W_down[n][c] h_c)
 *   dh_c     = sum_n W_down[n][c] dO_a[n]
 *   dg_c     = dh_c u_c silu'(g_c),  du_c = dh_c silu(g_c)
 *   dL/dW_gate[c][i] += dg_c x_t[i],  dL/dW_up[c][i] += du_c x_t[i]
 * with silu'(g) = s (1 + g (1 - s)), s = 1 / (1 + e^-g).  Channels c >= k_e
 * and experts with k_e = 0 take no part in the layer and get zero gradient.
 * The shared expert enters through y only.
 * g_gate, g_up [E][I][d], g_down [E][d][I] (fp64, overwritten); *loss = L.
 * Returns 0, or the error of oracle_layer_forward. */
int oracle_layer_grads(int T, int d, int E, int I, int k, int I_s, int dtype, int norm_topk,
                       const void *x, const float *logits, const void *w_gate, const void *w_up,
                       const void *w_down, const int32_t *keep, const void *ws_gate,
                       const void *ws_up, const void *ws_down, const float *y_target,
                       double *loss, double *g_gate, double *g_up, double *g_down)
{
    if (T < 0 || d < 1 || E < 1 || I < 1 || k < 1 || k > E || !y_target || !loss || !g_gate ||
        !g_up || !g_down)
        return -1;
    size_t nw = (size_t)E * I * d;
    memset(g_gate, 0, nw * sizeof(double));
    memset(g_up, 0, nw * sizeof(double));
    memset(g_down, 0, nw * sizeof(double));
    *loss = 0.0;
    if (T == 0)
        return 0;
    size_t A = (size_t)T * k;
    double *y = (double *)malloc((size_t)T * d * sizeof(double));
    double *w = (double *)malloc(A * sizeof(double));
    int32_t *idx = (int32_t *)malloc(A * sizeof(int32_t));
    int32_t *counts = (int32_t *)malloc((size_t)E * sizeof(int32_t));
    int32_t *offsets = (int32_t *)malloc((size_t)(E + 1) * sizeof(int32_t));
    int32_t *perm = (int32_t *)malloc(A * sizeof(int32_t));
    int32_t *pos = (int32_t *)malloc(A * sizeof(int32_t));
    int rc = -1;
    if (!y || !w || !idx || !counts || !offsets || !perm || !pos)
        goto done;
    rc = oracle_layer_forward(T, d, E, I, k, I_s, dtype, norm_topk, x, logits, w_gate, w_up,
                              w_down, keep, ws_gate, ws_up, ws_down, y, idx, w, counts, offsets,
                              perm, pos);
    if (rc != 0)
        goto done;

    /* dY = y - y_target (overwrites y) and the loss */
    double L = 0.0;
    for (size_t i = 0; i < (size_t)T * d; ++i) {
        y[i] -= (double)y_target[i];
        L += 0.5 * y[i] * y[i];
    }
    *loss = L;

    /* experts are independent: one thread per expert, its assignments in
     * dispatch order */
#pragma omp parallel for schedule(dynamic, 1)
    for (int e = 0; e < E; ++e) {
        int kk = keep[e];
        if (kk == 0 || offsets[e + 1] == offsets[e])
            continue;
        double *g = (double *)malloc((size_t)kk * sizeof(double));
        double *u = (double *)malloc((size_t)kk * sizeof(double));
        double *dO = (double *)malloc((size_t)d * sizeof(double));
        const size_t wb = (size_t)e * I * d; /* gate/up block [I][d], down block [d][I] */
        for (int p = offsets[e]; p < offsets[e + 1]; ++p) {
            int a = perm[p], t = a / k;
            const size_t xo = (size_t)t * d;
            for (int c = 0; c < kk; ++c) {
                double gc = 0.0, uc = 0.0;
                for (int i = 0; i < d; ++i) {
                    double xi = elem(x, dtype, xo + i);
                    gc += elem(w_gate, dtype, wb + (size_t)c * d + i) * xi;
                    uc += elem(w_up, dtype, wb + (size_t)c * d + i) * xi;
                }
                g[c] = gc;
                u[c] = uc;
            }
            for (int n = 0; n < d; ++n)
                dO[n] = w[a] * y[xo + n];
            for (int c = 0; c < kk; ++c) {
                double sg = 1.0 / (1.0 + exp(-g[c]));
                double silu = g[c] * sg, dsilu = sg * (1.0 + g[c] * (1.0 - sg));
                double h = silu * u[c], dh = 0.0;
                for (int n = 0; n < d; ++n) {
                    g_down[wb + (size_t)n * I + c] += dO[n] * h;
                    dh += elem(w_down, dtype, wb + (size_t)n * I + c) * dO[n];
                }
                double dg = dh * u[c] * dsilu, du = dh * silu;
                for (int i = 0; i < d; ++i) {
                    double xi = elem(x, dtype, xo + i);
                    g_gate[wb + (size_t)c * d + i] += dg * xi;
                    g_up[wb + (size_t)c * d + i] += du * xi;
                }
            }
        }
        free(g);
        free(u);
        free(dO);
    }
    rc = 0;
done:
    free(y);
    free(w);
    free(idx);
    free(counts);
    free(offsets);
    free(perm);
    free(pos);
    return rc;
}

/* Eq. 2 for one batch: the saliency of hidden channel j of expert e is the
 * sum over its parameter group -- gate row j, up row j, down column j -- of
 * (theta * dL/dtheta)^2 (a sum of squares, not the square of a sum).
 * s [E][I] fp64 (overwritten). */
int oracle_channel_saliency(int d, int E, int I, int dtype, const void *w_gate, const void *w_up,
                            const void *w_down, const double *g_gate, const double *g_up,
                            const double *g_down, double *s)
{
    if (d < 1 || E < 1 || I < 1 || !w_gate || !w_up || !w_down || !g_gate || !g_up || !g_down || !s)
        return -1;
#pragma omp parallel for schedule(static)
    for (int e = 0; e < E; ++e) {
        const size_t wb = (size_t)e * I * d;
        for (int j = 0; j < I; ++j) {
            double acc = 0.0;
            for (int i = 0; i < d; ++i) {
                double tg = elem(w_gate, dtype, wb + (size_t)j * d + i) * g_gate[wb + (size_t)j * d + i];
                double tu = elem(w_up, dtype, wb + (size_t)j * d + i) * g_up[wb + (size_t)j * d + i];
                acc += tg * tg + tu * tu;
            }
            for (int n = 0; n < d; ++n) {
                double td = elem(w_down, dtype, wb + (size_t)n * I + j) * g_down[wb + (size_t)n * I + j];
                acc += td * td;
            }
            s[(size_t)e * I + j] = acc;
        }
    }
    return 0;
}

/* Eq. 5: per expert, z_soft = softmax((alpha + g) / tau) over the K actions
 * and the hard action k* = argmax; the sampled width is ceil(r_k* * I).  The
 * argmax is taken on the fp32 sums alpha + g (the softmax is monotone in
 * them), the first index on ties.  alpha, gumbel [E][K] fp32; ratio [K];
 * keep [E], action [E] (int32), z_soft [E][K] fp64 (any may be NULL). */
int oracle_keep_from_ratio(double r, int I);
int oracle_sample_actions(int E, int K, const double *ratio, int I, const float *alpha,
                          const float *gumbel, double tau, int32_t *keep, double *z_soft,
                          int32_t *action)
{
    if (E < 1 || K < 1 || I < 1 || !ratio || !alpha || !gumbel || !(tau > 0.0))
        return -1;
    for (int e = 0; e < E; ++e) {
        const float *a = alpha + (size_t)e * K, *g = gumbel + (size_t)e * K;
        int best = 0;
        for (int k = 1; k < K; ++k)
            if (a[k] + g[k] > a[best] + g[best])
                best = k;
        double m = -INFINITY, z = 0.0;
        for (int k = 0; k < K; ++k)
            if (((double)a[k] + g[k]) / tau > m)
                m = ((double)a[k] + g[k]) / tau;
        for (int k = 0; k < K; ++k)
            z += exp(((double)a[k] + g[k]) / tau - m);
        if (z_soft)
            for (int k = 0; k < K; ++k)
                z_soft[(size_t)e * K + k] = exp(((double)a[k] + g[k]) / tau - m) / z;
        if (action)
            action[e] = best;
        if (keep)
            keep[e] = oracle_keep_from_ratio(ratio[best], I);
    }
    return 0;
}

/* Backward of the masked layer for an upstream gradient dY [T][d] (Sec. 3.2:
 * the sampled subnet's forward is the masked layer, h_c = M_c a_c with
 * a_c = silu(g_c) u_c and the prefix mask M_c = [c < k_e]).  With
 * dO_a = w_a dY_t and dh'_c = sum_n W_down[n][c] dO_a[n] for every channel:
 *   dM[e][c]    = sum over e's assignments of dh'_c a_c   (all c < I)
 *   dg_c, du_c  = M_c dh'_c u_c silu'(g_c),  M_c dh'_c silu(g_c)
 *   dx_t       += sum_c dg_c W_gate[c] + du_c W_up[c]  (+ the shared expert's
 *                 terms, with dO = dY_t and no mask)
 *   dw_a        = <dY_t, O_a>, then through the router weights of
 *                 oracle_route to the logits: with p = softmax(logits),
 *                 w_j = p_{i_j} (/ sum_j p_{i_j} if norm_topk).
 * Experts with k_e = 0 are skipped, as in the forward.  Outputs (fp64,
 * overwritten): dx [T][d], dlogits [T][E], dmask [E][I]. */
int oracle_masked_backward(int T, int d, int E, int I, int k, int I_s, int dtype, int norm_topk,
                           const void *x, const float *logits, const void *w_gate,
                           const void *w_up, const void *w_down, const int32_t *keep,
                           const void *ws_gate, const void *ws_up, const void *ws_down,
                           const float *dy, double *dx, double *dlogits, double *dmask)
{
    if (T < 0 || d < 1 || E < 1 || I < 1 || k < 1 || k > E || I_s < 0 || !keep || !dy || !dx ||
        !dlogits || !dmask)
        return -1;
    for (int e = 0; e < E; ++e)
        if (keep[e] < 0 || keep[e] > I)
            return -3;
    memset(dx, 0, (size_t)T * d * sizeof(double));
    memset(dlogits, 0, (size_t)T * E * sizeof(double));
    memset(dmask, 0, (size_t)E * I * sizeof(double));
    if (T == 0)
        return 0;
    size_t A = (size_t)T * k;
    int32_t *idx = (int32_t *)malloc(A * sizeof(int32_t));
    double *w = (double *)malloc(A * sizeof(double));
    int32_t *counts = (int32_t *)malloc((size_t)E * sizeof(int32_t));
    int32_t *offsets = (int32_t *)malloc((size_t)(E + 1) * sizeof(int32_t));
    int32_t *perm = (int32_t *)malloc(A * sizeof(int32_t));
    int32_t *pos = (int32_t *)malloc(A * sizeof(int32_t));
    double *dw = (double *)calloc(A, sizeof(double));
    double *dxa = (double *)calloc(A * (size_t)d, sizeof(double)); /* per-assignment dx */
    int rc = -1;
    if (!idx || !w || !counts || !offsets || !perm || !pos || !dw || !dxa)
        goto done;
    if (oracle_route(T, E, k, logits, norm_topk, idx, w) != 0)
        goto done;
    if (oracle_dispatch(T, E, k, idx, keep, counts, offsets, perm, pos) < 0)
        goto done;

#pragma omp parallel for schedule(dynamic, 1)
    for (int e = 0; e < E; ++e) {
        int kk = keep[e];
        if (kk == 0)
            continue;
        double *g = (double *)malloc((size_t)I * sizeof(double));
        double *u = (double *)malloc((size_t)I * sizeof(double));
        double *h = (double *)malloc((size_t)I * sizeof(double));
        const size_t wb = (size_t)e * I * d;
        for (int p = offsets[e]; p < offsets[e + 1]; ++p) {
            int a = perm[p], t = a / k;
            const size_t xo = (size_t)t * d;
            for (int c = 0; c < I; ++c) {
                double gc = 0.0, uc = 0.0;
                for (int i = 0; i < d; ++i) {
                    double xi = elem(x, dtype, xo + i);
                    gc += elem(w_gate, dtype, wb + (size_t)c * d + i) * xi;
                    uc += elem(w_up, dtype, wb + (size_t)c * d + i) * xi;
                }
                g[c] = gc;
                u[c] = uc;
            }
            /* dw_a = <dY_t, O_a>, O_a over the kept channels */
            for (int c = 0; c < kk; ++c)
                h[c] = g[c] / (1.0 + exp(-g[c])) * u[c];
            double dwa = 0.0;
            for (int n = 0; n < d; ++n) {
                double o = 0.0;
                for (int c = 0; c < kk; ++c)
                    o += h[c] * elem(w_down, dtype, wb + (size_t)n * I + c);
                dwa += (double)dy[xo + n] * o;
            }
            dw[a] = dwa;
            for (int c = 0; c < I; ++c) {
                double sg = 1.0 / (1.0 + exp(-g[c]));
                double silu = g[c] * sg, dsilu = sg * (1.0 + g[c] * (1.0 - sg));
                double dh = 0.0;
                for (int n = 0; n < d; ++n)
                    dh += elem(w_down, dtype, wb + (size_t)n * I + c) * w[a] * (double)dy[xo + n];
                dmask[(size_t)e * I + c] += dh * silu * u[c];
                if (c >= kk)
                    continue;
                double dg = dh * u[c] * dsilu, du = dh * silu;
                for (int i = 0; i < d; ++i)
                    dxa[(size_t)a * d + i] += dg * elem(w_gate, dtype, wb + (size_t)c * d + i) +
                                              du * elem(w_up, dtype, wb + (size_t)c * d + i);
            }
        }
        free(g);
        free(u);
        free(h);
    }

#pragma omp parallel for schedule(static)
    for (int t = 0; t < T; ++t) {
        double *dxt = dx + (size_t)t * d;
        for (int j = 0; j < k; ++j)
            for (int i = 0; i < d; ++i)
                dxt[i] += dxa[((size_t)t * k + j) * d + i];
        if (I_s > 0) {
            const size_t xo = (size_t)t * d;
            for (int c = 0; c < I_s; ++c) {
                double gc = 0.0, uc = 0.0;
                for (int i = 0; i < d; ++i) {
                    double xi = elem(x, dtype, xo + i);
                    gc += elem(ws_gate, dtype, (size_t)c * d + i) * xi;
                    uc += elem(ws_up, dtype, (size_t)c * d + i) * xi;
                }
                double sg = 1.0 / (1.0 + exp(-gc));
                double dh = 0.0;
                for (int n = 0; n < d; ++n)
                    dh += elem(ws_down, dtype, (size_t)n * I_s + c) * (double)dy[xo + n];
                double dg = dh * uc * sg * (1.0 + gc * (1.0 - sg)), du = dh * gc * sg;
                for (int i = 0; i < d; ++i)
                    dxt[i] += dg * elem(ws_gate, dtype, (size_t)c * d + i) +
                              du * elem(ws_up, dtype, (size_t)c * d + i);
            }
        }
        /* router: softmax over all E, then the optional renormalisation */
        const float *l = logits + (size_t)t * E;
        double m = -INFINITY, z = 0.0;
        for (int e = 0; e < E; ++e)
            if ((double)l[e] > m)
                m = (double)l[e];
        for (int e = 0; e < E; ++e)
            z += exp((double)l[e] - m);
        double S = 0.0;
        for (int j = 0; j < k; ++j)
            S += exp((double)l[idx[(size_t)t * k + j]] - m) / z;
        /* dL/dp_i for the selected experts */
        double dwsum = 0.0;
        for (int j = 0; j < k; ++j)
            dwsum += dw[(size_t)t * k + j] * w[(size_t)t * k + j];
        double dpp = 0.0; /* sum_i dL/dp_i * p_i */
        double *dp = (double *)calloc((size_t)E, sizeof(double));
        for (int j = 0; j < k; ++j) {
            int e = idx[(size_t)t * k + j];
            double g = norm_topk ? (dw[(size_t)t * k + j] - dwsum) / S : dw[(size_t)t * k + j];
            dp[e] = g;
            dpp += g * exp((double)l[e] - m) / z;
        }
        for (int e = 0; e < E; ++e) {
            double pe = exp((double)l[e] - m) / z;
            dlogits[(size_t)t * E + e] = pe * (dp[e] - dpp);
        }
        free(dp);
    }
    rc = 0;
done:
    free(idx);
    free(w);
    free(counts);
    free(offsets);
    free(perm);
    free(pos);
    free(dw);
    free(dxa);
    return rc;
}

/* Gradient of the action logits (Eqs. 5-8) for one layer:
 *   quality term through the straight-through estimator (Eq. 6): the forward
 *     mask is M = sum_k z~_k m(r_k), so dL/dz~_k = sum_{c < K_k} dmask[c]
 *     (K_k = ceil(r_k I)); z~ passes it to z_soft unchanged, and
 *     z_soft = softmax(s), s = (alpha + g) / tau gives
 *     dalpha_k = z_soft_k (dz_k - sum_j z_soft_j dz_j) / tau;
 *   cost (Eq. 7): C = sum_e q_e sum_k p_{e,k} r_k with p_e = softmax(alpha_e)
 *     and q_e = counts_e / (T * top_k), constant in alpha:
 *     dC/dalpha_{e,k} = q_e p_{e,k} (r_k - sum_j p_{e,j} r_j);
 *   entropy (Eq. 8 and the text after it): H = (1/E) sum_e -sum_k p log p,
 *     dH/dalpha_{e,k} = -(1/E) p_{e,k} (log p_{e,k} + H_e);
 *   dalpha = dalpha_quality + lambda_cost dC/dalpha - beta dH/dalpha.
 * dalpha [E][K] fp64; *cost = C, *entropy = H. */
int oracle_action_grad(int E, int K, const double *ratio, int I, const float *alpha,
                       const float *gumbel, double tau, const double *dmask,
                       const int32_t *counts, long long assignments, double lambda_cost,
                       double beta, double *dalpha, double *cost, double *entropy)
{
    if (E < 1 || K < 1 || I < 1 || !ratio || !alpha || !gumbel || !dmask || !counts || !dalpha ||
        !(tau > 0.0) || assignments < 1)
        return -1;
    double *zs = (double *)malloc((size_t)E * K * sizeof(double));
    if (!zs)
        return -1;
    oracle_sample_actions(E, K, ratio, I, alpha, gumbel, tau, NULL, zs, NULL);
    double C = 0.0, H = 0.0;
    for (int e = 0; e < E; ++e) {
        const float *a = alpha + (size_t)e * K;
        const double *z = zs + (size_t)e * K;
        double dz[64], p[64];
        if (K > 64) {
            free(zs);
            return -1;
        }
        for (int kk = 0; kk < K; ++kk) {
            int w = oracle_keep_from_ratio(ratio[kk], I);
            dz[kk] = 0.0;
            for (int c = 0; c < w; ++c)
                dz[kk] += dmask[(size_t)e * I + c];
        }
        double zdz = 0.0;
        for (int kk = 0; kk < K; ++kk)
            zdz += z[kk] * dz[kk];
        double m = -INFINITY, Z = 0.0;
        for (int kk = 0; kk < K; ++kk)
            if ((double)a[kk] > m)
                m = (double)a[kk];
        for (int kk = 0; kk < K; ++kk)
            Z += exp((double)a[kk] - m);
        double rbar = 0.0, He = 0.0;
        for (int kk = 0; kk < K; ++kk) {
            p[kk] = exp((double)a[kk] - m) / Z;
            rbar += p[kk] * ratio[kk];
            He -= p[kk] > 0.0 ? p[kk] * log(p[kk]) : 0.0;
        }
        double q = (double)counts[e] / (double)assignments;
        C += q * rbar;
        H += He / E;
        for (int kk = 0; kk < K; ++kk) {
            double g_quality = z[kk] * (dz[kk] - zdz) / tau;
            double g_cost = q * p[kk] * (ratio[kk] - rbar);
            double g_ent = p[kk] > 0.0 ? -p[kk] * (log(p[kk]) + He) / E : 0.0;
            dalpha[(size_t)e * K + kk] = g_quality + lambda_cost * g_cost - beta * g_ent;
        }
    }
    if (cost)
        *cost = C;
    if (entropy)
        *entropy = H;
    free(zs);
    return 0;
}

/* Eq. 3: sort scores in descending order to get pi, then
 *   W~_gate = P W_gate (rows), W~_up = P W_up (rows), W~_down = W_down P^T
 * (columns).  Ranked channel c holds original channel pi[c]. */
static const float *g_sort_scores;
static int rank_cmp(const void *pa, const void *pb)
{
    int a = *(const int32_t *)pa, b = *(const int32_t *)pb;
    float va = g_sort_scores[a], vb = g_sort_scores[b];
    int na = isnan(va), nb = isnan(vb);
    if (na != nb)
        return na ? 1 : -1;
    if (!na && va != vb)
        return va > vb ? -1 : 1;
    return a < b ? -1 : (a > b);
}

int oracle_rank_reorder(int E, int I, int d, int dtype, const float *scores,
                        const void *w_gate, const void *w_up, const void *w_down,
                        void *w_gate_r, void *w_up_r, void *w_down_r, int32_t *perm_out)
{
    if (E < 1 || I < 1 || d < 1 || !scores || !w_gate || !w_up || !w_down || !w_gate_r ||
        !w_up_r || !w_down_r)
        return -1;
    int32_t *pi = (int32_t *)malloc((size_t)I * sizeof(int32_t));
    if (!pi)
        return -1;
    for (int e = 0; e < E; ++e) {
        for (int c = 0; c < I; ++c)
            pi[c] = c;
        g_sort_scores = scores + (size_t)e * I;
        qsort(pi, (size_t)I, sizeof(int32_t), rank_cmp);
        for (int c = 0; c < I; ++c) {
            size_t src = ((size_t)e * I + pi[c]) * d, dst = ((size_t)e * I + c) * d;
            for (int i = 0; i < d; ++i) {
                store(w_gate_r, dtype, dst + i, w_gate, src + i);
                store(w_up_r, dtype, dst + i, w_up, src + i);
            }
        }
        for (int n = 0; n < d; ++n)
            for (int c = 0; c < I; ++c)
                store(w_down_r, dtype, ((size_t)e * d + n) * I + c, w_down,
                      ((size_t)e * d + n) * I + pi[c]);
        if (perm_out)
            memcpy(perm_out + (size_t)e * I, pi, (size_t)I * sizeof(int32_t));
    }
    free(pi);
    return 0;
}

/* k = ceil(r * d_ff) (Sec. 3.1).  A slack of 1e-9 absorbs the representation
 * error of decimal ratios such as 0.7 in binary floating point.
 * Returns -1 for r outside [0, 1], NaN or I < 1. */
int oracle_keep_from_ratio(double r, int I)
{
    if (!(r >= 0.0 && r <= 1.0) || I < 1)
        return -1;
    double k = ceil(r * (double)I - 1e-9);
    if (k < 0)
        k = 0;
    if (k > I)
        k = I;
    return (int)k;
}

/* Threads the OpenMP loops above run with (reported next to CPU timings). */
int oracle_num_threads(void)
{
    return omp_get_max_threads();
}

/* Sets the threads of the OpenMP loops (CPU-baseline timing at 1 thread and
 * at all cores); returns the new count. */
int oracle_set_threads(int n)
{
    if (n >= 1)
        omp_set_num_threads(n);
    return omp_get_max_threads();
}

/* 1 for the fp32-accumulator timing build, 0 for the fp64 parity build. */
int oracle_acc_f32(void)
{
    return (int)(sizeof(acc_t) == sizeof(float));
}
