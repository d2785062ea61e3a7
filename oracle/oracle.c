/*
 * fp64 CPU oracle for the dReLU feed-forward layer and its Mixture-of-Experts
 * form.  TEST INFRASTRUCTURE ONLY: it exists to check the HIP path, it is
 * called only by the tests, the smoke check and the CPU-baseline leg of the
 * benchmark, and nothing in the product links or loads it.  It shares no code
 * with the HIP library.
 *
 * What it computes (Turbo Sparse, arXiv 2406.05955):
 *   - Eq. (gated-MLP), section 2 "Gated-MLP Blocks": Gate = F_act(x W_gate),
 *     Up = x W_up, Combined = Gate * Up, out = Combined W_down.
 *   - Eq. (drelu), section 3.2: dReLU applies ReLU to both projections,
 *     Combined = max(0, x W_gate) * max(0, x W_up); no bias on either
 *     projection (section 3.2 footnote).
 *   - Section 6.2: a neuron is inactive when its Combined activation is zero;
 *     the MoE layer routes each token to 2 of 8 experts and each routed expert
 *     is itself a dReLU FFN.
 *
 * The method's sparse evaluation reaches exactly the dense result (skipped
 * terms are exact zeros), so this oracle is the plain dense definition.
 * Layout: the paper writes row vectors (x W); here every matrix is stored
 * neuron-major [I][H] and W_down_t[i][:] is the paper's W_down row i.
 * Summation order is fixed: j ascending for the projections, i ascending for
 * the output.  OpenMP splits neurons (projections) and output columns (down),
 * which does not change any sum's order.  Built with -ffp-contract=off so no
 * multiply-add is fused.
 *
 * Routing (the paper states only "2 out of 8 experts", section 6.2; the
 * softmax, top-k and renormalisation form is Mixtral's): logits = W_r x,
 * p = softmax(logits), S = the top_k experts by p (ties: lower index first),
 * w_e = p_e / sum_{e' in S} p_e', out = sum_{e in S, ascending e} w_e FFN_e(x).
 */
#define _GNU_SOURCE
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

enum { OR_F32 = 0, OR_BF16 = 1 };

/* Exact upcast of one stored weight: fp32 as is, bf16 via its fp32 bit pattern. */
static inline double load_w(const void *w, int dtype, size_t k)
{
    if (dtype == OR_F32)
        return (double)((const float *)w)[k];
    uint32_t bits = ((uint32_t)((const uint16_t *)w)[k]) << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

static int set_threads(int nthreads)
{
#ifdef _OPENMP
    if (nthreads <= 0)
        nthreads = omp_get_max_threads();
    return nthreads;
#else
    (void)nthreads;
    return 1;
#endif
}

/*
 * One token through one dReLU FFN.
 *   x [H]; wg, wu, wdt [I][H] in `dtype`; y [H] (written);
 *   g, u [I] (written, the gate and up projections before ReLU);
 *   h [I] scratch (written, the Combined activations).
 */
static void ffn_token(const float *x, const void *wg, const void *wu, const void *wdt, int dtype,
                      int H, int I, double *y, double *g, double *u, double *h, int nthreads)
{
    int i;
#pragma omp parallel for num_threads(nthreads) schedule(static)
    for (i = 0; i < I; ++i) {
        double sg = 0.0, su = 0.0;
        size_t row = (size_t)i * (size_t)H;
        for (int j = 0; j < H; ++j) {
            double xj = (double)x[j];
            sg += load_w(wg, dtype, row + j) * xj;
            su += load_w(wu, dtype, row + j) * xj;
        }
        g[i] = sg;
        u[i] = su;
        /* max(0, g) * max(0, u): zero unless both projections are positive. */
        h[i] = (sg > 0.0 && su > 0.0) ? sg * su : 0.0;
    }

    /* out[j] = sum_i h[i] * W_down_t[i][j], i ascending for every j. */
    int nblk = (H + 63) / 64;
    int b;
#pragma omp parallel for num_threads(nthreads) schedule(static)
    for (b = 0; b < nblk; ++b) {
        int j0 = b * 64, j1 = j0 + 64 < H ? j0 + 64 : H;
        for (int j = j0; j < j1; ++j)
            y[j] = 0.0;
        for (int ii = 0; ii < I; ++ii) {
            double hv = h[ii];
            size_t row = (size_t)ii * (size_t)H;
            for (int j = j0; j < j1; ++j)
                y[j] += load_w(wdt, dtype, row + j) * hv;
        }
    }
}

/*
 * Dense dReLU FFN over a batch of tokens.
 *   x [B][H] fp32; wg, wu, wdt [I][H] (fp32 or bf16 bits); y [B][H] fp64 out.
 *   g_out, u_out [B][I] fp64, nullable: the pre-ReLU gate / up projections.
 * Returns 0, or -1 on bad arguments / allocation failure.
 */
int or_ffn(const float *x, const void *wg, const void *wu, const void *wdt, int dtype, int B, int H,
           int I, double *y, double *g_out, double *u_out, int nthreads)
{
    if (!x || !wg || !wu || !wdt || !y || B < 0 || H <= 0 || I < 0 || (dtype != OR_F32 && dtype != OR_BF16))
        return -1;
    nthreads = set_threads(nthreads);
    size_t nI = I > 0 ? (size_t)I : 1;
    double *g = malloc(nI * sizeof *g), *u = malloc(nI * sizeof *u), *h = malloc(nI * sizeof *h);
    if (!g || !u || !h) {
        free(g); free(u); free(h);
        return -1;
    }
    for (int t = 0; t < B; ++t) {
        ffn_token(x + (size_t)t * H, wg, wu, wdt, dtype, H, I, y + (size_t)t * H, g, u, h, nthreads);
        if (g_out)
            memcpy(g_out + (size_t)t * I, g, (size_t)I * sizeof *g);
        if (u_out)
            memcpy(u_out + (size_t)t * I, u, (size_t)I * sizeof *u);
    }
    free(g); free(u); free(h);
    return 0;
}

/*
 * The FFN with a gate-only ReLU (section 2, Eq. gated-MLP with F_act = ReLU,
 * i.e. ReGLU, the ReLUfication baseline of section 3.1) or its shifted form
 * (section 3.1: shifted-ReLU moves the ReLU threshold of the gate to mask
 * more of it; read here as max(0, gate - tau)), next to dReLU:
 *   act 0 (dReLU):  Combined_i = max(0, g_i) * max(0, u_i)      (tau must be 0)
 *   act 1 (ReGLU):  Combined_i = max(0, g_i - tau) * u_i          (up unmasked)
 * Same layout, order and outputs as or_ffn (g_out / u_out: the projections
 * before any activation).  Returns 0, or -1 on bad arguments.
 */
int or_ffn_act(const float *x, const void *wg, const void *wu, const void *wdt, int dtype, int B, int H,
               int I, int act, double tau, double *y, double *g_out, double *u_out, int nthreads)
{
    if (!x || !wg || !wu || !wdt || !y || B < 0 || H <= 0 || I < 0 || (dtype != OR_F32 && dtype != OR_BF16) ||
        (act != 0 && act != 1) || (act == 0 && tau != 0.0) || !isfinite(tau))
        return -1;
    nthreads = set_threads(nthreads);
    size_t nI = I > 0 ? (size_t)I : 1;
    double *ha = malloc(nI * sizeof *ha);
    if (!ha)
        return -1;
    for (int t = 0; t < B; ++t) {
        const float *xt = x + (size_t)t * H;
        int i;
#pragma omp parallel for num_threads(nthreads) schedule(static)
        for (i = 0; i < I; ++i) {
            double sg = 0.0, su = 0.0;
            size_t row = (size_t)i * (size_t)H;
            for (int j = 0; j < H; ++j) {
                sg += load_w(wg, dtype, row + j) * (double)xt[j];
                su += load_w(wu, dtype, row + j) * (double)xt[j];
            }
            if (g_out)
                g_out[(size_t)t * I + i] = sg;
            if (u_out)
                u_out[(size_t)t * I + i] = su;
            if (act == 0)
                ha[i] = (sg > 0.0 && su > 0.0) ? sg * su : 0.0;
            else
                ha[i] = sg > tau ? (sg - tau) * su : 0.0;
        }
        double *yt = y + (size_t)t * H;
        int nblk = (H + 63) / 64;
        int b;
#pragma omp parallel for num_threads(nthreads) schedule(static)
        for (b = 0; b < nblk; ++b) {
            int j0 = b * 64, j1 = j0 + 64 < H ? j0 + 64 : H;
            for (int j = j0; j < j1; ++j)
                yt[j] = 0.0;
            for (int ii = 0; ii < I; ++ii) {
                double hv = ha[ii];
                size_t row = (size_t)ii * (size_t)H;
                for (int j = j0; j < j1; ++j)
                    yt[j] += load_w(wdt, dtype, row + j) * hv;
            }
        }
    }
    free(ha);
    return 0;
}

/*
 * The dReLU FFN with the top-k magnitude mask (section 3.2, Eq. mask and Eq.
 * sparsify-gated-MLP): per token only the `keep` neurons with the largest
 * |Combined| contribute (ties: the lower neuron index first; when keep
 * exceeds the number of non-zero activations the extra kept neurons are
 * zeros and change nothing):
 *   y_t[j] = sum over kept i, ascending, of Combined_i * W_down_t[i][j].
 *   n_kept [B] (nullable): kept neurons with a non-zero Combined activation.
 * Returns 0, or -1 on bad arguments / allocation failure.
 */
static int cmp_desc_then_index(const void *pa, const void *pb, void *ctx)
{
    const double *h = (const double *)ctx;
    int a = *(const int *)pa, b = *(const int *)pb;
    double va = fabs(h[a]), vb = fabs(h[b]);
    if (va > vb)
        return -1;
    if (va < vb)
        return 1;
    return (a > b) - (a < b);
}

int or_ffn_topk(const float *x, const void *wg, const void *wu, const void *wdt, int dtype, int B, int H, int I,
                int keep, double *y, int32_t *n_kept, int nthreads)
{
    if (!x || !wg || !wu || !wdt || !y || B < 0 || H <= 0 || I < 0 || keep < 0 ||
        (dtype != OR_F32 && dtype != OR_BF16))
        return -1;
    nthreads = set_threads(nthreads);
    size_t nI = I > 0 ? (size_t)I : 1;
    double *g = malloc(nI * sizeof *g), *u = malloc(nI * sizeof *u), *h = malloc(nI * sizeof *h);
    double *hk = malloc(nI * sizeof *hk);
    int *order = malloc(nI * sizeof *order);
    if (!g || !u || !h || !hk || !order) {
        free(g); free(u); free(h); free(hk); free(order);
        return -1;
    }
    for (int t = 0; t < B; ++t) {
        double *yt = y + (size_t)t * H;
        /* Combined for every neuron (dReLU), then its dense sum is not used:
           only the kept terms enter y. */
        ffn_token(x + (size_t)t * H, wg, wu, wdt, dtype, H, I, yt, g, u, h, nthreads);
        for (int i = 0; i < I; ++i)
            order[i] = i;
        qsort_r(order, (size_t)I, sizeof *order, cmp_desc_then_index, h);
        int k = keep < I ? keep : I, nk = 0;
        for (int i = 0; i < I; ++i)
            hk[i] = 0.0;
        for (int r = 0; r < k; ++r) {
            hk[order[r]] = h[order[r]];
            nk += h[order[r]] != 0.0;
        }
        if (n_kept)
            n_kept[t] = nk;
        int nblk = (H + 63) / 64;
        int b;
#pragma omp parallel for num_threads(nthreads) schedule(static)
        for (b = 0; b < nblk; ++b) {
            int j0 = b * 64, j1 = j0 + 64 < H ? j0 + 64 : H;
            for (int j = j0; j < j1; ++j)
                yt[j] = 0.0;
            for (int ii = 0; ii < I; ++ii) {
                double hv = hk[ii];
                if (hv == 0.0)
                    continue;
                size_t row = (size_t)ii * (size_t)H;
                for (int j = j0; j < j1; ++j)
                    yt[j] += load_w(wdt, dtype, row + j) * hv;
            }
        }
    }
    free(g); free(u); free(h); free(hk); free(order);
    return 0;
}

/*
 * The dReLU FFN evaluated over given neuron lists: the interface an
 * activation predictor drives (section 7 of the paper: the inference engine
 * evaluates only the neurons predicted active).  For token t only the
 * entries idx[t][0 .. min(count[t], maxc)) contribute, in list order;
 * entries outside [0, I) are skipped and a repeated entry counts again:
 *   y_t[j] = sum over listed i of max(0, g_i) max(0, u_i) W_down_t[i][j].
 * With a list that holds every neuron whose Combined activation is non-zero
 * (G_t, or all neurons ascending) this is the dense FFN term for term.
 *   idx [B][maxc], count [B] int32; y [B][H] fp64 out;
 *   n_open / n_active [B] (nullable): listed entries with g > 0, and with
 *   g > 0 and u > 0.
 * Returns 0, or -1 on bad arguments / allocation failure.
 */
int or_ffn_given(const float *x, const void *wg, const void *wu, const void *wdt, int dtype, int B, int H,
                 int I, const int32_t *idx, const int32_t *count, int maxc, double *y, int32_t *n_open,
                 int32_t *n_active, int nthreads)
{
    if (!x || !wg || !wu || !wdt || !idx || !count || !y || B < 0 || H <= 0 || I < 0 || maxc < 0 ||
        (dtype != OR_F32 && dtype != OR_BF16))
        return -1;
    nthreads = set_threads(nthreads);
    size_t nL = maxc > 0 ? (size_t)maxc : 1;
    double *hl = malloc(nL * sizeof *hl);
    if (!hl)
        return -1;
    for (int t = 0; t < B; ++t) {
        const float *xt = x + (size_t)t * H;
        const int32_t *lt = idx + (size_t)t * maxc;
        int n = count[t] < 0 ? 0 : (count[t] > maxc ? maxc : count[t]);
        int no = 0, na = 0;
        /* Combined activation of each list entry (0 for skipped entries). */
        int k;
#pragma omp parallel for num_threads(nthreads) schedule(static) reduction(+ : no, na)
        for (k = 0; k < n; ++k) {
            int i = lt[k];
            hl[k] = 0.0;
            if (i < 0 || i >= I)
                continue;
            double sg = 0.0, su = 0.0;
            size_t row = (size_t)i * (size_t)H;
            for (int j = 0; j < H; ++j) {
                sg += load_w(wg, dtype, row + j) * (double)xt[j];
                su += load_w(wu, dtype, row + j) * (double)xt[j];
            }
            no += sg > 0.0;
            na += sg > 0.0 && su > 0.0;
            hl[k] = (sg > 0.0 && su > 0.0) ? sg * su : 0.0;
        }
        if (n_open)
            n_open[t] = no;
        if (n_active)
            n_active[t] = na;
        /* y[j] = sum over the list, in list order, of h_k * W_down_t[idx_k][j]. */
        double *yt = y + (size_t)t * H;
        int nblk = (H + 63) / 64;
        int b;
#pragma omp parallel for num_threads(nthreads) schedule(static)
        for (b = 0; b < nblk; ++b) {
            int j0 = b * 64, j1 = j0 + 64 < H ? j0 + 64 : H;
            for (int j = j0; j < j1; ++j)
                yt[j] = 0.0;
            for (int kk = 0; kk < n; ++kk) {
                int i = lt[kk];
                if (i < 0 || i >= I)
                    continue;
                double hv = hl[kk];
                size_t row = (size_t)i * (size_t)H;
                for (int j = j0; j < j1; ++j)
                    yt[j] += load_w(wdt, dtype, row + j) * hv;
            }
        }
    }
    free(hl);
    return 0;
}

/*
 * Router of the MoE layer for one token: logits, softmax, top-k, renormalised
 * weights.  logits / probs [E] out; idx [K] ascending-by-rank (rank 0 = largest
 * p); w [K] the renormalised weight of idx[k].
 */
static void route_token(const float *x, const void *wr, int dtype, int H, int E, int K, double *logits,
                        double *probs, int32_t *idx, double *w)
{
    double m = -INFINITY;
    for (int e = 0; e < E; ++e) {
        double s = 0.0;
        for (int j = 0; j < H; ++j)
            s += load_w(wr, dtype, (size_t)e * H + j) * (double)x[j];
        logits[e] = s;
        if (s > m)
            m = s;
    }
    double z = 0.0;
    for (int e = 0; e < E; ++e) {
        probs[e] = exp(logits[e] - m);
        z += probs[e];
    }
    for (int e = 0; e < E; ++e)
        probs[e] /= z;

    /* Selection: repeatedly take the largest remaining p; a strict '>' keeps the
       lower index on ties. */
    char taken[256];
    memset(taken, 0, sizeof taken);
    double psum = 0.0;
    for (int k = 0; k < K; ++k) {
        int best = -1;
        for (int e = 0; e < E; ++e)
            if (!taken[e] && (best < 0 || probs[e] > probs[best]))
                best = e;
        taken[best] = 1;
        idx[k] = best;
        psum += probs[best];
    }
    for (int k = 0; k < K; ++k)
        w[k] = probs[idx[k]] / psum;
}

/*
 * Mixture-of-Experts layer with dReLU experts.
 *   x [B][H]; wr [E][H]; wg, wu, wdt [E][I][H]; y [B][H] fp64 out.
 *   topk_idx [B][K], topk_w [B][K], probs [B][E]: nullable outputs.
 *   g_out, u_out [B][K][I]: nullable, the routed experts' projections in
 *   rank order.
 */
int or_moe(const float *x, const void *wr, const void *wg, const void *wu, const void *wdt, int dtype,
           int B, int H, int I, int E, int K, double *y, int32_t *topk_idx, double *topk_w,
           double *probs_out, double *g_out, double *u_out, int nthreads)
{
    if (!x || !wr || !wg || !wu || !wdt || !y || B < 0 || H <= 0 || I < 0 || E < 1 || E > 256 || K < 1 ||
        K > E || (dtype != OR_F32 && dtype != OR_BF16))
        return -1;
    nthreads = set_threads(nthreads);
    size_t nI = I > 0 ? (size_t)I : 1;
    size_t esz = dtype == OR_F32 ? 4 : 2;
    size_t expert_bytes = (size_t)I * (size_t)H * esz;
    double *g = malloc(nI * sizeof *g), *u = malloc(nI * sizeof *u), *h = malloc(nI * sizeof *h);
    double *ye = malloc((size_t)H * sizeof *ye);
    double logits[256], probs[256], w[256];
    int32_t idx[256];
    if (!g || !u || !h || !ye) {
        free(g); free(u); free(h); free(ye);
        return -1;
    }
    for (int t = 0; t < B; ++t) {
        const float *xt = x + (size_t)t * H;
        double *yt = y + (size_t)t * H;
        route_token(xt, wr, dtype, H, E, K, logits, probs, idx, w);
        for (int j = 0; j < H; ++j)
            yt[j] = 0.0;
        /* Experts are combined in ascending expert index. */
        for (int e = 0; e < E; ++e) {
            int rank = -1;
            for (int k = 0; k < K; ++k)
                if (idx[k] == e)
                    rank = k;
            if (rank < 0)
                continue;
            const char *base_g = (const char *)wg + (size_t)e * expert_bytes;
            const char *base_u = (const char *)wu + (size_t)e * expert_bytes;
            const char *base_d = (const char *)wdt + (size_t)e * expert_bytes;
            ffn_token(xt, base_g, base_u, base_d, dtype, H, I, ye, g, u, h, nthreads);
            for (int j = 0; j < H; ++j)
                yt[j] += w[rank] * ye[j];
            if (g_out)
                memcpy(g_out + ((size_t)t * K + rank) * I, g, (size_t)I * sizeof *g);
            if (u_out)
                memcpy(u_out + ((size_t)t * K + rank) * I, u, (size_t)I * sizeof *u);
        }
        if (topk_idx)
            memcpy(topk_idx + (size_t)t * K, idx, (size_t)K * sizeof *idx);
        if (topk_w)
            memcpy(topk_w + (size_t)t * K, w, (size_t)K * sizeof *w);
        if (probs_out)
            memcpy(probs_out + (size_t)t * E, probs, (size_t)E * sizeof *probs);
    }
    free(g); free(u); free(h); free(ye);
    return 0;
}

/* Number of OpenMP threads a call with nthreads <= 0 would use. */
int or_max_threads(void)
{
    return set_threads(0);
}
