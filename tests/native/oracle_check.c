/*
 * Drives every function of the fp64 oracle (oracle/oracle.c, linked in
 * directly) on small random inputs, fp32 and bf16, so that the address and
 * undefined-behaviour sanitizers see all of its indexing.  Built with gcc and
 * -fsanitize=address,undefined by tests/test_plan_cpu.py; prints "ok" or the
 * first failed check.  Besides running clean under the sanitizers, the
 * calls must agree bitwise where the definitions coincide exactly:
 *   - the given-list FFN over all neurons (ascending) is the dense FFN;
 *   - the activation variant with act 0 (dReLU) is the dense FFN;
 *   - the top-k mask keeping every neuron is the dense FFN;
 *   - the MoE layer with one expert and top-1 is that expert's FFN.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int or_ffn(const float *x, const void *wg, const void *wu, const void *wdt, int dtype, int B, int H, int I,
           double *y, double *g, double *u, int nthreads);
int or_ffn_act(const float *x, const void *wg, const void *wu, const void *wdt, int dtype, int B, int H, int I,
               int act, double tau, double *y, double *g, double *u, int nthreads);
int or_ffn_topk(const float *x, const void *wg, const void *wu, const void *wdt, int dtype, int B, int H, int I,
                int keep, double *y, int32_t *n_kept, int nthreads);
int or_ffn_given(const float *x, const void *wg, const void *wu, const void *wdt, int dtype, int B, int H, int I,
                 const int32_t *idx, const int32_t *count, int maxc, double *y, int32_t *n_open,
                 int32_t *n_active, int nthreads);
int or_moe(const float *x, const void *wr, const void *wg, const void *wu, const void *wdt, int dtype, int B,
           int H, int I, int E, int K, double *y, int32_t *topk_idx, double *topk_w, double *probs, double *g,
           double *u, int nthreads);

static uint64_t rs = 0x9e3779b97f4a7c15ull;
static double urand(void)
{
    rs ^= rs << 13;
    rs ^= rs >> 7;
    rs ^= rs << 17;
    return (double)(rs >> 11) / 9007199254740992.0 * 2.0 - 1.0;
}

/* n random weights in dtype 0 (fp32) or 1 (bf16 bits, truncated); caller frees */
static void *weights(size_t n, int dtype, double scale)
{
    if (dtype == 0) {
        float *w = malloc(n * sizeof *w);
        for (size_t i = 0; i < n; ++i)
            w[i] = (float)(urand() * scale);
        return w;
    }
    uint16_t *w = malloc(n * sizeof *w);
    for (size_t i = 0; i < n; ++i) {
        float f = (float)(urand() * scale);
        uint32_t b;
        memcpy(&b, &f, 4);
        w[i] = (uint16_t)(b >> 16);
    }
    return w;
}

static int fail(const char *what, int dtype, int B, int H, int I)
{
    printf("FAIL %s dtype=%d B=%d H=%d I=%d\n", what, dtype, B, H, I);
    return 1;
}

static int one_case(int dtype, int B, int H, int I, int nthreads)
{
    size_t nx = (size_t)B * H, nw = (size_t)I * H;
    float *x = malloc(nx * sizeof *x);
    for (size_t i = 0; i < nx; ++i)
        x[i] = (float)urand();
    for (int t = 0; t < B; ++t)
        x[(size_t)t * H] = 1.0f;
    void *wg = weights(nw, dtype, 1.0), *wu = weights(nw, dtype, 1.0), *wd = weights(nw, dtype, 1.0);
    double *y = malloc(nx * sizeof *y), *y2 = malloc(nx * sizeof *y2);
    double *g = malloc((size_t)B * I * sizeof *g), *u = malloc((size_t)B * I * sizeof *u);
    int rc = 0;
    if (or_ffn(x, wg, wu, wd, dtype, B, H, I, y, g, u, nthreads))
        rc = fail("or_ffn", dtype, B, H, I);

    /* the given list of every neuron, ascending, plus one entry out of range */
    int maxc = I + 1;
    int32_t *idx = malloc((size_t)B * maxc * sizeof *idx), *cnt = malloc(B * sizeof *cnt);
    int32_t *no = malloc(B * sizeof *no), *na = malloc(B * sizeof *na);
    for (int t = 0; t < B; ++t) {
        for (int i = 0; i < I; ++i)
            idx[(size_t)t * maxc + i] = i;
        idx[(size_t)t * maxc + I] = I + 7; /* skipped */
        cnt[t] = maxc;
    }
    if (!rc && or_ffn_given(x, wg, wu, wd, dtype, B, H, I, idx, cnt, maxc, y2, no, na, nthreads))
        rc = fail("or_ffn_given", dtype, B, H, I);
    if (!rc && memcmp(y, y2, nx * sizeof *y))
        rc = fail("given(all) != dense", dtype, B, H, I);

    double *g2 = malloc((size_t)B * I * sizeof *g2), *u2 = malloc((size_t)B * I * sizeof *u2);
    if (!rc && or_ffn_act(x, wg, wu, wd, dtype, B, H, I, 0, 0.0, y2, g2, u2, nthreads))
        rc = fail("or_ffn_act", dtype, B, H, I);
    if (!rc && memcmp(y, y2, nx * sizeof *y))
        rc = fail("act 0 != dense", dtype, B, H, I);
    if (!rc && or_ffn_act(x, wg, wu, wd, dtype, B, H, I, 1, 0.25, y2, g2, u2, nthreads))
        rc = fail("or_ffn_act shifted", dtype, B, H, I);

    int32_t *nk = malloc(B * sizeof *nk);
    if (!rc && or_ffn_topk(x, wg, wu, wd, dtype, B, H, I, I, y2, nk, nthreads))
        rc = fail("or_ffn_topk", dtype, B, H, I);
    if (!rc && memcmp(y, y2, nx * sizeof *y))
        rc = fail("topk(keep all) != dense", dtype, B, H, I);
    if (!rc && or_ffn_topk(x, wg, wu, wd, dtype, B, H, I, I / 3, y2, nk, nthreads))
        rc = fail("or_ffn_topk partial", dtype, B, H, I);

    /* MoE with one expert and top-1 is that expert's FFN */
    void *wr = weights((size_t)H, dtype, 1.0);
    int32_t *ti = malloc(B * sizeof *ti);
    double *tw = malloc(B * sizeof *tw), *pr = malloc(B * sizeof *pr);
    if (!rc && or_moe(x, wr, wg, wu, wd, dtype, B, H, I, 1, 1, y2, ti, tw, pr, g2, u2, nthreads))
        rc = fail("or_moe E=1", dtype, B, H, I);
    if (!rc && memcmp(y, y2, nx * sizeof *y))
        rc = fail("moe(E=1,K=1) != dense", dtype, B, H, I);

    /* MoE with 4 experts, top-2 */
    {
        int E = 4, K = 2;
        void *wr4 = weights((size_t)E * H, dtype, 1.0);
        void *eg = weights((size_t)E * nw, dtype, 1.0), *eu = weights((size_t)E * nw, dtype, 1.0);
        void *ed = weights((size_t)E * nw, dtype, 1.0);
        int32_t *ti4 = malloc((size_t)B * K * sizeof *ti4);
        double *tw4 = malloc((size_t)B * K * sizeof *tw4), *pr4 = malloc((size_t)B * E * sizeof *pr4);
        double *g4 = malloc((size_t)B * K * I * sizeof *g4), *u4 = malloc((size_t)B * K * I * sizeof *u4);
        if (!rc && or_moe(x, wr4, eg, eu, ed, dtype, B, H, I, E, K, y2, ti4, tw4, pr4, g4, u4, nthreads))
            rc = fail("or_moe E=4", dtype, B, H, I);
        for (int t = 0; !rc && t < B; ++t)
            if (ti4[t * K] == ti4[t * K + 1] || ti4[t * K] < 0 || ti4[t * K] >= E)
                rc = fail("moe routing", dtype, B, H, I);
        free(wr4), free(eg), free(eu), free(ed), free(ti4), free(tw4), free(pr4), free(g4), free(u4);
    }
    free(x), free(wg), free(wu), free(wd), free(y), free(y2), free(g), free(u), free(idx), free(cnt);
    free(no), free(na), free(g2), free(u2), free(nk), free(wr), free(ti), free(tw), free(pr);
    return rc;
}

int main(void)
{
    const int shapes[][3] = {{1, 8, 1}, {1, 8, 7}, {2, 40, 65}, {3, 64, 130}, {1, 200, 333}, {4, 16, 5}};
    for (int dtype = 0; dtype < 2; ++dtype)
        for (size_t s = 0; s < sizeof shapes / sizeof shapes[0]; ++s)
            for (int th = 1; th <= 3; th += 2)
                if (one_case(dtype, shapes[s][0], shapes[s][1], shapes[s][2], th))
                    return 1;
    /* rejected arguments return -1 without touching anything */
    double y;
    if (or_ffn(NULL, NULL, NULL, NULL, 0, 1, 8, 1, &y, NULL, NULL, 1) != -1) {
        printf("FAIL null arguments accepted\n");
        return 1;
    }
    printf("ok\n");
    return 0;
}
