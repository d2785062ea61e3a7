/*
 * The C ABI used from plain C, without Python or PyTorch: device memory from
 * the HIP runtime, one ts_ffn_sparse call (fp32 weights, two tokens), the
 * result checked against a direct double-precision evaluation of the dReLU
 * FFN (Eq. gated-MLP with ReLU on both projections), one argument error
 * that must leave the output untouched, and the allocation-free entry point,
 * which must give the same bits.  Prints "c_smoke ok" and exits 0 on success.
 */
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>
#include <stdlib.h>

#include "turbosparse.h"

#define B 2
#define H 256
#define I 600

static uint64_t state = 0x9E3779B97F4A7C15ull;
static float uniform(void)  /* xorshift64*, in [-1, 1) */
{
    state ^= state >> 12;
    state ^= state << 25;
    state ^= state >> 27;
    return (float)((double)((state * 0x2545F4914F6CDD1Dull) >> 11) / 9007199254740992.0 * 2.0 - 1.0);
}

#define CHECK(call)                                                   \
    do {                                                              \
        hipError_t e_ = (call);                                       \
        if (e_ != hipSuccess) {                                       \
            fprintf(stderr, "%s: %s\n", #call, hipGetErrorString(e_)); \
            return 2;                                                 \
        }                                                             \
    } while (0)

int main(void)
{
    static float x[B * H], wg[I * H], wu[I * H], wd[I * H], out[B * H];
    for (int k = 0; k < B * H; ++k) x[k] = uniform();
    for (int k = 0; k < I * H; ++k) {
        wg[k] = uniform() * 0.0625f;
        wu[k] = uniform() * 0.0625f;
        wd[k] = uniform() * 0.0625f;
    }
    for (int t = 0; t < B; ++t) x[t * H] = 1.0f;
    for (int i = 0; i < I; ++i) wg[i * H] = -0.1f;  /* a bias column: fewer open gates */

    /* direct evaluation */
    static double ref[B * H];
    int active = 0;
    for (int t = 0; t < B; ++t) {
        for (int j = 0; j < H; ++j) ref[t * H + j] = 0.0;
        for (int i = 0; i < I; ++i) {
            double g = 0.0, u = 0.0;
            for (int j = 0; j < H; ++j) {
                g += (double)wg[i * H + j] * x[t * H + j];
                u += (double)wu[i * H + j] * x[t * H + j];
            }
            if (g > 0.0 && u > 0.0) {
                ++active;
                for (int j = 0; j < H; ++j) ref[t * H + j] += g * u * wd[i * H + j];
            }
        }
    }

    size_t wsb = ts_ffn_workspace_bytes(B, H, I, TS_F32);
    if (wsb == 0) {
        fprintf(stderr, "workspace size 0\n");
        return 1;
    }
    float *dx, *dg, *du, *dd, *dout;
    void *ws;
    CHECK(hipMalloc((void **)&dx, sizeof x));
    CHECK(hipMalloc((void **)&dg, sizeof wg));
    CHECK(hipMalloc((void **)&du, sizeof wu));
    CHECK(hipMalloc((void **)&dd, sizeof wd));
    CHECK(hipMalloc((void **)&dout, sizeof out));
    CHECK(hipMalloc(&ws, wsb));
    CHECK(hipMemcpy(dx, x, sizeof x, hipMemcpyHostToDevice));
    CHECK(hipMemcpy(dg, wg, sizeof wg, hipMemcpyHostToDevice));
    CHECK(hipMemcpy(du, wu, sizeof wu, hipMemcpyHostToDevice));
    CHECK(hipMemcpy(dd, wd, sizeof wd, hipMemcpyHostToDevice));

    ts_status s = ts_ffn_sparse(dx, dg, du, dd, TS_F32, B, H, I, dout, NULL, ws, wsb, NULL);
    if (s != TS_OK) {
        fprintf(stderr, "ts_ffn_sparse: %s (%s)\n", ts_status_str(s), ts_last_error());
        return 1;
    }
    CHECK(hipDeviceSynchronize());
    CHECK(hipMemcpy(out, dout, sizeof out, hipMemcpyDeviceToHost));
    double num = 0.0, den = 0.0;
    for (int k = 0; k < B * H; ++k) {
        num += (out[k] - ref[k]) * (out[k] - ref[k]);
        den += ref[k] * ref[k];
    }
    double rel = sqrt(num / den);
    if (!(rel <= 1e-5) || active == 0) {
        fprintf(stderr, "rel L2 %g, active %d\n", rel, active);
        return 1;
    }

    /* an argument error enqueues nothing and leaves the output untouched */
    s = ts_ffn_sparse(dx, dg, du, dd, TS_F32, B, H, I, (float *)((char *)dout + 4), NULL, ws, wsb, NULL);
    if (s != TS_ERR_ALIGN) {
        fprintf(stderr, "misaligned out: got %s\n", ts_status_str(s));
        return 1;
    }
    static float again[B * H];
    CHECK(hipDeviceSynchronize());
    CHECK(hipMemcpy(again, dout, sizeof again, hipMemcpyDeviceToHost));
    for (int k = 0; k < B * H; ++k)
        if (again[k] != out[k]) {
            fprintf(stderr, "output changed by a rejected call\n");
            return 1;
        }

    /* the allocation-free entry point: same kernels on the library's own
       scratch, so the same bits */
    s = ts_ffn_sparse_noalloc(dx, dg, du, dd, TS_F32, B, H, I, dout, NULL, NULL);
    if (s != TS_OK) {
        fprintf(stderr, "ts_ffn_sparse_noalloc: %s (%s)\n", ts_status_str(s), ts_last_error());
        return 1;
    }
    CHECK(hipDeviceSynchronize());
    CHECK(hipMemcpy(again, dout, sizeof again, hipMemcpyDeviceToHost));
    if (memcmp(again, out, sizeof again) != 0) {
        fprintf(stderr, "ts_ffn_sparse_noalloc differs from ts_ffn_sparse\n");
        return 1;
    }

    hipFree(dx);
    hipFree(dg);
    hipFree(du);
    hipFree(dd);
    hipFree(dout);
    hipFree(ws);
    printf("c_smoke ok: rel L2 %.3g, %d active neurons, %s\n", rel, active, ts_version());
    return 0;
}
