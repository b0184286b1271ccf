/*
 * A plain C caller of the library: device memory from the HIP runtime's C API,
 * one mb_scan_fwd call through include/mbscan.h, and the result compared with
 * the fp64 oracle (oracle/liboracle.so) on the same inputs.  Test
 * infrastructure: the GPU test suite runs it after build() has compiled it.
 *
 * Shape: batch 2, dim 40 (the last 8-channel group has dead lanes), L 528 (the
 * tiled kernel, ending in a half chunk), dstate 16, fp32 in and out, with a
 * gate, a skip term, a timestep bias, h0 in and h_last out.
 * Exit status 0 when y and h_last meet the parity bars (2e-3 and 1e-4 under
 * |g - r| / (|r| + rms(r))), 1 otherwise, 2 on a runtime or argument error.
 */
#include <hip/hip_runtime_api.h>

#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include "mbscan.h"

int mbo_scan_rows(int64_t R, int64_t L, int64_t N, int delta_softplus,
                  const double *u, const double *delta, const double *z,
                  const double *A, const double *Dskip, const double *dt_bias,
                  const double *h0, const int64_t *bidx, int64_t nbatch,
                  const double *Bm, const double *Cm, double *y, double *h_last);

enum { NB = 2, DIM = 40, L = 528, N = 16 };

/* splitmix64: a counter-based generator, used here only to draw inputs */
static uint64_t sm_state = 0x2401136600000001ull;
static double uniform(double lo, double hi) {
    uint64_t z = (sm_state += 0x9e3779b97f4a7c15ull);
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    z ^= z >> 31;
    return lo + (hi - lo) * (double)(z >> 11) * (1.0 / 9007199254740992.0);
}

static float *to_device(const float *h, size_t n) {
    void *d = NULL;
    if (hipMalloc(&d, n * sizeof(float)) != hipSuccess) return NULL;
    if (hipMemcpy(d, h, n * sizeof(float), hipMemcpyHostToDevice) != hipSuccess) return NULL;
    return (float *)d;
}

static double rel_err(const float *g, const double *r, size_t n) {
    double ss = 0.0, worst = 0.0;
    for (size_t i = 0; i < n; ++i) ss += r[i] * r[i];
    const double rms = sqrt(ss / (double)n);
    for (size_t i = 0; i < n; ++i) {
        if (!isfinite(g[i])) return INFINITY;
        const double den = fabs(r[i]) + rms;
        const double e = fabs((double)g[i] - r[i]) / (den > 0.0 ? den : 1.0);
        if (e > worst) worst = e;
    }
    return worst;
}

int main(void) {
    const size_t act = (size_t)NB * DIM * L, bc = (size_t)NB * N * L, st = (size_t)NB * DIM * N;
    float *u = malloc(act * 4), *dl = malloc(act * 4), *z = malloc(act * 4), *Bm = malloc(bc * 4),
          *Cm = malloc(bc * 4), *A = malloc((size_t)DIM * N * 4), *Ds = malloc(DIM * 4), *bias = malloc(DIM * 4),
          *h0 = malloc(st * 4), *y = malloc(act * 4), *hl = malloc(st * 4);
    double *du = malloc(act * 8), *ddl = malloc(act * 8), *dz = malloc(act * 8), *dB = malloc(bc * 8),
           *dC = malloc(bc * 8), *dA = malloc((size_t)NB * DIM * N * 8), *dDs = malloc(NB * DIM * 8),
           *dbias = malloc(NB * DIM * 8), *dh0 = malloc(st * 8), *yr = malloc(act * 8), *hr = malloc(st * 8);
    int64_t *bidx = malloc(NB * DIM * sizeof(int64_t));
    if (!u || !dl || !z || !Bm || !Cm || !A || !Ds || !bias || !h0 || !y || !hl || !du || !ddl || !dz || !dB ||
        !dC || !dA || !dDs || !dbias || !dh0 || !yr || !hr || !bidx)
        return 2;

    for (size_t i = 0; i < act; ++i) {
        u[i] = (float)uniform(-1.0, 1.0);
        dl[i] = (float)uniform(-1.0, 1.0);
        z[i] = (float)uniform(-2.0, 2.0);
    }
    for (size_t i = 0; i < bc; ++i) {
        Bm[i] = (float)uniform(-1.0, 1.0);
        Cm[i] = (float)uniform(-1.0, 1.0);
    }
    for (int d = 0; d < DIM; ++d) {
        for (int n = 0; n < N; ++n) A[d * N + n] = -(float)(n + 1);
        Ds[d] = (float)uniform(0.5, 1.5);
        bias[d] = (float)log(expm1(uniform(1e-3, 0.1)));
    }
    for (size_t i = 0; i < st; ++i) h0[i] = (float)uniform(-0.1, 0.1);

    /* the oracle sees the same fp32 values, widened */
    for (size_t i = 0; i < act; ++i) { du[i] = u[i]; ddl[i] = dl[i]; dz[i] = z[i]; }
    for (size_t i = 0; i < bc; ++i) { dB[i] = Bm[i]; dC[i] = Cm[i]; }
    for (int r = 0; r < NB * DIM; ++r) {
        const int d = r % DIM;
        bidx[r] = r / DIM;
        dDs[r] = Ds[d];
        dbias[r] = bias[d];
        for (int n = 0; n < N; ++n) dA[r * N + n] = A[d * N + n];
    }
    for (size_t i = 0; i < st; ++i) dh0[i] = h0[i];
    if (mbo_scan_rows(NB * DIM, L, N, 1, du, ddl, dz, dA, dDs, dbias, dh0, bidx, NB, dB, dC, yr, hr) != 0) {
        fprintf(stderr, "oracle rejected its arguments\n");
        return 2;
    }

    float *gu = to_device(u, act), *gdl = to_device(dl, act), *gz = to_device(z, act), *gB = to_device(Bm, bc),
          *gC = to_device(Cm, bc), *gA = to_device(A, (size_t)DIM * N), *gDs = to_device(Ds, DIM),
          *gbias = to_device(bias, DIM), *gh0 = to_device(h0, st), *gy = to_device(y, act), *ghl = to_device(hl, st);
    if (!gu || !gdl || !gz || !gB || !gC || !gA || !gDs || !gbias || !gh0 || !gy || !ghl) {
        fprintf(stderr, "device allocation or copy failed\n");
        return 2;
    }
    hipStream_t stream = NULL;
    if (hipStreamCreate(&stream) != hipSuccess) return 2;

    if (mb_scan_fwd(NULL, gu, gdl, gA, gB, gC, gDs, gbias, gz, gh0, gy, ghl, (void *)stream) != MB_ERR_NULL) {
        fprintf(stderr, "a null descriptor was not rejected\n");
        return 2;
    }
    mb_scan_desc desc = {NB, DIM, L, N, MB_F32, MB_F32, 1, 0};
    const int status = mb_scan_fwd(&desc, gu, gdl, gA, gB, gC, gDs, gbias, gz, gh0, gy, ghl, (void *)stream);
    if (status != MB_OK) {
        fprintf(stderr, "mb_scan_fwd: %s\n", mb_status_string(status));
        return 2;
    }
    if (hipStreamSynchronize(stream) != hipSuccess) return 2;
    if (hipMemcpy(y, gy, act * 4, hipMemcpyDeviceToHost) != hipSuccess ||
        hipMemcpy(hl, ghl, st * 4, hipMemcpyDeviceToHost) != hipSuccess)
        return 2;

    const double ey = rel_err(y, yr, act), eh = rel_err(hl, hr, st);
    printf("c caller: ABI version %d, y error %.2e, h_last error %.2e\n", mb_abi_version(), ey, eh);
    (void)hipStreamDestroy(stream);
    return (ey <= 2e-3 && eh <= 1e-4) ? 0 : 1;
}
