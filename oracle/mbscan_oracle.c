/*
 * mbscan_oracle.c -- TEST INFRASTRUCTURE ONLY (the parity oracle).
 *
 * A plain, slow, obviously correct fp64 CPU implementation of the selective
 * scan that MambaByte runs in every layer (MambaByte, Section 2 "Selective
 * SSMs", eq. (2); Appendix D "Discretization and selection"; Table 8, MambaByte
 * rows "Discretization", "Recurrence", "Output", "Element-wise gating").
 *
 * Only the test-suite, the smoke check and the benchmark's CPU-baseline leg
 * may load this file.  It shares no source with the HIP library: no headers,
 * no helpers, no constants.  It is a time-ordered loop, nothing is blocked,
 * fused or reordered, and every number is an IEEE double.
 *
 * What is computed, for every row r (one (batch, channel) pair) and every
 * state index n < N, starting from h[n] = h0[r][n] (zeros when h0 is absent):
 *
 *   v      = delta[r][t] + dt_bias[r]                       (dt_bias absent => 0)
 *   dlt    = softplus(v) if delta_softplus else v           (eq. (3): softplus makes the step positive)
 *   abar   = exp(dlt * A[r][n])                             (App. D: zero-order hold on A)
 *   bbar_x = (dlt * B[b][n][t]) * u[r][t]                   (App. D footnote: simplified Euler on B)
 *   h[n]   = abar * h[n] + bbar_x                           (eq. (2): h[k] = Abar h[k-1] + Bbar x[k])
 *   yv     = sum_n C[b][n][t] * h[n] + Dskip[r] * u[r][t]   (eq. (2) y = C h, plus the skip term of Table 8)
 *   y[r][t]= yv * silu(z[r][t]) if z is given, else yv      (Table 8 "Element-wise gating"; Fig. 5 Swish gate)
 *
 * and h_last[r] = h after the final step.  Optionally the state is also
 * recorded at requested positions: h_pos[r][k] = h after timestep pos[r][k],
 * where position -1 is the initial state and a position outside [-1, L-1]
 * reads NaN (the verifier of Appendix F, Algorithm 1, resumes from the state
 * at the bifurcation position c; Section 3, speculative decoding paragraph).
 * b = bidx[r] selects the batch
 * element whose B and C rows (shape N x L, time contiguous) the row reads:
 * B and C are shared by all channels of a batch element (Section 2, after
 * eq. (3)); A, Dskip and dt_bias are per channel.
 *
 * The single-step entry point is the loop body above for one t, updating h
 * in place (Section 2: the recurrence is run directly during generation).
 *
 * The file also holds the oracle of the step upstream of the scan: the causal
 * depthwise 1D convolution of the Mamba block (Table 8, "Pre-SSM 1D
 * convolution"; Fig. 5, right, followed by the Swish activation; kernel size
 * k = 4 in Table 9), with a carried state of the last k - 1 inputs so that a
 * sequence can be resumed or decoded byte by byte:
 *
 *   xin(s)   = x[r][s] for s >= 0, state_in[r][k - 1 + s] for -(k-1) <= s < 0
 *              (zeros when state_in is absent)
 *   pre[t]   = bias[r] + sum_{i < k} w[r][i] * xin(t - (k-1) + i)
 *   y[r][t]  = silu(pre[t]) if apply_silu else pre[t]
 *   state_out[r][j] = xin(L - (k-1) + j)   for j < k - 1
 *
 * And the backward of the scan (training at the 8,192-byte context, Section 4,
 * Appendix C): given dy (and optionally dh_last), the gradients with respect to
 * every input, by reverse-mode differentiation of the loop above.  With
 * lambda_t[n] the total gradient of the loss with respect to h_t[n]:
 *
 *   ds_t        = dy_t * silu(z_t)  (dy_t without a gate)
 *   dz_t        = dy_t * s_t * silu'(z_t),  s_t = sum_n C_t[n] h_t[n] + Dskip u_t
 *   lambda_t[n] = ds_t C_t[n] + abar_{t+1}[n] lambda_{t+1}[n]   (+ dh_last at t = L-1)
 *   dC_t[n]    += ds_t h_t[n]                    (summed over the channels of a batch element)
 *   dB_t[n]    += lambda_t[n] dlt_t u_t          (idem)
 *   du_t        = ds_t Dskip + sum_n lambda_t[n] dlt_t B_t[n]
 *   ddlt_t      = sum_n lambda_t[n] (A[n] abar_t[n] h_{t-1}[n] + B_t[n] u_t)
 *   ddelta_t    = ddlt_t * sigmoid(v_t) with softplus, ddlt_t without; dbias += ddelta_t
 *   dA[n]      += lambda_t[n] dlt_t abar_t[n] h_{t-1}[n];  dDskip += ds_t u_t
 *   dh0[n]      = abar_0[n] lambda_0[n]
 *
 * Parity pinned by tests/test_oracle_pins.py (brute-force materialisation on
 * the time grid t_k = sum Delta, geometric closed form, B = 0, split
 * invariance, the eq. (4) gated-recurrence special case, the associative
 * tuple scan, N-separability, linearity, step == forward, the Delta limits,
 * states at positions against the time-grid closed form of every state).
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define MBO_MAX_N 256

#define MBO_OK 0
#define MBO_ERR_ARG (-1)

static double softplus(double v)
{
    /* log(1 + exp(v)), written so that neither exp overflows nor the log
     * loses the small argument: max(v, 0) + log1p(exp(-|v|)). */
    return fmax(v, 0.0) + log1p(exp(-fabs(v)));
}

static double silu(double z)
{
    /* z * sigmoid(z), the Swish gate of Fig. 5. */
    return z / (1.0 + exp(-z));
}

/* Copy the state after timestep t (t = -1: before the first step) into every
 * slot k whose requested position is t; when t = -1 also mark the slots whose
 * position lies outside [-1, L-1] with NaN. */
static void record_states(int64_t t, int64_t L, int64_t N, const double *h,
                          const int64_t *pos, int64_t P, double *out)
{
    for (int64_t k = 0; k < P; ++k) {
        if (pos[k] == t) {
            for (int64_t n = 0; n < N; ++n)
                out[k * N + n] = h[n];
        } else if (t == -1 && (pos[k] < -1 || pos[k] >= L)) {
            for (int64_t n = 0; n < N; ++n)
                out[k * N + n] = NAN;
        }
    }
}

static void scan_one_row(int64_t r, int64_t L, int64_t N, int delta_softplus,
                         const double *u, const double *delta, const double *z,
                         const double *A, const double *Dskip, const double *dt_bias,
                         const double *h0, const int64_t *bidx,
                         const double *Bm, const double *Cm,
                         double *y, double *h_last,
                         const int64_t *pos, int64_t P, double *h_pos)
{
    double h[MBO_MAX_N];
    const int64_t b = bidx[r];
    for (int64_t n = 0; n < N; ++n)
        h[n] = h0 ? h0[r * N + n] : 0.0;
    const int64_t *row_pos = P > 0 ? pos + r * P : NULL;
    double *row_out = P > 0 ? h_pos + r * P * N : NULL;
    record_states(-1, L, N, h, row_pos, P, row_out);

    for (int64_t t = 0; t < L; ++t) {
        const double x = u[r * L + t];
        double v = delta[r * L + t] + (dt_bias ? dt_bias[r] : 0.0);
        const double dlt = delta_softplus ? softplus(v) : v;
        double acc = 0.0;
        for (int64_t n = 0; n < N; ++n) {
            const double abar = exp(dlt * A[r * N + n]);
            const double bbar_x = (dlt * Bm[(b * N + n) * L + t]) * x;
            h[n] = abar * h[n] + bbar_x;
            acc += Cm[(b * N + n) * L + t] * h[n];
        }
        const double yv = acc + (Dskip ? Dskip[r] * x : 0.0);
        y[r * L + t] = z ? yv * silu(z[r * L + t]) : yv;
        record_states(t, L, N, h, row_pos, P, row_out);
    }
    if (h_last)
        for (int64_t n = 0; n < N; ++n)
            h_last[r * N + n] = h[n];
}

/*
 * Forward scan over R independent rows of length L.
 *   u, delta, z : R x L     (z may be NULL: no gate)
 *   A           : R x N     (the per-channel diagonal of A for each row)
 *   Dskip       : R         (may be NULL: no skip term)
 *   dt_bias     : R         (may be NULL: no bias)
 *   h0          : R x N     (may be NULL: zero initial state)
 *   bidx        : R         (batch element of each row, 0 <= bidx[r] < nbatch)
 *   Bm, Cm      : nbatch x N x L
 *   y           : R x L     (output)
 *   h_last      : R x N     (output, may be NULL)
 *   pos         : R x P     (requested positions of each row, may be NULL when P = 0)
 *   h_pos       : R x P x N (output: the state at each requested position)
 * Returns 0, or -1 on a bad argument (nothing written).
 */
int mbo_scan_rows_states(int64_t R, int64_t L, int64_t N, int delta_softplus,
                         const double *u, const double *delta, const double *z,
                         const double *A, const double *Dskip, const double *dt_bias,
                         const double *h0, const int64_t *bidx, int64_t nbatch,
                         const double *Bm, const double *Cm,
                         double *y, double *h_last,
                         const int64_t *pos, int64_t P, double *h_pos)
{
    if (R < 0 || L < 0 || N < 1 || N > MBO_MAX_N || nbatch < 1 || P < 0)
        return MBO_ERR_ARG;
    if (R == 0)
        return MBO_OK;
    if (!u || !delta || !A || !bidx || !Bm || !Cm || (!y && L > 0))
        return MBO_ERR_ARG;
    if (P > 0 && (!pos || !h_pos))
        return MBO_ERR_ARG;
    for (int64_t r = 0; r < R; ++r)
        if (bidx[r] < 0 || bidx[r] >= nbatch)
            return MBO_ERR_ARG;

#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t r = 0; r < R; ++r)
        scan_one_row(r, L, N, delta_softplus, u, delta, z, A, Dskip, dt_bias,
                     h0, bidx, Bm, Cm, y, h_last, pos, P, h_pos);
    return MBO_OK;
}

/* The forward scan without recorded positions. */
int mbo_scan_rows(int64_t R, int64_t L, int64_t N, int delta_softplus,
                  const double *u, const double *delta, const double *z,
                  const double *A, const double *Dskip, const double *dt_bias,
                  const double *h0, const int64_t *bidx, int64_t nbatch,
                  const double *Bm, const double *Cm,
                  double *y, double *h_last)
{
    return mbo_scan_rows_states(R, L, N, delta_softplus, u, delta, z, A, Dskip, dt_bias,
                                h0, bidx, nbatch, Bm, Cm, y, h_last, NULL, 0, NULL);
}

/*
 * One recurrent step for R rows, h updated in place.
 *   u_t, delta_t, z_t : R       (z_t may be NULL)
 *   A                 : R x N
 *   Dskip, dt_bias    : R       (may be NULL)
 *   bidx              : R
 *   B_t, C_t          : nbatch x N
 *   h                 : R x N   (in/out)
 *   y_t               : R       (output)
 * This is the forward scan with L = 1, h0 = h and h_last = h.
 */
int mbo_scan_step(int64_t R, int64_t N, int delta_softplus,
                  const double *u_t, const double *delta_t, const double *z_t,
                  const double *A, const double *Dskip, const double *dt_bias,
                  const int64_t *bidx, int64_t nbatch,
                  const double *B_t, const double *C_t,
                  double *h, double *y_t)
{
    if (R < 0 || N < 1 || N > MBO_MAX_N || nbatch < 1)
        return MBO_ERR_ARG;
    if (R == 0)
        return MBO_OK;
    if (!u_t || !delta_t || !A || !bidx || !B_t || !C_t || !h || !y_t)
        return MBO_ERR_ARG;
    for (int64_t r = 0; r < R; ++r)
        if (bidx[r] < 0 || bidx[r] >= nbatch)
            return MBO_ERR_ARG;

    for (int64_t r = 0; r < R; ++r) {
        /* B_t and C_t are (nbatch, N): the L = 1 case of the (nbatch, N, L) layout. */
        scan_one_row(r, 1, N, delta_softplus, u_t, delta_t, z_t, A, Dskip, dt_bias,
                     h, bidx, B_t, C_t, y_t, h, NULL, 0, NULL);
    }
    return MBO_OK;
}

/* ---- the backward of the scan ---------------------------------------------- */

static double sigmoid(double v)
{
    return 1.0 / (1.0 + exp(-v));
}

/* Per-row outputs (du, ddelta, dz, dA_row, dD_row, dbias_row, dh0) are written;
 * dB and dC (nbatch x N x L) are accumulated into the calling thread's buffers. */
static void bwd_one_row(int64_t r, int64_t L, int64_t N, int delta_softplus,
                        const double *u, const double *delta, const double *z,
                        const double *A, const double *Dskip, const double *dt_bias,
                        const double *h0, const int64_t *bidx,
                        const double *Bm, const double *Cm,
                        const double *dy, const double *dh_last,
                        double *du, double *ddelta, double *dz, double *dA, double *dD,
                        double *dbias, double *dh0, double *dB, double *dC)
{
    const int64_t b = bidx[r];
    /* forward, keeping every state (hs[t + 1] = h_t, hs[0] = h_{-1}) */
    double *hs = malloc(sizeof(double) * (size_t)(L + 1) * (size_t)N);
    double *dl = malloc(sizeof(double) * (size_t)(L > 0 ? L : 1));
    double *sv = malloc(sizeof(double) * (size_t)(L > 0 ? L : 1));
    for (int64_t n = 0; n < N; ++n)
        hs[n] = h0 ? h0[r * N + n] : 0.0;
    for (int64_t t = 0; t < L; ++t) {
        const double x = u[r * L + t];
        const double v = delta[r * L + t] + (dt_bias ? dt_bias[r] : 0.0);
        dl[t] = delta_softplus ? softplus(v) : v;
        double acc = Dskip ? Dskip[r] * x : 0.0;
        for (int64_t n = 0; n < N; ++n) {
            const double ab = exp(dl[t] * A[r * N + n]);
            hs[(t + 1) * N + n] = ab * hs[t * N + n] + (dl[t] * Bm[(b * N + n) * L + t]) * x;
            acc += Cm[(b * N + n) * L + t] * hs[(t + 1) * N + n];
        }
        sv[t] = acc;
    }
    /* reverse */
    double lam_next[MBO_MAX_N];      /* abar_{t+1} lambda_{t+1}: the gradient reaching h_t through h_{t+1} */
    for (int64_t n = 0; n < N; ++n) {
        lam_next[n] = dh_last ? dh_last[r * N + n] : 0.0;
        dA[r * N + n] = 0.0;
    }
    double sum_dD = 0.0, sum_dbias = 0.0;
    for (int64_t t = L - 1; t >= 0; --t) {
        const double x = u[r * L + t];
        const double g = z ? silu(z[r * L + t]) : 1.0;
        const double ds = dy[r * L + t] * g;
        if (z) {
            const double zz = z[r * L + t], sg = sigmoid(zz);
            dz[r * L + t] = dy[r * L + t] * sv[t] * sg * (1.0 + zz * (1.0 - sg));
        }
        sum_dD += ds * x;
        double dut = ds * (Dskip ? Dskip[r] : 0.0);
        double ddl = 0.0;
        for (int64_t n = 0; n < N; ++n) {
            const double Bv = Bm[(b * N + n) * L + t], Cv = Cm[(b * N + n) * L + t];
            const double ab = exp(dl[t] * A[r * N + n]);
            const double hprev = hs[t * N + n], hcur = hs[(t + 1) * N + n];
            const double lam = ds * Cv + lam_next[n];
            dC[(b * N + n) * L + t] += ds * hcur;
            dB[(b * N + n) * L + t] += lam * dl[t] * x;
            dut += lam * dl[t] * Bv;
            ddl += lam * (A[r * N + n] * ab * hprev + Bv * x);
            dA[r * N + n] += lam * dl[t] * ab * hprev;
            lam_next[n] = lam * ab;
        }
        du[r * L + t] = dut;
        const double v = delta[r * L + t] + (dt_bias ? dt_bias[r] : 0.0);
        const double dv = delta_softplus ? ddl * sigmoid(v) : ddl;
        ddelta[r * L + t] = dv;
        sum_dbias += dv;
    }
    dD[r] = sum_dD;
    dbias[r] = sum_dbias;
    if (dh0)
        for (int64_t n = 0; n < N; ++n)
            dh0[r * N + n] = lam_next[n];
    free(hs);
    free(dl);
    free(sv);
}

/*
 * Backward over R rows.  Inputs as for mbo_scan_rows, plus
 *   dy        : R x L       gradient of the loss with respect to y
 *   dh_last   : R x N       gradient with respect to h_last (may be NULL: zero)
 * Outputs
 *   du, ddelta: R x L;  dz: R x L (may be NULL when z is NULL)
 *   dA        : R x N       per row (the caller sums the rows of a channel)
 *   dD, dbias : R           per row (idem)
 *   dh0       : R x N       (may be NULL)
 *   dB, dC    : nbatch x N x L, overwritten with the sums over the rows of each batch element
 */
int mbo_scan_bwd_rows(int64_t R, int64_t L, int64_t N, int delta_softplus,
                      const double *u, const double *delta, const double *z,
                      const double *A, const double *Dskip, const double *dt_bias,
                      const double *h0, const int64_t *bidx, int64_t nbatch,
                      const double *Bm, const double *Cm,
                      const double *dy, const double *dh_last,
                      double *du, double *ddelta, double *dz, double *dA, double *dD,
                      double *dbias, double *dh0, double *dB, double *dC)
{
    if (R < 0 || L < 0 || N < 1 || N > MBO_MAX_N || nbatch < 1)
        return MBO_ERR_ARG;
    if (!u || !delta || !A || !bidx || !Bm || !Cm || !dy || !du || !ddelta || !dA || !dD || !dbias ||
        !dB || !dC || (z && !dz))
        return MBO_ERR_ARG;
    for (int64_t r = 0; r < R; ++r)
        if (bidx[r] < 0 || bidx[r] >= nbatch)
            return MBO_ERR_ARG;
    const int64_t nbc = nbatch * N * L;
    for (int64_t i = 0; i < nbc; ++i) {
        dB[i] = 0.0;
        dC[i] = 0.0;
    }
    /* each thread sums its rows' dB / dC into buffers of its own, merged at the end */
#pragma omp parallel
    {
        double *myB = calloc((size_t)(nbc > 0 ? nbc : 1), sizeof(double));
        double *myC = calloc((size_t)(nbc > 0 ? nbc : 1), sizeof(double));
#pragma omp for schedule(dynamic, 1)
        for (int64_t r = 0; r < R; ++r)
            bwd_one_row(r, L, N, delta_softplus, u, delta, z, A, Dskip, dt_bias, h0, bidx, Bm, Cm,
                        dy, dh_last, du, ddelta, dz, dA, dD, dbias, dh0, myB, myC);
#pragma omp critical
        for (int64_t i = 0; i < nbc; ++i) {
            dB[i] += myB[i];
            dC[i] += myC[i];
        }
        free(myB);
        free(myC);
    }
    return MBO_OK;
}

/* ---- the causal depthwise convolution ------------------------------------ */

#define MBO_MAX_K 64

static void conv_one_row(int64_t r, int64_t L, int64_t K, int apply_silu,
                         const double *x, const double *w, const double *bias,
                         const double *state_in, double *y, double *state_out)
{
    /* xin(s) for s in [-(K-1), L): the carried inputs, then this row's inputs */
    const int64_t H = K - 1;
    for (int64_t t = 0; t < L; ++t) {
        double pre = bias ? bias[r] : 0.0;
        for (int64_t i = 0; i < K; ++i) {
            const int64_t src = t - H + i;
            double xv;
            if (src >= 0)
                xv = x[r * L + src];
            else
                xv = state_in ? state_in[r * H + (H + src)] : 0.0;
            pre += w[r * K + i] * xv;
        }
        y[r * L + t] = apply_silu ? silu(pre) : pre;
    }
    if (state_out) {
        for (int64_t j = 0; j < H; ++j) {
            const int64_t src = L - H + j;
            state_out[r * H + j] = src >= 0 ? x[r * L + src]
                                            : (state_in ? state_in[r * H + (H + src)] : 0.0);
        }
    }
}

/*
 * Convolution over R independent rows of length L.
 *   x          : R x L       (input)
 *   w          : R x K       (taps of each row's channel; w[.][K-1] multiplies the current input)
 *   bias       : R           (may be NULL)
 *   state_in   : R x (K-1)   (the K-1 inputs before x, oldest first; may be NULL: zeros)
 *   y          : R x L       (output)
 *   state_out  : R x (K-1)   (output, may be NULL: the last K-1 inputs)
 */
int mbo_conv1d_rows(int64_t R, int64_t L, int64_t K, int apply_silu,
                    const double *x, const double *w, const double *bias,
                    const double *state_in, double *y, double *state_out)
{
    if (R < 0 || L < 0 || K < 1 || K > MBO_MAX_K)
        return MBO_ERR_ARG;
    if (R == 0)
        return MBO_OK;
    if (!w || (L > 0 && (!x || !y)))
        return MBO_ERR_ARG;
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t r = 0; r < R; ++r)
        conv_one_row(r, L, K, apply_silu, x, w, bias, state_in, y, state_out);
    return MBO_OK;
}

/* One step: the convolution with L = 1, the state updated in place. */
int mbo_conv1d_step(int64_t R, int64_t K, int apply_silu, const double *x_t,
                    const double *w, const double *bias, double *state, double *y_t)
{
    if (R < 0 || K < 1 || K > MBO_MAX_K)
        return MBO_ERR_ARG;
    if (R == 0)
        return MBO_OK;
    if (!x_t || !w || !y_t || (K > 1 && !state))
        return MBO_ERR_ARG;
    for (int64_t r = 0; r < R; ++r) {
        /* row r seen as row 0 of one-row arrays, so that the new state can go
         * to a local buffer before it replaces the old one */
        double next[MBO_MAX_K];
        double *st = K > 1 ? state + r * (K - 1) : NULL;
        conv_one_row(0, 1, K, apply_silu, x_t + r, w + r * K, bias ? bias + r : NULL, st,
                     y_t + r, next);
        for (int64_t j = 0; j < K - 1; ++j)
            st[j] = next[j];
    }
    return MBO_OK;
}

/* Threads the row loop runs on (reported next to the oracle's timing). */
int mbo_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Set the number of threads later row loops use (the single-threaded timing). */
void mbo_set_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}
