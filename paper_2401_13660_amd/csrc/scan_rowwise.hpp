// scan_rowwise.hpp -- the plain forward scan: one thread per (batch, channel) row.
//
// Each thread walks its row in time order, holding the N-state of eq. (2) in
// registers.  It is the fallback for shapes the tiled kernel does not take
// (dstate < 16, unaligned rows) and the baseline the tiled kernel is measured
// against; it is correct for every legal argument combination.
#pragma once

#include "device_math.hpp"
#include "scan_params.hpp"

namespace mbs {

template <int IN, int OUT, int N>
__global__ __launch_bounds__(64) void scan_fwd_rowwise(ScanParams p) {
    const int64_t row = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (row >= p.batch * p.dim) return;
    const int64_t b = row / p.dim;
    const int64_t d = row - b * p.dim;
    const int64_t L = p.seqlen;

    float a2[N], h[N];
#pragma unroll
    for (int n = 0; n < N; ++n) {
        a2[n] = p.A[d * N + n] * kLog2e;            // exp(dlt A) = 2^(dlt A log2 e)
        h[n] = p.h0 ? p.h0[row * N + n] : 0.0f;
    }
    const float dskip = p.Dskip ? p.Dskip[d] : 0.0f;
    const float bias = p.dt_bias ? p.dt_bias[d] : 0.0f;
    const int64_t base = row * L;
    const int64_t bc = b * N * L;

    for (int64_t t = 0; t < L; ++t) {
        const float x = Act<IN>::ld(p.u, base + t);
        const float v = Act<IN>::ld(p.delta, base + t) + bias;
        const float dlt = p.delta_softplus ? softplus_f32(v) : v;
        const float dx = dlt * x;
        float acc = 0.0f;
#pragma unroll
        for (int n = 0; n < N; ++n) {
            const float abar = hw_exp2(dlt * a2[n]);                         // ZOH on A
            const float bx = dx * Act<IN>::ld(p.Bm, bc + n * L + t);         // Euler on B
            h[n] = __builtin_fmaf(abar, h[n], bx);
            acc = __builtin_fmaf(Act<IN>::ld(p.Cm, bc + n * L + t), h[n], acc);
        }
        float yv = __builtin_fmaf(dskip, x, acc);
        if (p.z) yv *= silu_f32(Act<IN>::ld(p.z, base + t));
        st_out<OUT>(p.y, base + t, yv);
        for (int64_t k = 0; k < p.npos; ++k) {          // states at requested positions
            if (p.pos[k * p.batch + b] != t) continue;
            float *dst = p.h_pos + ((k * p.batch + b) * p.dim + d) * N;
#pragma unroll
            for (int n = 0; n < N; ++n) dst[n] = h[n];
        }
    }
    if (p.h_last) {
#pragma unroll
        for (int n = 0; n < N; ++n) p.h_last[row * N + n] = h[n];
    }
}

// The slots of h_pos the scan kernels do not write: position -1 is the state
// before the first timestep (h0, or zeros), and a position outside
// [-1, seqlen - 1] reads NaN.  One thread per (k, b, d, n).
__global__ void init_positions(ScanParams p, int64_t N) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t per_k = p.batch * p.dim * N;
    if (i >= p.npos * per_k) return;
    const int64_t k = i / per_k;
    const int64_t rest = i - k * per_k;                 // (b * dim + d) * N + n
    const int64_t b = rest / (p.dim * N);
    const int32_t pos = p.pos[k * p.batch + b];
    if (pos == -1) p.h_pos[i] = p.h0 ? p.h0[rest] : 0.0f;
    else if (pos < -1 || pos >= p.seqlen) p.h_pos[i] = __builtin_nanf("");
}

// seqlen == 0: the final state is the initial one.
__global__ void copy_state(const float *h0, float *h_last, int64_t count) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < count) h_last[i] = h0 ? h0[i] : 0.0f;
}

}  // namespace mbs
