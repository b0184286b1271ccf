// scan_step.hpp -- one recurrent step (generation mode), state updated in place.
//
// Four lanes share a (batch, channel) row, each holding N/4 of its states, so
// that the fp32 state (the dominant traffic: 2 x 64 B per row) moves as
// coalesced 16-byte accesses; the partial outputs are summed across the four
// lanes with cross-lane shuffles.
#pragma once

#include "device_math.hpp"
#include "scan_params.hpp"

namespace mbs {

template <int IN, int OUT, int N>
__global__ __launch_bounds__(256) void scan_step_kernel(StepParams p) {
    constexpr int LANES = N >= 4 ? 4 : 1;      // lanes per row
    constexpr int S = N / LANES;               // states per lane
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t rows = p.batch * p.dim;
    const int64_t row = gid / LANES;
    const int part = (int)(gid - row * LANES);
    const bool live = row < rows;
    const int64_t r = live ? row : 0;           // dead lanes still take part in the shuffles
    const int64_t b = r / p.dim;
    const int64_t d = r - b * p.dim;

    const float x = Act<IN>::ld(p.u, r);
    const float v = Act<IN>::ld(p.delta, r) + (p.dt_bias ? p.dt_bias[d] : 0.0f);
    const float dlt = p.delta_softplus ? softplus_f32(v) : v;
    const float dx = dlt * x;

    float acc = 0.0f;
    float hs[S];
#pragma unroll
    for (int s = 0; s < S; ++s) {
        const int n = part * S + s;
        const float abar = hw_exp2(dlt * (p.A[d * N + n] * kLog2e));
        const float bx = dx * Act<IN>::ld(p.Bt, b * N + n);
        hs[s] = __builtin_fmaf(abar, p.h[r * N + n], bx);
        acc = __builtin_fmaf(Act<IN>::ld(p.Ct, b * N + n), hs[s], acc);
    }
    if (LANES == 4) {
        acc += __shfl_xor(acc, 1, 4);
        acc += __shfl_xor(acc, 2, 4);
    }
    if (!live) return;
#pragma unroll
    for (int s = 0; s < S; ++s) p.h[r * N + part * S + s] = hs[s];
    if (part == 0) {
        float yv = __builtin_fmaf(p.Dskip ? p.Dskip[d] : 0.0f, x, acc);
        if (p.z) yv *= silu_f32(Act<IN>::ld(p.z, r));
        st_out<OUT>(p.y, r, yv);
    }
}

}  // namespace mbs
