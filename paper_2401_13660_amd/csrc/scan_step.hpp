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

// Launch: 256-thread blocks, grid.x = ceil(dim / (256 / lanes)) channel blocks,
// grid.y = min(batch, 65535); each block steps its channels for batch elements
// blockIdx.y, blockIdx.y + gridDim.y, ...  No thread divides: the channel and the
// lane's share of the states come from the thread index by shifts.
template <int N> constexpr int kStepLanes = N >= 4 ? 4 : 1;      // lanes per row
template <int N> constexpr int kStepRowsPerBlock = 256 / kStepLanes<N>;

template <int IN, int OUT, int N>
__global__ __launch_bounds__(256) void scan_step_kernel(StepParams p) {
    constexpr int LANES = kStepLanes<N>;
    constexpr int S = N / LANES;               // states per lane
    const int tid = threadIdx.x;
    const int part = tid % LANES;
    const int64_t d = (int64_t)blockIdx.x * kStepRowsPerBlock<N> + tid / LANES;
    const bool dlive = d < p.dim;
    const int64_t dc = dlive ? d : 0;          // dead lanes still take part in the shuffles
    for (int64_t b = blockIdx.y; b < p.batch; b += gridDim.y) {
        const int64_t r = b * p.dim + dc;
        // Every load is issued before the first use of any of them, so that a
        // step costs one round trip to memory instead of several (activations,
        // state, gate and the per-channel operands).  The per-channel operands
        // are loaded inside the loop, after the state, for that reason: loaded
        // (and scaled) before it, the compiler waited for them before issuing
        // the loop's loads.  An absent gate reads u instead, an absent bias or
        // skip reads A, each discarded.  The lanes of a row read the same
        // activation words.
        float hs[S], bv[S], cv[S], ar[S];
#pragma unroll
        for (int s = 0; s < S; ++s) {
            const int n = part * S + s;
            hs[s] = p.h[r * N + n];
            bv[s] = Act<IN>::ld(p.Bt, b * N + n);
            cv[s] = Act<IN>::ld(p.Ct, b * N + n);
        }
        const float x = Act<IN>::ld(p.u, r);
        const float draw = Act<IN>::ld(p.delta, r);
        const float z_raw = Act<IN>::ld(p.z ? p.z : p.u, r);
#pragma unroll
        for (int s = 0; s < S; ++s) ar[s] = p.A[dc * N + part * S + s];
        const float bias_raw = (p.dt_bias ? p.dt_bias : p.A)[dc];
        const float dskip_raw = (p.Dskip ? p.Dskip : p.A)[dc];
        const float bias = p.dt_bias ? bias_raw : 0.0f;
        const float dskip = p.Dskip ? dskip_raw : 0.0f;
        const float v = draw + bias;
        const float dlt = p.delta_softplus ? softplus_f32(v) : v;
        const float dx = dlt * x;
        float acc = 0.0f;
#pragma unroll
        for (int s = 0; s < S; ++s) {
            const float abar = hw_exp2(dlt * (ar[s] * kLog2e));
            hs[s] = __builtin_fmaf(abar, hs[s], dx * bv[s]);
            acc = __builtin_fmaf(cv[s], hs[s], acc);
        }
        if (LANES == 4) {
            acc += __shfl_xor(acc, 1, 4);
            acc += __shfl_xor(acc, 2, 4);
        }
        if (dlive) {
#pragma unroll
            for (int s = 0; s < S; ++s) p.h[r * N + part * S + s] = hs[s];
            if (part == 0) {
                float yv = __builtin_fmaf(dskip, x, acc);
                if (p.z) yv *= silu_f32(z_raw);
                st_out<OUT>(p.y, r, yv);
            }
        }
    }
}

}  // namespace mbs
