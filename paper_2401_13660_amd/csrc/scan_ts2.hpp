// scan_ts2.hpp -- the forward selective scan with each chunk cut into two time
// slices inside the wave, for shapes with too few (batch, channel) rows to give
// every SIMD two waves of the plain tiled kernel (one wave issues at about half
// the rate two interleaved waves reach).
//
// A wave owns 4 channels of one batch element (half the channels of a plain
// wave, so twice the waves).  Lane l = 16 j + 2 q + k holds channel j's states
// 2q and 2q+1 for slice k of every 32-byte chunk: timesteps 16 k .. 16 k + 15.
// The associative operator of the parallel scan (Section 2, "Implementation")
// is applied between the two slices without materialising the pair aggregate:
//
//   A  per-element work as in the plain kernel: lane (j, q, k) takes channel j
//      at timesteps 16 k + 2q, 16 k + 2q + 1 and publishes (dlt, dx); the wave
//      stages the chunk's B and C rows, widened to fp32;
//   L  every lane computes abar = 2^(dlt A log2 e) and dx B for its slice and
//      keeps them (and C) in registers; the lanes of slice 0 also run the state
//      chain h = abar h + dx B from the state entering the chunk;
//   X  a DPP move within each lane pair hands slice 0's end state to slice 1;
//   T  every lane runs the chain from its slice's true entering state with the
//      kept factors (one FMA per state and step, no exponential) and forms the
//      partial contraction C_t[2q] h_t[2q] + C_t[2q+1] h_t[2q+1];
//   C  as in the plain kernel, through LDS: lane (j, q, k) sums the eight
//      partials of channel j at its own two timesteps, adds Dskip * u, applies
//      the gate and stores y.
//
// Each state h_t is produced by the same operations in the same order as in the
// plain kernel, so y and h_last are its bits exactly.  The cost over the plain
// kernel is the chain of slice 0 run twice (one FMA per state and step).
// Requires seqlen % 16 == 0 and 16-byte aligned activation rows, like the plain
// kernel; one time segment (the host uses the plain kernel otherwise).  With
// p.ck it also stores the backward's checkpoints, the state before every 16th
// timestep, which are the slices' entering states (the same bits as the plain
// kernel's checkpoints).
#pragma once

#include <hip/hip_runtime.h>

#include "device_math.hpp"
#include "scan_params.hpp"
#include "scan_tiled.hpp"

namespace mbs {
namespace ts2 {

using tiled::kN;
using tiled::kT;
using tiled::kWavesPerGroup;
using tiled::kThreads;
using tiled::Raw2;
using tiled::Raw4;
using tiled::lds_wait;

constexpr int kCh = 4;            // channels per wave
constexpr int kS = kT / 2;        // timesteps per slice

// Private LDS area of one wave, in 16-byte entries.  The pads follow the bank
// rules measured on gfx950 (lds_banks.hip: one dispatch per access pattern under
// the SQ_LDS_BANK_CONFLICT counter): a 16-byte write serves 8 consecutive lanes at
// a time from 32 banks of 4 bytes (a 128-byte period), an 8-byte read 32 lanes at
// a time from 64 banks (256 bytes).  In every write below, the 8 lanes of a group
// are 4 state pairs of both slices of one channel; in every read the two slices'
// entries fall in different banks.  Each access of the kernel, measured in that
// program, runs without a bank conflict.
//   dd    row r = chunk timesteps 2r, 2r+1 (slice k: rows 8k .. 8k+7) at 5 r
//         (+ 4 when r >= 8); entry j = (dlt, dx, dlt, dx) of channel j
//   bc    entry q of chunk timestep t at 9 t + q (+ 8 when t >= 16) =
//         (B[2q], B[2q+1], C[2q], C[2q+1])
//   part  row 8 j + 4 k + i = channel j, timesteps 16 k + 4 i .. + 3; entry q =
//         the partial output of state pair q (9 entries per row, 8 used)
struct WaveSmem {
    f32x4 dd[5 * (kT / 2) + 4];   // 1.3 KB
    f32x4 bc[9 * kT + 8];         // 4.6 KB
    f32x4 part[kCh * 8][9];       // 4.5 KB
};
// row c of slice k's dd rows (c < 8), and chunk timestep t or row c of slice k in bc
__device__ __forceinline__ int dd_at(int k, int c) { return (5 * kS / 2 + 4) * k + 5 * c; }
__device__ __forceinline__ int bc_at(int t) { return 9 * t + (t >= kS ? 8 : 0); }
__device__ __forceinline__ int bc_at(int k, int c) { return (9 * kS + 8) * k + 9 * c; }

// The value of lane l ^ 1 (a DPP quad permutation).
__device__ __forceinline__ float pair_swap(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xf, 0xf, false));
}

// CK = true: also store the backward's checkpoints in p.ck.
template <int IN, int OUT, bool GATE, bool SOFTPLUS, bool CK = false>
__global__ __launch_bounds__(kThreads) void scan_fwd_ts2(ScanParams p) {
    extern __shared__ __align__(16) unsigned char smem_raw[];
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    WaveSmem &sm = reinterpret_cast<WaveSmem *>(smem_raw)[wave];

    const int lane = threadIdx.x & 63;
    const int k = lane & 1;               // time slice
    const int q = (lane >> 1) & 7;        // state pair
    const int j = lane >> 4;              // channel within the wave
    const int jj = 2 * j + k;             // this lane's quad of B/C staging rows
    const uint32_t n_cg = (uint32_t)((p.dim + kCh - 1) / kCh);
    // workgroups renumbered so that each XCD (own L2) takes a contiguous range
    const uint32_t per_xcd = gridDim.x / 8;
    const uint32_t blk = blockIdx.x;
    const uint32_t lwg = blk < per_xcd * 8 ? (blk % 8) * per_xcd + blk / 8 : blk;
    const uint32_t wid = lwg * kWavesPerGroup + wave;
    if (wid >= n_cg * (uint32_t)p.batch) return;          // whole wave leaves together
    const uint32_t b32 = wid / n_cg;
    const int64_t cg = wid - b32 * n_cg;
    const int64_t b = b32;

    const int64_t d = cg * kCh + j;
    const bool live = d < p.dim;
    const int64_t dcl = live ? d : p.dim - 1;           // dead lanes read a valid row, never store
    const int64_t row = b * p.dim + dcl, rows = p.batch * p.dim;
    const int64_t L = p.seqlen;
    const int n0 = 2 * q;

    float a2[2], h[2];
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        a2[s] = p.A[dcl * kN + n0 + s] * kLog2e;
        h[s] = p.h0 ? p.h0[row * kN + n0 + s] : 0.0f;
    }
    const float dskip = p.Dskip ? p.Dskip[dcl] : 0.0f;
    const float bias = p.dt_bias ? p.dt_bias[dcl] : 0.0f;

    constexpr int kEl = IN == 1 ? 2 : 4;
    const int64_t act0 = (b * p.dim + cg * kCh) * L;                 // wave-uniform
    const int64_t bc0 = b * kN * L;
    const char *ub = static_cast<const char *>(p.u) + act0 * kEl;
    const char *db = static_cast<const char *>(p.delta) + act0 * kEl;
    const char *zb = GATE ? static_cast<const char *>(p.z) + act0 * kEl : nullptr;
    const char *bb = static_cast<const char *>(p.Bm) + bc0 * kEl;
    const char *cb = static_cast<const char *>(p.Cm) + bc0 * kEl;
    char *yb = static_cast<char *>(p.y) + act0 * (OUT == 1 ? 2 : 4);
    const uint32_t seq_n = (uint32_t)L;                              // a multiple of 16
    const uint32_t act_row = (uint32_t)((dcl - cg * kCh) * L);
    const int t_a = kS * k + 2 * q;                 // phase A / C timesteps t_a, t_a + 1 of a chunk
    const uint32_t bc_row = (uint32_t)(2 * q * L);  // B/C staging: rows 2q, 2q+1 at timesteps 4 jj ..

    struct Slot { Raw2<IN> u, dl, z; Raw4<IN> B0, B1, C0, C1; };
    Slot s0, s1;
    // Loads never branch: past the end a lane reads the last valid pair or quad
    // again (those values are never stored).
    auto issue_loads = [&](Slot &sl, uint32_t t0) {
        const uint32_t ta = t0 + t_a < seq_n - 2 ? t0 + t_a : seq_n - 2;
        const uint32_t oa = act_row + ta;
        sl.u.load(ub, oa);
        sl.dl.load(db, oa);
        if (GATE) sl.z.load(zb, oa);
        const uint32_t tb = t0 + 4 * jj < seq_n - 4 ? t0 + 4 * jj : seq_n - 4;
        const uint32_t ob = bc_row + tb;
        sl.B0.load(bb, ob);
        sl.B1.load(bb, ob + (uint32_t)L);
        sl.C0.load(cb, ob);
        sl.C1.load(cb, ob + (uint32_t)L);
    };

    auto wave_sync = [] {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    };

    // Pass L, step TQ: slice timesteps 4 TQ .. 4 TQ + 3.
    float ab[kS][2], bx[kS][2], cc[kS][2];
    float hl[2];
    auto loadL = [&](f32x4 (&ddv)[2], f32x4 (&bcv)[4], auto tq_c) {
        constexpr int TQ = decltype(tq_c)::value;
#pragma unroll
        for (int i = 0; i < 2; ++i) ddv[i] = sm.dd[dd_at(k, 2 * TQ + i) + j];
#pragma unroll
        for (int i = 0; i < 4; ++i) bcv[i] = sm.bc[bc_at(k, 4 * TQ + i) + q];
    };
    auto stepL = [&](const f32x4 (&ddv)[2], const f32x4 (&bcv)[4], auto tq_c) {
        constexpr int TQ = decltype(tq_c)::value;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int t = 4 * TQ + i;
            const float dl = (i & 1) ? ddv[i >> 1].z : ddv[i >> 1].x;
            const float dx = (i & 1) ? ddv[i >> 1].w : ddv[i >> 1].y;
            ab[t][0] = hw_exp2(dl * a2[0]);
            ab[t][1] = hw_exp2(dl * a2[1]);
            bx[t][0] = dx * bcv[i][0];
            bx[t][1] = dx * bcv[i][1];
            cc[t][0] = bcv[i][2];
            cc[t][1] = bcv[i][3];
            hl[0] = __builtin_fmaf(ab[t][0], hl[0], bx[t][0]);
            hl[1] = __builtin_fmaf(ab[t][1], hl[1], bx[t][1]);
        }
    };
    // Pass T, step TQ: the chain from the true entering state, and the partials.
    auto stepT = [&](float (&g)[2], auto tq_c) {
        constexpr int TQ = decltype(tq_c)::value;
        float acc4[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int t = 4 * TQ + i;
            g[0] = __builtin_fmaf(ab[t][0], g[0], bx[t][0]);
            g[1] = __builtin_fmaf(ab[t][1], g[1], bx[t][1]);
            acc4[i] = __builtin_fmaf(cc[t][1], g[1], cc[t][0] * g[0]);
        }
        sm.part[8 * j + 4 * k + TQ][q] = f32x4{acc4[0], acc4[1], acc4[2], acc4[3]};
    };

    auto chunk = [&](Slot &sl, uint32_t t0) {
        const int nt = seq_n - t0 < (uint32_t)kT ? (int)(seq_n - t0) : kT;       // 16 or 32

        // ---- A: per-element work of timesteps t_a, t_a + 1 and B/C staging
        float xs[2], gs[2];
        {
            float dl[2], dx[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const float x = sl.u.get(i);
                const float v = sl.dl.get(i) + bias;
                dl[i] = SOFTPLUS ? softplus_f32(v) : v;
                dx[i] = dl[i] * x;
                xs[i] = x;
                if (GATE) gs[i] = silu_f32(sl.z.get(i));
            }
            sm.dd[dd_at(k, q) + j] = f32x4{dl[0], dx[0], dl[1], dx[1]};
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
            sm.bc[bc_at(4 * jj + i) + q] = f32x4{sl.B0.get(i), sl.B1.get(i), sl.C0.get(i), sl.C1.get(i)};
        wave_sync();

        // refill this slot with the chunk after next while the recurrence runs
        issue_loads(sl, t0 + 2 * kT);

        // ---- L: the slice's factors; slice 0 also carries the chunk's state
        hl[0] = k ? 0.0f : h[0];
        hl[1] = k ? 0.0f : h[1];
        {
            f32x4 ddA[2], bcA[4], ddB[2], bcB[4];
            using I0 = std::integral_constant<int, 0>;
            using I1 = std::integral_constant<int, 1>;
            using I2 = std::integral_constant<int, 2>;
            using I3 = std::integral_constant<int, 3>;
            loadL(ddA, bcA, I0{});
            lds_wait<0>();
            loadL(ddB, bcB, I1{});
            stepL(ddA, bcA, I0{});
            lds_wait<0>();
            loadL(ddA, bcA, I2{});
            stepL(ddB, bcB, I1{});
            lds_wait<0>();
            loadL(ddB, bcB, I3{});
            stepL(ddA, bcA, I2{});
            lds_wait<0>();
            stepL(ddB, bcB, I3{});
        }

        // ---- X: slice 1 starts from slice 0's end state
        float g[2];
        {
            const float e0 = pair_swap(hl[0]), e1 = pair_swap(hl[1]);
            g[0] = k ? e0 : h[0];
            g[1] = k ? e1 : h[1];
        }
        // checkpoints for the backward: the states before timesteps t0 and t0 + 16
        // are the two slices' entering states
        if (CK && live && t0 + kS * k < seq_n)
            *reinterpret_cast<float2 *>(p.ck + (((int64_t)(t0 / kS) + k) * rows + row) * kN + n0) =
                float2{g[0], g[1]};

        // ---- T: the chain again from the true entering state, with the partials
        {
            using I0 = std::integral_constant<int, 0>;
            using I1 = std::integral_constant<int, 1>;
            using I2 = std::integral_constant<int, 2>;
            using I3 = std::integral_constant<int, 3>;
            stepT(g, I0{});
            stepT(g, I1{});
            stepT(g, I2{});
            stepT(g, I3{});
        }
        // the state leaving the chunk: slice 1's end, or slice 0's for a half chunk
        {
            const float f0 = pair_swap(g[0]), f1 = pair_swap(g[1]);
            const bool mine = (nt == kT) == (k == 1);
            h[0] = mine ? g[0] : f0;
            h[1] = mine ? g[1] : f1;
        }
        wave_sync();

        // ---- C: sum the 8 partials of channel j at timesteps t_a, t_a + 1
        {
            const float2 *src =
                reinterpret_cast<const float2 *>(&sm.part[8 * j + 4 * k + (q >> 1)][0]) + (q & 1);
            float2 acc = src[0];
#pragma unroll
            for (int w = 1; w < 8; ++w) {
                acc.x += src[2 * w].x;
                acc.y += src[2 * w].y;
            }
            float yv[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                float y = __builtin_fmaf(dskip, xs[i], i ? acc.y : acc.x);
                if (GATE) y *= gs[i];
                yv[i] = y;
            }
            if (live && t_a < nt) {
                const uint32_t oy = act_row + t0 + t_a;
                if (OUT == 0)
                    *reinterpret_cast<float2 *>(yb + oy * 4u) = float2{yv[0], yv[1]};
                else
                    *reinterpret_cast<uint32_t *>(yb + oy * 2u) = bf16x2_pack(yv[0], yv[1]);
            }
        }
        __builtin_amdgcn_wave_barrier();    // the tables are rewritten by the next chunk
    };

    issue_loads(s0, 0);
    issue_loads(s1, kT);
    uint32_t t0 = 0;
    for (; t0 + 2 * kT <= seq_n; t0 += 2 * kT) {      // pairs of full chunks
        chunk(s0, t0);
        chunk(s1, t0 + kT);
    }
    if (t0 < seq_n) chunk(s0, t0);                    // a full chunk and/or a half chunk remain
    if (t0 + kT < seq_n) chunk(s1, t0 + kT);

    if (p.h_last && live && k == 0) {
#pragma unroll
        for (int s = 0; s < 2; ++s) p.h_last[row * kN + n0 + s] = h[s];
    }
}

}  // namespace ts2
}  // namespace mbs

namespace mbs {
namespace ts2 {

// Whether the time-split kernel takes p: one time segment, no recorded states,
// at least one full chunk, and no more plain-kernel waves than SIMDs (where the
// plain kernel would leave every SIMD with one wave at most).  Checkpoints (p.ck)
// are the slices' entering states, stored after the hand-over.
inline bool takes(const ScanParams &p) {
    if (p.npos > 0 || p.seqlen < kT) return false;
    int64_t seg_len, pieces;
    if (tiled::fwd_segments(p, &seg_len, &pieces) != 1) return false;
    const int64_t plain_waves = (p.dim + tiled::kCh - 1) / tiled::kCh * p.batch;
    return plain_waves <= 4 * tiled::device_cus();
}

template <int IN, int OUT, bool GATE>
hipError_t fwd_ts2(ScanParams &p, void *stream) {
    const int64_t waves = (p.dim + kCh - 1) / kCh * p.batch;
    const int64_t blocks = (waves + kWavesPerGroup - 1) / kWavesPerGroup;
    void *args[] = {&p};
    const void *fn =
        p.ck ? (p.delta_softplus ? reinterpret_cast<const void *>(&scan_fwd_ts2<IN, OUT, GATE, true, true>)
                                 : reinterpret_cast<const void *>(&scan_fwd_ts2<IN, OUT, GATE, false, true>))
             : (p.delta_softplus ? reinterpret_cast<const void *>(&scan_fwd_ts2<IN, OUT, GATE, true>)
                                 : reinterpret_cast<const void *>(&scan_fwd_ts2<IN, OUT, GATE, false>));
    return hipLaunchKernel(fn, dim3((unsigned)blocks), dim3(kThreads), args, sizeof(WaveSmem) * kWavesPerGroup,
                           static_cast<hipStream_t>(stream));
}

}  // namespace ts2
}  // namespace mbs
