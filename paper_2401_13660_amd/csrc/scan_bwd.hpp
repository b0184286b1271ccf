// scan_bwd.hpp -- the backward of the selective scan (training, Section 4 and
// Appendix C: MambaByte is trained at 8,192-byte contexts), for dstate 16.
//
// With lambda_t[n] the gradient of the loss with respect to h_t[n], reverse-mode
// differentiation of eq. (2) with the discretisation of Appendix D and the
// output and gating rows of Table 8 gives
//
//   ds_t        = dy_t g_t,  g_t = silu(z_t) (1 without a gate);  dz_t = dy_t s_t silu'(z_t)
//   lambda_t[n] = ds_t C_t[n] + abar_{t+1}[n] lambda_{t+1}[n]        (+ dh_last at t = L-1)
//   dC_t[n]    += ds_t h_t[n],   dB_t[n] += lambda_t[n] dlt_t u_t    (summed over channels)
//   du_t        = ds_t Dskip + dlt_t sum_n lambda_t[n] B_t[n]
//   ddlt_t      = sum_n lambda_t[n] (A[n] abar_t[n] h_{t-1}[n] + u_t B_t[n]);  ddelta = ddlt sigma(v)
//   dA[n]      += dlt_t lambda_t[n] abar_t[n] h_{t-1}[n],  dDskip += ds_t u_t,  dbias += ddelta_t
//   dh0[n]      = abar_0[n] lambda_0[n]
//
// Three kernels:
//   scan_ckpt   forward recurrence (no output) storing h at the start of every
//               16-step chunk: ck[(chunk * rows + row) * 16 + n];
//   scan_bwd    the lanes of a wave own 8 channels x 16 states as in the forward
//               kernel (lane 8j + q: channel j, states 2q, 2q+1).  Chunks run in
//               reverse; per chunk: the per-element terms (A), the chunk's forward
//               from its checkpoint keeping h_t and abar_t in VGPRs (F), s_t and
//               dz (C1), the adjoint recurrence backwards (R), then du and ddelta
//               (C2).  dB and dC are summed over the wave's 8 channels in
//               registers (lane swaps) and written as one partial per wave;
//   bwd_finish  sums the dB / dC partials over channel groups and dA, dDskip,
//               dbias over the batch and the time segments (no atomics: results
//               are deterministic).
// With few (batch, channel) rows, time is cut into segments so that more waves
// share the chip: bwd_seg_aggregate runs the adjoint recurrence of every segment
// but the first from a zero carry (in pieces), and the wave of segment s starts
// from dh_last folded with the aggregates of the pieces after it.
#pragma once

#include <hip/hip_runtime.h>

#include "device_math.hpp"
#include "scan_params.hpp"

#include <type_traits>

namespace mbs {
namespace bwd {

constexpr int kN = 16;
constexpr int kCh = 8;                 // channels per wave
constexpr int kQ = 8;                  // lanes per channel
constexpr int kT = 16;                 // timesteps per chunk
constexpr int kWaves = 4;
constexpr int kThreads = kWaves * 64;

struct BwdParams {
    int64_t batch, dim, seqlen;
    const void *u, *delta, *Bm, *Cm, *z;
    const float *A, *Dskip, *dt_bias, *h0;
    const void *dy;
    const float *dh_last;
    void *du, *ddelta, *dz;            // (batch, dim, L), out dtype
    float *dh0;                        // (batch, dim, N) or null
    // workspace
    float *ck;                         // (L / 16, batch * dim, 16) checkpoints
    float *part_bc;                    // (ncg, batch, L, 8, 4): per wave, summed over its channels:
                                       // (dB[2q], dC[2q], dB[2q+1], dC[2q+1]) of state pair q
    float *part_row;                   // (nseg, batch * dim, 16 + 2): dA (16), dDskip, dbias per row
                                       // and time segment
    // Time segments (few rows): segment s covers [s seg_len, (s + 1) seg_len) of L.
    // Segments 1 .. nseg-1 are cut into agg_pieces pieces each, of seg_len /
    // agg_pieces timesteps (piece i of segment s is number (s - 1) agg_pieces + i;
    // pieces past L are empty).  agg[((i * rows + row) * 16 + n) * 2 + {0, 1}] =
    // (P, H) of piece i: the carry abar_{t_b} lambda_{t_b} it hands to the timestep
    // before it is P c + H, for the carry c = abar_{t_e} lambda_{t_e} that enters its
    // last timestep.
    // scan_ckpt's own segments, of ck_seg_len (>= L: none):
    // fagg[((s * rows + row) * 16 + n) * 2 + {0, 1}] = the forward aggregate (P, H)
    // of its segment s < nseg - 1 (the forward pre-pass's layout); it starts
    // segment s from h0 folded with those of segments 0 .. s-1.
    int64_t seg_len;
    int64_t agg_pieces;
    float *agg;
    int64_t ck_seg_len;
    const float *fagg;
    int delta_softplus;
};

// 2 consecutive activations (4 bytes bf16, 8 bytes fp32).
// Global addressing: a wave-uniform byte base (the wave's first row) plus a
// 32-bit lane offset in elements, so that loads and stores take the
// scalar-base form.  The host keeps L below 2^25, so 16 rows of 4-byte
// elements stay below 2^32 bytes.
template <int DT> constexpr uint32_t kElBytes = DT == 1 ? 2u : 4u;
template <int DT> __device__ __forceinline__ const char *wave_base(const void *p, int64_t el) {
    return static_cast<const char *>(p) + el * (int64_t)kElBytes<DT>;
}

template <int DT> struct Raw2;
template <> struct Raw2<1> {
    uint32_t v;
    __device__ __forceinline__ void load(const char *base, uint32_t off) {
        v = *reinterpret_cast<const uint32_t *>(base + off * 2u);
    }
    __device__ __forceinline__ float get(int i) const { return i ? bf16_hi(v) : bf16_lo(v); }
};
template <> struct Raw2<0> {
    float v0, v1;
    __device__ __forceinline__ void load(const char *base, uint32_t off) {
        const float *f = reinterpret_cast<const float *>(base + off * 4u);
        v0 = f[0];
        v1 = f[1];
    }
    __device__ __forceinline__ float get(int i) const { return i ? v1 : v0; }
};

template <int DT> __device__ __forceinline__ void store2(const char *base, uint32_t off, float a, float b) {
    char *at = const_cast<char *>(base) + off * kElBytes<DT>;
    if (DT == 0) {
        *reinterpret_cast<u32x2 *>(at) = u32x2{__builtin_bit_cast(uint32_t, a), __builtin_bit_cast(uint32_t, b)};
    } else {
        *reinterpret_cast<uint32_t *>(at) = bf16x2_pack(a, b);
    }
}

// Private LDS area of one wave (13.75 KB); padded rows spread reads and writes
// over the banks.  A 16-byte write serves 8 consecutive lanes (one channel) at a
// time from 32 banks (a 128-byte period, measured); lane q writes timesteps 2q and
// 2q + 1, so the dd rows are permuted (dd_row) to put those 8 writes in 8
// different bank quads.
__device__ __forceinline__ constexpr int dd_row(int t) { return (t >> 1) + (t & 1) * (kT / 2); }
struct WaveSmem {
    f32x4 dd[kT][kCh + 1];            // row dd_row(t): (dlt, dlt*u, ds, u) of timestep t, channel j
    f32x4 bc[kT][kQ + 2];             // (B[2q], B[2q+1], C[2q], C[2q+1]) of timestep t
    f32x4 pa[kCh * (kT / 4)][kQ + 1]; // per-state-pair partials, 4 timesteps per entry
    f32x4 pb[kCh * (kT / 4)][kQ + 1];
};

// softplus(v) (as softplus_f32) and its derivative sigmoid(v) from the one
// exponential e = e^-|v|: sigmoid(v) = 1 / (1 + e) for v >= 0, e / (1 + e) below.
__device__ __forceinline__ void softplus_and_sigmoid(float v, float &sp, float &sg) {
    const float e = hw_exp2(-__builtin_fabsf(v) * kLog2e);
    const float w = 1.0f + e;
    const float c = e - (w - 1.0f);
    sp = __builtin_fmaxf(v, 0.0f) + __builtin_fmaf(hw_log2(w), kLn2, c);
    sg = (v >= 0.0f ? 1.0f : e) * hw_rcp(w);
}

// The first two words of a 16-byte LDS entry, as one 8-byte read.  (Reading the
// whole entry when two words are used lets the compiler reuse the unused half of
// the destination for the next read, which then has to wait for this one.)
__device__ __forceinline__ float2 lo2(const f32x4 &e) { return *reinterpret_cast<const float2 *>(&e); }

__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Sum over the 8 state-pair lanes of channel j of the per-4-timestep partials in
// part[4j + t/4][lane][t%4], for the lane's own timesteps t = 2q and 2q + 1 (the
// two are adjacent in one entry, so each partial is one 8-byte read).
__device__ __forceinline__ void part_sum(const f32x4 (&part)[kCh * (kT / 4)][kQ + 1], int j, int q,
                                         float (&out)[2]) {
    const float *base = reinterpret_cast<const float *>(&part[4 * j + (q >> 1)][0]) + 2 * (q & 1);
    const float2 v0 = *reinterpret_cast<const float2 *>(base);
    float s0 = v0.x, s1 = v0.y;
#pragma unroll
    for (int w = 1; w < kQ; ++w) {
        const float2 v = *reinterpret_cast<const float2 *>(base + 4 * w);
        s0 += v.x;
        s1 += v.y;
    }
    out[0] = s0;
    out[1] = s1;
}

// Sums over lanes l and l + 32 of two values at once: lanes 0-31 receive a's,
// lanes 32-63 b's (v_permlane32_swap exchanges lanes 32-63 of its first
// operand with lanes 0-31 of its second).  The halves are copied to scalars
// before reinterpreting them.
__device__ __forceinline__ float half_swap_sum(float a, float b) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(a), __float_as_uint(b), false, false);
    const unsigned r0 = r[0], r1 = r[1];
    return __uint_as_float(r0) + __uint_as_float(r1);
}

// The same over lanes l and l ^ 16 (v_permlane16_swap exchanges the odd 16-lane
// rows of its first operand with the even rows of its second): even rows receive
// a's sum, odd rows b's.
__device__ __forceinline__ float row_swap_sum(float a, float b) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(a), __float_as_uint(b), false, false);
    const unsigned r0 = r[0], r1 = r[1];
    return __uint_as_float(r0) + __uint_as_float(r1);
}

// v + the value of lane l ^ 8 (a DPP rotation by 8 inside each 16-lane row).
__device__ __forceinline__ float add_xor8(float v) {
    return v + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x128, 0xf, 0xf, false));
}

// The wave's (batch, channel group) from a workgroup renumbered so that each of
// the 8 XCDs works on a contiguous range of groups.
__device__ __forceinline__ int64_t wave_id() {
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t per_xcd = (int64_t)gridDim.x / 8;
    const int64_t k = blockIdx.x;
    const int64_t lwg = k < per_xcd * 8 ? (k % 8) * per_xcd + k / 8 : k;
    return lwg * kWaves + wave;
}

// ---- the checkpoint pass ------------------------------------------------------
// Loads run two chunks ahead in two static register slots (clamped, never
// branched), as in the forward kernel.
template <int IN, bool SOFTPLUS>
__global__ __launch_bounds__(kThreads) void scan_ckpt(BwdParams p) {
    extern __shared__ __align__(16) unsigned char smem_raw[];
    WaveSmem &sm = reinterpret_cast<WaveSmem *>(smem_raw)[__builtin_amdgcn_readfirstlane(threadIdx.x >> 6)];
    const int lane = threadIdx.x & 63, j = lane >> 3, q = lane & 7, n0 = 2 * q;
    const int64_t n_cg = (p.dim + kCh - 1) / kCh, L = p.seqlen;
    const int64_t nseg = (L + p.ck_seg_len - 1) / p.ck_seg_len;
    const int64_t wid = wave_id();
    if (wid >= n_cg * p.batch * nseg) return;
    const int64_t cg = wid % n_cg, b = (wid / n_cg) % p.batch, seg = wid / (n_cg * p.batch);
    const int64_t t_begin = seg * p.ck_seg_len;
    const int64_t t_end = t_begin + p.ck_seg_len < L ? t_begin + p.ck_seg_len : L;
    const int64_t d = cg * kCh + j;
    const bool live = d < p.dim;
    const int64_t dcl = live ? d : p.dim - 1;
    const int64_t row = b * p.dim + dcl, rows = p.batch * p.dim;
    const float bias = p.dt_bias ? p.dt_bias[dcl] : 0.0f;
    float a2[2], h[2];
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        a2[s] = p.A[dcl * kN + n0 + s] * kLog2e;
        h[s] = p.h0 ? p.h0[row * kN + n0 + s] : 0.0f;
        for (int64_t s2 = 0; s2 < seg; ++s2) {           // carry-in of the earlier segments
            const float *f = p.fagg + ((s2 * rows + row) * kN + n0 + s) * 2;
            h[s] = __builtin_fmaf(f[0], h[s], f[1]);
        }
    }
    const int64_t row0 = b * p.dim + cg * kCh;          // the wave's first row
    const uint32_t lrow = (uint32_t)((dcl - cg * kCh) * L), brow = (uint32_t)(n0 * L);
    const uint32_t lck = (uint32_t)((dcl - cg * kCh) * kN + n0);
    const char *ub = wave_base<IN>(p.u, row0 * L), *db = wave_base<IN>(p.delta, row0 * L);
    const char *bb = wave_base<IN>(p.Bm, b * kN * L);

    // per element: lane (j, q) takes timesteps 2q, 2q+1; B staging: timesteps 2j, 2j+1
    struct Slot { Raw2<IN> u, dl, b0, b1; };
    auto issue = [&](Slot &sl, int64_t t0) {
        const uint32_t tc = (uint32_t)(t0 < t_end ? t0 : t_end - kT);   // past the end: reload the last chunk
        sl.u.load(ub, lrow + tc + 2 * q);
        sl.dl.load(db, lrow + tc + 2 * q);
        sl.b0.load(bb, brow + tc + 2 * j);
        sl.b1.load(bb, brow + (uint32_t)L + tc + 2 * j);
    };
    auto chunk = [&](Slot &sl, int64_t t0) {
#pragma unroll
        for (int k = 0; k < 2; ++k) {
            const float v = sl.dl.get(k) + bias;
            const float dl = SOFTPLUS ? softplus_f32(v) : v;
            sm.dd[dd_row(2 * q + k)][j] = f32x4{dl, dl * sl.u.get(k), 0.0f, 0.0f};
            sm.bc[2 * j + k][q] = f32x4{sl.b0.get(k), sl.b1.get(k), 0.0f, 0.0f};
        }
        issue(sl, t0 + 2 * kT);
        if (live)
            *reinterpret_cast<u32x2 *>(p.ck + ((t0 / kT) * rows + row0) * kN + lck) =
                u32x2{__builtin_bit_cast(uint32_t, h[0]), __builtin_bit_cast(uint32_t, h[1])};
        wave_sync();
#pragma unroll
        for (int tq = 0; tq < kT / 4; ++tq) {
            float2 dvs[4], bvs[4];                      // (dlt, dlt*u), (B0, B1) of 4 steps, read together
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                dvs[k] = lo2(sm.dd[dd_row(4 * tq + k)][j]);
                bvs[k] = lo2(sm.bc[4 * tq + k][q]);
            }
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                h[0] = __builtin_fmaf(hw_exp2(dvs[k].x * a2[0]), h[0], dvs[k].y * bvs[k].x);
                h[1] = __builtin_fmaf(hw_exp2(dvs[k].x * a2[1]), h[1], dvs[k].y * bvs[k].y);
            }
        }
        wave_sync();
    };
    Slot s0, s1;
    issue(s0, t_begin);
    issue(s1, t_begin + kT);
    int64_t t0 = t_begin;
    for (; t0 + 2 * kT <= t_end; t0 += 2 * kT) {
        chunk(s0, t0);
        chunk(s1, t0 + kT);
    }
    if (t0 < t_end) chunk(s0, t0);
}

// ---- the adjoint aggregate of a piece of a time segment -----------------------------
// The adjoint recurrence is linear in its carry: within [t_b, t_e),
// lambda_t = ds_t C_t + carry and the next carry is abar_t lambda_t, so the carry
// handed on, abar_{t_b} lambda_{t_b}, is P c + H for the carry c entering t_e - 1,
// with P = prod_t abar_t = 2^(A log2 e sum_t dlt_t) and H the carry from c = 0.
// (The associative operator of Section 2 applied to the adjoint, backwards.)
// Lanes own channel j, states 2q, 2q+1 as in scan_bwd; per 16-step chunk the
// wave stages (dlt, ds) and C, then runs the recurrence backwards.  One wave per
// piece and 8 channels: with few rows a whole segment per wave would leave a lone
// wave on a SIMD, which waits on its chain (two dependent operations per step),
// so the host cuts each segment into up to 4 pieces.
struct AggSmem {
    float2 dd[kT][kCh + 1];           // (dlt, ds) of timestep t, channel j
    float2 cc[kT][kQ + 1];            // (C[2q], C[2q+1]) at timestep t
};

template <int IN, int OUT, bool GATE, bool SOFTPLUS>
__global__ __launch_bounds__(kThreads) void bwd_seg_aggregate(BwdParams p) {
    extern __shared__ __align__(16) unsigned char smem_raw[];
    AggSmem &sm = reinterpret_cast<AggSmem *>(smem_raw)[__builtin_amdgcn_readfirstlane(threadIdx.x >> 6)];
    const int lane = threadIdx.x & 63, j = lane >> 3, q = lane & 7, n0 = 2 * q;
    const int64_t n_cg = (p.dim + kCh - 1) / kCh, L = p.seqlen;
    const int64_t nseg = (L + p.seg_len - 1) / p.seg_len;
    const int64_t npieces = p.agg_pieces * (nseg - 1), piece_len = p.seg_len / p.agg_pieces;
    const int64_t wid = wave_id();
    if (wid >= n_cg * p.batch * npieces) return;       // the pieces of segments 1 .. nseg-1
    const int64_t cg = wid % n_cg, b = (wid / n_cg) % p.batch, piece = wid / (n_cg * p.batch);
    const int64_t t_begin = p.seg_len + piece * piece_len;
    const int64_t t_end = t_begin + piece_len < L ? t_begin + piece_len : L;
    const int64_t d = cg * kCh + j;
    const bool live = d < p.dim;
    const int64_t dcl = live ? d : p.dim - 1;
    const int64_t row = b * p.dim + dcl, rows = p.batch * p.dim;
    if (t_begin >= L) {                                 // an empty piece of the last segment: (1, 0)
        if (live) {
#pragma unroll
            for (int s = 0; s < 2; ++s) {                 // (the planes are 8-byte aligned only)
                float *o = p.agg + ((piece * rows + row) * kN + n0 + s) * 2;
                o[0] = 1.0f;
                o[1] = 0.0f;
            }
        }
        return;
    }
    const float bias = p.dt_bias ? p.dt_bias[dcl] : 0.0f;
    float a2[2], carry[2] = {0.0f, 0.0f}, dsum = 0.0f;
#pragma unroll
    for (int s = 0; s < 2; ++s) a2[s] = p.A[dcl * kN + n0 + s] * kLog2e;
    const int64_t row0 = b * p.dim + cg * kCh;
    const uint32_t lrow = (uint32_t)((dcl - cg * kCh) * L), brow = (uint32_t)(n0 * L);
    const char *db = wave_base<IN>(p.delta, row0 * L);
    const char *zb = GATE ? wave_base<IN>(p.z, row0 * L) : nullptr;
    const char *cb = wave_base<IN>(p.Cm, b * kN * L);
    const char *dyb = wave_base<OUT>(p.dy, row0 * L);

    // per element: lane (j, q) takes timesteps 2q, 2q+1; C staging: timesteps 2j, 2j+1
    struct Slot { Raw2<IN> dl, z, c0, c1; Raw2<OUT> dy; };
    auto issue = [&](Slot &sl, int64_t t0) {                // clamped at the piece start
        const uint32_t tc = (uint32_t)(t0 >= t_begin ? t0 : t_begin);
        const uint32_t oa = lrow + tc + 2 * q, ob = brow + tc + 2 * j;
        sl.dl.load(db, oa);
        if (GATE) sl.z.load(zb, oa);
        sl.dy.load(dyb, oa);
        sl.c0.load(cb, ob);
        sl.c1.load(cb, ob + (uint32_t)L);
    };
    auto chunk = [&](Slot &sl, int64_t t0) {
#pragma unroll
        for (int k = 0; k < 2; ++k) {
            const float v = sl.dl.get(k) + bias;
            const float dl = SOFTPLUS ? softplus_f32(v) : v;
            const float g = GATE ? silu_f32(sl.z.get(k)) : 1.0f;
            dsum += dl;
            // a dead lane has ds = 0, so its carry stays exactly 0
            sm.dd[2 * q + k][j] = float2{dl, live ? sl.dy.get(k) * g : 0.0f};
            sm.cc[2 * j + k][q] = float2{sl.c0.get(k), sl.c1.get(k)};
        }
        wave_sync();
        issue(sl, t0 - 2 * kT);                          // the chunk two further back
#pragma unroll
        for (int t = kT - 1; t >= 0; --t) {
            const float2 dv = sm.dd[t][j];
            const float2 cv = sm.cc[t][q];
            const float lam0 = __builtin_fmaf(dv.y, cv.x, carry[0]);
            const float lam1 = __builtin_fmaf(dv.y, cv.y, carry[1]);
            carry[0] = hw_exp2(dv.x * a2[0]) * lam0;
            carry[1] = hw_exp2(dv.x * a2[1]) * lam1;
        }
        wave_sync();                                     // dd / cc are rewritten
    };

    Slot s0, s1;
    issue(s0, t_end - kT);
    issue(s1, t_end - 2 * kT);
    int64_t t0 = t_end - kT;
    for (; t0 - kT >= t_begin; t0 -= 2 * kT) {
        chunk(s0, t0);
        chunk(s1, t0 - kT);
    }
    if (t0 >= t_begin) chunk(s0, t0);

    dsum += __shfl_xor(dsum, 1);                         // the piece's sum of dlt for channel j
    dsum += __shfl_xor(dsum, 2);
    dsum += __shfl_xor(dsum, 4);
    if (live) {
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            float *o = p.agg + ((piece * rows + row) * kN + n0 + s) * 2;
            o[0] = hw_exp2(a2[s] * dsum);
            o[1] = carry[s];
        }
    }
}

// ---- the backward pass -----------------------------------------------------------
// Floats of the workgroup's dB/dC exchange area (WG = true): two buffers of
// 4 waves x 2 step pairs x 64 lanes.
constexpr int kWgXchg = 2 * kWaves * 2 * 64;

// WG = true (the number of 8-channel groups is a multiple of 4, so the 4 waves of
// a workgroup are 4 consecutive groups of one batch element): the waves also
// sum their dB/dC terms with each other through LDS every 4 steps, one barrier
// per 4 steps, and the workgroup writes one partial per 32 channels.
template <int IN, int OUT, bool GATE, bool SOFTPLUS, bool WG = false>
__global__ __launch_bounds__(kThreads, 2) void scan_bwd(BwdParams p) {     // 2 waves per SIMD: <= 256 VGPRs
    extern __shared__ __align__(16) unsigned char smem_raw[];
    __shared__ float wg_sums[WG ? kWgXchg : 1];         // WG: the workgroup's dB/dC exchange area
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    WaveSmem &sm = reinterpret_cast<WaveSmem *>(smem_raw)[wave];
    const int lane = threadIdx.x & 63, j = lane >> 3, q = lane & 7, n0 = 2 * q;
    const int64_t n_cg = (p.dim + kCh - 1) / kCh, L = p.seqlen;
    const int64_t nseg = (L + p.seg_len - 1) / p.seg_len;
    const int64_t wid = wave_id();
    if (wid >= n_cg * p.batch * nseg) return;
    const int64_t cg = wid % n_cg, b = (wid / n_cg) % p.batch, seg = wid / (n_cg * p.batch);
    const int64_t t_begin = seg * p.seg_len;
    const int64_t t_end = t_begin + p.seg_len < L ? t_begin + p.seg_len : L;
    const int64_t d = cg * kCh + j;
    const bool live = d < p.dim;
    const int64_t dcl = live ? d : p.dim - 1;
    const int64_t row = b * p.dim + dcl, rows = p.batch * p.dim;
    const float bias = p.dt_bias ? p.dt_bias[dcl] : 0.0f;
    const float dskip = p.Dskip ? p.Dskip[dcl] : 0.0f;
    float a2[2], Av[2], carry[2], dA[2] = {0.0f, 0.0f};
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        Av[s] = p.A[dcl * kN + n0 + s];
        a2[s] = Av[s] * kLog2e;
        carry[s] = (p.dh_last && live) ? p.dh_last[row * kN + n0 + s] : 0.0f;   // abar_{t+1} lambda_{t+1}
        // carry-in: fold the aggregates of the later segments' pieces, the last one first
        for (int64_t i = p.agg_pieces * (nseg - 1) - 1; i >= p.agg_pieces * seg; --i) {
            const float *a = p.agg + ((i * rows + row) * kN + n0 + s) * 2;
            carry[s] = live ? __builtin_fmaf(a[0], carry[s], a[1]) : 0.0f;
        }
    }
    float sum_dD = 0.0f, sum_dbias = 0.0f;
    const int64_t row0 = b * p.dim + cg * kCh;          // the wave's first row
    const uint32_t lrow = (uint32_t)((dcl - cg * kCh) * L), brow = (uint32_t)(n0 * L);
    const uint32_t lck = (uint32_t)((dcl - cg * kCh) * kN + n0);
    const char *ub = wave_base<IN>(p.u, row0 * L), *db = wave_base<IN>(p.delta, row0 * L);
    const char *zb = GATE ? wave_base<IN>(p.z, row0 * L) : nullptr;
    const char *bb = wave_base<IN>(p.Bm, b * kN * L), *cb = wave_base<IN>(p.Cm, b * kN * L);
    const char *dyb = wave_base<OUT>(p.dy, row0 * L);
    const char *dub = wave_base<OUT>(p.du, row0 * L), *ddb = wave_base<OUT>(p.ddelta, row0 * L);
    const char *dzb = GATE ? wave_base<OUT>(p.dz, row0 * L) : nullptr;
    float *pbc = p.part_bc + (((WG ? cg / kWaves : cg) * p.batch + b) * L) * (kQ * 4);
    int buf = 0;                                        // WG: the exchange buffer in use

    // Loads run two chunks ahead (in processing order: backwards in time) in two
    // static register slots, clamped at the segment start, never branched.
    struct Slot {
        Raw2<IN> u, dl, z, b0, b1, c0, c1;
        Raw2<OUT> dy;
        float ck0, ck1;
    };
    auto issue = [&](Slot &sl, int64_t t0) {
        const int64_t tc = t0 >= t_begin ? t0 : t_begin;
        const uint32_t oa = lrow + (uint32_t)tc + 2 * q, ob = brow + (uint32_t)tc + 2 * j;
        sl.u.load(ub, oa);
        sl.dl.load(db, oa);
        if (GATE) sl.z.load(zb, oa);
        sl.dy.load(dyb, oa);
        sl.b0.load(bb, ob);
        sl.b1.load(bb, ob + (uint32_t)L);
        sl.c0.load(cb, ob);
        sl.c1.load(cb, ob + (uint32_t)L);
        const float *ckp = p.ck + ((tc / kT) * rows + row0) * kN + lck;
        sl.ck0 = ckp[0];
        sl.ck1 = ckp[1];
    };

    auto chunk = [&](Slot &sl, int64_t t0) {
        // ---- A: per-element terms of timesteps 2q, 2q+1 and B/C staging ----------
        // A dead lane (channel beyond dim) starts from h = 0 with lambda = 0 and has
        // dlt*u = ds = 0, so every term it computes is exactly 0 and it adds nothing
        // to the dB / dC sums over channels.
        float hb[kT + 1][2], ab[kT][2];                 // h_{t-1} .. h_{t+15}; abar_t
        hb[0][0] = live ? sl.ck0 : 0.0f;
        hb[0][1] = live ? sl.ck1 : 0.0f;
        float xs[2], dyv[2], dsilu[2], sg[2], dlv[2], dsv[2];
#pragma unroll
        for (int k = 0; k < 2; ++k) {
            const float x = sl.u.get(k);
            const float v = sl.dl.get(k) + bias;
            float dl = v;
            sg[k] = 1.0f;
            if (SOFTPLUS) softplus_and_sigmoid(v, dl, sg[k]);          // softplus'(v) = sigmoid(v)
            dyv[k] = sl.dy.get(k);
            float g = 1.0f;
            if (GATE) {                                 // silu(z) and silu'(z) from one sigmoid
                const float z = sl.z.get(k);
                const float sz = hw_rcp(1.0f + hw_exp2(-z * kLog2e));
                g = z * sz;
                dsilu[k] = sz * __builtin_fmaf(z, 1.0f - sz, 1.0f);
            }
            const float ds = dyv[k] * g;
            xs[k] = x;
            dlv[k] = dl;
            dsv[k] = ds;
            sum_dD = __builtin_fmaf(ds, x, sum_dD);
            sm.dd[dd_row(2 * q + k)][j] = live ? f32x4{dl, dl * x, ds, x} : f32x4{dl, 0.0f, 0.0f, x};
            sm.bc[2 * j + k][q] = f32x4{sl.b0.get(k), sl.b1.get(k), sl.c0.get(k), sl.c1.get(k)};
        }
        issue(sl, t0 - 2 * kT);                         // refill with the chunk two further back
        wave_sync();

        // ---- F: the chunk's forward from its checkpoint -------------------------
#pragma unroll
        for (int tq = 0; tq < kT / 4; ++tq) {
            float acc[4];
            // the 4 steps' operands, read together; only the words used are read
            float2 dvs[4];                              // (dlt, dlt*u)
            f32x4 bvs[4];                               // (B0, B1, C0, C1); C only with a gate
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                dvs[k] = lo2(sm.dd[dd_row(4 * tq + k)][j]);
                if (GATE) {
                    bvs[k] = sm.bc[4 * tq + k][q];
                } else {
                    const float2 b2 = lo2(sm.bc[4 * tq + k][q]);
                    bvs[k] = f32x4{b2.x, b2.y, 0.0f, 0.0f};
                }
            }
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int t = 4 * tq + k;
                const float2 dv = dvs[k];
                const f32x4 bv = bvs[k];
#pragma unroll
                for (int s = 0; s < 2; ++s) {
                    ab[t][s] = hw_exp2(dv.x * a2[s]);
                    hb[t + 1][s] = __builtin_fmaf(ab[t][s], hb[t][s], dv.y * bv[s]);
                }
                if (GATE) acc[k] = __builtin_fmaf(bv.w, hb[t + 1][1], bv.z * hb[t + 1][0]);
            }
            if (GATE) sm.pa[4 * j + tq][q] = f32x4{acc[0], acc[1], acc[2], acc[3]};   // C . h, for dz
        }
        wave_sync();

        // ---- C1: s_t = C_t . h_t + Dskip u_t and dz for timesteps 2q, 2q+1 -------
        if (GATE) {
            float dzv[2], sp[2];
            part_sum(sm.pa, j, q, sp);
#pragma unroll
            for (int k = 0; k < 2; ++k) {
                const float s = __builtin_fmaf(dskip, xs[k], sp[k]);
                dzv[k] = dyv[k] * s * dsilu[k];
            }
            if (live) store2<OUT>(dzb, lrow + (uint32_t)t0 + 2 * q, dzv[0], dzv[1]);
        }
        wave_sync();                                    // pa is rewritten below

        // ---- R: the adjoint recurrence, timesteps 15 .. 0 -------------------------
        // The dB / dC terms of each step are summed over the wave's 8 channels in
        // registers: the channel bits 5, 4 and 3 of the lane meet in a 32-lane swap,
        // a 16-lane swap and a rotation by 8, after which lane (b5, b4, b3, q) holds
        // entry 2 b5 + b4 of state pair q's (dB[2q], dC[2q], dB[2q+1], dC[2q+1]),
        // the same for b3 = 0 and 1; lanes with b3 = 0 store the even step of a pair,
        // lanes with b3 = 1 the odd one.
        const int b3 = (lane >> 3) & 1;
        const uint32_t pl = ((uint32_t)t0 + b3) * (kQ * 4) + q * 4 + (((lane >> 5) << 1) | ((lane >> 4) & 1));
#pragma unroll
        for (int tq = kT / 4 - 1; tq >= 0; --tq) {
            float pu[4], pd[4], tot_hi = 0.0f;
            f32x4 dvs[4], bvs[4];                       // the 4 steps' operands, read together
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                dvs[k] = sm.dd[dd_row(4 * tq + k)][j];
                bvs[k] = sm.bc[4 * tq + k][q];
            }
#pragma unroll
            for (int k = 3; k >= 0; --k) {
                const int t = 4 * tq + k;
                const f32x4 dv = dvs[k];               // (dlt, dlt*u, ds, u)
                const f32x4 bv = bvs[k];               // (B0, B1, C0, C1)
                const float lam0 = __builtin_fmaf(dv.z, bv.z, carry[0]);
                const float lam1 = __builtin_fmaf(dv.z, bv.w, carry[1]);
                const float pb0 = lam0 * dv.y, pb1 = lam1 * dv.y;                          // dB terms
                const float pc0 = dv.z * hb[t + 1][0], pc1 = dv.z * hb[t + 1][1];          // dC terms
                const float u0 = __builtin_fmaf(lam1, bv.y, lam0 * bv.x);
                const float w0 = lam0 * ab[t][0] * hb[t][0];
                const float w1 = lam1 * ab[t][1] * hb[t][1];
                pu[k] = u0;                             // sum_n lambda B      (du; u * it in ddelta)
                pd[k] = __builtin_fmaf(Av[1], w1, Av[0] * w0);   // sum_n A lambda abar h_{t-1}
                dA[0] = __builtin_fmaf(dv.x, w0, dA[0]);
                dA[1] = __builtin_fmaf(dv.x, w1, dA[1]);
                carry[0] = lam0 * ab[t][0];
                carry[1] = lam1 * ab[t][1];
                // the channel sums after the step's other work, so the swaps do not
                // wait on the products just formed
                const float sb = half_swap_sum(pb0, pb1);                                   // dB: b5 picks the state
                const float sc = half_swap_sum(pc0, pc1);                                   // dC
                const float tot = add_xor8(row_swap_sum(sb, sc));                          // b4 picks dB or dC
                if (k & 1) {
                    tot_hi = tot;
                } else {                                // steps k, k + 1: b3 = 0 stores k, b3 = 1 stores k + 1
                    const float v = b3 ? tot_hi : tot;
                    if (WG) wg_sums[((buf * kWaves + wave) * 2 + (k >> 1)) * 64 + lane] = v;
                    else pbc[pl + (4 * tq + k) * (kQ * 4)] = v;
                }
            }
            sm.pa[4 * j + tq][q] = f32x4{pu[0], pu[1], pu[2], pu[3]};
            sm.pb[4 * j + tq][q] = f32x4{pd[0], pd[1], pd[2], pd[3]};
            if (WG) {
                // Every wave's 128 sums of this group are in wg_sums[buf]; wave w adds up
                // the 4 waves' values of source lanes 32 (w & 1) .. + 31 of step pair
                // w >> 1 (fixed order: deterministic) and writes them.  The buffers
                // alternate, so the next group's writes never meet these reads: a wave
                // passes the next barrier only after all have finished reading here.
                __syncthreads();
                if (lane < 32) {
                    const int i = wave >> 1, l = (wave & 1) * 32 + lane;
                    const float *x0 = wg_sums + (buf * kWaves * 2 + i) * 64 + l;
                    const float sum = (x0[0] + x0[2 * 64]) + (x0[4 * 64] + x0[6 * 64]);
                    const int lslot = ((l >> 5) << 1) | ((l >> 4) & 1);
                    pbc[((uint32_t)t0 + 4 * tq + 2 * i + ((l >> 3) & 1)) * (kQ * 4) + (l & 7) * 4 + lslot] = sum;
                }
                buf ^= 1;
            }
        }
        wave_sync();                                    // pa / pb are read below

        // ---- C2: du and ddelta of timesteps 2q, 2q+1 ------------------------------
        {
            float duv[2], ddv[2], su[2], sd[2];
            part_sum(sm.pa, j, q, su);
            part_sum(sm.pb, j, q, sd);
#pragma unroll
            for (int k = 0; k < 2; ++k) {
                duv[k] = __builtin_fmaf(dlv[k], su[k], dsv[k] * dskip);
                ddv[k] = __builtin_fmaf(xs[k], su[k], sd[k]) * sg[k];
                sum_dbias += ddv[k];
            }
            if (live) {
                store2<OUT>(dub, lrow + (uint32_t)t0 + 2 * q, duv[0], duv[1]);
                store2<OUT>(ddb, lrow + (uint32_t)t0 + 2 * q, ddv[0], ddv[1]);
            }
        }
        wave_sync();                                    // dd / bc / pa / pb are rewritten
    };

    Slot s0, s1;
    issue(s0, t_end - kT);
    issue(s1, t_end - 2 * kT);
    int64_t t0 = t_end - kT;
    for (; t0 - kT >= t_begin; t0 -= 2 * kT) {         // pairs of chunks, backwards
        chunk(s0, t0);
        chunk(s1, t0 - kT);
    }
    if (t0 >= t_begin) chunk(s0, t0);

    // ---- per-row results: dh0, dA (per state), dDskip and dbias (per channel) ----
#pragma unroll
    for (int off = 1; off < kQ; off <<= 1) {            // sum over the 8 lanes of channel j
        sum_dD += __shfl_xor(sum_dD, off, 64);
        sum_dbias += __shfl_xor(sum_dbias, off, 64);
    }
    if (live) {
        if (p.dh0 && seg == 0) {
            p.dh0[row * kN + n0] = carry[0];
            p.dh0[row * kN + n0 + 1] = carry[1];
        }
        float *pr = p.part_row + (seg * rows + row) * (kN + 2);
        pr[n0] = dA[0];
        pr[n0 + 1] = dA[1];
        if (q == 0) {
            pr[kN] = sum_dD;
            pr[kN + 1] = sum_dbias;
        }
    }
}

// ---- the reductions ---------------------------------------------------------------
// dB[b][n][t], dC[b][n][t]: thread (b, t, q) sums the ncg channel-group partials.
__global__ __launch_bounds__(256) void bwd_finish_bc(BwdParams p, float *dB, float *dC, int64_t ncg) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;   // (b, t, q)
    const int64_t L = p.seqlen;
    if (i >= p.batch * L * kQ) return;
    const int64_t qq = i % kQ, t = (i / kQ) % L, b = i / (kQ * L);
    const int64_t stride = p.batch * L * kQ * 4;
    const float *src = p.part_bc + ((b * L + t) * kQ + qq) * 4;
    f32x4 sum = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    for (int64_t c = 0; c < ncg; ++c) sum += *reinterpret_cast<const f32x4 *>(src + c * stride);
    const int64_t n0 = 2 * qq;
    dB[(b * kN + n0) * L + t] = sum.x;
    dC[(b * kN + n0) * L + t] = sum.y;
    dB[(b * kN + n0 + 1) * L + t] = sum.z;
    dC[(b * kN + n0 + 1) * L + t] = sum.w;
}

// dA[d][n], dDskip[d], dbias[d]: thread (d, slot) sums over the batch and the
// time segments.
__global__ __launch_bounds__(256) void bwd_finish_rows(BwdParams p, float *dA, float *dD, float *dbias) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;   // (d, slot)
    if (i >= p.dim * (kN + 2)) return;
    const int64_t d = i / (kN + 2), slot = i % (kN + 2);
    const int64_t nseg = (p.seqlen + p.seg_len - 1) / p.seg_len;
    float sum = 0.0f;
    for (int64_t s = 0; s < nseg; ++s)
        for (int64_t b = 0; b < p.batch; ++b)
            sum += p.part_row[((s * p.batch + b) * p.dim + d) * (kN + 2) + slot];
    if (slot < kN) dA[d * kN + slot] = sum;
    else if (slot == kN) { if (dD) dD[d] = sum; }
    else if (dbias) dbias[d] = sum;
}

}  // namespace bwd
}  // namespace mbs
