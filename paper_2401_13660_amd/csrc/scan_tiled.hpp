// scan_tiled.hpp -- the forward selective scan for dstate = 16, tiled for gfx950.
//
// Each wavefront works alone (no workgroup barrier anywhere): it owns 8
// channels of one batch element over one time segment, and lane l = 8 j + q
// holds channel j's states 2q and 2q+1 of eq. (2) in VGPRs.  Time advances in
// chunks of T = 32 bytes; per chunk the wave
//
//   A  does the per-element work once: lane (j, q) widens u, delta and z of
//      channel j at timesteps 4q .. 4q+3 (eight lanes read 64 contiguous bytes
//      of a row), computes dlt = softplus(delta + dt_bias) (eq. (3)),
//      dx = dlt * u and silu(z) (Table 8), and publishes (dlt, dx) in its
//      private LDS area; the wave also stages the chunk's B and C rows there,
//      time-major and widened to fp32;
//   B  runs the recurrence for its two states over the 32 timesteps --
//      abar = 2^(dlt A log2 e) (zero-order hold on A), h = abar h + dx B
//      (simplified Euler on B) -- reading the next four timesteps' operands
//      from LDS while computing the current four, and publishes its partial
//      contraction C_t[2q] h_t[2q] + C_t[2q+1] h_t[2q+1] per timestep;
//   C  lane (j, q) sums the eight partials of channel j at its own timesteps
//      4q .. 4q+3, adds Dskip * u, applies the gate and stores y (eight lanes
//      write 128 contiguous bytes of a row).
//
// Global loads run two chunks ahead.  Arithmetic is fp32; the state never
// leaves VGPRs except through h0 / h_last.  Requires seqlen % 16 == 0 and
// 16-byte aligned activation rows (the host checks; otherwise it uses the
// row-per-thread kernel).
#pragma once

#include <hip/hip_runtime.h>

#include "device_math.hpp"
#include "scan_params.hpp"

#include <type_traits>

namespace mbs {
namespace tiled {

constexpr int kN = 16;                // states per channel
constexpr int kCh = 8;                // channels per wave
constexpr int kQ = 8;                 // state pairs per channel (lanes per channel)
constexpr int kT = 32;                // timesteps per chunk
constexpr int kWavesPerGroup = 4;     // independent waves per workgroup
constexpr int kThreads = kWavesPerGroup * 64;

// 4 consecutive activations of one row (8 bytes bf16, 16 bytes fp32).
template <int IN> struct Raw4;
template <> struct Raw4<1> {
    u32x2 v;
    __device__ __forceinline__ void load(const void *base, uint32_t off) {
        v = *reinterpret_cast<const u32x2 *>(static_cast<const char *>(base) + off * 2u);
    }
    __device__ __forceinline__ void zero() { v = u32x2{0, 0}; }
    __device__ __forceinline__ float get(int i) const {
        const uint32_t w = (i >> 1) ? v.y : v.x;
        return (i & 1) ? bf16_hi(w) : bf16_lo(w);
    }
};
template <> struct Raw4<0> {
    f32x4 v;
    __device__ __forceinline__ void load(const void *base, uint32_t off) {
        v = *reinterpret_cast<const f32x4 *>(static_cast<const char *>(base) + off * 4u);
    }
    __device__ __forceinline__ void zero() { v = f32x4{0, 0, 0, 0}; }
    __device__ __forceinline__ float get(int i) const { return v[i]; }
};

// 2 consecutive activations of one row (4 bytes bf16, 8 bytes fp32): the
// per-lane share of a 16-timestep sequence.
template <int IN> struct Raw2;
template <> struct Raw2<1> {
    uint32_t v;
    __device__ __forceinline__ void load(const void *base, uint32_t off) {
        v = *reinterpret_cast<const uint32_t *>(static_cast<const char *>(base) + off * 2u);
    }
    __device__ __forceinline__ float get(int i) const { return i ? bf16_hi(v) : bf16_lo(v); }
};
template <> struct Raw2<0> {
    float2 v;
    __device__ __forceinline__ void load(const void *base, uint32_t off) {
        v = *reinterpret_cast<const float2 *>(static_cast<const char *>(base) + off * 4u);
    }
    __device__ __forceinline__ float get(int i) const { return i ? v.y : v.x; }
};

// Private LDS area of one wave.  Rows are padded so that the reads of every
// table touch distinct banks (16-byte entries, 64 banks), and the dd rows are
// permuted (dd_row) so that its writes do too: a 16-byte write serves 8
// consecutive lanes at a time from 32 banks (a 128-byte period, measured), and
// the 8 lanes of one channel write timestep pairs 2q and 2q + 1; rows of 9
// entries in natural order put those 8 writes in pairs on 4 bank quads.
//   dd    row dd_row(r) = timesteps 2r, 2r+1; entry j = (dlt, dx, dlt, dx) of channel j
//   bc    row t; entry q = (B[2q], B[2q+1], C[2q], C[2q+1]) at timestep t
//   part  row 8 j + tq = channel j, timesteps 4 tq .. 4 tq + 3; entry q = the
//         partial output of state pair q at those four timesteps
constexpr int kDdRow = 9;       // 16-byte entries per row: 8 used + 1 pad
constexpr int kBcRow = 10;      // 8 used + 2 pad
constexpr int kPartRow = 9;     // 8 used + 1 pad
// SHORT: the tables of a sequence of one 16-timestep half chunk (the verify
// shape), about a third the size, so that 7 workgroups fit in a CU's LDS instead
// of 2.  Their B/C rows have no pad (every write and read of a row covers its 8
// entries at once), and lanes q and q ^ 1 add their partial outputs in registers
// before the write, so a partial row holds 4 sums (+ 1 pad entry).
// The dd row of timestep pair r: pairs 2q and 2q + 1 go to rows q and 8 + q, so
// that the 8 lanes of a channel write 8 different bank quads.  (The 16-timestep
// tables have 8 rows; lane q writes row q only.)
template <bool SHORT> __device__ __forceinline__ constexpr int dd_row(int r) {
    return SHORT ? r : (r >> 1) + (r & 1) * (kT / 4);
}
template <bool SHORT> struct WaveSmemT {
    static constexpr int kSteps = SHORT ? kT / 2 : kT;
    static constexpr int kPartW = SHORT ? kQ / 2 + 1 : kPartRow;
    f32x4 dd[kSteps / 2][kDdRow];                    // 2.25 KB (SHORT: 1.1 KB)
    f32x4 bc[kSteps][SHORT ? kQ : kBcRow];           // 5 KB (SHORT: 2 KB)
    f32x4 part[kCh * (kSteps / 4)][kPartW];          // 9 KB (SHORT: 2.5 KB)
};
using WaveSmem = WaveSmemT<false>;
static_assert(sizeof(WaveSmemT<true>) * kWavesPerGroup * 7 <= 160 * 1024,
              "seven workgroups of the 16-timestep tables fit the 160 KB of a CU's LDS");

// v + the value of lane l ^ 1 (a DPP quad permutation): the same sum in both lanes.
__device__ __forceinline__ float add_lane_xor1(float v) {
    return v + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xf, 0xf, false));
}
// The segment aggregate pass (scan_seg_agg) needs neither C nor the output
// partials.  It stages B two timesteps per entry, and the smaller area lets more
// waves share a CU:
//   b2    row dd_row(r) = timesteps 2r, 2r+1; entry q = (B[2q], B[2q+1]) at 2r, then at 2r+1
// (the dd rows are permuted as in the scan's tables)
struct WaveSmemPre {
    static constexpr int kSteps = kT;
    f32x4 dd[kT / 2][kDdRow];                 // 2.25 KB
    f32x4 b2[kT / 2][kDdRow];                 // 2.25 KB
};

// The scan.  With several time segments, each cut into `pieces` equal pieces for
//   the pre-pass, the wave of segment s starts from the copy of h0 that
//   scan_seg_agg leaves in carry plane pieces (nseg - 1), folded with the
//   aggregates of pieces 0 .. pieces s - 1 (carry planes 0 .. pieces s - 1), those
//   of the segments before it in time order.  It never reads h0
//   itself: the wave of the last segment may then write h_last over h0 while the
//   waves of earlier segments of the same rows have not started (workgroups are
//   not ordered).
// POS = true: also record the states at p.pos (p.npos > 0).
// CK = true: also store the state at every 16-timestep boundary in p.ck, the
//   checkpoints the backward recomputes its chunks from.
// SHORT = true (seqlen 16): one half chunk per wave, with the half-size tables
//   of WaveSmemT<true>; phases A and C give every lane two timesteps (2q, 2q+1)
//   instead of four to half of them.
template <int N> __device__ __forceinline__ void lds_wait() {
    static_assert(N >= 0 && N < 16, "lgkmcnt is a 4-bit field");
    // nothing may be scheduled across the wait, so that the reads issued after
    // it stay after it and the operands read before it need no further wait
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(0xC07F | (N << 8));
    __builtin_amdgcn_sched_barrier(0);
}

template <int IN, int OUT, bool GATE, bool SOFTPLUS, bool POS, bool CK = false, bool SHORT = false>
__global__ __launch_bounds__(kThreads) void scan_fwd_tiled(ScanParams p, int64_t seg_len, int64_t pieces,
                                                      const float *carry) {
    extern __shared__ __align__(16) unsigned char smem_raw[];
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    using Smem = WaveSmemT<SHORT>;
    Smem &sm = reinterpret_cast<Smem *>(smem_raw)[wave];
    constexpr int kPS = Smem::kSteps / 4;              // part rows per channel

    const int lane = threadIdx.x & 63;
    const int j = lane >> 3;          // channel within the wave
    const int q = lane & 7;           // state pair; also the timestep quad of phases A and C
    // Wave indexing in 32 bits: the host launches fewer than 2^31 waves and
    // sends sequences shorter than 2^25 bytes here, so every quotient below fits.
    const uint32_t n_cg = (uint32_t)((p.dim + kCh - 1) / kCh);
    // (a 16-byte sequence is never cut into time segments: no division for it)
    const uint32_t nseg = SHORT ? 1u : ((uint32_t)p.seqlen + (uint32_t)seg_len - 1) / (uint32_t)seg_len;
    // Workgroups are dealt round-robin to the 8 XCDs (each with its own L2);
    // renumber them so that an XCD works on a contiguous range of (batch,
    // channel) groups and the B/C rows of a batch stay in one or two L2s.
    // Time segment innermost: the waves resident together work on every segment.
    // Their loads then spread over the L2 sets even when the row stride is a
    // multiple of 128 KB (L = 65536), where the same timestep of every row falls
    // in the same sets: ordered by segment, the 1.6B layer's scan fetched 2.54 GB
    // for 1.81 GB of activations, in this order 1.99 GB.
    // SHORT: a two-dimensional grid (channel groups x batch), so that a wave finds
    // its group without a division (its B/C rows are too few for the XCD order
    // to matter).
    uint32_t seg32 = 0, bq, cg32;
    if constexpr (SHORT) {
        cg32 = blockIdx.x * kWavesPerGroup + wave;
        bq = blockIdx.y;
        if (cg32 >= n_cg) return;                    // whole wave leaves together
    } else {
        const uint32_t per_xcd = gridDim.x / 8;
        const uint32_t blk = blockIdx.x;
        const uint32_t lwg = blk < per_xcd * 8 ? (blk % 8) * per_xcd + blk / 8 : blk;
        const uint32_t wid = lwg * kWavesPerGroup + wave;
        if (wid >= n_cg * (uint32_t)p.batch * nseg) return;   // whole wave leaves together
        const uint32_t rest = wid / nseg;
        seg32 = wid - rest * nseg;
        bq = rest / n_cg;
        cg32 = rest - bq * n_cg;
    }
    const int64_t seg = seg32;
    const int64_t cg = cg32;
    const int64_t b = bq;
    const int64_t t_begin = seg * seg_len;
    const int64_t t_end = t_begin + seg_len < p.seqlen ? t_begin + seg_len : p.seqlen;

    const int64_t d = cg * kCh + j;
    const bool live = d < p.dim;
    const int64_t dcl = live ? d : p.dim - 1;           // dead lanes read a valid row, never store
    const int64_t row = b * p.dim + dcl;
    const int64_t L = p.seqlen;
    const int n0 = 2 * q;

    // Global addressing: wave-uniform 64-bit bases (the wave's first channel
    // row, or state row 0 of B and C, at the segment start) plus 32-bit lane
    // offsets in elements, so the loads use the scalar-base form.
    constexpr int kEl = IN == 1 ? 2 : 4;
    const int64_t row0 = b * p.dim + cg * kCh;                       // wave-uniform
    const int64_t act0 = row0 * L + t_begin;
    const int64_t bc0 = b * kN * L + t_begin;
    const char *ub = static_cast<const char *>(p.u) + act0 * kEl;
    const char *db = static_cast<const char *>(p.delta) + act0 * kEl;
    const char *zb = GATE ? static_cast<const char *>(p.z) + act0 * kEl : nullptr;
    const char *bb = static_cast<const char *>(p.Bm) + bc0 * kEl;
    const char *cb = static_cast<const char *>(p.Cm) + bc0 * kEl;
    char *yb = static_cast<char *>(p.y) + act0 * (OUT == 1 ? 2 : 4);
    const uint32_t seg_n = (uint32_t)(t_end - t_begin);             // a multiple of 16
    const uint32_t act_row = (uint32_t)((dcl - cg * kCh) * L);       // lane's channel row
    // Elements per lane in phases A and C: timesteps kE q .. kE q + kE - 1.
    constexpr int kE = SHORT ? 2 : 4;
    // B/C staging: lane (j, q) moves timesteps kE j .. kE j + kE - 1 of state
    // rows 2q and 2q+1 of B and C, i.e. the entries bc[kE j + i][q].
    const int st_t = kE * j;
    const uint32_t bc_row = (uint32_t)(2 * q * L);

    using Raw = std::conditional_t<SHORT, Raw2<IN>, Raw4<IN>>;
    struct Slot { Raw u, dl, z, B0, B1, C0, C1; };
    Slot s0, s1;
    // Loads never branch: a chunk past the end of the segment reads the last
    // valid quad again (those values are never consumed), so the prefetch
    // registers are written in place every time.
    auto issue_loads = [&](Slot &sl, uint32_t tr) {            // tr: chunk start within the segment
        const uint32_t ta = tr + kE * q < seg_n - kE ? tr + kE * q : seg_n - kE;
        const uint32_t oa = act_row + ta;
        sl.u.load(ub, oa);
        sl.dl.load(db, oa);
        if (GATE) sl.z.load(zb, oa);
        const uint32_t tb = tr + st_t < seg_n - kE ? tr + st_t : seg_n - kE;
        const uint32_t ob = bc_row + tb;
        sl.B0.load(bb, ob);
        sl.B1.load(bb, ob + (uint32_t)L);
        sl.C0.load(cb, ob);
        sl.C1.load(cb, ob + (uint32_t)L);
    };
    // The activation loads of the first chunks go out before the per-row
    // operands below, whose loads are conditional (null pointers are allowed):
    // in the other order the compiler made the activation addresses wait for
    // them, two memory round trips before the first chunk (a whole call of the
    // 16-byte verify shape).
    issue_loads(s0, 0);
    if constexpr (!SHORT) issue_loads(s1, kT);

    const int64_t rows = p.batch * p.dim;
    float a2[2], h[2];
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        a2[s] = p.A[dcl * kN + n0 + s] * kLog2e;
        h[s] = (nseg == 1 && p.h0) ? p.h0[row * kN + n0 + s] : 0.0f;
    }
    if (nseg > 1) {
        // carry-in: the copy of h0, then the aggregates of the earlier segments'
        // pieces; folding (1, h0) into the zero state gives h0 exactly
        auto fold = [&](int64_t plane) {
            const f32x4 ph = *reinterpret_cast<const f32x4 *>(carry + ((plane * rows + row) * kN + n0) * 2);
            h[0] = __builtin_fmaf(ph.x, h[0], ph.y);
            h[1] = __builtin_fmaf(ph.z, h[1], ph.w);
        };
        fold(pieces * (nseg - 1));
        for (int64_t s2 = 0; s2 < pieces * seg; ++s2) fold(s2);
    }
    const float dskip = p.Dskip ? p.Dskip[dcl] : 0.0f;
    const float bias = p.dt_bias ? p.dt_bias[dcl] : 0.0f;


    // Phase B step TQ: timesteps 4 TQ .. 4 TQ + 3, operands already in registers.
    auto recur4 = [&](const f32x4 (&ddv)[2], const f32x4 (&bcv)[4], auto tq_c) {
        constexpr int TQ = decltype(tq_c)::value;
        float acc4[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const float dl = (k & 1) ? ddv[k >> 1].z : ddv[k >> 1].x;
            const float dx = (k & 1) ? ddv[k >> 1].w : ddv[k >> 1].y;
            const float b0 = bcv[k][0];
            const float b1 = bcv[k][1];
            const float a0 = hw_exp2(dl * a2[0]);
            const float a1 = hw_exp2(dl * a2[1]);
            h[0] = __builtin_fmaf(a0, h[0], dx * b0);
            h[1] = __builtin_fmaf(a1, h[1], dx * b1);
            acc4[k] = __builtin_fmaf(bcv[k][3], h[1], bcv[k][2] * h[0]);
        }
        if constexpr (SHORT) {
            // state pairs q and q ^ 1 summed; both lanes write the same entry
#pragma unroll
            for (int k = 0; k < 4; ++k) acc4[k] = add_lane_xor1(acc4[k]);
            sm.part[kPS * j + TQ][q >> 1] = f32x4{acc4[0], acc4[1], acc4[2], acc4[3]};
        } else {
            sm.part[kPS * j + TQ][q] = f32x4{acc4[0], acc4[1], acc4[2], acc4[3]};
        }
    };
    auto load4 = [&](f32x4 (&ddv)[2], f32x4 (&bcv)[4], auto tq_c) {
        constexpr int TQ = decltype(tq_c)::value;
#pragma unroll
        for (int k = 0; k < 2; ++k) ddv[k] = sm.dd[dd_row<SHORT>(2 * TQ + k)][j];
#pragma unroll
        for (int k = 0; k < 4; ++k) bcv[k] = sm.bc[4 * TQ + k][q];
    };
    // s_waitcnt lgkmcnt(N) (vmcnt and expcnt left alone): wait until at most N of
    // this wave's LDS operations are outstanding.
    constexpr int kW = 1;      // the scan writes one partial row per step
    // Order this wave's LDS writes before its later reads of other lanes' data.
    auto wave_sync = [] {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    };

    // States at requested positions inside the chunk at t0: starting from the
    // state before the chunk, replay the chunk's first timesteps from the
    // (dlt, dx) and B tables, which phase B has finished reading and the next
    // phase A has not yet rewritten.  The replay repeats phase B's operations
    // in the same order, so the recorded state equals the one the scan carries.
    auto record_positions = [&](int64_t t0, int nt, float r0, float r1) {
        if constexpr (POS) for (int64_t k = 0; k < p.npos; ++k) {
            const int64_t pk = p.pos[k * p.batch + b];              // wave-uniform
            if (pk < t0 || pk >= t0 + nt) continue;
            const int cnt = (int)(pk - t0) + 1;
            float g0 = r0, g1 = r1;
            for (int i = 0; i < cnt; ++i) {
                const f32x4 dv = sm.dd[dd_row<SHORT>(i >> 1)][j];
                const float dl = (i & 1) ? dv.z : dv.x;
                const float dx = (i & 1) ? dv.w : dv.y;
                const f32x4 bv = sm.bc[i][q];
                const float a0 = hw_exp2(dl * a2[0]);
                const float a1 = hw_exp2(dl * a2[1]);
                g0 = __builtin_fmaf(a0, g0, dx * bv[0]);
                g1 = __builtin_fmaf(a1, g1, dx * bv[1]);
            }
            if (live) {
                float *dst = p.h_pos + ((k * p.batch + b) * p.dim + d) * kN + n0;
                dst[0] = g0;
                dst[1] = g1;
            }
        }
    };

    // Checkpoints are stored in time order, one per 16 timesteps, so a lane's
    // pointer steps by one checkpoint plane (rows x kN floats) per store.
    float *ck_at = CK ? p.ck + ((t_begin / 16) * rows + row) * kN + n0 : nullptr;
    const int64_t ck_plane = rows * kN;
    auto store_ck = [&] {                            // the state before the next 16 timesteps
        if (live) *reinterpret_cast<float2 *>(ck_at) = float2{h[0], h[1]};
        ck_at += ck_plane;
    };

    auto chunk = [&](Slot &sl, int64_t t0) {
        const int nt = SHORT ? kT / 2 : (int)(t_end - t0 < kT ? t_end - t0 : kT);   // multiple of 16

        // ---- A: per-element work of timesteps kE q .. kE q + kE - 1 and B/C staging
        float xs[kE], gs[kE];
        {
            float dl[kE], dx[kE];
#pragma unroll
            for (int k = 0; k < kE; ++k) {
                const float x = sl.u.get(k);
                const float v = sl.dl.get(k) + bias;
                dl[k] = SOFTPLUS ? softplus_f32(v) : v;
                dx[k] = dl[k] * x;
                xs[k] = x;
                if (GATE) gs[k] = silu_f32(sl.z.get(k));
            }
            if constexpr (SHORT) {
                sm.dd[q][j] = f32x4{dl[0], dx[0], dl[1], dx[1]};
            } else {
                sm.dd[dd_row<false>(2 * q)][j] = f32x4{dl[0], dx[0], dl[1], dx[1]};
                sm.dd[dd_row<false>(2 * q + 1)][j] = f32x4{dl[2], dx[2], dl[3], dx[3]};
            }
        }
#pragma unroll
        for (int k = 0; k < kE; ++k)
            sm.bc[st_t + k][q] = f32x4{sl.B0.get(k), sl.B1.get(k), sl.C0.get(k), sl.C1.get(k)};
        wave_sync();

        // refill this slot with the chunk after next while the recurrence runs
        // (a 16-byte sequence has no next chunk)
        if constexpr (!SHORT) issue_loads(sl, (uint32_t)(t0 - t_begin) + 2 * kT);

        // ---- B: the recurrence, fully unrolled over the chunk; the operands of
        //      step i + 1 are read from LDS while step i computes ----------------
        const float hs0 = POS ? h[0] : 0.0f;        // the state before this chunk
        const float hs1 = POS ? h[1] : 0.0f;
        if (CK) store_ck();
        {
            f32x4 ddA[2], bcA[4], ddB[2], bcB[4];
            using I0 = std::integral_constant<int, 0>;
            using I1 = std::integral_constant<int, 1>;
            using I2 = std::integral_constant<int, 2>;
            using I3 = std::integral_constant<int, 3>;
            using I4 = std::integral_constant<int, 4>;
            using I5 = std::integral_constant<int, 5>;
            using I6 = std::integral_constant<int, 6>;
            using I7 = std::integral_constant<int, 7>;
            // One wait per step: before step i computes, its operands (read
            // during step i - 1) must have arrived, while the partial row that
            // step i - 1 wrote may still be in flight (LDS operations complete
            // in order).  The reads of step i + 1 go out right after the wait.
            load4(ddA, bcA, I0{});
            lds_wait<0>();
            load4(ddB, bcB, I1{});
            recur4(ddA, bcA, I0{});
            lds_wait<kW>();
            load4(ddA, bcA, I2{});
            recur4(ddB, bcB, I1{});
            lds_wait<kW>();
            load4(ddB, bcB, I3{});
            recur4(ddA, bcA, I2{});
            if (!SHORT && nt == kT) {
                lds_wait<kW>();
                load4(ddA, bcA, I4{});
                recur4(ddB, bcB, I3{});
                if (CK) store_ck();
                lds_wait<kW>();
                load4(ddB, bcB, I5{});
                recur4(ddA, bcA, I4{});
                lds_wait<kW>();
                load4(ddA, bcA, I6{});
                recur4(ddB, bcB, I5{});
                lds_wait<kW>();
                load4(ddB, bcB, I7{});
                recur4(ddA, bcA, I6{});
                lds_wait<kW>();
                recur4(ddB, bcB, I7{});
            } else {                                // nt == 16: the last, half chunk
                lds_wait<kW>();
                recur4(ddB, bcB, I3{});
            }
        }
        wave_sync();

        // ---- C: sum the 4 partial sums of channel j at timesteps 2q, 2q+1 ------
        if constexpr (SHORT) {
            // the partials of timesteps 2q, 2q+1 are one half of entry (j, q >> 1)
            const float2 *src = reinterpret_cast<const float2 *>(&sm.part[kPS * j + (q >> 1)][0]) + (q & 1);
            float2 acc = src[0];
#pragma unroll
            for (int w = 1; w < kQ / 2; ++w) {
                acc.x += src[2 * w].x;
                acc.y += src[2 * w].y;
            }
            float yv[2];
#pragma unroll
            for (int k = 0; k < 2; ++k) {
                float y = __builtin_fmaf(dskip, xs[k], k ? acc.y : acc.x);
                if (GATE) y *= gs[k];
                yv[k] = y;
            }
            if (live) {
                const uint32_t oy = act_row + (uint32_t)(t0 - t_begin) + 2 * q;
                if (OUT == 0)
                    *reinterpret_cast<float2 *>(yb + oy * 4u) = float2{yv[0], yv[1]};
                else
                    *reinterpret_cast<uint32_t *>(yb + oy * 2u) = bf16x2_pack(yv[0], yv[1]);
            }
        } else {
            if (4 * q < nt) {
                // ---- C: sum the 8 partials of channel j at timesteps 4q .. 4q+3 ----
                f32x4 acc = sm.part[kPS * j + q][0];
#pragma unroll
                for (int w = 1; w < kQ; ++w) acc += sm.part[kPS * j + q][w];
                float yv[4];
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    float y = __builtin_fmaf(dskip, xs[k], acc[k]);
                    if (GATE) y *= gs[k];
                    yv[k] = y;
                }
                if (live) {
                    const uint32_t oy = act_row + (uint32_t)(t0 - t_begin) + 4 * q;
                    if (OUT == 0) {
                        *reinterpret_cast<f32x4 *>(yb + oy * 4u) = f32x4{yv[0], yv[1], yv[2], yv[3]};
                    } else {
                        const uint32_t w0 = bf16x2_pack(yv[0], yv[1]);
                        const uint32_t w1 = bf16x2_pack(yv[2], yv[3]);
                        *reinterpret_cast<u32x2 *>(yb + oy * 2u) = u32x2{w0, w1};
                    }
                }
            }
        }
        if (POS) record_positions(t0, nt, hs0, hs1);
        wave_sync();   // part / dd / bc are rewritten by the next chunk
    };

    if constexpr (SHORT) {
        chunk(s0, t_begin);                         // the one half chunk
    } else {
        int64_t t0 = t_begin;
        for (; t0 + 2 * kT <= t_end; t0 += 2 * kT) {   // pairs of full chunks
            chunk(s0, t0);
            chunk(s1, t0 + kT);
        }
        if (t0 < t_end) chunk(s0, t0);                  // a full chunk and/or a half chunk remain
        if (t0 + kT < t_end) chunk(s1, t0 + kT);
    }

    if (p.h_last && live && seg == nseg - 1) {
#pragma unroll
        for (int s = 0; s < 2; ++s) p.h_last[row * kN + n0 + s] = h[s];
    }
}

// ---- segment aggregates ------------------------------------------------------
//
// The scan's segments but the last are cut into pieces of piece_len timesteps
// (a multiple of 32), npieces in all.  For every piece and every state n of a
// row, the piece's element of the associative operator of
// Section 2 ("Implementation"):
//   P[n] = prod_t abar_t[n] = 2^(A[n] log2 e sum_t dlt_t),
//   H[n] = sum_t (prod_{r > t} abar_r[n]) dlt_t B_t[n] x_t,
// so that the state at the piece's end is P h_start + H.  H is the state the
// recurrence reaches from a zero state at the piece's start; P is one
// exponential of the piece's summed dlt, not a product of hundreds of
// hardware exponentials near 1, whose rounding would drift and be carried into
// every later segment by the fold P h + H.  The pairs (P, H) go to
// carry[((piece * rows + row) * 16 + n) * 2 + {0, 1}].
//
// Pieces smaller than the scan's segments balance the pass: one wave per piece
// and 8 channels, and with one piece per segment the 1.6B layer's 3,456 waves
// leave 4 on some SIMDs and 3 on others, while 6,912 half-length pieces make 6.75
// per SIMD against at most 7.
//
// A walk from the segment's end that stops once the running product of abar is
// exactly zero in fp32 gives the same (P, H) with fewer timesteps, but with the
// timestep bias of the MambaByte layers (dt down to 1e-3) some channel of almost
// every 8-channel wave decays too slowly for that within a segment, and the walk
// costs a multiply more per step: measured slower on the 1.6B layer.
//
// The waves of piece 0 also copy h0 (or zeros) into plane npieces as the pairs
// (1, h0[n]), which the scan folds first.
//
// Lane l = 8 j + q as in the scan: channel j, states 2q and 2q+1.  Per chunk,
// lane (j, q) forms dlt and dx of channel j at timesteps 4q .. 4q+3 and stages B
// rows 2j and 2j+1 at those timesteps (the dd and b2 tables of WaveSmemPre).
template <int IN, bool SOFTPLUS>
__global__ __launch_bounds__(kThreads) void scan_seg_agg(ScanParams p, int64_t piece_len, int64_t npieces,
                                                    float *carry) {
    extern __shared__ __align__(16) unsigned char smem_raw[];
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    WaveSmemPre &sm = reinterpret_cast<WaveSmemPre *>(smem_raw)[wave];

    const int lane = threadIdx.x & 63;
    const int j = lane >> 3;
    const int q = lane & 7;
    const uint32_t n_cg = (uint32_t)((p.dim + kCh - 1) / kCh);
    const uint32_t nsg = (uint32_t)npieces;             // the pieces that have an aggregate
    const uint32_t per_xcd = gridDim.x / 8;
    const uint32_t blk = blockIdx.x;
    const uint32_t lwg = blk < per_xcd * 8 ? (blk % 8) * per_xcd + blk / 8 : blk;
    const uint32_t wid = lwg * kWavesPerGroup + wave;
    if (wid >= n_cg * (uint32_t)p.batch * nsg) return;   // whole wave leaves together
    const uint32_t rest = wid / nsg;
    const int64_t piece = wid - rest * nsg;
    const uint32_t bq = rest / n_cg;
    const int64_t cg = rest - bq * n_cg;
    const int64_t b = bq;
    const int64_t t_begin = piece * piece_len;

    const int64_t d = cg * kCh + j;
    const bool live = d < p.dim;
    const int64_t dcl = live ? d : p.dim - 1;           // dead lanes read a valid row, never store
    const int64_t row = b * p.dim + dcl;
    const int64_t L = p.seqlen;
    const int n0 = 2 * q;
    const int64_t rows = p.batch * p.dim;

    float a2[2], h[2] = {0.0f, 0.0f};
    float dsum = 0.0f;      // this lane's share of the piece's sum of dlt
#pragma unroll
    for (int s = 0; s < 2; ++s) a2[s] = p.A[dcl * kN + n0 + s] * kLog2e;
    if (piece == 0 && live) {
        const float g0 = p.h0 ? p.h0[row * kN + n0] : 0.0f;
        const float g1 = p.h0 ? p.h0[row * kN + n0 + 1] : 0.0f;
        *reinterpret_cast<f32x4 *>(carry + (((int64_t)nsg * rows + row) * kN + n0) * 2) =
            f32x4{1.0f, g0, 1.0f, g1};
    }
    const float bias = p.dt_bias ? p.dt_bias[dcl] : 0.0f;

    constexpr int kEl = IN == 1 ? 2 : 4;
    const int64_t row0 = b * p.dim + cg * kCh;                       // wave-uniform
    const int64_t act0 = row0 * L + t_begin;
    const char *ub = static_cast<const char *>(p.u) + act0 * kEl;
    const char *db = static_cast<const char *>(p.delta) + act0 * kEl;
    const char *bb = static_cast<const char *>(p.Bm) + (b * kN * L + t_begin) * kEl;
    const uint32_t act_row = (uint32_t)((dcl - cg * kCh) * L);       // lane's channel row
    const uint32_t bc_row = (uint32_t)(2 * j * L);                   // B rows 2j, 2j+1
    const uint32_t nch = (uint32_t)(piece_len / kT);

    struct Slot { Raw4<IN> u, dl, B0, B1; };
    Slot s0, s1;
    // Chunk k starts at 32 k; past the piece's end the loads read the last
    // chunk again (never consumed).
    auto issue_loads = [&](Slot &sl, uint32_t k) {
        const uint32_t tr = (k < nch ? k : nch - 1) * kT + 4 * q;
        sl.u.load(ub, act_row + tr);
        sl.dl.load(db, act_row + tr);
        sl.B0.load(bb, bc_row + tr);
        sl.B1.load(bb, bc_row + tr + (uint32_t)L);
    };
    // Four timesteps: table rows 2 TQ and 2 TQ + 1, the even timestep of a row first.
    auto fwd4 = [&](const f32x4 (&dv)[2], const f32x4 (&bv)[2]) {
#pragma unroll
        for (int k = 0; k < 2; ++k) {
#pragma unroll
            for (int o = 0; o < 2; ++o) {
                const float dl = o ? dv[k].z : dv[k].x;
                const float dx = o ? dv[k].w : dv[k].y;
                const float b0 = o ? bv[k].z : bv[k].x;
                const float b1 = o ? bv[k].w : bv[k].y;
                h[0] = __builtin_fmaf(hw_exp2(dl * a2[0]), h[0], dx * b0);
                h[1] = __builtin_fmaf(hw_exp2(dl * a2[1]), h[1], dx * b1);
            }
        }
    };
    auto load2 = [&](f32x4 (&dv)[2], f32x4 (&bv)[2], int tq) {
#pragma unroll
        for (int k = 0; k < 2; ++k) {
            dv[k] = sm.dd[dd_row<false>(2 * tq + k)][j];
            bv[k] = sm.b2[dd_row<false>(2 * tq + k)][q];
        }
    };
    auto wave_sync = [] {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    };

    auto chunk = [&](Slot &sl, uint32_t k) {
        float dl[4], dx[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float v = sl.dl.get(i) + bias;
            dl[i] = SOFTPLUS ? softplus_f32(v) : v;
            dx[i] = dl[i] * sl.u.get(i);
        }
        // pairwise within the quad, then across chunks and lanes: the rounding
        // of the piece's sum stays small
        dsum += (dl[0] + dl[1]) + (dl[2] + dl[3]);
        sm.dd[dd_row<false>(2 * q)][j] = f32x4{dl[0], dx[0], dl[1], dx[1]};
        sm.dd[dd_row<false>(2 * q + 1)][j] = f32x4{dl[2], dx[2], dl[3], dx[3]};
        sm.b2[dd_row<false>(2 * q)][j] = f32x4{sl.B0.get(0), sl.B1.get(0), sl.B0.get(1), sl.B1.get(1)};
        sm.b2[dd_row<false>(2 * q + 1)][j] = f32x4{sl.B0.get(2), sl.B1.get(2), sl.B0.get(3), sl.B1.get(3)};
        wave_sync();
        issue_loads(sl, k + 2);
        {
            f32x4 dA[2], bA[2], dB[2], bB[2];
            load2(dA, bA, 0);
            lds_wait<0>();
            load2(dB, bB, 1);
            fwd4(dA, bA);
            lds_wait<0>();
            load2(dA, bA, 2);
            fwd4(dB, bB);
            lds_wait<0>();
            load2(dB, bB, 3);
            fwd4(dA, bA);
            lds_wait<0>();
            load2(dA, bA, 4);
            fwd4(dB, bB);
            lds_wait<0>();
            load2(dB, bB, 5);
            fwd4(dA, bA);
            lds_wait<0>();
            load2(dA, bA, 6);
            fwd4(dB, bB);
            lds_wait<0>();
            load2(dB, bB, 7);
            fwd4(dA, bA);
            lds_wait<0>();
            fwd4(dB, bB);
        }
        wave_sync();                                  // dd / b2 are rewritten by the next chunk
    };

    issue_loads(s0, 0);
    issue_loads(s1, 1);
    uint32_t k = 0;
    for (; k + 2 <= nch; k += 2) {                  // pairs of chunks
        chunk(s0, k);
        chunk(s1, k + 1);
    }
    if (k < nch) chunk(s0, k);                      // an odd chunk count leaves one
    // the eight lanes of channel j hold its timesteps 4q .. 4q+3 of every chunk:
    // after the butterfly each holds the whole piece's sum
    dsum += __shfl_xor(dsum, 1);
    dsum += __shfl_xor(dsum, 2);
    dsum += __shfl_xor(dsum, 4);
    if (live) {
        const float P0 = hw_exp2(a2[0] * dsum), P1 = hw_exp2(a2[1] * dsum);
        *reinterpret_cast<f32x4 *>(carry + ((piece * rows + row) * kN + n0) * 2) = f32x4{P0, h[0], P1, h[1]};
    }
}

// ---- host side: launch configuration -------------------------------------

// Time segments for the tiled path.  One wave covers 8 channels of one batch
// element, and a CU holds two workgroups of the scan at once (its LDS area
// allows no more): `resident` = 8 waves per CU.  With fewer than 3/8 of that
// per segment most of the chip idles, so the sequence is cut into segments
// (each a multiple of 32 bytes, at least 256).  A pre-pass computes each
// segment's aggregate from a zero state; the scan of segment s then starts
// from h0 folded with the aggregates of segments 0 .. s-1.  The count is the
// largest that fills the chip at most twice over: a third round, partly
// filled, costs more than its shorter segments return.  Above the threshold
// the pre-pass costs more than the extra occupancy returns.
// The pre-pass cuts each segment into `pieces` (1 or 2) equal pieces, one wave
// per piece and 8 channels.  A SIMD takes as long as its largest number of
// waves times the piece length, so 2 pieces are taken where that is shorter:
// ceil(2 w / simds) / 2 below ceil(w / simds), for the w waves of whole
// segments.  That takes 2 pieces only up to 7 waves per SIMD, as many as fit
// with bf16 inputs (70 VGPRs), so those waves are all resident at once.
inline int64_t choose_segments(int64_t waves_base, int64_t L, int64_t resident, int64_t simds, int64_t *seg_len,
                               int64_t *pieces) {
    int64_t nseg = 1;
    if (waves_base > 0 && waves_base * 8 < resident * 3) nseg = 2 * resident / waves_base;
    const int64_t max_seg = L / 256;
    if (nseg > max_seg) nseg = max_seg;
    if (nseg < 1) nseg = 1;
    int64_t m = 1;
    if (nseg > 1) {
        const int64_t w = waves_base * (nseg - 1);
        if ((2 * w + simds - 1) / simds < 2 * ((w + simds - 1) / simds)) m = 2;
    }
    int64_t len = (L + nseg - 1) / nseg;
    len = (len + 32 * m - 1) / (32 * m) * (32 * m);     // pieces of a multiple of 32 timesteps
    *seg_len = len;
    *pieces = m;
    return (L + len - 1) / len;
}

// Compute units of the current device; 256 (MI355X) if the runtime cannot say.
inline int64_t device_cus() {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
        cus = 256;
    return cus;
}

// Waves of the scan resident at once on the current device (2 workgroups of
// 4 waves per CU).
inline int64_t resident_waves() { return 2 * kWavesPerGroup * device_cus(); }

// The time segments the forward takes for p (1: none), their length and the
// pre-pass pieces per segment.
inline int64_t fwd_segments(const ScanParams &p, int64_t *seg_len, int64_t *pieces) {
    const int64_t n_cg = (p.dim + kCh - 1) / kCh;
    *seg_len = p.seqlen;
    *pieces = 1;
    return p.seqlen >= 512
               ? choose_segments(n_cg * p.batch, p.seqlen, resident_waves(), 4 * device_cus(), seg_len, pieces)
               : 1;
}

// Device bytes of the segment carry: the aggregates of the pieces of segments
// 0 .. nseg-2, then the copy of h0 (rows x 16 states x 2 floats per plane).
inline size_t fwd_carry_bytes(const ScanParams &p, int64_t nseg, int64_t pieces) {
    return nseg > 1 ? (size_t)(pieces * (nseg - 1) + 1) * (size_t)(p.batch * p.dim) * kN * 2 * sizeof(float) : 0;
}

// lent: device memory of at least fwd_carry_bytes() for the carry, or null for
// an allocation on the stream (hipMallocAsync, freed after the scan).
template <int IN, int OUT, bool GATE, bool SP>
hipError_t fwd_tiled_sp(ScanParams &p, void *stream, float *lent) {
    hipStream_t st = static_cast<hipStream_t>(stream);
    const int64_t n_cg = (p.dim + kCh - 1) / kCh;
    int64_t seg_len = p.seqlen, pieces = 1;
    const int64_t nseg = fwd_segments(p, &seg_len, &pieces);
    float *carry = nullptr;
    const size_t lds = sizeof(WaveSmem) * kWavesPerGroup;
    hipError_t e;
    if (nseg > 1) {
        if (lent) {
            carry = lent;
        } else {
            e = hipMallocAsync(reinterpret_cast<void **>(&carry), fwd_carry_bytes(p, nseg, pieces), st);
            if (e != hipSuccess) return e;
        }
        int64_t piece_len = seg_len / pieces, npieces = pieces * (nseg - 1);
        const int64_t waves = n_cg * p.batch * npieces;
        const int64_t blocks = (waves + kWavesPerGroup - 1) / kWavesPerGroup;
        void *args[] = {&p, &piece_len, &npieces, &carry};
        e = hipLaunchKernel(reinterpret_cast<const void *>(&scan_seg_agg<IN, SP>), dim3((unsigned)blocks),
                            dim3(kThreads), args, sizeof(WaveSmemPre) * kWavesPerGroup, st);
        if (e != hipSuccess) {
            if (!lent) (void)hipFreeAsync(carry, st);
            return e;
        }
    }
    const int64_t waves = n_cg * p.batch * nseg;
    const int64_t blocks = (waves + kWavesPerGroup - 1) / kWavesPerGroup;
    void *args[] = {&p, &seg_len, &pieces, &carry};
    // One 16-timestep half chunk per wave (the verify shape): half-size tables.
    const bool short_seq = p.seqlen == kT / 2 && nseg == 1 && !p.ck && p.batch <= 65535;
    const void *main_fn =
        short_seq ? (p.npos > 0
                         ? reinterpret_cast<const void *>(&scan_fwd_tiled<IN, OUT, GATE, SP, true, false, true>)
                         : reinterpret_cast<const void *>(&scan_fwd_tiled<IN, OUT, GATE, SP, false, false, true>))
        : p.npos > 0 ? reinterpret_cast<const void *>(&scan_fwd_tiled<IN, OUT, GATE, SP, true>)
        : p.ck       ? reinterpret_cast<const void *>(&scan_fwd_tiled<IN, OUT, GATE, SP, false, true>)
                     : reinterpret_cast<const void *>(&scan_fwd_tiled<IN, OUT, GATE, SP, false>);
    const size_t main_lds = short_seq ? sizeof(WaveSmemT<true>) * kWavesPerGroup : lds;
    const dim3 grid = short_seq ? dim3((unsigned)((n_cg + kWavesPerGroup - 1) / kWavesPerGroup), (unsigned)p.batch)
                                : dim3((unsigned)blocks);
    e = hipLaunchKernel(main_fn, grid, dim3(kThreads), args, main_lds, st);
    if (carry && !lent) {
        const hipError_t f = hipFreeAsync(carry, st);
        if (e == hipSuccess) e = f;
    }
    return e;
}

template <int IN, int OUT, bool GATE>
hipError_t fwd_tiled(ScanParams &p, void *stream, float *lent) {
    return p.delta_softplus ? fwd_tiled_sp<IN, OUT, GATE, true>(p, stream, lent)
                            : fwd_tiled_sp<IN, OUT, GATE, false>(p, stream, lent);
}

}  // namespace tiled
}  // namespace mbs
