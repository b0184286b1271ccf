// conv1d.hpp -- the causal depthwise convolution upstream of the scan.
//
// In the Mamba block the x branch passes through a per-channel causal 1D
// convolution with kernel size k and a bias, then the Swish activation, before
// it becomes the scan's input u (Table 8, "Pre-SSM 1D convolution"; Fig. 5,
// right; k = 4 in every MambaByte model, Table 9):
//
//   pre[t] = bias[d] + sum_{i < k} w[d][i] * x[t - (k-1) + i]
//   y[t]   = silu(pre[t])            (or pre[t] without the activation)
//
// with the k - 1 inputs before t = 0 taken from a carried state (oldest first),
// so that a sequence resumes exactly where the previous call stopped; the call
// returns the last k - 1 inputs as the next state.  The work is streaming
// (2 + 2 bytes per element for bf16 in and out, 2k + 7 flops): HBM-bound.
#pragma once

#include <hip/hip_runtime.h>

#include "device_math.hpp"

namespace mbs {
namespace conv {

constexpr int kSpan = 8;          // outputs per thread
constexpr int kThreads = 256;
constexpr int kMaxK = 4;

struct ConvParams {
    int64_t batch, dim, seqlen;
    const void *x;                // (batch, dim, L) act
    const float *w;               // (dim, K)
    const float *bias;            // (dim) or null
    const float *state_in;        // (batch, dim, K-1) or null: zeros
    void *y;                      // (batch, dim, L) out
    float *state_out;             // (batch, dim, K-1) or null
    int apply_silu;
};

// 8 consecutive activations starting at element offset off of an aligned row.
template <int DT> __device__ __forceinline__ void load8(const void *base, int64_t off, float (&v)[kSpan]);
template <> __device__ __forceinline__ void load8<1>(const void *base, int64_t off, float (&v)[kSpan]) {
    const u32x4 r = *reinterpret_cast<const u32x4 *>(static_cast<const uint16_t *>(base) + off);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        v[2 * i] = bf16_lo(r[i]);
        v[2 * i + 1] = bf16_hi(r[i]);
    }
}
template <> __device__ __forceinline__ void load8<0>(const void *base, int64_t off, float (&v)[kSpan]) {
    const f32x4 *p = reinterpret_cast<const f32x4 *>(static_cast<const float *>(base) + off);
    const f32x4 a = p[0], b = p[1];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        v[i] = a[i];
        v[4 + i] = b[i];
    }
}

// The last H (1..3) activations of the span of 8 at element offset off, t[j] =
// activation 8 - H + j.  Only the words that hold them are loaded: a loaded word
// that is never used frees its register at once, and the compiler then waits
// for the load to land before reusing it (a memory round trip per span).
template <int DT, int H> __device__ __forceinline__ void load_tail(const void *base, int64_t off, float (&t)[H]) {
    static_assert(H >= 1 && H <= 3, "kernel sizes 2..4");
    if constexpr (DT == 1) {
        const uint16_t *b = static_cast<const uint16_t *>(base) + off;
        if constexpr (H == 3) {
            const u32x2 r = *reinterpret_cast<const u32x2 *>(b + 4);      // activations 4..7
            t[0] = bf16_hi(r[0]);
            t[1] = bf16_lo(r[1]);
            t[2] = bf16_hi(r[1]);
        } else {
            const uint32_t r = *reinterpret_cast<const uint32_t *>(b + 6);   // activations 6, 7
            if constexpr (H == 2) t[0] = bf16_lo(r);
            t[H - 1] = bf16_hi(r);
        }
    } else {
        const float *f = static_cast<const float *>(base) + off + (kSpan - H);
#pragma unroll
        for (int j = 0; j < H; ++j) t[j] = f[j];
    }
}

template <int DT> __device__ __forceinline__ void store8(void *base, int64_t off, const float (&v)[kSpan]);
template <> __device__ __forceinline__ void store8<1>(void *base, int64_t off, const float (&v)[kSpan]) {
    u32x4 r;
#pragma unroll
    for (int i = 0; i < 4; ++i)
        r[i] = bf16x2_pack(v[2 * i], v[2 * i + 1]);
    *reinterpret_cast<u32x4 *>(static_cast<uint16_t *>(base) + off) = r;
}
template <> __device__ __forceinline__ void store8<0>(void *base, int64_t off, const float (&v)[kSpan]) {
    f32x4 *p = reinterpret_cast<f32x4 *>(static_cast<float *>(base) + off);
    p[0] = f32x4{v[0], v[1], v[2], v[3]};
    p[1] = f32x4{v[4], v[5], v[6], v[7]};
}

// The common shape: every row of x and y starts 16-byte aligned and L % 8 == 0,
// so spans of 8 move as 16-byte vectors, and rows follow each other in memory,
// so the spans of all rows form one sequence g = row * nspan + span.  Lane i of
// wave w of block blk takes spans g = ((blk * 4 + w) * kVecPerThread + v) * 64 + i
// for v < kVecPerThread: each load instruction of a wave reads one contiguous
// 1 KB (bf16), across row ends too, and all of a thread's loads (its spans and,
// for the k-1 inputs before each, the neighbouring span, a cache hit) are in
// flight before any arithmetic.  Short rows (the 16-byte verify chunk) pack
// densely.
constexpr int kVecPerThread = 2;

template <int IN, int OUT, int K>
__global__ __launch_bounds__(kThreads) void conv1d_fwd_vec(ConvParams p, uint32_t nspan, uint32_t total) {
    constexpr int H = K - 1;
    const int64_t L = p.seqlen;
    const uint32_t first = (blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6)) * (64 * kVecPerThread) +
                           (threadIdx.x & 63);

    // Every load of the thread (its spans, the neighbouring spans' last inputs,
    // the taps, bias and carried state of their rows) is issued before any of
    // them is used: one memory round trip per thread.
    float cur[kVecPerThread][kSpan], prev[kVecPerThread][H > 0 ? H : 1];
    float w[kVecPerThread][K], bv[kVecPerThread], st[kVecPerThread][H > 0 ? H : 1];
    uint32_t row[kVecPerThread], sp[kVecPerThread];
#pragma unroll
    for (int v = 0; v < kVecPerThread; ++v) {
        // a span past the last one reads the last span again (never stored)
        const uint32_t g = first + v * 64 < total ? first + v * 64 : total - 1;
        load8<IN>(p.x, (int64_t)g * kSpan, cur[v]);
        if constexpr (H > 0) load_tail<IN, H>(p.x, (int64_t)(g > 0 ? g - 1 : 0) * kSpan, prev[v]);
    }
#pragma unroll
    for (int v = 0; v < kVecPerThread; ++v) {
        const uint32_t g = first + v * 64 < total ? first + v * 64 : total - 1;
        row[v] = g / nspan;
        sp[v] = g - row[v] * nspan;
        const uint32_t d = row[v] % (uint32_t)p.dim;
#pragma unroll
        for (int i = 0; i < K; ++i) w[v][i] = p.w[d * K + i];
        bv[v] = p.bias ? p.bias[d] : 0.0f;
#pragma unroll
        for (int j = 0; j < H; ++j)
            st[v][j] = (sp[v] == 0 && p.state_in) ? p.state_in[(int64_t)row[v] * H + j] : 0.0f;
    }

#pragma unroll
    for (int v = 0; v < kVecPerThread; ++v) {
        if (first + v * 64 >= total) break;
        const int64_t base = (int64_t)row[v] * L;
        float xin[H + kSpan];
#pragma unroll
        for (int i = 0; i < kSpan; ++i) xin[H + i] = cur[v][i];
#pragma unroll
        for (int j = 0; j < H; ++j) xin[j] = sp[v] > 0 ? prev[v][j] : st[v][j];
        float out[kSpan];
#pragma unroll
        for (int i = 0; i < kSpan; ++i) {
            float acc = bv[v];
#pragma unroll
            for (int k = 0; k < K; ++k) acc = __builtin_fmaf(w[v][k], xin[i + k], acc);
            out[i] = p.apply_silu ? silu_f32(acc) : acc;
        }
        store8<OUT>(p.y, base + (int64_t)sp[v] * kSpan, out);
        // the span holding the last input writes the next state: inputs L-H .. L-1
        if (H > 0 && p.state_out && sp[v] == nspan - 1) {
#pragma unroll
            for (int j = 0; j < H; ++j) p.state_out[(int64_t)row[v] * H + j] = xin[kSpan + j];
        }
    }
}

// Every other shape: one span of 8 per thread, element loads with bounds checks.
// A block covers 256 consecutive spans of one row.
template <int IN, int OUT, int K>
__global__ __launch_bounds__(kThreads) void conv1d_fwd(ConvParams p, uint32_t blocks_per_row) {
    constexpr int H = K - 1;
    const int64_t L = p.seqlen;
    const uint32_t blk = blockIdx.x;
    const int64_t row = blk / blocks_per_row;                        // wave-uniform
    const int64_t c = (int64_t)(blk - (uint32_t)row * blocks_per_row) * kThreads + threadIdx.x;
    const int64_t d = (uint32_t)row % (uint32_t)p.dim;
    const int64_t t0 = c * kSpan;
    const int64_t base = row * L;
    if (t0 >= L) return;                         // the row's last block may run past its end

    // xin[0 .. H-1] = inputs t0-H .. t0-1, xin[H .. H+7] = inputs t0 .. t0+7
    float xin[H + kSpan];
#pragma unroll
    for (int i = 0; i < kSpan; ++i) xin[H + i] = t0 + i < L ? Act<IN>::ld(p.x, base + t0 + i) : 0.0f;
#pragma unroll
    for (int j = 0; j < H; ++j) {
        const int64_t s = t0 - H + j;
        xin[j] = s >= 0 ? Act<IN>::ld(p.x, base + s) : (p.state_in ? p.state_in[row * H + (H + s)] : 0.0f);
    }

    float w[K];
#pragma unroll
    for (int i = 0; i < K; ++i) w[i] = p.w[d * K + i];
    const float b = p.bias ? p.bias[d] : 0.0f;
    float out[kSpan];
#pragma unroll
    for (int i = 0; i < kSpan; ++i) {
        float acc = b;
#pragma unroll
        for (int k = 0; k < K; ++k) acc = __builtin_fmaf(w[k], xin[i + k], acc);
        out[i] = p.apply_silu ? silu_f32(acc) : acc;
    }
#pragma unroll
    for (int i = 0; i < kSpan; ++i)
        if (t0 + i < L) st_out<OUT>(p.y, base + t0 + i, out[i]);

    // The span holding the last input writes the next state: inputs L-H .. L-1.
    if (H > 0 && p.state_out && t0 + kSpan >= L) {
#pragma unroll
        for (int j = 0; j < H; ++j) {
            const int64_t s = L - H + j;                  // >= t0 - H: inside xin
            p.state_out[row * H + j] = xin[s - t0 + H];
        }
    }
}

// One byte per row, the state shifted in place: thread per row.
template <int IN, int OUT, int K>
__global__ __launch_bounds__(kThreads) void conv1d_step(ConvParams p) {
    constexpr int H = K - 1;
    const int64_t row = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (row >= p.batch * p.dim) return;
    const int64_t d = row % p.dim;
    float xin[K];
#pragma unroll
    for (int j = 0; j < H; ++j) xin[j] = p.state_out[row * H + j];
    xin[H] = Act<IN>::ld(p.x, row);
    float acc = p.bias ? p.bias[d] : 0.0f;
#pragma unroll
    for (int k = 0; k < K; ++k) acc = __builtin_fmaf(p.w[d * K + k], xin[k], acc);
    st_out<OUT>(p.y, row, p.apply_silu ? silu_f32(acc) : acc);
#pragma unroll
    for (int j = 0; j < H; ++j) p.state_out[row * H + j] = xin[j + 1];
}

}  // namespace conv
}  // namespace mbs
