// verify_rank.hpp -- the top-beta check that ends a speculative verification.
//
// After the byte-level model has scanned the drafted bytes in parallel, each
// drafted byte x_i is accepted when it is among the model's top-beta candidates
// for position i, and the draft is kept up to the furthest position whose bytes
// all pass (Section 3, "Speculative decoding through subword drafting";
// Appendix F, Algorithm 1; beta = 3 in Table 6):
//
//   rank_i   = 1 + #{y : logit_i[y] > logit_i[x_i]}   (vocab + 1 if x_i is out of
//              range or its logit is NaN; a softmax is monotone, so logits suffice)
//   accepted = number of leading positions with rank_i <= beta
//
// One workgroup per batch element with up to 16 waves (one per drafted byte for
// the usual short drafts); wave w ranks positions w, w + nwaves, ...: each lane
// compares vocab/64 logits with the drafted byte's, and the counts are summed
// across the wave.  The first rejected position is folded with an LDS atomic
// minimum, so any draft length works.
#pragma once

#include <hip/hip_runtime.h>

#include "device_math.hpp"

namespace mbs {
namespace rank {

constexpr int kMaxThreads = 1024;

struct RankParams {
    int64_t batch, ndraft, vocab;
    const void *logits;          // (batch, ndraft, vocab) act
    const int32_t *draft;        // (batch, ndraft)
    int32_t beta;
    int32_t *ranks;              // (batch, ndraft) or null
    int32_t *accepted;           // (batch)
    int32_t *last_pos;           // (batch) or null: accepted - 1
};

template <int DT>
__global__ __launch_bounds__(kMaxThreads) void verify_rank(RankParams p) {
    __shared__ int first_reject;
    const int64_t b = blockIdx.x;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    if (threadIdx.x == 0) first_reject = (int)p.ndraft;
    __syncthreads();

    const int nwaves = blockDim.x >> 6;
    for (int64_t i = wave; i < p.ndraft; i += nwaves) {
        const int64_t row = b * p.ndraft + i;
        const int32_t x = p.draft[row];
        const int64_t base = row * p.vocab;
        const bool in_range = x >= 0 && x < p.vocab;
        const float lx = in_range ? Act<DT>::ld(p.logits, base + x) : 0.0f;
        int count = 0;
        for (int64_t y = lane; y < p.vocab; y += 64) count += Act<DT>::ld(p.logits, base + y) > lx ? 1 : 0;
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) count += __shfl_xor(count, off, 64);
        const int32_t r = (in_range && lx == lx) ? 1 + count : (int32_t)(p.vocab + 1);
        if (lane == 0) {
            if (p.ranks) p.ranks[row] = r;
            if (r > p.beta) atomicMin(&first_reject, (int)i);
        }
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        p.accepted[b] = first_reject;
        if (p.last_pos) p.last_pos[b] = first_reject - 1;
    }
}

}  // namespace rank
}  // namespace mbs
