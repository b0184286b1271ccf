// bf16_pack_check.hip -- the hardware bf16 pair conversion against the bit-level one.
//
// A stand-alone program, built by build.py as paper_2401_13660_amd/bf16_pack_check
// and run on the GPU by tests/test_gpu_bf16_pack.py.  The kernels store bf16
// outputs through bf16x2_pack (one v_cvt_pk_bf16_f32 per pair); this program
// checks that it gives the bits of f32_to_bf16 (round to nearest even, a NaN kept
// a quiet NaN with its sign) for every one of the 2^32 fp32 patterns, in both
// halves of the pair.  It prints the number of differing results and exits with
// status 0 only when there are none.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstring>
#include <vector>

#include "device_math.hpp"

namespace {

constexpr unsigned kThreads = 1u << 18;                        // 2^14 patterns each
constexpr unsigned kPerThread = (unsigned)((1ull << 32) / kThreads);

// Thread t checks patterns t * kPerThread .. + kPerThread - 1, two per conversion:
// pattern x in the low half and x ^ 0x80000001 (another pattern, so both halves
// see every value) in the high half.
__global__ __launch_bounds__(256) void check(unsigned *bad, unsigned *first) {
    const unsigned tid = blockIdx.x * 256 + threadIdx.x;
    unsigned n = 0, fst = 0xffffffffu;
    for (unsigned i = 0; i < kPerThread; ++i) {
        const unsigned x = tid * kPerThread + i, x2 = x ^ 0x80000001u;
        const float a = __uint_as_float(x), b = __uint_as_float(x2);
        const uint32_t hw = mbs::bf16x2_pack(a, b);
        const uint32_t sw = (uint32_t)mbs::f32_to_bf16(a) | ((uint32_t)mbs::f32_to_bf16(b) << 16);
        if (hw != sw) {
            ++n;
            if (fst == 0xffffffffu) fst = x;
        }
    }
    bad[tid] = n;
    first[tid] = fst;
}

bool ok(hipError_t e, const char *what) {
    if (e == hipSuccess) return true;
    std::fprintf(stderr, "%s: %s\n", what, hipGetErrorString(e));
    return false;
}

}  // namespace

int main() {
    unsigned *d_bad = nullptr, *d_first = nullptr;
    if (!ok(hipMalloc(&d_bad, kThreads * sizeof(unsigned)), "hipMalloc") ||
        !ok(hipMalloc(&d_first, kThreads * sizeof(unsigned)), "hipMalloc"))
        return 2;
    hipLaunchKernelGGL(check, dim3(kThreads / 256), dim3(256), 0, 0, d_bad, d_first);
    if (!ok(hipGetLastError(), "launch") || !ok(hipDeviceSynchronize(), "kernel")) return 2;
    std::vector<unsigned> bad(kThreads), first(kThreads);
    if (!ok(hipMemcpy(bad.data(), d_bad, kThreads * sizeof(unsigned), hipMemcpyDeviceToHost), "copy") ||
        !ok(hipMemcpy(first.data(), d_first, kThreads * sizeof(unsigned), hipMemcpyDeviceToHost), "copy"))
        return 2;
    unsigned long long total = 0;
    int shown = 0;
    for (unsigned t = 0; t < kThreads; ++t) {
        total += bad[t];
        if (first[t] != 0xffffffffu && shown < 8) {
            std::printf("differs at pattern 0x%08x\n", first[t]);
            ++shown;
        }
    }
    std::printf("bf16 pair conversion: %llu of %llu results differ\n", total, 2ull << 32);
    (void)hipFree(d_bad);
    (void)hipFree(d_first);
    return total == 0 ? 0 : 1;
}
