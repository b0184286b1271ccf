// lds_banks.hip -- LDS bank behaviour of gfx950 for the access widths the scan
// kernels use, measured.
//
// A stand-alone program, built by build.py as paper_2401_13660_amd/lds_banks and
// run on the GPU as it is (it prints a markdown table).  Each access pattern gives
// the byte address of every lane of a wave; one dispatch per pattern runs 256
// workgroups of 2 waves, each wave issuing 8,000 LDS instructions of the pattern
// (8 back to back, then a wait) into its own 32 KB of LDS.  The table gives the
// shader cycles per instruction and wave (two waves share a CU's LDS); the bank
// conflicts of each dispatch come from the SQ_LDS_BANK_CONFLICT counter of the
// same program under rocprofv3 --pmc (dispatch 1 is a warm-up, dispatch n + 1 the
// table's row n).
//
// Patterns: strided lanes and groups of consecutive lanes (the bank rules), and
// every LDS access of the time-split forward kernel, in the table layout it had
// first ("old") and in the one laid out by these rules ("new").
#include <hip/hip_runtime.h>

#include <cstdio>
#include <functional>
#include <string>
#include <type_traits>
#include <vector>

namespace {

typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

#define READ8(OP)                                                                                              \
    asm volatile(OP " %0, %8\n " OP " %1, %8\n " OP " %2, %8\n " OP " %3, %8\n " OP " %4, %8\n " OP " %5, %8\n " \
                 OP " %6, %8\n " OP " %7, %8\n s_waitcnt lgkmcnt(0)"                                           \
                 : "=v"(r0), "=v"(r1), "=v"(r2), "=v"(r3), "=v"(r4), "=v"(r5), "=v"(r6), "=v"(r7)            \
                 : "v"(a))
#define WRITE8(OP)                                                                                             \
    asm volatile(OP " %0, %1\n " OP " %0, %2\n " OP " %0, %3\n " OP " %0, %4\n " OP " %0, %5\n " OP " %0, %6\n " \
                 OP " %0, %7\n " OP " %0, %8\n s_waitcnt lgkmcnt(0)"                                           \
                 :: "v"(a), "v"(r0), "v"(r1), "v"(r2), "v"(r3), "v"(r4), "v"(r5), "v"(r6), "v"(r7) : "memory")

constexpr int kIters = 1000;       // x 8 instructions per wave
constexpr int kRegion = 32768;     // LDS bytes per wave

// NB bytes per lane; WRITE: ds_write, else ds_read.  The dynamic LDS area starts
// at offset 0 (the kernel has no static LDS), so wave w's region starts at w * 32 KB.
template <int NB, bool WRITE>
__global__ __launch_bounds__(128) void probe(const unsigned *addrs, float *out, unsigned long long *clk) {
    extern __shared__ __align__(16) unsigned char lds[];
    float *f = reinterpret_cast<float *>(lds);
    for (int i = threadIdx.x; i < 2 * kRegion / 4; i += 128) f[i] = (float)i;
    __syncthreads();
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const unsigned a = wave * (unsigned)kRegion + addrs[lane];
    using T = typename std::conditional<NB == 16, f32x4_t, typename std::conditional<NB == 8, f32x2_t, float>::type>::type;
    T r0{}, r1{}, r2{}, r3{}, r4{}, r5{}, r6{}, r7{};
    r0 += (float)lane;
    const unsigned long long m0 = __builtin_amdgcn_s_memtime();
    for (int i = 0; i < kIters; ++i) {
        if constexpr (!WRITE) {
            if constexpr (NB == 16) READ8("ds_read_b128");
            else if constexpr (NB == 8) READ8("ds_read_b64");
            else READ8("ds_read_b32");
        } else {
            if constexpr (NB == 16) WRITE8("ds_write_b128");
            else if constexpr (NB == 8) WRITE8("ds_write_b64");
            else WRITE8("ds_write_b32");
        }
    }
    const unsigned long long m1 = __builtin_amdgcn_s_memtime();
    const T s = r0 + r1 + r2 + r3 + r4 + r5 + r6 + r7;
    float sv;
    if constexpr (NB == 16) sv = s.x + s.y + s.z + s.w;
    else if constexpr (NB == 8) sv = s.x + s.y;
    else sv = s;
    out[blockIdx.x * 128 + threadIdx.x] = sv;
    if (lane == 0) clk[blockIdx.x * 2 + wave] = m1 - m0;
}

struct Pattern {
    std::string name;
    bool write;
    int nb;
    std::vector<unsigned> a;
};

void add(std::vector<Pattern> &v, const std::string &name, bool write, int nb,
         const std::function<unsigned(int)> &addr) {
    Pattern p{name, write, nb, {}};
    for (int l = 0; l < 64; ++l) p.a.push_back(addr(l));
    v.push_back(p);
}

// The time-split kernel's tables: lane l = 16 j + 2 q + k (channel j, state pair
// q, slice k); 16-byte entries.  Layout: bc row stride and slice pad, dd row
// stride and slice pad, part row stride.
struct Ts2Layout { int s_bc, pad_bc, s_dd, pad_dd, p; };

void add_ts2(std::vector<Pattern> &v, const char *tag, Ts2Layout y) {
    auto J = [](int l) { return l >> 4; };
    auto Q = [](int l) { return (l >> 1) & 7; };
    auto K = [](int l) { return l & 1; };
    auto bc = [&](int t) { return y.s_bc * t + (t >= 16 ? y.pad_bc : 0); };
    auto dd = [&](int r) { return y.s_dd * r + (r >= 8 ? y.pad_dd : 0); };
    auto mk = [&](const std::string &name, bool write, int nb, const std::function<unsigned(int)> &addr) {
        add(v, std::string(tag) + " " + name, write, nb, addr);
    };
    mk("dd write", true, 16, [&](int l) { return (unsigned)(dd(8 * K(l) + Q(l)) + J(l)) * 16; });
    for (int i = 0; i < 4; ++i)
        mk("bc write " + std::to_string(i), true, 16, [&](int l) { return (unsigned)(bc(4 * (2 * J(l) + K(l)) + i) + Q(l)) * 16; });
    for (int tq = 0; tq < 4; ++tq) {
        for (int i = 0; i < 2; ++i)
            mk("dd read " + std::to_string(2 * tq + i), false, 16, [&](int l) { return (unsigned)(dd(8 * K(l) + 2 * tq + i) + J(l)) * 16; });
        for (int i = 0; i < 4; ++i)
            mk("bc read " + std::to_string(4 * tq + i), false, 16, [&](int l) { return (unsigned)(bc(16 * K(l) + 4 * tq + i) + Q(l)) * 16; });
        mk("part write " + std::to_string(tq), true, 16, [&](int l) { return (unsigned)((8 * J(l) + 4 * K(l) + tq) * y.p + Q(l)) * 16; });
    }
    for (int w = 0; w < 8; ++w)
        mk("partial read " + std::to_string(w), false, 8,
           [&](int l) { return (unsigned)((8 * J(l) + 4 * K(l) + (Q(l) >> 1)) * y.p * 16 + (2 * w + (Q(l) & 1)) * 8); });
}

bool ok(hipError_t e, const char *what) {
    if (e == hipSuccess) return true;
    std::fprintf(stderr, "%s: %s\n", what, hipGetErrorString(e));
    return false;
}

}  // namespace

int main() {
    std::vector<Pattern> pats;
    for (int nb : {16, 8}) {
        for (bool w : {false, true}) {
            if (nb == 8 && w) continue;
            const std::string op = std::string("b") + std::to_string(nb * 8) + (w ? " write" : " read");
            for (int stride : {1, 2, 4, 8, 16})
                add(pats, op + ", lanes " + std::to_string(stride * nb) + " bytes apart", w, nb,
                    [=](int l) { return (unsigned)(l * stride * nb); });
            for (int g : {4, 8, 16, 32})
                add(pats, op + ", groups of " + std::to_string(g) + " consecutive lanes 1 KB apart", w, nb,
                    [=](int l) { return (unsigned)((l % g) * nb + 1024 * (l / g)); });
        }
    }
    add_ts2(pats, "time-split, old:", Ts2Layout{10, 8, 5, 0, 10});
    add_ts2(pats, "time-split, new:", Ts2Layout{9, 8, 5, 4, 9});
    for (const Pattern &p : pats)
        for (unsigned x : p.a)
            if (x % p.nb || x + p.nb > (unsigned)kRegion) {
                std::fprintf(stderr, "pattern %s leaves its region\n", p.name.c_str());
                return 2;
            }

    const int blocks = 256;
    unsigned *d_a = nullptr;
    float *d_out = nullptr;
    unsigned long long *d_clk = nullptr;
    if (!ok(hipMalloc(&d_a, 64 * sizeof(unsigned)), "hipMalloc") ||
        !ok(hipMalloc(&d_out, blocks * 128 * sizeof(float)), "hipMalloc") ||
        !ok(hipMalloc(&d_clk, blocks * 2 * sizeof(unsigned long long)), "hipMalloc"))
        return 2;
    std::vector<unsigned long long> clk(blocks * 2);
    auto run = [&](const Pattern &p, double *cycles) {
        if (!ok(hipMemcpy(d_a, p.a.data(), 64 * sizeof(unsigned), hipMemcpyHostToDevice), "copy")) return false;
        const dim3 g(blocks), b(128);
        const size_t sh = 2 * kRegion;
        if (!p.write && p.nb == 16) hipLaunchKernelGGL((probe<16, false>), g, b, sh, 0, d_a, d_out, d_clk);
        if (!p.write && p.nb == 8) hipLaunchKernelGGL((probe<8, false>), g, b, sh, 0, d_a, d_out, d_clk);
        if (p.write && p.nb == 16) hipLaunchKernelGGL((probe<16, true>), g, b, sh, 0, d_a, d_out, d_clk);
        if (!ok(hipGetLastError(), "launch") || !ok(hipDeviceSynchronize(), "kernel")) return false;
        if (!ok(hipMemcpy(clk.data(), d_clk, clk.size() * sizeof(unsigned long long), hipMemcpyDeviceToHost), "copy"))
            return false;
        double s = 0;
        for (unsigned long long c : clk) s += (double)c;
        *cycles = s / (double)clk.size() / (kIters * 8.0);
        return true;
    };
    double c;
    if (!run(pats[0], &c)) return 2;                    // warm-up: dispatch 1
    std::printf("| row | pattern | cycles per instruction and wave |\n|---|---|---|\n");
    for (size_t i = 0; i < pats.size(); ++i) {
        if (!run(pats[i], &c)) return 2;
        std::printf("| %zu | %s | %.2f |\n", i + 1, pats[i].name.c_str(), c);
    }
    (void)hipFree(d_a);
    (void)hipFree(d_out);
    (void)hipFree(d_clk);
    return 0;
}
