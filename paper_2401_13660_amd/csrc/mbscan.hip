// mbscan.hip -- the C ABI of libmbscan.so: argument checks and kernel dispatch.
//
// Every entry point validates its arguments on the host, enqueues its kernels
// on the caller's stream and returns; see include/mbscan.h for the contract.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include <mutex>

#include "conv1d.hpp"
#include "mbscan.h"
#include "scan_bwd.hpp"
#include "scan_params.hpp"
#include "scan_rowwise.hpp"
#include "scan_step.hpp"
#include "scan_tiled.hpp"
#include "scan_ts2.hpp"
#include "verify_rank.hpp"

namespace {

using mbs::ScanParams;
using mbs::StepParams;

// Every element count the entry points form stays below 2^56, so that byte
// counts (at most 4 bytes per element, times the position count's factor
// already inside the count) and the address ranges of the alias checks stay far
// from overflow.  No device memory comes near it.
constexpr int64_t kMaxElems = int64_t(1) << 56;

bool valid_dtype(int32_t t) { return t == MB_F32 || t == MB_BF16; }
size_t dtype_size(int32_t t) { return t == MB_BF16 ? 2 : 4; }

bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Does [a, a+na) overlap [b, b+nb)?  Null or empty ranges never overlap.
bool overlaps(const void *a, size_t na, const void *b, size_t nb) {
    if (!a || !b || na == 0 || nb == 0) return false;
    const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
    return x < y + nb && y < x + na;
}

// a * b without overflow past kMaxElems (both non-negative).
bool mul_ok(int64_t a, int64_t b, int64_t *out) {
    if (a != 0 && b > kMaxElems / a) return false;
    *out = a * b;
    return true;
}

bool supported_dstate(int64_t n) { return n == 1 || n == 2 || n == 4 || n == 8 || n == 16; }

hipError_t launch(const void *fn, dim3 grid, dim3 block, void *params, void *stream) {
    void *args[] = {params};
    return hipLaunchKernel(fn, grid, block, args, 0, static_cast<hipStream_t>(stream));
}

template <int IN, int OUT, int N>
hipError_t fwd_rowwise(ScanParams &p, void *stream) {
    const int64_t rows = p.batch * p.dim;
    const dim3 block(64), grid((unsigned)((rows + 63) / 64));
    return launch(reinterpret_cast<const void *>(&mbs::scan_fwd_rowwise<IN, OUT, N>), grid, block, &p,
                  stream);
}

// The tiled kernel takes dstate 16 with 16-byte aligned activation rows.
bool tiled_ok(const ScanParams &p, int64_t N, int32_t in_dtype, int32_t out_dtype) {
    // 32-bit lane offsets inside a wave's rows: (16 rows) x L x 4 bytes < 2^32
    if (N != 16 || p.seqlen % 16 != 0 || p.seqlen >= (int64_t(1) << 25)) return false;
    const void *ptrs[] = {p.u, p.delta, p.z, p.Bm, p.Cm, p.y};
    for (const void *q : ptrs)
        if (q && !aligned(q, 16)) return false;
    (void)in_dtype; (void)out_dtype;
    // fewer than 2^30 eight-channel waves: the kernel indexes its waves in 32 bits
    // (with time segments, only shapes of a few thousand waves are multiplied)
    return p.batch * ((p.dim + 7) / 8) < (int64_t(1) << 30);
}

template <int IN, int OUT>
hipError_t fwd_dispatch_n(ScanParams &p, int64_t N, void *stream, float *lent) {
    if (tiled_ok(p, N, IN, OUT)) {
        if (mbs::ts2::takes(p))
            return p.z ? mbs::ts2::fwd_ts2<IN, OUT, true>(p, stream) : mbs::ts2::fwd_ts2<IN, OUT, false>(p, stream);
        return p.z ? mbs::tiled::fwd_tiled<IN, OUT, true>(p, stream, lent)
                   : mbs::tiled::fwd_tiled<IN, OUT, false>(p, stream, lent);
    }
    switch (N) {
        case 1: return fwd_rowwise<IN, OUT, 1>(p, stream);
        case 2: return fwd_rowwise<IN, OUT, 2>(p, stream);
        case 4: return fwd_rowwise<IN, OUT, 4>(p, stream);
        case 8: return fwd_rowwise<IN, OUT, 8>(p, stream);
        default: return fwd_rowwise<IN, OUT, 16>(p, stream);
    }
}

template <int IN, int OUT, int N>
hipError_t step_launch(StepParams &p, void *stream) {
    constexpr int64_t per_block = mbs::kStepRowsPerBlock<N>;
    const dim3 block(256);
    const dim3 grid((unsigned)((p.dim + per_block - 1) / per_block), (unsigned)(p.batch < 65535 ? p.batch : 65535));
    return launch(reinterpret_cast<const void *>(&mbs::scan_step_kernel<IN, OUT, N>), grid, block, &p,
                  stream);
}

template <int IN, int OUT>
hipError_t step_dispatch_n(StepParams &p, int64_t N, void *stream) {
    switch (N) {
        case 1: return step_launch<IN, OUT, 1>(p, stream);
        case 2: return step_launch<IN, OUT, 2>(p, stream);
        case 4: return step_launch<IN, OUT, 4>(p, stream);
        case 8: return step_launch<IN, OUT, 8>(p, stream);
        default: return step_launch<IN, OUT, 16>(p, stream);
    }
}

template <int IN, int OUT, int K>
hipError_t conv_fwd_k(mbs::conv::ConvParams &p, bool vec, void *stream) {
    namespace C = mbs::conv;
    const int64_t nspan = (p.seqlen + C::kSpan - 1) / C::kSpan;
    const dim3 block(C::kThreads);
    if (vec) {
        uint32_t ns = (uint32_t)nspan, total = (uint32_t)(p.batch * p.dim * nspan);
        const int64_t per_block = C::kThreads * C::kVecPerThread;
        const dim3 grid((unsigned)((total + per_block - 1) / per_block));
        void *args[] = {&p, &ns, &total};
        return hipLaunchKernel(reinterpret_cast<const void *>(&C::conv1d_fwd_vec<IN, OUT, K>), grid, block,
                               args, 0, static_cast<hipStream_t>(stream));
    }
    uint32_t per_row = (uint32_t)((nspan + C::kThreads - 1) / C::kThreads);
    const dim3 grid((unsigned)(p.batch * p.dim * (int64_t)per_row));
    void *args[] = {&p, &per_row};
    return hipLaunchKernel(reinterpret_cast<const void *>(&C::conv1d_fwd<IN, OUT, K>), grid, block, args, 0,
                           static_cast<hipStream_t>(stream));
}

template <int IN, int OUT, int K>
hipError_t conv_step_k(mbs::conv::ConvParams &p, void *stream) {
    namespace C = mbs::conv;
    const int64_t rows = p.batch * p.dim;
    const dim3 block(C::kThreads), grid((unsigned)((rows + C::kThreads - 1) / C::kThreads));
    return launch(reinterpret_cast<const void *>(&C::conv1d_step<IN, OUT, K>), grid, block, &p, stream);
}

template <int IN, int OUT>
hipError_t conv_dispatch(mbs::conv::ConvParams &p, int K, bool step, bool vec, void *stream) {
    switch (K) {
        case 1: return step ? conv_step_k<IN, OUT, 1>(p, stream) : conv_fwd_k<IN, OUT, 1>(p, vec, stream);
        case 2: return step ? conv_step_k<IN, OUT, 2>(p, stream) : conv_fwd_k<IN, OUT, 2>(p, vec, stream);
        case 3: return step ? conv_step_k<IN, OUT, 3>(p, stream) : conv_fwd_k<IN, OUT, 3>(p, vec, stream);
        default: return step ? conv_step_k<IN, OUT, 4>(p, stream) : conv_fwd_k<IN, OUT, 4>(p, vec, stream);
    }
}

hipError_t conv_launch(mbs::conv::ConvParams &p, int32_t in_dtype, int32_t out_dtype, int K, bool step,
                       bool vec, void *stream) {
    if (in_dtype == MB_F32)
        return out_dtype == MB_F32 ? conv_dispatch<0, 0>(p, K, step, vec, stream)
                                   : conv_dispatch<0, 1>(p, K, step, vec, stream);
    return out_dtype == MB_F32 ? conv_dispatch<1, 0>(p, K, step, vec, stream)
                               : conv_dispatch<1, 1>(p, K, step, vec, stream);
}

__global__ void zero_f32(float *p, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0.0f;
}

hipError_t zero_async(float *p, int64_t n, hipStream_t st) {
    if (!p || n <= 0) return hipSuccess;
    void *args[] = {&p, &n};
    return hipLaunchKernel(reinterpret_cast<const void *>(&zero_f32), dim3((unsigned)((n + 255) / 256)),
                           dim3(256), args, 0, st);
}

// The backward's dB/dC partials come one per 8-channel group, or one per
// workgroup of 4 groups: when the group count is a multiple of 4 (no workgroup
// spans two batch elements) and there are at least 1,536 waves (1.5 per SIMD, so
// that the other workgroup's waves fill a SIMD while one waits at the
// workgroup's barrier every 4 steps), the workgroup sums its waves' terms in LDS.
bool bwd_workgroup_sum(int64_t batch, int64_t dim, int64_t nseg) {
    namespace W = mbs::bwd;
    const int64_t n_cg = (dim + W::kCh - 1) / W::kCh;
    return n_cg % W::kWaves == 0 && n_cg * batch * nseg >= 1536;
}

int64_t bwd_partial_groups(int64_t batch, int64_t dim, int64_t nseg) {
    namespace W = mbs::bwd;
    const int64_t n_cg = (dim + W::kCh - 1) / W::kCh;
    return bwd_workgroup_sum(batch, dim, nseg) ? n_cg / W::kWaves : n_cg;
}

// Time segments of the backward.  Its kernel needs up to 256 VGPRs, so 2 waves
// share a SIMD; with at most half that many 8-channel waves the sequence is cut
// into the most segments that fill the chip once, each at least 256 bytes and a
// multiple of 32.  The aggregate pre-pass costs about a quarter of the backward's
// work per timestep, well below what the extra waves return.  The pre-pass cuts
// each segment into `pieces` (1, 2 or 4), the most that keep its waves at 4 per
// SIMD or fewer: one wave alone on a SIMD waits on its chain of dependent
// operations, and up to 4 interleave.  Segments are then a multiple of 16 x pieces
// timesteps (and of 32).
int64_t bwd_segments(int64_t batch, int64_t dim, int64_t L, int64_t *seg_len, int64_t *pieces) {
    namespace W = mbs::bwd;
    const int64_t waves = (dim + W::kCh - 1) / W::kCh * batch;
    int64_t nseg = 1;
    if (L >= 512 && waves > 0) {
        const int64_t resident = mbs::tiled::resident_waves();   // 2 waves per SIMD, as here
        if (2 * waves <= resident) nseg = resident / waves;
        if (nseg > L / 256) nseg = L / 256;
        if (nseg < 1) nseg = 1;
    }
    int64_t m = 1;
    if (nseg > 1) {
        const int64_t simds = 4 * mbs::tiled::device_cus();
        while (m < 4 && 2 * m * waves * (nseg - 1) <= 4 * simds) m *= 2;
    }
    const int64_t unit = 16 * m > 32 ? 16 * m : 32;
    int64_t len = (L + nseg - 1) / nseg;
    len = (len + unit - 1) / unit * unit;
    *seg_len = len;
    *pieces = m;
    return (L + len - 1) / len;
}

template <int IN, int OUT, bool GATE, bool SP>
hipError_t bwd_launch(mbs::bwd::BwdParams &p, bool have_ck, float *dA, float *dB, float *dC, float *dD,
                      float *dbias, hipStream_t st) {
    namespace W = mbs::bwd;
    const int64_t n_cg = (p.dim + W::kCh - 1) / W::kCh;
    const int64_t nseg = (p.seqlen + p.seg_len - 1) / p.seg_len;
    const int64_t ck_nseg = (p.seqlen + p.ck_seg_len - 1) / p.ck_seg_len;
    const int64_t waves = n_cg * p.batch;
    const dim3 grid((unsigned)((waves + W::kWaves - 1) / W::kWaves)), block(W::kThreads);
    const dim3 grid_seg((unsigned)((waves * nseg + W::kWaves - 1) / W::kWaves));
    const size_t lds = sizeof(W::WaveSmem) * W::kWaves;
    void *args[] = {&p};
    hipError_t e = hipSuccess;
    if (!have_ck && ck_nseg > 1) {
        // the forward pre-pass: each segment's state aggregate, for scan_ckpt's carry-in
        mbs::ScanParams f{};
        f.batch = p.batch; f.dim = p.dim; f.seqlen = p.seqlen;
        f.u = p.u; f.delta = p.delta; f.Bm = p.Bm; f.Cm = p.Cm;
        f.A = p.A; f.dt_bias = p.dt_bias;
        f.delta_softplus = p.delta_softplus;
        int64_t seg_len = p.ck_seg_len, npieces = ck_nseg - 1;   // one piece per segment
        float *fagg = const_cast<float *>(p.fagg);
        void *fargs[] = {&f, &seg_len, &npieces, &fagg};
        namespace T = mbs::tiled;
        const dim3 grid_pre((unsigned)((waves * (ck_nseg - 1) + T::kWavesPerGroup - 1) / T::kWavesPerGroup));
        e = hipLaunchKernel(reinterpret_cast<const void *>(&T::scan_seg_agg<IN, SP>), grid_pre, dim3(T::kThreads),
                            fargs, sizeof(T::WaveSmemPre) * T::kWavesPerGroup, st);
        if (e != hipSuccess) return e;
    }
    if (!have_ck) {
        const dim3 grid_ck((unsigned)((waves * ck_nseg + W::kWaves - 1) / W::kWaves));
        e = hipLaunchKernel(reinterpret_cast<const void *>(&W::scan_ckpt<IN, SP>), grid_ck, block, args, lds, st);
    }
    if (e != hipSuccess) return e;
    if (nseg > 1) {
        const dim3 grid_agg((unsigned)((waves * p.agg_pieces * (nseg - 1) + W::kWaves - 1) / W::kWaves));
        e = hipLaunchKernel(reinterpret_cast<const void *>(&W::bwd_seg_aggregate<IN, OUT, GATE, SP>), grid_agg,
                            block, args, sizeof(W::AggSmem) * W::kWaves, st);
        if (e != hipSuccess) return e;
    }
    if (bwd_workgroup_sum(p.batch, p.dim, nseg))
        e = hipLaunchKernel(reinterpret_cast<const void *>(&W::scan_bwd<IN, OUT, GATE, SP, true>), grid_seg,
                            block, args, lds, st);               // + its static exchange area
    else
        e = hipLaunchKernel(reinterpret_cast<const void *>(&W::scan_bwd<IN, OUT, GATE, SP, false>), grid_seg,
                            block, args, lds, st);
    if (e != hipSuccess) return e;
    int64_t ncg = bwd_partial_groups(p.batch, p.dim, nseg);
    void *fargs[] = {&p, &dB, &dC, &ncg};
    const int64_t nbc = p.batch * p.seqlen * W::kQ;
    e = hipLaunchKernel(reinterpret_cast<const void *>(&W::bwd_finish_bc), dim3((unsigned)((nbc + 255) / 256)),
                        dim3(256), fargs, 0, st);
    if (e != hipSuccess) return e;
    void *rargs[] = {&p, &dA, &dD, &dbias};
    const int64_t nr = p.dim * (W::kN + 2);
    return hipLaunchKernel(reinterpret_cast<const void *>(&W::bwd_finish_rows), dim3((unsigned)((nr + 255) / 256)),
                           dim3(256), rargs, 0, st);
}

template <int IN, int OUT>
hipError_t bwd_dispatch(mbs::bwd::BwdParams &p, bool have_ck, float *dA, float *dB, float *dC, float *dD,
                        float *dbias, hipStream_t st) {
    if (p.z)
        return p.delta_softplus ? bwd_launch<IN, OUT, true, true>(p, have_ck, dA, dB, dC, dD, dbias, st)
                                : bwd_launch<IN, OUT, true, false>(p, have_ck, dA, dB, dC, dD, dbias, st);
    return p.delta_softplus ? bwd_launch<IN, OUT, false, true>(p, have_ck, dA, dB, dC, dD, dbias, st)
                            : bwd_launch<IN, OUT, false, false>(p, have_ck, dA, dB, dC, dD, dbias, st);
}

}  // namespace

extern "C" {

int mb_abi_version(void) { return MB_ABI_VERSION; }

const char *mb_status_string(int status) {
    switch (status) {
        case MB_OK: return "ok";
        case MB_ERR_NULL: return "a required pointer is NULL";
        case MB_ERR_SHAPE: return "a size is negative or too large";
        case MB_ERR_DTYPE: return "unknown element type";
        case MB_ERR_ALIGN: return "a pointer is not aligned to its element size";
        case MB_ERR_UNSUPPORTED: return "unsupported dstate or convolution width, or reserved field set";
        case MB_ERR_HIP: return "the HIP runtime failed to launch a kernel";
        case MB_ERR_ALIAS: return "an output overlaps an input";
        default: return "unknown status";
    }
}

}  // extern "C"

namespace {

// ---- the scratch array of mb_scan_fwd_noalloc ------------------------------
//
// Each GPU the library runs on holds one copy of `scratch` until the process
// ends.  In host code the name is only a stand-in for the device symbol: the
// device address of this GPU's copy comes from hipGetSymbolAddress, looked up
// once per device with that device current and kept in scratch_dev[].
constexpr size_t kScratchBytes = size_t(8) << 20;
constexpr int kMaxDevices = 64;
void *scratch_dev[kMaxDevices];
std::mutex scratch_mu;

}  // namespace

__device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

// The device address of the current device's scratch array.
int scratch_for_current_device(void **out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return MB_ERR_HIP;
    if (dev < 0 || dev >= kMaxDevices) return MB_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(scratch_mu);
    if (!scratch_dev[dev]) {
        void *ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return MB_ERR_HIP;
        scratch_dev[dev] = ptr;
    }
    *out = scratch_dev[dev];
    return MB_OK;
}

// The forward scan behind mb_scan_fwd, mb_scan_fwd_states and mb_scan_fwd_ckpt.
int scan_fwd_impl(const mb_scan_desc *desc, const void *u, const void *delta, const float *A,
                  const void *Bmat, const void *Cmat, const float *Dskip, const float *dt_bias,
                  const void *z, const float *h0, void *y, float *h_last, const int32_t *pos,
                  int64_t npos, float *h_pos, float *ck, void *stream, bool no_alloc = false) {
    if (!desc) return MB_ERR_NULL;
    const int64_t B = desc->batch, D = desc->dim, L = desc->seqlen, N = desc->dstate;
    if (B < 0 || D < 0 || L < 0 || N < 0) return MB_ERR_SHAPE;
    if (!valid_dtype(desc->in_dtype) || !valid_dtype(desc->out_dtype)) return MB_ERR_DTYPE;
    if (desc->reserved != 0 || !supported_dstate(N)) return MB_ERR_UNSUPPORTED;
    int64_t rows, elems, bn, bc_elems, state_elems, pos_elems = 0, hpos_elems = 0;
    if (npos < 0) return MB_ERR_SHAPE;
    if (!mul_ok(B, D, &rows) || !mul_ok(rows, L, &elems) || !mul_ok(B, N, &bn) || !mul_ok(bn, L, &bc_elems) ||
        !mul_ok(rows, N, &state_elems) || !mul_ok(npos, B, &pos_elems) ||
        !mul_ok(npos, state_elems, &hpos_elems))
        return MB_ERR_SHAPE;
    if (rows == 0) return MB_OK;

    if (!A) return MB_ERR_NULL;
    if (L > 0 && (!u || !delta || !Bmat || !Cmat || !y)) return MB_ERR_NULL;
    if (npos > 0 && (!pos || !h_pos)) return MB_ERR_NULL;
    if (npos > 0 && (!aligned(pos, 4) || !aligned(h_pos, 4))) return MB_ERR_ALIGN;

    const size_t in_sz = dtype_size(desc->in_dtype), out_sz = dtype_size(desc->out_dtype);
    const void *act[] = {u, delta, Bmat, Cmat, z};
    for (const void *p : act)
        if (p && !aligned(p, in_sz)) return MB_ERR_ALIGN;
    const void *f32s[] = {A, Dskip, dt_bias, h0, h_last};
    for (const void *p : f32s)
        if (p && !aligned(p, 4)) return MB_ERR_ALIGN;
    if (y && !aligned(y, out_sz)) return MB_ERR_ALIGN;

    // y may overlap nothing; h_last may only coincide exactly with h0.
    const size_t act_bytes = (size_t)elems * in_sz, bc_bytes = (size_t)bc_elems * in_sz;
    const size_t st_bytes = (size_t)state_elems * 4, a_bytes = (size_t)(D * N) * 4, v_bytes = (size_t)D * 4;
    struct Range { const void *p; size_t n; } ins[] = {
        {u, act_bytes}, {delta, act_bytes}, {z, act_bytes}, {Bmat, bc_bytes}, {Cmat, bc_bytes},
        {A, a_bytes}, {Dskip, v_bytes}, {dt_bias, v_bytes}, {h0, st_bytes}};
    const size_t y_bytes = (size_t)elems * out_sz;
    for (const Range &r : ins) {
        if (overlaps(y, y_bytes, r.p, r.n)) return MB_ERR_ALIAS;
        if (r.p == h0) continue;
        if (overlaps(h_last, st_bytes, r.p, r.n)) return MB_ERR_ALIAS;
    }
    if (overlaps(h_last, st_bytes, y, y_bytes)) return MB_ERR_ALIAS;
    if (h0 && h_last && h0 != h_last && overlaps(h_last, st_bytes, h0, st_bytes)) return MB_ERR_ALIAS;
    if (npos > 0) {
        // h_pos overlaps nothing; pos is an input like the others.
        const size_t pos_bytes = (size_t)pos_elems * 4, hpos_bytes = (size_t)hpos_elems * 4;
        for (const Range &r : ins)
            if (overlaps(h_pos, hpos_bytes, r.p, r.n)) return MB_ERR_ALIAS;
        if (overlaps(h_pos, hpos_bytes, pos, pos_bytes) || overlaps(h_pos, hpos_bytes, y, y_bytes) ||
            overlaps(h_pos, hpos_bytes, h_last, st_bytes) || overlaps(pos, pos_bytes, y, y_bytes) ||
            overlaps(pos, pos_bytes, h_last, st_bytes))
            return MB_ERR_ALIAS;
    }

    ScanParams p{};
    p.batch = B; p.dim = D; p.seqlen = L;
    p.u = u; p.delta = delta; p.Bm = Bmat; p.Cm = Cmat; p.z = z;
    p.A = A; p.Dskip = Dskip; p.dt_bias = dt_bias; p.h0 = h0;
    p.y = y; p.h_last = h_last;
    p.pos = npos > 0 ? pos : nullptr; p.npos = npos; p.h_pos = npos > 0 ? h_pos : nullptr;
    p.ck = nullptr;
    p.delta_softplus = desc->delta_softplus ? 1 : 0;

    if (ck) {
        // checkpoints exist on the tiled path only: dstate 16, L a multiple of 16,
        // 16-byte aligned activations and y
        if (N != 16 || L % 16 != 0 || L >= (int64_t(1) << 25)) return MB_ERR_UNSUPPORTED;
        const void *a16[] = {u, delta, z, Bmat, Cmat, y};
        for (const void *q : a16)
            if (q && !aligned(q, 16)) return MB_ERR_ALIGN;
        if (!aligned(ck, 8)) return MB_ERR_ALIGN;
        const size_t ck_bytes = (size_t)elems * 4;        // (L / 16) x rows x 16 floats
        for (const Range &r : ins)
            if (overlaps(ck, ck_bytes, r.p, r.n)) return MB_ERR_ALIAS;
        if (overlaps(ck, ck_bytes, y, y_bytes) || overlaps(ck, ck_bytes, h_last, st_bytes)) return MB_ERR_ALIAS;
        if (L > 0 && !tiled_ok(p, N, desc->in_dtype, desc->out_dtype)) return MB_ERR_UNSUPPORTED;
        p.ck = ck;
    }

    if (npos > 0) {
        // Position -1 and invalid positions, before h_last (which may be h0) is written.
        const dim3 block(256), grid((unsigned)((hpos_elems + 255) / 256));
        int64_t n_arg = N;
        void *args[] = {&p, &n_arg};
        const hipError_t e = hipLaunchKernel(reinterpret_cast<const void *>(&mbs::init_positions), grid,
                                             block, args, 0, static_cast<hipStream_t>(stream));
        if (e != hipSuccess) return MB_ERR_HIP;
    }

    if (L == 0) {
        if (!h_last || h_last == h0) return MB_OK;
        struct { const float *h0; float *h_last; int64_t n; } cp{h0, h_last, state_elems};
        void *args[] = {&cp.h0, &cp.h_last, &cp.n};
        const dim3 block(256), grid((unsigned)((state_elems + 255) / 256));
        const hipError_t e = hipLaunchKernel(reinterpret_cast<const void *>(&mbs::copy_state), grid, block,
                                             args, 0, static_cast<hipStream_t>(stream));
        return e == hipSuccess ? MB_OK : MB_ERR_HIP;
    }

    float *lent = nullptr;
    if (no_alloc && tiled_ok(p, N, desc->in_dtype, desc->out_dtype)) {
        // the segment carry lives in this device's copy of the static scratch array
        int64_t seg_len, pieces;
        const int64_t nseg = mbs::tiled::fwd_segments(p, &seg_len, &pieces);
        const size_t need = mbs::tiled::fwd_carry_bytes(p, nseg, pieces);
        if (need > kScratchBytes) return MB_ERR_SHAPE;
        if (need > 0) {
            const int st = scratch_for_current_device(reinterpret_cast<void **>(&lent));
            if (st != MB_OK) return st;
        }
    }

    hipError_t e;
    if (desc->in_dtype == MB_F32)
        e = desc->out_dtype == MB_F32 ? fwd_dispatch_n<0, 0>(p, N, stream, lent)
                                      : fwd_dispatch_n<0, 1>(p, N, stream, lent);
    else
        e = desc->out_dtype == MB_F32 ? fwd_dispatch_n<1, 0>(p, N, stream, lent)
                                      : fwd_dispatch_n<1, 1>(p, N, stream, lent);
    return e == hipSuccess ? MB_OK : MB_ERR_HIP;
}

}  // namespace

extern "C" {

int mb_scan_fwd(const mb_scan_desc *desc, const void *u, const void *delta, const float *A,
                const void *Bmat, const void *Cmat, const float *Dskip, const float *dt_bias,
                const void *z, const float *h0, void *y, float *h_last, void *stream) {
    return scan_fwd_impl(desc, u, delta, A, Bmat, Cmat, Dskip, dt_bias, z, h0, y, h_last, nullptr, 0, nullptr,
                         nullptr, stream);
}

int mb_scan_fwd_noalloc(const mb_scan_desc *desc, const void *u, const void *delta, const float *A,
                        const void *Bmat, const void *Cmat, const float *Dskip, const float *dt_bias,
                        const void *z, const float *h0, void *y, float *h_last, void *stream) {
    return scan_fwd_impl(desc, u, delta, A, Bmat, Cmat, Dskip, dt_bias, z, h0, y, h_last, nullptr, 0, nullptr,
                         nullptr, stream, true);
}

int mb_scan_fwd_states(const mb_scan_desc *desc, const void *u, const void *delta, const float *A,
                       const void *Bmat, const void *Cmat, const float *Dskip, const float *dt_bias,
                       const void *z, const float *h0, void *y, float *h_last, const int32_t *pos,
                       int64_t npos, float *h_pos, void *stream) {
    return scan_fwd_impl(desc, u, delta, A, Bmat, Cmat, Dskip, dt_bias, z, h0, y, h_last, pos, npos, h_pos,
                         nullptr, stream);
}

int mb_scan_fwd_ckpt(const mb_scan_desc *desc, const void *u, const void *delta, const float *A,
                     const void *Bmat, const void *Cmat, const float *Dskip, const float *dt_bias,
                     const void *z, const float *h0, void *y, float *h_last, float *ck, void *stream) {
    if (!ck) return MB_ERR_NULL;
    return scan_fwd_impl(desc, u, delta, A, Bmat, Cmat, Dskip, dt_bias, z, h0, y, h_last, nullptr, 0, nullptr,
                         ck, stream);
}

int mb_conv1d_fwd(const mb_conv_desc *desc, const void *x, const float *w, const float *bias,
                  const float *state_in, void *y, float *state_out, void *stream) {
    if (!desc) return MB_ERR_NULL;
    const int64_t B = desc->batch, D = desc->dim, L = desc->seqlen, K = desc->width;
    if (B < 0 || D < 0 || L < 0) return MB_ERR_SHAPE;
    if (!valid_dtype(desc->in_dtype) || !valid_dtype(desc->out_dtype)) return MB_ERR_DTYPE;
    if (K < 1 || K > mbs::conv::kMaxK || desc->reserved != 0 || desc->reserved2 != 0) return MB_ERR_UNSUPPORTED;
    int64_t rows, elems, st_elems;
    if (!mul_ok(B, D, &rows) || !mul_ok(rows, L, &elems) || !mul_ok(rows, K - 1, &st_elems))
        return MB_ERR_SHAPE;
    if (rows == 0) return MB_OK;
    if (!w) return MB_ERR_NULL;
    if (L > 0 && (!x || !y)) return MB_ERR_NULL;
    const size_t in_sz = dtype_size(desc->in_dtype), out_sz = dtype_size(desc->out_dtype);
    if ((x && !aligned(x, in_sz)) || (y && !aligned(y, out_sz))) return MB_ERR_ALIGN;
    const void *f32s[] = {w, bias, state_in, state_out};
    for (const void *q : f32s)
        if (q && !aligned(q, 4)) return MB_ERR_ALIGN;
    // Outputs overlap nothing (state_out may not even be state_in: the span that
    // writes it is not the one that reads state_in).
    const size_t x_bytes = (size_t)elems * in_sz, y_bytes = (size_t)elems * out_sz;
    const size_t st_bytes = (size_t)st_elems * 4;
    struct Range { const void *p; size_t n; } ins[] = {
        {x, x_bytes}, {w, (size_t)(D * K) * 4}, {bias, (size_t)D * 4}, {state_in, st_bytes}};
    for (const Range &r : ins)
        if (overlaps(y, y_bytes, r.p, r.n) || overlaps(state_out, st_bytes, r.p, r.n)) return MB_ERR_ALIAS;
    if (overlaps(y, y_bytes, state_out, st_bytes)) return MB_ERR_ALIAS;

    mbs::conv::ConvParams p{};
    p.batch = B; p.dim = D; p.seqlen = L;
    p.x = x; p.w = w; p.bias = bias; p.state_in = state_in; p.y = y; p.state_out = state_out;
    p.apply_silu = desc->apply_silu ? 1 : 0;
    hipError_t e;
    if (L == 0) {
        // nothing to convolve: the next state is the carried one (or zeros)
        if (!state_out || K == 1) return MB_OK;
        void *args[] = {&p.state_in, &p.state_out, &st_elems};
        const dim3 block(256), grid((unsigned)((st_elems + 255) / 256));
        e = hipLaunchKernel(reinterpret_cast<const void *>(&mbs::copy_state), grid, block, args, 0,
                            static_cast<hipStream_t>(stream));
        return e == hipSuccess ? MB_OK : MB_ERR_HIP;
    }
    // 32-bit span and block indices: rows * ceil(L / 8) spans below 2^31
    const int64_t nspan = (L + mbs::conv::kSpan - 1) / mbs::conv::kSpan;
    if (nspan > (int64_t(1) << 31) / rows) return MB_ERR_SHAPE;
    const bool vec = L % mbs::conv::kSpan == 0 && aligned(x, 16) && aligned(y, 16);
    e = conv_launch(p, desc->in_dtype, desc->out_dtype, (int)K, false, vec, stream);
    return e == hipSuccess ? MB_OK : MB_ERR_HIP;
}

int mb_conv1d_step(int64_t batch, int64_t dim, int32_t width, int32_t in_dtype, int32_t out_dtype,
                   int32_t apply_silu, const void *x_t, const float *w, const float *bias, float *state,
                   void *y_t, void *stream) {
    if (batch < 0 || dim < 0) return MB_ERR_SHAPE;
    if (!valid_dtype(in_dtype) || !valid_dtype(out_dtype)) return MB_ERR_DTYPE;
    if (width < 1 || width > mbs::conv::kMaxK) return MB_ERR_UNSUPPORTED;
    int64_t rows, st_elems;
    if (!mul_ok(batch, dim, &rows) || !mul_ok(rows, width - 1, &st_elems)) return MB_ERR_SHAPE;
    if (rows == 0) return MB_OK;
    if (!x_t || !w || !y_t || (width > 1 && !state)) return MB_ERR_NULL;
    const size_t in_sz = dtype_size(in_dtype), out_sz = dtype_size(out_dtype);
    if (!aligned(x_t, in_sz) || !aligned(y_t, out_sz)) return MB_ERR_ALIGN;
    const void *f32s[] = {w, bias, state};
    for (const void *q : f32s)
        if (q && !aligned(q, 4)) return MB_ERR_ALIGN;
    const size_t st_bytes = (size_t)st_elems * 4, y_bytes = (size_t)rows * out_sz;
    struct Range { const void *p; size_t n; } ins[] = {
        {x_t, (size_t)rows * in_sz}, {w, (size_t)(dim * width) * 4}, {bias, (size_t)dim * 4}};
    for (const Range &r : ins)
        if (overlaps(y_t, y_bytes, r.p, r.n) || overlaps(state, st_bytes, r.p, r.n)) return MB_ERR_ALIAS;
    if (overlaps(y_t, y_bytes, state, st_bytes)) return MB_ERR_ALIAS;

    mbs::conv::ConvParams p{};
    p.batch = batch; p.dim = dim; p.seqlen = 1;
    p.x = x_t; p.w = w; p.bias = bias; p.state_in = state; p.y = y_t; p.state_out = state;
    p.apply_silu = apply_silu ? 1 : 0;
    const hipError_t e = conv_launch(p, in_dtype, out_dtype, width, true, false, stream);
    return e == hipSuccess ? MB_OK : MB_ERR_HIP;
}

int mb_scan_bwd(const mb_scan_desc *desc, const void *u, const void *delta, const float *A,
                const void *Bmat, const void *Cmat, const float *Dskip, const float *dt_bias,
                const void *z, const float *h0, const void *dy, const float *dh_last, const float *ck,
                void *du, void *ddelta, void *dz, float *dA, float *dB, float *dC, float *dDskip,
                float *ddt_bias, float *dh0, void *stream) {
    if (!desc) return MB_ERR_NULL;
    const int64_t B = desc->batch, D = desc->dim, L = desc->seqlen, N = desc->dstate;
    if (B < 0 || D < 0 || L < 0 || N < 0) return MB_ERR_SHAPE;
    if (!valid_dtype(desc->in_dtype) || !valid_dtype(desc->out_dtype)) return MB_ERR_DTYPE;
    // 32-bit lane offsets inside a wave's rows: (16 rows) x L x 4 bytes < 2^32
    if (desc->reserved != 0 || N != 16 || L % 16 != 0 || L >= (int64_t(1) << 25)) return MB_ERR_UNSUPPORTED;
    int64_t rows, elems, bn, bc_elems, state_elems;
    if (!mul_ok(B, D, &rows) || !mul_ok(rows, L, &elems) || !mul_ok(B, N, &bn) || !mul_ok(bn, L, &bc_elems) ||
        !mul_ok(rows, N, &state_elems))
        return MB_ERR_SHAPE;
    if (L >= (int64_t(1) << 31) || rows >= (int64_t(1) << 31)) return MB_ERR_SHAPE;
    if (rows == 0) {
        // no row: the parameter gradients are sums over nothing
        if (D == 0) return MB_OK;
        if (!dA || (Dskip && !dDskip) || (dt_bias && !ddt_bias)) return MB_ERR_NULL;
        const void *f32z[] = {dA, dDskip, ddt_bias};
        for (const void *q : f32z)
            if (q && !aligned(q, 4)) return MB_ERR_ALIGN;
        hipStream_t st0 = static_cast<hipStream_t>(stream);
        hipError_t e0 = zero_async(dA, D * N, st0);
        if (e0 == hipSuccess) e0 = zero_async(Dskip ? dDskip : nullptr, D, st0);
        if (e0 == hipSuccess) e0 = zero_async(dt_bias ? ddt_bias : nullptr, D, st0);
        return e0 == hipSuccess ? MB_OK : MB_ERR_HIP;
    }
    if (!A || !dA || (Dskip && !dDskip) || (dt_bias && !ddt_bias)) return MB_ERR_NULL;
    if (L > 0 && (!u || !delta || !Bmat || !Cmat || !dy || !du || !ddelta || !dB || !dC || (z && !dz)))
        return MB_ERR_NULL;
    const size_t in_sz = dtype_size(desc->in_dtype), out_sz = dtype_size(desc->out_dtype);
    const void *act_in[] = {u, delta, z, Bmat, Cmat};
    for (const void *q : act_in)
        if (q && !aligned(q, 16)) return MB_ERR_ALIGN;
    const void *act_out[] = {dy, du, ddelta, dz};
    for (const void *q : act_out)
        if (q && !aligned(q, 16)) return MB_ERR_ALIGN;
    const void *f32s[] = {A, Dskip, dt_bias, h0, dh_last, ck, dA, dB, dC, dDskip, ddt_bias, dh0};
    for (const void *q : f32s)
        if (q && !aligned(q, 8)) return MB_ERR_ALIGN;
    // outputs overlap nothing
    const size_t in_b = (size_t)elems * in_sz, out_b = (size_t)elems * out_sz, bc_b = (size_t)bc_elems * in_sz;
    const size_t st_b = (size_t)state_elems * 4, a_b = (size_t)(D * N) * 4, v_b = (size_t)D * 4;
    struct Range { const void *p; size_t n; };
    const Range ins[] = {{u, in_b}, {delta, in_b}, {z, in_b}, {Bmat, bc_b}, {Cmat, bc_b}, {A, a_b},
                         {Dskip, v_b}, {dt_bias, v_b}, {h0, st_b}, {dy, out_b}, {dh_last, st_b},
                         {ck, (size_t)elems * 4}};
    const Range outs[] = {{du, out_b}, {ddelta, out_b}, {dz, z ? out_b : 0}, {dA, a_b},
                          {dB, (size_t)bc_elems * 4}, {dC, (size_t)bc_elems * 4}, {dDskip, v_b},
                          {ddt_bias, v_b}, {dh0, st_b}};
    const int n_out = sizeof(outs) / sizeof(outs[0]);
    for (int i = 0; i < n_out; ++i) {
        for (const Range &r : ins)
            if (overlaps(outs[i].p, outs[i].n, r.p, r.n)) return MB_ERR_ALIAS;
        for (int k = i + 1; k < n_out; ++k)
            if (overlaps(outs[i].p, outs[i].n, outs[k].p, outs[k].n)) return MB_ERR_ALIAS;
    }

    hipStream_t st = static_cast<hipStream_t>(stream);
    hipError_t e;
    if (L == 0) {
        // no timestep: the state passes straight through; parameter gradients are zero
        e = zero_async(dA, D * N, st);
        if (e == hipSuccess) e = zero_async(dDskip, Dskip ? D : 0, st);
        if (e == hipSuccess) e = zero_async(ddt_bias, dt_bias ? D : 0, st);
        if (e == hipSuccess && dh0) {
            void *args[] = {const_cast<float **>(&dh_last), &dh0, &state_elems};
            e = hipLaunchKernel(reinterpret_cast<const void *>(&mbs::copy_state),
                                dim3((unsigned)((state_elems + 255) / 256)), dim3(256), args, 0, st);
        }
        return e == hipSuccess ? MB_OK : MB_ERR_HIP;
    }

    namespace W = mbs::bwd;
    int64_t seg_len = L, agg_pieces = 1;
    const int64_t nseg = bwd_segments(B, D, L, &seg_len, &agg_pieces);
    const int64_t n_cg = bwd_partial_groups(B, D, nseg);       // dB/dC partials per (batch, t)
    // each area of the workspace starts on a 256-byte boundary (the kernels move
    // 16-byte vectors in the partials and the forward aggregates)
    auto pad = [](size_t n) { return (n + 255) / 256 * 256; };
    const size_t ck_b = ck ? 0 : pad((size_t)(L / W::kT) * (size_t)rows * W::kN * 4);
    const size_t bcp_b = pad((size_t)n_cg * (size_t)B * (size_t)L * W::kQ * 4 * 4);
    const size_t row_b = pad((size_t)nseg * (size_t)rows * (W::kN + 2) * 4);
    const size_t agg_b = nseg > 1 ? pad((size_t)(agg_pieces * (nseg - 1)) * (size_t)rows * W::kN * 2 * 4) : 0;
    // The checkpoint pass is a forward recurrence: its pre-pass costs as much per
    // timestep as the pass itself, so it takes the segments only with at most a
    // third as many waves as the chip holds.
    const int64_t ck_nseg = (!ck && 3 * ((D + W::kCh - 1) / W::kCh * B) <= mbs::tiled::resident_waves()) ? nseg : 1;
    // the forward pre-pass writes ck_nseg planes: the aggregates of segments
    // 0 .. ck_nseg-2 and a copy of h0 (which scan_ckpt does not need)
    const size_t fagg_b = ck_nseg > 1 ? pad((size_t)ck_nseg * (size_t)rows * W::kN * 2 * 4) : 0;
    char *ws = nullptr;
    e = hipMallocAsync(reinterpret_cast<void **>(&ws), ck_b + bcp_b + row_b + agg_b + fagg_b, st);
    if (e != hipSuccess) return MB_ERR_HIP;
    W::BwdParams p{};
    p.batch = B; p.dim = D; p.seqlen = L;
    p.u = u; p.delta = delta; p.Bm = Bmat; p.Cm = Cmat; p.z = z;
    p.A = A; p.Dskip = Dskip; p.dt_bias = dt_bias; p.h0 = h0;
    p.dy = dy; p.dh_last = dh_last;
    p.du = du; p.ddelta = ddelta; p.dz = dz; p.dh0 = dh0;
    p.ck = ck ? const_cast<float *>(ck) : reinterpret_cast<float *>(ws);   // given: read only
    p.part_bc = reinterpret_cast<float *>(ws + ck_b);
    p.part_row = reinterpret_cast<float *>(ws + ck_b + bcp_b);
    p.seg_len = seg_len;
    p.agg_pieces = agg_pieces;
    p.ck_seg_len = ck_nseg > 1 ? seg_len : (L + 31) / 32 * 32;
    p.agg = nseg > 1 ? reinterpret_cast<float *>(ws + ck_b + bcp_b + row_b) : nullptr;
    p.fagg = fagg_b ? reinterpret_cast<float *>(ws + ck_b + bcp_b + row_b + agg_b) : nullptr;
    p.delta_softplus = desc->delta_softplus ? 1 : 0;
    float *dD = Dskip ? dDskip : nullptr, *dbias = dt_bias ? ddt_bias : nullptr;
    if (desc->in_dtype == MB_F32)
        e = desc->out_dtype == MB_F32 ? bwd_dispatch<0, 0>(p, ck != nullptr, dA, dB, dC, dD, dbias, st)
                                      : bwd_dispatch<0, 1>(p, ck != nullptr, dA, dB, dC, dD, dbias, st);
    else
        e = desc->out_dtype == MB_F32 ? bwd_dispatch<1, 0>(p, ck != nullptr, dA, dB, dC, dD, dbias, st)
                                      : bwd_dispatch<1, 1>(p, ck != nullptr, dA, dB, dC, dD, dbias, st);
    const hipError_t f = hipFreeAsync(ws, st);
    if (e == hipSuccess) e = f;
    return e == hipSuccess ? MB_OK : MB_ERR_HIP;
}

int mb_verify_rank(int64_t batch, int64_t ndraft, int64_t vocab, int32_t logit_dtype, int32_t beta,
                   const void *logits, const int32_t *draft, int32_t *ranks, int32_t *accepted,
                   int32_t *last_pos, void *stream) {
    if (batch < 0 || ndraft < 0 || vocab < 1) return MB_ERR_SHAPE;
    if (ndraft >= (int64_t(1) << 31) || vocab >= (int64_t(1) << 31) - 1 || batch >= (int64_t(1) << 31))
        return MB_ERR_SHAPE;
    if (!valid_dtype(logit_dtype)) return MB_ERR_DTYPE;
    int64_t pairs, elems;
    if (!mul_ok(batch, ndraft, &pairs) || !mul_ok(pairs, vocab, &elems)) return MB_ERR_SHAPE;
    if (batch == 0) return MB_OK;
    if (!accepted || (ndraft > 0 && (!logits || !draft))) return MB_ERR_NULL;
    const size_t lsz = dtype_size(logit_dtype);
    if ((logits && !aligned(logits, lsz)) || (draft && !aligned(draft, 4)) || !aligned(accepted, 4) ||
        (ranks && !aligned(ranks, 4)) || (last_pos && !aligned(last_pos, 4)))
        return MB_ERR_ALIGN;
    const size_t l_bytes = (size_t)elems * lsz, d_bytes = (size_t)pairs * 4, b_bytes = (size_t)batch * 4;
    struct Range { const void *p; size_t n; } outs[] = {{ranks, d_bytes}, {accepted, b_bytes}, {last_pos, b_bytes}};
    for (int i = 0; i < 3; ++i) {
        if (overlaps(outs[i].p, outs[i].n, logits, l_bytes) || overlaps(outs[i].p, outs[i].n, draft, d_bytes))
            return MB_ERR_ALIAS;
        for (int j = i + 1; j < 3; ++j)
            if (overlaps(outs[i].p, outs[i].n, outs[j].p, outs[j].n)) return MB_ERR_ALIAS;
    }
    mbs::rank::RankParams p{};
    p.batch = batch; p.ndraft = ndraft; p.vocab = vocab; p.logits = logits; p.draft = draft; p.beta = beta;
    p.ranks = ranks; p.accepted = accepted; p.last_pos = last_pos;
    const void *fn = logit_dtype == MB_F32 ? reinterpret_cast<const void *>(&mbs::rank::verify_rank<0>)
                                           : reinterpret_cast<const void *>(&mbs::rank::verify_rank<1>);
    const int waves = ndraft < 1 ? 1 : (ndraft > mbs::rank::kMaxThreads / 64 ? mbs::rank::kMaxThreads / 64
                                                                               : (int)ndraft);
    const hipError_t e = launch(fn, dim3((unsigned)batch), dim3(64 * waves), &p, stream);
    return e == hipSuccess ? MB_OK : MB_ERR_HIP;
}

int mb_scan_step(int64_t batch, int64_t dim, int64_t dstate, int32_t in_dtype, int32_t out_dtype,
                 int32_t delta_softplus, const void *u_t, const void *delta_t, const float *A,
                 const void *B_t, const void *C_t, const float *Dskip, const float *dt_bias,
                 const void *z_t, float *h, void *y_t, void *stream) {
    // dim below 2^36: at most 2^30 channel blocks of 64 along the grid's x
    if (batch < 0 || dim < 0 || dstate < 0 || dim >= (int64_t(1) << 36)) return MB_ERR_SHAPE;
    if (!valid_dtype(in_dtype) || !valid_dtype(out_dtype)) return MB_ERR_DTYPE;
    if (!supported_dstate(dstate)) return MB_ERR_UNSUPPORTED;
    int64_t rows, state_elems, bc_elems;
    if (!mul_ok(batch, dim, &rows) || !mul_ok(rows, dstate, &state_elems) ||
        !mul_ok(batch, dstate, &bc_elems))
        return MB_ERR_SHAPE;
    if (rows == 0) return MB_OK;
    if (!u_t || !delta_t || !A || !B_t || !C_t || !h || !y_t) return MB_ERR_NULL;

    const size_t in_sz = dtype_size(in_dtype), out_sz = dtype_size(out_dtype);
    const void *act[] = {u_t, delta_t, B_t, C_t, z_t};
    for (const void *p : act)
        if (p && !aligned(p, in_sz)) return MB_ERR_ALIGN;
    const void *f32s[] = {A, Dskip, dt_bias, h};
    for (const void *p : f32s)
        if (p && !aligned(p, 4)) return MB_ERR_ALIGN;
    if (!aligned(y_t, out_sz)) return MB_ERR_ALIGN;

    const size_t act_bytes = (size_t)rows * in_sz, bc_bytes = (size_t)bc_elems * in_sz;
    const size_t st_bytes = (size_t)state_elems * 4;
    struct Range { const void *p; size_t n; } ins[] = {
        {u_t, act_bytes}, {delta_t, act_bytes}, {z_t, act_bytes}, {B_t, bc_bytes}, {C_t, bc_bytes},
        {A, (size_t)(dim * dstate) * 4}, {Dskip, (size_t)dim * 4}, {dt_bias, (size_t)dim * 4}};
    const size_t y_bytes = (size_t)rows * out_sz;
    for (const Range &r : ins)
        if (overlaps(y_t, y_bytes, r.p, r.n) || overlaps(h, st_bytes, r.p, r.n)) return MB_ERR_ALIAS;
    if (overlaps(y_t, y_bytes, h, st_bytes)) return MB_ERR_ALIAS;

    StepParams p{};
    p.batch = batch; p.dim = dim;
    p.u = u_t; p.delta = delta_t; p.Bt = B_t; p.Ct = C_t; p.z = z_t;
    p.A = A; p.Dskip = Dskip; p.dt_bias = dt_bias; p.h = h; p.y = y_t;
    p.delta_softplus = delta_softplus ? 1 : 0;

    hipError_t e;
    if (in_dtype == MB_F32)
        e = out_dtype == MB_F32 ? step_dispatch_n<0, 0>(p, dstate, stream) : step_dispatch_n<0, 1>(p, dstate, stream);
    else
        e = out_dtype == MB_F32 ? step_dispatch_n<1, 0>(p, dstate, stream) : step_dispatch_n<1, 1>(p, dstate, stream);
    return e == hipSuccess ? MB_OK : MB_ERR_HIP;
}

}  // extern "C"
