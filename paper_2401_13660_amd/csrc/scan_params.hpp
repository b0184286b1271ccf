// scan_params.hpp -- argument block passed to every scan kernel.
#pragma once

#include <stdint.h>

namespace mbs {

struct ScanParams {
    int64_t batch, dim, seqlen;
    const void *u, *delta, *Bm, *Cm, *z;
    const float *A, *Dskip, *dt_bias, *h0;
    void *y;
    float *h_last;
    // States at requested positions: pos[k * batch + b] is position k of batch
    // element b; h_pos[((k * batch + b) * dim + d) * N + n] receives the state
    // after that timestep.  npos == 0 disables them.  The scan kernels write
    // only positions in [0, seqlen); init_positions fills the other slots.
    const int32_t *pos;
    int64_t npos;
    float *h_pos;
    // Checkpoints for the backward (tiled path only): ck[((t / 16) * batch * dim
    // + row) * 16 + n] receives the state before timestep t for every t that is a
    // multiple of 16 (h0 at t = 0).  Null disables them.
    float *ck;
    int delta_softplus;
};

struct StepParams {
    int64_t batch, dim;
    const void *u, *delta, *Bt, *Ct, *z;
    const float *A, *Dskip, *dt_bias;
    float *h;
    void *y;
    int delta_softplus;
};

}  // namespace mbs
