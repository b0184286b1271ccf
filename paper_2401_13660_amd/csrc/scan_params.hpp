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
