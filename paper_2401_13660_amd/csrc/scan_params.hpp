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
