// Internal interface between the host entry points (bdlm_api.cpp) and the HIP
// kernels (bdlm_scan.hip).  Plain C++; no HIP types.
#pragma once

#include <stdint.h>

#include "bdlm.h"

namespace bdlm {

struct LaunchArgs {
    const void *x, *dt, *Bm, *Cm;
    const float *A, *D, *D_rev;
    float *h_pool;   // read only for a step, updated in place by a commit
    float *y;        // step: required; commit: optional (NULL skips y_clean)
    int64_t xs_b, xs_t, xs_h;
    int64_t dts_b, dts_t;
    int64_t bcs_b, bcs_t, bcs_g;
    int32_t batch, nheads, ngroups, L, dstate;
    int32_t bf16;          // activation storage: 1 bf16, 0 fp32
    const int32_t *slots;  // host [batch] or NULL (identity)
};

// Enqueue one block step (commit == false) or one commit (commit == true).
// Arguments are already validated.  Returns BDLM_OK or BDLM_E_LAUNCH.
int launch_block(const LaunchArgs &a, bool commit, void *stream);

// Full-window bidirectional scan over T tokens (a.L is ignored): forward pass,
// then reverse pass adding into a.y.
int launch_full_window(const LaunchArgs &a, int64_t T, void *stream);

// Forward chain over T tokens continuing the states in a.h_pool (via a.slots),
// writing them back; a.y (optional) receives the forward outputs.
int launch_prefill(const LaunchArgs &a, int64_t T, void *stream);

// Permute nstates states between row-major [64][dstate] and the pool layout.
int launch_state_permute(const float *src, float *dst, int64_t nstates, int64_t dstate,
                         bool to_pool, void *stream);

// Zero nreset states of state_elems floats each (slots NULL: all nslots).
int launch_reset(float *h_pool, int64_t nslots, int64_t state_elems, const int32_t *slots,
                 int64_t nreset, void *stream);

}  // namespace bdlm
