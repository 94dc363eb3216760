// Algorithm 1 ("Adaptive Threshold Caching", Section 3.3): one gate step,
// shared by the host gate (gate.cpp) and the device-resident gate kernel
// (elementwise.hip), so both take their decisions with the same IEEE-double
// operations: one addition into the accumulator, one subtraction, absolute
// value and comparison for the stability test, one comparison against the
// threshold.  No product appears, so floating-point contraction cannot
// change a result; the host build also disables it.
#pragma once

#include <stdint.h>

#include "acid.h"

#if defined(__HIPCC__)
#define ACID_HD __host__ __device__
#else
#define ACID_HD
#endif

namespace acid {

// Advances st by one step with signal s_t (ignored during warmup).  Returns
// the decision (1: run the model, 0: reuse the cache) and stores the active
// threshold in *tau (NaN during warmup).
ACID_HD inline int32_t gate_step(acid_gate_state* st, const acid_gate_params* p, double s_t,
                                 double* tau) {
  const int32_t step = st->step;
  st->step = step + 1;
  if (step < p->n_warmup) {
    // Leading steps of the base method: always run, state left as it was.
    *tau = __builtin_nan("");
    return 1;
  }
  st->sigma_sum = st->sigma_sum + s_t;
  const double adiff = __builtin_fabs(s_t - st->s_prev);
  // A signal that moved by at most delta picks the larger threshold.
  const double t = (st->has_prev && adiff <= p->delta) ? p->tau_high : p->tau_low;
  int32_t compute;
  if (st->sigma_sum <= t) {
    compute = 0;
  } else {
    compute = 1;  // a computed step restarts the accumulation
    st->sigma_sum = 0.0;
  }
  st->s_prev = s_t;
  st->has_prev = 1;
  *tau = t;
  return compute;
}

}  // namespace acid
