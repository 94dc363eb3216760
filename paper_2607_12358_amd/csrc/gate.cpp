// Algorithm 1 ("Adaptive Threshold Caching", Section 3.3): one gate step.
//
// Pure host code in IEEE double.  Built with -ffp-contract=off and without
// fast-math so every sum and comparison is the plain IEEE operation; fed the
// same drift values, its decisions are bit-identical to any other IEEE-double
// implementation of the algorithm.
#include <math.h>

#include "acid.h"

extern "C" acid_status acid_gate(acid_gate_state* st, const acid_gate_params* p, double s_t,
                                 int32_t* compute_out, double* tau_used_out) {
  if (!st || !p || !compute_out) return ACID_ERR_INVALID_ARG;
  const int32_t step = st->step;
  st->step = step + 1;
  if (step < p->n_warmup) {
    // Warmup: the base method runs the full model; the gate state is untouched.
    *compute_out = 1;
    if (tau_used_out) *tau_used_out = NAN;
    return ACID_OK;
  }
  st->sigma_sum = st->sigma_sum + s_t;
  double tau;
  if (st->has_prev && fabs(s_t - st->s_prev) <= p->delta)
    tau = p->tau_high;  // stable phase: cache aggressively
  else
    tau = p->tau_low;   // dynamic phase: cache conservatively
  int32_t compute;
  if (st->sigma_sum <= tau) {
    compute = 0;        // reuse the cached residual
  } else {
    compute = 1;        // run the model, reset the accumulator
    st->sigma_sum = 0.0;
  }
  st->s_prev = s_t;
  st->has_prev = 1;
  *compute_out = compute;
  if (tau_used_out) *tau_used_out = tau;
  return ACID_OK;
}
