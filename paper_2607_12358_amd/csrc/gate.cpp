// Algorithm 1 ("Adaptive Threshold Caching", Section 3.3): the host gate.
//
// Pure host code in IEEE double, built with -ffp-contract=off and without
// fast-math.  The step itself lives in gate_step.h, which the device-resident
// gate kernel also uses, so host and device decisions agree bit for bit on
// the same drift values.
#include "gate_step.h"

extern "C" acid_status acid_gate(acid_gate_state* st, const acid_gate_params* p, double s_t,
                                 int32_t* compute_out, double* tau_used_out) {
  if (!st || !p || !compute_out) return ACID_ERR_INVALID_ARG;
  double tau;
  *compute_out = acid::gate_step(st, p, s_t, &tau);
  if (tau_used_out) *tau_used_out = tau;
  return ACID_OK;
}
