// Host-only checks shared by the library's translation units (defined in host_checks.cpp): the
// per-thread error text behind dit_last_error_message(), block-configuration validation and the
// coefficients of the flow-step update. No HIP types, so host-only code can include it.
#pragma once
#include "status.h"

namespace dit {
// DIT_OK or the first violated rule of the configuration (message set).
dit_status check_config(const dit_block_config* c);
// x' = cx x + cv v + ce noise for one sampler step from t to t_next with noise scale a (the Euler
// ODE step when a == 0, the SDE step otherwise); domain errors as documented for flow_step.
dit_status flow_coefficients(float t, float t_next, float a, bool has_noise, float* cx, float* cv, float* ce);
}  // namespace dit
