// Backward pass of the non-gated ReLU-sparse FFN (launch interface).
#pragma once

#include <hip/hip_runtime.h>

#include "../../include/sfl.h"

namespace sfl {

sfl_status_t backward_workspace(const sfl_ffn_bwd_args_t* a, size_t* bytes);
sfl_status_t backward_run(const sfl_ffn_bwd_args_t* a, hipStream_t s);

}  // namespace sfl
