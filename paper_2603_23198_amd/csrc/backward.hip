// Backward pass of the non-gated ReLU-sparse FFN.
#include "backward.h"
#include "common.h"
#include "internal.h"

namespace sfl {

sfl_status_t backward_workspace(const sfl_ffn_bwd_args_t* a, size_t* bytes) {
  if (!a || !bytes) return SFL_E_ARG;
  *bytes = 0;
  return SFL_E_UNSUPPORTED;
}

sfl_status_t backward_run(const sfl_ffn_bwd_args_t* a, hipStream_t) {
  if (!a) return SFL_E_ARG;
  return SFL_E_UNSUPPORTED;
}

}  // namespace sfl
