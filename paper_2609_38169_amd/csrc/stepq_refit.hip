// Launcher of the decode step with the online Key-Row-Aware Dual-Axis refit
// (the kernel body is in stepq_refit_body.h).
#include "stepq_refit_body.h"

namespace stepq {

hipError_t launch_decode_refit(const DecodeArgs &a, bool bf16, bool diag, int pool_layout, hipStream_t stream)
{
    return launch_refit_mode<Refit::DualAxis>(a, bf16, diag, pool_layout, stream);
}

}  // namespace stepq
