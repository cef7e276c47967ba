// Launcher of the decode step with the row-wise absmax requantization of
// the INT-b baseline (the kernel body is in stepq_refit_body.h).
#include "stepq_refit_body.h"

namespace stepq {

hipError_t launch_decode_rowmax(const DecodeArgs &a, bool bf16, bool diag, int pool_layout, hipStream_t stream)
{
    return launch_refit_mode<Refit::RowAbsmax>(a, bf16, diag, pool_layout, stream);
}

}  // namespace stepq
