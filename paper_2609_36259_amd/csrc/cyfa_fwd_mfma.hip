// Matrix-core (bf16 MFMA) chunk-wise forward -- placeholder until implemented.
#include "cyfa_internal.h"

namespace cyfa {

bool mfma_supported(const FwdParams &) { return false; }
size_t mfma_workspace_bytes(const FwdParams &, int) { return 0; }
int mfma_auto_segments(const FwdParams &) { return 1; }
hipError_t launch_fwd_mfma(const FwdParams &, int, void *, hipStream_t, hipEvent_t, hipEvent_t) {
    return hipErrorNotSupported;
}

}  // namespace cyfa
