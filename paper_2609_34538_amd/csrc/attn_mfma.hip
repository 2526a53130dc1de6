// Matrix-core (MFMA) policy-attention kernel for bf16 caches.
#include "das_internal.h"

namespace das {

int mfma_rows_per_wg(int rows) { return rows < 64 ? 64 : 64; }

hipError_t launch_attn_mfma(const AttnParams &, int, hipStream_t) {
  return hipErrorNotSupported;
}

}  // namespace das
