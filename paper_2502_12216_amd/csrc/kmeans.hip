// Prefill K-means clustering (Sec. 4.2) -- placeholder until the kernels land.
#include "kmeans.hpp"

namespace tactic {

size_t kmeans_workspace_bytes(int, int, int64_t, int64_t, int, int64_t) { return 256; }

hipError_t run_kmeans(const uint16_t*, const uint16_t*, const int64_t*, const int64_t*, int, int, int64_t,
                      int64_t, int64_t, int, const int32_t*, int, uint16_t*, int32_t*, int32_t*, int32_t*,
                      uint16_t*, uint16_t*, void*, hipStream_t) {
  return hipErrorNotSupported;
}

}  // namespace tactic
