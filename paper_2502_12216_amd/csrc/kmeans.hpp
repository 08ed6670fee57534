// Prefill K-means clustering (Sec. 4.2): internal entry points.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace tactic {

size_t kmeans_workspace_bytes(int B, int Hkv, int64_t total, int64_t Ct, int Cm, int64_t nmax);

hipError_t run_kmeans(const uint16_t* K, const uint16_t* V, const int64_t* kv_indptr, const int64_t* seq_len,
                      const int64_t* cl_indptr, int B, int Hkv, int64_t total, int64_t nmax,
                      int64_t Ct, int Cm, const int32_t* init_idx, int max_iters,
                      const uint16_t* prev_centroids, const int64_t* prev_cl_indptr,
                      uint16_t* centroids, int32_t* assign, int32_t* offsets, int32_t* perm,
                      uint16_t* K_sorted, uint16_t* V_sorted, void* workspace, hipStream_t st);

}  // namespace tactic
