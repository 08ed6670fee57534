// Kernel argument blocks and launchers (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.hpp"

namespace tactic {

struct ScoreArgs {
  const uint16_t* q;          // bf16 [B][Hq][128]
  const uint16_t* centroids;  // bf16 [Hkv][Ct][128]
  const int64_t* cl_indptr;   // [B+1]
  int B, Hq, Hkv, Cm;
  int64_t Ct;
  float* scores;              // [B*Hq][Cm]
};

struct SortArgs {
  const float* scores;        // [B*Hq][Cm]
  const int32_t* offsets;     // [Hkv][Ct + B]
  const int64_t* kv_indptr;
  const int64_t* seq_len;     // [B] or null (see tactic_kv_shape)
  const int64_t* cl_indptr;
  int B, Hq, Hkv, G, Cm, nb_max;
  int64_t Ct, S_cap;
  int max_tail;               // recent tokens per sequence beyond the clusters (capacity)
  SelParams prm;
  uint64_t* g_keys;           // sort scratch when the sort does not fit LDS
  uint32_t* g_cnt;
  uint32_t* g_start;
  int32_t* order;             // [B*Hq][Cm]
  int32_t* rank_of;           // [B*Hq][Cm]
  int32_t* rprefix;           // [B*Hq][Cm+1]
  int32_t* sample_rows;       // [B*Hq][S_cap]
  int32_t* head_meta;         // [B*Hq][16]
  int per_head;               // 1: per-head selections (no union); sel_count_kv is then a sum
  int32_t* sel_count_kv;      // [B*Hkv], zeroed here in per-head mode
};

struct FitArgs {
  const uint16_t* q;
  const uint16_t* K;          // cluster-sorted keys [Hkv][total][128]
  const int64_t* kv_indptr;
  const int64_t* cl_indptr;
  const int32_t* offsets;
  int B, Hq, Hkv, G, Cm, BH, split;
  // selection groups: NV per sequence of GV query heads each; group j reads KV
  // head j / kv_div (union: NV = Hkv, GV = G, kv_div = 1; per head: NV = Hq, GV = 1, kv_div = G)
  int NV, kv_div, per_head;
  int64_t Ct, total, S_cap, chunk_tokens, max_chunks;
  double P;
  const int32_t* head_meta;
  const int32_t* sample_rows;
  const int32_t* rprefix;
  const int32_t* rank_of;
  double* logits;             // [B*Hq][S_cap]
  double* lse;                // [B*Hq][split][4 regions][max, sum exp(l - max)]
  double* fit;                // [B*Hq][16]
  int32_t* cut;               // [B*Hq][2]
  int32_t* sel_count_q;       // [B*Hq]
  int32_t* sel_count_kv;      // [B*Hkv]
  int32_t* union_len;         // [NV][Ct]
  int32_t* gmeta;             // [B*NV][4]: ranges, union tokens, work items, tokens per item
  int32_t* rstart;            // [B*NV][Cm+2]: first row of each selected range
  int32_t* rupos;             // [B*NV][Cm+2]: its first position in the group's token list
  int32_t* cfr;               // [B*NV][max_chunks]
};

struct AttnArgs {
  const uint16_t* q;
  const uint16_t* K;
  const uint16_t* V;
  const int64_t* kv_indptr;
  const int64_t* seq_len;     // [B] or null
  int B, Hq, Hkv, Cm, dense;
  int NV, kv_div;             // selection groups per sequence and KV head divisor (as in FitArgs)
  int64_t total, chunk_tokens, max_chunks;
  const int32_t* gmeta;
  const int32_t* rstart;
  const int32_t* rupos;
  const int32_t* cfr;
  float* partials;            // [B*NV + grid][GV*130]: one slot per (group, workgroup) pair
  int64_t* ameta;             // [B*NV + 2]: tokens per workgroup, then the groups' token offsets
  float* out;                 // [B][Hq][128]
};

hipError_t launch_score(const ScoreArgs& a, int G, int grid_x, int grid_y, hipStream_t st);
hipError_t launch_sort(const SortArgs& a, bool lds, int n_heads, hipStream_t st);
hipError_t launch_sample(const FitArgs& a, int split, int n_heads, hipStream_t st);
hipError_t launch_fit_union(const FitArgs& a, int G, int n_groups, hipStream_t st);
hipError_t launch_attn(const AttnArgs& a, int G, int grid, hipStream_t st);
hipError_t launch_combine(const AttnArgs& a, int G, hipStream_t st);
hipError_t attn_resident_grid(int G, int n_groups, int* grid);

}  // namespace tactic
