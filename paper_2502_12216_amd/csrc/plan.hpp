// Host/device description of one sparse-decode launch sequence: sizes and
// workspace offsets, derived once from the shape and parameters.
#pragma once

#include <stdint.h>

#include "common.hpp"

namespace tactic {

constexpr int64_t kPlanMagic = 0x54414354494331LL;  // "TACTIC1"
constexpr int kTile = 64;              // tokens per attention tile
constexpr int kMaxChunkTokens = 2048;  // tokens whose rows the attention stages in LDS at once
constexpr int kCfrTokens = 256;        // granularity of the union's position -> range index
constexpr int kMaxAttnGrid = 4096;     // attention workgroups the partials are sized for (cap)
constexpr int kSortLdsBuckets = 8192;  // largest cluster count sorted in LDS
constexpr int kMaxGroups = 4096;       // B * Hkv limit of the attention work list
constexpr int kFitFields = 16;
constexpr int kStageEvents = 7;        // start + after each of the six decode kernels
constexpr int kUnionLdsMax = 32768;     // clusters whose union lengths are staged in LDS
constexpr int kMaxUnionSlices = 8;    // workgroups per selection group of the sliced union
constexpr int kScoreRows = 64;         // centroids per scoring workgroup (4096 workgroups at 8192 x 32)
#ifndef TACTIC_SAMPLE_CHUNK
#define TACTIC_SAMPLE_CHUNK 64
#endif
constexpr int kSampleChunk = TACTIC_SAMPLE_CHUNK;  // sampled rows per sampling workgroup

struct DecodePlan {
  int64_t magic;
  int64_t B, Hq, Hkv, G, Cm, Ct, nmax, total;
  int64_t S_cap;         // sampled rows per head (capacity)
  int64_t chunk_tokens;  // kCfrTokens: positions per entry of the position -> range index
  int64_t max_chunks;    // entries of that index per selection group (capacity)
  int64_t split;         // sampling workgroups per query head
  int64_t attn_grid;     // attention workgroups the partials are sized for (resident capacity)
  int64_t sort_lds;      // 1: sort in LDS, 0: sort scratch in the workspace
  int64_t nb_max;        // bucket capacity of the sort
  // workspace byte offsets
  int64_t off_scores, off_order, off_rank, off_rprefix, off_headmeta, off_rows, off_logit;
  int64_t off_fit, off_cut, off_union_len, off_gmeta, off_rstart, off_rupos, off_cfr, off_lse;
  int64_t off_partials, off_sort_keys, off_sort_cnt, off_sort_start, off_ameta, off_slice_tot;
  int64_t ws_bytes;
  int64_t exact_bp, win_bp, win_min, p1_bp, p2_bp;
  int64_t events[kStageEvents];  // optional hipEvent_t recorded between the kernels
  int64_t use_union;     // 1: GQA union (Sec. 4.5); 0: every query head over its own selection
  int64_t NV, GV;        // selection groups per sequence, query heads per selection group
  int64_t max_tail;      // capacity for recent (unclustered) tokens per sequence
  int64_t attn_dev;      // device the resident attention grids below were measured on (-1: none)
  int64_t attn_res[2];   // attention workgroups resident at once on it: contiguous, paged
  int64_t pad[64 - 57];
};
static_assert(sizeof(DecodePlan) == 64 * sizeof(int64_t), "plan must fill tactic_decode_plan");

}  // namespace tactic
