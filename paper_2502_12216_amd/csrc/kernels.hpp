// Kernel argument blocks and launchers (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.hpp"

namespace tactic {

// A paged K/V cache: page p holds page_size consecutive tokens of one
// sequence for every KV head, bf16 [num_pages][Hkv][page_size][128]; the
// page of a sequence's tokens [i * page_size, (i + 1) * page_size) is
// page_table[b * max_pages + i].  perm (or null for the identity) maps a
// cluster-sorted row of the first c_b rows to its token; rows from c_b on
// (the recent tokens) are their own tokens.
struct PagedKV {
  const int32_t* page_table;  // [B][max_pages]
  const int32_t* perm;        // [Hkv][total] sequence-relative token per cluster-sorted row, or null
  int page_size, max_pages;
  int64_t num_pages;
};

// Element offset of the 128-wide K/V row of (sequence b, KV head kvh) at
// cluster-sorted row `row` (the token itself when dense); n_c = clustered rows.
__device__ __forceinline__ int64_t paged_row(const PagedKV& pk, int Hkv, int64_t total, int64_t kvb, int b,
                                             int kvh, int row, int n_c) {
  int tok = (pk.perm && row < n_c) ? pk.perm[(int64_t)kvh * total + kvb + row] : row;
  tok = min(max(tok, 0), pk.max_pages * pk.page_size - 1);  // in bounds whatever the tables hold
  int64_t page = pk.page_table[(int64_t)b * pk.max_pages + tok / pk.page_size];
  page = min(max(page, (int64_t)0), pk.num_pages - 1);
  return (page * Hkv + kvh) * pk.page_size + tok % pk.page_size;
}

// paged_row for K rows at once, each row in [0, n) of a sequence of n tokens
// (kvb + n <= total): the K permutation loads are issued together (row >= n_c
// reads an entry it then ignores, so no load sits behind a per-row guard),
// then the K page-table loads.  Same clamps and results as paged_row.
template <int K>
__device__ __forceinline__ void paged_rows(const PagedKV& pk, int Hkv, int64_t total, int64_t kvb, int b,
                                           int kvh, const int (&row)[K], int n_c, int64_t (&out)[K]) {
  int tok[K];
  if (pk.perm) {
#pragma unroll
    for (int e = 0; e < K; ++e) tok[e] = pk.perm[(int64_t)kvh * total + kvb + row[e]];
#pragma unroll
    for (int e = 0; e < K; ++e) tok[e] = row[e] < n_c ? tok[e] : row[e];
  } else {
#pragma unroll
    for (int e = 0; e < K; ++e) tok[e] = row[e];
  }
  int64_t page[K];
#pragma unroll
  for (int e = 0; e < K; ++e) {
    tok[e] = min(max(tok[e], 0), pk.max_pages * pk.page_size - 1);
    page[e] = pk.page_table[(int64_t)b * pk.max_pages + tok[e] / pk.page_size];
  }
#pragma unroll
  for (int e = 0; e < K; ++e) {
    const int64_t pg = min(max(page[e], (int64_t)0), pk.num_pages - 1);
    out[e] = (pg * Hkv + kvh) * pk.page_size + tok[e] % pk.page_size;
  }
}

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
  const int32_t* order;       // [B*Hq][Cm]: cluster at each rank
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
  uint64_t* slice_tot;        // [B*NV][kMaxUnionSlices]: (ranges << 32) | tokens of each union slice
  int union_slice;            // clusters per union slice (set by the launcher; 0: not sliced)
  PagedKV pk;                 // used by the paged launches (K then points at the pages)
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
  const int32_t* head_meta;   // [B*Hq][16] (sparse, paged: clustered rows per head in field 0)
  PagedKV pk;                 // used by the paged launches (K, V then point at the pages)
  float* out;                 // [B][Hq][128]
};

hipError_t launch_score(const ScoreArgs& a, int G, int grid_x, int grid_y, hipStream_t st);
hipError_t launch_sort(const SortArgs& a, bool lds, int n_heads, hipStream_t st);
hipError_t launch_sample(const FitArgs& a, int split, int n_heads, bool paged, hipStream_t st);
hipError_t launch_fit_union(const FitArgs& a, int G, int n_groups, hipStream_t st);
hipError_t launch_attn(const AttnArgs& a, int G, int grid, bool paged, hipStream_t st);
hipError_t launch_combine(const AttnArgs& a, int G, hipStream_t st);
hipError_t attn_resident_grid(int G, int n_groups, bool paged, int* grid);
hipError_t launch_stream_read(const void* buf, int64_t n16, int workgroups, uint32_t* sink, hipStream_t st);

}  // namespace tactic
