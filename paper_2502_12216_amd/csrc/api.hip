// Host side of the C ABI declared in include/tactic.h: validation, launch
// plans, workspace layout and the launch sequence of each call.
#include <hip/hip_runtime.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <string>

#include "../../include/tactic.h"
#include "common.hpp"
#include "kernels.hpp"
#include "kmeans.hpp"
#include "plan.hpp"

namespace {

thread_local std::string g_last_error;

tactic_status fail(tactic_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
tactic_status fail(tactic_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

tactic_status hip_fail(hipError_t e, const char* what) {
  return fail(TACTIC_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

int64_t align_up(int64_t x, int64_t a) { return (x + a - 1) / a * a; }

struct Layout {
  int64_t cur = 0;
  int64_t take(int64_t bytes) {
    const int64_t o = cur;
    cur = align_up(cur + bytes, 256);
    return o;
  }
};

tactic::SelParams sel_params(const tactic_decode_params* p) {
  tactic::SelParams s;
  s.target_frac = p->target_frac;
  s.exact_bp = p->exact_bp;
  s.win_bp = p->win_bp;
  s.win_min = p->win_min;
  s.p1_bp = p->p1_bp;
  s.p2_bp = p->p2_bp;
  return s;
}

tactic_status check_shape(const tactic_kv_shape* s) {
  if (!s) return fail(TACTIC_ERR_INVALID_ARG, "shape is null");
  if (s->batch < 1) return fail(TACTIC_ERR_INVALID_ARG, "batch must be >= 1 (got %d)", s->batch);
  if (s->n_kv_heads < 1 || s->n_q_heads < 1)
    return fail(TACTIC_ERR_INVALID_ARG, "head counts must be >= 1");
  if (s->n_q_heads % s->n_kv_heads != 0)
    return fail(TACTIC_ERR_INVALID_ARG, "n_q_heads (%d) is not a multiple of n_kv_heads (%d)",
                s->n_q_heads, s->n_kv_heads);
  const int G = s->n_q_heads / s->n_kv_heads;
  if (G != 1 && G != 2 && G != 4 && G != 8)
    return fail(TACTIC_ERR_UNSUPPORTED, "group size %d not in {1, 2, 4, 8}", G);
  if (s->head_dim != tactic::kHeadDim)
    return fail(TACTIC_ERR_UNSUPPORTED, "head_dim %d != 128", s->head_dim);
  if (s->total_tokens < 0 || s->max_seq_len < 0 || s->max_seq_len > s->total_tokens)
    return fail(TACTIC_ERR_INVALID_ARG, "inconsistent total_tokens / max_seq_len");
  if (s->max_seq_len >= (int64_t)1 << 31)
    return fail(TACTIC_ERR_UNSUPPORTED, "sequence length >= 2^31");
  if ((int64_t)s->batch * s->n_kv_heads > tactic::kMaxGroups)
    return fail(TACTIC_ERR_UNSUPPORTED, "batch * n_kv_heads > %d", tactic::kMaxGroups);
  if (!s->kv_indptr) return fail(TACTIC_ERR_INVALID_ARG, "kv_indptr is null");
  return TACTIC_OK;
}

tactic_status check_params(const tactic_decode_params* p) {
  if (!p) return fail(TACTIC_ERR_INVALID_ARG, "params is null");
  if (!(p->target_frac > 0.f && p->target_frac <= 1.f))
    return fail(TACTIC_ERR_INVALID_ARG, "target_frac must be in (0, 1] (got %g)", (double)p->target_frac);
  if (p->exact_bp < 0 || p->exact_bp > 10000 || p->win_bp < 0 || p->win_bp > 10000 || p->win_min < 1 ||
      p->p1_bp < 0 || p->p1_bp > 10000 || p->p2_bp < 0 || p->p2_bp > 10000)
    return fail(TACTIC_ERR_INVALID_ARG, "fit parameters out of range");
  if (p->use_union != 0 && p->use_union != 1) return fail(TACTIC_ERR_INVALID_ARG, "use_union must be 0 or 1");
  if (p->max_tail < 0) return fail(TACTIC_ERR_INVALID_ARG, "max_tail must be >= 0");
  return TACTIC_OK;
}

tactic_status paged_args(const tactic_paged_kv* kv, const tactic_kv_shape* s, tactic::PagedKV* pk) {
  if (!kv || !kv->K_pages || !kv->V_pages || !kv->page_table) return fail(TACTIC_ERR_INVALID_ARG, "null paged-KV pointer");
  if (kv->page_size < 1 || kv->max_pages < 1 || kv->num_pages < 1)
    return fail(TACTIC_ERR_INVALID_ARG, "page_size, max_pages and num_pages must be >= 1");
  if ((int64_t)kv->page_size * kv->max_pages < s->max_seq_len)
    return fail(TACTIC_ERR_INVALID_ARG, "max_pages * page_size < max_seq_len");
  if ((int64_t)kv->page_size * kv->max_pages >= ((int64_t)1 << 31))
    return fail(TACTIC_ERR_UNSUPPORTED, "max_pages * page_size >= 2^31");
  if (kv->num_pages * s->n_kv_heads * kv->page_size >= ((int64_t)1 << 31))
    return fail(TACTIC_ERR_UNSUPPORTED, "num_pages * n_kv_heads * page_size >= 2^31 rows");
  pk->page_table = kv->page_table;
  pk->perm = kv->perm;
  pk->page_size = kv->page_size;
  pk->max_pages = kv->max_pages;
  pk->num_pages = kv->num_pages;
  return TACTIC_OK;
}

const tactic::DecodePlan* as_plan(const tactic_decode_plan* p) {
  return reinterpret_cast<const tactic::DecodePlan*>(p);
}

// Workspace of a dense launch on `grid` attention workgroups: a partial slot
// per (KV group, workgroup) pair that can meet, and the split's offsets.
size_t dense_workspace_bytes(const tactic_kv_shape* s, int64_t grid) {
  const int64_t BG = (int64_t)s->batch * s->n_kv_heads;
  const int64_t G = s->n_q_heads / s->n_kv_heads;
  Layout L;
  L.take((BG + grid) * G * (tactic::kHeadDim + 2) * 4);
  L.take((BG + 2) * 8);
  return (size_t)L.cur;
}

}  // namespace

extern "C" {

void tactic_decode_params_default(tactic_decode_params* p) {
  if (!p) return;
  p->target_frac = 0.9f;
  p->exact_bp = 100;
  p->win_bp = 50;
  p->win_min = 8;
  p->p1_bp = 1000;
  p->p2_bp = 6000;
  p->use_union = 1;
  p->max_tail = 0;
}

const char* tactic_status_string(tactic_status s) {
  switch (s) {
    case TACTIC_OK: return "ok";
    case TACTIC_ERR_INVALID_ARG: return "invalid argument";
    case TACTIC_ERR_UNSUPPORTED: return "unsupported";
    case TACTIC_ERR_WORKSPACE: return "workspace too small";
    case TACTIC_ERR_HIP: return "HIP error";
  }
  return "unknown status";
}

const char* tactic_last_error(void) { return g_last_error.c_str(); }

tactic_status tactic_sparse_decode_plan(const tactic_kv_shape* shape, const tactic_cluster_meta* meta,
                                        const tactic_decode_params* params, tactic_decode_plan* plan_out,
                                        size_t* workspace_bytes) {
  tactic_status st = check_shape(shape);
  if (st != TACTIC_OK) return st;
  if ((st = check_params(params)) != TACTIC_OK) return st;
  if (!meta || !plan_out || !workspace_bytes) return fail(TACTIC_ERR_INVALID_ARG, "null argument");
  if (meta->max_clusters < 1 || meta->total_clusters < meta->max_clusters ||
      meta->total_clusters > (int64_t)meta->max_clusters * shape->batch)
    return fail(TACTIC_ERR_INVALID_ARG, "inconsistent total_clusters / max_clusters");
  if (meta->max_clusters > (1 << 24)) return fail(TACTIC_ERR_UNSUPPORTED, "more than 2^24 clusters");

  tactic::DecodePlan p;
  memset(&p, 0, sizeof(p));
  p.magic = tactic::kPlanMagic;
  p.B = shape->batch;
  p.Hq = shape->n_q_heads;
  p.Hkv = shape->n_kv_heads;
  p.G = p.Hq / p.Hkv;
  p.Cm = meta->max_clusters;
  p.Ct = meta->total_clusters;
  p.nmax = shape->max_seq_len;
  p.total = shape->total_tokens;
  p.exact_bp = params->exact_bp;
  p.win_bp = params->win_bp;
  p.win_min = params->win_min;
  p.p1_bp = params->p1_bp;
  p.p2_bp = params->p2_bp;
  p.use_union = params->use_union;
  p.max_tail = params->max_tail;
  p.NV = p.use_union ? p.Hkv : p.Hq;
  p.GV = p.use_union ? p.G : 1;
  // the attention keeps one prefix entry per selection group in LDS
  if (p.B * p.NV > tactic::kMaxGroups)
    return fail(TACTIC_ERR_UNSUPPORTED, "batch * %s = %lld selection groups > %d",
                p.use_union ? "n_kv_heads" : "n_q_heads (use_union = 0)", (long long)(p.B * p.NV),
                tactic::kMaxGroups);
  // sampled rows per head: the largest list any length <= nmax can need
  const tactic::SelParams sp = sel_params(params);
  int64_t S_cap = 1;
  for (int64_t n = 1; n <= p.nmax; ++n) {
    const tactic::Geometry g = tactic::make_geometry(n, sp);
    if (g.samples > S_cap) S_cap = g.samples;
  }
  p.S_cap = S_cap + p.max_tail;  // the recent tokens follow the sampled rows
  p.chunk_tokens = tactic::kCfrTokens;
  p.max_chunks = std::max<int64_t>(1, (p.nmax + p.chunk_tokens - 1) / p.chunk_tokens);
  p.split = std::max<int64_t>(1, (p.S_cap + tactic::kSampleChunk - 1) / tactic::kSampleChunk);
  // the partials hold one slot per (selection group, attention workgroup) pair
  // that can meet: at most groups + workgroups; the grid (the device's resident
  // capacity) is capped so that the plan does not depend on the device
  p.attn_grid = tactic::kMaxAttnGrid;
  int64_t nb = 1;
  while (nb < p.Cm) nb <<= 1;
  p.sort_lds = nb <= tactic::kSortLdsBuckets ? 1 : 0;
  p.nb_max = p.sort_lds ? tactic::kSortLdsBuckets : nb;

  const int64_t BH = p.B * p.Hq, BG = p.B * p.NV;  // BG: selection groups
  Layout L;
  p.off_scores = L.take(BH * p.Cm * 4);
  p.off_order = L.take(BH * p.Cm * 4);
  p.off_rank = L.take(BH * p.Cm * 4);
  p.off_rprefix = L.take(BH * (p.Cm + 1) * 4);
  p.off_headmeta = L.take(BH * 16 * 4);
  p.off_rows = L.take(BH * p.S_cap * 4);
  p.off_logit = L.take(BH * p.S_cap * 8);
  p.off_fit = L.take(BH * tactic::kFitFields * 8);
  p.off_lse = L.take(BH * p.split * 8 * 8);
  p.off_cut = L.take(BH * 2 * 4);
  p.off_union_len = L.take(p.NV * p.Ct * 4);
  p.off_gmeta = L.take(BG * 4 * 4);
  p.off_rstart = L.take(BG * (p.Cm + 2) * 4);  // ranges: clusters, then the recent tokens
  p.off_rupos = L.take(BG * (p.Cm + 2) * 4);
  p.off_cfr = L.take(BG * p.max_chunks * 4);
  p.off_slice_tot = L.take(BG * tactic::kMaxUnionSlices * 8);
  p.off_partials = L.take((BG + p.attn_grid) * p.GV * (tactic::kHeadDim + 2) * 4);
  p.off_ameta = L.take((BG + 2) * 8);
  if (!p.sort_lds) {
    p.off_sort_keys = L.take(BH * p.nb_max * 8);
    p.off_sort_cnt = L.take(BH * (p.nb_max + 4) * 4);
    p.off_sort_start = L.take(BH * (p.nb_max + 4) * 4);
  }
  p.ws_bytes = L.cur;
  // resident attention workgroups on the current device, so that decode calls
  // on it need no occupancy query; without a usable device the calls query
  p.attn_dev = -1;
  int dev = -1, g0 = 0, g1 = 0;
  if (hipGetDevice(&dev) == hipSuccess &&
      tactic::attn_resident_grid((int)p.GV, (int)(p.B * p.NV), false, &g0) == hipSuccess &&
      tactic::attn_resident_grid((int)p.GV, (int)(p.B * p.NV), true, &g1) == hipSuccess) {
    p.attn_dev = dev;
    p.attn_res[0] = g0;
    p.attn_res[1] = g1;
  } else {
    (void)hipGetLastError();  // leave no error behind for the next launch check
  }
  memcpy(plan_out, &p, sizeof(p));
  *workspace_bytes = (size_t)p.ws_bytes;
  return TACTIC_OK;
}

// The sparse decode launch sequence; pk non-null reads K/V through a page table.
static tactic_status sparse_decode_impl(const uint16_t* q, const uint16_t* K_sorted, const uint16_t* V_sorted,
                                   const tactic::PagedKV* pk,
                                   const tactic_kv_shape* shape, const tactic_cluster_meta* meta,
                                   const tactic_decode_params* params, const tactic_decode_plan* plan_in,
                                   float* out, int32_t* sel_count_q, int32_t* sel_count_kv, void* workspace,
                                   size_t workspace_bytes, hipStream_t stream) {
  tactic_status st = check_shape(shape);
  if (st != TACTIC_OK) return st;
  if ((st = check_params(params)) != TACTIC_OK) return st;
  if (!q || !K_sorted || !V_sorted || !meta || !out || !sel_count_q || !sel_count_kv || !plan_in)
    return fail(TACTIC_ERR_INVALID_ARG, "null argument");
  if (!meta->cl_indptr || !meta->centroids || !meta->offsets)
    return fail(TACTIC_ERR_INVALID_ARG, "null cluster meta pointer");
  const tactic::DecodePlan& p = *as_plan(plan_in);
  if (p.magic != tactic::kPlanMagic || p.B != shape->batch || p.Hq != shape->n_q_heads ||
      p.Hkv != shape->n_kv_heads || p.nmax != shape->max_seq_len || p.total != shape->total_tokens ||
      p.Cm != meta->max_clusters || p.Ct != meta->total_clusters || p.exact_bp != params->exact_bp ||
      p.win_bp != params->win_bp || p.win_min != params->win_min || p.p1_bp != params->p1_bp ||
      p.p2_bp != params->p2_bp || p.use_union != params->use_union || p.max_tail != params->max_tail)
    return fail(TACTIC_ERR_INVALID_ARG, "plan does not match the shape / meta / params");
  if (!workspace || (int64_t)workspace_bytes < p.ws_bytes)
    return fail(TACTIC_ERR_WORKSPACE, "workspace has %zu bytes, needs %lld", workspace_bytes,
                (long long)p.ws_bytes);

  char* ws = static_cast<char*>(workspace);
  const int BH = (int)(p.B * p.Hq), BG = (int)(p.B * p.Hkv), BV = (int)(p.B * p.NV);
  const bool timed = p.events[0] != 0;
  auto record = [&](int i) -> hipError_t {
    return timed ? hipEventRecord(reinterpret_cast<hipEvent_t>(p.events[i]), stream) : hipSuccess;
  };
  hipError_t e = record(0);
  if (e != hipSuccess) return hip_fail(e, "event record");

  tactic::ScoreArgs sa{};
  sa.q = q;
  sa.centroids = meta->centroids;
  sa.cl_indptr = meta->cl_indptr;
  sa.B = (int)p.B;
  sa.Hq = (int)p.Hq;
  sa.Hkv = (int)p.Hkv;
  sa.Cm = (int)p.Cm;
  sa.Ct = p.Ct;
  sa.scores = reinterpret_cast<float*>(ws + p.off_scores);
  e = tactic::launch_score(sa, (int)p.G, (int)((p.Cm + tactic::kScoreRows - 1) / tactic::kScoreRows), BG, stream);
  if (e == hipSuccess) e = record(1);
  if (e != hipSuccess) return hip_fail(e, "score_clusters launch");

  tactic::SortArgs so{};
  so.scores = sa.scores;
  so.offsets = meta->offsets;
  so.kv_indptr = shape->kv_indptr;
  so.seq_len = shape->seq_len;
  so.cl_indptr = meta->cl_indptr;
  so.B = (int)p.B;
  so.Hq = (int)p.Hq;
  so.Hkv = (int)p.Hkv;
  so.G = (int)p.G;
  so.Cm = (int)p.Cm;
  so.nb_max = (int)p.nb_max;
  so.Ct = p.Ct;
  so.S_cap = p.S_cap;
  so.max_tail = (int)p.max_tail;
  so.prm = sel_params(params);
  so.g_keys = p.sort_lds ? nullptr : reinterpret_cast<uint64_t*>(ws + p.off_sort_keys);
  so.g_cnt = p.sort_lds ? nullptr : reinterpret_cast<uint32_t*>(ws + p.off_sort_cnt);
  so.g_start = p.sort_lds ? nullptr : reinterpret_cast<uint32_t*>(ws + p.off_sort_start);
  so.order = reinterpret_cast<int32_t*>(ws + p.off_order);
  so.rank_of = reinterpret_cast<int32_t*>(ws + p.off_rank);
  so.rprefix = reinterpret_cast<int32_t*>(ws + p.off_rprefix);
  so.sample_rows = reinterpret_cast<int32_t*>(ws + p.off_rows);
  so.head_meta = reinterpret_cast<int32_t*>(ws + p.off_headmeta);
  so.per_head = p.use_union ? 0 : 1;
  so.sel_count_kv = sel_count_kv;
  e = tactic::launch_sort(so, p.sort_lds != 0, BH, stream);
  if (e == hipSuccess) e = record(2);
  if (e != hipSuccess) return hip_fail(e, "sort_clusters launch");

  tactic::FitArgs fa{};
  fa.q = q;
  fa.K = K_sorted;
  fa.kv_indptr = shape->kv_indptr;
  fa.cl_indptr = meta->cl_indptr;
  fa.offsets = meta->offsets;
  fa.B = (int)p.B;
  fa.Hq = (int)p.Hq;
  fa.Hkv = (int)p.Hkv;
  fa.G = (int)p.G;
  fa.Cm = (int)p.Cm;
  fa.BH = BH;
  fa.split = (int)p.split;
  fa.NV = (int)p.NV;
  fa.kv_div = p.use_union ? 1 : (int)p.G;
  fa.per_head = p.use_union ? 0 : 1;
  fa.Ct = p.Ct;
  fa.total = p.total;
  fa.S_cap = p.S_cap;
  fa.chunk_tokens = p.chunk_tokens;
  fa.max_chunks = p.max_chunks;
  fa.P = (double)params->target_frac;
  fa.head_meta = so.head_meta;
  fa.sample_rows = so.sample_rows;
  fa.rprefix = so.rprefix;
  fa.rank_of = so.rank_of;
  fa.order = so.order;
  fa.logits = reinterpret_cast<double*>(ws + p.off_logit);
  fa.fit = reinterpret_cast<double*>(ws + p.off_fit);
  fa.lse = reinterpret_cast<double*>(ws + p.off_lse);
  fa.cut = reinterpret_cast<int32_t*>(ws + p.off_cut);
  fa.sel_count_q = sel_count_q;
  fa.sel_count_kv = sel_count_kv;
  fa.union_len = reinterpret_cast<int32_t*>(ws + p.off_union_len);
  fa.gmeta = reinterpret_cast<int32_t*>(ws + p.off_gmeta);
  fa.rstart = reinterpret_cast<int32_t*>(ws + p.off_rstart);
  fa.rupos = reinterpret_cast<int32_t*>(ws + p.off_rupos);
  fa.cfr = reinterpret_cast<int32_t*>(ws + p.off_cfr);
  fa.slice_tot = reinterpret_cast<uint64_t*>(ws + p.off_slice_tot);
  if (pk) fa.pk = *pk;
  e = tactic::launch_sample(fa, (int)p.split, BH, pk != nullptr, stream);
  if (e == hipSuccess) e = record(3);
  if (e != hipSuccess) return hip_fail(e, "sample_logits launch");
  e = tactic::launch_fit_union(fa, (int)p.GV, BV, stream);
  if (e == hipSuccess) e = record(4);
  if (e != hipSuccess) return hip_fail(e, "fit_union launch");

  tactic::AttnArgs aa{};
  aa.q = q;
  aa.K = K_sorted;
  aa.V = V_sorted;
  aa.kv_indptr = shape->kv_indptr;
  aa.seq_len = shape->seq_len;
  aa.B = (int)p.B;
  aa.Hq = (int)p.Hq;
  aa.Hkv = (int)p.Hkv;
  aa.Cm = (int)p.Cm;
  aa.dense = 0;
  aa.NV = fa.NV;
  aa.kv_div = fa.kv_div;
  aa.total = p.total;
  aa.chunk_tokens = p.chunk_tokens;
  aa.max_chunks = p.max_chunks;
  aa.gmeta = fa.gmeta;
  aa.rstart = fa.rstart;
  aa.rupos = fa.rupos;
  aa.cfr = fa.cfr;
  aa.partials = reinterpret_cast<float*>(ws + p.off_partials);
  aa.ameta = reinterpret_cast<int64_t*>(ws + p.off_ameta);
  aa.head_meta = so.head_meta;
  if (pk) aa.pk = *pk;
  aa.out = out;
  int grid = 0, dev = -1;
  e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev == p.attn_dev) {
    grid = (int)p.attn_res[pk != nullptr ? 1 : 0];
  } else {
    e = tactic::attn_resident_grid((int)p.GV, BV, pk != nullptr, &grid);
    if (e != hipSuccess) return hip_fail(e, "attention occupancy query");
  }
  grid = (int)std::min<int64_t>(grid, p.attn_grid);  // the partials are sized for attn_grid
  e = tactic::launch_attn(aa, (int)p.GV, grid, pk != nullptr, stream);
  if (e == hipSuccess) e = record(5);
  if (e != hipSuccess) return hip_fail(e, "attention launch");
  e = tactic::launch_combine(aa, (int)p.GV, stream);
  if (e == hipSuccess) e = record(6);
  if (e != hipSuccess) return hip_fail(e, "combine launch");
  return TACTIC_OK;
}

tactic_status tactic_sparse_decode(const uint16_t* q, const uint16_t* K_sorted, const uint16_t* V_sorted,
                                   const tactic_kv_shape* shape, const tactic_cluster_meta* meta,
                                   const tactic_decode_params* params, const tactic_decode_plan* plan_in,
                                   float* out, int32_t* sel_count_q, int32_t* sel_count_kv, void* workspace,
                                   size_t workspace_bytes, hipStream_t stream) {
  return sparse_decode_impl(q, K_sorted, V_sorted, nullptr, shape, meta, params, plan_in, out, sel_count_q,
                            sel_count_kv, workspace, workspace_bytes, stream);
}

}  // extern "C"

// Scratch of the no-alloc decode: one array per device, from the code object's
// own data (allocated when the library is loaded on that device, held until the
// process ends).  Host code never uses the array's name as an address: the
// device address of each device's copy comes from hipGetSymbolAddress.
namespace {
constexpr size_t kScratchBytes = TACTIC_NOALLOC_SCRATCH_BYTES;
__device__ __align__(256) unsigned char scratch[kScratchBytes];
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxScratchDevices];  // device address of `scratch` per device, or null

tactic_status scratch_on_current_device(void** addr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxScratchDevices)
    return fail(TACTIC_ERR_UNSUPPORTED, "device %d: the scratch table holds %d devices", dev, kMaxScratchDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!p) return fail(TACTIC_ERR_HIP, "hipGetSymbolAddress(scratch) returned a null address");
    g_scratch_addr[dev] = p;
  }
  *addr = g_scratch_addr[dev];
  return TACTIC_OK;
}
}  // namespace

extern "C" {

tactic_status tactic_sparse_decode_noalloc(const uint16_t* q, const uint16_t* K_sorted, const uint16_t* V_sorted,
                                           const tactic_kv_shape* shape, const tactic_cluster_meta* meta,
                                           const tactic_decode_params* params, const tactic_decode_plan* plan_in,
                                           float* out, int32_t* sel_count_q, int32_t* sel_count_kv,
                                           hipStream_t stream) {
  if (!plan_in) return fail(TACTIC_ERR_INVALID_ARG, "null plan");
  const tactic::DecodePlan& p = *as_plan(plan_in);
  if (p.magic != tactic::kPlanMagic) return fail(TACTIC_ERR_INVALID_ARG, "not a decode plan");
  if (p.ws_bytes > (int64_t)kScratchBytes)
    return fail(TACTIC_ERR_WORKSPACE, "the shape needs %lld bytes of workspace; the static scratch of "
                "tactic_sparse_decode_noalloc holds %zu", (long long)p.ws_bytes, kScratchBytes);
  void* ws = nullptr;
  const tactic_status st = scratch_on_current_device(&ws);
  if (st != TACTIC_OK) return st;
  // the decode needs no zeroed workspace: every kernel writes what it reads later
  return sparse_decode_impl(q, K_sorted, V_sorted, nullptr, shape, meta, params, plan_in, out, sel_count_q,
                            sel_count_kv, ws, kScratchBytes, stream);
}

tactic_status tactic_sparse_decode_paged(const uint16_t* q, const tactic_paged_kv* kv,
                                         const tactic_kv_shape* shape, const tactic_cluster_meta* meta,
                                         const tactic_decode_params* params, const tactic_decode_plan* plan_in,
                                         float* out, int32_t* sel_count_q, int32_t* sel_count_kv,
                                         void* workspace, size_t workspace_bytes, hipStream_t stream) {
  tactic_status st = check_shape(shape);
  if (st != TACTIC_OK) return st;
  tactic::PagedKV pk;
  if ((st = paged_args(kv, shape, &pk)) != TACTIC_OK) return st;
  return sparse_decode_impl(q, kv->K_pages, kv->V_pages, &pk, shape, meta, params, plan_in, out, sel_count_q,
                            sel_count_kv, workspace, workspace_bytes, stream);
}

tactic_status tactic_sparse_decode_plan_set_events(tactic_decode_plan* plan_in, hipEvent_t* events) {
  if (!plan_in) return fail(TACTIC_ERR_INVALID_ARG, "null plan");
  tactic::DecodePlan* p = reinterpret_cast<tactic::DecodePlan*>(plan_in);
  if (p->magic != tactic::kPlanMagic) return fail(TACTIC_ERR_INVALID_ARG, "not a decode plan");
  for (int i = 0; i < tactic::kStageEvents; ++i) {
    if (events && !events[i]) return fail(TACTIC_ERR_INVALID_ARG, "event %d is null", i);
    p->events[i] = events ? reinterpret_cast<int64_t>(events[i]) : 0;
  }
  return TACTIC_OK;
}

tactic_status tactic_sparse_decode_view(const tactic_decode_plan* plan_in, const void* workspace,
                                        tactic_decode_view* view) {
  if (!plan_in || !workspace || !view) return fail(TACTIC_ERR_INVALID_ARG, "null argument");
  const tactic::DecodePlan& p = *as_plan(plan_in);
  if (p.magic != tactic::kPlanMagic) return fail(TACTIC_ERR_INVALID_ARG, "not a decode plan");
  const char* ws = static_cast<const char*>(workspace);
  view->scores = reinterpret_cast<const float*>(ws + p.off_scores);
  view->order = reinterpret_cast<const int32_t*>(ws + p.off_order);
  view->rank_prefix = reinterpret_cast<const int32_t*>(ws + p.off_rprefix);
  view->fit = reinterpret_cast<const double*>(ws + p.off_fit);
  view->union_len = reinterpret_cast<const int32_t*>(ws + p.off_union_len);
  view->sample_rows = reinterpret_cast<const int32_t*>(ws + p.off_rows);
  view->sample_cap = p.S_cap;
  return TACTIC_OK;
}

size_t tactic_dense_decode_workspace_size(const tactic_kv_shape* shape) {
  if (check_shape(shape) != TACTIC_OK) return 0;
  return dense_workspace_bytes(shape, tactic::kMaxAttnGrid);
}

static tactic_status dense_decode_impl(const uint16_t* q, const uint16_t* K, const uint16_t* V,
                                       const tactic::PagedKV* pk, const tactic_kv_shape* shape, float* out,
                                       void* workspace, size_t workspace_bytes, hipStream_t stream) {
  tactic_status st = check_shape(shape);
  if (st != TACTIC_OK) return st;
  if (!q || !K || !V || !out) return fail(TACTIC_ERR_INVALID_ARG, "null argument");
  const int64_t BG = (int64_t)shape->batch * shape->n_kv_heads;
  const int G = shape->n_q_heads / shape->n_kv_heads;
  const size_t need = dense_workspace_bytes(shape, tactic::kMaxAttnGrid);
  if (!workspace || workspace_bytes < need)
    return fail(TACTIC_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, need);
  int resident = 0;
  hipError_t e = tactic::attn_resident_grid(G, (int)BG, pk != nullptr, &resident);
  if (e != hipSuccess) return hip_fail(e, "attention occupancy query");
  resident = std::min(resident, tactic::kMaxAttnGrid);
  tactic::AttnArgs aa{};
  memset(&aa, 0, sizeof(aa));
  aa.q = q;
  aa.K = K;
  aa.V = V;
  aa.kv_indptr = shape->kv_indptr;
  aa.seq_len = shape->seq_len;
  aa.B = shape->batch;
  aa.Hq = shape->n_q_heads;
  aa.Hkv = shape->n_kv_heads;
  aa.dense = 1;
  aa.NV = shape->n_kv_heads;
  aa.kv_div = 1;
  aa.total = shape->total_tokens;
  aa.partials = static_cast<float*>(workspace);
  {
    Layout L;  // same layout as dense_workspace_bytes
    L.take((BG + tactic::kMaxAttnGrid) * G * (tactic::kHeadDim + 2) * 4);
    aa.ameta = reinterpret_cast<int64_t*>(static_cast<char*>(workspace) + L.take((BG + 2) * 8));
  }
  if (pk) aa.pk = *pk;
  aa.out = out;
  e = tactic::launch_attn(aa, G, resident, pk != nullptr, stream);
  if (e == hipSuccess) e = tactic::launch_combine(aa, G, stream);
  if (e != hipSuccess) return hip_fail(e, "dense attention launch");
  return TACTIC_OK;
}

tactic_status tactic_dense_decode(const uint16_t* q, const uint16_t* K, const uint16_t* V,
                                  const tactic_kv_shape* shape, float* out, void* workspace,
                                  size_t workspace_bytes, hipStream_t stream) {
  return dense_decode_impl(q, K, V, nullptr, shape, out, workspace, workspace_bytes, stream);
}

tactic_status tactic_dense_decode_paged(const uint16_t* q, const tactic_paged_kv* kv,
                                        const tactic_kv_shape* shape, float* out, void* workspace,
                                        size_t workspace_bytes, hipStream_t stream) {
  tactic_status st = check_shape(shape);
  if (st != TACTIC_OK) return st;
  tactic::PagedKV pk;
  if ((st = paged_args(kv, shape, &pk)) != TACTIC_OK) return st;
  pk.perm = nullptr;  // dense decode reads positions: no cluster order
  return dense_decode_impl(q, kv->K_pages, kv->V_pages, &pk, shape, out, workspace, workspace_bytes, stream);
}

tactic_status tactic_probe_stream_read(const void* buf, size_t bytes, int32_t workgroups, uint32_t* sink,
                                       hipStream_t stream) {
  if (!buf || !sink || bytes == 0 || bytes % 16 != 0 || workgroups < 0)
    return fail(TACTIC_ERR_INVALID_ARG, "stream read probe: null pointer, a size that is not a multiple of 16 "
                "or a negative workgroup count");
  const hipError_t e = tactic::launch_stream_read(buf, bytes / 16, workgroups, sink, stream);
  if (e != hipSuccess) return hip_fail(e, "stream read launch");
  return TACTIC_OK;
}

size_t tactic_build_clusters_workspace_size(const tactic_kv_shape* shape, int64_t total_clusters,
                                            int32_t max_clusters) {
  if (check_shape(shape) != TACTIC_OK || max_clusters < 1 || total_clusters < max_clusters) return 0;
  return tactic::kmeans_workspace_bytes(shape->batch, shape->n_kv_heads, shape->total_tokens,
                                        total_clusters, max_clusters, shape->max_seq_len);
}

tactic_status tactic_build_clusters(const uint16_t* K, const uint16_t* V, const tactic_kv_shape* shape,
                                    const int64_t* cl_indptr, int64_t total_clusters, int32_t max_clusters,
                                    const int32_t* init_idx, const tactic_kmeans_params* params,
                                    uint16_t* centroids, int32_t* assign, int32_t* offsets, int32_t* perm,
                                    uint16_t* K_sorted, uint16_t* V_sorted, void* workspace,
                                    size_t workspace_bytes, hipStream_t stream) {
  tactic_status st = check_shape(shape);
  if (st != TACTIC_OK) return st;
  if (!K || !cl_indptr || !init_idx || !params || !centroids || !assign || !offsets || !perm)
    return fail(TACTIC_ERR_INVALID_ARG, "null argument");
  if ((K_sorted != nullptr || V_sorted != nullptr) && (V_sorted != nullptr) && !V)
    return fail(TACTIC_ERR_INVALID_ARG, "V_sorted requested without V");
  if (max_clusters < 1 || total_clusters < max_clusters ||
      total_clusters > (int64_t)max_clusters * shape->batch)
    return fail(TACTIC_ERR_INVALID_ARG, "inconsistent total_clusters / max_clusters");
  if (params->max_iters < 1 || params->max_iters > 1000)
    return fail(TACTIC_ERR_INVALID_ARG, "max_iters must be in [1, 1000]");
  if (max_clusters >= (1 << 21)) return fail(TACTIC_ERR_UNSUPPORTED, "more than 2^21 - 1 clusters");
  if ((params->prev_centroids == nullptr) != (params->prev_cl_indptr == nullptr))
    return fail(TACTIC_ERR_INVALID_ARG, "prev_centroids and prev_cl_indptr must be set together");
  const size_t need = tactic_build_clusters_workspace_size(shape, total_clusters, max_clusters);
  if (!workspace || workspace_bytes < need)
    return fail(TACTIC_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, need);
  hipError_t e = tactic::run_kmeans(K, V, shape->kv_indptr, shape->seq_len, cl_indptr, shape->batch, shape->n_kv_heads,
                                    shape->total_tokens, shape->max_seq_len, total_clusters, max_clusters,
                                    init_idx, params->max_iters, params->prev_centroids, params->prev_cl_indptr,
                                    centroids, assign, offsets, perm, K_sorted,
                                    V_sorted, workspace, stream);
  if (e != hipSuccess) return hip_fail(e, "k-means launch");
  return TACTIC_OK;
}

}  // extern "C"
