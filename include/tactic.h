/*
 * tactic.h - C ABI of the MI355X (gfx950) library for Tactic's decode-time
 * sparse attention ("Tactic: Adaptive Sparse Attention with Clustering and
 * Distribution Fitting for Long-Context LLMs").
 *
 * Problem statement (Sec. 3.3 - 3.5): given a decode query q, the cached keys
 * K and values V of n tokens and a target fraction P, return the attention
 * output over a small index set I whose cumulative attention score p(I)
 * (Eq. 5) reaches P.  The set is found as in Sec. 4: keys are grouped by
 * K-means at prefill (Sec. 4.2); at decode every query head ranks the clusters
 * by q . centroid (Sec. 4.3), fits y = a/x + b to sampled scores to estimate
 * its token budget (Sec. 4.4, Algorithm 1), the query heads of a GQA group
 * take the union of their selections (Sec. 4.5), and attention runs over the
 * selected tokens only (Sec. 4.6, Eq. 3).
 *
 * Conventions for every call
 *  - All tensor arguments are DEVICE pointers unless a field says "host".
 *  - bf16 values are passed as uint16_t bit patterns.  head_dim must be 128.
 *  - A ragged batch of B sequences: sequence b owns tokens
 *    [kv_indptr[b], kv_indptr[b+1]) of every per-KV-head array; K and V are
 *    laid out [Hkv][total_tokens][128] (head-major).  Query head h uses KV
 *    head h / (Hq / Hkv).  Sequence lengths must be below 2^31.
 *  - Every call is asynchronous on `stream` and does not synchronise with
 *    the host.  Argument checks that need only host data are done before any
 *    launch; a failed check returns an error and launches nothing.  Device
 *    arrays are trusted to match the host-side sizes given (a mismatch is
 *    undefined behaviour).
 *  - The library allocates no memory and keeps no global state: the caller
 *    owns every buffer, including the workspace.  Calls that share a
 *    workspace must be ordered on one stream.  The one exception is the
 *    static scratch of tactic_sparse_decode_noalloc (see there).
 */
#ifndef TACTIC_H_
#define TACTIC_H_

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  TACTIC_OK = 0,
  TACTIC_ERR_INVALID_ARG = 1,  /* a null pointer, a size out of range, P outside (0, 1] ... */
  TACTIC_ERR_UNSUPPORTED = 2,  /* a valid request the library does not implement (e.g. head_dim != 128) */
  TACTIC_ERR_WORKSPACE = 3,    /* workspace smaller than the size query returned */
  TACTIC_ERR_HIP = 4           /* a HIP launch failed; tactic_last_error() has the message */
} tactic_status;

/* Shape of a ragged decode batch. */
typedef struct {
  int32_t batch;               /* B >= 1 */
  int32_t n_q_heads;           /* Hq, a multiple of n_kv_heads; Hq / Hkv in {1, 2, 4, 8} */
  int32_t n_kv_heads;          /* Hkv >= 1 */
  int32_t head_dim;            /* must be 128 */
  int64_t total_tokens;        /* host: kv_indptr[B], the row count of every per-KV-head array */
  int64_t max_seq_len;         /* host: largest kv_indptr[b+1] - kv_indptr[b] */
  const int64_t* kv_indptr;    /* device [B+1], kv_indptr[0] = 0, non-decreasing: sequence b's
                                  rows start at kv_indptr[b] */
  const int64_t* seq_len;      /* device [B] or NULL: sequence b holds rows kv_indptr[b] ..
                                  kv_indptr[b] + seq_len[b] - 1 (clamped to kv_indptr[b+1]); the
                                  rest of its span is spare room for new tokens.  NULL: the
                                  whole span kv_indptr[b] .. kv_indptr[b+1] - 1. */
} tactic_kv_shape;

/* Cluster description of a cluster-sorted KV cache (the output of
 * tactic_build_clusters, or any caller-made grouping).  Sequence b has C_b
 * clusters per KV head (C_b >= 1 when the sequence is non-empty); they are
 * clusters [cl_indptr[b], cl_indptr[b+1]) of every per-KV-head cluster array.
 * Cluster j of (b, g) owns the rows offsets_bg[j] .. offsets_bg[j+1]-1 of the
 * sequence's cluster-sorted K/V, where offsets_bg = offsets + g*(total_clusters
 * + B) + cl_indptr[b] + b holds C_b + 1 sequence-relative offsets from 0 to
 * c_b <= n_b.  Within a cluster, rows keep their original token order (Sec.
 * 4.3 unpacks clusters in that stored order).  Rows c_b .. n_b-1 are the
 * recent tokens generated since the clustering (the same count for every KV
 * head of the sequence): every head attends to all of them and their exact
 * attention mass counts toward the target (Sec. 1: full attention on newly
 * generated tokens until the next re-clustering). */
typedef struct {
  int64_t total_clusters;      /* host: sum of C_b */
  int32_t max_clusters;        /* host: largest C_b */
  const int64_t* cl_indptr;    /* device [B+1] */
  const uint16_t* centroids;   /* device bf16 [Hkv][total_clusters][128] */
  const int32_t* offsets;      /* device int32 [Hkv][total_clusters + B] */
} tactic_cluster_meta;

/* Parameters of the decode selection.  The fractions are integers in basis
 * points (1 bp = 1e-4) so that the library and any checker derive identical
 * integer sizes.  For a list of n tokens:
 *   exact head  N = min(n, max(1, ceil(n * exact_bp / 1e4)))     (Sec. 4.4: 1-2%)
 *   window      W = max(win_min, ceil(n * win_bp / 1e4))
 *   centres     c_j = floor((n * p_j_bp + 5000) / 1e4)           (Sec. 4.4: 10%, 60%)
 *   window j    s_j = max(c_j - floor(W/2), N + 1), t_j = min(s_j + W - 1, n)
 * If a window is empty, the windows overlap or N = n, every score of the list
 * is computed exactly instead of fitted. */
typedef struct {
  float target_frac;           /* P in (0, 1]; P = 1 selects every token (dense) */
  int32_t exact_bp;            /* default 100  (N = 1% of the tokens) */
  int32_t win_bp;              /* default 50   (W = 0.5% of the tokens) */
  int32_t win_min;             /* default 8 */
  int32_t p1_bp;               /* default 1000 */
  int32_t p2_bp;               /* default 6000 */
  int32_t use_union;           /* 1 (default): every head of a GQA group attends over the union
                                  of the group's selections, loaded once (Sec. 4.5).  0: every
                                  query head attends over its own selection only (the ablation
                                  partner of the union, Sec. 5.3); sel_count_kv then counts the
                                  K/V rows loaded for the KV head, i.e. the sum of the group's
                                  per-head counts.  Other values: TACTIC_ERR_INVALID_ARG. */
  int32_t max_tail;            /* default 0: the most recent (unclustered) tokens any sequence
                                  may have, n_b - c_b.  Sizes the workspace; a longer tail is
                                  cut to its first max_tail tokens (memory-safe, but then the
                                  result leaves the rest out).  Negative: INVALID_ARG. */
} tactic_decode_params;

/* Host-side launch plan of a sparse decode: sizes derived from the shape,
 * the cluster counts and the parameters (done once per shape; it costs
 * O(max_seq_len) host time).  Plain data owned by the caller. */
typedef struct {
  int64_t v[64];
} tactic_decode_plan;

/* Fills `p` with the defaults listed above and target_frac = 0.9. */
void tactic_decode_params_default(tactic_decode_params* p);

/* Validates shape, cluster counts and parameters and fills `plan`.
 * *workspace_bytes receives the workspace size tactic_sparse_decode needs.
 * meta's device pointers are not read and may be null here.  The plan also
 * records how many attention workgroups fit at once on the device current at
 * this call, so that decode calls on that device make no occupancy query
 * (calls on another device make it).  At most 4096 selection groups: B * Hkv,
 * or B * Hq with use_union = 0.
 * Errors: TACTIC_ERR_INVALID_ARG, TACTIC_ERR_UNSUPPORTED. */
tactic_status tactic_sparse_decode_plan(const tactic_kv_shape* shape,
                                        const tactic_cluster_meta* meta,
                                        const tactic_decode_params* params,
                                        tactic_decode_plan* plan,
                                        size_t* workspace_bytes);

/* Tactic's decode for one layer (Sec. 4.3 - 4.6, Algorithm 1).
 *   q          bf16 [B][Hq][128]
 *   K_sorted,  bf16 [Hkv][total_tokens][128], rows in the cluster-sorted
 *   V_sorted   order that `meta` describes
 *   out        fp32 [B][Hq][128]: attention of each query head over the
 *              union of its group's selected tokens (use_union = 1) or over
 *              its own selection (use_union = 0), softmax renormalised over
 *              that set (Eq. 3); zeros for an empty sequence
 *   sel_count_q   int32 [B][Hq]: tokens head h attends to of its own selection:
 *              the budget k_h of Algorithm 1 plus the recent tokens
 *   sel_count_kv  int32 [B][Hkv]: size of the group union |U_g| (use_union = 1),
 *              or the sum of the group's k_h (use_union = 0): K/V rows loaded
 *   workspace  at least the bytes reported by tactic_sparse_decode_plan for
 *              the same arguments; contents on entry are irrelevant.
 * The plan must come from the same shape, meta sizes and params. */
tactic_status tactic_sparse_decode(const uint16_t* q, const uint16_t* K_sorted,
                                   const uint16_t* V_sorted, const tactic_kv_shape* shape,
                                   const tactic_cluster_meta* meta,
                                   const tactic_decode_params* params,
                                   const tactic_decode_plan* plan, float* out,
                                   int32_t* sel_count_q, int32_t* sel_count_kv,
                                   void* workspace, size_t workspace_bytes,
                                   hipStream_t stream);

/* The same decode for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * it takes no workspace and calls no allocating routine.  Its workspace is a
 * static scratch array of TACTIC_NOALLOC_SCRATCH_BYTES in the library's device
 * code, one copy per GPU, held from the library's load on that GPU until the
 * process ends (its device address is looked up once per device, at the first
 * call there).  A plan whose workspace exceeds it gives TACTIC_ERR_WORKSPACE
 * before any launch.  Every call on a GPU uses that GPU's one array, which
 * keeps the last call's contents: calls that overlap on one GPU (other
 * streams, other threads) race and must be ordered by the caller.  The
 * decode needs no zeroed workspace.  Arguments, outputs and errors are those
 * of tactic_sparse_decode. */
#define TACTIC_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
tactic_status tactic_sparse_decode_noalloc(const uint16_t* q, const uint16_t* K_sorted,
                                           const uint16_t* V_sorted, const tactic_kv_shape* shape,
                                           const tactic_cluster_meta* meta,
                                           const tactic_decode_params* params,
                                           const tactic_decode_plan* plan, float* out,
                                           int32_t* sel_count_q, int32_t* sel_count_kv,
                                           hipStream_t stream);

/* Optional per-stage timing: with events set (an array of 7 created events,
 * or NULL to clear), every tactic_sparse_decode with this plan records
 * events[0] before its first kernel and events[1..6] after each of its six
 * kernels (centroid scoring, cluster sort, sampled logits, fit + union,
 * attention, combine) on the call's stream.  The events stay owned by the
 * caller. */
tactic_status tactic_sparse_decode_plan_set_events(tactic_decode_plan* plan, hipEvent_t* events);

/* Number of fp64 fields per query head in the fit record of the view below:
 *   0 m (logit shift: max over the exact head)   1 mu_1   2 mu_2   3 a   4 b
 *   5 S_n (estimated total)   6 T = P * S_n   7 k   8 N   9 n   10 exact mode
 *   11 sampled rows   12 E_N (exact-head sum)   13 cutoff rank   14 cutoff length
 *   15 E_t (exact mass of the recent tokens; S_n and T include it) */
#define TACTIC_FIT_FIELDS 16

/* Device pointers into a workspace after tactic_sparse_decode, for
 * inspecting the intermediate stages (cluster order, fit, union).  Valid
 * until the workspace is reused. */
typedef struct {
  const float* scores;         /* [B][Hq][max_clusters]: q . centroid (fp32) */
  const int32_t* order;        /* [B][Hq][max_clusters]: cluster ids by rank */
  const int32_t* rank_prefix;  /* [B][Hq][max_clusters + 1]: tokens ahead of each rank */
  const double* fit;           /* [B][Hq][TACTIC_FIT_FIELDS] */
  const int32_t* union_len;    /* [Hkv][total_clusters] (use_union = 1) or
                                  [Hq][total_clusters] (use_union = 0): rows of each cluster
                                  in the group's union or the head's selection (a prefix of
                                  the cluster) */
  const int32_t* sample_rows;  /* [B][Hq][sample_cap]: sequence-relative cache rows whose keys the
                                  head sampled (exact head 1..N, window 1, window 2, then the
                                  recent tokens); the first `sampled rows` (fit field 11) are valid */
  int64_t sample_cap;
} tactic_decode_view;

tactic_status tactic_sparse_decode_view(const tactic_decode_plan* plan, const void* workspace,
                                        tactic_decode_view* view);

/* Dense decode attention over every token (Eq. 2), the baseline.  Same
 * layouts as tactic_sparse_decode (any row order works: attention does not
 * depend on it).  Workspace contents on entry are irrelevant. */
size_t tactic_dense_decode_workspace_size(const tactic_kv_shape* shape);
tactic_status tactic_dense_decode(const uint16_t* q, const uint16_t* K, const uint16_t* V,
                                  const tactic_kv_shape* shape, float* out, void* workspace,
                                  size_t workspace_bytes, hipStream_t stream);

/* A paged K/V cache (Sec. 4.6 reads the selected tokens from a paged cache
 * through sub-requests): instead of a cluster-sorted copy, the keys and
 * values stay in pages in token order and the cluster order reaches them
 * through `perm`.  Page p holds page_size consecutive tokens of one sequence
 * for every KV head; tokens [i*page_size, (i+1)*page_size) of sequence b are
 * in page page_table[b*max_pages + i].  Out-of-range table entries are
 * clamped (reads stay inside the arrays; the result is then meaningless). */
typedef struct {
  const uint16_t* K_pages;     /* device bf16 [num_pages][Hkv][page_size][128] */
  const uint16_t* V_pages;     /* device bf16, same layout */
  const int32_t* page_table;   /* device int32 [B][max_pages] */
  const int32_t* perm;         /* device int32 [Hkv][total_tokens]: sequence-relative token at each
                                  cluster-sorted row (the perm output of tactic_build_clusters),
                                  for the first c_b rows; rows from c_b on (recent tokens) are
                                  their own tokens.  NULL: the pages hold the tokens in cluster
                                  order already. */
  int32_t page_size;           /* tokens per page, >= 1 */
  int32_t max_pages;           /* page-table entries per sequence; max_pages * page_size >=
                                  max_seq_len and < 2^31 */
  int64_t num_pages;           /* host: pages in K_pages / V_pages; num_pages * Hkv * page_size < 2^31 */
} tactic_paged_kv;

/* tactic_sparse_decode over a paged cache: same selection, outputs, plan and
 * workspace; `shape` gives the sequence lengths (kv_indptr / seq_len) and the
 * row stride of `perm`. */
tactic_status tactic_sparse_decode_paged(const uint16_t* q, const tactic_paged_kv* kv,
                                         const tactic_kv_shape* shape,
                                         const tactic_cluster_meta* meta,
                                         const tactic_decode_params* params,
                                         const tactic_decode_plan* plan, float* out,
                                         int32_t* sel_count_q, int32_t* sel_count_kv,
                                         void* workspace, size_t workspace_bytes,
                                         hipStream_t stream);

/* tactic_dense_decode over a paged cache (perm is ignored: dense attention
 * reads every token); workspace as tactic_dense_decode_workspace_size. */
tactic_status tactic_dense_decode_paged(const uint16_t* q, const tactic_paged_kv* kv,
                                        const tactic_kv_shape* shape, float* out, void* workspace,
                                        size_t workspace_bytes, hipStream_t stream);

/* Prefill clustering (Sec. 4.2): per (sequence, KV head) K-means on the keys
 * with C_b clusters, started from the keys of the tokens init_idx names,
 * alternating nearest-centroid assignment (squared Euclidean distance, ties to
 * the smaller id) and centroid = mean of members (an empty cluster keeps its
 * centroid), for at most max_iters iterations or until an assignment step
 * changes nothing.  Centroids are stored in bf16 and each assignment measures
 * distances to the stored values.
 *   K, V          bf16 [Hkv][total_tokens][128], original token order
 *   cl_indptr     device [B+1] (C_b = cl_indptr[b+1] - cl_indptr[b], 1 <= C_b <= n_b)
 *   init_idx      device int32 [Hkv][total_clusters]: C_b distinct sequence-relative
 *                 token ids per (b, g) (entries of warm-started centroids are ignored)
 * Outputs: centroids bf16 [Hkv][total_clusters][128], assign int32 [Hkv][total_tokens]
 * (cluster of each original token), offsets int32 [Hkv][total_clusters + B] and perm
 * int32 [Hkv][total_tokens] (original token of each cluster-sorted row, ascending
 * within a cluster), K_sorted / V_sorted (the cache rows permuted by perm; either may
 * be null to skip it). */
typedef struct {
  int32_t max_iters;           /* default 10 (Sec. 4.2) */
  int32_t reserved;            /* 0 */
  /* Warm start (re-clustering, Sec. 1: the cache is re-clustered periodically
   * while decoding).  NULL: every centroid starts from init_idx.  Otherwise a
   * previous clustering of the same sequences and KV heads: prev_cl_indptr is
   * device int64 [B+1] (prev C_b = prev_cl_indptr[b+1] - prev_cl_indptr[b]) and
   * prev_centroids bf16 [Hkv][prev_cl_indptr[B]][128]; centroid j of (b, g)
   * starts from previous centroid j of (b, g) for j < min(C_b, prev C_b) (its
   * init_idx entry is ignored) and from the key init_idx names for the rest.
   * Both pointers are set or both are NULL (else TACTIC_ERR_INVALID_ARG); the
   * arrays are read by the first kernel only and must not overlap the
   * centroids output; prev C_b may be smaller or larger than C_b.  An all-zero
   * struct with max_iters set is a cold start. */
  const uint16_t* prev_centroids;
  const int64_t* prev_cl_indptr;
} tactic_kmeans_params;

size_t tactic_build_clusters_workspace_size(const tactic_kv_shape* shape, int64_t total_clusters,
                                            int32_t max_clusters);
tactic_status tactic_build_clusters(const uint16_t* K, const uint16_t* V,
                                    const tactic_kv_shape* shape, const int64_t* cl_indptr,
                                    int64_t total_clusters, int32_t max_clusters,
                                    const int32_t* init_idx, const tactic_kmeans_params* params,
                                    uint16_t* centroids, int32_t* assign, int32_t* offsets,
                                    int32_t* perm, uint16_t* K_sorted, uint16_t* V_sorted,
                                    void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Measurement helper, not part of the method: reads every 16-byte word of
 * `buf` (bytes, a multiple of 16) once with streaming loads from `workgroups`
 * workgroups of 256 threads (0: as many as fit on the device at once) and
 * stores nothing unless a read value equals a magic word (then one word to
 * *sink, a device uint32).  Its best rate over launch shapes is the device's
 * practical streaming-read ceiling, the yardstick of the bandwidth-bound
 * decode kernels.  Errors: TACTIC_ERR_INVALID_ARG, TACTIC_ERR_HIP. */
tactic_status tactic_probe_stream_read(const void* buf, size_t bytes, int32_t workgroups, uint32_t* sink,
                                       hipStream_t stream);

/* Static description of a status code. */
const char* tactic_status_string(tactic_status s);
/* Message of the last failure on the calling thread ("" if none). */
const char* tactic_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* TACTIC_H_ */
