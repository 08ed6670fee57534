// Token selection of Tactic's decode (Sec. 4.3 - 4.5, Algorithm 1) for gfx950.
//
//   score_clusters     q . centroid for every (query head, cluster)       Sec. 4.3
//   sort_clusters      per query head: cluster order (score desc, id asc),
//                      tokens ahead of every rank, sampled-row list        Sec. 4.3, Alg. 1 input
//   sample_logits      exact logits of the sampled rows (fp64)             Alg. 1
//   fit_union          per GQA group: fit y = a/x + b and the budget k of
//                      every head, then the union of the group's selections
//                      and the attention work list                         Sec. 4.4, 4.5, Alg. 1
//   union_ranges       (8192 to 65536 clusters per group, up to 4 heads: the
//                      union in slices) the slices' ranges end to end      Sec. 4.5, 4.6
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "common.hpp"
#include "kernels.hpp"
#include "plan.hpp"

namespace tactic {

// ============================================================================
// Block-wide helpers (any blockDim that is a multiple of 64, at most 1024)
// ============================================================================

// Exclusive scan in place of a[0..count) (LDS or global); returns the total.
// `s_wave` must hold 17 elements of T in LDS.  Ends with a barrier.
template <typename T>
__device__ T block_exclusive_scan(T* a, int count, T* s_wave) {
  const int tid = threadIdx.x, nt = blockDim.x, nw = nt / kWave;
  const int seg = (count + nt - 1) / nt;
  const int beg = min(count, tid * seg), end = min(count, beg + seg);
  T local = 0;
  for (int i = beg; i < end; ++i) local += a[i];
  T incl = wave_incl_scan(local);  // DPP, no LDS
  if ((tid & (kWave - 1)) == kWave - 1) s_wave[tid / kWave] = incl;
  __syncthreads();
  if (tid == 0) {
    T run = 0;
    for (int w = 0; w < nw; ++w) {
      const T t = s_wave[w];
      s_wave[w] = run;
      run += t;
    }
    s_wave[16] = run;
  }
  __syncthreads();
  T run = s_wave[tid / kWave] + incl - local;
  for (int i = beg; i < end; ++i) {
    const T t = a[i];
    a[i] = run;
    run += t;
  }
  const T total = s_wave[16];
  __syncthreads();
  return total;
}

// ============================================================================
// 1. Centroid scoring: s[b][h][j] = q_h . c_{b,g,j}, fp32 accumulation of
//    bf16 products (v_dot2).  grid (ceil(Cm/kScoreRows), B*Hkv), 256 threads;
//    16 lanes own one centroid row (16 B each), a wave scores 4 rows per step
//    with 4 steps of loads in flight; the group's G query heads sit in
//    registers.
// ============================================================================
template <int G>
__global__ __launch_bounds__(256) void score_clusters_kernel(ScoreArgs a) {
  const int bg = blockIdx.y;
  const int b = bg / a.Hkv, g = bg % a.Hkv;
  const int64_t cb = a.cl_indptr[b];
  const int C = min((int)(a.cl_indptr[b + 1] - cb), a.Cm);
  const int j0 = blockIdx.x * kScoreRows;
  if (j0 >= C) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, sl = lane & 15, grp = lane >> 4;

  uint32_t qw[G][4];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const uint4 v = *reinterpret_cast<const uint4*>(a.q + ((int64_t)b * a.Hq + g * G + h) * kHeadDim + sl * 8);
    qw[h][0] = v.x; qw[h][1] = v.y; qw[h][2] = v.z; qw[h][3] = v.w;
  }
  const uint16_t* cbase = a.centroids + ((int64_t)g * a.Ct + cb) * kHeadDim + sl * 8;
  float* sc = a.scores + ((int64_t)b * a.Hq + g * G) * a.Cm;
  constexpr int kPerWave = kScoreRows / 4;  // rows per wave, 4 per step
  constexpr int kSteps = kPerWave / 4;
  // after sum16 all 16 lanes of a row hold its G scores; lane sl keeps the
  // score of head sl % G of step sl / G of a window of P steps, and the
  // window goes out as one store of P * 4 consecutive rows per head
  constexpr int P = 16 / G;
  float keep = 0.f;
  auto flush = [&](int s0, int ns) {
    const int sp = sl / G, h = sl % G;
    const int j = j0 + wave * kPerWave + (s0 + sp) * 4 + grp;
    if (sp < ns && j < C) sc[(int64_t)h * a.Cm + j] = keep;
  };
#pragma unroll
  for (int it0 = 0; it0 < kSteps; it0 += 4) {
    uint4 c[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      // unconditional loads at clamped rows (C > j0 >= 0), masked after, so
      // that the four are in flight together
      const int j = j0 + wave * kPerWave + (it0 + k) * 4 + grp;
      const uint4 x = load_stream16(cbase + (int64_t)min(j, C - 1) * kHeadDim);
      c[k] = j < C ? x : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int st = it0 + k;
#pragma unroll
      for (int h = 0; h < G; ++h) {
        float d = dot2_bf16(c[k].x, qw[h][0], 0.f);
        d = dot2_bf16(c[k].y, qw[h][1], d);
        d = dot2_bf16(c[k].z, qw[h][2], d);
        d = dot2_bf16(c[k].w, qw[h][3], d);
        d = sum16(d);
        if (sl == (st % P) * G + h) keep = d;
      }
      if ((st + 1) % P == 0 || st + 1 == kSteps) flush(st - st % P, st % P + 1);
    }
  }
}

// ============================================================================
// 2. Per-head cluster order by a bucket sort.  Key = (descending-orderable
//    score bits, cluster id): ascending keys give score descending, ties by
//    ascending id.  The bucket of a score is a monotone function of it, so
//    bucket order agrees with key order and every element's rank is its
//    bucket start plus the number of smaller keys in its bucket.  The map
//    squashes the standardised score z = (s - mean) / sd through
//    z / (1 + |z|), which spreads a bell-shaped score distribution with far
//    outliers evenly over the buckets (about one element per bucket), where a
//    linear map over [min, max] would crowd the bulk into a few buckets.  Then
//    the tokens ahead of every rank (exclusive prefix of cluster sizes in rank
//    order) and the rows of the sampled positions: exact head 1..N and the
//    two windows (Alg. 1).  One workgroup (1024 threads) per query head (up
//    to eight per head beyond 8192 clusters, see the workspace sort below).
// ============================================================================
__device__ __forceinline__ uint32_t desc_key_bits(float s) {
  const uint32_t u = __float_as_uint(s + 0.0f);  // -0 -> +0
  const uint32_t ord = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ~ord;
}

// Monotone non-increasing in s (NaN last).  With r = 1 / (1 + |z|) in (0, 1]
// the bucket is (nb / 2) r for z >= 0 and nb - (nb / 2) r for z < 0, i.e.
// (1 - u) nb for u = 1/2 + sign(z) (1 - r) / 2.  Every step is monotone in its
// input: fp32 subtract, scale by a positive constant, absolute value, add,
// correctly rounded divide, scale by a power of two (exact), subtract from
// nb, truncation and clamp; the two branches meet at nb / 2.
__device__ __forceinline__ int squash_bucket(float s, float mu, float inv_sd, int nb) {
  if (!(s == s)) return nb - 1;
  const float z = (s - mu) * inv_sd;
  const float half = 0.5f * (float)nb;
  const float x = half * (1.0f / (1.0f + fabsf(z)));  // (0, nb/2], non-increasing in |z|
  const int bk = (int)(z >= 0.f ? x : (float)nb - x);
  return min(max(bk, 0), nb - 1);
}

// Exclusive scan in place of a[0..1024 kPer) in LDS by 1024 threads, kPer
// consecutive entries each (16-byte LDS accesses when kPer is 8); returns the
// total.  Ends with a barrier.
template <int kPer>
__device__ uint32_t scan_lds(uint32_t* a, uint32_t* s_wave) {
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  uint32_t v[kPer];
  if constexpr (kPer == 8) {
    const uint4* a4 = reinterpret_cast<const uint4*>(a) + tid * 2;
    const uint4 x = a4[0], y = a4[1];
    v[0] = x.x, v[1] = x.y, v[2] = x.z, v[3] = x.w, v[4] = y.x, v[5] = y.y, v[6] = y.z, v[7] = y.w;
  } else {
#pragma unroll
    for (int e = 0; e < kPer; ++e) v[e] = a[tid * kPer + e];
  }
  uint32_t local = 0;
#pragma unroll
  for (int e = 0; e < kPer; ++e) local += v[e];
  uint32_t incl = wave_incl_scan(local);  // DPP, no LDS
  if (lane == kWave - 1) s_wave[wave] = incl;
  __syncthreads();
  if (wave == 0) {
    const uint32_t w = lane < 16 ? s_wave[lane] : 0u;
    uint32_t wi = row_incl_scan(w);  // DPP, no LDS
    if (lane < 16) s_wave[lane] = wi - w;
    if (lane == 15) s_wave[16] = wi;
  }
  __syncthreads();
  uint32_t run = s_wave[wave] + incl - local;
  uint32_t o[kPer];
#pragma unroll
  for (int e = 0; e < kPer; ++e) {
    o[e] = run;
    run += v[e];
  }
  if constexpr (kPer == 8) {
    uint4* a4 = reinterpret_cast<uint4*>(a) + tid * 2;
    a4[0] = make_uint4(o[0], o[1], o[2], o[3]);
    a4[1] = make_uint4(o[4], o[5], o[6], o[7]);
  } else {
#pragma unroll
    for (int e = 0; e < kPer; ++e) a[tid * kPer + e] = o[e];
  }
  const uint32_t total = s_wave[16];
  __syncthreads();
  return total;
}
__device__ __forceinline__ uint32_t scan8k_lds(uint32_t* a, uint32_t* s_wave) { return scan_lds<8>(a, s_wave); }

// Inverse of desc_key_bits: the score (with -0 read as +0; NaN bits kept).
__device__ __forceinline__ float key_score(uint32_t k) {
  const uint32_t ord = ~k;
  return __uint_as_float((ord & 0x80000000u) ? (ord & 0x7fffffffu) : ~ord);
}

// Workspace sort of 8192 < C <= kPieceMaxC clusters: the scores and sizes of
// a thread's 32 clusters stay in registers; the bucket counts (kPieceBuckets)
// sit in LDS, and counting them gives each cluster its place in its bucket,
// so after the scan each cluster knows its position in bucket order.  The
// buckets are then taken in pieces of consecutive buckets holding at most
// kPieceCap clusters, whose keys are staged in LDS at those positions: every
// access of the rank computation is an LDS access, and the global accesses
// are coalesced.  A piece's ranks are consecutive, so its order, rank-prefix
// and size entries leave in order.  A head's buckets are shared by the
// workgroups of its grid column (blockIdx.y): each counts every cluster (the
// bucket starts must be known everywhere), then ranks only the pieces of its
// own run of whole buckets, its prefix starting at the tokens of the
// clusters before them, and finds the sampled rows that fall in its ranks.
// The workgroups exchange nothing; the first one also writes the head record.
constexpr int kPieceBuckets = 4096;
constexpr int kPiecePer = 6;                    // entries per thread in the piece scan
constexpr int kPieceCap = kPiecePer * 1024;     // clusters per piece
constexpr int kPieceMaxC = 32 * 1024;           // 32 clusters per thread
constexpr size_t kPieceLdsBytes = (size_t)kPieceBuckets * 8 + (size_t)kPieceCap * 20;
// dynamic LDS of the workspace sort: the pieces, or 8192 bucket counts and
// starts on the general path; then the rank prefix for the sample search
constexpr size_t kSortWsLdsBytes = kPieceLdsBytes > (size_t)kSortLdsBuckets * 8 ? kPieceLdsBytes : (size_t)kSortLdsBuckets * 8;

template <bool kLds>
__global__ __launch_bounds__(1024) void sort_clusters_kernel(SortArgs a) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  __shared__ uint32_t s_wave_u[17];
  __shared__ float s_wave_f[17];
  __shared__ float s_red[16][4];
  const int tid = threadIdx.x, nt = blockDim.x;
  const int bh = blockIdx.x;
  const int b = bh / a.Hq, h = bh % a.Hq, g = h / a.G;
  const float* sc = a.scores + (int64_t)bh * a.Cm;
  // LDS path: the head's scores, loaded first and unconditionally at indices
  // clamped to the stride Cm (>= C; the entries past C are masked later), so
  // that they travel with the cluster-count load instead of after it
  float raw[8];
  if constexpr (kLds) {
#pragma unroll
    for (int e = 0; e < 8; ++e) raw[e] = sc[min(tid + e * 1024, a.Cm - 1)];
  }
  const int64_t cb = a.cl_indptr[b];
  const int C = min((int)(a.cl_indptr[b + 1] - cb), a.Cm);
  const int n = (int)seq_tokens(a.kv_indptr, a.seq_len, b);
  const int32_t* off = a.offsets + (int64_t)g * (a.Ct + a.B) + cb + b;
  int32_t* rank_of = a.rank_of + (int64_t)bh * a.Cm;
  int32_t* order = a.order + (int64_t)bh * a.Cm;

  uint32_t* cnt;      // per rank: cluster size, then the exclusive prefix
  int32_t* ostart;    // per rank: first row of the cluster
  uint32_t total = 0; // tokens of the sequence (prefix at rank C)
  // ranks [rk_lo, rk_hi) of this workgroup, holding token positions
  // (tok_lo, tok_hi]; the whole order except when a head's pieces are shared
  int rk_lo = 0, rk_hi = -1;
  uint32_t tok_lo = 0, tok_hi = 0;
  if constexpr (kLds) {
    // LDS: keys u64[8192] (after ranking: ostart i32[8192], ord_s i32[8192]),
    // cnt u32[8192], start u32[8192]
    uint64_t* keys = reinterpret_cast<uint64_t*>(smem_raw);
    cnt = reinterpret_cast<uint32_t*>(keys + kSortLdsBuckets);
    uint32_t* start = cnt + kSortLdsBuckets;
    ostart = reinterpret_cast<int32_t*>(keys);
    int32_t* ord_s = ostart + kSortLdsBuckets;
    constexpr int nb = kSortLdsBuckets;
    // every thread keeps its 8 elements in registers (C <= 8192 = 8 * 1024)
    float v[8];
    int o0[8], o1[8], bk[8], pos[8];
    // the offsets too are loaded unconditionally, at indices clamped into the
    // (b, g) list, so that all of them are in flight together (a guarded load
    // whose value is used inside its guard waits there); they are first used
    // after the ranking, so their latency hides behind the phases before it
#pragma unroll
    for (int e = 0; e < 8; ++e) {  // the (b, g) list holds C + 1 entries (one when C = 0)
      const int jc = max(min(tid + e * 1024, C - 1), 0);
      o0[e] = off[jc];
      o1[e] = off[min(jc + 1, C)];
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = tid + e * 1024 < C ? raw[e] : NAN;
    {
      uint4* c4 = reinterpret_cast<uint4*>(cnt) + tid * 2;
      c4[0] = make_uint4(0, 0, 0, 0);
      c4[1] = make_uint4(0, 0, 0, 0);
    }
    // moments and range of the finite scores (one barrier)
    float sm = 0.f, sq = 0.f, lo = INFINITY, hi = -INFINITY, nf = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if (v[e] == v[e]) {
        sm += v[e];
        sq += v[e] * v[e];
        lo = fminf(lo, v[e]);
        hi = fmaxf(hi, v[e]);
        nf += 1.f;
      }
    }
    sm = wave_allsum_f(sm);  // DPP, no LDS
    sq = wave_allsum_f(sq);
    nf = wave_allsum_f(nf);
    lo = wave_allmin_f(lo);
    hi = wave_allmax_f(hi);
    if ((tid & (kWave - 1)) == 0) {
      s_red[tid / kWave][0] = sm;
      s_red[tid / kWave][1] = sq;
      s_red[tid / kWave][2] = lo;
      s_red[tid / kWave][3] = hi;
      s_wave_f[tid / kWave] = nf;
    }
    __syncthreads();
    sm = 0.f, sq = 0.f, lo = INFINITY, hi = -INFINITY, nf = 0.f;
    for (int w = 0; w < 16; ++w) {
      sm += s_red[w][0];
      sq += s_red[w][1];
      lo = fminf(lo, s_red[w][2]);
      hi = fmaxf(hi, s_red[w][3]);
      nf += s_wave_f[w];
    }
    if (lo == hi && nf == (float)C) {
      // all scores equal: the order is the cluster id
#pragma unroll
      for (int e = 0; e < 8; ++e) pos[e] = tid + e * 1024;
    } else {
      const float mu = nf > 0.f ? sm / nf : 0.f;
      const float var = nf > 0.f ? fmaxf(sq / nf - mu * mu, 0.f) : 0.f;
      const float sd = sqrtf(var);
      const float inv_sd = sd > 0.f ? 1.f / sd : (hi > lo ? 1.f / (hi - lo) : 1.f);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        bk[e] = squash_bucket(v[e], mu, inv_sd, nb);
        if (tid + e * 1024 < C) atomicAdd(&cnt[bk[e]], 1u);
      }
      __syncthreads();
      {
        const uint4* c4 = reinterpret_cast<const uint4*>(cnt) + tid * 2;
        uint4* s4 = reinterpret_cast<uint4*>(start) + tid * 2;
        s4[0] = c4[0];
        s4[1] = c4[1];
      }
      scan8k_lds(start, s_wave_u);  // (each thread copied the entries it scans)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int j = tid + e * 1024;
        if (j < C) keys[atomicAdd(&start[bk[e]], 1u)] = ((uint64_t)desc_key_bits(v[e]) << 32) | (uint32_t)j;
      }
      __syncthreads();
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int j = tid + e * 1024;
        pos[e] = 0;
        if (j < C) {
          const uint64_t key = ((uint64_t)desc_key_bits(v[e]) << 32) | (uint32_t)j;
          const uint32_t end = start[bk[e]], beg = end - cnt[bk[e]];
          uint32_t r = 0, t = beg;
          for (; t + 1 < end; t += 2) {  // two LDS reads in flight per step
            const uint64_t k0 = keys[t], k1 = keys[t + 1];
            r += (k0 < key ? 1u : 0u) + (k1 < key ? 1u : 0u);
          }
          if (t < end) r += keys[t] < key ? 1u : 0u;
          pos[e] = (int)(beg + r);
        }
      }
      __syncthreads();
    }
    // sizes, starts and ids by rank; ranks >= C hold size 0
    {
      uint4* c4 = reinterpret_cast<uint4*>(cnt) + tid * 2;
      c4[0] = make_uint4(0, 0, 0, 0);
      c4[1] = make_uint4(0, 0, 0, 0);
    }
    __syncthreads();
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if (tid + e * 1024 < C) {
        cnt[pos[e]] = (uint32_t)(o1[e] - o0[e]);
        ostart[pos[e]] = o0[e];
        ord_s[pos[e]] = tid + e * 1024;
      }
    }
    __syncthreads();
    total = scan8k_lds(cnt, s_wave_u);  // cnt has no entry C when C == 8192
    // global results after the last barrier (no barrier waits on these
    // stores); the LDS reads first, unconditional (every index is inside the
    // 8192-entry arrays), so that they are in flight together
    int os[8];
    uint32_t pv[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      os[e] = ord_s[tid + e * 1024];
      pv[e] = cnt[tid + e * 1024];
    }
    int32_t* rpre = a.rprefix + (int64_t)bh * (a.Cm + 1);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int j = tid + e * 1024;
      if (j < C) {
        rank_of[j] = pos[e];
        order[j] = os[e];
      }
      if (j <= C) rpre[j] = (int32_t)(j < C ? pv[e] : total);
    }
    if (tid == 0 && C == kSortLdsBuckets) rpre[C] = (int32_t)total;  // the one entry past the 8192
  } else {
    cnt = a.g_cnt + (int64_t)bh * (a.nb_max + 4);  // per rank: size, then prefix
    ostart = nullptr;                              // the sample rows start from off[order[r]]
    bool pieces_done = false;
    if (C > 0 && C <= kPieceMaxC) {  // uniform; its loads clamp indices to C - 1
      constexpr int nbk = kPieceBuckets, kE = kPieceMaxC / 1024;
      uint32_t* cnt_l = reinterpret_cast<uint32_t*>(smem_raw);  // bucket sizes
      uint32_t* st_l = cnt_l + nbk;                             // bucket starts
      uint64_t* s_keys = reinterpret_cast<uint64_t*>(st_l + nbk);  // the piece's keys by bucket position
      uint32_t* s_aux = reinterpret_cast<uint32_t*>(s_keys + kPieceCap);  // size by position, then rank
      int32_t* s_ord = reinterpret_cast<int32_t*>(s_aux + kPieceCap);     // cluster by rank in the piece
      uint32_t* s_sz = reinterpret_cast<uint32_t*>(s_ord + kPieceCap);    // size, then prefix, by rank
      float v[kE];     // the score, then the rank
      uint32_t ps[kE];  // size (low 16 bits) | place in its bucket, then bucket position (high 16 bits)
      uint32_t size_or = 0;  // OR of the sizes: any bit above 15 sends the head to the general path
      const int nv = C > tid ? (C - tid + 1023) / 1024 : 0;  // clusters of this thread: tid + 1024 e, e < nv
      // the cluster id, rebuilt at each use rather than kept in 32 registers
      auto cid = [&](int e) {
        int t = tid;
        asm volatile("" : "+v"(t));
        return t + e * 1024;
      };
#pragma unroll
      for (int e = 0; e < kE; ++e) v[e] = sc[min(cid(e), C - 1)];
#pragma unroll
      for (int e0 = 0; e0 < kE; e0 += kE / 2) {  // sizes: 32 offset loads in flight per batch
        int o0[kE / 2], o1[kE / 2];
#pragma unroll
        for (int e = 0; e < kE / 2; ++e) {
          const int jc = min(cid(e0 + e), C - 1);
          o0[e] = off[jc];
          o1[e] = off[jc + 1];
        }
#pragma unroll
        for (int e = 0; e < kE / 2; ++e) {
          uint32_t x = (uint32_t)(o1[e] - o0[e]);
          size_or |= x;
          // taken now, so that the loaded offsets die here
          asm volatile("" : "+v"(x), "+v"(size_or));
          ps[e0 + e] = x & 0xffffu;
        }
      }
      reinterpret_cast<uint4*>(cnt_l)[tid] = make_uint4(0, 0, 0, 0);
      float sm = 0.f, sq = 0.f, lo = INFINITY, hi = -INFINITY, nf = 0.f;
#pragma unroll
      for (int e = 0; e < kE; ++e) {
        if (e < nv && v[e] == v[e]) {
          sm += v[e];
          sq += v[e] * v[e];
          lo = fminf(lo, v[e]);
          hi = fmaxf(hi, v[e]);
          nf += 1.f;
        }
      }
      sm = wave_allsum_f(sm);  // DPP, no LDS
      sq = wave_allsum_f(sq);
      nf = wave_allsum_f(nf);
      lo = wave_allmin_f(lo);
      hi = wave_allmax_f(hi);
      if ((tid & (kWave - 1)) == 0) {
        s_red[tid / kWave][0] = sm;
        s_red[tid / kWave][1] = sq;
        s_red[tid / kWave][2] = lo;
        s_red[tid / kWave][3] = hi;
        s_wave_f[tid / kWave] = nf;
      }
      __syncthreads();  // also orders the count clears before the counting below
      sm = 0.f, sq = 0.f, lo = INFINITY, hi = -INFINITY, nf = 0.f;
      for (int w = 0; w < 1024 / kWave; ++w) {
        sm += s_red[w][0];
        sq += s_red[w][1];
        lo = fminf(lo, s_red[w][2]);
        hi = fmaxf(hi, s_red[w][3]);
        nf += s_wave_f[w];
      }
      const bool all_equal = lo == hi && nf == (float)C;  // the general path orders them by id
      const float mu = nf > 0.f ? sm / nf : 0.f;
      const float var = nf > 0.f ? fmaxf(sq / nf - mu * mu, 0.f) : 0.f;
      const float sd = sqrtf(var);
      const float inv_sd = sd > 0.f ? 1.f / sd : (hi > lo ? 1.f / (hi - lo) : 1.f);
      if (!all_equal) {
        // counting: each cluster's place in its bucket (arrival order)
#pragma unroll
        for (int e0 = 0; e0 < kE; e0 += 8) {  // unconditional (adding 0 past C): 8 returns in flight
#pragma unroll
          for (int e = e0; e < e0 + 8; ++e)
            ps[e] |= atomicAdd(&cnt_l[squash_bucket(v[e], mu, inv_sd, nbk)], e < nv ? 1u : 0u) << 16;
#pragma unroll
          for (int e = e0; e < e0 + 8; ++e) asm volatile("" : "+v"(ps[e]));  // done before the next 8
        }
        __syncthreads();
        // the largest bucket must fit a piece
        const uint4 c4 = reinterpret_cast<const uint4*>(cnt_l)[tid];
        reinterpret_cast<uint4*>(st_l)[tid] = c4;
        float mb = (float)max(max(c4.x, c4.y), max(c4.z, c4.w));  // counts <= 2^15: exact
        mb = wave_allmax_f(size_or > 0xffffu ? INFINITY : mb);
        if ((tid & (kWave - 1)) == 0) s_wave_f[tid / kWave] = mb;
        scan_lds<nbk / 1024>(st_l, s_wave_u);  // bucket starts; its barriers publish s_wave_f
        float maxb = 0.f;
        for (int w = 0; w < 1024 / kWave; ++w) maxb = fmaxf(maxb, s_wave_f[w]);
        pieces_done = maxb <= (float)kPieceCap;
        // bucket position = bucket start + place (C <= 2^15: 16 bits)
#pragma unroll
        for (int e0 = 0; e0 < kE; e0 += 8) {  // 8 reads in flight
#pragma unroll
          for (int e = e0; e < e0 + 8; ++e) ps[e] += st_l[squash_bucket(v[e], mu, inv_sd, nbk)] << 16;
#pragma unroll
          for (int e = e0; e < e0 + 8; ++e) asm volatile("" : "+v"(ps[e]));
        }
      }
      if (pieces_done) {
        int32_t* rpre = a.rprefix + (int64_t)bh * (a.Cm + 1);
        // the head's rank order is shared by the gridDim.y workgroups of the
        // head: workgroup kw takes the buckets [b_lo, b_hi), b_lo the largest
        // bucket whose start is at most kw C / nw (counted as b1 below), so
        // the ranges are whole buckets, disjoint and cover every cluster; its
        // first rank carries the tokens of the clusters before b_lo
        const int nw = (int)gridDim.y, kw = (int)blockIdx.y;
        const uint32_t t_lo = (uint32_t)((int64_t)kw * C / nw), t_hi = (uint32_t)((int64_t)(kw + 1) * C / nw);
        uint32_t* s_cnt2 = reinterpret_cast<uint32_t*>(&s_red[0][0]);  // 64 words: three wave-total slots of 16
        int b_lo, b_hi;
        {
          const uint4 s4 = reinterpret_cast<const uint4*>(st_l)[tid];
          auto count_le = [&](uint32_t lim) {
            return (tid > 0 && s4.x <= lim ? 1u : 0u) + (s4.y <= lim ? 1u : 0u) + (s4.z <= lim ? 1u : 0u) +
                   (s4.w <= lim ? 1u : 0u) + (tid == 1023 && (uint32_t)C <= lim ? 1u : 0u);
          };
          const uint32_t clo = (uint32_t)__builtin_amdgcn_readlane((int)wave_incl_scan(count_le(t_lo)), kWave - 1);
          const uint32_t chi = (uint32_t)__builtin_amdgcn_readlane((int)wave_incl_scan(count_le(t_hi)), kWave - 1);
          if ((tid & (kWave - 1)) == 0) {
            s_wave_u[tid / kWave] = clo;
            s_cnt2[tid / kWave] = chi;
          }
        }
        __syncthreads();
        b_lo = 0;
        b_hi = 0;
        for (int w = 0; w < 1024 / kWave; ++w) {
          b_lo += (int)s_wave_u[w];
          b_hi += (int)s_cnt2[w];
        }
        if (kw == 0) b_lo = 0;        // (the buckets before are empty)
        if (kw == nw - 1) b_hi = nbk;  // (every bucket start is at most C)
        // uniform over the workgroup: kept in scalar registers (the thread's
        // 32 scores and sizes fill its vector registers)
        b_lo = __builtin_amdgcn_readfirstlane(b_lo);
        b_hi = __builtin_amdgcn_readfirstlane(b_hi);
        const uint32_t r_lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(b_lo < nbk ? st_l[b_lo] : (uint32_t)C));
        const uint32_t r_hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(b_hi < nbk ? st_l[b_hi] : (uint32_t)C));
        {
          // tokens of the clusters ranked before r_lo, and of all clusters
          uint32_t before = 0, all = 0;
#pragma unroll
          for (int e = 0; e < kE; ++e) {
            const uint32_t sz = e < nv ? (ps[e] & 0xffffu) : 0u;
            all += sz;
            before += (ps[e] >> 16) < r_lo ? sz : 0u;
          }
          before = (uint32_t)__builtin_amdgcn_readlane((int)wave_incl_scan(before), kWave - 1);
          all = (uint32_t)__builtin_amdgcn_readlane((int)wave_incl_scan(all), kWave - 1);
          if ((tid & (kWave - 1)) == 0) {
            s_cnt2[16 + tid / kWave] = before;
            s_cnt2[32 + tid / kWave] = all;
          }
        }
        __syncthreads();  // (s_wave_u was read before it: the piece loop may write it)
        uint32_t carry = 0;
        total = 0;
        for (int w = 0; w < 1024 / kWave; ++w) {
          carry += s_cnt2[16 + w];
          total += s_cnt2[32 + w];
        }
        carry = (uint32_t)__builtin_amdgcn_readfirstlane((int)carry);
        total = (uint32_t)__builtin_amdgcn_readfirstlane((int)total);
        rk_lo = (int)r_lo;
        rk_hi = (int)r_hi;
        tok_lo = carry;
        for (int b0 = b_lo; b0 < b_hi;) {
          // the piece: buckets [b0, b1), the last b1 whose start is within
          // kPieceCap of the piece's start (the bucket b0 alone fits)
          // (starts are non-decreasing: b1 counts the b in [1, nbk] with
          // start(b) <= p0 + kPieceCap, start(nbk) = C)
          const uint32_t p0 = st_l[b0];
          {
            const uint4 s4 = reinterpret_cast<const uint4*>(st_l)[tid];
            const uint32_t lim = p0 + (uint32_t)kPieceCap;
            uint32_t c = (tid > 0 && s4.x <= lim ? 1u : 0u) + (s4.y <= lim ? 1u : 0u) + (s4.z <= lim ? 1u : 0u) +
                         (s4.w <= lim ? 1u : 0u) + (tid == 1023 && (uint32_t)C <= lim ? 1u : 0u);
            c = (uint32_t)__builtin_amdgcn_readlane((int)wave_incl_scan(c), kWave - 1);  // DPP, no LDS
            if ((tid & (kWave - 1)) == 0) s_wave_u[tid / kWave] = c;
          }
          __syncthreads();  // also: the previous piece's LDS reads are done
          int b1 = 0;
          for (int w = 0; w < 1024 / kWave; ++w) b1 += (int)s_wave_u[w];
          b1 = min(b1, b_hi);
          const uint32_t len = (b1 < nbk ? st_l[b1] : (uint32_t)C) - p0;
#pragma unroll
          for (int e = 0; e < kPiecePer; ++e) s_sz[tid * kPiecePer + e] = 0u;
          // the owners place the piece's keys and sizes at their bucket positions
#pragma unroll
          for (int e = 0; e < kE; ++e) {
            const uint32_t pos = (ps[e] >> 16) - p0;
            if (e < nv && pos < len) {
              s_keys[pos] = ((uint64_t)desc_key_bits(v[e]) << 32) | (uint32_t)cid(e);
              s_aux[pos] = ps[e] & 0xffffu;
            }
          }
          __syncthreads();
          // by position: rank = bucket start + smaller keys of the bucket
          for (int t = tid; t < (int)len; t += 1024) {
            const uint64_t key = s_keys[t];
            const int bk = squash_bucket(key_score((uint32_t)(key >> 32)), mu, inv_sd, nbk);
            const uint32_t beg = st_l[bk] - p0, end = beg + cnt_l[bk];
            uint32_t r = beg, i = beg;
            for (; i + 4 <= end; i += 4) {  // four reads in flight
              const uint64_t k0 = s_keys[i], k1 = s_keys[i + 1], k2 = s_keys[i + 2], k3 = s_keys[i + 3];
              r += (k0 < key ? 1u : 0u) + (k1 < key ? 1u : 0u) + (k2 < key ? 1u : 0u) + (k3 < key ? 1u : 0u);
            }
            for (; i < end; ++i) r += s_keys[i] < key ? 1u : 0u;
            s_ord[r] = (int32_t)(uint32_t)key;
            s_sz[r] = s_aux[t];
            s_aux[t] = p0 + r;
          }
          __syncthreads();
#pragma unroll
          for (int e0 = 0; e0 < kE; e0 += 8) {  // reads at clamped positions, 8 in flight
#pragma unroll
            for (int e = e0; e < e0 + 8; ++e) {
              const uint32_t pos = (ps[e] >> 16) - p0;
              const uint32_t rk = s_aux[min(pos, (uint32_t)kPieceCap - 1)];
              v[e] = (e < nv && pos < len) ? __uint_as_float(rk) : v[e];
            }
#pragma unroll
            for (int e = e0; e < e0 + 8; ++e) asm volatile("" : "+v"(v[e]));
          }
          const uint32_t tot = scan_lds<kPiecePer>(s_sz, s_wave_u);
          for (int t = tid; t < (int)len; t += 1024) {
            const uint32_t pf = carry + s_sz[t];
            order[p0 + t] = s_ord[t];
            cnt[p0 + t] = pf;
            rpre[p0 + t] = (int32_t)pf;
          }
          carry += tot;
          b0 = b1;
        }
#pragma unroll
        for (int e = 0; e < kE; ++e) {
          const uint32_t pos = ps[e] >> 16;
          if (e < nv && pos >= r_lo && pos < r_hi) rank_of[cid(e)] = (int32_t)__float_as_uint(v[e]);
        }
        if (tid == 0 && kw == 0) rpre[C] = (int32_t)total;
        tok_hi = carry;
      }
      __syncthreads();  // the general path below reuses the LDS and s_red
    }
    // the general path runs in the head's first workgroup; after the pieces
    // every workgroup finds the sampled rows of its own ranks
    if (!pieces_done && blockIdx.y != 0) return;
    if (!pieces_done) {
      // C > 8192: the bucket counts (8192 buckets) in LDS, the keys and the
      // per-rank sizes / starts in the workspace.  Every loop over the elements
      // takes 8 (4 in the ranking) per thread per step with their global loads
      // issued together, so a step costs one memory round trip.
      uint32_t* cnt_l = reinterpret_cast<uint32_t*>(smem_raw);
      uint32_t* start_l = cnt_l + kSortLdsBuckets;
      constexpr int nb = kSortLdsBuckets;
      constexpr int kB = 8;
      uint64_t* keys = a.g_keys + (int64_t)bh * a.nb_max;
      {
        uint4* c4 = reinterpret_cast<uint4*>(cnt_l) + tid * 2;
        c4[0] = make_uint4(0, 0, 0, 0);
        c4[1] = make_uint4(0, 0, 0, 0);
      }
      // moments and range of the finite scores, as in the LDS path
      float sm = 0.f, sq = 0.f, lo = INFINITY, hi = -INFINITY, nf = 0.f;
      for (int j0 = tid; j0 < C; j0 += kB * nt) {
        float v[kB];
#pragma unroll
        for (int e = 0; e < kB; ++e) v[e] = sc[min(j0 + e * nt, C - 1)];
#pragma unroll
        for (int e = 0; e < kB; ++e) {
          if (j0 + e * nt < C && v[e] == v[e]) {
            sm += v[e];
            sq += v[e] * v[e];
            lo = fminf(lo, v[e]);
            hi = fmaxf(hi, v[e]);
            nf += 1.f;
          }
        }
      }
      sm = wave_allsum_f(sm);  // DPP, no LDS
      sq = wave_allsum_f(sq);
      nf = wave_allsum_f(nf);
      lo = wave_allmin_f(lo);
      hi = wave_allmax_f(hi);
      if ((tid & (kWave - 1)) == 0) {
        s_red[tid / kWave][0] = sm;
        s_red[tid / kWave][1] = sq;
        s_red[tid / kWave][2] = lo;
        s_red[tid / kWave][3] = hi;
        s_wave_f[tid / kWave] = nf;
      }
      __syncthreads();  // also orders the count clears before the counting below
      sm = 0.f, sq = 0.f, lo = INFINITY, hi = -INFINITY, nf = 0.f;
      for (int w = 0; w < nt / kWave; ++w) {
        sm += s_red[w][0];
        sq += s_red[w][1];
        lo = fminf(lo, s_red[w][2]);
        hi = fmaxf(hi, s_red[w][3]);
        nf += s_wave_f[w];
      }
      const bool all_equal = lo == hi && nf == (float)C;  // then the order is the cluster id
      const float mu = nf > 0.f ? sm / nf : 0.f;
      const float var = nf > 0.f ? fmaxf(sq / nf - mu * mu, 0.f) : 0.f;
      const float sd = sqrtf(var);
      const float inv_sd = sd > 0.f ? 1.f / sd : (hi > lo ? 1.f / (hi - lo) : 1.f);
      if (!all_equal) {
        for (int j0 = tid; j0 < C; j0 += kB * nt) {
          float v[kB];
#pragma unroll
          for (int e = 0; e < kB; ++e) v[e] = sc[min(j0 + e * nt, C - 1)];
#pragma unroll
          for (int e = 0; e < kB; ++e)
            if (j0 + e * nt < C) atomicAdd(&cnt_l[squash_bucket(v[e], mu, inv_sd, nb)], 1u);
        }
        __syncthreads();
        {
          const uint4* c4 = reinterpret_cast<const uint4*>(cnt_l) + tid * 2;
          uint4* s4 = reinterpret_cast<uint4*>(start_l) + tid * 2;
          s4[0] = c4[0];
          s4[1] = c4[1];
        }
        scan8k_lds(start_l, s_wave_u);  // (each thread copied the entries it scans)
        for (int j0 = tid; j0 < C; j0 += kB * nt) {
          float v[kB];
#pragma unroll
          for (int e = 0; e < kB; ++e) v[e] = sc[min(j0 + e * nt, C - 1)];
#pragma unroll
          for (int e = 0; e < kB; ++e) {
            const int j = j0 + e * nt;
            if (j < C)
              keys[atomicAdd(&start_l[squash_bucket(v[e], mu, inv_sd, nb)], 1u)] =
                  ((uint64_t)desc_key_bits(v[e]) << 32) | (uint32_t)j;
          }
        }
        __syncthreads();  // the keys are visible to the workgroup; start_l holds the bucket ends
      }
      // rank of every element: its bucket start plus the smaller keys in its
      // bucket.  Four elements per step: the first four keys of each one's
      // bucket load together with the elements' cluster offsets; longer buckets
      // are walked after.  Then its size and first row go to its rank.
      {
        constexpr int kE = 4, kK = 4;
        for (int j0 = tid; j0 < C; j0 += kE * nt) {
          uint64_t key[kE];
          uint32_t beg[kE], end[kE], r[kE];
          int o_lo[kE], o_hi[kE];
#pragma unroll
          for (int e = 0; e < kE; ++e) {
            const int jc = min(j0 + e * nt, C - 1);
            const float sv = sc[jc];
            key[e] = ((uint64_t)desc_key_bits(sv) << 32) | (uint32_t)jc;
            o_lo[e] = off[jc];
            o_hi[e] = off[jc + 1];
            const int bk = all_equal ? 0 : squash_bucket(sv, mu, inv_sd, nb);
            end[e] = all_equal ? 1u : start_l[bk];
            beg[e] = all_equal ? 0u : end[e] - cnt_l[bk];
            r[e] = 0;
          }
          if (!all_equal) {
            uint64_t kk[kE][kK];
#pragma unroll
            for (int e = 0; e < kE; ++e)
#pragma unroll
              for (int i = 0; i < kK; ++i) kk[e][i] = keys[min(beg[e] + i, end[e] - 1)];  // the element is in it
#pragma unroll
            for (int e = 0; e < kE; ++e) {
#pragma unroll
              for (int i = 0; i < kK; ++i) r[e] += (beg[e] + i < end[e] && kk[e][i] < key[e]) ? 1u : 0u;
              for (uint32_t t = beg[e] + kK; t < end[e]; ++t) r[e] += keys[t] < key[e] ? 1u : 0u;
            }
          }
#pragma unroll
          for (int e = 0; e < kE; ++e) {
            const int j = j0 + e * nt;
            if (j < C) {
              const int p2 = all_equal ? j : (int)(beg[e] + r[e]);
              order[p2] = j;
              rank_of[j] = p2;
              cnt[p2] = (uint32_t)(o_hi[e] - o_lo[e]);
            }
          }
        }
      }
      __syncthreads();  // sizes and starts by rank are visible
      // exclusive prefix of the sizes in rank order: 32 consecutive ranks per
      // thread per pass, loaded together
      {
        constexpr int kS = 32;
        uint32_t carry = 0;
        for (int base = 0; base < C; base += kS * nt) {
          const int r0 = base + tid * kS;
          uint32_t v[kS];
#pragma unroll
          for (int e = 0; e < kS; ++e) v[e] = r0 + e < C ? cnt[r0 + e] : 0u;
          uint32_t local = 0;
#pragma unroll
          for (int e = 0; e < kS; ++e) local += v[e];
          const uint32_t incl = wave_incl_scan(local);  // DPP, no LDS
          if ((tid & (kWave - 1)) == kWave - 1) s_wave_u[tid / kWave] = incl;
          __syncthreads();
          uint32_t run = carry + incl - local, tot = 0;
          for (int w = 0; w < nt / kWave; ++w) {
            const uint32_t t = s_wave_u[w];
            if (w < tid / kWave) run += t;
            tot += t;
          }
#pragma unroll
          for (int e = 0; e < kS; ++e) {
            if (r0 + e < C) cnt[r0 + e] = run;
            run += v[e];
          }
          carry += tot;
          __syncthreads();  // s_wave_u is reused; the prefix is visible
        }
        total = carry;
      }
      int32_t* rpre = a.rprefix + (int64_t)bh * (a.Cm + 1);
      for (int r0 = tid; r0 <= C; r0 += kB * nt) {
        uint32_t v[kB];
#pragma unroll
        for (int e = 0; e < kB; ++e) v[e] = cnt[min(r0 + e * nt, max(C - 1, 0))];  // (entry 0 when C = 0: unused)
#pragma unroll
        for (int e = 0; e < kB; ++e) {
          const int r = r0 + e * nt;
          if (r <= C) rpre[r] = (int32_t)(r < C ? v[e] : total);
        }
      }
    }
  }

  // the clusters hold the first n_c rows; the rest are recent tokens, sampled
  // (all of them) after the exact head and the windows of the clustered list
  const int n_c = (int)min((int64_t)total, (int64_t)n);
  const int tail = min(max(n - n_c, 0), a.max_tail);
  const Geometry geo = make_geometry(n_c, a.prm);
  const int64_t S_main = min(geo.samples, a.S_cap);
  const int64_t S = min(S_main + tail, a.S_cap);
  const bool first_wg = blockIdx.y == 0;  // (more than one only when the pieces are shared)
  if (tid == 0 && first_wg) {
    int32_t* hm = a.head_meta + (int64_t)bh * 16;
    hm[0] = n_c;
    hm[1] = (int32_t)geo.N;
    hm[2] = geo.exact ? 0 : (int32_t)(geo.t1 - geo.s1 + 1);
    hm[3] = geo.exact ? 0 : (int32_t)(geo.t2 - geo.s2 + 1);
    hm[4] = (int32_t)geo.s1;
    hm[5] = (int32_t)geo.t1;
    hm[6] = (int32_t)geo.s2;
    hm[7] = (int32_t)geo.t2;
    hm[8] = geo.exact;
    hm[9] = (int32_t)S;
    hm[10] = C;
    hm[11] = tail;
    hm[12] = (int32_t)S_main;
    if (a.per_head && h % a.G == 0) a.sel_count_kv[b * a.Hkv + g] = 0;  // summed by fit_union
  }
  int32_t* rows = a.sample_rows + (int64_t)bh * a.S_cap;
  if (first_wg)
    for (int64_t u = S_main + tid; u < S; u += nt) rows[u] = n_c + (int32_t)(u - S_main);
  if (C <= 0) return;
  const int64_t N = geo.exact ? n_c : geo.N;
  const int64_t W1 = geo.exact ? 0 : geo.t1 - geo.s1 + 1;
  if constexpr (!kLds) {
    // workspace path: ranks [r0, r0 + R) of the order (the whole order, or
    // this workgroup's share of it), every kStr-th of their prefix entries in
    // LDS (every entry up to kSortWsLdsBytes / 4 clusters; the bucket arrays
    // are dead), a binary search there, then the last kStr entries from
    // memory, for the sampled positions in (p_lo, p_hi], the tokens of those
    // ranks.  The row of position i in rank r's cluster is
    // off[order[r]] + i - 1 - prefix[r].
    const bool whole = rk_hi < 0;
    const int r0 = whole ? 0 : rk_lo, R = whole ? C : rk_hi - rk_lo;
    const int64_t p_lo = whole ? 0 : tok_lo, p_hi = whole ? (int64_t)total : tok_hi;
    if (R <= 0) return;
    uint32_t* s_pre = reinterpret_cast<uint32_t*>(smem_raw);
    constexpr int kPreCap = (int)(kSortWsLdsBytes / 4);
    const int kStr = (R + kPreCap - 1) / kPreCap;
    const int nsp = (R + kStr - 1) / kStr;
    for (int i0 = tid; i0 < nsp; i0 += 16 * nt) {
      uint32_t v[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) v[e] = cnt[r0 + min((i0 + e * nt) * kStr, R - 1)];
#pragma unroll
      for (int e = 0; e < 16; ++e)
        if (i0 + e * nt < nsp) s_pre[i0 + e * nt] = v[e];
    }
    __syncthreads();
    int top = 1;
    while (top * 2 <= nsp) top <<= 1;
    constexpr int kU = 8;  // independent searches in flight per thread
    // positions and prefixes in 32 bits (a sequence holds fewer than 2^31
    // tokens).  The sampled positions of each region (exact head 1..N, the
    // two windows) that fall in (p_lo, p_hi] are a run of sample indices.
    const int N32 = (int)N, NW = (int)(N + W1), s1 = (int)geo.s1, s2 = (int)geo.s2, Sm = (int)S_main;
    for (int rg = 0; rg < 3; ++rg) {
      const int u_beg = rg == 0 ? 0 : (rg == 1 ? min(N32, Sm) : min(NW, Sm));
      const int u_end = rg == 0 ? min(N32, Sm) : (rg == 1 ? min(NW, Sm) : Sm);
      const int64_t pos0 = rg == 0 ? 1 : (rg == 1 ? s1 : s2);  // position of sample u_beg
      // the samples u in [u_beg, u_end) whose position pos0 + (u - u_beg) is in (p_lo, p_hi]
      const int ua = (int)max((int64_t)u_beg, u_beg + (p_lo + 1 - pos0));
      const int ub = (int)min((int64_t)u_end, u_beg + (p_hi + 1 - pos0));
      for (int u0 = ua + tid; u0 < ub; u0 += kU * nt) {
        uint32_t iv[kU];
        int li[kU];
#pragma unroll
        for (int k = 0; k < kU; ++k) {
          const int u = min(u0 + k * nt, ub - 1);  // (past ub: the last sample again, not stored)
          iv[k] = (uint32_t)(pos0 + (u - u_beg));
          li[k] = 0;
        }
        // largest i with s_pre[i] < position (s_pre[0] = prefix[r0] = p_lo <
        // position); the reads at clamped indices, so that the kU of a step
        // are in flight together
        for (int step = top; step > 0; step >>= 1) {
          uint32_t pv[kU];
#pragma unroll
          for (int k = 0; k < kU; ++k) pv[k] = s_pre[min(li[k] + step, nsp - 1)];
#pragma unroll
          for (int k = 0; k < kU; ++k) {
            const int t = li[k] + step;
            li[k] = (t < nsp && pv[k] < iv[k]) ? t : li[k];
          }
        }
        // then the largest r in [li * kStr, li * kStr + kStr) with prefix[r] < position
        int lr[kU];
#pragma unroll
        for (int k = 0; k < kU; ++k) lr[k] = li[k] * kStr;
        for (int d = 1; d < kStr; ++d) {
          uint32_t pv[kU];
#pragma unroll
          for (int k = 0; k < kU; ++k) pv[k] = cnt[r0 + min(li[k] * kStr + d, R - 1)];
#pragma unroll
          for (int k = 0; k < kU; ++k) {
            const int t = li[k] * kStr + d;
            lr[k] = (t < R && pv[k] < iv[k]) ? t : lr[k];
          }
        }
        int first[kU];
        uint32_t pr[kU];
#pragma unroll
        for (int k = 0; k < kU; ++k) {
          lr[k] = min(lr[k], R - 1);
          first[k] = off[order[r0 + lr[k]]];
        }
        // the rank's prefix from LDS when every entry is there (kept apart from
        // the memory read so that each compiles to its own instruction kind)
        if (kStr == 1) {
#pragma unroll
          for (int k = 0; k < kU; ++k) pr[k] = s_pre[lr[k]];
        } else {
#pragma unroll
          for (int k = 0; k < kU; ++k) pr[k] = cnt[r0 + lr[k]];
        }
#pragma unroll
        for (int k = 0; k < kU; ++k) {
          const int u = u0 + k * nt;
          if (u < ub) rows[u] = min(max(first[k] + (int32_t)(iv[k] - 1 - pr[k]), 0), n - 1);
        }
      }
    }
    return;
  }
  // the prefix array holds the total at every rank from C to 8191 (those
  // ranks have size 0), so steps from 4096 down never leave it and need no
  // clamp or end case: every entry there is >= any position searched
  int top = 1;
  while (top * 2 <= C) top <<= 1;
  top = min(top, kSortLdsBuckets / 2);
  // positions and prefixes in 32 bits (a sequence holds fewer than 2^31
  // tokens); three searches per thread, which covers the timed shape's 2623
  // samples in one round
  constexpr int kU = 3;  // independent searches in flight per thread
  const int N32 = (int)N, NW = (int)(N + W1), s1 = (int)geo.s1, s2 = (int)geo.s2, Sm = (int)S_main;
  for (int u0 = tid; u0 < Sm; u0 += kU * nt) {
    uint32_t iv[kU];  // 1-based position in the unpacked list
    int lr[kU];
#pragma unroll
    for (int k = 0; k < kU; ++k) {
      const int u = u0 + k * nt;
      iv[k] = (uint32_t)(u < N32 ? u + 1 : (u < NW ? s1 + (u - N32) : s2 + (u - NW)));
      lr[k] = 0;
    }
    // largest r in [0, C) with prefix[r] < i (prefix[0] = 0 < i); branch-free
    // so that the kU lookups of a step are in flight together
    for (int step = top; step > 0; step >>= 1) {
      uint32_t pv[kU];
#pragma unroll
      for (int k = 0; k < kU; ++k) pv[k] = cnt[lr[k] + step];
#pragma unroll
      for (int k = 0; k < kU; ++k) lr[k] = pv[k] < iv[k] ? lr[k] + step : lr[k];
    }
    int32_t first[kU];
    uint32_t pr[kU];
#pragma unroll
    for (int k = 0; k < kU; ++k) {  // read together (r < C: C only with offsets that disagree with kv_indptr)
      const int r = min(lr[k], C - 1);
      first[k] = ostart[r];
      pr[k] = cnt[r];
    }
#pragma unroll
    for (int k = 0; k < kU; ++k) {
      const int u = u0 + k * nt;
      if (u < Sm) rows[u] = min(max(first[k] + (int32_t)(iv[k] - 1 - pr[k]), 0), n - 1);
    }
  }
}

// ============================================================================
// 3. Sampled logits, fit, cutoff, union.
// ============================================================================
__device__ double harmonic(int64_t x) {
  if (x <= 0) return 0.0;
  if (x < 64) {
    double s = 0.0;
    for (int64_t i = 1; i <= x; ++i) s += 1.0 / (double)i;
    return s;
  }
  const double X = (double)x, r = 1.0 / X, r2 = r * r;
  // Euler-Maclaurin expansion of H(x) = psi(x + 1) + gamma
  return log(X) + 0.57721566490153286061 + 0.5 * r -
         r2 * (1.0 / 12.0 - r2 * (1.0 / 120.0 - r2 * (1.0 / 252.0 - r2 * (1.0 / 240.0))));
}

// Positive interval [L, R] of a/i + b over integer i in [lo, hi]; false when
// it is empty.  a/i + b evaluated in fp64 is monotone in i (non-increasing for
// a >= 0, non-decreasing for a < 0: correctly rounded division and addition
// are monotone), so the positive set is a prefix or a suffix of [lo, hi] and
// a binary search finds its end in O(log n) steps for any a and b (NaN
// coefficients give an empty interval).
__device__ bool positive_interval(double a, double b, int64_t lo, int64_t hi, int64_t* L, int64_t* R) {
  if (hi < lo || !(a == a) || !(b == b)) return false;
  auto pos = [&](int64_t i) { return a / (double)i + b > 0.0; };
  if (a >= 0.0) {  // prefix [lo, R]
    if (!pos(lo)) return false;
    if (pos(hi)) {
      *L = lo;
      *R = hi;
      return true;
    }
    // the real root -a/b (b < 0 here) usually lands on the answer
    const double z = a / -b;
    if (z >= (double)lo && z < (double)hi) {
      const int64_t r = (int64_t)z;
      if (pos(r) && !pos(r + 1)) {
        *L = lo;
        *R = r;
        return true;
      }
    }
    int64_t l = lo, h = hi;  // pos(l) holds; last positive index
    while (l < h) {
      const int64_t m = l + (h - l + 1) / 2;
      if (pos(m)) l = m;
      else h = m - 1;
    }
    *L = lo;
    *R = l;
  } else {  // suffix [L, hi]
    if (!pos(hi)) return false;
    if (pos(lo)) {
      *L = lo;
      *R = hi;
      return true;
    }
    const double z = -a / b;  // b > 0 here
    if (z >= (double)lo && z < (double)hi) {
      const int64_t l0 = (int64_t)z + 1;
      if (pos(l0) && !pos(l0 - 1)) {
        *L = l0;
        *R = hi;
        return true;
      }
    }
    int64_t l = lo, h = hi;  // pos(h) holds; first positive index
    while (l < h) {
      const int64_t m = l + (h - l) / 2;
      if (pos(m)) h = m;
      else l = m + 1;
    }
    *L = l;
    *R = hi;
  }
  return true;
}

// 3a. Logits of the sampled rows: each lane sums its 8 bf16 products in fp32
//     (v_dot2, error at most a few ulp of the lane's sum of |products|), the
//     16 lane sums add in fp64.  grid (ceil(S_cap/128), B*Hq), 256 threads:
//     workgroup c owns samples [128c, 128c + 128); 16 lanes per row, each wave
//     gathers 32 rows with all loads in flight together.  The workgroup also
//     reduces its logits per region (exact head, window 1, window 2, recent
//     tokens) to (max, sum of exp(l - max)), so the fit needs one exponential
//     per chunk instead of one per sample.
// wave-wide fp64 sum / max, identical in every lane (DPP scans, no LDS)
__device__ __forceinline__ double wave_sum_d(double v) { return wave_allsum_d(v); }
__device__ __forceinline__ double wave_max_d(double v) { return wave_allmax_d(v); }

template <bool kPaged>
__global__ __launch_bounds__(256) void sample_logits_kernel(FitArgs a) {
  __shared__ double s_lg[kSampleChunk];
  constexpr int kRW = kSampleChunk / kWave;  // samples per lane in the chunk reduction
  static_assert(kSampleChunk % kWave == 0 && kRW <= 4, "chunk must be 1 to 4 waves of samples");
  const int tid = threadIdx.x;
  const int bh = blockIdx.y;
  const int b = bh / a.Hq, h = bh % a.Hq, g = h / a.G;
  const int32_t* hm = a.head_meta + (int64_t)bh * 16;
  const int64_t u0 = (int64_t)blockIdx.x * kSampleChunk;
  const int lane = tid & 63, wave = tid >> 6, sl = lane & 15, grp = lane >> 4;
  // one sampled row per lane, coalesced (the wave's kSpw samples), loaded
  // together with the head's metadata: entries past the head's sample count
  // (but inside its S_cap) are read and then ignored.  Each lane-group then
  // takes its rows from the lanes that hold them (cross-lane permute), so
  // only the K data stays in registers while every load is in flight.
  constexpr int kSpw = kSampleChunk / 4;  // samples per wave
  constexpr int kR = kSampleChunk / 16;   // rows per lane-group
  static_assert(kSpw <= kWave, "one sample per lane");
  const int64_t uw = u0 + wave * kSpw + lane;  // this lane's sample
  const int32_t* rows = a.sample_rows + (int64_t)bh * a.S_cap;
  int32_t rl = (lane < kSpw && uw < a.S_cap) ? rows[uw] : -1;
  const int64_t S = hm[9];
  if (u0 >= S) return;
  if (uw >= S) rl = -1;
  const uint4 qv = *reinterpret_cast<const uint4*>(a.q + (int64_t)bh * kHeadDim + sl * 8);
  const int64_t kvb = a.kv_indptr[b];
  double* lg = a.logits + (int64_t)bh * a.S_cap;
  uint4 kv[kR];  // sample wave * kSpw + k * 4 + grp of the chunk
  if constexpr (kPaged) {
    const int64_t ro = rl >= 0 ? paged_row(a.pk, a.Hkv, a.total, kvb, b, g, rl, hm[0]) : -1;
    const uint16_t* Kl = a.K + sl * 8;
#pragma unroll
    for (int k = 0; k < kR; ++k) {  // unconditional loads (row 0 for no sample), then masked
      const int64_t rk = __shfl(ro, k * 4 + grp, kWave);
      const uint4 x = load_stream16(Kl + max(rk, (int64_t)0) * kHeadDim);
      kv[k] = rk >= 0 ? x : make_uint4(0, 0, 0, 0);
    }
  } else {
    const uint16_t* Kg = a.K + ((int64_t)g * a.total + kvb) * kHeadDim + sl * 8;
#pragma unroll
    for (int k = 0; k < kR; ++k) {  // unconditional loads (the sequence's row 0 for no sample), then masked
      const int rk = __shfl(rl, k * 4 + grp, kWave);
      const uint4 x = load_stream16(Kg + (int64_t)max(rk, 0) * kHeadDim);
      kv[k] = rk >= 0 ? x : make_uint4(0, 0, 0, 0);
    }
  }
#pragma unroll
  for (int k = 0; k < kR; ++k) {
    // the lane's 8 products summed in fp32 (v_dot2), the 16 lane sums in fp64
    float d = dot2_bf16(kv[k].x, qv.x, 0.f);
    d = dot2_bf16(kv[k].y, qv.y, d);
    d = dot2_bf16(kv[k].z, qv.z, d);
    d = dot2_bf16(kv[k].w, qv.w, d);
    const double acc = sum16d((double)d) * 0.088388347648318440550;  // 1 / sqrt(128), within 1 ulp of the quotient
    const int t = wave * kSpw + k * 4 + grp;
    if (sl == 0) s_lg[t] = acc;
  }
  __syncthreads();
  if (tid < kSampleChunk && u0 + tid < S) lg[u0 + tid] = s_lg[tid];  // contiguous stores
  // per-region (max, sum exp(l - max)) of this chunk, wave r taking region r
  // (4 waves, 4 regions: exact head, window 1, window 2, recent tokens), kRW
  // samples per lane
  const int64_t S_main = hm[12];
  const int64_t N = hm[8] ? S_main : hm[1];
  const int64_t N1 = N + hm[2];
  auto region = [&](int64_t u) {
    return u < N ? 0 : (u < N1 ? 1 : (u < S_main ? 2 : (u < S ? 3 : 4)));
  };
  const int rg_lo = region(u0), rg_hi = region(min(S, u0 + kSampleChunk) - 1);  // regions present
  double l[kRW];
  int reg[kRW];
#pragma unroll
  for (int i = 0; i < kRW; ++i) {
    l[i] = s_lg[i * kWave + lane];
    reg[i] = region(u0 + i * kWave + lane);
  }
  double* out = a.lse + ((int64_t)bh * a.split + blockIdx.x) * 8;
  const int rg = wave;
  double mx = -INFINITY, sm = 0.0;
  if (rg >= rg_lo && rg <= rg_hi) {
    double m0 = -INFINITY;
#pragma unroll
    for (int i = 0; i < kRW; ++i) m0 = fmax(m0, reg[i] == rg ? l[i] : -INFINITY);
    mx = wave_max_d(m0);
    double e = 0.0;
#pragma unroll
    for (int i = 0; i < kRW; ++i) e += reg[i] == rg ? exp(l[i] - mx) : 0.0;
    sm = wave_sum_d(e);
  }
  if (lane == 0) {
    out[rg * 2] = mx;
    out[rg * 2 + 1] = mx == -INFINITY ? 0.0 : sm;
  }
}

// Fit and budget of one query head (Algorithm 1) by one wave, fp64.  Lane 0
// writes the head's record and returns the cutoff (rank, length) in cut[2].
// Region sums come from the per-chunk (max, sum) partials of the sampling
// kernel: with M the maximum over the exact head (the shift m), a region's sum
// of exp(l - m) is sum_c exp(M_c - m) S_c.
// (store: write the head's budget and fit record; false where another
// workgroup fitting the same head writes them)
__device__ void fit_head_wave(const FitArgs& a, int bh, int lane, int* cut, bool store) {
  constexpr int kRg = 4;  // regions: exact head, window 1, window 2, recent tokens
  const int32_t* hm = a.head_meta + (int64_t)bh * 16;
  const double* lg = a.logits + (int64_t)bh * a.S_cap;
  const double* lse = a.lse + (int64_t)bh * a.split * (2 * kRg);
  // the partials of the first 64 chunks, the first chunk's logits and the
  // first 64 rank-prefix entries load together with the head's metadata (a
  // small budget ends in the first chunk and the first clusters)
  double pre[2 * kRg];
#pragma unroll
  for (int i = 0; i < 2 * kRg; ++i) pre[i] = lane < a.split ? lse[lane * 2 * kRg + i] : 0.0;
  constexpr int kLg0 = kSampleChunk / kWave;
  double lg0[kLg0];
#pragma unroll
  for (int i = 0; i < kLg0; ++i) lg0[i] = i * kWave + lane < a.S_cap ? lg[i * kWave + lane] : 0.0;
  const int32_t* rpre = a.rprefix + (int64_t)bh * (a.Cm + 1);
  const int rp0 = lane <= a.Cm ? rpre[lane] : 0;
  const int n = hm[0];          // clustered tokens (the list of Algorithm 1)
  const int64_t S = hm[9];      // sampled rows, the recent tokens included
  const int tail = hm[11];      // recent tokens, all selected
  const int exact = hm[8];
  const int64_t N = exact ? (int64_t)hm[12] : (int64_t)hm[1];
  const int64_t W1 = hm[2], W2 = hm[3];
  const int nch = min((int)((S + kSampleChunk - 1) / kSampleChunk), a.split);  // S <= S_cap
  int k = 0;
  double m = 0.0, mu1 = 0.0, mu2 = 0.0, fa = 0.0, fb = 0.0, Sn = 0.0, T = 0.0, EN = 0.0, Et = 0.0;
  if (S > 0) {
    double M[kRg];
#pragma unroll
    for (int rg = 0; rg < kRg; ++rg) M[rg] = lane < nch ? pre[rg * 2] : -INFINITY;
    for (int c = lane + kWave; c < nch; c += kWave)
#pragma unroll
      for (int rg = 0; rg < kRg; ++rg) M[rg] = fmax(M[rg], lse[(c * kRg + rg) * 2]);
#pragma unroll
    for (int rg = 0; rg < kRg; ++rg) M[rg] = wave_max_d(M[rg]);
    m = fmax(M[0], M[3]);  // shift: largest exact score (head and recent tokens)
    double R[kRg];
#pragma unroll
    for (int rg = 0; rg < kRg; ++rg)
      R[rg] = (lane < nch && pre[rg * 2] != -INFINITY) ? pre[rg * 2 + 1] * exp(pre[rg * 2] - m) : 0.0;
    for (int c = lane + kWave; c < nch; c += kWave) {
      double ms[2 * kRg];  // all 8 loads in flight before any is used
#pragma unroll
      for (int i = 0; i < 2 * kRg; ++i) ms[i] = lse[c * 2 * kRg + i];
#pragma unroll
      for (int rg = 0; rg < kRg; ++rg)
        if (ms[rg * 2] != -INFINITY) R[rg] += ms[rg * 2 + 1] * exp(ms[rg * 2] - m);
    }
#pragma unroll
    for (int rg = 0; rg < kRg; ++rg) R[rg] = wave_sum_d(R[rg]);
    EN = R[0];
    Et = R[3];
    mu1 = R[1];
    mu2 = R[2];
  }
  double Tc = 0.0;  // the part of the target the clustered list must supply
  // positive interval [L, R] of the fitted curve over (N, n] and H(R), H(L - 1):
  // the tail sum S_n and the budget search share them
  bool any = false;
  int64_t L = 0, Rr = 0;
  double HL = 0.0, HR = 0.0;
  if (n > 0) {
    if (exact) {
      Sn = EN;
      mu1 = mu2 = 0.0;
    } else {
      mu1 /= (double)W1;
      mu2 /= (double)W2;
      const double x1 = (double)(hm[4] + hm[5]) / 2.0, x2 = (double)(hm[6] + hm[7]) / 2.0;
      fa = (mu1 - mu2) / (1.0 / x1 - 1.0 / x2);
      fb = mu1 - fa / x1;
      any = positive_interval(fa, fb, N + 1, n, &L, &Rr);
      if (any) {  // the two harmonic numbers in two lanes at once
        const double hx = harmonic(lane == 0 ? Rr : L - 1);
        HR = readlane_d(hx, 0);
        HL = readlane_d(hx, 1);
      }
      Sn = EN + (any ? fa * (HR - HL) + fb * (double)(Rr - L + 1) : 0.0);  // the tail sum over (N, n]
    }
  } else {
    mu1 = mu2 = 0.0;
  }
  Sn += Et;
  if (n > 0) {
    if (a.P >= 1.0) {
      k = n;
    } else {
      T = a.P * Sn;
      Tc = T - Et;
      if (tail > 0 && Tc <= 0.0) {
        k = 0;  // the recent tokens alone reach the target
      } else if (Tc <= EN) {
        // the budget lies in the exact head: find the chunk whose head part
        // crosses Tc, then scan that chunk in position order
        const int nhc = (int)((N + kSampleChunk - 1) / kSampleChunk);
        double base = 0.0;
        int cstar = nhc - 1;
        for (int c0 = 0; c0 < nhc; c0 += kWave) {
          const int c = c0 + lane, cc = min(c, nhc - 1);  // loads at clamped chunks, in flight together
          const double ml = c0 == 0 ? pre[0] : lse[(cc * kRg) * 2], sl_ = c0 == 0 ? pre[1] : lse[(cc * kRg) * 2 + 1];
          const double mc = c < nhc ? ml : -INFINITY;
          const double sc = c < nhc ? sl_ : 0.0;
          const double v = (c < nhc && mc != -INFINITY) ? sc * exp(mc - m) : 0.0;
          double incl = wave_incl_scan(v);  // DPP, no LDS
          // the running sum only grows, so the crossing is the first lane that reaches Tc
          const uint64_t hb = __ballot(c < nhc && base + incl >= Tc);
          const int hit = hb ? c0 + __ffsll((long long)hb) - 1 : 0x7fffffff;
          if (hit != 0x7fffffff) {
            cstar = hit;
            base += __shfl(incl - v, hit - c0, kWave);
            break;
          }
          base += __shfl(incl, kWave - 1, kWave);
        }
        const int64_t ub = (int64_t)cstar * kSampleChunk, ue = min(N, ub + kSampleChunk);
        int cand = 0x7fffffff;
        double run = base;
        for (int64_t v0 = ub; v0 < ue && cand == 0x7fffffff; v0 += kWave) {
          const int64_t u = v0 + lane;
          double lu = 0.0;
          if (cstar == 0) {
#pragma unroll
            for (int i = 0; i < kLg0; ++i)
              if (v0 == i * kWave) lu = lg0[i];
          } else {
            lu = lg[min(u, ue - 1)];  // unconditional (u >= ue is masked below)
          }
          const double e = u < ue ? exp(lu - m) : 0.0;
          double incl = wave_incl_scan(e);  // DPP, no LDS
          const uint64_t hb = __ballot(u < ue && run + incl >= Tc);
          cand = hb ? (int)(v0 + __ffsll((long long)hb)) : 0x7fffffff;  // u + 1 of the first such lane
          run += __shfl(incl, kWave - 1, kWave);
        }
        k = cand == 0x7fffffff ? (int)ue : cand;  // ue only if rounding lost the crossing
      } else {
        // minimal k in (N, n] with E_N + tail(N+1..k) >= Tc: 64-way parallel
        // search on the closed form over the positive interval [L, R]
        auto reached = [&](int64_t kk) -> bool {
          const int64_t r = min(kk, Rr);
          const double t = (!any || r < L) ? 0.0 : fa * (harmonic(r) - HL) + fb * (double)(r - L + 1);
          return EN + t >= Tc;
        };
        int64_t lo = N + 1, hi = n;  // the answer lies in [lo, hi]
        while (lo < hi) {
          const int64_t step = (hi - lo + kWave) / kWave;
          const int64_t cand = min(hi, lo + (int64_t)lane * step);
          const uint64_t rb = __ballot(reached(cand));  // the first reached candidate
          const int first = rb ? __ffsll((long long)rb) - 1 : kWave;
          const int64_t chi = first < kWave ? min(hi, lo + (int64_t)first * step) : hi;
          // a reached candidate bounds the answer above; if rounding left none
          // reached, the clamp ends the search at hi
          const int64_t clo = first > 0 ? min(hi, min(hi, lo + (int64_t)(first - 1) * step) + 1) : lo;
          lo = clo;
          hi = chi;
        }
        k = (int)lo;
      }
    }
  }
  // cutoff cluster: largest rank r in [0, C] with prefix[r] < k, by a 64-way
  // search of the whole wave over the prefix (prefix[0] = 0 < k keeps lane 0's
  // candidate true, and the prefix is non-decreasing)
  int cut_r = -1, cut_len = 0;
  if (k > 0) {
    const int C = hm[10];
    int lo = 0, hi = C, vlo = 0;
    // the first 64 entries settle it when prefix[63] >= k or C <= 63
    const int v63 = __shfl(rp0, kWave - 1, kWave);
    if (C <= kWave - 1 || v63 >= k) {
      const uint64_t ok = __ballot(lane <= C && rp0 < k);
      const int j = 63 - __clzll((long long)ok);
      vlo = __shfl(rp0, j, kWave);
      lo = hi = j;
    }
    while (lo < hi) {
      const int step = (hi - lo + kWave) / kWave;
      const int cand = lo + lane * step;
      const int v = cand <= hi ? rpre[cand] : 0x7fffffff;
      const uint64_t ok = __ballot(v < k);
      const int j = 63 - __clzll((long long)ok);
      vlo = __shfl(v, j, kWave);
      hi = min(hi, lo + (j + 1) * step - 1);
      lo = lo + j * step;
    }
    cut_r = lo;
    cut_len = k - vlo;
  }
  if (lane == 0) {
    cut[0] = cut_r;
    cut[1] = cut_len;
  }
  if (lane == 0 && store) {
    a.sel_count_q[bh] = k + tail;  // tokens the head attends to
    double* fit = a.fit + (int64_t)bh * kFitFields;
    fit[0] = m; fit[1] = mu1; fit[2] = mu2; fit[3] = fa; fit[4] = fb; fit[5] = Sn; fit[6] = T;
    fit[7] = (double)k; fit[8] = (double)N; fit[9] = (double)n; fit[10] = (double)exact;
    fit[11] = (double)S; fit[12] = EN; fit[13] = (double)cut_r; fit[14] = (double)cut_len;
    fit[15] = Et;
  }
}

// 3b. Fit of the G heads of a group (one wave each), then the union of their
//     selections (Sec. 4.5) and the attention work list.  grid B*Hkv, 1024
//     threads (the first G waves fit).  Staged form (G <= 4, Cm <= 8192):
//     while the first G waves fit, the other waves copy the heads' cluster
//     ranks (u16) and the cluster offsets to LDS; then every thread takes 8
//     consecutive clusters and keeps their union lengths and offsets in
//     registers through the scan and the range list.  Up to 65536 clusters
//     the staged form runs in slices (grid B*Hkv x slices) and
//     union_ranges_kernel writes the ranges.  Otherwise (G = 8), up to
//     32768 clusters: offsets to LDS while the fit runs, the heads' first
//     cut-rank clusters marked there from the sort order, 32-cluster segments
//     per thread through the scan; beyond that the union lengths go through
//     the output array between the passes.
constexpr int kUnionSeg = 8;              // clusters per thread in the staged union
constexpr int kUnionStagedMax = 8 * 1024;  // clusters of one workgroup of the staged union (kUnionSeg per thread)
__host__ __device__ inline bool union_staged(int G, int64_t Cm) {
  return G <= 4 && Cm <= (int64_t)kUnionStagedMax * kMaxUnionSlices;
}
__host__ __device__ inline bool union_sliced(int G, int64_t Cm) { return union_staged(G, Cm) && Cm > kUnionStagedMax; }

// The group's range list ends with the recent tokens (rows n_c .. n_c + tail
// - 1, the same for every head of the group) as one more range; then the
// group's counts.  tot = (cluster ranges << 32) | their tokens.
__device__ void union_close(const FitArgs& a, int bg, int b, int kvh, int n_c, int tail, uint64_t tot,
                            int32_t* rstart, int32_t* rupos, int32_t* cfr) {
  const int64_t T = kCfrTokens;
  int R = (int)(tot >> 32);
  const int64_t U = (int64_t)(tot & 0xffffffffu);
  int64_t Ut = U;
  if (tail > 0) {
    rstart[R] = n_c;
    rupos[R] = (int32_t)U;
    for (int64_t c = (U + T - 1) / T; c * T < U + tail && c < a.max_chunks; ++c) cfr[c] = R;
    ++R;
    Ut += tail;
  }
  rupos[R] = (int32_t)Ut;
  a.gmeta[bg * 4 + 0] = R;
  a.gmeta[bg * 4 + 1] = (int32_t)Ut;
  a.gmeta[bg * 4 + 2] = (int32_t)((Ut + T - 1) / T);
  a.gmeta[bg * 4 + 3] = (int32_t)T;
  if (a.per_head) atomicAdd(&a.sel_count_kv[b * a.Hkv + kvh], (int32_t)Ut);  // rows loaded per KV head
  else a.sel_count_kv[bg] = (int32_t)Ut;
}

template <int G>
__global__ __launch_bounds__(1024) void fit_union_kernel(FitArgs a) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  __shared__ uint64_t s_wave_u[17];
  __shared__ int s_cut[G][2];
  const int tid = threadIdx.x, nt = blockDim.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int bg = blockIdx.x;  // selection group: G query heads reading KV head kvh
  const int b = bg / a.NV, jg = bg % a.NV, kvh = jg / a.kv_div;
  const int h0 = b * a.Hq + jg * G;  // first query head of the group
  const int64_t T = kCfrTokens;
  int32_t* rstart = a.rstart + (int64_t)bg * (a.Cm + 2);
  int32_t* rupos = a.rupos + (int64_t)bg * (a.Cm + 2);
  int32_t* cfr = a.cfr + (int64_t)bg * a.max_chunks;
  // the sequence's clusters and the group's clustered rows / recent tokens
  // (the same for every head of the group), loaded before the fit so that
  // no global load waits behind it
  const int64_t cb = a.cl_indptr[b];
  const int C = min((int)(a.cl_indptr[b + 1] - cb), a.Cm);
  const int n_c = a.head_meta[(int64_t)h0 * 16 + 0], tail = a.head_meta[(int64_t)h0 * 16 + 11];

  if (union_staged(G, a.Cm)) {
    // up to kUnionStagedMax clusters one workgroup measures and lays out the
    // whole union; beyond that (sliced) the clusters come in slices of
    // a.union_slice, one per workgroup of the grid column (blockIdx.y): every
    // workgroup fits the group's heads, stages and measures its own slice,
    // and leaves the slice's union lengths and (ranges, tokens) total, and
    // union_ranges_kernel lays the slices' ranges end to end
    const bool sliced = a.Cm > kUnionStagedMax;
    const int kw = sliced ? (int)blockIdx.y : 0;
    const int Cp = sliced ? a.union_slice : (a.Cm + kUnionSeg - 1) / kUnionSeg * kUnionSeg;
    const int jb = kw * Cp, ns = sliced ? max(0, min(C - jb, Cp)) : C;  // clusters jb .. jb + ns - 1
    uint16_t* s_rk = reinterpret_cast<uint16_t*>(smem_raw);        // [G][Cp]
    int32_t* s_off = reinterpret_cast<int32_t*>(s_rk + G * Cp);  // [Cp + 1]
    int32_t* s_L = s_off + Cp + 4;                                // [Cp]: union lengths (16-byte aligned)
    if (wave < G) {
      fit_head_wave(a, h0 + wave, lane, s_cut[wave], kw == 0);
    } else {
      const int32_t* off = a.offsets + (int64_t)kvh * (a.Ct + a.B) + cb + b + jb;
      // all loads of a thread are issued before its LDS stores
      constexpr int nw = 1024 - G * kWave;
      constexpr int kW = (kUnionStagedMax + nw) / nw;  // covers j in [0, ns] for ns <= kUnionStagedMax
      const int w = tid - G * kWave;
      int32_t ov[kW];
#pragma unroll
      for (int i = 0; i < kW; ++i) ov[i] = w + i * nw <= ns ? off[w + i * nw] : 0;
      int32_t rv[G][kW];
#pragma unroll
      for (int hh = 0; hh < G; ++hh)
#pragma unroll
        for (int i = 0; i < kW; ++i)
          rv[hh][i] = w + i * nw < ns ? a.rank_of[(int64_t)(h0 + hh) * a.Cm + jb + w + i * nw] : 0;
#pragma unroll
      for (int i = 0; i < kW; ++i)
        if (w + i * nw <= ns) s_off[w + i * nw] = ov[i];
#pragma unroll
      for (int hh = 0; hh < G; ++hh)
#pragma unroll
        for (int i = 0; i < kW; ++i)
          if (w + i * nw < ns) s_rk[hh * Cp + w + i * nw] = (uint16_t)rv[hh][i];
    }
    __syncthreads();
    int32_t* ulen = a.union_len + (int64_t)jg * a.Ct + cb + jb;
    // union length of the thread's clusters jb + j0 .. jb + j0 + 7: the whole cluster
    // when some head ranks it before its cut (rank - cut < 0), the largest
    // cut length among the heads whose cut cluster it is (rank - cut = 0)
    const int j0 = tid * kUnionSeg;
    int32_t o[kUnionSeg + 1], L[kUnionSeg];
    uint64_t loc = 0;  // (ranges << 32) | tokens
    if (j0 < ns) {
      {  // two 16-byte LDS reads (j0 is a multiple of 8) and the next thread's first entry
        const int4 x = *reinterpret_cast<const int4*>(s_off + j0);
        const int4 y = *reinterpret_cast<const int4*>(s_off + j0 + 4);
        o[0] = x.x; o[1] = x.y; o[2] = x.z; o[3] = x.w;
        o[4] = y.x; o[5] = y.y; o[6] = y.z; o[7] = y.w;
      }
      o[kUnionSeg] = j0 + kUnionSeg <= ns ? s_off[j0 + kUnionSeg] : 0;
      int dmin[kUnionSeg];
#pragma unroll
      for (int e = 0; e < kUnionSeg; ++e) dmin[e] = 0x7fffffff;
#pragma unroll
      for (int hh = 0; hh < G; ++hh) {
        const uint4 rw = *reinterpret_cast<const uint4*>(s_rk + hh * Cp + j0);
        const uint32_t r2[4] = {rw.x, rw.y, rw.z, rw.w};
        const int c0 = s_cut[hh][0];
#pragma unroll
        for (int e = 0; e < kUnionSeg; ++e)
          dmin[e] = min(dmin[e], (int)((r2[e >> 1] >> (16 * (e & 1))) & 0xffffu) - c0);
      }
#pragma unroll
      for (int e = 0; e < kUnionSeg; ++e) {
        L[e] = dmin[e] < 0 ? o[e + 1] - o[e] : 0;
        if (dmin[e] == 0) {  // some head's cut cluster (at most G per group)
          for (int hh = 0; hh < G; ++hh)
            if ((int)s_rk[hh * Cp + j0 + e] == s_cut[hh][0]) L[e] = max(L[e], s_cut[hh][1]);
        }
      }
#pragma unroll
      for (int e = 0; e < kUnionSeg; ++e) {
        if (j0 + e < ns) {
          if (L[e] > 0) loc += (1ull << 32) | (uint64_t)L[e];
        } else {
          L[e] = 0;
        }
      }
      // the lengths go out through LDS so that the global stores are contiguous
      *reinterpret_cast<int4*>(s_L + j0) = make_int4(L[0], L[1], L[2], L[3]);
      *reinterpret_cast<int4*>(s_L + j0 + 4) = make_int4(L[4], L[5], L[6], L[7]);
    }
    uint64_t incl = wave_incl_scan(loc);  // DPP, no LDS
    if (lane == kWave - 1) s_wave_u[wave] = incl;
    __syncthreads();
    uint64_t base = incl - loc, tot = 0;
    for (int w = 0; w < 16; ++w) {
      const uint64_t t = s_wave_u[w];
      if (w < wave) base += t;
      tot += t;
    }
#pragma unroll
    for (int i = 0; i < kUnionSeg; ++i)
      if (tid + i * 1024 < ns) ulen[tid + i * 1024] = s_L[tid + i * 1024];
    if (sliced) {
      if (tid == 0) a.slice_tot[(int64_t)bg * kMaxUnionSlices + kw] = tot;
      return;
    }
    if (j0 < ns) {
      int idx = (int)(base >> 32);
      int64_t upos = (int64_t)(base & 0xffffffffu);
#pragma unroll
      for (int e = 0; e < kUnionSeg; ++e) {
        if (L[e] > 0) {
          rstart[idx] = o[e];
          rupos[idx] = (int32_t)upos;
          for (int64_t c = (upos + T - 1) / T; c * T < upos + L[e] && c < a.max_chunks; ++c) cfr[c] = idx;
          ++idx;
          upos += L[e];
        }
      }
    }
    if (tid == 0) union_close(a, bg, b, kvh, n_c, tail, tot, rstart, rupos, cfr);
    return;
  }

  const int32_t* off = a.offsets + (int64_t)kvh * (a.Ct + a.B) + cb + b;
  int32_t* ulen = a.union_len + (int64_t)jg * a.Ct + cb;
  const int mc = (int)min((int64_t)a.max_chunks, (int64_t)INT32_MAX), Ti = (int)T;
  uint64_t tot;  // (ranges << 32) | tokens of the clustered union
  // exclusive block scan of (ranges << 32) | tokens: DPP within the wave,
  // then the wave totals; returns the thread's base and sets tot
  auto block_scan = [&](uint64_t loc) {
    const uint64_t incl = wave_incl_scan(loc);
    if (lane == kWave - 1) s_wave_u[wave] = incl;
    __syncthreads();
    if (tid == 0) {
      uint64_t run = 0;
      for (int w = 0; w < nt / kWave; ++w) {
        const uint64_t t = s_wave_u[w];
        s_wave_u[w] = run;
        run += t;
      }
      s_wave_u[16] = run;
    }
    __syncthreads();
    tot = s_wave_u[16];
    return s_wave_u[wave] + incl - loc;
  };

  if (a.Cm <= kUnionLdsMax) {
    // One workgroup per group runs every pass here, so the passes are kept
    // short in instructions per cluster. LDS holds the cluster offsets (one
    // pad entry after every 32, so that the threads' 32-entry segments start
    // in different banks), their top bit set for clusters some head takes
    // whole; later each cluster's union length or position. With many
    // ranges: per 32 clusters a bit per non-empty cluster and the count of
    // non-empty clusters before them.
    static_assert(kUnionLdsMax <= 32 * 1024, "one 32-cluster segment per thread");
    const int Cp = (a.Cm + 31) / 32 * 32;                      // whole segments
    int32_t* const Lo = reinterpret_cast<int32_t*>(smem_raw);  // [Cp + Cp / 32 + 1]
    auto li = [](int j) { return j + (j >> 5); };
    uint32_t* s_nz = reinterpret_cast<uint32_t*>(Lo + Cp + Cp / 32 + 1);  // [Cp / 32]
    int32_t* s_wb = reinterpret_cast<int32_t*>(s_nz + Cp / 32);           // [Cp / 32]
    __shared__ int s_cutj[G];                                                  // cut cluster, -1: none
    if (wave < G) {
      fit_head_wave(a, h0 + wave, lane, s_cut[wave], true);
      if (lane == 0) s_cutj[wave] = -1;
    } else {
      // offsets 0 .. C into LDS while the fit runs (8 per thread and step loaded together)
      constexpr int nw = 1024 - G * kWave;
      const int w = tid - G * kWave;
      for (int k0 = 0; k0 * nw <= C; k0 += 8) {
        int o[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] = off[min((k0 + e) * nw + w, C)];
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if ((k0 + e) * nw + w <= C) Lo[li((k0 + e) * nw + w)] = o[e];
      }
    }
    __syncthreads();
    {
      // marks: every head's clusters ranked before its cut (its first
      // cut-rank entries of the sort order) get the top bit, and the cut
      // cluster is noted; the heads' entries taken as one list, 8 per thread
      // and step loaded together
      int pre[G + 1];
      pre[0] = 0;
#pragma unroll
      for (int hh = 0; hh < G; ++hh) {
        const int c0 = s_cut[hh][0];
        pre[hh + 1] = pre[hh] + (c0 < C ? c0 + 1 : C);  // c0 = -1: no cluster
      }
      const int NR = pre[G];
      auto head_of = [&](int t) {
        int hh = 0;
#pragma unroll
        for (int k = 1; k < G; ++k) hh += t >= pre[k] ? 1 : 0;
        return hh;
      };
      for (int t0 = 0; t0 < NR; t0 += 8 * nt) {
        int jv[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int t = min(t0 + e * nt + tid, NR - 1);
          const int hh = head_of(t);
          jv[e] = a.order[(int64_t)(h0 + hh) * a.Cm + (t - pre[hh])];
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int t = t0 + e * nt + tid;
          if (t < NR) {
            const int hh = head_of(t);
            if (t - pre[hh] == s_cut[hh][0]) s_cutj[hh] = jv[e];
            else atomicOr(reinterpret_cast<unsigned int*>(Lo) + li(jv[e]), 0x80000000u);
          }
        }
      }
    }
    __syncthreads();
    // segments of 32 clusters (C <= 32 * 1024): union length = the size for
    // a marked cluster, at least the cut length at a head's cut cluster
    constexpr int kSeg = 32;
    const int beg = tid * kSeg;
    int L[kSeg];
    uint64_t loc = 0;  // (ranges << 32) | tokens
    if (beg < C) {
      int o[kSeg + 1];
#pragma unroll
      for (int e = 0; e <= kSeg; ++e) o[e] = Lo[li(min(beg + e, C))];
#pragma unroll
      for (int e = 0; e < kSeg; ++e) {
        L[e] = (o[e] < 0 && beg + e < C) ? (o[e + 1] & 0x7fffffff) - (o[e] & 0x7fffffff) : 0;
        loc += L[e];
      }
      bool has_cut = false;
#pragma unroll
      for (int hh = 0; hh < G; ++hh) has_cut |= (unsigned)(s_cutj[hh] - beg) < (unsigned)kSeg;
      if (has_cut) {
        loc = 0;
#pragma unroll
        for (int hh = 0; hh < G; ++hh) {
          const int cj = s_cutj[hh], cl = s_cut[hh][1];
#pragma unroll
          for (int e = 0; e < kSeg; ++e)
            if (beg + e == cj) L[e] = max(L[e], cl);
        }
#pragma unroll
        for (int e = 0; e < kSeg; ++e) loc += L[e];
      }
      int nr = 0;
#pragma unroll
      for (int e = 0; e < kSeg; ++e) nr += L[e] > 0 ? 1 : 0;
      loc |= (uint64_t)nr << 32;
    }
    const uint64_t base = block_scan(loc);
    // few ranges (the common case with this many clusters): each thread
    // writes its segment's ranges, scattered across the lanes but rare;
    // else a coalesced pass writes them, neighbouring lanes writing
    // neighbouring ranges
    const bool few = (tot >> 32) * 8 <= (uint64_t)C;
    if (beg < C) {
      int idx = (int)(base >> 32), upos = (int)(base & 0xffffffffu);
      if (few) {
        // each cluster's union length replaces its offset (the last segment
        // also writes entries past C, which nothing reads); a non-empty
        // cluster's range and the position -> range index, one entry per
        // kCfrTokens positions
#pragma unroll
        for (int e0 = 0; e0 < kSeg; e0 += 8) {
          int o[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) o[e] = Lo[li(beg + e0 + e)];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int Le = L[e0 + e];
            Lo[li(beg + e0 + e)] = Le;
            if (Le > 0) {
              rstart[idx] = o[e] & 0x7fffffff;
              rupos[idx] = upos;
              for (int c = (upos + Ti - 1) / Ti; c * Ti < upos + Le && c < mc; ++c) cfr[c] = idx;
              ++idx;
            }
            upos += Le;
          }
        }
      } else {
        // each cluster's union position replaces its offset (the last
        // segment writes C's entry, the total, and entries past it, which
        // nothing reads); the segment's non-empty bits and the range count
        // before it
        uint32_t nzb = 0;
#pragma unroll
        for (int e = 0; e < kSeg; ++e) {
          Lo[li(beg + e)] = upos;
          upos += L[e];
          nzb |= (L[e] > 0 ? 1u : 0u) << e;
        }
        s_nz[tid] = nzb;
        s_wb[tid] = idx;
      }
    }
    if (!few && tid == 0 && (C & 31) == 0) Lo[li(C)] = (int)(tot & 0xffffffffu);  // no segment holds C
    __syncthreads();
    if (few) {
      // union lengths out (coalesced)
      for (int k0 = 0; k0 * nt < C; k0 += 8) {
        int v[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = Lo[li(min((k0 + e) * nt + tid, C - 1))];
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if ((k0 + e) * nt + tid < C) ulen[(k0 + e) * nt + tid] = v[e];
      }
    } else {
      // coalesced: union lengths out, and per non-empty cluster its range
      // (index = non-empty clusters before it) and the position -> range
      // index; the cluster starts are loaded with the step's LDS reads, so
      // that no load waits behind the stores
      for (int k0 = 0; k0 * nt < C; k0 += 4) {
        int u0[4], u1[4], wb[4], ov[4];
        uint32_t m[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int jj = min((k0 + e) * nt + tid, C - 1);
          ov[e] = off[jj];
          u0[e] = Lo[li(jj)];
          u1[e] = Lo[li(jj + 1)];
          m[e] = s_nz[jj >> 5];
          wb[e] = s_wb[jj >> 5];
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int j = (k0 + e) * nt + tid;
          const int Lj = u1[e] - u0[e];
          if (j < C) {
            ulen[j] = Lj;
            if (Lj > 0) {
              const int r = wb[e] + __popc(m[e] & ((1u << (j & 31)) - 1u));
              rstart[r] = ov[e];
              rupos[r] = u0[e];
              for (int c = (u0[e] + Ti - 1) / Ti; c * Ti < u0[e] + Lj && c < mc; ++c) cfr[c] = r;
            }
          }
        }
      }
    }
  } else {
    if (wave < G) fit_head_wave(a, h0 + wave, lane, s_cut[wave], true);
    __syncthreads();
    // pass 1 (coalesced, kB clusters per thread and step loaded together at
    // clamped indices): selected prefix length of every cluster = max over
    // heads, into the union-length output
    constexpr int kB = G >= 8 ? 4 : 8;
    for (int k0 = 0; k0 * nt < C; k0 += kB) {
      int o0[kB], o1[kB], rk[kB][G];
#pragma unroll
      for (int e = 0; e < kB; ++e) {
        const int jj = min((k0 + e) * nt + tid, C - 1);
        o0[e] = off[jj];
        o1[e] = off[jj + 1];
#pragma unroll
        for (int hh = 0; hh < G; ++hh) rk[e][hh] = a.rank_of[(int64_t)(h0 + hh) * a.Cm + jj];
      }
#pragma unroll
      for (int e = 0; e < kB; ++e) {
        const int j = (k0 + e) * nt + tid;
        const int size = o1[e] - o0[e];
        int L = 0;
#pragma unroll
        for (int hh = 0; hh < G; ++hh) {
          const int r = rk[e][hh];
          L = max(L, r < s_cut[hh][0] ? size : (r == s_cut[hh][0] ? s_cut[hh][1] : 0));
        }
        if (j < C) ulen[j] = L;
      }
    }
    __syncthreads();
    // pass 2: compact the non-empty clusters into ranges (contiguous segment
    // per thread), 8 entries per step read together
    const int seg = (C + nt - 1) / nt;
    const int beg = min(C, tid * seg), end = min(C, beg + seg);
    uint64_t loc = 0;  // (ranges << 32) | tokens
    for (int j0 = beg; j0 < end; j0 += 8) {
      int Lv[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) Lv[e] = ulen[min(j0 + e, end - 1)];
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (j0 + e < end && Lv[e] > 0) loc += (1ull << 32) | (uint64_t)Lv[e];
    }
    const uint64_t base = block_scan(loc);
    // the thread writes its own segment's ranges, 8 lengths and cluster
    // starts per step loaded together (union positions fit 32 bits: a
    // sequence holds fewer than 2^31 tokens)
    int idx = (int)(base >> 32), upos = (int)(base & 0xffffffffu);
    for (int j0 = beg; j0 < end; j0 += 8) {
      int Lv[8], ov[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int jj = min(j0 + e, end - 1);
        Lv[e] = ulen[jj];
        ov[e] = off[jj];
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        if (j0 + e < end && Lv[e] > 0) {
          rstart[idx] = ov[e];
          rupos[idx] = upos;
          for (int c = (upos + Ti - 1) / Ti; c * Ti < upos + Lv[e] && c < mc; ++c) cfr[c] = idx;
          ++idx;
          upos += Lv[e];
        }
      }
    }
  }
  if (tid == 0) union_close(a, bg, b, kvh, n_c, tail, tot, rstart, rupos, cfr);
}

// Ranges of the sliced staged union: workgroup kw of group bg takes its
// slice of clusters, starts from the (ranges, tokens) of the slices before
// it, and writes the slice's (row, position) ranges and the chunk-index
// entries whose first position falls in them; the last slice's workgroup
// closes the group's list.
__global__ __launch_bounds__(1024) void union_ranges_kernel(FitArgs a) {
  __shared__ uint64_t s_wave_u[16];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int bg = blockIdx.x, kw = blockIdx.y, nwu = gridDim.y;
  const int b = bg / a.NV, jg = bg % a.NV, kvh = jg / a.kv_div;
  const int h0 = b * a.Hq + jg * (a.Hq / a.NV);  // first query head of the group
  const int64_t T = kCfrTokens;
  int32_t* rstart = a.rstart + (int64_t)bg * (a.Cm + 2);
  int32_t* rupos = a.rupos + (int64_t)bg * (a.Cm + 2);
  int32_t* cfr = a.cfr + (int64_t)bg * a.max_chunks;
  const int64_t cb = a.cl_indptr[b];
  const int C = min((int)(a.cl_indptr[b + 1] - cb), a.Cm);
  const int Cs = a.union_slice, jb = kw * Cs, ns = max(0, min(C - jb, Cs));
  const int32_t* off = a.offsets + (int64_t)kvh * (a.Ct + a.B) + cb + b + jb;
  const int32_t* ulen = a.union_len + (int64_t)jg * a.Ct + cb + jb;
  uint64_t base = 0, all = 0;  // the slices before this one; all of them
  for (int w = 0; w < nwu; ++w) {
    const uint64_t t = a.slice_tot[(int64_t)bg * kMaxUnionSlices + w];
    base += w < kw ? t : 0ull;
    all += t;
  }
  const int j0 = tid * kUnionSeg;  // the thread's clusters jb + j0 .. jb + j0 + 7
  int32_t o[kUnionSeg], L[kUnionSeg];
  uint64_t loc = 0;
#pragma unroll
  for (int e = 0; e < kUnionSeg; ++e) {
    const bool in = j0 + e < ns;
    o[e] = in ? off[j0 + e] : 0;
    L[e] = in ? ulen[j0 + e] : 0;
  }
#pragma unroll
  for (int e = 0; e < kUnionSeg; ++e)
    if (L[e] > 0) loc += (1ull << 32) | (uint64_t)L[e];
  const uint64_t incl = wave_incl_scan(loc);  // DPP, no LDS
  if (lane == kWave - 1) s_wave_u[wave] = incl;
  __syncthreads();
  uint64_t mine = base + incl - loc;
  for (int w = 0; w < wave; ++w) mine += s_wave_u[w];
  int idx = (int)(mine >> 32);
  int64_t upos = (int64_t)(mine & 0xffffffffu);
#pragma unroll
  for (int e = 0; e < kUnionSeg; ++e) {
    if (L[e] > 0) {
      rstart[idx] = o[e];
      rupos[idx] = (int32_t)upos;
      for (int64_t c = (upos + T - 1) / T; c * T < upos + L[e] && c < a.max_chunks; ++c) cfr[c] = idx;
      ++idx;
      upos += L[e];
    }
  }
  if (kw == nwu - 1 && tid == 0) {
    const int n_c = a.head_meta[(int64_t)h0 * 16 + 0], tail = a.head_meta[(int64_t)h0 * 16 + 11];
    union_close(a, bg, b, kvh, n_c, tail, all, rstart, rupos, cfr);
  }
}

// ============================================================================
// Launchers
// ============================================================================
hipError_t launch_score(const ScoreArgs& a, int G, int grid_x, int grid_y, hipStream_t st) {
  dim3 grid(grid_x, grid_y);
  switch (G) {
    case 1: hipLaunchKernelGGL(score_clusters_kernel<1>, grid, dim3(256), 0, st, a); break;
    case 2: hipLaunchKernelGGL(score_clusters_kernel<2>, grid, dim3(256), 0, st, a); break;
    case 4: hipLaunchKernelGGL(score_clusters_kernel<4>, grid, dim3(256), 0, st, a); break;
    case 8: hipLaunchKernelGGL(score_clusters_kernel<8>, grid, dim3(256), 0, st, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_sort(const SortArgs& a, bool lds, int n_heads, hipStream_t st) {
  if (lds) {
    const size_t bytes = (size_t)kSortLdsBuckets * 16;  // keys u64, cnt u32, start u32
    hipLaunchKernelGGL(sort_clusters_kernel<true>, dim3(n_heads), dim3(1024), bytes, st, a);
  } else {
    // beyond 8192 clusters a head's pieces are shared by up to 8 workgroups,
    // so that few heads still occupy the device's 256 compute units
    const int nw = max(1, min(8, 256 / max(n_heads, 1)));
    hipLaunchKernelGGL(sort_clusters_kernel<false>, dim3(n_heads, nw), dim3(1024), kSortWsLdsBytes, st, a);
  }
  return hipGetLastError();
}

hipError_t launch_sample(const FitArgs& a, int split, int n_heads, bool paged, hipStream_t st) {
  if (paged) hipLaunchKernelGGL(sample_logits_kernel<true>, dim3(split, n_heads), dim3(256), 0, st, a);
  else hipLaunchKernelGGL(sample_logits_kernel<false>, dim3(split, n_heads), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_fit_union(const FitArgs& args, int G, int n_groups, hipStream_t st) {
  FitArgs a = args;
  const bool sliced = union_sliced(G, a.Cm);
  // beyond kUnionStagedMax clusters the staged union runs in slices of at
  // most that many, up to kMaxUnionSlices workgroups per group (as many as
  // fill the device's 256 compute units), then a second kernel lays out the
  // ranges
  int nwu = 1;
  a.union_slice = 0;
  if (sliced) {
    nwu = (int)max((a.Cm + kUnionStagedMax - 1) / kUnionStagedMax, (int64_t)min(kMaxUnionSlices, 256 / max(n_groups, 1)));
    nwu = min(nwu, kMaxUnionSlices);
    a.union_slice = (int)(((a.Cm + nwu - 1) / nwu + kUnionSeg - 1) / kUnionSeg * kUnionSeg);
    nwu = (int)((a.Cm + a.union_slice - 1) / a.union_slice);
  }
  const int64_t Cp = sliced ? a.union_slice : (a.Cm + kUnionSeg - 1) / kUnionSeg * kUnionSeg;
  const int64_t C32 = (a.Cm + 31) / 32 * 32;
  const size_t lds = union_staged(G, a.Cm) ? (size_t)(G * Cp * 2 + (Cp + 4) * 4 + Cp * 4)
                                           : (a.Cm <= kUnionLdsMax ? (size_t)(C32 + 3 * (C32 / 32) + 1) * 4 : 0);
  const dim3 grid(n_groups, nwu);
  switch (G) {
    case 1: hipLaunchKernelGGL(fit_union_kernel<1>, grid, dim3(1024), lds, st, a); break;
    case 2: hipLaunchKernelGGL(fit_union_kernel<2>, grid, dim3(1024), lds, st, a); break;
    case 4: hipLaunchKernelGGL(fit_union_kernel<4>, grid, dim3(1024), lds, st, a); break;
    case 8: hipLaunchKernelGGL(fit_union_kernel<8>, grid, dim3(1024), lds, st, a); break;
    default: return hipErrorInvalidValue;
  }
  if (sliced) {
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(union_ranges_kernel, grid, dim3(1024), 0, st, a);
  }
  return hipGetLastError();
}

}  // namespace tactic
