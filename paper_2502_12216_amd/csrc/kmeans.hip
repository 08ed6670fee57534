// Prefill K-means clustering of the keys (Sec. 4.2) for gfx950.
//
// One problem per (sequence b, KV head g): n_b keys, C_b clusters, started
// from the keys of the sampled tokens init_idx.  Each iteration:
//   km_assign   nearest stored centroid of every key: the largest
//               k.c - ||c||^2 / 2, contracted on MFMA (v_mfma_f32_32x32x16_bf16,
//               fp32 accumulation) with a fused argmax (ties to the smaller id);
//               counts assignments that changed.
//   km_hist     per tile of 2048 tokens: sort (cluster, token) keys in LDS,
//               giving each token its rank among same-cluster tokens of the
//               tile, and the tile's count of every cluster.  An iteration
//               whose assignment step changed nothing ends the problem.
//   km_scan*    exclusive scan of the (cluster, tile) counts: start row of
//               every cluster and of every (cluster, tile) run.
//   km_perm     stable counting-sort scatter: perm[row] = token.
//   km_mean     centroid = mean of the members, summed in row order (fixed,
//               so results are deterministic), rounded to bf16; an empty
//               cluster keeps its centroid.
// After the last iteration the K/V rows are permuted into cluster order.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <algorithm>

#include "common.hpp"
#include "kmeans.hpp"

namespace tactic {

constexpr int kKmTile = 2048;       // tokens per counting tile
constexpr int kKmChunk = 16384;     // table entries per scan chunk
constexpr int kKmMaxIters = 1000;
constexpr int kAsgTok = 256;        // tokens per assignment workgroup (4 waves x 64)
constexpr int kAsgCen = 96;         // centroids staged in LDS per step

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

struct KmArgs {
  const uint16_t* K;
  const uint16_t* V;
  const int64_t* kv_indptr;
  const int64_t* seq_len;     // [B] or null (see tactic_kv_shape)
  const int64_t* cl_indptr;
  int B, Hkv, Cm, tiles_max, chunks_max, iter, max_iters;
  int64_t total, Ct;
  const int32_t* init_idx;
  const uint16_t* prev_centroids;  // warm start, or null
  const int64_t* prev_cl_indptr;
  uint16_t* centroids;
  float* cnorm;
  int32_t* assign;
  int32_t* offsets;
  int32_t* perm;
  int32_t* local_rank;
  int32_t* table;
  int32_t* chunk_sums;
  int32_t* changed;  // [max_iters + 1][BG]
  int32_t* done;     // [BG]
  uint16_t* K_sorted;
  uint16_t* V_sorted;
};

struct Problem {
  int b, g, n, C, tiles;
  int64_t tok_base, cl_base, off_base;
};

__device__ __forceinline__ Problem problem(const KmArgs& a, int p) {
  Problem q;
  q.b = p / a.Hkv;
  q.g = p % a.Hkv;
  const int64_t s0 = a.kv_indptr[q.b], c0 = a.cl_indptr[q.b];
  q.n = (int)seq_tokens(a.kv_indptr, a.seq_len, q.b);
  q.C = min((int)(a.cl_indptr[q.b + 1] - c0), a.Cm);
  q.tiles = (q.n + kKmTile - 1) / kKmTile;
  q.tok_base = (int64_t)q.g * a.total + s0;
  q.cl_base = (int64_t)q.g * a.Ct + c0;
  q.off_base = (int64_t)q.g * (a.Ct + a.B) + c0 + q.b;
  return q;
}

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// ---------------------------------------------------------------------------
// init: c0 = K[init_idx] (or the previous clustering's centroid j for a warm
// start), ||c0||^2, per-problem flags.  grid (ceil(Cm/4), BG)
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void km_init_kernel(KmArgs a) {
  const int p = blockIdx.y;
  const Problem q = problem(a, p);
  if (blockIdx.x == 0) {
    for (int i = threadIdx.x; i <= a.max_iters; i += blockDim.x) a.changed[(int64_t)i * a.B * a.Hkv + p] = 0;
    if (threadIdx.x == 0) a.done[p] = 0;
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, sl = lane & 15, grp = lane >> 4;
  const int j = blockIdx.x * 4 + wave;
  if (j >= q.C || grp != 0 || q.n == 0) return;
  uint4 v;
  const int64_t pc0 = a.prev_centroids ? a.prev_cl_indptr[q.b] : 0;
  const int64_t pc1 = a.prev_centroids ? a.prev_cl_indptr[q.b + 1] : 0;
  if (j < pc1 - pc0) {
    // warm start: the previous clustering's centroid j of this (b, g)
    const int64_t prev_total = a.prev_cl_indptr[a.B];
    v = *reinterpret_cast<const uint4*>(a.prev_centroids + ((int64_t)q.g * prev_total + pc0 + j) * kHeadDim + sl * 8);
  } else {
    const int t = min(max(a.init_idx[q.cl_base + j], 0), q.n - 1);
    v = *reinterpret_cast<const uint4*>(a.K + (q.tok_base + t) * kHeadDim + sl * 8);
  }
  *reinterpret_cast<uint4*>(a.centroids + (q.cl_base + j) * kHeadDim + sl * 8) = v;
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
  float s = 0.f;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float x = bf16lo(w[e]), y = bf16hi(w[e]);
    s = fmaf(x, x, s);
    s = fmaf(y, y, s);
  }
  s = sum16(s);
  if (sl == 0) a.cnorm[q.cl_base + j] = s;
}

// ---------------------------------------------------------------------------
// assignment: grid (ceil(nmax/256), BG), 256 threads.  A wave owns 64 tokens
// (two 32-token MFMA B operands held in registers for the whole pass);
// centroids stream through LDS 96 at a time as the A operand, each tile
// loaded from memory straight into the other of two LDS buffers while the
// one before it is contracted (one barrier per tile).  The nearest
// centroid maximises s = k.c - ||c||^2 / 2; the accumulators of a block start
// at the fp32 -||c||^2 / 2 of their centroid row, so the contraction ends on
// finished scores and the epilogue is a 3-input max over each lane's 16
// scores of a block, and the search for the row that holds it only when some
// lane of the wave improved on its best (strict, so the smaller centroid id
// wins a tie).
// ---------------------------------------------------------------------------
// three waves per SIMD: the B operands and accumulators live in VGPRs (a
// few registers of the unrolled tile staging spill; rolling that loop to
// avoid it was slower)
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3))) void km_assign_kernel(KmArgs a) {
  // two centroid tiles (the next one loads while this one is contracted):
  // rows of 16 chunks of 16 bytes, logical chunk c of row r stored at chunk
  // c ^ (r & 15), so that the 32 rows an A-operand read touches at one
  // logical chunk fall in distinct LDS bank groups
  __shared__ __align__(16) uint16_t s_c[2][kAsgCen * kHeadDim];
  __shared__ __align__(16) float s_nh[2][kAsgCen];  // -||c||^2 / 2 (-inf past the last centroid)
  const int p = blockIdx.y;
  if (a.done[p]) return;
  const Problem q = problem(a, p);
  const int i0 = blockIdx.x * kAsgTok;
  if (i0 >= q.n) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, col = lane & 31;

  bf16x8 bt[2][8];
#pragma unroll
  for (int bb = 0; bb < 2; ++bb) {
    const int tok = i0 + wave * 64 + bb * 32 + col;
    const uint16_t* src = a.K + (q.tok_base + min(tok, q.n - 1)) * kHeadDim + 64 * half;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (tok < q.n) v = *reinterpret_cast<const uint4*>(src + 8 * s);
      bt[bb][s] = __builtin_bit_cast(bf16x8, v);
    }
  }
  float best_v[2] = {-INFINITY, -INFINITY};
  int best_j[2] = {0x7fffffff, 0x7fffffff};
  const uint16_t* cbase = a.centroids + q.cl_base * kHeadDim;
  // a tile goes from memory straight to LDS (no registers): each wave moves
  // four blocks of 64 chunks; lane L of block blk fills stored chunk
  // blk * 64 + L, i.e. row (blk * 64 + L) / 16, with the row's logical chunk
  // that the swizzle puts there; rows past C load a valid row (their scores
  // are -inf through the norm term)
  auto stage = [&](int c0, int buf) {
#pragma unroll
    for (int i = 0; i < kAsgCen * 16 / 256; ++i) {
      const int blk = wave * (kAsgCen * 16 / 256) + i, qq = blk * 64 + lane, row = qq >> 4;
      const int grow = min(c0 + row, q.C - 1);
      __builtin_amdgcn_global_load_lds(cbase + (int64_t)grow * kHeadDim + ((qq & 15) ^ (row & 15)) * 8,
                                       (__attribute__((address_space(3))) void*)(s_c[buf] + blk * 512), 16, 0, 0);
    }
  };
  float pfn = (tid < kAsgCen && tid < q.C) ? a.cnorm[q.cl_base + tid] : 0.f;
  if (q.C > 0) stage(0, 0);
  int buf = 0;
  for (int c0 = 0; c0 < q.C; c0 += kAsgCen, buf ^= 1) {
    if (tid < kAsgCen) s_nh[buf][tid] = c0 + tid < q.C ? -0.5f * pfn : -INFINITY;
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wave's tile loads have reached LDS
    __syncthreads();  // every wave's part of the tile and the norms in place; the other buffer free
    if (c0 + kAsgCen < q.C) {
      stage(c0 + kAsgCen, buf ^ 1);
      if (tid < kAsgCen && c0 + kAsgCen + tid < q.C) pfn = a.cnorm[q.cl_base + c0 + kAsgCen + tid];
    }
    const int nblk = min(kAsgCen / 32, (q.C - c0 + 31) / 32);
    for (int cb = 0; cb < nblk; ++cb) {
      // accumulator i of a lane is row 8 (i / 4) + 4 half + i % 4 of the block
      f32x16 acc[2];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const float4 x = *reinterpret_cast<const float4*>(s_nh[buf] + cb * 32 + 8 * k + 4 * half);
        acc[0][4 * k] = acc[1][4 * k] = x.x;
        acc[0][4 * k + 1] = acc[1][4 * k + 1] = x.y;
        acc[0][4 * k + 2] = acc[1][4 * k + 2] = x.z;
        acc[0][4 * k + 3] = acc[1][4 * k + 3] = x.w;
      }
      const uint16_t* arow = s_c[buf] + (cb * 32 + col) * kHeadDim;  // row cb * 32 + col: swizzle col & 15
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const bf16x8 av = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(arow + (((8 * half + s) ^ (col & 15)) * 8)));
        acc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bt[0][s], acc[0], 0, 0, 0);
        acc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bt[1][s], acc[1], 0, 0, 0);
      }
#pragma unroll
      for (int bb = 0; bb < 2; ++bb) {
        const f32x16 v = acc[bb];
        float m = fmaxf(fmaxf(v[0], v[1]), v[2]);
        m = fmaxf(fmaxf(m, v[3]), v[4]);
        m = fmaxf(fmaxf(m, v[5]), v[6]);
        m = fmaxf(fmaxf(m, v[7]), v[8]);
        m = fmaxf(fmaxf(m, v[9]), v[10]);
        m = fmaxf(fmaxf(m, v[11]), v[12]);
        m = fmaxf(fmaxf(m, v[13]), v[14]);
        m = fmaxf(m, v[15]);
        const bool imp = m > best_v[bb];
        if (__any(imp)) {
          int r = 0;  // the smallest row of this lane that holds m
#pragma unroll
          for (int i = 15; i >= 0; --i) r = v[i] == m ? 8 * (i / 4) + 4 * half + (i % 4) : r;
          if (imp) {
            best_v[bb] = m;
            best_j[bb] = c0 + cb * 32 + r;
          }
        }
      }
    }
  }
  int nchg = 0;
#pragma unroll
  for (int bb = 0; bb < 2; ++bb) {
    const float ov = __shfl_xor(best_v[bb], 32, 64);
    const int oj = __shfl_xor(best_j[bb], 32, 64);
    if (ov > best_v[bb] || (ov == best_v[bb] && oj < best_j[bb])) {
      best_v[bb] = ov;
      best_j[bb] = oj;
    }
    const int tok = i0 + wave * 64 + bb * 32 + col;
    if (half == 0 && tok < q.n) {
      const int jn = min(max(best_j[bb], 0), q.C - 1);
      int32_t* dst = a.assign + q.tok_base + tok;
      if (a.iter > 1 && *dst != jn) ++nchg;
      *dst = jn;
    }
  }
  for (int o = 32; o > 0; o >>= 1) nchg += __shfl_xor(nchg, o, 64);
  if (lane == 0 && nchg > 0) atomicAdd(a.changed + (int64_t)a.iter * a.B * a.Hkv + p, nchg);
}

// ---------------------------------------------------------------------------
// counting tile: grid (tiles_max, BG), 1024 threads
// ---------------------------------------------------------------------------
__device__ __forceinline__ int lower_bound_u32(const uint32_t* s, int n, uint32_t key) {
  int lo = 0, hi = n;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (s[mid] < key) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

constexpr int kHistLdsCounts = 8192;  // clusters whose tile counts are gathered in LDS

__global__ __launch_bounds__(1024) void km_hist_kernel(KmArgs a) {
  __shared__ uint32_t s_key[kKmTile];
  __shared__ int32_t s_cnt[kHistLdsCounts];
  const int p = blockIdx.y;
  if (a.done[p]) return;
  if (a.iter > 1 && a.changed[(int64_t)a.iter * a.B * a.Hkv + p] == 0) {
    if (blockIdx.x == 0 && threadIdx.x == 0) a.done[p] = 1;  // converged: nothing changed
    return;
  }
  const Problem q = problem(a, p);
  const int t = blockIdx.x;
  const int i0 = t * kKmTile;
  if (i0 >= q.n) return;
  const int m = min(kKmTile, q.n - i0);
  const int tid = threadIdx.x;
  const bool lds_counts = q.C <= kHistLdsCounts;
  if (lds_counts)
    for (int c = tid; c < q.C; c += 1024) s_cnt[c] = 0;  // ordered before use by the sort's barriers
  for (int x = tid; x < kKmTile; x += 1024)
    s_key[x] = x < m ? ((uint32_t)a.assign[q.tok_base + i0 + x] << 11) | (uint32_t)x : 0xffffffffu;
  // bitonic sort of 2048 keys, one compare-exchange per thread per step
  for (int k = 2; k <= kKmTile; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      __syncthreads();
      const int i = 2 * tid - (tid & (j - 1));  // lower index of this thread's pair
      const int l = i + j;
      const uint32_t x = s_key[i], y = s_key[l];
      const bool up = (i & k) == 0;
      if ((x > y) == up) {
        s_key[i] = y;
        s_key[l] = x;
      }
    }
  }
  __syncthreads();
  // rank of each token among the tile's tokens of its cluster (offset from
  // the start of its run of equal clusters); the last token of a run holds
  // the cluster's count in this tile
  for (int s = tid; s < m; s += 1024) {
    const uint32_t key = s_key[s];
    const uint32_t c = key >> 11;
    const int lb = lower_bound_u32(s_key, m, c << 11);
    a.local_rank[q.tok_base + i0 + (key & 2047u)] = s - lb;
    if (lds_counts && (s == m - 1 || (s_key[s + 1] >> 11) != c)) s_cnt[c] = s - lb + 1;
  }
  int32_t* tab = a.table + (int64_t)p * a.Cm * a.tiles_max + (int64_t)t * q.C;  // this tile's row
  if (lds_counts) {
    __syncthreads();
    for (int c = tid; c < q.C; c += 1024) tab[c] = s_cnt[c];
  } else {
    for (int c = tid; c < q.C; c += 1024) {
      const int lo = lower_bound_u32(s_key, m, (uint32_t)c << 11);
      const int hi = lower_bound_u32(s_key, m, (uint32_t)(c + 1) << 11);
      tab[c] = hi - lo;
    }
  }
}

// ---------------------------------------------------------------------------
// exclusive scan of the (cluster, tile) counts in cluster-major order
// (x = c * tiles + t); the table is stored tile-major (entry t * C + c), so
// that each counting tile writes one contiguous row
// ---------------------------------------------------------------------------

__device__ __forceinline__ bool km_active(const KmArgs& a, int p) {
  return !a.done[p];
}

__global__ __launch_bounds__(1024) void km_scan1_kernel(KmArgs a) {
  __shared__ int s_w[16];
  const int p = blockIdx.y;
  if (!km_active(a, p)) return;
  const Problem q = problem(a, p);
  const int64_t E = (int64_t)q.C * q.tiles;
  const int64_t x0 = (int64_t)blockIdx.x * kKmChunk;
  if (x0 >= E) return;
  const int32_t* tab = a.table + (int64_t)p * a.Cm * a.tiles_max;
  // 16 consecutive entries per thread, their (tile, cluster) stepped from
  // the first one's
  const int64_t b0 = x0 + (int64_t)threadIdx.x * 16, b1 = min(E, b0 + 16);
  const int t0 = (int)(b0 % q.tiles), c0 = (int)(b0 / q.tiles);
  // every load unconditional (entries past the end read entry 0 and count
  // nothing) so that the 16 are in flight together
  int s = 0;
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const int te = t0 + e;
    const bool in = b0 + e < b1;
    const int v = tab[in ? (int64_t)(te % q.tiles) * q.C + c0 + te / q.tiles : 0];
    s += in ? v : 0;
  }
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
  if ((threadIdx.x & 63) == 0) s_w[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    int t = 0;
    for (int w = 0; w < 16; ++w) t += s_w[w];
    a.chunk_sums[(int64_t)p * a.chunks_max + blockIdx.x] = t;
  }
}

__global__ __launch_bounds__(64) void km_scan2_kernel(KmArgs a) {
  const int p = blockIdx.x;
  if (!km_active(a, p)) return;
  const Problem q = problem(a, p);
  const int64_t E = (int64_t)q.C * q.tiles;
  const int nch = (int)((E + kKmChunk - 1) / kKmChunk);
  int32_t* cs = a.chunk_sums + (int64_t)p * a.chunks_max;
  if (threadIdx.x == 0) {
    int run = 0;
    for (int c = 0; c < nch; ++c) {
      const int t = cs[c];
      cs[c] = run;
      run += t;
    }
  }
}

__global__ __launch_bounds__(1024) void km_scan3_kernel(KmArgs a) {
  __shared__ int s_w[17];
  const int p = blockIdx.y;
  if (!km_active(a, p)) return;
  const Problem q = problem(a, p);
  const int64_t E = (int64_t)q.C * q.tiles;
  const int64_t x0 = (int64_t)blockIdx.x * kKmChunk;
  if (blockIdx.x == 0 && threadIdx.x == 0) a.offsets[q.off_base + q.C] = q.n;
  if (x0 >= E) return;
  int32_t* tab = a.table + (int64_t)p * a.Cm * a.tiles_max;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t b0 = x0 + (int64_t)tid * 16, b1 = min(E, b0 + 16);
  // the 16 entries' (tile, cluster), stepped from the first one's
  const int t0 = (int)(b0 % q.tiles), c0 = (int)(b0 / q.tiles);
  int64_t ix[16];
  int v[16];
  int loc = 0;
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const int te = t0 + e;  // e < 16: at most ceil(16 / tiles) wraps, folded below
    const int ce = c0 + te / q.tiles;
    ix[e] = (int64_t)(te % q.tiles) * q.C + ce;
    v[e] = b0 + e < b1 ? tab[ix[e]] : 0;
    loc += v[e];
  }
  int incl = wave_incl_scan(loc);  // DPP, no LDS
  if (lane == 63) s_w[wave] = incl;
  __syncthreads();
  if (tid == 0) {
    int run = a.chunk_sums[(int64_t)p * a.chunks_max + blockIdx.x];
    for (int w = 0; w < 16; ++w) {
      const int t = s_w[w];
      s_w[w] = run;
      run += t;
    }
  }
  __syncthreads();
  int run = s_w[wave] + incl - loc;
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const int64_t x = b0 + e;
    if (x < b1) {
      tab[ix[e]] = run;
      if (x % q.tiles == 0) a.offsets[q.off_base + x / q.tiles] = run;  // start of cluster x / tiles
      run += v[e];
    }
  }
}

// ---------------------------------------------------------------------------
// stable scatter: perm[row] = token.  grid (tiles_max, BG), 1024 threads
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(1024) void km_perm_kernel(KmArgs a) {
  const int p = blockIdx.y;
  if (!km_active(a, p)) return;
  const Problem q = problem(a, p);
  const int t = blockIdx.x;
  const int i0 = t * kKmTile;
  if (i0 >= q.n) return;
  const int32_t* tab = a.table + (int64_t)p * a.Cm * a.tiles_max;
  for (int x = threadIdx.x; x < min(kKmTile, q.n - i0); x += 1024) {
    const int i = i0 + x;
    const int c = a.assign[q.tok_base + i];
    const int row = tab[(int64_t)t * q.C + c] + a.local_rank[q.tok_base + i];
    a.perm[q.tok_base + min(max(row, 0), q.n - 1)] = i;
  }
}

// ---------------------------------------------------------------------------
// centroid = bf16(mean of members).  grid (ceil(Cm/4), BG), a wave per cluster
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void km_mean_kernel(KmArgs a) {
  const int p = blockIdx.y;
  if (!km_active(a, p)) return;
  const Problem q = problem(a, p);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, sl = lane & 15, grp = lane >> 4;
  const int j = blockIdx.x * 4 + wave;
  if (j >= q.C) return;
  const int o0 = a.offsets[q.off_base + j], o1 = a.offsets[q.off_base + j + 1];
  if (o1 <= o0) return;  // empty cluster keeps its centroid
  // lane-group grp sums rows grp, grp + 4, grp + 8, ... in that order; 16
  // rows per step, their token ids and then their key rows loaded together
  float s[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int r0 = o0; r0 < o1; r0 += 16) {
    int tok[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int r = r0 + grp + 4 * k;
      tok[k] = r < o1 ? a.perm[q.tok_base + r] : -1;
    }
    uint4 v[4];
#pragma unroll
    for (int k = 0; k < 4; ++k)
      v[k] = tok[k] >= 0 ? *reinterpret_cast<const uint4*>(a.K + (q.tok_base + tok[k]) * kHeadDim + sl * 8)
                         : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (tok[k] < 0) continue;
      const uint32_t w[4] = {v[k].x, v[k].y, v[k].z, v[k].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        s[2 * e] += bf16lo(w[e]);
        s[2 * e + 1] += bf16hi(w[e]);
      }
    }
  }
  const float inv = 1.f / (float)(o1 - o0);
  float cn = 0.f;
  uint32_t out[4];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    float v = s[e];
    v += __shfl_xor(v, 16, 64);
    v += __shfl_xor(v, 32, 64);
    const uint16_t hb = f32_to_bf16_rne(v * inv);
    const float r = __uint_as_float((uint32_t)hb << 16);
    cn = fmaf(r, r, cn);
    if (e & 1) out[e >> 1] |= (uint32_t)hb << 16;
    else out[e >> 1] = hb;
  }
  cn = sum16(cn);
  if (grp == 0) *reinterpret_cast<uint4*>(a.centroids + (q.cl_base + j) * kHeadDim + sl * 8) =
      make_uint4(out[0], out[1], out[2], out[3]);
  if (lane == 0) a.cnorm[q.cl_base + j] = cn;
}

// ---------------------------------------------------------------------------
// K_sorted[row] = K[perm[row]] (and V).  grid (ceil(nmax/16), BG), 256 threads
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void km_permute_kv_kernel(KmArgs a) {
  const int p = blockIdx.y;
  const Problem q = problem(a, p);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, sl = lane & 15, grp = lane >> 4;
  const int r = blockIdx.x * 16 + wave * 4 + grp;
  if (r >= q.n) return;
  const int tok = min(max(a.perm[q.tok_base + r], 0), q.n - 1);
  const int64_t src = (q.tok_base + tok) * kHeadDim + sl * 8, dst = (q.tok_base + r) * kHeadDim + sl * 8;
  if (a.K_sorted) *reinterpret_cast<uint4*>(a.K_sorted + dst) = load_stream16(a.K + src);
  if (a.V_sorted) *reinterpret_cast<uint4*>(a.V_sorted + dst) = load_stream16(a.V + src);
}

// ---------------------------------------------------------------------------
// host driver
// ---------------------------------------------------------------------------
namespace {

struct KmLayout {
  int tiles_max, chunks_max;
  int64_t off_cnorm, off_rank, off_table, off_chunks, off_changed, off_done, bytes;
};

KmLayout km_layout(int B, int Hkv, int64_t total, int64_t Ct, int Cm, int64_t nmax) {
  KmLayout L;
  const int64_t BG = (int64_t)B * Hkv;
  L.tiles_max = (int)std::max<int64_t>(1, (nmax + kKmTile - 1) / kKmTile);
  L.chunks_max = (int)std::max<int64_t>(1, ((int64_t)Cm * L.tiles_max + kKmChunk - 1) / kKmChunk);
  int64_t cur = 0;
  auto take = [&](int64_t bytes) {
    const int64_t o = cur;
    cur = (cur + bytes + 255) / 256 * 256;
    return o;
  };
  L.off_cnorm = take((int64_t)Hkv * Ct * 4);
  L.off_rank = take((int64_t)Hkv * total * 4);
  L.off_table = take(BG * Cm * (int64_t)L.tiles_max * 4);
  L.off_chunks = take(BG * L.chunks_max * 4);
  L.off_changed = take((int64_t)(kKmMaxIters + 1) * BG * 4);
  L.off_done = take(BG * 4);
  L.bytes = cur;
  return L;
}

}  // namespace

size_t kmeans_workspace_bytes(int B, int Hkv, int64_t total, int64_t Ct, int Cm, int64_t nmax) {
  return (size_t)km_layout(B, Hkv, total, Ct, Cm, nmax).bytes;
}

hipError_t run_kmeans(const uint16_t* K, const uint16_t* V, const int64_t* kv_indptr, const int64_t* seq_len,
                      const int64_t* cl_indptr, int B, int Hkv, int64_t total, int64_t nmax,
                      int64_t Ct, int Cm, const int32_t* init_idx, int max_iters,
                      const uint16_t* prev_centroids, const int64_t* prev_cl_indptr, uint16_t* centroids, int32_t* assign, int32_t* offsets, int32_t* perm,
                      uint16_t* K_sorted, uint16_t* V_sorted, void* workspace, hipStream_t st) {
  if (max_iters > kKmMaxIters) return hipErrorInvalidValue;
  const KmLayout L = km_layout(B, Hkv, total, Ct, Cm, nmax);
  char* ws = static_cast<char*>(workspace);
  KmArgs a;
  a.K = K;
  a.V = V;
  a.kv_indptr = kv_indptr;
  a.seq_len = seq_len;
  a.cl_indptr = cl_indptr;
  a.B = B;
  a.Hkv = Hkv;
  a.Cm = Cm;
  a.tiles_max = L.tiles_max;
  a.chunks_max = L.chunks_max;
  a.iter = 0;
  a.max_iters = max_iters;
  a.total = total;
  a.Ct = Ct;
  a.init_idx = init_idx;
  a.prev_centroids = prev_centroids;
  a.prev_cl_indptr = prev_cl_indptr;
  a.centroids = centroids;
  a.cnorm = reinterpret_cast<float*>(ws + L.off_cnorm);
  a.assign = assign;
  a.offsets = offsets;
  a.perm = perm;
  a.local_rank = reinterpret_cast<int32_t*>(ws + L.off_rank);
  a.table = reinterpret_cast<int32_t*>(ws + L.off_table);
  a.chunk_sums = reinterpret_cast<int32_t*>(ws + L.off_chunks);
  a.changed = reinterpret_cast<int32_t*>(ws + L.off_changed);
  a.done = reinterpret_cast<int32_t*>(ws + L.off_done);
  a.K_sorted = K_sorted;
  a.V_sorted = V_sorted;
  const int BG = B * Hkv;
  const dim3 g_cl((Cm + 3) / 4, BG), g_tok((unsigned)((nmax + kAsgTok - 1) / kAsgTok), BG);
  const dim3 g_tile(L.tiles_max, BG), g_chunk(L.chunks_max, BG);
  hipLaunchKernelGGL(km_init_kernel, g_cl, dim3(256), 0, st, a);
  hipError_t e = hipGetLastError();
  for (int it = 1; it <= max_iters && e == hipSuccess; ++it) {
    a.iter = it;
    hipLaunchKernelGGL(km_assign_kernel, g_tok, dim3(256), 0, st, a);
    hipLaunchKernelGGL(km_hist_kernel, g_tile, dim3(1024), 0, st, a);
    hipLaunchKernelGGL(km_scan1_kernel, g_chunk, dim3(1024), 0, st, a);
    hipLaunchKernelGGL(km_scan2_kernel, dim3(BG), dim3(64), 0, st, a);
    hipLaunchKernelGGL(km_scan3_kernel, g_chunk, dim3(1024), 0, st, a);
    hipLaunchKernelGGL(km_perm_kernel, g_tile, dim3(1024), 0, st, a);
    hipLaunchKernelGGL(km_mean_kernel, g_cl, dim3(256), 0, st, a);
    e = hipGetLastError();
  }
  if (e == hipSuccess && (K_sorted || V_sorted)) {
    if (!V) a.V_sorted = nullptr;
    hipLaunchKernelGGL(km_permute_kv_kernel, dim3((unsigned)((nmax + 15) / 16), BG), dim3(256), 0, st, a);
    e = hipGetLastError();
  }
  return e;
}

}  // namespace tactic
