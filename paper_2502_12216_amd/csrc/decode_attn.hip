// Gather split-K flash decoding over the selected tokens (Sec. 4.6, Eq. 3).
//
// Work items are (sequence b, KV head g, chunk c): chunk c covers tokens
// [c*T, (c+1)*T) of the group's union, stored as ranges of cluster-sorted rows
// (every cluster contributes a prefix of its rows).  A persistent grid walks
// the items.  Inside an item the 16 lane-groups of a workgroup (16 lanes x
// 16 B = one 256-byte K or V row) each stream their own share of the rows,
// four tokens per tile, with the next tile's rows already in flight, and keep
// their own online-softmax state for the G query heads of the group, so the
// tile loop needs no barrier.  The 16 states are merged through LDS into one
// partial (running max, running sum, unnormalised output) per item.  A second
// kernel combines a group's partials in chunk order, so results do not depend
// on scheduling.  Dense decode (Eq. 2) is the same pair of kernels with one
// range covering the whole sequence.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "common.hpp"
#include "kernels.hpp"
#include "plan.hpp"

namespace tactic {

// log2(e) / sqrt(128): logits are kept in base-2 units for exp2
constexpr float kScaleLog2 = 0.12751743074880046f;

// Tokens of selection group bg: its union (sparse) or its sequence (dense).
__device__ __forceinline__ int64_t group_tokens(const AttnArgs& a, int bg) {
  if (a.dense) {
    return seq_tokens(a.kv_indptr, a.seq_len, bg / a.NV);
  }
  return (int64_t)a.gmeta[bg * 4 + 1];
}

// The attention splits "units" evenly over its workgroups: a group's tokens
// plus kSegmentCost units standing for the fixed work of a group segment
// (query load, range lookup, merge, partial store; about the time of 96
// streamed tokens), so a workgroup that straddles groups gets fewer tokens.
constexpr int64_t kSegmentCost = 96;
constexpr int64_t kMinShare = 256;  // smallest split share (units) of a workgroup
__device__ __forceinline__ int64_t split_units(const AttnArgs& a, int bg) {
  const int64_t n = group_tokens(a, bg);
  return n > 0 ? n + kSegmentCost : 0;
}

__device__ __forceinline__ void load_words(const uint16_t* p, uint32_t* w) {
  const uint4 v = load_stream16(p);
  w[0] = v.x; w[1] = v.y; w[2] = v.z; w[3] = v.w;
}

// Sum over the 16 lanes of a DPP row of G per-lane values (one per query
// head), returning in every lane the total of head sl / (16 / G).  Each
// butterfly step pairs lanes across one lane bit with a mirror or quad DPP
// move; while more than one head is left, the lower lane of a pair keeps the
// lower half of the heads and receives its partner's copy of them, so the G
// sums take log2(16) steps of G/2, G/4, ... adds instead of 4 steps of G.
// Lanes that end on the same head hold bitwise identical sums (each step adds
// the same two operands in both partners).
template <int G>
__device__ __forceinline__ float reduce_heads(const float (&v)[G], int sl) {
  static_assert(G == 1 || G == 2 || G == 4 || G == 8, "heads per group: 1, 2, 4 or 8");
  if constexpr (G == 1) {
    return sum16(v[0]);
  } else {
    constexpr int G1 = G / 2;
    float a[G1];
    const bool up1 = sl & 8;  // row_mirror pairs lane i with 15 - i
#pragma unroll
    for (int i = 0; i < G1; ++i) {
      const float keep = up1 ? v[G1 + i] : v[i], send = up1 ? v[i] : v[G1 + i];
      a[i] = keep + dpp<0x140>(send);
    }
    if constexpr (G1 == 1) {
      float x = a[0];
      x += dpp<0x141>(x);
      x += dpp<0x4E>(x);
      x += dpp<0xB1>(x);
      return x;
    } else {
      constexpr int G2 = G1 / 2;
      float c[G2];
      const bool up2 = sl & 4;  // row_half_mirror pairs lane i with 7 - i in each half
#pragma unroll
      for (int i = 0; i < G2; ++i) {
        const float keep = up2 ? a[G2 + i] : a[i], send = up2 ? a[i] : a[G2 + i];
        c[i] = keep + dpp<0x141>(send);
      }
      if constexpr (G2 == 1) {
        float x = c[0];
        x += dpp<0x4E>(x);
        x += dpp<0xB1>(x);
        return x;
      } else {
        const bool up3 = sl & 2;  // quad_perm [2,3,0,1]
        const float keep = up3 ? c[1] : c[0], send = up3 ? c[0] : c[1];
        float x = keep + dpp<0x4E>(send);
        x += dpp<0xB1>(x);
        return x;
      }
    }
  }
}

// Value of head h (h < G, a constant after unrolling) from a lane that holds
// it: DPP row_newbcast of the first lane of head h's lanes (lane h * 16 / G of
// the row) to the whole row.
template <int G>
__device__ __forceinline__ float head_value(float x, int h) {
  constexpr int S = 16 / G;
  switch (h) {
    case 0: return G == 1 ? x : dpp<0x150>(x);
    case 1: return dpp<0x150 + 1 * S>(x);
    case 2: return dpp<0x150 + (2 * S & 15)>(x);
    case 3: return dpp<0x150 + (3 * S & 15)>(x);
    case 4: return dpp<0x150 + (4 * S & 15)>(x);
    case 5: return dpp<0x150 + (5 * S & 15)>(x);
    case 6: return dpp<0x150 + (6 * S & 15)>(x);
    default: return dpp<0x150 + (7 * S & 15)>(x);
  }
}

// 16 lanes share one 256-byte row (16 B per lane); a lane-group streams TOK
// rows per tile.
#ifndef TACTIC_ATTN_TOK
#define TACTIC_ATTN_TOK 2
#endif
#ifndef TACTIC_ATTN_DEPTH
#define TACTIC_ATTN_DEPTH 2  // tiles in flight while one is consumed
#endif
#ifndef TACTIC_ATTN_WPE
#define TACTIC_ATTN_WPE 3  // resident waves per SIMD the register budget must allow
#endif

template <int G, int TOK, bool kPaged>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(G >= 8 ? 2 : TACTIC_ATTN_WPE)))
void attn_splitk_kernel(AttnArgs a) {
  constexpr int LPR = 16;                 // lanes per 256-byte row
  constexpr int kPart = G * (kHeadDim + 2);
  constexpr int EPL = kHeadDim / LPR;     // bf16 elements per lane
  constexpr int W = EPL / 2;              // 32-bit words per lane
  constexpr int GPW = kWave / LPR;        // lane-groups per wave
  constexpr int NG = 4 * GPW;             // lane-groups per workgroup
  constexpr int kTileTok = NG * TOK;      // tokens per workgroup tile
  extern __shared__ int64_t s_prefix[];  // [B * NV + 1] split units before each selection group
  // the row table of a sub-range is dead once the merge starts, so the
  // merge's partial sums reuse its storage
  union ItemShared {
    struct {
      int rows[kMaxChunkTokens];
      int rupos[kMaxChunkTokens + 1];
      int rstart[kMaxChunkTokens + 1];
    } r;
    // the merge: every lane-group's rescaled accumulators (G <= 4), else the
    // four waves' sums after an in-wave reduction
    float red[G <= 4 ? NG : 4][G][kHeadDim];
  };
  __shared__ __align__(16) ItemShared sh;  // 16-byte LDS accesses to the row table
  int* s_rows = sh.r.rows;
  int* s_rupos = sh.r.rupos;
  int* s_rstart = sh.r.rstart;
  auto s_red = sh.red;
  __shared__ float s_ml[NG][2][G];
  __shared__ float s_M[G], s_L[G];
  __shared__ int64_t s_wsum[4];
  __shared__ int s_wmax[4];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, sl = lane % LPR, grp = lane / LPR;
  const int gid = wave * GPW + grp;
  const int BG = a.B * a.NV;

  // exclusive prefix of the groups' split units (tokens plus kSegmentCost for
  // a non-empty group): every thread sums a contiguous run of groups, then a
  // wave scan and the four wave totals
  {
    const int per = (BG + 255) / 256, g0 = min(BG, tid * per), g1 = min(BG, g0 + per);
    // the first group's units are kept (up to 256 groups it is the thread's
    // only one), so the second pass does not load them again
    const int64_t u_first = g0 < g1 ? split_units(a, g0) : 0;
    int64_t loc = u_first;
    for (int bg = g0 + 1; bg < g1; ++bg) loc += split_units(a, bg);
    int64_t incl = wave_incl_scan(loc);  // DPP, no LDS
    if (lane == kWave - 1) s_wsum[wave] = incl;
    __syncthreads();
    int64_t run = incl - loc;
    for (int w = 0; w < wave; ++w) run += s_wsum[w];
    for (int bg = g0; bg < g1; ++bg) {
      s_prefix[bg] = run;
      run += bg == g0 ? u_first : split_units(a, bg);
    }
    if (tid == 255) s_prefix[BG] = run;
    __syncthreads();
  }
  const int64_t total = s_prefix[BG];
  // a small selection is not spread thinner than kMinShare units per
  // workgroup: below that the fixed work of a workgroup and the partials the
  // combine must merge cost more than the extra workgroups stream
  const int64_t share = max((total + gridDim.x - 1) / gridDim.x, kMinShare);
  if (blockIdx.x == 0) {  // for the combine: the split and the group offsets
    if (tid == 0) a.ameta[0] = share;
    for (int bg = tid; bg <= BG; bg += 256) a.ameta[1 + bg] = s_prefix[bg];
  }
  const int64_t t0 = (int64_t)blockIdx.x * share, t1 = min(total, t0 + share);
  if (t0 >= t1) return;
  int bg0 = 0, bgh = BG - 1;  // largest group with s_prefix <= t0 (it holds t0)
  while (bg0 < bgh) {
    const int mid = (bg0 + bgh + 1) >> 1;
    if (s_prefix[mid] <= t0) bg0 = mid;
    else bgh = mid - 1;
  }

  for (int bg = bg0; bg < BG && s_prefix[bg] < t1; ++bg) {
    // the group's tokens follow its kSegmentCost units of setup in the split
    const int64_t first = s_prefix[bg] + kSegmentCost;
    const int64_t seg_lo = max(t0, first) - first;
    const int64_t seg_hi = min(t1, s_prefix[bg + 1]) - first;
    if (seg_lo >= seg_hi) continue;  // no token of this group in the range
    const int b = bg / a.NV, jg = bg % a.NV, kvh = jg / a.kv_div;
    const int64_t kvb = a.kv_indptr[b];
    const int nseq = (int)seq_tokens(a.kv_indptr, a.seq_len, b);

    uint32_t qw[G][W];
#pragma unroll
    for (int h = 0; h < G; ++h)
      load_words(a.q + ((int64_t)b * a.Hq + jg * G + h) * kHeadDim + sl * EPL, qw[h]);

    // online-softmax state: the running max and sum of this lane's head hl
    // (identical in the 16 / G lanes of that head), the accumulators of every head
    const int hl = sl / (16 / G);
    float m = -INFINITY, l = 0.f, acc[G][EPL];
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[h][e] = 0.f;

    // contiguous: rows of this (sequence, KV head); paged: row indices into the page array
    const int64_t rbase = kPaged ? 0 : (int64_t)kvh * a.total + kvb;
    const uint16_t* Kb = a.K + rbase * kHeadDim + sl * EPL;
    const uint16_t* Vb = a.V + rbase * kHeadDim + sl * EPL;
    // clustered rows of the group (paged: rows from there on are their own tokens)
    const int n_c = (kPaged && !a.dense) ? a.head_meta[(int64_t)(b * a.Hq + jg * G) * 16] : nseq;
    int cnt = 0;      // tokens of the current sub-range
    int64_t p0 = 0;   // its first position in the group's token list
    struct Tile {
      uint32_t k[TOK][W];
      uint32_t v[TOK][W];
    };
    auto load_tile = [&](int tile) -> Tile {
      Tile r;
#pragma unroll
      for (int i = 0; i < TOK; ++i) {
        const int t = tile * kTileTok + gid * TOK + i;
        if (t < cnt) {
          const int64_t row = (a.dense && !kPaged) ? p0 + t : (int64_t)s_rows[t];
          load_words(Kb + row * kHeadDim, r.k[i]);
          load_words(Vb + row * kHeadDim, r.v[i]);
        } else {
#pragma unroll
          for (int w = 0; w < W; ++w) r.k[i][w] = r.v[i][w] = 0u;
        }
      }
      return r;
    };
    // one tile of TOK tokens per lane-group: logits of the G heads (each lane
    // ends with its own head's), running max (rescale only when some group's
    // max grows), p * v with each head's weight broadcast from its lanes
    auto consume = [&](const Tile& x, int tile) {
      float s[TOK];
#pragma unroll
      for (int i = 0; i < TOK; ++i) {
        const bool valid = tile * kTileTok + gid * TOK + i < cnt;
        float d[G];
#pragma unroll
        for (int h = 0; h < G; ++h) {
          d[h] = 0.f;
#pragma unroll
          for (int w = 0; w < W; ++w) d[h] = dot2_bf16(x.k[i][w], qw[h][w], d[h]);
        }
        const float r = reduce_heads<G>(d, sl);
        s[i] = valid ? r * kScaleLog2 : -INFINITY;
      }
      float mn = m;
#pragma unroll
      for (int i = 0; i < TOK; ++i) mn = fmaxf(mn, s[i]);
      if (__any(mn > m)) {
        const float corr = mn > m ? fast_exp2(m - mn) : 1.f;
        m = mn;
        l *= corr;
#pragma unroll
        for (int h = 0; h < G; ++h) {
          const float c = head_value<G>(corr, h);
#pragma unroll
          for (int e = 0; e < EPL; ++e) acc[h][e] *= c;
        }
      }
#pragma unroll
      for (int i = 0; i < TOK; ++i) {
        const float p = s[i] == -INFINITY ? 0.f : fast_exp2(s[i] - m);
        l += p;
        float vf[EPL];
#pragma unroll
        for (int w = 0; w < W; ++w) {
          vf[2 * w] = bf16lo(x.v[i][w]);
          vf[2 * w + 1] = bf16hi(x.v[i][w]);
        }
#pragma unroll
        for (int h = 0; h < G; ++h) {
          const float ph = head_value<G>(p, h);
#pragma unroll
          for (int e = 0; e < EPL; ++e) acc[h][e] = fmaf(ph, vf[e], acc[h][e]);
        }
      }
    };
    // the group's part of this workgroup's range, in sub-ranges whose row
    // table fits LDS (dense rows are positions: one sub-range)
    for (int64_t p = seg_lo; p < seg_hi; p += cnt) {
      p0 = p;
      if (a.dense && !kPaged) {
        cnt = (int)(seg_hi - p);
      } else if (a.dense) {
        // paged dense: the row table holds each position's page row
        cnt = (int)min(seg_hi - p, (int64_t)kMaxChunkTokens);
        // a thread's positions (stride 256; cnt >= 1) looked up as one batch
        // of loads, those past the sub-range at its last position
        constexpr int kPer = kMaxChunkTokens / 256;
        int rr[kPer];
        int64_t pr[kPer];
#pragma unroll
        for (int e = 0; e < kPer; ++e) rr[e] = (int)(p + min(tid + e * 256, cnt - 1));
        paged_rows(a.pk, a.Hkv, a.total, kvb, b, kvh, rr, 0, pr);
#pragma unroll
        for (int e = 0; e < kPer; ++e)
          if (tid + e * 256 < cnt) s_rows[tid + e * 256] = (int)pr[e];
        __syncthreads();
      } else {
        const int64_t c = p / kCfrTokens, in = p - c * kCfrTokens;
        cnt = (int)min(seg_hi - p, (int64_t)kMaxChunkTokens - in);
        // ranges that can touch [p, p + cnt): from the one holding position
        // c * kCfrTokens to the one holding the first position of the chunk
        // after the sub-range's last (or the group's last range), at most
        // in + cnt of them (every range after r0 starts at its own position)
        const int R = a.gmeta[bg * 4 + 0], nchunk = a.gmeta[bg * 4 + 2];
        const int64_t c_end = (p + cnt - 1) / kCfrTokens + 1;
        const int32_t* cf = a.cfr + (int64_t)bg * a.max_chunks;
        const int r0 = cf[c];
        // loaded unconditionally (clamped into the group's chunk index) so that
        // it travels with the group's metadata instead of after it
        const int cf_end = cf[min(c_end, a.max_chunks - 1)];
        const int r_hi = c_end < min((int64_t)nchunk, a.max_chunks) ? cf_end : R - 1;
        const int nr = max(1, min(min(R - r0, r_hi - r0 + 1), (int)(in + cnt)));
        const int32_t* rup = a.rupos + (int64_t)bg * (a.Cm + 2) + r0;
        const int32_t* rst = a.rstart + (int64_t)bg * (a.Cm + 2) + r0;
        constexpr int kRun = kMaxChunkTokens / 256;  // positions per thread
        const int t_lo = tid * kRun;
        // the row table starts as range markers: all zero, then each range's
        // index at its first position (the ranges starting at or before p
        // all mark position 0, and the largest index wins)
        *reinterpret_cast<int4*>(s_rows + t_lo) = make_int4(0, 0, 0, 0);
        *reinterpret_cast<int4*>(s_rows + t_lo + 4) = make_int4(0, 0, 0, 0);
        // loads and stores unconditional so that the two loads are in flight
        // together: entry nr of the starts (a copy of range nr - 1's) is
        // never read, since every marker is a range index below nr
#pragma unroll 4
        for (int i = tid; i <= nr; i += 256) {
          const int up = rup[i], st = rst[min(i, nr - 1)];
          s_rupos[i] = up;
          s_rstart[i] = st;
        }
        __syncthreads();
        for (int i = tid; i < nr; i += 256) {
          const int64_t q = (int64_t)s_rupos[i] - p;
          if (q < cnt) atomicMax(&s_rows[max(q, (int64_t)0)], i);
        }
        __syncthreads();
        // each position's range is the largest marker at or before it: a
        // running max over the thread's positions, a DPP max-scan over the
        // wave, the maxima of the earlier waves
        int mk[kRun];
        {
          const int4 x = *reinterpret_cast<const int4*>(s_rows + t_lo);
          const int4 y = *reinterpret_cast<const int4*>(s_rows + t_lo + 4);
          mk[0] = x.x; mk[1] = x.y; mk[2] = x.z; mk[3] = x.w;
          mk[4] = y.x; mk[5] = y.y; mk[6] = y.z; mk[7] = y.w;
        }
#pragma unroll
        for (int e = 1; e < kRun; ++e) mk[e] = max(mk[e], mk[e - 1]);
        const int wincl = wave_incl_max(mk[kRun - 1]);
        if (lane == kWave - 1) s_wmax[wave] = wincl;
        __syncthreads();
        int run = dpp_zero<0x138, 0xF>(wincl);  // wave_shr:1, the lanes before this one
        for (int w = 0; w < wave; ++w) run = max(run, s_wmax[w]);
        int rw[kRun];
#pragma unroll
        for (int e = 0; e < kRun; ++e) {
          const int idx = max(mk[e], run);
          const int pos = (int)(p + t_lo + e);
          rw[e] = min(max(s_rstart[idx] + (pos - s_rupos[idx]), 0), nseq - 1);  // clamp: bad meta only
        }
        if constexpr (kPaged) {  // the group holds tokens here, so nseq >= 1 and every row is valid
          int64_t pr[kRun];
          paged_rows(a.pk, a.Hkv, a.total, kvb, b, kvh, rw, n_c, pr);
#pragma unroll
          for (int e = 0; e < kRun; ++e) rw[e] = (int)pr[e];
        }
        *reinterpret_cast<int4*>(s_rows + t_lo) = make_int4(rw[0], rw[1], rw[2], rw[3]);
        *reinterpret_cast<int4*>(s_rows + t_lo + 4) = make_int4(rw[4], rw[5], rw[6], rw[7]);
        __syncthreads();
      }
      const int ntile = (cnt + kTileTok - 1) / kTileTok;
#if TACTIC_ATTN_DEPTH == 2
      // two tiles in flight while one is consumed (rotation unrolled by three)
      Tile t0 = load_tile(0), t1 = load_tile(1);
#pragma unroll 1
      for (int tile = 0; tile < ntile; tile += 3) {
        Tile t2 = load_tile(tile + 2);
        consume(t0, tile);
        if (tile + 1 >= ntile) break;
        t0 = load_tile(tile + 3);
        consume(t1, tile + 1);
        if (tile + 2 >= ntile) break;
        t1 = load_tile(tile + 4);
        consume(t2, tile + 2);
      }
#elif TACTIC_ATTN_DEPTH == 3
      Tile t0 = load_tile(0), t1 = load_tile(1), t2 = load_tile(2);
#pragma unroll 1
      for (int tile = 0; tile < ntile; tile += 4) {
        Tile t3 = load_tile(tile + 3);
        consume(t0, tile);
        if (tile + 1 >= ntile) break;
        t0 = load_tile(tile + 4);
        consume(t1, tile + 1);
        if (tile + 2 >= ntile) break;
        t1 = load_tile(tile + 5);
        consume(t2, tile + 2);
        if (tile + 3 >= ntile) break;
        t2 = load_tile(tile + 6);
        consume(t3, tile + 3);
      }
#else
      Tile cur = load_tile(0);
#pragma unroll 1
      for (int tile = 0; tile < ntile; ++tile) {
        const Tile nxt = load_tile(tile + 1);  // zeros past the end
        consume(cur, tile);
        cur = nxt;
      }
#endif
      if (!a.dense || kPaged) __syncthreads();  // the next sub-range rewrites the row table
    }

    // ---- merge the lane-group states: common max, rescale, sum
    if (sl == hl * (16 / G)) {
      s_ml[gid][0][hl] = m;
      s_ml[gid][1][hl] = l;
    }
    __syncthreads();
    if (tid < G) {
      float mm = -INFINITY;
      for (int q2 = 0; q2 < NG; ++q2) mm = fmaxf(mm, s_ml[q2][0][tid]);
      float ll = 0.f;
      for (int q2 = 0; q2 < NG; ++q2) {
        const float mq = s_ml[q2][0][tid];
        ll += mq == -INFINITY ? 0.f : s_ml[q2][1][tid] * fast_exp2(mq - mm);
      }
      s_M[tid] = mm;
      s_L[tid] = ll;
    }
    __syncthreads();
    const float sc_own = m == -INFINITY ? 0.f : fast_exp2(m - s_M[hl]);
    float* part = a.partials + ((int64_t)bg + blockIdx.x) * kPart;  // slot bg + w is unique
    if constexpr (G <= 4) {
      // every lane-group's rescaled accumulators to LDS, then 4 consecutive
      // outputs per thread summed over the NG lane-groups
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float sc = head_value<G>(sc_own, h);
#pragma unroll
        for (int e = 0; e < EPL; e += 4)
          *reinterpret_cast<float4*>(&s_red[gid][h][sl * EPL + e]) =
              make_float4(acc[h][e] * sc, acc[h][e + 1] * sc, acc[h][e + 2] * sc, acc[h][e + 3] * sc);
      }
      __syncthreads();
      if (tid * 4 < G * kHeadDim) {
        const int h = tid * 4 / kHeadDim, d = tid * 4 % kHeadDim;
        float4 sum = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int q2 = 0; q2 < NG; ++q2) {
          const float4 v = *reinterpret_cast<const float4*>(&s_red[q2][h][d]);
          sum.x += v.x;
          sum.y += v.y;
          sum.z += v.z;
          sum.w += v.w;
        }
        *reinterpret_cast<float4*>(part + tid * 4) = sum;
      }
    } else {
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float sc = head_value<G>(sc_own, h);
#pragma unroll
        for (int e = 0; e < EPL; ++e) {
          float v = acc[h][e] * sc;
          v += __shfl_xor(v, 16, 64);
          v += __shfl_xor(v, 32, 64);
          acc[h][e] = v;
        }
      }
      if (grp == 0) {
#pragma unroll
        for (int h = 0; h < G; ++h)
#pragma unroll
          for (int e = 0; e < EPL; ++e) s_red[wave][h][sl * EPL + e] = acc[h][e];
      }
      __syncthreads();
      for (int i = tid; i < G * kHeadDim; i += 256) {
        const int h = i / kHeadDim, d = i % kHeadDim;
        part[i] = s_red[0][h][d] + s_red[1][h][d] + s_red[2][h][d] + s_red[3][h][d];
      }
    }
    if (tid < G) {
      part[G * kHeadDim + tid] = s_M[tid];
      part[G * kHeadDim + G + tid] = s_L[tid];
    }
    __syncthreads();
  }
}

// Combine the partials of every (b, g): out = sum_c acc_c 2^(m_c - M) /
// sum_c l_c 2^(m_c - M).  grid (B*NV, G), 512 threads: four slices of the
// partials (c = slice mod 4) x 128 output dimensions.  The partials'
// (maximum, sum) pairs go to LDS and a block reduction gives M; each
// partial's weight 2^(m_c - M) then replaces its maximum in LDS and a block
// reduction gives the denominator; each slice sums weight x accumulator over
// its partials in ascending order (the first eight loaded before the
// reductions, all loads independent of one another) and the slices add in
// order.  Every sum has a fixed order, so results do not depend on
// scheduling.  Groups without tokens get zeros.
template <int G>
__global__ __launch_bounds__(512) void combine_kernel(AttnArgs a) {
  constexpr int kPart = G * (kHeadDim + 2);
  __shared__ float s_w[kMaxAttnGrid];     // running maximum, then weight, of each partial
  __shared__ float s_l[kMaxAttnGrid];     // running sum of each partial
  __shared__ float s_num[4][kHeadDim];
  __shared__ float s_red[8];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid >> 6;
  const int bg = blockIdx.x, h = blockIdx.y;
  const int b = bg / a.NV, jg = bg % a.NV;
  const int d = tid & (kHeadDim - 1), slice = tid >> 7;
  float* out = a.out + ((int64_t)b * a.Hq + jg * G + h) * kHeadDim;
  // workgroups w0..w1 covered this group's tokens; their partials sit in slots bg + w
  const int64_t share = a.ameta[0], P0 = a.ameta[1 + bg], P1 = a.ameta[2 + bg];
  if (P1 <= P0 || share <= 0) {
    if (slice == 0) out[d] = 0.f;
    return;
  }
  const int64_t w0 = (P0 + kSegmentCost) / share, w1 = (P1 - 1) / share;
  const int np = (int)min(w1 - w0 + 1, (int64_t)kMaxAttnGrid);
  const float* pb = a.partials + (bg + w0) * kPart;
  const float* pd = pb + h * kHeadDim + d;  // this thread's output dimension of partial 0
  constexpr int kPre = 8;                   // numerator loads issued before the reductions
  float pre[kPre];
#pragma unroll
  for (int i = 0; i < kPre; ++i) {
    const int c = slice + 4 * i;
    pre[i] = c < np ? pd[(int64_t)c * kPart] : 0.f;
  }
  // 1. every partial's (maximum, sum) to LDS, and the common maximum
  float mx = -INFINITY;
  for (int c = tid; c < np; c += 512) {
    const float mc = pb[(int64_t)c * kPart + G * kHeadDim + h];
    s_w[c] = mc;
    s_l[c] = pb[(int64_t)c * kPart + G * kHeadDim + G + h];
    mx = fmaxf(mx, mc);
  }
  mx = wave_allmax_f(mx);
  if (lane == 0) s_red[wave] = mx;
  __syncthreads();
  float M = s_red[0];
#pragma unroll
  for (int w = 1; w < 8; ++w) M = fmaxf(M, s_red[w]);
  __syncthreads();  // s_red is reused below
  // 2. weights and denominator
  float den = 0.f;
  for (int c = tid; c < np; c += 512) {  // the entries this thread wrote
    const float mc = s_w[c];
    const float wc = mc == -INFINITY ? 0.f : fast_exp2(mc - M);
    s_w[c] = wc;
    den = fmaf(s_l[c], wc, den);
  }
  den = wave_allsum_f(den);
  if (lane == 0) s_red[wave] = den;
  __syncthreads();
  // 3. numerator: slice s sums partials s, s + 4, ... for dimension d
  float num = 0.f;
#pragma unroll
  for (int i = 0; i < kPre; ++i) {
    const int c = slice + 4 * i;
    if (c < np) num = fmaf(s_w[c], pre[i], num);
  }
#pragma unroll 8
  for (int c = slice + 4 * kPre; c < np; c += 4) num = fmaf(s_w[c], pd[(int64_t)c * kPart], num);
  s_num[slice][d] = num;
  __syncthreads();
  if (slice == 0) {
    float dd = 0.f;
#pragma unroll
    for (int w = 0; w < 8; ++w) dd += s_red[w];
    out[d] = (((s_num[0][d] + s_num[1][d]) + s_num[2][d]) + s_num[3][d]) / dd;
  }
}

static size_t attn_dyn_lds(const AttnArgs& a) { return ((size_t)a.B * a.NV + 1) * sizeof(int64_t); }

template <bool kPaged>
static hipError_t launch_attn_t(const AttnArgs& a, int G, int grid, hipStream_t st) {
  constexpr int TOK = TACTIC_ATTN_TOK;
  const size_t lds = attn_dyn_lds(a);
  switch (G) {
    case 1: hipLaunchKernelGGL((attn_splitk_kernel<1, TOK, kPaged>), dim3(grid), dim3(256), lds, st, a); break;
    case 2: hipLaunchKernelGGL((attn_splitk_kernel<2, TOK, kPaged>), dim3(grid), dim3(256), lds, st, a); break;
    case 4: hipLaunchKernelGGL((attn_splitk_kernel<4, TOK, kPaged>), dim3(grid), dim3(256), lds, st, a); break;
    case 8: hipLaunchKernelGGL((attn_splitk_kernel<8, TOK, kPaged>), dim3(grid), dim3(256), lds, st, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_attn(const AttnArgs& a, int G, int grid, bool paged, hipStream_t st) {
  return paged ? launch_attn_t<true>(a, G, grid, st) : launch_attn_t<false>(a, G, grid, st);
}

// Workgroups of the attention kernel that fit on the device at once: the
// persistent grid is sized to exactly this, so every workgroup streams its
// share of the tokens from the start.
template <bool kPaged>
static hipError_t resident_t(int G, size_t lds, int* per) {
  constexpr int TOK = TACTIC_ATTN_TOK;
  switch (G) {
    case 1: return hipOccupancyMaxActiveBlocksPerMultiprocessor(per, attn_splitk_kernel<1, TOK, kPaged>, 256, lds);
    case 2: return hipOccupancyMaxActiveBlocksPerMultiprocessor(per, attn_splitk_kernel<2, TOK, kPaged>, 256, lds);
    case 4: return hipOccupancyMaxActiveBlocksPerMultiprocessor(per, attn_splitk_kernel<4, TOK, kPaged>, 256, lds);
    case 8: return hipOccupancyMaxActiveBlocksPerMultiprocessor(per, attn_splitk_kernel<8, TOK, kPaged>, 256, lds);
    default: return hipErrorInvalidValue;
  }
}

hipError_t attn_resident_grid(int G, int n_groups, bool paged, int* grid) {
  int dev = 0, cus = 0, per = 0;
  const size_t lds = ((size_t)n_groups + 1) * sizeof(int64_t);
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  e = paged ? resident_t<true>(G, lds, &per) : resident_t<false>(G, lds, &per);
  *grid = (per > 0 ? per : 1) * (cus > 0 ? cus : 1);
  return e;
}

hipError_t launch_combine(const AttnArgs& a, int G, hipStream_t st) {
  const dim3 grid(a.B * a.NV, G);
  switch (G) {
    case 1: hipLaunchKernelGGL(combine_kernel<1>, grid, dim3(512), 0, st, a); break;
    case 2: hipLaunchKernelGGL(combine_kernel<2>, grid, dim3(512), 0, st, a); break;
    case 4: hipLaunchKernelGGL(combine_kernel<4>, grid, dim3(512), 0, st, a); break;
    case 8: hipLaunchKernelGGL(combine_kernel<8>, grid, dim3(512), 0, st, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace tactic
