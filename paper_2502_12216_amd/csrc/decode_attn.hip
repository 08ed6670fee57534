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

__device__ __forceinline__ int64_t item_tokens(const AttnArgs& a, int bg) {
  return a.dense ? a.chunk_tokens : (int64_t)a.gmeta[bg * 4 + 3];
}

__device__ __forceinline__ int item_count(const AttnArgs& a, int bg) {
  if (a.dense) {
    const int b = bg / a.Hkv;
    const int64_t n = a.kv_indptr[b + 1] - a.kv_indptr[b];
    return (int)((n + a.chunk_tokens - 1) / a.chunk_tokens);
  }
  return a.gmeta[bg * 4 + 2];
}

template <int G, int TOK>
__global__ __launch_bounds__(256) void attn_splitk_kernel(AttnArgs a) {
  constexpr int kPart = G * (kHeadDim + 2);
  constexpr int kTileTok = 16 * TOK;  // tokens per workgroup tile
  __shared__ int s_prefix[kMaxGroups + 1];
  __shared__ int s_rows[kMaxChunkTokens];
  __shared__ int s_rupos[kMaxChunkTokens + 1];
  __shared__ int s_rstart[kMaxChunkTokens + 1];
  __shared__ float s_ml[16][2][G];
  __shared__ float s_M[G], s_L[G];
  __shared__ float s_red[4][G][kHeadDim];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, sl = lane & 15, grp = lane >> 4;
  const int gid = wave * 4 + grp;  // 16 lane-groups of 16 lanes
  const int BG = a.B * a.Hkv;

  for (int i = tid; i < BG; i += 256) s_prefix[i + 1] = item_count(a, i);
  if (tid == 0) s_prefix[0] = 0;
  __syncthreads();
  if (tid == 0) {
    for (int i = 0; i < BG; ++i) s_prefix[i + 1] += s_prefix[i];
  }
  __syncthreads();
  const int total_items = s_prefix[BG];

  for (int item = blockIdx.x; item < total_items; item += gridDim.x) {
    int lo = 0, hi = BG - 1;  // largest bg with s_prefix[bg] <= item
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (s_prefix[mid] <= item) lo = mid;
      else hi = mid - 1;
    }
    const int bg = lo, c = item - s_prefix[bg];
    const int b = bg / a.Hkv, g = bg % a.Hkv;
    const int64_t kvb = a.kv_indptr[b];
    const int nseq = (int)(a.kv_indptr[b + 1] - kvb);
    const int64_t T = item_tokens(a, bg);
    const int64_t U = a.dense ? (int64_t)nseq : (int64_t)a.gmeta[bg * 4 + 1];
    const int64_t p0 = (int64_t)c * T;
    const int cnt = (int)min(T, U - p0);

    uint32_t qw[G][4];
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const uint4 v = *reinterpret_cast<const uint4*>(a.q + ((int64_t)b * a.Hq + g * G + h) * kHeadDim + sl * 8);
      qw[h][0] = v.x; qw[h][1] = v.y; qw[h][2] = v.z; qw[h][3] = v.w;
    }

    // rows of this item (sequence-relative)
    if (a.dense) {
      for (int t = tid; t < cnt; t += 256) s_rows[t] = (int)(p0 + t);
    } else {
      const int R = a.gmeta[bg * 4 + 0];
      const int r0 = a.cfr[(int64_t)bg * a.max_chunks + c];
      const int nr = max(1, min(R - r0, (int)T));  // ranges that can touch this item
      const int32_t* rup = a.rupos + (int64_t)bg * (a.Cm + 1) + r0;
      const int32_t* rst = a.rstart + (int64_t)bg * a.Cm + r0;
      for (int i = tid; i <= nr; i += 256) {
        s_rupos[i] = rup[i];
        if (i < nr) s_rstart[i] = rst[i];
      }
      __syncthreads();
      for (int t = tid; t < cnt; t += 256) {
        const int pos = (int)(p0 + t);
        int l2 = 0, h2 = nr - 1;  // largest i with s_rupos[i] <= pos
        while (l2 < h2) {
          const int mid = (l2 + h2 + 1) >> 1;
          if (s_rupos[mid] <= pos) l2 = mid;
          else h2 = mid - 1;
        }
        const int row = s_rstart[l2] + (pos - s_rupos[l2]);
        s_rows[t] = min(max(row, 0), nseq - 1);  // in range unless the cluster meta is inconsistent
      }
    }
    __syncthreads();

    float m[G], l[G], acc[G][8];
#pragma unroll
    for (int h = 0; h < G; ++h) {
      m[h] = -INFINITY;
      l[h] = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[h][e] = 0.f;
    }

    const uint16_t* Kb = a.K + ((int64_t)g * a.total + kvb) * kHeadDim + sl * 8;
    const uint16_t* Vb = a.V + ((int64_t)g * a.total + kvb) * kHeadDim + sl * 8;
    const int ntile = (cnt + kTileTok - 1) / kTileTok;
    auto load_tile = [&](int tile, uint4* kk, uint4* vv) {
#pragma unroll
      for (int i = 0; i < TOK; ++i) {
        const int t = tile * kTileTok + gid * TOK + i;
        if (t < cnt) {
          const int64_t row = s_rows[t];
          kk[i] = load_stream16(Kb + row * kHeadDim);
          vv[i] = load_stream16(Vb + row * kHeadDim);
        } else {
          kk[i] = make_uint4(0, 0, 0, 0);
          vv[i] = make_uint4(0, 0, 0, 0);
        }
      }
    };
    // one tile of TOK tokens per lane-group: logits of the G heads, running max
    // (rescale only when some group's max grows), p * v
    auto consume = [&](const uint4* kx, const uint4* vx, int tile) {
      float s[TOK][G];
#pragma unroll
      for (int i = 0; i < TOK; ++i) {
        const bool valid = tile * kTileTok + gid * TOK + i < cnt;
#pragma unroll
        for (int h = 0; h < G; ++h) {
          float d = dot2_bf16(kx[i].x, qw[h][0], 0.f);
          d = dot2_bf16(kx[i].y, qw[h][1], d);
          d = dot2_bf16(kx[i].z, qw[h][2], d);
          d = dot2_bf16(kx[i].w, qw[h][3], d);
          s[i][h] = valid ? sum16(d) * kScaleLog2 : -INFINITY;
        }
      }
      float mn[G];
      bool grow = false;
#pragma unroll
      for (int h = 0; h < G; ++h) {
        float mt = s[0][h];
#pragma unroll
        for (int i = 1; i < TOK; ++i) mt = fmaxf(mt, s[i][h]);
        mn[h] = fmaxf(m[h], mt);
        grow |= mn[h] > m[h];
      }
      if (__any(grow)) {
#pragma unroll
        for (int h = 0; h < G; ++h) {
          const float corr = mn[h] > m[h] ? fast_exp2(m[h] - mn[h]) : 1.f;
          m[h] = mn[h];
          l[h] *= corr;
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[h][e] *= corr;
        }
      }
#pragma unroll
      for (int i = 0; i < TOK; ++i) {
        const float vf[8] = {bf16lo(vx[i].x), bf16hi(vx[i].x), bf16lo(vx[i].y), bf16hi(vx[i].y),
                             bf16lo(vx[i].z), bf16hi(vx[i].z), bf16lo(vx[i].w), bf16hi(vx[i].w)};
#pragma unroll
        for (int h = 0; h < G; ++h) {
          const float p = s[i][h] == -INFINITY ? 0.f : fast_exp2(s[i][h] - m[h]);
          l[h] += p;
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[h][e] = fmaf(p, vf[e], acc[h][e]);
        }
      }
    };
    uint4 kc[TOK], vc[TOK], kn[TOK], vn[TOK];
    load_tile(0, kc, vc);
#pragma unroll 1
    for (int tile = 0; tile < ntile; ++tile) {
      load_tile(tile + 1, kn, vn);  // zeros past the end
      consume(kc, vc, tile);
#pragma unroll
      for (int i = 0; i < TOK; ++i) {
        kc[i] = kn[i];
        vc[i] = vn[i];
      }
    }

    // ---- merge the 16 lane-group states: common max, rescale, sum
    if (sl == 0) {
#pragma unroll
      for (int h = 0; h < G; ++h) {
        s_ml[gid][0][h] = m[h];
        s_ml[gid][1][h] = l[h];
      }
    }
    __syncthreads();
    if (tid < G) {
      float mm = -INFINITY;
      for (int q2 = 0; q2 < 16; ++q2) mm = fmaxf(mm, s_ml[q2][0][tid]);
      float ll = 0.f;
      for (int q2 = 0; q2 < 16; ++q2) {
        const float mq = s_ml[q2][0][tid];
        ll += mq == -INFINITY ? 0.f : s_ml[q2][1][tid] * fast_exp2(mq - mm);
      }
      s_M[tid] = mm;
      s_L[tid] = ll;
    }
    __syncthreads();
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float sc = m[h] == -INFINITY ? 0.f : fast_exp2(m[h] - s_M[h]);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
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
        for (int e = 0; e < 8; ++e) s_red[wave][h][sl * 8 + e] = acc[h][e];
    }
    __syncthreads();
    float* part = a.partials + ((int64_t)bg * a.max_chunks + c) * kPart;
    for (int i = tid; i < G * kHeadDim; i += 256) {
      const int h = i / kHeadDim, d = i % kHeadDim;
      part[i] = s_red[0][h][d] + s_red[1][h][d] + s_red[2][h][d] + s_red[3][h][d];
    }
    if (tid < G) {
      part[G * kHeadDim + tid] = s_M[tid];
      part[G * kHeadDim + G + tid] = s_L[tid];
    }
    __syncthreads();
  }
}

// Combine the partials of every (b, g) in chunk order: out = sum_c acc_c 2^(m_c - M)
// / sum_c l_c 2^(m_c - M).  Groups without tokens get zeros.  grid (B*Hkv, G),
// 128 threads: one head per workgroup, one output dimension per thread.
template <int G>
__global__ __launch_bounds__(128) void combine_kernel(AttnArgs a) {
  constexpr int kPart = G * (kHeadDim + 2);
  constexpr int kMaxC = 1024;
  __shared__ float s_w[kMaxC];
  __shared__ float s_red[2];
  const int bg = blockIdx.x, h = blockIdx.y;
  const int b = bg / a.Hkv, g = bg % a.Hkv;
  const int tid = threadIdx.x;
  const int nchunks = item_count(a, bg);
  float* out = a.out + ((int64_t)b * a.Hq + g * G + h) * kHeadDim;
  if (nchunks == 0) {
    out[tid] = 0.f;
    return;
  }
  const float* pb = a.partials + (int64_t)bg * a.max_chunks * kPart;
  float M = -INFINITY;
  for (int c = tid; c < nchunks; c += 128) M = fmaxf(M, pb[(int64_t)c * kPart + G * kHeadDim + h]);
  for (int o = 32; o > 0; o >>= 1) M = fmaxf(M, __shfl_xor(M, o, 64));
  if ((tid & 63) == 0) s_red[tid >> 6] = M;
  __syncthreads();
  M = fmaxf(s_red[0], s_red[1]);
  __syncthreads();
  float den = 0.f;
  for (int c0 = 0; c0 < nchunks; c0 += kMaxC) {
    const int nc = min(kMaxC, nchunks - c0);
    for (int c = tid; c < nc; c += 128) {
      const float* pc = pb + (int64_t)(c0 + c) * kPart;
      const float w = fast_exp2(pc[G * kHeadDim + h] - M);
      s_w[c] = w;
      den = fmaf(pc[G * kHeadDim + G + h], w, den);
    }
    __syncthreads();
    float num = 0.f;
    const float* pa = pb + (int64_t)c0 * kPart + h * kHeadDim + tid;
#pragma unroll 8
    for (int c = 0; c < nc; ++c) num = fmaf(pa[(int64_t)c * kPart], s_w[c], num);
    if (c0 == 0) out[tid] = num;
    else out[tid] += num;
    __syncthreads();
  }
  for (int o = 32; o > 0; o >>= 1) den += __shfl_xor(den, o, 64);
  if ((tid & 63) == 0) s_red[tid >> 6] = den;
  __syncthreads();
  den = s_red[0] + s_red[1];
  out[tid] = out[tid] / den;
}

#ifndef TACTIC_ATTN_TOK
#define TACTIC_ATTN_TOK 2
#endif

hipError_t launch_attn(const AttnArgs& a, int G, int grid, hipStream_t st) {
  constexpr int TOK = TACTIC_ATTN_TOK;
  switch (G) {
    case 1: hipLaunchKernelGGL((attn_splitk_kernel<1, TOK>), dim3(grid), dim3(256), 0, st, a); break;
    case 2: hipLaunchKernelGGL((attn_splitk_kernel<2, TOK>), dim3(grid), dim3(256), 0, st, a); break;
    case 4: hipLaunchKernelGGL((attn_splitk_kernel<4, TOK>), dim3(grid), dim3(256), 0, st, a); break;
    case 8: hipLaunchKernelGGL((attn_splitk_kernel<8, TOK>), dim3(grid), dim3(256), 0, st, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_combine(const AttnArgs& a, int G, hipStream_t st) {
  const dim3 grid(a.B * a.Hkv, G);
  switch (G) {
    case 1: hipLaunchKernelGGL(combine_kernel<1>, grid, dim3(128), 0, st, a); break;
    case 2: hipLaunchKernelGGL(combine_kernel<2>, grid, dim3(128), 0, st, a); break;
    case 4: hipLaunchKernelGGL(combine_kernel<4>, grid, dim3(128), 0, st, a); break;
    case 8: hipLaunchKernelGGL(combine_kernel<8>, grid, dim3(128), 0, st, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace tactic
