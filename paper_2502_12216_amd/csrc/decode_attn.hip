// Gather split-K flash decoding over the selected tokens (Sec. 4.6, Eq. 3).
//
// Work items are (sequence b, KV head g, chunk c): chunk c covers tokens
// [c*T, (c+1)*T) of the group's union, laid out as ranges of cluster-sorted
// rows (every cluster contributes a prefix of its rows).  A persistent grid
// walks the items; each item streams its K/V rows in tiles of 64 tokens with
// an online softmax for the G query heads of the group and writes a partial
// (running max, running sum, unnormalised output).  The workgroup finishing a
// group's last item combines the group's partials into the output, in chunk
// order, so the result does not depend on scheduling.  Dense decode (Eq. 2)
// is the same kernel with one range covering the whole sequence.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "common.hpp"
#include "kernels.hpp"
#include "plan.hpp"

namespace tactic {

// log2(e) / sqrt(128): logits are kept in base-2 units for exp2
constexpr float kScaleLog2 = 0.12751743074880046f;

template <int G>
__global__ __launch_bounds__(256) void attn_splitk_kernel(AttnArgs a) {
  constexpr int kPart = G * (kHeadDim + 2);
  __shared__ int s_prefix[kMaxGroups + 1];
  __shared__ int s_rows[kMaxChunkTokens];
  __shared__ int s_rupos[kMaxChunkTokens + 1];
  __shared__ int s_rstart[kMaxChunkTokens + 1];
  __shared__ float s_logit[G][kTile];
  __shared__ float s_p[kTile][G];
  __shared__ float s_m[G], s_l[G], s_corr[G];
  __shared__ float s_red[4][G][kHeadDim];
  __shared__ int s_flag;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, sl = lane & 15, grp = lane >> 4;
  const int gid = wave * 4 + grp;  // 16 groups of 16 lanes
  const int BG = a.B * a.Hkv;
  const int64_t T = a.chunk_tokens;

  // work-item prefix over (b, g)
  for (int i = tid; i < BG; i += 256) {
    int chunks;
    if (a.dense) {
      const int b = i / a.Hkv;
      const int64_t n = a.kv_indptr[b + 1] - a.kv_indptr[b];
      chunks = (int)((n + T - 1) / T);
    } else {
      chunks = a.gmeta[i * 4 + 2];
    }
    s_prefix[i + 1] = chunks;
  }
  if (tid == 0) s_prefix[0] = 0;
  __syncthreads();
  if (tid == 0) {
    for (int i = 0; i < BG; ++i) s_prefix[i + 1] += s_prefix[i];
  }
  __syncthreads();
  const int total_items = s_prefix[BG];

  // groups with nothing to attend to (empty sequences) get zeros
  if (blockIdx.x == 0) {
    for (int bg = 0; bg < BG; ++bg) {
      if (s_prefix[bg + 1] != s_prefix[bg]) continue;
      const int b = bg / a.Hkv, g = bg % a.Hkv;
      for (int i = tid; i < G * kHeadDim; i += 256)
        a.out[((int64_t)b * a.Hq + g * G) * kHeadDim + i] = 0.f;
    }
  }

  for (int item = blockIdx.x; item < total_items; item += gridDim.x) {
    int lo = 0, hi = BG - 1;  // largest bg with s_prefix[bg] <= item
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (s_prefix[mid] <= item) lo = mid;
      else hi = mid - 1;
    }
    const int bg = lo, c = item - s_prefix[bg];
    const int nchunks = s_prefix[bg + 1] - s_prefix[bg];
    const int b = bg / a.Hkv, g = bg % a.Hkv;
    const int64_t kvb = a.kv_indptr[b];
    const int nseq = (int)(a.kv_indptr[b + 1] - kvb);
    const int64_t U = a.dense ? (a.kv_indptr[b + 1] - kvb) : (int64_t)a.gmeta[bg * 4 + 1];
    const int64_t p0 = (int64_t)c * T;
    const int cnt = (int)min(T, U - p0);

    // rows of this chunk (sequence-relative)
    if (a.dense) {
      for (int t = tid; t < cnt; t += 256) s_rows[t] = (int)(p0 + t);
    } else {
      const int R = a.gmeta[bg * 4 + 0];
      const int r0 = a.cfr[(int64_t)bg * a.max_chunks + c];
      const int nr = max(1, min(R - r0, (int)T));  // ranges that can touch this chunk
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
    if (tid < G) {
      s_m[tid] = -INFINITY;
      s_l[tid] = 0.f;
    }

    uint32_t qw[G][4];
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const uint4 v = *reinterpret_cast<const uint4*>(a.q + ((int64_t)b * a.Hq + g * G + h) * kHeadDim + sl * 8);
      qw[h][0] = v.x; qw[h][1] = v.y; qw[h][2] = v.z; qw[h][3] = v.w;
    }
    float acc[G][8];
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[h][e] = 0.f;
    __syncthreads();

    const uint16_t* Kb = a.K + ((int64_t)g * a.total + kvb) * kHeadDim + sl * 8;
    const uint16_t* Vb = a.V + ((int64_t)g * a.total + kvb) * kHeadDim + sl * 8;
    for (int tb = 0; tb < cnt; tb += kTile) {
      // ---- phase 1: logits of this group's 4 tokens, V prefetch
      uint4 vv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = tb + gid * 4 + i;
        uint4 kv = make_uint4(0, 0, 0, 0);
        vv[i] = make_uint4(0, 0, 0, 0);
        if (t < cnt) {
          const int64_t row = s_rows[t];
          kv = *reinterpret_cast<const uint4*>(Kb + row * kHeadDim);
          vv[i] = *reinterpret_cast<const uint4*>(Vb + row * kHeadDim);
        }
#pragma unroll
        for (int h = 0; h < G; ++h) {
          float s = dot2_bf16(kv.x, qw[h][0], 0.f);
          s = dot2_bf16(kv.y, qw[h][1], s);
          s = dot2_bf16(kv.z, qw[h][2], s);
          s = dot2_bf16(kv.w, qw[h][3], s);
          s = sum16(s);
          if (sl == h) s_logit[h][gid * 4 + i] = s;
        }
      }
      __syncthreads();
      // ---- phase 2: tile max / probabilities / running sums per head
      for (int h = wave; h < G; h += 4) {
        const bool valid = tb + lane < cnt;
        const float s = valid ? s_logit[h][lane] * kScaleLog2 : -INFINITY;
        const float mt = wave_max(s);
        const float m_old = s_m[h];
        const float m_new = fmaxf(m_old, mt);
        const float p = valid ? exp2f(s - m_new) : 0.f;
        const float lt = wave_sum(p);
        const float corr = exp2f(m_old - m_new);
        s_p[lane][h] = p;
        if (lane == 0) {
          s_m[h] = m_new;
          s_l[h] = s_l[h] * corr + lt;
          s_corr[h] = corr;
        }
      }
      __syncthreads();
      // ---- phase 3: rescale and accumulate p * v
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float cr = s_corr[h];
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[h][e] *= cr;
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = gid * 4 + i;
        const float vf[8] = {bf16lo(vv[i].x), bf16hi(vv[i].x), bf16lo(vv[i].y), bf16hi(vv[i].y),
                             bf16lo(vv[i].z), bf16hi(vv[i].z), bf16lo(vv[i].w), bf16hi(vv[i].w)};
#pragma unroll
        for (int h = 0; h < G; ++h) {
          const float p = s_p[t][h];
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[h][e] = fmaf(p, vf[e], acc[h][e]);
        }
      }
      __syncthreads();
    }

    // ---- reduce the 16 groups: 4 groups of a wave by shuffles, 4 waves in LDS
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float v = acc[h][e];
        v += __shfl_xor(v, 16, 64);
        v += __shfl_xor(v, 32, 64);
        acc[h][e] = v;
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
      part[G * kHeadDim + tid] = s_m[tid];
      part[G * kHeadDim + G + tid] = s_l[tid];
    }

    // ---- the last item of the group combines all its partials
    if (arrive_last(a.done + bg, nchunks, &s_flag)) {
      const float* pb = a.partials + (int64_t)bg * a.max_chunks * kPart;
      for (int i = tid; i < G * kHeadDim; i += 256) {
        const int h = i / kHeadDim;
        float M = -INFINITY;
        for (int cc = 0; cc < nchunks; ++cc) M = fmaxf(M, pb[(int64_t)cc * kPart + G * kHeadDim + h]);
        float num = 0.f, den = 0.f;
        for (int cc = 0; cc < nchunks; ++cc) {
          const float* pc = pb + (int64_t)cc * kPart;
          const float w = exp2f(pc[G * kHeadDim + h] - M);
          num = fmaf(pc[i], w, num);
          den = fmaf(pc[G * kHeadDim + G + h], w, den);
        }
        a.out[((int64_t)b * a.Hq + g * G) * kHeadDim + i] = num / den;
      }
      if (tid == 0) __hip_atomic_store(a.done + bg, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
  }
}

hipError_t launch_attn(const AttnArgs& a, int G, int grid, hipStream_t st) {
  switch (G) {
    case 1: hipLaunchKernelGGL(attn_splitk_kernel<1>, dim3(grid), dim3(256), 0, st, a); break;
    case 2: hipLaunchKernelGGL(attn_splitk_kernel<2>, dim3(grid), dim3(256), 0, st, a); break;
    case 4: hipLaunchKernelGGL(attn_splitk_kernel<4>, dim3(grid), dim3(256), 0, st, a); break;
    case 8: hipLaunchKernelGGL(attn_splitk_kernel<8>, dim3(grid), dim3(256), 0, st, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace tactic
