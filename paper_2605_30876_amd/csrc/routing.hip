// Expert selection.
//
// Block routing (Sec. 4.2 aggregation; Alg. 1 with a coreset of size k):
// one workgroup per block sums the block's token probabilities in token order
// (the mean is the aggregate, so no separate normalisation is needed), picks
// the k best experts and the (k+1)-th for the gap, then renormalises every
// token's probabilities over the picked set.
// Token routing (the baseline): one wave per token does the same on its own
// probability row.
//
// Selection uses the total order (score desc, id asc), so an exact tie goes
// to the lower id.  Block routing (one workgroup per block): for E <=
// kRankMaxE each element's rank is counted directly (how many elements
// precede it), one pass with no serial rounds; above that, and for token
// routing (one wave per token), a top-k walks the order: round r picks the
// best element strictly after round r-1's pick.
#include <algorithm>

#include "dmoe_common.h"

namespace dmoe {
namespace {

struct Cand {
  float v;
  int i;
};

// (v, i) ranks before (w, j) in (score desc, id asc) order.
__device__ __forceinline__ bool ranks_before(float v, int i, float w, int j) {
  return v > w || (v == w && i < j);
}

__device__ __forceinline__ Cand wave_best(Cand c) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    float ov = __shfl_xor(c.v, m);
    int oi = __shfl_xor(c.i, m);
    if (ranks_before(ov, oi, c.v, c.i)) {
      c.v = ov;
      c.i = oi;
    }
  }
  return c;
}

constexpr int kMaxK = 64;
constexpr int kNone = 0x7fffffff;
constexpr int kRankMaxE = 1024;

__device__ __forceinline__ int precedes(float u, int e, float v, int i) {
  return (u > v || (u == v && e < i)) ? 1 : 0;
}

// Rank of (v, i) among vals[0..E) (LDS, 16-byte aligned): the number of
// elements that precede it.  Sixteen values per step, four 128-bit reads.
__device__ __forceinline__ int rank_of(const float* vals, int E, float v, int i) {
  int r = 0;
  int e = 0;
  const f32x4* v4 = reinterpret_cast<const f32x4*>(vals);
  for (; e + 16 <= E; e += 16) {
    f32x4 a[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) a[j] = v4[(e >> 2) + j];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int l = 0; l < 4; ++l) r += precedes(a[j][l], e + 4 * j + l, v, i);
  }
  for (; e < E; ++e) r += precedes(vals[e], e, v, i);
  return r;
}

constexpr int kWChunk = 64;  // tokens whose selected probabilities are staged at once

// One workgroup (256 threads) per block.  Dynamic LDS: E floats of S, then the
// selected probabilities of kWChunk tokens (kWChunk * k floats).
__global__ __launch_bounds__(256) void block_topk_kernel(const float* __restrict__ probs, int bs,
                                                         int E, int k, float* __restrict__ scores,
                                                         int32_t* __restrict__ experts,
                                                         float* __restrict__ w,
                                                         float* __restrict__ gap) {
  extern __shared__ float S[];
  float* V = S + E;  // kWChunk * k floats
  __shared__ int sel[kMaxK + 1];
  __shared__ float selv[kMaxK + 1];
  __shared__ Cand wbest[4];
  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int b = blockIdx.x;
  const float* pb = probs + static_cast<size_t>(b) * bs * E;

  const float n_tok = static_cast<float>(bs);
  for (int e = tid; e < E; e += blockDim.x) {
    float acc = 0.f;
#pragma unroll 8
    for (int t = 0; t < bs; ++t) acc += pb[static_cast<size_t>(t) * E + e];  // token order
    const float v = acc / n_tok;
    S[e] = v;
    if (scores) scores[static_cast<size_t>(b) * E + e] = v;
  }
  __syncthreads();

  const int rounds = k < E ? k + 1 : k;
  if (E <= kRankMaxE) {
    for (int e = tid; e < E; e += blockDim.x) {
      const float v = S[e];
      const int r = rank_of(S, E, v, e);
      if (r < rounds) {
        sel[r] = e;
        selv[r] = v;
      }
    }
    __syncthreads();
  } else {
    float pv = INFINITY;
    int pi = -1;
    for (int r = 0; r < rounds; ++r) {
      Cand best{-INFINITY, kNone};
      for (int e = tid; e < E; e += blockDim.x) {
        const float v = S[e];
        if (ranks_before(pv, pi, v, e) && ranks_before(v, e, best.v, best.i)) best = Cand{v, e};
      }
      best = wave_best(best);
      if (lane == 0) wbest[wave] = best;
      __syncthreads();
      best = wbest[0];
#pragma unroll
      for (int ww = 1; ww < 4; ++ww)
        if (ranks_before(wbest[ww].v, wbest[ww].i, best.v, best.i)) best = wbest[ww];
      if (tid == 0) {
        sel[r] = best.i;
        selv[r] = best.v;
      }
      pv = best.v;
      pi = best.i;
      __syncthreads();
    }
  }

  if (tid == 0) {
    if (gap) gap[b] = k < E ? selv[k - 1] - selv[k] : INFINITY;
  }
  if (tid < k) experts[static_cast<size_t>(b) * k + tid] = sel[tid];

  // Combine weights, kWChunk tokens at a time: all (token, slot) loads of the
  // chunk are independent and issued together, then each token sums its k
  // values in slot order.
  for (int t0 = 0; t0 < bs; t0 += kWChunk) {
    const int nt = min(kWChunk, bs - t0);
    for (int i = tid; i < nt * k; i += blockDim.x) {
      const int tl = i / k, j = i - tl * k;
      V[i] = pb[static_cast<size_t>(t0 + tl) * E + sel[j]];
    }
    __syncthreads();
    if (tid < nt) {
      const float* v = V + tid * k;
      float denom = 0.f;
      for (int j = 0; j < k; ++j) denom += v[j];
      float* wr = w + (static_cast<size_t>(b) * bs + t0 + tid) * k;
      for (int j = 0; j < k; ++j) wr[j] = v[j] / denom;
    }
    __syncthreads();
  }
}

// One wave per token, four tokens per workgroup; the token's row is staged in
// LDS (dynamic: 4*E floats) so the k+1 rounds do not go back to memory.
__global__ __launch_bounds__(256) void token_topk_kernel(const float* __restrict__ probs, int T,
                                                         int E, int k,
                                                         int32_t* __restrict__ experts,
                                                         float* __restrict__ w,
                                                         float* __restrict__ gap) {
  extern __shared__ float rows[];
  __shared__ int sel[4][kMaxK + 1];
  __shared__ float selv[4][kMaxK + 1];
  __shared__ float denom_s[4];
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + wave;
  // Waves past the last token skip the work but still reach both barriers.
  const bool live = t < T;
  const float* grow = probs + static_cast<size_t>(live ? t : 0) * E;
  float* row = rows + static_cast<size_t>(wave) * E;
  for (int e = lane; e < E; e += kWave) row[e] = grow[e];

  const int rounds = live ? (k < E ? k + 1 : k) : 0;
  float pv = INFINITY;
  int pi = -1;
  for (int r = 0; r < rounds; ++r) {
    Cand best{-INFINITY, kNone};
    for (int e = lane; e < E; e += kWave) {
      const float v = row[e];
      if (ranks_before(pv, pi, v, e) && ranks_before(v, e, best.v, best.i)) best = Cand{v, e};
    }
    best = wave_best(best);
    if (lane == 0) {
      sel[wave][r] = best.i;
      selv[wave][r] = best.v;
    }
    pv = best.v;
    pi = best.i;
  }
  __syncthreads();
  if (live && lane == 0) {
    float denom = 0.f;
    for (int j = 0; j < k; ++j) denom += selv[wave][j];
    if (gap) gap[t] = k < E ? selv[wave][k - 1] - selv[wave][k] : INFINITY;
    denom_s[wave] = denom;
  }
  __syncthreads();
  if (live && lane < k) {
    experts[static_cast<size_t>(t) * k + lane] = sel[wave][lane];
    w[static_cast<size_t>(t) * k + lane] = selv[wave][lane] / denom_s[wave];
  }
}

}  // namespace

hipError_t launch_block_topk(const float* probs, int nb, int bs, int E, int k, float* scores,
                             int32_t* experts, float* w, float* gap, hipStream_t s) {
  const size_t lds = (static_cast<size_t>(E) + static_cast<size_t>(kWChunk) * k) * sizeof(float);
  block_topk_kernel<<<nb, 256, lds, s>>>(probs, bs, E, k, scores, experts, w, gap);
  return hipGetLastError();
}

hipError_t launch_token_topk(const float* probs, int T, int E, int k, int32_t* experts, float* w,
                             float* gap, hipStream_t s) {
  token_topk_kernel<<<(T + 3) / 4, 256, static_cast<size_t>(4) * E * sizeof(float), s>>>(
      probs, T, E, k, experts, w, gap);
  return hipGetLastError();
}

}  // namespace dmoe
