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
// A top-k walks the total order (score desc, id asc): round r picks the best
// element that comes strictly after round r-1's pick, so nothing has to be
// removed or marked, and an exact tie goes to the lower id.
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

// One workgroup (256 threads) per block.  Dynamic LDS: E floats of S.
__global__ __launch_bounds__(256) void block_topk_kernel(const float* __restrict__ probs, int bs,
                                                         int E, int k, float* __restrict__ scores,
                                                         int32_t* __restrict__ experts,
                                                         float* __restrict__ w,
                                                         float* __restrict__ gap) {
  extern __shared__ float S[];
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
    for (int t = 0; t < bs; ++t) acc += pb[static_cast<size_t>(t) * E + e];
    const float v = acc / n_tok;
    S[e] = v;
    if (scores) scores[static_cast<size_t>(b) * E + e] = v;
  }
  __syncthreads();

  const int rounds = k < E ? k + 1 : k;
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

  if (tid == 0) {
    if (gap) gap[b] = k < E ? selv[k - 1] - selv[k] : INFINITY;
  }
  if (tid < k) experts[static_cast<size_t>(b) * k + tid] = sel[tid];

  for (int t = tid; t < bs; t += blockDim.x) {
    const float* row = pb + static_cast<size_t>(t) * E;
    float denom = 0.f;
    for (int j = 0; j < k; ++j) denom += row[sel[j]];
    float* wr = w + (static_cast<size_t>(b) * bs + t) * k;
    for (int j = 0; j < k; ++j) wr[j] = row[sel[j]] / denom;
  }
}

// One wave per token, four tokens per workgroup.
__global__ __launch_bounds__(256) void token_topk_kernel(const float* __restrict__ probs, int T,
                                                         int E, int k,
                                                         int32_t* __restrict__ experts,
                                                         float* __restrict__ w,
                                                         float* __restrict__ gap) {
  __shared__ int sel[4][kMaxK + 1];
  __shared__ float selv[4][kMaxK + 1];
  __shared__ float denom_s[4];
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + wave;
  // Waves past the last token skip the work but still reach both barriers.
  const bool live = t < T;
  const float* row = probs + static_cast<size_t>(live ? t : 0) * E;

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
  block_topk_kernel<<<nb, 256, static_cast<size_t>(E) * sizeof(float), s>>>(probs, bs, E, k, scores,
                                                                             experts, w, gap);
  return hipGetLastError();
}

hipError_t launch_token_topk(const float* probs, int T, int E, int k, int32_t* experts, float* w,
                             float* gap, hipStream_t s) {
  token_topk_kernel<<<(T + 3) / 4, 256, 0, s>>>(probs, T, E, k, experts, w, gap);
  return hipGetLastError();
}

}  // namespace dmoe
