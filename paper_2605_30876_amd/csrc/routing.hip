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
// to the lower id.  Up to 1024 experts a wave selects by radix search over
// order-preserving keys (dev::wave_topk_radix); above that a top-k walks the
// order: round r picks the best element strictly after round r-1's pick.
#include <algorithm>

#include "route_dev.h"

namespace dmoe {
namespace {

using dev::Cand;
using dev::key_before;
using dev::kMaxK;
using dev::wave_best;

constexpr int kRadixMaxE = 64 * dev::kRadixMaxPerLane;
constexpr int kSumBatch = 32;  // token loads of a block sum issued together

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
  __shared__ float bufv[kMaxK + 1];
  __shared__ int bufi[kMaxK + 1];
  __shared__ Cand wbest[4];
  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int b = blockIdx.x;
  const float* pb = probs + static_cast<size_t>(b) * bs * E;

  // Block mean in token order; a batch of token loads is in flight at once.
  const float n_tok = static_cast<float>(bs);
  for (int e = tid; e < E; e += blockDim.x) {
    float acc = 0.f;
    for (int t0 = 0; t0 < bs; t0 += kSumBatch) {
      float v[kSumBatch];
#pragma unroll
      for (int u = 0; u < kSumBatch; ++u)
        if (t0 + u < bs) v[u] = pb[static_cast<size_t>(t0 + u) * E + e];
#pragma unroll
      for (int u = 0; u < kSumBatch; ++u)
        if (t0 + u < bs) acc += v[u];
    }
    const float v = acc / n_tok;
    S[e] = v;
    if (scores) scores[static_cast<size_t>(b) * E + e] = v;
  }
  __syncthreads();

  const int rounds = k < E ? k + 1 : k;
  if (E <= kRadixMaxE) {
    if (wave == 0) dev::wave_topk_radix(S, E, rounds, sel, selv, bufv, bufi);
    __syncthreads();
  } else {
    Cand prev = dev::kCandTop;
    for (int r = 0; r < rounds; ++r) {
      Cand best = dev::kCandNone;
      for (int e = tid; e < E; e += blockDim.x) {
        const uint32_t kv = dev::order_key(S[e]);
        if (key_before(prev.key, prev.i, kv, e) && key_before(kv, e, best.key, best.i)) best = Cand{kv, e};
      }
      best = wave_best(best);
      if (lane == 0) wbest[wave] = best;
      __syncthreads();
      best = wbest[0];
#pragma unroll
      for (int ww = 1; ww < 4; ++ww)
        if (key_before(wbest[ww].key, wbest[ww].i, best.key, best.i)) best = wbest[ww];
      if (tid == 0) {
        sel[r] = best.i;
        selv[r] = dev::key_value(best.key);
      }
      prev = best;
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
// LDS (dynamic: 4*E floats) so the selection does not go back to memory.
__global__ __launch_bounds__(256) void token_topk_kernel(const float* __restrict__ probs, int T,
                                                         int E, int k,
                                                         int32_t* __restrict__ experts,
                                                         float* __restrict__ w,
                                                         float* __restrict__ gap, int raw) {
  extern __shared__ float rows[];
  __shared__ int sel[4][kMaxK + 1];
  __shared__ float selv[4][kMaxK + 1];
  __shared__ float bufv[4][kMaxK + 1];
  __shared__ int bufi[4][kMaxK + 1];
  __shared__ float denom_s[4];
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + wave;
  // Waves past the last token skip the work but still reach both barriers.
  const bool live = t < T;
  const float* grow = probs + static_cast<size_t>(live ? t : 0) * E;
  float* row = rows + static_cast<size_t>(wave) * E;
  for (int e = lane; e < E; e += kWave) row[e] = grow[e];

  const int rounds = k < E ? k + 1 : k;
  if (live) {
    if (E <= kRadixMaxE)
      dev::wave_topk_radix(row, E, rounds, sel[wave], selv[wave], bufv[wave], bufi[wave]);
    else
      dev::wave_topk(row, E, rounds, sel[wave], selv[wave]);
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
    // raw: the staged row's own value (the stored probability, bit for bit)
    w[static_cast<size_t>(t) * k + lane] = raw ? row[sel[wave][lane]] : selv[wave][lane] / denom_s[wave];
  }
}

// Token routing straight from the router's partial logits: one wave per
// token sums the partials, takes the softmax in registers (the routine the
// separate softmax kernel uses, so probs are bit-identical), stages the row in
// LDS and selects from it as token_topk_kernel does (one launch instead of
// two).  E <= 512.
template <int NQ>
__global__ __launch_bounds__(256) void softmax_token_topk_kernel(const float* part, int S,
                                                                 const float* __restrict__ bias, int T, int E, int k,
                                                                 float* probs, float* __restrict__ logits,
                                                                 int32_t* __restrict__ experts,
                                                                 float* __restrict__ w, float* __restrict__ gap,
                                                                 int raw) {
  extern __shared__ float rows[];
  __shared__ int sel[4][kMaxK + 1];
  __shared__ float selv[4][kMaxK + 1];
  __shared__ float bufv[4][kMaxK + 1];
  __shared__ int bufi[4][kMaxK + 1];
  __shared__ float denom_s[4];
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + wave;
  // Waves past the last token skip the work but still reach the barriers.
  const bool live = t < T;
  float* row = rows + static_cast<size_t>(wave) * E;
  if (live) {
    dev::RowPartials<NQ> r[1];
    dev::load_row<NQ>(part, static_cast<size_t>(T) * E, S, bias, E, t, r[0]);
    const bool lv[1] = {true};
    float* const out[1] = {probs + static_cast<size_t>(t) * E};
    float* const lds[1] = {row};
    float* const lo[1] = {logits ? logits + static_cast<size_t>(t) * E : nullptr};
    dev::softmax_loaded<NQ, 1>(r, lv, S, bias != nullptr, E, out, lds, lo);
  }
  __syncthreads();  // the staged rows (and, with S == 1, part aliasing probs) are complete

  const int rounds = k < E ? k + 1 : k;
  if (live) dev::wave_topk_radix(row, E, rounds, sel[wave], selv[wave], bufv[wave], bufi[wave]);
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
    // raw: the staged row's own value (the stored probability, bit for bit)
    w[static_cast<size_t>(t) * k + lane] = raw ? row[sel[wave][lane]] : selv[wave][lane] / denom_s[wave];
  }
}

}  // namespace

bool softmax_token_topk_fits(int E) { return E <= dev::kRegSoftmaxMaxE && E <= kRadixMaxE; }

hipError_t launch_softmax_token_topk(const float* part, int S, const float* bias, int T, int E, int k, float* probs,
                                     float* logits, int32_t* experts, float* w, float* gap, hipStream_t s,
                                     bool raw) {
  const unsigned blocks = (T + 3) / 4;
  const size_t lds = static_cast<size_t>(4) * E * sizeof(float);
  if (E <= 256)
    softmax_token_topk_kernel<1><<<blocks, 256, lds, s>>>(part, S, bias, T, E, k, probs, logits, experts, w, gap,
                                                           raw ? 1 : 0);
  else
    softmax_token_topk_kernel<2><<<blocks, 256, lds, s>>>(part, S, bias, T, E, k, probs, logits, experts, w, gap,
                                                           raw ? 1 : 0);
  return hipGetLastError();
}

hipError_t launch_block_topk(const float* probs, int nb, int bs, int E, int k, float* scores,
                             int32_t* experts, float* w, float* gap, hipStream_t s) {
  const size_t lds = (static_cast<size_t>(E) + static_cast<size_t>(kWChunk) * k) * sizeof(float);
  block_topk_kernel<<<nb, 256, lds, s>>>(probs, bs, E, k, scores, experts, w, gap);
  return hipGetLastError();
}

hipError_t launch_token_topk(const float* probs, int T, int E, int k, int32_t* experts, float* w,
                             float* gap, hipStream_t s, bool raw) {
  token_topk_kernel<<<(T + 3) / 4, 256, static_cast<size_t>(4) * E * sizeof(float), s>>>(
      probs, T, E, k, experts, w, gap, raw ? 1 : 0);
  return hipGetLastError();
}

}  // namespace dmoe
