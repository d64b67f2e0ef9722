// Alg. 1 (Sec. 4.2) on each block of tokens, with the Top-P coreset:
//   S[e]  = sum over the block's tokens, in token order, of TopKMask(p_t, k)[e]
//   Sn[e] = S[e] / sum_e' S[e']                (the sum in expert-id order)
//   C     = the shortest prefix of the experts ranked by Sn (desc, id asc)
//           whose cumulative Sn, in that order, reaches p; at least
//           min_coreset experts
//   R_t   = top-k of p_t restricted to C; weights renormalised over R_t.
// One workgroup (4 waves) per block.  Token selections use the wave radix
// select of route_dev.h (same total order and tie rule as the other paths);
// the sums and the Top-P walk are sequential in the stated orders, so the
// float32 decisions are those of the definition.
#include "route_dev.h"

namespace dmoe {
namespace {

constexpr int kTopPThreads = 256;
constexpr int kTopPWaves = kTopPThreads / kWave;

__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Dynamic LDS (4-byte words): rows [4][Ep] (a wave's staged token row; row 0
// also holds Sn), S [Ep], order [Ep], inside [Ep], sel [bs][k].
__global__ __launch_bounds__(kTopPThreads) void block_topp_kernel(
    const float* __restrict__ probs, int bs, int E, int k, float p, int min_c,
    float* __restrict__ block_scores, int32_t* __restrict__ coreset, int32_t* __restrict__ coreset_size,
    int32_t* __restrict__ experts, float* __restrict__ cw, float* __restrict__ gap) {
  extern __shared__ float lds[];
  const int Ep = dev::pad4(E);
  float* rows = lds;
  float* S = rows + 4 * Ep;
  int* order = reinterpret_cast<int*>(S + Ep);
  int* inside = order + Ep;
  int* sel = inside + Ep;
  __shared__ int wsel[kTopPWaves][dev::kMaxK + 1];
  __shared__ float wselv[kTopPWaves][dev::kMaxK + 1];
  __shared__ float bufv[kTopPWaves][dev::kMaxK + 1];
  __shared__ int bufi[kTopPWaves][dev::kMaxK + 1];
  __shared__ float s_total;
  __shared__ int s_csize;

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int b = blockIdx.x;
  const float* pb = probs + static_cast<size_t>(b) * bs * E;
  float* row = rows + wave * Ep;

  // 1. every token's own top-k (the support of TopKMask), one wave per token
  for (int t = wave; t < bs; t += kTopPWaves) {
    for (int e = lane; e < E; e += kWave) row[e] = pb[static_cast<size_t>(t) * E + e];
    wave_sync();
    dev::wave_topk_radix(row, E, k, sel + t * k, wselv[wave], bufv[wave], bufi[wave]);
    wave_sync();
  }
  for (int e = tid; e < E; e += kTopPThreads) inside[e] = 0;
  __syncthreads();

  // 2. S[e]: the masked sums in token order
  for (int e = tid; e < E; e += kTopPThreads) {
    float acc = 0.f;
    for (int t = 0; t < bs; ++t) {
      const int* st = sel + t * k;
      bool hit = false;
      for (int j = 0; j < k; ++j) hit |= st[j] == e;
      if (hit) acc += pb[static_cast<size_t>(t) * E + e];
    }
    S[e] = acc;
  }
  __syncthreads();

  // 3. the sum, in expert-id order
  if (tid == 0) {
    float total = 0.f;
    for (int e = 0; e < E; ++e) total += S[e];
    s_total = total;
  }
  __syncthreads();

  // 4. Sn and its ranking (Sn desc, id asc)
  float* Sn = rows;
  const float total = s_total;
  for (int e = tid; e < E; e += kTopPThreads) {
    const float v = S[e] / total;
    Sn[e] = v;
    if (block_scores) block_scores[static_cast<size_t>(b) * E + e] = v;
  }
  __syncthreads();
  for (int e = tid; e < E; e += kTopPThreads) {
    const float v = Sn[e];
    int r = 0;
    for (int m = 0; m < E; ++m) r += dev::precedes(Sn[m], m, v, e);
    order[r] = e;
  }
  __syncthreads();

  // 5. the Top-P cut: cumulative Sn in rank order reaches p, at least min_c
  if (tid == 0) {
    float acc = 0.f;
    int n = 0;
    for (int i = 0; i < E; ++i) {
      n = i + 1;
      acc += Sn[order[i]];
      if (acc >= p && n >= min_c) break;
    }
    s_csize = max(n, min_c);
  }
  __syncthreads();
  const int csize = s_csize;
  if (tid == 0) coreset_size[b] = csize;
  for (int i = tid; i < csize; i += kTopPThreads) {
    coreset[static_cast<size_t>(b) * E + i] = order[i];
    inside[order[i]] = 1;
  }
  __syncthreads();

  // 6. every token's top-k inside the coreset, and its renormalised weights
  const int rounds = csize > k ? k + 1 : k;
  for (int t = wave; t < bs; t += kTopPWaves) {
    for (int e = lane; e < E; e += kWave) row[e] = inside[e] ? pb[static_cast<size_t>(t) * E + e] : -INFINITY;
    wave_sync();
    dev::wave_topk_radix(row, E, rounds, wsel[wave], wselv[wave], bufv[wave], bufi[wave]);
    wave_sync();
    float denom = 0.f;
    for (int j = 0; j < k; ++j) denom += wselv[wave][j];  // slot order
    const size_t tk = (static_cast<size_t>(b) * bs + t) * k;
    for (int j = lane; j < k; j += kWave) {
      experts[tk + j] = wsel[wave][j];
      cw[tk + j] = wselv[wave][j] / denom;
    }
    if (gap && lane == 0) gap[static_cast<size_t>(b) * bs + t] = csize > k ? wselv[wave][k - 1] - wselv[wave][k] : INFINITY;
    wave_sync();
  }
}

}  // namespace

size_t topp_lds_bytes(int bs, int E, int k) {
  return (static_cast<size_t>(dev::pad4(E)) * 7 + static_cast<size_t>(bs) * k) * sizeof(float);
}

hipError_t launch_block_topp(const float* probs, int nb, int bs, int E, int k, float p, int min_c,
                             float* block_scores, int32_t* coreset, int32_t* coreset_size, int32_t* experts,
                             float* w, float* gap, hipStream_t s) {
  block_topp_kernel<<<nb, kTopPThreads, topp_lds_bytes(bs, E, k), s>>>(probs, bs, E, k, p, min_c, block_scores,
                                                                      coreset, coreset_size, experts, w, gap);
  return hipGetLastError();
}

}  // namespace dmoe
