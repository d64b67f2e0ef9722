// Alg. 1 (Sec. 4.2) on each block of tokens, with the Top-P coreset:
//   S[e]  = sum over the block's tokens, in token order, of TopKMask(p_t, k)[e]
//   Sn[e] = S[e] / sum_e' S[e']                (the sum in expert-id order)
//   C     = the shortest prefix of the experts ranked by Sn (desc, id asc)
//           whose cumulative Sn, in that order, reaches p; at least
//           min_coreset experts
//   R_t   = top-k of p_t restricted to C; weights renormalised over R_t.
// Three launches: every token's own top-k (the support of TopKMask) by the
// token-routing selection kernel, one wave per token across many CUs; one
// workgroup per block for S, Sn, the ranking and the Top-P cut; then one wave
// per token again for its top-k inside its block's coreset.  Selections use
// the wave radix select of route_dev.h (same total order and tie rule as the
// other paths).  The sums and the Top-P walk are sequential in the stated
// orders, so the float32 decisions are those of the definition; everything
// else is spread over the threads.
#include "route_dev.h"

namespace dmoe {
namespace {

constexpr int kCoreThreads = 512;
constexpr size_t kCoreLdsBudget = 64 * 1024 - 256;  // dynamic LDS bytes (the kernel has no static LDS)

// Dynamic LDS of the coreset kernel, in 4-byte words (the only LDS of the
// kernel, so word 0 is 16-byte aligned).  Rows of Ep = pad4(E) words keep
// the 128-bit reads of S and Sv aligned.
struct CoreLayout {
  int Ep, tc;  // padded row, tokens per masked-sum chunk
  size_t misc, S, Sv, order, M, total;
};

__host__ __device__ inline CoreLayout core_layout(int bs, int E) {
  CoreLayout L;
  L.Ep = dev::pad4(E);
  L.misc = 0;              // the block's total, the coreset size
  L.S = 4;                 // block sums, then Sn in place
  L.Sv = L.S + L.Ep;       // Sn in rank order
  L.order = L.Sv + L.Ep;   // expert ids in rank order
  L.M = L.order + L.Ep;    // [tc][Ep] masked-sum chunk, then rank counters
  const size_t budget = kCoreLdsBudget / 4;
  const size_t room = budget > L.M ? (budget - L.M) / L.Ep : 0;
  L.tc = static_cast<int>(room < static_cast<size_t>(bs) ? room : static_cast<size_t>(bs));
  L.total = L.M + static_cast<size_t>(L.tc) * L.Ep;
  return L;
}

// One workgroup per block: S from the tokens' own top-k (own_sel [T][k], in
// token order), Sn, the ranking, the Top-P cut and the coreset.
__global__ __launch_bounds__(kCoreThreads) void block_coreset_kernel(
    const float* __restrict__ probs, const int32_t* __restrict__ own_sel, int bs, int E, int k, float p,
    int min_c, float* __restrict__ block_scores, int32_t* __restrict__ coreset,
    int32_t* __restrict__ coreset_size) {
  extern __shared__ __align__(16) float lds[];
  const CoreLayout L = core_layout(bs, E);
  const int Ep = L.Ep;
  float* S = lds + L.S;
  float* Sv = lds + L.Sv;
  int* order = reinterpret_cast<int*>(lds + L.order);
  float* M = lds + L.M;
  float& s_total = lds[L.misc];
  int& s_csize = reinterpret_cast<int*>(lds)[L.misc + 1];

  const int tid = threadIdx.x;
  const int b = blockIdx.x;
  const float* pb = probs + static_cast<size_t>(b) * bs * E;
  const int32_t* sb = own_sel + static_cast<size_t>(b) * bs * k;

  // 1. S[e]: the masked sums in token order.  Chunks of tc tokens are
  //    scattered into a dense [tc][Ep] matrix (zero where a token did not
  //    select e, so adding it is exact), then each thread adds its column.
  float acc[2] = {0.f, 0.f};  // columns tid and tid + 512 (E <= 1024)
  for (int c0 = 0; c0 < bs; c0 += L.tc) {
    const int nt = min(L.tc, bs - c0);
    for (int i = tid; i < nt * Ep; i += kCoreThreads) M[i] = 0.f;
    __syncthreads();
    for (int i = tid; i < nt * k; i += kCoreThreads) {
      const int tl = i / k;
      const int e = sb[c0 * k + i];
      M[tl * Ep + e] = pb[static_cast<size_t>(c0 + tl) * E + e];
    }
    __syncthreads();
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int e = tid + h * kCoreThreads;
      if (e < Ep)
        for (int tl = 0; tl < nt; ++tl) acc[h] += M[tl * Ep + e];
    }
    __syncthreads();
  }
#pragma unroll
  for (int h = 0; h < 2; ++h)
    if (tid + h * kCoreThreads < Ep) S[tid + h * kCoreThreads] = acc[h];  // padding: 0
  __syncthreads();

  // 2. the sum, in expert-id order (padding adds exact zeros); the rank
  //    counters of step 3 (in M, free now) start at zero
  int* rankc = reinterpret_cast<int*>(M);
  for (int e = tid; e < Ep; e += kCoreThreads) rankc[e] = 0;
  if (tid == 0) {
    const float4* S4 = reinterpret_cast<const float4*>(S);
    float total = 0.f;
#pragma unroll 8
    for (int i = 0; i < Ep / 4; ++i) {
      const float4 q = S4[i];
      total += q.x;
      total += q.y;
      total += q.z;
      total += q.w;
    }
    s_total = total;
  }
  __syncthreads();

  // 3. Sn in place, then each expert's rank (Sn desc, id asc) by counting
  //    over the order keys of Sn (staged in Sv, free until the ranks are
  //    known); padding (ids >= E) takes key 0 and never ranks before a real
  //    expert, so the ranks of the E experts are 0 .. E-1
  const float total = s_total;
  uint32_t* Sk = reinterpret_cast<uint32_t*>(Sv);
  for (int e = tid; e < Ep; e += kCoreThreads) {
    const float v = S[e] / total;
    S[e] = v;
    Sk[e] = e < E ? max(dev::order_key(v), 1u) : 0u;
    if (block_scores && e < E) block_scores[static_cast<size_t>(b) * E + e] = v;
  }
  __syncthreads();
  {
    // `parts` threads per expert (a power of two, all 512 threads busy when
    // E <= 256) each count the experts ranked before it in a slice of the
    // row; the counts meet in LDS.
    const int parts = Ep <= 64 ? 8 : Ep <= 128 ? 4 : Ep <= 256 ? 2 : 1;
    const int n4 = Ep / 4, len = (n4 + parts - 1) / parts;
    const uint4* K4 = reinterpret_cast<const uint4*>(Sk);
    for (int idx = tid; idx < E * parts; idx += kCoreThreads) {
      const int e = idx / parts, h = idx - e * parts;
      const uint32_t kv = Sk[e];
      const int m1 = min(n4, (h + 1) * len);
      int r = 0;
#pragma unroll 4
      for (int m = h * len; m < m1; ++m) {
        const uint4 q = K4[m];
        r += (dev::key_before(q.x, 4 * m, kv, e) ? 1 : 0) + (dev::key_before(q.y, 4 * m + 1, kv, e) ? 1 : 0) +
             (dev::key_before(q.z, 4 * m + 2, kv, e) ? 1 : 0) + (dev::key_before(q.w, 4 * m + 3, kv, e) ? 1 : 0);
      }
      if (r) atomicAdd(&rankc[e], r);
    }
  }
  __syncthreads();
  for (int e = tid; e < E; e += kCoreThreads) {
    const int r = rankc[e];
    order[r] = e;
    Sv[r] = S[e];
  }
  __syncthreads();

  // 4. the Top-P cut: cumulative Sn in rank order reaches p, at least min_c.
  //    One thread adds in rank order, 32 values per batch: a straight chain
  //    of adds (entries past E add an exact zero), then the first prefix
  //    that qualifies.
  if (tid == 0) {
    const float4* Sv4 = reinterpret_cast<const float4*>(Sv);
    float cum = 0.f;
    int n = 0;
    for (int i0 = 0; i0 < E && n == 0; i0 += 32) {
      float c[32];
#pragma unroll
      for (int q = 0; q < 8; ++q) {  // within the Ep-word row
        const float4 f = i0 + 4 * q < Ep ? Sv4[i0 / 4 + q] : float4{0.f, 0.f, 0.f, 0.f};
        c[4 * q] = f.x;
        c[4 * q + 1] = f.y;
        c[4 * q + 2] = f.z;
        c[4 * q + 3] = f.w;
      }
#pragma unroll
      for (int u = 0; u < 32; ++u) {
        cum += i0 + u < E ? c[u] : 0.f;
        c[u] = cum;
      }
#pragma unroll
      for (int u = 31; u >= 0; --u)
        if (i0 + u < E && c[u] >= p && i0 + u + 1 >= min_c) n = i0 + u + 1;
    }
    s_csize = n > 0 ? n : E;
  }
  __syncthreads();
  const int csize = s_csize;
  if (tid == 0) coreset_size[b] = csize;
  for (int i = tid; i < csize; i += kCoreThreads) coreset[static_cast<size_t>(b) * E + i] = order[i];
}

__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// One wave per token, four per workgroup: the token's top-k inside its
// block's coreset (and the next one for the gap), then its weights
// renormalised over them, summed in slot order.  Dynamic LDS (words): four
// coreset-flag rows of Ep, then per wave sel, selv and the radix gather
// buffers (k + 1 each).
template <int NJ>
__global__ __launch_bounds__(256) void topp_select_kernel(const float* __restrict__ probs, int T, int bs, int E,
                                                          int k, const int32_t* __restrict__ coreset,
                                                          const int32_t* __restrict__ coreset_size,
                                                          int32_t* __restrict__ experts, float* __restrict__ cw,
                                                          float* __restrict__ gap) {
  extern __shared__ __align__(16) int ldsi[];
  const int Ep = dev::pad4(E), K1 = k + 1;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + wave;
  if (t >= T) return;  // only wave-level synchronisation below
  int* inside = ldsi + wave * Ep;
  int* wsel = ldsi + 4 * Ep + wave * 4 * K1;
  float* wselv = reinterpret_cast<float*>(wsel + K1);
  float* bufv = reinterpret_cast<float*>(wsel + 2 * K1);
  int* bufi = wsel + 3 * K1;
  const int b = t / bs;
  const int csize = coreset_size[b];
  for (int e = lane; e < Ep; e += kWave) inside[e] = 0;
  wave_sync();
  for (int i = lane; i < csize; i += kWave) inside[coreset[static_cast<size_t>(b) * E + i]] = 1;
  wave_sync();
  const int rounds = csize > k ? K1 : k;
  const float* const rows[1] = {probs + static_cast<size_t>(t) * E};
  const bool live[1] = {true};
  int* const s[1] = {wsel};
  float* const sv[1] = {wselv};
  dev::wave_topk_radix_rows<NJ, 1, true>(rows, live, E, rounds, s, sv, bufv, bufi, inside);
  float denom = 0.f;
  for (int j = 0; j < k; ++j) denom += wselv[j];
  const size_t tk = static_cast<size_t>(t) * k;
  for (int j = lane; j < k; j += kWave) {
    experts[tk + j] = wsel[j];
    cw[tk + j] = wselv[j] / denom;
  }
  if (gap && lane == 0) gap[t] = csize > k ? wselv[k - 1] - wselv[k] : INFINITY;
}

}  // namespace

bool topp_supported(int bs, int E, int k) {
  return E <= 64 * dev::kRadixMaxPerLane && k <= dev::kMaxK && core_layout(bs, E).tc >= 1;
}

hipError_t launch_block_topp(const float* probs, int nb, int bs, int E, int k, float p, int min_c,
                             float* block_scores, int32_t* coreset, int32_t* coreset_size, int32_t* experts,
                             float* w, float* gap, hipStream_t s, bool own_done) {
  if (!topp_supported(bs, E, k)) return hipErrorInvalidValue;
  const int T = nb * bs;
  hipError_t err;
  // 1. every token's own top-k, into `experts` (overwritten by step 3;
  //    own_done: the caller's launch already put it there)
  if (!own_done) {
    err = launch_token_topk(probs, T, E, k, experts, w, nullptr, s);
    if (err != hipSuccess) return err;
  }
  // 2. one workgroup per block
  block_coreset_kernel<<<nb, kCoreThreads, core_layout(bs, E).total * sizeof(float), s>>>(
      probs, experts, bs, E, k, p, min_c, block_scores, coreset, coreset_size);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  // 3. one wave per token
  const size_t lds = (4 * static_cast<size_t>(dev::pad4(E)) + 16 * static_cast<size_t>(k + 1)) * sizeof(int);
  const unsigned grid = static_cast<unsigned>((T + 3) / 4);
#define DMOE_TOPP(NJ)                                                                                         \
  topp_select_kernel<NJ><<<grid, 256, lds, s>>>(probs, T, bs, E, k, coreset, coreset_size, experts, w, gap)
  if (E <= 64)
    DMOE_TOPP(1);
  else if (E <= 128)
    DMOE_TOPP(2);
  else if (E <= 256)
    DMOE_TOPP(4);
  else if (E <= 512)
    DMOE_TOPP(8);
  else
    DMOE_TOPP(16);
#undef DMOE_TOPP
  return hipGetLastError();
}

}  // namespace dmoe
