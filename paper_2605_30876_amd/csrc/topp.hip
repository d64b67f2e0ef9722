// Alg. 1 (Sec. 4.2) on each block of tokens, with the Top-P coreset:
//   S[e]  = sum over the block's tokens, in token order, of TopKMask(p_t, k)[e]
//   Sn[e] = S[e] / sum_e' S[e']                (the sum in expert-id order)
//   C     = the shortest prefix of the experts ranked by Sn (desc, id asc)
//           whose cumulative Sn, in that order, reaches p; at least
//           min_coreset experts
//   R_t   = top-k of p_t restricted to C; weights renormalised over R_t.
// One workgroup (8 waves) per block.  Token selections use the wave radix
// select of route_dev.h (same total order and tie rule as the other paths),
// kRB token rows per wave at once.  The sums and the Top-P walk are
// sequential in the stated orders, so the float32 decisions are those of the
// definition; everything else is spread over the workgroup.
#include "route_dev.h"

namespace dmoe {
namespace {

constexpr int kTopPThreads = 512;
constexpr int kTopPWaves = kTopPThreads / kWave;
constexpr int kRB = 4;                              // token rows a wave selects together
constexpr size_t kTopPLdsBudget = 64 * 1024 - 256;  // dynamic LDS bytes (the kernel has no static LDS)

// Dynamic LDS of one workgroup, in 4-byte words (the only LDS of the kernel,
// so word 0 is 16-byte aligned).  Rows of Ep = pad4(E) words keep the 128-bit
// reads of S and Sv aligned.
struct TopPLayout {
  int Ep, K1, tc;  // padded row, k + 1, tokens per masked-sum chunk
  size_t misc, S, Sv, order, inside, sel, selv, wsel, wselv, bufv, bufi, M, total;
};

__host__ __device__ inline TopPLayout topp_layout(int bs, int E, int k) {
  TopPLayout L;
  L.Ep = dev::pad4(E);
  L.K1 = k + 1;
  const size_t bk = static_cast<size_t>(bs) * k;
  const size_t wk = static_cast<size_t>(kTopPWaves) * kRB * L.K1;
  L.misc = 0;                             // the block's total, the coreset size
  L.S = 4;                                // block sums, then Sn in place
  L.Sv = L.S + L.Ep;                      // Sn in rank order
  L.order = L.Sv + L.Ep;                  // expert ids in rank order
  L.inside = L.order + L.Ep;              // coreset flags
  L.sel = L.inside + L.Ep;                // [bs][k] each token's own top-k
  L.selv = L.sel + bk;                    // [bs][k] their probabilities
  L.wsel = L.selv + bk;                   // [waves][kRB][k+1] in-coreset selections
  L.wselv = L.wsel + wk;
  L.bufv = L.wselv + wk;                  // [waves][k+1] radix gather buffers
  L.bufi = L.bufv + static_cast<size_t>(kTopPWaves) * L.K1;
  L.M = (L.bufi + static_cast<size_t>(kTopPWaves) * L.K1 + 3) & ~static_cast<size_t>(3);  // [tc][Ep]
  const size_t budget = kTopPLdsBudget / 4;
  const size_t room = budget > L.M ? (budget - L.M) / L.Ep : 0;
  L.tc = static_cast<int>(room < static_cast<size_t>(bs) ? room : static_cast<size_t>(bs));
  L.total = L.M + static_cast<size_t>(L.tc) * L.Ep;
  return L;
}

template <int NJ>
__global__ __launch_bounds__(kTopPThreads) void block_topp_kernel(
    const float* __restrict__ probs, int bs, int E, int k, float p, int min_c,
    float* __restrict__ block_scores, int32_t* __restrict__ coreset, int32_t* __restrict__ coreset_size,
    int32_t* __restrict__ experts, float* __restrict__ cw, float* __restrict__ gap) {
  extern __shared__ __align__(16) float lds[];
  const TopPLayout L = topp_layout(bs, E, k);
  const int Ep = L.Ep, K1 = L.K1;
  float* S = lds + L.S;
  float* Sv = lds + L.Sv;
  int* order = reinterpret_cast<int*>(lds + L.order);
  int* inside = reinterpret_cast<int*>(lds + L.inside);
  int* sel = reinterpret_cast<int*>(lds + L.sel);
  float* selv = lds + L.selv;
  float* M = lds + L.M;
  float& s_total = lds[L.misc];
  int& s_csize = reinterpret_cast<int*>(lds)[L.misc + 1];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int b = blockIdx.x;
  const float* pb = probs + static_cast<size_t>(b) * bs * E;
  int* wsel = reinterpret_cast<int*>(lds + L.wsel) + wave * kRB * K1;
  float* wselv = lds + L.wselv + wave * kRB * K1;
  float* bufv = lds + L.bufv + wave * K1;
  int* bufi = reinterpret_cast<int*>(lds + L.bufi) + wave * K1;

  // 1. every token's own top-k (the support of TopKMask), kRB rows per wave
  for (int t0 = wave; t0 < bs; t0 += kTopPWaves * kRB) {
    const float* rows[kRB];
    bool live[kRB];
    int* s[kRB];
    float* sv[kRB];
#pragma unroll
    for (int u = 0; u < kRB; ++u) {
      const int t = t0 + u * kTopPWaves;
      live[u] = t < bs;
      const int tt = live[u] ? t : t0;
      rows[u] = pb + static_cast<size_t>(tt) * E;
      s[u] = sel + tt * k;
      sv[u] = selv + tt * k;
    }
    dev::wave_topk_radix_rows<NJ, kRB>(rows, live, E, k, s, sv, bufv, bufi);
  }
  for (int e = tid; e < Ep; e += kTopPThreads) inside[e] = 0;
  __syncthreads();

  // 2. S[e]: the masked sums in token order.  Chunks of tc tokens are
  //    scattered into a dense [tc][Ep] matrix (zero where a token did not
  //    select e, so adding it is exact), then each thread adds its column.
  float acc[2] = {0.f, 0.f};  // columns tid and tid + 512 (E <= 1024)
  for (int c0 = 0; c0 < bs; c0 += L.tc) {
    const int nt = min(L.tc, bs - c0);
    for (int i = tid; i < nt * Ep; i += kTopPThreads) M[i] = 0.f;
    __syncthreads();
    for (int i = tid; i < nt * k; i += kTopPThreads) {
      const int tl = i / k;
      M[tl * Ep + sel[c0 * k + i]] = selv[c0 * k + i];
    }
    __syncthreads();
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int e = tid + h * kTopPThreads;
      if (e < Ep)
        for (int tl = 0; tl < nt; ++tl) acc[h] += M[tl * Ep + e];
    }
    __syncthreads();
  }
#pragma unroll
  for (int h = 0; h < 2; ++h)
    if (tid + h * kTopPThreads < Ep) S[tid + h * kTopPThreads] = acc[h];  // padding: 0
  __syncthreads();

  // 3. the sum, in expert-id order (padding adds exact zeros); the rank
  //    counters of step 4 (in M, free now) start at zero
  int* rankc = reinterpret_cast<int*>(M);
  for (int e = tid; e < Ep; e += kTopPThreads) rankc[e] = 0;
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

  // 4. Sn in place, then each expert's rank (Sn desc, id asc) by counting;
  //    padding (Sn = 0 at ids >= E) never ranks before a real expert
  const float total = s_total;
  for (int e = tid; e < Ep; e += kTopPThreads) {
    const float v = S[e] / total;
    S[e] = v;
    if (block_scores && e < E) block_scores[static_cast<size_t>(b) * E + e] = v;
  }
  __syncthreads();
  {
    // `parts` threads per expert (a power of two, all 512 threads busy when
    // E <= 256) each count the experts ranked before it in a slice of the
    // row; the counts meet in LDS.
    const int parts = Ep <= 64 ? 8 : Ep <= 128 ? 4 : Ep <= 256 ? 2 : 1;
    const int n4 = Ep / 4, len = (n4 + parts - 1) / parts;
    const float4* S4 = reinterpret_cast<const float4*>(S);
    for (int idx = tid; idx < E * parts; idx += kTopPThreads) {
      const int e = idx / parts, h = idx - e * parts;
      const float v = S[e];
      const int m1 = min(n4, (h + 1) * len);
      int r = 0;
#pragma unroll 4
      for (int m = h * len; m < m1; ++m) {
        const float4 q = S4[m];
        r += dev::precedes(q.x, 4 * m, v, e) + dev::precedes(q.y, 4 * m + 1, v, e) +
             dev::precedes(q.z, 4 * m + 2, v, e) + dev::precedes(q.w, 4 * m + 3, v, e);
      }
      if (r) atomicAdd(&rankc[e], r);
    }
  }
  __syncthreads();
  for (int e = tid; e < E; e += kTopPThreads) {
    const int r = rankc[e];
    order[r] = e;
    Sv[r] = S[e];
  }
  __syncthreads();

  // 5. the Top-P cut: cumulative Sn in rank order reaches p, at least min_c.
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
  for (int i = tid; i < csize; i += kTopPThreads) {
    const int e = order[i];
    coreset[static_cast<size_t>(b) * E + i] = e;
    inside[e] = 1;
  }
  __syncthreads();

  // 6. every token's top-k inside the coreset (and the next one for the
  //    gap), then its weights renormalised over them, summed in slot order
  const int rounds = csize > k ? K1 : k;
  for (int t0 = wave; t0 < bs; t0 += kTopPWaves * kRB) {
    const float* rows[kRB];
    bool live[kRB];
    int* s[kRB];
    float* sv[kRB];
#pragma unroll
    for (int u = 0; u < kRB; ++u) {
      const int t = t0 + u * kTopPWaves;
      live[u] = t < bs;
      rows[u] = pb + static_cast<size_t>(live[u] ? t : t0) * E;
      s[u] = wsel + u * K1;
      sv[u] = wselv + u * K1;
    }
    dev::wave_topk_radix_rows<NJ, kRB, true>(rows, live, E, rounds, s, sv, bufv, bufi, inside);
#pragma unroll
    for (int u = 0; u < kRB; ++u) {
      const int t = t0 + u * kTopPWaves;
      if (t >= bs) continue;
      const float* v = wselv + u * K1;
      float denom = 0.f;
      for (int j = 0; j < k; ++j) denom += v[j];
      const size_t tk = (static_cast<size_t>(b) * bs + t) * k;
      for (int j = lane; j < k; j += kWave) {
        experts[tk + j] = wsel[u * K1 + j];
        cw[tk + j] = v[j] / denom;
      }
      if (gap && lane == 0) gap[static_cast<size_t>(b) * bs + t] = csize > k ? v[k - 1] - v[k] : INFINITY;
    }
    // the per-wave selection buffers are reused by the next rows
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
}

}  // namespace

size_t topp_lds_bytes(int bs, int E, int k) {
  const TopPLayout L = topp_layout(bs, E, k);
  return L.tc >= 1 ? L.total * sizeof(float) : 0;  // 0: does not fit
}

hipError_t launch_block_topp(const float* probs, int nb, int bs, int E, int k, float p, int min_c,
                             float* block_scores, int32_t* coreset, int32_t* coreset_size, int32_t* experts,
                             float* w, float* gap, hipStream_t s) {
  const size_t lds = topp_lds_bytes(bs, E, k);
  if (lds == 0 || E > 64 * dev::kRadixMaxPerLane) return hipErrorInvalidValue;
#define DMOE_TOPP(NJ)                                                                                        \
  block_topp_kernel<NJ><<<nb, kTopPThreads, lds, s>>>(probs, bs, E, k, p, min_c, block_scores, coreset,     \
                                                      coreset_size, experts, w, gap)
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
