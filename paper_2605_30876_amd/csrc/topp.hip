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
constexpr int kCoreWaves = kCoreThreads / kWave;
constexpr int kCoreCols = 2;        // experts per thread (E <= 1024)
constexpr int kCoreTokChunk = 32;   // tokens per masked-sum chunk, at most
constexpr int kCoreMWords = 8192;   // LDS words of a chunk's masked probability rows (32 KiB)

__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Dynamic LDS of the coreset kernel, in 4-byte words (the only LDS of the
// kernel, so word 0 is 16-byte aligned).  Rows of Ep = pad4(E) words keep
// the 128-bit reads aligned.  tc: tokens per masked-sum chunk (at most one
// selection entry per thread, at most kCoreMWords of probabilities).
struct CoreLayout {
  int Ep, tc, tc8;
  size_t misc, wcnt, S, Sv, order, keys, rankc, M, total;
};

__host__ __device__ inline CoreLayout core_layout(int bs, int E, int k) {
  CoreLayout L;
  L.Ep = dev::pad4(E);
  int tc = kCoreThreads / (k > 0 ? k : 1);
  tc = tc < kCoreTokChunk ? tc : kCoreTokChunk;
  tc = tc < kCoreMWords / L.Ep ? tc : kCoreMWords / L.Ep;
  L.tc = tc < bs ? tc : bs;
  L.misc = 0;                             // the block's total, the coreset size, keys below +0's
  L.wcnt = 4;                             // per-wave ballot counts, kCoreCols * kCoreWaves
  L.S = L.wcnt + kCoreCols * kCoreWaves;  // block sums, then Sn in place
  L.Sv = L.S + L.Ep;                      // Sn in rank order, zeros up to a multiple of 64
  L.order = L.Sv + ((L.Ep + kWave - 1) & ~(kWave - 1));  // expert ids in rank order
  L.keys = L.order + L.Ep;                // the nonzero sums (total), then the listed experts'
                                          // 64-bit ranking keys (2 Ep words)
  L.rankc = L.keys + 2 * L.Ep;            // rank counters, then the Top-P walk's prefix sums
  L.tc8 = (L.tc + 7) & ~7;                // rows of M, read in groups of 8
  L.M = L.rankc + (L.Ep > kWave ? L.Ep : kWave);  // [tc8][Ep] masked probabilities of a chunk
  L.total = L.M + static_cast<size_t>(L.tc8) * L.Ep;
  return L;
}

// One workgroup per block: S from the tokens' own top-k (own_sel [T][k], in
// token order), Sn, the ranking, the Top-P cut and the coreset.  Every float
// sum runs in the order the definition states; zeros are skipped only where
// adding them is exact.
__global__ __launch_bounds__(kCoreThreads) void block_coreset_kernel(
    const float* __restrict__ own_p, const int32_t* __restrict__ own_sel, int bs, int E, int k, float p,
    int min_c, float* __restrict__ block_scores, int32_t* __restrict__ coreset,
    int32_t* __restrict__ coreset_size) {
  extern __shared__ __align__(16) float lds[];
  const CoreLayout L = core_layout(bs, E, k);
  const int Ep = L.Ep;
  float* S = lds + L.S;
  float* Sv = lds + L.Sv;
  int* order = reinterpret_cast<int*>(lds + L.order);
  float* nzv = lds + L.keys;  // step 2 (the keys come later)
  uint64_t* keys = reinterpret_cast<uint64_t*>(lds + L.keys);
  int* rankc = reinterpret_cast<int*>(lds + L.rankc);
  float* cumv = lds + L.rankc;  // step 6 (the counters are read by then)
  int* wcnt = reinterpret_cast<int*>(lds + L.wcnt);
  float& s_total = lds[L.misc];
  int& s_csize = reinterpret_cast<int*>(lds)[L.misc + 1];
  int& s_nbelow = reinterpret_cast<int*>(lds)[L.misc + 2];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int b = blockIdx.x;
  const float* pb = own_p + static_cast<size_t>(b) * bs * k;
  const int32_t* sb = own_sel + static_cast<size_t>(b) * bs * k;

  // 1. S[e]: the masked sums in token order.  Chunks of tc tokens are
  //    scattered into a dense [tc][Ep] matrix (zero where a token did not
  //    select e, so adding it is exact), then each thread adds its column,
  //    eight rows per batch with all reads first (rows past the chunk are
  //    zero too).
  float* M = lds + L.M;
  if (tid == 0) s_nbelow = 0;
  float acc[kCoreCols] = {0.f, 0.f};
  for (int c0 = 0; c0 < bs; c0 += L.tc) {
    const int nt = min(L.tc, bs - c0);
    const bool has_sel = tid < nt * k;
    const int e_sel = has_sel ? sb[static_cast<size_t>(c0) * k + tid] : 0;
    const float p_sel = has_sel ? pb[static_cast<size_t>(c0) * k + tid] : 0.f;
    for (int i = tid; i < L.tc8 * Ep; i += kCoreThreads) M[i] = 0.f;
    __syncthreads();
    if (has_sel && static_cast<unsigned>(e_sel) < static_cast<unsigned>(E)) M[(tid / k) * Ep + e_sel] = p_sel;
    __syncthreads();
#pragma unroll
    for (int h = 0; h < kCoreCols; ++h) {
      const int e = tid + h * kCoreThreads;
      if (e < Ep)
        for (int t0 = 0; t0 < nt; t0 += 8) {
          float pv[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) pv[u] = M[(t0 + u) * Ep + e];
#pragma unroll
          for (int u = 0; u < 8; ++u) acc[h] += pv[u];
        }
    }
    __syncthreads();  // the next chunk clears M
  }

  // 2. the total, in expert-id order.  Experts that no token selected have
  //    S = +0, which adds nothing exactly, so only the nonzero sums are added
  //    (listed in id order).
  uint64_t m[kCoreCols];
  bool fl[kCoreCols];
#pragma unroll
  for (int h = 0; h < kCoreCols; ++h) {
    const int e = tid + h * kCoreThreads;
    if (e < Ep) S[e] = acc[h];  // padding: 0
    fl[h] = e < E && __float_as_uint(acc[h]) != 0u;
    m[h] = __builtin_amdgcn_ballot_w64(fl[h]);
    if (lane == 0) wcnt[h * kCoreWaves + wave] = __popcll(m[h]);
  }
  __syncthreads();
  int before[kCoreCols] = {0, 0}, nlist = 0;
#pragma unroll
  for (int g = 0; g < kCoreCols * kCoreWaves; ++g) {
    const int c = wcnt[g];
#pragma unroll
    for (int h = 0; h < kCoreCols; ++h) before[h] += g < h * kCoreWaves + wave ? c : 0;
    nlist += c;
  }
#pragma unroll
  for (int h = 0; h < kCoreCols; ++h)
    if (fl[h]) nzv[before[h] + dev::lanes_below(m[h])] = acc[h];
  if (tid < kWave) nzv[nlist + tid] = 0.f;  // exact zeros up to a multiple of 64
  __syncthreads();
  if (tid == 0) {
    // 64 values per round, all 16 reads first, then the chain
    const float4* z4 = reinterpret_cast<const float4*>(nzv);
    float total = 0.f;
    for (int r0 = 0; r0 < nlist; r0 += kWave) {
      float4 q[kWave / 4];
#pragma unroll
      for (int j = 0; j < kWave / 4; ++j) q[j] = z4[r0 / 4 + j];
#pragma unroll
      for (int j = 0; j < kWave / 4; ++j) {
        total += q[j].x;
        total += q[j].y;
        total += q[j].z;
        total += q[j].w;
      }
    }
    s_total = total;
  }
  __syncthreads();

  // 3. Sn in place and each expert's order key (the key of Sn, at least 1).
  //    The experts whose key differs from that of +0 -- those with a positive
  //    Sn -- are listed in id order; the others all share +0's key and so
  //    rank among themselves by id.  A listed expert's 64-bit ranking key is
  //    its order key above the complement of its list index: a larger one
  //    ranks first, so key ties go to the lower index, i.e. the lower id.
  const float total = s_total;
  const uint32_t key0 = max(dev::order_key(0.f), 1u);
  uint32_t kv[kCoreCols];
#pragma unroll
  for (int h = 0; h < kCoreCols; ++h) {
    const int e = tid + h * kCoreThreads;
    float v = 0.f;
    if (e < Ep) {
      v = S[e] / total;
      S[e] = v;
      if (block_scores && e < E) block_scores[static_cast<size_t>(b) * E + e] = v;
    }
    kv[h] = e < E ? max(dev::order_key(v), 1u) : 0u;
    fl[h] = e < E && kv[h] != key0;
    m[h] = __builtin_amdgcn_ballot_w64(fl[h]);
    if (lane == 0) wcnt[h * kCoreWaves + wave] = __popcll(m[h]);
    if (fl[h] && kv[h] < key0) atomicAdd(&s_nbelow, 1);  // below +0: a NaN with its sign bit set
  }
  for (int i = tid; i < Ep; i += kCoreThreads) {
    keys[i] = 0u;  // padding: below every real key, never counted
    rankc[i] = 0;
  }
  __syncthreads();
  nlist = 0;
  int below[kCoreCols] = {0, 0};  // listed experts with a lower id
#pragma unroll
  for (int g = 0; g < kCoreCols * kCoreWaves; ++g) {
    const int c = wcnt[g];
#pragma unroll
    for (int h = 0; h < kCoreCols; ++h) below[h] += g < h * kCoreWaves + wave ? c : 0;
    nlist += c;
  }
#pragma unroll
  for (int h = 0; h < kCoreCols; ++h) {
    below[h] += dev::lanes_below(m[h]);
    if (fl[h]) keys[below[h]] = (static_cast<uint64_t>(kv[h]) << 32) | (0xFFFFFFFFu - static_cast<uint32_t>(below[h]));
  }
  __syncthreads();

  // 4. ranks (Sn desc, id asc): a listed expert counts the listed ranking
  //    keys above its own, `parts` threads per expert over slices of the
  //    list, the counts meeting in LDS.
  {
    const int n2 = (nlist + 1) / 2;  // pairs of keys (the padding key is 0)
    const int parts = nlist > 0 ? max(1, min(8, kCoreThreads / nlist)) : 1;
    const int len = (n2 + parts - 1) / parts;
    const ulonglong2* K2 = reinterpret_cast<const ulonglong2*>(keys);
    for (int idx = tid; idx < nlist * parts; idx += kCoreThreads) {
      const int i = idx / parts, hh = idx - i * parts;
      const uint64_t ki = keys[i];
      const int m1 = min(n2, (hh + 1) * len);
      int r = 0;
#pragma unroll 4
      for (int mm = hh * len; mm < m1; ++mm) {
        const ulonglong2 q = K2[mm];
        r += (q.x > ki ? 1 : 0) + (q.y > ki ? 1 : 0);
      }
      if (r) atomicAdd(&rankc[i], r);
    }
  }
  __syncthreads();

  // 5. the ranked order.  Listed experts above +0's key take their count;
  //    the unlisted ones follow in id order; listed ones below +0's key
  //    (NaNs with the sign bit) come after those.
  {
    const int n_unlisted = E - nlist, n_above = nlist - s_nbelow;
#pragma unroll
    for (int h = 0; h < kCoreCols; ++h) {
      const int e = tid + h * kCoreThreads;
      if (e < E) {
        const int r = fl[h] ? rankc[below[h]] + (kv[h] < key0 ? n_unlisted : 0) : n_above + (e - below[h]);
        order[r] = e;
        Sv[r] = S[e];
      }
    }
    const int e64 = (E + kWave - 1) & ~(kWave - 1);
    if (E + tid < e64) Sv[E + tid] = 0.f;  // the walk adds these exact zeros
  }
  __syncthreads();

  // 6. the Top-P cut: cumulative Sn in rank order reaches p, at least min_c.
  //    Lane 0 of wave 0 adds 64 ranked values per round, in rank order (a
  //    straight chain; entries past E add exact zeros), into LDS; the wave
  //    then finds the first prefix that qualifies with one ballot.
  if (wave == 0) {
    float cum = 0.f;
    int n = 0;
    for (int r0 = 0; r0 < E && n == 0; r0 += kWave) {
      if (lane == 0) {
        // all 16 reads first, then the chain (Sv holds exact zeros from E up
        // to the next multiple of 64)
        const float4* Sv4 = reinterpret_cast<const float4*>(Sv + r0);
        float4* C4 = reinterpret_cast<float4*>(cumv);
        float4 f[kWave / 4];
#pragma unroll
        for (int q = 0; q < kWave / 4; ++q) f[q] = Sv4[q];
#pragma unroll
        for (int q = 0; q < kWave / 4; ++q) {
          float4 o;
          cum += f[q].x;
          o.x = cum;
          cum += f[q].y;
          o.y = cum;
          cum += f[q].z;
          o.z = cum;
          cum += f[q].w;
          o.w = cum;
          C4[q] = o;
        }
      }
      wave_sync();
      const int r = r0 + lane;
      const uint64_t hit = __builtin_amdgcn_ballot_w64(r < E && cumv[lane] >= p && r + 1 >= min_c);
      if (hit) n = r0 + __builtin_ctzll(hit) + 1;  // uniform
      wave_sync();  // every lane has read cumv before lane 0 overwrites it
    }
    if (lane == 0) s_csize = n > 0 ? n : E;
  }
  __syncthreads();
  const int csize = s_csize;
  if (tid == 0) coreset_size[b] = csize;
  for (int i = tid; i < csize; i += kCoreThreads) coreset[static_cast<size_t>(b) * E + i] = order[i];
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
  return E <= 64 * dev::kRadixMaxPerLane && k <= dev::kMaxK && core_layout(bs, E, k).tc >= 1;
}

hipError_t launch_block_topp(const float* probs, int nb, int bs, int E, int k, float p, int min_c,
                             float* block_scores, int32_t* coreset, int32_t* coreset_size, int32_t* experts,
                             float* w, float* gap, hipStream_t s, bool own_done) {
  if (!topp_supported(bs, E, k)) return hipErrorInvalidValue;
  const int T = nb * bs;
  hipError_t err;
  // 1. every token's own top-k, into `experts`, and the selected
  //    probabilities into `w` (both overwritten by step 3; own_done: the
  //    caller's launch already put them there)
  if (!own_done) {
    err = launch_token_topk(probs, T, E, k, experts, w, nullptr, s, true);
    if (err != hipSuccess) return err;
  }
  // 2. one workgroup per block
  block_coreset_kernel<<<nb, kCoreThreads, core_layout(bs, E, k).total * sizeof(float), s>>>(
      w, experts, bs, E, k, p, min_c, block_scores, coreset, coreset_size);
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
