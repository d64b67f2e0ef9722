// The whole block-routed MoE layer forward of ONE block (a decode step of one
// sequence) in three launches.
//
// A decode step's layer is a chain of small dependent phases -- router,
// routing, gate/up, down, combine -- and on gfx950 each kernel boundary costs
// a launch plus a memory round trip to data another XCD wrote, while a
// cross-XCD barrier inside a kernel costs more (cache write-back and
// invalidation).  So the phases are merged where the merge needs no
// synchronisation at all:
//
//  1. router.  Router tiles of 16 tokens x 16 experts over one of up to four
//     slices of the hidden dimension write partial logits (a decode step's
//     router is bound by what each CU can load, so the slices spread it over
//     more CUs); the workgroups of the first expert tile also write x in the
//     chunk-major layout.
//  2. routing + gate/up.  The shared expert needs only x: its workgroups
//     stream its gate/up tiles at once.  Every other workgroup recomputes the block's
//     routing from the logits -- the slices' partial logits added in slice
//     order, softmax of each token row, the block mean
//     in token order, the top-(k+1) by radix selection, the weights -- with
//     the device routines of the routing kernels, so every workgroup reaches
//     the same bits (workgroup (0, 0) writes the routing outputs and the
//     closed-form schedule).  Workgroup (x, j) then streams two packed tiles of
//     the j-th selected expert's gate/up weights over all tokens of the block
//     and stores the SwiGLU activations already multiplied by the token's
//     combine weight, w[t][j] * silu(g) * u, as bf16.
//  3. down + combine.  With every token using the same k experts, the
//     weighted sum over experts of the down projections is ONE product with a
//     reduction over k*I + I_s: y[t] = [Wd_1 .. Wd_k Wsd] [w_1 h_1; ..; w_k
//     h_k; h_s](t).  A workgroup owns 16 output features; wave j reduces over
//     the j-th expert's intermediate units (the last wave over the shared
//     expert's), and the waves' partial tiles are added in wave order, so y
//     is deterministic and there is no per-slot output and no combine launch.
//     With a residual the same epilogue writes res_in + y (the next layer's
//     input) as well.
//
// Activations between the launches are chunk-major over the concatenated
// reduction index: hk[(kk/8)*T + t][kk%8], kk = j*I + i for routed slot j and
// unit i, kk = k*I + i for the shared expert.
#include <algorithm>

#include "ffn_dev.h"
#include "route_dev.h"

namespace dmoe {
namespace {

using fdev::kFrag;

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kTok = 16;  // tokens per MFMA tile
// K-steps of token fragments loaded per chunk: with one or two token tiles
// all 16 steps go out with the weight burst (one memory round trip per
// product); four tiles would not fit in registers, so they take chunks of 4.
template <int NT>
constexpr int kTokChunk = NT <= 2 ? 16 : 4;

struct LayerParams {
  const bf16_t* x;     // [T][H] row-major
  const bf16_t* wr;    // router [E][H]
  const float* bias;   // [E] or nullptr
  const bf16_t* w13;   // routed gate/up, packed
  const bf16_t* w2;    // routed down, packed
  const bf16_t* ws13;  // shared gate/up, packed (nullptr: no shared expert)
  const bf16_t* ws2;   // shared down, packed
  int T, H, E, I, I_s, k;
  float* z;            // [nz][T][E] partial logits without the bias (workspace)
  int nz;              // slices of the hidden dimension in the router (1, 2 or 4)
  bf16_t* xk;          // x chunk-major [H/8][T][8] (output)
  bf16_t* hk;          // activations chunk-major [(k*I + I_s)/8][T][8] (workspace)
  float* logits;       // [T][E] or nullptr
  float* probs;        // [T][E]
  float* block_scores; // [E] or nullptr
  int32_t* experts;    // [k]
  float* cw;           // [T][k]
  float* gap;          // [1] or nullptr
  dmoe_schedule sched;
  void* y;             // [T][H], float32 or bf16
  const bf16_t* res_in;  // [T][H] or nullptr: res_out = bf16(res_in + y), y in fp32
  bf16_t* res_out;
};

// ---- launch 1: router tiles and the shared expert's gate/up -----------------

constexpr int kRouterBurst = 16;  // K-steps of 32 loaded at once per wave
// Slices of the hidden dimension (when H is a multiple of 512): the router's
// workgroups each read half of the bytes of a whole-dimension tile, over
// twice the CUs (a decode step's router is bound by the loads each CU can
// take); the softmax adds the slices' partial logits in slice order.
constexpr int kRouterSlices = 4;
template <int NQ>
constexpr int kSlicesOf = NQ == 1 ? 4 : 2;  // partial rows a softmax lane can hold (E <= 256: 4)
constexpr int router_slices(int H, int E) {  // 8: the router's waves
  const int most = E <= 256 ? 4 : 2;
  return most >= 4 && H % (32 * 8 * 4) == 0 ? 4 : (H % (32 * 8 * 2) == 0 ? 2 : 1);
}

// Logits of 16 tokens x 16 experts over the whole hidden dimension (the four
// waves each reduce a quarter, summed in wave order).  A = x rows (tokens),
// B = router rows (experts): lane (q, c) ends with tokens 4q..4q+3 of expert
// column c.
template <int NW>
__device__ void router_tile(const LayerParams& p, int tile, int slice, f32x4 (*red)[kWave]) {
  const int T = p.T, H = p.H, E = p.E;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, q = lane >> 4, c = lane & 15;
  const int ntt = (T + kTok - 1) / kTok;
  const int tt = tile % ntt, et = tile / ntt;
  const int kq = H / (p.nz * NW), k0 = (slice * NW + wave) * kq, steps = kq / 32;
  const int t = min(tt * kTok + c, T - 1), e = min(et * kTok + c, E - 1);
  const bf16_t* pa = p.x + static_cast<size_t>(t) * H + k0 + q * 8;
  const bf16_t* pb = p.wr + static_cast<size_t>(e) * H + k0 + q * 8;
  const bool write_x = et == 0 && tt * kTok + c < T;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < steps; s0 += kRouterBurst) {
    const int ns = min(kRouterBurst, steps - s0);
    bf16x8 a[kRouterBurst], b[kRouterBurst];
#pragma unroll
    for (int s = 0; s < kRouterBurst; ++s)
      if (s < ns) {
        a[s] = ld_bf16x8(pa + (s0 + s) * 32);
        b[s] = ld_bf16x8(pb + (s0 + s) * 32);
      }
#pragma unroll
    for (int s = 0; s < kRouterBurst; ++s)
      if (s < ns) acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[s], b[s], acc, 0, 0, 0);
    if (write_x) {
#pragma unroll
      for (int s = 0; s < kRouterBurst; ++s)
        if (s < ns) {
          const int j = ((k0 + (s0 + s) * 32) >> 3) + q;  // chunk of 8 features
          *reinterpret_cast<bf16x8*>(p.xk + (static_cast<size_t>(j) * T + tt * kTok + c) * 8) = a[s];
        }
    }
  }
  if (wave > 0) red[wave - 1][lane] = acc;
  __syncthreads();
  if (wave != 0) return;
#pragma unroll
  for (int w = 0; w < NW - 1; ++w) acc += red[w][lane];
  const int ec = et * kTok + c;
  if (ec >= E) return;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int tr = tt * kTok + 4 * q + r;
    if (tr < T) p.z[(static_cast<size_t>(slice) * T + tr) * E + ec] = acc[r];
  }
}

// SwiGLU of one lane's accumulators (g_i, g_i+1, u_i, u_i+1), scaled by w,
// stored as the two bf16 activations of units i, i+1 of token `col`.
__device__ __forceinline__ void store_h(bf16_t* hk, int T, int chunk, int col, int q, const f32x4& v, float w) {
  const uint32_t h0 = f32_to_bf16(silu_f32(v[0]) * v[2] * w);
  const uint32_t h1 = f32_to_bf16(silu_f32(v[1]) * v[3] * w);
  *reinterpret_cast<uint32_t*>(hk + (static_cast<size_t>(chunk) * T + col) * 8 + 2 * q) = h0 | (h1 << 16);
}

// Eight waves split one of the nz slices of the hidden dimension
// (two K-steps each for H = 2048 in four slices).
constexpr int kRouterWaves = 8;
__global__ __launch_bounds__(kRouterWaves * kWave) void layer_router_kernel(LayerParams p) {
  __shared__ f32x4 red[kRouterWaves - 1][kWave];
  router_tile<kRouterWaves>(p, blockIdx.x, blockIdx.y, red);
}

// ---- launch 2: the block's routing, then the routed gate/up ------------------

constexpr int kRoundsMax = dev::kMaxK + 1;

// The first `rounds` of S[0..E) (LDS; E <= kThreads, rounds <= 16) in (score
// desc, id asc) order, by all threads of the workgroup; the same selection
// as dev::wave_topk_radix.  Thread e holds expert e's order key.  A lower
// bound of the rounds-th largest key: the rounds-th largest of the maxima of
// the 16-lane groups (each of those groups holds an element at least that
// large).  Only keys at or above it are candidates, and each candidate's rank
// among them, by (key, id), is its rank in the row.  Called by all threads.
constexpr int kCandMax = kThreads;
__device__ void block_topk_small(const float* S, int E, int rounds, int* sel, float* selv, uint32_t* gmax,
                                 uint32_t* ckey, int* cid, int* wcount) {
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  // excluded threads (e >= E) take key 0, below every real key (real keys >= 1)
  const uint32_t key = tid < E ? max(dev::order_key(S[tid]), 1u) : 0u;
  uint32_t g = key;  // max over the 16 lanes of the row: rotations by 1, 2, 4, 8
  g = max(g, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(g), 0x121, 0xF, 0xF, false)));
  g = max(g, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(g), 0x122, 0xF, 0xF, false)));
  g = max(g, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(g), 0x124, 0xF, 0xF, false)));
  g = max(g, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(g), 0x128, 0xF, 0xF, false)));
  if ((lane & 15) == 0) gmax[tid >> 4] = g;
  __syncthreads();
  if (tid < 16) {  // rank of group tid's maximum among the 16 (ties by group index)
    const uint32_t mine = gmax[tid];
    int r = 0;
#pragma unroll
    for (int i = 0; i < 16; ++i) r += dev::key_before(gmax[i], i, mine, tid) ? 1 : 0;
    if (r == rounds - 1) gmax[16] = mine;
  }
  __syncthreads();
  const uint32_t bound = gmax[16];
  const bool cand = key >= bound && tid < E;
  const uint64_t m = __ballot(cand);
  if (lane == 0) wcount[wave] = __popcll(m);
  __syncthreads();
  int base = 0, ncand = 0;
#pragma unroll
  for (int w = 0; w < kThreads / kWave; ++w) {
    base += w < wave ? wcount[w] : 0;
    ncand += wcount[w];
  }
  if (cand) {
    const int pos = base + dev::lanes_below(m);
    ckey[pos] = key;
    cid[pos] = tid;
  }
  if (tid < 3) {  // pad to a multiple of 4 with entries that rank after everything
    ckey[ncand + tid] = 0u;
    cid[ncand + tid] = dev::kNone;
  }
  __syncthreads();
  if (cand) {
    int r = 0;
    const uint4* k4 = reinterpret_cast<const uint4*>(ckey);
    const int4* i4 = reinterpret_cast<const int4*>(cid);
    for (int i = 0; i < (ncand + 3) / 4; ++i) {
      const uint4 kk = k4[i];
      const int4 ii = i4[i];
      r += (dev::key_before(kk.x, ii.x, key, tid) ? 1 : 0) + (dev::key_before(kk.y, ii.y, key, tid) ? 1 : 0) +
           (dev::key_before(kk.z, ii.z, key, tid) ? 1 : 0) + (dev::key_before(kk.w, ii.w, key, tid) ? 1 : 0);
    }
    if (r < rounds) {
      sel[r] = tid;
      selv[r] = dev::key_value(key);
    }
  }
}

// LDS of the routing prologue (4-byte words): P [T][Es] probabilities, then
// S [Es] block means.  Es = E rounded up to a multiple of 4.
__host__ __device__ inline size_t prologue_words(int T, int E) {
  const size_t Es = static_cast<size_t>(dev::pad4(E));
  return (static_cast<size_t>(T) + 1) * Es;
}

// Softmax of the T logit rows (p.z, plus the bias), max-subtracted, with the
// hardware exp2 on z*log2(e) - m*log2(e) and one reciprocal per row.  Eight
// lanes share a row: lane l of wave w takes row 8*(w + 4*pass) + l/8 and the
// experts 4*(s + 8*i) + c (s = l%8, i < 8*NQ, c < 4), so each of its float4
// loads is one 16-byte piece of a 128-byte run the row's 8 lanes read
// together, and a row's max and sum take three lane exchanges (within the 8
// lanes) instead of six.  A wave handles 8 rows in one pass, all of their
// loads in flight together.  Probabilities go to P (LDS, row stride Es) and,
// for the first workgroup, to probs (and the logits to logits when requested).
template <int NQ, int NPASS>
__device__ void rows_softmax(const LayerParams& p, float* P, int Es, bool first) {
  // E % 4 == 0 (checked by layer_fused_fits): a lane's pieces lie wholly in
  // or past the row, and pieces past it are masked, not branched around, so
  // all loads of a pass are issued before the first wait.
  constexpr int NV = 8 * NQ;  // float4 pieces per lane
  const int T = p.T, E = p.E;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int sl = lane & 7;
  const f32x4 zero4 = {0.f, 0.f, 0.f, 0.f};
  f32x4 b[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) b[i] = zero4;
  if (p.bias) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int e0 = 4 * (sl + 8 * i);
      const f32x4 v = *reinterpret_cast<const f32x4*>(p.bias + min(e0, E - 4));
      b[i] = e0 < E ? v : zero4;
    }
  }
#pragma unroll
  for (int pass = 0; pass < NPASS; ++pass) {
    const int t = 8 * (wave + kWaves * pass) + (lane >> 3);
    const float* src = p.z + static_cast<size_t>(min(t, T - 1)) * E;
    // the second slice (slice 0 again, not added, with one slice): every
    // load is issued before the first wait
    constexpr int NS = kSlicesOf<NQ>;
    f32x4 z[NV], zs[NS - 1][NV];
#pragma unroll
    for (int i = 0; i < NV; ++i) z[i] = *reinterpret_cast<const f32x4*>(src + min(4 * (sl + 8 * i), E - 4));
#pragma unroll
    for (int h = 1; h < NS; ++h) {
      const float* sh = src + static_cast<size_t>(min(h, p.nz - 1)) * T * E;
#pragma unroll
      for (int i = 0; i < NV; ++i) zs[h - 1][i] = *reinterpret_cast<const f32x4*>(sh + min(4 * (sl + 8 * i), E - 4));
    }
#pragma unroll
    for (int h = 1; h < NS; ++h)  // slice order
#pragma unroll
      for (int i = 0; i < NV; ++i) z[i] += h < p.nz ? zs[h - 1][i] : zero4;
    float* lo = first && p.logits && t < T ? p.logits + static_cast<size_t>(t) * E : nullptr;
    float m = -INFINITY;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const bool in = 4 * (sl + 8 * i) < E;
      z[i] += b[i];
#pragma unroll
      for (int c = 0; c < 4; ++c) m = fmaxf(m, in ? z[i][c] : -INFINITY);
    }
    if (lo) {
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        const int e0 = 4 * (sl + 8 * i);
        if (e0 < E) *reinterpret_cast<f32x4*>(lo + e0) = z[i];
      }
    }
    // max over the row's 8 lanes: xor 1, xor 2, then mirror within the 8
    m = fmaxf(m, dev::dppf<dev::kDppXor1>(m, m));
    m = fmaxf(m, dev::dppf<dev::kDppXor2>(m, m));
    m = fmaxf(m, dev::dppf<dev::kDppHalfMirror>(m, m));
    const float ml = m * dev::kLog2e;
    float sum = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const bool in = 4 * (sl + 8 * i) < E;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        z[i][c] = dev::exp2_hw(fmaf(z[i][c], dev::kLog2e, -ml));
        sum += in ? z[i][c] : 0.f;
      }
    }
    sum += dev::dppf<dev::kDppXor1>(sum, sum);
    sum += dev::dppf<dev::kDppXor2>(sum, sum);
    sum += dev::dppf<dev::kDppHalfMirror>(sum, sum);
    const float rs = __builtin_amdgcn_rcpf(sum);
    if (t < T) {
      float* prow = P + static_cast<size_t>(t) * Es;
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        const int e0 = 4 * (sl + 8 * i);
        if (e0 < E) *reinterpret_cast<f32x4*>(prow + e0) = z[i] * rs;
      }
      if (first) {
        float* out = p.probs + static_cast<size_t>(t) * E;
#pragma unroll
        for (int i = 0; i < NV; ++i) {
          const int e0 = 4 * (sl + 8 * i);
          if (e0 < E) *reinterpret_cast<f32x4*>(out + e0) = z[i] * rs;
        }
      }
    }
  }
}

// Workgroups (x, j): slot j < k streams packed tiles kRT*x .. kRT*x+kRT-1 of
// the j-th selected expert; slot j == k (when there is a shared expert)
// streams the shared expert's tiles and needs no routing.
// 16-row weight tiles per wave: two (half the workgroups, so each CU reads
// the token operand once per two tiles) unless four token tiles would not
// fit in registers.
template <int NT>
constexpr int kRTof = NT <= 2 ? 2 : 1;

// The shared expert's gate/up tiles over all T tokens (chunk-major x).
template <int NT>
__device__ void shared_gateup_tiles(const LayerParams& p, int it0, f32x4 (*red)[kRTof<NT>][NT][kWave]) {
  constexpr int kRT = kRTof<NT>;
  const int T = p.T, H = p.H;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, q = lane >> 4, c = lane & 15;
  const int ksteps = H >> 5, steps = ksteps >> 2;
  const bf16_t* pa = p.ws13 + (static_cast<size_t>(it0) * ksteps + wave * steps) * kFrag + lane * 8;
  const int chunk0 = wave * steps * 4 + q;
  const bf16_t* pb[NT];
#pragma unroll
  for (int ct = 0; ct < NT; ++ct) {
    const int tok = min(ct * kTok + c, T - 1);
    pb[ct] = p.xk + (static_cast<size_t>(chunk0) * T + tok) * 8;
  }
  f32x4 acc[kRT][NT];
  fdev::zero(acc);
  fdev::WaveOps<NT, 16, 4, kRT> w;
  fdev::wave_dot<true>(w, pa, static_cast<size_t>(ksteps) * kFrag, pb, 32 * T, steps, acc, false);
  fdev::reduce_waves(acc, red, wave, lane);
  if (wave != 0) return;
#pragma unroll
  for (int r = 0; r < kRT; ++r)
#pragma unroll
    for (int ct = 0; ct < NT; ++ct) {
      const int col = ct * kTok + c;
      if (col < T) store_h(p.hk, T, (p.k * p.I) / 8 + it0 + r, col, q, acc[r][ct], 1.f);
    }
}

template <int NQ, int NT>
__global__ __launch_bounds__(kThreads, 2) void layer_route_gateup_kernel(LayerParams p) {
  extern __shared__ float lds[];
  __shared__ int sel[kRoundsMax];
  __shared__ float selv[kRoundsMax];
  __shared__ float bufv[kRoundsMax];
  __shared__ int bufi[kRoundsMax];
  __shared__ int slds[kWave];
  __shared__ float wslot[NT * kTok];
  __shared__ f32x4 red[kWaves - 1][kRTof<NT>][NT][kWave];
  __shared__ uint32_t gmax[17];
  __shared__ __align__(16) uint32_t ckey[kCandMax + 4];
  __shared__ __align__(16) int cid[kCandMax + 4];
  __shared__ int wcount[kWaves];
  constexpr int kRT = kRTof<NT>;
  const int T = p.T, E = p.E, k = p.k;
  const int Es = dev::pad4(E);
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int it = blockIdx.x * kRT, j = blockIdx.y;
  if (j == k) {  // the shared expert: no routing needed
    if (it * 8 < p.I_s) shared_gateup_tiles<NT>(p, it, red);
    return;
  }
  if (it * 8 >= p.I) return;  // past this expert's tiles (I < I_s)
  const bool first = it == 0 && j == 0;  // writes the routing outputs
  float* P = lds;
  float* S = lds + static_cast<size_t>(T) * Es;

  // 1. softmax of each token row: wave w owns rows w, w + 4, ..., all of
  //    whose loads are issued at once (one memory round trip)
  rows_softmax<NQ, (NT * kTok + 8 * kWaves - 1) / (8 * kWaves)>(p, P, Es, first);
  __syncthreads();

  // 2. block means in token order, 3. top-(k+1) by one wave
  const float n_tok = static_cast<float>(T);
  for (int e = tid; e < E; e += kThreads) {
    const float* pe = P + e;
    float acc = 0.f;
#pragma unroll 8
    for (int t = 0; t < T; ++t) acc += pe[static_cast<size_t>(t) * Es];  // token order
    const float v = acc / n_tok;
    S[e] = v;
    if (first && p.block_scores) p.block_scores[e] = v;
  }
  __syncthreads();
  const int rounds = k < E ? k + 1 : k;
  if (E <= kThreads && rounds <= 16) {
    block_topk_small(S, E, rounds, sel, selv, gmax, ckey, cid, wcount);
  } else if (wave == 0) {
    dev::wave_topk_radix_n<4 * NQ>(S, E, rounds, sel, selv, bufv, bufi);
  }
  __syncthreads();

  // 5. packed tile `it` of expert sel[j]'s gate/up over all tokens
  const int H = p.H, q = lane >> 4, c = lane & 15;
  const int ksteps = H >> 5, steps = ksteps >> 2;
  const bf16_t* W = p.w13 + static_cast<size_t>(sel[j]) * 2 * p.I * H;
  const bf16_t* pa = W + (static_cast<size_t>(it) * ksteps + wave * steps) * kFrag + lane * 8;
  const int chunk0 = wave * steps * 4 + q;
  const bf16_t* pb[NT];
#pragma unroll
  for (int ct = 0; ct < NT; ++ct) {
    const int tok = min(ct * kTok + c, T - 1);
    pb[ct] = p.xk + (static_cast<size_t>(chunk0) * T + tok) * 8;
  }
  f32x4 acc[kRT][NT];
  fdev::zero(acc);
  fdev::WaveOps<NT, 16, 4, kRT> w;
  fdev::wave_dot<true>(w, pa, static_cast<size_t>(ksteps) * kFrag, pb, 32 * T, steps, acc, false);

  // 6. the routing outputs (workgroup (0, 0), while the other workgroups
  //    stream): the selection, gap, every token's combine weights (its
  //    probabilities on the selection, renormalised, summed in slot order) and
  //    the closed-form schedule
  if (first) {
    for (int i = tid; i < T * k; i += kThreads) {
      const int t = i / k, jj = i - t * k;
      const float* prow = P + static_cast<size_t>(t) * Es;
      float denom = 0.f;
      for (int j2 = 0; j2 < k; ++j2) denom += prow[sel[j2]];
      p.cw[i] = prow[sel[jj]] / denom;
    }
    for (int jj = tid; jj < k; jj += kThreads) p.experts[jj] = sel[jj];
    if (p.gap && tid == 0) p.gap[0] = k < E ? selv[k - 1] - selv[k] : INFINITY;
    dev::schedule_one_group(sel, T, k, slds, p.sched);  // all threads; synchronises
  }
  // 7. slot j's combine weight of every token, a quarter of the tokens per
  //    wave (read by wave 0 after the barrier of the reduction)
  {
    constexpr int kPer = NT * kTok / kWaves;  // tokens per wave
    const int t = wave * kPer + lane;
    if (lane < kPer && t < T) {
      const float* prow = P + static_cast<size_t>(t) * Es;
      float denom = 0.f;
#pragma unroll 8
      for (int j2 = 0; j2 < k; ++j2) denom += prow[sel[j2]];  // slot order
      wslot[t] = prow[sel[j]] / denom;
    }
  }
  fdev::reduce_waves(acc, red, wave, lane);
  if (wave != 0) return;
  // 8. SwiGLU scaled by the weights
#pragma unroll
  for (int r = 0; r < kRT; ++r)
#pragma unroll
    for (int ct = 0; ct < NT; ++ct) {
      const int col = ct * kTok + c;
      if (col < T) store_h(p.hk, T, (j * p.I) / 8 + it + r, col, q, acc[r][ct], wslot[col]);
    }
}

// ---- launch 3: down projection of every expert and the combine ---------------

// Waves of the down kernel: k routed experts + the shared expert, at most 12
// (three waves per SIMD leave each wave room for a 16-step weight burst).
constexpr int kMaxSegments = 12;

__device__ __forceinline__ void store_y(float* y, const f32x4& v) { *reinterpret_cast<f32x4*>(y) = v; }
__device__ __forceinline__ void store_y(bf16_t* y, const f32x4& v) {
  const uint32_t lo = f32_to_bf16(v[0]) | (static_cast<uint32_t>(f32_to_bf16(v[1])) << 16);
  const uint32_t hi = f32_to_bf16(v[2]) | (static_cast<uint32_t>(f32_to_bf16(v[3])) << 16);
  *reinterpret_cast<uint2*>(y) = make_uint2(lo, hi);
}

// Workgroup = one packed down tile jt (16 output features) x one tile of 16
// tokens; wave j < k reduces over slot j's expert, wave k (when present) over
// the shared expert.  Grid index tt * (H/16) + jt: the token tiles of one
// feature tile are dispatched to the same XCD (H/16 is a multiple of the 8
// XCDs), so their second read of the tile's weights is served by its L2.
template <typename OutT>
__global__ __launch_bounds__(kMaxSegments * kWave) void layer_down_combine_kernel(LayerParams p) {
  constexpr int NT = 1;
  __shared__ f32x4 red[kMaxSegments - 1][NT][kWave];
  const int T = p.T, H = p.H, k = p.k;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, q = lane >> 4, c = lane & 15;
  const int nw = blockDim.x >> 6;
  const int jt = blockIdx.x % (H / 16), tt = blockIdx.x / (H / 16);
  const bool shared = wave == k;
  const int Kd = shared ? p.I_s : p.I;
  const int ksteps = Kd >> 5;
  // token operand first (it does not depend on the routing), then the expert
  const int chunk0 = (wave * p.I) / 8 + q;  // wave == k: the shared block starts at k*I
  const bf16_t* pb[NT];
#pragma unroll
  for (int ct = 0; ct < NT; ++ct) {
    const int tok = min((tt + ct) * kTok + c, T - 1);
    pb[ct] = p.hk + (static_cast<size_t>(chunk0) * T + tok) * 8;
  }
  const bf16_t* W = shared ? p.ws2 : p.w2 + static_cast<size_t>(p.experts[wave]) * H * p.I;
  const bf16_t* pa = W + static_cast<size_t>(jt) * ksteps * kFrag + lane * 8;
  // the residual's four inputs of this lane (wave 0 writes the outputs),
  // loaded before the product so that their latency is hidden
  uint2 rin[NT];
#pragma unroll
  for (int ct = 0; ct < NT; ++ct) {
    rin[ct] = make_uint2(0u, 0u);
    const int tok = min((tt + ct) * kTok + c, T - 1);
    if (p.res_out && wave == 0)
      rin[ct] = *reinterpret_cast<const uint2*>(p.res_in + static_cast<size_t>(tok) * H + jt * 16 + 4 * q);
  }
  f32x4 acc[1][NT];
  fdev::zero(acc);
  fdev::WaveOps<NT, 16, kTokChunk<NT>, 1> w;
  fdev::wave_dot<true>(w, pa, 0, pb, 32 * T, ksteps, acc, false);
  if (wave > 0) {
#pragma unroll
    for (int ct = 0; ct < NT; ++ct) red[wave - 1][ct][lane] = acc[0][ct];
  }
  __syncthreads();
  if (wave != 0) return;
  for (int ww = 0; ww < nw - 1; ++ww)
#pragma unroll
    for (int ct = 0; ct < NT; ++ct) acc[0][ct] += red[ww][ct][lane];  // wave order
  OutT* y = static_cast<OutT*>(p.y);
#pragma unroll
  for (int ct = 0; ct < NT; ++ct) {
    const int col = (tt + ct) * kTok + c;
    if (col >= T) continue;
    store_y(y + static_cast<size_t>(col) * H + jt * 16 + 4 * q, acc[0][ct]);
    if (p.res_out) {
      const f32x4 r = {bf16_to_f32(static_cast<bf16_t>(rin[ct].x & 0xFFFFu)),
                       bf16_to_f32(static_cast<bf16_t>(rin[ct].x >> 16)),
                       bf16_to_f32(static_cast<bf16_t>(rin[ct].y & 0xFFFFu)),
                       bf16_to_f32(static_cast<bf16_t>(rin[ct].y >> 16))};
      store_y(p.res_out + static_cast<size_t>(col) * H + jt * 16 + 4 * q, r + acc[0][ct]);
    }
  }
}

template <int NT>
hipError_t launch_nt(const LayerParams& p, dmoe_dtype y_dt, hipStream_t s) {
  const int n_router = ((p.T + kTok - 1) / kTok) * ((p.E + kTok - 1) / kTok);
  layer_router_kernel<<<dim3(n_router, p.nz), kRouterWaves * kWave, 0, s>>>(p);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  const size_t lds = prologue_words(p.T, p.E) * sizeof(float);
  const dim3 gu_grid(std::max(p.I, p.ws13 ? p.I_s : 0) / (8 * kRTof<NT>), p.k + (p.ws13 ? 1 : 0));
  if (p.E <= 256)
    layer_route_gateup_kernel<1, NT><<<gu_grid, kThreads, lds, s>>>(p);
  else
    layer_route_gateup_kernel<2, NT><<<gu_grid, kThreads, lds, s>>>(p);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  const int waves = p.k + (p.ws13 ? 1 : 0);
  const unsigned down_grid = (p.H / 16) * ((p.T + kTok - 1) / kTok);
  if (y_dt == DMOE_F32)
    layer_down_combine_kernel<float><<<down_grid, waves * kWave, 0, s>>>(p);
  else
    layer_down_combine_kernel<bf16_t><<<down_grid, waves * kWave, 0, s>>>(p);
  return hipGetLastError();
}

}  // namespace

bool layer_fused_fits(dmoe_dtype dt, int n_blocks, int T, int H, int E, int I, int I_s, int k) {
  if (dt != DMOE_BF16 || n_blocks != 1) return false;
  if (T < 1 || T > 4 * kTok || E > dev::kRegSoftmaxMaxE || k > dev::kMaxK) return false;
  if (k + (I_s > 0 ? 1 : 0) > kMaxSegments) return false;
  if (H % (32 * kRouterWaves) || I % 128 || I_s % 128 || E % 4) return false;
  return prologue_words(T, E) * sizeof(float) <= 48 * 1024;
}

size_t layer_fused_workspace_bytes(int T, int E, int I, int I_s, int k) {
  const size_t z = (static_cast<size_t>(kRouterSlices) * T * E * sizeof(float) + 255) & ~static_cast<size_t>(255);
  return z + (static_cast<size_t>(k) * I + I_s) * T * sizeof(bf16_t);
}

hipError_t launch_layer_fused(const LayerArgs& a, hipStream_t s) {
  const size_t zb = (static_cast<size_t>(kRouterSlices) * a.T * a.E * sizeof(float) + 255) & ~static_cast<size_t>(255);
  LayerParams p{static_cast<const bf16_t*>(a.x), static_cast<const bf16_t*>(a.w_router), a.bias,
                static_cast<const bf16_t*>(a.w13), static_cast<const bf16_t*>(a.w2),
                static_cast<const bf16_t*>(a.ws13), static_cast<const bf16_t*>(a.ws2), a.T, a.H, a.E, a.I, a.I_s,
                a.k, static_cast<float*>(a.workspace), router_slices(a.H, a.E),
                static_cast<bf16_t*>(a.x_chunked),
                reinterpret_cast<bf16_t*>(static_cast<char*>(a.workspace) + zb), a.logits, a.probs, a.block_scores,
                a.experts, a.combine_w, a.gap, a.sched, a.y, static_cast<const bf16_t*>(a.res_in),
                static_cast<bf16_t*>(a.res_out)};
  if (a.T <= kTok) return launch_nt<1>(p, a.y_dt, s);
  if (a.T <= 2 * kTok) return launch_nt<2>(p, a.y_dt, s);
  return launch_nt<4>(p, a.y_dt, s);
}

}  // namespace dmoe
