// The routing stage of one forward: router scores (Sec. 4.2), expert
// selection (block routing, Sec. 4.2 aggregation and Alg. 1 with a coreset
// of size k; or the token-level baseline), combine weights and the
// unique-expert schedule.
//
// A decode step routes few tokens; its routing kernels are bound by memory
// round trips (each kernel boundary adds a write, a cache flush and a re-read
// from another XCD), not by arithmetic.  When the forward's logits fit in
// LDS (T*E <= 8192), everything after the router runs in ONE workgroup with a
// single round trip: all partial logits are loaded at once, then softmax
// rows (into LDS), block sums, radix-select top-k per block, combine weights
// and the schedule run on chip.  (Token routing has T rows to select; spread
// over T/4 workgroups it is faster, so it runs the softmax and each token's
// selection in one launch of T/4 workgroups, then the schedule.)  The
// arithmetic is that of
// the separate kernels (same device routines, same summation orders), so the
// results are bit-identical to dmoe_router_logits +
// dmoe_block_aggregate_topk / dmoe_token_topk + dmoe_build_expert_schedule.
// Larger forwards chain those kernels.
#include "route_dev.h"

namespace dmoe {
namespace {

constexpr int kThreads = dev::kSchedThreads;  // the schedule's workgroup size
constexpr int kWaves = kThreads / kWave;
constexpr int kFusedMaxTE = 8192;                   // logits of the forward kept in LDS
constexpr size_t kMaxLdsBytes = 64 * 1024 - 1024;   // headroom for static LDS

// LDS words of the fused kernel (4-byte words; rows padded to a multiple of 4
// floats for 128-bit reads).
struct FusedLayout {
  int Es;  // padded row stride
  size_t sb, sel, selv, expc, bufv, bufi, sched, total;
};

__host__ __device__ inline FusedLayout fused_layout(int T, int E, int k, int G) {
  FusedLayout L;
  L.Es = (E + 3) & ~3;
  L.sb = static_cast<size_t>(T) * L.Es;                        // P [T][Es]
  L.sel = L.sb + static_cast<size_t>(G) * L.Es;                // S [G][Es]
  L.selv = L.sel + static_cast<size_t>(G) * (k + 1);           // sel [G][k+1]
  L.expc = L.selv + static_cast<size_t>(G) * (k + 1);          // selv [G][k+1]
  L.bufv = L.expc + static_cast<size_t>(G) * k;                // expert lists [G][k]
  L.bufi = L.bufv + static_cast<size_t>(kWaves) * (k + 1);     // per-wave top-k gather
  L.sched = (L.bufi + static_cast<size_t>(kWaves) * (k + 1) + 3) & ~static_cast<size_t>(3);  // 16-byte aligned
  L.total = L.sched + dev::schedule_lds_ints(E);               // schedule scratch
  return L;
}

constexpr int kWBatch = 8;  // selected probabilities of a token loaded together

// kPerBlock: workgroup b routes block b alone (T = gs rows of the forward's
// T_all; the partial planes keep T_all rows) and the schedule is left to a
// launch of its own.
template <int NQ, bool kPerBlock = false>
__global__ __launch_bounds__(kThreads) void route_small_kernel(
    const float* part, int S, const float* __restrict__ bias, int T, int E, int k, int gs,
    float* probs, float* __restrict__ logits, float* __restrict__ block_scores,
    int32_t* __restrict__ experts, float* __restrict__ cw, float* __restrict__ gap,
    dmoe_schedule sched, int T_all) {
  extern __shared__ float lds[];
  if (kPerBlock) {
    const size_t b = blockIdx.x;
    part += b * gs * E;
    probs += b * gs * E;
    if (logits) logits += b * gs * E;
    if (block_scores) block_scores += b * E;
    experts += b * k;
    cw += b * gs * k;
    if (gap) gap += b;
  }
  const int G = T / gs;
  const int K1 = k + 1;
  const FusedLayout L = fused_layout(T, E, k, G);
  const int Es = L.Es;
  float* P = lds;
  float* Sb = lds + L.sb;
  int* sel = reinterpret_cast<int*>(lds + L.sel);
  float* selv = lds + L.selv;
  int* expc = reinterpret_cast<int*>(lds + L.expc);
  const int tid = threadIdx.x, wave = tid >> 6;
  float* bufv = lds + L.bufv + wave * K1;
  int* bufi = reinterpret_cast<int*>(lds + L.bufi) + wave * K1;
  int* slds = reinterpret_cast<int*>(lds + L.sched);

  // 1. router softmax: wave w owns rows w, w + 8, ...; a batch of RB rows
  //    has all of its partial loads in flight together, then each row is
  //    reduced in registers into probs and P.  (part may alias probs: a row
  //    is read only by the wave that writes it, before it writes it.)
  {
    constexpr int RB = 4 / NQ;
    const size_t plane = static_cast<size_t>(T_all) * E;
    for (int t0 = wave; t0 < T; t0 += kWaves * RB) {
      dev::RowPartials<NQ> r[RB];
#pragma unroll
      for (int u = 0; u < RB; ++u) {
        const int t = t0 + u * kWaves;
        if (t < T) dev::load_row<NQ>(part, plane, S, bias, E, t, r[u]);
      }
      bool live[RB];
      float* out[RB];
      float* prow[RB];
      float* lo[RB];
#pragma unroll
      for (int u = 0; u < RB; ++u) {
        const int t = min(t0 + u * kWaves, T - 1);
        live[u] = t0 + u * kWaves < T;
        out[u] = probs + static_cast<size_t>(t) * E;
        prow[u] = P + static_cast<size_t>(t) * Es;
        lo[u] = logits ? logits + static_cast<size_t>(t) * E : nullptr;
      }
      dev::softmax_loaded<NQ, RB>(r, live, S, bias != nullptr, E, out, prow, lo);
    }
  }
  __syncthreads();

  // 2. selection: block means in token order, then sel[b][0..rounds) in
  //    (score desc, id asc) order, one wave per block by radix selection
  const int rounds = k < E ? K1 : k;
  const float n_tok = static_cast<float>(gs);
  for (int i = tid; i < G * E; i += kThreads) {
    const int b = i / E, e = i - b * E;
    const float* pb = P + static_cast<size_t>(b) * gs * Es + e;
    float acc = 0.f;
#pragma unroll 8
    for (int t = 0; t < gs; ++t) acc += pb[static_cast<size_t>(t) * Es];  // token order
    const float v = acc / n_tok;
    Sb[static_cast<size_t>(b) * Es + e] = v;
    if (block_scores) block_scores[i] = v;
  }
  __syncthreads();
  for (int b = wave; b < G; b += kWaves)
    dev::wave_topk_radix_n<4 * NQ>(Sb + static_cast<size_t>(b) * Es, E, rounds, sel + b * K1, selv + b * K1, bufv,
                                   bufi);
  __syncthreads();

  // 3. expert lists, gaps, and every token's weights renormalised over its
  //    group's selection (summed in slot order)
  for (int i = tid; i < G * k; i += kThreads) {
    const int g = i / k, j = i - g * k;
    const int e = sel[g * K1 + j];
    experts[i] = e;
    expc[i] = e;
  }
  if (gap)
    for (int g = tid; g < G; g += kThreads) gap[g] = k < E ? selv[g * K1 + k - 1] - selv[g * K1 + k] : INFINITY;
  // one thread per (token, slot); each sums its token's k values in slot order
  for (int i = tid; i < T * k; i += kThreads) {
    const int t = i / k, j = i - t * k;
    const int g = t / gs;
    const float* prow = P + static_cast<size_t>(t) * Es;
    const int* sg = sel + g * K1;
    float denom = 0.f;
    for (int j0 = 0; j0 < k; j0 += kWBatch) {
      float v[kWBatch];
#pragma unroll
      for (int u = 0; u < kWBatch; ++u)
        if (j0 + u < k) v[u] = prow[sg[j0 + u]];
#pragma unroll
      for (int u = 0; u < kWBatch; ++u)
        if (j0 + u < k) denom += v[u];
    }
    cw[i] = prow[sg[j]] / denom;
  }
  __syncthreads();

  // 4. unique-expert schedule of the G expert lists (one block: closed form)
  if (kPerBlock) return;
  if (G == 1 && k <= kWave)
    dev::schedule_one_group(expc, gs, k, slds, sched);
  else
    dev::schedule_wg(expc, G, gs, k, E, slds, sched);
}

}  // namespace

bool route_fused_fits(int T, int E, int k, int gs, bool block) {
  // Token routing selects T rows serially per wave on one CU, slower than the
  // separate kernels spread over T/4 workgroups: only block routing is fused.
  if (!block) return false;
  if (E > dev::kRegSoftmaxMaxE || k > dev::kMaxK) return false;
  if (static_cast<long>(T) * E > kFusedMaxTE) return false;
  return fused_layout(T, E, k, T / gs).total * sizeof(float) <= kMaxLdsBytes;
}

// One workgroup per block when a block's rows fit in LDS.
static bool route_block_fits(int gs, int E, int k, bool block) {
  if (!block) return false;
  if (E > dev::kRegSoftmaxMaxE || k > dev::kMaxK) return false;
  return fused_layout(gs, E, k, 1).total * sizeof(float) <= kMaxLdsBytes;
}

// Alg. 1 with the Top-P coreset: the router, every token's own top-k (with
// the softmax in one launch when the router's partial logits allow it), the
// coreset of each block, each token's top-k inside it, then the token-level
// schedule.
static hipError_t launch_route_topp(const RouteArgs& a, dmoe_dtype dt, hipStream_t s) {
  hipError_t err;
  bool own_done = false;
  if (dt == DMOE_BF16 && softmax_token_topk_fits(a.E)) {
    float* part = nullptr;
    int S = 1;
    err = launch_router_partials(a.x, a.w, dt, a.T, a.H, a.E, a.probs, a.x_chunked, a.workspace, a.ws_bytes, s,
                                 &part, &S);
    if (err != hipSuccess) return err;
    err = launch_softmax_token_topk(part, S, a.bias, a.T, a.E, a.k, a.probs, a.logits, a.experts, a.combine_w,
                                    nullptr, s, true);  // the selected probabilities, for the coreset
    own_done = true;
  } else {
    err = launch_router(a.x, a.w, a.bias, dt, a.T, a.H, a.E, a.logits, a.probs, a.x_chunked, a.workspace,
                        a.ws_bytes, s);
  }
  if (err != hipSuccess) return err;
  err = launch_block_topp(a.probs, a.T / a.gs, a.gs, a.E, a.k, a.top_p, a.min_coreset, a.block_scores, a.coreset,
                          a.coreset_size, a.experts, a.combine_w, a.gap, s, own_done);
  if (err != hipSuccess) return err;
  return launch_schedule(a.experts, a.T, 1, a.k, a.E, a.sched, s);
}

hipError_t launch_route(const RouteArgs& a, dmoe_dtype dt, hipStream_t s) {
  if (a.topp) return launch_route_topp(a, dt, s);
  const int G = a.block ? a.T / a.gs : a.T;
  if (route_fused_fits(a.T, a.E, a.k, a.gs, a.block)) {
    float* part = nullptr;
    int S = 1;
    hipError_t err = launch_router_partials(a.x, a.w, dt, a.T, a.H, a.E, a.probs, a.x_chunked, a.workspace,
                                            a.ws_bytes, s, &part, &S);
    if (err != hipSuccess) return err;
    const size_t lds = fused_layout(a.T, a.E, a.k, G).total * sizeof(float);
    if (a.E <= 256)
      route_small_kernel<1><<<1, kThreads, lds, s>>>(part, S, a.bias, a.T, a.E, a.k, a.gs, a.probs, a.logits,
                                                     a.block_scores, a.experts, a.combine_w, a.gap, a.sched, a.T);
    else
      route_small_kernel<2><<<1, kThreads, lds, s>>>(part, S, a.bias, a.T, a.E, a.k, a.gs, a.probs, a.logits,
                                                     a.block_scores, a.experts, a.combine_w, a.gap, a.sched, a.T);
    return hipGetLastError();
  }
  if (route_block_fits(a.gs, a.E, a.k, a.block)) {
    // larger block-routed forwards: one workgroup per block (softmax rows,
    // block mean, top-k, weights), then the schedule
    float* part = nullptr;
    int S = 1;
    hipError_t err = launch_router_partials(a.x, a.w, dt, a.T, a.H, a.E, a.probs, a.x_chunked, a.workspace,
                                            a.ws_bytes, s, &part, &S);
    if (err != hipSuccess) return err;
    const size_t lds = fused_layout(a.gs, a.E, a.k, 1).total * sizeof(float);
    if (a.E <= 256)
      route_small_kernel<1, true><<<G, kThreads, lds, s>>>(part, S, a.bias, a.gs, a.E, a.k, a.gs, a.probs,
                                                           a.logits, a.block_scores, a.experts, a.combine_w,
                                                           a.gap, a.sched, a.T);
    else
      route_small_kernel<2, true><<<G, kThreads, lds, s>>>(part, S, a.bias, a.gs, a.E, a.k, a.gs, a.probs,
                                                           a.logits, a.block_scores, a.experts, a.combine_w,
                                                           a.gap, a.sched, a.T);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
    return launch_schedule(a.experts, G, a.gs, a.k, a.E, a.sched, s);
  }
  hipError_t err;
  if (!a.block && dt == DMOE_BF16 && softmax_token_topk_fits(a.E)) {
    // token routing: the softmax and each token's selection in one launch
    float* part = nullptr;
    int S = 1;
    err = launch_router_partials(a.x, a.w, dt, a.T, a.H, a.E, a.probs, a.x_chunked, a.workspace, a.ws_bytes, s,
                                 &part, &S);
    if (err != hipSuccess) return err;
    err = launch_softmax_token_topk(part, S, a.bias, a.T, a.E, a.k, a.probs, a.logits, a.experts, a.combine_w,
                                    a.gap, s);
    if (err != hipSuccess) return err;
    return launch_schedule(a.experts, G, 1, a.k, a.E, a.sched, s);
  }
  err = launch_router(a.x, a.w, a.bias, dt, a.T, a.H, a.E, a.logits, a.probs, a.x_chunked, a.workspace,
                      a.ws_bytes, s);
  if (err != hipSuccess) return err;
  if (a.block)
    err = launch_block_topk(a.probs, G, a.gs, a.E, a.k, a.block_scores, a.experts, a.combine_w, a.gap, s);
  else
    err = launch_token_topk(a.probs, a.T, a.E, a.k, a.experts, a.combine_w, a.gap, s);
  if (err != hipSuccess) return err;
  return launch_schedule(a.experts, G, a.block ? a.gs : 1, a.k, a.E, a.sched, s);
}

}  // namespace dmoe
