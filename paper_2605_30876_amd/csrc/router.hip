// Router scores s_i = Router(t_i) (Sec. 4.2): linear router + softmax over
// all experts.
//
// bf16: logits = x Wr^T on the matrix cores (v_mfma_f32_16x16x32_bf16, fp32
// accumulation; a bf16 x bf16 product is exact in fp32).  A workgroup owns a
// 32-token x 32-expert tile of one of S slices of the hidden dimension; its
// four waves split the slice in quarters and issue all their operand loads
// at once, and the partial tiles are summed in wave order through LDS.  With
// few tokens (a decode step) the hidden dimension is split over S <= 4
// workgroups so that more CUs share the router matrix; the S partial logits
// go to the workspace and the softmax sums them in slice order, so the result
// does not depend on scheduling.
// f32: one thread per (token, expert) dot product.
// Softmax: one wave per token row; all partial loads of a pass are issued
// together and the row is staged in LDS (one read pass, one write pass).
// Optionally the kernel also stores x in the chunk-major layout the expert
// FFN reads ([H/c][T][c], c elements per 16-byte chunk): the workgroups of the
// first expert tile already hold every 16-byte chunk of x in registers.
// Larger forwards (T >= 256) use LDS-staged tiles of up to 128 tokens x 64
// experts instead (router_tile_bf16_kernel): far fewer re-reads of x and the
// router matrix, and whole-line loads.
#include <algorithm>
#include <type_traits>

#include "route_dev.h"

namespace dmoe {
namespace {

using dev::kMaxSplits;

constexpr int kRouterTile = 32;
constexpr int kRouterSteps = 8;  // K steps of 32 per load burst

__global__ __launch_bounds__(256) void router_logits_bf16_kernel(
    const bf16_t* __restrict__ x, const bf16_t* __restrict__ w, int T, int H, int E, int S,
    float* __restrict__ part, bf16_t* __restrict__ xk) {
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int q = lane >> 4;   // k-group of the MFMA operand / row group of the result
  const int c = lane & 15;   // row of A (token) / column of B (expert)
  const int t0 = blockIdx.x * kRouterTile;
  const int e0 = blockIdx.y * kRouterTile;
  const int slice = H / S;
  const int kw = slice >> 2;
  const int kbeg = blockIdx.z * slice + wave * kw;
  const int steps = kw >> 5;

  const bf16_t* pa[2];
  const bf16_t* pb[2];
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    // ragged token / expert tails: clamp the rows read, skip the writes
    const int t = min(t0 + r * 16 + c, T - 1);
    const int e = min(e0 + r * 16 + c, E - 1);
    pa[r] = x + static_cast<size_t>(t) * H + kbeg + q * 8;
    pb[r] = w + static_cast<size_t>(e) * H + kbeg + q * 8;
  }
  f32x4 acc[2][2];
#pragma unroll
  for (int r = 0; r < 2; ++r)
#pragma unroll
    for (int s = 0; s < 2; ++s) acc[r][s] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int sc = 0; sc < steps; sc += kRouterSteps) {
    const int ns = min(kRouterSteps, steps - sc);
    bf16x8 a[kRouterSteps][2], b[kRouterSteps][2];
#pragma unroll
    for (int s = 0; s < kRouterSteps; ++s)
      if (s < ns)
#pragma unroll
        for (int r = 0; r < 2; ++r) {
          a[s][r] = ld_bf16x8(pa[r] + (sc + s) * 32);
          b[s][r] = ld_bf16x8(pb[r] + (sc + s) * 32);
        }
#pragma unroll
    for (int s = 0; s < kRouterSteps; ++s)
      if (s < ns)
#pragma unroll
        for (int r = 0; r < 2; ++r)
#pragma unroll
          for (int u = 0; u < 2; ++u)
            acc[r][u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[s][r], b[s][u], acc[r][u], 0, 0, 0);
    if (xk && blockIdx.y == 0) {
      // chunk (kbeg + 32*(sc+s))/8 + q of token t0 + 16r + c
#pragma unroll
      for (int s = 0; s < kRouterSteps; ++s)
        if (s < ns)
#pragma unroll
          for (int r = 0; r < 2; ++r) {
            const int t = t0 + r * 16 + c;
            const int j = ((kbeg + (sc + s) * 32) >> 3) + q;
            if (t < T)
              *reinterpret_cast<bf16x8*>(xk + (static_cast<size_t>(j) * T + t) * 8) = a[s][r];
          }
    }
  }

  __shared__ f32x4 red[3][4][kWave];
  if (wave > 0) {
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
      for (int s = 0; s < 2; ++s) red[wave - 1][r * 2 + s][lane] = acc[r][s];
  }
  __syncthreads();
  if (wave != 0) return;
  float* out = part + static_cast<size_t>(blockIdx.z) * T * E;
#pragma unroll
  for (int r = 0; r < 2; ++r) {
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      f32x4 v = acc[r][s];
#pragma unroll
      for (int ww = 0; ww < 3; ++ww) v += red[ww][r * 2 + s][lane];
      const int e = e0 + s * 16 + c;
      if (e >= E) continue;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = t0 + r * 16 + q * 4 + i;
        if (t < T) out[static_cast<size_t>(t) * E + e] = v[i];
      }
    }
  }
}

// ---- larger forwards: LDS-staged tiles -------------------------------------
//
// A workgroup owns TT tokens x TE experts of one of S slices of the hidden
// dimension.  Each stage of 64 reduction elements is loaded with whole-line
// loads (eight threads per 128-byte piece of a row) into a double-buffered
// LDS stage, from which every wave reads its matrix-core fragments.  Loading
// the fragments straight from the row-major x and router matrix touches 16
// rows x 64 bytes per instruction, which caps the L2 -> CU rate, and a
// 32 x 32 tile re-reads x once per 32 experts and the router matrix once per
// 32 tokens.  The global loads run RING - 1 stages ahead of the matrix work
// through a ring of registers (one stage of matrix work is far shorter than
// a memory round trip).  The waves split the tile (never the reduction), so each output is
// one accumulator summed over the slice in ascending order.
constexpr int kStageK = 64;           // reduction elements per LDS stage
constexpr int kLdsRow = kStageK + 8;  // bf16 per LDS row (16 bytes of padding against bank conflicts)
template <int TT, int TE, int RING = 4>
__global__ __launch_bounds__(256) void router_tile_bf16_kernel(
    const bf16_t* __restrict__ x, const bf16_t* __restrict__ w, int T, int H, int E, int S,
    float* __restrict__ part, bf16_t* __restrict__ xk) {
  constexpr int TTt = TT / 16, TEt = TE / 16;           // 16 x 16 output tiles
  constexpr int WT = TTt < 4 ? TTt : 4, WE = 4 / WT;    // waves along tokens / experts
  constexpr int NTw = TTt / WT, NEw = TEt / WE;         // output tiles per wave
  constexpr int XP = TT * 8 / 256, WP = TE * 8 / 256;   // 16-byte pieces per thread per stage
  static_assert(NTw * WT == TTt && NEw * WE == TEt && XP >= 1 && WP >= 1, "tile shape");
  static_assert(RING == 4 || RING == 8, "register ring");
  __shared__ __align__(16) bf16_t lx[2][TT][kLdsRow];
  __shared__ __align__(16) bf16_t lw[2][TE][kLdsRow];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, q = lane >> 4, c = lane & 15;
  const int t0 = blockIdx.x * TT, e0 = blockIdx.y * TE;
  const int slice = H / S, kbeg = blockIdx.z * slice, nst = slice / kStageK;
  // loader: piece i of a stage is row pr + 32 i, elements 8 pc .. 8 pc + 7
  // (ragged token / expert tails: the rows read are clamped, the writes skipped)
  const int pr = tid >> 3, pc = tid & 7;
  const bf16_t* px[XP];
  const bf16_t* pw[WP];
#pragma unroll
  for (int i = 0; i < XP; ++i)
    px[i] = x + static_cast<size_t>(min(t0 + pr + 32 * i, T - 1)) * H + kbeg + pc * 8;
#pragma unroll
  for (int i = 0; i < WP; ++i)
    pw[i] = w + static_cast<size_t>(min(e0 + pr + 32 * i, E - 1)) * H + kbeg + pc * 8;
  const int ny = gridDim.y, ey = blockIdx.y;  // x chunk-major: stage st is written by expert tile st % ny
  bf16x8 rx[RING][XP], rw[RING][WP];
  // stages past the last reload the last one (straight-line loads keep the
  // compiler's memory-counter waits exact); they are never stored
  auto load = [&](int st, bf16x8 (&ax)[XP], bf16x8 (&aw)[WP]) {
    st = min(st, nst - 1);
#pragma unroll
    for (int i = 0; i < XP; ++i) ax[i] = ld_bf16x8(px[i] + st * kStageK);
#pragma unroll
    for (int i = 0; i < WP; ++i) aw[i] = ld_bf16x8(pw[i] + st * kStageK);
  };
  auto store = [&](int buf, int st, const bf16x8 (&ax)[XP], const bf16x8 (&aw)[WP]) {
#pragma unroll
    for (int i = 0; i < XP; ++i) *reinterpret_cast<bf16x8*>(&lx[buf][pr + 32 * i][pc * 8]) = ax[i];
#pragma unroll
    for (int i = 0; i < WP; ++i) *reinterpret_cast<bf16x8*>(&lw[buf][pr + 32 * i][pc * 8]) = aw[i];
    if (xk && st % ny == ey) {  // uniform; every expert tile writes a share
      const int j = ((kbeg + st * kStageK) >> 3) + pc;  // chunk of 8 features
#pragma unroll
      for (int i = 0; i < XP; ++i) {
        const int t = t0 + pr + 32 * i;
        if (t < T) *reinterpret_cast<bf16x8*>(xk + (static_cast<size_t>(j) * T + t) * 8) = ax[i];
      }
    }
  };
  const int wt = wave % WT, we = wave / WT;
  f32x4 acc[NTw][NEw];
#pragma unroll
  for (int i = 0; i < NTw; ++i)
#pragma unroll
    for (int j = 0; j < NEw; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int r = 0; r < RING - 1; ++r) load(r, rx[r], rw[r]);
  store(0, 0, rx[0], rw[0]);
  __syncthreads();
  // Stage st: register slot st % RING (a compile-time index: RING stages per
  // trip).  Its loads went out RING - 1 stages earlier; the slot it frees
  // takes the loads of stage st + RING - 1.  LDS buffer st & 1 is stored
  // again two stages later, after the barrier that ends every wave's reads.
  auto run_stage = [&](auto slot, int st) {
    constexpr int R = decltype(slot)::value;
    load(st + RING - 1, rx[(R + RING - 1) % RING], rw[(R + RING - 1) % RING]);
    const int buf = st & 1;
#pragma unroll
    for (int s = 0; s < kStageK / 32; ++s) {
      bf16x8 a[NTw], b[NEw];
#pragma unroll
      for (int i = 0; i < NTw; ++i)
        a[i] = *reinterpret_cast<const bf16x8*>(&lx[buf][(wt * NTw + i) * 16 + c][32 * s + 8 * q]);
#pragma unroll
      for (int j = 0; j < NEw; ++j)
        b[j] = *reinterpret_cast<const bf16x8*>(&lw[buf][(we * NEw + j) * 16 + c][32 * s + 8 * q]);
#pragma unroll
      for (int i = 0; i < NTw; ++i)
#pragma unroll
        for (int j = 0; j < NEw; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    if (st + 1 < nst) store(buf ^ 1, st + 1, rx[(R + 1) % RING], rw[(R + 1) % RING]);
    __syncthreads();
  };
  for (int st = 0; st < nst; st += RING) {
    run_stage(std::integral_constant<int, 0>{}, st);
    if (st + 1 < nst) run_stage(std::integral_constant<int, 1>{}, st + 1);
    if (st + 2 < nst) run_stage(std::integral_constant<int, 2>{}, st + 2);
    if (st + 3 < nst) run_stage(std::integral_constant<int, 3>{}, st + 3);
    if constexpr (RING == 8) {
      if (st + 4 < nst) run_stage(std::integral_constant<int, 4 % RING>{}, st + 4);
      if (st + 5 < nst) run_stage(std::integral_constant<int, 5 % RING>{}, st + 5);
      if (st + 6 < nst) run_stage(std::integral_constant<int, 6 % RING>{}, st + 6);
      if (st + 7 < nst) run_stage(std::integral_constant<int, 7 % RING>{}, st + 7);
    }
  }
  // lane (q, c) holds tokens 4q .. 4q+3 of expert column c of each output tile
  float* out = part + static_cast<size_t>(blockIdx.z) * T * E;
#pragma unroll
  for (int j = 0; j < NEw; ++j) {
    const int e = e0 + (we * NEw + j) * 16 + c;
    if (e >= E) continue;
#pragma unroll
    for (int i = 0; i < NTw; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = t0 + (wt * NTw + i) * 16 + 4 * q + r;
        if (t < T) out[static_cast<size_t>(t) * E + e] = acc[i][j][r];
      }
  }
}

// fp32 router: grid (ceil(E / 16), T).  Wave w of a workgroup computes the
// logits of experts 16*bx + w, + 4, ... for token t: each lane accumulates
// the features h = lane, lane + 64, ... of x[t] . w[e] (coalesced row reads),
// then the wave sums its lanes in a fixed order (dev::wave_sum).
constexpr int kF32RouterExperts = 16;

__global__ __launch_bounds__(256) void router_logits_f32_kernel(
    const float* __restrict__ x, const float* __restrict__ w, int T, int H, int E,
    float* __restrict__ part, float* __restrict__ xk) {
  const int t = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const float* xr = x + static_cast<size_t>(t) * H;
  if (xk && blockIdx.x == 0)
    for (int h = threadIdx.x; h < H; h += blockDim.x) xk[(static_cast<size_t>(h >> 2) * T + t) * 4 + (h & 3)] = xr[h];
  const int e1 = min(E, static_cast<int>(blockIdx.x + 1) * kF32RouterExperts);
  for (int e = blockIdx.x * kF32RouterExperts + wave; e < e1; e += 4) {
    const float* wr = w + static_cast<size_t>(e) * H;
    float acc = 0.f;
    for (int h = lane; h < H; h += kWave) acc = fmaf(xr[h], wr[h], acc);
    acc = dev::wave_sum(acc);
    if (lane == 0) part[static_cast<size_t>(t) * E + e] = acc;
  }
}

// One wave per token row, four rows per workgroup.  Up to 512 experts the
// row is reduced in registers (dev::softmax_loaded, the routine the fused
// routing kernel uses); wider rows are staged in LDS (dynamic: 4*E floats).
// part may alias probs (S == 1): a row is read whole before it is written.
template <int NQ>
__global__ __launch_bounds__(256) void softmax_rows_reg_kernel(const float* part, int S,
                                                               const float* __restrict__ bias, int T, int E,
                                                               float* probs, float* logits) {
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  dev::RowPartials<NQ> r[1];
  dev::load_row<NQ>(part, static_cast<size_t>(T) * E, S, bias, E, t, r[0]);
  const bool live[1] = {true};
  float* const out[1] = {probs + static_cast<size_t>(t) * E};
  float* const lds[1] = {nullptr};
  float* const lo[1] = {logits ? logits + static_cast<size_t>(t) * E : nullptr};
  dev::softmax_loaded<NQ, 1>(r, live, S, bias != nullptr, E, out, lds, lo);
}

__global__ __launch_bounds__(256) void softmax_rows_kernel(const float* part, int S,
                                                           const float* __restrict__ bias, int T,
                                                           int E, float* probs, float* logits) {
  extern __shared__ float zrow[];
  const int wave = threadIdx.x >> 6;
  const int t = blockIdx.x * 4 + wave;
  if (t >= T) return;
  dev::softmax_row(part + static_cast<size_t>(t) * E, static_cast<size_t>(T) * E, S, bias, E,
                   zrow + static_cast<size_t>(wave) * E, probs + static_cast<size_t>(t) * E,
                   logits ? logits + static_cast<size_t>(t) * E : nullptr);
}

// Launch shape of the bf16 router.  Smaller forwards: 32 x 32 tiles, the
// hidden dimension in enough slices (multiples of 128) to spread the router
// matrix over about half the CUs.  T >= 256: LDS-staged tiles of tt tokens x
// te experts in S slices, the shape with the fewest bytes moved (x once per
// expert tile, the router matrix once per token tile, the partial planes
// written and read back) among those with at least 256 workgroups (one per
// CU), else the one with the most workgroups.
struct RouterShape {
  bool tiled;
  int tt;  // tokens per workgroup
  int te;  // experts per workgroup
  int S;   // slices of the hidden dimension
};

constexpr int kTiledMinT = 256;

RouterShape router_shape(int T, int H, int E) {
  if (T < kTiledMinT) {
    const long tiles = static_cast<long>((T + kRouterTile - 1) / kRouterTile) * ((E + kRouterTile - 1) / kRouterTile);
    int S = 1;
    while (S < kMaxSplits && tiles * S < 128 && (H / 128) % (2 * S) == 0) S *= 2;
    return {false, kRouterTile, kRouterTile, S};
  }
  RouterShape best{true, 32, 32, 1};
  long best_wg = -1;
  double best_bytes = 0;
  for (int tt : {128, 64, 32})
    for (int te : {64, 32})
      for (int S = 1; S <= kMaxSplits && H % S == 0 && (H / S) % kStageK == 0; S *= 2) {
        const long nt = (T + tt - 1) / tt, ne = (E + te - 1) / te, wg = nt * ne * S;
        const double bytes = 2.0 * H * (static_cast<double>(T) * ne + static_cast<double>(E) * nt) +
                             (S > 1 ? 8.0 * S * T * E : 0.0);
        const bool full = wg >= 256, best_full = best_wg >= 256;
        const bool better = full != best_full ? full
                            : full        ? bytes < best_bytes
                                          : (wg > best_wg || (wg == best_wg && bytes < best_bytes));
        if (better) {
          best = {true, tt, te, S};
          best_wg = wg;
          best_bytes = bytes;
        }
      }
  return best;
}
}  // namespace

size_t router_workspace_bytes(int T, int H, int E, dmoe_dtype dt) {
  if (dt != DMOE_BF16) return 0;
  const int S = router_shape(T, H, E).S;
  return S > 1 ? static_cast<size_t>(S) * T * E * sizeof(float) : 0;
}

hipError_t launch_router_partials(const void* x, const void* w, dmoe_dtype dt, int T, int H, int E,
                                  float* probs, void* x_chunked, void* workspace, size_t ws_bytes,
                                  hipStream_t s, float** part_out, int* S_out) {
  int S = 1;
  float* part = probs;  // S == 1: the logits go to probs, read back in place by the softmax
  if (dt == DMOE_BF16) {
    const RouterShape rs = router_shape(T, H, E);
    const size_t need = router_workspace_bytes(T, H, E, dt);
    if (need > 0 && workspace && ws_bytes >= need) {
      S = rs.S;
      part = static_cast<float*>(workspace);
    }
    const bf16_t* xb = static_cast<const bf16_t*>(x);
    const bf16_t* wb = static_cast<const bf16_t*>(w);
    bf16_t* xkb = static_cast<bf16_t*>(x_chunked);
    if (rs.tiled) {
      const dim3 grid((T + rs.tt - 1) / rs.tt, (E + rs.te - 1) / rs.te, S);
#define DMOE_ROUTER_TILE(TT_, TE_)                                                          \
  if (rs.tt == TT_ && rs.te == TE_)                                                         \
    router_tile_bf16_kernel<TT_, TE_><<<grid, 256, 0, s>>>(xb, wb, T, H, E, S, part, xkb); \
  else
      DMOE_ROUTER_TILE(128, 64)
      DMOE_ROUTER_TILE(128, 32)
      DMOE_ROUTER_TILE(64, 64)
      DMOE_ROUTER_TILE(64, 32)
      DMOE_ROUTER_TILE(32, 64)
      // the smallest tile has the fewest loads per stage: a deeper ring
      // (measured 11.4 -> 10.3 us at 256 tokens, hidden 4096)
      router_tile_bf16_kernel<32, 32, 8><<<grid, 256, 0, s>>>(xb, wb, T, H, E, S, part, xkb);
#undef DMOE_ROUTER_TILE
    } else {
      dim3 grid((T + kRouterTile - 1) / kRouterTile, (E + kRouterTile - 1) / kRouterTile, S);
      router_logits_bf16_kernel<<<grid, 256, 0, s>>>(xb, wb, T, H, E, S, part, xkb);
    }
  } else {
    dim3 grid((E + kF32RouterExperts - 1) / kF32RouterExperts, T);
    router_logits_f32_kernel<<<grid, 256, 0, s>>>(static_cast<const float*>(x),
                                                   static_cast<const float*>(w), T, H, E, part,
                                                   static_cast<float*>(x_chunked));
  }
  *part_out = part;
  *S_out = S;
  return hipGetLastError();
}

hipError_t launch_router(const void* x, const void* w, const float* bias, dmoe_dtype dt, int T,
                         int H, int E, float* logits, float* probs, void* x_chunked,
                         void* workspace, size_t ws_bytes, hipStream_t s) {
  float* part = nullptr;
  int S = 1;
  hipError_t err = launch_router_partials(x, w, dt, T, H, E, probs, x_chunked, workspace, ws_bytes, s,
                                          &part, &S);
  if (err != hipSuccess) return err;
  const unsigned blocks = (T + 3) / 4;
  if (E <= 256) {
    softmax_rows_reg_kernel<1><<<blocks, 256, 0, s>>>(part, S, bias, T, E, probs, logits);
  } else if (E <= dev::kRegSoftmaxMaxE) {
    softmax_rows_reg_kernel<2><<<blocks, 256, 0, s>>>(part, S, bias, T, E, probs, logits);
  } else {
    const size_t lds = static_cast<size_t>(4) * E * sizeof(float);
    softmax_rows_kernel<<<blocks, 256, lds, s>>>(part, S, bias, T, E, probs, logits);
  }
  return hipGetLastError();
}

}  // namespace dmoe
