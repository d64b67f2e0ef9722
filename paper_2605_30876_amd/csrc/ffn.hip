// Expert execution: the SwiGLU FFN of every unique expert of the forward over
// the rows that selected it, plus the always-on shared expert over all tokens.
//
//   h    = silu(Wg x) * (Wu x)        gate/up kernel -> h rows (workspace)
//   out  = Wd h                       down kernel    -> slot_out[t][j] / shared_out[t]
//
// Work items: max_work grid rows for the schedule's work items (up to
// DMOE_WORK_ROWS rows of one routed expert; rows past n_work exit at once)
// and rows for the shared expert's T tokens cut into pieces of
// DMOE_WORK_ROWS.  One-tile launches (schedules of many small items, whose
// max_work bound is loose) put the shared pieces first so that the rows that
// exit at once are dispatched last; the others put them last (measured
// faster for block-routed decode steps).  A decode workgroup owns one or two
// 16-row weight tiles of one item, streams them from HBM and applies them to
// the item's rows (tokens); a tile workgroup owns 64 or 128 weight rows and
// up to 128 tokens.  Each selected expert's weights are read once per forward
// per piece of its rows.
//
// bf16 path (matrix cores, v_mfma_f32_16x16x32_bf16, fp32 accumulation):
//  * A operand = weight rows, B operand = token rows, C = [weight row][token].
//  * A gate/up tile interleaves the gate and up rows of 8 intermediate units,
//    so a lane's four accumulators are (g_i, g_i+1, u_i, u_i+1) of one token
//    and SwiGLU is applied in registers.
//  * Tiles of 16 weight rows give many small workgroups: a burst of weight
//    reads spread over several workgroups per CU keeps every HBM channel busy
//    and the CUs evenly loaded (32-row tiles left a third of the bandwidth
//    unused on small forwards).
//  * The four waves of a workgroup split the reduction dimension in quarters.
//    Each wave issues all of its weight loads at once (one burst per up to
//    KMAX 32-wide K steps), with the token operand double-buffered in chunks
//    behind it; partial tiles are summed in wave order through LDS, so
//    results do not depend on scheduling.
//  * Operand layouts are chosen so that consecutive lanes read consecutive
//    memory: weights are pre-packed in fragment order (a wave's load of one
//    16 x 32 tile is 1 KiB contiguous, its burst a contiguous run), and token
//    rows (x, and the h rows between the two kernels) are chunk-major
//    [K/8][rows][8], so 16 consecutive rows read 256 contiguous bytes per
//    8-element chunk.  Lane (q, c) of a K-step holds chunk 4*step + q of its
//    row in both operands, which is all the matrix instruction needs.
//    Scattered token rows (token-level routing) may instead be read from the
//    row-major x, one 64-byte piece per token and K-step (tile_gathered).
// f32 path: reduction-major weights, each lane one output unit, the waves
// splitting the reduction (small fp32 layers).
#include <algorithm>
#include <type_traits>

#include "dmoe_common.h"
#include "ffn_dev.h"

namespace dmoe {
namespace {

constexpr int kThreads = 256;

struct Group {
  int r0;          // first row of the item in the row space (h buffer row)
  int n;           // rows (tokens) in the item
  int expert;      // routed expert id, or -1 for the shared expert
  const int* tok;  // token of each row (routed), or nullptr: row c is token t0 + c
  int t0;
  int piece;       // index of the item among its expert's items (0, 1, ...)
};

// Grid row y: the schedule's max_work items, then the shared expert's pieces
// (kSharedFirst: the pieces first).  One memory round trip: the item count
// and the item are loaded together (the index stays inside the work array;
// an item past n_work is loaded but not used).  An item naming an expert
// outside [0, E) is skipped, so no schedule can steer a weight read outside
// the expert arrays.
template <bool kSharedFirst = false>
__device__ __forceinline__ bool decode_item(int y, int shared_items, int max_work, const int* n_work,
                                            const int* work, const int* row_token, int T, int Tk, int E, Group& g) {
  const int w = kSharedFirst ? y - shared_items : y;
  if (kSharedFirst ? w >= 0 : w < max_work) {
    const int nw = *n_work;
    const int4 it = reinterpret_cast<const int4*>(work)[w];
    g.expert = it.x;
    g.r0 = it.y;
    g.n = (w < nw && static_cast<unsigned>(it.x) < static_cast<unsigned>(E)) ? it.z : 0;
    g.tok = row_token + it.y;
    g.t0 = 0;
    g.piece = it.w;
  } else {
    const int c = kSharedFirst ? y : y - max_work;
    g.expert = -1;
    g.piece = c;
    g.t0 = c * DMOE_WORK_ROWS;
    g.r0 = Tk + g.t0;
    g.n = min(DMOE_WORK_ROWS, T - g.t0);
    g.tok = nullptr;
  }
  return g.n > 0;
}

// ---- bf16 kernels ----------------------------------------------------------

// Which copy of x serves a token tile's B loads better.  Lane (q, c) of
// each 16-lane row holds the token of column c (ascending within an item).
// Per K-step the chunk-major copy touches 4 * D8 cache lines (D8: distinct
// groups of 8 consecutive tokens among the 16; one group per line and chunk),
// the row-major copy D lines (D: distinct tokens, one 64-byte piece each).
// Tiles of fewer than 4 distinct tokens stay chunk-major (measured slightly
// faster there: 32-token decode steps under token routing).  Wave-uniform.
__device__ __forceinline__ bool tile_gathered(int tok) {
  // token of lane c - 1 in the same row (lane c = 0 sees its own)
  const int prev = __builtin_amdgcn_update_dpp(tok, tok, 0x111, 0xF, 0xF, false);  // row_shr:1
  const uint32_t new_tok = static_cast<uint32_t>(__builtin_amdgcn_ballot_w64(tok != prev)) & 0xFFFFu;
  const uint32_t new_grp = static_cast<uint32_t>(__builtin_amdgcn_ballot_w64((tok >> 3) != (prev >> 3))) & 0xFFFFu;
  const int d = 1 + __builtin_popcount(new_tok), d8 = 1 + __builtin_popcount(new_grp);
  return d >= 4 && d < 4 * d8;
}

struct FfnParams {
  const bf16_t* xk;    // activations, chunk-major [H/8][T][8]
  const bf16_t* xr;    // the same row-major [T][H] (gathered rows read it), or nullptr
  const bf16_t* w13;   // routed gate/up, fragment-packed
  const bf16_t* w2;    // routed down, fragment-packed
  const bf16_t* ws13;  // shared gate/up, fragment-packed
  const bf16_t* ws2;   // shared down, fragment-packed
  const int* n_work;
  const int* work;
  const int* row_token;
  const int* row_slot;
  int T, H, E, I, I_s, k, Tk, R, max_work;  // R: rows of the h buffer
  int shared_items;                        // grid rows of the shared expert's pieces (0: none)
  bf16_t* hk;                              // SwiGLU activations, chunk-major [ldh/8][R][8]
  void* slot_out;                          // [T][k][H], float32 or scaled half (slot_f16s)
  float* shared_out;
  int slot_f16s;
};

// Four consecutive outputs j0 .. j0+3 of schedule row r (token row_token[r],
// slot row_slot[r]) into the slot outputs, float32 or scaled half with the
// exponent e of their 16-feature group (written by the group's lane j0 % 16
// == 0).
__device__ __forceinline__ void store_slot(const FfnParams& p, int r, int j0, const f32x4& v, int e) {
  const size_t row = static_cast<size_t>(p.row_token[r]) * p.k + p.row_slot[r];
  if (p.slot_f16s) {
    uint16_t* hv = static_cast<uint16_t*>(p.slot_out);
    *reinterpret_cast<uint2*>(hv + row * p.H + j0) = f16s_encode(v, e);
    if ((j0 & 15) == 0) {
      int8_t* ev = reinterpret_cast<int8_t*>(hv + static_cast<size_t>(p.T) * p.k * p.H);
      ev[row * (p.H >> 4) + (j0 >> 4)] = static_cast<int8_t>(e);
    }
  } else {
    *reinterpret_cast<f32x4*>(static_cast<float*>(p.slot_out) + row * p.H + j0) = v;
  }
}

// The shared exponent of the 16-feature group a lane's outputs belong to
// (scaled-half slot outputs only; 0 otherwise).  All 64 lanes call it.
__device__ __forceinline__ int slot_exponent(const FfnParams& p, const f32x4& v) {
  return p.slot_f16s ? f16s_exponent(f16s_group_max(v)) : 0;
}

using namespace fdev;  // the wave-level operand helpers of ffn_dev.h

// Occupancy floors (waves per SIMD) for the two-tile variants, which serve
// block-routed decode steps: 3 (gate/up and down) keep every workgroup of
// such a launch resident at once instead of leaving a second partial round.
// grid (ldh / (8 RT), groups): packed gate/up tiles it .. it + RT - 1, tile
// `it` = 8 intermediate units.
// Wave w reduces over hidden chunks [w*H/32, (w+1)*H/32) (K-steps
// [w*H/128, (w+1)*H/128)).
template <int NT, int KMAX, int BC, int MINW, bool kSharedFirst, int RT>
__global__ __launch_bounds__(kThreads, MINW) void ffn_gateup_bf16_kernel(FfnParams p) {
  Group g;
  if (!decode_item<kSharedFirst>(blockIdx.y, p.shared_items, p.max_work, p.n_work, p.work, p.row_token, p.T,
                                 p.Tk, p.E, g))
    return;
  const int Iw = g.expert >= 0 ? p.I : p.I_s;
  const int it = blockIdx.x * RT;  // first of the RT packed tiles (Iw / 8 is a multiple of 16)
  if (it * 8 >= Iw) return;
  const int H = p.H;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int q = lane >> 4, c = lane & 15;
  const int ksteps = H >> 5, steps = ksteps >> 2;
  const bf16_t* W = g.expert >= 0 ? p.w13 + static_cast<size_t>(g.expert) * 2 * p.I * H : p.ws13;
  const bf16_t* pa = W + (static_cast<size_t>(it) * ksteps + wave * steps) * kFrag + lane * 8;
  const size_t tstride = static_cast<size_t>(ksteps) * kFrag;  // next packed tile
  const int bstep = 32 * p.T;  // 4 chunks of T tokens per K-step
  const int chunk0 = wave * steps * 4 + q;

  __shared__ f32x4 red[3][RT][NT][kWave];
  WaveOps<NT, KMAX, BC, RT> w;  // a one-burst weight slice stays here across passes
  // At two token tiles (items of whole blocks) a one-burst slice is loaded
  // before the token rows are known: the weights wait only for the work
  // item, not for its row list and then x.  With one token tile (many small
  // items) the token fragments going first measured faster.
  bool a_held = false;
  if constexpr (NT == 2) {
    if (steps <= KMAX) {
      issue_a<true>(w, pa, tstride, steps);
      a_held = true;
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  for (int p0 = 0; p0 < g.n; p0 += 16 * NT) {
    const bf16_t* pb[NT];
    int tok[NT];
    bool gathered = false;
#pragma unroll
    for (int ct = 0; ct < NT; ++ct) {
      const int col = min(p0 + ct * 16 + c, g.n - 1);
      tok[ct] = g.tok ? g.tok[col] : g.t0 + col;
      if (p.xr && g.tok) gathered |= tile_gathered(tok[ct]);
    }
#pragma unroll
    for (int ct = 0; ct < NT; ++ct)
      pb[ct] = gathered ? p.xr + static_cast<size_t>(tok[ct]) * H + chunk0 * 8
                        : p.xk + (static_cast<size_t>(chunk0) * p.T + tok[ct]) * 8;
    f32x4 acc[RT][NT];
    zero(acc);
    wave_dot<true>(w, pa, tstride, pb, gathered ? 32 : bstep, steps, acc, a_held || (p0 > 0 && steps <= KMAX));
    reduce_waves(acc, red, wave, lane);
    if (wave == 0) {
#pragma unroll
      for (int r = 0; r < RT; ++r)
#pragma unroll
        for (int ct = 0; ct < NT; ++ct) {
          const int col = p0 + ct * 16 + c;
          if (col < g.n) {
            // accumulators: (g_i, g_i+1, u_i, u_i+1) with i = 8*(it + r) + 2q
            const f32x4 v = acc[r][ct];
            const uint32_t h0 = f32_to_bf16(silu_f32(v[0]) * v[2]);
            const uint32_t h1 = f32_to_bf16(silu_f32(v[1]) * v[3]);
            bf16_t* dst = p.hk + (static_cast<size_t>(it + r) * p.R + g.r0 + col) * 8 + 2 * q;
            *reinterpret_cast<uint32_t*>(dst) = h0 | (h1 << 16);
          }
        }
    }
    __syncthreads();  // red is reused by the next pass
  }
}

// grid (H / (16 RT), groups): packed down tiles jt .. jt + RT - 1, tile `jt`
// = 16 output features.
template <int NT, int KMAX, int BC, int MINW, bool kSharedFirst, int RT>
__global__ __launch_bounds__(kThreads, MINW) void ffn_down_bf16_kernel(FfnParams p) {
  Group g;
  if (!decode_item<kSharedFirst>(blockIdx.y, p.shared_items, p.max_work, p.n_work, p.work, p.row_token, p.T,
                                 p.Tk, p.E, g))
    return;
  const int Kd = g.expert >= 0 ? p.I : p.I_s;
  const int H = p.H;
  const int jt = blockIdx.x * RT;  // first of the RT packed tiles (H / 16 is a multiple of 8)
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int q = lane >> 4, c = lane & 15;
  const int ksteps = Kd >> 5, steps = ksteps >> 2;
  const bf16_t* W = g.expert >= 0 ? p.w2 + static_cast<size_t>(g.expert) * H * p.I : p.ws2;
  const bf16_t* pa = W + (static_cast<size_t>(jt) * ksteps + wave * steps) * kFrag + lane * 8;
  const size_t tstride = static_cast<size_t>(ksteps) * kFrag;  // next packed tile
  const int bstep = 32 * p.R;
  const int chunk0 = wave * steps * 4 + q;

  __shared__ f32x4 red[3][RT][NT][kWave];
  WaveOps<NT, KMAX, BC, RT> w;  // a one-burst weight slice stays here across passes
  for (int p0 = 0; p0 < g.n; p0 += 16 * NT) {
    const bf16_t* pb[NT];
#pragma unroll
    for (int ct = 0; ct < NT; ++ct) {
      const int col = min(p0 + ct * 16 + c, g.n - 1);
      pb[ct] = p.hk + (static_cast<size_t>(chunk0) * p.R + g.r0 + col) * 8;
    }
    f32x4 acc[RT][NT];
    zero(acc);
    wave_dot<true>(w, pa, tstride, pb, bstep, steps, acc, p0 > 0 && steps <= KMAX);
    reduce_waves(acc, red, wave, lane);
    if (wave == 0) {
#pragma unroll
      for (int ct = 0; ct < NT; ++ct) {
        const int col = p0 + ct * 16 + c;
        int ex[RT];
#pragma unroll
        for (int r = 0; r < RT; ++r) ex[r] = g.tok ? slot_exponent(p, acc[r][ct]) : 0;  // whole wave
        if (col < g.n) {
          if (g.tok) {
#pragma unroll
            for (int r = 0; r < RT; ++r) store_slot(p, g.r0 + col, (jt + r) * 16 + 4 * q, acc[r][ct], ex[r]);
          } else {
            float* dst = p.shared_out + static_cast<size_t>(g.t0 + col) * H;
#pragma unroll
            for (int r = 0; r < RT; ++r) *reinterpret_cast<f32x4*>(dst + (jt + r) * 16 + 4 * q) = acc[r][ct];
          }
        }
      }
    }
    __syncthreads();
  }
}

// Workgroups are dispatched to the 8 XCDs round-robin by linear id, and each
// XCD has its own L2.  The 1-D grid of gx * items8 workgroups (gx row blocks
// per item, items8: the grid rows rounded up to a multiple of 8) is mapped
// onto the schedule's live items (the first n_work, then the shared
// expert's) so that each item's row blocks run on S XCDs: its token rows
// enter S L2 caches.  Schedules of many live items (>= 256: thousands of
// tokens, whose token rows per XCD copy cost about as much traffic as the
// weights) take S = 1; the others S = 8 (every XCD shares every item's
// work, the most even load; measured faster for 16 blocks of 32 tokens and
// for the Zipf-biased large layer).  With S = 1, XCD x runs a contiguous
// run of ceil(live / 8) items, one item (all its row blocks) after the
// other: the items of one expert are adjacent in the schedule, so its pieces
// run back to back on one XCD and share that L2's copy of its weights.  With
// S > 1, XCD x of group x / S runs row blocks x % S, x % S + S, ... of the
// group's items (an expert's pieces again meet on the XCDs of each row
// block).
__device__ __forceinline__ bool map_item(const FfnParams& p, int gx, int& item, int& rb) {
  const int nw = min(*p.n_work, p.max_work);
  const int live = nw + p.shared_items;
  const int S = min(live >= 256 ? 1 : 8, gx & -gx);  // a power of two dividing gx
  const int x = blockIdx.x & 7, slot = blockIdx.x >> 3;
  int j;
  if (S == 1) {
    const int q = (live + 7) >> 3, i = slot / gx;  // q items per XCD
    rb = slot % gx;
    if (i >= q) return false;
    j = x * q + i;
  } else {
    const int per = gx / S;  // row blocks of an item on each of its XCDs
    j = (slot / per) * (8 / S) + x / S;
    rb = x % S + S * (slot % per);
  }
  if (j >= live) return false;
  item = j < nw ? j : p.max_work + (j - nw);
  return true;
}

// ---- tile kernels: many tokens per work item --------------------------------
//
// A workgroup covers 4 * kRowTiles (one or two) 16-row weight tiles (wave w: packed tiles
// kRowTiles * (4*bx + w) + m, m < kRowTiles, over the whole reduction) x up
// to 128 tokens of one work item (8 token tiles).  The reduction runs in
// stages of kStageSteps K-steps: the stage's token fragments are loaded from
// global memory once per workgroup into a double-buffered LDS stage read by
// all four waves, each fragment read once per wave and applied to the
// wave's kRowTiles weight tiles, while each wave streams its own weight tiles
// into registers two stages ahead (HBM latency spans more than one stage's
// matrix work).  Accumulation order (K ascending) and the epilogues match the
// decode kernels.
constexpr int kTileTok = 8;       // token tiles per workgroup (128 tokens)
constexpr int kStageSteps = 2;    // K-steps per LDS stage (two: 32 KB of LDS, three workgroups per CU)
static_assert(kTileTok * 16 == DMOE_WORK_ROWS, "a tile workgroup covers one work item's rows");

// The workgroup's work once its item is known (kStream: weights loaded
// non-temporally).
template <bool kGateUp, int kRowTiles, bool kStream>
__device__ __forceinline__ void tile_body(const FfnParams& p, const Group& g, int bx,
                                          bf16x8 (&stage)[2][kStageSteps][kTileTok][kWave]) {
  constexpr int kTileRows = 4 * kRowTiles;  // weight tiles per workgroup
  const int H = p.H;
  const int Iw = g.expert >= 0 ? p.I : p.I_s;
  const int Kd = kGateUp ? H : Iw;                    // reduction length
  const int tiles = kGateUp ? Iw / 8 : H / 16;        // packed 16-row tiles of the matrix
  if (bx * kTileRows >= tiles) return;  // uniform: past the matrix
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  // tiles % kTileRows == 0 (H, I, I_s multiples of 128)
  const int tile0 = (bx * 4 + wave) * kRowTiles;
  const int ksteps = Kd >> 5;                         // multiple of kStageSteps
  const bf16_t* W;
  if (kGateUp)
    W = g.expert >= 0 ? p.w13 + static_cast<size_t>(g.expert) * 2 * p.I * H : p.ws13;
  else
    W = g.expert >= 0 ? p.w2 + static_cast<size_t>(g.expert) * H * p.I : p.ws2;
  const bf16_t* pa = W + static_cast<size_t>(tile0) * ksteps * kFrag + lane * 8;
  const size_t tstride = static_cast<size_t>(ksteps) * kFrag;  // next packed tile
  const int nt = (g.n + 15) >> 4;  // live token tiles

  // Token-fragment producer: thread t loads pieces (tile t/64, lane t%64) and
  // (tile t/64 + 4, same lane) of every K-step of a stage.  Tiles past the
  // item's last token load its last row again (straight-line code; those
  // fragments are never used).
  const int tid = threadIdx.x;
  const int pl = tid & 63, pq = pl >> 4, pc = pl & 15;
  const int pct = __builtin_amdgcn_readfirstlane(tid >> 6);  // the wave (uniform)
  const int rows_b = kGateUp ? p.T : p.R;  // rows of the chunk-major source
  const bf16_t* src = kGateUp ? p.xk : p.hk;
  const bf16_t* pb[2];
  int row[2];
  bool gathered = false;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int ct = pct + 4 * h;
    const int col = min(ct * 16 + pc, g.n - 1);
    if (kGateUp) {
      row[h] = g.tok ? g.tok[col] : g.t0 + col;
      if (p.xr && g.tok) gathered |= tile_gathered(row[h]);
    } else {
      row[h] = g.r0 + col;
    }
  }
#pragma unroll
  for (int h = 0; h < 2; ++h)
    pb[h] = gathered ? p.xr + static_cast<size_t>(row[h]) * H + pq * 8
                     : src + (static_cast<size_t>(pq) * rows_b + row[h]) * 8;
  const int bstep = gathered ? 32 : 32 * rows_b;

  f32x4 acc[kRowTiles][kTileTok];
#pragma unroll
  for (int m = 0; m < kRowTiles; ++m)
#pragma unroll
    for (int ct = 0; ct < kTileTok; ++ct) acc[m][ct] = f32x4{0.f, 0.f, 0.f, 0.f};
  // Weights (from HBM) run two stages ahead in a three-slot register ring,
  // token fragments (mostly from L2) one stage ahead through registers into
  // the LDS double buffer.  Loads are issued tokens first, then weights, so
  // waiting for the next stage's tokens never waits for the newest weights.
  bf16x8 a_reg[3][kStageSteps][kRowTiles], b_nxt[kStageSteps][2];

  auto load_a = [&](int st, bf16x8 (&a)[kStageSteps][kRowTiles]) {
#pragma unroll
    for (int s = 0; s < kStageSteps; ++s)
#pragma unroll
      for (int m = 0; m < kRowTiles; ++m)
        a[s][m] = kStream ? ld_bf16x8_stream(pa + m * tstride + (st * kStageSteps + s) * kFrag)
                          : ld_bf16x8(pa + m * tstride + (st * kStageSteps + s) * kFrag);
  };
  auto load_b = [&](int st) {
#pragma unroll
    for (int s = 0; s < kStageSteps; ++s)
#pragma unroll
      for (int h = 0; h < 2; ++h) b_nxt[s][h] = ld_bf16x8(pb[h] + (st * kStageSteps + s) * bstep);
  };
  auto store_b = [&](int buf) {
#pragma unroll
    for (int h = 0; h < 2; ++h)
      if (pct + 4 * h < nt)  // uniform: the wave's tile holds tokens
#pragma unroll
        for (int s = 0; s < kStageSteps; ++s) stage[buf][s][pct + 4 * h][pl] = b_nxt[s][h];
  };

  const int nstages = ksteps / kStageSteps;
  load_b(0);
  load_a(0, a_reg[0]);
  if (nstages > 1) load_a(1, a_reg[1]);
  store_b(0);
  __syncthreads();
  // stage st uses ring slot R = st % 3 (a compile-time index: the loop runs
  // three stages per trip)
  auto run_stage = [&](auto slot, int st) {
    constexpr int R = decltype(slot)::value;
    const bool more = st + 1 < nstages;
    if (more) load_b(st + 1);
    __builtin_amdgcn_sched_barrier(0);  // tokens before weights
    if (st + 2 < nstages) load_a(st + 2, a_reg[(R + 2) % 3]);
    __builtin_amdgcn_sched_barrier(0);
    const int buf = st & 1;
    // token tile by token tile over the item's nt live tiles: the next
    // tile's fragments are read from LDS while this tile's matrix
    // instructions run.  Each accumulator still sums K in order.
    bf16x8 bc[kStageSteps], bn[kStageSteps];
#pragma unroll
    for (int s = 0; s < kStageSteps; ++s) bc[s] = stage[buf][s][0][lane];
#pragma unroll
    for (int ct = 0; ct < kTileTok; ++ct) {
      if (ct >= nt) break;  // uniform
      if (ct + 1 < nt)
#pragma unroll
        for (int s = 0; s < kStageSteps; ++s) bn[s] = stage[buf][s][ct + 1][lane];
#pragma unroll
      for (int s = 0; s < kStageSteps; ++s)
#pragma unroll
        for (int m = 0; m < kRowTiles; ++m)
          acc[m][ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a_reg[R][s][m], bc[s], acc[m][ct], 0, 0, 0);
#pragma unroll
      for (int s = 0; s < kStageSteps; ++s) bc[s] = bn[s];
    }
    if (more) store_b(buf ^ 1);
    __syncthreads();
  };
  for (int st = 0; st < nstages; st += 3) {
    run_stage(std::integral_constant<int, 0>{}, st);
    if (st + 1 < nstages) run_stage(std::integral_constant<int, 1>{}, st + 1);
    if (st + 2 < nstages) run_stage(std::integral_constant<int, 2>{}, st + 2);
  }

  const int q = lane >> 4, c = lane & 15;
#pragma unroll
  for (int m = 0; m < kRowTiles; ++m) {
    const int tile = tile0 + m;
#pragma unroll
    for (int ct = 0; ct < kTileTok; ++ct) {
      const int col = ct * 16 + c;
      if (ct >= nt) continue;  // uniform
      const f32x4 v = acc[m][ct];
      const int ex = !kGateUp && g.tok ? slot_exponent(p, v) : 0;  // whole wave, before the row guard
      if (col >= g.n) continue;
      if (kGateUp) {
        // accumulators: (g_i, g_i+1, u_i, u_i+1) with i = 8*tile + 2q
        const uint32_t h0 = f32_to_bf16(silu_f32(v[0]) * v[2]);
        const uint32_t h1 = f32_to_bf16(silu_f32(v[1]) * v[3]);
        bf16_t* dst = p.hk + (static_cast<size_t>(tile) * p.R + g.r0 + col) * 8 + 2 * q;
        *reinterpret_cast<uint32_t*>(dst) = h0 | (h1 << 16);
      } else {
        const int j = tile * 16 + 4 * q;
        if (g.tok)
          store_slot(p, g.r0 + col, j, v, ex);
        else
          *reinterpret_cast<f32x4*>(p.shared_out + static_cast<size_t>(g.t0 + col) * H + j) = v;
      }
    }
  }
}


template <bool kGateUp, int kRowTiles>
__global__ __launch_bounds__(kThreads, 2) void ffn_tile_bf16_kernel(FfnParams p, int gx) {
  int item, bx;
  if (!map_item(p, gx, item, bx)) return;
  Group g;
  if (!decode_item(item, p.shared_items, p.max_work, p.n_work, p.work, p.row_token, p.T, p.Tk, p.E, g)) return;
  __shared__ bf16x8 stage[2][kStageSteps][kTileTok][kWave];  // 32 KiB
  // An expert whose rows are one item is the only reader of its weights in
  // the launch (each row block reads its own rows once): they are streamed
  // non-temporally, which measured faster.  The items of an expert with more
  // rows read the same weights one after the other, through the L2 of the
  // XCD they share (non-temporal loads there measured slower).
  bool single;
  if (g.expert >= 0) {
    const int nw = min(*p.n_work, p.max_work);
    single = g.piece == 0 && !(item + 1 < nw && reinterpret_cast<const int4*>(p.work)[item + 1].x == g.expert);
  } else {
    single = p.T <= DMOE_WORK_ROWS;
  }
  if (single)
    tile_body<kGateUp, kRowTiles, true>(p, g, bx, stage);
  else
    tile_body<kGateUp, kRowTiles, false>(p, g, bx, stage);
}

// ---- f32 path -------------------------------------------------------------
//
// Weights are reduction-major (w13[e][h][u], w2[e][i][j]), so the 64 lanes of
// a wave, one output unit each, read 256 contiguous bytes per reduction
// index.  The four waves of a workgroup split the reduction in quarters and
// keep kF32Tok tokens' partial sums in registers; the token values are the
// same for every lane (scalar loads).  Partial sums are added in wave order
// through LDS.

constexpr int kF32Tok = 8;  // tokens per pass

// grid (ceil(max(I, I_s) / 64), groups): units 64*bx + lane of item g.
__global__ __launch_bounds__(kThreads) void ffn_gateup_f32_kernel(
    const float* __restrict__ xk, const float* __restrict__ w13, const float* __restrict__ ws13,
    const int* __restrict__ n_work, const int* __restrict__ work, const int* __restrict__ row_token, int T, int H,
    int E, int I, int I_s, int Tk, int max_work, int ldh, float* __restrict__ hbuf) {
  Group g;
  if (!decode_item(blockIdx.y, 0, max_work, n_work, work, row_token, T, Tk, E, g)) return;
  const int Iw = g.expert >= 0 ? I : I_s;
  if (static_cast<int>(blockIdx.x) * kWave >= Iw) return;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int u = blockIdx.x * kWave + lane;
  const bool live = u < Iw;
  const int uc = live ? u : Iw - 1;
  const float* W = g.expert >= 0 ? w13 + static_cast<size_t>(g.expert) * 2 * I * H : ws13;
  const size_t ldw = 2 * static_cast<size_t>(Iw);
  const int nch = H >> 2, per = (nch + 3) >> 2;  // 4-feature chunks, a quarter per wave
  const int c0 = wave * per, c1 = min(nch, c0 + per);
  __shared__ float red[3][2][kF32Tok][kWave];
  for (int p0 = 0; p0 < g.n; p0 += kF32Tok) {
    float ag[kF32Tok], au[kF32Tok];
    int tok[kF32Tok];
#pragma unroll
    for (int t = 0; t < kF32Tok; ++t) {
      ag[t] = au[t] = 0.f;
      const int col = min(p0 + t, g.n - 1);
      tok[t] = g.tok ? g.tok[col] : g.t0 + col;
    }
#pragma unroll 4
    for (int c = c0; c < c1; ++c) {
      float wg[4], wu[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float* wr = W + static_cast<size_t>(4 * c + q) * ldw;
        wg[q] = wr[uc];
        wu[q] = wr[Iw + uc];
      }
#pragma unroll
      for (int t = 0; t < kF32Tok; ++t) {
        const f32x4 xv = *reinterpret_cast<const f32x4*>(xk + (static_cast<size_t>(c) * T + tok[t]) * 4);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          ag[t] = fmaf(xv[q], wg[q], ag[t]);
          au[t] = fmaf(xv[q], wu[q], au[t]);
        }
      }
    }
    if (wave > 0) {
#pragma unroll
      for (int t = 0; t < kF32Tok; ++t) {
        red[wave - 1][0][t][lane] = ag[t];
        red[wave - 1][1][t][lane] = au[t];
      }
    }
    __syncthreads();
    if (wave == 0) {
#pragma unroll
      for (int t = 0; t < kF32Tok; ++t) {
#pragma unroll
        for (int ww = 0; ww < 3; ++ww) {
          ag[t] += red[ww][0][t][lane];
          au[t] += red[ww][1][t][lane];
        }
        if (live && p0 + t < g.n) hbuf[static_cast<size_t>(g.r0 + p0 + t) * ldh + u] = silu_f32(ag[t]) * au[t];
      }
    }
    __syncthreads();  // red is reused by the next pass
  }
}

// grid (ceil(H / 64), groups): output features 64*bx + lane of item g.
__global__ __launch_bounds__(kThreads) void ffn_down_f32_kernel(
    const float* __restrict__ w2, const float* __restrict__ ws2, const int* __restrict__ n_work,
    const int* __restrict__ work, const int* __restrict__ row_token, const int* __restrict__ row_slot, int T,
    int H, int E, int I, int I_s, int k, int Tk, int max_work, int ldh, const float* __restrict__ hbuf,
    float* __restrict__ slot_out, float* __restrict__ shared_out) {
  Group g;
  if (!decode_item(blockIdx.y, 0, max_work, n_work, work, row_token, T, Tk, E, g)) return;
  const int Kd = g.expert >= 0 ? I : I_s;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int j = blockIdx.x * kWave + lane;
  const bool live = j < H;
  const int jc = live ? j : H - 1;
  const float* W = g.expert >= 0 ? w2 + static_cast<size_t>(g.expert) * H * I : ws2;
  const int per = (Kd + 3) >> 2;
  const int i0 = wave * per, i1 = min(Kd, i0 + per);
  __shared__ float red[3][kF32Tok][kWave];
  for (int p0 = 0; p0 < g.n; p0 += kF32Tok) {
    float acc[kF32Tok];
    const float* hr[kF32Tok];
#pragma unroll
    for (int t = 0; t < kF32Tok; ++t) {
      acc[t] = 0.f;
      hr[t] = hbuf + static_cast<size_t>(g.r0 + min(p0 + t, g.n - 1)) * ldh;
    }
#pragma unroll 8
    for (int i = i0; i < i1; ++i) {
      const float wv = W[static_cast<size_t>(i) * H + jc];
#pragma unroll
      for (int t = 0; t < kF32Tok; ++t) acc[t] = fmaf(hr[t][i], wv, acc[t]);
    }
    if (wave > 0) {
#pragma unroll
      for (int t = 0; t < kF32Tok; ++t) red[wave - 1][t][lane] = acc[t];
    }
    __syncthreads();
    if (wave == 0) {
#pragma unroll
      for (int t = 0; t < kF32Tok; ++t) {
#pragma unroll
        for (int ww = 0; ww < 3; ++ww) acc[t] += red[ww][t][lane];
        const int col = p0 + t;
        if (!live || col >= g.n) continue;
        if (g.tok) {
          const int r = g.r0 + col;
          slot_out[(static_cast<size_t>(row_token[r]) * k + row_slot[r]) * H + j] = acc[t];
        } else {
          shared_out[static_cast<size_t>(g.t0 + col) * H + j] = acc[t];
        }
      }
    }
    __syncthreads();
  }
}

// ---- launch ---------------------------------------------------------------

// Token columns per pass: enough 16-wide tiles for the expected rows of a
// work item (the rows of the forward spread over max_work items, at most
// DMOE_WORK_ROWS), at most 4.
// rows per item of the launch: the routed rows spread over max_work items, or
// (max_work == 0, the shared expert alone) its pieces of up to DMOE_WORK_ROWS.
long rows_per_item(int T, int k, int max_work) {
  if (max_work == 0) return std::min<long>(DMOE_WORK_ROWS, T);
  return std::min<long>(DMOE_WORK_ROWS, (static_cast<long>(T) * k + max_work - 1) / max_work);
}

int pick_ntiles(int T, int k, int max_work) {
  const long rows = rows_per_item(T, k, max_work);
  return rows <= 16 ? 1 : (rows <= 32 ? 2 : 4);
}

// Launch shapes per token-tile count NT: weight burst KMAX steps, token
// chunks of BC steps, occupancy floor MINW (waves per SIMD), weight tiles
// per wave (kGuRows / kDnRows: each token fragment feeds that many matrix
// instructions), and the order of the grid rows (kSharedFirst, see the top
// of the file).  The one-tile variants serve token-level schedules, items of
// a few rows over many experts: two weight tiles per wave in both kernels
// halve the token-fragment reads from L2 per weight byte (measured 12 %
// faster at 512 tokens over 256 experts, equal at 32 tokens).  The two-tile
// variants serve block-routed decode steps, whose launches are small enough
// that a higher floor keeps every workgroup resident at once; their down
// kernel applies each h fragment to two weight tiles (half the h reads from
// L2; measured 0.4 us faster per step than one tile, while two gate/up tiles
// per wave measured 1.2 us slower).
template <int NT>
struct Shape;
template <>
struct Shape<1> {
  static constexpr int kGuMax = 16, kGuChunk = 4, kGuWaves = 2, kDnMax = 8, kDnChunk = 4, kDnWaves = 3;
  static constexpr int kGuRows = 2, kDnRows = 2;
  static constexpr bool kSharedFirst = true;
};
template <>
struct Shape<2> {
  static constexpr int kGuMax = 16, kGuChunk = 4, kGuWaves = 3, kDnMax = 4, kDnChunk = 4, kDnWaves = 3;
  static constexpr int kGuRows = 1, kDnRows = 2;
  static constexpr bool kSharedFirst = false;
};
template <>
struct Shape<4> {
  static constexpr int kGuMax = 8, kGuChunk = 4, kGuWaves = 1, kDnMax = 8, kDnChunk = 4, kDnWaves = 1;
  static constexpr int kGuRows = 1, kDnRows = 1;
  static constexpr bool kSharedFirst = false;
};

template <int NT>
hipError_t launch_bf16(const FfnParams& p, int ldh, int groups, hipStream_t s) {
  using S = Shape<NT>;
  ffn_gateup_bf16_kernel<NT, S::kGuMax, S::kGuChunk, S::kGuWaves, S::kSharedFirst, S::kGuRows>
      <<<dim3(ldh / (8 * S::kGuRows), groups), kThreads, 0, s>>>(p);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  ffn_down_bf16_kernel<NT, S::kDnMax, S::kDnChunk, S::kDnWaves, S::kSharedFirst, S::kDnRows>
      <<<dim3(p.H / (16 * S::kDnRows), groups), kThreads, 0, s>>>(p);
  return hipGetLastError();
}

// Tile kernels, one item per workgroup: two weight tiles per wave
// halve the LDS reads per weight byte; one tile per wave doubles the
// workgroups.  A gate/up grid of fewer than two rounds of the chip (three
// resident workgroups on each of 256 CUs) ends in a long partial round, which
// the finer split shortens.  The down projection always takes two tiles per
// wave: its reduction (I) is short, and at one tile per wave a workgroup
// reads twice as many token bytes as weight bytes.
constexpr long kTileRound = 3L * 256;
template <bool kGateUp>
hipError_t launch_tile_bf16(const FfnParams& p, int ldh, int items, hipStream_t s) {
  const int tiles = kGateUp ? ldh / 8 : p.H / 16;  // packed 16-row tiles
  const int items8 = (items + 7) / 8 * 8;
  if constexpr (kGateUp) {
    if (static_cast<long>(ldh / 64) * items < 2 * kTileRound) {
      ffn_tile_bf16_kernel<true, 1><<<dim3(tiles / 4 * items8), kThreads, 0, s>>>(p, tiles / 4);
      return hipGetLastError();
    }
  }
  ffn_tile_bf16_kernel<kGateUp, 2><<<dim3(tiles / 8 * items8), kThreads, 0, s>>>(p, tiles / 8);
  return hipGetLastError();
}

constexpr int kPassRows = 16;  // token rows of one decode-kernel pass

bool use_tile_kernels(int T, int k, int max_work, int items, int ldh) {
  return rows_per_item(T, k, max_work) >= 32 && static_cast<long>(ldh / 32) * items >= 512;
}

}  // namespace

size_t ffn_workspace_bytes(int T, int I, int I_s, int k, dmoe_dtype dt) {
  const size_t rows = static_cast<size_t>(T) * k + (I_s > 0 ? T : 0);
  const size_t ldh = static_cast<size_t>(std::max(I, I_s));
  return rows * ldh * (dt == DMOE_F32 ? 4 : 2);
}

hipError_t launch_ffn(const FfnArgs& a, dmoe_dtype dt, hipStream_t s) {
  const int Tk = a.T * a.k;
  const int R = Tk + (a.I_s > 0 ? a.T : 0);
  const int ldh = std::max(a.I, a.I_s);
  const int shared_items = a.I_s > 0 ? (a.T + DMOE_WORK_ROWS - 1) / DMOE_WORK_ROWS : 0;
  const int items = a.max_work + shared_items;
  if (dt == DMOE_BF16) {
    FfnParams p{static_cast<const bf16_t*>(a.x), static_cast<const bf16_t*>(a.xr),
                static_cast<const bf16_t*>(a.w13), static_cast<const bf16_t*>(a.w2),
                static_cast<const bf16_t*>(a.ws13),
                static_cast<const bf16_t*>(a.ws2), a.sched.n_work, a.sched.work, a.sched.row_token,
                a.sched.row_slot, a.T, a.H, a.E, a.I, a.I_s, a.k, Tk, R, a.max_work, shared_items,
                static_cast<bf16_t*>(a.workspace), a.slot_out, a.shared_out,
                a.slot_fmt == DMOE_SLOT_F16S ? 1 : 0};
    if (use_tile_kernels(a.T, a.k, a.max_work, items, ldh)) {
      const hipError_t err = launch_tile_bf16<true>(p, ldh, items, s);
      if (err != hipSuccess) return err;
      return launch_tile_bf16<false>(p, ldh, items, s);
    }
    switch (pick_ntiles(a.T, a.k, a.max_work)) {
      case 1: {
        // Items of a one-tile schedule average few rows, but an expert can
        // still collect many (a popular expert, a small Top-P coreset, the
        // shared expert over more than 16 tokens).  The decode kernels keep a
        // wave's weight slice in registers across 16-row passes when it is
        // one burst; when it is not, they would stream the weights once per
        // pass, so such layers run every item on the tile kernels (measured
        // faster than leaving the items of one pass to the decode kernels,
        // whose grids, sized for the worst case, cost ~17 us each when few
        // items are that small).  So do schedules of at least one pass per
        // expert on average (T*k >= 16 E), where the tile kernels measured
        // faster too (512 tokens over 256 experts at hidden 2048: token
        // routing 321 -> 283 us, Top-P 317 -> 306; 256 tokens and fewer
        // favour the decode kernels).
        const bool multi_burst = a.H / 128 > Shape<1>::kGuMax || ldh / 128 > Shape<1>::kDnMax;
        const bool pass_per_expert = static_cast<long>(a.T) * a.k >= static_cast<long>(kPassRows) * a.E;
        if (a.T > kPassRows && (multi_burst || pass_per_expert)) {
          const hipError_t err = launch_tile_bf16<true>(p, ldh, items, s);
          if (err != hipSuccess) return err;
          return launch_tile_bf16<false>(p, ldh, items, s);
        }
        return launch_bf16<1>(p, ldh, items, s);
      }
      case 2: return launch_bf16<2>(p, ldh, items, s);
      default: return launch_bf16<4>(p, ldh, items, s);
    }
  }
  float* hbuf = static_cast<float*>(a.workspace);
  dim3 g_gu((ldh + kWave - 1) / kWave, items), g_dn((a.H + kWave - 1) / kWave, items);
  ffn_gateup_f32_kernel<<<g_gu, kThreads, 0, s>>>(
      static_cast<const float*>(a.x), static_cast<const float*>(a.w13), static_cast<const float*>(a.ws13),
      a.sched.n_work, a.sched.work, a.sched.row_token, a.T, a.H, a.E, a.I, a.I_s, Tk, a.max_work, ldh, hbuf);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  ffn_down_f32_kernel<<<g_dn, kThreads, 0, s>>>(
      static_cast<const float*>(a.w2), static_cast<const float*>(a.ws2), a.sched.n_work, a.sched.work,
      a.sched.row_token, a.sched.row_slot, a.T, a.H, a.E, a.I, a.I_s, a.k, Tk, a.max_work, ldh, hbuf,
      static_cast<float*>(a.slot_out), a.shared_out);  // f32 layers: float32 slot outputs (checked by the API)
  return hipGetLastError();
}

}  // namespace dmoe
