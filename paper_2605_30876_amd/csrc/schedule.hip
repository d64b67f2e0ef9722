// Unique-expert schedule of one forward.
//
// The set of experts selected anywhere in the forward is the unique-expert
// set whose size the paper reports per forward (Sec. 3); each of its experts
// must be streamed from HBM exactly once.  One workgroup of 512 threads:
//   1. counts the selections of every expert (LDS integer atomics),
//   2. scans the counts: ascending unique ids, their row offsets, n_unique,
//   3. places every (group, slot) entry's rows.  Entries are taken in rounds
//      of 512 in index order; an entry's rank among earlier entries of the
//      same expert comes from a per-expert bitmask of the round plus a
//      running count, so rows of one expert end up in token order and the
//      schedule is identical on every run.
#include "dmoe_common.h"

namespace dmoe {
namespace {

constexpr int kSchedThreads = 512;
constexpr int kMaskWords = kSchedThreads / 32;

__device__ __forceinline__ int wave_incl_scan(int v, int lane) {
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    int o = __shfl_up(v, d);
    if (lane >= d) v += o;
  }
  return v;
}

__global__ __launch_bounds__(kSchedThreads) void schedule_kernel(
    const int32_t* __restrict__ experts, int n_groups, int gs, int k, int E,
    int32_t* __restrict__ n_unique, int32_t* __restrict__ unique, int32_t* __restrict__ offsets,
    int32_t* __restrict__ row_token, int32_t* __restrict__ row_slot) {
  extern __shared__ int lds[];
  int* cnt = lds;                                            // [E] selections
  int* base = cnt + E;                                       // [E] first row
  int* run = base + E;                                       // [E] rows placed so far / gs
  unsigned* mask = reinterpret_cast<unsigned*>(run + E);     // [E][kMaskWords]
  __shared__ int wrows[kSchedThreads / kWave];
  __shared__ int wuniq[kSchedThreads / kWave];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  for (int e = tid; e < E; e += kSchedThreads) {
    cnt[e] = 0;
    run[e] = 0;
#pragma unroll
    for (int w = 0; w < kMaskWords; ++w) mask[e * kMaskWords + w] = 0u;
  }
  __syncthreads();

  const int n_entries = n_groups * k;
  for (int i = tid; i < n_entries; i += kSchedThreads) {
    const int e = experts[i];
    if (e >= 0 && e < E) atomicAdd(&cnt[e], 1);
  }
  __syncthreads();

  // Exclusive scans over experts (E <= kSchedThreads: one expert per thread).
  const int c = tid < E ? cnt[tid] : 0;
  const int rows = c * gs;
  const int pres = c > 0 ? 1 : 0;
  const int r_incl = wave_incl_scan(rows, lane);
  const int u_incl = wave_incl_scan(pres, lane);
  if (lane == kWave - 1) {
    wrows[wave] = r_incl;
    wuniq[wave] = u_incl;
  }
  __syncthreads();
  int r_off = 0, u_off = 0;
  for (int w = 0; w < wave; ++w) {
    r_off += wrows[w];
    u_off += wuniq[w];
  }
  const int r_excl = r_off + r_incl - rows;
  const int u_excl = u_off + u_incl - pres;
  if (tid < E) {
    base[tid] = r_excl;
    if (pres) {
      unique[u_excl] = tid;
      offsets[u_excl] = r_excl;
    }
  }
  if (tid == kSchedThreads - 1) {
    offsets[u_excl + pres] = r_excl + rows;
    *n_unique = u_excl + pres;
  }
  __syncthreads();

  const int word = tid >> 5;
  const unsigned bit = 1u << (tid & 31);
  for (int r0 = 0; r0 < n_entries; r0 += kSchedThreads) {
    const int i = r0 + tid;
    const int e = i < n_entries ? experts[i] : -1;
    const bool active = e >= 0 && e < E;
    if (active) atomicOr(&mask[e * kMaskWords + word], bit);
    __syncthreads();
    int below = 0;
    bool last = true;
    if (active) {
      const unsigned* m = mask + e * kMaskWords;
      for (int w = 0; w < word; ++w) below += __popc(m[w]);
      below += __popc(m[word] & (bit - 1u));
      if (m[word] & ~(bit | (bit - 1u))) last = false;
      for (int w = word + 1; w < kMaskWords; ++w)
        if (m[w]) last = false;
      const int g = i / k;
      const int s = i - g * k;
      const int pos = base[e] + (run[e] + below) * gs;
      for (int tl = 0; tl < gs; ++tl) {
        row_token[pos + tl] = g * gs + tl;
        row_slot[pos + tl] = s;
      }
    }
    __syncthreads();
    if (active) {
      if (last) run[e] += below + 1;
      atomicAnd(&mask[e * kMaskWords + word], ~bit);
    }
    __syncthreads();
  }
}

}  // namespace

hipError_t launch_schedule(const int32_t* experts, int n_groups, int gs, int k, int E,
                           dmoe_schedule sched, hipStream_t s) {
  const size_t lds = static_cast<size_t>(E) * (3 + kMaskWords) * sizeof(int);
  schedule_kernel<<<1, kSchedThreads, lds, s>>>(experts, n_groups, gs, k, E, sched.n_unique,
                                                sched.unique, sched.offsets, sched.row_token,
                                                sched.row_slot);
  return hipGetLastError();
}

}  // namespace dmoe
