// Unique-expert schedule of one forward.
//
// The set of experts selected anywhere in the forward is the unique-expert
// set whose size the paper reports per forward (Sec. 3); each of its experts
// must be streamed from HBM exactly once.  One workgroup of 512 threads runs
// dev::schedule_wg (counts, scans, deterministic token-ordered placement, and
// the expert FFN's work items).  Token schedules with many entries and a
// scratch array run the same steps over many workgroups (count, scan,
// place); the placement rule is the same, so the results are identical.
// Block schedules with many rows leave the rows to one workgroup per group
// (the single workgroup's stores of thousands of rows were the long pole:
// 64 blocks of 64 tokens, 32768 rows, took ~20 us).
#include <algorithm>

#include "route_dev.h"

namespace dmoe {
namespace {

__global__ __launch_bounds__(dev::kSchedThreads) void schedule_kernel(
    const int32_t* __restrict__ experts, int n_groups, int gs, int k, int E, dmoe_schedule sched, int place_rows) {
  extern __shared__ int lds[];
  dev::schedule_wg(experts, n_groups, gs, k, E, lds, sched, place_rows != 0);
}

// ---- rows of a block schedule, one workgroup per group --------------------
// Entry (g, j) (expert e = experts[g*k + j]) starts at row
//   offsets[u] + gs * (entries before it, in index order, naming e),
// u the rank of e among the unique ids: the rows dev::schedule_wg places.
// Workgroup g counts the earlier entries naming each of its k experts (LDS
// counters), finds u by binary search in the ascending unique list, and
// writes the gs rows of each of its entries.
constexpr int kRowsThreads = 256;
// Rows (n_groups * gs * k) from which the rows get their own launch: below it
// the second launch costs more than the single workgroup's stores (16 x 32
// tokens x top-8: 6.3 us in one kernel, 4.6 + 4.9 us in two; 64 x 64 x 8:
// 20.5 us in one, 4.9 + 5.6 us in two).
constexpr int kRowsMinRows = 16384;

__global__ __launch_bounds__(kRowsThreads) void schedule_rows_kernel(const int32_t* __restrict__ experts, int gs,
                                                                     int k, int E, dmoe_schedule sched) {
  __shared__ int mine[kWave], cnt[kWave], pos[kWave];
  const int g = blockIdx.x, tid = threadIdx.x;
  if (tid < k) {
    mine[tid] = experts[static_cast<size_t>(g) * k + tid];
    cnt[tid] = 0;
  }
  __syncthreads();
  const int before = g * k;
  for (int i = tid; i < before; i += kRowsThreads) {
    const int v = experts[i];
    for (int j = 0; j < k; ++j)
      if (mine[j] == v) atomicAdd(&cnt[j], 1);
  }
  __syncthreads();
  if (tid < k) {
    const int e = mine[tid];
    int p = -1;  // an id outside [0, E): no rows
    if (e >= 0 && e < E) {
      int r = cnt[tid];
      for (int j = 0; j < tid; ++j) r += mine[j] == e ? 1 : 0;  // earlier entries of this group
      int lo = 0, hi = *sched.n_unique;
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (sched.unique[mid] < e)
          lo = mid + 1;
        else
          hi = mid;
      }
      p = sched.offsets[lo] + r * gs;
    }
    pos[tid] = p;
  }
  __syncthreads();
  for (int idx = tid; idx < k * gs; idx += kRowsThreads) {
    const int j = idx / gs, tl = idx - j * gs;
    const int p = pos[j];
    if (p < 0) continue;
    sched.row_token[p + tl] = g * gs + tl;
    sched.row_slot[p + tl] = j;
  }
}

// ---- many workgroups (group size 1, many entries) -------------------------
// Entries (token, slot) in index order are cut into chunks of kSchedThreads,
// one workgroup each.  scratch: [C][E] per-chunk counts, turned into each
// chunk's first rank per expert, then [E] each expert's first row.
constexpr int kChunk = dev::kSchedThreads;

// 1. each chunk's selections per expert
__global__ __launch_bounds__(kChunk) void schedule_count_kernel(const int32_t* __restrict__ experts,
                                                                int n_entries, int E, int32_t* __restrict__ scratch) {
  extern __shared__ int cnt[];
  const int tid = threadIdx.x, c = blockIdx.x;
  for (int e = tid; e < E; e += kChunk) cnt[e] = 0;
  __syncthreads();
  const int i = c * kChunk + tid;
  if (i < n_entries) {
    const int e = experts[i];
    if (e >= 0 && e < E) atomicAdd(&cnt[e], 1);
  }
  __syncthreads();
  for (int e = tid; e < E; e += kChunk) scratch[static_cast<size_t>(c) * E + e] = cnt[e];
}

// 2. one workgroup: per expert, exclusive scan over the chunks (chunk order
//    = entry order), then the schedule's totals from the expert counts
__global__ __launch_bounds__(kChunk) void schedule_scan_kernel(int n_chunks, int E, dmoe_schedule sched) {
  int32_t* scratch = sched.scratch;
  const int tid = threadIdx.x;
  int total = 0;
  if (tid < E) {
    constexpr int kBatch = 16;  // chunk counts loaded together
    for (int c0 = 0; c0 < n_chunks; c0 += kBatch) {
      int v[kBatch];
#pragma unroll
      for (int u = 0; u < kBatch; ++u)
        if (c0 + u < n_chunks) v[u] = scratch[static_cast<size_t>(c0 + u) * E + tid];
#pragma unroll
      for (int u = 0; u < kBatch; ++u)
        if (c0 + u < n_chunks) {
          scratch[static_cast<size_t>(c0 + u) * E + tid] = total;
          total += v[u];
        }
    }
  }
  dev::schedule_totals(total, 1, E, sched, scratch + static_cast<size_t>(n_chunks) * E);
}

// 3. each chunk places its entries: row = expert's first row + the chunk's
//    first rank + the entry's rank among the chunk's earlier entries of the
//    same expert (per-expert bitmasks in LDS, as in dev::schedule_wg)
__global__ __launch_bounds__(kChunk) void schedule_place_kernel(const int32_t* __restrict__ experts, int n_entries,
                                                                int k, int E, int n_chunks, dmoe_schedule sched) {
  extern __shared__ unsigned mask[];  // [E'][kMaskWords]
  const int tid = threadIdx.x, c = blockIdx.x;
  const int Ep = dev::pad4(E);
  for (int e = tid; e < Ep; e += kChunk) {
    uint4* m4 = reinterpret_cast<uint4*>(mask + e * dev::kMaskWords);
#pragma unroll
    for (int w = 0; w < dev::kMaskWords / 4; ++w) m4[w] = make_uint4(0u, 0u, 0u, 0u);
  }
  __syncthreads();
  const int i = c * kChunk + tid;
  const int e = i < n_entries ? experts[i] : -1;
  const bool active = e >= 0 && e < E;
  const int word = tid >> 5;
  const unsigned bit = 1u << (tid & 31);
  if (active) atomicOr(&mask[e * dev::kMaskWords + word], bit);
  __syncthreads();
  if (!active) return;
  const uint4* m4 = reinterpret_cast<const uint4*>(mask + e * dev::kMaskWords);
  int below = 0;
#pragma unroll
  for (int w4 = 0; w4 < dev::kMaskWords / 4; ++w4) {
    const uint4 q = m4[w4];
    const unsigned m[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int w = 4 * w4 + u;
      if (w < word) below += __popc(m[u]);
      if (w == word) below += __popc(m[u] & (bit - 1u));
    }
  }
  const int32_t* scratch = sched.scratch;
  const int row = scratch[static_cast<size_t>(n_chunks) * E + e] + scratch[static_cast<size_t>(c) * E + e] + below;
  sched.row_token[row] = i / k;
  sched.row_slot[row] = i - (i / k) * k;
}

}  // namespace

size_t schedule_scratch_ints(long n_groups, long k, long E) {
  const long n = n_groups * k;
  return static_cast<size_t>(((n + kChunk - 1) / kChunk + 1) * E);
}

// Each unique expert's rows come in whole groups (multiples of group_size), so
// every work item holds at least gcd(group_size, DMOE_WORK_ROWS) rows; and at
// most one item per expert is not full.
long schedule_max_work(long n_groups, long group_size, long k, long E) {
  const long rows = n_groups * group_size * k;
  const long umax = std::min(E, n_groups * k);
  long a = group_size, b = DMOE_WORK_ROWS;
  while (b) {
    const long t = a % b;
    a = b;
    b = t;
  }
  return std::min((rows + DMOE_WORK_ROWS - 1) / DMOE_WORK_ROWS + umax, rows / a);
}

hipError_t launch_schedule(const int32_t* experts, int n_groups, int gs, int k, int E,
                           dmoe_schedule sched, hipStream_t s) {
  const int n_entries = n_groups * k;
  if (gs == 1 && n_entries >= DMOE_SCHED_SPLIT_MIN && sched.scratch) {
    const int C = (n_entries + kChunk - 1) / kChunk;
    schedule_count_kernel<<<C, kChunk, static_cast<size_t>(E) * sizeof(int), s>>>(experts, n_entries, E,
                                                                                  sched.scratch);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    schedule_scan_kernel<<<1, kChunk, 0, s>>>(C, E, sched);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
    const size_t lds = static_cast<size_t>(dev::pad4(E)) * dev::kMaskWords * sizeof(unsigned);
    schedule_place_kernel<<<C, kChunk, lds, s>>>(experts, n_entries, k, E, C, sched);
    return hipGetLastError();
  }
  const size_t lds = dev::schedule_lds_ints(E) * sizeof(int);
  const bool rows_apart = gs > 1 && n_groups > 1 && static_cast<long>(n_entries) * gs >= kRowsMinRows;
  schedule_kernel<<<1, dev::kSchedThreads, lds, s>>>(experts, n_groups, gs, k, E, sched, rows_apart ? 0 : 1);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || !rows_apart) return err;
  schedule_rows_kernel<<<n_groups, kRowsThreads, 0, s>>>(experts, gs, k, E, sched);
  return hipGetLastError();
}

}  // namespace dmoe
