// Unique-expert schedule of one forward.
//
// The set of experts selected anywhere in the forward is the unique-expert
// set whose size the paper reports per forward (Sec. 3); each of its experts
// must be streamed from HBM exactly once.  One workgroup of 512 threads runs
// dev::schedule_wg (counts, scans, deterministic token-ordered placement, and
// the expert FFN's work items).
#include <algorithm>

#include "route_dev.h"

namespace dmoe {
namespace {

__global__ __launch_bounds__(dev::kSchedThreads) void schedule_kernel(
    const int32_t* __restrict__ experts, int n_groups, int gs, int k, int E, dmoe_schedule sched) {
  extern __shared__ int lds[];
  dev::schedule_wg(experts, n_groups, gs, k, E, lds, sched);
}

}  // namespace

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
  const size_t lds = dev::schedule_lds_ints(E) * sizeof(int);
  schedule_kernel<<<1, dev::kSchedThreads, lds, s>>>(experts, n_groups, gs, k, E, sched);
  return hipGetLastError();
}

}  // namespace dmoe
