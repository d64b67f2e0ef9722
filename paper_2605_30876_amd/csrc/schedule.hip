// Unique-expert schedule of one forward.
//
// The set of experts selected anywhere in the forward is the unique-expert
// set whose size the paper reports per forward (Sec. 3); each of its experts
// must be streamed from HBM exactly once.  One workgroup of 512 threads runs
// dev::schedule_wg (counts, scans, deterministic token-ordered placement).
#include "route_dev.h"

namespace dmoe {
namespace {

__global__ __launch_bounds__(dev::kSchedThreads) void schedule_kernel(
    const int32_t* __restrict__ experts, int n_groups, int gs, int k, int E,
    int32_t* __restrict__ n_unique, int32_t* __restrict__ unique, int32_t* __restrict__ offsets,
    int32_t* __restrict__ row_token, int32_t* __restrict__ row_slot) {
  extern __shared__ int lds[];
  dev::schedule_wg(experts, n_groups, gs, k, E, lds, n_unique, unique, offsets, row_token, row_slot);
}

}  // namespace

hipError_t launch_schedule(const int32_t* experts, int n_groups, int gs, int k, int E,
                           dmoe_schedule sched, hipStream_t s) {
  const size_t lds = dev::schedule_lds_ints(E) * sizeof(int);
  schedule_kernel<<<1, dev::kSchedThreads, lds, s>>>(experts, n_groups, gs, k, E, sched.n_unique,
                                                     sched.unique, sched.offsets, sched.row_token,
                                                     sched.row_slot);
  return hipGetLastError();
}

}  // namespace dmoe
