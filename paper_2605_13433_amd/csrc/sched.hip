// Standalone launch of the seq_offsets tile scheduler (device body and the
// description of the lists in sched_impl.h): the forward call and the
// inspection entry point use it; the backward call builds its lists inside
// the LayerNorm-backward launch instead.
#include "internal.h"
#include "sched_impl.h"

namespace hstu {

namespace {

constexpr int SCHED_THREADS = 1024;

__global__ void __launch_bounds__(SCHED_THREADS) schedule_kernel(SchedArgs a) {
  __shared__ SchedSmem sm;
  build_schedule<SCHED_THREADS>(a, sm, threadIdx.x);
}

}  // namespace

hipError_t launch_schedule(const int64_t *seq_offsets, const Problem &p,
                           void *ws, const Layout &L, hipStream_t s) {
  hipLaunchKernelGGL(schedule_kernel, dim3(1), dim3(SCHED_THREADS), 0, s,
                     sched_args(seq_offsets, p, ws, L));
  return hipGetLastError();
}

}  // namespace hstu
