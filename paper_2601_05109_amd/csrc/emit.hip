// Final gather: the sorted (key, position) pairs become the caller's
// order / slack / route / cost arrays (the priorities of set_priority and the
// decisions of route / migrate, Table 2).
#include "internal.hpp"

namespace nalar {

namespace {

constexpr int kEmitThreads = 256;

__global__ __launch_bounds__(kEmitThreads) void k_emit(EmitArgs a) {
  const Ctrl* ctrl = a.ctrl;
  if (ctrl->status) return;
  const int64_t R = ctrl->n_ready;
  const int fin = (int(ctrl->sort_npass) - 1) & 1;   // at least one pass ran when R > 0
  const int64_t smin = ctrl->slack_min;
  const int64_t stride = int64_t(gridDim.x) * kEmitThreads;
  for (int64_t i = int64_t(blockIdx.x) * kEmitThreads + threadIdx.x; i < R; i += stride) {
    const uint32_t pos = a.pay_buf[fin][i];
    a.order[i] = a.node_of_pos ? a.node_of_pos[pos] : int32_t(pos);
    a.slack[i] = int64_t(a.key_buf[fin][i] + uint64_t(smin));
    a.route[i] = a.stg_route[pos];
    if (a.cost) a.cost[i] = a.stg_cost[pos];
  }
}

}  // namespace

hipError_t launch_emit(hipStream_t s, const EmitArgs& a, int64_t max_count) {
  int64_t b = (max_count + kEmitThreads * 4 - 1) / (kEmitThreads * 4);
  if (b < 1) b = 1;
  if (b > 4096) b = 4096;
  hipLaunchKernelGGL(k_emit, dim3(unsigned(b)), dim3(kEmitThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace nalar
