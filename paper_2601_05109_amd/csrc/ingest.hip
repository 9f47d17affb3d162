// Graph-store ingest: per-pass control reset, instance table, validation of
// every node attribute and of the dependency offsets, and the first position
// of each workflow.  (Table 3's future metadata arrives as a struct of arrays
// in HBM; the rules checked here are those of nalar_problem.)
#include "internal.hpp"

namespace nalar {

namespace {

constexpr int kSetupThreads = 1024;
constexpr int kNodeThreads = 256;

// One workgroup: reset the control block, check the instance table and sort it
// by (type, index) so each future's candidates form one contiguous run.
__global__ __launch_bounds__(kSetupThreads) void k_setup(ProblemDev p, Ctrl* ctrl, ITab it,
                                                         uint32_t* ghist_slack,
                                                         uint32_t* ghist_group) {
  const int tid = threadIdx.x;
  if (tid == 0) {
    ctrl->status = 0;
    ctrl->sort_npass = 0;
    ctrl->n_ready = 0;
    ctrl->slack_min = INT64_MAX;
    ctrl->slack_max = INT64_MIN;
    for (int i = 0; i < 16; ++i) ctrl->tile_ticket[i] = 0;
  }
  for (int i = tid; i < kParts; i += kSetupThreads) {
    ctrl->part_min[i] = INT64_MAX;
    ctrl->part_max[i] = INT64_MIN;
    ctrl->part_cnt[i] = 0;
  }
  for (int i = tid; i < kMaxSortPasses * kRadixBuckets; i += kSetupThreads) ghist_slack[i] = 0;
  for (int i = tid; i < kMaxGroupPasses * kRadixBuckets; i += kSetupThreads) ghist_group[i] = 0;
  __syncthreads();
  const int M = int(p.M);
  __shared__ int32_t s_type[NALAR_MAX_INSTANCES];
  bool bad = false;
  for (int i = tid; i < M; i += kSetupThreads) {
    const int32_t t = p.inst_type[i];
    const int32_t sp = p.inst_speed[i];
    const int64_t ld = p.inst_load[i];
    bad |= (t < 0) | (sp < 1) | (ld < 0) | (ld > NALAR_LOAD_MAX);
    s_type[i] = t;
  }
  if (bad) flag_status(ctrl, kStInval);
  __syncthreads();
  for (int i = tid; i < M; i += kSetupThreads) {
    const int32_t t = s_type[i];
    int rank = 0;
    for (int j = 0; j < M; ++j) {
      const int32_t u = s_type[j];
      rank += (u < t) | ((u == t) & (j < i));
    }
    const int32_t sp = p.inst_speed[i];
    it.type[rank] = t;
    it.idx[rank] = i;
    it.load[rank] = p.inst_load[i];
    it.speed[rank] = sp;
    it.inv_speed[rank] = sp >= 1 ? 1.0 / double(sp) : 0.0;
    it.pos_of[i] = rank;
  }
}

// Grid-stride over nodes (attribute and offset rules), workflows (deadline
// rule) and, for the contiguous layout, workflow start positions.
__global__ __launch_bounds__(kNodeThreads) void k_nodes(ProblemDev p, Ctrl* ctrl, int32_t* wf_off,
                                                       int contiguous) {
  const int64_t N = p.N, W = p.W;
  const int64_t stride = int64_t(gridDim.x) * kNodeThreads;
  const int64_t g0 = int64_t(blockIdx.x) * kNodeThreads + threadIdx.x;
  bool bad = false;
  for (int64_t v = g0; v < N; v += stride) {
    const int32_t w = p.wf[v];
    const int32_t t = p.type[v];
    const int32_t l = p.loc[v];
    const int64_t e = p.est[v];
    const uint8_t d = p.done[v];
    const int32_t o0 = p.dep_off[v];
    const int32_t o1 = p.dep_off[v + 1];
    bad |= (w < 0) | (int64_t(w) >= W) | (t < 0) | (l < -1) | (int64_t(l) >= p.M) | (e < 0) |
           (e > NALAR_EST_MAX) | (d > 1) | (o0 > o1);
    if (v == 0) bad |= (o0 != 0);
    if (v == N - 1) bad |= (int64_t(o1) != p.E);
    if (contiguous && v + 1 < N) bad |= (p.wf[v + 1] < w);
  }
  for (int64_t w = g0; w < W; w += stride) {
    const int64_t dl = p.deadline[w];
    bad |= (dl < p.now - NALAR_HORIZON_MAX) | (dl > p.now + NALAR_HORIZON_MAX);
  }
  if (contiguous) {
    // first position of workflow w = first v with wf[v] >= w (wf non-decreasing;
    // if it is not, the pass fails with EINVAL and the offsets are never used)
    for (int64_t w = g0; w <= W; w += stride) {
      int64_t lo = 0, hi = N;
      while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (int64_t(p.wf[mid]) < w) lo = mid + 1; else hi = mid;
      }
      wf_off[w] = int32_t(lo);
    }
  }
  if (__ballot(bad) != 0 && lane_id() == 0) flag_status(ctrl, kStInval);
}

// After the stable sort of (wf, id) pairs: position of every node and first
// position of every workflow.
__global__ __launch_bounds__(kNodeThreads) void k_group_finish(ProblemDev p, Ctrl* ctrl,
                                                              const uint32_t* sorted_wf,
                                                              const uint32_t* sorted_ids,
                                                              int32_t* pos_of_node,
                                                              int32_t* wf_off) {
  if (ctrl->status) return;
  const int64_t N = p.N, W = p.W;
  const int64_t stride = int64_t(gridDim.x) * kNodeThreads;
  const int64_t g0 = int64_t(blockIdx.x) * kNodeThreads + threadIdx.x;
  for (int64_t q = g0; q < N; q += stride) pos_of_node[sorted_ids[q]] = int32_t(q);
  for (int64_t w = g0; w <= W; w += stride) {
    int64_t lo = 0, hi = N;
    while (lo < hi) {
      const int64_t mid = (lo + hi) >> 1;
      if (int64_t(sorted_wf[mid]) < w) lo = mid + 1; else hi = mid;
    }
    wf_off[w] = int32_t(lo);
  }
}

int grid_for(int64_t n, int threads, int cap) {
  int64_t b = (n + threads - 1) / threads;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return int(b);
}

}  // namespace

hipError_t launch_setup(hipStream_t s, const ProblemDev& p, Ctrl* ctrl, ITab itab,
                        uint32_t* ghist_slack, uint32_t* ghist_group) {
  hipLaunchKernelGGL(k_setup, dim3(1), dim3(kSetupThreads), 0, s, p, ctrl, itab, ghist_slack,
                     ghist_group);
  return hipGetLastError();
}

hipError_t launch_nodes(hipStream_t s, const ProblemDev& p, Ctrl* ctrl, int32_t* wf_off,
                        int contiguous) {
  int64_t n = p.N > p.W + 1 ? p.N : p.W + 1;
  hipLaunchKernelGGL(k_nodes, dim3(grid_for(n, kNodeThreads, 4096)), dim3(kNodeThreads), 0, s,
                     p, ctrl, wf_off, contiguous);
  return hipGetLastError();
}

hipError_t launch_group_finish(hipStream_t s, const ProblemDev& p, Ctrl* ctrl,
                               const uint32_t* sorted_wf, const uint32_t* sorted_ids,
                               int32_t* pos_of_node, int32_t* wf_off) {
  int64_t n = p.N > p.W + 1 ? p.N : p.W + 1;
  hipLaunchKernelGGL(k_group_finish, dim3(grid_for(n, kNodeThreads, 4096)), dim3(kNodeThreads),
                     0, s, p, ctrl, sorted_wf, sorted_ids, pos_of_node, wf_off);
  return hipGetLastError();
}

}  // namespace nalar
