// Graph-store ingest: validation of every node attribute, dependency offset,
// deadline and instance (the rules of nalar_problem), the instance table
// sorted by (type, index), and the first position of each workflow.  Table 3's
// future metadata arrives as a struct of arrays in HBM.
#include "internal.hpp"

namespace nalar {

namespace {

constexpr int kNodeThreads = 256;

// Instance table sorted by (type, original index) and the run of each small
// type; resets the next pass's control block (one workgroup).
__device__ void instance_table(const ProblemDev& p, ITab it, Ctrl* next_ctrl) {
  const int64_t M = p.M;
  reset_ctrl(next_ctrl);  // unused by this pass; ready for the next one
  __shared__ int32_t s_type[NALAR_MAX_INSTANCES];
  __shared__ int32_t s_sorted[NALAR_MAX_INSTANCES];
  for (int i = threadIdx.x; i < M; i += kNodeThreads) s_type[i] = p.inst_type[i];
  for (int t = threadIdx.x; t < kTypeDirect; t += kNodeThreads) it.run[t] = 0;
  __syncthreads();
  for (int i = threadIdx.x; i < M; i += kNodeThreads) {
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
    s_sorted[rank] = t;
  }
  __syncthreads();
  // run of sorted positions per small type: from where the type starts to
  // where the next one does (or M)
  for (int r = threadIdx.x; r < M; r += kNodeThreads) {
    const int32_t t = s_sorted[r];
    if (t >= 0 && t < kTypeDirect && (r == 0 || s_sorted[r - 1] != t)) {
      int e = r + 1;
      while (e < M && s_sorted[e] == t) ++e;
      it.run[t] = uint32_t(r) | (uint32_t(e) << 16);
    }
  }
}

// Grid-stride over nodes, workflows and instances.  The last workgroup only
// sorts the instance table by (type, index), so each future's candidates form
// one contiguous run, and resets the control block of the next pass.
__global__ __launch_bounds__(kNodeThreads) void k_nodes(ProblemDev p, Ctrl* ctrl, Ctrl* next_ctrl,
                                                       ITab it, int32_t* wf_off, int contiguous) {
  const int64_t N = p.N, W = p.W, M = p.M;
  if (blockIdx.x == gridDim.x - 1) {
    instance_table(p, it, next_ctrl);
    return;
  }
  const int64_t stride = int64_t(gridDim.x - 1) * kNodeThreads;
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
    bad |= (w < 0) | (int64_t(w) >= W) | (t < 0) | (l < -1) | (int64_t(l) >= M) | (e < 0) |
           (e > NALAR_EST_MAX) | (d > 1) | (o0 > o1);
    if (v == 0) bad |= (o0 != 0);
    if (v == N - 1) bad |= (int64_t(o1) != p.E);
    if (contiguous && v + 1 < N) bad |= (p.wf[v + 1] < w);
  }
  for (int64_t w = g0; w < W; w += stride) {
    const int64_t dl = p.deadline[w];
    bad |= (dl < p.now - NALAR_HORIZON_MAX) | (dl > p.now + NALAR_HORIZON_MAX) |
           (p.prio != nullptr && p.prio[w] > NALAR_PRIORITY_MAX);
  }
  for (int64_t i = g0; i < M; i += stride) {
    const int64_t ld = p.inst_load[i];
    bad |= (p.inst_type[i] < 0) | (p.inst_speed[i] < 1) | (ld < 0) | (ld > NALAR_LOAD_MAX);
  }
  if (contiguous) {
    // first position of workflow w = first v with wf[v] >= w (wf non-decreasing;
    // if it is not, the pass fails with EINVAL and the offsets are never used)
    for (int64_t w = g0; w <= W; w += stride) {
      const int64_t guess = W > 0 ? (w * N) / W : 0;
      wf_off[w] = int32_t(lower_bound_from(p.wf, N, w, guess));
    }
  }
  if (__ballot(bad) != 0 && lane_id() == 0) flag_status(ctrl, kStInval);

}

int grid_for(int64_t n, int threads, int cap) {
  int64_t b = (n + threads - 1) / threads;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return int(b);
}

}  // namespace

hipError_t launch_nodes(hipStream_t s, const ProblemDev& p, Ctrl* ctrl, Ctrl* next_ctrl, ITab itab,
                        int32_t* wf_off, int contiguous) {
  int64_t n = p.N > p.W + 1 ? p.N : p.W + 1;
  hipLaunchKernelGGL(k_nodes, dim3(grid_for(n, kNodeThreads, 4096) + 1), dim3(kNodeThreads), 0, s, p,
                     ctrl, next_ctrl, itab, wf_off, contiguous);
  return hipGetLastError();
}

}  // namespace nalar
