// Graph-store ingest: validation of every node attribute, dependency offset,
// deadline and instance (the rules of nalar_problem), the instance table
// sorted by (type, index), and the first position of each workflow.  Table 3's
// future metadata arrives as a struct of arrays in HBM.
#include "internal.hpp"

namespace nalar {

namespace {

constexpr int kNodeThreads = 256;
constexpr int kNodeItems = 4;

// Instance table sorted by (type, original index) and the run of each small
// type; resets the next pass's control block (one workgroup).
__device__ void instance_table(const ProblemDev& p, ITab it, Ctrl* next_ctrl) {
  const int64_t M = p.M;
  reset_ctrl(next_ctrl);  // unused by this pass; ready for the next one
  __shared__ __align__(16) int32_t s_type[NALAR_MAX_INSTANCES];
  __shared__ int32_t s_sorted[NALAR_MAX_INSTANCES];
  __shared__ uint32_t s_run[kTypeDirect];
  const int M4 = int((M + 3) & ~int64_t(3));
  // padding past M compares as neither below nor equal to any entry's rank
  for (int i = threadIdx.x; i < M4; i += kNodeThreads) s_type[i] = i < M ? p.inst_type[i] : INT32_MAX;
  for (int t = threadIdx.x; t < kTypeDirect; t += kNodeThreads) s_run[t] = 0;
  __syncthreads();
  const int4* s_type4 = reinterpret_cast<const int4*>(s_type);
  for (int i = threadIdx.x; i < M; i += kNodeThreads) {
    const int32_t t = s_type[i];
    // rank = entries of a smaller type, plus entries of this type before i;
    // four entries per LDS read, unrolled so that the reads overlap
    int rank = 0;
#pragma unroll 4
    for (int q = 0; q < M4 / 4; ++q) {
      const int4 u = s_type4[q];
      const int j = 4 * q;
      rank += (u.x < t) | ((u.x == t) & (j < i));
      rank += (u.y < t) | ((u.y == t) & (j + 1 < i));
      rank += (u.z < t) | ((u.z == t) & (j + 2 < i));
      rank += (u.w < t) | ((u.w == t) & (j + 3 < i));
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
  // run of sorted positions per small type: its first position, from the
  // entry that starts it, and the end, from the entry that ends it
  for (int r = threadIdx.x; r < M; r += kNodeThreads) {
    const int32_t t = s_sorted[r];
    if (t >= 0 && t < kTypeDirect) {
      if (r == 0 || s_sorted[r - 1] != t) atomicOr(&s_run[t], uint32_t(r));
      if (r == M - 1 || s_sorted[r + 1] != t) atomicOr(&s_run[t], uint32_t(r + 1) << 16);
    }
  }
  __syncthreads();
  for (int t = threadIdx.x; t < kTypeDirect; t += kNodeThreads) it.run[t] = s_run[t];
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
  // kNodeItems nodes a stride apart per thread, every load issued before the
  // first check, so that each thread keeps that many lines in flight
  for (int64_t v0 = g0; v0 < N; v0 += kNodeItems * stride) {
    int32_t w[kNodeItems], t[kNodeItems], l[kNodeItems], o0[kNodeItems], o1[kNodeItems], wn[kNodeItems];
    int64_t e[kNodeItems];
    uint8_t d[kNodeItems];
#pragma unroll
    for (int u = 0; u < kNodeItems; ++u) {
      const int64_t v = v0 + u * stride;
      const bool in = v < N;
      const int64_t vs = in ? v : v0;
      w[u] = p.wf[vs];
      t[u] = p.type[vs];
      l[u] = p.loc[vs];
      e[u] = p.est[vs];
      d[u] = p.done[vs];
      o0[u] = p.dep_off[vs];
      o1[u] = p.dep_off[vs + 1];
      wn[u] = contiguous && vs + 1 < N ? p.wf[vs + 1] : INT32_MAX;
    }
#pragma unroll
    for (int u = 0; u < kNodeItems; ++u) {
      const int64_t v = v0 + u * stride;
      if (v >= N) continue;
      bad |= (w[u] < 0) | (int64_t(w[u]) >= W) | (t[u] < 0) | (l[u] < -1) | (int64_t(l[u]) >= M) |
             (e[u] < 0) | (e[u] > NALAR_EST_MAX) | (d[u] > 1) | (o0[u] > o1[u]) | (wn[u] < w[u]);
      if (v == 0) bad |= (o0[u] != 0);
      if (v == N - 1) bad |= (int64_t(o1[u]) != p.E);
    }
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
  const int64_t nv = (p.N + kNodeItems - 1) / kNodeItems;
  int64_t n = nv > p.W + 1 ? nv : p.W + 1;
  hipLaunchKernelGGL(k_nodes, dim3(grid_for(n, kNodeThreads, 4096) + 1), dim3(kNodeThreads), 0, s, p,
                     ctrl, next_ctrl, itab, wf_off, contiguous);
  return hipGetLastError();
}

}  // namespace nalar
