// Graph-store ingest: validation of every node attribute, dependency offset,
// deadline and instance (the rules of nalar_problem), the instance table
// sorted by (type, index), and the first position of each workflow.  Table 3's
// future metadata arrives as a struct of arrays in HBM.
#include "internal.hpp"

namespace nalar {

namespace {

constexpr int kNodeThreads = 256;
constexpr int kNodeItems = 4;

// Instance table sorted by type, and the run of each small type; resets the
// next pass's control block (one workgroup).  Inside a type's run the
// instances that no other instance of the type dominates come first, in
// ascending index, then the dominated ones (see route_future); prun marks the
// end of the first part.  Types with more than kPruneRun instances are not
// pruned (their run is in ascending index and prun is its end).
constexpr int kPruneRun = 128;

__device__ void instance_table(const ProblemDev& p, ITab it, Ctrl* next_ctrl) {
  const int64_t M = p.M;
  reset_ctrl(next_ctrl);  // unused by this pass; ready for the next one
  __shared__ __align__(16) int32_t s_type[NALAR_MAX_INSTANCES];
  __shared__ int64_t s_load[NALAR_MAX_INSTANCES];
  __shared__ int32_t s_speed[NALAR_MAX_INSTANCES];
  __shared__ int32_t s_sorted[NALAR_MAX_INSTANCES];  // position by (type, index) -> index
  __shared__ uint8_t s_dom[NALAR_MAX_INSTANCES];     // by index: dominated in its type
  const int M4 = int((M + 3) & ~int64_t(3));
  // padding past M compares as neither below nor equal to any entry's rank
  for (int i = threadIdx.x; i < M4; i += kNodeThreads) {
    s_type[i] = i < M ? p.inst_type[i] : INT32_MAX;
    if (i < M) {
      s_load[i] = p.inst_load[i];
      s_speed[i] = p.inst_speed[i];
    }
  }
  __syncthreads();
  const int4* s_type4 = reinterpret_cast<const int4*>(s_type);
  // pass 1: rank by (type, index), the type's first position and its size
  constexpr int kPer = (NALAR_MAX_INSTANCES + kNodeThreads - 1) / kNodeThreads;
  int below[kPer], same[kPer];
  for (int u = 0; u < kPer; ++u) {
    const int i = threadIdx.x + u * kNodeThreads;
    below[u] = 0;
    same[u] = 0;
    if (i >= M) continue;
    const int32_t t = s_type[i];
    // four entries per LDS read, unrolled so that the reads overlap
    int bl = 0, sm = 0, before = 0;
#pragma unroll 4
    for (int q = 0; q < M4 / 4; ++q) {
      const int4 v = s_type4[q];
      const int j = 4 * q;
      bl += (v.x < t) + (v.y < t) + (v.z < t) + (v.w < t);
      sm += (v.x == t) + (v.y == t) + (v.z == t) + (v.w == t);
      before += ((v.x == t) & (j < i)) + ((v.y == t) & (j + 1 < i)) + ((v.z == t) & (j + 2 < i)) +
                ((v.w == t) & (j + 3 < i));
    }
    below[u] = bl;
    same[u] = sm;
    s_sorted[bl + before] = i;
  }
  __syncthreads();
  // pass 2: dominated instances of small runs
  for (int u = 0; u < kPer; ++u) {
    const int i = threadIdx.x + u * kNodeThreads;
    if (i >= M) continue;
    bool dom = false;
    if (same[u] <= kPruneRun) {
      const int64_t li = s_load[i];
      const int32_t si = s_speed[i];
      for (int r = below[u]; r < below[u] + same[u]; ++r) {
        const int j = s_sorted[r];
        const int64_t lj = s_load[j];
        const int32_t sj = s_speed[j];
        dom |= sj >= si && (lj < li || (lj == li && j < i));
      }
    }
    s_dom[i] = dom ? 1 : 0;
  }
  __syncthreads();
  // pass 3: undominated first, each part in ascending index
  for (int u = 0; u < kPer; ++u) {
    const int i = threadIdx.x + u * kNodeThreads;
    if (i >= M) continue;
    const int32_t t = s_type[i];
    const bool dom = s_dom[i] != 0;
    int und = 0, rank = 0;
    for (int r = below[u]; r < below[u] + same[u]; ++r) {
      const int j = s_sorted[r];
      const bool dj = s_dom[j] != 0;
      und += dj ? 0 : 1;
      rank += (dj == dom && j < i) ? 1 : 0;
    }
    const int pos = below[u] + (dom ? und + rank : rank);
    const int32_t sp = s_speed[i];
    it.type[pos] = t;
    it.idx[pos] = i;
    it.load[pos] = s_load[i];
    it.speed[pos] = sp;
    it.inv_speed[pos] = sp >= 1 ? 1.0 / double(sp) : 0.0;
    it.pos_of[i] = pos;
    // the run of a small type, written by the type's lowest index
    if (t >= 0 && t < kTypeDirect && s_sorted[below[u]] == i) {
      it.run[t] = uint32_t(below[u]) | (uint32_t(below[u] + same[u]) << 16);
      it.prun[t] = uint32_t(below[u] + und);
    }
  }
  // types without an instance
  for (int t = threadIdx.x; t < kTypeDirect; t += kNodeThreads) {
    bool present = false;
    for (int q = 0; q < M4 / 4 && !present; ++q) {
      const int4 v = s_type4[q];
      present = v.x == t || v.y == t || v.z == t || v.w == t;
    }
    if (!present) {
      it.run[t] = 0;
      it.prun[t] = 0;
    }
  }
}

// Grid-stride over nodes, workflows and instances.  Workgroup 0 (dispatched
// first, so that its longer work overlaps the others) only builds the
// instance table sorted by type, so each future's candidates form one
// contiguous run, and resets the control block of the next pass.
__global__ __launch_bounds__(kNodeThreads) void k_nodes(ProblemDev p, Ctrl* ctrl, Ctrl* next_ctrl,
                                                       ITab it, int32_t* wf_off, int contiguous) {
  const int64_t N = p.N, W = p.W, M = p.M;
  if (blockIdx.x == 0) {
    instance_table(p, it, next_ctrl);
    return;
  }
  const int64_t stride = int64_t(gridDim.x - 1) * kNodeThreads;
  const int64_t g0 = int64_t(blockIdx.x - 1) * kNodeThreads + threadIdx.x;
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
