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
//
// With every type below kTypeDirect (the usual case) the (type, index) order
// is a counting sort: inside each group of 64 instances, ballots over the type
// bits find the lanes of equal type and the rank among them; per-group type
// counts, summed over earlier groups and earlier types, give the run starts.
// Otherwise each instance counts the entries before it (O(M^2), any types).
// The dominance checks then run per sorted position, so the lanes of one run
// read the same LDS entries.
constexpr int kPruneRun = 128;

struct TabLds {
  int32_t* type;    // by index
  int32_t* sorted;  // by (type, index) position: the index
  int64_t* sload;   // by position
  int32_t* sspeed;  // by position
  uint32_t* rng;    // by position: its run, lo | hi << 16
  uint8_t* sdom;    // by position: dominated inside its run
  uint32_t* wh;     // [groups][kTypeDirect]: per group type counts, then offsets
};

size_t tab_lds_bytes(int64_t M) {
  const size_t m4 = size_t((M + 3) & ~int64_t(3));
  const size_t groups = size_t((M + kWave - 1) / kWave);
  return 8 * m4 + 4 * m4 * 4 + ((m4 + 15) & ~size_t(15)) + 4 * groups * kTypeDirect;
}

__device__ inline TabLds carve_tab(unsigned char* sp, int64_t M) {
  const size_t m4 = size_t((M + 3) & ~int64_t(3));
  TabLds t;
  t.sload = reinterpret_cast<int64_t*>(sp); sp += 8 * m4;
  t.type = reinterpret_cast<int32_t*>(sp); sp += 4 * m4;
  t.sorted = reinterpret_cast<int32_t*>(sp); sp += 4 * m4;
  t.sspeed = reinterpret_cast<int32_t*>(sp); sp += 4 * m4;
  t.rng = reinterpret_cast<uint32_t*>(sp); sp += 4 * m4;
  t.sdom = sp; sp += (m4 + 15) & ~size_t(15);
  t.wh = reinterpret_cast<uint32_t*>(sp);
  return t;
}

// A workgroup barrier that orders LDS accesses only: it waits for this wave's
// LDS operations, not for its global loads and stores in flight (which
// __syncthreads also waits for).
__device__ inline void lds_barrier() {
  __asm__ __volatile__("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

__device__ void instance_table(const ProblemDev& p, ITab it, unsigned char* smem) {
  const int M = int(p.M);
  const int tid = threadIdx.x;
  __shared__ uint32_t s_run[kTypeDirect], s_prun[kTypeDirect], s_tstart[kTypeDirect];
  const TabLds S = carve_tab(smem, M);
  const int M4 = (M + 3) & ~3;
  const int groups = (M + kWave - 1) / kWave;
  constexpr int kPer = (NALAR_MAX_INSTANCES + kNodeThreads - 1) / kNodeThreads;
  // padding past M compares as neither below nor equal to any entry's rank
  bool general = false;
  int32_t ty[kPer];
  int64_t ld[kPer];
  int32_t sp[kPer];
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int i = tid + u * kNodeThreads;
    ty[u] = INT32_MAX;
    ld[u] = 0;
    sp[u] = 0;
    if (i < M) {
      ty[u] = p.inst_type[i];
      ld[u] = p.inst_load[i];
      sp[u] = p.inst_speed[i];
      general |= uint32_t(ty[u]) >= uint32_t(kTypeDirect);
    }
    if (i < M4) S.type[i] = ty[u];
  }
  for (int t = tid; t < kTypeDirect; t += kNodeThreads) {
    s_run[t] = 0;  // types without an instance keep an empty run
    s_prun[t] = 0;
  }
  for (int q = tid; q < groups * kTypeDirect; q += kNodeThreads) S.wh[q] = 0;
  general = __syncthreads_or(general ? 1 : 0) != 0;

  int at[kPer], lo[kPer], hi[kPer];
  if (!general) {
    // rank among the equal types of the group, and each group's type counts
    uint32_t below[kPer];
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int i = tid + u * kNodeThreads;
      below[u] = 0;
      if (u * kNodeThreads >= M) continue;  // the same on every lane
      const bool in = i < M;
      uint64_t peers = ballot(in);
#pragma unroll
      for (int bit = 0; bit < 6; ++bit) {
        static_assert(kTypeDirect == 64, "six type bits");
        const bool on = (ty[u] >> bit) & 1;
        const uint64_t m = ballot(on);
        peers &= on ? m : ~m;
      }
      below[u] = uint32_t(__popcll(peers & lanemask_lt()));
      if (in && below[u] == 0) S.wh[(i / kWave) * kTypeDirect + ty[u]] = uint32_t(__popcll(peers));
    }
    lds_barrier();
    // per type: offsets of the groups, then the run starts (one wave)
    if (tid < kTypeDirect) {
      uint32_t tot = 0;
      for (int g = 0; g < groups; ++g) {
        const uint32_t c = S.wh[g * kTypeDirect + tid];
        S.wh[g * kTypeDirect + tid] = tot;
        tot += c;
      }
      const uint32_t inc = wave_incl_scan_u32(tot);
      s_tstart[tid] = inc - tot;
    }
    lds_barrier();
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int i = tid + u * kNodeThreads;
      at[u] = lo[u] = hi[u] = 0;
      if (i >= M) continue;
      lo[u] = int(s_tstart[ty[u]]);
      hi[u] = ty[u] + 1 < kTypeDirect ? int(s_tstart[ty[u] + 1]) : M;
      at[u] = lo[u] + int(S.wh[(i / kWave) * kTypeDirect + ty[u]] + below[u]);
    }
  } else {
    const int4* type4 = reinterpret_cast<const int4*>(S.type);
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int i = tid + u * kNodeThreads;
      at[u] = lo[u] = hi[u] = 0;
      if (i >= M) continue;
      const int32_t t = ty[u];
      int bl = 0, sm = 0, before = 0;
#pragma unroll 4
      for (int q = 0; q < M4 / 4; ++q) {
        const int4 v = type4[q];
        const int j = 4 * q;
        bl += (v.x < t) + (v.y < t) + (v.z < t) + (v.w < t);
        sm += (v.x == t) + (v.y == t) + (v.z == t) + (v.w == t);
        before += ((v.x == t) & (j < i)) + ((v.y == t) & (j + 1 < i)) + ((v.z == t) & (j + 2 < i)) +
                  ((v.w == t) & (j + 3 < i));
      }
      lo[u] = bl;
      hi[u] = bl + sm;
      at[u] = bl + before;
    }
  }
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int i = tid + u * kNodeThreads;
    if (i >= M) continue;
    S.sorted[at[u]] = i;
    S.sload[at[u]] = ld[u];
    S.sspeed[at[u]] = sp[u];
    S.rng[at[u]] = uint32_t(lo[u]) | (uint32_t(hi[u]) << 16);
  }
  lds_barrier();
  // dominated instances of small runs, per sorted position r (j < i is q < r)
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int r = tid + u * kNodeThreads;
    if (r >= M) continue;
    const uint32_t rg = S.rng[r];
    const int a = int(rg & 0xFFFFu), e = int(rg >> 16);
    bool dom = false;
    if (e - a <= kPruneRun) {
      const int64_t li = S.sload[r];
      const int32_t si = S.sspeed[r];
      // eight entries per step, their LDS reads in flight together (a step
      // past the run rereads its first entry and ignores it)
      for (int q0 = a; q0 < e; q0 += 8) {
#pragma unroll
        for (int d = 0; d < 8; ++d) {
          const int q = q0 + d < e ? q0 + d : a;
          const int64_t lj = S.sload[q];
          dom |= (q0 + d < e) & (S.sspeed[q] >= si) & ((lj < li) | ((lj == li) & (q < r)));
        }
      }
    }
    S.sdom[r] = dom ? 1 : 0;
  }
  lds_barrier();
  // undominated first, each part in ascending index
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int r = tid + u * kNodeThreads;
    if (r >= M) continue;
    const uint32_t rg = S.rng[r];
    const int a = int(rg & 0xFFFFu), e = int(rg >> 16);
    const int dom = S.sdom[r];
    int und = 0, rank = 0;
    for (int q0 = a; q0 < e; q0 += 8) {
#pragma unroll
      for (int d = 0; d < 8; ++d) {
        const int q = q0 + d < e ? q0 + d : a;
        const int in = q0 + d < e ? 1 : 0;
        const int dq = S.sdom[q];
        und += in & (1 - dq);
        rank += in & (dq == dom) & (q < r);
      }
    }
    const int pos = a + (dom ? und + rank : rank);
    const int32_t i = S.sorted[r];
    const int32_t t = S.type[i];
    const int32_t spd = S.sspeed[r];
    it.type[pos] = t;
    it.idx[pos] = i;
    it.load[pos] = S.sload[r];
    it.speed[pos] = spd;
    it.inv_speed[pos] = spd >= 1 ? 1.0 / double(spd) : 0.0;
    it.pos_of[i] = pos;
    if (t >= 0 && t < kTypeDirect && r == a) {  // the run of a small type
      s_run[t] = uint32_t(a) | (uint32_t(e) << 16);
      s_prun[t] = uint32_t(a + und);
    }
  }
  lds_barrier();
  for (int t = tid; t < kTypeDirect; t += kNodeThreads) {
    it.run[t] = s_run[t];
    it.prun[t] = s_prun[t];
  }
}

// Grid-stride over nodes, workflows and instances.  Workgroup 0 (dispatched
// first, so that its longer work overlaps the others) only builds the
// instance table sorted by type, so each future's candidates form one
// contiguous run; workgroup 1 also resets the control block of the next pass
// (the grid always has a second workgroup).
__global__ __launch_bounds__(kNodeThreads) void k_nodes(ProblemDev p, Ctrl* ctrl, Ctrl* next_ctrl,
                                                       ITab it, int32_t* wf_off, int contiguous,
                                                       int64_t v_begin, uint64_t* done_bits) {
  const int64_t N = p.N, W = p.W, M = p.M;
  if (blockIdx.x == 0) {
    extern __shared__ __align__(16) unsigned char smem[];
    instance_table(p, it, smem);
    return;
  }
  if (blockIdx.x == 1) reset_ctrl(next_ctrl);  // unused by this pass; ready for the next one
  const int64_t stride = int64_t(gridDim.x - 1) * kNodeThreads;
  const int64_t g0 = int64_t(blockIdx.x - 1) * kNodeThreads + threadIdx.x;
  bool bad = false;
  // kNodeItems nodes a stride apart per thread, every load issued before the
  // first check, so that each thread keeps that many lines in flight
  for (int64_t v0 = v_begin + g0; v0 < N; v0 += kNodeItems * stride) {
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
    if (done_bits) {  // a wave holds 64 consecutive futures (lane 0's a multiple of 64)
#pragma unroll
      for (int u = 0; u < kNodeItems; ++u) {
        const int64_t v = v0 + u * stride;
        const uint64_t m = ballot(v < N && d[u] != 0);
        if (lane_id() == 0 && v < N) done_bits[v >> 6] = m;
      }
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
                        int32_t* wf_off, int contiguous, int64_t v_begin, uint64_t* done_bits) {
  if (v_begin % kWave != 0) done_bits = nullptr;  // a wave's futures must fill whole words
  const int64_t nv = (p.N - v_begin + kNodeItems - 1) / kNodeItems;
  int64_t n = nv > p.W + 1 ? nv : p.W + 1;
  hipLaunchKernelGGL(k_nodes, dim3(grid_for(n, kNodeThreads, 4096) + 1), dim3(kNodeThreads), tab_lds_bytes(p.M), s, p,
                     ctrl, next_ctrl, itab, wf_off, contiguous, v_begin, done_bits);
  return hipGetLastError();
}

}  // namespace nalar
