// Load-aware routing (NALAR_ROUTE_GREEDY): the ready futures, already in
// output order, are routed one at a time; each takes the cheapest candidate of
// its type under the loads left by the futures before it and adds its service
// time on the chosen instance to that instance's load (routing that balances
// load across instances, Section 6.1).
//
// Futures of different types never share a candidate, so each type is an
// independent sequence: one wavefront per type walks the output order, picks
// its own futures with a ballot, and routes them in turn.  The candidates of
// the type and their running loads stay in the wave's LDS; a future's costs are
// evaluated lane-parallel over the candidates and the lexicographic minimum of
// (cost, candidate index) is found with a wave reduction and a ballot.
#include "internal.hpp"

namespace nalar {

namespace {

constexpr int kGreedyThreads = kWave;  // one wavefront per workgroup

__global__ __launch_bounds__(kGreedyThreads) void k_route_greedy(GreedyArgs g) {
  __shared__ int64_t s_load[NALAR_MAX_INSTANCES];   // running load of candidate q
  __shared__ double s_inv[NALAR_MAX_INSTANCES];
  __shared__ int32_t s_speed[NALAR_MAX_INSTANCES];
  __shared__ int32_t s_idx[NALAR_MAX_INSTANCES];    // instance id of candidate q
  __shared__ int32_t s_q[NALAR_MAX_INSTANCES];      // candidate of instance i (type t only)
  __shared__ int32_t s_itype[NALAR_MAX_INSTANCES];  // type of every instance
  const int w = blockIdx.x;
  const int ln = lane_id();
  const int M = g.M;
  const int32_t t = g.inst_type[w];
  for (int j = ln; j < M; j += kWave) s_itype[j] = g.inst_type[j];
  __syncthreads();
  // only the lowest-index instance of each type runs its type's sequence
  for (int j0 = 0; j0 < w; j0 += kWave) {
    const int j = j0 + ln;
    if (ballot(j < w && s_itype[j] == t) != 0) return;  // wave-uniform
  }
  int nc = 0;
  for (int j0 = 0; j0 < M; j0 += kWave) {
    const int j = j0 + ln;
    const bool m = j < M && s_itype[j] == t;
    const uint64_t mk = ballot(m);
    if (m) {
      const int q = nc + int(lanes_below(mk));
      const int32_t sp = g.inst_speed[j];
      s_idx[q] = j;
      s_load[q] = g.inst_load[j];
      s_speed[q] = sp;
      s_inv[q] = sp >= 1 ? 1.0 / double(sp) : 0.0;
      s_q[j] = q;
    }
    nc += int(__popcll(mk));
  }
  __syncthreads();

  // Up to 64 candidates live in registers (lane q holds candidate q and its
  // running load); more stay in LDS.
  const bool in_regs = nc <= kWave;
  int64_t my_load = 0;
  int32_t my_speed = 1, my_idx = -1;
  double my_inv = 0.0;
  if (in_regs && ln < nc) {
    my_load = s_load[ln];
    my_speed = s_speed[ln];
    my_inv = s_inv[ln];
    my_idx = s_idx[ln];
  }

  // The output order is read a chunk of 64 ahead (ids two chunks ahead, their
  // attributes one chunk ahead), so its latency overlaps the routing.
  bool bad = false;
  const int64_t R = g.R;
  int32_t v_next = ln < R ? g.order[ln] : 0;
  int32_t v_after = kWave + ln < R ? g.order[kWave + ln] : 0;
  int32_t t_cur = ln < R ? g.type[v_next] : -1;
  int64_t e_cur = ln < R ? g.est[v_next] : 0;
  int32_t l_cur = ln < R ? g.loc[v_next] : -1;
  for (int64_t k0 = 0; k0 < R; k0 += kWave) {
    const int32_t t_this = t_cur;
    const int64_t e_this = e_cur;
    const int32_t l_this = l_cur;
    {  // prefetch
      const int64_t k1 = k0 + kWave + ln, k2 = k0 + 2 * kWave + ln;
      const int32_t v1 = v_after;
      t_cur = k1 < R ? g.type[v1] : -1;
      e_cur = k1 < R ? g.est[v1] : 0;
      l_cur = k1 < R ? g.loc[v1] : -1;
      v_after = k2 < R ? g.order[k2] : 0;
    }
    uint64_t mk = ballot(t_this == t);
    while (mk != 0) {  // this chunk's futures of type t, in order
      const int src = __builtin_ctzll(mk);
      mk &= mk - 1;
      const int64_t e = readlane_i64(e_this, src);
      const int32_t l = readlane_i32(l_this, src);
      const double a = double(e * 1000);
      const bool pinned = g.stateful && l >= 0 && s_itype[l] == t;
      if (in_regs) {
        const int64_t svc = ln < nc ? floordiv_exact(a, my_speed, my_inv) : 0;
        int64_t c = INT64_MAX;
        if (ln < nc) c = my_load + svc + ((!pinned && l >= 0 && l != my_idx) ? g.mig : 0);
        int qb;
        int64_t cb;
        if (pinned) {
          qb = s_q[l];
          cb = readlane_i64(c, qb);
        } else {
          cb = wave_min_i64(c);
          qb = __builtin_ctzll(ballot(c == cb));  // lanes ascend with the index: lowest wins
        }
        if (ln == qb) {
          g.route[k0 + src] = my_idx;
          if (g.cost) g.cost[k0 + src] = cb;
          my_load += svc;
          bad |= my_load > NALAR_REM_MAX;
        }
      } else {
        int qb;
        int64_t cb;
        if (pinned) {
          qb = s_q[l];
          cb = s_load[qb] + floordiv_exact(a, s_speed[qb], s_inv[qb]);
        } else {
          int64_t bc = INT64_MAX;
          int bq = INT32_MAX;
          for (int q = ln; q < nc; q += kWave) {  // ascending q per lane: strict < keeps the lowest
            int64_t c = s_load[q] + floordiv_exact(a, s_speed[q], s_inv[q]);
            if (l >= 0 && l != s_idx[q]) c += g.mig;
            if (c < bc) { bc = c; bq = q; }
          }
          cb = wave_min_i64(bc);
          qb = int(wave_min_i64(bc == cb ? int64_t(bq) : int64_t(INT32_MAX)));
        }
        if (ln == 0) {
          g.route[k0 + src] = s_idx[qb];
          if (g.cost) g.cost[k0 + src] = cb;
          const int64_t nl = s_load[qb] + floordiv_exact(a, s_speed[qb], s_inv[qb]);
          s_load[qb] = nl;
          bad |= nl > NALAR_REM_MAX;
        }
        // One wavefront: its LDS accesses complete in program order, so the
        // next future's reads see this update; only the compiler must not
        // move them (a barrier would also wait for the stores above).
        __asm__ __volatile__("" ::: "memory");
      }
    }
    (void)v_next;
  }
  bad = ballot(bad) != 0;
  if (ln == 0 && bad)
    __hip_atomic_fetch_or(&g.host->aux_status, kStRange, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

}  // namespace

hipError_t launch_route_greedy(hipStream_t s, const GreedyArgs& g) {
  if (g.M <= 0 || g.R <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_route_greedy, dim3(g.M), dim3(kGreedyThreads), 0, s, g);
  return hipGetLastError();
}

}  // namespace nalar
