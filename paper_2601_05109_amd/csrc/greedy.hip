// Load-aware routing (NALAR_ROUTE_GREEDY): the ready futures, already in
// output order, are routed one at a time; each takes the cheapest candidate of
// its type under the loads left by the futures before it and adds its service
// time on the chosen instance to that instance's load (routing that balances
// load across instances, Section 6.1).
//
// Futures of different types never share a candidate, so each type is an
// independent sequence: one wavefront per type walks the output order and
// picks its own futures with a ballot.  With at most 64 candidates, lane q
// holds candidate q and its running load; the type's futures are queued in LDS
// and routed in batches of 64:
//   1. lane j takes future j of the batch and computes its service time on
//      every candidate (independent work, all lanes busy) into an LDS table;
//   2. the futures are then routed in order: lane q adds its running load to
//      the table entry of (future, q), the lexicographic minimum of (cost,
//      candidate) comes from a reduction over as few lanes as there are
//      candidates and a ballot, and the winner updates its load.
// Only step 2 is sequential, and its chain per future is an add, the
// reduction and a compare.  More than 64 candidates stay in LDS and each
// future scans them lane-parallel.
#include "internal.hpp"

namespace nalar {

namespace {

constexpr int kGreedyThreads = kWave;       // one wavefront per workgroup
constexpr int kWalk = 16;                   // chunks of the output order loaded at once
constexpr int kGreedyRing = 2048;           // queued futures of the type: under 64 + one walk block
constexpr int kSvStride = kWave + 1;        // padded row: lanes writing one column spread over banks
static_assert(kGreedyRing >= kWave - 1 + kWalk * kWave, "the queue holds a batch's remainder and a block");

// DPP controls that stay inside a row of 16 lanes.
constexpr int kDppHalfMirror = 0x141;       // lane i <- lane 7 - i within each 8 lanes
constexpr int kDppMirror = 0x140;           // lane i <- lane 15 - i within each 16 lanes

// A DPP move whose pattern reads a lane of the same row for every lane (the
// quad permutations and mirrors), so no lane keeps its old value.
template <int kCtrl>
__device__ inline int64_t row_dpp_i64(int64_t x) {
  const int lo = __builtin_amdgcn_mov_dpp(int(uint32_t(uint64_t(x))), kCtrl, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_mov_dpp(int(uint32_t(uint64_t(x) >> 32)), kCtrl, 0xF, 0xF, false);
  return int64_t((uint64_t(uint32_t(hi)) << 32) | uint32_t(lo));
}

// Minimum of lanes [0, W) (lanes past the candidates hold INT64_MAX), read
// from lane 0.
template <int W>
__device__ inline int64_t lanes_min_i64(int64_t x) {
  auto mn = [](int64_t u, int64_t v) { return u < v ? u : v; };
  if constexpr (W > 16) {
    return wave_min_i64(x);
  } else {
    x = mn(x, row_dpp_i64<kDppXor1>(x));
    x = mn(x, row_dpp_i64<kDppXor2>(x));
    x = mn(x, row_dpp_i64<kDppHalfMirror>(x));
    if constexpr (W > 8) x = mn(x, row_dpp_i64<kDppMirror>(x));
    return readlane_i64(x, 0);
  }
}

struct Cand {  // the type's candidates in LDS (candidate q = the q-th instance of the type)
  int64_t* load;
  double* inv;
  int32_t* speed;
  int32_t* idx;
  int32_t* q_of;   // candidate of an instance of the type
  int32_t* itype;  // type of every instance
};

// Routes the queued futures [head, head + B) of type t (B <= 64): lane q < nc
// holds candidate q's index and running load.
template <int W>
__device__ inline void route_batch(const GreedyArgs& g, const Cand& cd, int32_t t, int nc, int head, int B,
                                   const int32_t* r_out, const int64_t* r_est, const int32_t* r_loc,
                                   int64_t* sv, int64_t& my_load, int32_t my_idx, bool& bad) {
  const int ln = lane_id();
  const int slot = (head + ln) & (kGreedyRing - 1);
  const bool act = ln < B;
  const int32_t out_j = act ? r_out[slot] : 0;
  const int64_t e_j = act ? r_est[slot] : 0;
  const int32_t l_j = act ? r_loc[slot] : -1;
  // a future whose state lives on an instance of its own type runs there
  const int32_t pin_j = (g.stateful && l_j >= 0 && cd.itype[l_j] == t) ? cd.q_of[l_j] : -1;
  // 1. service times of future j (lane j) on every candidate
  const double a = double(e_j * 1000);
  for (int q = 0; q < nc; ++q) sv[ln * kSvStride + q] = floordiv_exact(a, cd.speed[q], cd.inv[q]);
  // One wavefront: its LDS accesses complete in program order; only the
  // compiler must not move the reads below above these writes.
  __asm__ __volatile__("" ::: "memory");
  // 2. in order.  Only the running loads carry from one future to the next;
  // the winner and cost of future j go to lane j and the batch's outputs are
  // stored together at the end.
  const bool cand = ln < nc;
  int32_t qv = 0;
  int64_t cv = 0;
  int64_t svc_next = sv[ln];  // the next future's entry is read one step ahead
  for (int j = 0; j < B; ++j) {
    const int64_t svc = svc_next;  // a lane past the candidates reads a spare entry
    if (j + 1 < B) svc_next = sv[(j + 1) * kSvStride + ln];
    const int32_t l = readlane_i32(l_j, j);
    const int32_t pq = readlane_i32(pin_j, j);
    const int64_t mt = (pq < 0 && l >= 0 && l != my_idx) ? g.mig : 0;
    const int64_t c = cand ? my_load + svc + mt : INT64_MAX;
    int qb;
    int64_t cb;
    if (pq >= 0) {
      qb = pq;
      cb = readlane_i64(c, qb);
    } else {
      cb = lanes_min_i64<W>(c);
      qb = __builtin_ctzll(ballot(c == cb));  // lanes ascend with the index: lowest wins
    }
    my_load += ln == qb ? svc : 0;
    qv = ln == j ? qb : qv;
    cv = ln == j ? cb : cv;
  }
  if (act) {
    g.route[out_j] = cd.idx[qv];
    if (g.cost) g.cost[out_j] = cv;
  }
  // loads only grow, and a batch adds at most 64 service times (each below
  // 2^50), so one check per batch sees every load that passes the limit
  bad |= cand && my_load > NALAR_REM_MAX;
  __asm__ __volatile__("" ::: "memory");  // the next batch overwrites the table
}

struct Queue {  // LDS: the queued futures and the batch's service-time table
  int32_t out[kGreedyRing];
  int64_t est[kGreedyRing];
  int32_t loc[kGreedyRing];
  int64_t sv[kWave * kSvStride];
};

// The type's futures in output order, queued through LDS and routed in
// batches of 64 (candidates in registers, nc <= W <= 64).
template <int W>
__device__ void route_type_regs(const GreedyArgs& g, const Cand& cd, int32_t t, int nc, Queue& Q, bool& bad) {
  int32_t* r_out = Q.out;
  int64_t* r_est = Q.est;
  int32_t* r_loc = Q.loc;
  int64_t* sv = Q.sv;
  const int ln = lane_id();
  int64_t my_load = 0;
  int32_t my_idx = -1;
  if (ln < nc) {
    my_load = cd.load[ln];
    my_idx = cd.idx[ln];
  }
  // The output order is walked kWalk chunks of 64 at a time: every attribute
  // load of a block is issued before any is used, and the next block's ids are
  // loaded while this block is routed, so a block costs one memory latency.
  const int64_t R = g.R;
  constexpr int64_t kBlock = int64_t(kWalk) * kWave;
  int32_t vn[kWalk];
#pragma unroll
  for (int u = 0; u < kWalk; ++u) vn[u] = u * kWave + ln < R ? g.order[u * kWave + ln] : 0;
  int head = 0, tail = 0;  // queue positions (the same on every lane)
  for (int64_t k0 = 0; k0 < R; k0 += kBlock) {
    int32_t tt[kWalk], ll[kWalk];
    int64_t ee[kWalk];
#pragma unroll
    for (int u = 0; u < kWalk; ++u) {
      const bool in = k0 + u * kWave + ln < R;
      tt[u] = in ? g.type[vn[u]] : -1;
      ee[u] = in ? g.est[vn[u]] : 0;
      ll[u] = in ? g.loc[vn[u]] : -1;
    }
#pragma unroll
    for (int u = 0; u < kWalk; ++u) {
      const int64_t k = k0 + kBlock + u * kWave + ln;
      vn[u] = k < R ? g.order[k] : 0;
    }
#pragma unroll
    for (int u = 0; u < kWalk; ++u) {
      const uint64_t mk = ballot(tt[u] == t);
      if (tt[u] == t) {
        const int s = (tail + int(lanes_below(mk))) & (kGreedyRing - 1);
        r_out[s] = int32_t(k0 + u * kWave + ln);
        r_est[s] = ee[u];
        r_loc[s] = ll[u];
      }
      tail += int(__popcll(mk));
    }
    __asm__ __volatile__("" ::: "memory");
    for (; tail - head >= kWave; head += kWave)
      route_batch<W>(g, cd, t, nc, head, kWave, r_out, r_est, r_loc, sv, my_load, my_idx, bad);
  }
  if (tail > head) route_batch<W>(g, cd, t, nc, head, tail - head, r_out, r_est, r_loc, sv, my_load, my_idx, bad);
}

// More than 64 candidates: every future scans them lane-parallel in LDS.
__device__ void route_type_lds(const GreedyArgs& g, const Cand& cd, int32_t t, int nc, bool& bad) {
  const int ln = lane_id();
  const int64_t R = g.R;
  for (int64_t k0 = 0; k0 < R; k0 += kWave) {
    const int64_t k = k0 + ln;
    int32_t tk = -1, lk = -1;
    int64_t ek = 0;
    if (k < R) {
      const int32_t v = g.order[k];
      tk = g.type[v];
      ek = g.est[v];
      lk = g.loc[v];
    }
    uint64_t mk = ballot(tk == t);
    while (mk != 0) {  // this chunk's futures of type t, in order
      const int src = __builtin_ctzll(mk);
      mk &= mk - 1;
      const int64_t e = readlane_i64(ek, src);
      const int32_t l = readlane_i32(lk, src);
      const double a = double(e * 1000);
      const bool pinned = g.stateful && l >= 0 && cd.itype[l] == t;
      int qb;
      int64_t cb;
      if (pinned) {
        qb = cd.q_of[l];
        cb = cd.load[qb] + floordiv_exact(a, cd.speed[qb], cd.inv[qb]);
      } else {
        int64_t bc = INT64_MAX;
        int bq = INT32_MAX;
        for (int q = ln; q < nc; q += kWave) {  // ascending q per lane: strict < keeps the lowest
          int64_t c = cd.load[q] + floordiv_exact(a, cd.speed[q], cd.inv[q]);
          if (l >= 0 && l != cd.idx[q]) c += g.mig;
          if (c < bc) { bc = c; bq = q; }
        }
        cb = wave_min_i64(bc);
        qb = int(wave_min_i64(bc == cb ? int64_t(bq) : int64_t(INT32_MAX)));
      }
      if (ln == 0) {
        g.route[k0 + src] = cd.idx[qb];
        if (g.cost) g.cost[k0 + src] = cb;
        const int64_t nl = cd.load[qb] + floordiv_exact(a, cd.speed[qb], cd.inv[qb]);
        cd.load[qb] = nl;
        bad |= nl > NALAR_REM_MAX;
      }
      // One wavefront: its LDS accesses complete in program order, so the
      // next future's reads see this update; only the compiler must not
      // move them (a barrier would also wait for the stores above).
      __asm__ __volatile__("" ::: "memory");
    }
  }
}

__global__ __launch_bounds__(kGreedyThreads) void k_route_greedy(GreedyArgs g) {
  __shared__ int64_t s_load[NALAR_MAX_INSTANCES];   // running load of candidate q
  __shared__ double s_inv[NALAR_MAX_INSTANCES];
  __shared__ int32_t s_speed[NALAR_MAX_INSTANCES];
  __shared__ int32_t s_idx[NALAR_MAX_INSTANCES];    // instance id of candidate q
  __shared__ int32_t s_q[NALAR_MAX_INSTANCES];      // candidate of instance i (type t only)
  __shared__ int32_t s_itype[NALAR_MAX_INSTANCES];  // type of every instance
  __shared__ Queue Q;
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

  const Cand cd{s_load, s_inv, s_speed, s_idx, s_q, s_itype};
  bool bad = false;
  if (nc <= 8)
    route_type_regs<8>(g, cd, t, nc, Q, bad);
  else if (nc <= 16)
    route_type_regs<16>(g, cd, t, nc, Q, bad);
  else if (nc <= kWave)
    route_type_regs<kWave>(g, cd, t, nc, Q, bad);
  else
    route_type_lds(g, cd, t, nc, bad);
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
