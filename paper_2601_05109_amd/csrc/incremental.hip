// Incremental pass over the graph store.  Between two passes the store only
// changes by deltas (Section 4.3.1: futures created with their dependencies,
// values materialising): futures appended, futures marked done.  A future's
// remaining critical path rem(v) = est'(v) + max over its consumers c of
// rem(c) (est' = 0 once done) depends only on v and its descendants, so after
// a delta it can change only for the changed futures (the seeds: appended or
// completed since the last pass) and their ancestors (every future a seed
// depends on, transitively): the closure.  Everything else keeps the rem of
// the last pass, persisted in the store.
//
// The pass, after validating the appended futures (k_nodes over the appended
// range):
//   1. closure: from every seed, its dependencies are marked (one bit per
//      future) and visited in turn;
//   2. scan (every future, O(N + E)): readiness (not done, every dependency
//      done) into a list of ready futures; for a closure member, one count per
//      dependency (its consumers inside the closure); for a future outside
//      the closure, its unchanged rem pushed to each dependency inside the
//      closure (max);
//   3. sweep of the closure: the members without closure consumers listed,
//      then a member whose closure consumers are all finalised takes rem =
//      est' + max, and pushes it to its dependencies;
//   4. the ready futures keyed, routed and dropped into the bins of the
//      partition sort (the splitters of the previous pass), which then orders
//      them by (key, wf, id).
// Steps 1 and 3 let a thread follow a chain of single dependencies itself (the
// common shape: a future created as the child of one future), so a chain of
// any length costs one launch; a future with several new dependencies hands
// all but one to its workgroup's LDS queue, and a future with more than
// kIncHeavy dependencies goes to a second LDS queue whose futures the whole
// workgroup expands together; the workgroup drains both before it ends.  A
// full queue spills into the next round's lists; the host launches kIncRounds
// rounds, and work left after the last one makes the pass fall back to a
// full pass (kStIncomplete).
#include "internal.hpp"

namespace nalar {

namespace {

constexpr int kIncThreads = 256;
constexpr int kIncTail = 3;       // rounds from here on run in one workgroup (k_inc_*_tail)
constexpr int kIncHeavy = 64;     // more dependencies: one workgroup expands the future
constexpr int kScanPer = 8;       // futures per thread in the scan (kIncThreads apart)
constexpr int kReadyPer = 4;      // ready futures per thread and chunk in the ready kernel

__device__ inline bool bit_set_new(uint32_t* bits, int32_t v) {
  const uint32_t m = 1u << (uint32_t(v) & 31u);
  return (atomicOr(&bits[uint32_t(v) >> 5], m) & m) == 0u;
}

__device__ inline bool bit_get(const uint32_t* bits, int32_t v) {
  return ((bits[uint32_t(v) >> 5] >> (uint32_t(v) & 31u)) & 1u) != 0u;
}

// A round's count, read where the atomics that wrote it are coherent (the
// tail kernel reads counts its own earlier rounds wrote).
__device__ inline uint32_t ld_count(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Start of round r's items in a list whose rounds are appended one after the
// other (counts of rounds 0 .. r-1, stable once round r runs).
__device__ inline uint32_t round_base(const uint32_t* cnt, int r) {
  uint32_t b = 0;
  for (int i = 0; i < r; ++i) b += ld_count(&cnt[i]);
  return b;
}

__device__ inline void push_round(int32_t* list, uint32_t* cnt, int r, int32_t v) {
  if (r > kIncRounds) return;  // cannot happen: rounds past the last are never appended to
  const uint32_t at = round_base(cnt, r) + atomicAdd(&cnt[r], 1u);
  list[at] = v;
}

// Appends the lanes' futures with one atomic per workgroup: thread t holds the
// futures first + j * stride for the set bits j of mask (every thread of the
// workgroup calls).  s_tmp holds one word per wave and two more.
__device__ inline void push_block(uint32_t mask, int64_t first, int32_t* list, uint32_t* n, uint32_t base,
                                  uint32_t* s_tmp, int64_t stride = 1) {
  const int nw = int(blockDim.x) / kWave;
  const int wv = int(threadIdx.x) / kWave;
  const uint32_t k = uint32_t(__popc(mask));
  const uint32_t inc = wave_incl_scan_u32(k);
  if (lane_id() == kWave - 1) s_tmp[wv] = inc;
  __syncthreads();
  uint32_t off = 0, tot = 0;
  for (int w = 0; w < nw; ++w) {
    off += w < wv ? s_tmp[w] : 0u;
    tot += s_tmp[w];
  }
  if (threadIdx.x == 0) s_tmp[nw] = tot ? atomicAdd(n, tot) : 0u;
  __syncthreads();
  uint32_t at = base + s_tmp[nw] + off + inc - k;
  while (mask) {
    const int j = __builtin_ctz(mask);
    mask &= mask - 1;
    list[at++] = int32_t(first + int64_t(j) * stride);
  }
  __syncthreads();  // s_tmp is free again
}

// One future (or none) per thread, appended as push_block does.
__device__ inline void push_block1(bool in, int32_t v, int32_t* list, uint32_t* n, uint32_t base,
                                   uint32_t* s_tmp) {
  push_block(in ? 1u : 0u, v, list, n, base, s_tmp);
}

__device__ inline void flag(Ctrl* c, uint32_t bits) {
  __hip_atomic_fetch_or(&c->status_sweep, bits, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// A dependency d of closure member u, checked: in range and not u itself;
// for an appended future (u >= n_prev, never validated before) also of u's
// workflow.
__device__ inline bool dep_ok(const IncArgs& a, int32_t u, int32_t d) {
  if (d < 0 || int64_t(d) >= a.p.N) {
    flag(a.ctrl, kStInval);
    return false;
  }
  if (d == u) {
    flag(a.ctrl, kStCycle);
    return false;
  }
  if (int64_t(u) >= a.n_prev && a.p.wf[d] != a.p.wf[u]) {
    flag(a.ctrl, kStInval);
    return false;
  }
  return true;
}

__device__ inline void join(const IncArgs& a, int32_t d) {
  a.mxA[d] = 0;
  a.cntA[d] = 0;
}

// A workgroup's queues of futures to continue from (LDS): single ones and
// heavy ones; past a queue's capacity a future goes to the next round's list
// instead.
constexpr int kIncQueue = 2048;
constexpr int kIncHeavyQueue = 64;

struct WgQueue {
  int32_t* q;       // [kIncQueue]
  int* n;
  int32_t* hq;      // [kIncHeavyQueue]
  int* hn;
  uint32_t* tmp;    // [waves + 2] for push_block
  int* htaken;      // heavy futures this workgroup kept (at most kIncHeavyKeep)
  bool keep_all;    // one workgroup for every round left: keep every heavy future
};

__device__ inline void wg_push(const WgQueue& wq, int32_t* list, uint32_t* cnt, int round, int32_t v) {
  const int at = atomicAdd(wq.n, 1);
  if (at < kIncQueue) wq.q[at] = v;
  else push_round(list, cnt, round + 1, v);
}

// A workgroup expands heavy futures itself while its queue has room, but at
// most kIncHeavyKeep of those with more than kIncHugeDeps dependencies (a
// reduction over thousands of futures); the others go to the next round,
// whose workgroups expand them side by side.
constexpr int kIncHeavyKeep = 1;
constexpr int kIncHugeDeps = 1024;

__device__ inline void wg_push_heavy(const WgQueue& wq, int32_t* list, uint32_t* cnt, int round, int32_t v,
                                     int32_t deg) {
  if (wq.keep_all || deg <= kIncHugeDeps || atomicAdd(wq.htaken, 1) < kIncHeavyKeep) {
    const int at = atomicAdd(wq.hn, 1);
    if (at < kIncHeavyQueue) {
      wq.hq[at] = v;
      return;
    }
  }
  push_round(list, cnt, round + 1, v);
}

// ------------------------------------------------------------------ closure

// Marks the lanes' dependencies d (d < 0: none) with one atomic per group of
// lanes holding the same d (a fan-in: many consumers of one future walking
// at once), else one per lane; returns whether this lane made d a member
// (one lane per d).  Every lane of the wave calls.
__device__ inline bool wave_mark(uint32_t* bits, int32_t d) {
  uint64_t pend = ballot(d >= 0);
  bool fresh = false;
  for (int it = 0; it < 2 && pend != 0; ++it) {
    const int lead = __builtin_ctzll(pend);
    const int32_t t = readlane_i32(d, lead);
    const uint64_t grp = ballot(((pend >> lane_id()) & 1u) && d == t);
    if (__popcll(grp) < 2) break;
    if (lane_id() == lead) fresh = bit_set_new(bits, t);
    pend &= ~grp;
  }
  if ((pend >> lane_id()) & 1u) fresh = bit_set_new(bits, d);
  return fresh;
}

// u has just joined the closure: visit its dependencies, following the chain
// while exactly one of them is new.  Every lane of the wave calls (u = -1:
// nothing), so that the lanes whose single dependency is one future mark it
// together.
__device__ void close_walk(const IncArgs& a, int32_t u, int round, const WgQueue& wq) {
  while (ballot(u >= 0) != 0) {
    int32_t d1 = -1;  // the one dependency of a single-dependency future
    if (u >= 0) {
      const int32_t o0 = a.p.dep_off[u], o1 = a.p.dep_off[u + 1];
      if (o1 - o0 > kIncHeavy) {
        wg_push_heavy(wq, a.heavy, a.ic->ch, round, u, o1 - o0);
        u = -1;
      } else if (o1 - o0 == 1) {
        const int32_t d = a.p.dep_idx[o0];
        if (dep_ok(a, u, d)) d1 = d;
        u = -1;
      } else {
        int32_t next = -1;
        for (int32_t e = o0; e < o1; ++e) {
          const int32_t d = a.p.dep_idx[e];
          if (!dep_ok(a, u, d)) continue;
          if (bit_set_new(a.inA, d)) {
            join(a, d);
            if (next < 0) next = d;
            else wg_push(wq, a.light, a.ic->cl, round, d);
          }
        }
        u = next;
      }
    }
    if (wave_mark(a.inA, d1)) {
      join(a, d1);
      u = d1;
    }
  }
}

// Drains the workgroup's queues (every thread of the workgroup calls): a heavy
// future is expanded by the whole workgroup (expand(v) on every thread), else
// up to one single future per thread is taken from the top, until both are
// empty.
template <typename Walk, typename Expand>
__device__ void wg_drain(const WgQueue& wq, Walk walk, Expand expand) {
  for (;;) {
    __syncthreads();
    const int hc = *wq.hn, c = *wq.n;
    const int hn = hc < kIncHeavyQueue ? hc : kIncHeavyQueue;
    const int n = c < kIncQueue ? c : kIncQueue;
    if (hn == 0 && n == 0) break;  // the same on every thread
    if (hn > 0) {
      const int32_t h = wq.hq[hn - 1];
      __syncthreads();
      if (threadIdx.x == 0) *wq.hn = hn - 1;
      __syncthreads();
      expand(h);
      continue;
    }
    int32_t mine = -1;
    if (int(threadIdx.x) < n) mine = wq.q[n - 1 - int(threadIdx.x)];
    __syncthreads();
    if (threadIdx.x == 0) *wq.n = n > int(blockDim.x) ? n - int(blockDim.x) : 0;
    __syncthreads();
    walk(mine);  // every lane: the walks work wave by wave
  }
}

// A heavy member's dependencies visited by the whole workgroup; the new
// members go to the next round, where every workgroup shares their walks.
__device__ inline void close_expand(const IncArgs& a, int32_t u, int round, const WgQueue& wq) {
  const int32_t o0 = a.p.dep_off[u], o1 = a.p.dep_off[u + 1];
  for (int32_t e0 = o0; e0 < o1; e0 += int32_t(blockDim.x)) {
    const int32_t e = e0 + int32_t(threadIdx.x);
    bool fresh = false;
    int32_t d = -1;
    if (e < o1) {
      d = a.p.dep_idx[e];
      if (dep_ok(a, u, d) && bit_set_new(a.inA, d)) {
        join(a, d);
        fresh = true;
      }
    }
    const int rn = round + 1 <= kIncRounds ? round + 1 : kIncRounds;
    push_block1(fresh, d, a.light, &a.ic->cl[rn], round_base(a.ic->cl, rn), wq.tmp);
  }
}

// Every kernel leaves the snapshot alone once validation has failed (the
// dependency offsets of the appended futures are trusted only then).
__device__ inline bool invalid(const IncArgs& a) { return a.ctrl->status != 0; }

// The appended futures' membership bits, one word per thread (every bit is
// clear when this runs).
__global__ __launch_bounds__(kIncThreads) void k_inc_mark(IncArgs a) {
  if (invalid(a)) return;
  const int64_t lo = a.n_prev, hi = a.p.N;
  if (hi <= lo) return;
  const int64_t w0 = lo >> 5, w1 = (hi - 1) >> 5;
  for (int64_t w = w0 + int64_t(blockIdx.x) * kIncThreads + threadIdx.x; w <= w1;
       w += int64_t(gridDim.x) * kIncThreads) {
    const int64_t b0 = w * 32 > lo ? w * 32 : lo, b1 = w * 32 + 32 < hi ? w * 32 + 32 : hi;
    const uint32_t hi_mask = b1 - w * 32 >= 32 ? 0xFFFFFFFFu : ((1u << uint32_t(b1 - w * 32)) - 1u);
    const uint32_t lo_mask = ~((1u << uint32_t(b0 - w * 32)) - 1u);
    a.inA[w] = hi_mask & lo_mask;
  }
}

// Round 0 takes the seeds (completed ids of the log, then the appended
// range); round r >= 1 the futures handed on: heavy ones expanded one per
// workgroup, the others one per thread.  Then the workgroup drains its queue.
// One round of the closure, this workgroup's share of it (every thread of the
// workgroup calls; the workgroup's queues are empty on entry and on return).
__device__ void close_round(const IncArgs& a, int r, const WgQueue& wq) {
  const uint32_t nh = r ? ld_count(&a.ic->ch[r]) : 0u, nl = r ? ld_count(&a.ic->cl[r]) : 0u;
  const int64_t n_app = a.p.N - a.n_prev;
  const int64_t n_seed = r ? 0 : a.n_log + (n_app > 0 ? n_app : 0);
  if (nh == 0 && nl == 0 && n_seed == 0) return;  // the same on every thread
  if (threadIdx.x == 0) {
    *wq.n = 0;
    *wq.hn = 0;
    *wq.htaken = 0;
  }
  __syncthreads();
  // every lane of a wave runs each iteration (the walks work wave by wave)
  for (int64_t i0 = int64_t(blockIdx.x) * kIncThreads; i0 < n_seed; i0 += int64_t(gridDim.x) * kIncThreads) {
    const int64_t i = i0 + threadIdx.x;
    int32_t v = -1;
    if (i < n_seed) {
      if (i >= a.n_log) {  // appended: already members (k_inc_mark)
        v = int32_t(a.n_prev + (i - a.n_log));
        join(a, v);
      } else {
        const int32_t c = a.log[i];
        // an id out of range is counted by the completion kernel
        if (c >= 0 && int64_t(c) < a.p.N && bit_set_new(a.inA, c)) {
          join(a, c);
          v = c;
        }
      }
    }
    close_walk(a, v, r, wq);
  }
  const uint32_t bh = round_base(a.ic->ch, r), bl = round_base(a.ic->cl, r);
  for (uint32_t h = blockIdx.x; h < nh; h += gridDim.x) close_expand(a, a.heavy[bh + h], r, wq);
  for (uint32_t i0 = blockIdx.x * kIncThreads; i0 < nl; i0 += gridDim.x * kIncThreads) {
    const uint32_t i = i0 + threadIdx.x;
    close_walk(a, i < nl ? a.light[bl + i] : -1, r, wq);
  }
  wg_drain(wq, [&](int32_t v) { close_walk(a, v, r, wq); }, [&](int32_t v) { close_expand(a, v, r, wq); });
}

// The workgroup's LDS queues.
#define NALAR_INC_QUEUES(keep)                                                  \
  __shared__ int32_t s_q[kIncQueue], s_hq[kIncHeavyQueue];                      \
  __shared__ int s_n, s_hn, s_htaken;                                           \
  __shared__ uint32_t s_tmp[kIncThreads / kWave + 2];                           \
  const WgQueue wq{s_q, &s_n, s_hq, &s_hn, s_tmp, &s_htaken, keep}

__global__ __launch_bounds__(kIncThreads) void k_inc_close(IncArgs a, int r) {
  if (invalid(a)) return;
  NALAR_INC_QUEUES(false);
  close_round(a, r, wq);
}

// Rounds kIncTail .. kIncRounds - 1 by one workgroup (they are usually empty,
// and one launch costs less than one per round).  What a round hands on is
// read by the same workgroup in the next one.
__global__ __launch_bounds__(kIncThreads) void k_inc_close_tail(IncArgs a) {
  if (invalid(a)) return;
  NALAR_INC_QUEUES(true);
  for (int r = kIncTail; r < kIncRounds; ++r) {
    close_round(a, r, wq);
    __syncthreads();
  }
}

// --------------------------------------------------------------------- scan

// Pending pushes of one lane to one dependency: merged while the target
// repeats (children of one future are appended next to one another).
struct Pend {
  int32_t d = -1;
  int64_t v = 0;
};

__device__ inline void flush_max(int64_t* mx, Pend& p) {
  if (p.d >= 0) atomicMax(reinterpret_cast<long long*>(&mx[p.d]), (long long)p.v);
  p.d = -1;
}

__device__ inline void flush_cnt(int32_t* cnt, Pend& p) {
  if (p.d >= 0) atomicAdd(&cnt[p.d], int32_t(p.v));
  p.d = -1;
}

// The last pushes of a wave: one atomic when every lane holds the same target.
__device__ inline void flush_wave_max(int64_t* mx, Pend& p) {
  const uint64_t act = ballot(p.d >= 0);
  if (act == 0) return;
  const int lead = __builtin_ctzll(act);
  const int32_t first = readlane_i32(p.d, lead);
  if ((act & (act - 1)) != 0 && ballot(p.d >= 0 && p.d != first) == 0) {
    const int64_t m = wave_max_i64(p.d >= 0 ? p.v : INT64_MIN);
    if (lane_id() == lead) atomicMax(reinterpret_cast<long long*>(&mx[first]), (long long)m);
    p.d = -1;
    return;
  }
  flush_max(mx, p);
}

__device__ inline void flush_wave_cnt(int32_t* cnt, Pend& p) {
  const uint64_t act = ballot(p.d >= 0);
  if (act == 0) return;
  const int lead = __builtin_ctzll(act);
  const int32_t first = readlane_i32(p.d, lead);
  if ((act & (act - 1)) != 0 && ballot(p.d >= 0 && p.d != first) == 0) {
    const int64_t s = wave_sum_i64(p.d >= 0 ? p.v : 0);
    if (lane_id() == lead) atomicAdd(&cnt[first], int32_t(s));
    p.d = -1;
    return;
  }
  flush_cnt(cnt, p);
}

// Appends the lanes' values to a list with one atomic per wave (every lane of
// the wave calls).
__device__ inline void push_wave(bool in, int32_t v, int32_t* list, uint32_t* n) {
  const uint64_t m = ballot(in);
  if (m == 0) return;
  const int lead = __builtin_ctzll(m);
  uint32_t b = 0;
  if (lane_id() == lead) b = atomicAdd(n, uint32_t(__popcll(m)));
  b = uint32_t(readlane_i32(int32_t(b), lead));
  if (in) list[b + lanes_below(m)] = v;
}

// A workgroup takes kScanPer x kIncThreads consecutive futures, thread t the
// futures t, t + kIncThreads, ... of them (so every load of a wave is
// coalesced), and issues the loads of all of them together, stage by stage
// (offsets, membership and done flags; the first dependency; its done flag
// and membership), so that the gathers of a thread overlap; further
// dependencies (rare in the graphs this serves) are visited one by one after.
// A thread's futures lie kIncThreads apart, so a run of futures with one
// common dependency (the children of a hub) still merges its pushes per lane.
__global__ __launch_bounds__(kIncThreads) void k_inc_scan(IncArgs a) {
  if (invalid(a)) return;
  __shared__ uint32_t s_tmp[kIncThreads / kWave + 2];
  const int64_t N = a.p.N;
  Pend pm, pc;
  uint32_t members = 0;
  const int64_t step = int64_t(gridDim.x) * kIncThreads * kScanPer;
  for (int64_t g0 = int64_t(blockIdx.x) * kIncThreads * kScanPer; g0 < N; g0 += step) {
    const int64_t v0 = g0 + int64_t(threadIdx.x);
    int32_t o0[kScanPer], o1[kScanPer], d0[kScanPer];
    bool in[kScanPer], dn[kScanPer], dd[kScanPer], din[kScanPer];
#pragma unroll
    for (int j = 0; j < kScanPer; ++j) {
      const int64_t v = v0 + int64_t(j) * kIncThreads;
      const bool ok = v < N;
      o0[j] = ok ? a.p.dep_off[v] : 0;
      o1[j] = ok ? a.p.dep_off[v + 1] : 0;
      in[j] = ok && bit_get(a.inA, int32_t(v));
      dn[j] = ok ? a.p.done[v] != 0 : true;
    }
#pragma unroll
    for (int j = 0; j < kScanPer; ++j) {
      const bool one = o1[j] > o0[j] && o1[j] - o0[j] <= kIncHeavy;
      d0[j] = one ? a.p.dep_idx[o0[j]] : -1;
    }
#pragma unroll
    for (int j = 0; j < kScanPer; ++j) {
      const bool okd = d0[j] >= 0 && int64_t(d0[j]) < N;
      dd[j] = okd ? bit_get(a.dnb, d0[j]) : true;
      din[j] = okd && bit_get(a.inA, d0[j]);
    }
    uint32_t rmask = 0;
#pragma unroll
    for (int j = 0; j < kScanPer; ++j) {
      const int64_t v = v0 + int64_t(j) * kIncThreads;
      bool ready = false, heavy = false;
      if (v < N) {
        members += in[j] ? 1u : 0u;
        if (o1[j] - o0[j] > kIncHeavy) {
          heavy = true;
        } else {
          bool blocked = false;
          int64_t rv = 0;
          bool have_rv = false;
          for (int32_t e = o0[j]; e < o1[j]; ++e) {
            int32_t d;
            bool d_done, d_in;
            if (e == o0[j]) {  // the first dependency, loaded above
              d = d0[j];
              d_done = dd[j];
              d_in = din[j];
            } else {
              d = a.p.dep_idx[e];
              const bool okd = d >= 0 && int64_t(d) < N;
              d_done = okd ? bit_get(a.dnb, d) : true;
              d_in = okd && bit_get(a.inA, d);
            }
            if (d < 0 || int64_t(d) >= N) continue;  // reported by the closure or an earlier pass
            blocked |= !d_done;
            if (in[j]) {
              if (d != pc.d) {
                flush_cnt(a.cntA, pc);
                pc.d = d;
                pc.v = 0;
              }
              pc.v += 1;
            } else if (d_in) {
              if (!have_rv) {
                rv = a.rem[v];
                have_rv = true;
              }
              if (d != pm.d) {
                flush_max(a.mxA, pm);
                pm.d = d;
                pm.v = rv;
              }
              pm.v = rv > pm.v ? rv : pm.v;
            }
          }
          ready = !dn[j] && !blocked;
        }
      }
      if (ready) rmask |= 1u << j;
      push_wave(heavy, int32_t(v), a.heavy, &a.ic->scan_heavy);  // rare
    }
    push_block(rmask, v0, a.rlist, &a.ic->r_n, 0u, s_tmp, kIncThreads);
  }
  flush_wave_cnt(a.cntA, pc);
  flush_wave_max(a.mxA, pm);
  const int64_t mt = wave_sum_i64(int64_t(members));
  if (lane_id() == 0 && mt) atomicAdd(&a.ic->a_n, uint32_t(mt));
}

// The futures with more than kIncHeavy dependencies, one per workgroup.
__global__ __launch_bounds__(kIncThreads) void k_inc_scan_heavy(IncArgs a) {
  if (invalid(a)) return;
  __shared__ int s_blocked;
  const uint32_t nh = a.ic->scan_heavy;
  for (uint32_t h = blockIdx.x; h < nh; h += gridDim.x) {
    const int32_t v = a.heavy[h];
    if (threadIdx.x == 0) s_blocked = 0;
    __syncthreads();
    const bool in = bit_get(a.inA, v);
    const int32_t o0 = a.p.dep_off[v], o1 = a.p.dep_off[v + 1];
    bool blocked = false;
    int64_t rv = 0;
    if (!in && int64_t(v) < a.n_prev) rv = a.rem[v];
    for (int32_t e = o0 + int32_t(threadIdx.x); e < o1; e += kIncThreads) {
      const int32_t d = a.p.dep_idx[e];
      if (d < 0 || int64_t(d) >= a.p.N) continue;
      blocked |= !bit_get(a.dnb, d);
      if (in) atomicAdd(&a.cntA[d], 1);
      else if (bit_get(a.inA, d)) atomicMax(reinterpret_cast<long long*>(&a.mxA[d]), (long long)rv);
    }
    if (blocked) s_blocked = 1;
    __syncthreads();
    if (threadIdx.x == 0 && a.p.done[v] == 0 && s_blocked == 0) a.rlist[atomicAdd(&a.ic->r_n, 1u)] = v;
    __syncthreads();
  }
}

// -------------------------------------------------------------------- sweep

// A device-scope max that is skipped when a plain read of the location
// already shows a value at least as large.  Within the sweep a member's max
// only grows (the closure zeroed it, the scan and the sweep only raise it),
// so a stale read is never above the true value and skipping stays exact; it
// saves a memory-side atomic whenever an earlier push was larger.  (In the
// scan the extra reads cost more than the atomics they save.)
__device__ inline void max_if_larger(int64_t* p, int64_t v) {
  if (v > __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP))
    __hip_atomic_fetch_max(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// One push of a finalised member: its rem into d's max, then d's count down
// by k; returns the count before.  Every access to the maxima and counts in
// the sweep is a device-scope atomic, so their values meet where such
// atomics are coherent, and the only order needed is the max before the
// count: the wait makes the max complete there before the count is touched,
// so the member that sees the count reach zero (and then loads the max
// atomically) sees every push.  No cache write-back or invalidation is
// needed: the only other access is the read that lets max_if_larger skip a
// max, and a stale value there is never above the true one.
__device__ inline int32_t push_count(const IncArgs& a, int32_t d, int64_t r, int32_t k) {
  max_if_larger(&a.mxA[d], r);
  __asm__ __volatile__("s_waitcnt vmcnt(0)" ::: "memory");
  return __hip_atomic_fetch_add(&a.cntA[d], -k, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Pushes the lanes' rem r to their dependencies d (d < 0: none) with one
// pair of atomics per group of lanes holding the same d (a fan-in), else one
// pair per lane; returns whether this lane brought d's count to zero (one
// lane per d).  Every lane of the wave calls.
__device__ inline bool wave_push(const IncArgs& a, int32_t d, int64_t r) {
  uint64_t pend = ballot(d >= 0);
  bool zero = false;
  for (int it = 0; it < 2 && pend != 0; ++it) {
    const int lead = __builtin_ctzll(pend);
    const int32_t t = readlane_i32(d, lead);
    const bool in = ((pend >> lane_id()) & 1u) && d == t;
    const uint64_t grp = ballot(in);
    const int n = __popcll(grp);
    if (n < 2) break;
    const int64_t m = wave_max_i64(in ? r : INT64_MIN);
    if (lane_id() == lead) zero = push_count(a, t, m, n) == n;
    pend &= ~grp;
  }
  if ((pend >> lane_id()) & 1u) zero = push_count(a, d, r, 1) == 1;
  return zero;
}

// u's closure consumers are all finalised: rem(u) = est' + max, pushed to its
// dependencies; a dependency whose count reaches zero is finalised next (by
// this lane if it is the first, else through the workgroup's queue).  Every
// lane of the wave calls (u = -1: nothing).
__device__ void sweep_walk(const IncArgs& a, int32_t u, int round, uint32_t& fin, const WgQueue& wq) {
  while (ballot(u >= 0) != 0) {
    int32_t d1 = -1;  // the one dependency of a single-dependency future
    int64_t r = 0;
    if (u >= 0) {
      const int64_t est = bit_get(a.dnb, u) ? 0 : a.p.est[u];
      const int64_t m = __hip_atomic_load(&a.mxA[u], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      r = est + m;
      if (r > NALAR_REM_MAX) {
        r = NALAR_REM_MAX + 1;
        flag(a.ctrl, kStRange);
      }
      a.rem[u] = r;
      ++fin;
      const int32_t o0 = a.p.dep_off[u], o1 = a.p.dep_off[u + 1];
      if (o1 - o0 > kIncHeavy) {
        wg_push_heavy(wq, a.heavy, a.ic->sh, round, u, o1 - o0);
        u = -1;
      } else if (o1 - o0 == 1) {
        const int32_t d = a.p.dep_idx[o0];
        if (d >= 0 && int64_t(d) < a.p.N && d != u) d1 = d;
        u = -1;
      } else {
        int32_t next = -1;
        for (int32_t e = o0; e < o1; ++e) {
          const int32_t d = a.p.dep_idx[e];
          if (d < 0 || int64_t(d) >= a.p.N || d == u) continue;
          if (push_count(a, d, r, 1) == 1) {
            if (next < 0) next = d;
            else wg_push(wq, a.light, a.ic->sl, round, d);
          }
        }
        u = next;
      }
    }
    if (wave_push(a, d1, r)) u = d1;
  }
}

__device__ inline void add_fin(const IncArgs& a, uint32_t fin) {
  const int64_t t = wave_sum_i64(int64_t(fin));
  if (lane_id() == 0 && t) atomicAdd(&a.ic->fin, uint32_t(t));
}

// The sweep's first round: every closure member without closure consumers,
// listed before any member is finalised (a walk may bring another member's
// count to zero while this list is taken, and that member is then the
// walker's), one thread per word of the membership bits.
__global__ __launch_bounds__(kIncThreads) void k_inc_front0(IncArgs a) {
  if (invalid(a)) return;
  __shared__ uint32_t s_tmp[kIncThreads / kWave + 2];
  const int64_t words = (a.p.N + 31) / 32;
  const int64_t step = int64_t(gridDim.x) * kIncThreads;
  // the loop runs the same number of times on every thread of the workgroup
  for (int64_t w0 = int64_t(blockIdx.x) * kIncThreads; w0 < words; w0 += step) {
    const int64_t w = w0 + threadIdx.x;
    uint32_t bits = w < words ? a.inA[w] : 0u;
    uint32_t zmask = 0;
    while (bits) {
      const int b = __builtin_ctz(bits);
      bits &= bits - 1;
      if (a.cntA[w * 32 + b] == 0) zmask |= 1u << b;
    }
    push_block(zmask, w * 32, a.light, &a.ic->sl[0], 0u, s_tmp);
  }
}

// A finalised heavy member's rem pushed to its dependencies by the whole
// workgroup; the dependencies it finalises go to the next round, where every
// workgroup shares their walks.
__device__ inline void sweep_expand(const IncArgs& a, int32_t u, int round, uint32_t& fin, const WgQueue& wq) {
  const int64_t ru = a.rem[u];
  const int32_t o0 = a.p.dep_off[u], o1 = a.p.dep_off[u + 1];
  const int rn = round + 1 <= kIncRounds ? round + 1 : kIncRounds;
  for (int32_t e0 = o0; e0 < o1; e0 += int32_t(blockDim.x)) {
    const int32_t e = e0 + int32_t(threadIdx.x);
    bool zero = false;
    int32_t d = -1;
    if (e < o1) {
      d = a.p.dep_idx[e];
      if (d >= 0 && int64_t(d) < a.p.N && d != u) zero = push_count(a, d, ru, 1) == 1;
    }
    push_block1(zero, d, a.light, &a.ic->sl[rn], round_base(a.ic->sl, rn), wq.tmp);
  }
  (void)fin;
}

// One round of the sweep, this workgroup's share of it (as close_round).
__device__ void sweep_round(const IncArgs& a, int r, const WgQueue& wq, uint32_t& fin) {
  const uint32_t nh = ld_count(&a.ic->sh[r]), nl = ld_count(&a.ic->sl[r]);
  if (nh == 0 && nl == 0) return;  // the same on every thread
  if (threadIdx.x == 0) {
    *wq.n = 0;
    *wq.hn = 0;
    *wq.htaken = 0;
  }
  __syncthreads();
  const uint32_t bh = round_base(a.ic->sh, r), bl = round_base(a.ic->sl, r);
  for (uint32_t h = blockIdx.x; h < nh; h += gridDim.x) sweep_expand(a, a.heavy[bh + h], r, fin, wq);
  for (uint32_t i0 = blockIdx.x * kIncThreads; i0 < nl; i0 += gridDim.x * kIncThreads) {
    const uint32_t i = i0 + threadIdx.x;
    sweep_walk(a, i < nl ? a.light[bl + i] : -1, r, fin, wq);
  }
  wg_drain(wq, [&](int32_t v) { sweep_walk(a, v, r, fin, wq); },
           [&](int32_t v) { sweep_expand(a, v, r, fin, wq); });
}

__global__ __launch_bounds__(kIncThreads) void k_inc_sweep(IncArgs a, int r) {
  if (invalid(a)) return;
  NALAR_INC_QUEUES(false);
  uint32_t fin = 0;
  sweep_round(a, r, wq, fin);
  add_fin(a, fin);
}

// Rounds kIncTail .. kIncRounds - 1 of the sweep by one workgroup.
__global__ __launch_bounds__(kIncThreads) void k_inc_sweep_tail(IncArgs a) {
  if (invalid(a)) return;
  NALAR_INC_QUEUES(true);
  uint32_t fin = 0;
  for (int r = kIncTail; r < kIncRounds; ++r) {
    sweep_round(a, r, wq, fin);
    __syncthreads();
  }
  add_fin(a, fin);
}

// -------------------------------------------------------------------- ready

// Incomplete rounds or an unfinished closure: status for the host.
__device__ inline void check_rounds(const IncArgs& a) {
  const IncCtrl* ic = a.ic;
  if (ic->cl[kIncRounds] | ic->ch[kIncRounds] | ic->sl[kIncRounds] | ic->sh[kIncRounds])
    flag(a.ctrl, kStIncomplete);
  else if (ic->fin != ic->a_n)
    flag(a.ctrl, kStCycle);  // some member's closure consumers never all finalised
}

__device__ inline int64_t key_of(uint32_t policy, int64_t rem, int64_t dl) {
  if (policy & NALAR_ORDER_LPT) return -rem;
  if (policy & NALAR_ORDER_SRTF) return rem;
  return dl - rem;
}

// The ready futures: key, bin (splitters in LDS), route, slot.  Per chunk of
// kReadyPer * T futures, the bins' LDS counts give each future its rank
// inside the chunk's part of its bin, and one atomic per bin claims that part.
__global__ __launch_bounds__(kIncThreads) void k_inc_ready(IncArgs a) {
  constexpr int T = kIncThreads;
  for (int64_t i = int64_t(blockIdx.x) * T + threadIdx.x; i < a.bk_clear_n; i += int64_t(gridDim.x) * T)
    a.bk_clear[i] = 0;  // the next pass's bin counters
  Ctrl* ctrl = a.ctrl;
  if (ctrl->status != 0) return;
  if (blockIdx.x == 0 && threadIdx.x == 0) check_rounds(a);
  if ((ctrl->status | ctrl->status_sweep) != 0) return;
  extern __shared__ __align__(16) unsigned char smem[];
  const int M = int(a.p.M);
  const int nb = a.bk.nb;
  unsigned char* sp = smem;
  int64_t* s_split = reinterpret_cast<int64_t*>(sp); sp += 8 * size_t(kBinMax);
  int64_t* s_load = reinterpret_cast<int64_t*>(sp); sp += 8 * size_t(M);
  double* s_inv = reinterpret_cast<double*>(sp); sp += 8 * size_t(M);
  int32_t* s_type = reinterpret_cast<int32_t*>(sp); sp += 4 * size_t(M);
  int32_t* s_idx = reinterpret_cast<int32_t*>(sp); sp += 4 * size_t(M);
  int32_t* s_speed = reinterpret_cast<int32_t*>(sp); sp += 4 * size_t(M);
  int32_t* s_pos = reinterpret_cast<int32_t*>(sp); sp += 4 * size_t(M);
  uint32_t* s_run = reinterpret_cast<uint32_t*>(sp); sp += 4 * size_t(kTypeDirect);
  uint32_t* s_prun = reinterpret_cast<uint32_t*>(sp); sp += 4 * size_t(kTypeDirect);
  uint32_t* s_cnt = reinterpret_cast<uint32_t*>(sp); sp += 4 * size_t(kBinMax);
  uint32_t* s_base = reinterpret_cast<uint32_t*>(sp);
  __shared__ int64_t s_red[3][T / kWave];
  const int tid = threadIdx.x;
  for (int i = tid; i < M; i += T) {
    s_load[i] = a.itab.load[i];
    s_inv[i] = a.itab.inv_speed[i];
    s_type[i] = a.itab.type[i];
    s_idx[i] = a.itab.idx[i];
    s_speed[i] = a.itab.speed[i];
    s_pos[i] = a.itab.pos_of[i];
  }
  for (int t = tid; t < kTypeDirect; t += T) {
    s_run[t] = a.itab.run[t];
    s_prun[t] = a.itab.prun[t];
  }
  for (int i = tid; i < nb - 1; i += T) s_split[i] = a.bk.split[i];
  for (int i = tid; i < nb; i += T) s_cnt[i] = 0;
  __syncthreads();
  const uint32_t policy = a.p.policy;
  const bool out_slack = (policy & (NALAR_ORDER_LPT | NALAR_ORDER_SRTF)) != 0;
  const int64_t R = a.ic->r_n;
  int64_t tmin = INT64_MAX, tmax = INT64_MIN, tready = 0;
  constexpr int64_t kChunk = int64_t(kReadyPer) * T;
  for (int64_t c0 = int64_t(blockIdx.x) * kChunk; c0 < R; c0 += int64_t(gridDim.x) * kChunk) {
    int32_t v[kReadyPer];
    int64_t key[kReadyPer], rem[kReadyPer], dl[kReadyPer];
    uint32_t bin[kReadyPer], rk[kReadyPer];
#pragma unroll
    for (int j = 0; j < kReadyPer; ++j) {
      const int64_t i = c0 + j * T + tid;
      v[j] = -1;
      key[j] = rem[j] = dl[j] = 0;
      bin[j] = rk[j] = 0;
      if (i < R) {
        v[j] = a.rlist[i];
        rem[j] = a.rem[v[j]];
        dl[j] = a.p.deadline[a.p.wf[v[j]]] - a.p.now;
        key[j] = key_of(policy, rem[j], dl[j]);
      }
    }
    for (int st = nb >> 1; st > 0; st >>= 1) {
#pragma unroll
      for (int j = 0; j < kReadyPer; ++j)
        if (v[j] >= 0 && s_split[bin[j] + st - 1] <= key[j]) bin[j] += st;
    }
#pragma unroll
    for (int j = 0; j < kReadyPer; ++j)
      if (v[j] >= 0) rk[j] = atomicAdd(&s_cnt[bin[j]], 1u);
    __syncthreads();
    {  // one segment per bin for the chunk: every thread's atomics in flight together
      constexpr int kPerT = kBinMax / T;
      uint32_t c[kPerT];
#pragma unroll
      for (int q = 0; q < kPerT; ++q) {
        const int t = tid + q * T;
        c[q] = t < nb ? s_cnt[t] : 0u;
      }
#pragma unroll
      for (int q = 0; q < kPerT; ++q) c[q] = c[q] ? add_agent(a.bk.cnt + tid + q * T, c[q]) : 0u;
#pragma unroll
      for (int q = 0; q < kPerT; ++q) {
        const int t = tid + q * T;
        if (t < nb) {
          s_base[t] = c[q];
          s_cnt[t] = 0;
        }
      }
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kReadyPer; ++j) {
      if (v[j] < 0) continue;
      const int32_t u = v[j];
      int32_t route;
      int64_t cost;
      route_future(a.p.type[u], a.p.est[u], a.p.loc[u], int32_t(M), a.p.mig, s_type, s_idx, s_load, s_speed,
                   s_inv, s_pos, s_run, (policy & NALAR_ROUTE_STATEFUL) != 0, route, cost, s_prun);
      const uint32_t slot = rk[j] + s_base[bin[j]];
      if (slot < uint32_t(a.bk.cap)) {
        int64_t* sl = reinterpret_cast<int64_t*>(a.bk.slot + int64_t(bin[j]) * a.bk.cap + slot);
        sl[0] = key[j];
        sl[1] = cost;
        sl[2] = int64_t(uint64_t(uint32_t(u)) | (uint64_t(uint32_t(slot_pack(route, 0))) << 32));
      } else {
        st_relaxed_agent(&ctrl->bucket_overflow, 1u);
      }
      if (out_slack) a.stg_oslack[u] = dl[j] - rem[j];
      tmin = key[j] < tmin ? key[j] : tmin;
      tmax = key[j] > tmax ? key[j] : tmax;
      tready += 1;
    }
    __syncthreads();  // the counters are clean again before the next chunk
  }
  const int64_t mn = wave_min_i64(tmin), mx = wave_max_i64(tmax), rd = wave_sum_i64(tready);
  const int wv = tid / kWave;
  if (lane_id() == 0) {
    s_red[0][wv] = mn;
    s_red[1][wv] = mx;
    s_red[2][wv] = rd;
  }
  __syncthreads();
  if (tid == 0) {
    int64_t a0 = INT64_MAX, a1 = INT64_MIN, a2 = 0;
    for (int x = 0; x < T / kWave; ++x) {
      a0 = s_red[0][x] < a0 ? s_red[0][x] : a0;
      a1 = s_red[1][x] > a1 ? s_red[1][x] : a1;
      a2 += s_red[2][x];
    }
    if (a2 > 0) {
      const int slot = blockIdx.x & (kParts - 1);
      __hip_atomic_fetch_min(&ctrl->part_min[slot], a0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_fetch_max(&ctrl->part_max[slot], a1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      add_agent(&ctrl->part_cnt[slot], a2);
    }
  }
}

// Word i of the membership bits cleared, and of the done bits packed from
// the done flags of futures 32i .. 32i+31 (the gathers of dependencies' flags
// then read 1/8 of the bytes, a bitmap that stays in the L2).
__global__ __launch_bounds__(kIncThreads) void k_inc_pack(IncArgs a) {
  const int64_t N = a.p.N, nw = (N + 31) / 32;
  for (int64_t i = int64_t(blockIdx.x) * kIncThreads + threadIdx.x; i < nw; i += int64_t(gridDim.x) * kIncThreads) {
    const int64_t v0 = 32 * i;
    uint32_t bits = 0;
    if (v0 + 32 <= N) {  // 32 flags in two aligned 16-byte loads (the array is 256-byte aligned)
      const uint4* q = reinterpret_cast<const uint4*>(a.p.done + v0);
      const uint4 x = q[0], y = q[1];
      const uint32_t w[8] = {x.x, x.y, x.z, x.w, y.x, y.y, y.z, y.w};
#pragma unroll
      for (int k = 0; k < 8; ++k)
#pragma unroll
        for (int b = 0; b < 4; ++b) bits |= uint32_t(((w[k] >> (8 * b)) & 0xFFu) != 0u) << (4 * k + b);
    } else {
      for (int64_t v = v0; v < N; ++v) bits |= uint32_t(a.p.done[v] != 0) << uint32_t(v - v0);
    }
    a.inA[i] = 0;
    a.dnb[i] = bits;
  }
}

__global__ __launch_bounds__(kIncThreads) void k_inc_clear(uint32_t* p, int64_t n) {
  for (int64_t i = int64_t(blockIdx.x) * kIncThreads + threadIdx.x; i < n; i += int64_t(gridDim.x) * kIncThreads)
    p[i] = 0;
}

int inc_grid(int64_t n, int cap) {
  int64_t g = (n + kIncThreads - 1) / kIncThreads;
  if (g < 1) g = 1;
  if (g > cap) g = cap;
  return int(g);
}

}  // namespace

size_t inc_ready_lds(int64_t M) {
  return 8 * size_t(kBinMax) + 32 * size_t(M) + 8 * size_t(kTypeDirect) + 8 * size_t(kBinMax);
}

hipError_t prepare_inc_kernels() {
  return hipFuncSetAttribute(reinterpret_cast<const void*>(&k_inc_ready),
                             hipFuncAttributeMaxDynamicSharedMemorySize, int(inc_ready_lds(NALAR_MAX_INSTANCES)));
}

hipError_t launch_inc_clear(hipStream_t s, uint32_t* p, int64_t n) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_inc_clear, dim3(inc_grid(n, 2048)), dim3(kIncThreads), 0, s, p, n);
  return hipGetLastError();
}

hipError_t launch_inc_pack(hipStream_t s, const IncArgs& a) {
  const int64_t nw = (a.p.N + 31) / 32;
  if (nw <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_inc_pack, dim3(inc_grid(nw, 2048)), dim3(kIncThreads), 0, s, a);
  return hipGetLastError();
}

constexpr const char* kCloseNames[kIncRounds] = {"inc_close_r0", "inc_close_r1", "inc_close_r2", "inc_close_r3",
                                                  "inc_close_r4", "inc_close_r5", "inc_close_r6", "inc_close_r7"};
constexpr const char* kSweepNames[kIncRounds] = {"inc_sweep_r0", "inc_sweep_r1", "inc_sweep_r2", "inc_sweep_r3",
                                                  "inc_sweep_r4", "inc_sweep_r5", "inc_sweep_r6", "inc_sweep_r7"};
static_assert(kIncRounds == 8, "one name per round");

hipError_t launch_inc_closure(hipStream_t s, const IncArgs& a, int cus, void (*mark)(void*, const char*),
                              void* ctx) {
  const int64_t seeds = a.n_log + (a.p.N - a.n_prev);
  mark(ctx, "inc_mark");
  hipLaunchKernelGGL(k_inc_mark, dim3(inc_grid((a.p.N - a.n_prev) / 32 + 2, 1024)), dim3(kIncThreads), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  mark(ctx, kCloseNames[0]);
  hipLaunchKernelGGL(k_inc_close, dim3(inc_grid(seeds, 4096)), dim3(kIncThreads), 0, s, a, 0);
  e = hipGetLastError();
  for (int r = 1; r < kIncTail && e == hipSuccess; ++r) {
    mark(ctx, kCloseNames[r]);
    hipLaunchKernelGGL(k_inc_close, dim3(r < 2 ? 4 * cus : cus), dim3(kIncThreads), 0, s, a, r);
    e = hipGetLastError();
  }
  if (e != hipSuccess) return e;
  mark(ctx, "inc_close_tail");
  hipLaunchKernelGGL(k_inc_close_tail, dim3(1), dim3(kIncThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_inc_scan(hipStream_t s, const IncArgs& a, int cus) {
  hipLaunchKernelGGL(k_inc_scan, dim3(inc_grid((a.p.N + kScanPer - 1) / kScanPer, 16 * cus)),
                     dim3(kIncThreads), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_inc_scan_heavy, dim3(2 * cus), dim3(kIncThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_inc_sweep(hipStream_t s, const IncArgs& a, int cus, void (*mark)(void*, const char*),
                            void* ctx) {
  mark(ctx, "inc_front0");
  hipLaunchKernelGGL(k_inc_front0, dim3(inc_grid((a.p.N + 31) / 32, 8 * cus)), dim3(kIncThreads), 0, s, a);
  hipError_t e = hipGetLastError();
  for (int r = 0; r < kIncTail && e == hipSuccess; ++r) {
    mark(ctx, kSweepNames[r]);
    hipLaunchKernelGGL(k_inc_sweep, dim3(4 * cus), dim3(kIncThreads), 0, s, a, r);
    e = hipGetLastError();
  }
  if (e != hipSuccess) return e;
  mark(ctx, "inc_sweep_tail");
  hipLaunchKernelGGL(k_inc_sweep_tail, dim3(1), dim3(kIncThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_inc_ready(hipStream_t s, const IncArgs& a, int cus) {
  hipLaunchKernelGGL(k_inc_ready, dim3(4 * cus), dim3(kIncThreads), inc_ready_lds(a.p.M), s, a);
  return hipGetLastError();
}

}  // namespace nalar
