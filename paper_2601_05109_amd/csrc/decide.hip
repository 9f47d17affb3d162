// Per-event decisions: the one-level design of Section 6.3 (Table 4), in
// which the central controller decides every future event itself instead of
// installing a policy once per pass.  For each event future v, against the
// view the last pass produced (every future's remaining critical path and the
// current order of the ready futures):
//   slack[v] = deadline[wf[v]] - now - rem[v]
//   route[v] = the argmin of (cost, instance) over the instances of v's type,
//              cost = load + floor(est*1000/speed) + migration penalty unless
//              the instance holds v's state (or v's stateful pin)
//   rank[v]  = the number of entries of the current order that come before v
//              under the pass's order: (-level, key, wf, id), key the slack,
//              -rem (LPT) or rem (SRTF); i.e. v's place in that order
// A future's remaining critical path does not change when it becomes ready
// (its dependencies finishing changes only their own estimates), so the last
// pass's rem is the one a decision needs.
//
// The snapshot is not validated again, but every index a decision follows is
// checked before it is used (an event's workflow and state location, each
// candidate's speed, each order entry's id and workflow), so a snapshot that
// does not match the view gives NALAR_EINVAL rather than a stray access.
//
// One wavefront per event: the instance table is scanned lane-parallel (lane l
// takes instances l, l + 64, ...) and reduced to the lexicographic minimum of
// (cost, instance) with DPP minimum reductions; the rank comes from a 64-way
// search in which every lane probes one entry per round, so an order of R
// entries takes about log_65 R rounds of two dependent loads.
#include "internal.hpp"

namespace nalar {

namespace {

// Whether order entry j comes before the event (its level, key, wf and id).
struct EventKey {
  int lvl;
  int64_t key;
  int32_t wf;
  int32_t v;
};

__device__ inline bool entry_before(const DecideArgs& a, int64_t j, const EventKey& e, bool& bad) {
  const int32_t u = a.order[j];
  if (u < 0 || int64_t(u) >= a.p.N) {
    bad = true;
    return false;
  }
  const int32_t wu = a.p.wf[u];
  if (wu < 0 || int64_t(wu) >= a.p.W) {
    bad = true;
    return false;
  }
  const int lu = a.p.prio ? int(a.p.prio[wu]) : 0;
  int64_t ku;
  if (a.p.policy & NALAR_ORDER_LPT) ku = -a.rem[u];
  else if (a.p.policy & NALAR_ORDER_SRTF) ku = a.rem[u];
  else ku = a.slack[j];
  if (lu != e.lvl) return lu > e.lvl;
  if (ku != e.key) return ku < e.key;
  if (wu != e.wf) return wu < e.wf;
  return u < e.v;
}

__device__ inline void reject(const DecideArgs& a, int64_t ev) {
  if (lane_id() == 0) {
    __hip_atomic_fetch_or(&a.host->aux_status, kStInval, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    a.slack_out[ev] = 0;
    a.route_out[ev] = -1;
    if (a.cost_out) a.cost_out[ev] = INT64_MAX;
    if (a.rank_out) a.rank_out[ev] = -1;
  }
}

__global__ __launch_bounds__(kWave) void k_decide(DecideArgs a) {
  const int ln = lane_id();
  const int64_t ev = blockIdx.x;
  const int32_t v = a.events[ev];
  if (v < 0 || int64_t(v) >= a.p.N) return reject(a, ev);
  const int32_t w = a.p.wf[v];
  const int32_t t = a.p.type[v];
  const int64_t est = a.p.est[v];
  const int32_t loc = a.p.loc[v];
  const int64_t rem = a.rem[v];
  if (w < 0 || int64_t(w) >= a.p.W || loc < -1 || int64_t(loc) >= a.p.M) return reject(a, ev);
  const int64_t slack = (a.p.deadline[w] - a.p.now) - rem;

  // route: stateful pin, else the lexicographic minimum of (cost, instance)
  int32_t route = -1;
  int64_t cost = INT64_MAX;
  const bool pinned = (a.p.policy & NALAR_ROUTE_STATEFUL) && loc >= 0 && a.p.inst_type[loc] == t;
  bool bad = false;
  if (pinned) {
    const int32_t sp = a.p.inst_speed[loc];
    if (sp < 1) return reject(a, ev);
    route = loc;
    cost = a.p.inst_load[loc] + (est * 1000) / int64_t(sp);
  } else {
    int64_t best = INT64_MAX;
    int32_t arg = INT32_MAX;
    for (int64_t i = ln; i < a.p.M; i += kWave) {
      if (a.p.inst_type[i] != t) continue;
      const int32_t sp = a.p.inst_speed[i];
      if (sp < 1) {
        bad = true;
        continue;
      }
      const int64_t c = a.p.inst_load[i] + (est * 1000) / int64_t(sp) +
                        ((loc >= 0 && loc != int32_t(i)) ? a.p.mig : 0);
      if (c < best) {  // ascending i per lane: strict, so a lane keeps its lowest index
        best = c;
        arg = int32_t(i);
      }
    }
    const int64_t m = wave_min_i64(best);
    const int64_t who = wave_min_i64(best == m ? int64_t(arg) : int64_t(INT32_MAX));
    if (m != INT64_MAX) {
      route = int32_t(who);
      cost = m;
    }
    if (ballot(bad) != 0) return reject(a, ev);
  }

  // rank: every j < lo comes before the event, no j >= hi does
  int64_t rank = 0;
  if (a.rank_out) {
    EventKey e;
    e.lvl = a.p.prio ? int(a.p.prio[w]) : 0;
    e.key = (a.p.policy & NALAR_ORDER_LPT) ? -rem : ((a.p.policy & NALAR_ORDER_SRTF) ? rem : slack);
    e.wf = w;
    e.v = v;
    int64_t lo = 0, hi = a.n_order;
    while (lo < hi) {
      const int64_t span = hi - lo;
      // probes: every entry when the range fits the wave, else 64 evenly spaced
      const int64_t q = span <= kWave ? lo + ln : lo + (span * (ln + 1)) / (kWave + 1);
      const bool live = span <= kWave ? ln < span : true;
      const bool before = live && entry_before(a, q, e, bad);
      if (ballot(bad) != 0) return reject(a, ev);
      const uint64_t m = ballot(before);
      const int c = __popcll(m);  // probes ascend, so the "before" ones are lanes [0, c)
      if (span <= kWave) {
        lo += c;
        break;
      }
      const int64_t nlo = c == 0 ? lo : readlane_i64(q, c - 1) + 1;
      const int64_t nhi = c == kWave ? hi : readlane_i64(q, c);
      lo = nlo;
      hi = nhi;
    }
    rank = lo;
  }
  if (ln == 0) {
    a.slack_out[ev] = slack;
    a.route_out[ev] = route;
    if (a.cost_out) a.cost_out[ev] = cost;
    if (a.rank_out) a.rank_out[ev] = rank;
  }
}

}  // namespace

hipError_t launch_decide(hipStream_t s, const DecideArgs& a) {
  if (a.n_events <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_decide, dim3(unsigned(a.n_events)), dim3(kWave), 0, s, a);
  return hipGetLastError();
}

}  // namespace nalar
