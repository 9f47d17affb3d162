// Reference ("oracle") implementation of Nalar's global policy pass.
//
// TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, obviously correct
// CPU definition that the HIP implementation is checked against.  Only the test
// suite, the package smoke check and the benchmark's CPU-baseline leg may load
// it; the product path never calls it.  It shares no source, header, helper or
// constant table with the GPU library.
//
// One single-threaded pass over a snapshot of the global view (the paper's
// global controller runs one single-threaded policy loop, Section 4.2):
//
//   O1  validate the snapshot                                  -> -1 (EINVAL)
//   O2  est'[v] = done[v] ? 0 : est[v]
//   O3  successor lists = transpose of the dependency lists (Table 3:
//       "dependencies" and "consumers")
//   O4  reverse topological order by iterative depth-first post-order over
//       successors; meeting a node still on the stack is a cycle  -> -2 (ECYCLE)
//   O5  remaining critical path, visited in that post-order:
//         rem[v] = est'[v] + max(0, max over successors s of rem[s])
//       (the remaining work by which the SRTF policy ranks jobs, Section 6.2,
//       generalised from a chain of stages to a DAG); rem > 2^62 -> -3 (ERANGE)
//   O6  ready[v] = !done[v] and every dependency of v is done (push-based
//       readiness, Section 4.3.1, property 3)
//   O7  slack[v] = (deadline[wf[v]] - now) - rem[v]              (set_priority,
//       Table 2)
//   O8  route[v] = the instance i of type type[v] minimising
//         cost = load[i] + est[v]*1000/speed[i]   (integer division)
//              + (loc[v] >= 0 and loc[v] != i ? migration cost : 0)
//       scanning i upward with a strict "<", so the lowest index wins ties;
//       route = -1 and cost = INT64_MAX when no instance has the type
//       (route / migrate, Table 2; state locality, Section 4.3.2)
//   O9  order = the ready futures sorted by (slack, wf, v) ascending
//   O10 write rem, order, slack, route, cost and the ready count.
//
// Policy variants (the policy word of nalar_oracle_pass_policy):
//   kLpt       O9 sorts by (-rem, wf, v) instead: the future with the longest
//              remaining processing first (the LPT policy, Section 6.2); slack
//              is still reported as in O7
//   kStateful  O8 for a future whose state lives on an instance of its own
//              type: route = that instance, cost without migration penalty,
//              no other candidate (the stateful directive, Table 1, and the
//              managed-state routing guarantee, Section 4.3.2); other futures
//              are routed as in O8
//   kGreedy    routing is redone after O9, one future at a time in the output
//              order: each takes the cheapest candidate (the O8 rule, or its
//              pin under kStateful) under the loads left by the futures before
//              it, then adds its service time on that instance,
//              est*1000/speed, to that instance's load (routing that balances
//              load across instances, Section 6.1); a load above 2^62 -> -3
//   kSrtf      O9 sorts by (rem, wf, v) instead: the future with the least
//              remaining work first (shortest remaining time first, the
//              policy that minimises job completion time, Section 6.2); slack
//              is still reported as in O7.  kLpt and kSrtf together -> -1
//   kWeighted  after O9, the ready futures of each type that has instances of
//              positive weight are dealt to those instances in proportion to
//              their weights (route with a list of instances and weights,
//              Table 2): the futures of type t, taken in output order, get
//              sequence numbers j = 0, 1, 2, ...; with the instances of type t
//              and positive weight listed by ascending index and S their total
//              weight, future j goes to the instance whose run of w[i]
//              consecutive numbers in 0..S-1 holds j mod S (the first w[0]
//              numbers to the first instance, the next w[1] to the second,
//              ...).  Its cost is that instance's O8 cost.  A future pinned by
//              kStateful keeps its pin and takes no number; a type without a
//              positive weight keeps the O8 route.  Weights above 2^20 -> -1;
//              kWeighted with kGreedy -> -1
//   priorities (a per-workflow level 0..15, set_priority of Table 2): O9
//              sorts by (-priority[wf], key, wf, v), the higher level first,
//              for any key; a level above 15 -> -1
//
// Precedence of errors: EINVAL, then ECYCLE, then ERANGE.
#include <algorithm>
#include <cstdint>
#include <cstring>
#include <map>
#include <vector>

namespace {

constexpr int kOk = 0;
constexpr int kEinval = -1;
constexpr int kEcycle = -2;
constexpr int kErange = -3;

constexpr uint32_t kLpt = 2u;
constexpr uint32_t kStateful = 4u;
constexpr uint32_t kGreedy = 8u;
constexpr uint32_t kSrtf = 16u;
constexpr uint32_t kWeighted = 32u;
constexpr int kMaxPriority = 15;
constexpr uint32_t kMaxWeight = 1u << 20;

constexpr int64_t kMaxNodes = int64_t(1) << 30;
constexpr int64_t kMaxEdges = (int64_t(1) << 31) - 1;
constexpr int64_t kMaxWorkflows = int64_t(1) << 30;
constexpr int64_t kMaxInstances = 1024;
constexpr int64_t kEstMax = int64_t(1) << 40;
constexpr int64_t kLoadMax = int64_t(1) << 60;
constexpr int64_t kMigMax = int64_t(1) << 60;
constexpr int64_t kHorizon = int64_t(1) << 61;   // |now| and |deadline - now|
constexpr int64_t kRemMax = int64_t(1) << 62;

// O1: every rule the snapshot must satisfy.  A self-dependency is left to the
// cycle check (it is a cycle of length one).
int validate(int64_t N, int64_t E, int64_t W, int64_t M, int64_t now, int64_t mig,
             const int32_t* wf, const int32_t* type, const int64_t* est,
             const uint8_t* done, const int32_t* loc, const int32_t* dep_off,
             const int32_t* dep_idx, const int64_t* deadline, const int32_t* inst_type,
             const int64_t* inst_load, const int32_t* inst_speed) {
  if (N < 0 || N > kMaxNodes || E < 0 || E > kMaxEdges || W < 0 || W > kMaxWorkflows ||
      M < 0 || M > kMaxInstances)
    return kEinval;
  if (now < -kHorizon || now > kHorizon || mig < 0 || mig > kMigMax) return kEinval;
  if (N == 0 && E != 0) return kEinval;
  if (N > 0 && (!wf || !type || !est || !done || !loc || !dep_off)) return kEinval;
  if (E > 0 && !dep_idx) return kEinval;
  if (W > 0 && !deadline) return kEinval;
  if (M > 0 && (!inst_type || !inst_load || !inst_speed)) return kEinval;
  for (int64_t w = 0; w < W; ++w)
    if (deadline[w] < now - kHorizon || deadline[w] > now + kHorizon) return kEinval;
  for (int64_t i = 0; i < M; ++i) {
    if (inst_type[i] < 0) return kEinval;
    if (inst_speed[i] < 1) return kEinval;
    if (inst_load[i] < 0 || inst_load[i] > kLoadMax) return kEinval;
  }
  if (N == 0) return kOk;
  if (dep_off[0] != 0 || dep_off[N] != E) return kEinval;
  for (int64_t v = 0; v < N; ++v) {
    if (dep_off[v] > dep_off[v + 1]) return kEinval;
    if (wf[v] < 0 || wf[v] >= W) return kEinval;
    if (type[v] < 0) return kEinval;
    if (loc[v] < -1 || loc[v] >= M) return kEinval;
    if (est[v] < 0 || est[v] > kEstMax) return kEinval;
    if (done[v] > 1) return kEinval;
  }
  for (int64_t v = 0; v < N; ++v) {
    for (int32_t e = dep_off[v]; e < dep_off[v + 1]; ++e) {
      int32_t p = dep_idx[e];
      if (p < 0 || p >= N) return kEinval;
      if (wf[p] != wf[v]) return kEinval;
    }
  }
  return kOk;
}

}  // namespace

extern "C" {

// The boundary of the oracle: host arrays in, host arrays out.  Output arrays
// must hold n_nodes entries (rem) and n_nodes entries (order, slack, route,
// cost); rem_out and cost_out may be NULL.  Returns 0 or a negative error code.
int nalar_oracle_pass_policy(int64_t N, int64_t E, int64_t W, int64_t M, int64_t now, int64_t mig,
                             uint32_t policy, const uint8_t* priority,
                             const uint32_t* inst_weight, const int32_t* wf, const int32_t* type,
                             const int64_t* est, const uint8_t* done, const int32_t* loc,
                             const int32_t* dep_off, const int32_t* dep_idx,
                             const int64_t* deadline, const int32_t* inst_type,
                             const int64_t* inst_load, const int32_t* inst_speed, int64_t* rem_out,
                             int32_t* order_out, int64_t* slack_out, int32_t* route_out,
                             int64_t* cost_out, int64_t* n_ready_out) {
  if ((policy & ~(kLpt | kStateful | kGreedy | kSrtf | kWeighted)) != 0) return kEinval;
  if ((policy & kLpt) && (policy & kSrtf)) return kEinval;
  if ((policy & kGreedy) && (policy & kWeighted)) return kEinval;
  if ((policy & kWeighted) && M > 0) {
    if (!inst_weight) return kEinval;
    for (int64_t i = 0; i < M; ++i)
      if (inst_weight[i] > kMaxWeight) return kEinval;
  }
  if (priority)
    for (int64_t w = 0; w < W; ++w)
      if (priority[w] > kMaxPriority) return kEinval;
  int rc = validate(N, E, W, M, now, mig, wf, type, est, done, loc, dep_off, dep_idx,
                    deadline, inst_type, inst_load, inst_speed);
  if (rc != kOk) return rc;
  if (n_ready_out) *n_ready_out = 0;
  if (N == 0) return kOk;
  if (!order_out || !slack_out || !route_out) return kEinval;

  // O2
  std::vector<int64_t> est_eff(N);
  for (int64_t v = 0; v < N; ++v) est_eff[v] = done[v] ? 0 : est[v];

  // O3: successor CSR (counting sort of the edges by parent)
  std::vector<int64_t> succ_off(N + 1, 0);
  for (int64_t e = 0; e < E; ++e) succ_off[dep_idx[e] + 1]++;
  for (int64_t v = 0; v < N; ++v) succ_off[v + 1] += succ_off[v];
  std::vector<int32_t> succ(E);
  {
    std::vector<int64_t> fill(succ_off.begin(), succ_off.end() - 1);
    for (int64_t v = 0; v < N; ++v)
      for (int32_t e = dep_off[v]; e < dep_off[v + 1]; ++e) succ[fill[dep_idx[e]]++] = int32_t(v);
  }

  // O4 + O5: iterative DFS, post-order evaluation of rem.
  enum : uint8_t { kWhite = 0, kGray = 1, kBlack = 2 };
  std::vector<uint8_t> color(N, kWhite);
  std::vector<int64_t> rem(N, 0);
  bool overflow = false;
  struct Frame { int64_t v; int64_t next; };
  std::vector<Frame> stack;
  for (int64_t root = 0; root < N; ++root) {
    if (color[root] != kWhite) continue;
    color[root] = kGray;
    stack.push_back({root, succ_off[root]});
    while (!stack.empty()) {
      Frame& f = stack.back();
      if (f.next < succ_off[f.v + 1]) {
        int64_t s = succ[f.next++];
        if (color[s] == kGray) return kEcycle;
        if (color[s] == kWhite) {
          color[s] = kGray;
          stack.push_back({s, succ_off[s]});
        }
        continue;
      }
      // post-visit: every successor is finished
      int64_t v = f.v;
      int64_t best = 0;
      for (int64_t k = succ_off[v]; k < succ_off[v + 1]; ++k) best = std::max(best, rem[succ[k]]);
      int64_t r;
      if (__builtin_add_overflow(est_eff[v], best, &r) || r > kRemMax) {
        overflow = true;
        r = kRemMax + 1;  // keep later sums finite; the pass fails anyway
      }
      rem[v] = r;
      color[v] = kBlack;
      stack.pop_back();
    }
  }
  if (overflow) return kErange;

  // O6 + O7 + O8
  std::vector<int32_t> ready_ids;
  for (int64_t v = 0; v < N; ++v) {
    if (done[v]) continue;
    bool all_done = true;
    for (int32_t e = dep_off[v]; e < dep_off[v + 1]; ++e)
      if (!done[dep_idx[e]]) { all_done = false; break; }
    if (all_done) ready_ids.push_back(int32_t(v));
  }
  const int64_t R = int64_t(ready_ids.size());
  std::vector<int64_t> slack(N, 0), cost(N, 0);
  std::vector<int32_t> route(N, -1);
  for (int64_t k = 0; k < R; ++k) {
    int32_t v = ready_ids[k];
    slack[v] = (deadline[wf[v]] - now) - rem[v];
    if ((policy & kStateful) && loc[v] >= 0 && inst_type[loc[v]] == type[v]) {
      const int32_t i = loc[v];
      route[v] = i;
      cost[v] = inst_load[i] + (est[v] * 1000) / inst_speed[i];
      continue;
    }
    int64_t best = INT64_MAX;
    int32_t arg = -1;
    for (int64_t i = 0; i < M; ++i) {
      if (inst_type[i] != type[v]) continue;
      int64_t c = inst_load[i] + (est[v] * 1000) / inst_speed[i];
      if (loc[v] >= 0 && loc[v] != i) c += mig;
      if (c < best) { best = c; arg = int32_t(i); }
    }
    route[v] = arg;
    cost[v] = best;
  }

  // O9: the full key (slack, wf, v), or (-rem, wf, v) under kLpt, or
  // (rem, wf, v) under kSrtf, behind the workflow's priority level when given,
  // is a total order, so the result is unique.
  const bool lpt = (policy & kLpt) != 0;
  const bool srtf = (policy & kSrtf) != 0;
  auto key_of = [&](int32_t v) { return lpt ? -rem[v] : (srtf ? rem[v] : slack[v]); };
  std::vector<int32_t> order(ready_ids);
  std::sort(order.begin(), order.end(), [&](int32_t a, int32_t b) {
    if (priority && priority[wf[a]] != priority[wf[b]]) return priority[wf[a]] > priority[wf[b]];
    const int64_t ka = key_of(a);
    const int64_t kb = key_of(b);
    if (ka != kb) return ka < kb;
    if (wf[a] != wf[b]) return wf[a] < wf[b];
    return a < b;
  });

  // O9b (kGreedy): route again in the output order with running loads.
  if (policy & kGreedy) {
    std::vector<int64_t> load(inst_load, inst_load + M);
    for (int32_t v : order) {
      int32_t arg = -1;
      int64_t best = INT64_MAX;
      if ((policy & kStateful) && loc[v] >= 0 && inst_type[loc[v]] == type[v]) {
        arg = loc[v];
        best = load[arg] + (est[v] * 1000) / inst_speed[arg];
      } else {
        for (int64_t i = 0; i < M; ++i) {
          if (inst_type[i] != type[v]) continue;
          int64_t c = load[i] + (est[v] * 1000) / inst_speed[i];
          if (loc[v] >= 0 && loc[v] != i) c += mig;
          if (c < best) { best = c; arg = int32_t(i); }
        }
      }
      route[v] = arg;
      cost[v] = best;
      if (arg >= 0) {
        load[arg] += (est[v] * 1000) / inst_speed[arg];
        if (load[arg] > kRemMax) return kErange;
      }
    }
  }

  // O9c (kWeighted): deal each weighted type's futures, in output order, to
  // its instances by their weights.
  if ((policy & kWeighted) && M > 0) {
    std::map<int32_t, int64_t> next_seq;  // next sequence number of each type
    for (int32_t v : order) {
      if ((policy & kStateful) && loc[v] >= 0 && inst_type[loc[v]] == type[v]) continue;
      int64_t total = 0;
      for (int64_t i = 0; i < M; ++i)
        if (inst_type[i] == type[v]) total += inst_weight[i];
      if (total == 0) continue;
      int64_t r = next_seq[type[v]]++ % total;
      int32_t pick = -1;
      for (int64_t i = 0; i < M && pick < 0; ++i) {
        if (inst_type[i] != type[v]) continue;
        if (r < int64_t(inst_weight[i])) pick = int32_t(i);
        else r -= inst_weight[i];
      }
      route[v] = pick;
      cost[v] = inst_load[pick] + (est[v] * 1000) / inst_speed[pick] +
                ((loc[v] >= 0 && loc[v] != pick) ? mig : 0);
    }
  }

  // O10
  if (rem_out) std::memcpy(rem_out, rem.data(), sizeof(int64_t) * N);
  for (int64_t k = 0; k < R; ++k) {
    int32_t v = order[k];
    order_out[k] = v;
    slack_out[k] = slack[v];
    route_out[k] = route[v];
    if (cost_out) cost_out[k] = cost[v];
  }
  if (n_ready_out) *n_ready_out = R;
  return kOk;
}

// The default policy (least slack first, load-and-locality routing).
int nalar_oracle_pass(int64_t N, int64_t E, int64_t W, int64_t M, int64_t now, int64_t mig,
                      const int32_t* wf, const int32_t* type, const int64_t* est,
                      const uint8_t* done, const int32_t* loc, const int32_t* dep_off,
                      const int32_t* dep_idx, const int64_t* deadline,
                      const int32_t* inst_type, const int64_t* inst_load,
                      const int32_t* inst_speed, int64_t* rem_out, int32_t* order_out,
                      int64_t* slack_out, int32_t* route_out, int64_t* cost_out,
                      int64_t* n_ready_out) {
  return nalar_oracle_pass_policy(N, E, W, M, now, mig, 0u, nullptr, nullptr, wf, type, est, done, loc, dep_off,
                                  dep_idx, deadline, inst_type, inst_load, inst_speed, rem_out,
                                  order_out, slack_out, route_out, cost_out, n_ready_out);
}

}  // extern "C"
