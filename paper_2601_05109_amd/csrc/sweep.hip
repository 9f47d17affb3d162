// Per-workflow sweep: remaining critical path, readiness, order key and
// routing of every future, in one kernel.
//
// Futures of different workflows never depend on each other (one global
// controller per workflow, Section 4.1; cross-workflow dependencies are
// rejected), so workflows are swept independently, each by the reverse
// level-synchronous max-plus sweep:
//
//   cnt[u] = number of consumers of u (atomic out-degree counters)
//   level 0 = futures with no consumer; a future joins a level when its last
//   consumer is finalised; finalising u sets
//       rem[u] = est'[u] + mx[u],   mx = running max of the consumers' rem
//   and pushes rem[u] into mx[p] / decrements cnt[p] for each dependency p.
//
// Pushes (max, then decrement) and counter increments are order-free integer
// atomics, so the result does not depend on scheduling.  When a whole wave
// targets the same future (a fan-in such as a map/reduce root), the wave
// reduces first and one lane issues a single atomic.
//
// Three shapes:
//  * k_sweep_wave: one wavefront per workflow of at most 512 futures, or per
//    pair of consecutive workflows of at most 64 futures together when
//    workflows average 32 or fewer (four independent waves per workgroup, no
//    workgroup barrier in the sweep), the slice's state in a
//    14-byte-per-future LDS slice, each lane owning up to eight futures with
//    their dependencies in registers; the levels are rounds of LDS atomics.
//    In fused mode it also validates the snapshot, finds each workflow's
//    bounds and builds the routing table itself.
//  * k_sweep: one workgroup per workflow of up to 5,120 futures (LDS state).
//  * workflows larger than that (or all, under NALAR_FORCE_GLOBAL_SWEEP) keep
//    their state in HBM by position.  When every dependency of such a
//    workflow lies at a lower position than its consumer, its positions are
//    taken in chunks from the last to the first (sweep_hbm_ordered); else it
//    processes explicit frontier lists (sweep_hbm).  Either way the workgroup
//    that met the workflow sweeps it.
//
// Every ready future is routed against the pass-start instance table and then
// either dropped into its order-key bucket (one returning atomic for a slot)
// or, when the tiled sort is planned, staged by position.
#include "internal.hpp"

namespace nalar {

namespace {

constexpr int kPmax = 3;          // dependencies held in registers per future
constexpr int kHeavyCap = 64;     // cooperative list capacity per phase
constexpr int kHeavyBatch = 2;    // cooperative dependency loads a thread keeps in flight
constexpr int kHbmLight = 32;     // HBM path: more dependencies -> cooperative
constexpr size_t kStaticLdsReserve = 4096;

struct Layout {
  const int32_t* node_of_pos;
  const int32_t* pos_of_node;
  int64_t N;
};

__device__ inline int32_t node_at(const Layout& L, int64_t q) {
  return L.node_of_pos ? L.node_of_pos[q] : int32_t(q);
}

// Index of dependency p inside the workflow occupying positions [b, b+n), or
// -1 if p lies outside it (out of range or another workflow).
__device__ inline int32_t local_of(const Layout& L, int32_t p, int64_t b, int n) {
  int64_t q;
  if (L.pos_of_node) {
    if (p < 0 || int64_t(p) >= L.N) return -1;
    q = L.pos_of_node[p];
  } else {
    q = p;
  }
  const int64_t lp = q - b;
  return (lp >= 0 && lp < n) ? int32_t(lp) : -1;
}

__device__ inline int32_t checked_dep(const Layout& L, int32_t p, int64_t b, int n, int k,
                                      Ctrl* ctrl) {
  const int32_t lp = local_of(L, p, b, n);
  if (lp < 0) {
    flag_sweep(ctrl, kStInval);
    return -1;
  }
  if (lp == k) {
    flag_sweep(ctrl, kStCycle);
    return -1;
  }
  return lp;
}

// A dependency that must also lie in the workflow's own part [lo, hi) of a
// slice holding several workflows (a dependency on another workflow of the
// slice is one outside the future's workflow).
__device__ inline int32_t checked_dep_seg(const Layout& L, int32_t p, int64_t b, int n, int lo, int hi,
                                          int k, Ctrl* ctrl) {
  const int32_t lp = checked_dep(L, p, b, n, k, ctrl);
  if (lp >= 0 && (lp < lo || lp >= hi)) {
    flag_sweep(ctrl, kStInval);
    return -1;
  }
  return lp;
}

// ---------------------------------------------------------------- LDS atomics

__device__ inline void agg_count_lds(int32_t* cnt, int lp) {
  const uint64_t act = ballot(lp >= 0);
  if (act == 0) return;
  if ((act & (act - 1)) != 0) {
    const int lead = __builtin_ctzll(act);
    const int first = readlane_i32(lp, lead);
    if (ballot(lp >= 0 && lp != first) == 0) {  // the whole wave feeds one future
      if (lane_id() == lead) atomicAdd(&cnt[first], int(__popcll(act)));
      return;
    }
  }
  if (lp >= 0) atomicAdd(&cnt[lp], 1);
}

// Called with every lane of the wave active.
__device__ inline void agg_push_lds(int64_t* mx, int32_t* cnt, int lp, int64_t r) {
  const uint64_t act = ballot(lp >= 0);
  if (act == 0) return;
  if ((act & (act - 1)) != 0) {
    const int lead = __builtin_ctzll(act);
    const int first = readlane_i32(lp, lead);
    if (ballot(lp >= 0 && lp != first) == 0) {  // fan-in: reduce, then one atomic
      const int64_t m = wave_max_i64(lp >= 0 ? r : INT64_MIN);
      if (lane_id() == lead) {
        atomicMax(reinterpret_cast<long long*>(&mx[first]), (long long)m);
        atomicSub(&cnt[first], int(__popcll(act)));
      }
      return;
    }
  }
  if (lp >= 0) {
    atomicMax(reinterpret_cast<long long*>(&mx[lp]), (long long)r);
    atomicSub(&cnt[lp], 1);
  }
}

// A push of n merged contributions (max rem r) to dependency lp; called with
// every lane of the wave active.
__device__ inline void agg_push_lds_n(int64_t* mx, int32_t* cnt, int lp, int64_t r, int32_t n) {
  const uint64_t act = ballot(lp >= 0);
  if (act == 0) return;
  if ((act & (act - 1)) != 0) {
    const int lead = __builtin_ctzll(act);
    const int first = readlane_i32(lp, lead);
    if (ballot(lp >= 0 && lp != first) == 0) {  // fan-in: reduce, then one atomic
      const int64_t m = wave_max_i64(lp >= 0 ? r : INT64_MIN);
      const int64_t c = wave_sum_i64(lp >= 0 ? int64_t(n) : 0);
      if (lane_id() == lead) {
        atomicMax(reinterpret_cast<long long*>(&mx[first]), (long long)m);
        atomicSub(&cnt[first], int(c));
      }
      return;
    }
  }
  if (lp >= 0) {
    atomicMax(reinterpret_cast<long long*>(&mx[lp]), (long long)r);
    atomicSub(&cnt[lp], n);
  }
}

// ---------------------------------------------------------------- HBM atomics

__device__ inline void agg_count_hbm(int32_t* cnt, int lp) {
  const uint64_t act = ballot(lp >= 0);
  if (act == 0) return;
  if ((act & (act - 1)) != 0) {
    const int lead = __builtin_ctzll(act);
    const int first = readlane_i32(lp, lead);
    if (ballot(lp >= 0 && lp != first) == 0) {
      if (lane_id() == lead) add_wg(&cnt[first], int32_t(__popcll(act)));
      return;
    }
  }
  if (lp >= 0) add_wg(&cnt[lp], int32_t(1));
}

__device__ inline void append_wave(bool in, int32_t val, int32_t* list, int* s_count) {
  const uint64_t am = ballot(in);
  if (am == 0) return;
  const int lead = __builtin_ctzll(am);
  int base = 0;
  if (lane_id() == lead) base = atomicAdd(s_count, int(__popcll(am)));
  base = readlane_i32(base, lead);
  if (in) list[base + int(lanes_below(am))] = val;
}

// Called with every lane of the wave active.  A dependency whose counter
// reaches zero is appended to the next frontier.
__device__ inline void agg_push_hbm(int64_t* mx, int32_t* cnt, int lp, int64_t r, int32_t* nxt,
                                    int* s_fnext) {
  const uint64_t act = ballot(lp >= 0);
  bool app = false;
  int32_t app_lp = 0;
  if (act != 0) {
    const int lead = __builtin_ctzll(act);
    const int first = readlane_i32(lp, lead);
    if ((act & (act - 1)) != 0 && ballot(lp >= 0 && lp != first) == 0) {
      const int64_t m = wave_max_i64(lp >= 0 ? r : INT64_MIN);
      if (lane_id() == lead) {
        max_wg(&mx[first], m);
        const int32_t c = int32_t(__popcll(act));
        if (add_wg(&cnt[first], -c) == c) { app = true; app_lp = first; }
      }
    } else if (lp >= 0) {
      max_wg(&mx[lp], r);
      if (add_wg(&cnt[lp], int32_t(-1)) == 1) { app = true; app_lp = lp; }
    }
  }
  append_wave(app, app_lp, nxt, s_fnext);
}

__device__ inline int64_t clamp_rem(int64_t r, bool& overflow) {
  if (r > NALAR_REM_MAX) {
    overflow = true;
    return NALAR_REM_MAX + 1;
  }
  return r;
}

// Workgroup-shared bookkeeping of the sweep (one instance per workgroup).
struct Shared {
  int bad;
  int hcount;
  int fcount;
  int fnext;
  int proc;
  int32_t hk[kHeavyCap];
  int32_t ho[kHeavyCap];
  int32_t hd[kHeavyCap];
  int64_t red[3][16];
};

struct ITabLds {
  int64_t* load;
  double* inv;
  int32_t* type;
  int32_t* idx;
  int32_t* speed;
  int32_t* pos;
  uint32_t* run;    // [kTypeDirect]
  uint32_t* prun;   // [kTypeDirect] undominated ends (tables from the node kernel), or NULL
};

struct Acc {
  int64_t tmin = INT64_MAX;
  int64_t tmax = INT64_MIN;
  int64_t tready = 0;
};

// Bucket of a key under this pass's bucket boundaries (lvl: the priority
// level of its workflow), and a slot in it (one returning atomic; claim early
// so that its latency overlaps other work).  Every result lies in [0, nb).
// kLevels: the mapping may have level groups (the block kernel takes none,
// which keeps it within its registers; the host then plans no buckets).
template <bool kLevels>
__device__ inline uint32_t bucket_of(const BucketArgs& bk, int64_t key, int lvl) {
  // the workflow's part (the same on every lane): its level's group of
  // buckets [base, base + last]
  uint32_t base = 0, last = uint32_t(bk.nb - 1);
  if (kLevels && bk.ngroups > 0) {
    const int32_t g = bk.lvl_hi - int32_t(lvl);
    const bool in = g >= 0 && g < bk.ngroups;
    base = g < 0 ? 0u : (in ? uint32_t(g) << bk.lshift : last);
    last = in ? (1u << bk.lshift) - 1u : 0u;
  }
  const uint64_t d = key > bk.lo ? uint64_t(key) - uint64_t(bk.lo) : 0;
  const uint64_t q = d >> bk.shift;
  return base + (q < uint64_t(last) ? uint32_t(q) : last);
}

// Bin of a key: the number of splitters at or below it (splitters ascending,
// in LDS), so bins ascend with the key and equal keys share a bin.
// Bin of a key: the number of splitters <= key (nb - 1 ascending splitters,
// nb a power of two), by binary lifting so that every lane takes the same
// log2(nb) steps.
__device__ inline uint32_t bin_of(const int64_t* split, int nb, int64_t key) {
  uint32_t at = 0;
  for (int step = nb >> 1; step > 0; step >>= 1)
    if (split[at + step - 1] <= key) at += step;
  return at;
}

__device__ inline void bucket_put(const SweepArgs& a, uint32_t bkt, uint32_t slot, int64_t key,
                                  int64_t pos, int32_t route, int lvl, int64_t cost) {
  const uint32_t cap = a.bk.bins ? uint32_t(a.bk.cap) : uint32_t(kBucketCap);
  if (slot < cap) {
    // three 8-byte stores: key, cost, and position | packed route (the
    // struct's last two fields)
    int64_t* sl = reinterpret_cast<int64_t*>(a.bk.slot + int64_t(bkt) * cap + slot);
    sl[0] = key;
    sl[1] = cost;
    sl[2] = int64_t(uint64_t(uint32_t(pos)) | (uint64_t(uint32_t(slot_pack(route, lvl))) << 32));
  } else {
    st_relaxed_agent(&a.ctrl->bucket_overflow, 1u);
  }
}

// The key the ready futures are ordered by (behind their workflow's priority
// level): the slack, or the remaining critical path negated under
// NALAR_ORDER_LPT (longest first) or as it is under NALAR_ORDER_SRTF
// (shortest first).
// Written as base - (+-rem) with both chosen by the policy word (the same on
// every lane), which keeps the block sweep within its registers.
__device__ inline int64_t order_key(const SweepArgs& a, int64_t rem, int64_t dl) {
  const int64_t base = (a.p.policy & (NALAR_ORDER_LPT | NALAR_ORDER_SRTF)) ? 0 : dl;
  const int64_t r = (a.p.policy & NALAR_ORDER_SRTF) ? -rem : rem;
  return base - r;
}

// Workflow w's priority level (0 without levels); w is the same on every
// lane, so the level goes to a scalar register.
__device__ inline int prio_level(const SweepArgs& a, int64_t w) {
  return a.p.prio ? __builtin_amdgcn_readfirstlane(int(a.p.prio[w])) : 0;
}

__device__ inline uint32_t level_bit(int lvl) { return 1u << (uint32_t(lvl) & 31u); }

// Stores of one ready future: its bucket slot (bucketed sort) or its staged
// values by position (tiled sort), and its slack by position when the key is
// not the slack.
__device__ inline void store_ready(const SweepArgs& a, uint32_t bkt, uint32_t slot, int64_t key,
                                   int lvl, int64_t slack, int64_t pos, int32_t route, int64_t cost,
                                   Acc& acc) {
  if (a.bk.nb > 0) {
    bucket_put(a, bkt, slot, key, pos, route, lvl, cost);
  } else {
    a.stg_slack[pos] = key;
    a.stg_route[pos] = route;
    a.stg_cost[pos] = cost;
  }
  if ((a.p.policy & (NALAR_ORDER_LPT | NALAR_ORDER_SRTF)) || a.p.prio) a.stg_oslack[pos] = slack;
  acc.tmin = key < acc.tmin ? key : acc.tmin;
  acc.tmax = key > acc.tmax ? key : acc.tmax;
  acc.tready += 1;
}

// split_l: the splitters in LDS when the pass uses bins (block kernel only).
template <bool kLevels>
__device__ inline void write_ready(const SweepArgs& a, const ITabLds& it, int64_t pos, int32_t type,
                                   int32_t loc, int64_t rem, int64_t est, int64_t dl, int lvl,
                                   Acc& acc, const int64_t* split_l) {
  const int64_t key = order_key(a, rem, dl);
  const BucketArgs& bk = a.bk;
  uint32_t bkt = 0, slot = 0;
  if (bk.nb > 0) {
    bkt = bk.bins ? bin_of(split_l, bk.nb, key) : bucket_of<kLevels>(bk, key, lvl);
    slot = add_agent(bk.cnt + bkt, 1u);
  }
  int32_t route;
  int64_t cost;
  route_future(type, est, loc, int32_t(a.p.M), a.p.mig, it.type, it.idx, it.load, it.speed,
               it.inv, it.pos, it.run, (a.p.policy & NALAR_ROUTE_STATEFUL) != 0, route, cost, it.prun);
  store_ready(a, bkt, slot, key, lvl, dl - rem, pos, route, cost, acc);
}

// ------------------------------------------------------------ LDS workflow

// Owned-future registers of the LDS path.  Local indices are below 2^16 there
// (lds_cap < 65535), so the three dependency slots and the degree pack into two
// words: p01 = d0 | d1 << 16, p2 = d2 | deg << 16 | heavy << 31 (0xFFFF = none).
constexpr uint32_t kNoDep = 0xFFFFu;
constexpr uint32_t kHeavyBit = 0x80000000u;

__device__ inline int dep_at(uint32_t p01, uint32_t p2, int q) {
  const uint32_t x = q == 0 ? (p01 & 0xFFFFu) : q == 1 ? (p01 >> 16) : (p2 & 0xFFFFu);
  return x == kNoDep ? -1 : int(x);
}

// With bins, bl holds the splitters and two per-bin counter arrays in LDS
// (zero on entry, left zero on return).
struct BinLds {
  const int64_t* split;   // [nb - 1]
  uint32_t* cnt;          // [nb] this workflow's ready futures in each bin
  uint32_t* base;         // [nb] the segment each bin gave this workflow
};

template <int T, int NPT>
__device__ __attribute__((always_inline)) void sweep_lds(const SweepArgs& a, const Layout& L, const ITabLds& it, Shared& S,
                          int64_t* mx, int32_t* cnt, uint8_t* dn, uint8_t* nr, int lds_cap, int64_t b,
                          int n, int64_t dl, int lvl, Acc& acc, const BinLds& bl) {
  const int tid = threadIdx.x;
  Ctrl* ctrl = a.ctrl;

  int32_t vv[NPT];
  int64_t ee[NPT];
  int32_t off[NPT], deg[NPT], ty[NPT], lc[NPT];
  uint32_t p01[NPT], p2[NPT];
  uint32_t own = 0, fin = 0, ready = 0;

  // A: everything the workflow needs from HBM about its own futures, in one
  // round trip; reset their counters
#pragma unroll
  for (int j = 0; j < NPT; ++j) {
    const int k = j * T + tid;
    vv[j] = 0; ee[j] = 0; off[j] = 0; deg[j] = 0; ty[j] = 0; lc[j] = -1;
    p01[j] = 0xFFFFFFFFu; p2[j] = kNoDep;
    if (k < n) {
      own |= 1u << j;
      const int32_t v = node_at(L, b + k);
      const uint8_t d = a.p.done[v];
      vv[j] = v;
      ee[j] = d ? 0 : a.p.est[v];
      off[j] = a.p.dep_off[v];
      deg[j] = a.p.dep_off[v + 1] - off[j];
      ty[j] = a.p.type[v];
      lc[j] = a.p.loc[v];
      cnt[k] = 0;
      mx[k] = 0;
      dn[k] = d;
      nr[k] = 0;
    }
  }
  if (tid == 0) { S.hcount = 0; S.proc = 0; }
  __syncthreads();

  // B: out-degree counters and readiness (one pass over the dependencies)
#pragma unroll
  for (int j = 0; j < NPT; ++j) {
    if (ballot((own >> j) & 1u) == 0) continue;   // wave-uniform: no future in this slot
    const int k = j * T + tid;
    const bool mine = (own >> j) & 1u;
    const bool light = mine && deg[j] <= kPmax;
    if (mine && !light) {
      p2[j] = kHeavyBit | kNoDep;
      const int slot = atomicAdd(&S.hcount, 1);
      if (slot < kHeavyCap) {
        S.hk[slot] = k; S.ho[slot] = off[j]; S.hd[slot] = deg[j];
      } else {
        bool blocked = false;
        for (int e = 0; e < deg[j]; ++e) {
          const int32_t lp = checked_dep(L, a.p.dep_idx[off[j] + e], b, n, k, ctrl);
          if (lp >= 0) { atomicAdd(&cnt[lp], 1); blocked |= dn[lp] == 0; }
        }
        if (blocked) nr[k] = 1;
      }
    }
    bool blocked = false;
    uint32_t packed[kPmax];
#pragma unroll
    for (int q = 0; q < kPmax; ++q) {
      int32_t lp = -1;
      if (light && q < deg[j]) lp = checked_dep(L, a.p.dep_idx[off[j] + q], b, n, k, ctrl);
      packed[q] = lp >= 0 ? uint32_t(lp) : kNoDep;
      agg_count_lds(cnt, lp);
      if (lp >= 0 && dn[lp] == 0) blocked = true;
    }
    if (light) {
      p01[j] = packed[0] | (packed[1] << 16);
      p2[j] = packed[2] | (uint32_t(deg[j]) << 16);
      if (blocked) nr[k] = 1;
    }
  }
  __syncthreads();
  const int hc0 = S.hcount;          // futures with many dependencies, if any
  const bool any_heavy = hc0 > 0;
  {
    const int hc = hc0 < kHeavyCap ? hc0 : kHeavyCap;
    for (int h = 0; h < hc; ++h) {
      const int k = S.hk[h], o = S.ho[h], dg = S.hd[h];
      bool blocked = false;
      for (int e0 = 0; e0 < dg; e0 += kHeavyBatch * T) {
        int32_t raw[kHeavyBatch];
#pragma unroll
        for (int u = 0; u < kHeavyBatch; ++u) {  // the batch's loads in flight together
          const int e = e0 + u * T + tid;
          raw[u] = e < dg ? a.p.dep_idx[o + e] : 0;
        }
#pragma unroll
        for (int u = 0; u < kHeavyBatch; ++u) {
          int32_t lp = -1;
          if (e0 + u * T + tid < dg) lp = checked_dep(L, raw[u], b, n, k, ctrl);
          agg_count_lds(cnt, lp);
          if (lp >= 0 && dn[lp] == 0) blocked = true;
        }
      }
      if (blocked) nr[k] = 1;
    }
  }
  __syncthreads();

  // ready flags (staged by position for the sort's first pass)
#pragma unroll
  for (int j = 0; j < NPT; ++j) {
    if ((own >> j) & 1u) {
      const int k = j * T + tid;
      const bool rd = dn[k] == 0 && nr[k] == 0;
      if (rd) ready |= 1u << j;
      if (a.bk.nb == 0) a.stg_ready[b + k] = rd ? uint8_t(1 + lvl) : 0;
    }
  }
  if (tid == 0) S.hcount = 0;

  // C: levels.  A future whose consumers are all finalised (cnt == 0) is
  // finalised and pushes its rem to its dependencies.
  bool overflow = false;
  for (;;) {
    int32_t cv[NPT];
#pragma unroll
    for (int j = 0; j < NPT; ++j) cv[j] = (j * T + tid < lds_cap) ? cnt[j * T + tid] : 1;
    uint32_t cand = 0;
#pragma unroll
    for (int j = 0; j < NPT; ++j)
      if ((((own & ~fin) >> j) & 1u) && cv[j] == 0) cand |= 1u << j;
    if (!__syncthreads_or(cand != 0)) break;
    // A lane's pushes to one dependency are merged before they reach LDS
    // (pending: target, max rem, count), so that a fan-in (every future of
    // the wave feeding one future) costs one wave reduction per round, not
    // one per slot.  A future finalised this round is no push target in it
    // (its consumers were all finalised before), so the pushes may wait for
    // the end of the round.
    int32_t pend_lp = -1;
    int64_t pend_r = INT64_MIN;
    int32_t pend_n = 0;
#pragma unroll
    for (int j = 0; j < NPT; ++j) {
      const bool c = (cand >> j) & 1u;
      if (ballot(c) == 0) continue;               // wave-uniform
      const bool hv = (p2[j] & kHeavyBit) != 0;
      const int k = j * T + tid;
      int64_t r = 0;
      if (c) {
        r = clamp_rem(ee[j] + mx[k], overflow);
        mx[k] = r;
        fin |= 1u << j;
        if (hv) {
          // the dependency list read again (phase B's registers for it are
          // not kept through the levels)
          const int32_t ho = a.p.dep_off[vv[j]];
          const int32_t hd = a.p.dep_off[vv[j] + 1] - ho;
          const int hs = atomicAdd(&S.hcount, 1);
          if (hs < kHeavyCap) {
            S.hk[hs] = k; S.ho[hs] = ho; S.hd[hs] = hd;
          } else {
            for (int e = 0; e < hd; ++e) {
              const int32_t lp = local_of(L, a.p.dep_idx[ho + e], b, n);
              if (lp >= 0 && lp != k) {
                atomicMax(reinterpret_cast<long long*>(&mx[lp]), (long long)r);
                atomicSub(&cnt[lp], 1);
              }
            }
          }
        }
      }
      if (c && !hv) {
#pragma unroll
        for (int q = 0; q < kPmax; ++q) {
          const int lp = dep_at(p01[j], p2[j], q);
          if (lp < 0) continue;
          if (lp == pend_lp) {
            pend_r = r > pend_r ? r : pend_r;
            ++pend_n;
          } else {
            if (pend_lp >= 0) {
              atomicMax(reinterpret_cast<long long*>(&mx[pend_lp]), (long long)pend_r);
              atomicSub(&cnt[pend_lp], pend_n);
            }
            pend_lp = lp;
            pend_r = r;
            pend_n = 1;
          }
        }
      }
    }
    agg_push_lds_n(mx, cnt, pend_lp, pend_r, pend_n);
    if (any_heavy) {
      __syncthreads();
      const int hc = S.hcount < kHeavyCap ? S.hcount : kHeavyCap;
      for (int h = 0; h < hc; ++h) {
        const int k = S.hk[h], o = S.ho[h], dg = S.hd[h];
        const int64_t r = mx[k];
        for (int e0 = 0; e0 < dg; e0 += kHeavyBatch * T) {
          int32_t raw[kHeavyBatch];
#pragma unroll
          for (int u = 0; u < kHeavyBatch; ++u) {
            const int e = e0 + u * T + tid;
            raw[u] = e < dg ? a.p.dep_idx[o + e] : 0;
          }
#pragma unroll
          for (int u = 0; u < kHeavyBatch; ++u) {
            int32_t lp = -1;
            if (e0 + u * T + tid < dg) {
              lp = local_of(L, raw[u], b, n);
              if (lp == k) lp = -1;
            }
            agg_push_lds(mx, cnt, lp, r);
          }
        }
      }
      __syncthreads();
      if (tid == 0) S.hcount = 0;
    }
    __syncthreads();
  }
  if (overflow) flag_sweep(ctrl, kStRange);
  {  // one LDS atomic per wave
    const int64_t nf = wave_sum_i64(int64_t(__popc(fin)));
    if (lane_id() == 0 && nf != 0) atomicAdd(&S.proc, int(nf));
  }
  __syncthreads();  // nothing is in flight here, so this barrier waits for no store
  if (tid == 0 && S.proc != n) flag_sweep(ctrl, kStCycle);

  if (a.rem_out) {  // rem stayed in LDS during the levels; store it once
#pragma unroll
    for (int j = 0; j < NPT; ++j)
      if ((fin >> j) & 1u) a.rem_out[vv[j]] = mx[j * T + tid];
  }
  const BucketArgs& bk = a.bk;
  if (bk.bins) {
    // D (bins): the bin of each ready future and its rank inside this
    // workflow's part of the bin (LDS counters), kept in the consumer
    // counters, which the levels left at zero: bin | rank << 16 (rank <
    // lds_cap < 2^16, bin < kBinMax).  Then one segment of each bin for the
    // whole workflow (one atomic per bin), and each future is routed and
    // stored into its segment.
    // the searches of all NPT futures in lockstep (independent LDS reads)
    int64_t key[NPT];
    uint32_t at[NPT];
#pragma unroll
    for (int j = 0; j < NPT; ++j) {
      at[j] = 0;
      key[j] = ((ready >> j) & 1u) ? order_key(a, mx[j * T + tid], dl) : 0;
    }
    for (int step = bk.nb >> 1; step > 0; step >>= 1) {
#pragma unroll
      for (int j = 0; j < NPT; ++j)
        if (((ready >> j) & 1u) && bl.split[at[j] + step - 1] <= key[j]) at[j] += step;
    }
#pragma unroll
    for (int j = 0; j < NPT; ++j) {
      if (!((ready >> j) & 1u)) continue;
      cnt[j * T + tid] = int32_t(at[j] | (atomicAdd(&bl.cnt[at[j]], 1u) << 16));
    }
    __syncthreads();
    for (int t = tid; t < bk.nb; t += T) {
      const uint32_t c = bl.cnt[t];
      bl.base[t] = c ? add_agent(bk.cnt + t, c) : 0u;
      bl.cnt[t] = 0;  // clean for the next workflow
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < NPT; ++j) {
      if (!((ready >> j) & 1u)) continue;
      const int k = j * T + tid;
      int32_t route;
      int64_t cost;
      route_future(ty[j], ee[j], lc[j], int32_t(a.p.M), a.p.mig, it.type, it.idx, it.load, it.speed,
                   it.inv, it.pos, it.run, (a.p.policy & NALAR_ROUTE_STATEFUL) != 0, route, cost, it.prun);
      const uint32_t pk = uint32_t(cnt[k]);
      const uint32_t bn = pk & 0xFFFFu;
      const int64_t r = mx[k];
      store_ready(a, bn, (pk >> 16) + bl.base[bn], order_key(a, r, dl), lvl, dl - r, b + k, route, cost, acc);
      cnt[k] = 0;  // the next workflow starts from zero counters
    }
    return;
  }

  // D (buckets or staging): every bucket-slot atomic first, then the
  // routing (LDS and arithmetic only) while the atomics are in flight, then
  // the stores of the ready futures.  No barrier follows: the next workflow of
  // this workgroup touches only its own threads' LDS entries before its first
  // barrier.
  uint32_t bkt[NPT], slot[NPT];
#pragma unroll
  for (int j = 0; j < NPT; ++j) {
    bkt[j] = 0;
    slot[j] = 0;
    if (bk.nb > 0 && ((ready >> j) & 1u)) {
      bkt[j] = bucket_of<false>(bk, order_key(a, mx[j * T + tid], dl), lvl);
      slot[j] = add_agent(bk.cnt + bkt[j], 1u);
    }
  }
  int32_t route[NPT];
  int64_t cost[NPT];
#pragma unroll
  for (int j = 0; j < NPT; ++j) {
    route[j] = -1;
    cost[j] = 0;
    if ((ready >> j) & 1u)
      route_future(ty[j], ee[j], lc[j], int32_t(a.p.M), a.p.mig, it.type, it.idx, it.load, it.speed,
                   it.inv, it.pos, it.run, (a.p.policy & NALAR_ROUTE_STATEFUL) != 0, route[j],
                   cost[j], it.prun);
  }
#pragma unroll
  for (int j = 0; j < NPT; ++j) __asm__ __volatile__("" : "+v"(slot[j]) :: "memory");
#pragma unroll
  for (int j = 0; j < NPT; ++j) {
    if (!((ready >> j) & 1u)) continue;
    const int k = j * T + tid;
    store_ready(a, bkt[j], slot[j], order_key(a, mx[k], dl), lvl, dl - mx[k], b + k, route[j],
                cost[j], acc);
  }
}

// ------------------------------------------------------------ HBM workflow

template <int T, bool kFused, bool kLevels>
__device__ __attribute__((always_inline)) void sweep_hbm(const SweepArgs& a, const Layout& L, const ITabLds& it, Shared& S,
                          int w, int64_t b, int n, int64_t dl, int lvl, Acc& acc,
                          const int64_t* split_l) {
  const int tid = threadIdx.x;
  Ctrl* ctrl = a.ctrl;
  int32_t* cnt = a.g_cnt + b;
  int64_t* mx = a.g_mx + b;
  uint8_t* dn = a.g_dn + b;
  uint8_t* nr = a.g_nr + b;

  for (int k = tid; k < n; k += T) {
    const int32_t v = node_at(L, b + k);
    st_wg(&cnt[k], int32_t(0));
    st_wg(&mx[k], int64_t(0));
    dn[k] = a.p.done[v];
    nr[k] = 0;
  }
  if (tid == 0) { S.hcount = 0; S.fcount = 0; S.bad = 0; }
  __syncthreads();
  if (kFused) {  // the rules of nalar_problem for this workflow's futures
    for (int k = tid; k < n; k += T) {
      const int32_t v = node_at(L, b + k);
      const int32_t o0 = a.p.dep_off[v], o1 = a.p.dep_off[v + 1];
      const int32_t t = a.p.type[v], l = a.p.loc[v];
      const int64_t e = a.p.est[v];
      if ((a.p.wf[v] != w) | (t < 0) | (l < -1) | (int64_t(l) >= a.p.M) | (e < 0) |
          (e > NALAR_EST_MAX) | (dn[k] > 1) | (o0 < 0) | (o1 < o0) | (int64_t(o1) > a.p.E))
        S.bad = 1;
    }
    __syncthreads();
    if (S.bad) {  // reported; the workflow is left alone (the pass fails)
      __syncthreads();  // everyone has read the flag before it is reused
      if (tid == 0) flag_sweep(ctrl, kStInval);
      return;
    }
  }

  // out-degree counters and readiness
  for (int k0 = 0; k0 < n; k0 += T) {
    const int k = k0 + tid;
    const bool own = k < n;
    int32_t v = 0, off = 0, deg = 0;
    if (own) {
      v = node_at(L, b + k);
      off = a.p.dep_off[v];
      deg = a.p.dep_off[v + 1] - off;
    }
    const bool light = own && deg <= kHbmLight;
    if (own && !light) {
      const int slot = atomicAdd(&S.hcount, 1);
      if (slot < kHeavyCap) {
        S.hk[slot] = k; S.ho[slot] = off; S.hd[slot] = deg;
      } else {
        bool blocked = false;
        for (int e = 0; e < deg; ++e) {
          const int32_t lp = checked_dep(L, a.p.dep_idx[off + e], b, n, k, ctrl);
          if (lp >= 0) { add_wg(&cnt[lp], int32_t(1)); blocked |= dn[lp] == 0; }
        }
        if (blocked) nr[k] = 1;
      }
    }
    bool blocked = false;
    for (int q = 0;; ++q) {
      const bool has = light && q < deg;
      if (ballot(has) == 0) break;
      int32_t lp = -1;
      if (has) lp = checked_dep(L, a.p.dep_idx[off + q], b, n, k, ctrl);
      agg_count_hbm(cnt, lp);
      if (lp >= 0 && dn[lp] == 0) blocked = true;
    }
    if (light && blocked) nr[k] = 1;
  }
  __syncthreads();
  {
    const int hc = S.hcount < kHeavyCap ? S.hcount : kHeavyCap;
    for (int h = 0; h < hc; ++h) {
      const int k = S.hk[h], off = S.ho[h], deg = S.hd[h];
      bool blocked = false;
      for (int e0 = 0; e0 < deg; e0 += T) {
        const int e = e0 + tid;
        int32_t lp = -1;
        if (e < deg) lp = checked_dep(L, a.p.dep_idx[off + e], b, n, k, ctrl);
        agg_count_hbm(cnt, lp);
        if (lp >= 0 && dn[lp] == 0) blocked = true;
      }
      if (blocked) nr[k] = 1;
    }
  }
  __syncthreads();

  if (a.bk.nb == 0)
    for (int k = tid; k < n; k += T) a.stg_ready[b + k] = (dn[k] == 0 && nr[k] == 0) ? uint8_t(1 + lvl) : 0;
  if (tid == 0) S.hcount = 0;

  // frontier 0: futures without consumers
  int32_t* cur = a.g_front0 + b;
  int32_t* nxt = a.g_front1 + b;
  for (int k0 = 0; k0 < n; k0 += T) {
    const int k = k0 + tid;
    append_wave(k < n && ld_wg(&cnt[k]) == 0, k, cur, &S.fcount);
  }
  __syncthreads();
  int fsize = S.fcount;
  int64_t processed = 0;
  bool overflow = false;
  while (fsize > 0) {
    processed += fsize;
    if (tid == 0) { S.fnext = 0; S.hcount = 0; }
    __syncthreads();
    for (int i0 = 0; i0 < fsize; i0 += T) {
      const int i = i0 + tid;
      const bool act = i < fsize;
      int32_t k = 0, off = 0, deg = 0;
      int64_t r = 0;
      if (act) {
        k = cur[i];
        const int32_t v = node_at(L, b + k);
        r = clamp_rem((dn[k] ? 0 : a.p.est[v]) + ld_wg(&mx[k]), overflow);
        st_wg(&mx[k], r);
        if (a.rem_out) a.rem_out[v] = r;
        off = a.p.dep_off[v];
        deg = a.p.dep_off[v + 1] - off;
        if (deg > kHbmLight) {
          const int hs = atomicAdd(&S.hcount, 1);
          if (hs < kHeavyCap) {
            S.hk[hs] = k; S.ho[hs] = off; S.hd[hs] = deg;
          } else {
            for (int e = 0; e < deg; ++e) {
              const int32_t lp = local_of(L, a.p.dep_idx[off + e], b, n);
              if (lp >= 0 && lp != k) {
                max_wg(&mx[lp], r);
                if (add_wg(&cnt[lp], int32_t(-1)) == 1) {
                  nxt[atomicAdd(&S.fnext, 1)] = lp;
                }
              }
            }
          }
        }
      }
      const bool light = act && deg <= kHbmLight;
      for (int q = 0;; ++q) {
        const bool has = light && q < deg;
        if (ballot(has) == 0) break;
        int32_t lp = -1;
        if (has) {
          lp = local_of(L, a.p.dep_idx[off + q], b, n);
          if (lp == k) lp = -1;
        }
        agg_push_hbm(mx, cnt, lp, r, nxt, &S.fnext);
      }
    }
    __syncthreads();
    const int hc = S.hcount < kHeavyCap ? S.hcount : kHeavyCap;
    for (int h = 0; h < hc; ++h) {
      const int k = S.hk[h], off = S.ho[h], deg = S.hd[h];
      const int64_t r = ld_wg(&mx[k]);
      for (int e0 = 0; e0 < deg; e0 += T) {
        const int e = e0 + tid;
        int32_t lp = -1;
        if (e < deg) {
          lp = local_of(L, a.p.dep_idx[off + e], b, n);
          if (lp == k) lp = -1;
        }
        agg_push_hbm(mx, cnt, lp, r, nxt, &S.fnext);
      }
    }
    __syncthreads();
    fsize = S.fnext;
    int32_t* t = cur; cur = nxt; nxt = t;
    __syncthreads();
  }
  if (overflow) flag_sweep(ctrl, kStRange);
  if (tid == 0 && processed != n) flag_sweep(ctrl, kStCycle);

  // slack, route, staged at the future's position
  for (int k = tid; k < n; k += T) {
    if (dn[k] == 0 && nr[k] == 0) {
      const int32_t v = node_at(L, b + k);
      write_ready<kLevels>(a, it, b + k, a.p.type[v], a.p.loc[v], ld_wg(&mx[k]), a.p.est[v], dl, lvl, acc,
                           split_l);
    }
  }
  __syncthreads();
}

// ------------------------------------------------------------ ordered workflow

// Futures a thread carries through one step of the ordered pass's counting,
// their loads issued together.
constexpr int kHbmU = 4;
// The one-dependency summary the counting leaves by position (positions of a
// workflow on this path stay below 2^22, the chunk table's limit).
constexpr int32_t kOneNone = -1;
constexpr int32_t kOneMany = -2;
constexpr int32_t kOneBlocked = 1 << 30;

// Future v's done flag from the packed copy the node kernel wrote (1.5 MB per
// 12M futures, so that the random reads of dependencies' flags stay in L2).
__device__ inline bool done_bit(const uint32_t* bits, int32_t v) {
  return ((bits[uint32_t(v) >> 5] >> (uint32_t(v) & 31u)) & 1u) != 0u;
}

// A workflow in HBM whose every dependency lies at a lower position than its
// consumer (ids in topological order within the workflow, as when futures are
// appended after their dependencies) needs no out-degree counters and no
// frontiers: taking its positions in chunks of T from the last chunk to the
// first, every consumer of a future in an earlier chunk has already pushed its
// rem when that chunk is reached.  Inside a chunk, a future waits until its
// consumers in the same chunk (counted beforehand) have pushed; these rounds
// end because the pending future at the highest position never waits.
//
// The chunk being swept keeps its futures' running maxima in LDS.  A push
// into an earlier chunk is not an atomic on a random line of HBM: it is
// appended to that chunk's segment of a log (the segments sized by a count
// taken with the order check), and the chunk folds its segment into LDS when
// its turn comes.  A workflow of n futures costs about n / T chunks of a few
// round trips each, plus one write and one read of 12 bytes per dependency.
//
// Returns false, having written only its own scratch (the in-chunk counters),
// when some dependency does not lie lower, when there is no log, or when the
// chunk table does not fit; the caller then runs the level-synchronous sweep.
// lc: T ints of LDS; mxl: lds_cap int64 of LDS (T maxima, then the table).
template <int T>
__device__ __attribute__((always_inline)) bool sweep_hbm_ordered(const SweepArgs& a, const Layout& L, const ITabLds& it,
                                                                 const BlockSweepArgs& ba, Shared& S, int64_t b, int n,
                                                                 int64_t dl, int lvl, Acc& acc, const int64_t* split_l,
                                                                 int32_t* lc, int64_t* mxl, int lds_cap) {
  const int tid = threadIdx.x;
  Ctrl* ctrl = a.ctrl;
  const int nc = (n + T - 1) / T;
  if (ba.plog_lp == nullptr || T + nc > lds_cap || nc > 4 * T) return false;  // the same on every thread
  uint32_t* cseg = reinterpret_cast<uint32_t*>(mxl + T);  // [nc] pushes into each chunk, then its segment's start
  uint32_t* cfill = cseg + nc;                             // [nc] pushes appended to each segment so far
  int32_t* cnt = a.g_cnt + b;                              // consumers in the same chunk, by position
  // by position, what the second step needs of a future with one dependency:
  // that dependency's position, and kOneBlocked if it is not done; else
  // kOneNone (no valid dependency) or kOneMany (gather the list again)
  int32_t* one = a.g_front0 + b;
  __shared__ int64_t s_base;
  __shared__ uint32_t s_total;

  // 1: check the order and count each dependency's push: into its own
  // counter (HBM, by position) if the consumer is in the same chunk, else into
  // the count of its chunk's segment (LDS).  No chunk order is needed here:
  // kHbmU futures per thread, their loads issued together.  A future with a
  // single dependency also leaves its summary in `one`, so that the second
  // step reads one coalesced word instead of gathering the list again.
  for (int k = tid; k < n; k += T) st_wg(&cnt[k], int32_t(0));
  for (int i = tid; i < nc; i += T) { cseg[i] = 0; cfill[i] = 0; }
  if (tid == 0) { S.bad = 0; S.hcount = 0; }
  __syncthreads();
  // a dependency at position lp of the future at position k
  auto count = [&](int32_t lp, int k) -> bool {
    if (lp > k) return true;  // not below its consumer: not ordered
    if (lp >= (k / T) * T) add_wg(&cnt[lp], int32_t(1));
    else if (lp >= 0) atomicAdd(&cseg[lp / T], 1u);
    return false;
  };
  bool up = false;
  for (int k0 = 0; k0 < n; k0 += T * kHbmU) {
    int32_t v[kHbmU], off[kHbmU], deg[kHbmU], d0[kHbmU];
#pragma unroll
    for (int j = 0; j < kHbmU; ++j) {
      const int k = k0 + j * T + tid;
      v[j] = k < n ? node_at(L, b + k) : 0;
    }
#pragma unroll
    for (int j = 0; j < kHbmU; ++j) {
      const bool own = k0 + j * T + tid < n;
      off[j] = own ? a.p.dep_off[v[j]] : 0;
      deg[j] = own ? a.p.dep_off[v[j] + 1] - off[j] : 0;
    }
#pragma unroll
    for (int j = 0; j < kHbmU; ++j)
      d0[j] = deg[j] > 0 && deg[j] <= kHbmLight ? a.p.dep_idx[off[j]] : 0;
#pragma unroll
    for (int j = 0; j < kHbmU; ++j) {
      const int k = k0 + j * T + tid;
      if (k < n) one[k] = deg[j] == 0 ? kOneNone : kOneMany;
      if (deg[j] <= 0) continue;
      if (deg[j] <= kHbmLight) {
        const int32_t lp = checked_dep(L, d0[j], b, n, k, ctrl);
        up |= count(lp, k);
        if (deg[j] == 1)
          one[k] = lp < 0 || lp > k ? kOneNone : lp | (done_bit(ba.done_bits, d0[j]) ? 0 : kOneBlocked);
        for (int e = 1; e < deg[j]; ++e) up |= count(checked_dep(L, a.p.dep_idx[off[j] + e], b, n, k, ctrl), k);
        continue;
      }
      const int slot = atomicAdd(&S.hcount, 1);
      if (slot < kHeavyCap) {
        S.hk[slot] = k; S.ho[slot] = off[j]; S.hd[slot] = deg[j];
      } else {  // the list is full: this thread counts them itself
        for (int e = 0; e < deg[j]; ++e) up |= count(checked_dep(L, a.p.dep_idx[off[j] + e], b, n, k, ctrl), k);
      }
    }
  }
  if (up) S.bad = 1;
  __syncthreads();
  {
    const int hc = S.hcount < kHeavyCap ? S.hcount : kHeavyCap;
    bool hup = false;
    for (int h = 0; h < hc; ++h) {
      const int hk = S.hk[h], ho = S.ho[h], hd = S.hd[h];
      for (int e = tid; e < hd; e += T) hup |= count(checked_dep(L, a.p.dep_idx[ho + e], b, n, hk, ctrl), hk);
    }
    if (hup) S.bad = 1;
  }
  __syncthreads();
  const bool unordered = S.bad != 0;

  // the segments: an exclusive scan of the counts (up to four per thread),
  // and one stretch of the log for the whole workflow
  {
    constexpr int Q = 4;
    const int q = (nc + T - 1) / T;
    uint32_t x[Q], sum = 0;
#pragma unroll
    for (int j = 0; j < Q; ++j) {
      const int i = tid * q + j;
      x[j] = j < q && i < nc ? cseg[i] : 0u;
      sum += x[j];
    }
    const uint32_t inc = wave_incl_scan_u32(sum);
    if (lane_id() == kWave - 1) S.hk[tid / kWave] = int32_t(inc);
    __syncthreads();
    uint32_t run = 0;
    for (int w = 0; w < tid / kWave; ++w) run += uint32_t(S.hk[w]);
    run += inc - sum;
#pragma unroll
    for (int j = 0; j < Q; ++j) {
      const int i = tid * q + j;
      if (j < q && i < nc) cseg[i] = run;
      run += x[j];
    }
    if (tid == T - 1) {
      s_total = run;
      s_base = unordered ? 0 : int64_t(atomicAdd(reinterpret_cast<unsigned long long*>(&ctrl->plog_fill),
                                                 (unsigned long long)run));
    }
    __syncthreads();
  }
  const uint32_t total = s_total;
  const int64_t base = s_base;
  __syncthreads();  // every thread has read the flags before the caller reuses them
  if (unordered || base + int64_t(total) > ba.plog_cap) return false;
  int64_t* pr = ba.plog_r + base;
  int32_t* plp = ba.plog_lp + base;

  // a push of r into the future at position lp (lp < the consumer's)
  auto push = [&](int32_t lp, int64_t r, int c0) {
    if (lp >= c0) {
      atomicMax(reinterpret_cast<long long*>(&mxl[lp - c0]), (long long)r);
      atomicSub(&lc[lp - c0], 1);
    } else {
      const int cj = lp / T;
      const uint32_t at = cseg[cj] + atomicAdd(&cfill[cj], 1u);
      const uint32_t end = cj + 1 < nc ? cseg[cj + 1] : total;
      if (at < end) {
        plp[at] = lp;
        pr[at] = r;
      } else {
        flag_sweep(ctrl, kStCycle);  // cannot happen: the counts above are exact
      }
    }
  };

  // 2: the chunks from the last to the first.  Everything a future needs
  // except its consumers' max is loaded when its chunk starts (its first two
  // dependencies, their positions and done flags), while the chunk folds in
  // the pushes its futures received from later chunks.  A thread's ready
  // future is routed and stored while the loads of its next chunk are in
  // flight, off the rounds' critical path.
  bool overflow = false;
  bool prd = false;  // the thread's ready future of the previous chunk, not yet stored
  int32_t pty = 0, plo = -1;
  int64_t prem = 0, pest = 0, ppos = 0;
  for (int c0 = ((n - 1) / T) * T; c0 >= 0; c0 -= T) {
    const int k = c0 + tid;
    const bool own = k < n;
    int32_t v = 0, off = 0, deg = 0;
    bool dnk = true;
    int64_t est = 0;
    const int32_t o = own ? one[k] : kOneNone;
    if (own) {
      v = node_at(L, b + k);
      dnk = done_bit(ba.done_bits, v);
      est = a.p.est[v];
      lc[tid] = ld_wg(&cnt[k]);
    }
    if (o == kOneMany) {
      off = a.p.dep_off[v];
      deg = a.p.dep_off[v + 1] - off;
    } else if (o >= 0) {
      deg = 1;
    }
    const bool light = own && deg <= kHbmLight;
    int32_t p0 = 0, p1 = 0, lp0 = o >= 0 ? o & ~kOneBlocked : -1, lp1 = -1;
    bool blocked = o >= 0 && (o & kOneBlocked) != 0;
    if (o == kOneMany && light) {
      p0 = a.p.dep_idx[off];
      p1 = a.p.dep_idx[off + 1];  // deg >= 2
      lp0 = local_of(L, p0, b, n);
      lp1 = local_of(L, p1, b, n);
      if (lp0 == k) lp0 = -1;  // reported by the first step
      if (lp1 == k) lp1 = -1;
      if (lp0 >= 0) blocked |= !done_bit(ba.done_bits, p0);
      if (lp1 >= 0) blocked |= !done_bit(ba.done_bits, p1);
    }
    if (prd) {
      write_ready<false>(a, it, ppos, pty, plo, prem, pest, dl, lvl, acc, split_l);
      prd = false;
    }
    mxl[tid] = 0;
    if (tid == 0) { S.fcount = 0; S.hcount = 0; }
    __syncthreads();
    {
      const int ci = c0 / T;
      const uint32_t s0 = cseg[ci], s1 = s0 + cfill[ci];
      for (uint32_t i = s0 + uint32_t(tid); i < s1; i += T) {
        const int32_t lp = plp[i];
        atomicMax(reinterpret_cast<long long*>(&mxl[lp - c0]), (long long)pr[i]);
      }
    }
    bool pending = own;
    __syncthreads();
    for (int round = 0;; ++round) {
      const bool go = pending && lc[tid] == 0;
      __syncthreads();  // every count is read before this round's pushes
      if (go) {
        pending = false;
        const int64_t r = clamp_rem((dnk ? 0 : est) + mxl[tid], overflow);
        mxl[tid] = r;
        if (a.rem_out) a.rem_out[v] = r;
        // a heavy future goes to the workgroup's list; when that is full, its
        // thread pushes alone, as for a light one
        const int slot = light ? -1 : atomicAdd(&S.hcount, 1);
        if (slot >= 0 && slot < kHeavyCap) {
          S.hk[slot] = k; S.ho[slot] = off; S.hd[slot] = deg;
        } else {
          if (lp0 >= 0) push(lp0, r, c0);
          if (lp1 >= 0) push(lp1, r, c0);
          for (int e = light ? 2 : 0; e < deg; ++e) {
            const int32_t p = a.p.dep_idx[off + e];
            const int32_t lp = local_of(L, p, b, n);
            if (lp < 0 || lp == k) continue;
            blocked |= !done_bit(ba.done_bits, p);
            push(lp, r, c0);
          }
          const bool rd = !dnk && !blocked;
          if (a.bk.nb == 0) a.stg_ready[b + k] = rd ? uint8_t(1 + lvl) : 0;
          if (rd) {  // stored at the next chunk's start
            prd = true;
            pty = a.p.type[v];
            plo = a.p.loc[v];
            prem = r;
            pest = est;
            ppos = b + k;
          }
        }
      }
      if (pending) atomicAdd(&S.fcount, 1);
      __syncthreads();
      const int hc = S.hcount < kHeavyCap ? S.hcount : kHeavyCap;
      for (int h = 0; h < hc; ++h) {  // heavy futures: the workgroup pushes together
        const int hk = S.hk[h], ho = S.ho[h], hd = S.hd[h];
        const int64_t hr = mxl[hk - c0];
        if (tid == 0) S.proc = 0;
        __syncthreads();
        bool hb = false;
        for (int e = tid; e < hd; e += T) {
          const int32_t p = a.p.dep_idx[ho + e];
          const int32_t lp = local_of(L, p, b, n);
          if (lp < 0 || lp == hk) continue;
          hb |= !done_bit(ba.done_bits, p);
          push(lp, hr, c0);
        }
        if (hb) S.proc = 1;
        __syncthreads();
        if (tid == 0) {
          const int32_t hv = node_at(L, b + hk);
          const bool rd = !done_bit(ba.done_bits, hv) && S.proc == 0;
          if (a.bk.nb == 0) a.stg_ready[b + hk] = rd ? uint8_t(1 + lvl) : 0;
          if (rd) write_ready<false>(a, it, b + hk, a.p.type[hv], a.p.loc[hv], hr, a.p.est[hv], dl, lvl, acc, split_l);
        }
      }
      __syncthreads();
      const int pend = S.fcount;
      __syncthreads();  // every thread has read the counts before they are reset
      if (pend == 0) break;
      if (round > T) {  // cannot happen: some pending future never waits
        if (tid == 0) flag_sweep(ctrl, kStCycle);
        break;
      }
      if (tid == 0) { S.fcount = 0; S.hcount = 0; }
    }
  }
  if (prd) write_ready<false>(a, it, ppos, pty, plo, prem, pest, dl, lvl, acc, split_l);
  if (overflow) flag_sweep(ctrl, kStRange);
  __syncthreads();
  return true;
}

// ------------------------------------------------------------ wave workflow

// The LDS operations of one wave complete in program order, so a wave working
// on LDS of its own needs no barrier: each read observes every earlier write
// and atomic of the same wave.  wave_order() only keeps the compiler from
// moving LDS accesses across a phase boundary; it emits no wait, so
// outstanding HBM stores never stall the wave.
__device__ inline void wave_order() { __asm__ __volatile__("" ::: "memory"); }

// Instance tables of at most kWaveItabMax entries get one LDS copy per wave:
// the wave loads its entries into registers at kernel start and writes them
// to its copy just before it first routes, so the load's latency hides behind
// the sweep and no workgroup barrier is needed.
constexpr int kWaveItabMax = 2 * kWave;

struct ItabStage {
  int64_t load[2];
  double inv[2];
  int32_t type[2], idx[2], speed[2], pos[2];
  uint32_t run;
  bool pending;
  bool build;   // entry `lane` of the caller's table is in type/speed/load[0]: sort it here
};

__device__ inline void itab_stage_load(ItabStage& st, const ITab& g, int M, int ln) {
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int i = ln + u * kWave;
    if (i < M) {
      st.load[u] = g.load[i];
      st.inv[u] = g.inv_speed[i];
      st.type[u] = g.type[i];
      st.idx[u] = g.idx[i];
      st.speed[u] = g.speed[i];
      st.pos[u] = g.pos_of[i];
    }
  }
  st.run = g.run[ln];  // kTypeDirect == kWave entries
  st.pending = true;
}

// Sorts an instance table of at most 64 entries (entry l held by lane l) into
// the wave's LDS copy, with no workgroup barrier.  Types in [0, 64) (the usual
// case) are ranked with ballots: lanes of equal type from six bit ballots, the
// count of each type through LDS and one wave scan.  Other types fall back to a
// comparison against every entry.
__device__ inline void itab_wave_build(const ItabStage& st, const ITabLds& it, int M, int ln) {
  const bool valid = ln < M;
  const int32_t t = valid ? st.type[0] : 0;
  int less = 0, eq = 0, eq_below = 0;
  if (ballot(valid && uint32_t(t) >= uint32_t(kTypeDirect)) == 0) {
    uint64_t peers = ballot(valid);
#pragma unroll
    for (int bit = 0; bit < 6; ++bit) {
      const bool on = (t >> bit) & 1;
      const uint64_t m = ballot(valid && on);
      peers &= on ? m : ~m;
    }
    eq = valid ? int(__popcll(peers)) : 0;
    eq_below = valid ? int(__popcll(peers & lanemask_lt())) : 0;
    it.run[ln] = 0;                       // count of each type, then its run
    wave_order();
    if (valid && eq_below == 0) it.run[t] = uint32_t(eq);
    wave_order();
    const uint32_t c = it.run[ln];
    const uint32_t base = wave_incl_scan_u32(c) - c;
    wave_order();
    it.run[ln] = base | ((base + c) << 16);
    wave_order();
    less = valid ? int(it.run[t] & 0xFFFFu) : 0;
  } else {
    for (int j = 0; j < M; ++j) {
      const int32_t o = readlane_i32(t, j);
      less += o < t;
      eq += o == t;
      eq_below += (o == t) & (j < ln);
    }
    it.run[ln] = 0;
    wave_order();
    if (valid && t >= 0 && t < kTypeDirect && eq_below == 0)
      it.run[t] = uint32_t(less) | (uint32_t(less + eq) << 16);
  }
  if (valid) {
    const int rank = less + eq_below;
    const int32_t sp = st.speed[0];
    it.type[rank] = t;
    it.idx[rank] = ln;
    it.load[rank] = st.load[0];
    it.speed[rank] = sp;
    it.inv[rank] = sp >= 1 ? 1.0 / double(sp) : 0.0;
    it.pos[ln] = rank;
  }
  wave_order();
}

__device__ inline void itab_stage_store(ItabStage& st, const ITabLds& it, int M, int ln) {
  if (!st.pending) return;
  if (st.build) {
    itab_wave_build(st, it, M, ln);
    st.pending = false;
    return;
  }
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int i = ln + u * kWave;
    if (i < M) {
      it.load[i] = st.load[u];
      it.inv[i] = st.inv[u];
      it.type[i] = st.type[u];
      it.idx[i] = st.idx[u];
      it.speed[i] = st.speed[u];
      it.pos[i] = st.pos[u];
    }
  }
  it.run[ln] = st.run;
  st.pending = false;
}

// One wave sweeps a workflow of at most 64 * NPTW futures on its own LDS slice.

// LDS slice of one wave (cap futures).
struct WaveSlice {
  int64_t* mx;      // running max of the consumers' rem, then rem
  int32_t* cnt;     // consumers not yet finalised
  uint8_t* dn;      // done
  uint8_t* nr;      // some dependency not done (bit 0); finalised (bit 1, frontier rounds)
  // frontier rounds only (kFrontierMinNpt futures per lane and more)
  int64_t* est;     // est'
  uint32_t* d01;    // dependency slots 0 and 1 (as p01)
  uint32_t* d2;     // dependency slot 2 (as p2), or kHeavyMark
  uint16_t* q0;     // frontier queues (ping-pong)
  uint16_t* q1;
};

// From this many futures per lane the rounds follow a frontier (deep
// workflows: many levels, few futures finalised per level).
constexpr int kFrontierMinNpt = 4;
constexpr uint32_t kHeavyMark = 0xFFFFFFFFu;

// Rounds of the wave sweep: every owned future whose consumers are all
// finalised (counter zero) is finalised, rem = est' + running max, and pushed
// into its dependencies.  kHeavy adds whole-wave pushes for futures with more
// than kPmax dependencies, read from the dependency list in global memory.
template <int NPTW, bool kHeavy>
__device__ __attribute__((always_inline)) inline void rounds(
    const SweepArgs& a, const Layout& L, const WaveSlice& W, int64_t b, int n, uint32_t own,
    uint32_t heavy, const int64_t* ee, const uint32_t* p01, const uint32_t* p2, int64_t* rr,
    uint32_t& fin, bool& overflow) {
  const int ln = lane_id();
  fin = 0;
#pragma unroll
  for (int j = 0; j < NPTW; ++j) rr[j] = 0;
  for (;;) {
    uint32_t act = 0;
    int64_t mv[NPTW];
#pragma unroll
    for (int j = 0; j < NPTW; ++j) {
      mv[j] = 0;
      if (((own & ~fin) >> j) & 1u) {  // counter and running max in one round trip
        const int k = j * kWave + ln;
        const int32_t c = W.cnt[k];
        const int64_t m = W.mx[k];
        act |= uint32_t(c == 0) << j;
        mv[j] = m;
      }
    }
    if (ballot(act != 0) == 0) break;
#pragma unroll
    for (int j = 0; j < NPTW; ++j) {
      if ((act >> j) & 1u) {
        const int k = j * kWave + ln;
        const int64_t r = clamp_rem(ee[j] + mv[j], overflow);
        rr[j] = r;
        if ((heavy >> j) & 1u) {
          W.mx[k] = r;  // read by the whole wave below
        } else {
#pragma unroll
          for (int q = 0; q < kPmax; ++q) {
            const int lp = dep_at(p01[j], p2[j], q);
            if (lp >= 0) {
              atomicMax(reinterpret_cast<long long*>(&W.mx[lp]), (long long)r);
              atomicSub(&W.cnt[lp], 1);
            }
          }
        }
      }
    }
    fin |= act;
    // futures with many dependencies: the whole wave pushes each one
    if (kHeavy) {
      const uint32_t hact = act & heavy;
      for (uint64_t hs = ballot(hact != 0); hs; hs &= hs - 1) {
        const int src = __builtin_ctzll(hs);
        for (uint32_t hj = uint32_t(readlane_i32(int(hact), src)); hj; hj &= hj - 1) {
          const int kh = __builtin_ctz(hj) * kWave + src;
          const int64_t r = W.mx[kh];
          const int32_t vh = node_at(L, b + kh);
          const int o = a.p.dep_off[vh];
          const int d = a.p.dep_off[vh + 1] - o;
          for (int e0 = 0; e0 < d; e0 += kWave) {
            const int e = e0 + ln;
            if (e < d) {
              const int32_t lp = local_of(L, a.p.dep_idx[o + e], b, n);
              if (lp >= 0 && lp != kh) {
                atomicMax(reinterpret_cast<long long*>(&W.mx[lp]), (long long)r);
                atomicSub(&W.cnt[lp], 1);
              }
            }
          }
        }
      }
    }
    wave_order();
  }
}

// The workflows one wave sweeps together: ns consecutive workflows w[0] ..
// occupying positions [b, b + n), workflow i at local indices [c[i], c[i+1])
// (c[0] = 0, c[ns] = n), with their deadlines (less now) and key offsets.
// Every field is the same on every lane.
template <int G>
struct Seg {
  int64_t b;
  int n;
  int ns;
  int c[G + 1];
  int64_t w[G];
  int64_t dl[G];
  int lvl[G];
  // the part of local index k
  __device__ int part(int k) const {
    int s = 0;
#pragma unroll
    for (int i = 1; i < G; ++i) s += (i < ns && k >= c[i]) ? 1 : 0;
    return s;
  }
};

// Rounds that follow a frontier instead of rescanning every owned future:
// a future enters the next frontier when the push that drops its consumer
// counter to zero (a returning LDS atomic) sees it, so each round touches
// only the futures it finalises, processed by whichever lanes take the queue
// entries (estimates and dependency slots are copied to LDS first).  Futures
// with more than kPmax dependencies push their list with the whole wave.
// Results as for rounds(): rem of every finalised future in rr, fin bits.
template <int NPTW>
__device__ __attribute__((always_inline)) inline void rounds_frontier(
    const SweepArgs& a, const Layout& L, const WaveSlice& W, int64_t b, int n, uint32_t own,
    uint32_t heavy, const int64_t* ee, const uint32_t* p01, const uint32_t* p2, int64_t* rr,
    uint32_t& fin, bool& overflow) {
  const int ln = lane_id();
#pragma unroll
  for (int j = 0; j < NPTW; ++j) {
    if ((own >> j) & 1u) {
      const int k = j * kWave + ln;
      W.est[k] = ee[j];
      W.d01[k] = p01[j];
      W.d2[k] = ((heavy >> j) & 1u) ? kHeavyMark : p2[j];
    }
  }
  // the first frontier: futures with no consumer left to wait for
  int qn = 0;
#pragma unroll
  for (int j = 0; j < NPTW; ++j) {
    const int k = j * kWave + ln;
    const bool z = ((own >> j) & 1u) && W.cnt[k] == 0;
    const uint64_t m = ballot(z);
    if (z) W.q0[qn + int(lanes_below(m))] = uint16_t(k);
    qn += int(__popcll(m));
  }
  wave_order();
  uint16_t* cq = W.q0;
  uint16_t* nq = W.q1;
  while (qn > 0) {
    int nn = 0;
    for (int base = 0; base < qn; base += kWave) {
      const int e = base + ln;
      const bool act = e < qn;
      int k = 0;
      int64_t r = 0;
      uint32_t d01 = 0xFFFFFFFFu, d2 = 0xFFFFFFFFu;
      if (act) {
        k = cq[e];
        r = clamp_rem(W.est[k] + W.mx[k], overflow);
        W.mx[k] = r;  // rem from here on
        W.nr[k] |= 2u;
        d01 = W.d01[k];
        d2 = W.d2[k];
      }
      const bool hv = act && d2 == kHeavyMark;
      int32_t lps[kPmax];
      bool nw[kPmax];
#pragma unroll
      for (int q = 0; q < kPmax; ++q) {
        const int lp = (act && !hv) ? dep_at(d01, d2, q) : -1;
        lps[q] = lp;
        nw[q] = false;
        if (lp >= 0) {
          atomicMax(reinterpret_cast<long long*>(&W.mx[lp]), (long long)r);
          nw[q] = atomicSub(&W.cnt[lp], 1) == 1;
        }
      }
#pragma unroll
      for (int q = 0; q < kPmax; ++q) {
        const uint64_t m = ballot(nw[q]);
        if (nw[q]) nq[nn + int(lanes_below(m))] = uint16_t(lps[q]);
        nn += int(__popcll(m));
      }
      for (uint64_t hs = ballot(hv); hs; hs &= hs - 1) {
        const int src = __builtin_ctzll(hs);
        const int kh = readlane_i32(k, src);
        const int64_t rh = readlane_i64(r, src);
        const int32_t vh = node_at(L, b + kh);
        const int o = a.p.dep_off[vh];
        const int d = a.p.dep_off[vh + 1] - o;
        for (int e0 = 0; e0 < d; e0 += kWave) {
          const int ex = e0 + ln;
          bool nwh = false;
          int32_t lp = -1;
          if (ex < d) {
            lp = local_of(L, a.p.dep_idx[o + ex], b, n);
            if (lp >= 0 && lp != kh) {
              atomicMax(reinterpret_cast<long long*>(&W.mx[lp]), (long long)rh);
              nwh = atomicSub(&W.cnt[lp], 1) == 1;
            }
          }
          const uint64_t m = ballot(nwh);
          if (nwh) nq[nn + int(lanes_below(m))] = uint16_t(lp);
          nn += int(__popcll(m));
        }
      }
    }
    wave_order();
    uint16_t* t = cq;
    cq = nq;
    nq = t;
    qn = nn;
  }
  fin = 0;
#pragma unroll
  for (int j = 0; j < NPTW; ++j) {
    rr[j] = 0;
    if ((own >> j) & 1u) {
      const int k = j * kWave + ln;
      if (W.nr[k] & 2u) {
        fin |= 1u << j;
        rr[j] = W.mx[k];
      }
    }
  }
  wave_order();
}

// Attributes of future spec + lane loaded before the workflow's bounds are
// known, spec being the bound that equal workflow sizes would give (the
// fused one-future-per-lane wave sweep; valid when the bound turns out so).
struct PreAttr {
  int64_t e = 0;
  int32_t o0 = 0, o1 = 0, t = 0, l = -1, wfv = -1;
  uint8_t d = 1;
};

// Sweep of one workflow by one wave.  Lane l owns futures l, l+64, ... of the
// workflow and keeps their estimate and (up to three) dependencies in
// registers.  Each round, every owned future whose consumers are all finalised
// (counter zero) is finalised: rem = est' + running max, pushed into its
// dependencies' running max, whose counters drop by one.  Pushes return
// nothing, so a round costs one LDS round trip (the counter and running-max
// reads) however many futures it finalises.  Futures with more dependencies
// are pushed by the whole wave from the dependency list.
template <int NPTW, bool kFused, int G>
__device__ __attribute__((always_inline)) void sweep_wave(const SweepArgs& a, const Layout& L, const ITabLds& it,
                           const WaveSlice& W, const Seg<G>& sg, Acc& acc, ItabStage& st,
                           const PreAttr& pre, bool use_pre) {
  const int64_t b = sg.b;
  const int n = sg.n;
  const int ln = lane_id();
  Ctrl* ctrl = a.ctrl;
  int32_t vv[NPTW], ty[NPTW], lc[NPTW], off[NPTW], deg[NPTW];
  int64_t ee[NPTW];
  uint32_t p01[NPTW], p2[NPTW];
  uint32_t own = 0, ready = 0, heavy = 0;

  // A: attributes in one round trip; reset the state
#pragma unroll
  for (int j = 0; j < NPTW; ++j) {
    const int k = j * kWave + ln;
    vv[j] = 0; ty[j] = 0; lc[j] = -1; off[j] = 0; deg[j] = 0; ee[j] = 0;
    p01[j] = 0xFFFFFFFFu; p2[j] = kNoDep;
    if (k < n) {
      own |= 1u << j;
      const int32_t v = node_at(L, b + k);
      uint8_t d;
      int32_t o0, o1, t, l, wfv = 0;
      int64_t e;
      if (NPTW == 1 && kFused && use_pre) {  // loaded ahead (the same future: b is the guess)
        d = pre.d;
        o0 = pre.o0;
        o1 = pre.o1;
        t = pre.t;
        l = pre.l;
        e = pre.e;
        wfv = pre.wfv;
      } else {
        d = a.p.done[v];
        o0 = a.p.dep_off[v];
        o1 = a.p.dep_off[v + 1];
        t = a.p.type[v];
        l = a.p.loc[v];
        e = a.p.est[v];
        if (kFused) wfv = a.p.wf[v];
      }
      if (kFused) {  // the rules of nalar_problem for this future
        const bool bad = (wfv != sg.w[sg.part(k)]) | (t < 0) | (l < -1) | (int64_t(l) >= a.p.M) | (e < 0) |
                         (e > NALAR_EST_MAX) | (d > 1) | (o0 < 0) | (o1 < o0) | (int64_t(o1) > a.p.E);
        if (bad) {  // reported; neutralised so that no access leaves its array
          flag_sweep(ctrl, kStInval);
          o0 = o1 = 0;
          l = -1;
          d = 1;
        }
      }
      vv[j] = v;
      off[j] = o0;
      deg[j] = o1 - o0;
      ty[j] = t;
      lc[j] = l;
      ee[j] = d ? 0 : e;
      W.cnt[k] = 0;
      W.mx[k] = 0;
      W.dn[k] = d;
      W.nr[k] = 0;
    }
  }
  wave_order();

  // B: out-degree counters, readiness, dependency lists into registers
#pragma unroll
  for (int j = 0; j < NPTW; ++j) {
    if (ballot((own >> j) & 1u) == 0) continue;
    const int k = j * kWave + ln;
    const bool mine = (own >> j) & 1u;
    const bool light = mine && deg[j] <= kPmax;
    bool blocked = false;
    uint32_t packed[kPmax];
#pragma unroll
    for (int q = 0; q < kPmax; ++q) {
      int32_t lp = -1;
      if (light && q < deg[j]) {
        if (G == 1) {
          lp = checked_dep(L, a.p.dep_idx[off[j] + q], b, n, k, ctrl);
        } else {
          const int pk = sg.part(k);
          lp = checked_dep_seg(L, a.p.dep_idx[off[j] + q], b, n, sg.c[pk], sg.c[pk + 1], k, ctrl);
        }
      }
      packed[q] = lp >= 0 ? uint32_t(lp) : kNoDep;
      if (lp >= 0) {
        atomicAdd(&W.cnt[lp], 1);
        blocked |= W.dn[lp] == 0;
      }
    }
    if (light) {
      p01[j] = packed[0] | (packed[1] << 16);
      p2[j] = packed[2];
      if (blocked) W.nr[k] = 1;
    }
    if (mine && !light) heavy |= 1u << j;
    for (uint64_t hm = ballot(mine && !light); hm; hm &= hm - 1) {
      const int src = __builtin_ctzll(hm);
      const int kh = j * kWave + src;
      const int o = readlane_i32(off[j], src);
      const int d = readlane_i32(deg[j], src);
      const int ph = sg.part(kh);
      bool blk = false;
      for (int e0 = 0; e0 < d; e0 += kWave) {
        const int e = e0 + ln;
        if (e < d) {
          const int32_t lp = G == 1 ? checked_dep(L, a.p.dep_idx[o + e], b, n, kh, ctrl)
                                    : checked_dep_seg(L, a.p.dep_idx[o + e], b, n, sg.c[ph], sg.c[ph + 1], kh, ctrl);
          if (lp >= 0) {
            atomicAdd(&W.cnt[lp], 1);
            blk |= W.dn[lp] == 0;
          }
        }
      }
      if (ballot(blk) != 0 && ln == 0) W.nr[kh] = 1;
    }
  }
  wave_order();

  // the instance table's LDS copy, now that its loads have long returned and
  // no store is in flight (a wait here costs nothing)
  itab_stage_store(st, it, int(a.p.M), ln);

  // readiness (stored after the rounds: no store may be in flight during
  // them, or every round would wait for it)
#pragma unroll
  for (int j = 0; j < NPTW; ++j) {
    if ((own >> j) & 1u) {
      const int k = j * kWave + ln;
      if (W.dn[k] == 0 && W.nr[k] == 0) ready |= 1u << j;
    }
  }
  wave_order();

  // C: rounds of finalisation (the variant without futures of many
  // dependencies touches no global memory inside its loop, so nothing there
  // waits on outstanding loads or stores)
  bool overflow = false;
  uint32_t fin = 0;
  int64_t rr[NPTW];
  if constexpr (NPTW >= kFrontierMinNpt)
    rounds_frontier<NPTW>(a, L, W, b, n, own, heavy, ee, p01, p2, rr, fin, overflow);
  else if (ballot(heavy != 0) != 0)  // a future with many dependencies: the variant that pushes it
    rounds<NPTW, true>(a, L, W, b, n, own, heavy, ee, p01, p2, rr, fin, overflow);
  else
    rounds<NPTW, false>(a, L, W, b, n, own, heavy, ee, p01, p2, rr, fin, overflow);
  if (overflow) flag_sweep(ctrl, kStRange);
  // a future never finalised lies on a cycle (or depends on one)
  if (ballot((own & ~fin) != 0) != 0 && ln == 0) flag_sweep(ctrl, kStCycle);

  // D: bucket slots first, then the routing (LDS only) while the slot
  // atomics are in flight, then every store.  No store is issued between the
  // atomics and the routing, so nothing makes the routing wait for them.
  const BucketArgs& bk = a.bk;
  uint32_t bkt[NPTW], slot[NPTW];
#pragma unroll
  for (int j = 0; j < NPTW; ++j) {
    bkt[j] = 0;
    slot[j] = 0;
    if (bk.nb > 0 && ((ready >> j) & 1u)) {
      const int pk = sg.part(j * kWave + ln);
      bkt[j] = bucket_of<true>(bk, order_key(a, rr[j], sg.dl[pk]), sg.lvl[pk]);
      slot[j] = add_agent(bk.cnt + bkt[j], 1u);
    }
  }
  int32_t route[NPTW];
  int64_t cost[NPTW];
#pragma unroll
  for (int j = 0; j < NPTW; ++j) {
    route[j] = -1;
    cost[j] = 0;
    if ((ready >> j) & 1u)
      route_future(ty[j], ee[j], lc[j], int32_t(a.p.M), a.p.mig, it.type, it.idx, it.load,
                   it.speed, it.inv, it.pos, it.run, (a.p.policy & NALAR_ROUTE_STATEFUL) != 0,
                   route[j], cost[j]);
  }
#pragma unroll
  for (int j = 0; j < NPTW; ++j) __asm__ __volatile__("" : "+v"(slot[j]) :: "memory");
#pragma unroll
  for (int j = 0; j < NPTW; ++j) {
    if (!((own >> j) & 1u)) continue;
    const int64_t pos = b + j * kWave + ln;
    if (bk.nb == 0) a.stg_ready[pos] = ((ready >> j) & 1u) ? uint8_t(1 + sg.lvl[sg.part(j * kWave + ln)]) : uint8_t(0);
    if (a.rem_out) a.rem_out[vv[j]] = rr[j];
    if ((ready >> j) & 1u) {
      const int pk = sg.part(j * kWave + ln);
      const int64_t dl = sg.dl[pk];
      store_ready(a, bkt[j], slot[j], order_key(a, rr[j], dl), sg.lvl[pk], dl - rr[j], pos, route[j],
                  cost[j], acc);
    }
  }
  wave_order();
}

// ------------------------------------------------------------ kernel

template <int T, int NPT>
__global__ __launch_bounds__(T) void k_sweep(SweepArgs a, int lds_cap, BlockSweepArgs ba) {
  constexpr int NW = T / kWave;
  Ctrl* ctrl = a.ctrl;
  for (int64_t i = int64_t(blockIdx.x) * T + threadIdx.x; i < a.bk_clear_n; i += int64_t(gridDim.x) * T)
    a.bk_clear[i] = 0;  // the next pass's bucket counters
  if (ctrl->status != 0) return;  // written by earlier kernels only
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ Shared S;

  const int M = int(a.p.M);
  const int tid = threadIdx.x;
  unsigned char* sp = smem;
  ITabLds it;
  it.load = reinterpret_cast<int64_t*>(sp); sp += 8 * size_t(M);
  it.inv = reinterpret_cast<double*>(sp); sp += 8 * size_t(M);
  int64_t* mx = reinterpret_cast<int64_t*>(sp); sp += 8 * size_t(lds_cap);
  it.type = reinterpret_cast<int32_t*>(sp); sp += 4 * size_t(M);
  it.idx = reinterpret_cast<int32_t*>(sp); sp += 4 * size_t(M);
  it.speed = reinterpret_cast<int32_t*>(sp); sp += 4 * size_t(M);
  it.pos = reinterpret_cast<int32_t*>(sp); sp += 4 * size_t(M);
  it.run = reinterpret_cast<uint32_t*>(sp); sp += 4 * size_t(kTypeDirect);
  it.prun = reinterpret_cast<uint32_t*>(sp); sp += 4 * size_t(kTypeDirect);
  BinLds bl;
  int64_t* split_l = reinterpret_cast<int64_t*>(sp); sp += 8 * size_t(kBinMax);
  bl.split = split_l;
  bl.cnt = reinterpret_cast<uint32_t*>(sp); sp += 4 * size_t(kBinMax);
  bl.base = reinterpret_cast<uint32_t*>(sp); sp += 4 * size_t(kBinMax);
  int32_t* cnt = reinterpret_cast<int32_t*>(sp); sp += 4 * size_t(lds_cap);
  uint8_t* dn = sp; sp += lds_cap;
  uint8_t* nr = sp;

  for (int i = tid; i < M; i += T) {
    it.load[i] = a.itab.load[i];
    it.inv[i] = a.itab.inv_speed[i];
    it.type[i] = a.itab.type[i];
    it.idx[i] = a.itab.idx[i];
    it.speed[i] = a.itab.speed[i];
    it.pos[i] = a.itab.pos_of[i];
  }
  for (int t = tid; t < kTypeDirect; t += blockDim.x) {
    it.run[t] = a.itab.run[t];
    it.prun[t] = a.itab.prun[t];
  }
  if (a.bk.bins) {  // the splitters; the counters start at zero
    for (int i = tid; i < a.bk.nb - 1; i += T) split_l[i] = a.bk.split[i];
    for (int i = tid; i < a.bk.nb; i += T) bl.cnt[i] = 0;
  }

  const Layout L{a.node_of_pos, a.pos_of_node, a.p.N};
  Acc acc;
  uint32_t lmask = 0;  // priority levels of the block's workflows
  for (int64_t w = blockIdx.x; w < a.p.W; w += gridDim.x) {
    const int64_t b = a.wf_off[w];
    const int n = a.wf_off[w + 1] - int32_t(b);
    if (n <= 0) continue;
    const int64_t dl = a.p.deadline[w] - a.p.now;
    const int lvl = prio_level(a, w);
    lmask |= level_bit(lvl);
    if (!a.force_global && n <= lds_cap)
      sweep_lds<T, NPT>(a, L, it, S, mx, cnt, dn, nr, lds_cap, b, n, dl, lvl, acc, bl);
    else if (!(ba.ordered && sweep_hbm_ordered<T>(a, L, it, ba, S, b, n, dl, lvl, acc, split_l, cnt, mx, lds_cap)))
      sweep_hbm<T, false, false>(a, L, it, S, int(w), b, n, dl, lvl, acc, split_l);
  }

  // fold the block's slack range and ready count into the control block
  const int64_t mn = wave_min_i64(acc.tmin);
  const int64_t mxv = wave_max_i64(acc.tmax);
  const int64_t rd = wave_sum_i64(acc.tready);
  const int wv = tid / kWave;
  if (lane_id() == 0) { S.red[0][wv] = mn; S.red[1][wv] = mxv; S.red[2][wv] = rd; }
  __syncthreads();
  if (tid == 0) {
    int64_t a0 = INT64_MAX, a1 = INT64_MIN, a2 = 0;
    for (int x = 0; x < NW; ++x) {
      a0 = S.red[0][x] < a0 ? S.red[0][x] : a0;
      a1 = S.red[1][x] > a1 ? S.red[1][x] : a1;
      a2 += S.red[2][x];
    }
    if (a2 > 0) {
      const int slot = blockIdx.x & (kParts - 1);
      __hip_atomic_fetch_min(&ctrl->part_min[slot], a0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_fetch_max(&ctrl->part_max[slot], a1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      add_agent(&ctrl->part_cnt[slot], a2);
      if (a.p.prio)
        __hip_atomic_fetch_or(&ctrl->part_lvl[slot], lmask, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

constexpr int kWaveNpt = 8;                  // futures per lane in the wave path
constexpr int kWaveCap = kWave * kWaveNpt;     // at most 512 futures per wave
constexpr int kWaveBlock = 256;                // four independent waves per workgroup
constexpr int kWavesPerBlock = kWaveBlock / kWave;
static_assert(kWavesPerBlock == 4, "the wave kernel's flags assume four waves");
constexpr size_t kWaveSliceBytesPerFuture = 8 + 4 + 1 + 1;
constexpr size_t kWaveFrontierBytesPerFuture = 8 + 4 + 4 + 2 + 2;  // est', slots, two queues

// Instance table of the fused mode, built by the whole workgroup into its LDS
// (M <= kWaveItabMax, entry i held by thread i, loaded by the caller): rank by
// (type, index), and the run of each small type from the counts of smaller
// and equal types.  Every thread of the workgroup calls it; two barriers.
__device__ __attribute__((always_inline)) void build_itab_block(const ITabLds& it, int M, int32_t t,
                                                                int32_t sp, int64_t ld,
                                                                int32_t* s_type) {
  const int i = threadIdx.x;
  if (i < M) s_type[i] = t;
  if (i < kTypeDirect) it.run[i] = 0;
  __syncthreads();
  if (i < M) {
    // four types per LDS read; the bound lives in a vector register (as a
    // scalar it would be reloaded from the arguments, waiting on every LDS
    // read in flight).  Each comparison feeds one add right away, so no
    // comparison mask stays live (those live in scalar registers).
    int mv;
    __asm__ __volatile__("v_mov_b32 %0, %1" : "=v"(mv) : "s"(M));
    int less = 0, eq_below = 0, eq = 0;
    const int4* s4 = reinterpret_cast<const int4*>(s_type);
#pragma unroll 1
    for (int j0 = 0; j0 < mv; j0 += 4) {
      const int4 v = s4[j0 >> 2];
      const int32_t o[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int j = j0 + q;
        const int in = j < mv ? 1 : 0;
        const int lt = o[q] < t ? in : 0;
        const int e = o[q] == t ? in : 0;
        less += lt;
        eq += e;
        eq_below += j < i ? e : 0;
      }
    }
    const int rank = less + eq_below;
    it.type[rank] = t;
    it.idx[rank] = i;
    it.load[rank] = ld;
    it.speed[rank] = sp;
    it.inv[rank] = sp >= 1 ? 1.0 / double(sp) : 0.0;
    it.pos[i] = rank;
    if (t >= 0 && t < kTypeDirect && eq_below == 0)
      it.run[t] = uint32_t(less) | (uint32_t(less + eq) << 16);
  }
  __syncthreads();
}

// Bounds of workflow w: from the offsets computed before the sweep, or (fused
// mode, ids grouped by workflow) as lower bounds of w and w + 1 in wf, found
// by lanes 0 and 1 of the wave (wave-uniform call).
__device__ inline void wf_bounds(const SweepArgs& a, int64_t w, int64_t& b, int& n) {
  if (!a.fused) {
    b = a.wf_off[w];
    n = a.wf_off[w + 1] - int32_t(b);
    return;
  }
  const int64_t N = a.p.N, Wn = a.p.W;
  const int ln = lane_id();
  int32_t lb = 0;
  if (ln < 2) lb = int32_t(lower_bound_from(a.p.wf, N, w + ln, ((w + ln) * N) / Wn));
  const int32_t lo = readlane_i32(lb, 0), hi = readlane_i32(lb, 1);
  b = lo;
  n = hi - lo;
  // the ranges must tile [0, N): none negative, the first at 0, the last at N
  if (ln == 0 && ((n < 0) | ((w == 0) & (lo != 0)) | ((w == Wn - 1) & (int64_t(hi) != N))))
    flag_sweep(a.ctrl, kStInval);
}

// LDS of the instance tables of one wave workgroup.
__host__ __device__ inline size_t itab_lds_wave(int64_t M) {
  const size_t one = 32 * size_t(M) + 4 * kTypeDirect;
  return M <= kWaveItabMax ? one * kWavesPerBlock : one;
}

__device__ inline ITabLds carve_itab(unsigned char* sp, int M) {
  ITabLds it;
  it.load = reinterpret_cast<int64_t*>(sp); sp += 8 * size_t(M);
  it.inv = reinterpret_cast<double*>(sp); sp += 8 * size_t(M);
  it.type = reinterpret_cast<int32_t*>(sp); sp += 4 * size_t(M);
  it.idx = reinterpret_cast<int32_t*>(sp); sp += 4 * size_t(M);
  it.speed = reinterpret_cast<int32_t*>(sp); sp += 4 * size_t(M);
  it.pos = reinterpret_cast<int32_t*>(sp); sp += 4 * size_t(M);
  it.run = reinterpret_cast<uint32_t*>(sp);
  it.prun = nullptr;  // the wave tables scan whole runs
  return it;
}

// The first things a wave reads: the pointers and sizes its opening loads
// need, passed as the wave kernel's leading scalar arguments so that they
// arrive preloaded in scalar registers (the library is built with
// kernel-argument preloading; fourteen dwords fit beside the segment
// pointer) and the opening loads start at once.
struct WaveHead {
  const int32_t* inst_type;
  const int32_t* inst_speed;
  const int64_t* inst_load;
  const int64_t* deadline;
  const int32_t* wf;
  int64_t N;
  int32_t W;
  int32_t M;
};
static_assert(sizeof(WaveHead) == 14 * 4, "the preloaded arguments fill fourteen dwords");

// The wave kernel's arguments as they lie in the kernel-argument segment
// (explicit arguments in order at their natural alignment, from offset 0).
struct WaveKernArgs {
  WaveHead head;
  SweepArgs a;
  int wcap;
};
constexpr int kKernArgLines = int((sizeof(WaveKernArgs) + 63) / 64);
static_assert(kKernArgLines == 8, "warm_kernargs loads eight lines");

// The eight 64-byte lines of the wave kernel's arguments are brought into the
// scalar cache with loads that are all in flight at once (issued before the
// opening loads, waited for after them), and the argument block is then read
// through a pointer the compiler cannot read ahead of the wait: the block is
// large and its fields are reloaded on demand, so every field read is a
// scalar-cache hit instead of a round trip per cold line.
typedef __attribute__((address_space(4))) const WaveKernArgs* WaveKernArgsPtr;
struct KernArgWarm {
  uint32_t v[kKernArgLines];
  WaveKernArgsPtr kp;
};

__device__ inline void warm_kernargs_issue(KernArgWarm& w) {
  w.kp = (WaveKernArgsPtr)__builtin_amdgcn_kernarg_segment_ptr();
  __asm__ __volatile__(
      "s_load_dword %0, %8, 0\n"
      "s_load_dword %1, %8, 64\n"
      "s_load_dword %2, %8, 128\n"
      "s_load_dword %3, %8, 192\n"
      "s_load_dword %4, %8, 256\n"
      "s_load_dword %5, %8, 320\n"
      "s_load_dword %6, %8, 384\n"
      "s_load_dword %7, %8, 448"
      : "=&s"(w.v[0]), "=&s"(w.v[1]), "=&s"(w.v[2]), "=&s"(w.v[3]), "=&s"(w.v[4]), "=&s"(w.v[5]),
        "=&s"(w.v[6]), "=&s"(w.v[7])
      : "s"(w.kp));
}

// The destinations of the loads above stay reserved until this wait (they are
// its inputs), so nothing else lands in a register a load is still writing.
__device__ inline const WaveKernArgs* warm_kernargs_wait(KernArgWarm& w) {
  __asm__ __volatile__("s_waitcnt lgkmcnt(0)"
                       : "+s"(w.kp)
                       : "s"(w.v[0]), "s"(w.v[1]), "s"(w.v[2]), "s"(w.v[3]), "s"(w.v[4]), "s"(w.v[5]),
                         "s"(w.v[6]), "s"(w.v[7]));
  return (const WaveKernArgs*)w.kp;
}

// The next pass's bucket counters and, in fused mode, its control block.
// Done last: a store in flight would make every later wait for a load wait
// for it too (one counter covers both).
template <bool kFused>
__device__ inline void clear_for_next_pass(const SweepArgs& a) {
  const int64_t gi = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t gstride = int64_t(gridDim.x) * blockDim.x;
  for (int64_t i = gi; i < a.bk_clear_n; i += gstride) a.bk_clear[i] = 0;
  if (kFused) reset_ctrl_spread(a.next_ctrl, gi, gstride);
}

// Bounds of group pw (workflows pw*G .. pw*G + G - 1): lane i <= G gets the
// first position of workflow pw*G + i (N past the last workflow), lane i < G
// that workflow's raw deadline.
template <int G>
__device__ inline void group_bounds(const SweepArgs& a, int64_t pw, int32_t& lbv, int64_t& rawv) {
  const int ln = lane_id();
  const int64_t W = a.p.W, N = a.p.N;
  const int64_t key = pw * G + ln < W ? pw * G + ln : W;
  lbv = 0;
  rawv = 0;
  if (ln <= G) {
    if (a.fused)
      lbv = key >= W ? int32_t(N) : int32_t(lower_bound_from(a.p.wf, N, key, (key * N) / W));
    else
      lbv = a.wf_off[key];
  }
  if (ln < G && pw * G + ln < W) rawv = a.p.deadline[pw * G + ln];
}

// The group's segment description from the per-lane bounds and deadlines, and
// (fused mode) the rules of nalar_problem for its workflows: the ranges tile
// [0, N) in workflow order, deadlines within the horizon, levels up to 15.
template <int G, bool kFused>
__device__ inline Seg<G> make_seg(const SweepArgs& a, int64_t pw, int32_t lbv, int64_t rawv, Ctrl* ctrl) {
  const int ln = lane_id();
  const int64_t W = a.p.W;
  Seg<G> sg;
  const int64_t w0 = pw * G;
  sg.ns = int(W - w0 < G ? W - w0 : G);
  int32_t lb[G + 1];
#pragma unroll
  for (int i = 0; i <= G; ++i) lb[i] = readlane_i32(lbv, i);
  sg.b = lb[0];
  sg.n = lb[sg.ns] - lb[0];
#pragma unroll
  for (int i = 0; i <= G; ++i) sg.c[i] = (i <= sg.ns ? lb[i] : lb[sg.ns]) - lb[0];
#pragma unroll
  for (int i = 0; i < G; ++i) {
    sg.w[i] = w0 + i;
    sg.dl[i] = readlane_i64(rawv, i) - a.p.now;
    sg.lvl[i] = i < sg.ns ? prio_level(a, w0 + i) : 0;
  }
  if (kFused && ln < sg.ns) {
    const int64_t w = w0 + ln;
    int32_t lo = 0, hi = 0;
#pragma unroll
    for (int i = 0; i < G; ++i)
      if (ln == i) {
        lo = lb[i];
        hi = lb[i + 1];
      }
    if ((hi < lo) | ((w == 0) & (lo != 0)) | ((w == W - 1) & (int64_t(hi) != a.p.N)) |
        (rawv < a.p.now - NALAR_HORIZON_MAX) | (rawv > a.p.now + NALAR_HORIZON_MAX) |
        (a.p.prio != nullptr && a.p.prio[w] > NALAR_PRIORITY_MAX))
      flag_sweep(ctrl, kStInval);
  }
  return sg;
}

// Small workflows: one wave each, no workgroup barrier on the way (fused mode:
// after the instance table is built).  With G > 1 a wave takes G consecutive
// workflows and sweeps them together as one slice of at most wcap futures
// (their DAGs are disjoint, so the rounds run side by side: half-empty waves
// of 32-future workflows become full ones), else one at a time.  Workflows
// larger than a wave's slice (wcap futures) are swept at the end by whole
// workgroups with HBM state.  Each wave folds its slack range and ready count
// into one of the control block's partial slots.
template <int NPTW, bool kFused, int G>
__global__ __launch_bounds__(kWaveBlock) void k_sweep_wave(
    const int32_t* inst_type, const int32_t* inst_speed, const int64_t* inst_load, const int64_t* deadline,
    const int32_t* wf, int64_t N, int32_t W, int32_t M_, SweepArgs a_arg, int wcap_arg) {
  (void)a_arg;
  (void)wcap_arg;
  // scalar arguments (an aggregate is not preloaded); the same fields as WaveHead
  const WaveHead h{inst_type, inst_speed, inst_load, deadline, wf, N, W, M_};
  KernArgWarm warm;
  warm_kernargs_issue(warm);
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ Shared S;
  __shared__ __align__(16) int32_t s_itype[kWaveItabMax];
  __shared__ int s_big[kWavesPerBlock];
  const int M = h.M;
  const int tid = threadIdx.x;
  const int wv = __builtin_amdgcn_readfirstlane(tid / kWave);  // wave-uniform: scalar registers
  const int ln = lane_id();
  const bool wave_itab = kFused && M <= kWave;  // sorted by each wave itself, no barrier
  const bool per_wave = (!kFused && M <= kWaveItabMax) || wave_itab;
  const int64_t gw = int64_t(blockIdx.x) * kWavesPerBlock + wv;
  const int64_t nwaves = int64_t(gridDim.x) * kWavesPerBlock;

  // one round trip, from the preloaded arguments: this wave's first group of
  // workflows (fused) and the instance table; every load is issued before any
  // is used
  int64_t raw0 = 0;
  int32_t it_t = 0, it_sp = 1, spec_before = INT32_MIN, spec_at = INT32_MAX;
  int64_t it_ld = 0, spec_g = 0, spec_lo = 0;
  int32_t off_first = 0, off_last = 0;
  if (kFused) {
    const int ie = wave_itab ? ln : tid;  // the instance this thread loads
    if (ie < M) {
      it_t = h.inst_type[ie];
      it_sp = h.inst_speed[ie];
      it_ld = h.inst_load[ie];
    }
    if (gw * G < h.W) {
      if (ln < G && gw * G + ln < h.W) raw0 = h.deadline[gw * G + ln];
      // bounds that equal workflow sizes would give: lane i <= G guesses the
      // first position of workflow gw*G + i and loads the ids around it
      const int64_t key = gw * G + ln < h.W ? gw * G + ln : int64_t(h.W);
      if (ln <= G) {
        spec_g = (key * h.N) / h.W;
        if (spec_g >= 1) spec_before = h.wf[spec_g - 1];
        if (spec_g < h.N) spec_at = h.wf[spec_g];
      }
      spec_lo = readlane_i64(spec_g, 0);
    }
  }
  const WaveKernArgs* kargs = warm_kernargs_wait(warm);  // the rest, read after the warm-up
  const SweepArgs& a = kargs->a;
  const int wcap = kargs->wcap;
  // one future per lane: the first group's attributes at the guessed
  // bound, in flight with the bound checks instead of after them
  PreAttr pre;
  if (kFused && NPTW == 1 && gw < h.W && spec_lo + ln < h.N) {
    const int64_t v = spec_lo + ln;
    pre.d = a.p.done[v];
    pre.o0 = a.p.dep_off[v];
    pre.o1 = a.p.dep_off[v + 1];
    pre.t = a.p.type[v];
    pre.l = a.p.loc[v];
    pre.e = a.p.est[v];
    pre.wfv = a.p.wf[v];
  }
  // the offsets' first and last entries (checked at the end: every future's
  // own offsets are checked where they are used, so nothing waits for these)
  if (kFused && gw == 0 && ln == 0) {
    off_first = a.p.dep_off[0];
    off_last = a.p.dep_off[a.p.N];
  }
  Ctrl* ctrl = a.ctrl;
  // (fused: nothing ran before this kernel in the pass; otherwise written by
  // earlier kernels only, so a plain load sees it; an uncached load of one
  // word by every wave would queue at the memory controller)
  const uint32_t status = kFused ? 0u : ctrl->status;
  int32_t lb0 = 0;  // lane i <= G: first position of workflow gw*G + i
  if (!kFused && gw * G < a.p.W) group_bounds<G>(a, gw, lb0, raw0);
  ItabStage st;
  st.pending = false;
  st.build = false;
  if (!kFused && per_wave) itab_stage_load(st, a.itab, M, ln);

  const size_t nw = size_t(kWavesPerBlock) * size_t(wcap);
  const size_t itab_one = 32 * size_t(M) + 4 * kTypeDirect;
  unsigned char* sp = smem;
  const ITabLds it = carve_itab(sp + (per_wave ? size_t(wv) * itab_one : 0), M);
  sp += itab_lds_wave(M);
  WaveSlice Wv{};
  Wv.mx = reinterpret_cast<int64_t*>(sp) + size_t(wv) * wcap; sp += 8 * nw;
  Wv.cnt = reinterpret_cast<int32_t*>(sp) + size_t(wv) * wcap; sp += 4 * nw;
  Wv.dn = sp + size_t(wv) * wcap; sp += nw;
  Wv.nr = sp + size_t(wv) * wcap; sp += nw;
  if (NPTW >= kFrontierMinNpt) {
    Wv.est = reinterpret_cast<int64_t*>(sp) + size_t(wv) * wcap; sp += 8 * nw;
    Wv.d01 = reinterpret_cast<uint32_t*>(sp) + size_t(wv) * wcap; sp += 4 * nw;
    Wv.d2 = reinterpret_cast<uint32_t*>(sp) + size_t(wv) * wcap; sp += 4 * nw;
    Wv.q0 = reinterpret_cast<uint16_t*>(sp) + size_t(wv) * wcap; sp += 2 * nw;
    Wv.q1 = reinterpret_cast<uint16_t*>(sp) + size_t(wv) * wcap;
  }
  if (kFused) {
    if ((wave_itab ? ln : tid) < M && ((it_t < 0) | (it_sp < 1) | (it_ld < 0) | (it_ld > NALAR_LOAD_MAX)))
      flag_sweep(ctrl, kStInval);
    if (gw * G < a.p.W && ln <= G) {
      // workflow bounds: the speculative guess, else a search (lanes 0 .. G)
      const int64_t key = gw * G + ln < a.p.W ? gw * G + ln : a.p.W;
      const bool ok = (spec_g == 0 || int64_t(spec_before) < key) &&
                      (spec_g >= a.p.N || int64_t(spec_at) >= key);
      lb0 = ok ? int32_t(spec_g) : int32_t(lower_bound_from(a.p.wf, a.p.N, key, spec_g));
    }
    if (wave_itab) {
      st.type[0] = it_t;
      st.speed[0] = it_sp;
      st.load[0] = it_ld;
      st.pending = true;
      st.build = true;
    } else {
      build_itab_block(it, M, it_t, it_sp, it_ld, s_itype);
    }
  } else {
    if (!per_wave) {  // one shared copy (every thread reaches this barrier)
      for (int i = tid; i < M; i += kWaveBlock) {
        it.load[i] = a.itab.load[i];
        it.inv[i] = a.itab.inv_speed[i];
        it.type[i] = a.itab.type[i];
        it.idx[i] = a.itab.idx[i];
        it.speed[i] = a.itab.speed[i];
        it.pos[i] = a.itab.pos_of[i];
      }
      for (int t = tid; t < kTypeDirect; t += kWaveBlock) it.run[t] = a.itab.run[t];
      __syncthreads();
    }
  }
  // the validation status read above cannot change during this kernel (the
  // sweep reports into its own word), so every wave of every workgroup
  // leaves together
  if (status != 0) {
    clear_for_next_pass<kFused>(a);
    return;
  }

  const Layout L{a.node_of_pos, a.pos_of_node, a.p.N};
  Acc acc;
  bool big = false;
  uint32_t lmask = 0;  // priority levels of the wave's workflows
  for (int64_t pw = gw; pw * G < a.p.W; pw += nwaves) {
    int32_t lbv = lb0;
    int64_t rawv = raw0;
    if (pw != gw) group_bounds<G>(a, pw, lbv, rawv);
    Seg<G> sg = make_seg<G, kFused>(a, pw, lbv, rawv, ctrl);
    bool any = false, gbig = false;  // a workflow of the group to sweep here / in HBM
#pragma unroll
    for (int i = 0; i < G; ++i) {
      const int ni = sg.c[i + 1] - sg.c[i];
      if (i < sg.ns && ni > 0) {
        lmask |= level_bit(sg.lvl[i]);
        if (ni > wcap || a.force_global) gbig = true;
        else any = true;
      }
    }
    big |= gbig;
    if (!any) continue;
    const bool use_pre = pw == gw && sg.b == spec_lo;
    if (!gbig && sg.n <= wcap) {  // the whole group in one slice
      sweep_wave<NPTW, kFused, G>(a, L, it, Wv, sg, acc, st, pre, use_pre);
      continue;
    }
    // one workflow at a time (a group too large for one slice)
#pragma unroll
    for (int i = 0; i < G; ++i) {
      const int ni = sg.c[i + 1] - sg.c[i];
      if (i >= sg.ns || ni <= 0 || ni > wcap || a.force_global) continue;
      Seg<G> one = sg;
      one.b = sg.b + sg.c[i];
      one.n = ni;
      one.ns = 1;
      one.c[0] = 0;
      one.c[1] = ni;
      one.w[0] = sg.w[i];
      one.dl[0] = sg.dl[i];
      one.lvl[0] = sg.lvl[i];
      sweep_wave<NPTW, kFused, G>(a, L, it, Wv, one, acc, st, pre, use_pre && i == 0);
    }
  }
  if (ln == 0) s_big[wv] = big ? 1 : 0;
  __syncthreads();
  if (s_big[0] | s_big[1] | s_big[2] | s_big[3]) {  // the workgroup's large workflows (HBM state)
    itab_stage_store(st, it, M, ln);
    __syncthreads();
    for (int64_t base = int64_t(blockIdx.x) * kWavesPerBlock * G; base < a.p.W; base += nwaves * G) {
      for (int i = 0; i < kWavesPerBlock * G; ++i) {
        const int64_t w = base + i;
        if (w >= a.p.W) break;
        int64_t b;
        int n;
        wf_bounds(a, w, b, n);
        if (n <= 0 || (n <= wcap && !a.force_global)) continue;
        const int lvl = prio_level(a, w);
        lmask |= level_bit(lvl);
        sweep_hbm<kWaveBlock, kFused, true>(a, L, it, S, int(w), b, n, a.p.deadline[w] - a.p.now, lvl, acc,
                                            nullptr);
      }
    }
  }

  if (kFused && gw == 0 && ln == 0 && (off_first != 0 || int64_t(off_last) != a.p.E))
    flag_sweep(ctrl, kStInval);
  const int64_t mn = wave_min_i64(acc.tmin);
  const int64_t mxv = wave_max_i64(acc.tmax);
  const int64_t rd = wave_sum_i64(acc.tready);
  if (ln == 0 && rd > 0) {
    const int slot = int(gw & (kParts - 1));
    __hip_atomic_fetch_min(&ctrl->part_min[slot], mn, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_fetch_max(&ctrl->part_max[slot], mxv, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    add_agent(&ctrl->part_cnt[slot], rd);
    if (a.p.prio)
      __hip_atomic_fetch_or(&ctrl->part_lvl[slot], lmask, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  clear_for_next_pass<kFused>(a);
}

constexpr int kBlockT = 1024;
constexpr int kBlockNpt = 5;

}  // namespace

SweepShape plan_sweep(int64_t N, int64_t W, int64_t M, int device_cus, size_t lds_limit) {
  const int64_t avg = W > 0 ? (N + W - 1) / W : 0;
  const size_t itab = 32 * size_t(M) + 4 * kTypeDirect;
  SweepShape s;
  if (avg <= kWaveCap) {  // one wave per workflow (or pair of workflows)
    int64_t wcap = 64;       // room for workflows up to twice the average size
    while (wcap < 2 * avg && wcap < kWaveCap) wcap *= 2;
    s.threads = kWaveBlock;
    s.npt = int(wcap / kWave);
    s.lds_cap = int(wcap);
    const size_t per = kWaveSliceBytesPerFuture +
                       (wcap / kWave >= kFrontierMinNpt ? kWaveFrontierBytesPerFuture : 0);
    s.lds_bytes = itab_lds_wave(M) + per * size_t(kWavesPerBlock) * size_t(wcap) + 16;
    s.wave_path = 1;
    // workflows of up to 32 futures on average: two per wave, side by side
    s.group = (wcap == kWave && 2 * avg <= kWave) ? 2 : 1;
    int64_t blocks = (W + int64_t(kWavesPerBlock) * s.group - 1) / (int64_t(kWavesPerBlock) * s.group);
    const int64_t most = int64_t(device_cus) * 8;
    if (blocks > most) blocks = most;
    s.blocks = int(blocks < 1 ? 1 : blocks);
    return s;
  }
  s.threads = kBlockT;
  s.npt = kBlockNpt;
  // and the undominated ends, the splitters and two bin counter arrays
  const size_t itab_b = itab + 4 * kTypeDirect + 16 * size_t(kBinMax);
  const size_t avail = lds_limit > kStaticLdsReserve + itab_b ? lds_limit - kStaticLdsReserve - itab_b : 0;
  int64_t cap = int64_t(avail / 14);
  if (cap > int64_t(kBlockT) * kBlockNpt) cap = int64_t(kBlockT) * kBlockNpt;
  s.lds_cap = int(cap);
  s.lds_bytes = itab_b + 14 * size_t(cap) + 16;
  s.wave_path = 0;
  int64_t blocks = int64_t(device_cus) * 2;
  if (blocks > W) blocks = W;
  s.blocks = int(blocks < 1 ? 1 : blocks);
  return s;
}

bool sweep_can_fuse(const SweepShape& shape, int64_t M, bool contiguous) {
  return contiguous && shape.wave_path && M <= kWaveItabMax;
}

hipError_t prepare_sweep_kernels(size_t lds_limit) {
  const size_t dyn = lds_limit > kStaticLdsReserve ? lds_limit - kStaticLdsReserve : 0;
  hipError_t e = hipSuccess;
  for (const void* k : {reinterpret_cast<const void*>(&k_sweep<kBlockT, kBlockNpt>),reinterpret_cast<const void*>(&k_sweep_wave<1, false, 1>),
                        reinterpret_cast<const void*>(&k_sweep_wave<1, false, 2>),
                        reinterpret_cast<const void*>(&k_sweep_wave<2, false, 1>),
                        reinterpret_cast<const void*>(&k_sweep_wave<4, false, 1>),
                        reinterpret_cast<const void*>(&k_sweep_wave<8, false, 1>),
                        reinterpret_cast<const void*>(&k_sweep_wave<1, true, 1>),
                        reinterpret_cast<const void*>(&k_sweep_wave<1, true, 2>),
                        reinterpret_cast<const void*>(&k_sweep_wave<2, true, 1>),
                        reinterpret_cast<const void*>(&k_sweep_wave<4, true, 1>),
                        reinterpret_cast<const void*>(&k_sweep_wave<8, true, 1>)}) {
    e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, int(dyn));
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// The wave kernel with its preloaded leading arguments taken from a.
template <int NPTW, bool kFused, int G = 1>
void launch_wave(hipStream_t s, dim3 g, dim3 t, size_t lds, const SweepArgs& a, int cap) {
  hipLaunchKernelGGL((k_sweep_wave<NPTW, kFused, G>), g, t, lds, s, a.p.inst_type, a.p.inst_speed,
                     a.p.inst_load, a.p.deadline, a.p.wf, a.p.N, int32_t(a.p.W), int32_t(a.p.M), a, cap);
}

hipError_t launch_sweep(hipStream_t s, const SweepArgs& a, const BlockSweepArgs& ba, const SweepShape& sh) {
  if (sh.threads == kWaveBlock) {
    // futures per lane = slice capacity / 64 (a power of two up to kWaveNpt)
    const dim3 g(sh.blocks), t(kWaveBlock);
    const size_t lds = sh.lds_bytes;
    const int cap = sh.lds_cap;
    if (a.fused) {
      switch (sh.npt) {
        case 1:
          if (sh.group == 2) launch_wave<1, true, 2>(s, g, t, lds, a, cap);
          else launch_wave<1, true>(s, g, t, lds, a, cap);
          break;
        case 2: launch_wave<2, true>(s, g, t, lds, a, cap); break;
        case 4: launch_wave<4, true>(s, g, t, lds, a, cap); break;
        default: launch_wave<kWaveNpt, true>(s, g, t, lds, a, cap); break;
      }
    } else {
      switch (sh.npt) {
        case 1:
          if (sh.group == 2) launch_wave<1, false, 2>(s, g, t, lds, a, cap);
          else launch_wave<1, false>(s, g, t, lds, a, cap);
          break;
        case 2: launch_wave<2, false>(s, g, t, lds, a, cap); break;
        case 4: launch_wave<4, false>(s, g, t, lds, a, cap); break;
        default: launch_wave<kWaveNpt, false>(s, g, t, lds, a, cap); break;
      }
    }
  } else {
    hipLaunchKernelGGL((k_sweep<kBlockT, kBlockNpt>), dim3(sh.blocks), dim3(kBlockT), sh.lds_bytes, s,
                       a, sh.lds_cap, ba);
  }
  return hipGetLastError();
}

}  // namespace nalar
