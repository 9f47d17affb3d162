// Device-side helpers shared by the policy-pass kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "nalar_policy.h"

namespace nalar {

// Status word bits (ORed by any kernel that finds a problem).
constexpr uint32_t kStInval = 1u;
constexpr uint32_t kStCycle = 2u;
constexpr uint32_t kStRange = 4u;
constexpr uint32_t kStIncomplete = 8u;  // incremental pass: work left after the last round (fall back)

constexpr int kWave = 64;
constexpr int kRadixBits = 8;
constexpr int kRadixBuckets = 1 << kRadixBits;
constexpr int kMaxKeyPasses = 8;     // 64-bit keys
constexpr int kMaxSortPasses = 9;    // key passes, then one priority-level pass
constexpr int kMaxGroupPasses = 4;   // workflow ids < 2^30
constexpr int kSortThreads = 256;
constexpr int kSortItems = 16;
constexpr int kSortTile = kSortThreads * kSortItems;

// Decoupled look-back words: [63:40] epoch, [39:38] flag, [37:0] value.
constexpr int kLbValueBits = 38;
constexpr uint64_t kLbValueMask = (uint64_t(1) << kLbValueBits) - 1;
constexpr uint64_t kLbAgg = uint64_t(1) << 38;    // aggregate of this tile only
constexpr uint64_t kLbInc = uint64_t(2) << 38;    // inclusive prefix
constexpr uint32_t kEpochMask = (1u << 24) - 1;

__host__ __device__ inline uint64_t lb_pack(uint32_t epoch, uint64_t flag, uint64_t value) {
  return (uint64_t(epoch & kEpochMask) << 40) | flag | (value & kLbValueMask);
}

// Per-pass control block in device memory.  Two of them alternate between
// passes: the last kernel of a pass resets the block the next pass will use.
// The sweep folds each workgroup's slack range and ready count into one of
// kParts slots (spreading the atomics over many addresses); the sort reduces
// the slots with one wave.  With priority levels the slots also hold a mask of
// the levels seen.
constexpr int kParts = 64;

struct Ctrl {
  uint32_t status;               // problems found before the sweep (validation)
  uint32_t status_sweep;         // problems found by the sweep (cycles, ranges)
  uint32_t sort_npass;           // digit passes the slack sort runs
  uint32_t bucket_overflow;      // a bucket of the bucketed sort overflowed
  uint32_t level_mask;           // priority levels seen (the next pass's bucket hint)
  uint32_t sort_level_pass;      // the last digit pass orders by priority level
  int64_t n_ready;
  int64_t slack_min;             // key range of the ready futures (all keys lie inside)
  int64_t slack_max;
  int64_t hint_min;              // the range the host plans the next buckets from
  int64_t hint_max;              //   (the key range)
  uint64_t plog_fill;            // entries of the push log taken by the ordered HBM sweep
  uint32_t tile_ticket[16];      // per radix pass: [0,9) slack sort, [9,13) grouping
  int64_t part_min[kParts];
  int64_t part_max[kParts];
  int64_t part_cnt[kParts];
  uint32_t part_lvl[kParts];
  uint32_t part_crowd[kParts];   // fullest bucket seen by the large-bucket totals kernel
  uint32_t ghist_slack[kMaxSortPasses * kRadixBuckets];
  uint32_t ghist_group[kMaxGroupPasses * kRadixBuckets];
};

// Slack-sort digit passes launched before the host looks at the status; a
// wider slack range reports kStatusContinue and the host launches the rest.
constexpr int kSortLaunched = 4;
constexpr uint32_t kStatusContinue = 0x40000000u;

// Bucketed slack sort.  With the slack range of the previous pass as a hint,
// the sweep drops each ready future into one of nb buckets of increasing slack
// (kBucketCap slots each, unordered inside a bucket); one kernel then orders
// every bucket and writes it at its offset.  A bucket that overflows reports
// kStatusTiled and the host runs the tiled radix sort instead.
constexpr int kBucketCap = 64;            // slots per bucket
constexpr int kBucketGroup = 16;          // buckets per workgroup of the small bucket kernel
constexpr int kBucketMin = 64;            // bucket counts are powers of two in
constexpr int kBucketMax = 1 << 19;       //   [kBucketMin, kBucketMax]
constexpr int64_t kBucketMaxReady = int64_t(1) << 22;  // larger ready sets use the tiled sort
constexpr int64_t kBucketDense = 131072;  // up to here about 2 futures per bucket, then 4
// From kBucketLbMin buckets on, a first kernel totals each group of
// kBucketLbGroup buckets and the sort kernel (one workgroup per group) adds up
// the totals of earlier groups instead of every earlier bucket counter.
constexpr int kBucketLbMin = 16384;
constexpr int kBucketLbGroup = 256;
constexpr int kBucketLbGroups = kBucketMax / kBucketLbGroup;
static_assert(kBucketLbGroup == 4 * kWave, "one uint4 of counters per lane and group");
// A bucket with more futures than this after a large-bucket sort asks for a
// denser plan next time (the sort still succeeded), up to sixteen times the
// base bucket count.
constexpr uint32_t kBucketCrowded = 8;
static_assert(kBucketLbMin % kBucketLbGroup == 0, "whole groups");
constexpr uint32_t kStatusTiled = 0x20000000u;

// Partition sort of large ready sets (the block sweep): the previous pass's
// key quantiles split the keys into nb bins (a power of two with at most
// kBinTarget ready futures each on average); every workgroup of the sweep
// counts its ready futures per bin in LDS, claims one segment of each bin with
// one atomic, and writes them there; k_bin_sort then orders each bin in LDS
// (k_bin_sort_big the bins of more than kBinCap futures; more than the bins'
// capacity, at most kBinAlloc, is an overflow, like a full bucket) and writes
// the outputs at the bin's offset.
constexpr int64_t kBinMinReady = 65536;   // smaller ready sets keep the buckets
constexpr int kBinTarget = 1024;          // futures per bin on average
constexpr int kBinCap = 2048;             // records per bin in one workgroup's LDS (k_bin_sort)
constexpr int kBinAlloc = 8192;           // records per bin in HBM (more than kBinCap: k_bin_sort_big)
constexpr int kBinMin = 64;               // bins: a power of two in [kBinMin, kBinMax]
constexpr int kBinMax = 2048;
// bins for a ready count (the same rule on the host and on the device)
__host__ __device__ inline int bins_for(int64_t R) {
  int nb = kBinMin;
  while (nb < kBinMax && int64_t(nb) * kBinTarget < R) nb *= 2;
  return nb;
}
__host__ __device__ inline int bin_cap_for(int64_t R, int nb) {
  const int64_t c = 8 * ((R + nb - 1) / nb) + 256;
  return int(c < kBinAlloc ? c : kBinAlloc);
}

struct BucketSlot {
  int64_t key;      // the order key: the slack, or -rem / rem under NALAR_ORDER_LPT / _SRTF
  int64_t cost;
  int32_t pos;
  int32_t route;    // slot_pack(route, priority level)
};
static_assert(sizeof(BucketSlot) == 24 && offsetof(BucketSlot, cost) == 8 && offsetof(BucketSlot, pos) == 16 &&
                  offsetof(BucketSlot, route) == 20,
              "the sweep writes a slot as three 8-byte words");

// A slot's route field holds the route (-1 .. 1023) in its low 16 bits and
// the future's priority level above them, so that a bucket holding futures of
// several levels ranks them by (level descending, key, position).
__host__ __device__ inline int32_t slot_pack(int32_t route, int lvl) {
  return int32_t((uint32_t(route) & 0xFFFFu) | (uint32_t(lvl) << 16));
}
__host__ __device__ inline int32_t slot_route(int32_t packed) { return int32_t(int16_t(packed & 0xFFFF)); }
__host__ __device__ inline int slot_level(int32_t packed) { return int((uint32_t(packed) >> 16) & 0xFFu); }

// Written by the last kernel of a pass into pinned host memory.
struct HostStatus {
  uint32_t status;
  uint32_t key_bits;   // significant bits of the slack range
  int64_t n_ready;
  int64_t slack_min;   // range of this pass (the next pass's bucket hint; with
  int64_t slack_max;   //   priority levels the range of the key within its level)
  uint32_t aux_status; // status bits of the load-aware routing kernel
  uint32_t level_mask; // priority levels of this pass (bit l: level l; with levels only)
  uint32_t max_bucket; // futures in the fullest bucket (large-bucket sort only, else 0)
  uint32_t split_nb;   // bins the splitters written by this pass are for (0: none)
};

// Resets a control block for a later pass (run by one workgroup).
__device__ inline void reset_ctrl(Ctrl* c) {
  const int tid = threadIdx.x;
  if (tid == 0) {
    c->status = 0;
    c->status_sweep = 0;
    c->sort_npass = 0;
    c->sort_level_pass = 0;
    c->bucket_overflow = 0;
    c->n_ready = 0;
    c->slack_min = INT64_MAX;
    c->slack_max = INT64_MIN;
    c->plog_fill = 0;
  }
  for (int i = tid; i < 16; i += blockDim.x) c->tile_ticket[i] = 0;
  for (int i = tid; i < kParts; i += blockDim.x) {
    c->part_min[i] = INT64_MAX;
    c->part_max[i] = INT64_MIN;
    c->part_cnt[i] = 0;
    c->part_lvl[i] = 0;
    c->part_crowd[i] = 0;
  }
  for (int i = tid; i < kMaxSortPasses * kRadixBuckets; i += blockDim.x) c->ghist_slack[i] = 0;
  for (int i = tid; i < kMaxGroupPasses * kRadixBuckets; i += blockDim.x) c->ghist_group[i] = 0;
}

// The same reset spread over a grid: thread gi of gstride writes every
// gstride-th word (gi = blockIdx.x * blockDim.x + threadIdx.x).
__device__ inline void reset_ctrl_spread(Ctrl* c, int64_t gi, int64_t gstride) {
  if (gi == 0) {
    c->status = 0;
    c->status_sweep = 0;
    c->sort_npass = 0;
    c->sort_level_pass = 0;
    c->bucket_overflow = 0;
    c->n_ready = 0;
    c->slack_min = INT64_MAX;
    c->slack_max = INT64_MIN;
    c->plog_fill = 0;
  }
  for (int64_t i = gi; i < 16; i += gstride) c->tile_ticket[i] = 0;
  for (int64_t i = gi; i < kParts; i += gstride) {
    c->part_min[i] = INT64_MAX;
    c->part_max[i] = INT64_MIN;
    c->part_cnt[i] = 0;
    c->part_lvl[i] = 0;
    c->part_crowd[i] = 0;
  }
  for (int64_t i = gi; i < kMaxSortPasses * kRadixBuckets; i += gstride) c->ghist_slack[i] = 0;
  for (int64_t i = gi; i < kMaxGroupPasses * kRadixBuckets; i += gstride) c->ghist_group[i] = 0;
}

// Instance table sorted by (type, original index), plus the sorted position of
// every original index (for the instance that holds a future's state) and,
// for types below kTypeDirect, the run of sorted positions holding that type.
constexpr int kTypeDirect = 64;

struct ITab {
  int64_t* load;      // [M]
  double* inv_speed;  // [M] 1.0 / speed
  int32_t* type;      // [M]
  int32_t* idx;       // [M] original index
  int32_t* speed;     // [M]
  int32_t* pos_of;    // [M] sorted position of original index i
  uint32_t* run;      // [kTypeDirect] first | end << 16 (0: no instance)
  uint32_t* prun;     // [kTypeDirect] end of the type's undominated instances,
                      //   which open its run (see route_future)
};

// ----------------------------------------------------------------- wave ops

__device__ inline int lane_id() { return __lane_id(); }

__device__ inline uint64_t ballot(bool p) { return __ballot(p); }

__device__ inline uint32_t lanes_below(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi(uint32_t(m >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(m), 0u));
}

__device__ inline uint64_t lanemask_lt() {
  const int l = lane_id();
  return l == 0 ? 0ull : (~0ull >> (64 - l));
}

__device__ inline int readlane_i32(int x, int lane) { return __builtin_amdgcn_readlane(x, lane); }

// Whole-wave reductions (all 64 lanes active): a butterfly inside each row of
// 16 lanes by DPP (quad swaps, then row rotations by 4 and 8), then the four
// row results through scalar registers.  No LDS traffic.
template <int kCtrl>
__device__ inline int64_t dpp_i64(int64_t x) {
  const int lo = __builtin_amdgcn_update_dpp(0, int(uint32_t(uint64_t(x))), kCtrl, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp(0, int(uint32_t(uint64_t(x) >> 32)), kCtrl, 0xF, 0xF, false);
  return int64_t((uint64_t(uint32_t(hi)) << 32) | uint32_t(lo));
}

__device__ inline int64_t readlane_i64(int64_t x, int lane) {
  const int lo = __builtin_amdgcn_readlane(int(uint32_t(uint64_t(x))), lane);
  const int hi = __builtin_amdgcn_readlane(int(uint32_t(uint64_t(x) >> 32)), lane);
  return int64_t((uint64_t(uint32_t(hi)) << 32) | uint32_t(lo));
}

constexpr int kDppXor1 = 0xB1;   // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;   // quad_perm [2,3,0,1]
constexpr int kDppRor4 = 0x124;  // row_ror:4
constexpr int kDppRor8 = 0x128;  // row_ror:8

template <typename Op>
__device__ inline int64_t wave_reduce_i64(int64_t x, Op op) {
  x = op(x, dpp_i64<kDppXor1>(x));
  x = op(x, dpp_i64<kDppXor2>(x));
  x = op(x, dpp_i64<kDppRor4>(x));
  x = op(x, dpp_i64<kDppRor8>(x));
  const int64_t r01 = op(readlane_i64(x, 0), readlane_i64(x, 16));
  const int64_t r23 = op(readlane_i64(x, 32), readlane_i64(x, 48));
  return op(r01, r23);
}

__device__ inline int64_t wave_max_i64(int64_t x) {
  return wave_reduce_i64(x, [](int64_t u, int64_t v) { return u > v ? u : v; });
}

__device__ inline int64_t wave_min_i64(int64_t x) {
  return wave_reduce_i64(x, [](int64_t u, int64_t v) { return u < v ? u : v; });
}

__device__ inline int64_t wave_sum_i64(int64_t x) {
  return wave_reduce_i64(x, [](int64_t u, int64_t v) { return u + v; });
}

__device__ inline uint32_t wave_or_u32(uint32_t x) {
  return uint32_t(wave_reduce_i64(int64_t(x), [](int64_t u, int64_t v) { return u | v; }));
}

// Inclusive scan over the wave (all 64 lanes active).
__device__ inline uint32_t wave_incl_scan_u32(uint32_t x) {
  const int l = lane_id();
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    uint32_t y = __shfl_up(x, d, kWave);
    if (l >= d) x += y;
  }
  return x;
}

// ----------------------------------------------------------------- atomics

template <typename T>
__device__ inline T ld_relaxed_agent(const T* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <typename T>
__device__ inline void st_relaxed_agent(T* p, T v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <typename T>
__device__ inline T ld_wg(const T* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
template <typename T>
__device__ inline void st_wg(T* p, T v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
template <typename T>
__device__ inline T add_wg(T* p, T v) {
  return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
template <typename T>
__device__ inline T max_wg(T* p, T v) {
  return __hip_atomic_fetch_max(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
template <typename T>
__device__ inline T add_agent(T* p, T v) {
  return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ inline void flag_status(Ctrl* c, uint32_t bits) {
  __hip_atomic_fetch_or(&c->status, bits, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The sweep reports into a word of its own, so that the status it reads at its
// start (validation) cannot change while it runs.
__device__ inline void flag_sweep(Ctrl* c, uint32_t bits) {
  __hip_atomic_fetch_or(&c->status_sweep, bits, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Exclusive prefix over earlier tiles by decoupled look-back.  The caller has
// already published its own aggregate.  Every earlier tile was claimed (by
// ticket) before the caller's, by a workgroup that publishes its aggregate
// without waiting on anything, so every spin ends.  The predecessors are read a
// window of kLbWindow at a time (independent loads), so walking back over t
// tiles costs about t / kLbWindow load round trips instead of t.
constexpr int kLbWindow = 16;

__device__ inline uint64_t lookback_exclusive(const uint64_t* words, int64_t slot, int64_t stride,
                                              uint32_t epoch) {
  uint64_t excl = 0;
  const uint64_t want = uint64_t(epoch & kEpochMask);
  int64_t t = slot - 1;
  while (t >= 0) {
    uint64_t w[kLbWindow];
#pragma unroll
    for (int i = 0; i < kLbWindow; ++i) w[i] = (t - i >= 0) ? ld_relaxed_agent(words + (t - i) * stride) : 0;
    bool found = false;
#pragma unroll
    for (int i = 0; i < kLbWindow; ++i) {
      if (found || t - i < 0) continue;
      while ((w[i] >> 40) != want || (w[i] & (kLbAgg | kLbInc)) == 0)
        w[i] = ld_relaxed_agent(words + (t - i) * stride);
      excl += w[i] & kLbValueMask;
      found = (w[i] & kLbInc) != 0;
    }
    if (found) break;
    t -= kLbWindow;
  }
  return excl;
}

// First index i in [0, n] with a[i] >= key for non-decreasing a, found by
// galloping from `guess`.  a[guess - 1] and a[guess] are read together, so an
// exact guess (equal-sized workflows) costs one round trip.
__device__ inline int64_t lower_bound_from(const int32_t* a, int64_t n, int64_t key, int64_t guess) {
  guess = guess < 0 ? 0 : (guess > n ? n : guess);
  const int32_t before = guess >= 1 && guess - 1 < n ? a[guess - 1] : INT32_MIN;
  const int32_t at = guess < n ? a[guess] : INT32_MAX;
  const bool ok_before = guess == 0 || int64_t(before) < key;
  const bool ok_at = guess >= n || int64_t(at) >= key;
  if (ok_before && ok_at) return guess;
  int64_t lo, hi;
  if (!ok_before) {  // answer below guess
    hi = guess - 1;
    int64_t step = 1;
    lo = hi - 1;
    while (lo >= 0 && int64_t(a[lo]) >= key) {
      hi = lo;
      lo = hi - step;
      step <<= 1;
    }
    lo = lo < 0 ? 0 : lo + 1;
  } else {           // answer above guess
    lo = guess + 1;
    hi = lo;
    int64_t step = 1;
    while (hi < n && int64_t(a[hi]) < key) {
      lo = hi + 1;
      hi = lo + step;
      if (hi > n) hi = n;
      step <<= 1;
    }
  }
  while (lo < hi) {
    const int64_t mid = (lo + hi) >> 1;
    if (int64_t(a[mid]) < key) lo = mid + 1; else hi = mid;
  }
  return lo;
}

// ----------------------------------------------------------------- routing

// floor(A / d) for 0 <= A < 2^53, 1 <= d < 2^31, exact.  The double product
// A * RN(1/d) is within 0.25 of A/d (relative error <= 2^-52, A < 2^50 here),
// so its floor is off by at most one; the remainder, computed exactly by an
// FMA (it is an integer below 2^33 in magnitude), corrects it.
__host__ __device__ inline int64_t floordiv_exact(double a, int32_t d, double inv_d) {
  double q = floor(a * inv_d);
  double r = fma(-q, double(d), a);
  q += (r < 0.0) ? -1.0 : ((r >= double(d)) ? 1.0 : 0.0);
  return int64_t(q);
}

// Route one ready future against the sorted instance table (in LDS).
// Candidates are the instances of type t, visited in ascending original index.
// The migration penalty applies to every candidate except the one holding the
// future's state, so the best candidate is either the unpenalised holder or the
// best candidate overall plus the penalty (ties broken by index).  With
// `stateful`, a future whose state lives on an instance of its own type runs
// there, at that instance's cost and with no other candidate.
//
// With s_prun, the run of a small type opens with its undominated instances
// (ascending index) and only those are scanned: instance j of the type is
// dominated when another instance i of it has load_i <= load_j and speed_i >=
// speed_j, with i < j or load_i < load_j.  Then for every estimate i's service
// time is at most j's, so i's cost is at most j's and i wins every tie on
// index, or its cost is strictly lower: j can never be the lexicographic
// minimum of (cost, index), and leaving it out changes no result.
__host__ __device__ inline void route_future(int32_t t, int64_t est, int32_t loc, int32_t M, int64_t mig,
                                    const int32_t* s_type, const int32_t* s_idx,
                                    const int64_t* s_load, const int32_t* s_speed,
                                    const double* s_inv, const int32_t* s_pos,
                                    const uint32_t* s_run, bool stateful, int32_t& route,
                                    int64_t& cost, const uint32_t* s_prun = nullptr) {
  if (stateful && loc >= 0) {
    const int pl = s_pos[loc];
    if (s_type[pl] == t) {
      route = loc;
      cost = s_load[pl] + floordiv_exact(double(est * 1000), s_speed[pl], s_inv[pl]);
      return;
    }
  }
  int lo, hi;
  if (uint32_t(t) < uint32_t(kTypeDirect)) {
    const uint32_t rn = s_run[t];
    lo = int(rn & 0xFFFFu);
    hi = s_prun ? int(s_prun[t]) : int(rn >> 16);
  } else {
    lo = 0;
    hi = M;
    while (lo < hi) {  // first position with type >= t
      int mid = (lo + hi) >> 1;
      if (s_type[mid] < t) lo = mid + 1; else hi = mid;
    }
    hi = lo;
    while (hi < M && s_type[hi] == t) ++hi;
  }
  const double a = double(est * 1000);
  int64_t best = INT64_MAX;
  int bj = -1;
  // candidates four at a time (independent LDS reads), compared in index order
  for (int j0 = lo; j0 < hi; j0 += 4) {
    int64_t c[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int j = j0 + u < hi ? j0 + u : j0;
      c[u] = s_load[j] + floordiv_exact(a, s_speed[j], s_inv[j]);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (j0 + u < hi && c[u] < best) { best = c[u]; bj = j0 + u; }
  }
  if (bj < 0) { route = -1; cost = INT64_MAX; return; }
  const int32_t bidx = s_idx[bj];
  if (loc >= 0) {
    const int pl = s_pos[loc];
    if (s_type[pl] == t) {
      const int64_t cl = s_load[pl] + floordiv_exact(a, s_speed[pl], s_inv[pl]);
      const int64_t cm = best + mig;
      if (cl < cm || (cl == cm && loc < bidx)) { route = loc; cost = cl; }
      else { route = bidx; cost = cm; }
    } else {
      route = bidx;
      cost = best + mig;
    }
  } else {
    route = bidx;
    cost = best;
  }
}

}  // namespace nalar
