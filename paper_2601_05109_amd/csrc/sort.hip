// The order of the ready futures, and the grouping of ids by workflow.
//
// Bucketed sort (the usual pass): the sweep has dropped every ready future
// into one of nb buckets of its order key, planned from the previous pass's
// range; k_bucket_sort (or k_bucket_totals + k_bucket_sort_lb for many
// buckets) finds each bucket's offset, ranks the futures inside a bucket by
// (key, position) and writes order, slack, route and cost in place.
//
// Tiled sort (first pass, bucket overflow, very large ready sets):
// stable LSD radix sort of (key, payload) pairs.  Each 8-bit digit pass is one
// launch that ranks tiles of 4096 items in LDS and finds their global offsets
// by decoupled look-back over earlier tiles ("onesweep": one upfront histogram
// of every digit instead of a scan per pass).  Passes beyond what the key
// range needs return at once; for the slack sort only kSortLaunched passes
// (32-bit key ranges, the usual case) are launched up front.
//
// Two sorts use it:
//  * the slack sort (set_priority, Table 2): key = slack - min slack, payload =
//    position of the ready future.  Its first pass reads the futures staged by
//    position and skips positions that are not ready, so it also compacts them;
//    the passes are stable, so equal slacks keep (wf, id) order, which makes the
//    order exactly ascending (slack, wf, id).  With priority levels of more
//    than one value, one more pass follows the key passes, whose digit is
//    15 - level (read from the staged ready byte of the item's position), so
//    that a higher level comes first and each level keeps its key order.  Its
//    last pass gathers each ready future's id, slack, route and cost straight
//    into the caller's arrays;
//  * grouping futures by workflow when the caller's ids are not grouped:
//    key = wf, payload = id; it ends by recording each node's position and
//    each workflow's first position.
//
// Tile layout: 256 threads (4 waves), 16 items per thread, wave w owning a
// contiguous run of 1024 items with item j of lane l at offset j*64 + l, so
// loads are coalesced and the in-wave ranking visits items in input order.
#include "internal.hpp"

namespace nalar {

namespace {

constexpr int kWavesPerTile = kSortThreads / kWave;

template <typename K>
struct TileSmem {
  uint32_t whist[kWavesPerTile][kRadixBuckets];
  uint32_t tprefix[kRadixBuckets];
  uint64_t gstart[kRadixBuckets];
  uint32_t tmp[kWavesPerTile];
  uint32_t intile;
  uint32_t tile;
  K key[kSortTile];
  uint32_t pay[kSortTile];
};

// Where the first pass reads its items.
struct FirstSource {
  int mode;                 // kSrcStaged or kSrcWf
  const int64_t* stg_slack;
  const uint8_t* stg_ready;
  const int32_t* wf;
  int64_t span;             // positions scanned
  int64_t smin;             // staged: key = slack - smin
};

__device__ inline bool first_valid(const FirstSource& f, int64_t i) {
  return i < f.span && (f.mode != kSrcStaged || f.stg_ready[i] != 0);
}

template <typename K>
__device__ inline K first_key(const FirstSource& f, int64_t i) {
  if (f.mode == kSrcStaged) return K(uint64_t(f.stg_slack[i] - f.smin));
  return K(uint32_t(f.wf[i]));
}

// Exclusive scan of one value per thread over the 256-thread block.
__device__ inline uint32_t block_excl_scan(uint32_t x, uint32_t* s_tmp) {
  const int w = threadIdx.x / kWave;
  const uint32_t inc = wave_incl_scan_u32(x);
  if (lane_id() == kWave - 1) s_tmp[w] = inc;
  __syncthreads();
  uint32_t off = 0;
  for (int i = 0; i < w; ++i) off += s_tmp[i];
  __syncthreads();
  return off + inc - x;
}

// Digit histograms (the npass key digits, and the level digit in row
// level_row when it is not negative) of the first pass's items, added into
// ghist.  H is a workgroup-private [kMaxSortPasses][256] array.  Each thread
// takes kHistItems items per step, all loaded before any is used, so a
// workgroup covers many items per memory round trip and few workgroups (few
// flushes of 256 x npass global adds) cover the span.
constexpr int kHistItems = 8;

template <typename K>
__device__ void histogram(const FirstSource& f, int npass, int level_row, uint32_t (*H)[kRadixBuckets],
                          uint32_t* ghist) {
  for (int i = threadIdx.x; i < kMaxSortPasses * kRadixBuckets; i += kSortThreads) (&H[0][0])[i] = 0;
  __syncthreads();
  const int64_t stride = int64_t(gridDim.x) * kSortThreads * kHistItems;
  for (int64_t base = int64_t(blockIdx.x) * kSortThreads * kHistItems; base < f.span; base += stride) {
    bool valid[kHistItems];
    K key[kHistItems];
    uint32_t ldg[kHistItems];  // level digit: 15 - level
#pragma unroll
    for (int u = 0; u < kHistItems; ++u) {  // every load first (in bounds; stale keys are dropped)
      const int64_t i = base + int64_t(u) * kSortThreads + threadIdx.x;
      const bool in = i < f.span;
      ldg[u] = 0;
      if (f.mode == kSrcStaged) {
        const uint32_t rd = f.stg_ready[in ? i : 0];
        valid[u] = in && rd != 0;
        ldg[u] = (16u - rd) & 15u;
        key[u] = K(uint64_t(f.stg_slack[in ? i : 0] - f.smin));
      } else {
        valid[u] = in;
        key[u] = K(uint32_t(f.wf[in ? i : 0]));
      }
    }
#pragma unroll
    for (int u = 0; u < kHistItems; ++u) {
      for (int ps = 0; ps < npass; ++ps) {
        const uint32_t dg = uint32_t(key[u] >> (ps * kRadixBits)) & (kRadixBuckets - 1);
        // most high digits are shared by the whole wave: one add instead of 64
        const uint64_t act = ballot(valid[u]);
        const int first = readlane_i32(int(dg), act ? __builtin_ctzll(act) : 0);
        const uint64_t same = ballot(valid[u] && int(dg) == first);
        if (same == act) {
          if (act && lane_id() == __builtin_ctzll(act)) atomicAdd(&H[ps][dg], uint32_t(__popcll(act)));
        } else if (valid[u]) {
          atomicAdd(&H[ps][dg], 1u);
        }
      }
      if (level_row >= 0 && valid[u]) atomicAdd(&H[level_row][ldg[u]], 1u);
    }
  }
  __syncthreads();
  if (level_row >= 0)
    for (int b = threadIdx.x; b < 16; b += kSortThreads)
      if (H[level_row][b]) atomicAdd(&ghist[level_row * kRadixBuckets + b], H[level_row][b]);
  for (int ps = 0; ps < npass; ++ps)
    for (int b = threadIdx.x; b < kRadixBuckets; b += kSortThreads)
      if (H[ps][b]) atomicAdd(&ghist[ps * kRadixBuckets + b], H[ps][b]);
}

// One tile of one digit pass.  Every thread of the workgroup calls it.
// Where the last pass of the slack sort writes: the caller's arrays.
struct FinalOut {
  bool on;
  const int32_t* node_of_pos;   // NULL: position == node id
  const int64_t* out_slack;     // by position, or NULL: the slack is the key
  const int32_t* stg_route;
  const int64_t* stg_cost;
  int64_t smin;
  int32_t* order;
  int64_t* slack;
  int32_t* route;
  int64_t* cost;
};

// level_of: non-NULL in the priority-level pass, whose digit is 15 - level
// read from level_of[payload] (1 + level), instead of a digit of the key.
template <typename K>
__device__ void radix_tile(TileSmem<K>& S, const FirstSource& f, bool first, int pass, int64_t tile,
                           int64_t span, int64_t R, const K* kin, const uint32_t* pin, K* kout,
                           uint32_t* pout, const uint32_t* ghist_row, uint64_t* lb_pass,
                           uint32_t epoch, const FinalOut& fo, const uint8_t* level_of = nullptr) {
  const int tid = threadIdx.x;
  const int wv = tid / kWave;
  const int ln = lane_id();
  const int shift = level_of ? 0 : pass * kRadixBits;
  for (int i = tid; i < kWavesPerTile * kRadixBuckets; i += kSortThreads) (&S.whist[0][0])[i] = 0;
  __syncthreads();
  const int64_t seg = tile * kSortTile + int64_t(wv) * (kWave * kSortItems);

  K key[kSortItems];
  uint32_t pay[kSortItems];
  uint32_t rank[kSortItems];
  uint32_t validm = 0;
#pragma unroll
  for (int j = 0; j < kSortItems; ++j) {
    const int64_t i = seg + j * kWave + ln;
    key[j] = K(0);
    pay[j] = 0;
    if (first) {
      if (first_valid(f, i)) {
        key[j] = first_key<K>(f, i);
        pay[j] = uint32_t(i);
        validm |= 1u << j;
      }
    } else if (i < span) {
      key[j] = kin[i];
      pay[j] = pin[i];
      validm |= 1u << j;
    }
  }
  if (level_of) {  // the key's digits are done: the level decides this pass
#pragma unroll
    for (int j = 0; j < kSortItems; ++j)
      if ((validm >> j) & 1u) key[j] = K((16u - uint32_t(level_of[pay[j]])) & 15u);
  }

  // In-wave stable ranking: lanes with equal digits found by 8 ballots; the
  // per-wave running count of each digit lives in LDS.
  uint32_t* wh = S.whist[wv];
#pragma unroll
  for (int j = 0; j < kSortItems; ++j) {
    const bool valid = (validm >> j) & 1u;
    const uint32_t dg = uint32_t(key[j] >> shift) & (kRadixBuckets - 1);
    uint64_t peers = ballot(valid);
#pragma unroll
    for (int b = 0; b < kRadixBits; ++b) {
      const bool bit = (dg >> b) & 1u;
      const uint64_t m = ballot(bit);
      peers &= bit ? m : ~m;
    }
    const uint64_t below = peers & lanemask_lt();
    uint32_t cnt = 0;
    if (valid) cnt = wh[dg];
    rank[j] = cnt + uint32_t(__popcll(below));
    if (valid && below == 0) wh[dg] = cnt + uint32_t(__popcll(peers));
  }
  __syncthreads();

  // Digit totals of the tile; per-wave counts become exclusive offsets.
  const int dg = tid;  // 256 threads, 256 digits
  uint32_t tot = 0;
#pragma unroll
  for (int w = 0; w < kWavesPerTile; ++w) {
    const uint32_t c = S.whist[w][dg];
    S.whist[w][dg] = tot;
    tot += c;
  }
  uint64_t* lb = lb_pass + dg;
  st_relaxed_agent(lb + tile * kRadixBuckets, lb_pack(epoch, tile == 0 ? kLbInc : kLbAgg, tot));
  const uint32_t gexcl = block_excl_scan(ghist_row[dg], S.tmp);
  const uint32_t texcl = block_excl_scan(tot, S.tmp);
  uint64_t excl = 0;
  if (tile > 0) {
    excl = lookback_exclusive(lb, tile, kRadixBuckets, epoch);
    st_relaxed_agent(lb + tile * kRadixBuckets, lb_pack(epoch, kLbInc, excl + tot));
  }
  S.tprefix[dg] = texcl;
  S.gstart[dg] = uint64_t(gexcl) + excl;
  if (dg == kRadixBuckets - 1) S.intile = texcl + tot;
  __syncthreads();

  // Stage the tile in digit order in LDS, then write runs of equal digits to
  // consecutive global addresses.
#pragma unroll
  for (int j = 0; j < kSortItems; ++j) {
    if ((validm >> j) & 1u) {
      const uint32_t dgt = uint32_t(key[j] >> shift) & (kRadixBuckets - 1);
      const uint32_t pos = S.tprefix[dgt] + S.whist[wv][dgt] + rank[j];
      S.key[pos] = key[j];
      S.pay[pos] = pay[j];
    }
  }
  __syncthreads();
  const int in_tile = int(S.intile);
  for (int i = tid; i < in_tile; i += kSortThreads) {
    const K k = S.key[i];
    const uint32_t dgt = uint32_t(k >> shift) & (kRadixBuckets - 1);
    const uint64_t g = S.gstart[dgt] + uint64_t(i - int(S.tprefix[dgt]));
    if (g >= uint64_t(R)) continue;
    if (fo.on) {  // last pass: gather the ready future's decision into place
      const uint32_t pos = S.pay[i];
      fo.order[g] = fo.node_of_pos ? fo.node_of_pos[pos] : int32_t(pos);
      fo.slack[g] = fo.out_slack ? fo.out_slack[pos] : int64_t(uint64_t(k) + uint64_t(fo.smin));
      fo.route[g] = fo.stg_route[pos];
      if (fo.cost) fo.cost[g] = fo.stg_cost[pos];
    } else {
      kout[g] = k;
      pout[g] = S.pay[i];
    }
  }
}

// Resets a control block (workgroup 0, if given) and clears n counters.
__global__ __launch_bounds__(kSortThreads) void k_reset(Ctrl* c, uint32_t* clear, int64_t n) {
  if (c && blockIdx.x == 0) reset_ctrl(c);
  for (int64_t i = int64_t(blockIdx.x) * kSortThreads + threadIdx.x; i < n;
       i += int64_t(gridDim.x) * kSortThreads)
    clear[i] = 0;
}

// The sweep's per-slot range, count and level words as one wave holds them
// (lane l: slot l; other threads hold the identities), loaded ahead of use.
struct RangeLanes {
  int64_t mn = INT64_MAX, mx = INT64_MIN, ct = 0;
  uint32_t lm = 0;
};

__device__ inline RangeLanes load_range_lanes(const Ctrl* ctrl, bool levels) {
  RangeLanes r;
  if (threadIdx.x < kWave) {
    r.mn = ctrl->part_min[threadIdx.x];
    r.mx = ctrl->part_max[threadIdx.x];
    r.ct = ctrl->part_cnt[threadIdx.x];
    if (levels) r.lm = ctrl->part_lvl[threadIdx.x];
  }
  return r;
}

// Slack range, ready count and pass count from the sweep's slots (one wave;
// every thread of the workgroup calls it).  s_range = {min key, ready count,
// digit passes, significant key bits, max key, hint min, hint max, level
// mask, level pass}.  The hint is the key range; with levels the mask of the
// levels seen goes with it, and when more than one level is present the
// passes end with the level pass.
constexpr int kRangeWords = 9;

__device__ void settle_range(const RangeLanes& rl, Ctrl* ctrl, int64_t* s_range, bool write,
                             bool levels) {
  if (threadIdx.x < kWave) {
    const int64_t mn = wave_min_i64(rl.mn);
    const int64_t mx = wave_max_i64(rl.mx);
    const int64_t ct = wave_sum_i64(rl.ct);
    const uint32_t lm = levels ? wave_or_u32(rl.lm) : 0u;
    if (threadIdx.x == 0) {
      const int64_t hmin = mn, hmax = mx;
      int npass = 0, nbits = 0, lpass = 0;
      if (ct > 0) {
        const uint64_t range = uint64_t(mx) - uint64_t(mn);
        nbits = range ? 64 - __builtin_clzll(range) : 0;
        npass = (nbits + kRadixBits - 1) / kRadixBits;
        if (npass == 0) npass = 1;  // the first pass also compacts
        lpass = (lm & (lm - 1)) != 0 ? 1 : 0;
        npass += lpass;
      }
      s_range[0] = mn;
      s_range[1] = ct;
      s_range[2] = npass;
      s_range[3] = nbits;
      s_range[4] = mx;
      s_range[5] = hmin;
      s_range[6] = hmax;
      s_range[7] = int64_t(lm);
      s_range[8] = lpass;
      if (write) {
        ctrl->n_ready = ct;
        ctrl->slack_min = mn;
        ctrl->slack_max = mx;
        ctrl->hint_min = hmin;
        ctrl->hint_max = hmax;
        ctrl->level_mask = lm;
        ctrl->sort_npass = uint32_t(npass);
        ctrl->sort_level_pass = uint32_t(lpass);
      }
    }
  }
  __syncthreads();
}

__device__ void settle_range(Ctrl* ctrl, int64_t* s_range, bool write, bool levels) {
  settle_range(load_range_lanes(ctrl, levels), ctrl, s_range, write, levels);
}

// Status, ready count, the next pass's bucket hint (key range, levels) and the
// significant key bits for the host (one thread).
__device__ inline void publish_status(HostStatus* host, uint32_t status, int64_t n_ready,
                                      int key_bits, int64_t hmin, int64_t hmax, uint32_t lmask) {
  __hip_atomic_store(&host->n_ready, n_ready, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  __hip_atomic_store(&host->key_bits, uint32_t(key_bits), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  __hip_atomic_store(&host->slack_min, hmin, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  __hip_atomic_store(&host->slack_max, hmax, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  __hip_atomic_store(&host->level_mask, lmask, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  __hip_atomic_store(&host->status, status, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

__device__ inline void publish_range(HostStatus* host, uint32_t status, const int64_t* s_range) {
  publish_status(host, status, s_range[1], int(s_range[3]), s_range[5], s_range[6],
                 uint32_t(s_range[7]));
}

// ------------------------------------------------------------ bucketed sort

constexpr int kBucketThreads = 256;
constexpr int kGroupSlots = kBucketGroup * kBucketCap;

// One workgroup per group of kBucketGroup buckets.  Buckets ascend in slack, so
// a future's place in the order is: futures in earlier groups (a sum of group
// counts), plus futures in earlier buckets of its group, plus its rank among
// its bucket-mates by (slack, position).  Positions ascend in (workflow, id),
// so that is the rank by (slack, workflow, id).
__global__ __launch_bounds__(kBucketThreads) void k_bucket_sort(SortArgs a, BucketArgs bk) {
  __shared__ int64_t s_range[kRangeWords];
  __shared__ uint32_t s_off[kBucketGroup + 1];
  __shared__ uint32_t s_red[kBucketThreads / kWave];
  __shared__ int64_t s_slack[kGroupSlots];
  __shared__ int64_t s_cost[kGroupSlots];
  __shared__ int32_t s_pos[kGroupSlots];
  __shared__ int32_t s_route[kGroupSlots];
  __shared__ uint8_t s_bkt[kGroupSlots];
  const int tid = threadIdx.x;
  const int g = blockIdx.x;
  Ctrl* ctrl = a.ctrl;
  // Every load of the prologue is issued before any of them decides anything
  // (they all read memory that exists whatever the status says): the status
  // words, the sweep's range slots (workgroup 0, which reports to the host),
  // the counts of buckets [0, 16 g) four at a time, and this group's counts.
  const uint32_t status = ctrl->status | ctrl->status_sweep;
  const uint32_t overflow = ctrl->bucket_overflow;  // written by the sweep, an earlier kernel
  RangeLanes rl;
  if (g == 0) rl = load_range_lanes(ctrl, a.levels != 0);
  uint32_t part = 0;
  const uint4* cnt4 = reinterpret_cast<const uint4*>(bk.cnt);
#pragma unroll 4
  for (int i = tid; i < g * (kBucketGroup / 4); i += kBucketThreads) {
    const uint4 c = cnt4[i];
    part += c.x + c.y + c.z + c.w;
  }
  uint32_t cg = tid < kBucketGroup ? bk.cnt[g * kBucketGroup + tid] : 0u;
  if (status) {
    if (g == 0 && tid == 0) publish_status(a.host, status, 0, 0, 0, 0, 0u);
    return;
  }
  if (g == 0) {
    settle_range(rl, ctrl, s_range, true, a.levels != 0);
    if (tid == 0) publish_range(a.host, overflow ? kStatusTiled : 0u, s_range);
  }
  if (overflow) return;

  // futures in earlier groups
  part = uint32_t(wave_sum_i64(int64_t(part)));
  if (lane_id() == 0) s_red[tid / kWave] = part;
  if (tid < kWave) {  // bucket offsets inside the group (wave 0)
    uint32_t c = cg;
    c = c < uint32_t(kBucketCap) ? c : uint32_t(kBucketCap);  // overflow was handled above
    const uint32_t inc = wave_incl_scan_u32(c);
    if (tid < kBucketGroup) s_off[tid + 1] = inc;
    if (tid == 0) s_off[0] = 0;
  }
  __syncthreads();
  int64_t base = 0;
#pragma unroll
  for (int w = 0; w < kBucketThreads / kWave; ++w) base += s_red[w];
  const int T = int(s_off[kBucketGroup]);
  if (T == 0) return;

  // this group's futures into LDS, bucket by bucket
  for (int i = tid; i < T; i += kBucketThreads) {
    int b = 0;
#pragma unroll
    for (int k = 1; k < kBucketGroup; ++k) b += int(s_off[k]) <= i;
    const BucketSlot* sl = bk.slot + (int64_t(g) * kBucketGroup + b) * kBucketCap + (i - int(s_off[b]));
    s_slack[i] = sl->key;
    s_cost[i] = sl->cost;
    s_pos[i] = sl->pos;
    s_route[i] = sl->route;
    s_bkt[i] = uint8_t(b);
  }
  __syncthreads();
  for (int i = tid; i < T; i += kBucketThreads) {
    const int b = s_bkt[i];
    const int lo = int(s_off[b]), hi = int(s_off[b + 1]);
    const int64_t sk = s_slack[i];
    const int32_t ps = s_pos[i];
    int rank = 0;
    if (a.levels) {  // a bucket may hold several levels: (level desc, key, position)
      const int sl = slot_level(s_route[i]);
#pragma unroll 4
      for (int j = lo; j < hi; ++j) {
        const int64_t o = s_slack[j];
        const int ol = slot_level(s_route[j]);
        rank += (ol > sl) | ((ol == sl) & ((o < sk) | ((o == sk) & (s_pos[j] < ps))));
      }
    } else {
#pragma unroll 8
      for (int j = lo; j < hi; ++j) {  // independent LDS loads: unrolled, they overlap
        const int64_t o = s_slack[j];
        rank += (o < sk) | ((o == sk) & (s_pos[j] < ps));
      }
    }
    const int64_t out = base + lo + rank;
    a.order[out] = a.node_of_pos ? a.node_of_pos[ps] : ps;
    a.slack[out] = a.out_slack ? a.out_slack[ps] : sk;
    a.route[out] = slot_route(s_route[i]);
    if (a.cost) a.cost[out] = s_cost[i];
  }
}

// Large bucket counts.  k_bucket_totals writes the number of futures in each
// group of kBucketLbGroup buckets; k_bucket_sort_lb then runs one workgroup per
// group (one bucket per thread), whose base is the sum of the totals of all
// earlier groups (plain loads: the totals come from the previous kernel, so
// they are cached like any input).  A future's rank inside its bucket is
// counted against its bucket-mates' slots directly (a few on average).
__global__ __launch_bounds__(kBucketLbGroup) void k_bucket_totals(SortArgs a, BucketArgs bk) {
  constexpr int kPerBlock = kBucketLbGroup / kWave;  // groups per workgroup, one per wave
  Ctrl* ctrl = a.ctrl;
  const int wv = threadIdx.x / kWave;
  const int64_t grp = int64_t(blockIdx.x) * kPerBlock + wv;
  if (grp * kBucketLbGroup >= bk.nb) return;
  const uint32_t bad = ctrl->status | ctrl->status_sweep | ctrl->bucket_overflow;
  const uint4 c = reinterpret_cast<const uint4*>(bk.cnt + grp * kBucketLbGroup)[lane_id()];
  if (bad != 0) return;
  const uint32_t cap = uint32_t(kBucketCap);
  const int64_t t = int64_t((c.x < cap ? c.x : cap) + (c.y < cap ? c.y : cap) +
                            (c.z < cap ? c.z : cap) + (c.w < cap ? c.w : cap));
  const int64_t sum = wave_sum_i64(t);
  if (lane_id() == 0) a.bagg[grp] = uint64_t(sum);
  // the fullest bucket (how crowded the plan is: the host adds buckets when
  // it is), folded into one of kParts slots; not needed once the plan has
  // the most buckets it can have
  if (bk.nb < kBucketMax) {
    const uint32_t m01 = c.x > c.y ? c.x : c.y, m23 = c.z > c.w ? c.z : c.w;
    const int64_t mx = wave_max_i64(int64_t(m01 > m23 ? m01 : m23));
    if (lane_id() == 0)
      __hip_atomic_fetch_max(&ctrl->part_crowd[grp & (kParts - 1)], uint32_t(mx), __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
  }
}

constexpr int kLbStage = 2048;  // futures of a bucket group staged in LDS at once
static_assert(kLbStage % kBucketLbGroup == 0, "whole rows of the workgroup");

__global__ __launch_bounds__(kBucketLbGroup) void k_bucket_sort_lb(SortArgs a, BucketArgs bk) {
  __shared__ int64_t s_range[kRangeWords];
  __shared__ uint32_t s_off[kBucketLbGroup + 1];
  __shared__ uint32_t s_red[kBucketLbGroup / kWave];
  __shared__ int64_t s_base[kBucketLbGroup / kWave];
  __shared__ int64_t s_slack[kLbStage];
  __shared__ int32_t s_pos[kLbStage];
  __shared__ uint8_t s_b[kLbStage];
  __shared__ uint8_t s_lv[kLbStage];  // priority level (with levels only)
  const int tid = threadIdx.x;
  const int wv = tid / kWave;
  const int g = blockIdx.x;
  Ctrl* ctrl = a.ctrl;
  // every load of the prologue first (as in k_bucket_sort): status words,
  // range slots (workgroup 0), the totals of earlier groups, this bucket's count
  const uint32_t status = ctrl->status | ctrl->status_sweep;
  const uint32_t overflow = ctrl->bucket_overflow;  // written by the sweep, an earlier kernel
  RangeLanes rl;
  uint32_t crowd = 0;
  if (g == 0) {
    rl = load_range_lanes(ctrl, a.levels != 0);
    if (tid < kWave) crowd = ctrl->part_crowd[tid];
  }
  int64_t part = 0;
#pragma unroll 4
  for (int j = tid; j < g; j += kBucketLbGroup) part += int64_t(a.bagg[j]);
  const int64_t b0 = int64_t(g) * kBucketLbGroup;
  uint32_t c = bk.cnt[b0 + tid];
  if (status) {
    if (g == 0 && tid == 0) publish_status(a.host, status, 0, 0, 0, 0, 0u);
    return;
  }
  if (g == 0) {
    crowd = uint32_t(wave_max_i64(int64_t(crowd)));  // wave 0 holds the slots
    if (tid == 0) __hip_atomic_store(&a.host->max_bucket, crowd, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    settle_range(rl, ctrl, s_range, true, a.levels != 0);
    if (tid == 0) publish_range(a.host, overflow ? kStatusTiled : 0u, s_range);
  }
  if (overflow) return;

  // futures in earlier groups
  part = wave_sum_i64(part);
  // bucket offsets inside the group
  c = c < uint32_t(kBucketCap) ? c : uint32_t(kBucketCap);  // overflow was handled above
  const uint32_t inc = wave_incl_scan_u32(c);
  if (lane_id() == kWave - 1) s_red[wv] = inc;
  if (lane_id() == 0) s_base[wv] = part;
  __syncthreads();
  uint32_t before = 0;
  int64_t base = 0;
#pragma unroll
  for (int w = 0; w < kBucketLbGroup / kWave; ++w) {
    before += w < wv ? s_red[w] : 0u;
    base += s_base[w];
  }
  s_off[tid + 1] = before + inc;
  if (tid == 0) s_off[0] = 0;
  __syncthreads();

  // The group's futures go through LDS in chunks of at most kLbStage that end
  // at a bucket boundary (a bucket holds at most kBucketCap < kLbStage, so
  // every chunk holds at least one whole bucket): bucket ids first (each
  // thread writes its own bucket's), then every slot of the chunk with
  // independent loads, then each future is ranked among its bucket-mates.
  const int T = int(s_off[kBucketLbGroup]);
  const int my0 = int(before + inc - c), my1 = int(before + inc);
  for (int cs = 0, ce = 0; cs < T; cs = ce) {
    ce = T;
    if (T - cs > kLbStage) {  // the last boundary within kLbStage of cs
      int lo = 0, hi = kBucketLbGroup;  // s_off[lo] <= cs + kLbStage < s_off[hi]
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (int(s_off[mid]) <= cs + kLbStage) lo = mid; else hi = mid;
      }
      ce = int(s_off[lo]);
    }
    for (int i = my0 > cs ? my0 : cs; i < (my1 < ce ? my1 : ce); ++i) s_b[i - cs] = uint8_t(tid);
    __syncthreads();
    // Addresses first, then every load with no per-lane branch between them
    // (such a branch makes the compiler wait for the previous load before the
    // next address).  Only the rows the chunk fills are loaded (a bound the
    // same on every lane); a lane past the chunk's end loads the group's first
    // slot, which always exists, and drops it (one line per group, not one
    // address that every group queues on).
    const int rows = (ce - cs + kBucketLbGroup - 1) / kBucketLbGroup;
    int64_t at[kLbStage / kBucketLbGroup];
#pragma unroll
    for (int u = 0; u < kLbStage / kBucketLbGroup; ++u) {
      const int i = cs + u * kBucketLbGroup + tid;
      const bool ok = i < ce;
      const int lb = s_b[ok ? i - cs : 0];
      const int64_t q = (b0 + lb) * kBucketCap + (i - int(s_off[lb]));
      at[u] = ok ? q : b0 * kBucketCap;
    }
    BucketSlot v[kLbStage / kBucketLbGroup];
#pragma unroll
    for (int u = 0; u < kLbStage / kBucketLbGroup; ++u)
      if (u < rows) v[u] = bk.slot[at[u]];
    // the gathers by position (output slack, node id) are issued here, so
    // that their latency overlaps the staging and the ranking
    int64_t os[kLbStage / kBucketLbGroup];
    int32_t on[kLbStage / kBucketLbGroup];
#pragma unroll
    for (int u = 0; u < kLbStage / kBucketLbGroup; ++u) {
      if (u >= rows) continue;
      const bool ok = cs + u * kBucketLbGroup + tid < ce;
      const int32_t ps = ok ? v[u].pos : 0;  // a dropped lane's slot may be stale
      os[u] = a.out_slack ? a.out_slack[ps] : v[u].key;
      on[u] = a.node_of_pos ? a.node_of_pos[ps] : ps;
    }
#pragma unroll
    for (int u = 0; u < kLbStage / kBucketLbGroup; ++u) {
      const int i = cs + u * kBucketLbGroup + tid;
      if (i < ce) {
        s_slack[i - cs] = v[u].key;
        s_pos[i - cs] = v[u].pos;
        if (a.levels) s_lv[i - cs] = uint8_t(slot_level(v[u].route));
      }
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kLbStage / kBucketLbGroup; ++u) {
      const int i = cs + u * kBucketLbGroup + tid;
      if (i >= ce) continue;
      const int lb = s_b[i - cs];
      const int k0 = int(s_off[lb]);
      const int k1 = int(s_off[lb + 1]);  // inside [cs, ce]: chunks end at bucket boundaries
      int rank = 0;
      if (a.levels) {  // a bucket may hold several levels: (level desc, key, position)
        const int sl = slot_level(v[u].route);
#pragma unroll 4
        for (int j = k0 - cs; j < k1 - cs; ++j) {
          const int64_t o = s_slack[j];
          const int ol = s_lv[j];
          rank += (ol > sl) | ((ol == sl) & ((o < v[u].key) | ((o == v[u].key) & (s_pos[j] < v[u].pos))));
        }
      } else {
#pragma unroll 8
        for (int j = k0 - cs; j < k1 - cs; ++j) {  // independent LDS loads: unrolled, they overlap
          const int64_t o = s_slack[j];
          rank += (o < v[u].key) | ((o == v[u].key) & (s_pos[j] < v[u].pos));
        }
      }
      const int64_t out = base + k0 + rank;
      a.order[out] = on[u];
      a.slack[out] = os[u];
      a.route[out] = slot_route(v[u].route);
      if (a.cost) a.cost[out] = v[u].cost;
    }
    __syncthreads();
  }
}

// ------------------------------------------------------------ bin sort

constexpr int kBinThreads = 256;

// The key a pass orders by, recovered from its output at rank g: the slack,
// or the remaining critical path (deadline - now - slack) negated under LPT or
// as it is under SRTF.
__device__ inline int64_t output_key(const SortArgs& a, int64_t g) {
  const int64_t sl = a.slack[g];
  if (!(a.p.policy & (NALAR_ORDER_LPT | NALAR_ORDER_SRTF))) return sl;
  const int32_t v = a.order[g];
  const int64_t rem = (a.p.deadline[a.p.wf[v]] - a.p.now) - sl;
  return (a.p.policy & NALAR_ORDER_LPT) ? -rem : rem;
}

// One workgroup per bin: its records (claimed by the sweep in any order) are
// put in (key, position) order, which is the (key, wf, id) order since
// positions follow (wf, id), by a counting sort over kBinSub sub-buckets of
// the bin's key range (the top bits of key minus the bin's lowest key; the
// lowest and highest bins, whose keys may trail off away from their one
// splitter, count again on a log-linear scale of the distance from that
// splitter, 16 sub-buckets per octave, if the first count crowds): one
// LDS counter per sub-bucket, their exclusive scan, and a scatter of (key,
// position) to LDS; a future's rank is then its sub-bucket's start plus the
// number of sub-bucket mates of smaller (key, position).  Sub-buckets hold
// about one future each, since the bins are cut at quantiles; one holding
// more than kBinRun (many equal keys, or a bin whose keys crowd at one end of
// its range, as the lowest and highest bins' tails do) is sorted in place by
// the whole workgroup with a bitonic network whose comparators all put the
// smaller entry first, so that the missing entries of the padded size never
// move (comparators reaching past the segment are skipped).  The futures are
// then in LDS by rank, and the sorted bin is written at its offset (the
// records of all lower bins) with consecutive lanes on consecutive ranks.  The workgroups also write the next pass's
// splitters (this pass's key quantiles: the key at rank (q + 1) * R / nb' for
// nb' = bins_for(R)): the future of that rank writes it.  Workgroup 0
// publishes the status.
// Two kernels share the work: k_bin_sort (kBinThreads threads, a bin of up
// to kBinCap futures in LDS, one workgroup per bin) and k_bin_sort_big (four
// times the threads and the LDS) for the few bins holding more: the bins hold up to
// kBinAlloc records, so that a ready set whose keys moved since the splitters
// were taken (a whole workflow's futures shifting together) still fits.
constexpr int kBinBigThreads = 4 * kBinThreads;
constexpr int kBinBigCap = 4 * kBinCap;
static_assert(kBinBigCap >= kBinAlloc, "the big-bin kernel holds a full bin");
constexpr int kBinJ = (kBinCap + kBinThreads - 1) / kBinThreads;  // items per lane (both kernels)
static_assert(kBinJ * kBinBigThreads >= kBinBigCap, "items per lane of the big-bin kernel");
constexpr int kBinSub = 1024;
constexpr int kBinSubLog = 10;
static_assert(kBinSub == 1 << kBinSubLog && kBinSub % kBinBigThreads == 0, "sub-buckets");

constexpr int kBinRun = 32;
constexpr int kBinCrowdMax = kBinBigCap / (kBinRun + 1) + 1;  // crowded sub-buckets a bin can hold

template <int NW>
struct BinFixed {
  uint32_t sub[kBinSub];  // sub-bucket counts, then starts
  uint32_t crowd[kBinCrowdMax];  // crowded sub-buckets: start | end << 16
  int ncrowd;
  uint32_t tmp[NW];
  int64_t range[kRangeWords];
  int64_t red[4][NW];
};

__host__ __device__ constexpr size_t bin_align(size_t b) { return (b + 15) & ~size_t(15); }

// LDS of a workgroup holding lc futures: keys, positions, record indices,
// (with workflow ties) the positions' workflows, and the fixed part.
template <int NW>
__host__ __device__ constexpr size_t bin_lds_bytes(int lc, bool tie_wf) {
  return bin_align(8 * size_t(lc)) + bin_align(4 * size_t(lc)) + bin_align(2 * size_t(lc)) +
         (tie_wf ? bin_align(4 * size_t(lc)) : 0) + sizeof(BinFixed<NW>);
}

template <int NW>
struct BinLds {
  int64_t* key;
  int32_t* pos;
  uint16_t* rec;
  int32_t* wf;
  BinFixed<NW>* F;
};

template <int NW>
__device__ inline BinLds<NW> carve_bin(unsigned char* sp, int lc, bool tie_wf) {
  BinLds<NW> L;
  L.key = reinterpret_cast<int64_t*>(sp); sp += bin_align(8 * size_t(lc));
  L.pos = reinterpret_cast<int32_t*>(sp); sp += bin_align(4 * size_t(lc));
  L.rec = reinterpret_cast<uint16_t*>(sp); sp += bin_align(2 * size_t(lc));
  L.wf = nullptr;
  if (tie_wf) {
    L.wf = reinterpret_cast<int32_t*>(sp);
    sp += bin_align(4 * size_t(lc));
  }
  L.F = reinterpret_cast<BinFixed<NW>*>(sp);
  return L;
}

// Sub-bucket of a key: mode 0, (key - base) >> sshift (base the bin's lowest
// key); mode 1 (lowest bin, base = its splitter - 1 >= key) and mode 2
// (highest bin, base = its splitter <= key) a log-linear scale of the
// distance d from base (d below 16 as it is, else 16 steps per octave),
// reversed in mode 1 so that sub-buckets ascend with the key.
__device__ inline uint32_t bin_sub(int64_t key, int mode, int64_t base, int sshift) {
  if (mode == 0) return uint32_t((uint64_t(key) - uint64_t(base)) >> sshift);
  const uint64_t d = mode == 1 ? uint64_t(base) - uint64_t(key) : uint64_t(key) - uint64_t(base);
  uint32_t f = uint32_t(d);
  if (d >= 16) {
    const int e = 63 - __builtin_clzll(d);  // 4 .. 63, so f < 976
    f = uint32_t(e - 3) * 16u + uint32_t((d >> (e - 4)) & 15u);
  }
  return mode == 1 ? uint32_t(kBinSub - 1) - f : f;
}

// Entries x < y of an LDS segment: (key, workflow, position) ascending (no
// workflow array: (key, position)), the record index moving along.
__device__ inline void bin_cmpx(int64_t* k, int32_t* p, uint16_t* r, int32_t* w, int x, int y) {
  const int64_t kx = k[x], ky = k[y];
  const int32_t px = p[x], py = p[y];
  const int32_t wx = w ? w[x] : 0, wy = w ? w[y] : 0;
  if (ky < kx || (ky == kx && (wy < wx || (wy == wx && py < px)))) {
    k[x] = ky;
    k[y] = kx;
    p[x] = py;
    p[y] = px;
    if (w) {
      w[x] = wy;
      w[y] = wx;
    }
    const uint16_t rx = r[x];
    r[x] = r[y];
    r[y] = rx;
  }
}

// Sorts the segment [0, L) of the three LDS arrays in place (every thread of
// the workgroup takes part): sizes 2, 4, ..., P (P the power of two >= L),
// each a mirror step (entry i of a block against the block's entry k - 1 - i)
// and then half-cleaners at distances k/4 ... 1.
__device__ void bin_bitonic(int64_t* k, int32_t* p, uint16_t* r, int32_t* w, int L) {
  int lp = 0;
  while ((1 << lp) < L) ++lp;
  const int P = 1 << lp;
  for (int ls = 1; ls <= lp; ++ls) {  // size 2^ls, half 2^(ls - 1)
    const int lh = ls - 1;
    for (int c = threadIdx.x; c < P / 2; c += int(blockDim.x)) {
      const int base = (c >> lh) << ls, off = c & ((1 << lh) - 1);
      const int x = base + off, y = base + (1 << ls) - 1 - off;
      if (y < L) bin_cmpx(k, p, r, w, x, y);
    }
    __syncthreads();
    for (int ld = lh - 1; ld >= 0; --ld) {  // distance 2^ld
      for (int c = threadIdx.x; c < P / 2; c += int(blockDim.x)) {
        const int x = ((c >> ld) << (ld + 1)) + (c & ((1 << ld) - 1)), y = x + (1 << ld);
        if (y < L) bin_cmpx(k, p, r, w, x, y);
      }
      __syncthreads();
    }
  }
}

// Sorts bin b (n records, n <= LC) with T threads and writes it out.
template <int T, int LC>
__device__ void bin_sort_one(const SortArgs& a, const BucketArgs& bk, int b, int n, const BinLds<T / kWave>& L) {
  constexpr int kBinThreads = T;
  constexpr int kBinWaves = T / kWave;
  const int cap = bk.cap;
  const int32_t* tw = a.tie_wf;
  int64_t* s_key = L.key;
  int32_t* s_pos = L.pos;
  uint16_t* s_rec = L.rec;
  int32_t* s_wf = L.wf;
  BinFixed<kBinWaves>* F = L.F;
  const int tid = threadIdx.x;
  const int wv = tid / kWave;
  const int ln = lane_id();
  uint32_t before = 0, total = 0;
  for (int i = tid; i < bk.nb; i += kBinThreads) {
    uint32_t c = bk.cnt[i];
    c = c < uint32_t(cap) ? c : uint32_t(cap);
    total += c;
    before += i < b ? c : 0u;
  }
  const BucketSlot* rec = bk.slot + int64_t(b) * cap;
  // item j of lane l of wave w: record w * C + j * 64 + l
  const int J = (n + kBinThreads - 1) / kBinThreads;
  const int C = J * kWave;
  int64_t key[kBinJ];
  int32_t pos[kBinJ], wfj[kBinJ];
  int64_t kmin = INT64_MAX, kmax = INT64_MIN;
#pragma unroll
  for (int j = 0; j < kBinJ; ++j) {
    const int i = wv * C + j * kWave + ln;
    key[j] = 0;
    pos[j] = 0;
    wfj[j] = 0;
    if (j < J && i < n) {
      key[j] = rec[i].key;
      pos[j] = rec[i].pos;
      if (tw) wfj[j] = tw[pos[j]];
      kmin = key[j] < kmin ? key[j] : kmin;
      kmax = key[j] > kmax ? key[j] : kmax;
    }
  }
  // for (for the sub-bucket counters) and block sums: records before this
  // bin and in total, and the bin's key range
  for (int i = tid; i < kBinSub; i += kBinThreads) F->sub[i] = 0;
  {
    const int64_t s0 = wave_sum_i64(int64_t(before)), s1 = wave_sum_i64(int64_t(total));
    const int64_t m0 = wave_min_i64(kmin), m1 = wave_max_i64(kmax);
    if (ln == 0) {
      F->red[0][wv] = s0;
      F->red[1][wv] = s1;
      F->red[2][wv] = m0;
      F->red[3][wv] = m1;
    }
    __syncthreads();
    before = 0;
    total = 0;
    kmin = INT64_MAX;
    kmax = INT64_MIN;
    for (int w = 0; w < kBinWaves; ++w) {
      before += uint32_t(F->red[0][w]);
      total += uint32_t(F->red[1][w]);
      kmin = F->red[2][w] < kmin ? F->red[2][w] : kmin;
      kmax = F->red[3][w] > kmax ? F->red[3][w] : kmax;
    }
  }
  const int64_t R = total;
  const uint64_t kr = n > 0 ? uint64_t(kmax) - uint64_t(kmin) : 0;
  // sub-bucket scale: linear over [kmin, kmax], or log-linear from the one
  // splitter of the lowest or highest bin (below)
  const int kbits = kr ? 64 - __builtin_clzll(kr) : 0;
  const int sshift = kbits > kBinSubLog ? kbits - kBinSubLog : 0;
  int smode = 0;
  int64_t sbase = kmin;
  uint32_t at[kBinJ];  // slot inside the sub-bucket, then the rank in the bin
  for (;;) {
#pragma unroll
    for (int j = 0; j < kBinJ; ++j) {
      at[j] = 0;
      if (j < J && wv * C + j * kWave + ln < n)
        at[j] = atomicAdd(&F->sub[bin_sub(key[j], smode, sbase, sshift)], 1u);
    }
    __syncthreads();
    if (smode != 0 || (b != 0 && b != bk.nb - 1)) break;
    // the lowest or highest bin with a crowded sub-bucket counts again on
    // the log-linear scale
    bool crowded = false;
    for (int i = tid; i < kBinSub; i += kBinThreads) crowded |= F->sub[i] > uint32_t(kBinRun);
    if (!__syncthreads_or(crowded ? 1 : 0)) break;
    smode = b == 0 ? 1 : 2;
    sbase = b == 0 ? bk.split[0] - 1 : bk.split[bk.nb - 2];
    for (int i = tid; i < kBinSub; i += kBinThreads) F->sub[i] = 0;
    __syncthreads();
  }
  {
    constexpr int kPerT = kBinSub / kBinThreads;
    uint32_t c[kPerT], sum = 0;
#pragma unroll
    for (int u = 0; u < kPerT; ++u) {
      c[u] = F->sub[tid * kPerT + u];
      sum += c[u];
    }
    uint32_t run = block_excl_scan(sum, F->tmp);  // every count is read before its barrier
#pragma unroll
    for (int u = 0; u < kPerT; ++u) {
      F->sub[tid * kPerT + u] = run;
      run += c[u];
    }
  }
  __syncthreads();
  uint32_t span[kBinJ];  // the sub-bucket's [start, end) as start | end << 16 (n < 2^16)
#pragma unroll
  for (int j = 0; j < kBinJ; ++j) {
    span[j] = 0;
    if (j >= J || wv * C + j * kWave + ln >= n) continue;
    const uint32_t sb = bin_sub(key[j], smode, sbase, sshift);
    const uint32_t st = F->sub[sb];
    const uint32_t en = sb + 1 < uint32_t(kBinSub) ? F->sub[sb + 1] : uint32_t(n);
    span[j] = st | (en << 16);
    s_key[st + at[j]] = key[j];
    s_pos[st + at[j]] = pos[j];
    s_rec[st + at[j]] = uint16_t(wv * C + j * kWave + ln);
    if (tw) s_wf[st + at[j]] = wfj[j];
  }
  if (tid == 0) F->ncrowd = 0;
  __syncthreads();
  {
    constexpr int kPerT = kBinSub / kBinThreads;
#pragma unroll
    for (int u = 0; u < kPerT; ++u) {
      const int sb = tid * kPerT + u;
      const uint32_t st = F->sub[sb];
      const uint32_t en = sb + 1 < kBinSub ? F->sub[sb + 1] : uint32_t(n);
      if (en - st > uint32_t(kBinRun)) F->crowd[atomicAdd(&F->ncrowd, 1)] = st | (en << 16);
    }
  }
  // rank: the sub-bucket's start plus its mates of smaller (key, position)
  // (crowded sub-buckets are sorted below)
#pragma unroll
  for (int j = 0; j < kBinJ; ++j) {
    at[j] = 0xFFFFFFFFu;
    if (j >= J || wv * C + j * kWave + ln >= n) continue;
    const int st = int(span[j] & 0xFFFFu), en = int(span[j] >> 16);
    if (en - st > kBinRun) continue;
    uint32_t r = uint32_t(st);
    if (tw) {
      for (int q = st; q < en; ++q) {
        const int64_t kq = s_key[q];
        const int32_t wq = s_wf[q];
        r += (kq < key[j]) | ((kq == key[j]) & ((wq < wfj[j]) | ((wq == wfj[j]) & (s_pos[q] < pos[j]))));
      }
    } else {
      for (int q = st; q < en; ++q) {
        const int64_t kq = s_key[q];
        r += (kq < key[j]) | ((kq == key[j]) & (s_pos[q] < pos[j]));
      }
    }
    at[j] = r;
  }
  // by rank in LDS (every mate has been read), then written rank by rank; the
  // future at a splitter rank G = (q + 1) * R / nb' also writes splitter q
  // (q + 1 = ceil(G nb' / R); at most one q per rank since R / nb' >= 1)
  __syncthreads();
#pragma unroll
  for (int j = 0; j < kBinJ; ++j) {
    const int i = wv * C + j * kWave + ln;
    if (j >= J || i >= n || at[j] == 0xFFFFFFFFu) continue;
    s_key[at[j]] = key[j];
    s_pos[at[j]] = pos[j];
    s_rec[at[j]] = uint16_t(i);
  }
  // the crowded sub-buckets (other ranges of LDS than the moves above)
  const int ncrowd = F->ncrowd;
  for (int c = 0; c < ncrowd; ++c) {
    const uint32_t cs = F->crowd[c];
    const int st = int(cs & 0xFFFFu);
    bin_bitonic(s_key + st, s_pos + st, s_rec + st, s_wf ? s_wf + st : nullptr, int(cs >> 16) - st);
  }
  __syncthreads();
  const int nbn = R >= a.split_min ? bins_for(R) : 0;
  for (int r = tid; r < n; r += kBinThreads) {
    const int64_t g = int64_t(before) + r;
    const int64_t k = s_key[r];
    const int32_t ps = s_pos[r];
    const BucketSlot& src = rec[s_rec[r]];
    a.order[g] = a.node_of_pos ? a.node_of_pos[ps] : ps;
    a.slack[g] = a.out_slack ? a.out_slack[ps] : k;
    a.route[g] = slot_route(src.route);
    if (a.cost) a.cost[g] = src.cost;
    if (nbn > 0) {
      const int64_t q1 = (g * nbn + R - 1) / R;
      if (q1 >= 1 && q1 <= nbn - 1 && (q1 * R) / nbn == g) a.split_next[q1 - 1] = k;
    }
  }
  if (b == 0 && tid == 0)
    __hip_atomic_store(&a.host->split_nb, uint32_t(nbn), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

// One workgroup per bin; bins of more than kBinCap records are left to
// k_bin_sort_big.  Workgroup 0 settles and publishes the status and range,
// and the size of the largest bin (in max_bucket), from which the host plans
// the next pass's bin capacity.
__global__ __launch_bounds__(kBinThreads) void k_bin_sort(SortArgs a, BucketArgs bk) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int NW = kBinThreads / kWave;
  const BinLds<NW> L = carve_bin<NW>(smem, kBinCap, a.tie_wf != nullptr);
  const int b = blockIdx.x;
  if (b == 0) {
    __shared__ uint32_t s_mx[NW];
    uint32_t mx = 0;
    for (int i = int(threadIdx.x); i < bk.nb; i += kBinThreads) mx = bk.cnt[i] > mx ? bk.cnt[i] : mx;
    mx = uint32_t(wave_max_i64(int64_t(mx)));
    if (lane_id() == 0) s_mx[threadIdx.x / kWave] = mx;
    __syncthreads();
    if (threadIdx.x == 0) {
      for (int w = 1; w < NW; ++w) mx = s_mx[w] > mx ? s_mx[w] : mx;
      __hip_atomic_store(&a.host->max_bucket, mx, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    }
  }
  Ctrl* ctrl = a.ctrl;
  const uint32_t status = ctrl->status | ctrl->status_sweep;
  const uint32_t overflow = ctrl->bucket_overflow;
  RangeLanes rl;
  if (b == 0) rl = load_range_lanes(ctrl, a.levels != 0);
  if (status) {
    if (b == 0 && threadIdx.x == 0) publish_status(a.host, status, 0, 0, 0, 0, 0u);
    return;
  }
  if (b == 0) {
    settle_range(rl, ctrl, L.F->range, true, a.levels != 0);
    if (threadIdx.x == 0) publish_range(a.host, overflow ? kStatusTiled : 0u, L.F->range);
  }
  if (overflow) return;
  const uint32_t nraw = bk.cnt[b];
  const int n = int(nraw < uint32_t(bk.cap) ? nraw : uint32_t(bk.cap));
  if (n > kBinCap) return;
  bin_sort_one<kBinThreads, kBinCap>(a, bk, b, n, L);
}

// The bins of more than kBinCap records: every workgroup lists them in bin
// order and takes every gridDim-th.
constexpr int kBinBigGroups = 64;

__global__ __launch_bounds__(kBinBigThreads) void k_bin_sort_big(SortArgs a, BucketArgs bk) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int NW = kBinBigThreads / kWave;
  const BinLds<NW> L = carve_bin<NW>(smem, kBinBigCap, a.tie_wf != nullptr);
  __shared__ int32_t s_big[kBinMax];
  __shared__ int s_nbig;
  Ctrl* ctrl = a.ctrl;
  if ((ctrl->status | ctrl->status_sweep) != 0 || ctrl->bucket_overflow != 0) return;
  int nbig = 0;
  for (int i0 = 0; i0 < bk.nb; i0 += kBinBigThreads) {
    const int i = i0 + int(threadIdx.x);
    const uint32_t c = i < bk.nb ? bk.cnt[i] : 0u;
    const bool big = c > uint32_t(kBinCap) && c <= uint32_t(bk.cap);
    const uint32_t at = block_excl_scan(big ? 1u : 0u, L.F->tmp);
    if (big) s_big[nbig + int(at)] = i;
    if (threadIdx.x == kBinBigThreads - 1) s_nbig = nbig + int(at) + (big ? 1 : 0);
    __syncthreads();
    nbig = s_nbig;
    __syncthreads();
  }
  for (int k = int(blockIdx.x); k < nbig; k += int(gridDim.x)) {
    const int b = s_big[k];
    bin_sort_one<kBinBigThreads, kBinBigCap>(a, bk, b, int(bk.cnt[b]), L);
    __syncthreads();
  }
}

// The next pass's splitters from the output of the tiled or bucketed sort
// (one workgroup; R from the control block the sort settled).
__global__ __launch_bounds__(kSortThreads) void k_splitters(SortArgs a) {
  Ctrl* ctrl = a.ctrl;
  // nothing when the pass failed, a bucket overflowed (the host sorts again),
  // or the tiled sort has passes still to run
  if (ctrl->bucket_overflow || int(ctrl->sort_npass) > a.passes_launched) return;
  const uint32_t bad = ctrl->status | ctrl->status_sweep;
  const int64_t R = ctrl->n_ready;
  const int nbn = (bad == 0 && R >= a.split_min) ? bins_for(R) : 0;
  for (int q = threadIdx.x; q < nbn - 1; q += kSortThreads)
    a.split_next[q] = output_key(a, (int64_t(q) + 1) * R / nbn);
  if (threadIdx.x == 0)
    __hip_atomic_store(&a.host->split_nb, uint32_t(nbn), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

__global__ __launch_bounds__(kSortThreads) void k_slack_hist(SortArgs a) {
  __shared__ uint32_t H[kMaxSortPasses][kRadixBuckets];
  __shared__ int64_t s_range[kRangeWords];
  Ctrl* ctrl = a.ctrl;
  const uint32_t status = ctrl->status | ctrl->status_sweep;
  if (status) {
    if (blockIdx.x == 0 && threadIdx.x == 0) publish_status(a.host, status, 0, 0, 0, 0, 0u);
    return;
  }
  settle_range(ctrl, s_range, blockIdx.x == 0, a.levels != 0);
  const int npass = int(s_range[2]);
  if (npass == 0) {  // nothing ready: no pass runs, so report here
    if (blockIdx.x == 0 && threadIdx.x == 0) publish_status(a.host, 0, 0, 0, 0, 0, 0u);
    return;
  }
  const FirstSource f{kSrcStaged, a.stg_slack, a.stg_ready, nullptr, a.span, s_range[0]};
  const int lpass = int(s_range[8]);
  histogram<uint64_t>(f, npass - lpass, lpass ? npass - 1 : -1, H, ctrl->ghist_slack);
}

// One digit pass of the slack sort.  The last pass the key range needs writes
// the caller's arrays and the host status; pass kSortLaunched-1 of a wider range
// asks the host for the remaining passes instead.
__global__ __launch_bounds__(kSortThreads) void k_slack_pass(SortArgs a, int pass) {
  __shared__ TileSmem<uint64_t> S;
  Ctrl* ctrl = a.ctrl;
  if (ctrl->status | ctrl->status_sweep) return;
  const int npass = int(ctrl->sort_npass);
  if (pass >= npass) return;
  const int64_t R = ctrl->n_ready;
  const bool first = pass == 0;
  const bool last = pass == npass - 1;
  const bool level_pass = last && ctrl->sort_level_pass != 0;
  const int64_t span = first ? a.span : R;
  const int64_t ntiles = (span + kSortTile - 1) / kSortTile;
  if (threadIdx.x == 0) S.tile = atomicAdd(&ctrl->tile_ticket[pass], 1u);
  __syncthreads();
  const int64_t tile = S.tile;
  if (tile >= ntiles) return;
  const int64_t smin = ctrl->slack_min;
  const FirstSource f{kSrcStaged, a.stg_slack, a.stg_ready, nullptr, a.span, smin};
  const FinalOut fo{last, a.node_of_pos, a.out_slack, a.stg_route, a.stg_cost, smin,
                    a.order, a.slack, a.route, a.cost};
  radix_tile<uint64_t>(S, f, first, pass, tile, span, R, a.key[(pass + 1) & 1],
                       a.pay[(pass + 1) & 1], a.key[pass & 1], a.pay[pass & 1],
                       ctrl->ghist_slack + pass * kRadixBuckets,
                       a.lookback + int64_t(pass) * a.tiles_cap * kRadixBuckets, a.epoch, fo,
                       level_pass ? a.stg_ready : nullptr);
  if (tile == 0 && threadIdx.x == 0) {
    const int64_t smax = ctrl->slack_max;
    const int nbits = 64 - __builtin_clzll(uint64_t(smax - smin) | 1);
    const uint32_t st = last ? 0u : kStatusContinue;
    if (last || pass == kSortLaunched - 1)
      publish_status(a.host, st, R, nbits, ctrl->hint_min, ctrl->hint_max, ctrl->level_mask);
  }
}

// Grouping by workflow in one digit (at most 256 workflows), without the
// onesweep look-back: its tiles wait on each other in a chain, about 40 ns
// each, which at 12M futures (3,000 tiles) costs more than the data does.
// Three kernels instead, each parallel over tiles or workflows:
//   count  per tile of kSortTile ids, the futures of each workflow
//          (workflow-major, so that a workflow's counts are contiguous);
//   scan   per workflow, its tiles' counts into offsets, and its total;
//   place  per tile, the workflows' starts from the totals, then each
//          future's stable rank in its tile by ballots, its position =
//          start + tile offset + rank, and both maps.
// The counts take the first key buffer, the totals the second.
constexpr int kGroup1Items = kSortTile / kSortThreads;

__global__ __launch_bounds__(kSortThreads) void k_group1_count(GroupArgs a) {
  __shared__ uint32_t H[kRadixBuckets];
  if (a.ctrl->status) return;
  const int64_t N = a.p.N;
  const int64_t ntiles = (N + kSortTile - 1) / kSortTile;
  const int64_t tile = blockIdx.x;
  H[threadIdx.x] = 0;
  __syncthreads();
  const int64_t t0 = tile * kSortTile;
  uint32_t d[kGroup1Items];
#pragma unroll
  for (int j = 0; j < kGroup1Items; ++j) {
    const int64_t i = t0 + j * kSortThreads + threadIdx.x;
    d[j] = i < N ? uint32_t(a.p.wf[i]) & (kRadixBuckets - 1) : kRadixBuckets;
  }
#pragma unroll
  for (int j = 0; j < kGroup1Items; ++j)
    if (d[j] < kRadixBuckets) atomicAdd(&H[d[j]], 1u);
  __syncthreads();
  a.key[0][int64_t(threadIdx.x) * ntiles + tile] = H[threadIdx.x];
}

__global__ __launch_bounds__(kSortThreads) void k_group1_scan(GroupArgs a) {
  __shared__ uint32_t s_tmp[kSortThreads / kWave + 2];
  __shared__ uint32_t s_sum;
  if (a.ctrl->status) return;
  const int64_t ntiles = (a.p.N + kSortTile - 1) / kSortTile;
  uint32_t* row = a.key[0] + int64_t(blockIdx.x) * ntiles;
  uint32_t carry = 0;
  for (int64_t t0 = 0; t0 < ntiles; t0 += kSortThreads) {
    const int64_t t = t0 + threadIdx.x;
    const uint32_t x = t < ntiles ? row[t] : 0u;
    const uint32_t ex = block_excl_scan(x, s_tmp);
    if (t < ntiles) row[t] = carry + ex;
    if (threadIdx.x == kSortThreads - 1) s_sum = ex + x;
    __syncthreads();
    carry += s_sum;
    __syncthreads();
  }
  if (threadIdx.x == 0) a.key[1][blockIdx.x] = carry;
}

__global__ __launch_bounds__(kSortThreads) void k_group1_place(GroupArgs a) {
  __shared__ uint32_t s_tmp[kSortThreads / kWave + 2];
  __shared__ uint32_t base[kRadixBuckets];   // first position of each workflow, then of its part of this tile
  __shared__ uint32_t wcnt[kSortThreads / kWave][kRadixBuckets];  // this round's futures per wave and workflow
  __shared__ uint32_t run[kRadixBuckets];    // this tile's futures per workflow in earlier rounds
  if (a.ctrl->status) return;
  const int64_t N = a.p.N;
  const int64_t ntiles = (N + kSortTile - 1) / kSortTile;
  const int64_t tile = blockIdx.x;
  const int tid = threadIdx.x, wv = tid / kWave;
  {
    const uint32_t tot = a.key[1][tid];
    const uint32_t start = block_excl_scan(tot, s_tmp);
    if (tile == 0 && tid <= a.p.W) a.wf_off[tid] = int32_t(start);
    if (tile == 0 && tid == kSortThreads - 1 && a.p.W == kRadixBuckets) a.wf_off[kRadixBuckets] = int32_t(N);
    base[tid] = start + a.key[0][int64_t(tid) * ntiles + tile];
    run[tid] = 0;
    for (int w = 0; w < kSortThreads / kWave; ++w) wcnt[w][tid] = 0;
  }
  __syncthreads();
  const int64_t t0 = tile * kSortTile;
  for (int j = 0; j < kGroup1Items; ++j) {
    const int64_t i = t0 + j * kSortThreads + tid;
    const bool in = i < N;
    const uint32_t d = in ? uint32_t(a.p.wf[i]) & (kRadixBuckets - 1) : 0u;
    uint64_t m = ballot(in);  // the wave's lanes holding the same workflow
#pragma unroll
    for (int bit = 0; bit < kRadixBits; ++bit) {
      const uint64_t b = ballot(in && ((d >> bit) & 1u));
      m &= ((d >> bit) & 1u) ? b : ~b;
    }
    if (in && lanes_below(m) == 0) wcnt[wv][d] = uint32_t(__popcll(m));
    __syncthreads();
    if (in) {
      uint32_t r = run[d] + lanes_below(m);
      for (int w = 0; w < wv; ++w) r += wcnt[w][d];
      const uint32_t q = base[d] + r;
      a.pay[0][q] = uint32_t(i);
      a.pos_of_node[i] = int32_t(q);
    }
    __syncthreads();
    {
      uint32_t s = 0;
      for (int w = 0; w < kSortThreads / kWave; ++w) {
        s += wcnt[w][tid];
        wcnt[w][tid] = 0;
      }
      run[tid] += s;
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(kSortThreads) void k_group_hist(GroupArgs a) {
  __shared__ uint32_t H[kMaxSortPasses][kRadixBuckets];
  if (a.ctrl->status) return;
  const FirstSource f{kSrcWf, nullptr, nullptr, a.p.wf, a.p.N, 0};
  histogram<uint32_t>(f, a.npass, -1, H, a.ctrl->ghist_group);
}

__global__ __launch_bounds__(kSortThreads) void k_group_pass(GroupArgs a, int pass) {
  __shared__ TileSmem<uint32_t> S;
  Ctrl* ctrl = a.ctrl;
  if (ctrl->status) return;
  const int64_t N = a.p.N;
  const int64_t ntiles = (N + kSortTile - 1) / kSortTile;
  if (threadIdx.x == 0) S.tile = atomicAdd(&ctrl->tile_ticket[kMaxSortPasses + pass], 1u);
  __syncthreads();
  const int64_t tile = S.tile;
  if (tile >= ntiles) return;
  const FirstSource f{kSrcWf, nullptr, nullptr, a.p.wf, N, 0};
  radix_tile<uint32_t>(S, f, pass == 0, pass, tile, N, N, a.key[(pass + 1) & 1],
                       a.pay[(pass + 1) & 1], a.key[pass & 1], a.pay[pass & 1],
                       ctrl->ghist_group + pass * kRadixBuckets,
                       a.lookback + int64_t(pass) * a.tiles_cap * kRadixBuckets, a.epoch,
                       FinalOut{false, nullptr, nullptr, nullptr, nullptr, 0, nullptr, nullptr, nullptr, nullptr});
}

// Position of every node and first position of every workflow.
__global__ __launch_bounds__(kSortThreads) void k_group_finish(GroupArgs a) {
  if (a.ctrl->status) return;
  const int64_t N = a.p.N, W = a.p.W;
  const int fin = (a.npass - 1) & 1;
  const uint32_t* sorted_wf = a.key[fin];
  const uint32_t* sorted_id = a.pay[fin];
  const int64_t stride = int64_t(gridDim.x) * kSortThreads;
  const int64_t g0 = int64_t(blockIdx.x) * kSortThreads + threadIdx.x;
  for (int64_t q = g0; q < N; q += stride) a.pos_of_node[sorted_id[q]] = int32_t(q);
  for (int64_t w = g0; w <= W; w += stride) {
    int64_t lo = 0, hi = N;
    while (lo < hi) {
      const int64_t mid = (lo + hi) >> 1;
      if (int64_t(sorted_wf[mid]) < w) lo = mid + 1; else hi = mid;
    }
    a.wf_off[w] = int32_t(lo);
  }
}

unsigned grid_of(int64_t n, int64_t per, int64_t cap) {
  int64_t b = (n + per - 1) / per;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return unsigned(b);
}

}  // namespace

hipError_t launch_reset(hipStream_t s, Ctrl* c, uint32_t* clear, int64_t n_clear) {
  hipLaunchKernelGGL(k_reset, dim3(grid_of(n_clear, kSortThreads, 256)), dim3(kSortThreads), 0, s, c,
                     clear, n_clear);
  return hipGetLastError();
}

hipError_t launch_bucket_sort(hipStream_t s, const SortArgs& a, const BucketArgs& bk) {
  if (bk.nb >= kBucketLbMin) {
    const int groups = bk.nb / kBucketLbGroup;
    const int per_block = kBucketLbGroup / kWave;
    hipLaunchKernelGGL(k_bucket_totals, dim3((groups + per_block - 1) / per_block), dim3(kBucketLbGroup),
                       0, s, a, bk);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_bucket_sort_lb, dim3(groups), dim3(kBucketLbGroup), 0, s, a, bk);
  } else
    hipLaunchKernelGGL(k_bucket_sort, dim3(bk.nb / kBucketGroup), dim3(kBucketThreads), 0, s, a, bk);
  return hipGetLastError();
}

hipError_t launch_bin_sort(hipStream_t s, const SortArgs& a, const BucketArgs& bk) {
  hipLaunchKernelGGL(k_bin_sort, dim3(bk.nb), dim3(kBinThreads),
                     bin_lds_bytes<kBinThreads / kWave>(kBinCap, a.tie_wf != nullptr), s, a, bk);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || bk.cap <= kBinCap) return e;
  hipLaunchKernelGGL(k_bin_sort_big, dim3(kBinBigGroups), dim3(kBinBigThreads),
                     bin_lds_bytes<kBinBigThreads / kWave>(kBinBigCap, a.tie_wf != nullptr), s, a, bk);
  return hipGetLastError();
}

hipError_t prepare_sort_kernels() {
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_bin_sort),
                                     hipFuncAttributeMaxDynamicSharedMemorySize,
                                     int(bin_lds_bytes<kBinThreads / kWave>(kBinCap, true)));
  if (e != hipSuccess) return e;
  return hipFuncSetAttribute(reinterpret_cast<const void*>(&k_bin_sort_big),
                             hipFuncAttributeMaxDynamicSharedMemorySize,
                             int(bin_lds_bytes<kBinBigThreads / kWave>(kBinBigCap, true)));
}

hipError_t launch_splitters(hipStream_t s, const SortArgs& a) {
  hipLaunchKernelGGL(k_splitters, dim3(1), dim3(kSortThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_slack_sort(hipStream_t s, const SortArgs& a, int first_pass, int last_pass,
                             void (*mark)(void*, const char*), void* ctx) {
  hipError_t e;
  if (first_pass == 0) {
    mark(ctx, "sort_hist");
    hipLaunchKernelGGL(k_slack_hist, dim3(grid_of(a.span, kHistItems * kSortThreads, 256)),
                       dim3(kSortThreads), 0, s, a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  static const char* names[kMaxSortPasses] = {"sort_pass0", "sort_pass1", "sort_pass2",
                                              "sort_pass3", "sort_pass4", "sort_pass5",
                                              "sort_pass6", "sort_pass7", "sort_pass8"};
  for (int ps = first_pass; ps <= last_pass; ++ps) {
    mark(ctx, names[ps]);
    hipLaunchKernelGGL(k_slack_pass, dim3(grid_of(a.span, kSortTile, INT32_MAX)), dim3(kSortThreads),
                       0, s, a, ps);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_group(hipStream_t s, const GroupArgs& a, void (*mark)(void*, const char*),
                        void* ctx) {
  const int64_t ntiles = (a.p.N + kSortTile - 1) / kSortTile;
  if (a.npass == 1 && int64_t(kRadixBuckets) * ntiles <= a.cap_n) {  // at most 256 workflows
    mark(ctx, "group_count");
    hipLaunchKernelGGL(k_group1_count, dim3(ntiles), dim3(kSortThreads), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    mark(ctx, "group_scan");
    hipLaunchKernelGGL(k_group1_scan, dim3(kRadixBuckets), dim3(kSortThreads), 0, s, a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    mark(ctx, "group_place");
    hipLaunchKernelGGL(k_group1_place, dim3(ntiles), dim3(kSortThreads), 0, s, a);
    return hipGetLastError();
  }
  mark(ctx, "group_hist");
  hipLaunchKernelGGL(k_group_hist, dim3(grid_of(a.p.N, kHistItems * kSortThreads, 256)), dim3(kSortThreads), 0, s,
                     a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  for (int ps = 0; ps < a.npass; ++ps) {
    mark(ctx, "group_pass");
    hipLaunchKernelGGL(k_group_pass, dim3(grid_of(a.p.N, kSortTile, INT32_MAX)), dim3(kSortThreads),
                       0, s, a, ps);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  mark(ctx, "group_finish");
  hipLaunchKernelGGL(k_group_finish, dim3(grid_of(a.p.N + a.p.W + 1, kSortThreads, 4096)),
                     dim3(kSortThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace nalar
