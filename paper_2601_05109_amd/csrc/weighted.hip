// Weighted routing (NALAR_ROUTE_WEIGHTED): route with a list of instances and
// weights (Table 2).  After ordering, the ready futures of each type that has
// instances of positive weight are dealt to those instances in proportion to
// their weights: the futures of type t, in output order, take sequence numbers
// j = 0, 1, 2, ...; with the weighted instances of t listed by ascending index,
// w[i] their weights and S their total, future j goes to the instance whose run
// of w[i] consecutive numbers in 0 .. S-1 holds j mod S.
//
// A future's sequence number is its rank among the futures of its type before
// it in the output order, which is a per-type prefix count over the order:
//   k_weighted_table   (one workgroup) the weighted instances sorted by
//                      (type, index) with the weight before each entry inside
//                      its type, the type's total and its first entry (the
//                      type's slot, which names it in the counts below);
//   k_weighted_count   one wavefront per tile of kWTile output positions counts
//                      the tile's futures per slot;
//   k_weighted_scan    one workgroup per slot turns the tile counts into
//                      exclusive prefixes over the tiles;
//   k_weighted_assign  each tile again: every future's rank inside the tile
//                      (in order: 16 steps of 64 positions, lanes of equal slot
//                      ranked by ballots) plus the tile prefix is its sequence
//                      number; the instance whose weight run holds it is found
//                      by a binary search, and route and cost are written.
// Futures pinned by NALAR_ROUTE_STATEFUL and futures of types with no weighted
// instance keep the route the pass gave them.
#include "internal.hpp"

namespace nalar {

namespace {

constexpr int kWThreads = 256;
constexpr int kWWaves = kWThreads / kWave;
constexpr int kWItems = 16;
constexpr int kWTile = kWave * kWItems;   // positions per wavefront tile
constexpr int kWTableThreads = 1024;
constexpr int kSlotBits = 10;             // slots < NALAR_MAX_INSTANCES = 2^10
static_assert((1 << kSlotBits) == NALAR_MAX_INSTANCES, "slot bits");

// The table of weighted instances in LDS (n entries).
struct WTab {
  int32_t type[NALAR_MAX_INSTANCES];
  int32_t idx[NALAR_MAX_INSTANCES];
  uint32_t cum[NALAR_MAX_INSTANCES];   // weight of the type's entries before this one
  uint32_t tot[NALAR_MAX_INSTANCES];   // total weight of the entry's type
  int32_t first[NALAR_MAX_INSTANCES];  // first entry of the entry's type (its slot)
  int32_t cnt[NALAR_MAX_INSTANCES];    // entries of the entry's type
};

// Within one wavefront LDS operations complete in program order; this only
// keeps the compiler from moving LDS accesses across it.
__device__ inline void wave_barrier() { __asm__ __volatile__("" ::: "memory"); }

__global__ __launch_bounds__(kWTableThreads) void k_weighted_table(WeightedArgs g) {
  __shared__ int32_t s_type[NALAR_MAX_INSTANCES];
  __shared__ uint32_t s_w[NALAR_MAX_INSTANCES];
  const int M = g.M;
  bool bad = false;
  for (int i = threadIdx.x; i < M; i += kWTableThreads) {
    s_type[i] = g.inst_type[i];
    const uint32_t w = g.inst_weight[i];
    bad |= w > NALAR_WEIGHT_MAX;
    s_w[i] = bad ? 0u : w;
  }
  if (ballot(bad) != 0 && lane_id() == 0) flag_status(g.ctrl, kStInval);
  __syncthreads();
  int n = 0;
  for (int i = threadIdx.x; i < M; i += kWTableThreads) {
    const uint32_t w = s_w[i];
    const int32_t t = s_type[i];
    int rank = 0, before_type = 0, in_type = 0;
    uint32_t cum = 0, tot = 0;
    for (int j = 0; j < M; ++j) {
      if (s_w[j] == 0) continue;
      const int32_t u = s_type[j];
      rank += (u < t || (u == t && j < i)) ? 1 : 0;
      before_type += u < t ? 1 : 0;
      if (u == t) {
        in_type += 1;
        tot += s_w[j];
        cum += j < i ? s_w[j] : 0u;
      }
    }
    if (w == 0) continue;
    g.wt_type[rank] = t;
    g.wt_idx[rank] = i;
    g.wt_cum[rank] = cum;
    g.wt_tot[rank] = tot;
    g.wt_first[rank] = before_type;
    g.wt_cnt[rank] = in_type;
    n += 1;
  }
  // the number of entries: the weighted instances
  n = int(wave_sum_i64(int64_t(n)));
  __shared__ int s_n[kWTableThreads / kWave];
  if (lane_id() == 0) s_n[threadIdx.x / kWave] = n;
  __syncthreads();
  if (threadIdx.x == 0) {
    int tot = 0;
    for (int w = 0; w < kWTableThreads / kWave; ++w) tot += s_n[w];
    *g.n_wt = tot;
  }
}

__device__ inline void load_table(const WeightedArgs& g, WTab& T, int n) {
  for (int i = threadIdx.x; i < n; i += kWThreads) {
    T.type[i] = g.wt_type[i];
    T.idx[i] = g.wt_idx[i];
    T.cum[i] = g.wt_cum[i];
    T.tot[i] = g.wt_tot[i];
    T.first[i] = g.wt_first[i];
    T.cnt[i] = g.wt_cnt[i];
  }
}

// Slot of type t (its first weighted entry), or -1 without weighted instances.
__device__ inline int slot_of(const WTab& T, int n, int32_t t) {
  int lo = 0, hi = n;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (T.type[mid] < t) lo = mid + 1; else hi = mid;
  }
  return (lo < n && T.type[lo] == t) ? lo : -1;
}

// Slot of the future at output position k, or -1 when it keeps its route.
__device__ inline int slot_at(const WeightedArgs& g, const WTab& T, int n, int64_t k) {
  if (k >= g.R) return -1;
  const int32_t v = g.order[k];
  const int32_t t = g.type[v];
  if (g.stateful) {
    const int32_t l = g.loc[v];
    if (l >= 0 && g.inst_type[l] == t) return -1;
  }
  return slot_of(T, n, t);
}

__global__ __launch_bounds__(kWThreads) void k_weighted_count(WeightedArgs g) {
  __shared__ WTab T;
  __shared__ uint32_t hist[kWWaves][NALAR_MAX_INSTANCES];
  const int n = *g.n_wt;
  const int wv = threadIdx.x / kWave;
  const int ln = lane_id();
  load_table(g, T, n);
  for (int i = ln; i < n; i += kWave) hist[wv][i] = 0;
  __syncthreads();
  const int64_t tile = int64_t(blockIdx.x) * kWWaves + wv;
  if (tile >= g.tiles || n == 0) return;
  const int64_t base = tile * kWTile;
  int sl[kWItems];
#pragma unroll
  for (int j = 0; j < kWItems; ++j) sl[j] = slot_at(g, T, n, base + j * kWave + ln);
#pragma unroll
  for (int j = 0; j < kWItems; ++j)
    if (sl[j] >= 0) atomicAdd(&hist[wv][sl[j]], 1u);
  wave_barrier();
  uint32_t* row = g.counts + tile * NALAR_MAX_INSTANCES;
  for (int i = ln; i < n; i += kWave) row[i] = hist[wv][i];
}

// Exclusive prefix over the tiles of one slot (one workgroup per slot; slots
// that are no type's first entry have no futures and return).
__global__ __launch_bounds__(kWThreads) void k_weighted_scan(WeightedArgs g) {
  __shared__ uint32_t s_part[kWWaves];
  const int s = blockIdx.x;
  if (s >= *g.n_wt || g.wt_first[s] != s) return;
  uint32_t carry = 0;
  for (int64_t t0 = 0; t0 < g.tiles; t0 += kWThreads) {
    const int64_t t = t0 + threadIdx.x;
    const uint32_t c = t < g.tiles ? g.counts[t * NALAR_MAX_INSTANCES + s] : 0u;
    const uint32_t inc = wave_incl_scan_u32(c);
    if (lane_id() == kWave - 1) s_part[threadIdx.x / kWave] = inc;
    __syncthreads();
    uint32_t before = carry;
    uint32_t total = 0;
    for (int w = 0; w < kWWaves; ++w) {
      before += w < int(threadIdx.x / kWave) ? s_part[w] : 0u;
      total += s_part[w];
    }
    if (t < g.tiles) g.counts[t * NALAR_MAX_INSTANCES + s] = before + inc - c;
    carry += total;
    __syncthreads();
  }
}

__global__ __launch_bounds__(kWThreads) void k_weighted_assign(WeightedArgs g) {
  __shared__ WTab T;
  __shared__ uint32_t run[kWWaves][NALAR_MAX_INSTANCES];
  const int n = *g.n_wt;
  const int wv = threadIdx.x / kWave;
  const int ln = lane_id();
  load_table(g, T, n);
  const int64_t tile = int64_t(blockIdx.x) * kWWaves + wv;
  const bool live = tile < g.tiles && n > 0;
  if (live) {
    const uint32_t* row = g.counts + tile * NALAR_MAX_INSTANCES;
    for (int i = ln; i < n; i += kWave) run[wv][i] = row[i];
  }
  __syncthreads();
  if (!live) return;
  const int64_t base = tile * kWTile;
  int sl[kWItems];
#pragma unroll
  for (int j = 0; j < kWItems; ++j) sl[j] = slot_at(g, T, n, base + j * kWave + ln);
#pragma unroll 1
  for (int j = 0; j < kWItems; ++j) {
    // lanes of equal slot, ranked by lane (positions ascend with the lane)
    const bool valid = sl[j] >= 0;
    const uint32_t s = valid ? uint32_t(sl[j]) : 0u;
    uint64_t peers = ballot(valid);
#pragma unroll
    for (int b = 0; b < kSlotBits; ++b) {
      const bool bit = (s >> b) & 1u;
      const uint64_t m = ballot(bit);
      peers &= bit ? m : ~m;
    }
    const uint64_t below = peers & lanemask_lt();
    uint32_t seq = 0;
    if (valid) seq = run[wv][s] + uint32_t(__popcll(below));
    wave_barrier();
    if (valid && below == 0) run[wv][s] += uint32_t(__popcll(peers));
    wave_barrier();
    if (!valid) continue;
    // the entry whose weight run holds seq mod S
    const uint32_t r = seq % T.tot[s];
    int lo = int(s), hi = int(s) + T.cnt[s] - 1;  // last entry with cum <= r
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (T.cum[mid] <= r) lo = mid; else hi = mid - 1;
    }
    const int32_t inst = T.idx[lo];
    const int64_t k = base + j * kWave + ln;
    const int32_t v = g.order[k];
    const int32_t l = g.loc[v];
    g.route[k] = inst;
    if (g.cost)
      g.cost[k] = g.inst_load[inst] + (g.est[v] * 1000) / int64_t(g.inst_speed[inst]) +
                  ((l >= 0 && l != inst) ? g.mig : 0);
  }
}

}  // namespace

int64_t weighted_tiles(int64_t R) { return (R + kWTile - 1) / kWTile; }

hipError_t launch_weighted_table(hipStream_t s, const WeightedArgs& g) {
  if (g.M <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_weighted_table, dim3(1), dim3(kWTableThreads), 0, s, g);
  return hipGetLastError();
}

hipError_t launch_route_weighted(hipStream_t s, const WeightedArgs& g, void (*mark)(void*, const char*),
                                 void* ctx) {
  if (g.M <= 0 || g.R <= 0) return hipSuccess;
  hipError_t e;
  const unsigned blocks = unsigned((g.tiles + kWWaves - 1) / kWWaves);
  mark(ctx, "weighted_count");
  hipLaunchKernelGGL(k_weighted_count, dim3(blocks), dim3(kWThreads), 0, s, g);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  mark(ctx, "weighted_scan");
  hipLaunchKernelGGL(k_weighted_scan, dim3(unsigned(g.M)), dim3(kWThreads), 0, s, g);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  mark(ctx, "weighted_assign");
  hipLaunchKernelGGL(k_weighted_assign, dim3(blocks), dim3(kWThreads), 0, s, g);
  return hipGetLastError();
}

}  // namespace nalar
