// C ABI of the policy pass: handle, scratch arena, launch sequence, status.
//
// A pass is a short sequence of launches on the handle's stream:
//   [reset]  -> only when a control block or bucket counters are stale
//   [nodes]  -> unless the sweep is fused: validate the snapshot, sort the
//               instance table, workflow offsets
//   [group]  -> only when the caller's ids are not grouped by workflow: stable
//               radix sort of the ids by workflow
//   sweep    -> remaining critical path, readiness, order key and routing;
//               in fused mode (contiguous ids, workflows of at most 512
//               futures, at most 128 instances) also validation, workflow
//               bounds, the instance table and the reset of the next pass's
//               control block and bucket counters
//   sort     -> bucketed: the sweep has dropped every ready future into a
//               bucket of a key range planned from the previous pass, and one
//               kernel (two for many buckets) orders each bucket and writes it
//               at its offset; or tiled: key histogram and range, then up to
//               four digit passes.  The last kernel writes the caller's arrays
//               and the status into pinned host memory
//   [greedy] -> NALAR_ROUTE_GREEDY only: routing again in output order
//   [weighted] -> NALAR_ROUTE_WEIGHTED only: the weighted instances are
//               tabulated before the sweep (their weights validated), and the
//               weighted types' futures are dealt out after the sort
// with one stream synchronisation after the sort (and one after greedy or
// weighted routing).  The bucketed sort is used once a previous pass has given a key
// range and at most kBucketMaxReady futures were ready; if a bucket
// overflows, the kernel reports "tiled", and after the synchronisation the
// host resets the control block, sweeps again without buckets and runs the
// tiled sort (then skips the bucketed sort for a few passes).  A key range
// wider than 32 bits reports "continue" from the tiled sort and its remaining
// passes follow after another synchronisation.
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>

#include "internal.hpp"

using namespace nalar;

// The static scratch array of nalar_policy_pass_static (NALAR_STATIC_SCRATCH_BYTES
// per device; see below for how host code reaches it).
static __device__ __align__(256) char scratch[NALAR_STATIC_SCRATCH_BYTES];

namespace {

constexpr int kMaxTimed = 48;

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

int64_t tiles_of(int64_t n) { return (n + kSortTile - 1) / kSortTile + 1; }

// Device scratch, carved from one allocation.
struct Arena {
  void* base = nullptr;
  size_t bytes = 0;
  size_t lookback_off = 0, lookback_bytes = 0;
  Ctrl* ctrl[2] = {nullptr, nullptr};
  ITab itab{};
  int32_t* wf_off = nullptr;
  uint8_t* stg_ready = nullptr;
  int64_t* stg_slack = nullptr;
  int32_t* stg_route = nullptr;
  int64_t* stg_cost = nullptr;
  int64_t* stg_oslack = nullptr;  // slack by position when the order key is not the slack
  uint64_t* skey[2] = {nullptr, nullptr};
  uint32_t* spay[2] = {nullptr, nullptr};
  uint64_t* slb = nullptr;
  uint32_t* gkey[2] = {nullptr, nullptr};
  uint32_t* gpay[2] = {nullptr, nullptr};
  uint64_t* glb = nullptr;
  uint64_t* bagg = nullptr;  // bucket-group totals of the look-back bucket kernel
  int32_t* wt_i32 = nullptr;   // weighted routing: type, idx, first, cnt tables and the entry count
  uint32_t* wt_u32 = nullptr;  // weighted routing: cum, tot tables
  uint32_t* wcounts = nullptr; // weighted routing: per-tile counts
  int32_t* pos_of_node = nullptr;
  int32_t* g_cnt = nullptr;
  int64_t* g_mx = nullptr;
  uint8_t* g_dn = nullptr;
  uint8_t* g_nr = nullptr;
  int32_t* g_front[2] = {nullptr, nullptr};
  uint64_t* done_bits = nullptr;  // [N / 64] the done flags, one bit per future
  uint32_t* bcnt[2] = {nullptr, nullptr};  // bucket counters, by pass parity
  BucketSlot* bslot = nullptr;
  int64_t* split[2] = {nullptr, nullptr};   // bin splitters: read by one pass, written for the next
  int64_t capN = -1, capW = -1, capB = -1, capRec = -1;
};

// The scratch a pass runs in: an arena and the state of what it holds (the
// look-back tag of the last pass, the control block the next pass uses, and
// which control blocks and bucket counters are stale).
struct ArenaState {
  Arena ar;
  // the ordered HBM sweep's log of pushes into earlier chunks (one entry per
  // dependency at most): allocated apart from the arena, for this handle's
  // own passes only (null for the static scratch)
  void* plog = nullptr;
  int64_t plog_cap = 0;
  uint32_t epoch = 0;
  uint64_t passes = 0;                 // selects the control block of the next pass
  bool ctrl_dirty[2] = {true, true};
  bool bcnt_clean[2] = {true, true};   // bucket counters known to be zero
};

// Scratch of nalar_policy_pass_static: one fixed array per device, laid out
// once for the largest snapshot it takes.  `scratch` names the array only in
// device code; host code uses the address hipGetSymbolAddress returns for it
// on each device (kept in g_static), never the name.
constexpr size_t kStaticScratchBytes = size_t(NALAR_STATIC_SCRATCH_BYTES);
constexpr int64_t kStaticBuckets = 16384;
constexpr int kMaxDevices = 64;

struct StaticScratch {
  std::mutex mu;          // serialises the calls on this device
  bool ready = false;     // address resolved and arena laid out
  bool cleared = false;   // look-back words untagged
  ArenaState st;
};

StaticScratch g_static[kMaxDevices];

}  // namespace

struct nalar_policy {
  int device = 0;
  uint32_t flags = 0;
  hipStream_t stream = nullptr;
  int cus = 0;
  size_t lds_limit = 0;
  // slack range and ready count of the last successful pass (bucket hint)
  bool hint_valid = false;
  int64_t hint_ready = 0, hint_min = 0, hint_max = 0;
  uint32_t hint_levels = 0;      // priority levels of the previous pass (bit l: level l)
  int bucket_skip = 0;           // passes left before the bucketed sort is tried again
  int bucket_backoff = 1;
  int bucket_dense = 0;          // buckets doubled this many times (overflows: up to 3, crowding: 4)
  int bucket_calm = 0;           // bucketed passes without overflow since the last change
  int bucket_relax = 64;         // calm passes before fewer buckets are tried again
  bool bucket_relaxed = false;   // the last pass tried fewer buckets
  int split_nb = 0;              // bins the current splitters are for (0: none)
  int split_cur = 0;             // the splitter buffer the next pass reads
  int bin_skip = 0;              // passes left before bins are tried again
  int bin_backoff = 1;
  bool split_any = false;        // splitters for any ready count, any sweep (graph store)
  uint32_t bin_max = 0;          // records in the largest bin of the last bin sort (0: unknown)
  std::string err;
  ArenaState own;                // scratch allocated by the library for this handle
  HostStatus* host = nullptr;    // pinned, written by the sort kernel
  bool timing = false;
  int n_timed = 0;
  bool timed_valid = false;
  hipEvent_t ev[kMaxTimed + 1] = {};
  const char* names[kMaxTimed] = {};
  float ms[kMaxTimed] = {};
};

namespace {

thread_local std::string g_create_error;

int fail(nalar_policy* h, int code, const std::string& msg) {
  if (h) h->err = msg;
  return code;
}

int hip_fail(nalar_policy* h, hipError_t e, const char* what) {
  std::string m = std::string(what) + ": " + hipGetErrorString(e);
  return fail(h, e == hipErrorOutOfMemory ? NALAR_ENOMEM : NALAR_EDEVICE, m);
}

// Lay out (or measure, when base is null) the arena for the given capacities.
size_t carve(Arena& a, char* base, int64_t N, int64_t W, int64_t B, int64_t Rec) {
  size_t off = 0;
  auto take = [&](size_t bytes) {
    off = align_up(off, 256);
    char* p = base ? base + off : nullptr;
    off += bytes;
    return p;
  };
  const int64_t n1 = N > 0 ? N : 1;
  const int64_t w1 = W > 0 ? W : 1;
  const int64_t tiles = tiles_of(n1);
  a.ctrl[0] = reinterpret_cast<Ctrl*>(take(sizeof(Ctrl)));
  a.ctrl[1] = reinterpret_cast<Ctrl*>(take(sizeof(Ctrl)));
  a.itab.load = reinterpret_cast<int64_t*>(take(8 * NALAR_MAX_INSTANCES));
  a.itab.inv_speed = reinterpret_cast<double*>(take(8 * NALAR_MAX_INSTANCES));
  a.itab.type = reinterpret_cast<int32_t*>(take(4 * NALAR_MAX_INSTANCES));
  a.itab.idx = reinterpret_cast<int32_t*>(take(4 * NALAR_MAX_INSTANCES));
  a.itab.speed = reinterpret_cast<int32_t*>(take(4 * NALAR_MAX_INSTANCES));
  a.itab.pos_of = reinterpret_cast<int32_t*>(take(4 * NALAR_MAX_INSTANCES));
  a.itab.run = reinterpret_cast<uint32_t*>(take(4 * kTypeDirect));
  a.itab.prun = reinterpret_cast<uint32_t*>(take(4 * kTypeDirect));
  a.wf_off = reinterpret_cast<int32_t*>(take(4 * size_t(w1 + 1)));
  a.stg_slack = reinterpret_cast<int64_t*>(take(8 * size_t(n1)));
  a.stg_cost = reinterpret_cast<int64_t*>(take(8 * size_t(n1)));
  a.stg_route = reinterpret_cast<int32_t*>(take(4 * size_t(n1)));
  a.stg_ready = reinterpret_cast<uint8_t*>(take(size_t(n1)));
  a.stg_oslack = reinterpret_cast<int64_t*>(take(8 * size_t(n1)));
  for (int i = 0; i < 2; ++i) a.skey[i] = reinterpret_cast<uint64_t*>(take(8 * size_t(n1)));
  for (int i = 0; i < 2; ++i) a.spay[i] = reinterpret_cast<uint32_t*>(take(4 * size_t(n1)));
  for (int i = 0; i < 2; ++i) a.gkey[i] = reinterpret_cast<uint32_t*>(take(4 * size_t(n1)));
  for (int i = 0; i < 2; ++i) a.gpay[i] = reinterpret_cast<uint32_t*>(take(4 * size_t(n1)));
  a.pos_of_node = reinterpret_cast<int32_t*>(take(4 * size_t(n1)));
  a.g_mx = reinterpret_cast<int64_t*>(take(8 * size_t(n1)));
  a.g_cnt = reinterpret_cast<int32_t*>(take(4 * size_t(n1)));
  for (int i = 0; i < 2; ++i) a.g_front[i] = reinterpret_cast<int32_t*>(take(4 * size_t(n1)));
  a.g_dn = reinterpret_cast<uint8_t*>(take(size_t(n1)));
  a.g_nr = reinterpret_cast<uint8_t*>(take(size_t(n1)));
  a.done_bits = reinterpret_cast<uint64_t*>(take(8 * size_t((n1 + 63) / 64)));
  const int64_t b1 = B > 0 ? B : 0;
  for (int i = 0; i < 2; ++i) a.bcnt[i] = reinterpret_cast<uint32_t*>(take(4 * size_t(b1 + 1)));
  const int64_t r1 = Rec > b1 * kBucketCap ? Rec : b1 * kBucketCap;
  a.bslot = reinterpret_cast<BucketSlot*>(take(sizeof(BucketSlot) * size_t(r1)));
  for (int i = 0; i < 2; ++i) a.split[i] = reinterpret_cast<int64_t*>(take(8 * size_t(kBinMax)));
  off = align_up(off, 256);
  a.lookback_off = off;
  a.slb = reinterpret_cast<uint64_t*>(take(8 * size_t(kMaxSortPasses) * tiles * kRadixBuckets));
  a.glb = reinterpret_cast<uint64_t*>(take(8 * size_t(kMaxGroupPasses) * tiles * kRadixBuckets));
  a.bagg = reinterpret_cast<uint64_t*>(take(8 * size_t(kBucketLbGroups)));
  a.lookback_bytes = off - a.lookback_off;
  a.wt_i32 = reinterpret_cast<int32_t*>(take(4 * size_t(4 * NALAR_MAX_INSTANCES + 1)));
  a.wt_u32 = reinterpret_cast<uint32_t*>(take(4 * size_t(2 * NALAR_MAX_INSTANCES)));
  a.wcounts = reinterpret_cast<uint32_t*>(take(4 * size_t(weighted_tiles(n1)) * NALAR_MAX_INSTANCES));
  return align_up(off, 256);
}

int ensure_capacity(nalar_policy* h, int64_t N, int64_t W, int64_t B, int64_t Rec) {
  Arena& a = h->own.ar;
  if (a.base && N <= a.capN && W <= a.capW && B <= a.capB && Rec <= a.capRec) return NALAR_OK;
  int64_t newN = a.capN > N ? a.capN : N;
  int64_t newW = a.capW > W ? a.capW : W;
  int64_t newB = a.capB > B ? a.capB : B;
  int64_t newRec = a.capRec > Rec ? a.capRec : Rec;
  int64_t keep_split[kBinMax];  // the current splitters move to the new arena
  if (a.base) {  // grow geometrically so a slowly growing graph (or ready set) reallocates rarely
    if (N > a.capN) newN = N + N / 4;
    if (W > a.capW) newW = W + W / 4;
    if (B > a.capB) newB = B + B / 4;
    if (Rec > a.capRec) newRec = Rec + Rec / 4;
    hipError_t e = hipStreamSynchronize(h->stream);
    if (e != hipSuccess) return hip_fail(h, e, "hipStreamSynchronize");
    if (h->split_nb > 0) {
      e = hipMemcpy(keep_split, a.split[h->split_cur], sizeof(int64_t) * size_t(h->split_nb - 1),
                    hipMemcpyDeviceToHost);
      if (e != hipSuccess) h->split_nb = 0;
    }
    (void)hipFree(a.base);
    a.base = nullptr;
  } else {
    h->split_nb = 0;
  }
  Arena fresh;
  const size_t bytes = carve(fresh, nullptr, newN, newW, newB, newRec);
  void* p = nullptr;
  hipError_t e = hipMalloc(&p, bytes);
  if (e != hipSuccess) {
    a.capN = a.capW = a.capB = -1;
    return hip_fail(h, e, "hipMalloc(scratch)");
  }
  e = hipMemset(p, 0, bytes);  // look-back words must start untagged
  if (e != hipSuccess) {
    (void)hipFree(p);
    return hip_fail(h, e, "hipMemset(scratch)");
  }
  carve(fresh, static_cast<char*>(p), newN, newW, newB, newRec);
  fresh.base = p;
  fresh.bytes = bytes;
  fresh.capN = newN;
  fresh.capW = newW;
  fresh.capB = newB;
  fresh.capRec = newRec;
  if (h->split_nb > 0) {
    e = hipMemcpy(fresh.split[h->split_cur], keep_split, sizeof(int64_t) * size_t(h->split_nb - 1),
                  hipMemcpyHostToDevice);
    if (e != hipSuccess) h->split_nb = 0;
  }
  h->own.ar = fresh;
  h->own.epoch = 0;
  h->own.ctrl_dirty[0] = h->own.ctrl_dirty[1] = true;
  h->own.bcnt_clean[0] = h->own.bcnt_clean[1] = true;
  return NALAR_OK;
}

// Buckets for this pass from the previous pass's ready count and key range
// (nb == 0: use the tiled sort).  With priority levels the buckets form one
// group per level between the lowest and the highest level seen, each spread
// over the range of the key within its level; only the one-wave-per-workflow
// sweep maps keys to level groups, so with the block sweep levels take the
// tiled sort.
BucketArgs plan_buckets(const nalar_policy* h, int64_t N, bool levels, bool wave_sweep) {
  BucketArgs bk{};
  if ((h->flags & NALAR_FORCE_TILED_SORT) || !h->hint_valid || h->bucket_skip > 0 || N == 0 ||
      h->hint_ready > kBucketMaxReady || (levels && (h->hint_levels == 0 || !wave_sweep)))
    return bk;
  int groups = 1, lvl_hi = 0;
  if (levels) {
    const int l0 = __builtin_ctz(h->hint_levels);
    lvl_hi = 31 - __builtin_clz(h->hint_levels);
    groups = lvl_hi - l0 + 1;
  }
  // about two futures per bucket, four for large ready sets (fewer buckets to
  // scan and clear; the 64 slots of a bucket still leave ample headroom)
  // after an overflow (keys crowded into a few buckets, e.g. a long-tailed
  // key), later passes try twice, four or eight times as many buckets
  const int64_t per = h->hint_ready <= kBucketDense ? 2 : 4;
  int64_t nb = kBucketMin;
  while (nb < kBucketMax && nb * per <= h->hint_ready) nb *= 2;
  for (int i = 0; i < h->bucket_dense && nb < kBucketMax; ++i) nb *= 2;
  // per level group: a power of two, at least one small-kernel group of
  // buckets, all groups together within kBucketMax
  int64_t nbl = kBucketGroup;
  while (nbl * groups < nb && nbl * 2 * groups <= kBucketMax) nbl *= 2;
  int lognb = 0;
  while ((int64_t(1) << lognb) < nbl) ++lognb;
  const uint64_t range = uint64_t(h->hint_max) - uint64_t(h->hint_min);
  const int bits = range ? 64 - __builtin_clzll(range) : 0;
  bk.lo = h->hint_min;
  bk.shift = bits > lognb ? bits - lognb : 0;
  bk.nb = int32_t(nbl * groups);
  if (levels) {
    bk.lvl_hi = lvl_hi;
    bk.ngroups = int16_t(groups);
    bk.lshift = int16_t(lognb);
  }
  return bk;
}

// Bins for this pass (the block sweep of a large ready set, splitters from the
// previous pass of this handle; bins == 0: not used).
// Records per bin for a full pass: one workgroup's LDS worth (kBinCap, one
// sort launch) when the largest bin of the last bin sort left a third of that
// to spare, else room for eight times the average bin (the large-bin kernel
// sorts the bins above kBinCap).  A bin past its capacity is an overflow: the
// pass sorts again another way, and the next plan is the roomy one.  (The
// store's incremental passes always plan the roomy bins: the keys of the
// futures they recompute move between passes.)
int bin_cap_plan(const nalar_policy* h, int nb) {
  if (h->bin_max > 0 && h->bin_max + h->bin_max / 2 + 128 <= uint32_t(kBinCap)) return kBinCap;
  return bin_cap_for(h->hint_ready, nb);
}

BucketArgs plan_bins(const nalar_policy* h, const SweepShape& sh, bool levels) {
  BucketArgs bk{};
  if ((h->flags & NALAR_FORCE_TILED_SORT) || sh.wave_path || levels || h->split_nb <= 0 ||
      !h->hint_valid || h->hint_ready < kBinMinReady || h->bin_skip > 0 ||
      (h->split_nb & (h->split_nb - 1)) != 0)  // bins_for gives powers of two
    return bk;
  bk.bins = 1;
  bk.nb = h->split_nb;
  bk.cap = bin_cap_plan(h, bk.nb);
  return bk;
}

int64_t records_of(const BucketArgs& bk) {
  return bk.bins ? int64_t(bk.nb) * bk.cap : int64_t(bk.nb) * kBucketCap;
}

bool in_range(int64_t v, int64_t lo, int64_t hi) { return v >= lo && v <= hi; }

int check_snapshot(nalar_policy* h, const nalar_problem* p) {
  if (!p) return fail(h, NALAR_EINVAL, "NULL problem");
  const int64_t N = p->n_nodes, E = p->n_edges, W = p->n_workflows, M = p->n_instances;
  if (!in_range(N, 0, NALAR_MAX_NODES)) return fail(h, NALAR_EINVAL, "n_nodes out of range");
  if (!in_range(E, 0, NALAR_MAX_EDGES)) return fail(h, NALAR_EINVAL, "n_edges out of range");
  if (!in_range(W, 0, NALAR_MAX_WORKFLOWS)) return fail(h, NALAR_EINVAL, "n_workflows out of range");
  if (!in_range(M, 0, NALAR_MAX_INSTANCES)) return fail(h, NALAR_EINVAL, "n_instances out of range");
  if (!in_range(p->now_us, -NALAR_HORIZON_MAX, NALAR_HORIZON_MAX))
    return fail(h, NALAR_EINVAL, "now_us out of range");
  if (!in_range(p->migration_cost_us, 0, NALAR_MIG_MAX))
    return fail(h, NALAR_EINVAL, "migration_cost_us out of range");
  if ((p->flags & ~(NALAR_WF_CONTIGUOUS | NALAR_ORDER_LPT | NALAR_ORDER_SRTF | NALAR_ROUTE_STATEFUL |
                    NALAR_ROUTE_GREEDY | NALAR_ROUTE_WEIGHTED)) != 0 ||
      p->reserved != 0)
    return fail(h, NALAR_EINVAL, "unknown problem flags");
  if ((p->flags & NALAR_ORDER_LPT) && (p->flags & NALAR_ORDER_SRTF))
    return fail(h, NALAR_EINVAL, "NALAR_ORDER_LPT and NALAR_ORDER_SRTF together");
  if ((p->flags & NALAR_ROUTE_GREEDY) && (p->flags & NALAR_ROUTE_WEIGHTED))
    return fail(h, NALAR_EINVAL, "NALAR_ROUTE_GREEDY and NALAR_ROUTE_WEIGHTED together");
  if ((p->flags & NALAR_ROUTE_WEIGHTED) && M > 0 && !p->inst_weight)
    return fail(h, NALAR_EINVAL, "NALAR_ROUTE_WEIGHTED without inst_weight");
  if (N == 0 && E != 0) return fail(h, NALAR_EINVAL, "edges without nodes");
  if (N > 0 && (!p->wf || !p->type || !p->est_us || !p->done || !p->loc || !p->dep_off))
    return fail(h, NALAR_EINVAL, "NULL node array");
  if (E > 0 && !p->dep_idx) return fail(h, NALAR_EINVAL, "NULL dep_idx");
  if (W > 0 && !p->deadline_us) return fail(h, NALAR_EINVAL, "NULL deadline_us");
  if (W == 0 && p->wf_priority) return fail(h, NALAR_EINVAL, "wf_priority without workflows");
  if (M > 0 && (!p->inst_type || !p->inst_load_us || !p->inst_speed_permille))
    return fail(h, NALAR_EINVAL, "NULL instance array");
  return NALAR_OK;
}

int check_problem(nalar_policy* h, const nalar_problem* p, const nalar_result* r) {
  if (!p || !r) return fail(h, NALAR_EINVAL, "NULL problem or result");
  const int rc = check_snapshot(h, p);
  if (rc != NALAR_OK) return rc;
  if (p->n_nodes > 0 && (!r->order || !r->slack_us || !r->route))
    return fail(h, NALAR_EINVAL, "NULL output array");
  return NALAR_OK;
}

ProblemDev device_view(const nalar_problem* p, uint32_t policy) {
  return ProblemDev{p->n_nodes, p->n_edges, p->n_workflows, p->n_instances, p->now_us,
                    p->migration_cost_us, policy, 0u, p->wf, p->type, p->est_us, p->done, p->loc,
                    p->dep_off, p->dep_idx, p->deadline_us, p->inst_type, p->inst_load_us,
                    p->inst_speed_permille, p->wf_priority, p->inst_weight};
}

struct Timer {
  nalar_policy* h;
  int n = 0;
  void mark(const char* name) {
    if (!h->timing || n >= kMaxTimed) return;
    (void)hipEventRecord(h->ev[n], h->stream);
    h->names[n] = name;
    ++n;
  }
  static void cb(void* self, const char* name) { static_cast<Timer*>(self)->mark(name); }
  void end() {
    if (!h->timing) return;
    (void)hipEventRecord(h->ev[n < kMaxTimed ? n : kMaxTimed], h->stream);
  }
};

}  // namespace

hipStream_t nalar::policy_stream(const nalar_policy* h) { return h->stream; }
int nalar::policy_device(const nalar_policy* h) { return h->device; }
int nalar::policy_fail(nalar_policy* h, int code, const char* msg) { return fail(h, code, msg); }

extern "C" {

int nalar_policy_create(const nalar_policy_config* cfg, nalar_policy** out) {
  g_create_error.clear();
  if (out) *out = nullptr;
  if (!cfg || !out) {
    g_create_error = "NULL config or output";
    return NALAR_EINVAL;
  }
  if ((cfg->flags & ~(NALAR_FORCE_GLOBAL_SWEEP | NALAR_FORCE_TILED_SORT | NALAR_FORCE_LEVEL_SWEEP)) != 0 || cfg->reserve_nodes < 0 ||
      cfg->reserve_edges < 0 || cfg->reserve_workflows < 0 ||
      cfg->reserve_nodes > NALAR_MAX_NODES || cfg->reserve_workflows > NALAR_MAX_WORKFLOWS) {
    g_create_error = "invalid config";
    return NALAR_EINVAL;
  }
  nalar_policy* h = new (std::nothrow) nalar_policy();
  if (!h) {
    g_create_error = "out of host memory";
    return NALAR_ENOMEM;
  }
  h->device = cfg->device;
  h->flags = cfg->flags;
  h->stream = static_cast<hipStream_t>(cfg->stream);
  auto bail = [&](hipError_t e, const char* what) {
    g_create_error = std::string(what) + ": " + hipGetErrorString(e);
    nalar_policy_destroy(h);
    return e == hipErrorOutOfMemory ? NALAR_ENOMEM : NALAR_EDEVICE;
  };
  hipError_t e = hipSetDevice(h->device);
  if (e != hipSuccess) return bail(e, "hipSetDevice");
  hipDeviceProp_t prop;
  e = hipGetDeviceProperties(&prop, h->device);
  if (e != hipSuccess) return bail(e, "hipGetDeviceProperties");
  h->cus = prop.multiProcessorCount;
  h->lds_limit = prop.sharedMemPerBlock;
  if (h->device < 0 || h->device >= kMaxDevices) {
    g_create_error = "device ordinal beyond the library's limit";
    nalar_policy_destroy(h);
    return NALAR_EINVAL;
  }
  {  // the static scratch of this device: resolve its address once
    StaticScratch& ss = g_static[h->device];
    std::lock_guard<std::mutex> lock(ss.mu);
    if (!ss.ready) {
      void* ptr = nullptr;
      e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
      if (e != hipSuccess) return bail(e, "hipGetSymbolAddress(scratch)");
      Arena& a = ss.st.ar;
      const size_t need = carve(a, nullptr, NALAR_STATIC_MAX_NODES, NALAR_STATIC_MAX_WORKFLOWS, kStaticBuckets, 0);
      if (need > kStaticScratchBytes) {
        g_create_error = "static scratch layout exceeds its array";
        nalar_policy_destroy(h);
        return NALAR_EDEVICE;
      }
      carve(a, static_cast<char*>(ptr), NALAR_STATIC_MAX_NODES, NALAR_STATIC_MAX_WORKFLOWS, kStaticBuckets, 0);
      a.base = ptr;
      a.bytes = need;
      a.capN = NALAR_STATIC_MAX_NODES;
      a.capW = NALAR_STATIC_MAX_WORKFLOWS;
      a.capB = kStaticBuckets;
      a.capRec = int64_t(kStaticBuckets) * kBucketCap;
      ss.st.bcnt_clean[0] = ss.st.bcnt_clean[1] = false;  // cleared by the first pass
      ss.ready = true;
    }
  }
  e = prepare_sweep_kernels(h->lds_limit);
  if (e != hipSuccess) return bail(e, "hipFuncSetAttribute");
  e = prepare_sort_kernels();
  if (e != hipSuccess) return bail(e, "hipFuncSetAttribute(sort)");
  e = prepare_inc_kernels();
  if (e != hipSuccess) return bail(e, "hipFuncSetAttribute(incremental)");
  e = hipHostMalloc(reinterpret_cast<void**>(&h->host), sizeof(HostStatus), hipHostMallocCoherent);
  if (e != hipSuccess) return bail(e, "hipHostMalloc");
  for (int i = 0; i <= kMaxTimed; ++i) {
    e = hipEventCreate(&h->ev[i]);
    if (e != hipSuccess) return bail(e, "hipEventCreate");
  }
  int rc = ensure_capacity(h, cfg->reserve_nodes, cfg->reserve_workflows, 0, 0);
  if (rc != NALAR_OK) {
    g_create_error = h->err;
    nalar_policy_destroy(h);
    return rc;
  }
  *out = h;
  return NALAR_OK;
}

void nalar_policy_destroy(nalar_policy* h) {
  if (!h) return;
  (void)hipSetDevice(h->device);
  (void)hipStreamSynchronize(h->stream);
  if (h->own.ar.base) (void)hipFree(h->own.ar.base);
  if (h->own.plog) (void)hipFree(h->own.plog);
  if (h->host) (void)hipHostFree(h->host);
  for (int i = 0; i <= kMaxTimed; ++i)
    if (h->ev[i]) (void)hipEventDestroy(h->ev[i]);
  delete h;
}

const char* nalar_policy_last_error(const nalar_policy* h) {
  return h ? h->err.c_str() : g_create_error.c_str();
}

int nalar_policy_set_timing(nalar_policy* h, int enable) {
  if (!h) return NALAR_EINVAL;
  h->timing = enable != 0;
  h->timed_valid = false;
  return NALAR_OK;
}

int nalar_policy_get_timing(const nalar_policy* h, const char** names, float* ms, int cap,
                            int* count) {
  if (!h || !h->timing || !h->timed_valid || cap < 0 || !count) return NALAR_EINVAL;
  *count = h->n_timed;
  for (int i = 0; i < h->n_timed && i < cap; ++i) {
    if (names) names[i] = h->names[i];
    if (ms) ms[i] = h->ms[i];
  }
  return NALAR_OK;
}

int nalar_policy_decide(nalar_policy* h, const nalar_problem* p, const nalar_view* view,
                        int64_t n_events, const int32_t* events, nalar_decisions* out) {
  if (!h) return NALAR_EINVAL;
  h->err.clear();
  h->timed_valid = false;
  int rc = check_snapshot(h, p);
  if (rc != NALAR_OK) return rc;
  if (p->flags & (NALAR_ROUTE_GREEDY | NALAR_ROUTE_WEIGHTED))
    return fail(h, NALAR_EINVAL, "decide: greedy and weighted routing need a whole order");
  if (!view || !out || n_events < 0) return fail(h, NALAR_EINVAL, "decide: NULL view or output");
  if (n_events == 0) return NALAR_OK;
  const int64_t N = p->n_nodes;
  if (view->n_order < 0 || view->n_order > N) return fail(h, NALAR_EINVAL, "decide: n_order out of range");
  if (!events || !out->slack_us || !out->route || !view->rem_us ||
      (view->n_order > 0 && (!view->order || !view->slack_us)))
    return fail(h, NALAR_EINVAL, "decide: NULL array");
  if (n_events > INT32_MAX) return fail(h, NALAR_EINVAL, "decide: too many events");
  hipError_t e = hipSetDevice(h->device);
  if (e != hipSuccess) return hip_fail(h, e, "hipSetDevice");
  const uint32_t policy = p->flags & (NALAR_ORDER_LPT | NALAR_ORDER_SRTF | NALAR_ROUTE_STATEFUL);
  DecideArgs a{device_view(p, policy), view->rem_us, view->order, view->slack_us, view->n_order,
               events, n_events, out->slack_us, out->route, out->cost_us, out->rank, h->host};
  __atomic_store_n(&h->host->aux_status, 0u, __ATOMIC_RELEASE);
  e = launch_decide(h->stream, a);
  if (e != hipSuccess) return hip_fail(h, e, "decide");
  e = hipStreamSynchronize(h->stream);
  if (e != hipSuccess) return hip_fail(h, e, "hipStreamSynchronize");
  if (__atomic_load_n(&h->host->aux_status, __ATOMIC_ACQUIRE) & kStInval)
    return fail(h, NALAR_EINVAL, "decide: an event id is out of range");
  return NALAR_OK;
}

}  // extern "C"

namespace {

// Zero the look-back words of an arena (a fill kernel rather than a memset, so
// that a caller may capture the pass into a graph).
hipError_t clear_lookback(hipStream_t s, const Arena& A) {
  return launch_reset(s, nullptr, reinterpret_cast<uint32_t*>(static_cast<char*>(A.base) + A.lookback_off),
                      int64_t(A.lookback_bytes / 4));
}

// The push log of the ordered HBM sweep, for E dependencies (grown by a
// quarter beyond the need, like the arena).
int ensure_push_log(nalar_policy* h, int64_t E) {
  ArenaState& as = h->own;
  if (E <= as.plog_cap) return NALAR_OK;
  const int64_t cap = E + E / 4;
  hipError_t e = hipStreamSynchronize(h->stream);
  if (e != hipSuccess) return hip_fail(h, e, "hipStreamSynchronize");
  if (as.plog) (void)hipFree(as.plog);
  as.plog = nullptr;
  as.plog_cap = 0;
  e = hipMalloc(&as.plog, size_t(cap) * (sizeof(int32_t) + sizeof(int64_t)) + 256);
  if (e != hipSuccess) {
    as.plog = nullptr;
    return hip_fail(h, e, "hipMalloc push log");
  }
  as.plog_cap = cap;
  return NALAR_OK;
}

// The pass proper, in the scratch of `as` (sized for the snapshot and for the
// buckets of bk), after the checks of the entry point.
// own_splitters: the arena belongs to the handle, so the bin splitters it
// holds are this handle's (bins and their splitters are used only then).
int run_pass(nalar_policy* h, const nalar_problem* p, nalar_result* r, ArenaState& as, BucketArgs bk,
             const SweepShape& sh, bool own_splitters) {
  hipError_t e;
  const int64_t N = p->n_nodes, W = p->n_workflows, M = p->n_instances;
  Arena& A = as.ar;
  hipStream_t s = h->stream;
  const int cur = int(as.passes & 1);
  const int nxt = cur ^ 1;
  bk.cnt = A.bcnt[cur];
  bk.slot = A.bslot;
  if (bk.bins) bk.split = A.split[h->split_cur];
  Ctrl* ctrl = A.ctrl[cur];
  // the next pass's splitters: after the sort, from its output (block sweep,
  // no priority levels, the handle's own arena)
  const bool want_split = own_splitters && (!sh.wave_path || h->split_any) && !p->wf_priority;

  as.epoch = (as.epoch + 1) & kEpochMask;
  if (as.epoch == 0) {  // tags wrapped: forget every old look-back word
    e = clear_lookback(s, A);
    if (e != hipSuccess) return hip_fail(h, e, "clear look-back");
    as.epoch = 1;
  }
  const uint32_t epoch = as.epoch;
  // This pass uses block `cur` (reset first if an earlier pass left it stale)
  // and its sort kernel resets block `nxt`; until that has run, both are stale.
  const bool need_reset = as.ctrl_dirty[cur];
  as.ctrl_dirty[cur] = true;
  as.ctrl_dirty[nxt] = true;

  const uint32_t policy = p->flags & (NALAR_ORDER_LPT | NALAR_ORDER_SRTF | NALAR_ROUTE_STATEFUL |
                                      NALAR_ROUTE_GREEDY | NALAR_ROUTE_WEIGHTED);
  const ProblemDev pd = device_view(p, policy);
  const bool contiguous = (p->flags & NALAR_WF_CONTIGUOUS) != 0 || W <= 1;

  Timer tm{h};
#define NALAR_LAUNCH(name, call)                            \
  do {                                                      \
    tm.mark(name);                                          \
    hipError_t le_ = (call);                                \
    if (le_ != hipSuccess) return hip_fail(h, le_, name);   \
  } while (0)

  // bucket counters of this pass: zeroed by the previous pass's sweep, else here
  const bool need_clear = bk.nb > 0 && !as.bcnt_clean[cur];
  if (need_reset || need_clear)
    NALAR_LAUNCH("reset", launch_reset(s, need_reset ? ctrl : nullptr, bk.cnt, need_clear ? bk.nb : 0));
  if (bk.nb > 0) as.bcnt_clean[cur] = false;
  WeightedArgs wa{};
  if (policy & NALAR_ROUTE_WEIGHTED) {
    wa.type = p->type;
    wa.est = p->est_us;
    wa.loc = p->loc;
    wa.inst_type = p->inst_type;
    wa.inst_load = p->inst_load_us;
    wa.inst_speed = p->inst_speed_permille;
    wa.inst_weight = p->inst_weight;
    wa.M = int32_t(M);
    wa.stateful = (policy & NALAR_ROUTE_STATEFUL) ? 1 : 0;
    wa.mig = p->migration_cost_us;
    wa.route = r->route;
    wa.cost = r->cost_us;
    wa.ctrl = ctrl;
    wa.wt_type = A.wt_i32;
    wa.wt_idx = A.wt_i32 + NALAR_MAX_INSTANCES;
    wa.wt_first = A.wt_i32 + 2 * NALAR_MAX_INSTANCES;
    wa.wt_cnt = A.wt_i32 + 3 * NALAR_MAX_INSTANCES;
    wa.n_wt = A.wt_i32 + 4 * NALAR_MAX_INSTANCES;
    wa.wt_cum = A.wt_u32;
    wa.wt_tot = A.wt_u32 + NALAR_MAX_INSTANCES;
    wa.counts = A.wcounts;
    NALAR_LAUNCH("weighted_table", launch_weighted_table(s, wa));
  }
  const bool fused = N > 0 && sweep_can_fuse(sh, M, contiguous);
  if (!fused)
    NALAR_LAUNCH("nodes", launch_nodes(s, pd, ctrl, A.ctrl[nxt], A.itab, A.wf_off, contiguous ? 1 : 0, 0,
                                       sh.wave_path ? nullptr : A.done_bits));

  const int32_t* node_of_pos = nullptr;
  const int32_t* pos_of_node = nullptr;
  if (N > 0 && !contiguous) {
    int bits = 0;
    while ((int64_t(1) << bits) < W) ++bits;
    GroupArgs g{};
    g.p = pd;
    g.ctrl = ctrl;
    g.npass = (bits + kRadixBits - 1) / kRadixBits;
    for (int i = 0; i < 2; ++i) {
      g.key[i] = A.gkey[i];
      g.pay[i] = A.gpay[i];
    }
    g.lookback = A.glb;
    g.tiles_cap = tiles_of(A.capN);
    g.epoch = epoch;
    g.pos_of_node = A.pos_of_node;
    g.wf_off = A.wf_off;
    g.cap_n = A.capN > 0 ? A.capN : 1;
    e = launch_group(s, g, Timer::cb, &tm);
    if (e != hipSuccess) return hip_fail(h, e, "group");
    node_of_pos = reinterpret_cast<const int32_t*>(A.gpay[(g.npass - 1) & 1]);
    pos_of_node = A.pos_of_node;
  }

  SweepArgs sw{};
  BlockSweepArgs ba{};
  if (N > 0) {
    sw.p = pd;
    sw.itab = A.itab;
    sw.wf_off = A.wf_off;
    sw.node_of_pos = node_of_pos;
    sw.pos_of_node = pos_of_node;
    sw.rem_out = r->rem_us;
    sw.stg_ready = A.stg_ready;
    sw.stg_slack = A.stg_slack;
    sw.stg_route = A.stg_route;
    sw.stg_cost = A.stg_cost;
    sw.stg_oslack = A.stg_oslack;
    sw.g_cnt = A.g_cnt;
    sw.g_mx = A.g_mx;
    sw.g_dn = A.g_dn;
    sw.g_nr = A.g_nr;
    sw.g_front0 = A.g_front[0];
    sw.g_front1 = A.g_front[1];
    sw.ctrl = ctrl;
    sw.bk = bk;
    sw.fused = fused ? 1 : 0;
    sw.next_ctrl = A.ctrl[nxt];
    sw.bk_clear = A.bcnt[nxt];
    sw.bk_clear_n = A.capB > 0 ? A.capB : 0;
    sw.force_global = (h->flags & NALAR_FORCE_GLOBAL_SWEEP) ? 1 : 0;
    ba.ordered = (h->flags & NALAR_FORCE_LEVEL_SWEEP) ? 0 : 1;
    ba.done_bits = reinterpret_cast<const uint32_t*>(A.done_bits);
    if (as.plog && as.plog_cap >= p->n_edges) {
      ba.plog_r = static_cast<int64_t*>(as.plog);
      ba.plog_lp = reinterpret_cast<int32_t*>(static_cast<char*>(as.plog) + align_up(size_t(as.plog_cap) * 8, 256));
      ba.plog_cap = as.plog_cap;
    }
    NALAR_LAUNCH("sweep", launch_sweep(s, sw, ba, sh));
    as.bcnt_clean[nxt] = true;  // the sweep cleared them for the next pass
  }

  SortArgs sa{};
  sa.ctrl = ctrl;
  sa.next_ctrl = A.ctrl[nxt];
  sa.host = h->host;
  sa.stg_slack = A.stg_slack;
  sa.stg_ready = A.stg_ready;
  sa.stg_route = A.stg_route;
  sa.stg_cost = A.stg_cost;
  sa.node_of_pos = node_of_pos;
  sa.out_slack = ((policy & (NALAR_ORDER_LPT | NALAR_ORDER_SRTF)) || p->wf_priority) ? A.stg_oslack : nullptr;
  sa.span = N;
  for (int i = 0; i < 2; ++i) {
    sa.key[i] = A.skey[i];
    sa.pay[i] = A.spay[i];
  }
  sa.lookback = A.slb;
  sa.tiles_cap = tiles_of(A.capN);
  sa.bagg = A.bagg;
  sa.epoch = epoch;
  sa.levels = p->wf_priority ? 1u : 0u;
  sa.order = r->order;
  sa.slack = r->slack_us;
  sa.route = r->route;
  sa.cost = r->cost_us;
  sa.split_next = A.split[h->split_cur ^ 1];
  sa.split_min = h->split_any ? 1 : kBinMinReady;
  sa.p = pd;
  sa.passes_launched = kMaxSortPasses;  // the bucketed and bin sorts finish in one launch
  __atomic_store_n(&h->host->max_bucket, 0u, __ATOMIC_RELAXED);       // written by the large-bucket sort
  __atomic_store_n(&h->host->split_nb, 0u, __ATOMIC_RELAXED);         // written with new splitters
  __atomic_store_n(&h->host->status, 0xFFFFFFFFu, __ATOMIC_RELEASE);  // the kernels overwrite it
  bool tiled = bk.nb == 0;
  if (!tiled) {
    if (bk.bins) {
      NALAR_LAUNCH("sort_bin", launch_bin_sort(s, sa, bk));
    } else {
      NALAR_LAUNCH("sort_bucket", launch_bucket_sort(s, sa, bk));
      if (want_split) NALAR_LAUNCH("splitters", launch_splitters(s, sa));
    }
    tm.end();
    e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(h, e, "hipStreamSynchronize");
    if (__atomic_load_n(&h->host->status, __ATOMIC_ACQUIRE) == kStatusTiled) {
      // A bucket overflowed.  With buckets planned the sweep staged nothing
      // for the tiled sort, so sweep again without buckets (same results,
      // staged by position) after resetting the control block it accumulates
      // into; the next pass's control block and counters are reset again too.
      __atomic_store_n(&h->host->status, 0xFFFFFFFFu, __ATOMIC_RELEASE);
      tiled = true;
      if (bk.bins) {  // a bin overflowed: new splitters come from the tiled sort; back off
        h->bin_max = 0;
        h->bin_skip = h->bin_backoff;
        h->bin_backoff = h->bin_backoff < 64 ? 2 * h->bin_backoff : 64;
      } else {
        h->bucket_calm = 0;
        // fewer buckets overflowed at once: wait twice as long before trying again
        if (h->bucket_relaxed && h->bucket_relax < 4096) h->bucket_relax *= 2;
        h->bucket_relaxed = false;
        if (h->bucket_dense < 3) {  // retry at once with more buckets
          ++h->bucket_dense;
        } else {                    // then back off
          h->bucket_skip = h->bucket_backoff;
          h->bucket_backoff = h->bucket_backoff < 64 ? 2 * h->bucket_backoff : 64;
        }
      }
      NALAR_LAUNCH("reset", launch_reset(s, ctrl, nullptr, 0));
      if (policy & NALAR_ROUTE_WEIGHTED)  // its weight check reports into the block just reset
        NALAR_LAUNCH("weighted_table", launch_weighted_table(s, wa));
      sw.bk = BucketArgs{};
      NALAR_LAUNCH("sweep", launch_sweep(s, sw, ba, sh));
    } else if (bk.bins) {
      h->bin_backoff = 1;
      h->bin_max = __atomic_load_n(&h->host->max_bucket, __ATOMIC_ACQUIRE);
    } else {
      h->bucket_backoff = 1;
      const bool crowded = __atomic_load_n(&h->host->max_bucket, __ATOMIC_ACQUIRE) > kBucketCrowded;
      const bool was_relaxed = h->bucket_relaxed;
      h->bucket_relaxed = false;
      if (crowded && h->bucket_dense < 4 && bk.nb < kBucketMax) {
        // sorted, but a bucket is crowded (its futures rank one another one by
        // one, and its group of buckets outweighs the rest): add buckets, and
        // if fewer buckets were just tried, wait longer before trying again
        ++h->bucket_dense;
        h->bucket_calm = 0;
        if (was_relaxed && h->bucket_relax < 4096) h->bucket_relax *= 2;
      } else if (h->bucket_dense > 0 && ++h->bucket_calm >= h->bucket_relax) {  // try fewer buckets again
        --h->bucket_dense;
        h->bucket_calm = 0;
        h->bucket_relaxed = true;
      }
    }
  }
  if (tiled) {
    sa.passes_launched = kSortLaunched;
    e = launch_slack_sort(s, sa, 0, kSortLaunched - 1, Timer::cb, &tm);
    if (e != hipSuccess) return hip_fail(h, e, "sort");
    if (want_split) NALAR_LAUNCH("splitters", launch_splitters(s, sa));
    tm.end();
    e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(h, e, "hipStreamSynchronize");
    if (__atomic_load_n(&h->host->status, __ATOMIC_ACQUIRE) == kStatusContinue) {
      __atomic_store_n(&h->host->status, 0xFFFFFFFFu, __ATOMIC_RELEASE);
      sa.passes_launched = kMaxSortPasses;
      e = launch_slack_sort(s, sa, kSortLaunched, kMaxSortPasses - 1, Timer::cb, &tm);
      if (e != hipSuccess) return hip_fail(h, e, "sort");
      if (want_split) NALAR_LAUNCH("splitters", launch_splitters(s, sa));
      tm.end();
      e = hipStreamSynchronize(s);
      if (e != hipSuccess) return hip_fail(h, e, "hipStreamSynchronize");
    }
  }
  as.passes += 1;
  as.ctrl_dirty[nxt] = false;
  const uint32_t st = __atomic_load_n(&h->host->status, __ATOMIC_ACQUIRE);
  if (st == 0xFFFFFFFFu) return fail(h, NALAR_EDEVICE, "status was not written");
  if (st & kStInval) return fail(h, NALAR_EINVAL, "invalid problem data");
  if (st & kStCycle) return fail(h, NALAR_ECYCLE, "dependency cycle");
  if (st & kStRange) return fail(h, NALAR_ERANGE, "remaining critical path exceeds 2^62 us");
  r->n_ready = __atomic_load_n(&h->host->n_ready, __ATOMIC_ACQUIRE);
  if (want_split || bk.bins) {  // splitters written for the next pass: read them from now on
    const uint32_t snb = __atomic_load_n(&h->host->split_nb, __ATOMIC_ACQUIRE);
    h->split_nb = int(snb);
    if (snb > 0) h->split_cur ^= 1;
  }
  if ((policy & NALAR_ROUTE_GREEDY) && r->n_ready > 0 && M > 0) {
    // route again in output order with running loads (one wavefront per type)
    __atomic_store_n(&h->host->aux_status, 0u, __ATOMIC_RELEASE);
    GreedyArgs g{r->order, r->n_ready, p->type, p->est_us, p->loc, p->inst_type, p->inst_load_us,
                 p->inst_speed_permille, int32_t(M), (policy & NALAR_ROUTE_STATEFUL) ? 1 : 0,
                 p->migration_cost_us, r->route, r->cost_us, h->host};
    NALAR_LAUNCH("route_greedy", launch_route_greedy(s, g));
    tm.end();
    e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(h, e, "hipStreamSynchronize");
    if (__atomic_load_n(&h->host->aux_status, __ATOMIC_ACQUIRE) & kStRange)
      return fail(h, NALAR_ERANGE, "an instance load exceeds 2^62 us under load-aware routing");
  }
  if ((policy & NALAR_ROUTE_WEIGHTED) && r->n_ready > 0 && M > 0) {
    wa.order = r->order;
    wa.R = r->n_ready;
    wa.tiles = weighted_tiles(r->n_ready);
    e = launch_route_weighted(s, wa, Timer::cb, &tm);
    if (e != hipSuccess) return hip_fail(h, e, "weighted");
    tm.end();
    e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(h, e, "hipStreamSynchronize");
  }
#undef NALAR_LAUNCH
  if (h->timing) {
    h->n_timed = tm.n;
    for (int i = 0; i < tm.n; ++i) (void)hipEventElapsedTime(&h->ms[i], h->ev[i], h->ev[i + 1]);
    h->timed_valid = true;
  }
  h->hint_valid = true;
  h->hint_ready = r->n_ready;
  h->hint_min = r->n_ready ? __atomic_load_n(&h->host->slack_min, __ATOMIC_ACQUIRE) : 0;
  h->hint_max = r->n_ready ? __atomic_load_n(&h->host->slack_max, __ATOMIC_ACQUIRE) : 0;
  h->hint_levels = r->n_ready && p->wf_priority ? __atomic_load_n(&h->host->level_mask, __ATOMIC_ACQUIRE) : 0u;
  return NALAR_OK;
}

}  // namespace

void nalar::policy_split_any(nalar_policy* h, bool on) { h->split_any = on; }

int nalar::policy_reserve(nalar_policy* h, int64_t N, int64_t E, int64_t W) {
  const Arena& a = h->own.ar;
  if (h->own.plog && E > h->own.plog_cap) {  // once a pass has used it, the push log follows the graph
    hipError_t e = hipSetDevice(h->device);
    if (e != hipSuccess) return hip_fail(h, e, "hipSetDevice");
    const int rc = ensure_push_log(h, E);
    if (rc != NALAR_OK) return rc;
  }
  if (!a.base) return NALAR_OK;  // the first pass sizes it
  // the incremental pass's bins at the last pass's ready count, kept at least
  BucketArgs bk{};
  bk.bins = 1;
  bk.nb = h->split_nb > 0 ? h->split_nb : 0;
  bk.cap = bk.nb > 0 ? bin_cap_for(h->hint_ready, bk.nb) : 0;
  const int64_t B = a.capB > bk.nb ? a.capB : bk.nb;
  const int64_t rec = bk.nb > 0 ? records_of(bk) : 0;
  const int64_t Rec = a.capRec > rec ? a.capRec : rec;
  // also when only the bins grew: a reallocation (and its clearing fill) inside
  // the next pass costs more than the pass
  if (N <= a.capN && W <= a.capW && B <= a.capB && Rec <= a.capRec) return NALAR_OK;
  hipError_t e = hipSetDevice(h->device);
  if (e != hipSuccess) return hip_fail(h, e, "hipSetDevice");
  return ensure_capacity(h, N, W, B, Rec);
}

// The incremental pass over the graph store (the kernels in incremental.hip):
// the appended futures validated, the closure of the changed futures and its
// sweep, readiness of every future, the ready futures binned by the previous
// pass's splitters and sorted with ties by (wf, id).  Everything the store
// keeps is its own; the rest is this handle's arena, as in a full pass.
int nalar::policy_pass_incremental(nalar_policy* h, const nalar_problem* p, nalar_result* r,
                                   const IncStore& st) {
  h->err.clear();
  h->timed_valid = false;
  int rc = check_problem(h, p, r);
  if (rc != NALAR_OK) return rc;
  const int64_t N = p->n_nodes, W = p->n_workflows, M = p->n_instances;
  if (N == 0 || h->split_nb <= 0 || (h->split_nb & (h->split_nb - 1)) != 0 || !h->hint_valid ||
      (h->flags & NALAR_FORCE_TILED_SORT) || p->wf_priority ||
      (p->flags & NALAR_ROUTE_WEIGHTED) || st.n_prev > N)
    return kIncFallback;
  hipError_t e = hipSetDevice(h->device);
  if (e != hipSuccess) return hip_fail(h, e, "hipSetDevice");
  BucketArgs bk{};
  bk.bins = 1;
  bk.nb = h->split_nb;
  bk.cap = bin_cap_for(h->hint_ready, bk.nb);
  rc = ensure_capacity(h, N, W, bk.nb, records_of(bk));
  if (rc != NALAR_OK) return rc;
  ArenaState& as = h->own;
  Arena& A = as.ar;
  hipStream_t s = h->stream;
  const int cur = int(as.passes & 1);
  const int nxt = cur ^ 1;
  bk.cnt = A.bcnt[cur];
  bk.slot = A.bslot;
  bk.split = A.split[h->split_cur];
  Ctrl* ctrl = A.ctrl[cur];
  const bool need_reset = as.ctrl_dirty[cur];
  as.ctrl_dirty[cur] = true;
  as.ctrl_dirty[nxt] = true;
  const uint32_t policy = p->flags & (NALAR_ORDER_LPT | NALAR_ORDER_SRTF | NALAR_ROUTE_STATEFUL | NALAR_ROUTE_GREEDY);
  const ProblemDev pd = device_view(p, policy);
  const bool contiguous = (p->flags & NALAR_WF_CONTIGUOUS) != 0 || W <= 1;

  Timer tm{h};
#define NALAR_LAUNCH(name, call)                            \
  do {                                                      \
    tm.mark(name);                                          \
    hipError_t le_ = (call);                                \
    if (le_ != hipSuccess) return hip_fail(h, le_, name);   \
  } while (0)

  const bool need_clear = !as.bcnt_clean[cur];
  if (need_reset || need_clear)
    NALAR_LAUNCH("reset", launch_reset(s, need_reset ? ctrl : nullptr, bk.cnt, need_clear ? bk.nb : 0));
  as.bcnt_clean[cur] = false;
  // the appended futures (and the one before them, for the contiguity rule)
  NALAR_LAUNCH("nodes", launch_nodes(s, pd, ctrl, A.ctrl[nxt], A.itab, A.wf_off, contiguous ? 1 : 0,
                                     st.n_prev > 0 ? st.n_prev - 1 : 0));
  IncArgs ia{};
  ia.p = pd;
  ia.n_prev = st.n_prev;
  ia.log = st.log;
  ia.n_log = st.n_log;
  ia.rem = st.rem;
  ia.inA = st.inA;
  ia.dnb = st.dnb;
  ia.mxA = st.mxA;
  ia.cntA = st.cntA;
  ia.light = st.light;
  ia.heavy = st.heavy;
  ia.rlist = st.rlist;
  ia.ic = st.ic;
  ia.ctrl = ctrl;
  ia.itab = A.itab;
  ia.bk = bk;
  ia.bk_clear = A.bcnt[nxt];
  ia.bk_clear_n = A.capB > 0 ? A.capB : 0;
  ia.stg_oslack = A.stg_oslack;
  NALAR_LAUNCH("inc_pack", launch_inc_pack(s, ia));
  NALAR_LAUNCH("inc_clear", launch_inc_clear(s, reinterpret_cast<uint32_t*>(st.ic), sizeof(IncCtrl) / 4));
  e = launch_inc_closure(s, ia, h->cus, Timer::cb, &tm);
  if (e != hipSuccess) return hip_fail(h, e, "inc_closure");
  NALAR_LAUNCH("inc_scan", launch_inc_scan(s, ia, h->cus));
  e = launch_inc_sweep(s, ia, h->cus, Timer::cb, &tm);
  if (e != hipSuccess) return hip_fail(h, e, "inc_sweep");
  NALAR_LAUNCH("inc_ready", launch_inc_ready(s, ia, h->cus));
  as.bcnt_clean[nxt] = true;

  SortArgs sa{};
  sa.ctrl = ctrl;
  sa.next_ctrl = A.ctrl[nxt];
  sa.host = h->host;
  sa.out_slack = (policy & (NALAR_ORDER_LPT | NALAR_ORDER_SRTF)) ? A.stg_oslack : nullptr;
  sa.span = N;
  sa.split_next = A.split[h->split_cur ^ 1];
  sa.split_min = 1;
  sa.tie_wf = p->wf;
  sa.p = pd;
  sa.passes_launched = kMaxSortPasses;
  sa.order = r->order;
  sa.slack = r->slack_us;
  sa.route = r->route;
  sa.cost = r->cost_us;
  __atomic_store_n(&h->host->max_bucket, 0u, __ATOMIC_RELAXED);
  __atomic_store_n(&h->host->split_nb, 0u, __ATOMIC_RELAXED);
  __atomic_store_n(&h->host->status, 0xFFFFFFFFu, __ATOMIC_RELEASE);
  NALAR_LAUNCH("sort_bin", launch_bin_sort(s, sa, bk));
  if (r->rem_us) NALAR_LAUNCH("rem_copy", hipMemcpyAsync(r->rem_us, st.rem, sizeof(int64_t) * size_t(N),
                                                         hipMemcpyDeviceToDevice, s));
  tm.end();
  e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(h, e, "hipStreamSynchronize");
  const uint32_t sts = __atomic_load_n(&h->host->status, __ATOMIC_ACQUIRE);
  if (sts == 0xFFFFFFFFu) return fail(h, NALAR_EDEVICE, "status was not written");
  if (sts == kStatusTiled) {
    h->bin_max = 0;
    return kIncFallbackOverflow;
  }
  h->bin_max = __atomic_load_n(&h->host->max_bucket, __ATOMIC_ACQUIRE);
  if (sts & kStIncomplete) return kIncFallbackRounds;
  as.passes += 1;
  as.ctrl_dirty[nxt] = false;
  if (sts & kStInval) return fail(h, NALAR_EINVAL, "invalid problem data");
  if (sts & kStCycle) return fail(h, NALAR_ECYCLE, "dependency cycle");
  if (sts & kStRange) return fail(h, NALAR_ERANGE, "remaining critical path exceeds 2^62 us");
  r->n_ready = __atomic_load_n(&h->host->n_ready, __ATOMIC_ACQUIRE);
  const uint32_t snb = __atomic_load_n(&h->host->split_nb, __ATOMIC_ACQUIRE);
  h->split_nb = int(snb);
  if (snb > 0) h->split_cur ^= 1;
  if ((policy & NALAR_ROUTE_GREEDY) && r->n_ready > 0 && M > 0) {
    __atomic_store_n(&h->host->aux_status, 0u, __ATOMIC_RELEASE);
    GreedyArgs g{r->order, r->n_ready, p->type, p->est_us, p->loc, p->inst_type, p->inst_load_us,
                 p->inst_speed_permille, int32_t(M), (policy & NALAR_ROUTE_STATEFUL) ? 1 : 0,
                 p->migration_cost_us, r->route, r->cost_us, h->host};
    NALAR_LAUNCH("route_greedy", launch_route_greedy(s, g));
    tm.end();
    e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(h, e, "hipStreamSynchronize");
    if (__atomic_load_n(&h->host->aux_status, __ATOMIC_ACQUIRE) & kStRange)
      return fail(h, NALAR_ERANGE, "an instance load exceeds 2^62 us under load-aware routing");
  }
#undef NALAR_LAUNCH
  if (h->timing) {
    h->n_timed = tm.n;
    for (int i = 0; i < tm.n; ++i) (void)hipEventElapsedTime(&h->ms[i], h->ev[i], h->ev[i + 1]);
    h->timed_valid = true;
  }
  h->hint_valid = true;
  h->hint_ready = r->n_ready;
  h->hint_min = r->n_ready ? __atomic_load_n(&h->host->slack_min, __ATOMIC_ACQUIRE) : 0;
  h->hint_max = r->n_ready ? __atomic_load_n(&h->host->slack_max, __ATOMIC_ACQUIRE) : 0;
  h->hint_levels = 0;
  return NALAR_OK;
}

extern "C" {

int nalar_policy_pass(nalar_policy* h, const nalar_problem* p, nalar_result* r) {
  if (!h) return NALAR_EINVAL;
  h->err.clear();
  h->timed_valid = false;
  int rc = check_problem(h, p, r);
  if (rc != NALAR_OK) return rc;
  hipError_t e = hipSetDevice(h->device);
  if (e != hipSuccess) return hip_fail(h, e, "hipSetDevice");
  const int64_t N = p->n_nodes, W = p->n_workflows, M = p->n_instances;
  const SweepShape sh = plan_sweep(N, W, M, h->cus, h->lds_limit);
  BucketArgs bk = plan_bins(h, sh, p->wf_priority != nullptr);
  if (!bk.bins) bk = plan_buckets(h, N, p->wf_priority != nullptr, sh.wave_path != 0);
  if (h->bucket_skip > 0) --h->bucket_skip;
  if (h->bin_skip > 0) --h->bin_skip;
  rc = ensure_capacity(h, N, W, bk.nb, records_of(bk));
  if (rc != NALAR_OK) return rc;
  if (!sh.wave_path && !(h->flags & NALAR_FORCE_LEVEL_SWEEP)) {
    rc = ensure_push_log(h, p->n_edges);
    if (rc != NALAR_OK) return rc;
  }
  return run_pass(h, p, r, h->own, bk, sh, true);
}

int nalar_policy_pass_static(nalar_policy* h, const nalar_problem* p, nalar_result* r) {
  if (!h) return NALAR_EINVAL;
  h->err.clear();
  h->timed_valid = false;
  int rc = check_problem(h, p, r);
  if (rc != NALAR_OK) return rc;
  if (p->n_nodes > NALAR_STATIC_MAX_NODES || p->n_workflows > NALAR_STATIC_MAX_WORKFLOWS)
    return fail(h, NALAR_EINVAL, "snapshot larger than the static scratch allows (n_nodes and n_workflows "
                                 "<= NALAR_STATIC_MAX_NODES / _WORKFLOWS)");
  hipError_t e = hipSetDevice(h->device);
  if (e != hipSuccess) return hip_fail(h, e, "hipSetDevice");
  StaticScratch& ss = g_static[h->device];
  std::lock_guard<std::mutex> lock(ss.mu);
  if (!ss.ready) return fail(h, NALAR_EDEVICE, "static scratch not set up on this device");
  const int64_t N = p->n_nodes, W = p->n_workflows, M = p->n_instances;
  const SweepShape sh = plan_sweep(N, W, M, h->cus, h->lds_limit);
  BucketArgs bk = plan_buckets(h, N, p->wf_priority != nullptr, sh.wave_path != 0);
  if (h->bucket_skip > 0) --h->bucket_skip;
  if (bk.nb > kStaticBuckets) bk = BucketArgs{};  // more buckets than the array holds: tiled sort
  if (!ss.cleared) {  // first use on this device: untag every look-back word
    e = clear_lookback(h->stream, ss.st.ar);
    if (e != hipSuccess) return hip_fail(h, e, "clear look-back");
    ss.cleared = true;
  }
  return run_pass(h, p, r, ss.st, bk, sh, false);
}

}  // extern "C"
