// Device-resident graph store: the global view kept in HBM across passes and
// updated by deltas (futures appended with their dependencies, futures
// completed, deadlines and instances replaced), so that a pass needs no
// upload or rebuild of the snapshot.  The arrays are the snapshot's own struct
// of arrays (ids in append order), grown geometrically.  A pass over the
// store gives the results of nalar_policy_pass over them: after a successful
// pass the store keeps every future's remaining critical path, and the next
// pass recomputes it only for the futures appended or completed since and
// their ancestors (incremental.hip), falling back to a full pass when it
// cannot (no earlier pass, no splitters, a bin overflow).
#include <cstring>

#include "internal.hpp"
#include "nalar_store.h"

using namespace nalar;

struct nalar_store {
  nalar_policy* h = nullptr;
  int64_t N = 0, E = 0, W = 0, M = 0;
  int64_t capN = 0, capE = 0, capW = 0, capM = 0;
  bool contiguous = true;
  int32_t* wf = nullptr;
  int32_t* type = nullptr;
  int64_t* est = nullptr;
  uint8_t* done = nullptr;
  int32_t* loc = nullptr;
  int32_t* dep_off = nullptr;   // [capN + 1]
  int32_t* dep_idx = nullptr;   // [capE]
  int64_t* deadline = nullptr;  // [capW]
  int32_t* inst_type = nullptr; // [capM]
  int64_t* inst_load = nullptr;
  int32_t* inst_speed = nullptr;
  uint32_t* bad = nullptr;      // pinned: count of completion calls with an id out of range,
                                //   and of appends whose offsets are malformed
  uint32_t bad_seen = 0;        // the count when last reported (only the device writes *bad)
  // incremental passes
  bool incremental = true;      // nalar_store_set_incremental
  bool rem_valid = false;       // rem holds [0, n_prev) from the last successful pass
  int last_incremental = 0;     // the last pass was an incremental one
  int last_fallback = 0;        // why the last pass was a full one (NALAR_STORE_FULL_*)
  int64_t n_prev = 0;
  int64_t W_prev = 0, M_prev = 0; // workflows and instances at the last pass (fewer now: the
                                //   stored futures must be validated again, in a full pass)
  int64_t capI = 0;             // futures the incremental buffers hold
  int64_t* rem = nullptr;       // [capI]
  uint32_t* inA = nullptr;      // [capI / 32 + 1]
  uint32_t* dnb = nullptr;      // [capI / 32 + 1] done flags as bits (pass scratch)
  int64_t* mxA = nullptr;
  int32_t* cntA = nullptr;
  int32_t* light = nullptr;
  int32_t* heavy = nullptr;
  int32_t* rlist = nullptr;
  IncCtrl* ic = nullptr;
  int32_t* log = nullptr;       // ids completed since the last pass
  int64_t n_log = 0, capLog = 0;
};

namespace {

constexpr int kStoreThreads = 256;

// dep_off of the appended futures: the store's edge count plus the offsets
// given relative to the call (dst[0], the previous end, is kept).  Offsets
// that do not start at 0, end at the call's edge count and never decrease are
// counted in *bad, so the next pass reports NALAR_EINVAL.
__global__ __launch_bounds__(kStoreThreads) void k_store_offsets(int32_t* dst, const int32_t* src,
                                                                 int64_t n, int32_t base, int64_t n_edges,
                                                                 uint32_t* bad) {
  bool b = false;
  for (int64_t i = int64_t(blockIdx.x) * kStoreThreads + threadIdx.x; i <= n;
       i += int64_t(gridDim.x) * kStoreThreads) {
    const int32_t x = src[i];
    if (i == 0) b |= x != 0;
    else {
      b |= x < src[i - 1];
      dst[i] = base + x;
    }
    if (i == n) b |= int64_t(x) != n_edges;
  }
  if (ballot(b) != 0 && lane_id() == 0)
    __hip_atomic_fetch_add(bad, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

__global__ __launch_bounds__(kStoreThreads) void k_store_complete(uint8_t* done, const int32_t* ids,
                                                                  int64_t n, int64_t N, uint32_t* bad) {
  bool b = false;
  for (int64_t i = int64_t(blockIdx.x) * kStoreThreads + threadIdx.x; i < n;
       i += int64_t(gridDim.x) * kStoreThreads) {
    const int32_t v = ids[i];
    if (v >= 0 && int64_t(v) < N) done[v] = 1;
    else b = true;
  }
  if (ballot(b) != 0 && lane_id() == 0)
    __hip_atomic_fetch_add(bad, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

int grid_for(int64_t n) {
  int64_t g = (n + kStoreThreads - 1) / kStoreThreads;
  return int(g < 1 ? 1 : (g > 4096 ? 4096 : g));
}

// Grow one array to hold `need` elements (geometric), keeping `keep` of them.
template <typename T>
hipError_t grow(T*& p, int64_t& cap, int64_t need, int64_t keep, hipStream_t s) {
  if (need <= cap) return hipSuccess;
  int64_t nc = cap > 0 ? cap + cap / 2 : 1024;
  if (nc < need) nc = need;
  T* q = nullptr;
  hipError_t e = hipMalloc(&q, sizeof(T) * size_t(nc));
  if (e != hipSuccess) return e;
  if (p && keep > 0) {
    e = hipMemcpyAsync(q, p, sizeof(T) * size_t(keep), hipMemcpyDeviceToDevice, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) { (void)hipFree(q); return e; }
  }
  if (p) (void)hipFree(p);
  p = q;
  cap = nc;
  return hipSuccess;
}

int store_fail(nalar_store* st, hipError_t e, const char* what) {
  std::string m = std::string(what) + ": " + hipGetErrorString(e);
  return policy_fail(st->h, e == hipErrorOutOfMemory ? NALAR_ENOMEM : NALAR_EDEVICE, m.c_str());
}

template <typename T>
hipError_t copy_in(T* dst, const T* src, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  return hipMemcpyAsync(dst, src, sizeof(T) * size_t(n), hipMemcpyDeviceToDevice, s);
}

// The incremental buffers for every stored future (rem keeps what the last
// pass computed).
int ensure_incremental(nalar_store* st) {
  hipError_t e = hipSetDevice(policy_device(st->h));
  if (e != hipSuccess) return store_fail(st, e, "hipSetDevice");
  hipStream_t s = policy_stream(st->h);
  if (!st->ic) {
    e = hipMalloc(&st->ic, sizeof(IncCtrl));
    if (e != hipSuccess) return store_fail(st, e, "store incremental");
  }
  const int64_t need = st->N > 0 ? st->N : 1;
  if (need <= st->capI) return NALAR_OK;
  int64_t nc = st->capI > 0 ? st->capI + st->capI / 2 : 1024;
  if (nc < need) nc = need;
  int64_t c;
  c = st->capI; e = grow(st->rem, c, nc, st->rem_valid ? st->n_prev : 0, s);
  if (e == hipSuccess) { c = st->capI / 32 + 1; e = grow(st->inA, c, nc / 32 + 1, 0, s); }
  if (e == hipSuccess) { c = st->capI / 32 + 1; e = grow(st->dnb, c, nc / 32 + 1, 0, s); }
  if (e == hipSuccess) { c = st->capI; e = grow(st->mxA, c, nc, 0, s); }
  if (e == hipSuccess) { c = st->capI; e = grow(st->cntA, c, nc, 0, s); }
  if (e == hipSuccess) { c = st->capI; e = grow(st->light, c, nc, 0, s); }
  if (e == hipSuccess) { c = st->capI; e = grow(st->heavy, c, nc, 0, s); }
  if (e == hipSuccess) { c = st->capI; e = grow(st->rlist, c, nc, 0, s); }
  if (e != hipSuccess) {
    st->rem_valid = false;
    return store_fail(st, e, "store incremental");
  }
  st->capI = nc;
  return NALAR_OK;
}

}  // namespace

extern "C" {

int nalar_store_create(nalar_policy* h, nalar_store** out) {
  if (out) *out = nullptr;
  if (!h || !out) return NALAR_EINVAL;
  nalar_store* st = new (std::nothrow) nalar_store();
  if (!st) return NALAR_ENOMEM;
  st->h = h;
  hipError_t e = hipSetDevice(policy_device(h));
  if (e == hipSuccess)
    e = hipHostMalloc(reinterpret_cast<void**>(&st->bad), sizeof(uint32_t), hipHostMallocCoherent);
  if (e != hipSuccess) {
    delete st;
    return policy_fail(h, NALAR_ENOMEM, "hipHostMalloc(store flag)");
  }
  *st->bad = 0;
  *out = st;
  return NALAR_OK;
}

void nalar_store_destroy(nalar_store* st) {
  if (!st) return;
  (void)hipSetDevice(policy_device(st->h));
  (void)hipStreamSynchronize(policy_stream(st->h));
  for (void* p : {static_cast<void*>(st->wf), static_cast<void*>(st->type), static_cast<void*>(st->est),
                  static_cast<void*>(st->done), static_cast<void*>(st->loc), static_cast<void*>(st->dep_off),
                  static_cast<void*>(st->dep_idx), static_cast<void*>(st->deadline),
                  static_cast<void*>(st->inst_type), static_cast<void*>(st->inst_load),
                  static_cast<void*>(st->inst_speed), static_cast<void*>(st->rem), static_cast<void*>(st->inA), static_cast<void*>(st->dnb),
                  static_cast<void*>(st->mxA), static_cast<void*>(st->cntA), static_cast<void*>(st->light),
                  static_cast<void*>(st->heavy), static_cast<void*>(st->rlist), static_cast<void*>(st->ic),
                  static_cast<void*>(st->log)})
    if (p) (void)hipFree(p);
  if (st->bad) (void)hipHostFree(st->bad);
  delete st;
}

int nalar_store_append(nalar_store* st, int64_t n_new, int64_t n_new_edges, const int32_t* wf,
                       const int32_t* type, const int64_t* est_us, const uint8_t* done,
                       const int32_t* loc, const int32_t* dep_off, const int32_t* dep_idx,
                       uint32_t flags) {
  if (!st) return NALAR_EINVAL;
  if (n_new < 0 || n_new_edges < 0 || (flags & ~NALAR_WF_CONTIGUOUS) != 0 ||
      st->N + n_new > NALAR_MAX_NODES || st->E + n_new_edges > NALAR_MAX_EDGES ||
      (n_new == 0 && n_new_edges != 0))
    return policy_fail(st->h, NALAR_EINVAL, "store append: sizes or flags out of range");
  if (n_new > 0 && (!wf || !type || !est_us || !done || !loc || !dep_off))
    return policy_fail(st->h, NALAR_EINVAL, "store append: NULL node array");
  if (n_new_edges > 0 && !dep_idx) return policy_fail(st->h, NALAR_EINVAL, "store append: NULL dep_idx");
  hipError_t e = hipSetDevice(policy_device(st->h));
  if (e != hipSuccess) return store_fail(st, e, "hipSetDevice");
  hipStream_t s = policy_stream(st->h);
  const int64_t N = st->N, E = st->E, need = N + n_new;
  if (need > st->capN) {  // every node array to the same new capacity
    int64_t nc = st->capN > 0 ? st->capN + st->capN / 2 : 1024;
    if (nc < need) nc = need;
    int64_t c0;
    c0 = st->capN; e = grow(st->wf, c0, nc, N, s);
    if (e == hipSuccess) { c0 = st->capN; e = grow(st->type, c0, nc, N, s); }
    if (e == hipSuccess) { c0 = st->capN; e = grow(st->est, c0, nc, N, s); }
    if (e == hipSuccess) { c0 = st->capN; e = grow(st->done, c0, nc, N, s); }
    if (e == hipSuccess) { c0 = st->capN; e = grow(st->loc, c0, nc, N, s); }
    if (e == hipSuccess) { c0 = st->capN + 1; e = grow(st->dep_off, c0, nc + 1, N + 1, s); }
    if (e != hipSuccess) return store_fail(st, e, "store grow");
    st->capN = nc;
  }
  if (E + n_new_edges > st->capE) {
    e = grow(st->dep_idx, st->capE, E + n_new_edges, E, s);
    if (e != hipSuccess) return store_fail(st, e, "store grow");
  }
  if (N == 0) {  // dep_off[0] = 0
    const int32_t zero = 0;
    e = hipMemcpyAsync(st->dep_off, &zero, sizeof(int32_t), hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return store_fail(st, e, "store init");
  }
  e = copy_in(st->wf + N, wf, n_new, s);
  if (e == hipSuccess) e = copy_in(st->type + N, type, n_new, s);
  if (e == hipSuccess) e = copy_in(st->est + N, est_us, n_new, s);
  if (e == hipSuccess) e = copy_in(st->done + N, done, n_new, s);
  if (e == hipSuccess) e = copy_in(st->loc + N, loc, n_new, s);
  if (e == hipSuccess) e = copy_in(st->dep_idx + E, dep_idx, n_new_edges, s);
  if (e != hipSuccess) return store_fail(st, e, "store copy");
  if (n_new > 0) {
    hipLaunchKernelGGL(k_store_offsets, dim3(grid_for(n_new + 1)), dim3(kStoreThreads), 0, s,
                       st->dep_off + N, dep_off, n_new, int32_t(E), n_new_edges, st->bad);
    e = hipGetLastError();
    if (e != hipSuccess) return store_fail(st, e, "store offsets");
  }
  st->N = need;
  st->E = E + n_new_edges;
  st->contiguous = st->contiguous && (flags & NALAR_WF_CONTIGUOUS);
  // the per-future buffers of the next pass grow here, with the store, and
  // not inside the pass
  int rc = ensure_incremental(st);
  if (rc == NALAR_OK) rc = policy_reserve(st->h, st->N, st->E, st->W);
  return rc;
}

int nalar_store_complete(nalar_store* st, int64_t n, const int32_t* ids) {
  if (!st) return NALAR_EINVAL;
  if (n < 0 || (n > 0 && !ids)) return policy_fail(st->h, NALAR_EINVAL, "store complete: bad arguments");
  if (n == 0) return NALAR_OK;
  hipError_t e = hipSetDevice(policy_device(st->h));
  if (e != hipSuccess) return store_fail(st, e, "hipSetDevice");
  hipStream_t s = policy_stream(st->h);
  hipLaunchKernelGGL(k_store_complete, dim3(grid_for(n)), dim3(kStoreThreads), 0, s, st->done, ids, n, st->N,
                     st->bad);
  e = hipGetLastError();
  if (e != hipSuccess) return store_fail(st, e, "store complete");
  // the completed ids seed the next incremental pass
  if (st->n_log + n > NALAR_MAX_NODES) {
    st->rem_valid = false;  // more completions than futures: the next pass is a full one
    st->n_log = 0;
    return NALAR_OK;
  }
  e = grow(st->log, st->capLog, st->n_log + n, st->n_log, s);
  if (e == hipSuccess) e = copy_in(st->log + st->n_log, ids, n, s);
  if (e != hipSuccess) return store_fail(st, e, "store complete log");
  st->n_log += n;
  return NALAR_OK;
}

int nalar_store_set_workflows(nalar_store* st, int64_t n_workflows, const int64_t* deadline_us) {
  if (!st) return NALAR_EINVAL;
  if (n_workflows < 0 || n_workflows > NALAR_MAX_WORKFLOWS || (n_workflows > 0 && !deadline_us))
    return policy_fail(st->h, NALAR_EINVAL, "store workflows: bad arguments");
  hipError_t e = hipSetDevice(policy_device(st->h));
  if (e == hipSuccess) e = grow(st->deadline, st->capW, n_workflows, 0, policy_stream(st->h));
  if (e == hipSuccess) e = copy_in(st->deadline, deadline_us, n_workflows, policy_stream(st->h));
  if (e != hipSuccess) return store_fail(st, e, "store workflows");
  st->W = n_workflows;
  return NALAR_OK;
}

int nalar_store_set_instances(nalar_store* st, int64_t n_instances, const int32_t* inst_type,
                              const int64_t* inst_load_us, const int32_t* inst_speed_permille) {
  if (!st) return NALAR_EINVAL;
  if (n_instances < 0 || n_instances > NALAR_MAX_INSTANCES ||
      (n_instances > 0 && (!inst_type || !inst_load_us || !inst_speed_permille)))
    return policy_fail(st->h, NALAR_EINVAL, "store instances: bad arguments");
  hipStream_t s = policy_stream(st->h);
  hipError_t e = hipSetDevice(policy_device(st->h));
  int64_t c1 = st->capM, c2 = st->capM;
  if (e == hipSuccess) e = grow(st->inst_type, st->capM, n_instances, 0, s);
  if (e == hipSuccess) e = grow(st->inst_load, c1, n_instances, 0, s);
  if (e == hipSuccess) e = grow(st->inst_speed, c2, n_instances, 0, s);
  if (e == hipSuccess) e = copy_in(st->inst_type, inst_type, n_instances, s);
  if (e == hipSuccess) e = copy_in(st->inst_load, inst_load_us, n_instances, s);
  if (e == hipSuccess) e = copy_in(st->inst_speed, inst_speed_permille, n_instances, s);
  if (e != hipSuccess) return store_fail(st, e, "store instances");
  st->M = n_instances;
  return NALAR_OK;
}

int64_t nalar_store_n_nodes(const nalar_store* st) { return st ? st->N : -1; }

int nalar_store_pass(nalar_store* st, int64_t now_us, int64_t migration_cost_us, uint32_t policy,
                     nalar_result* r) {
  if (!st) return NALAR_EINVAL;
  if ((policy & ~(NALAR_ORDER_LPT | NALAR_ORDER_SRTF | NALAR_ROUTE_STATEFUL | NALAR_ROUTE_GREEDY)) != 0)
    return policy_fail(st->h, NALAR_EINVAL, "store pass: unknown policy bits");
  nalar_problem p;
  std::memset(&p, 0, sizeof(p));
  p.n_nodes = st->N;
  p.n_edges = st->E;
  p.n_workflows = st->W;
  p.n_instances = st->M;
  p.now_us = now_us;
  p.migration_cost_us = migration_cost_us;
  p.flags = (st->contiguous ? NALAR_WF_CONTIGUOUS : 0u) | policy;
  p.wf = st->wf;
  p.type = st->type;
  p.est_us = st->est;
  p.done = st->done;
  p.loc = st->loc;
  p.dep_off = st->dep_off;
  p.dep_idx = st->dep_idx;
  p.deadline_us = st->deadline;
  p.inst_type = st->inst_type;
  p.inst_load_us = st->inst_load;
  p.inst_speed_permille = st->inst_speed;
  int rc = ensure_incremental(st);
  if (rc != NALAR_OK) return rc;
  st->last_incremental = 0;
  // a malformed append or completion since the last pass fails this one (the
  // pass has synchronised the stream, so every such call has been counted; the
  // host never writes the counter)
  auto bad_calls = [st]() {
    const uint32_t bad = __atomic_load_n(st->bad, __ATOMIC_ACQUIRE);
    const bool b = bad != st->bad_seen;
    st->bad_seen = bad;
    return b;
  };
  rc = kIncFallback;
  if (!st->incremental) st->last_fallback = NALAR_STORE_FULL_DISABLED;
  else if (!st->rem_valid || !r) st->last_fallback = NALAR_STORE_FULL_NO_STATE;
  else if (st->W < st->W_prev || st->M < st->M_prev) st->last_fallback = NALAR_STORE_FULL_SHRUNK;
  else {
    const IncStore is{st->n_prev, st->log, st->n_log, st->rem, st->inA, st->dnb, st->mxA, st->cntA,
                      st->light, st->heavy, st->rlist, st->ic};
    rc = policy_pass_incremental(st->h, &p, r, is);
    if (!inc_fallback(rc)) st->last_incremental = 1;
    st->last_fallback = rc == kIncFallback ? NALAR_STORE_FULL_NO_SPLITTERS
                      : rc == kIncFallbackOverflow ? NALAR_STORE_FULL_OVERFLOW
                      : rc == kIncFallbackRounds ? NALAR_STORE_FULL_ROUNDS : 0;
  }
  if (inc_fallback(rc)) {  // a full pass, its rem kept for the next one
    nalar_result r2{};
    if (r) r2 = *r;
    r2.rem_us = st->rem;
    policy_split_any(st->h, true);
    rc = nalar_policy_pass(st->h, &p, r ? &r2 : nullptr);
    policy_split_any(st->h, false);
    if (r) r->n_ready = r2.n_ready;
    if (rc == NALAR_OK && r && r->rem_us && st->N > 0) {
      hipError_t e = hipMemcpyAsync(r->rem_us, st->rem, sizeof(int64_t) * size_t(st->N), hipMemcpyDeviceToDevice,
                                    policy_stream(st->h));
      if (e == hipSuccess) e = hipStreamSynchronize(policy_stream(st->h));
      if (e != hipSuccess) rc = store_fail(st, e, "store rem");
    }
  }
  const bool bad = bad_calls();
  st->rem_valid = rc == NALAR_OK && !bad;
  st->n_prev = st->N;
  st->W_prev = st->W;
  st->M_prev = st->M;
  st->n_log = 0;
  if (bad) return policy_fail(st->h, NALAR_EINVAL, "a completed id was out of range, or appended offsets malformed");
  return rc;
}

int nalar_store_set_incremental(nalar_store* st, int enable) {
  if (!st) return NALAR_EINVAL;
  st->incremental = enable != 0;
  return NALAR_OK;
}

int nalar_store_last_pass_incremental(const nalar_store* st) { return st ? st->last_incremental : -1; }

int nalar_store_last_fallback(const nalar_store* st) { return st ? st->last_fallback : -1; }

}  // extern "C"
