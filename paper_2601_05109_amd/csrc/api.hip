// C ABI of the policy pass: handle, scratch arena, launch sequence, status.
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "internal.hpp"

using namespace nalar;

namespace {

constexpr int kMaxTimed = 32;

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

int64_t tiles_of(int64_t n) { return (n + kSortTile - 1) / kSortTile + 1; }

// Device scratch, carved from one allocation.
struct Arena {
  void* base = nullptr;
  size_t bytes = 0;
  size_t lookback_off = 0, lookback_bytes = 0;
  Ctrl* ctrl = nullptr;
  ITab itab{};
  uint32_t* ghist_slack = nullptr;
  uint32_t* ghist_group = nullptr;
  int32_t* wf_off = nullptr;
  uint8_t* stg_ready = nullptr;
  int64_t* stg_slack = nullptr;
  int32_t* stg_route = nullptr;
  int64_t* stg_cost = nullptr;
  uint64_t* skey[2] = {nullptr, nullptr};
  uint32_t* spay[2] = {nullptr, nullptr};
  uint64_t* slb = nullptr;
  uint32_t* gkey[2] = {nullptr, nullptr};
  uint32_t* gpay[2] = {nullptr, nullptr};
  uint64_t* glb = nullptr;
  int32_t* pos_of_node = nullptr;
  int32_t* g_cnt = nullptr;
  int64_t* g_mx = nullptr;
  uint8_t* g_dn = nullptr;
  uint8_t* g_nr = nullptr;
  int32_t* g_front[2] = {nullptr, nullptr};
  int64_t capN = -1, capW = -1;
};

}  // namespace

struct nalar_policy {
  int device = 0;
  uint32_t flags = 0;
  hipStream_t stream = nullptr;
  int cus = 0;
  size_t lds_limit = 0;
  uint32_t epoch = 0;
  std::string err;
  Arena ar;
  Ctrl* host_ctrl = nullptr;  // pinned readback
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
size_t carve(Arena& a, char* base, int64_t N, int64_t W) {
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
  a.ctrl = reinterpret_cast<Ctrl*>(take(sizeof(Ctrl)));
  a.itab.load = reinterpret_cast<int64_t*>(take(8 * NALAR_MAX_INSTANCES));
  a.itab.inv_speed = reinterpret_cast<double*>(take(8 * NALAR_MAX_INSTANCES));
  a.itab.type = reinterpret_cast<int32_t*>(take(4 * NALAR_MAX_INSTANCES));
  a.itab.idx = reinterpret_cast<int32_t*>(take(4 * NALAR_MAX_INSTANCES));
  a.itab.speed = reinterpret_cast<int32_t*>(take(4 * NALAR_MAX_INSTANCES));
  a.itab.pos_of = reinterpret_cast<int32_t*>(take(4 * NALAR_MAX_INSTANCES));
  a.ghist_slack = reinterpret_cast<uint32_t*>(take(4 * kMaxSortPasses * kRadixBuckets));
  a.ghist_group = reinterpret_cast<uint32_t*>(take(4 * kMaxGroupPasses * kRadixBuckets));
  a.wf_off = reinterpret_cast<int32_t*>(take(4 * size_t(w1 + 1)));
  a.stg_slack = reinterpret_cast<int64_t*>(take(8 * size_t(n1)));
  a.stg_cost = reinterpret_cast<int64_t*>(take(8 * size_t(n1)));
  a.stg_route = reinterpret_cast<int32_t*>(take(4 * size_t(n1)));
  a.stg_ready = reinterpret_cast<uint8_t*>(take(size_t(n1)));
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
  off = align_up(off, 256);
  a.lookback_off = off;
  a.slb = reinterpret_cast<uint64_t*>(take(8 * size_t(kMaxSortPasses) * tiles * kRadixBuckets));
  a.glb = reinterpret_cast<uint64_t*>(take(8 * size_t(kMaxGroupPasses) * tiles * kRadixBuckets));
  a.lookback_bytes = off - a.lookback_off;
  return align_up(off, 256);
}

int ensure_capacity(nalar_policy* h, int64_t N, int64_t W) {
  Arena& a = h->ar;
  if (a.base && N <= a.capN && W <= a.capW) return NALAR_OK;
  int64_t newN = a.capN > N ? a.capN : N;
  int64_t newW = a.capW > W ? a.capW : W;
  if (a.base) {  // grow geometrically so a slowly growing graph reallocates rarely
    if (N > a.capN) newN = N + N / 4;
    if (W > a.capW) newW = W + W / 4;
    hipError_t e = hipStreamSynchronize(h->stream);
    if (e != hipSuccess) return hip_fail(h, e, "hipStreamSynchronize");
    (void)hipFree(a.base);
    a.base = nullptr;
  }
  Arena fresh;
  const size_t bytes = carve(fresh, nullptr, newN, newW);
  void* p = nullptr;
  hipError_t e = hipMalloc(&p, bytes);
  if (e != hipSuccess) {
    a.capN = a.capW = -1;
    return hip_fail(h, e, "hipMalloc(scratch)");
  }
  e = hipMemset(p, 0, bytes);  // look-back words must start untagged
  if (e != hipSuccess) {
    (void)hipFree(p);
    return hip_fail(h, e, "hipMemset(scratch)");
  }
  carve(fresh, static_cast<char*>(p), newN, newW);
  fresh.base = p;
  fresh.bytes = bytes;
  fresh.capN = newN;
  fresh.capW = newW;
  h->ar = fresh;
  h->epoch = 0;
  return NALAR_OK;
}

bool in_range(int64_t v, int64_t lo, int64_t hi) { return v >= lo && v <= hi; }

int check_problem(nalar_policy* h, const nalar_problem* p, const nalar_result* r) {
  if (!p || !r) return fail(h, NALAR_EINVAL, "NULL problem or result");
  const int64_t N = p->n_nodes, E = p->n_edges, W = p->n_workflows, M = p->n_instances;
  if (!in_range(N, 0, NALAR_MAX_NODES)) return fail(h, NALAR_EINVAL, "n_nodes out of range");
  if (!in_range(E, 0, NALAR_MAX_EDGES)) return fail(h, NALAR_EINVAL, "n_edges out of range");
  if (!in_range(W, 0, NALAR_MAX_WORKFLOWS)) return fail(h, NALAR_EINVAL, "n_workflows out of range");
  if (!in_range(M, 0, NALAR_MAX_INSTANCES)) return fail(h, NALAR_EINVAL, "n_instances out of range");
  if (!in_range(p->now_us, -NALAR_HORIZON_MAX, NALAR_HORIZON_MAX))
    return fail(h, NALAR_EINVAL, "now_us out of range");
  if (!in_range(p->migration_cost_us, 0, NALAR_MIG_MAX))
    return fail(h, NALAR_EINVAL, "migration_cost_us out of range");
  if ((p->flags & ~NALAR_WF_CONTIGUOUS) != 0 || p->reserved != 0)
    return fail(h, NALAR_EINVAL, "unknown problem flags");
  if (N == 0 && E != 0) return fail(h, NALAR_EINVAL, "edges without nodes");
  if (N > 0 && (!p->wf || !p->type || !p->est_us || !p->done || !p->loc || !p->dep_off))
    return fail(h, NALAR_EINVAL, "NULL node array");
  if (E > 0 && !p->dep_idx) return fail(h, NALAR_EINVAL, "NULL dep_idx");
  if (W > 0 && !p->deadline_us) return fail(h, NALAR_EINVAL, "NULL deadline_us");
  if (M > 0 && (!p->inst_type || !p->inst_load_us || !p->inst_speed_permille))
    return fail(h, NALAR_EINVAL, "NULL instance array");
  if (N > 0 && (!r->order || !r->slack_us || !r->route))
    return fail(h, NALAR_EINVAL, "NULL output array");
  return NALAR_OK;
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
  void end() {
    if (!h->timing) return;
    const int k = n < kMaxTimed ? n : kMaxTimed;
    (void)hipEventRecord(h->ev[k], h->stream);
  }
};

const char* kSortPassNames[kMaxSortPasses] = {"sort_pass0", "sort_pass1", "sort_pass2",
                                              "sort_pass3", "sort_pass4", "sort_pass5",
                                              "sort_pass6", "sort_pass7"};
const char* kGroupPassNames[kMaxGroupPasses] = {"group_pass0", "group_pass1", "group_pass2",
                                                "group_pass3"};

}  // namespace

extern "C" {

int nalar_policy_create(const nalar_policy_config* cfg, nalar_policy** out) {
  g_create_error.clear();
  if (out) *out = nullptr;
  if (!cfg || !out) {
    g_create_error = "NULL config or output";
    return NALAR_EINVAL;
  }
  if ((cfg->flags & ~NALAR_FORCE_GLOBAL_SWEEP) != 0 || cfg->reserve_nodes < 0 ||
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
  e = prepare_sweep_kernels(h->lds_limit);
  if (e != hipSuccess) return bail(e, "hipFuncSetAttribute");
  e = hipHostMalloc(reinterpret_cast<void**>(&h->host_ctrl), sizeof(Ctrl), hipHostMallocDefault);
  if (e != hipSuccess) return bail(e, "hipHostMalloc");
  for (int i = 0; i <= kMaxTimed; ++i) {
    e = hipEventCreate(&h->ev[i]);
    if (e != hipSuccess) return bail(e, "hipEventCreate");
  }
  int rc = ensure_capacity(h, cfg->reserve_nodes, cfg->reserve_workflows);
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
  if (h->ar.base) (void)hipFree(h->ar.base);
  if (h->host_ctrl) (void)hipHostFree(h->host_ctrl);
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

int nalar_policy_pass(nalar_policy* h, const nalar_problem* p, nalar_result* r) {
  if (!h) return NALAR_EINVAL;
  h->err.clear();
  h->timed_valid = false;
  int rc = check_problem(h, p, r);
  if (rc != NALAR_OK) return rc;
  hipError_t e = hipSetDevice(h->device);
  if (e != hipSuccess) return hip_fail(h, e, "hipSetDevice");
  const int64_t N = p->n_nodes, W = p->n_workflows, M = p->n_instances;
  rc = ensure_capacity(h, N, W);
  if (rc != NALAR_OK) return rc;
  Arena& A = h->ar;
  hipStream_t s = h->stream;

  h->epoch = (h->epoch + 1) & kEpochMask;
  if (h->epoch == 0) {  // tags wrapped: forget every old look-back word
    e = hipMemsetAsync(static_cast<char*>(A.base) + A.lookback_off, 0, A.lookback_bytes, s);
    if (e != hipSuccess) return hip_fail(h, e, "hipMemsetAsync(look-back)");
    h->epoch = 1;
  }
  const uint32_t epoch = h->epoch;

  ProblemDev pd{N, p->n_edges, W, M, p->now_us, p->migration_cost_us,
                p->wf, p->type, p->est_us, p->done, p->loc, p->dep_off, p->dep_idx,
                p->deadline_us, p->inst_type, p->inst_load_us, p->inst_speed_permille};
  const bool contiguous = (p->flags & NALAR_WF_CONTIGUOUS) != 0 || W <= 1;

  Timer tm{h};
#define NALAR_LAUNCH(name, call)                  \
  do {                                            \
    tm.mark(name);                                \
    hipError_t le_ = (call);                      \
    if (le_ != hipSuccess) return hip_fail(h, le_, name); \
  } while (0)

  NALAR_LAUNCH("setup", launch_setup(s, pd, A.ctrl, A.itab, A.ghist_slack, A.ghist_group));
  NALAR_LAUNCH("nodes", launch_nodes(s, pd, A.ctrl, A.wf_off, contiguous ? 1 : 0));

  const int32_t* node_of_pos = nullptr;
  const int32_t* pos_of_node = nullptr;
  if (N > 0 && !contiguous) {
    int bits = 0;
    while ((int64_t(1) << bits) < W) ++bits;
    const int gpass = (bits + kRadixBits - 1) / kRadixBits;
    RadixDesc g{};
    g.wf = p->wf;
    g.key_buf[0] = A.gkey[0];
    g.key_buf[1] = A.gkey[1];
    g.pay_buf[0] = A.gpay[0];
    g.pay_buf[1] = A.gpay[1];
    g.count_dev = nullptr;
    g.count_host = N;
    g.first_span = N;
    g.lookback = A.glb;
    g.ghist = A.ghist_group;
    g.tiles_cap = tiles_of(A.capN);
    g.npass_host = gpass;
    g.ticket_base = 8;
    NALAR_LAUNCH("group_hist", launch_radix_hist(s, g, A.ctrl, kSrcWf, N, false));
    for (int ps = 0; ps < gpass; ++ps)
      NALAR_LAUNCH(kGroupPassNames[ps],
                   launch_radix_pass(s, g, A.ctrl, ps == 0 ? kSrcWf : kSrcBuffers, ps, epoch, N,
                                     false));
    const int fin = (gpass - 1) & 1;
    NALAR_LAUNCH("group_finish", launch_group_finish(s, pd, A.ctrl, A.gkey[fin], A.gpay[fin],
                                                     A.pos_of_node, A.wf_off));
    node_of_pos = reinterpret_cast<const int32_t*>(A.gpay[fin]);
    pos_of_node = A.pos_of_node;
  }

  if (N > 0) {
    SweepArgs sa{};
    sa.p = pd;
    sa.itab = A.itab;
    sa.wf_off = A.wf_off;
    sa.node_of_pos = node_of_pos;
    sa.pos_of_node = pos_of_node;
    sa.rem_out = r->rem_us;
    sa.stg_ready = A.stg_ready;
    sa.stg_slack = A.stg_slack;
    sa.stg_route = A.stg_route;
    sa.stg_cost = A.stg_cost;
    sa.g_cnt = A.g_cnt;
    sa.g_mx = A.g_mx;
    sa.g_dn = A.g_dn;
    sa.g_nr = A.g_nr;
    sa.g_front0 = A.g_front[0];
    sa.g_front1 = A.g_front[1];
    sa.ctrl = A.ctrl;
    sa.force_global = (h->flags & NALAR_FORCE_GLOBAL_SWEEP) ? 1 : 0;
    const SweepShape sh = plan_sweep(N, W, M, h->cus, h->lds_limit);
    NALAR_LAUNCH("sweep", launch_sweep(s, sa, sh));

    RadixDesc d{};
    d.stg_slack = A.stg_slack;
    d.stg_ready = A.stg_ready;
    d.key_buf[0] = A.skey[0];
    d.key_buf[1] = A.skey[1];
    d.pay_buf[0] = A.spay[0];
    d.pay_buf[1] = A.spay[1];
    d.count_dev = &A.ctrl->n_ready;
    d.count_host = 0;
    d.first_span = N;
    d.lookback = A.slb;
    d.ghist = A.ghist_slack;
    d.tiles_cap = tiles_of(A.capN);
    d.npass_host = -1;
    d.ticket_base = 0;
    NALAR_LAUNCH("sort_hist", launch_radix_hist(s, d, A.ctrl, kSrcStaged, N, true));
    for (int ps = 0; ps < kMaxSortPasses; ++ps)
      NALAR_LAUNCH(kSortPassNames[ps], launch_radix_pass(s, d, A.ctrl,
                                                         ps == 0 ? kSrcStaged : kSrcBuffers, ps,
                                                         epoch, N, true));
    EmitArgs ea{};
    ea.ctrl = A.ctrl;
    ea.node_of_pos = node_of_pos;
    ea.stg_route = A.stg_route;
    ea.stg_cost = A.stg_cost;
    ea.key_buf[0] = A.skey[0];
    ea.key_buf[1] = A.skey[1];
    ea.pay_buf[0] = A.spay[0];
    ea.pay_buf[1] = A.spay[1];
    ea.order = r->order;
    ea.slack = r->slack_us;
    ea.route = r->route;
    ea.cost = r->cost_us;
    NALAR_LAUNCH("emit", launch_emit(s, ea, N));
  }
#undef NALAR_LAUNCH
  tm.end();
  e = hipMemcpyAsync(h->host_ctrl, A.ctrl, sizeof(Ctrl), hipMemcpyDeviceToHost, s);
  if (e != hipSuccess) return hip_fail(h, e, "hipMemcpyAsync(status)");
  e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(h, e, "hipStreamSynchronize");
  if (h->timing) {
    h->n_timed = tm.n;
    for (int i = 0; i < tm.n; ++i) (void)hipEventElapsedTime(&h->ms[i], h->ev[i], h->ev[i + 1]);
    h->timed_valid = true;
  }
  const uint32_t st = h->host_ctrl->status;
  if (st & kStInval) return fail(h, NALAR_EINVAL, "invalid problem data");
  if (st & kStCycle) return fail(h, NALAR_ECYCLE, "dependency cycle");
  if (st & kStRange) return fail(h, NALAR_ERANGE, "remaining critical path exceeds 2^62 us");
  r->n_ready = N > 0 ? h->host_ctrl->n_ready : 0;
  return NALAR_OK;
}

}  // extern "C"
