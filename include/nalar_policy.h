/*
 * nalar_policy.h -- C ABI of the MI355X global policy pass.
 *
 * The global controller of Nalar's two-level control (Section 4.1) runs one
 * periodic, single-threaded policy loop (Section 4.2).  One iteration of its
 * policy computation over the dependency graph of every in-flight future is a
 * "pass":
 *
 *   1. remaining critical path of every future: the longest service-time
 *      path from the future through its consumers (the remaining-work key
 *      of the SRTF policy, Section 6.2, taken over the whole DAG);
 *   2. readiness: a future is runnable once it is not done and every future it
 *      depends on is done (push-based readiness, Section 4.3.1, property 3);
 *   3. priority: ready futures ranked by deadline slack, least slack first
 *      (set_priority, Table 2; the remaining-work orders of Section 6.2 are
 *      policy variants);
 *   4. routing: each ready future sent to the instance of its component type
 *      with the least load plus speed-scaled service time plus a migration
 *      penalty when its managed state lives on another instance (route and
 *      migrate, Table 2; state locality, Section 4.3.2).
 *
 * All times are int64 fixed-point microseconds and every result is an exact
 * integer: the GPU output is bit-identical to the plain definition.
 *
 * Calls are synchronous: nalar_policy_pass returns after its GPU work on the
 * handle's stream has finished.  A handle is not thread-safe; use one handle
 * per host thread.  All integers are little-endian and naturally aligned.
 */
#ifndef NALAR_POLICY_H
#define NALAR_POLICY_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Return codes.  On any non-OK return the outputs are unspecified and the
 * handle stays usable.  When several apply, the first in this order wins:
 * EINVAL, ECYCLE, ERANGE.  ENOMEM and EDEVICE report the library's own
 * failures (allocation, HIP runtime). */
enum {
  NALAR_OK = 0,
  NALAR_EINVAL = -1,  /* a rule of nalar_problem or nalar_policy_config broken  */
  NALAR_ECYCLE = -2,  /* the dependency graph has a cycle (a self-loop counts)  */
  NALAR_ERANGE = -3,  /* a remaining critical path exceeds NALAR_REM_MAX        */
  NALAR_ENOMEM = -4,  /* device or pinned host allocation failed                */
  NALAR_EDEVICE = -5  /* a HIP runtime call failed; see nalar_policy_last_error */
};

/* Limits of the ABI (values outside them are NALAR_EINVAL). */
#define NALAR_MAX_NODES      (INT64_C(1) << 30)
#define NALAR_MAX_EDGES      (INT64_C(2147483647))
#define NALAR_MAX_WORKFLOWS  (INT64_C(1) << 30)
#define NALAR_MAX_INSTANCES  1024
#define NALAR_EST_MAX        (INT64_C(1) << 40)  /* service time, us            */
#define NALAR_LOAD_MAX       (INT64_C(1) << 60)  /* instance load, us            */
#define NALAR_MIG_MAX        (INT64_C(1) << 60)  /* migration penalty, us        */
#define NALAR_HORIZON_MAX    (INT64_C(1) << 61)  /* |now|, |deadline - now|      */
#define NALAR_REM_MAX        (INT64_C(1) << 62)  /* remaining critical path, us  */
#define NALAR_PRIORITY_MAX   15                  /* highest priority level       */
#define NALAR_WEIGHT_MAX     (1u << 20)          /* routing weight of an instance */

/* nalar_problem.flags */
#define NALAR_WF_CONTIGUOUS  1u  /* the nodes of workflow w are exactly the ids
                                    [first_w, first_{w+1}) with first ascending in
                                    w, i.e. wf[] is non-decreasing.  The caller
                                    promises it; a violation is NALAR_EINVAL.
                                    Without it the library groups nodes by
                                    workflow itself (one extra sort).           */
/* Policy variants of the same pass (nalar_problem.flags; 0 = the default
 * least-slack-first order and load-and-locality routing): */
#define NALAR_ORDER_LPT      2u  /* order = ready futures by (-rem, wf, id)
                                    ascending: longest remaining processing
                                    first (the LPT policy, Section 6.2); the
                                    slack output is unchanged                   */
#define NALAR_ORDER_SRTF    16u  /* order = ready futures by (rem, wf, id)
                                    ascending: least remaining work first
                                    (shortest remaining time first, the policy
                                    that minimises job completion time, Section
                                    6.2); the slack output is unchanged; with
                                    NALAR_ORDER_LPT it is NALAR_EINVAL          */
#define NALAR_ROUTE_STATEFUL 4u  /* a ready future whose state lives on an
                                    instance of its own type (loc[v] >= 0 and
                                    inst_type[loc[v]] == type[v]) is routed there
                                    with no other candidate and no migration
                                    penalty (the stateful directive, Table 1;
                                    managed-state routing, Section 4.3.2); every
                                    other future is routed by the default rule */
#define NALAR_ROUTE_GREEDY   8u  /* load-aware routing: after ordering, the
                                    ready futures are routed one at a time in
                                    output order; each takes the (route rule)
                                    cheapest candidate under the loads left by
                                    the futures before it, then adds its service
                                    time floor(est*1000/speed) on the chosen
                                    instance to that instance's load (routing
                                    that balances load, Section 6.1).  A load
                                    past NALAR_REM_MAX is NALAR_ERANGE.  Futures
                                    of different types are independent
                                    sequences, so this runs one wavefront per
                                    component type                              */
#define NALAR_ROUTE_WEIGHTED 32u /* weighted routing (route with a list of
                                    instances and weights, Table 2): after
                                    ordering, the ready futures of each type
                                    that has instances of positive weight
                                    (inst_weight) are dealt to those instances
                                    in proportion to their weights.  The futures
                                    of type t, in output order, take sequence
                                    numbers j = 0, 1, 2, ...; with the instances
                                    of type t and positive weight listed by
                                    ascending index and S their total weight,
                                    future j goes to the instance whose run of
                                    w[i] consecutive numbers in 0..S-1 holds
                                    j mod S (the first w[0] numbers to the first
                                    instance, the next w[1] to the second, ...),
                                    at that instance's cost.  A future pinned by
                                    NALAR_ROUTE_STATEFUL keeps its pin and takes
                                    no number; a type without a positive weight
                                    keeps its default route.  With
                                    NALAR_ROUTE_GREEDY it is NALAR_EINVAL       */

/* nalar_policy_config.flags (tuning and testing; 0 is the normal setting) */
#define NALAR_FORCE_GLOBAL_SWEEP 1u  /* keep every workflow's sweep state in HBM
                                        instead of LDS (exercises the path used
                                        for workflows too large for LDS)         */
#define NALAR_FORCE_TILED_SORT   2u  /* always order the ready futures with the
                                        tiled radix sort (the path otherwise used
                                        on a handle's first pass, above 131072
                                        ready futures and when a bucket of the
                                        bucketed sort overflows)                 */
#define NALAR_FORCE_LEVEL_SWEEP  4u  /* sweep every workflow kept in HBM level
                                        by level with out-degree counters, also
                                        one whose dependencies all lie at lower
                                        ids (which otherwise takes one pass over
                                        its ids from the last to the first)      */

typedef struct nalar_policy nalar_policy;   /* opaque handle */

/* Creation-time settings.  Host memory, read during nalar_policy_create only. */
typedef struct {
  int32_t device;             /* HIP device ordinal                               */
  uint32_t flags;             /* NALAR_FORCE_* bits or 0                          */
  void* stream;               /* hipStream_t the pass runs on; NULL = null stream */
  int64_t reserve_nodes;      /* scratch pre-size hints (0 = size on first pass)  */
  int64_t reserve_edges;
  int64_t reserve_workflows;
} nalar_policy_config;

/* One snapshot of the global view (Table 3 future metadata, the managed
 * state layer's location of each future's state, and the instance table).
 * Struct in host memory; every array pointer is a DEVICE pointer, owned by the
 * caller and only read during the call.  N = n_nodes, E = n_edges,
 * W = n_workflows, M = n_instances. */
typedef struct {
  int64_t n_nodes;            /* [0, NALAR_MAX_NODES]                             */
  int64_t n_edges;            /* [0, NALAR_MAX_EDGES]; 0 when N = 0              */
  int64_t n_workflows;        /* [0, NALAR_MAX_WORKFLOWS]                         */
  int64_t n_instances;        /* [0, NALAR_MAX_INSTANCES]                         */
  int64_t now_us;             /* |now_us| <= NALAR_HORIZON_MAX                    */
  int64_t migration_cost_us;  /* penalty for running a future away from the
                                 instance holding its state, [0, NALAR_MIG_MAX]   */
  uint32_t flags;             /* NALAR_WF_CONTIGUOUS, NALAR_ORDER_* and
                                 NALAR_ROUTE_* bits, or 0                         */
  uint32_t reserved;          /* must be 0                                        */
  const int32_t* wf;          /* [N] workflow (session) of each future, [0, W)    */
  const int32_t* type;        /* [N] component type, >= 0                         */
  const int64_t* est_us;      /* [N] estimated service time, [0, NALAR_EST_MAX]   */
  const uint8_t* done;        /* [N] 1 = value materialised, 0 = not; else EINVAL */
  const int32_t* loc;         /* [N] instance holding the future's managed state,
                                 [0, M), or -1 for none                           */
  const int32_t* dep_off;     /* [N+1] dependency CSR: dep_off[0] = 0,
                                 non-decreasing, dep_off[N] = E                   */
  const int32_t* dep_idx;     /* [E] futures each future depends on, in [0, N),
                                 same workflow (else EINVAL), duplicates allowed;
                                 a future listing itself is a cycle (ECYCLE)      */
  const int64_t* deadline_us; /* [W] workflow deadline, |deadline - now| <=
                                 NALAR_HORIZON_MAX                                */
  const int32_t* inst_type;   /* [M] component type of each instance, >= 0       */
  const int64_t* inst_load_us;/* [M] queued work, [0, NALAR_LOAD_MAX]            */
  const int32_t* inst_speed_permille; /* [M] speed relative to nominal, >= 1      */
  const uint8_t* wf_priority; /* [W] priority level of each workflow (session),
                                 0..NALAR_PRIORITY_MAX, or NULL for none: the
                                 ready futures of a higher level come first in
                                 the order, whatever their key (set_priority,
                                 Table 2): the order is by (-level, key, wf, id) */
  const uint32_t* inst_weight;/* [M] routing weight of each instance,
                                 0..NALAR_WEIGHT_MAX; read only under
                                 NALAR_ROUTE_WEIGHTED (then required when M > 0),
                                 else may be NULL                                 */
} nalar_problem;

/* Outputs.  Struct in host memory; array pointers are DEVICE pointers, owned by
 * the caller, each with capacity >= n_nodes entries (the ready count R is not
 * known before the call).  Entries past R are left untouched. */
typedef struct {
  int64_t* rem_us;      /* [N] remaining critical path of every future, or NULL */
  int32_t* order;       /* [R] ready futures, ascending (slack, wf, id)          */
  int64_t* slack_us;    /* [R] deadline[wf] - now - rem, aligned with order      */
  int32_t* route;       /* [R] chosen instance, or -1 when no instance has the
                           future's type; aligned with order                     */
  int64_t* cost_us;     /* [R] cost of the chosen instance (INT64_MAX when route
                           is -1), aligned with order; or NULL                   */
  int64_t n_ready;      /* HOST field: R, written before a NALAR_OK return       */
} nalar_result;

/*
 * Create a handle bound to cfg->device and cfg->stream.  *out receives the
 * handle (NULL on failure).  Returns NALAR_OK, NALAR_EINVAL (NULL arguments,
 * negative reserve hints, unknown flags), NALAR_ENOMEM or NALAR_EDEVICE.
 * The library owns only its scratch memory (device and pinned host), which it
 * allocates here (sized by the reserve hints) and grows, never shrinks, inside
 * nalar_policy_pass.
 */
int nalar_policy_create(const nalar_policy_config* cfg, nalar_policy** out);

/*
 * Run one pass over the snapshot *p and write *r.  Definition of each output:
 *   est'[v]  = done[v] ? 0 : est_us[v]
 *   rem[v]   = est'[v] + max(0, max over futures s listing v in their
 *              dependencies of rem[s])
 *   ready[v] = !done[v] and done[u] for every u in v's dependencies
 *   slack[v] = (deadline_us[wf[v]] - now_us) - rem[v]
 *   cost(v,i)= inst_load_us[i] + floor(est_us[v]*1000 / inst_speed_permille[i])
 *              + (loc[v] >= 0 && loc[v] != i ? migration_cost_us : 0)
 *   route[v] = the instance i with inst_type[i] == type[v] minimising
 *              (cost(v,i), i) lexicographically (the lowest index wins ties),
 *              or -1 with cost INT64_MAX when there is none
 *   order    = the ready futures sorted by (slack, wf, id) ascending (behind
 *              the priority level of their workflow, highest first, when
 *              wf_priority is given)
 * (the NALAR_ORDER_* and NALAR_ROUTE_* bits change order and route as
 * described at their definitions).
 * Synchronous.  NULL p, r, or a required array (a node array when N > 0,
 * dep_idx when E > 0, deadline_us when W > 0, an instance array when M > 0,
 * order/slack_us/route when N > 0) is NALAR_EINVAL.  Error precedence and the
 * state of the outputs after an error are as described at the return codes.
 */
int nalar_policy_pass(nalar_policy* h, const nalar_problem* p, nalar_result* r);

/*
 * One-level decisions (the central, per-future control that Section 6.3 and
 * Table 4 contrast with installed policies): decide events one at a time (or
 * a batch of them) against the view the last pass left, instead of running a
 * pass.  The view is that pass's rem_us for every future and its order with
 * the slack of each entry (device pointers, read only).  For each event future
 * v = events[k]:
 *   slack_us[k] = deadline_us[wf[v]] - now_us - rem_us[v]
 *   route[k], cost_us[k] = v's route and cost under the routing rule of
 *              nalar_policy_pass (NALAR_ROUTE_STATEFUL honoured)
 *   rank[k]    = the number of entries of the view's order that come before v
 *              in the pass's order ((-level, key, wf, id) with the key of the
 *              NALAR_ORDER_* bits), i.e. where v enters the current order; a
 *              future already in the order gets its own index.
 * A future's rem does not change when it becomes ready, so the last pass's
 * rem is the one the decision needs.  p must be the snapshot the view came
 * from (its contents are not validated again); NALAR_ROUTE_GREEDY and
 * NALAR_ROUTE_WEIGHTED (which route by position in a whole order) are
 * NALAR_EINVAL.  Synchronous.  NALAR_EINVAL also for NULL or inconsistent
 * arguments (n_order outside [0, N], a NULL view array with entries, NULL
 * slack_us or route with events) and for an event id outside [0, N).
 */
typedef struct {
  const int64_t* rem_us;      /* [N] remaining critical path of every future     */
  const int32_t* order;       /* [n_order] ready futures in the pass's order      */
  const int64_t* slack_us;    /* [n_order] aligned with order                     */
  int64_t n_order;
} nalar_view;

typedef struct {              /* DEVICE arrays of n_events entries, caller-owned */
  int64_t* slack_us;
  int32_t* route;
  int64_t* cost_us;           /* or NULL                                          */
  int64_t* rank;              /* or NULL                                          */
} nalar_decisions;

int nalar_policy_decide(nalar_policy* h, const nalar_problem* p, const nalar_view* view,
                        int64_t n_events, const int32_t* events, nalar_decisions* out);

/*
 * For callers that cannot allocate (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): nalar_policy_pass without
 * any allocation.  Same arguments, results and return codes, but the scratch
 * is a fixed array of NALAR_STATIC_SCRATCH_BYTES of device memory that the
 * library holds on each device from the first handle created there until the
 * process ends, instead of memory allocated for the handle.  Limits:
 * n_nodes <= NALAR_STATIC_MAX_NODES and n_workflows <=
 * NALAR_STATIC_MAX_WORKFLOWS, else NALAR_EINVAL (the bucketed sort is skipped
 * for a ready set too large for the array's buckets).  Every call on one
 * device shares that device's array, which keeps the last call's contents;
 * the library serialises the calls on a device with a lock, so concurrent
 * callers wait for each other (calls are synchronous).
 */
#define NALAR_STATIC_SCRATCH_BYTES (64u << 20)
#define NALAR_STATIC_MAX_NODES     (INT64_C(1) << 18)
#define NALAR_STATIC_MAX_WORKFLOWS (INT64_C(1) << 18)
int nalar_policy_pass_static(nalar_policy* h, const nalar_problem* p, nalar_result* r);

/* Release the handle and its scratch.  NULL-safe.  Waits for the handle's
 * stream first. */
void nalar_policy_destroy(nalar_policy* h);

/* Message describing the last non-OK return on this handle ("" if none).  The
 * string is owned by the handle and valid until its next call.  h may be NULL
 * (returns the message of the last failed nalar_policy_create on this thread). */
const char* nalar_policy_last_error(const nalar_policy* h);

/* Per-kernel timing of the following passes, measured with HIP events recorded
 * on the handle's stream around each kernel (enable != 0 turns it on). */
int nalar_policy_set_timing(nalar_policy* h, int enable);

/* Kernel durations of the last timed pass, in milliseconds: names[i] (static
 * strings owned by the library) and ms[i] for i < *count.  cap is the capacity
 * of both arrays; *count receives the number of kernels the pass launched
 * (entries past cap are dropped).  Returns NALAR_EINVAL if timing is off or no
 * timed pass has run. */
int nalar_policy_get_timing(const nalar_policy* h, const char** names, float* ms, int cap,
                            int* count);

#ifdef __cplusplus
}
#endif

#endif /* NALAR_POLICY_H */
