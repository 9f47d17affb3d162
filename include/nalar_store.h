/*
 * nalar_store.h -- device-resident graph store of the global policy pass.
 *
 * The global controller keeps a view of every in-flight future, fed by
 * component-level controllers as futures are created with their dependencies
 * and as their values materialise (the future operations and dynamic graph
 * extraction of Section 4.3.1; Table 3's future metadata).  A store keeps
 * that view in HBM across passes and takes it in deltas: futures appended at
 * the end of the id space with their dependency lists, futures marked done,
 * workflow deadlines and the instance table replaced.  A pass over the store
 * is exactly nalar_policy_pass over the snapshot the deltas add up to, without
 * uploading or rebuilding that snapshot.
 *
 * Every array argument is a DEVICE pointer owned by the caller and only read
 * during the call (copied into the store on the handle's stream; the call
 * returns after the copies are enqueued, so the caller may reuse its buffers
 * once the stream has passed them).  Ids are assigned in append order: the
 * first appended future is id 0.  Validation of contents (ranges, workflows
 * of dependencies, cycles) happens in the pass, with the return codes of
 * nalar_policy_pass; the calls here check sizes and pointers only.
 */
#ifndef NALAR_STORE_H
#define NALAR_STORE_H

#include <stdint.h>

#include "nalar_policy.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct nalar_store nalar_store;   /* opaque; bound to one policy handle */

/* An empty store using h's device and stream (h must outlive it).  Returns
 * NALAR_OK, NALAR_EINVAL (NULL arguments) or NALAR_ENOMEM. */
int nalar_store_create(nalar_policy* h, nalar_store** out);

/* Release the store's device memory.  NULL-safe.  Waits for the stream. */
void nalar_store_destroy(nalar_store* s);

/* Append n_new futures (ids N .. N+n_new-1, N the current count) with
 * n_new_edges dependencies: wf, type, est_us, done, loc as in nalar_problem
 * ([n_new] each); dep_off [n_new+1] with dep_off[0] = 0 and dep_off[n_new] =
 * n_new_edges, relative to this call; dep_idx [n_new_edges] ids of any future
 * already stored or appended here.  flags: NALAR_WF_CONTIGUOUS if, after this
 * call, the nodes of every workflow still occupy one ascending id range in
 * workflow order (the store forgets the promise once a call omits it).
 * NALAR_EINVAL for negative sizes, NULL arrays with non-zero sizes or totals
 * past the limits of nalar_problem. */
int nalar_store_append(nalar_store* s, int64_t n_new, int64_t n_new_edges, const int32_t* wf,
                       const int32_t* type, const int64_t* est_us, const uint8_t* done,
                       const int32_t* loc, const int32_t* dep_off, const int32_t* dep_idx,
                       uint32_t flags);

/* Mark n futures done (their values materialised): ids [n], each in [0, N)
 * (an id out of range makes the next pass NALAR_EINVAL).  Duplicates are
 * allowed. */
int nalar_store_complete(nalar_store* s, int64_t n, const int32_t* ids);

/* Replace the workflow deadlines: deadline_us [n_workflows]. */
int nalar_store_set_workflows(nalar_store* s, int64_t n_workflows, const int64_t* deadline_us);

/* Replace the instance table: inst_type, inst_load_us, inst_speed_permille
 * [n_instances] as in nalar_problem. */
int nalar_store_set_instances(nalar_store* s, int64_t n_instances, const int32_t* inst_type,
                              const int64_t* inst_load_us, const int32_t* inst_speed_permille);

/* Number of futures stored (N), or -1 for a NULL store. */
int64_t nalar_store_n_nodes(const nalar_store* s);

/* One pass over the stored snapshot, as nalar_policy_pass on the policy
 * handle the store is bound to: now_us and migration_cost_us as in
 * nalar_problem, policy the NALAR_ORDER_LPT / NALAR_ORDER_SRTF /
 * NALAR_ROUTE_STATEFUL / NALAR_ROUTE_GREEDY bits (the store keeps no routing
 * weights: NALAR_ROUTE_WEIGHTED is NALAR_EINVAL); r as in nalar_policy_pass.
 * Synchronous.
 *
 * The results are those of nalar_policy_pass over the snapshot, however they
 * are computed.  After a successful pass the store keeps every future's
 * remaining critical path (Section 4.3.1's dynamic graph: a future's remaining
 * path depends only on it and on the futures that consume it, transitively),
 * and the next pass is incremental: it recomputes the remaining path only for
 * the futures appended or completed since and for the futures they depend on,
 * transitively; readiness, keys, routes and the order are computed afresh
 * for every ready future, ties broken by (workflow, id) without grouping the
 * ids.  A pass falls back to a full one when there was no successful earlier
 * pass, when the sort has no splitters from an earlier pass or its bins
 * overflow, or when the incremental rounds leave work.  The first failing
 * pass (any error code) also makes the next one full.  An appended
 * dependency list must start at 0, end at n_new_edges and never decrease;
 * otherwise the next pass returns NALAR_EINVAL. */
int nalar_store_pass(nalar_store* s, int64_t now_us, int64_t migration_cost_us, uint32_t policy,
                     nalar_result* r);

/* Incremental passes on (enable != 0, the default) or off (every pass a full
 * one).  NALAR_EINVAL for a NULL store. */
int nalar_store_set_incremental(nalar_store* s, int enable);

/* 1 if the last nalar_store_pass was incremental, 0 if it was a full pass,
 * -1 for a NULL store. */
int nalar_store_last_pass_incremental(const nalar_store* s);

/* Why the last pass was a full one: 0 (it was incremental) or one of the
 * NALAR_STORE_FULL_* reasons; -1 for a NULL store. */
#define NALAR_STORE_FULL_DISABLED      1  /* nalar_store_set_incremental(s, 0)                 */
#define NALAR_STORE_FULL_NO_STATE      2  /* no successful pass since the first append or an error */
#define NALAR_STORE_FULL_SHRUNK        3  /* fewer workflows or instances than at the last pass */
#define NALAR_STORE_FULL_NO_SPLITTERS  4  /* the handle has no splitters from an earlier pass  */
#define NALAR_STORE_FULL_OVERFLOW      5  /* a bin of the partition sort overflowed            */
#define NALAR_STORE_FULL_ROUNDS        6  /* the incremental rounds left work                  */
int nalar_store_last_fallback(const nalar_store* s);

#ifdef __cplusplus
}
#endif

#endif /* NALAR_STORE_H */
