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
 * Synchronous. */
int nalar_store_pass(nalar_store* s, int64_t now_us, int64_t migration_cost_us, uint32_t policy,
                     nalar_result* r);

#ifdef __cplusplus
}
#endif

#endif /* NALAR_STORE_H */
