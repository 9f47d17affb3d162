// Launch interface between the host orchestration (api.cpp) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.hpp"

namespace nalar {

// Device view of one snapshot (the arrays of nalar_problem).
struct ProblemDev {
  int64_t N, E, W, M;
  int64_t now, mig;
  uint32_t policy;              // NALAR_ORDER_* and NALAR_ROUTE_* bits
  uint32_t pad_;
  const int32_t* wf;
  const int32_t* type;
  const int64_t* est;
  const uint8_t* done;
  const int32_t* loc;
  const int32_t* dep_off;
  const int32_t* dep_idx;
  const int64_t* deadline;
  const int32_t* inst_type;
  const int64_t* inst_load;
  const int32_t* inst_speed;
  const uint8_t* prio;          // [W] priority level per workflow, or NULL
  const uint32_t* inst_weight;  // [M] routing weights (NALAR_ROUTE_WEIGHTED), or NULL
};

enum RadixSource : int {
  kSrcStaged = 1,   // ready futures staged by position (slack sort)
  kSrcWf = 2,       // workflow ids (grouping)
};

struct SortArgs {
  Ctrl* ctrl;
  Ctrl* next_ctrl;              // reset here for the following pass
  HostStatus* host;             // pinned: status and ready count for the host
  const int64_t* stg_slack;     // [N] by position
  const uint8_t* stg_ready;     // [N] by position: 1 + priority level if ready, else 0
  const int32_t* stg_route;
  const int64_t* stg_cost;
  const int32_t* node_of_pos;   // NULL: position == node id
  const int64_t* out_slack;     // [N] by position, or NULL: the slack is the key
  int64_t span;                 // N
  uint64_t* key[2];             // ping-pong buffers
  uint32_t* pay[2];
  uint64_t* lookback;           // [passes][tiles_cap][256]
  int64_t tiles_cap;
  uint64_t* bagg;               // [kBucketLbGroups] futures per group of buckets
  uint32_t epoch;
  uint32_t levels;              // nonzero: the keys carry priority levels
  int64_t* split_next;          // [kBinMax - 1] this pass's key quantiles, for the next pass
  int64_t split_min;            // fewest ready futures that get splitters
  int32_t passes_launched;      // tiled sort: digit passes launched so far (the
                                //   splitters wait for the last one)
  const int32_t* tie_wf;        // bin sort: positions are node ids, equal keys ordered by
                                //   (tie_wf[id], id); NULL: by position
  ProblemDev p;                 // the snapshot (deadline, wf and the key's policy for the splitters)
  int32_t* order;
  int64_t* slack;
  int32_t* route;
  int64_t* cost;
};

struct GroupArgs {
  ProblemDev p;
  Ctrl* ctrl;
  int npass;                    // digit passes over the workflow ids
  uint32_t* key[2];
  uint32_t* pay[2];
  uint64_t* lookback;
  int64_t tiles_cap;
  uint32_t epoch;
  int32_t* pos_of_node;
  int32_t* wf_off;
  int64_t cap_n;                // entries each key and payload buffer holds
};

// Buckets of the bucketed slack sort (nb == 0: not used this pass).  Bucket of
// a key k: min((k - lo) >> shift, nb - 1), 0 below lo.  With priority levels
// (ngroups > 0) the buckets form ngroups groups of 2^lshift, one per level from
// lvl_hi down; a key of level l falls into group lvl_hi - l (same mapping,
// 2^lshift buckets); a level above lvl_hi takes bucket 0 and one below the
// last group bucket nb - 1, so buckets still ascend in (-level, key), and the
// ranking inside a bucket compares levels first.
//
// Bins (bins != 0, the partition sort of large ready sets, block sweep only):
// nb bins of `cap` records, the bin of a key being the number of splitters
// (split, nb - 1 ascending keys: the previous pass's key quantiles) at or below
// it; cnt holds each bin's claimed records and slot its records.
struct BucketArgs {
  int64_t lo;
  int32_t shift;
  int32_t nb;
  uint32_t* cnt;                // [nb] futures dropped into each bucket (16-byte aligned)
  BucketSlot* slot;             // [nb * kBucketCap], or [nb * cap] with bins
  int32_t lvl_hi;
  int16_t ngroups;
  int16_t lshift;
  int32_t bins;                 // nonzero: key bins
  int32_t cap;                  // records per bin
  const int64_t* split;         // [nb - 1] splitters
};

struct SweepArgs {
  ProblemDev p;
  ITab itab;
  const int32_t* wf_off;        // [W+1] first position of each workflow
  const int32_t* node_of_pos;   // NULL: position == node id
  const int32_t* pos_of_node;   // NULL: position == node id
  int64_t* rem_out;             // [N] or NULL
  uint8_t* stg_ready;           // [N] by position: 1 + priority level if ready, else 0
  int64_t* stg_oslack;          // [N] by position: slack of ready futures when the
                                //   sort key is not the slack (NALAR_ORDER_LPT or
                                //   _SRTF, or priority levels)
  int64_t* stg_slack;           // [N] by position, written for ready futures
  int32_t* stg_route;
  int64_t* stg_cost;
  int32_t* g_cnt;               // HBM sweep state, by position
  int64_t* g_mx;
  uint8_t* g_dn;
  uint8_t* g_nr;
  int32_t* g_front0;
  int32_t* g_front1;
  Ctrl* ctrl;
  BucketArgs bk;
  int force_global;
  // fused mode (workflow-contiguous ids, wave path): the sweep itself
  // validates the snapshot, finds each workflow's bounds, builds the
  // instance table and resets the next pass's control block
  int fused;
  Ctrl* next_ctrl;
  uint32_t* bk_clear;           // bucket counters of the next pass, zeroed here
  int64_t bk_clear_n;
};

// What the block sweep alone takes besides SweepArgs (the wave kernel's
// arguments stay within eight 64-byte lines).
struct BlockSweepArgs {
  const uint32_t* done_bits;    // [N bits] done flags, one bit per future
  int ordered;                  // workflows kept in HBM may take the ordered chunk pass
  int64_t* plog_r;              // [plog_cap] the ordered pass's pushes into earlier chunks:
  int32_t* plog_lp;             //   value and target position (null: no log, no ordered pass)
  int64_t plog_cap;
};

// Load-aware routing over the ordered ready futures (greedy.hip).
struct GreedyArgs {
  const int32_t* order;         // [R] the pass's output order
  int64_t R;
  const int32_t* type;
  const int64_t* est;
  const int32_t* loc;
  const int32_t* inst_type;
  const int64_t* inst_load;
  const int32_t* inst_speed;
  int32_t M;
  int32_t stateful;             // NALAR_ROUTE_STATEFUL pins apply
  int64_t mig;
  int32_t* route;               // [R] overwritten, aligned with order
  int64_t* cost;                // [R] or NULL
  HostStatus* host;             // aux_status receives kStRange on a load overflow
};
hipError_t launch_route_greedy(hipStream_t s, const GreedyArgs& g);

// Weighted routing over the ordered ready futures (weighted.hip).  The table
// kernel also checks every weight against NALAR_WEIGHT_MAX (kStInval into
// ctrl->status, so it runs before the sweep and the error keeps its
// precedence); the other kernels run after a successful pass.
struct WeightedArgs {
  const int32_t* order;         // [R] the pass's output order
  int64_t R;
  const int32_t* type;
  const int64_t* est;
  const int32_t* loc;
  const int32_t* inst_type;
  const int64_t* inst_load;
  const int32_t* inst_speed;
  const uint32_t* inst_weight;
  int32_t M;
  int32_t stateful;             // NALAR_ROUTE_STATEFUL pins apply
  int64_t mig;
  int32_t* route;               // [R] overwritten for weighted futures
  int64_t* cost;                // [R] or NULL
  Ctrl* ctrl;                   // validation status of the pass
  // scratch: the weighted instances sorted by (type, index)
  int32_t* wt_type;
  int32_t* wt_idx;
  uint32_t* wt_cum;
  uint32_t* wt_tot;
  int32_t* wt_first;
  int32_t* wt_cnt;
  int32_t* n_wt;
  uint32_t* counts;             // [tiles][NALAR_MAX_INSTANCES]
  int64_t tiles;                // weighted_tiles(R)
};
int64_t weighted_tiles(int64_t R);
hipError_t launch_weighted_table(hipStream_t s, const WeightedArgs& g);
hipError_t launch_route_weighted(hipStream_t s, const WeightedArgs& g, void (*mark)(void*, const char*),
                                 void* ctx);

// Per-event decisions (decide.hip): one wavefront per event.
struct DecideArgs {
  ProblemDev p;
  const int64_t* rem;           // [N] remaining critical path (the last pass's)
  const int32_t* order;         // [n_order] the current order
  const int64_t* slack;         // [n_order] aligned with order
  int64_t n_order;
  const int32_t* events;        // [n_events] future ids
  int64_t n_events;
  int64_t* slack_out;           // [n_events]
  int32_t* route_out;
  int64_t* cost_out;            // or NULL
  int64_t* rank_out;            // or NULL
  HostStatus* host;             // aux_status receives kStInval for an id out of range
};
hipError_t launch_decide(hipStream_t s, const DecideArgs& a);

// Incremental pass over the graph store (incremental.hip).  Rounds of the
// closure and of its sweep append to per-round lists (items of round r follow
// those of rounds 0 .. r-1); the host launches kIncRounds rounds of each.
constexpr int kIncRounds = 8;

struct IncCtrl {
  uint32_t a_n;                  // closure members
  uint32_t r_n;                  // ready futures
  uint32_t fin;                  // closure members finalised by the sweep
  uint32_t scan_heavy;           // futures with many dependencies, for the scan
  uint32_t cl[kIncRounds + 1];   // closure: single futures per round
  uint32_t ch[kIncRounds + 1];   // closure: futures expanded by a workgroup
  uint32_t sl[kIncRounds + 1];   // sweep: single futures per round
  uint32_t sh[kIncRounds + 1];   // sweep: futures pushed by a workgroup
};

struct IncArgs {
  ProblemDev p;                  // the store's snapshot
  int64_t n_prev;                // futures rem covers from the last pass
  const int32_t* log;            // [n_log] ids completed since the last pass
  int64_t n_log;
  int64_t* rem;                  // [N] remaining critical path, kept across passes
  uint32_t* inA;                 // [ceil(N/32)] closure membership bits (cleared by the pack)
  uint32_t* dnb;                 // [ceil(N/32)] done flags as bits (written by the pack)
  int64_t* mxA;                  // [N] max rem over consumers (closure members)
  int32_t* cntA;                 // [N] closure consumers not yet finalised (members)
  int32_t* light;                // [N] per-round lists
  int32_t* heavy;                // [N]
  int32_t* rlist;                // [N] ready futures
  IncCtrl* ic;                   // zero on entry
  Ctrl* ctrl;                    // the pass's control block
  ITab itab;
  BucketArgs bk;                 // bins (the previous pass's splitters)
  uint32_t* bk_clear;            // the next pass's bin counters, zeroed here
  int64_t bk_clear_n;
  int64_t* stg_oslack;           // [N] slack by id when the key is not the slack
};
size_t inc_ready_lds(int64_t M);
hipError_t prepare_inc_kernels();
hipError_t launch_inc_clear(hipStream_t s, uint32_t* p, int64_t n_words);
// Clears the membership bits and packs the done flags into bits.
hipError_t launch_inc_pack(hipStream_t s, const IncArgs& a);
// (mark(ctx, name) before each launch, for timing)
hipError_t launch_inc_closure(hipStream_t s, const IncArgs& a, int cus, void (*mark)(void*, const char*), void* ctx);
hipError_t launch_inc_scan(hipStream_t s, const IncArgs& a, int cus);
hipError_t launch_inc_sweep(hipStream_t s, const IncArgs& a, int cus, void (*mark)(void*, const char*), void* ctx);
hipError_t launch_inc_ready(hipStream_t s, const IncArgs& a, int cus);

// The store's side of an incremental pass (defined in api.hip): its buffers,
// and the pass.  Returns a NALAR_* code, or one of the kIncFallback codes when
// the pass must be a full one instead.
constexpr int kIncFallback = 1000;          // no splitters or another precondition
constexpr int kIncFallbackOverflow = 1001;  // a bin overflowed
constexpr int kIncFallbackRounds = 1002;    // the rounds left work
inline bool inc_fallback(int rc) { return rc >= kIncFallback && rc <= kIncFallbackRounds; }
struct IncStore {
  int64_t n_prev;
  const int32_t* log;
  int64_t n_log;
  int64_t* rem;
  uint32_t* inA;
  uint32_t* dnb;
  int64_t* mxA;
  int32_t* cntA;
  int32_t* light;
  int32_t* heavy;
  int32_t* rlist;
  IncCtrl* ic;
};
int policy_pass_incremental(nalar_policy* h, const nalar_problem* p, nalar_result* r, const IncStore& st);
// Full passes of the store leave splitters for any number of ready futures.
void policy_split_any(nalar_policy* h, bool on);
// Grows the handle's pass arena ahead of a pass over N futures of W
// workflows (geometrically, like the pass itself), so that a store reallocates
// while taking in its deltas rather than inside a pass.
int policy_reserve(nalar_policy* h, int64_t N, int64_t E, int64_t W);

// Handle accessors for the graph store (store.hip), defined in api.hip.
hipStream_t policy_stream(const nalar_policy* h);
int policy_device(const nalar_policy* h);
int policy_fail(nalar_policy* h, int code, const char* msg);

// ingest.hip
// Validates the futures from v_begin on (and every deadline and instance).
// done_bits (or null, and only with v_begin = 0): the done flags packed one
// bit per future, bit v % 64 of word v / 64.
hipError_t launch_nodes(hipStream_t s, const ProblemDev& p, Ctrl* ctrl, Ctrl* next_ctrl, ITab itab,
                        int32_t* wf_off, int contiguous, int64_t v_begin = 0, uint64_t* done_bits = nullptr);

// sort.hip (mark(ctx, name) is called before each launch, for timing)
hipError_t launch_reset(hipStream_t s, Ctrl* c, uint32_t* clear, int64_t n_clear);
hipError_t launch_bucket_sort(hipStream_t s, const SortArgs& a, const BucketArgs& bk);
hipError_t launch_bin_sort(hipStream_t s, const SortArgs& a, const BucketArgs& bk);
hipError_t prepare_sort_kernels();  // LDS limits of the sort kernels (at handle creation)
// The next pass's splitters from this pass's output (after the tiled or the
// bucketed sort of a large ready set).
hipError_t launch_splitters(hipStream_t s, const SortArgs& a);
hipError_t launch_slack_sort(hipStream_t s, const SortArgs& a, int first_pass, int last_pass,
                             void (*mark)(void*, const char*), void* ctx);
hipError_t launch_group(hipStream_t s, const GroupArgs& a, void (*mark)(void*, const char*),
                        void* ctx);

// sweep.hip
struct SweepShape {
  int threads;    // workgroup size
  int npt;        // futures owned per thread in the LDS path
  int lds_cap;    // largest workflow handled in LDS
  size_t lds_bytes;
  int blocks;
  int wave_path;      // one wave per workflow or group of workflows (k_sweep_wave)
  int group = 1;      // wave path: consecutive workflows swept together by one wave
};
SweepShape plan_sweep(int64_t N, int64_t W, int64_t M, int device_cus, size_t lds_limit);
hipError_t prepare_sweep_kernels(size_t lds_limit);
hipError_t launch_sweep(hipStream_t s, const SweepArgs& a, const BlockSweepArgs& ba, const SweepShape& shape);
// Whether the sweep can do validation, workflow bounds and the instance table
// itself (no node kernel): ids grouped by workflow, wave path, small table.
bool sweep_can_fuse(const SweepShape& shape, int64_t M, bool contiguous);

}  // namespace nalar
