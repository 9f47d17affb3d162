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
};

// Radix-sort plumbing shared by the slack sort and the workflow grouping.
enum RadixSource : int {
  kSrcBuffers = 0,  // keys/payloads from the ping-pong buffers (passes >= 1)
  kSrcStaged = 1,   // ready futures staged by position: key = slack - min slack,
                    // payload = position; non-ready positions are skipped, so the
                    // first pass also compacts (slack sort, pass 0)
  kSrcWf = 2,       // key = workflow id, payload = node id (grouping, pass 0)
};

struct RadixDesc {
  const int64_t* stg_slack; // kSrcStaged source
  const uint8_t* stg_ready; // kSrcStaged validity
  const int32_t* wf;        // kSrcWf source
  void* key_buf[2];         // ping-pong keys (uint64 or uint32)
  uint32_t* pay_buf[2];     // ping-pong payloads
  const int64_t* count_dev; // dense element count in device memory, or NULL
  int64_t count_host;       // dense element count when count_dev is NULL
  int64_t first_span;       // positions scanned by the histogram and pass 0
  uint64_t* lookback;       // [passes][tiles_cap][256]
  uint32_t* ghist;          // [passes][256]
  int64_t tiles_cap;
  int npass_host;           // -1: the histogram kernel decides (slack sort)
  int ticket_base;          // first Ctrl::tile_ticket slot of this sort
};

struct SweepArgs {
  ProblemDev p;
  ITab itab;
  const int32_t* wf_off;        // [W+1] first position of each workflow
  const int32_t* node_of_pos;   // NULL: position == node id
  const int32_t* pos_of_node;   // NULL: position == node id
  int64_t* rem_out;             // [N] or NULL
  uint8_t* stg_ready;           // [N] by position: 1 = ready
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
  int force_global;
};

struct EmitArgs {
  Ctrl* ctrl;
  const int32_t* node_of_pos;   // NULL: position == node id
  const int32_t* stg_route;
  const int64_t* stg_cost;
  const uint64_t* key_buf[2];
  const uint32_t* pay_buf[2];
  int32_t* order;
  int64_t* slack;
  int32_t* route;
  int64_t* cost;
};

// ingest.hip
hipError_t launch_setup(hipStream_t s, const ProblemDev& p, Ctrl* ctrl, ITab itab,
                        uint32_t* ghist_slack, uint32_t* ghist_group);
hipError_t launch_nodes(hipStream_t s, const ProblemDev& p, Ctrl* ctrl, int32_t* wf_off,
                        int contiguous);
hipError_t launch_group_finish(hipStream_t s, const ProblemDev& p, Ctrl* ctrl,
                               const uint32_t* sorted_wf, const uint32_t* sorted_ids,
                               int32_t* pos_of_node, int32_t* wf_off);

// sort.hip
hipError_t launch_radix_hist(hipStream_t s, const RadixDesc& d, Ctrl* ctrl, int src,
                             int64_t max_count, bool key64);
hipError_t launch_radix_pass(hipStream_t s, const RadixDesc& d, Ctrl* ctrl, int src, int pass,
                             uint32_t epoch, int64_t max_count, bool key64);

// sweep.hip
struct SweepShape {
  int threads;    // workgroup size
  int npt;        // futures owned per thread in the LDS path
  int lds_cap;    // largest workflow handled in LDS
  size_t lds_bytes;
  int blocks;
};
SweepShape plan_sweep(int64_t N, int64_t W, int64_t M, int device_cus, size_t lds_limit);
hipError_t prepare_sweep_kernels(size_t lds_limit);
hipError_t launch_sweep(hipStream_t s, const SweepArgs& a, const SweepShape& shape);

// emit.hip
hipError_t launch_emit(hipStream_t s, const EmitArgs& a, int64_t max_count);

}  // namespace nalar
