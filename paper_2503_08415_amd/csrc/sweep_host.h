// sweep_host.h -- host-side plumbing shared by the entry points of the
// serving-simulation sweep: the plan derived on the host from a call's
// inputs, the device buffers a sweep runs in, and the launch sequence.
// Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <vector>

#include "sweep_internal.h"

namespace tsw {

constexpr int kClasses = 3;                       // register chunks per lane: 1, 2, 4
constexpr int kLaunches = kStages * kClasses;     // launch 3 * stage + class
static_assert(kLaunches == TS_N_SIM_KERNELS, "one timing entry per launch");

// What a sweep needs, derived on the host at create time: validated inputs,
// simulation units (one per one-worker point, one per device of a
// disaggregated point), the per-launch work order, and the records to upload.
struct Plan {
  int device = 0;
  int32_t count = 0;       // design points of the handle
  int32_t max_n = 1;       // longest trace (row stride of the per-request buffers)
  int32_t n_pd = 0;        // disaggregated points
  int64_t n_extra = 0;     // device result records after the points' own
  int64_t pd_reqs = 0;     // per-request entries of the disaggregated points
  uint32_t flags = 0;
  int64_t iter_cap = 0, slo_ttft = 0, slo_tpot = 0, time_limit_ms = 0;
  CostCoef coef{};
  LaneCoef lc{};
  std::vector<TraceRec> recs;   // traces, prefill-device shares, decode-arrival regions
  std::vector<DevPoint> dp;     // simulation units
  std::vector<int32_t> order;   // units per launch, longest expected first, concatenated
  std::vector<PdAux> aux;
  std::vector<PointInfo> pinfo;  // per design point: its trace (statistics kernel)
  int class_off[kLaunches] = {}, class_n[kLaunches] = {};
  int grid[kLaunches] = {};     // persistent workgroups per launch
  bool simple[kLaunches] = {};  // the launch's points are all simple (compile-time policy)
  // The one-worker points are all simple and some are wider than 64 slots:
  // launch 0 takes every one-worker point and hands those needing more than
  // 64 running slots to launch 1 or 2 (class_n[1], class_n[2] bound them).
  bool hand_over = false;
  int n_resume = 0;             // hand-over state slots (points a launch may hand on)
  int stats_grid = 1;
  int max_grid() const;
};

// Element counts of every device buffer of a plan.
struct BufCounts {
  size_t recs, points, order, counter, queue, res, req, lat, pd, s1, sub, gids, pinfo,
      handed, work, resume, claim;
  double bytes() const;  // total, in bytes
};
BufCounts buf_counts(const Plan& P);

// The device buffers a sweep runs in: owned by a handle, or carved out of
// the library's static scratch.
struct DevBufs {
  TraceRec* recs = nullptr;
  DevPoint* points = nullptr;
  int32_t* order = nullptr;
  unsigned int* counter = nullptr;  // work-queue tickets, one per launch, then the handed counts
  unsigned long long* work = nullptr;  // simulated iterations completed per launch
  int32_t* handed = nullptr;        // points handed from launch 0 to launches 1 and 2
  unsigned char* resume = nullptr;  // their hand-over states, kResumeBytes each
  unsigned int* claim = nullptr;    // per hand-over state: taken by a launch
  QEntry* queue = nullptr;          // kQueueCap per workgroup, shared by the launches
  ts_point_result* res = nullptr;
  ts_req_result* req = nullptr;     // the request records, max_n per point (always)
  int64_t* e2e = nullptr;           // max_n per point: latencies for the percentile pass
  int64_t* ttft = nullptr;
  PdAux* pd = nullptr;
  int64_t* s1_admit = nullptr;
  int64_t* s1_first = nullptr;
  int64_t* sub_a2 = nullptr;
  int32_t* sub_gid = nullptr;
  int32_t* gids = nullptr;
  PointInfo* pinfo = nullptr;
};

// HIP events around the launches (timing); any may be null.
struct LaunchEvents {
  hipEvent_t t0 = nullptr, t1 = nullptr, t2 = nullptr;
  hipEvent_t k0[kLaunches] = {};
  hipEvent_t k1[kLaunches] = {};
};

// Validates every input on the host, before any device call, then derives
// the plan (the grid sizes query the current device).
int make_plan(const ts_model* model, const ts_trace* traces, int32_t n_traces,
              const ts_point* points, int32_t n_points, const ts_options* opt, Plan* P);

// Copies the plan's records to the device buffers: synchronously, or on
// stream s (the host vectors must then outlive the copies).
int upload(const Plan& P, const DevBufs& B, bool async, hipStream_t s);

// Enqueues one run on stream s: counter reset, the simulation launches
// (with the merge and combine kernels of disaggregated points), then the
// statistics kernel.
int enqueue(const Plan& P, const DevBufs& B, hipStream_t s, const LaunchEvents* ev);

// Error text for ts_status_str (per thread).
int device_error(hipError_t e, const char* what);
void set_error_text(const char* text);
void clear_error_text();

}  // namespace tsw
