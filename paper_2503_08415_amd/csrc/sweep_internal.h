// sweep_internal.h -- device data layout shared by the host library and the
// gfx950 kernels of the serving-simulation sweep.  Not part of the public ABI.
#pragma once

#include <stdint.h>

#include "ts_sweep.h"

namespace tsw {

// One request of a trace, 16 bytes: a wave reads 64 consecutive records as
// one contiguous 1 KiB window (one 16-byte load per lane).
struct __attribute__((aligned(16))) TraceRec {
  int64_t arrival_ns;
  int32_t prompt;
  int32_t output;
};

// Per design point constants, derived on the host at create time.
struct __attribute__((aligned(16))) DevPoint {
  double inv_flops_ns;  // 1e9 / peak FLOP/s
  double inv_bw_ns;     // 1e9 / bytes per second
  int64_t cap_tokens;   // num_blocks * block_size: a request with more tokens is rejected
  int32_t num_blocks;
  int32_t block;
  int32_t max_batch;
  int32_t chunk;        // 0 = unlimited per-iteration token budget
  int32_t trace_off;    // first record of the point's trace
  int32_t n;            // requests in the trace
  int32_t out_index;    // index of the point's results
  int32_t may_reject;   // 1 if some request of the trace is rejected
  int32_t lg_iter;      // every iteration takes less than 2^lg_iter ns
  int64_t cap_prompt;   // a prompt above this many tokens is rejected (admission ratio)
  int32_t policy;       // TS_POLICY_*
  int32_t adm_reserve;  // blocks a first admission must leave free
  double inv_link_ns;   // swap preemption: 1e9 / host link bytes per second
  int64_t block_bytes;  // KV bytes of one block
  int32_t swap;         // 1: preemption by swap, 0: by recompute
  int32_t swap_overlap; // 1: transfers overlap the iteration's compute
};

// Integer coefficients of the per-operator roofline (exact below 2^53):
// every FLOP and byte count is an affine function of the batch sums
//   T (tokens), TP (prefill tokens), AP (causal prefill pairs), CP (prefill
//   keys), nD (decodes), CD (decode keys), R (sequences emitting a token).
struct CostCoef {
  int64_t f_qkv, b_qkv0, b_qkv;    // QKV projection: F = f*T, B = b0 + b*T
  int64_t f_attp, b_attp_c, b_attp_t;  // prefill attention: F = f*AP, B = bc*CP + bt*TP
  int64_t f_attd, b_attd_c, b_attd_n;  // decode attention: F = f*CD, B = bc*CD + bn*nD
  int64_t f_out, b_out0, b_out;    // output projection
  int64_t f_up, b_up0, b_up;       // FFN up (+gate)
  int64_t f_dn, b_dn0, b_dn;       // FFN down
  int64_t f_lm, b_lm0, b_lm;       // LM head: F = f*R, B = b0 + b*R (R > 0 only)
  double n_layers;
};

// A preempted request waiting for re-admission, 32 bytes.  After recompute
// preemption ctx is 0 and target covers prompt and decoded tokens; after swap
// preemption both keep the values the request had when it left.
struct __attribute__((aligned(16))) QEntry {
  int32_t id, target, rem, n_pre, flags, ctx;
  int64_t gap;
};

// Per-request times kept by the workgroup simulating a point, indexed by
// request: first admission, first token, and the last token before the
// latest preemption.  Written once per event, read when the request ends.
struct ReqTimes {
  int64_t admit, first, last;
};

// Per-lane roofline coefficients (doubles holding exact integers): lane j < 7
// prices operator j as F = f * X_j, B = (b0 + b1 * Y_j) + b2 * Z_j.
struct LaneCoef {
  double f[8], b0[8], b1[8], b2[8];
};

constexpr int kQueueCap = 256;  // >= max_batch: queue + running never exceed max_batch

struct SimArgs {
  const TraceRec* recs;
  const DevPoint* points;
  const int32_t* order;        // points of this launch, longest expected first
  int32_t n_order;
  int32_t max_n;               // row stride of the per-request buffers
  unsigned int* counter;       // work queue ticket counter (zeroed before launch)
  QEntry* queue;               // kQueueCap entries per workgroup
  ReqTimes* times;             // max_n entries per workgroup
  ts_point_result* res;
  ts_req_result* req;          // nullptr unless per-request records are requested
  int64_t* e2e;                // max_n per point: end-to-end latency of finished requests
  int64_t* ttft;               // max_n per point: time to first token
  int64_t iter_cap;
  int64_t slo_ttft_ns;
  int64_t slo_tpot_ns;
  uint64_t time_limit_ticks;   // 0 = none; 100 MHz device clock ticks per point
  double n_layers;
  LaneCoef lc;
};

}  // namespace tsw
