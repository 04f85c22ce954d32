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

// What a simulation unit is: a one-worker design point, or one device of a
// disaggregated point (a prefill device, or a decode device).
enum : int { kStageOne = 0, kStagePrefill = 1, kStageDecode = 2, kStages = 3 };

// Per simulation unit constants, derived on the host at create time.
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
  int64_t cap_po2;      // prefill device: a prompt + output above this never fits a decode device
  int32_t out_point;    // the design point's row (latencies, per-request records)
  int32_t pd;           // disaggregated point's PdAux index, -1 for a one-worker point
  int32_t unit;         // prefill or decode device index within its point
  int32_t resume;       // hand-over state slot of a point a launch may hand on, else -1
};

constexpr int kMaxDev = TS_MAX_DEVICES;

// One disaggregated design point: where its devices' data lives.  Prefill
// device w writes the requests it hands to decode device v, in completion
// order, to the sub-list (w, v) and its length to sub_cnt; the merge kernel
// orders each decode device's arrivals from those sub-lists.
struct __attribute__((aligned(16))) PdAux {
  int32_t n_p, n_d;       // prefill and decode devices
  int32_t point;          // the design point's row
  int32_t res0;           // result record of prefill device 0; decode device v at res0 + n_p + v
  int32_t dec_unit0;      // DevPoint of decode device 0 (its request count is set on the device)
  int32_t trace_off;      // the point's trace (original arrivals, prompt and output lengths)
  int32_t n;              // requests in the trace
  int32_t req_base;       // base of the point's per-request entries in the stage buffers
  int32_t no_kv;          // a prefill or decode device has no KV block
  int32_t num_blocks_d;   // a decode device's blocks
  int64_t kv_bpt;         // KV bytes per token
  double inv_link_ns;     // ns per byte of a prefill device's KV link; 0 = instant
  int32_t pad2;
  int32_t sub_off[kMaxDev * kMaxDev];  // (w, v) -> first entry of the sub-list
  int32_t sub_cnt[kMaxDev * kMaxDev];  // (w, v) -> entries written
  int32_t dec_off[kMaxDev];            // decode device v's trace records
};

// Where a design point's requests are: its trace's first record and length
// (the statistics kernel reads the arrivals there).
struct PointInfo {
  int32_t trace_off, n;
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

// Per-lane roofline coefficients (doubles holding exact integers): lane j < 7
// prices operator j as F = f * X_j, B = (b0 + b1 * Y_j) + b2 * Z_j.
struct LaneCoef {
  double f[8], b0[8], b1[8], b2[8];
};

constexpr int kQueueCap = 256;  // >= max_batch: queue + running never exceed max_batch
constexpr int kHandBuckets = 8;  // hand-over lists, by a point's remaining share of requests

// Hand-over state: a point's simulation at the start of the general-path
// iteration whose admissions needed more running slots than its launch has.
// The wider launch continues from this state instead of simulating the
// point again from the start.  Per slot: the head below,
// then up to kResumeSlots running requests, then the preempted queue.
struct __attribute__((aligned(16))) ResumeHead {
  int64_t t, n_iters, n_pre_tot, pf_tok, dec_tok;
  double ubns;
  int64_t counted;  // iterations the narrower launches counted as theirs
  int32_t freeb, nrun, npre, next, next_new, nwait, wbase, head_need, peak, n_done;
  int32_t valid;    // 0: the point starts over in the wider launch
};
struct __attribute__((aligned(8))) ResumeSlot {
  int32_t ctx, tgt, rem, room, fl, q, id, npre;
  int64_t gap;
};
constexpr int kResumeSlots = 128;  // the widest launch that hands points on has 128 slots
constexpr size_t kResumeHead = 128;
constexpr size_t kResumeBytes =
    kResumeHead + kResumeSlots * sizeof(ResumeSlot) + kQueueCap * sizeof(QEntry);
static_assert(sizeof(ResumeHead) <= kResumeHead, "hand-over head fits its space");

struct SimArgs {
  TraceRec* recs;              // traces, prefill devices' shares, decode devices' arrivals
  const DevPoint* points;
  const int32_t* order;        // points of this launch, longest expected first
  int32_t n_order;
  int32_t max_n;               // row stride of the per-request buffers
  unsigned int* counter;       // work queue ticket counter (zeroed before launch)
  QEntry* queue;               // kQueueCap entries per workgroup
  ts_point_result* res;
  // max_n per point (row = design point): the request records.  Admission
  // and first token are written when they happen, the rest at the finish;
  // until then finish_ns holds the time of the request's last token before a
  // preemption.
  ts_req_result* rec;
  int64_t iter_cap;
  uint64_t time_limit_ticks;   // 0 = none; 100 MHz device clock ticks per point
  unsigned long long* work;    // simulated iterations of the points completed by this launch
  // A narrow launch also takes points wider than its slots and hands those
  // that need more running slots to the launch with twice the slots: handed
  // (the lists the 64-slot launch fills at handed_off[0], the 128-slot one at
  // handed_off[1], one per remaining-work bucket, hand_cap entries apart) and
  // handed_n (their counts).  A launch taking over handed points reads its
  // bucket counts at n_dev (nullptr otherwise).
  int32_t* handed;
  int32_t handed_off[2];
  int32_t hand_cap[2];         // entries per bucket list of each hand-over level
  int32_t hand_cap_in;         // ... of the lists this launch takes its points from
  unsigned int* handed_n;      // [2][kHandBuckets] counts
  const unsigned int* n_dev;   // kHandBuckets counts of this launch's points
  // hand-over states (kResumeBytes per DevPoint::resume slot), nullptr when
  // no launch hands points on
  unsigned char* resume;
  // The 64-slot launch, once no point of its own is left, continues points
  // it handed over itself (128 slots) while the others still run: take holds
  // the positions of its kHandBuckets lists taken so far (nullptr when it
  // does not).  claim, per hand-over slot, marks a point that one launch has
  // taken, and the 128-slot launch skips those (nullptr: no claims).
  unsigned int* take;
  unsigned int* claim;
  double n_layers;
  LaneCoef lc;
  // disaggregated points
  PdAux* pd;
  int64_t* s1_admit;           // per request: admission on its prefill device
  int64_t* s1_first;           // per request: first token
  int64_t* sub_a2;             // sub-lists: when the KV reaches the decode device
  int32_t* sub_gid;            // sub-lists: request index
  const int32_t* gids;         // per trace record: request index (decode devices' arrivals)
};

}  // namespace tsw
