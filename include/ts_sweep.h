/*
 * ts_sweep.h -- C ABI of the MI355X serving-simulation sweep.
 *
 * The library evaluates TokenSim's per-iteration serving-simulation step
 * (arXiv 2503.08415) for many independent design points at once on one
 * gfx950 GPU.  A design point is one worker (Sec. III, system overview):
 * a local scheduler that re-forms the batch between iterations (continuous
 * batching, Sec. II-B and Sec. IV-A), a block-granular KV memory manager
 * (PagedAttention blocks, Sec. II-B and Sec. III-B) and a per-iteration
 * compute simulator priced as a per-operator roofline over the
 * transformer (Sec. III overview; prefill compute-bound and decode
 * memory-bound, Sec. II-A).  Its inputs follow the paper's statement of the
 * problem: a request trace of arrival time, prompt length and output length
 * (workload generator, Sec. III), a transformer shape, hardware FLOP/s,
 * bandwidth and capacity (Sec. V), and the scheduling / memory policy.
 *
 * Semantics, per design point, repeated until every request is finished or
 * rejected (integer state, int64 nanoseconds):
 *   1. intake: requests with arrival <= t join the waiting queue, ordered by
 *      (arrival, index); when nothing runs or waits the clock jumps to the
 *      next arrival;
 *   2. reserve: each running decode whose next token starts a new KV block
 *      takes one, in admission order; when none is free the most recently
 *      admitted running request is preempted (its blocks are freed and it
 *      waits again): by recompute, with target = prompt + tokens decoded and
 *      no KV, or by swap (swap_bw > 0), keeping its KV in host memory;
 *   3. budget: with chunk_size > 0, decodes take one token each and running
 *      prefills share what is left of chunk_size in admission order;
 *   4. admit (not in an iteration that preempted): FCFS, no skipping; the
 *      head joins while max_batch, budget and free blocks for its whole
 *      target allow;
 *   5. price the batch: per layer max(FLOPs/peak, bytes/BW) for the QKV
 *      projection, prefill attention, decode attention, output projection,
 *      FFN up(+gate) and FFN down, plus the LM head over sequences emitting
 *      a token; fp64, fixed order, no contraction;
 *      iter_ns = max(1, ceil(L * layer_sum + lm_head));
 *   6. advance: t += iter_ns; a completed first prefill emits the first
 *      token, each decode emits one; a request finishes after output_len
 *      decodes and frees its blocks.
 * A request is REJECTED up front when ceil((prompt + output) / block) is
 * above the point's block count.
 *
 * Threading and ownership: a handle must not be used by two threads at
 * once.  ts_sweep_create deep-copies every input, so the caller may free
 * its arrays when it returns.  The handle owns all device memory;
 * ts_sweep_destroy releases it.  Results go into caller-allocated host
 * arrays.  Every call returns TS_OK (0) or a negative TS_ERR_* code;
 * ts_status_str gives a static message for any code.
 */
#ifndef TS_SWEEP_H
#define TS_SWEEP_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TS_ABI_VERSION 4
#define TS_MAX_BATCH 256 /* running-set cap per design point */
#define TS_MAX_DEVICES 16 /* prefill, and decode, devices of a disaggregated point */

/* call status */
#define TS_OK 0
#define TS_ERR_ARG (-1)         /* invalid argument (NULL, range, unsorted trace, ...) */
#define TS_ERR_UNSUPPORTED (-2) /* valid but outside what the library supports */
#define TS_ERR_OOM (-3)         /* device or host allocation failed */
#define TS_ERR_DEVICE (-4)      /* HIP runtime error (no device, launch failure, ...) */
#define TS_ERR_STATE (-5)       /* call out of order (results before run) */

/* per design point status (ts_point_result.status) */
#define TS_POINT_OK 0
#define TS_POINT_NO_KV 1      /* KV budget below one block: every request rejected */
#define TS_POINT_ITER_LIMIT 2 /* stopped by the per-point iteration cap */
#define TS_POINT_TIME_LIMIT 3 /* stopped by the per-point wall-clock watchdog */

/* per request status (ts_req_result.status) */
#define TS_REQ_PENDING 0  /* not finished (iteration cap hit); other fields -1/0 */
#define TS_REQ_DONE 1
#define TS_REQ_REJECTED 2 /* could never fit; other fields -1/0 */

/* ts_point.policy: how the local scheduler forms each iteration.
 *   MIXED          continuous batching (Sec. II-B, Sec. IV-A): admissions join
 *                  every iteration, prefills and decodes share it;
 *   PREFILL_FIRST  an iteration either admits and prefills (running decodes
 *                  pause) when the waiting head can be admitted, or runs
 *                  every decode; the validation target's default scheduler
 *                  (Sec. III-C).  Requires chunk_size 0;
 *   STATIC         static batching (Sec. IV-A): a batch is admitted only into
 *                  an empty running set and runs until every member ends. */
#define TS_POLICY_MIXED 0
#define TS_POLICY_PREFILL_FIRST 1
#define TS_POLICY_STATIC 2

/* ts_options.flags */
#define TS_F_PER_REQUEST 1u /* also return per-request records */
/* The 64-slot launch leaves every point it hands over to the 128-slot
 * launch instead of continuing some itself (see ts_sweep_kernel_work): the
 * two-launch schedule, for measuring it; results are the same. */
#define TS_F_NO_TAKEOVER 2u

typedef struct ts_sweep ts_sweep; /* opaque; owns all device memory */

/* Transformer shape, shared by every point of a sweep.  Requires
 * d_model % n_heads == 0 and n_heads % n_kv_heads == 0; all fields >= 1
 * except ffn_gated / weights_in_capacity (0 or 1). */
typedef struct {
  int32_t n_layers, d_model, n_heads, n_kv_heads;
  int32_t ffn_dim;             /* FFN inner width */
  int32_t ffn_gated;           /* 1: gate + up + down matrices; 0: up + down */
  int32_t vocab;               /* LM head rows */
  int32_t w_bytes, kv_bytes;   /* bytes per weight / activation and per KV element */
  int32_t weights_in_capacity; /* 1: KV budget = capacity*util - weights; 0: capacity*util */
} ts_model;

/* One request trace, structure of arrays of length n (n >= 0), sorted by
 * arrival (ties keep index order).  arrival_ns >= 0; 1 <= prompt_len,
 * output_len <= TS_MAX_TOKENS. */
#define TS_MAX_TOKENS (1 << 20)
typedef struct {
  const int64_t *arrival_ns;
  const int32_t *prompt_len;
  const int32_t *output_len;
  int32_t n;
} ts_trace;

/* One design point (one simulated worker). */
typedef struct {
  double peak_flops;          /* FLOP/s, finite, > 0 */
  double mem_bw;              /* bytes/s, finite, > 0 */
  int64_t capacity_bytes;     /* > 0 */
  int32_t mem_util_permille;  /* 1..1000: share of capacity usable */
  int32_t block_size;         /* tokens per KV block, 1..65536 */
  int32_t max_batch;          /* 1..TS_MAX_BATCH running sequences */
  int32_t chunk_size;         /* 0: prompts prefill in one iteration; else per-iteration
                                 token budget, max_batch <= chunk_size <= TS_MAX_TOKENS */
  int32_t trace_id;           /* index into the traces passed to create */
  int32_t policy;             /* TS_POLICY_*; FCFS order in all */
  int32_t admit_mem_permille; /* 0: off; 1..1000: a first admission keeps used blocks
                                 <= floor(num_blocks * this / 1000), reserving the rest
                                 for requests already admitted (Sec. IV-B's maximum
                                 memory ratio for new requests); a request whose prompt
                                 needs more than that is rejected */
  int32_t swap_overlap;       /* swap transfers: 0 add to the iteration's compute time,
                                 1 overlap with it (the longer of the two) */
  double swap_bw;             /* 0: preemption by recompute.  > 0 (finite): preemption
                                 by swap over a host link of this many bytes/s
                                 (Sec. IV-B; priced by the communication model,
                                 Sec. III-B): the victim's blocks move to host memory
                                 and it keeps its tokens; re-admission moves them back
                                 (no re-prefill, no token budget) and the request works
                                 again from the next iteration.  An iteration's
                                 transfers take blocks * block bytes / swap_bw ns */
  /* Disaggregated prefill and decode (Sec. II-B; breakpoints and a global
   * scheduler, Sec. III-A; validated against DistServe, Sec. III-C; device
   * ratios and prefill hardware, Sec. V).  n_prefill = n_decode = 0: one
   * worker.  Otherwise the point is n_prefill prefill devices with hardware
   * p_* (same memory utilisation, block size, max_batch and chunk_size;
   * continuous batching over prefills only) and n_decode decode devices
   * with the hardware and memory policy above (policy MIXED only).  Request
   * i goes to prefill device i % n_prefill, which frees its blocks when its
   * prefill completes (the first token); its prompt's KV then crosses that
   * device's link, one transfer after another in completion order, each
   * ceil(prompt * KV bytes per token * 1e9 / kv_link_bw) ns (0 = instant).
   * At the transfer's end it reaches decode device i % n_decode and waits
   * in (arrival there, index) order; admission takes blocks for its KV and
   * the next token plus one token of budget, and it decodes at once.  A
   * request is rejected up front when its prompt does not fit a prefill
   * device or it could never fit a decode device. */
  int32_t n_prefill;          /* 0, or 1..TS_MAX_DEVICES */
  int32_t n_decode;           /* 0 with n_prefill 0, else 1..TS_MAX_DEVICES */
  double p_peak_flops;        /* prefill devices: FLOP/s, finite, > 0 */
  double p_mem_bw;            /* prefill devices: bytes/s, finite, > 0 */
  int64_t p_capacity_bytes;   /* prefill devices: > 0 */
  double kv_link_bw;          /* bytes/s of each prefill device's KV link, finite, >= 0 */
} ts_point;

/* Per-request record (TS_F_PER_REQUEST): 40 bytes. */
typedef struct {
  int64_t admit_ns;       /* first admission, -1 if none */
  int64_t first_token_ns; /* end of the iteration completing the first prefill */
  int64_t finish_ns;      /* end of the last decode */
  int64_t max_gap_ns;     /* largest interval between consecutive tokens */
  int32_t n_preempt;      /* times preempted */
  int32_t status;         /* TS_REQ_* */
} ts_req_result;

/* Per-point result: 176 bytes.  Percentiles are nearest rank over finished
 * requests (-1 when none); TTFT = first_token - arrival, E2E = finish -
 * arrival, TPOT numerator = finish - first_token.  slo_ok counts finished
 * requests with TTFT <= slo_ttft_ns and max gap <= slo_tpot_ns; slo_tpot_ok
 * those with max gap <= slo_tpot_ns (Sec. IV-B's two SLO throughputs are
 * these counts over last_finish_ns - first_arrival_ns).
 * used_block_ns = sum over iterations of used blocks * iteration time (fp64).
 * digest = sum mod 2^64 of a 64-bit hash of every finished or rejected
 * request's record and index. */
typedef struct {
  int32_t status, n_done, n_rejected, num_blocks;
  int64_t n_iters, n_preempt, prefill_tokens, decode_tokens, peak_used_blocks;
  int64_t first_arrival_ns, last_finish_ns, sum_ttft_ns, sum_e2e_ns, max_e2e_ns,
      sum_tpot_num_ns;
  int64_t p50_e2e_ns, p90_e2e_ns, p99_e2e_ns, p50_ttft_ns, p99_ttft_ns, slo_ok;
  double used_block_ns;
  uint64_t digest;
  int64_t slo_tpot_ok;
} ts_point_result;

/* Options; pass NULL for all defaults. */
typedef struct {
  uint32_t flags;        /* TS_F_* */
  int32_t first_point;   /* simulate points [first_point, first_point + n_points) */
  int32_t n_points;      /* 0 = through the last point */
  int32_t pad;
  int64_t iter_cap;      /* per-point iteration cap; 0 = 2^40 */
  int64_t slo_ttft_ns;   /* 0 = 15 s (TTFT SLO, Sec. IV-B) */
  int64_t slo_tpot_ns;   /* 0 = 0.3 s (mTPOT SLO, Sec. IV-B) */
  int64_t point_time_limit_ms; /* 0 = none; else a point still running after this much
                                  device wall-clock time stops with TS_POINT_TIME_LIMIT */
} ts_options;

/* Validate and upload a sweep.  traces[n_traces], points[n_points] (host
 * memory, copied).  The selected sub-range of points becomes the handle's
 * points, numbered from 0.  Every argument is checked before any device
 * call: TS_ERR_ARG for invalid input, TS_ERR_UNSUPPORTED when a cost-model
 * integer (a point's KV bytes, with swap) could exceed 2^53 (exact fp64) or a
 * block count exceeds 2^30.
 * Device memory it allocates: the traces (16 B per request), the request
 * records (40 B per point per request of the longest trace; the statistics
 * are computed from them, so they are kept with or without
 * TS_F_PER_REQUEST), the latency arrays of the percentile pass (16 B per
 * point per request of the longest trace), and a preempted-request queue
 * per workgroup (8 KiB); TS_ERR_OOM, before any allocation, when their sum
 * exceeds the device's free memory (or an allocation fails).
 * The handle belongs to the device current at create time; every later call
 * selects that device itself.
 * On success *out receives the handle; on failure *out is NULL. */
int ts_sweep_create(const ts_model *model, const ts_trace *traces, int32_t n_traces,
                    const ts_point *points, int32_t n_points, const ts_options *opt,
                    ts_sweep **out);

/* Enqueue the whole sweep (simulation kernels, then the statistics kernel)
 * on hip_stream (a hipStream_t; NULL = the default stream).  Returns once
 * the work is enqueued.  May be called again to re-run; each run restarts
 * every point from its initial state and replaces the previous results.  A
 * re-run on another stream first waits (on the device) for the previous
 * run, whose buffers it reuses. */
int ts_sweep_run(ts_sweep *h, void *hip_stream);

/* Wait for the last run and copy results to the host.  out_points receives
 * the handle's n_points records in point order.  out_requests is NULL or,
 * when created with TS_F_PER_REQUEST, an array of n_points * max_n records
 * (point-major, row stride max_n = the longest trace; rows of shorter
 * traces are padded with TS_REQ_PENDING records).  TS_ERR_STATE before the
 * first run, or when out_requests is given without TS_F_PER_REQUEST. */
int ts_sweep_results(ts_sweep *h, ts_point_result *out_points, ts_req_result *out_requests);

/* Sizes of the handle: points, longest trace. */
int ts_sweep_shape(const ts_sweep *h, int32_t *n_points, int32_t *max_n);

/* Device time of the last run in milliseconds, measured with HIP events on
 * the run's stream: sim_ms = simulation kernels, stats_ms = statistics
 * kernel.  Waits for the run.  TS_ERR_STATE before the first run. */
int ts_sweep_timing(ts_sweep *h, float *sim_ms, float *stats_ms);

/* Per-kernel device time of the last run.  The points are simulated by up
 * to TS_N_SIM_KERNELS kernel launches, one per stage and register-chunk
 * class, launched one after another on the run's stream: index
 * 3 * stage + class, stage 0 for one-worker points, 1 for the prefill
 * devices and 2 for the decode devices of disaggregated points, class 0, 1,
 * 2 for max_batch <= 64, <= 128, <= 256.  ms[k] receives launch k's duration
 * in milliseconds from HIP events recorded around it on that stream (0 when
 * it has no work) and n_points[k] its number of simulated workers (with the
 * hand-over described at ts_sweep_kernel_work: for k = 0 every one-worker
 * point, for k = 1, 2 the most it may be handed).  Waits for the run.
 * TS_ERR_STATE before the first run. */
#define TS_N_SIM_KERNELS 9
int ts_sweep_kernel_timing(ts_sweep *h, float *ms, int32_t *n_points);

/* Simulated iterations per launch of the last run: iters[k] receives the
 * iterations launch k simulated (index as for ts_sweep_kernel_timing); they
 * add up to the points' n_iters.  When every one-worker point is a simple
 * one (continuous batching, recompute preemption, no admission ratio, no
 * request that could never fit, no watchdog) and some allow more than 64
 * running requests, the max_batch <= 64 launch (k = 0) takes all of them
 * while at most 64 run at once; a point whose admissions need more slots is
 * handed on with 128 slots, and from there, if it needs more than 128, to
 * the 256-slot launch (k = 2).  Handed points are taken with the most
 * requests left first.  The 128-slot work runs in launch 0 itself, in each
 * workgroup that has no point of its own left, while the others still run
 * (counted as launch 0's iterations); the 128-slot launch (k = 1) takes the
 * points handed over after that.  The point continues from the start of
 * the iteration that needed the slots (each launch counts the iterations
 * it simulated), or, when the iteration had already admitted a full window,
 * is simulated again from the start (then only the launch that does counts
 * those iterations).  Waits for the run.  TS_ERR_STATE before the first run. */
int ts_sweep_kernel_work(ts_sweep *h, int64_t *iters);

/* For callers that cannot allocate device memory (tight serving loops,
 * harnesses that forbid hipMalloc): the whole sweep of ts_sweep_create +
 * ts_sweep_run + ts_sweep_results in one call that calls no hipMalloc,
 * hipFree or other allocating device routine.  Every buffer the kernels use
 * lives in one static device array of TS_STATIC_SCRATCH_BYTES that each GPU
 * the library runs on holds from the library's load until the process ends;
 * the first call on a device looks up its address there.  Inputs and
 * options are as for ts_sweep_create (host memory, validated before any
 * device call); out_points (n_points records) and out_requests (NULL, or
 * with TS_F_PER_REQUEST n_points * max_n records, max_n = the longest
 * trace) are caller-allocated host arrays, as for ts_sweep_results.  The
 * work is enqueued on hip_stream (NULL = the default stream) and the call
 * returns after synchronising it.  TS_ERR_UNSUPPORTED when the sweep's
 * buffers exceed the array even at one workgroup per kernel launch (the
 * per-workgroup queues shrink with the grid);
 * TS_ERR_STATE for out_requests without TS_F_PER_REQUEST.  All calls share
 * the one array of their GPU and it keeps the last call's contents (each
 * call clears what must start at zero): calls inside one process are
 * serialised by a lock, and calls that overlapped on one GPU would race.
 * Not for use under stream capture (it copies from pageable host memory and
 * synchronises the stream). */
#define TS_STATIC_SCRATCH_BYTES ((size_t)64 << 20)
int ts_sweep_run_static(const ts_model *model, const ts_trace *traces, int32_t n_traces,
                        const ts_point *points, int32_t n_points, const ts_options *opt,
                        void *hip_stream, ts_point_result *out_points,
                        ts_req_result *out_requests);

/* Release the handle and its device memory; NULL is accepted. */
void ts_sweep_destroy(ts_sweep *h);

/* Static message for a TS_* call status; for TS_ERR_DEVICE, the last HIP
 * error seen by this thread is appended when available. */
const char *ts_status_str(int status);

#ifdef __cplusplus
}
#endif
#endif
