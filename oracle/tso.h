/*
 * tso.h -- CPU oracle for the TokenSim serving-simulation step.
 *
 * TEST INFRASTRUCTURE ONLY.  This is the plain, slow, sequential reference
 * that the GPU sweep is checked against.  Only the test-suite, the smoke
 * check and the benchmark's CPU-baseline leg may load it; the product path
 * never calls it.  It shares no code, header or constant with the HIP
 * library.
 *
 * What it computes (TokenSim, arXiv 2503.08415):
 *   - a discrete-event simulation with one simulated clock (Sec. III, SimPy
 *     engine; requests released by a dispatcher at their arrival time);
 *   - one worker per design point whose local scheduler re-forms the batch
 *     between iterations (continuous batching, Sec. II-B and Sec. IV-A) and
 *     consults a block-granular memory manager (PagedAttention blocks,
 *     Sec. II-B; memory manager, Sec. III-B);
 *   - preemption of the newest requests when no free block remains
 *     (Sec. IV-B), taken here as recompute;
 *   - a per-iteration compute simulator fed the batch (Sec. III, overview):
 *     a per-operator roofline over the transformer's operators;
 *   - per-request latency records and per-point latency / SLO metrics
 *     (Sec. III-C, Sec. IV-B).
 * The paper gives no formulas or pseudocode for any of these; every point
 * it leaves open is resolved by a stated reading (see the design notes).
 *
 * Units: time in int64 nanoseconds, tokens and blocks in int32, the cost
 * model in IEEE fp64 with no contraction and a fixed evaluation order.
 */
#ifndef TSO_H
#define TSO_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { TSO_OK = 0, TSO_ERR_ARG = -1, TSO_ERR_UNSUPPORTED = -2, TSO_ERR_OOM = -3 };
enum { TSO_POINT_OK = 0, TSO_POINT_NO_KV = 1, TSO_POINT_ITER_LIMIT = 2 };
enum { TSO_REQ_PENDING = 0, TSO_REQ_DONE = 1, TSO_REQ_REJECTED = 2 };
/* Scheduling policies (Sec. IV-A compares continuous with static batching;
 * the prefill-first iteration is the validation target's default scheduler,
 * Sec. III-C):
 *   MIXED          continuous batching, prefill and decode in one iteration;
 *   PREFILL_FIRST  an iteration either admits and prefills (decodes pause) or
 *                  runs every decode; needs chunk_size 0;
 *   STATIC         a batch is admitted only when nothing runs. */
enum { TSO_POLICY_MIXED = 0, TSO_POLICY_PREFILL_FIRST = 1, TSO_POLICY_STATIC = 2 };
/* largest number of prefill, and of decode, devices of a disaggregated point */
enum { TSO_MAX_DEVICES = 16 };

typedef struct {
  int32_t n_layers, d_model, n_heads, n_kv_heads;
  int32_t ffn_dim, ffn_gated, vocab;
  int32_t w_bytes, kv_bytes;
  int32_t weights_in_capacity;
} tso_model;

typedef struct {
  const int64_t *arrival_ns;   /* non-decreasing */
  const int32_t *prompt_len;   /* >= 1 */
  const int32_t *output_len;   /* >= 1 */
  int32_t n;
} tso_trace;

typedef struct {
  double peak_flops;           /* FLOP/s */
  double mem_bw;               /* B/s */
  int64_t capacity_bytes;
  int32_t mem_util_permille;
  int32_t block_size;
  int32_t max_batch;
  int32_t chunk_size;          /* 0 = whole prompt in one iteration */
  int32_t trace_id;
  int32_t policy;              /* TSO_POLICY_* */
  int32_t admit_mem_permille;  /* 0 = off; else a first admission keeps used
                                  blocks <= floor(num_blocks * this / 1000)
                                  (Sec. IV-B, the maximum memory ratio for
                                  new requests) */
  int32_t swap_overlap;        /* swap transfers: 0 add to the iteration,
                                  1 overlap with its compute (Sec. III-B) */
  int32_t pad;
  double swap_bw;              /* B/s of the host link; 0 = recompute
                                  preemption, else preempted requests swap
                                  their KV blocks to host memory (Sec. IV-B)
                                  and back, priced by the communication model
                                  (Sec. III-B) */
  /* Disaggregated prefill and decode (Sec. II-B; Sec. III-C, Sec. V): with
   * n_prefill > 0 the point is n_prefill prefill devices with hardware p_*
   * and n_decode decode devices with the hardware and memory policy above
   * (policy MIXED only); each prefill device sends a prompt's KV over its
   * own link of kv_link_bw B/s (0 = instant) to the request's decode device. */
  int32_t n_prefill;           /* 0 = one worker; else 1..TSO_MAX_DEVICES */
  int32_t n_decode;            /* 1..TSO_MAX_DEVICES with n_prefill > 0, else 0 */
  double p_peak_flops;
  double p_mem_bw;
  int64_t p_capacity_bytes;
  double kv_link_bw;
} tso_point;

typedef struct {
  int64_t admit_ns, first_token_ns, finish_ns, max_gap_ns;
  int32_t n_preempt, status;
} tso_req;

typedef struct {
  int32_t status, n_done, n_rejected, num_blocks;
  int64_t n_iters, n_preempt, prefill_tokens, decode_tokens, peak_used_blocks;
  int64_t first_arrival_ns, last_finish_ns, sum_ttft_ns, sum_e2e_ns, max_e2e_ns,
      sum_tpot_num_ns;
  int64_t p50_e2e_ns, p90_e2e_ns, p99_e2e_ns, p50_ttft_ns, p99_ttft_ns, slo_ok;
  double used_block_ns;
  uint64_t digest;
  int64_t slo_tpot_ok;         /* finished with largest token gap <= the mTPOT SLO */
} tso_point_out;

typedef struct {
  int64_t kv_bytes_per_token;  /* K and V, all layers */
  int64_t weight_bytes;
  int64_t kv_budget_bytes;
  int32_t num_blocks;
  int32_t pad;
  double inv_flops_ns;         /* 1e9 / peak_flops */
  double inv_bw_ns;            /* 1e9 / mem_bw */
} tso_derived;

/* One simulated iteration, for tests that follow a schedule step by step. */
typedef struct {
  int64_t t_start, iter_ns;
  int32_t n_decode, n_prefill, tokens, used_blocks;
  int32_t n_running, n_preempted, n_admitted, n_finished;
} tso_iter_rec;

typedef struct {
  int64_t iter_cap;            /* 0 = 2^40 */
  int64_t slo_ttft_ns;         /* 0 = 15 s */
  int64_t slo_tpot_ns;         /* 0 = 0.3 s */
  int32_t n_threads;           /* 0 = all online cores */
  int32_t check_invariants;    /* 1 = check every iteration, count violations */
} tso_options;

/* Derived per-point constants (block budget, reciprocals). */
int tso_derive(const tso_model *m, const tso_point *p, tso_derived *out);

/* Cost of one iteration of the given scheduled set (each entry: tokens q
 * processed this iteration, context c0 before it, 1 if it is a prefill,
 * 1 if that prefill completes).  Returns the iteration time in ns. */
int64_t tso_iter_ns(const tso_model *m, double inv_flops_ns, double inv_bw_ns,
                    int32_t n, const int32_t *q, const int32_t *c0,
                    const int32_t *is_prefill, const int32_t *completes);

/* The same batch's compute time in ns before quantisation (no transfer). */
double tso_iter_total(const tso_model *m, double inv_flops_ns, double inv_bw_ns,
                      int32_t n, const int32_t *q, const int32_t *c0,
                      const int32_t *is_prefill, const int32_t *completes);

/* Simulate one design point, disaggregated or not.  out_req: trace.n
 * records (may be NULL);
 * log: up to log_cap iteration records (may be NULL); *n_log receives the
 * number of iterations logged (one-worker points only); *violations (may be
 * NULL) the number of invariant violations when opt->check_invariants is set. */
int tso_simulate_point(const tso_model *m, const tso_trace *tr, const tso_point *p,
                       const tso_options *opt, tso_point_out *out, tso_req *out_req,
                       tso_iter_rec *log, int64_t log_cap, int64_t *n_log,
                       int64_t *violations);

/* Simulate many points on a thread pool (threads across points only).
 * out_req: NULL or n_points * max_n records, point-major, row stride max_n. */
int tso_run_points(const tso_model *m, const tso_trace *traces, int32_t n_traces,
                   const tso_point *points, int32_t n_points, const tso_options *opt,
                   tso_point_out *out, tso_req *out_req, int32_t max_n);

/* Per-request record hash used for the per-point digest. */
uint64_t tso_record_hash(int64_t index, const tso_req *r);

#ifdef __cplusplus
}
#endif
#endif
