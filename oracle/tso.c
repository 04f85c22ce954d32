/*
 * tso.c -- CPU oracle for the TokenSim serving-simulation step.
 *
 * TEST INFRASTRUCTURE ONLY (see tso.h): a plain sequential event loop per
 * design point, written for a reader to check against the paper, not for
 * speed.  Threads are used only *across* design points.  Build with
 * -O2 -ffp-contract=off and no fast-math: the cost model is IEEE fp64
 * evaluated in the order written below.
 *
 * Sources in TokenSim (arXiv 2503.08415) for each part:
 *   event loop, one clock, dispatcher releasing arrivals   Sec. III (overview)
 *   local scheduler re-forming the batch per iteration     Sec. III-A, Sec. II-B
 *   continuous batching: arrivals join between iterations  Sec. II-B, Sec. IV-A
 *   block-granular KV memory manager (paged blocks)        Sec. II-B, Sec. III-B
 *   preempt the newest requests when blocks run out        Sec. IV-B
 *   compute simulator: iteration time from batch info      Sec. III (overview)
 *   prefill compute-bound, decode memory-bound             Sec. II-A
 *   latency percentiles, TTFT / mTPOT SLOs                 Sec. III-C, Sec. IV-B
 * The paper prints no formula or pseudocode for any of these.  Where it is
 * silent the reading used is stated next to the code.
 */
#define _GNU_SOURCE
#include "tso.h"

#include <math.h>
#include <pthread.h>
#include <stdlib.h>
#include <string.h>
#include <unistd.h>

enum { PH_FUTURE = 0, PH_WAITING, PH_RUNNING, PH_DONE, PH_REJECTED };

typedef struct {
  int phase;
  int32_t ctx;     /* KV tokens resident */
  int32_t target;  /* tokens to (re)fill before decoding: prompt + decodes done */
  int32_t gdone;   /* decode iterations done, 0..output_len */
  int32_t alloc;   /* KV blocks held while running */
  int32_t q;       /* tokens scheduled this iteration */
  int64_t admit, first, last, max_gap;
  int32_t n_pre;
  int32_t swapped; /* preempted by swap: its KV waits in host memory */
  int32_t fresh;   /* not yet admitted on this worker */
} rq;

#define DEFAULT_ITER_CAP (1LL << 40)
#define DEFAULT_SLO_TTFT 15000000000LL  /* 15 s TTFT SLO, Sec. IV-B */
#define DEFAULT_SLO_TPOT 300000000LL    /* 0.3 s mTPOT SLO, Sec. IV-B */

static int model_ok(const tso_model *m) {
  if (!m) return 0;
  if (m->n_layers < 1 || m->d_model < 1 || m->n_heads < 1 || m->n_kv_heads < 1) return 0;
  if (m->d_model % m->n_heads != 0 || m->n_heads % m->n_kv_heads != 0) return 0;
  if (m->ffn_dim < 1 || m->vocab < 1 || m->w_bytes < 1 || m->kv_bytes < 1) return 0;
  return 1;
}

int tso_derive(const tso_model *m, const tso_point *p, tso_derived *o) {
  if (!model_ok(m) || !p || !o) return TSO_ERR_ARG;
  if (!(p->peak_flops > 0) || !(p->mem_bw > 0) || !isfinite(p->peak_flops) ||
      !isfinite(p->mem_bw))
    return TSO_ERR_ARG;
  if (p->capacity_bytes <= 0 || p->mem_util_permille < 1 || p->mem_util_permille > 1000 ||
      p->block_size < 1)
    return TSO_ERR_ARG;
  const int64_t L = m->n_layers, d = m->d_model, h = m->n_heads, hkv = m->n_kv_heads;
  const int64_t dh = d / h, dkv = hkv * dh;
  const int64_t f = m->ffn_dim, g = 1 + (m->ffn_gated != 0), V = m->vocab;
  /* K and V, every layer, for one token */
  o->kv_bytes_per_token = 2 * L * dkv * m->kv_bytes;
  /* per layer: Q/K/V projections d x (d + 2 dkv), output projection d x d,
   * FFN (g + 1) matrices d x f; plus token embedding and LM head V x d each */
  o->weight_bytes =
      (int64_t)m->w_bytes * (L * (d * (d + 2 * dkv) + d * d + (g + 1) * d * f) + 2 * V * d);
  /* usable memory = floor(capacity * util / 1000); weights take their share
   * when they live in the same memory (Sec. V: capacity below the parameter
   * size is untestable) */
  __int128 usable = ((__int128)p->capacity_bytes * p->mem_util_permille) / 1000;
  int64_t budget = (int64_t)usable - (m->weights_in_capacity ? o->weight_bytes : 0);
  o->kv_budget_bytes = budget;
  int64_t per_block = (int64_t)p->block_size * o->kv_bytes_per_token;
  int64_t nb = budget > 0 ? budget / per_block : 0;
  if (nb > (1LL << 30)) return TSO_ERR_UNSUPPORTED;
  o->num_blocks = (int32_t)nb;
  o->pad = 0;
  o->inv_flops_ns = 1e9 / p->peak_flops;
  o->inv_bw_ns = 1e9 / p->mem_bw;
  return TSO_OK;
}

/* ---------------------------------------------------------------- cost model
 * Per-operator roofline: an operator takes max(FLOPs / peak, bytes / BW).
 * Operators per layer: QKV projection, attention over prefill tokens,
 * attention over decode tokens, output projection, FFN up(+gate), FFN down;
 * once per iteration: the LM head over the sequences that emit a token.
 * Elementwise work, embedding lookup and fixed overheads are not priced.
 */
typedef struct {
  int64_t T;    /* tokens processed */
  int64_t T_P;  /* prefill tokens */
  int64_t A_P;  /* causal query-key pairs of prefill tokens */
  int64_t C_P;  /* keys read by prefill sequences: sum of (c0 + q) */
  int64_t n_D;  /* decode sequences */
  int64_t C_D;  /* keys read by decode sequences: sum of (c0 + 1) */
  int64_t R_lm; /* sequences emitting a token (LM head rows) */
} batch_sums;

static double op_time(int64_t flops, int64_t bytes, double iF, double iB) {
  double tf = (double)flops * iF;
  double tb = (double)bytes * iB;
  return tf > tb ? tf : tb;
}

/* The iteration's compute time in ns before quantisation. */
static double compute_total(const tso_model *m, double iF, double iB, const batch_sums *s) {
  const int64_t L = m->n_layers, d = m->d_model, h = m->n_heads, hkv = m->n_kv_heads;
  const int64_t dh = d / h, dkv = hkv * dh;
  const int64_t f = m->ffn_dim, g = 1 + (m->ffn_gated != 0), V = m->vocab;
  const int64_t e = m->w_bytes, ekv = m->kv_bytes;
  const int64_t T = s->T, T_P = s->T_P, A_P = s->A_P, C_P = s->C_P;
  const int64_t n_D = s->n_D, C_D = s->C_D, R = s->R_lm;

  /* 1. QKV projection: weights, input activations, K/V written, Q written */
  double t1 = op_time(2 * T * d * (d + 2 * dkv),
                      e * (d * (d + 2 * dkv) + T * d) + ekv * T * 2 * dkv + e * T * d, iF, iB);
  /* 2. attention for prefill tokens: QK^T and PV over causal pairs; reads
   *    the K/V of the whole visible context, Q in and O out */
  double t2 = op_time(4 * d * A_P, ekv * 2 * dkv * C_P + e * 2 * d * T_P, iF, iB);
  /* 3. attention for decode tokens: one query against c0 + 1 keys */
  double t3 = op_time(4 * d * C_D, ekv * 2 * dkv * C_D + e * 2 * d * n_D, iF, iB);
  /* 4. output projection */
  double t4 = op_time(2 * T * d * d, e * (d * d + 2 * T * d), iF, iB);
  /* 5. FFN up (and gate when gated) */
  double t5 = op_time(2 * g * T * d * f, e * (g * d * f + T * d + g * T * f), iF, iB);
  /* 6. FFN down */
  double t6 = op_time(2 * T * f * d, e * (f * d + T * f + T * d), iF, iB);
  /* 7. LM head, once per iteration, only when some sequence emits a token */
  double t7 = R > 0 ? op_time(2 * R * d * V, e * (d * V + R * d + R * V), iF, iB) : 0.0;

  double layer = t1;
  layer = layer + t2;
  layer = layer + t3;
  layer = layer + t4;
  layer = layer + t5;
  layer = layer + t6;
  double total = (double)L * layer;
  total = total + t7;
  return total;
}

static int64_t cost_from_sums_x(const tso_model *m, double iF, double iB, const batch_sums *s,
                                double xfer, int overlap) {
  double total = compute_total(m, iF, iB, s);
  if (xfer > 0.0) total = overlap ? (xfer > total ? xfer : total) : total + xfer;
  int64_t ns = (int64_t)ceil(total);
  return ns < 1 ? 1 : ns;
}

/* xfer: swap transfer time of the iteration in ns (0 when none); overlap:
 * the transfer runs beside the compute instead of after it */
static int64_t cost_from_sums(const tso_model *m, double iF, double iB, const batch_sums *s) {
  return cost_from_sums_x(m, iF, iB, s, 0.0, 0);
}

static void sums_of(int32_t n, const int32_t *q, const int32_t *c0, const int32_t *is_prefill,
                    const int32_t *completes, batch_sums *out) {
  batch_sums s;
  memset(&s, 0, sizeof s);
  for (int32_t i = 0; i < n; i++) {
    int64_t qq = q[i], c = c0[i];
    if (is_prefill[i]) {
      s.T += qq;
      s.T_P += qq;
      s.A_P += qq * c + qq * (qq + 1) / 2;
      s.C_P += c + qq;
      if (completes[i]) s.R_lm += 1;
    } else {
      s.T += 1;
      s.n_D += 1;
      s.C_D += c + 1;
      s.R_lm += 1;
    }
  }
  *out = s;
}

int64_t tso_iter_ns(const tso_model *m, double iF, double iB, int32_t n, const int32_t *q,
                    const int32_t *c0, const int32_t *is_prefill, const int32_t *completes) {
  batch_sums s;
  sums_of(n, q, c0, is_prefill, completes, &s);
  return cost_from_sums(m, iF, iB, &s);
}

double tso_iter_total(const tso_model *m, double iF, double iB, int32_t n, const int32_t *q,
                      const int32_t *c0, const int32_t *is_prefill, const int32_t *completes) {
  batch_sums s;
  sums_of(n, q, c0, is_prefill, completes, &s);
  return compute_total(m, iF, iB, &s);
}

/* ------------------------------------------------------------ record hash
 * The digest is this library's own checksum of the per-request records (the
 * paper defines none): a multilinear combination of the record's fields with
 * fixed odd 64-bit multipliers, wrapped mod 2^64, then MurmurHash3's 64-bit
 * finaliser (fmix64). */
static uint64_t fmix64(uint64_t k) {
  k ^= k >> 33;
  k *= 0xff51afd7ed558ccdULL;
  k ^= k >> 33;
  k *= 0xc4ceb9fe1a85ec53ULL;
  k ^= k >> 33;
  return k;
}

uint64_t tso_record_hash(int64_t index, const tso_req *r) {
  const uint64_t tail = ((uint64_t)(uint32_t)r->n_preempt << 32) | (uint32_t)r->status;
  uint64_t h = (uint64_t)index * 0x9e3779b97f4a7c15ULL;
  h += (uint64_t)r->admit_ns * 0xbf58476d1ce4e5b9ULL;
  h += (uint64_t)r->first_token_ns * 0x94d049bb133111ebULL;
  h += (uint64_t)r->finish_ns * 0xd6e8feb86659fd93ULL;
  h += (uint64_t)r->max_gap_ns * 0xa0761d6478bd642fULL;
  h += tail * 0xe7037ed1a0b428dbULL;
  return fmix64(h);
}

/* ------------------------------------------------------------ simulation */
typedef struct {
  const int64_t *arr;
  rq *rs;
  int32_t *waiting;
  int32_t nw;
} waitq;

/* waiting is ordered by (arrival, index): FCFS */
static void waiting_insert(waitq *w, int32_t idx) {
  const int64_t *arr = w->arr;
  int32_t pos = w->nw;
  while (pos > 0) {
    int32_t o = w->waiting[pos - 1];
    if (arr[o] < arr[idx] || (arr[o] == arr[idx] && o < idx)) break;
    pos--;
  }
  memmove(&w->waiting[pos + 1], &w->waiting[pos], (size_t)(w->nw - pos) * sizeof(int32_t));
  w->waiting[pos] = idx;
  w->nw++;
}

static int cmp_i64(const void *a, const void *b) {
  int64_t x = *(const int64_t *)a, y = *(const int64_t *)b;
  return (x > y) - (x < y);
}

/* nearest rank: the smallest value with at least pct% of values <= it */
static int64_t nearest_rank(const int64_t *sorted, int64_t n, int pct) {
  if (n <= 0) return -1;
  int64_t rank = (pct * n + 99) / 100; /* ceil(pct * n / 100) */
  if (rank < 1) rank = 1;
  return sorted[rank - 1];
}

static int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

/* ------------------------------------------------------------ one worker */
/* What a worker does with the requests that reach it:
 *   WM_FULL     the whole request: prefill, first token, output decodes
 *               (a design point with one worker);
 *   WM_PREFILL  a prefill device of a disaggregated deployment (Sec. II-B;
 *               breakpoints after the first iteration, Sec. III-A): the
 *               request leaves when its prefill completes, and its KV
 *               crosses the device's link to a decode device;
 *   WM_DECODE   a decode device: the request arrives with its prompt's KV and
 *               first token, and runs its output decodes. */
enum { WM_FULL = 0, WM_PREFILL = 1, WM_DECODE = 2 };

typedef struct {
  int64_t n_iters, n_preempt, prefill_tokens, decode_tokens, peak_used;
  double used_block_ns;
  int32_t status;
  int64_t nviol, nlog;
} worker_out;

/* The KV link out of a prefill device.  Transfers run one after another in
 * the order the prefills complete: the sequential default of the
 * communication model (Sec. III-B), which prices a transfer as bytes over
 * bandwidth. */
typedef struct {
  int64_t kv_bytes_per_token;
  double inv_link_ns;  /* ns per byte; 0 = instant */
  int64_t free_at;     /* the link is busy until then */
  int64_t *arrive;     /* per request: when its KV reaches the decode device */
} kv_link;

/* ceil(prompt KV bytes * ns per byte), whole ns */
static int64_t kv_transfer_ns(const kv_link *lk, int32_t prompt) {
  if (lk->inv_link_ns == 0.0) return 0;
  return (int64_t)ceil((double)((int64_t)prompt * lk->kv_bytes_per_token) * lk->inv_link_ns);
}

/* Blocks a waiting request takes when admitted: a swapped request gets back
 * what it held; one that arrives ready to decode holds its KV plus the slot
 * of the token it decodes next; any other holds its whole prefill target. */
static int64_t admission_blocks(const rq *r, int64_t b) {
  const int64_t top = r->ctx > r->target ? r->ctx : r->target;
  if (r->swapped) return ceil_div(top, b);
  if (r->ctx >= r->target) return ceil_div((int64_t)r->ctx + 1, b);
  return ceil_div(r->target, b);
}

/* Run one worker (hardware and scheduler p, derived constants dv) over N
 * requests with arrival times arr (sorted), whose state rs the caller has
 * initialised (PH_FUTURE or PH_REJECTED, target, ctx, times). */
static int worker_loop(const tso_model *m, const tso_point *p, const tso_derived *dv, int wmode,
                       int32_t N, const int64_t *arr, const int32_t *plen, const int32_t *olen,
                       rq *rs, int64_t iter_cap, int check, kv_link *lk, tso_iter_rec *log,
                       int64_t log_cap, worker_out *wo) {
  const int64_t NB = dv->num_blocks, b = p->block_size, M = p->max_batch, K = p->chunk_size;
  const int policy = p->policy;
  /* blocks a first admission may leave in use, and the reserve it may not touch */
  const int64_t adm_cap = p->admit_mem_permille > 0 ? NB * p->admit_mem_permille / 1000 : NB;
  const int64_t adm_reserve = NB - adm_cap;
  /* swap preemption: KV bytes per block and ns per byte of the host link */
  const int swap = p->swap_bw > 0.0;
  const int64_t block_bytes = b * dv->kv_bytes_per_token;
  const double inv_link_ns = swap ? 1e9 / p->swap_bw : 0.0;
  const double iF = dv->inv_flops_ns, iB = dv->inv_bw_ns;
  int32_t *running = (int32_t *)malloc((size_t)M * sizeof(int32_t));
  int32_t *waiting = (int32_t *)malloc((size_t)(N > 0 ? N : 1) * sizeof(int32_t));
  if (!running || !waiting) {
    free(running); free(waiting);
    return TSO_ERR_OOM;
  }
  int64_t nviol = 0, nlog = 0;

  waitq wq = {arr, rs, waiting, 0};
  int64_t t = 0, free_blocks = NB;
  int32_t next = 0, nr = 0;
  int64_t n_iters = 0, n_preempt = 0, prefill_tokens = 0, decode_tokens = 0, peak_used = 0;
  double used_block_ns = 0.0;
  int32_t status = NB == 0 ? TSO_POINT_NO_KV : TSO_POINT_OK;

  while (NB > 0) {
    /* 1. the dispatcher releases every request that has arrived by t */
    while (next < N && arr[next] <= t) {
      if (rs[next].phase != PH_REJECTED) {
        rs[next].phase = PH_WAITING;
        waiting_insert(&wq, next);
      }
      next++;
    }
    /* 2. idle: jump the clock to the next arrival, or stop */
    if (nr == 0 && wq.nw == 0) {
      if (next == N) break;
      t = arr[next];
      continue;
    }
    if (n_iters >= iter_cap) {
      status = TSO_POINT_ITER_LIMIT;
      break;
    }

    /* Prefill-first: when the waiting head can be admitted now, the iteration
     * admits and prefills only, and the decodes pause. */
    int pf_iter = 0;
    if (policy == TSO_POLICY_PREFILL_FIRST && wq.nw > 0 && nr < M) {
      const rq *h = &rs[waiting[0]];
      const int64_t room = h->fresh ? free_blocks - adm_reserve : free_blocks;
      pf_iter = admission_blocks(h, b) <= room;
    }

    /* 3. decode sequences whose next token starts a new block reserve it, in
     *    admission order; when no block is free the most recently admitted
     *    running request is preempted (recompute: its KV is dropped and it
     *    waits again, ordered by arrival) until the block fits. */
    int preempted = 0;
    int32_t n_pre_now = 0;
    int64_t xfer_blocks = 0; /* blocks swapped out or in this iteration */
    for (int32_t i = 0; i < nr && !pf_iter; i++) {
      rq *r = &rs[running[i]];
      int need = (r->ctx >= r->target) && (r->ctx % b == 0);
      if (!need) continue;
      while (free_blocks == 0) {
        int32_t v = running[--nr];
        rq *pv = &rs[v];
        free_blocks += pv->alloc;
        if (swap) {
          /* swap: the KV moves to host memory and comes back on re-admission */
          xfer_blocks += pv->alloc;
          pv->swapped = 1;
        } else {
          /* recompute: the KV is dropped and refilled from the tokens so far */
          pv->ctx = 0;
          pv->target = plen[v] + pv->gdone;
        }
        pv->alloc = 0;
        pv->n_pre += 1;
        pv->phase = PH_WAITING;
        waiting_insert(&wq, v);
        n_preempt++;
        n_pre_now++;
        preempted = 1;
        if (nr == i) break; /* the requester itself was the newest */
      }
      if (i < nr) {
        free_blocks -= 1;
        r->alloc += 1;
      }
    }

    /* 4. token budget: decodes take one token each; running prefills take
     *    what is left of the chunk budget in admission order */
    const int unlimited = (K == 0);
    int64_t R = 0;
    if (!unlimited) {
      int64_t nd = 0;
      for (int32_t i = 0; i < nr; i++)
        if (rs[running[i]].ctx >= rs[running[i]].target) nd++;
      R = K - nd;
    }
    for (int32_t i = 0; i < nr; i++) {
      rq *r = &rs[running[i]];
      if (r->ctx >= r->target) {
        r->q = pf_iter ? 0 : 1;
      } else {
        int64_t left = r->target - r->ctx;
        int64_t q = unlimited ? left : (left < R ? left : R);
        r->q = (int32_t)q;
        if (!unlimited) R -= q;
      }
    }

    /* 5. FCFS admission (none in an iteration that preempted): the head of
     *    the waiting queue joins if its whole prefill target fits in free
     *    blocks (a first admission also leaves the reserve untouched), the
     *    running set is below max batch and budget remains; no skipping past
     *    a blocked head.  Static batching admits only into an empty running
     *    set; prefill-first only in a prefill iteration. */
    int32_t n_adm = 0;
    int may_admit = !preempted;
    if (policy == TSO_POLICY_STATIC && nr > 0) may_admit = 0;
    if (policy == TSO_POLICY_PREFILL_FIRST && !pf_iter) may_admit = 0;
    if (may_admit) {
      while (wq.nw > 0 && nr < M) {
        int32_t hidx = waiting[0];
        rq *r = &rs[hidx];
        /* a swapped request brings back the blocks it held and works from
         * the next iteration on; any other needs budget for its prefill, or
         * one token when it arrives ready to decode */
        if (!r->swapped && !unlimited && R <= 0) break;
        int64_t need = admission_blocks(r, b);
        if (need > (r->fresh ? free_blocks - adm_reserve : free_blocks)) break;
        free_blocks -= need;
        r->alloc = (int32_t)need;
        if (r->swapped) {
          xfer_blocks += need;
          r->swapped = 0;
          r->q = 0;
        } else if (r->ctx >= r->target) {
          /* its KV came from a prefill device: it decodes in this iteration */
          r->q = 1;
          if (!unlimited) R -= 1;
        } else {
          int64_t q = unlimited ? r->target : (r->target < R ? r->target : R);
          r->q = (int32_t)q;
          if (!unlimited) R -= q;
        }
        if (r->admit < 0) r->admit = t;
        r->fresh = 0;
        r->phase = PH_RUNNING;
        memmove(&waiting[0], &waiting[1], (size_t)(wq.nw - 1) * sizeof(int32_t));
        wq.nw--;
        running[nr++] = hidx;
        n_adm++;
      }
    }

    /* 6. price the iteration */
    batch_sums s;
    memset(&s, 0, sizeof s);
    int32_t n_dec = 0, n_pf = 0;
    for (int32_t i = 0; i < nr; i++) {
      rq *r = &rs[running[i]];
      int64_t c0 = r->ctx;
      if (r->ctx >= r->target) {
        if (r->q == 0) continue; /* paused, or swapped in this iteration */
        s.T += 1;
        s.n_D += 1;
        s.C_D += c0 + 1;
        s.R_lm += 1;
        n_dec++;
      } else if (r->q > 0) {
        int64_t q = r->q;
        s.T += q;
        s.T_P += q;
        s.A_P += q * c0 + q * (q + 1) / 2;
        s.C_P += c0 + q;
        if (c0 + q == r->target && r->first < 0) s.R_lm += 1; /* first token */
        n_pf++;
      }
    }
    /* swap transfers of the iteration, priced by the communication model */
    const double xfer = (double)(xfer_blocks * block_bytes) * inv_link_ns;
    const int64_t iter_ns = cost_from_sums_x(m, iF, iB, &s, xfer, p->swap_overlap);

    /* 7. advance the clock and every scheduled request */
    const int64_t t_end = t + iter_ns;
    const int64_t used = NB - free_blocks;
    if (used > peak_used) peak_used = used;
    used_block_ns = used_block_ns + (double)used * (double)iter_ns;
    n_iters++;
    int32_t j = 0, n_fin = 0;
    for (int32_t i = 0; i < nr; i++) {
      int32_t idx = running[i];
      rq *r = &rs[idx];
      if (r->ctx >= r->target && r->q > 0) {
        r->ctx += 1;
        r->gdone += 1;
        int64_t gap = t_end - r->last;
        if (gap > r->max_gap) r->max_gap = gap;
        r->last = t_end;
        decode_tokens++;
        if (r->gdone == olen[idx]) {
          r->phase = PH_DONE;
          free_blocks += r->alloc;
          r->alloc = 0;
          rs[idx].q = 0;
          /* finish time kept in 'last' */
          n_fin++;
          continue;
        }
      } else if (r->ctx < r->target && r->q > 0) {
        r->ctx += r->q;
        prefill_tokens += r->q;
        if (r->ctx == r->target && r->first < 0) {
          r->first = t_end; /* the full prefill emits the first token */
          r->last = t_end;
          if (wmode == WM_PREFILL) {
            /* a prefill device is done with the request: its blocks are
             * released and its KV queues for the device's link */
            r->phase = PH_DONE;
            free_blocks += r->alloc;
            r->alloc = 0;
            r->q = 0;
            const int64_t start = t_end > lk->free_at ? t_end : lk->free_at;
            lk->free_at = start + kv_transfer_ns(lk, plen[idx]);
            lk->arrive[idx] = lk->free_at;
            n_fin++;
            continue;
          }
        }
      }
      running[j++] = idx;
    }
    nr = j;
    if (log && nlog < log_cap) {
      tso_iter_rec *lr = &log[nlog];
      lr->t_start = t;
      lr->iter_ns = iter_ns;
      lr->n_decode = n_dec;
      lr->n_prefill = n_pf;
      lr->tokens = (int32_t)s.T;
      lr->used_blocks = (int32_t)used;
      lr->n_running = nr + n_fin;
      lr->n_preempted = n_pre_now;
      lr->n_admitted = n_adm;
      lr->n_finished = n_fin;
    }
    nlog++;
    t = t_end;

    if (check) {
      int64_t held = 0;
      if (nr > M) nviol++;
      if (!unlimited && s.T > K) nviol++;
      if (free_blocks < 0) nviol++;
      for (int32_t i = 0; i < nr; i++) {
        int32_t idx = running[i];
        rq *r = &rs[idx];
        held += r->alloc;
        int64_t top = r->ctx > r->target ? r->ctx : r->target;
        if (r->alloc != ceil_div(top, b)) nviol++;
        if (wmode != WM_DECODE && r->admit < arr[idx]) nviol++;
        if (r->first >= 0 && r->first <= r->admit) nviol++;
        if (r->ctx >= r->target && r->ctx != plen[idx] + r->gdone) nviol++;
        if (r->ctx < r->target && r->target != plen[idx] + r->gdone) nviol++;
        if (r->gdone >= olen[idx]) nviol++;
      }
      if (free_blocks + held != NB) nviol++;
      for (int32_t i = 1; i < wq.nw; i++) {
        int32_t a = waiting[i - 1], c = waiting[i];
        if (arr[a] > arr[c] || (arr[a] == arr[c] && a >= c)) nviol++;
      }
    }
  }


  if (check && status == TSO_POINT_OK && wmode != WM_PREFILL) {
    int64_t want = 0;
    for (int32_t i = 0; i < N; i++)
      if (rs[i].phase == PH_DONE) want += olen[i];
    if (want != decode_tokens) nviol++;
  }
  wo->n_iters = n_iters;
  wo->n_preempt = n_preempt;
  wo->prefill_tokens = prefill_tokens;
  wo->decode_tokens = decode_tokens;
  wo->peak_used = peak_used;
  wo->used_block_ns = used_block_ns;
  wo->status = status;
  wo->nviol = nviol;
  wo->nlog = nlog;
  free(running); free(waiting);
  return TSO_OK;
}

/* Per-request records, latency statistics and the digest of one point, from
 * every request's final state (arr: the trace's arrival times). */
static int point_stats(int32_t N, const int64_t *arr, const int32_t *olen, const rq *rs,
                       int64_t slo_ttft, int64_t slo_tpot, int check, tso_point_out *out,
                       tso_req *out_req, int64_t *nviol) {
  int64_t *e2e = (int64_t *)malloc((size_t)(N > 0 ? N : 1) * sizeof(int64_t));
  int64_t *ttft = (int64_t *)malloc((size_t)(N > 0 ? N : 1) * sizeof(int64_t));
  if (!e2e || !ttft) {
    free(e2e); free(ttft);
    return TSO_ERR_OOM;
  }
  /* per-request records and per-point statistics */
  int64_t n_done = 0, n_rej = 0;
  uint64_t digest = 0;
  for (int32_t i = 0; i < N; i++) {
    const rq *r = &rs[i];
    tso_req rec;
    rec.admit_ns = -1;
    rec.first_token_ns = -1;
    rec.finish_ns = -1;
    rec.max_gap_ns = 0;
    rec.n_preempt = 0;
    rec.status = TSO_REQ_PENDING;
    if (r->phase == PH_DONE) {
      rec.admit_ns = r->admit;
      rec.first_token_ns = r->first;
      rec.finish_ns = r->last;
      rec.max_gap_ns = r->max_gap;
      rec.n_preempt = r->n_pre;
      rec.status = TSO_REQ_DONE;
      int64_t tt = r->first - arr[i], ee = r->last - arr[i];
      ttft[n_done] = tt;
      e2e[n_done] = ee;
      n_done++;
      out->sum_ttft_ns += tt;
      out->sum_e2e_ns += ee;
      out->sum_tpot_num_ns += r->last - r->first;
      if (ee > out->max_e2e_ns) out->max_e2e_ns = ee;
      if (r->last > out->last_finish_ns) out->last_finish_ns = r->last;
      if (tt <= slo_ttft && r->max_gap <= slo_tpot) out->slo_ok++;
      if (r->max_gap <= slo_tpot) out->slo_tpot_ok++;
      if (check && r->gdone != olen[i]) (*nviol)++;
    } else if (r->phase == PH_REJECTED) {
      rec.status = TSO_REQ_REJECTED;
      n_rej++;
    }
    if (rec.status != TSO_REQ_PENDING) digest += tso_record_hash(i, &rec);
    if (out_req) out_req[i] = rec;
  }
  qsort(e2e, (size_t)n_done, sizeof(int64_t), cmp_i64);
  qsort(ttft, (size_t)n_done, sizeof(int64_t), cmp_i64);
  out->p50_e2e_ns = nearest_rank(e2e, n_done, 50);
  out->p90_e2e_ns = nearest_rank(e2e, n_done, 90);
  out->p99_e2e_ns = nearest_rank(e2e, n_done, 99);
  out->p50_ttft_ns = nearest_rank(ttft, n_done, 50);
  out->p99_ttft_ns = nearest_rank(ttft, n_done, 99);
  if (n_done == 0) out->max_e2e_ns = -1;
  out->n_done = (int32_t)n_done;
  out->n_rejected = (int32_t)n_rej;
  out->digest = digest;
  free(e2e); free(ttft);
  return TSO_OK;
}

/* ------------------------------------------------------------ disaggregated */
typedef struct {
  int64_t key;  /* when the request's KV reaches its decode device */
  int32_t idx;
} arrival_key;

static int cmp_arrival(const void *a, const void *b) {
  const arrival_key *x = (const arrival_key *)a, *y = (const arrival_key *)b;
  if (x->key != y->key) return (x->key > y->key) - (x->key < y->key);
  return (x->idx > y->idx) - (x->idx < y->idx);
}

/* A disaggregated design point (Sec. II-B; validated against DistServe in
 * Sec. III-C; device ratios and prefill-device hardware studied in Sec. V):
 * n_prefill prefill devices with hardware p_*, and n_decode decode devices
 * with the point's hardware and memory policy.  Readings:
 *   - the global scheduler sends request i to prefill device i mod n_prefill
 *     and then to decode device i mod n_decode (round robin in arrival
 *     order);
 *   - a prefill device runs continuous batching over prefills only; the
 *     iteration that completes a prompt emits the first token and frees the
 *     request's blocks; the prompt's KV then crosses the device's link
 *     (WM_PREFILL, kv_link);
 *   - the request reaches its decode device when that transfer ends, waits
 *     there in (arrival, index) order, and runs its output decodes as on a
 *     single worker (WM_DECODE), preemption included;
 *   - a request is rejected up front when its prompt does not fit a prefill
 *     device, or it could never fit a decode device.
 * Point totals: iterations, tokens and the used-block integral summed over
 * devices (prefill devices first, then decode devices, in index order), the
 * block peak of the busiest decode device, the decode devices' block count. */
static int simulate_pd(const tso_model *m, const tso_trace *tr, const tso_point *p,
                       const tso_options *opt, tso_point_out *out, tso_req *out_req,
                       int64_t *violations) {
  if (p->n_prefill < 1 || p->n_prefill > TSO_MAX_DEVICES || p->n_decode < 1 ||
      p->n_decode > TSO_MAX_DEVICES)
    return TSO_ERR_ARG;
  if (p->policy != TSO_POLICY_MIXED) return TSO_ERR_ARG;
  if (!isfinite(p->p_peak_flops) || !(p->p_peak_flops > 0) || !isfinite(p->p_mem_bw) ||
      !(p->p_mem_bw > 0) || p->p_capacity_bytes <= 0)
    return TSO_ERR_ARG;
  if (!isfinite(p->kv_link_bw) || !(p->kv_link_bw >= 0.0)) return TSO_ERR_ARG;
  /* a prefill device: its own hardware, continuous batching, nothing else */
  tso_point pp = *p;
  pp.peak_flops = p->p_peak_flops;
  pp.mem_bw = p->p_mem_bw;
  pp.capacity_bytes = p->p_capacity_bytes;
  pp.admit_mem_permille = 0;
  pp.swap_bw = 0.0;
  pp.swap_overlap = 0;
  tso_derived dvp, dvd;
  int rc = tso_derive(m, &pp, &dvp);
  if (rc != TSO_OK) return rc;
  rc = tso_derive(m, p, &dvd);
  if (rc != TSO_OK) return rc;
  const int64_t iter_cap = (opt && opt->iter_cap > 0) ? opt->iter_cap : DEFAULT_ITER_CAP;
  const int64_t slo_ttft = (opt && opt->slo_ttft_ns > 0) ? opt->slo_ttft_ns : DEFAULT_SLO_TTFT;
  const int64_t slo_tpot = (opt && opt->slo_tpot_ns > 0) ? opt->slo_tpot_ns : DEFAULT_SLO_TPOT;
  const int check = opt ? opt->check_invariants : 0;

  const int32_t N = tr->n;
  const int64_t *arr = tr->arrival_ns;
  const int32_t *plen = tr->prompt_len, *olen = tr->output_len;
  for (int32_t i = 0; i < N; i++) {
    if (plen[i] < 1 || olen[i] < 1 || arr[i] < 0) return TSO_ERR_ARG;
    if (i > 0 && arr[i] < arr[i - 1]) return TSO_ERR_ARG;
  }
  const int64_t NBp = dvp.num_blocks, NBd = dvd.num_blocks, b = p->block_size;
  const int64_t adm_cap = p->admit_mem_permille > 0 ? NBd * p->admit_mem_permille / 1000 : NBd;
  if (p->swap_bw > 0.0 && NBd * b * dvd.kv_bytes_per_token >= (1LL << 53))
    return TSO_ERR_UNSUPPORTED;

  memset(out, 0, sizeof *out);
  out->num_blocks = (int32_t)NBd;
  out->first_arrival_ns = N > 0 ? arr[0] : -1;
  out->last_finish_ns = -1;

  const size_t n1 = (size_t)(N > 0 ? N : 1);
  rq *g = (rq *)calloc(n1, sizeof(rq));        /* every request's final state */
  rq *rw = (rq *)calloc(n1, sizeof(rq));       /* one device's requests */
  int64_t *a2 = (int64_t *)malloc(n1 * sizeof(int64_t));
  int32_t *ids = (int32_t *)malloc(n1 * sizeof(int32_t));
  int64_t *arr_w = (int64_t *)malloc(n1 * sizeof(int64_t));
  int32_t *plen_w = (int32_t *)malloc(n1 * sizeof(int32_t));
  int32_t *olen_w = (int32_t *)malloc(n1 * sizeof(int32_t));
  int64_t *arrive_w = (int64_t *)malloc(n1 * sizeof(int64_t));
  arrival_key *keys = (arrival_key *)malloc(n1 * sizeof(arrival_key));
  int32_t *prefilled = (int32_t *)calloc(n1, sizeof(int32_t));
  if (!g || !rw || !a2 || !ids || !arr_w || !plen_w || !olen_w || !arrive_w || !keys ||
      !prefilled) {
    rc = TSO_ERR_OOM;
    goto done;
  }
  for (int32_t i = 0; i < N; i++) {
    rq *r = &g[i];
    r->phase = (NBp == 0 || NBd == 0 || ceil_div(plen[i], b) > NBp ||
                ceil_div((int64_t)plen[i] + olen[i], b) > NBd ||
                ceil_div((int64_t)plen[i] + 1, b) > adm_cap) ? PH_REJECTED : PH_FUTURE;
    r->target = plen[i];
    r->admit = r->first = r->last = -1;
  }
  int32_t status = (NBp == 0 || NBd == 0) ? TSO_POINT_NO_KV : TSO_POINT_OK;
  int64_t nviol = 0;
  double ubns = 0.0;
  const int32_t np = p->n_prefill, nd = p->n_decode;
  for (int32_t w = 0; w < np && NBp > 0 && NBd > 0; w++) {
    int32_t n = 0;
    for (int32_t i = w; i < N; i += np) {
      ids[n] = i;
      arr_w[n] = arr[i];
      plen_w[n] = plen[i];
      olen_w[n] = olen[i];
      memset(&rw[n], 0, sizeof(rq));
      rw[n].phase = g[i].phase;
      rw[n].target = plen[i];
      rw[n].admit = rw[n].first = rw[n].last = -1;
      rw[n].fresh = 1;
      n++;
    }
    kv_link lk = {dvp.kv_bytes_per_token, p->kv_link_bw > 0.0 ? 1e9 / p->kv_link_bw : 0.0, 0,
                  arrive_w};
    worker_out wo;
    rc = worker_loop(m, &pp, &dvp, WM_PREFILL, n, arr_w, plen_w, olen_w, rw, iter_cap, check,
                     &lk, NULL, 0, &wo);
    if (rc != TSO_OK) goto done;
    if (wo.status > status) status = wo.status;
    out->n_iters += wo.n_iters;
    out->prefill_tokens += wo.prefill_tokens;
    ubns = ubns + wo.used_block_ns;
    nviol += wo.nviol;
    for (int32_t k = 0; k < n; k++) {
      if (rw[k].phase != PH_DONE) continue;
      const int32_t i = ids[k];
      g[i].admit = rw[k].admit;
      g[i].first = rw[k].first;
      a2[i] = arrive_w[k];
      prefilled[i] = 1;
    }
  }
  for (int32_t v = 0; v < nd && NBp > 0 && NBd > 0; v++) {
    int32_t n = 0;
    for (int32_t i = v; i < N; i += nd)
      if (prefilled[i]) {
        keys[n].key = a2[i];
        keys[n].idx = i;
        n++;
      }
    qsort(keys, (size_t)n, sizeof(arrival_key), cmp_arrival);
    for (int32_t k = 0; k < n; k++) {
      const int32_t i = keys[k].idx;
      ids[k] = i;
      arr_w[k] = a2[i];
      plen_w[k] = plen[i];
      olen_w[k] = olen[i];
      memset(&rw[k], 0, sizeof(rq));
      rw[k].phase = PH_FUTURE;
      rw[k].ctx = plen[i];  /* the prompt's KV came over the link */
      rw[k].target = plen[i];
      rw[k].admit = g[i].admit;
      rw[k].first = g[i].first;
      rw[k].last = g[i].first;
      rw[k].fresh = 1;
    }
    worker_out wo;
    rc = worker_loop(m, p, &dvd, WM_DECODE, n, arr_w, plen_w, olen_w, rw, iter_cap, check, NULL,
                     NULL, 0, &wo);
    if (rc != TSO_OK) goto done;
    if (wo.status > status) status = wo.status;
    out->n_iters += wo.n_iters;
    out->n_preempt += wo.n_preempt;
    out->prefill_tokens += wo.prefill_tokens;
    out->decode_tokens += wo.decode_tokens;
    if (wo.peak_used > out->peak_used_blocks) out->peak_used_blocks = wo.peak_used;
    ubns = ubns + wo.used_block_ns;
    nviol += wo.nviol;
    for (int32_t k = 0; k < n; k++) {
      const int32_t i = ids[k];
      g[i].phase = rw[k].phase == PH_DONE ? PH_DONE : PH_RUNNING;
      g[i].last = rw[k].last;
      g[i].max_gap = rw[k].max_gap;
      g[i].n_pre = rw[k].n_pre;
      g[i].gdone = rw[k].gdone;
    }
  }
  {
    int64_t iters = out->n_iters, npre = out->n_preempt, pft = out->prefill_tokens,
            dct = out->decode_tokens, peak = out->peak_used_blocks;
    rc = point_stats(N, arr, olen, g, slo_ttft, slo_tpot, check, out, out_req, &nviol);
    out->n_iters = iters;
    out->n_preempt = npre;
    out->prefill_tokens = pft;
    out->decode_tokens = dct;
    out->peak_used_blocks = peak;
  }
  out->status = status;
  out->used_block_ns = ubns;
  if (violations) *violations = nviol;
done:
  free(g); free(rw); free(a2); free(ids); free(arr_w); free(plen_w); free(olen_w);
  free(arrive_w); free(keys); free(prefilled);
  return rc;
}

int tso_simulate_point(const tso_model *m, const tso_trace *tr, const tso_point *p,
                       const tso_options *opt, tso_point_out *out, tso_req *out_req,
                       tso_iter_rec *log, int64_t log_cap, int64_t *n_log,
                       int64_t *violations) {
  if (!m || !tr || !p || !out) return TSO_ERR_ARG;
  if (tr->n < 0 || (tr->n > 0 && (!tr->arrival_ns || !tr->prompt_len || !tr->output_len)))
    return TSO_ERR_ARG;
  if ((p->n_prefill != 0 || p->n_decode != 0) && log && log_cap > 0)
    return TSO_ERR_ARG;  /* iteration logs: one-worker points only */
  if (p->max_batch < 1 || p->block_size < 1) return TSO_ERR_ARG;
  if (p->policy < TSO_POLICY_MIXED || p->policy > TSO_POLICY_STATIC) return TSO_ERR_ARG;
  if (p->chunk_size != 0 && p->chunk_size < p->max_batch) return TSO_ERR_ARG;
  if (p->policy == TSO_POLICY_PREFILL_FIRST && p->chunk_size != 0) return TSO_ERR_ARG;
  if (p->admit_mem_permille < 0 || p->admit_mem_permille > 1000) return TSO_ERR_ARG;
  if (!(p->swap_bw >= 0.0) || !isfinite(p->swap_bw)) return TSO_ERR_ARG;
  if (p->swap_overlap != 0 && p->swap_overlap != 1) return TSO_ERR_ARG;
  if (p->n_prefill != 0 || p->n_decode != 0) {
    int64_t nv = 0;
    int rc = simulate_pd(m, tr, p, opt, out, out_req, &nv);
    if (n_log) *n_log = 0;
    if (violations) *violations = nv;
    return rc;
  }
  tso_derived dv;
  int rc = tso_derive(m, p, &dv);
  if (rc != TSO_OK) return rc;

  const int64_t iter_cap = (opt && opt->iter_cap > 0) ? opt->iter_cap : DEFAULT_ITER_CAP;
  const int64_t slo_ttft = (opt && opt->slo_ttft_ns > 0) ? opt->slo_ttft_ns : DEFAULT_SLO_TTFT;
  const int64_t slo_tpot = (opt && opt->slo_tpot_ns > 0) ? opt->slo_tpot_ns : DEFAULT_SLO_TPOT;
  const int check = opt ? opt->check_invariants : 0;

  const int32_t N = tr->n;
  const int64_t *arr = tr->arrival_ns;
  const int32_t *plen = tr->prompt_len, *olen = tr->output_len;
  for (int32_t i = 0; i < N; i++) {
    if (plen[i] < 1 || olen[i] < 1 || arr[i] < 0) return TSO_ERR_ARG;
    if (i > 0 && arr[i] < arr[i - 1]) return TSO_ERR_ARG;
  }
  const int64_t NB = dv.num_blocks, b = p->block_size;
  const int64_t adm_cap = p->admit_mem_permille > 0 ? NB * p->admit_mem_permille / 1000 : NB;
  if (p->swap_bw > 0.0 && NB * b * dv.kv_bytes_per_token >= (1LL << 53))
    return TSO_ERR_UNSUPPORTED;

  memset(out, 0, sizeof *out);
  out->num_blocks = (int32_t)NB;
  out->first_arrival_ns = N > 0 ? arr[0] : -1;
  out->last_finish_ns = -1;

  rq *rs = (rq *)calloc((size_t)(N > 0 ? N : 1), sizeof(rq));
  if (!rs) return TSO_ERR_OOM;

  /* A request that could not fit even alone is rejected up front: with
   * recompute preemption it would otherwise never finish.  So is one whose
   * prompt alone exceeds what a first admission may use. */
  for (int32_t i = 0; i < N; i++) {
    rq *r = &rs[i];
    r->phase = (NB == 0 || ceil_div((int64_t)plen[i] + olen[i], b) > NB ||
                ceil_div(plen[i], b) > adm_cap) ? PH_REJECTED : PH_FUTURE;
    r->target = plen[i];
    r->admit = r->first = r->last = -1;
    r->fresh = 1;
  }

  worker_out wo;
  int64_t nviol = 0;
  rc = worker_loop(m, p, &dv, WM_FULL, N, arr, plen, olen, rs, iter_cap, check, NULL, log,
                   log_cap, &wo);
  if (rc == TSO_OK)
    rc = point_stats(N, arr, olen, rs, slo_ttft, slo_tpot, check, out, out_req, &nviol);
  free(rs);
  if (rc != TSO_OK) return rc;
  out->status = wo.status;
  out->n_iters = wo.n_iters;
  out->n_preempt = wo.n_preempt;
  out->prefill_tokens = wo.prefill_tokens;
  out->decode_tokens = wo.decode_tokens;
  out->peak_used_blocks = wo.peak_used;
  out->used_block_ns = wo.used_block_ns;
  if (n_log) *n_log = wo.nlog;
  if (violations) *violations = nviol + wo.nviol;
  return TSO_OK;
}

/* ------------------------------------------------------------ thread pool */
typedef struct {
  const tso_model *m;
  const tso_trace *traces;
  int32_t n_traces;
  const tso_point *points;
  int32_t n_points;
  const tso_options *opt;
  tso_point_out *out;
  tso_req *out_req;
  int32_t max_n;
  int32_t next;   /* shared work counter */
  int rc;         /* first error */
} pool_job;

static void *pool_worker(void *arg) {
  pool_job *jb = (pool_job *)arg;
  for (;;) {
    int32_t i = __atomic_fetch_add(&jb->next, 1, __ATOMIC_RELAXED);
    if (i >= jb->n_points) break;
    const tso_point *p = &jb->points[i];
    int rc;
    if (p->trace_id < 0 || p->trace_id >= jb->n_traces) {
      rc = TSO_ERR_ARG;
    } else {
      const tso_trace *tr = &jb->traces[p->trace_id];
      tso_req *rq_out = jb->out_req ? jb->out_req + (size_t)i * (size_t)jb->max_n : NULL;
      if (rq_out && tr->n > jb->max_n) rc = TSO_ERR_ARG;
      else rc = tso_simulate_point(jb->m, tr, p, jb->opt, &jb->out[i], rq_out, NULL, 0, NULL, NULL);
    }
    if (rc != TSO_OK) {
      int zero = 0;
      __atomic_compare_exchange_n(&jb->rc, &zero, rc, 0, __ATOMIC_RELAXED, __ATOMIC_RELAXED);
    }
  }
  return NULL;
}

int tso_run_points(const tso_model *m, const tso_trace *traces, int32_t n_traces,
                   const tso_point *points, int32_t n_points, const tso_options *opt,
                   tso_point_out *out, tso_req *out_req, int32_t max_n) {
  if (!m || !traces || n_traces < 1 || !points || n_points < 0 || !out) return TSO_ERR_ARG;
  int nt = (opt && opt->n_threads > 0) ? opt->n_threads : (int)sysconf(_SC_NPROCESSORS_ONLN);
  if (nt < 1) nt = 1;
  if (nt > n_points) nt = n_points > 0 ? n_points : 1;
  pool_job jb = {m, traces, n_traces, points, n_points, opt, out, out_req, max_n, 0, 0};
  pthread_t *th = (pthread_t *)malloc((size_t)nt * sizeof(pthread_t));
  if (!th) return TSO_ERR_OOM;
  int started = 0;
  for (int k = 0; k < nt; k++) {
    if (pthread_create(&th[k], NULL, pool_worker, &jb) != 0) break;
    started++;
  }
  if (started == 0) pool_worker(&jb);
  for (int k = 0; k < started; k++) pthread_join(th[k], NULL);
  free(th);
  return jb.rc;
}
