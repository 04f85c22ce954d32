// host.hip -- C ABI of the serving-simulation sweep (see include/ts_sweep.h).
//
// ts_sweep_create validates every input on the host, derives each design
// point's block budget and reciprocals, checks that every cost-model integer
// stays exact in fp64, orders the points longest-expected-first and uploads
// traces and points.  ts_sweep_run enqueues the simulation kernels (one
// per register-chunk class, back to back on the caller's stream: each fills
// the whole GPU with persistent workgroups, so running them concurrently
// gains nothing) and the statistics kernel.  ts_sweep_results copies the results back.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <map>
#include <new>
#include <numeric>
#include <vector>

#include "sweep_host.h"

namespace tsw {
template <int NCH, int MODE, bool SIMPLE>
__global__ void sim_kernel(SimArgs A);
__global__ void pd_merge_kernel(const PdAux* aux, int n_aux, const int64_t* sub_a2,
                                const int32_t* sub_gid, TraceRec* recs, int32_t* gids,
                                DevPoint* units);
__global__ void pd_combine_kernel(const PdAux* aux, int n_aux, ts_point_result* res,
                                  const TraceRec* recs);
__global__ void stats_kernel(ts_req_result* rec, const TraceRec* recs, const PointInfo* pinfo,
                             ts_point_result* res, int64_t* e2e, int64_t* ttft, int max_n,
                             int n_points, int64_t slo_ttft_ns, int64_t slo_tpot_ns,
                             int pad_pending);
__global__ void reset_counters_kernel(unsigned int* c, int n, unsigned long long* w, int nw);
__global__ void fill_kernel(int32_t* p, int n, int32_t v);
}  // namespace tsw

using namespace tsw;

namespace {

thread_local char g_err[256];

constexpr int kClassChunks[kClasses] = {1, 2, 4};

// The kernel of launch 3 * stage + class; one-worker launches whose points
// are all simple (continuous batching, recompute preemption, no admission
// ratio, no request that could never fit, no watchdog) use the variant with
// that policy fixed at compile time.
const void* sim_kernel_fn(int launch, bool simple) {
  const int st = launch / kClasses, c = launch % kClasses;
  if (st == kStageOne && simple) {
    switch (kClassChunks[c]) {
      case 1: return (const void*)sim_kernel<1, kStageOne, true>;
      case 2: return (const void*)sim_kernel<2, kStageOne, true>;
      default: return (const void*)sim_kernel<4, kStageOne, true>;
    }
  }
  switch (st * 8 + kClassChunks[c]) {
    case 0 * 8 + 1: return (const void*)sim_kernel<1, kStageOne, false>;
    case 0 * 8 + 2: return (const void*)sim_kernel<2, kStageOne, false>;
    case 0 * 8 + 4: return (const void*)sim_kernel<4, kStageOne, false>;
    case 1 * 8 + 1: return (const void*)sim_kernel<1, kStagePrefill, false>;
    case 1 * 8 + 2: return (const void*)sim_kernel<2, kStagePrefill, false>;
    case 1 * 8 + 4: return (const void*)sim_kernel<4, kStagePrefill, false>;
    case 2 * 8 + 1: return (const void*)sim_kernel<1, kStageDecode, false>;
    case 2 * 8 + 2: return (const void*)sim_kernel<2, kStageDecode, false>;
    default: return (const void*)sim_kernel<4, kStageDecode, false>;
  }
}

int class_of(int max_batch) { return max_batch <= 64 ? 0 : (max_batch <= 128 ? 1 : 2); }

bool model_ok(const ts_model* m) {
  if (!m) return false;
  if (m->n_layers < 1 || m->n_layers > 4096) return false;
  if (m->d_model < 1 || m->d_model > 131072) return false;
  if (m->n_heads < 1 || m->n_kv_heads < 1) return false;
  if (m->d_model % m->n_heads != 0 || m->n_heads % m->n_kv_heads != 0) return false;
  if (m->ffn_dim < 1 || m->ffn_dim > 524288) return false;
  if (m->ffn_gated != 0 && m->ffn_gated != 1) return false;
  if (m->vocab < 1 || m->vocab > 4194304) return false;
  if (m->w_bytes < 1 || m->w_bytes > 16 || m->kv_bytes < 1 || m->kv_bytes > 16) return false;
  if (m->weights_in_capacity != 0 && m->weights_in_capacity != 1) return false;
  return true;
}

struct TraceStats {
  int64_t max_po = 0;     // largest prompt + output
  int64_t max_p = 0;      // largest prompt
  double mean_p = 0, mean_o = 0, span_s = 0;
};

struct Shape {
  int64_t L, d, dkv, f, g, V, e, ekv;
};

Shape shape_of(const ts_model* m) {
  Shape s;
  s.L = m->n_layers;
  s.d = m->d_model;
  s.dkv = (int64_t)m->n_kv_heads * (m->d_model / m->n_heads);
  s.f = m->ffn_dim;
  s.g = 1 + m->ffn_gated;
  s.V = m->vocab;
  s.e = m->w_bytes;
  s.ekv = m->kv_bytes;
  return s;
}

CostCoef make_coef(const Shape& s) {
  CostCoef c;
  c.f_qkv = 2 * s.d * (s.d + 2 * s.dkv);
  c.b_qkv0 = s.e * s.d * (s.d + 2 * s.dkv);
  c.b_qkv = s.e * s.d + s.ekv * 2 * s.dkv + s.e * s.d;
  c.f_attp = 4 * s.d;
  c.b_attp_c = s.ekv * 2 * s.dkv;
  c.b_attp_t = 2 * s.e * s.d;
  c.f_attd = 4 * s.d;
  c.b_attd_c = s.ekv * 2 * s.dkv;
  c.b_attd_n = 2 * s.e * s.d;
  c.f_out = 2 * s.d * s.d;
  c.b_out0 = s.e * s.d * s.d;
  c.b_out = 2 * s.e * s.d;
  c.f_up = 2 * s.g * s.d * s.f;
  c.b_up0 = s.e * s.g * s.d * s.f;
  c.b_up = s.e * (s.d + s.g * s.f);
  c.f_dn = 2 * s.f * s.d;
  c.b_dn0 = s.e * s.f * s.d;
  c.b_dn = s.e * (s.f + s.d);
  c.f_lm = 2 * s.d * s.V;
  c.b_lm0 = s.e * s.d * s.V;
  c.b_lm = s.e * (s.d + s.V);
  c.n_layers = (double)s.L;
  return c;
}

// Per-lane operator table of the device roofline (lane j prices operator j;
// X/Y/Z are selected on the device: T for the projections and FFN, AP/CP/TP
// for prefill attention, CD/CD/nD for decode attention, R/R for the LM head).
LaneCoef lane_coef(const CostCoef& c) {
  LaneCoef l;
  for (int j = 0; j < 8; ++j) l.f[j] = l.b0[j] = l.b1[j] = l.b2[j] = 0.0;
  const int64_t tab[7][4] = {
      {c.f_qkv, c.b_qkv0, c.b_qkv, 0},          {c.f_attp, 0, c.b_attp_c, c.b_attp_t},
      {c.f_attd, 0, c.b_attd_c, c.b_attd_n},    {c.f_out, c.b_out0, c.b_out, 0},
      {c.f_up, c.b_up0, c.b_up, 0},             {c.f_dn, c.b_dn0, c.b_dn, 0},
      {c.f_lm, c.b_lm0, c.b_lm, 0}};
  for (int j = 0; j < 7; ++j) {
    l.f[j] = (double)tab[j][0];   // all below 2^53: exact
    l.b0[j] = (double)tab[j][1];
    l.b1[j] = (double)tab[j][2];
    l.b2[j] = (double)tab[j][3];
  }
  return l;
}

// Upper bounds of every FLOP / byte count and of the iteration time for a
// point whose requests hold at most max_po tokens.
bool exact_and_bounded(const CostCoef& c, int64_t max_po, int M, int K, double iF, double iB,
                       double xfer_max, int* lg_iter) {
  const double po = (double)max_po;
  const double T = K > 0 ? (double)K : (double)M * po;   // tokens per iteration
  const double AP = T * po;                             // sum q*(c0+q) >= causal pairs
  const double CP = (double)M * po, CD = (double)M * po, nD = M, R = M;
  const double lim = 9007199254740992.0;                 // 2^53
  const double F[7] = {c.f_qkv * T, c.f_attp * AP, c.f_attd * CD, c.f_out * T, c.f_up * T,
                       c.f_dn * T, c.f_lm * R};
  const double Bv[7] = {c.b_qkv0 + c.b_qkv * T, c.b_attp_c * CP + c.b_attp_t * T,
                        c.b_attd_c * CD + c.b_attd_n * nD, c.b_out0 + c.b_out * T,
                        c.b_up0 + c.b_up * T, c.b_dn0 + c.b_dn * T, c.b_lm0 + c.b_lm * R};
  double tmax = 0;
  for (int i = 0; i < 7; ++i) {
    if (!(F[i] < lim) || !(Bv[i] < lim)) return false;
    const double t = std::max(F[i] * iF, Bv[i] * iB);
    tmax += i < 6 ? c.n_layers * t : t;
  }
  tmax += xfer_max;  // swap transfers of one iteration
  // per-lane int32 partial sums (tokens, keys) must not overflow either
  if (T * 4 > 2147483647.0 || CD * 4 > 2147483647.0) return false;
  if (!(tmax < 1125899906842624.0)) return false;  // 2^50 ns per iteration
  // a power of two above twice the bound (ceil and rounding order add less)
  int lg = 1;
  while ((double)((int64_t)1 << lg) < 2.0 * (tmax + 2.0)) ++lg;
  *lg_iter = lg;
  return true;
}

// Longest-expected-first ordering key: a rough count of iterations.  Under
// light load each request runs about prefill + output iterations on its own;
// under load the running set shares iterations.  Only the order of the
// points depends on it, never a result.
double work_estimate(const TraceStats& ts, int64_t n, int M, int K, double peak, double bw,
                     double weight_bytes) {
  const double chunks = K > 0 ? std::ceil(ts.mean_p / K) : 1.0;
  const double per_req = ts.mean_o + chunks;
  const double rate = ts.span_s > 0 ? (double)n / ts.span_s : 1.0;
  const double t_dec = weight_bytes / bw;
  const double t_pre = 2.0 * weight_bytes / 2.0 * ts.mean_p / peak;
  const double busy = rate * (t_pre + ts.mean_o * t_dec);  // mean concurrency
  const double conc = std::min((double)M, std::max(1.0, busy));
  return (double)n * per_req / conc;
}

}  // namespace

namespace tsw {

int device_error(hipError_t e, const char* what) {
  snprintf(g_err, sizeof g_err, "%s: %s", what, hipGetErrorString(e));
  return TS_ERR_DEVICE;
}
void set_error_text(const char* text) { snprintf(g_err, sizeof g_err, "%s", text); }
void clear_error_text() { g_err[0] = 0; }

int Plan::max_grid() const { return std::max(1, *std::max_element(grid, grid + kLaunches)); }

BufCounts buf_counts(const Plan& P) {
  BufCounts c;
  const size_t per_point = (size_t)P.max_n;
  c.recs = P.recs.size();
  c.points = P.dp.size();
  c.order = P.order.size();
  // tickets per launch, the handed points per wider class and bucket, then
  // the positions the 64-slot launch took of its own lists
  c.counter = kLaunches + 3 * kHandBuckets;
  // the 64-slot launch hands at most class_n[1] points on, the 128-slot one
  // at most class_n[2]
  c.handed = P.hand_over ? (size_t)kHandBuckets * (P.class_n[1] + P.class_n[2]) : 0;
  c.work = kLaunches;
  c.resume = (size_t)P.n_resume;
  c.claim = (size_t)P.n_resume;
  c.queue = (size_t)P.max_grid() * kQueueCap;
  c.res = (size_t)(P.count + P.n_extra);
  c.req = (size_t)P.count * per_point;  // the request records (always)
  c.pinfo = P.pinfo.size();
  c.lat = (size_t)P.count * per_point;
  c.pd = P.aux.size();
  c.s1 = (size_t)P.pd_reqs;
  c.sub = (size_t)P.pd_reqs;
  c.gids = P.recs.size();
  return c;
}

double BufCounts::bytes() const {
  return (double)recs * sizeof(TraceRec) + (double)points * sizeof(DevPoint) +
         (double)order * sizeof(int32_t) + (double)counter * sizeof(unsigned int) +
         (double)queue * sizeof(QEntry) +
         (double)res * sizeof(ts_point_result) + (double)req * sizeof(ts_req_result) +
         2.0 * (double)lat * sizeof(int64_t) + (double)pd * sizeof(PdAux) +
         2.0 * (double)s1 * sizeof(int64_t) + (double)sub * (sizeof(int64_t) + sizeof(int32_t)) +
         (double)gids * sizeof(int32_t) + (double)pinfo * sizeof(PointInfo) +
         (double)handed * sizeof(int32_t) + (double)work * sizeof(unsigned long long) +
         (double)resume * (double)kResumeBytes + (double)claim * sizeof(unsigned int);
}

}  // namespace tsw

struct ts_sweep {
  Plan P;
  DevBufs B;
  LaunchEvents ev;
  hipStream_t last_stream = nullptr;
  bool ran = false;
};

namespace {

void release(ts_sweep* h) {
  if (!h) return;
  DevBufs& b = h->B;
  (void)hipFree(b.recs);
  (void)hipFree(b.points);
  (void)hipFree(b.order);
  (void)hipFree(b.counter);
  (void)hipFree(b.queue);
  (void)hipFree(b.res);
  (void)hipFree(b.req);
  (void)hipFree(b.e2e);
  (void)hipFree(b.ttft);
  (void)hipFree(b.pd);
  (void)hipFree(b.s1_admit);
  (void)hipFree(b.s1_first);
  (void)hipFree(b.sub_a2);
  (void)hipFree(b.sub_gid);
  (void)hipFree(b.gids);
  (void)hipFree(b.pinfo);
  (void)hipFree(b.handed);
  (void)hipFree(b.work);
  (void)hipFree(b.resume);
  (void)hipFree(b.claim);
  for (int c = 0; c < kLaunches; ++c) {
    if (h->ev.k0[c]) (void)hipEventDestroy(h->ev.k0[c]);
    if (h->ev.k1[c]) (void)hipEventDestroy(h->ev.k1[c]);
  }
  if (h->ev.t0) (void)hipEventDestroy(h->ev.t0);
  if (h->ev.t1) (void)hipEventDestroy(h->ev.t1);
  if (h->ev.t2) (void)hipEventDestroy(h->ev.t2);
  delete h;
}

template <typename T>
hipError_t dev_alloc(T** p, size_t count) {
  *p = nullptr;
  if (count == 0) count = 1;
  return hipMalloc((void**)p, count * sizeof(T));
}

}  // namespace

namespace tsw {

int make_plan(const ts_model* model, const ts_trace* traces, int32_t n_traces,
              const ts_point* points, int32_t n_points, const ts_options* opt, Plan* P) {
  // ---------------------------------------------------------- validation
  if (!model_ok(model)) return TS_ERR_ARG;
  if (!traces || n_traces < 1 || !points || n_points < 0) return TS_ERR_ARG;
  int first = 0, count = n_points;
  uint32_t flags = 0;
  int64_t iter_cap = (int64_t)1 << 40, slo_ttft = 15000000000LL, slo_tpot = 300000000LL;
  int64_t time_limit_ms = 0;
  if (opt) {
    if (opt->flags & ~(TS_F_PER_REQUEST | TS_F_NO_TAKEOVER)) return TS_ERR_ARG;
    flags = opt->flags;
    if (opt->first_point < 0 || opt->n_points < 0) return TS_ERR_ARG;
    first = opt->first_point;
    if (first > n_points) return TS_ERR_ARG;
    count = opt->n_points == 0 ? n_points - first : opt->n_points;
    if ((int64_t)first + count > n_points) return TS_ERR_ARG;
    if (opt->iter_cap < 0 || opt->slo_ttft_ns < 0 || opt->slo_tpot_ns < 0) return TS_ERR_ARG;
    if (opt->iter_cap > 0) iter_cap = opt->iter_cap;
    if (opt->slo_ttft_ns > 0) slo_ttft = opt->slo_ttft_ns;
    if (opt->slo_tpot_ns > 0) slo_tpot = opt->slo_tpot_ns;
    if (opt->point_time_limit_ms < 0) return TS_ERR_ARG;
    time_limit_ms = opt->point_time_limit_ms;
  }
  std::vector<TraceStats> tstats((size_t)n_traces);
  std::vector<int64_t> toff((size_t)n_traces);
  int64_t total_recs = 0, max_n = 0;
  for (int k = 0; k < n_traces; ++k) {
    const ts_trace& tr = traces[k];
    if (tr.n < 0) return TS_ERR_ARG;
    if (tr.n > 0 && (!tr.arrival_ns || !tr.prompt_len || !tr.output_len)) return TS_ERR_ARG;
    TraceStats& s = tstats[(size_t)k];
    double sp = 0, so = 0;
    for (int i = 0; i < tr.n; ++i) {
      const int64_t a = tr.arrival_ns[i];
      const int32_t p = tr.prompt_len[i], o = tr.output_len[i];
      if (a < 0 || (i > 0 && a < tr.arrival_ns[i - 1])) return TS_ERR_ARG;
      if (p < 1 || o < 1 || p > TS_MAX_TOKENS || o > TS_MAX_TOKENS) return TS_ERR_ARG;
      s.max_po = std::max<int64_t>(s.max_po, (int64_t)p + o);
      s.max_p = std::max<int64_t>(s.max_p, p);
      sp += p;
      so += o;
    }
    if (tr.n > 0) {
      s.mean_p = sp / tr.n;
      s.mean_o = so / tr.n;
      s.span_s = (double)(tr.arrival_ns[tr.n - 1] - tr.arrival_ns[0]) * 1e-9;
    }
    toff[(size_t)k] = total_recs;
    total_recs += tr.n;
    max_n = std::max<int64_t>(max_n, tr.n);
  }
  if (total_recs > INT32_MAX) return TS_ERR_UNSUPPORTED;
  const Shape sh = shape_of(model);
  const CostCoef coef = make_coef(sh);
  const int64_t kv_tok = 2 * sh.L * sh.dkv * sh.ekv;
  const int64_t weights =
      sh.e * (sh.L * (sh.d * (sh.d + 2 * sh.dkv) + sh.d * sh.d + (sh.g + 1) * sh.d * sh.f) +
              2 * sh.V * sh.d);

  // KV blocks of a device: floor(capacity * util / 1000), minus the weights
  // when they share the memory, in whole blocks of block_size tokens
  auto blocks_of = [&](int64_t capacity, int32_t util, int32_t block, int64_t* nb) {
    const __int128 usable = ((__int128)capacity * util) / 1000;
    const __int128 budget = usable - (model->weights_in_capacity ? weights : 0);
    const __int128 per_block = (__int128)block * kv_tok;
    const __int128 v = budget > 0 ? budget / per_block : 0;
    if (v > ((__int128)1 << 30)) return false;
    *nb = (int64_t)v;
    return true;
  };

  // ---------------------------------------------------------- simulation units
  // A one-worker point is one unit.  A disaggregated point is n_prefill
  // prefill-device units, each over its share of the trace (request i goes
  // to prefill device i % n_prefill), and n_decode decode-device units, each
  // over the arrivals of the KV that the merge kernel writes on the device.
  std::vector<DevPoint>& dp = P->dp;
  std::vector<double> est;
  std::vector<int> stage;
  std::vector<PdAux>& aux = P->aux;
  dp.reserve((size_t)count);
  est.reserve((size_t)count);
  stage.reserve((size_t)count);
  int64_t& n_extra = P->n_extra;  // device result records, after the points' own
  int64_t& pd_reqs = P->pd_reqs;  // per-request entries of the disaggregated points
  int64_t extra_recs = 0;  // trace records after the traces: shares, then arrivals
  std::map<std::pair<int, int>, int64_t> share_at;  // (trace, n_prefill) -> first share record
  std::vector<std::pair<int, int>> shares;
  std::vector<int64_t> dec_region;  // per disaggregated point: its arrival records
  for (int i = 0; i < count; ++i) {
    const ts_point& p = points[first + i];
    if (!std::isfinite(p.peak_flops) || !(p.peak_flops > 0) || !std::isfinite(p.mem_bw) ||
        !(p.mem_bw > 0))
      return TS_ERR_ARG;
    if (p.capacity_bytes <= 0 || p.mem_util_permille < 1 || p.mem_util_permille > 1000)
      return TS_ERR_ARG;
    if (p.block_size < 1 || p.block_size > 65536) return TS_ERR_ARG;
    if (p.max_batch < 1) return TS_ERR_ARG;
    if (p.max_batch > TS_MAX_BATCH) return TS_ERR_UNSUPPORTED;
    if (p.chunk_size != 0 && (p.chunk_size < p.max_batch || p.chunk_size > TS_MAX_TOKENS))
      return TS_ERR_ARG;
    if (p.trace_id < 0 || p.trace_id >= n_traces) return TS_ERR_ARG;
    if (p.policy < TS_POLICY_MIXED || p.policy > TS_POLICY_STATIC) return TS_ERR_UNSUPPORTED;
    if (p.policy == TS_POLICY_PREFILL_FIRST && p.chunk_size != 0) return TS_ERR_ARG;
    if (p.admit_mem_permille < 0 || p.admit_mem_permille > 1000) return TS_ERR_ARG;
    if (!std::isfinite(p.swap_bw) || !(p.swap_bw >= 0.0)) return TS_ERR_ARG;
    if (p.swap_overlap != 0 && p.swap_overlap != 1) return TS_ERR_ARG;
    const bool disagg = p.n_prefill != 0 || p.n_decode != 0;
    if (disagg) {
      if (p.n_prefill < 1 || p.n_prefill > TS_MAX_DEVICES || p.n_decode < 1 ||
          p.n_decode > TS_MAX_DEVICES)
        return TS_ERR_ARG;
      if (p.policy != TS_POLICY_MIXED) return TS_ERR_ARG;
      if (!std::isfinite(p.p_peak_flops) || !(p.p_peak_flops > 0) ||
          !std::isfinite(p.p_mem_bw) || !(p.p_mem_bw > 0) || p.p_capacity_bytes <= 0)
        return TS_ERR_ARG;
      if (!std::isfinite(p.kv_link_bw) || !(p.kv_link_bw >= 0.0)) return TS_ERR_ARG;
    }
    int64_t nb = 0;
    if (!blocks_of(p.capacity_bytes, p.mem_util_permille, p.block_size, &nb))
      return TS_ERR_UNSUPPORTED;
    const TraceStats& ts = tstats[(size_t)p.trace_id];
    const int32_t N = traces[p.trace_id].n;
    // the worker (or decode devices) of the point: hardware and memory policy
    DevPoint d{};
    d.inv_flops_ns = 1e9 / p.peak_flops;
    d.inv_bw_ns = 1e9 / p.mem_bw;
    d.num_blocks = (int32_t)nb;
    d.block = p.block_size;
    d.cap_tokens = nb * p.block_size;
    d.max_batch = p.max_batch;
    d.chunk = p.chunk_size;
    d.trace_off = (int32_t)toff[(size_t)p.trace_id];
    d.n = N;
    d.out_index = i;
    d.out_point = i;
    P->pinfo.push_back(PointInfo{d.trace_off, N});
    d.pd = -1;
    // blocks a first admission may leave in use; the rest is reserved
    const int64_t adm_cap = p.admit_mem_permille > 0 ? nb * p.admit_mem_permille / 1000 : nb;
    d.policy = p.policy;
    d.adm_reserve = (int32_t)(nb - adm_cap);
    d.cap_prompt = adm_cap * p.block_size;
    d.may_reject = (ts.max_po > d.cap_tokens || ts.max_p > d.cap_prompt) ? 1 : 0;
    // swap preemption: an iteration moves at most every block once (out, or
    // in after an iteration that preempted nothing), exactly in int64 and fp64
    d.swap = p.swap_bw > 0.0 ? 1 : 0;
    d.swap_overlap = p.swap_overlap;
    d.block_bytes = (int64_t)p.block_size * kv_tok;
    d.inv_link_ns = d.swap ? 1e9 / p.swap_bw : 0.0;
    if (d.swap && (__int128)nb * d.block_bytes >= ((__int128)1 << 53)) return TS_ERR_UNSUPPORTED;
    const double xfer_max = (double)(nb * d.block_bytes) * d.inv_link_ns;
    if (!exact_and_bounded(coef, ts.max_po, p.max_batch, p.chunk_size, d.inv_flops_ns,
                           d.inv_bw_ns, xfer_max, &d.lg_iter))
      return TS_ERR_UNSUPPORTED;
    if (!disagg) {
      dp.push_back(d);
      est.push_back(work_estimate(ts, N, p.max_batch, p.chunk_size, p.peak_flops, p.mem_bw,
                                  (double)weights));
      stage.push_back(kStageOne);
      continue;
    }
    // ---- a disaggregated point
    int64_t nbp = 0;
    if (!blocks_of(p.p_capacity_bytes, p.mem_util_permille, p.block_size, &nbp))
      return TS_ERR_UNSUPPORTED;
    const int n_p = p.n_prefill, n_d = p.n_decode;
    if (pd_reqs + N > INT32_MAX) return TS_ERR_UNSUPPORTED;
    PdAux X{};
    X.n_p = n_p;
    X.n_d = n_d;
    X.point = i;
    X.res0 = (int32_t)(count + n_extra);
    X.trace_off = d.trace_off;
    X.n = N;
    X.req_base = (int32_t)pd_reqs;
    X.no_kv = (nbp == 0 || nb == 0) ? 1 : 0;
    X.num_blocks_d = (int32_t)nb;
    X.kv_bpt = kv_tok;
    X.inv_link_ns = p.kv_link_bw > 0.0 ? 1e9 / p.kv_link_bw : 0.0;
    // sub-list (w, v): the requests of prefill device w bound for decode device v
    std::vector<int64_t> cnt((size_t)n_p * n_d, 0), share_n((size_t)n_p, 0), dec_n((size_t)n_d, 0);
    for (int32_t r = 0; r < N; ++r) {
      cnt[(size_t)(r % n_p) * n_d + (size_t)(r % n_d)]++;
      share_n[(size_t)(r % n_p)]++;
      dec_n[(size_t)(r % n_d)]++;
    }
    int64_t acc = pd_reqs;
    for (int w = 0; w < n_p; ++w)
      for (int v = 0; v < n_d; ++v) {
        X.sub_off[w * kMaxDev + v] = (int32_t)acc;
        acc += cnt[(size_t)w * n_d + v];
      }
    pd_reqs += N;
    // the prefill devices' shares of the trace, once per (trace, n_prefill)
    const std::pair<int, int> key(p.trace_id, n_p);
    auto it = share_at.find(key);
    int64_t share0;
    if (it == share_at.end()) {
      share0 = total_recs + extra_recs;
      share_at[key] = share0;
      shares.push_back(key);
      extra_recs += N;
    } else {
      share0 = it->second;
    }
    // the decode devices' arrival records
    const int64_t dec0 = total_recs + extra_recs;
    extra_recs += N;
    dec_region.push_back(dec0);
    int64_t pos = 0;
    for (int v = 0; v < n_d; ++v) {
      X.dec_off[v] = (int32_t)(dec0 + pos);
      pos += dec_n[(size_t)v];
    }
    if (total_recs + extra_recs > INT32_MAX) return TS_ERR_UNSUPPORTED;
    const int pd_index = (int)aux.size();
    // prefill devices: their own hardware and memory, continuous batching
    // over prefills only; they reject what a prefill or a decode device can
    // never hold
    DevPoint dpp = d;
    dpp.inv_flops_ns = 1e9 / p.p_peak_flops;
    dpp.inv_bw_ns = 1e9 / p.p_mem_bw;
    dpp.num_blocks = (int32_t)nbp;
    dpp.cap_tokens = nbp * p.block_size;
    dpp.policy = TS_POLICY_MIXED;
    dpp.adm_reserve = 0;
    dpp.cap_prompt = adm_cap * p.block_size - 1;  // prompt + the next token within the ratio
    dpp.cap_po2 = nb * p.block_size;
    dpp.may_reject = (ts.max_p > dpp.cap_tokens || ts.max_po > dpp.cap_po2 ||
                      ts.max_p > dpp.cap_prompt) ? 1 : 0;
    dpp.swap = 0;
    dpp.swap_overlap = 0;
    dpp.inv_link_ns = 0.0;
    dpp.pd = pd_index;
    if (!exact_and_bounded(coef, ts.max_po, p.max_batch, p.chunk_size, dpp.inv_flops_ns,
                           dpp.inv_bw_ns, 0.0, &dpp.lg_iter))
      return TS_ERR_UNSUPPORTED;
    int64_t start = 0;
    for (int w = 0; w < n_p; ++w) {
      DevPoint u = dpp;
      u.trace_off = (int32_t)(share0 + start);
      u.n = (int32_t)share_n[(size_t)w];
      u.out_index = (int32_t)(count + n_extra++);
      u.unit = w;
      start += share_n[(size_t)w];
      dp.push_back(u);
      est.push_back(work_estimate(ts, u.n, p.max_batch, p.chunk_size, p.p_peak_flops,
                                  p.p_mem_bw, (double)weights));
      stage.push_back(kStagePrefill);
    }
    // decode devices: the point's hardware and memory policy; every request
    // that reaches them fits
    X.dec_unit0 = (int32_t)dp.size();
    for (int v = 0; v < n_d; ++v) {
      DevPoint u = d;
      u.trace_off = X.dec_off[v];
      u.n = 0;  // set on the device by the merge kernel
      u.out_index = (int32_t)(count + n_extra++);
      u.pd = pd_index;
      u.unit = v;
      u.may_reject = 0;
      dp.push_back(u);
      est.push_back(work_estimate(ts, dec_n[(size_t)v], p.max_batch, p.chunk_size, p.peak_flops,
                                  p.mem_bw, (double)weights));
      stage.push_back(kStageDecode);
    }
    aux.push_back(X);
  }
  if (count + n_extra > INT32_MAX) return TS_ERR_UNSUPPORTED;

  // ---------------------------------------------------------- launches + order
  std::vector<int32_t>& order = P->order;
  order.reserve(dp.size());
  for (int l = 0; l < kLaunches; ++l) {
    std::vector<int32_t> cls;
    for (size_t u = 0; u < dp.size(); ++u)
      if (stage[u] == l / kClasses && class_of(dp[u].max_batch) == l % kClasses)
        cls.push_back((int32_t)u);
    std::stable_sort(cls.begin(), cls.end(),
                     [&](int32_t a, int32_t b) { return est[(size_t)a] > est[(size_t)b]; });
    P->class_off[l] = (int)order.size();
    P->class_n[l] = (int)cls.size();
    // one-worker launches whose points are all simple take the kernel with
    // the policy fixed at compile time
    bool simple = l / kClasses == kStageOne && time_limit_ms == 0;
    for (const int32_t u : cls) {
      const DevPoint& d = dp[(size_t)u];
      simple = simple && d.policy == TS_POLICY_MIXED && d.swap == 0 && d.adm_reserve == 0 &&
               d.cap_prompt == d.cap_tokens && d.may_reject == 0;
    }
    P->simple[l] = simple;
    order.insert(order.end(), cls.begin(), cls.end());
  }
  // One-worker points wider than 64 slots that are simple run first in the
  // 64-slot launch (more waves per SIMD, fewer registers) while at most 64
  // run at once; the few that need more are handed to the 128-slot launch,
  // and from there those that need more than 128 to the 256-slot launch,
  // each continuing from its hand-over record.
  bool all_simple = true;
  for (int c = 0; c < kClasses; ++c)
    all_simple = all_simple && (P->class_n[c] == 0 || P->simple[c]);
  if (all_simple && P->class_n[1] + P->class_n[2] > 0) {
    std::vector<int32_t> all(order.begin(), order.begin() + P->class_n[0] + P->class_n[1] +
                                                               P->class_n[2]);
    std::stable_sort(all.begin(), all.end(),
                     [&](int32_t a, int32_t b) { return est[(size_t)a] > est[(size_t)b]; });
    std::copy(all.begin(), all.end(), order.begin());
    P->class_off[0] = 0;
    // class_n[2]: the points that may reach the 256-slot launch; class_n[1]:
    // those that may reach the 128-slot one
    P->class_n[1] = P->class_n[1] + P->class_n[2];
    P->class_n[0] = (int)all.size();
    P->simple[0] = P->simple[1] = P->simple[2] = true;
    P->hand_over = true;
  }
  // a hand-over state slot for each point a launch may hand on
  P->n_resume = 0;
  for (size_t u = 0; u < dp.size(); ++u) {
    const bool wide = P->hand_over && stage[u] == kStageOne && dp[u].max_batch > 64;
    dp[u].resume = wide ? P->n_resume++ : -1;
  }
  P->count = count;
  P->n_pd = (int32_t)aux.size();
  P->max_n = (int32_t)std::max<int64_t>(max_n, 1);
  P->flags = flags;
  P->iter_cap = iter_cap;
  P->slo_ttft = slo_ttft;
  P->slo_tpot = slo_tpot;
  P->time_limit_ms = time_limit_ms;
  P->coef = coef;
  P->lc = lane_coef(coef);

  // ---------------------------------------------------------- device
  hipError_t e = hipGetDevice(&P->device);
  if (e != hipSuccess) { return device_error(e, "hipGetDevice"); }
  hipDeviceProp_t prop;
  e = hipGetDeviceProperties(&prop, P->device);
  if (e != hipSuccess) { return device_error(e, "hipGetDeviceProperties"); }
  const int n_cu = prop.multiProcessorCount;
  for (int l = 0; l < kLaunches; ++l) {
    if (P->class_n[l] == 0) continue;
    int per_cu = 0;
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, sim_kernel_fn(l, P->simple[l]), 64,
                                                     0);
    if (e != hipSuccess) { return device_error(e, "occupancy query"); }
    per_cu = std::max(per_cu, 1);
    P->grid[l] = std::min(P->class_n[l], n_cu * per_cu);
  }
  {
    int per_cu = 0;
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, stats_kernel, 256, 0);
    if (e != hipSuccess) { return device_error(e, "occupancy query"); }
    P->stats_grid = std::max(1, std::min(count, n_cu * std::max(per_cu, 1)));
  }

  std::vector<TraceRec>& recs = P->recs;
  recs.assign((size_t)std::max<int64_t>(total_recs + extra_recs, 1), TraceRec{});
  for (int k = 0; k < n_traces; ++k) {
    const ts_trace& tr = traces[k];
    for (int i = 0; i < tr.n; ++i) {
      TraceRec& r = recs[(size_t)(toff[(size_t)k] + i)];
      r.arrival_ns = tr.arrival_ns[i];
      r.prompt = tr.prompt_len[i];
      r.output = tr.output_len[i];
    }
  }
  for (const auto& key : shares) {  // share w: requests w, w + n_p, ... in order
    const ts_trace& tr = traces[key.first];
    int64_t at = share_at[key];
    for (int w = 0; w < key.second; ++w)
      for (int i = w; i < tr.n; i += key.second) {
        TraceRec& r = recs[(size_t)at++];
        r.arrival_ns = tr.arrival_ns[i];
        r.prompt = tr.prompt_len[i];
        r.output = tr.output_len[i];
      }
  }
  return TS_OK;
}

int upload(const Plan& P, const DevBufs& B, bool async, hipStream_t s) {
  struct Part { void* dst; const void* src; size_t bytes; };
  const Part parts[5] = {
      {B.recs, P.recs.data(), P.recs.size() * sizeof(TraceRec)},
      {B.points, P.dp.data(), P.dp.size() * sizeof(DevPoint)},
      {B.order, P.order.data(), P.order.size() * sizeof(int32_t)},
      {B.pd, P.aux.data(), P.aux.size() * sizeof(PdAux)},
      {B.pinfo, P.pinfo.data(), P.pinfo.size() * sizeof(PointInfo)}};
  for (const Part& q : parts) {
    if (q.bytes == 0) continue;
    const hipError_t e = async ? hipMemcpyAsync(q.dst, q.src, q.bytes, hipMemcpyHostToDevice, s)
                               : hipMemcpy(q.dst, q.src, q.bytes, hipMemcpyHostToDevice);
    if (e != hipSuccess) return device_error(e, "upload");
  }
  return TS_OK;
}

int enqueue(const Plan& P, const DevBufs& B, hipStream_t s, const LaunchEvents* ev) {
  auto record = [&](hipEvent_t e) -> hipError_t {
    return (ev && e) ? hipEventRecord(e, s) : hipSuccess;
  };
  hipError_t e = record(ev ? ev->t0 : nullptr);
  if (e != hipSuccess) return device_error(e, "event record");
  reset_counters_kernel<<<1, 64, 0, s>>>(B.counter, kLaunches + 3 * kHandBuckets, B.work,
                                          kLaunches);
  if (P.hand_over) {
    // the 64-slot launch's lists start empty (-1: not written yet), as do
    // the claims, since it takes points from its lists while it fills them
    const int n_list = kHandBuckets * P.class_n[1];
    fill_kernel<<<std::max(1, std::min((n_list + 255) / 256, 1024)), 256, 0, s>>>(B.handed, n_list,
                                                                                 -1);
    fill_kernel<<<std::max(1, std::min((P.n_resume + 255) / 256, 1024)), 256, 0, s>>>(
        reinterpret_cast<int32_t*>(B.claim), P.n_resume, 0);
    e = hipGetLastError();
    if (e != hipSuccess) return device_error(e, "fill kernel launch");
  }
  SimArgs a;
  a.recs = B.recs;
  a.points = B.points;
  a.max_n = P.max_n;
  a.queue = B.queue;
  a.res = B.res;
  a.rec = B.req;
  a.iter_cap = P.iter_cap;
  a.work = nullptr;
  a.handed = B.handed;
  a.handed_off[0] = 0;
  a.handed_off[1] = kHandBuckets * P.class_n[1];
  a.hand_cap[0] = P.class_n[1];
  a.hand_cap[1] = P.class_n[2];
  a.hand_cap_in = 0;
  a.handed_n = B.counter + kLaunches;
  a.n_dev = nullptr;
  a.resume = P.hand_over ? B.resume : nullptr;
  a.take = nullptr;
  a.claim = nullptr;
  a.time_limit_ticks = (uint64_t)P.time_limit_ms * 100000ull;  // 100 MHz clock
  a.n_layers = P.coef.n_layers;
  a.lc = P.lc;
  a.pd = B.pd;
  a.s1_admit = B.s1_admit;
  a.s1_first = B.s1_first;
  a.sub_a2 = B.sub_a2;
  a.sub_gid = B.sub_gid;
  a.gids = B.gids;
  // one launch per (stage, class), back to back: one-worker points and
  // prefill devices, the merge of the prefill devices' hand-overs, the
  // decode devices, then the disaggregated points' records
  for (int l = 0; l < kLaunches; ++l) {
    if (l == kStageDecode * kClasses && P.n_pd > 0) {
      pd_merge_kernel<<<std::min(P.n_pd * kMaxDev, 65536), 256, 0, s>>>(
          B.pd, P.n_pd, B.sub_a2, B.sub_gid, B.recs, B.gids, B.points);
      e = hipGetLastError();
      if (e != hipSuccess) return device_error(e, "merge kernel launch");
    }
    if (P.class_n[l] == 0) continue;
    a.order = B.order + P.class_off[l];
    a.n_order = P.class_n[l];
    a.n_dev = nullptr;
    if (P.hand_over && (l == 1 || l == 2)) {  // the points launch 0 handed over
      a.order = B.handed + a.handed_off[l - 1];
      a.n_dev = B.counter + kLaunches + (l - 1) * kHandBuckets;
      a.hand_cap_in = a.hand_cap[l - 1];
    }
    // launch 0 also continues points it handed over; launch 1 skips those
    a.take = (P.hand_over && l == 0 && !(P.flags & TS_F_NO_TAKEOVER))
                 ? B.counter + kLaunches + 2 * kHandBuckets
                 : nullptr;
    a.claim = (P.hand_over && l <= 1) ? B.claim : nullptr;
    a.counter = B.counter + l;
    a.work = B.work + l;
    e = record(ev ? ev->k0[l] : nullptr);
    if (e != hipSuccess) return device_error(e, "event record");
    const int g = P.grid[l];
    switch (l + (P.simple[l] ? 100 : 0)) {
      case 0: sim_kernel<1, kStageOne, false><<<g, 64, 0, s>>>(a); break;
      case 1: sim_kernel<2, kStageOne, false><<<g, 64, 0, s>>>(a); break;
      case 2: sim_kernel<4, kStageOne, false><<<g, 64, 0, s>>>(a); break;
      case 100: sim_kernel<1, kStageOne, true><<<g, 64, 0, s>>>(a); break;
      case 101: sim_kernel<2, kStageOne, true><<<g, 64, 0, s>>>(a); break;
      case 102: sim_kernel<4, kStageOne, true><<<g, 64, 0, s>>>(a); break;
      case 3: sim_kernel<1, kStagePrefill, false><<<g, 64, 0, s>>>(a); break;
      case 4: sim_kernel<2, kStagePrefill, false><<<g, 64, 0, s>>>(a); break;
      case 5: sim_kernel<4, kStagePrefill, false><<<g, 64, 0, s>>>(a); break;
      case 6: sim_kernel<1, kStageDecode, false><<<g, 64, 0, s>>>(a); break;
      case 7: sim_kernel<2, kStageDecode, false><<<g, 64, 0, s>>>(a); break;
      default: sim_kernel<4, kStageDecode, false><<<g, 64, 0, s>>>(a); break;
    }
    e = hipGetLastError();
    if (e != hipSuccess) return device_error(e, "sim kernel launch");
    e = record(ev ? ev->k1[l] : nullptr);
    if (e != hipSuccess) return device_error(e, "event record");
  }
  if (P.n_pd > 0) {
    pd_combine_kernel<<<std::min((P.n_pd + 255) / 256, 65536), 256, 0, s>>>(B.pd, P.n_pd,
                                                                             B.res, B.recs);
    e = hipGetLastError();
    if (e != hipSuccess) return device_error(e, "combine kernel launch");
  }
  e = record(ev ? ev->t1 : nullptr);
  if (e != hipSuccess) return device_error(e, "event record");
  if (P.count > 0)
    stats_kernel<<<P.stats_grid, 256, 0, s>>>(B.req, B.recs, B.pinfo, B.res, B.e2e, B.ttft,
                                              P.max_n, P.count, P.slo_ttft, P.slo_tpot,
                                              (P.flags & TS_F_PER_REQUEST) ? 1 : 0);
  e = hipGetLastError();
  if (e != hipSuccess) return device_error(e, "stats kernel launch");
  e = record(ev ? ev->t2 : nullptr);
  if (e != hipSuccess) return device_error(e, "event record");
  return TS_OK;
}

}  // namespace tsw

extern "C" {

const char* ts_status_str(int status) {
  switch (status) {
    case TS_OK: return "ok";
    case TS_ERR_ARG: return "invalid argument";
    case TS_ERR_UNSUPPORTED:
      return g_err[0] ? g_err : "unsupported input (batch cap, policy, or exact-fp64 range)";
    case TS_ERR_OOM: return g_err[0] ? g_err : "out of memory";
    case TS_ERR_DEVICE: return g_err[0] ? g_err : "HIP device error";
    case TS_ERR_STATE: return "call out of order";
    default: return "unknown status";
  }
}

int ts_sweep_create(const ts_model* model, const ts_trace* traces, int32_t n_traces,
                    const ts_point* points, int32_t n_points, const ts_options* opt,
                    ts_sweep** out) {
  if (!out) return TS_ERR_ARG;
  *out = nullptr;
  g_err[0] = 0;
  ts_sweep* h = new (std::nothrow) ts_sweep();
  if (!h) return TS_ERR_OOM;
  int rc = make_plan(model, traces, n_traces, points, n_points, opt, &h->P);
  if (rc != TS_OK) {
    release(h);
    return rc;
  }
  const BufCounts n = buf_counts(h->P);
  // Everything the handle will hold on the device; more than the free
  // device memory is TS_ERR_OOM before any allocation is attempted.
  size_t mem_free = 0, mem_total = 0;
  hipError_t e = hipMemGetInfo(&mem_free, &mem_total);
  if (e != hipSuccess) { release(h); return device_error(e, "hipMemGetInfo"); }
  if (n.bytes() > (double)mem_free) {
    snprintf(g_err, sizeof g_err, "the sweep needs %.3g bytes of device memory, %.3g free",
             n.bytes(), (double)mem_free);
    release(h);
    return TS_ERR_OOM;
  }
  DevBufs& b = h->B;
  hipError_t ae = hipSuccess;
  if (ae == hipSuccess) ae = dev_alloc(&b.recs, n.recs);
  if (ae == hipSuccess) ae = dev_alloc(&b.points, n.points);
  if (ae == hipSuccess) ae = dev_alloc(&b.order, n.order);
  if (ae == hipSuccess) ae = dev_alloc(&b.counter, n.counter);
  if (ae == hipSuccess) ae = dev_alloc(&b.queue, n.queue);
  if (ae == hipSuccess) ae = dev_alloc(&b.res, n.res);
  if (ae == hipSuccess) ae = dev_alloc(&b.e2e, n.lat);
  if (ae == hipSuccess) ae = dev_alloc(&b.ttft, n.lat);
  if (ae == hipSuccess) ae = dev_alloc(&b.req, n.req);
  if (ae == hipSuccess) ae = dev_alloc(&b.pinfo, n.pinfo);
  if (ae == hipSuccess) ae = dev_alloc(&b.handed, n.handed);
  if (ae == hipSuccess) ae = dev_alloc(&b.work, n.work);
  if (ae == hipSuccess) ae = dev_alloc(&b.resume, n.resume * kResumeBytes);
  if (ae == hipSuccess) ae = dev_alloc(&b.claim, n.claim);
  if (ae == hipSuccess) ae = dev_alloc(&b.pd, n.pd);
  if (ae == hipSuccess) ae = dev_alloc(&b.s1_admit, n.s1);
  if (ae == hipSuccess) ae = dev_alloc(&b.s1_first, n.s1);
  if (ae == hipSuccess) ae = dev_alloc(&b.sub_a2, n.sub);
  if (ae == hipSuccess) ae = dev_alloc(&b.sub_gid, n.sub);
  if (ae == hipSuccess) ae = dev_alloc(&b.gids, n.gids);
  if (ae != hipSuccess) {
    const int rc2 = ae == hipErrorOutOfMemory ? TS_ERR_OOM : device_error(ae, "hipMalloc");
    if (rc2 == TS_ERR_OOM) snprintf(g_err, sizeof g_err, "device allocation failed");
    release(h);
    return rc2;
  }
  rc = upload(h->P, b, false, nullptr);
  if (rc != TS_OK) {
    release(h);
    return rc;
  }
  // the host copies of the uploaded records are no longer needed
  std::vector<TraceRec>().swap(h->P.recs);
  std::vector<DevPoint>().swap(h->P.dp);
  std::vector<int32_t>().swap(h->P.order);
  std::vector<PdAux>().swap(h->P.aux);
  for (int c = 0; c < kLaunches && e == hipSuccess; ++c) {
    e = hipEventCreate(&h->ev.k0[c]);
    if (e == hipSuccess) e = hipEventCreate(&h->ev.k1[c]);
  }
  if (e == hipSuccess) e = hipEventCreate(&h->ev.t0);
  if (e == hipSuccess) e = hipEventCreate(&h->ev.t1);
  if (e == hipSuccess) e = hipEventCreate(&h->ev.t2);
  if (e != hipSuccess) { release(h); return device_error(e, "stream/event create"); }
  *out = h;
  return TS_OK;
}

int ts_sweep_run(ts_sweep* h, void* hip_stream) {
  if (!h) return TS_ERR_ARG;
  hipStream_t s = (hipStream_t)hip_stream;
  hipError_t e = hipSetDevice(h->P.device);
  if (e != hipSuccess) return device_error(e, "hipSetDevice");
  // A re-run reuses the work-queue counters, queues, request records and result
  // buffers of the previous run: on another stream it must wait for that
  // run's last kernel.
  if (h->ran && s != h->last_stream) {
    e = hipStreamWaitEvent(s, h->ev.t2, 0);
    if (e != hipSuccess) return device_error(e, "stream wait");
  }
  const int rc = enqueue(h->P, h->B, s, &h->ev);
  if (rc != TS_OK) return rc;
  h->last_stream = s;
  h->ran = true;
  return TS_OK;
}

int ts_sweep_results(ts_sweep* h, ts_point_result* out_points, ts_req_result* out_requests) {
  if (!h) return TS_ERR_ARG;
  if (!h->ran) return TS_ERR_STATE;
  if (out_requests && !(h->P.flags & TS_F_PER_REQUEST)) return TS_ERR_STATE;
  if (!out_points && h->P.count > 0) return TS_ERR_ARG;
  hipError_t e = hipSetDevice(h->P.device);
  if (e == hipSuccess) e = hipStreamSynchronize(h->last_stream);
  if (e != hipSuccess) return device_error(e, "stream synchronize");
  if (h->P.count > 0) {
    e = hipMemcpy(out_points, h->B.res, (size_t)h->P.count * sizeof(ts_point_result),
                  hipMemcpyDeviceToHost);
    if (e != hipSuccess) return device_error(e, "copy results");
  }
  if (out_requests && h->P.count > 0) {
    e = hipMemcpy(out_requests, h->B.req,
                  (size_t)h->P.count * (size_t)h->P.max_n * sizeof(ts_req_result),
                  hipMemcpyDeviceToHost);
    if (e != hipSuccess) return device_error(e, "copy request records");
  }
  return TS_OK;
}

int ts_sweep_shape(const ts_sweep* h, int32_t* n_points, int32_t* max_n) {
  if (!h || !n_points || !max_n) return TS_ERR_ARG;
  *n_points = h->P.count;
  *max_n = h->P.max_n;
  return TS_OK;
}

int ts_sweep_timing(ts_sweep* h, float* sim_ms, float* stats_ms) {
  if (!h || !sim_ms || !stats_ms) return TS_ERR_ARG;
  if (!h->ran) return TS_ERR_STATE;
  hipError_t e = hipSetDevice(h->P.device);
  if (e == hipSuccess) e = hipEventSynchronize(h->ev.t2);
  if (e == hipSuccess) e = hipEventElapsedTime(sim_ms, h->ev.t0, h->ev.t1);
  if (e == hipSuccess) e = hipEventElapsedTime(stats_ms, h->ev.t1, h->ev.t2);
  if (e != hipSuccess) return device_error(e, "event timing");
  return TS_OK;
}

int ts_sweep_kernel_timing(ts_sweep* h, float* ms, int32_t* n_points) {
  if (!h || !ms || !n_points) return TS_ERR_ARG;
  if (!h->ran) return TS_ERR_STATE;
  hipError_t e = hipSetDevice(h->P.device);
  if (e == hipSuccess) e = hipEventSynchronize(h->ev.t2);
  for (int c = 0; c < kLaunches && e == hipSuccess; ++c) {
    ms[c] = 0.0f;
    n_points[c] = h->P.class_n[c];
    if (h->P.class_n[c] > 0) e = hipEventElapsedTime(&ms[c], h->ev.k0[c], h->ev.k1[c]);
  }
  if (e != hipSuccess) return device_error(e, "event timing");
  return TS_OK;
}

int ts_sweep_kernel_work(ts_sweep* h, int64_t* iters) {
  if (!h || !iters) return TS_ERR_ARG;
  if (!h->ran) return TS_ERR_STATE;
  hipError_t e = hipSetDevice(h->P.device);
  if (e == hipSuccess) e = hipEventSynchronize(h->ev.t2);
  if (e == hipSuccess)
    e = hipMemcpy(iters, h->B.work, kLaunches * sizeof(int64_t), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return device_error(e, "copy launch work");
  return TS_OK;
}

void ts_sweep_destroy(ts_sweep* h) { release(h); }

}  // extern "C"
