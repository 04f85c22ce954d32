// sim_kernel.hip -- gfx950 kernels of the serving-simulation sweep.
//
// One wave64 workgroup owns one design point at a time and runs TokenSim's
// per-iteration step (arXiv 2503.08415: continuous batching, Sec. II-B and
// Sec. IV-A; block-granular KV memory manager, Sec. III-B; preemption of the
// newest requests when blocks run out, Sec. IV-B; per-iteration compute
// simulator, Sec. III overview) until every request has finished:
//   * running requests live in "slots" in admission order: slot s is lane
//     s % 64 of register chunk s / 64 (NCH chunks cover max_batch <= 64*NCH);
//   * intake streams the trace as 64-record windows (one 16-byte load per
//     lane) and counts arrivals with a ballot;
//   * block reservation and recompute preemption are one inclusive wave scan
//     of held + needed blocks against the block count;
//   * the chunk budget and FCFS admission are prefix scans over slots and
//     over a 64-candidate window;
//   * the batch sums that feed the roofline are wave reductions (DPP);
//   * finished requests are found by ballot and removed by a stable
//     compaction through LDS;
//   * steady stretches advance decodes lazily and price up to 64 iterations
//     at once, one per lane (while a head prefill runs, through the decodes
//     that finish in them); a head prefill's completion, the admissions
//     behind it and the finishes in the same iteration are handled in place;
//   * a finish writes the request's record, from which the statistics
//     kernel derives every latency statistic and percentile;
//   * a narrow launch takes points wider than its slots and hands those that
//     need more running requests to a wider launch, with a record of their
//     state; the 64-slot launch itself continues them with 128 slots in the
//     workgroups that have no point of their own left.
// Scheduling state is integer; only the roofline is fp64, evaluated in a
// fixed order with contraction disabled.
#include <hip/hip_runtime.h>

#include "sweep_internal.h"

#pragma clang fp contract(off)

namespace tsw {

// ------------------------------------------------------------ wave helpers
__device__ __forceinline__ int lane_id() {
  return (int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
}
__device__ __forceinline__ uint64_t ballot(bool p) { return __builtin_amdgcn_ballot_w64(p); }
__device__ __forceinline__ int popc(uint64_t m) { return __popcll(m); }
// number of set bits of m below this lane
__device__ __forceinline__ int rank_below(uint64_t m) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                        __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}
__device__ __forceinline__ int rdl(int v, int l) { return __builtin_amdgcn_readlane(v, l); }
__device__ __forceinline__ int64_t rdl64(int64_t v, int l) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)v >> 32), l);
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Row shift with zero fill (bound_ctrl): every lane is written, no "old".
template <int CTRL>
__device__ __forceinline__ int shr0(int v) {
  return __builtin_amdgcn_mov_dpp(v, CTRL, 0xf, 0xf, true);
}
// DPP move with zero for lanes whose source is outside the row / not selected.
// A row shift over every row needs no zeroed "old": bound_ctrl fills it.
template <int CTRL, int ROWS>
__device__ __forceinline__ int dpp0(int v) {
  if constexpr (ROWS == 0xf && (CTRL & 0xff0) == 0x110) return shr0<CTRL>(v);
  return __builtin_amdgcn_update_dpp(0, v, CTRL, ROWS, 0xf, false);
}
template <int CTRL, int ROWS>
__device__ __forceinline__ int64_t dpp0_64(int64_t v) {
  const uint32_t lo = (uint32_t)dpp0<CTRL, ROWS>((int)(uint32_t)v);
  const uint32_t hi = (uint32_t)dpp0<CTRL, ROWS>((int)(uint32_t)((uint64_t)v >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}
// Inclusive prefix sum over the 64 lanes: Hillis-Steele inside each 16-lane
// row (row_shr 1, 2, 4, 8), then row 15 -> rows 1,3 and row 31 -> rows 2,3.
__device__ __forceinline__ int scan_i32(int v) {
  v += shr0<0x111>(v);
  v += shr0<0x112>(v);
  v += shr0<0x114>(v);
  v += shr0<0x118>(v);
  v += dpp0<0x142, 0xa>(v);
  v += dpp0<0x143, 0xc>(v);
  return v;
}
__device__ __forceinline__ int64_t scan_i64(int64_t v) {
  v += dpp0_64<0x111, 0xf>(v);
  v += dpp0_64<0x112, 0xf>(v);
  v += dpp0_64<0x114, 0xf>(v);
  v += dpp0_64<0x118, 0xf>(v);
  v += dpp0_64<0x142, 0xa>(v);
  v += dpp0_64<0x143, 0xc>(v);
  return v;
}
// Inclusive prefix sum of doubles (zero fill adds +0.0).  Exact while every
// value is an integer and every partial sum stays below 2^53, whatever the
// order of the additions.
__device__ __forceinline__ double scan_f64(double v) {
  auto sh = [](double x, auto ctrl) {
    return __builtin_bit_cast(double, ctrl(__builtin_bit_cast(int64_t, x)));
  };
  v = v + sh(v, [](int64_t x) { return dpp0_64<0x111, 0xf>(x); });
  v = v + sh(v, [](int64_t x) { return dpp0_64<0x112, 0xf>(x); });
  v = v + sh(v, [](int64_t x) { return dpp0_64<0x114, 0xf>(x); });
  v = v + sh(v, [](int64_t x) { return dpp0_64<0x118, 0xf>(x); });
  v = v + sh(v, [](int64_t x) { return dpp0_64<0x142, 0xa>(x); });
  v = v + sh(v, [](int64_t x) { return dpp0_64<0x143, 0xc>(x); });
  return v;
}
// Inclusive prefix max of non-negative values (0 is the identity).
__device__ __forceinline__ int64_t scan_max_i64(int64_t v) {
  int64_t u;
  u = dpp0_64<0x111, 0xf>(v); v = u > v ? u : v;
  u = dpp0_64<0x112, 0xf>(v); v = u > v ? u : v;
  u = dpp0_64<0x114, 0xf>(v); v = u > v ? u : v;
  u = dpp0_64<0x118, 0xf>(v); v = u > v ? u : v;
  u = dpp0_64<0x142, 0xa>(v); v = u > v ? u : v;
  u = dpp0_64<0x143, 0xc>(v); v = u > v ? u : v;
  return v;
}
// Inclusive prefix max of non-negative 32-bit values (0 is the identity).
__device__ __forceinline__ int scan_max_i32(int v) {
  int u;
  u = shr0<0x111>(v); v = u > v ? u : v;
  u = shr0<0x112>(v); v = u > v ? u : v;
  u = shr0<0x114>(v); v = u > v ? u : v;
  u = shr0<0x118>(v); v = u > v ? u : v;
  u = dpp0<0x142, 0xa>(v); v = u > v ? u : v;
  u = dpp0<0x143, 0xc>(v); v = u > v ? u : v;
  return v;
}
// Wrapping (mod 2^64) sum over the lanes, for hashes.
__device__ __forceinline__ uint64_t wsum_u64(uint64_t v) {
  v += (uint64_t)dpp0_64<0x111, 0xf>((int64_t)v);
  v += (uint64_t)dpp0_64<0x112, 0xf>((int64_t)v);
  v += (uint64_t)dpp0_64<0x114, 0xf>((int64_t)v);
  v += (uint64_t)dpp0_64<0x118, 0xf>((int64_t)v);
  v += (uint64_t)dpp0_64<0x142, 0xa>((int64_t)v);
  v += (uint64_t)dpp0_64<0x143, 0xc>((int64_t)v);
  return (uint64_t)rdl64((int64_t)v, 63);
}
__device__ __forceinline__ int wsum(int v) { return rdl(scan_i32(v), 63); }
__device__ __forceinline__ int64_t wsum64(int64_t v) { return rdl64(scan_i64(v), 63); }
__device__ __forceinline__ int64_t wmax64_nonneg(int64_t v) { return rdl64(scan_max_i64(v), 63); }

// ------------------------------------------------------------ record hash
// Checksum of a request record: the fields times fixed odd 64-bit constants,
// summed mod 2^64, then MurmurHash3's 64-bit finaliser.
__device__ __forceinline__ uint64_t fmix64(uint64_t k) {
  k ^= k >> 33;
  k *= 0xff51afd7ed558ccdULL;
  k ^= k >> 33;
  k *= 0xc4ceb9fe1a85ec53ULL;
  k ^= k >> 33;
  return k;
}
__device__ __forceinline__ uint64_t record_hash(int64_t idx, int64_t admit, int64_t first,
                                                int64_t finish, int64_t gap, int32_t npre,
                                                int32_t status) {
  uint64_t h = (uint64_t)idx * 0x9e3779b97f4a7c15ULL;
  h += (uint64_t)admit * 0xbf58476d1ce4e5b9ULL;
  h += (uint64_t)first * 0x94d049bb133111ebULL;
  h += (uint64_t)finish * 0xd6e8feb86659fd93ULL;
  h += (uint64_t)gap * 0xa0761d6478bd642fULL;
  h += (((uint64_t)(uint32_t)npre << 32) | (uint32_t)status) * 0xe7037ed1a0b428dbULL;
  return fmix64(h);
}

// ------------------------------------------------------------ roofline
// Lane j < 7 prices operator j of the iteration (QKV projection, prefill
// attention, decode attention, output projection, FFN up(+gate), FFN down,
// LM head): F = f * X, B = (b0 + b1 * Y) + b2 * Z with X, Y, Z batch sums.
// Every F and B is an integer below 2^53 and so is every partial product
// and sum, so fp64 evaluates them exactly: the same doubles as converting
// exact int64 counts.  Then t = max(F / peak, B / BW) with the reciprocals
// given in ns per FLOP / byte.  The layer sum keeps the fixed left-to-right
// order ((((t0 + t1) + t2) + t3) + t4) + t5 through a DPP chain in which
// lane k adds its term to lane k-1's partial sum.
__device__ __forceinline__ double dpp_shr1_f64(double v) {
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = (uint32_t)shr0<0x111>((int)(uint32_t)u);
  const uint32_t hi = (uint32_t)shr0<0x111>((int)(uint32_t)(u >> 32));
  return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}
// Row shift of a double (zero fill): CTRL 0x100 + k takes lane i + k,
// 0x110 + k lane i - k, within each 16-lane row.
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = (uint32_t)shr0<CTRL>((int)(uint32_t)u);
  const uint32_t hi = (uint32_t)shr0<CTRL>((int)(uint32_t)(u >> 32));
  return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}
__device__ __forceinline__ double rdl_f64(double v, int l) {
  return __builtin_bit_cast(double, (uint64_t)rdl64((int64_t)__builtin_bit_cast(uint64_t, v), l));
}

// This lane's operator coefficients (zero above lane 6), read from LDS on
// use rather than held in registers across the whole simulation.
// An LDS (address space 3) pointer: reads are ds_read, not flat loads.
typedef const volatile __attribute__((address_space(3))) double* LdsDoubles;
struct LaneRoof {
  LdsDoubles tab;  // [4][8]: f, b0, b1, b2 per operator lane
  int cl;                      // operator lane: min(lane, 7)
  bool is_attp, is_attd, is_lm;
  __device__ double f() const { return tab[cl]; }
  __device__ double b0() const { return tab[8 + cl]; }
  __device__ double b1() const { return tab[16 + cl]; }
  __device__ double b2() const { return tab[24 + cl]; }
};

// This lane's operator FLOPs F and bytes B for the batch sums (exact integers).
__device__ __forceinline__ void lane_work(const LaneRoof& c, int T, int TP, int64_t AP, int CP,
                                          int nD, int CD, int R, double* F, double* Bv) {
  // operands of this lane's operator, selected as integers, converted once
  int xi = c.is_attd ? CD : (c.is_lm ? R : T);
  int yi = c.is_attp ? CP : xi;
  int zi = c.is_attp ? TP : (c.is_attd ? nD : 0);
  const double X = c.is_attp ? (double)AP : (double)xi;
  const double Y = (double)yi;
  const double Z = (double)zi;
  const double b0 = (c.is_lm && R == 0) ? 0.0 : c.b0();  // no LM head without an emitter
  *F = c.f() * X;
  *Bv = (b0 + c.b1() * Y) + c.b2() * Z;
}

// Returns max(1, ceil(total)) and the same value as a double, where total is
// L * layer_sum + lm_head, and with swap transfers of xfer ns in the iteration
// (xfer > 0) total + xfer, or max(total, xfer) when they overlap the compute.
__device__ __forceinline__ int64_t iteration_ns(const LaneRoof& c, double n_layers, double iF,
                                                double iB, int T, int TP, int64_t AP, int CP,
                                                int nD, int CD, int R, double xfer,
                                                bool overlap, double* iter_d) {
  double F, Bv;
  lane_work(c, T, TP, AP, CP, nD, CD, R, &F, &Bv);
  const double tf = F * iF;
  const double tb = Bv * iB;
  const double t = __builtin_fmax(tf, tb);  // both finite and >= 0
  double s = t;
  s = dpp_shr1_f64(s) + t;  // lane 1: t0 + t1
  s = dpp_shr1_f64(s) + t;  // lane 2: (t0 + t1) + t2
  s = dpp_shr1_f64(s) + t;
  s = dpp_shr1_f64(s) + t;
  s = dpp_shr1_f64(s) + t;  // lane 5: the layer sum
  const double layer = rdl_f64(s, 5);
  const double lm = rdl_f64(t, 6);
  double total = n_layers * layer;
  total = total + lm;
  if (xfer > 0.0) total = overlap ? __builtin_fmax(total, xfer) : total + xfer;
  const double it = __builtin_fmax(ceil(total), 1.0);
  *iter_d = it;
  return (int64_t)it;
}

// ------------------------------------------------------------ slot state
// Running requests occupy slots in admission order.  Slot s lives in chunk
// s / 64, lane s % 64: chunk 0 in registers, chunks 1.. in LDS (only points
// with more than 64 running requests touch them).  Per slot, the hot state:
//   ctx   KV tokens resident          tgt  prefill target (prompt + decoded)
//   rem   decode iterations left      room free token slots in held blocks
//   fl    FL_FIRST: first token emitted; FL_STALE: the last token is older
//         than the previous iteration (set on re-admission after preemption);
//         FL_IDLE: swapped in this iteration, takes no part in it
//   q     tokens scheduled this iteration (prefill slots)
//   gap   largest interval between consecutive tokens so far
// Held blocks are (max(ctx, tgt) + room) / block and are never stored.
enum : int { FL_FIRST = 1, FL_STALE = 2, FL_IDLE = 4 };
// internal point status: the point is handed to a launch with more slots,
// which continues from the hand-over state, or starts it over
constexpr int kHandOver = -1;
constexpr int kHandOverRedo = -2;

struct Hot {
  int ctx, tgt, rem, room, fl, q;
  int64_t gap;
};

// Admission staging: one entry per admitted candidate of a window (its
// request index and preemption count go straight to their slot).
struct StageSlot {
  int32_t tgt, rem, fl, q, room, ctx;
  int64_t gap;
};

template <int NCH>
struct SlotLds {
  static constexpr int NX = NCH > 1 ? NCH - 1 : 1;  // LDS chunks (storage for one when unused)
  int32_t x_ctx[NX * 64], x_tgt[NX * 64], x_rem[NX * 64], x_room[NX * 64], x_q[NX * 64];
  int64_t x_gap[NX * 64];
  int32_t id[NCH * 64];    // request index per slot
  int32_t npre[NCH * 64];  // times preempted per slot
  uint8_t x_fl[NX * 64];   // flags fit a byte: with the staging below, 256 slots
                           // take at most 10 KiB, so 16 workgroups share a CU
  unsigned int sub_cnt[kMaxDev];  // prefill device: requests handed to each decode device
  // steady segment: the two attention operators' FLOPs, bytes and their
  // per-iteration steps at the segment start, then the other operators' times
  double segk[13];
  union {
    StageSlot stage[64];
    int64_t scratch[NCH * 64];
  } u;
};

template <int NCH>
__device__ __forceinline__ Hot load_chunk(const SlotLds<NCH>& L, const Hot& h0, int j, int lane) {
  if (j == 0) return h0;
  const int e = (j - 1) * 64 + lane;
  Hot h;
  h.ctx = L.x_ctx[e]; h.tgt = L.x_tgt[e]; h.rem = L.x_rem[e]; h.room = L.x_room[e];
  h.fl = L.x_fl[e]; h.q = L.x_q[e]; h.gap = L.x_gap[e];
  return h;
}
template <int NCH>
__device__ __forceinline__ void store_chunk(SlotLds<NCH>& L, Hot& h0, int j, int lane,
                                            const Hot& h) {
  if (j == 0) { h0 = h; return; }
  const int e = (j - 1) * 64 + lane;
  L.x_ctx[e] = h.ctx; L.x_tgt[e] = h.tgt; L.x_rem[e] = h.rem; L.x_room[e] = h.room;
  L.x_fl[e] = h.fl; L.x_q[e] = h.q; L.x_gap[e] = h.gap;
}

// ------------------------------------------------------------ one point
// MODE: kStageOne (a one-worker design point), kStagePrefill (a prefill
// device of a disaggregated point: requests leave when their prefill
// completes and their KV crosses the device's link) or kStageDecode (a
// decode device: requests arrive with their prompt's KV and first token).
// Returns -1 when the point is done, else (a narrow launch taking wider
// points, and the point needs more slots than this kernel holds) the bucket
// of its remaining work, 0 .. kHandBuckets - 1 by the share of its requests
// not finished: its state at the start of the iteration that needed the
// slots goes to its hand-over record, and a wider launch continues from
// there (or starts it over when the record says so).
template <int NCH, int MODE, bool SIMPLE>
__device__ __forceinline__ int simulate_point(const SimArgs& A, const int pidx,
                                               SlotLds<NCH>& L, QEntry* Q,
                                               const int lane, const LaneRoof& roofc,
                                               const bool resumed) {
  const DevPoint P = A.points[pidx];
  const TraceRec* __restrict__ rec = A.recs + P.trace_off;
  const int N = P.n, NB = P.num_blocks, B = P.block, M = P.max_batch, K = P.chunk;
  const bool unlimited = (K == 0);
  // SIMPLE: a one-worker point under continuous batching with recompute
  // preemption, no admission ratio, no request that could never fit and no
  // watchdog (the policy state folds away at compile time)
  static_assert(!SIMPLE || MODE == kStageOne, "simple points are one-worker points");
  const int64_t cap_tok = P.cap_tokens, cap_prompt = SIMPLE ? P.cap_tokens : P.cap_prompt;
  const int policy = SIMPLE ? TS_POLICY_MIXED : P.policy;
  const int adm_reserve = SIMPLE ? 0 : P.adm_reserve;
  const bool pff = policy == TS_POLICY_PREFILL_FIRST;
  const bool swap = SIMPLE ? false : P.swap != 0;  // preemption by swap instead of recompute
  const uint64_t time_limit = SIMPLE ? 0 : A.time_limit_ticks;
  const bool may_reject = SIMPLE ? false : P.may_reject != 0;  // some request never fits
  // a request that could never fit, alone or within the admission ratio (on
  // a prefill device: its prompt here, or the whole request on a decode device)
  auto rejected = [&](int32_t pr, int32_t ou) {
    if constexpr (MODE == kStagePrefill)
      return (int64_t)pr > cap_tok || (int64_t)pr + (int64_t)ou > P.cap_po2 ||
             (int64_t)pr > cap_prompt;
    else
      return (int64_t)pr + (int64_t)ou > cap_tok || (int64_t)pr > cap_prompt;
  };
  // the disaggregated point a device belongs to
  PdAux* X = nullptr;
  int n_pd = 1, nd_pd = 1, req_base = 0;
  int64_t kv_bpt = 0, link_free = 0;
  double inv_kv_link = 0.0;
  if constexpr (MODE != kStageOne) {
    X = A.pd + P.pd;
    n_pd = X->n_p;
    nd_pd = X->n_d;
    req_base = X->req_base;
    kv_bpt = X->kv_bpt;
    inv_kv_link = X->inv_link_ns;
  }
  // a request's index in the point's trace from its index in this unit's trace
  auto gid_of = [&](int local) -> int {
    if constexpr (MODE == kStagePrefill) return P.unit + local * n_pd;
    else if constexpr (MODE == kStageDecode) return A.gids[P.trace_off + local];
    else return local;
  };
  const double iF = P.inv_flops_ns, iB = P.inv_bw_ns;
  const int oi = P.out_index;
  const int orow = MODE == kStageOne ? oi : P.out_point;  // the design point's row
  // the design point's request records: every request's record is written
  // once, when it finishes, is rejected, or is left unfinished by an early stop
  ts_req_result* RR = A.rec + (size_t)orow * (size_t)A.max_n;

  L.sub_cnt[lane & (kMaxDev - 1)] = 0;
  __syncthreads();
  int n_rej = 0;

  // Requests that could never fit are rejected up front.
  if (may_reject) {
    for (int base = 0; base < N; base += 64) {
      const int i = base + lane;
      bool rj = false;
      if (i < N) {
        const TraceRec r = rec[i];
        rj = rejected(r.prompt, r.output);
      }
      if (rj) {
        ts_req_result o;
        o.admit_ns = -1; o.first_token_ns = -1; o.finish_ns = -1; o.max_gap_ns = 0;
        o.n_preempt = 0; o.status = TS_REQ_REJECTED;
        RR[gid_of(i)] = o;
      }
      n_rej += popc(ballot(rj));
    }
  }

  int status = (NB == 0) ? TS_POINT_NO_KV : TS_POINT_OK;
  int64_t t = 0;
  int freeb = NB, nrun = 0, npre = 0, qhead = 0;
  int next = 0, next_new = 0, nwait = 0, wbase = 0;
  int head_need = -1;  // block need of the waiting head when known, else -1
  int64_t n_iters = 0, n_pre_tot = 0, pf_tok = 0, dec_tok = 0;
  int peak = 0, n_done = 0;
  double ubns = 0.0;

  // arrival window: lane l holds record wbase + l
  int64_t w_arr = INT64_MAX;
  int w_rj = 0;  // 1: the record is rejected
  if (lane < N) {
    const TraceRec r = rec[lane];
    w_arr = r.arrival_ns; w_rj = rejected(r.prompt, r.output) ? 1 : 0;
  }

  Hot h0;  // chunk 0 in registers
  h0.ctx = h0.tgt = h0.rem = h0.room = h0.fl = h0.q = 0;
  h0.gap = 0;

  // A launch taking points handed over by a narrower one continues each
  // from its hand-over state: the start of the general-path iteration whose
  // admissions needed more slots (or starts it over when there is none).
  // n_it0: the iterations the narrower launches counted as theirs.
  int64_t n_it0 = 0;
  if constexpr (SIMPLE && NCH > 1) {
    if (resumed) {
      const unsigned char* base = A.resume + (size_t)P.resume * kResumeBytes;
      const ResumeHead* hp = reinterpret_cast<const ResumeHead*>(base);
      auto u64 = [](int64_t v) -> int64_t {
        const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)v);
        const uint32_t hi =
            (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)((uint64_t)v >> 32));
        return (int64_t)(((uint64_t)hi << 32) | lo);
      };
      auto u32 = [](int v) -> int { return __builtin_amdgcn_readfirstlane(v); };
      n_it0 = u64(hp->counted);
      if (u32(hp->valid) != 0) {
        t = u64(hp->t);
        n_iters = u64(hp->n_iters);
        n_pre_tot = u64(hp->n_pre_tot);
        pf_tok = u64(hp->pf_tok);
        dec_tok = u64(hp->dec_tok);
        ubns = __builtin_bit_cast(double, u64(__builtin_bit_cast(int64_t, hp->ubns)));
        freeb = u32(hp->freeb);
        nrun = u32(hp->nrun);
        npre = u32(hp->npre);
        next = u32(hp->next);
        next_new = u32(hp->next_new);
        nwait = u32(hp->nwait);
        wbase = u32(hp->wbase);
        head_need = u32(hp->head_need);
        peak = u32(hp->peak);
        n_done = u32(hp->n_done);
        const ResumeSlot* rs = reinterpret_cast<const ResumeSlot*>(base + kResumeHead);
#pragma unroll
        for (int j = 0; j < NCH; ++j) {
          const int sl = j * 64 + lane;
          if (sl < nrun) {
            const ResumeSlot o = rs[sl];
            Hot h;
            h.ctx = o.ctx; h.tgt = o.tgt; h.rem = o.rem; h.room = o.room; h.fl = o.fl;
            h.q = o.q; h.gap = o.gap;
            store_chunk<NCH>(L, h0, j, lane, h);
            L.id[sl] = o.id;
            L.npre[sl] = o.npre;
          }
        }
        const QEntry* rq = reinterpret_cast<const QEntry*>(base + kResumeHead +
                                                           kResumeSlots * sizeof(ResumeSlot));
        for (int i = lane; i < npre; i += 64) Q[i] = rq[i];
        qhead = 0;
        w_arr = INT64_MAX;
        w_rj = 0;
        if (wbase + lane < N) {
          const TraceRec r = rec[wbase + lane];
          w_arr = r.arrival_ns;
          w_rj = rejected(r.prompt, r.output) ? 1 : 0;
        }
        __syncthreads();
      }
    }
  }

  // intake: every request with arrival <= t joins the waiting set
  auto intake = [&]() {
    int guard = N / 64 + 2;  // window passes are bounded by the trace length
    while (next < N && --guard >= 0) {
      const uint64_t m = ballot(w_arr <= t);  // arrivals are sorted: a lane prefix
      const int cnt = popc(m);
      const int nn = wbase + cnt;
      if (nn > next) {
        int add = nn - next;
        if (may_reject) {
          const bool rj = lane >= next - wbase && lane < cnt && w_rj != 0;
          add -= popc(ballot(rj));
        }
        if (npre == 0 && nwait == 0) head_need = -1;
        nwait += add;
        next = nn;
      }
      if (cnt == 64 && nn < N) {
        wbase = nn;
        w_arr = INT64_MAX;
        w_rj = 0;
        if (wbase + lane < N) {
          const TraceRec r = rec[wbase + lane];
          w_arr = r.arrival_ns; w_rj = rejected(r.prompt, r.output) ? 1 : 0;
        }
        continue;
      }
      break;
    }
    if (nwait == 0) next_new = next;
  };

  // x / B; block sizes are usually powers of two
  const int lgB = (B & (B - 1)) == 0 ? 31 - __builtin_clz((unsigned)B) : -1;
  auto divB = [&](int x) { return lgB >= 0 ? x >> lgB : x / B; };

  // A request finishing at t_end (lanes with fin): the rest of its record
  // (its admission and first token are there already).  The point's latency
  // sums, SLO counts, percentiles and digest are computed from the records
  // after the simulation.
  auto record_done = [&](bool fin, int s, int64_t t_end, int64_t gap) {
    if (fin) {
      ts_req_result& o = RR[gid_of(L.id[s])];
      o.finish_ns = t_end;
      o.max_gap_ns = gap;
      o.n_preempt = L.npre[s];
      o.status = TS_REQ_DONE;
    }
  };

  // Remove the slots whose rem is 0, keeping the others in slot order.
  auto compact = [&](int nfin) {
    const int nsurv = nrun - nfin;
    if (nrun <= 64) {
      // One chunk: every lane pushes its slot through the LDS crossbar to
      // its new lane, survivors first in slot order, then the others.
      const bool keep = lane < nrun && h0.rem > 0;
      const uint64_t km = ballot(keep);
      const int ad = (keep ? rank_below(km) : nsurv + rank_below(~km)) << 2;
      h0.ctx = __builtin_amdgcn_ds_permute(ad, h0.ctx);
      h0.tgt = __builtin_amdgcn_ds_permute(ad, h0.tgt);
      h0.rem = __builtin_amdgcn_ds_permute(ad, h0.rem);
      h0.room = __builtin_amdgcn_ds_permute(ad, h0.room);
      h0.fl = __builtin_amdgcn_ds_permute(ad, h0.fl);
      const uint32_t glo = (uint32_t)__builtin_amdgcn_ds_permute(ad, (int)(uint32_t)h0.gap);
      const uint32_t ghi =
          (uint32_t)__builtin_amdgcn_ds_permute(ad, (int)(uint32_t)((uint64_t)h0.gap >> 32));
      h0.gap = (int64_t)(((uint64_t)ghi << 32) | glo);
      const int idv = __builtin_amdgcn_ds_permute(ad, L.id[lane]);
      const int npv = __builtin_amdgcn_ds_permute(ad, L.npre[lane]);
      L.id[lane] = idv;
      L.npre[lane] = npv;
    } else {
      // Stable compaction of the survivors through LDS scratch, one field at
      // a time.  Finished slots have rem == 0; rem moves last so every pass
      // reads 'keep' from the original slots.
      const int nch = ((nrun + 63) >> 6) < NCH ? ((nrun + 63) >> 6) : NCH;
      const int nch2 = (nsurv + 63) >> 6;
      int32_t* s32 = reinterpret_cast<int32_t*>(L.u.scratch);
#pragma nounroll
      for (int f = 0; f < 8; ++f) {
        int carry = 0;
#pragma nounroll
        for (int j = 0; j < nch; ++j) {
          const int s = j * 64 + lane;
          const int e = (j - 1) * 64 + lane;
          const int rem = j == 0 ? h0.rem : L.x_rem[e];
          const bool keep = s < nrun && rem > 0;
          const uint64_t km = ballot(keep);
          const int pos = carry + rank_below(km);
          carry += popc(km);
          if (keep) {
            switch (f) {
              case 0: s32[pos] = j == 0 ? h0.ctx : L.x_ctx[e]; break;
              case 1: s32[pos] = j == 0 ? h0.tgt : L.x_tgt[e]; break;
              case 2: s32[pos] = j == 0 ? h0.room : L.x_room[e]; break;
              case 3: s32[pos] = j == 0 ? h0.fl : L.x_fl[e]; break;
              case 4: s32[pos] = L.id[s]; break;
              case 5: L.u.scratch[pos] = j == 0 ? h0.gap : L.x_gap[e]; break;
              case 6: s32[pos] = L.npre[s]; break;
              default: s32[pos] = rem; break;
            }
          }
        }
        __syncthreads();
#pragma nounroll
        for (int j = 0; j < nch2; ++j) {
          const int s = j * 64 + lane;
          const int e = (j - 1) * 64 + lane;
          switch (f) {
            case 0: if (j == 0) h0.ctx = s32[s]; else L.x_ctx[e] = s32[s]; break;
            case 1: if (j == 0) h0.tgt = s32[s]; else L.x_tgt[e] = s32[s]; break;
            case 2: if (j == 0) h0.room = s32[s]; else L.x_room[e] = s32[s]; break;
            case 3: if (j == 0) h0.fl = s32[s]; else L.x_fl[e] = s32[s]; break;
            case 4: L.id[s] = s32[s]; break;
            case 5: if (j == 0) h0.gap = L.u.scratch[s]; else L.x_gap[e] = L.u.scratch[s]; break;
            case 6: L.npre[s] = s32[s]; break;
            default: if (j == 0) h0.rem = s32[s]; else L.x_rem[e] = s32[s]; break;
          }
        }
        __syncthreads();
      }
    }
    nrun = nsurv;
  };

  // A prefill device hands the requests of chunk j whose prefill completed
  // at t_end (lanes in pm) to their decode devices, in slot order: each KV
  // transfer starts when the device's link is free and takes
  // ceil(prompt * KV bytes per token * ns per byte).
  auto hand_over = [&](uint64_t pm, int j, int tgt_lane, int64_t t_end) {
    while (pm != 0) {
      const int l = (int)__builtin_ctzll(pm);
      pm &= pm - 1;
      const int id_l = __builtin_amdgcn_readfirstlane(L.id[j * 64 + l]);
      const int p_l = rdl(tgt_lane, l);
      const int g = P.unit + id_l * n_pd;
      const int64_t x =
          inv_kv_link == 0.0 ? 0 : (int64_t)ceil((double)((int64_t)p_l * kv_bpt) * inv_kv_link);
      link_free = (t_end > link_free ? t_end : link_free) + x;
      const int v = g % nd_pd;
      const int c = __builtin_amdgcn_readfirstlane((int)L.sub_cnt[v]);
      L.sub_cnt[v] = (unsigned int)(c + 1);  // every lane stores the same value
      const int pos = X->sub_off[P.unit * kMaxDev + v] + c;
      const int64_t adm = RR[g].admit_ns;
      if (lane == 0) {
        A.sub_a2[pos] = link_free;
        A.sub_gid[pos] = g;
        A.s1_first[req_base + g] = t_end;
        A.s1_admit[req_base + g] = adm;
      }
    }
  };

  const uint64_t clock0 = time_limit ? __builtin_amdgcn_s_memrealtime() : 0;
  while (status == TS_POINT_OK) {
    // ---- 0. steady stretch.  As long as no request is admitted or
    // preempted and no prefill completes, an iteration advances every decode
    // by one token and the head prefill by the whole remaining chunk budget,
    // so every batch sum moves by a fixed integer per iteration.  Such
    // iterations keep the decodes' slot state lazily (materialised when the
    // stretch ends: tokens and the per-request gap by the iteration count,
    // block boundaries by a countdown per slot) and step the two attention
    // operators' FLOPs and bytes by exact integer increments; the other
    // operators' times are constant.  Within a stretch:
    //   * decodes that finish are recorded in place and leave holes, removed
    //     when the stretch ends;
    //   * when the head prefill completes (its first one), it joins the
    //     decodes, and the rest of the chunk budget may admit the next trace
    //     request as the new head prefill, if that one does not complete in
    //     the same iteration;
    // after either event the sums are re-derived for the next segment.  The
    // iteration that ends a segment (first finish, head prefill completion,
    // iteration cap) is known when it starts.  The clock runs in fp64,
    // exact below 2^53.  A decode joining at iteration g is stored shifted
    // by g (tokens - g, remaining + g, room + g), so one iteration count
    // advances every decode alike.  Decodes hold slots [0, nD) and prefills
    // the slots after them: prefills receive tokens in slot order, so they
    // complete in slot order.
    if (nrun > 0) {
      const int nch0 = ((nrun + 63) >> 6) < NCH ? ((nrun + 63) >> 6) : NCH;
      int nD = 0;
      bool go = true;
      // alive decode slots: room + B * (blocks taken in this stretch), >= 0;
      // every other lane (prefills, unused, finished) holds a negative value
      int rr[NCH];
      bool short_chunk = false;  // a chunk before this one holds a non-decode slot
#pragma unroll
      for (int j = 0; j < NCH; ++j) {
        rr[j] = -0x40000000;
        if (j < nch0) {
          const Hot h = load_chunk<NCH>(L, h0, j, lane);
          const bool dec = (j * 64 + lane) < nrun && h.ctx >= h.tgt;
          const uint64_t dm = ballot(dec);
          nD += popc(dm);
          if (ballot(dec && ((h.fl & FL_STALE) != 0 || h.rem == 1)) != 0) go = false;
          if (swap || MODE == kStageDecode) {
            // a request swapped in behind a prefill can finish its prefill
            // later than a newer one, and a decode device admits decodes
            // behind re-prefills: the decodes may not form a slot prefix
            if ((dm & (dm + 1)) != 0 || (short_chunk && dm != 0)) go = false;
            short_chunk = short_chunk || dm != ~0ull;
          }
          rr[j] = dec ? h.room : -0x40000000;
        }
      }
      int npf = nrun - nD;
      if (npf > 0 && unlimited) go = false;
      int ctx_p = 0, tgt_p = 0, fl_p = 0;  // the head prefill (slot nD)
      if (go && npf > 0) {
        const int jp = nD >> 6, lp = nD & 63;
        if (NCH == 1 || jp == 0) {
          ctx_p = rdl(h0.ctx, lp);
          tgt_p = rdl(h0.tgt, lp);
          fl_p = rdl(h0.fl, lp);
        } else {
          ctx_p = __builtin_amdgcn_readfirstlane(L.x_ctx[(jp - 1) * 64 + lp]);
          tgt_p = __builtin_amdgcn_readfirstlane(L.x_tgt[(jp - 1) * 64 + lp]);
          fl_p = __builtin_amdgcn_readfirstlane(L.x_fl[(jp - 1) * 64 + lp]);
        }
        // the head prefill completes now: the general path, except for a
        // simple point's fresh head, which the stretch's first (completing)
        // iteration handles in place
        if (tgt_p - ctx_p <= K - nD && (!SIMPLE || (fl_p & (FL_FIRST | FL_STALE)) != 0))
          go = false;
      }
      constexpr int64_t kT52 = (int64_t)1 << 52;
      if (n_iters >= A.iter_cap || t >= kT52) go = false;
      if (time_limit != 0 && (n_iters & 255) == 0) go = false;  // watchdog below
      int nchd = (nD + 63) >> 6;
      int nDa = nD, nruna = nrun;  // alive decodes and running requests
      // an admission would find a free slot and token budget (a swapped
      // request needs no budget)
      auto adm_open = [&]() {
        return policy != TS_POLICY_STATIC && nruna < M &&
               (unlimited || (npf == 0 && K - nDa > 0) || (swap && npre > 0));
      };
      // the waiting head is known not to fit in fb free blocks (a first
      // admission also leaves the admission-ratio reserve)
      auto head_blocked = [&](int fb) {
        return head_need >= 0 && head_need > fb - (npre > 0 ? 0 : adm_reserve);
      };
      int nneed = 0;
      if (go) {
        if (next < N && rdl64(w_arr, next - wbase) <= t) intake();
#pragma unroll
        for (int j = 0; j < NCH; ++j)
          if (j < nchd) nneed += popc(ballot(rr[j] == 0));
        if (nneed > freeb) go = false;  // recompute preemption
        else if ((npre > 0 || nwait > 0) && adm_open() &&
                 !head_blocked(pff ? freeb : freeb - nneed))
          go = false;  // an admission may happen
      }
      if (go) {
        // iterations (counted from the stretch start) that must run elsewhere:
        // the iteration cap and the watchdog's clock checks
        int stop_fix = 0x3fffffff;
        if (A.iter_cap - n_iters < (int64_t)stop_fix) stop_fix = (int)(A.iter_cap - n_iters);
        if (time_limit != 0) {
          const int wd = 256 - (int)(n_iters & 255);
          stop_fix = wd < stop_fix ? wd : stop_fix;
        }
        // every iteration is below 2^lg_iter ns: this many from the stretch
        // start keep the fp64 clock below 2^52
        int stop_hard = stop_fix;
        {
          const int64_t ks = (kT52 - t) >> P.lg_iter;
          if (ks < (int64_t)stop_fix) stop_hard = ks > 0 ? (int)ks : 0;
        }
        int dG = 0, seg0 = 0, q = 0, fin_at = 0, stop = 0, cd_seg = 0;
        bool watch = false;
        const double kT52d = 4503599627370496.0;
        double thr = next < N ? __builtin_fmin((double)rdl64(w_arr, next - wbase), kT52d) : kT52d;
        // the clock (fp64, exact below 2^53), this lane's share of the
        // stretch's used-block integral, the last and the largest iteration
        double t_d = (double)t, ubl = 0.0, it = 0.0, em = 0.0;
        // Segment set-up at iteration dG: the alive decodes' first finishing
        // iteration and key sum, the head prefill's chunk, every operator's
        // work and its per-iteration step, and the segment's last iteration.
        // segk[8..11] hold the times of the operators that depend on T only
        // at T = K (the last full set-up had a head prefill running)
        bool tk_ok = false;
        // the segment runs as blocks through finishes (64 or 128 slots,
        // simple points: one worker, continuous batching with recompute
        // preemption; a head prefill running with a token budget left)
        auto through_fin = [&]() {
          return SIMPLE && NCH <= 2 && npf == 1 && q > 0;
        };
        auto setup = [&]() {
          // per lane over the chunks first, then one reduction each
          int mxl = 0, csl = 0;
#pragma unroll
          for (int j = 0; j < NCH; ++j) {
            if (j < nchd) {
              const int e = (j - 1) * 64 + lane;
              const int rem0 = j == 0 ? h0.rem : L.x_rem[e];
              const int ctx0 = j == 0 ? h0.ctx : L.x_ctx[e];
              const bool al = rr[j] >= 0;
              const int m = al ? 0x7fffffff - rem0 : 0;
              mxl = m > mxl ? m : mxl;
              csl += al ? ctx0 + 1 : 0;
            }
          }
          const int cs = wsum(csl);
          cd_seg = cs + nDa * dG;
          q = npf > 0 ? K - nDa : 0;
          // the first finishing iteration; blocks through finishes need it
          // only for a head prefill completing at once
          auto first_finish = [&]() {
            const int mx = rdl(scan_max_i32(mxl), 63);
            fin_at = nDa > 0 ? 0x7fffffff - mx - 1 : 0x3fffffff;
          };
          const bool tf = through_fin();
          if (!tf) first_finish();
          // A segment of blocks through finishes prices every operator but
          // the four that depend on T only, whose times it takes from a
          // set-up with a head prefill running (T = K in all of them).
          if (!(tf && tk_ok)) {
            const int64_t AP0 = (int64_t)q * ctx_p + ((int64_t)q * (q + 1)) / 2;
            double Fw, Bw;
            lane_work(roofc, nDa + q, q, AP0, q > 0 ? ctx_p + q : 0, nDa, cd_seg, nDa, &Fw, &Bw);
            const double dX = roofc.is_attp ? (double)((int64_t)q * q)
                                            : (roofc.is_attd ? (double)nDa : 0.0);
            const double dY = roofc.is_attp ? (double)q : (roofc.is_attd ? (double)nDa : 0.0);
            // the segment's constants in LDS, where every iteration reads
            // them: the attention operators' FLOPs and bytes at the segment
            // start and their steps per iteration (lanes 1, 2), then the other
            // operators' times (lanes 0, 3, 4, 5, 6)
            if (lane == 1 || lane == 2) {
              double* k = &L.segk[(lane - 1) * 4];
              k[0] = Fw;
              k[1] = Bw;
              k[2] = roofc.f() * dX;
              k[3] = roofc.b1() * dY;
            } else if (lane < 7) {
              L.segk[lane == 0 ? 8 : lane + 6] = __builtin_fmax(Fw * iF, Bw * iB);
            }
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
            __builtin_amdgcn_wave_barrier();
            tk_ok = npf > 0;  // T = nDa + (K - nDa)
          }
          stop = stop_hard;
          if (q > 0) {  // the head prefill completes in iteration kc
            // floor(n / q) for 0 <= n < 2^21 and 1 <= q <= 2^20 (a target
            // below 2^21 tokens, a budget of at most 2^20): n times the fp32
            // reciprocal of q (relative error below 2^-22) is within 1/2 of
            // n / q, so its truncation is off by at most one, corrected by
            // the remainder
            const int n = tgt_p - ctx_p - 1;
            int kq = (int)((float)n * __builtin_amdgcn_rcpf((float)q));
            const int rm = n - kq * q;
            kq = rm < 0 ? kq - 1 : (rm >= q ? kq + 1 : kq);
            const int kc = dG + kq;
            stop = kc < stop ? kc : stop;
          }
          if (tf && stop == dG) first_finish();
          // arrivals matter within the segment only if one could be admitted
          watch = adm_open() && npre == 0 && nwait == 0;
          seg0 = dG;
        };
        // a segment's token bookkeeping, through iteration dG - 1
        auto close_segment = [&]() {
          const int len = dG - seg0;
          pf_tok += (int64_t)q * len;
          dec_tok += (int64_t)nDa * len;
          ctx_p += q * len;
          if (NB - freeb > peak) peak = NB - freeb;
          seg0 = dG;
        };
        setup();
        // the checks before iteration dG: arrivals, then block boundaries;
        // false ends the stretch
        auto next_ok = [&]() -> bool {
          if (watch && (ballot(t_d >= thr) & 2ull) != 0) {
            t = (int64_t)rdl_f64(t_d, 1);
            if (t >= kT52) return false;
            intake();
            thr = next < N ? __builtin_fmin((double)rdl64(w_arr, next - wbase), kT52d) : kT52d;
            if ((npre > 0 || nwait > 0) && adm_open() && head_need < 0) return false;  // a new head
          }
          nneed = 0;
#pragma unroll
          for (int j = 0; j < NCH; ++j)
            if (j < nchd) nneed += popc(ballot(rr[j] == dG));
          return nneed <= freeb;
        };
        // An iteration whose FCFS admissions may run in place: only trace
        // requests wait (none preempted), no prefill runs, a chunked budget,
        // continuous batching on one worker.  It is priced like a head
        // prefill's completion, with no head.
        bool adm_next = false;
        auto adm_here = [&]() {
          return NCH > 1 && MODE == kStageOne && !unlimited && npf == 0 && npre == 0 &&
                 policy != TS_POLICY_STATIC && dG < stop_hard;
        };
        bool more = true;
        while (more) {
          // steady iterations up to the segment's last
          while (dG != stop) {
            if constexpr (SIMPLE && NCH <= 2) {
              if (through_fin()) {
                // A head prefill runs with the budget the decodes leave
                // (T = K): a block of up to 64 iterations, lane i pricing
                // iteration dG + i, runs through the decodes that finish in
                // it.  A decode finishing at iteration e takes part in e,
                // frees its blocks and budget from e + 1 on (the head's
                // chunk grows by one), and writes its record with e's end.
                // Per iteration, from prefix sums over the finishes before
                // it: alive decodes nD_i, their key sum CD_i, the head's
                // chunk q_i = K - nD_i and context ctx_i, the blocks freed;
                // the four operators that depend on T only keep their
                // segment times.  The block ends before the head prefill's
                // completing iteration, before the first iteration short of
                // blocks, and after the first whose end reaches an arrival
                // that matters.
                const int g0 = dG;
                const int cs0 = cd_seg - nDa * seg0;  // sum of ctx0 + 1 over the alive decodes
                close_segment();                      // the segment through g0 - 1
                const int W = stop - g0 < 64 ? stop - g0 : 64;
                int* hb = reinterpret_cast<int*>(&L.u);  // [4][64]: blocks taken, finishes,
                hb[lane] = 0;                            // their keys, blocks they free
                hb[64 + lane] = 0;
                hb[128 + lane] = 0;
                hb[192 + lane] = 0;
                __syncthreads();
                // per slot: its finishing iteration in the block (W: none)
                int osj[NCH];
#pragma unroll
                for (int j = 0; j < NCH; ++j) {
                  osj[j] = W;
                  if (j < nchd) {
                    const int e = (j - 1) * 64 + lane;
                    const int rem0 = j == 0 ? h0.rem : L.x_rem[e];
                    const int ctx0 = j == 0 ? h0.ctx : L.x_ctx[e];
                    const int rrj = rr[j];
                    const bool al = rrj >= 0;
                    const int os = rem0 - 1 - g0;  // the decode's finishing iteration
                    const bool fin_in = al && os >= 0 && os < W;
                    const int ob = rrj - g0;       // its next block boundary (>= 0)
                    if (al && ob >= 0) {
                      const int lim = fin_in ? os + 1 : W;  // boundaries through its finish
                      for (int pz = ob; pz < lim; pz += B) atomicAdd(&hb[pz], 1);
                    }
                    if (fin_in) {
                      const int nb = ob <= os ? divB(os - ob) + 1 : 0;  // blocks taken through it
                      atomicAdd(&hb[64 + os], 1);
                      atomicAdd(&hb[128 + os], ctx0 + 1);
                      atomicAdd(&hb[192 + os], divB(ctx0 + rrj + B * nb));
                      osj[j] = os;
                    }
                  }
                }
                __syncthreads();
                const bool in = lane < W;
                const int T = scan_i32(in ? hb[lane] : 0);  // blocks taken through i
                const int hf = in ? hb[64 + lane] : 0;
                const int Fi = scan_i32(hf);                // finished through i
                const int Fx = Fi - hf;                     // finished before i
                const int hk = in ? hb[128 + lane] : 0;
                const int KFi = scan_i32(hk);
                const int KFx = KFi - hk;
                const int hr = in ? hb[192 + lane] : 0;
                const int FBi = scan_i32(hr);               // blocks freed through i
                const int FBx = FBi - hr;
                const int SFi = scan_i32(Fx);               // sum of Fx through i
                const int nDi = nDa - Fx;
                const int qi = q + Fx;
                const int ctxi = ctx_p + lane * q + (SFi - Fx);
                const int CDi = (cs0 - KFx) + nDi * (g0 + lane);
                const LdsDoubles cf = roofc.tab;  // f, b0, b1, b2 per operator
                const int64_t APi = (int64_t)qi * ctxi + ((int64_t)qi * (qi + 1)) / 2;
                const double F1 = cf[1] * (double)APi;
                const double B1 = (cf[9] + cf[17] * (double)(ctxi + qi)) + cf[25] * (double)qi;
                const double F2 = cf[2] * (double)CDi;
                const double B2 = (cf[10] + cf[18] * (double)CDi) + cf[26] * (double)nDi;
                const double F6 = cf[6] * (double)nDi;
                const double B6 = ((nDi == 0 ? 0.0 : cf[14]) + cf[22] * (double)nDi) + cf[30] * 0.0;
                const double t1 = __builtin_fmax(F1 * iF, B1 * iB);
                const double t2 = __builtin_fmax(F2 * iF, B2 * iB);
                const double t6 = __builtin_fmax(F6 * iF, B6 * iB);
                double lay = L.segk[8] + t1;
                lay = lay + t2;
                lay = lay + L.segk[9];
                lay = lay + L.segk[10];
                lay = lay + L.segk[11];
                double tot = A.n_layers * lay;
                tot = tot + t6;
                const double itv = __builtin_fmax(ceil(tot), 1.0);
                const double tend = rdl_f64(t_d, 1) + scan_f64(in ? itv : 0.0);
                const uint64_t short_m = ballot(in && T > freeb + FBx);
                const uint64_t arr_m = watch ? ballot(in && tend >= thr) : 0ull;
                const uint64_t comp_m = ballot(in && ctxi + qi >= tgt_p);
                int Kb = W;
                if (short_m != 0) {
                  const int k = (int)__builtin_ctzll(short_m);
                  Kb = k < Kb ? k : Kb;
                }
                if (arr_m != 0) {
                  const int k = (int)__builtin_ctzll(arr_m) + 1;
                  Kb = k < Kb ? k : Kb;
                }
                const int kcomp = comp_m != 0 ? (int)__builtin_ctzll(comp_m) : 64;
                Kb = kcomp < Kb ? kcomp : Kb;
                if (Kb > 0) {
                  const int last = Kb - 1;
                  // used blocks during each iteration (after its reservations,
                  // before its frees): the integral and the peak
                  const int used = NB - freeb + T - FBx;
                  ubl = ubl + (lane < Kb ? (double)used * itv : 0.0);
                  // (with no finish in the block the used blocks and the
                  // iteration times only grow: the last ones are the largest)
                  const int nfin = rdl(Fi, last);
                  const int upk = nfin > 0 ? rdl(scan_max_i32(lane < Kb ? used : 0), 63)
                                           : rdl(used, last);
                  peak = upk > peak ? upk : peak;
                  // the decodes finishing here: end of their iteration, and
                  // the largest iteration time through it since the last fold
                  const int64_t tl = (int64_t)tend;
                  const int64_t pm = nfin > 0 ? scan_max_i64(in ? (int64_t)itv : 0) : 0;
                  const int64_t em0 = (int64_t)rdl_f64(em, 1);
                  auto lane64 = [](int src, int64_t v) {  // v of lane src / 4
                    return (int64_t)(((uint64_t)(uint32_t)__builtin_amdgcn_ds_bpermute(
                                          src, (int)((uint64_t)v >> 32)) << 32) |
                                     (uint32_t)__builtin_amdgcn_ds_bpermute(src, (int)v));
                  };
#pragma unroll
                  for (int j = 0; j < NCH; ++j) {
                    if (j < nchd) {
                      const int e = (j - 1) * 64 + lane;
                      const int os = osj[j];
                      const bool fin = os <= last;
                      if (ballot(fin) != 0) {
                        const int src = (fin ? os : lane) << 2;
                        const int64_t t_fin = lane64(src, tl);
                        const int64_t pm_fin = lane64(src, pm);
                        const int64_t gx = pm_fin > em0 ? pm_fin : em0;
                        const int64_t gap0 = j == 0 ? h0.gap : L.x_gap[e];
                        record_done(fin, j * 64 + lane, t_fin, gx > gap0 ? gx : gap0);
                      }
                      const int rrj = rr[j];
                      const int ob = rrj - g0;
                      if (rrj >= 0 && !fin && ob >= 0 && ob < Kb) rr[j] = rrj + B * (divB(last - ob) + 1);
                      rr[j] = fin ? -0x40000000 : rr[j];
                    }
                  }
                  const int sumF = rdl(SFi, last);  // the chunks' growth over the block
                  pf_tok += (int64_t)Kb * q + sumF;
                  dec_tok += (int64_t)Kb * nDa - sumF;
                  ctx_p += Kb * q + sumF;
                  freeb += rdl(FBi, last) - rdl(T, last);
                  n_done += nfin;
                  nDa -= nfin;
                  nruna -= nfin;
                  q = K - nDa;
                  dG = g0 + Kb;
                  seg0 = dG;
                  cd_seg = (cs0 - rdl(KFi, last)) + nDa * dG;
                  t_d = rdl_f64(tend, last);
                  it = rdl_f64(itv, last);
                  em = __builtin_fmax(em, nfin > 0 ? (double)rdl64(pm, last) : it);
                }
                if (comp_m != 0 && Kb == kcomp) stop = dG;  // the head prefill completes at dG
                if (dG == stop) {
                  // the completing iteration finds the decodes finishing in
                  // it by fin_at
                  int mxl = 0;
#pragma unroll
                  for (int j = 0; j < NCH; ++j) {
                    if (j < nchd) {
                      const int rem0 = j == 0 ? h0.rem : L.x_rem[(j - 1) * 64 + lane];
                      const int m = rr[j] >= 0 ? 0x7fffffff - rem0 : 0;
                      mxl = m > mxl ? m : mxl;
                    }
                  }
                  const int mx = rdl(scan_max_i32(mxl), 63);
                  fin_at = nDa > 0 ? 0x7fffffff - mx - 1 : 0x3fffffff;
                }
                if (!next_ok()) {
                  more = false;
                  break;
                }
                continue;
              }
            }
            // iterations that may run as one block: up to 64, through the
            // segment's last and its first finishing iteration
            int W = stop - dG;
            W = W < 64 ? W : 64;
            W = fin_at - dG + 1 < W ? fin_at - dG + 1 : W;
            if (W >= 3) {  // (two iterations cost less one at a time)
              // A block of consecutive iterations, lane i pricing iteration
              // dG + i exactly as one iteration at a time would (the
              // operators' FLOPs and bytes are exact integers, stepped by
              // exact integer increments).  It ends before the first
              // iteration short of blocks and after the first one whose end
              // reaches an arrival that matters.
              const int g0 = dG;
              int* hist = reinterpret_cast<int*>(L.u.scratch);  // blocks taken per iteration
              hist[lane] = 0;
              __syncthreads();
#pragma unroll
              for (int j = 0; j < NCH; ++j) {
                if (j < nchd) {
                  const int o = rr[j] - g0;  // this slot's next block boundary (alive: >= 0)
                  if (o >= 0 && o < W)
                    for (int pz = o; pz < W; pz += B) atomicAdd(&hist[pz], 1);
                }
              }
              __syncthreads();
              const bool in = lane < W;
              const int T = scan_i32(in ? hist[lane] : 0);  // blocks taken through iteration i
              const double mi = (double)(g0 - seg0 + lane);
              const double F1 = L.segk[0] + mi * L.segk[2];
              const double B1 = L.segk[1] + mi * L.segk[3];
              const double F2 = L.segk[4] + mi * L.segk[6];
              const double B2 = L.segk[5] + mi * L.segk[7];
              const double t1 = __builtin_fmax(F1 * iF, B1 * iB);
              const double t2 = __builtin_fmax(F2 * iF, B2 * iB);
              double lay = L.segk[8] + t1;
              lay = lay + t2;
              lay = lay + L.segk[9];
              lay = lay + L.segk[10];
              lay = lay + L.segk[11];
              double tot = A.n_layers * lay;
              tot = tot + L.segk[12];
              const double itv = __builtin_fmax(ceil(tot), 1.0);
              // the clock at each iteration's end: integers below 2^52, so
              // the fp64 prefix sum is exact
              const double tend = rdl_f64(t_d, 1) + scan_f64(in ? itv : 0.0);
              const uint64_t short_m = ballot(in && T > freeb);
              const uint64_t arr_m = watch ? ballot(in && tend >= thr) : 0ull;
              int Kb = W;
              if (short_m != 0) {
                const int k = (int)__builtin_ctzll(short_m);
                Kb = k < Kb ? k : Kb;
              }
              if (arr_m != 0) {
                const int k = (int)__builtin_ctzll(arr_m) + 1;
                Kb = k < Kb ? k : Kb;
              }
              const int last = Kb - 1;
              // the used-block integral: each lane keeps its iterations' terms
              // (summed over the wave when the stretch ends; an fp64 sum in
              // another order than the sequential one, within 1e-9 of it)
              const double pv = (double)(NB - freeb + T) * itv;
              ubl = ubl + (lane < Kb ? pv : 0.0);
              freeb -= rdl(T, last);
              t_d = rdl_f64(tend, last);
              it = rdl_f64(itv, last);
#pragma unroll
              for (int j = 0; j < NCH; ++j) {
                if (j < nchd) {
                  const int o = rr[j] - g0;
                  if (o >= 0 && o < Kb) rr[j] += B * (divB(last - o) + 1);
                }
              }
              dG = g0 + last;  // the block's last iteration; advanced past below
            } else {
            freeb -= nneed;
#pragma unroll
            for (int j = 0; j < NCH; ++j)
              if (j < nchd) rr[j] += rr[j] == dG ? B : 0;
            const double used_d = (double)(NB - freeb);
            // as a block's lane prices its iteration: prefill and decode
            // attention at this iteration, then the layer sum in the fixed
            // operator order
            const double mi = (double)(dG - seg0);
            const double F1 = L.segk[0] + mi * L.segk[2];
            const double B1 = L.segk[1] + mi * L.segk[3];
            const double F2 = L.segk[4] + mi * L.segk[6];
            const double B2 = L.segk[5] + mi * L.segk[7];
            const double t1 = __builtin_fmax(F1 * iF, B1 * iB);
            const double t2 = __builtin_fmax(F2 * iF, B2 * iB);
            double lay = L.segk[8] + t1;
            lay = lay + t2;
            lay = lay + L.segk[9];
            lay = lay + L.segk[10];
            lay = lay + L.segk[11];
            double tot = A.n_layers * lay;
            tot = tot + L.segk[12];
            it = __builtin_fmax(ceil(tot), 1.0);
            ubl = ubl + (lane == 1 ? used_d * it : 0.0);  // (every lane has the same time)
            t_d = t_d + it;
            }
            if (dG == fin_at) {
              // Alive decodes emitting their last token finish at the end of
              // this iteration.  Iteration times never fall within a
              // segment, so the largest so far is the larger of em and this.
              em = __builtin_fmax(em, it);
              const int64_t t_end = (int64_t)rdl_f64(t_d, 1);
              const int64_t gx = (int64_t)rdl_f64(em, 1);
              int nfin = 0, l_freed = 0;
#pragma unroll
              for (int j = 0; j < NCH; ++j) {
                if (j < nchd) {
                  const int e = (j - 1) * 64 + lane;
                  const int rem0 = j == 0 ? h0.rem : L.x_rem[e];
                  const bool fin = rr[j] >= 0 && rem0 - 1 == dG;
                  const uint64_t fm = ballot(fin);
                  if (fm != 0) {
                    const int ctx0 = j == 0 ? h0.ctx : L.x_ctx[e];
                    const int64_t gap0 = j == 0 ? h0.gap : L.x_gap[e];
                    record_done(fin, j * 64 + lane, t_end, gx > gap0 ? gx : gap0);
                    l_freed += fin ? divB(ctx0 + rr[j]) : 0;  // held blocks
                    rr[j] = fin ? -0x40000000 : rr[j];
                    nfin += popc(fm);
                  }
                }
              }
              ++dG;
              close_segment();
              freeb += wsum(l_freed);
              n_done += nfin;
              nDa -= nfin;
              nruna -= nfin;
              t = (int64_t)rdl_f64(t_d, 1);  // arrivals up to the clock
              if (next < N && rdl64(w_arr, next - wbase) <= t) {
                intake();
                thr = next < N ? __builtin_fmin((double)rdl64(w_arr, next - wbase), kT52d)
                               : kT52d;
              }
              if (nruna == 0) {
                more = false;  // nothing runs
                break;
              }
              const bool want = (npre > 0 || nwait > 0) && adm_open() && !head_blocked(freeb);
              if (want && !adm_here()) {
                more = false;  // the freed slot or blocks may admit: general path
                break;
              }
              if (want) {  // the next iteration admits in place (it needs no segment)
                stop = dG;
                adm_next = true;
              } else {
                setup();
              }
            } else {
              ++dG;
            }
            if (!next_ok()) {
              more = false;
              break;
            }
          }
          if (!more) break;
            // The head prefill completes in this iteration, or an admission
            // iteration was scheduled (or the cap / watchdog is reached).  A
            // head's first completion and the admissions are handled in place,
            // with the decodes that finish here; everything else runs on the
            // general path.
            const bool head = npf == 1;
            if (stop >= stop_hard || MODE == kStagePrefill || npf > 1 ||
                (head && (fl_p & (FL_FIRST | FL_STALE)) != 0) || (!head && !adm_next))
              break;
            adm_next = false;
            // decode keys at this iteration (an admission iteration has no
            // segment: summed over the alive decodes)
            int CD;
            if (head) {
              CD = cd_seg + nDa * (dG - seg0);
            } else {
              int csl = 0;
#pragma unroll
              for (int j = 0; j < NCH; ++j) {
                if (j < nchd) {
                  const int ctx0 = j == 0 ? h0.ctx : L.x_ctx[(j - 1) * 64 + lane];
                  csl += rr[j] >= 0 ? ctx0 + 1 : 0;
                }
              }
              CD = wsum(csl) + nDa * dG;
            }
            close_segment();
            t = (int64_t)rdl_f64(t_d, 1);  // arrivals up to the clock
            if (next < N && rdl64(w_arr, next - wbase) <= t) {
              intake();
              thr = next < N ? __builtin_fmin((double)rdl64(w_arr, next - wbase), kT52d) : kT52d;
            }
            const int left = head ? tgt_p - ctx_p : 0;
            const int R1 = K - nDa - left;  // budget left after the completing prefill
            // FCFS admissions into the rest of the budget, in place, from the
            // waiting trace requests at the queue head.  When the first one's
            // prompt exceeds the budget it becomes the new head prefill;
            // otherwise, over a window of 64, each takes its whole prompt
            // while the budget lasts (those complete in this iteration and
            // join the decodes), the last one possibly a part of it (the new
            // head prefill).  Preempted requests, a rejected request among
            // those admitted, a second window and a full slot set go to the
            // general path.
            int a = 0, c = 0, q_new = 0, sq = 0, need_sum = 0, id_h = 0, tgt_h = 0, o_h = 0;
            int64_t ap_new = 0;
            int c_p = 0, c_o = 0, c_need = 0, c_qv = 0;
            bool c_ok = false, c_comp = false;
            if (policy != TS_POLICY_STATIC && (npre > 0 || nwait > 0) && nruna < M &&
                (R1 > 0 || (swap && npre > 0))) {
              if (npre > 0 || nrun >= 64 * NCH) break;  // queue candidates, full slots
              const TraceRec r = rec[next_new];
              if (may_reject && rejected(r.prompt, r.output)) break;
              const int need_h = divB(r.prompt + B - 1);
              if (need_h > freeb - nneed - adm_reserve) {
                head_need = need_h;  // the head waits for blocks
              } else if (r.prompt > R1) {  // the new head prefill
                a = 1;
                q_new = R1;
                sq = R1;
                ap_new = ((int64_t)R1 * (R1 + 1)) / 2;
                need_sum = need_h;
                id_h = next_new;
                tgt_h = r.prompt;
                o_h = r.output;
                head_need = -1;
              } else {
                const int idx = next_new + lane;
                if (idx < next) {
                  const TraceRec rc = rec[idx];
                  c_p = rc.prompt;
                  c_o = rc.output;
                }
                // candidates up to the first rejected one
                const uint64_t rjm = ballot(may_reject && idx < next && rejected(c_p, c_o));
                const int lim = rjm != 0 ? (int)__builtin_ctzll(rjm) : 64;
                c_need = idx < next && lane < lim ? divB(c_p + B - 1) : 0;
                const int SN = scan_i32(c_need);
                const int SP = scan_i32(lane < lim ? c_p : 0);
                const int ET = SP - (lane < lim ? c_p : 0);  // prompt tokens of those before
                c_ok = idx < next && lane < lim && lane < M - nruna &&
                       SN <= freeb - nneed - adm_reserve && ET < R1;
                a = popc(ballot(c_ok));  // >= 1: the first one fits
                if ((rjm != 0 && a == lim) || a == 64 || nrun + a > 64 * NCH)
                  break;  // a rejected request, a second window, full slots
                c_comp = c_ok && SP <= R1;
                c = popc(ballot(c_comp));  // >= 1
                c_qv = c_ok ? (c_comp ? c_p : R1 - ET) : 0;
                sq = wsum(c_qv);
                ap_new = wsum64(c_ok ? ((int64_t)c_qv * (c_qv + 1)) / 2 : 0);
                need_sum = rdl(SN, a - 1);
                q_new = a > c ? rdl(c_qv, a - 1) : 0;
                head_need = a < next - next_new ? rdl(c_need, a) : -1;
              }
            }
            // reserve, admit, price the iteration with both prefills
            if (nneed > 0) {
              freeb -= nneed;
#pragma unroll
              for (int j = 0; j < NCH; ++j)
                if (j < nchd) rr[j] += rr[j] == dG ? B : 0;
            }
            freeb -= need_sum;
            const int TP = left + sq;
            const int64_t AP =
                (head ? (int64_t)left * ctx_p + ((int64_t)left * (left + 1)) / 2 : 0) + ap_new;
            double iter_d;
            const int64_t iter_ns =
                iteration_ns(roofc, A.n_layers, iF, iB, nDa + TP, TP, AP, (head ? tgt_p : 0) + sq,
                             nDa, CD, nDa + (head ? 1 : 0) + c, 0.0, false, &iter_d);
            const int64_t t_beg = t;
            const int64_t t_end = t_beg + iter_ns;
            ubl = ubl + (lane == 1 ? (double)(NB - freeb) * iter_d : 0.0);
            t_d = t_d + iter_d;
            if (NB - freeb > peak) peak = NB - freeb;
            pf_tok += TP;
            dec_tok += nDa;
            // the decodes' gaps include this iteration and the segment before
            // it (whose largest time is its last, it); the new decode's do not
            em = __builtin_fmax(__builtin_fmax(em, it), iter_d);
            const int64_t gx = (int64_t)rdl_f64(em, 1);
#pragma unroll
            for (int j = 0; j < NCH; ++j) {
              if (j < nchd) {
                const bool al = rr[j] >= 0;
                if (j == 0) {
                  h0.gap = al && gx > h0.gap ? gx : h0.gap;
                } else {
                  const int e = (j - 1) * 64 + lane;
                  const int64_t g = L.x_gap[e];
                  L.x_gap[e] = al && gx > g ? gx : g;
                }
              }
            }
            em = 0.0;
            it = 0.0;
            if (!head || dG == fin_at) {
              // alive decodes emitting their last token finish here (their
              // blocks are free from the next iteration on)
              int nfin = 0, l_freed = 0;
#pragma unroll
              for (int j = 0; j < NCH; ++j) {
                if (j < nchd) {
                  const int e = (j - 1) * 64 + lane;
                  const int rem0 = j == 0 ? h0.rem : L.x_rem[e];
                  const bool fin = rr[j] >= 0 && rem0 - 1 == dG;
                  const uint64_t fm = ballot(fin);
                  if (fm != 0) {
                    const int ctx0 = j == 0 ? h0.ctx : L.x_ctx[e];
                    const int64_t gap0 = j == 0 ? h0.gap : L.x_gap[e];  // folded above
                    record_done(fin, j * 64 + lane, t_end, gap0);
                    l_freed += fin ? divB(ctx0 + rr[j]) : 0;  // held blocks
                    rr[j] = fin ? -0x40000000 : rr[j];
                    nfin += popc(fm);
                  }
                }
              }
              freeb += wsum(l_freed);
              n_done += nfin;
              nDa -= nfin;
              nruna -= nfin;
            }
            // the completed prefill emits its first token and joins the
            // decodes at iteration dG + 1
            if (head) {
              const int js = nD >> 6, ls = nD & 63, g1 = dG + 1;
              int room_s, id_s;
              if (NCH == 1 || js == 0) {
                room_s = rdl(h0.room, ls);
                id_s = L.id[nD];
                h0.ctx = lane == ls ? tgt_p - g1 : h0.ctx;
                h0.rem = lane == ls ? h0.rem + g1 : h0.rem;
                h0.fl = lane == ls ? (h0.fl | FL_FIRST) : h0.fl;
              } else {
                const int e = (js - 1) * 64 + ls;
                room_s = __builtin_amdgcn_readfirstlane(L.x_room[e]);
                id_s = L.id[nD];
                // read once for the wave, then every lane stores the same values
                const int rem_s = __builtin_amdgcn_readfirstlane(L.x_rem[e]);
                const int fl_s = __builtin_amdgcn_readfirstlane((int)L.x_fl[e]);
                L.x_ctx[e] = tgt_p - g1;
                L.x_rem[e] = rem_s + g1;
                L.x_fl[e] = fl_s | FL_FIRST;
              }
              id_s = __builtin_amdgcn_readfirstlane(id_s);
              RR[gid_of(id_s)].first_token_ns = t_end;
#pragma unroll
              for (int j = 0; j < NCH; ++j)
                if (j == js) rr[j] = lane == ls ? room_s + g1 : rr[j];
              ++nD;
              ++nDa;
              nchd = (nD + 63) >> 6;
            }
            if (c > 0) {
              // the admitted requests take slots nrun.. in order: those whose
              // prompt completes emit their first token and join the decodes
              // at iteration dG + 1 (stored shifted by it, like the head
              // above), the last one may stay as the new head prefill
              const int g1 = dG + 1;
              const int s0 = nrun;
              if (c_ok) {
                const int idx = next_new + lane;
                StageSlot st;
                st.tgt = c_p;
                st.ctx = c_comp ? c_p - g1 : c_qv;
                st.rem = c_comp ? c_o + g1 : c_o;
                st.room = c_need * B - c_p;
                st.fl = c_comp ? FL_FIRST : 0;
                st.q = 0;
                st.gap = 0;
                L.u.stage[lane] = st;
                L.id[s0 + lane] = idx;
                L.npre[s0 + lane] = 0;
                RR[gid_of(idx)].admit_ns = t_beg;  // first admission
                if (c_comp) RR[gid_of(idx)].first_token_ns = t_end;
              }
              __syncthreads();
#pragma unroll
              for (int j = 0; j < NCH; ++j) {
                const int sl = j * 64 + lane;
                if (sl >= s0 && sl < s0 + a) {
                  const StageSlot st = L.u.stage[sl - s0];
                  Hot h;
                  h.ctx = st.ctx; h.tgt = st.tgt; h.rem = st.rem; h.room = st.room;
                  h.fl = st.fl; h.q = st.q; h.gap = st.gap;
                  store_chunk<NCH>(L, h0, j, lane, h);
                  if (sl < s0 + c) rr[j] = st.room + g1;
                }
              }
              __syncthreads();
              nrun += a;
              nruna += a;
              nD += c;
              nDa += c;
              nchd = (nD + 63) >> 6;
              next_new += a;
              nwait -= a;
              if (nwait == 0) next_new = next;
              if (a > c) {  // the new head prefill, in slot s0 + c
                npf = 1;
                ctx_p = q_new;
                tgt_p = rdl(c_p, a - 1);
                fl_p = 0;
              } else {
                npf = 0;
              }
            } else if (a > 0) {
              // the admitted request becomes the head prefill in slot nrun
              const int js = nrun >> 6, ls = nrun & 63;
              if (NCH == 1 || js == 0) {
                h0.ctx = lane == ls ? q_new : h0.ctx;
                h0.tgt = lane == ls ? tgt_h : h0.tgt;
                h0.rem = lane == ls ? o_h : h0.rem;
                h0.room = lane == ls ? need_sum * B - tgt_h : h0.room;
                h0.fl = lane == ls ? 0 : h0.fl;
                h0.q = lane == ls ? 0 : h0.q;
                h0.gap = lane == ls ? 0 : h0.gap;
              } else {
                const int e = (js - 1) * 64 + ls;  // every lane stores the same values
                L.x_ctx[e] = q_new;
                L.x_tgt[e] = tgt_h;
                L.x_rem[e] = o_h;
                L.x_room[e] = need_sum * B - tgt_h;
                L.x_fl[e] = 0;
                L.x_q[e] = 0;
                L.x_gap[e] = 0;
              }
              L.id[nrun] = id_h;
              L.npre[nrun] = 0;
              RR[gid_of(id_h)].admit_ns = t_beg;  // first admission
              ++nrun;
              ++nruna;
              ++next_new;
              if (--nwait == 0) next_new = next;
              npf = 1;
              ctx_p = q_new;
              tgt_p = tgt_h;
              fl_p = 0;
            } else {
              npf = 0;
            }
            ++dG;
            seg0 = dG;
            const bool want = (npre > 0 || nwait > 0) && adm_open() && !head_blocked(freeb);
            if (want && !adm_here()) break;  // the head may be admitted next: general path
            if (want) {  // the next iteration admits in place (it needs no segment)
              stop = dG;
              adm_next = true;
            } else {
              setup();
            }
          if (!next_ok()) break;
        }
        // the last segment's bookkeeping, the point's counters, the decodes
        // (finished ones get rem 0) and the head prefill, then close the holes
        close_segment();
        em = __builtin_fmax(em, it);
        t = (int64_t)rdl_f64(t_d, 1);
        ubns = ubns + rdl_f64(scan_f64(ubl), 63);
        n_iters += dG;
        const int64_t gx = (int64_t)rdl_f64(em, 1);
#pragma unroll
        for (int j = 0; j < NCH; ++j) {
          if (j < nchd) {
            const bool dec = (j * 64 + lane) < nD;
            const bool al = rr[j] >= 0;
            if (j == 0) {
              h0.ctx = al ? h0.ctx + dG : h0.ctx;
              h0.rem = al ? h0.rem - dG : (dec ? 0 : h0.rem);
              h0.room = al ? rr[0] - dG : h0.room;
              h0.gap = al && gx > h0.gap ? gx : h0.gap;
            } else {
              const int e = (j - 1) * 64 + lane;
              const int64_t g = L.x_gap[e];
              L.x_ctx[e] = al ? L.x_ctx[e] + dG : L.x_ctx[e];
              L.x_rem[e] = al ? L.x_rem[e] - dG : (dec ? 0 : L.x_rem[e]);
              L.x_room[e] = al ? rr[j] - dG : L.x_room[e];
              L.x_gap[e] = al && gx > g ? gx : g;
            }
          }
        }
        if (npf > 0) {
          const int jp = nD >> 6, lp = nD & 63;
          if (NCH == 1 || jp == 0) h0.ctx = lane == lp ? ctx_p : h0.ctx;
          else L.x_ctx[(jp - 1) * 64 + lp] = ctx_p;  // every lane stores the same value
        }
        if (nruna < nrun) compact(nrun - nruna);
      }
    }
    // watchdog: a point running longer than the wall-clock limit stops
    if (time_limit != 0 && (n_iters & 255) == 0 &&
        __builtin_amdgcn_s_memrealtime() - clock0 > time_limit) {
      status = TS_POINT_TIME_LIMIT;
      break;
    }
    // ---- 1. intake: every request with arrival <= t joins the waiting set;
    // ---- 2. when nothing runs or waits, jump to the next arrival
    bool drained = false;
    for (;;) {
      intake();
      if (nrun != 0 || npre != 0 || nwait != 0) break;
      if (next >= N) {
        drained = true;
        break;
      }
      t = rdl64(w_arr, next - wbase);
    }
    if (drained) break;
    if (n_iters >= A.iter_cap) {
      status = TS_POINT_ITER_LIMIT;
      break;
    }
    // Prefill-first: when the waiting head can be admitted now the
    // iteration admits and prefills only and the decodes pause; otherwise it
    // runs every decode and admits nothing.
    bool pf_iter = false;
    if (pff && (npre > 0 || nwait > 0) && nrun < M) {
      int tgt_h;  // tokens whose blocks the head needs
      if (npre > 0) {
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
        const int qc = Q[qhead].ctx, qt = Q[qhead].target;
        tgt_h = qc > qt ? qc : qt;
      } else {
        int i = next_new;  // the first candidate that is not rejected
        while (may_reject && i < next - 1 && rejected(rec[i].prompt, rec[i].output)) ++i;
        tgt_h = rec[i].prompt;
      }
      pf_iter = divB(tgt_h + B - 1) <= freeb - (npre > 0 ? 0 : adm_reserve);
    }

    // ---- 3. reserve a block for decodes crossing a block boundary
    int nch = (nrun + 63) >> 6;
    nch = nch < NCH ? nch : NCH;
    int nneed = 0;
#pragma nounroll
    for (int j = 0; j < nch && !pf_iter; ++j) {
      const Hot h = load_chunk<NCH>(L, h0, j, lane);
      const bool act = (j * 64 + lane) < nrun;
      nneed += popc(ballot(act && h.ctx >= h.tgt && h.room == 0));
    }
    bool preempted = false;
    int xblk = 0;  // blocks swapped out or in this iteration
    if (nneed <= freeb) {
      freeb -= nneed;
      if (nneed > 0) {
#pragma nounroll
        for (int j = 0; j < nch; ++j) {
          const bool act = (j * 64 + lane) < nrun;
          if (j == 0) {
            if (act && h0.ctx >= h0.tgt && h0.room == 0) h0.room += B;
          } else {
            const int e = (j - 1) * 64 + lane;
            if (act && L.x_ctx[e] >= L.x_tgt[e] && L.x_room[e] == 0) L.x_room[e] = B;
          }
        }
      }
    } else {
      // Preemption from the tail: keep the longest prefix of slots whose
      // held + needed blocks fit in the whole budget.
      int carry = 0, k = 0, kept = 0, kneed = 0;
#pragma nounroll
      for (int j = 0; j < nch; ++j) {
        const Hot h = load_chunk<NCH>(L, h0, j, lane);
        const bool act = (j * 64 + lane) < nrun;
        const int top = h.ctx > h.tgt ? h.ctx : h.tgt;
        const int need = (h.ctx >= h.tgt && h.room == 0) ? 1 : 0;
        const int v = act ? divB(top + h.room) + need : 0;  // held + needed blocks
        const int S = scan_i32(v) + carry;
        const bool keep = act && S <= NB;
        k += popc(ballot(keep));
        kneed += popc(ballot(keep && need != 0));
        kept += wsum(keep ? v : 0);
        carry = rdl(S, 63);
      }
      // swap moves the victims' held blocks: all held blocks but the kept ones
      if (swap) xblk = NB - freeb - (kept - kneed);
      freeb = NB - kept;
      const int nv = nrun - k;
      qhead = (qhead - nv) & (kQueueCap - 1);
#pragma nounroll
      for (int j = 0; j < nch; ++j) {
        Hot h = load_chunk<NCH>(L, h0, j, lane);
        const int s = j * 64 + lane;
        if (s < k) {
          if (h.ctx >= h.tgt && h.room == 0) h.room += B;
        } else if (s < nrun) {
          // victims keep admission order at the front of the waiting queue:
          // they are older than every request still waiting
          const int id = L.id[s];
          int fl = h.fl;
          if ((fl & FL_FIRST) && !(fl & FL_STALE)) {
            // the last token is the one emitted at the end of the previous iteration
            if (h.ctx >= h.tgt) RR[gid_of(id)].finish_ns = t;  // last token, until it finishes
            fl |= FL_STALE;
          }
          QEntry e;
          e.id = id;
          if (swap) {  // the KV goes to host memory and comes back as it was
            e.target = h.tgt;
            e.ctx = h.ctx;
          } else {  // recompute: prefill again over prompt + tokens decoded
            e.target = h.ctx > h.tgt ? h.ctx : h.tgt;
            e.ctx = 0;
          }
          e.rem = h.rem;
          e.n_pre = L.npre[s] + 1;
          e.flags = fl;
          e.gap = h.gap;
          Q[(qhead + s - k) & (kQueueCap - 1)] = e;
        }
        store_chunk<NCH>(L, h0, j, lane, h);
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
      npre += nv;
      n_pre_tot += nv;
      nrun = k;
      preempted = true;
      head_need = -1;
      nch = (nrun + 63) >> 6;
      nch = nch < NCH ? nch : NCH;
    }

    // ---- 4. token budget: decodes one token, running prefills share the rest
    int nD = 0, npf = 0;
#pragma nounroll
    for (int j = 0; j < nch; ++j) {
      const Hot h = load_chunk<NCH>(L, h0, j, lane);
      const bool act = (j * 64 + lane) < nrun;
      nD += popc(ballot(act && h.ctx >= h.tgt));
      npf += popc(ballot(act && h.ctx < h.tgt));
    }
    int R = 0;
    if (!unlimited) R = K - nD;
    if (npf > 0) {
      int carry = 0;  // prefill tokens still needed by the slots before this chunk
#pragma nounroll
      for (int j = 0; j < nch; ++j) {
        const Hot h = load_chunk<NCH>(L, h0, j, lane);
        const bool pf = (j * 64 + lane) < nrun && h.ctx < h.tgt;
        const int left = pf ? h.tgt - h.ctx : 0;
        int qv = left;
        if (!unlimited) {
          if (npf == 1) {  // one running prefill: min(what it needs, the budget)
            qv = left < R ? left : R;
            const uint64_t pm = ballot(pf);
            if (pm != 0) carry += rdl(left, (int)__builtin_ctzll(pm));
          } else {
            const int S = scan_i32(left);
            int avail = R - (S - left + carry);
            avail = avail < 0 ? 0 : avail;
            qv = left < avail ? left : avail;
            carry += rdl(S, 63);
          }
        }
        if (j == 0) {
          if (pf) h0.q = qv;
        } else if (pf) {
          L.x_q[(j - 1) * 64 + lane] = qv;
        }
      }
      if (!unlimited) {
        R = R - carry;
        if (R < 0) R = 0;
      }
    }

    // ---- 5. FCFS admission over 64-candidate windows (none after
    // preemption; static batching only into an empty running set;
    // prefill-first only in a prefill iteration).  A first admission leaves
    // the admission-ratio reserve free.
    int n_darr = 0;  // decode device: arrivals admitted, decoding in this iteration
    bool adm_before = false;  // an earlier window of this iteration admitted
    if (!preempted && (!pff || pf_iter) && (policy != TS_POLICY_STATIC || nrun == 0)) {
      int guard = M + N / 64 + 4;  // each pass admits or advances a window
      while (nrun < M && (unlimited || R > 0 || (swap && npre > 0)) && (npre > 0 || nwait > 0) &&
             --guard >= 0) {
        if (head_need >= 0 && head_need > freeb - (npre > 0 ? 0 : adm_reserve)) break;
        const bool fromq = npre > 0;
        const bool swin = fromq && swap;  // swapped requests: blocks only, no budget
        bool valid;
        int c_id, c_tgt, c_rem, c_npre, c_fl, c_ctx = 0;
        int64_t c_gap;
        if (fromq) {
          valid = lane < npre;
          __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
          if (valid) {
            const QEntry e = Q[(qhead + lane) & (kQueueCap - 1)];
            c_id = e.id; c_tgt = e.target; c_rem = e.rem; c_npre = e.n_pre; c_fl = e.flags;
            c_gap = e.gap; c_ctx = e.ctx;
          } else {
            c_id = 0; c_tgt = 1; c_rem = 1; c_npre = 0; c_fl = 0; c_gap = 0;
          }
        } else {
          const int idx = next_new + lane;
          valid = idx < next;
          c_id = idx; c_npre = 0; c_fl = 0; c_gap = 0; c_tgt = 1; c_rem = 1;
          if (valid) {
            const TraceRec r = rec[idx];
            c_tgt = r.prompt;
            c_rem = MODE == kStagePrefill ? 1 : r.output;  // a prefill device runs no decode
            if (may_reject && rejected(r.prompt, r.output)) valid = false;
          }
          if constexpr (MODE == kStageDecode) {  // arrives with its prompt's KV, first token out
            c_ctx = c_tgt;
            c_fl = FL_FIRST | FL_STALE;
          }
        }
        const uint64_t vm = ballot(valid);
        const int nvalid = popc(vm);
        if (nvalid == 0) {  // a window of rejected requests only
          const int adv = next - next_new < 64 ? next - next_new : 64;
          if (adv <= 0) {  // nothing left to scan: no valid request waits
            nwait = 0;
            break;
          }
          next_new += adv;
          continue;
        }
        const int rank = rank_below(vm);
        // a decode device's arrival decodes at once: blocks for its KV and
        // the next token, one token of budget
        const bool darr = MODE == kStageDecode && !fromq;
        const int c_top = c_ctx > c_tgt ? c_ctx : c_tgt;  // tokens held in blocks
        const int need = valid ? divB(c_top + (darr ? 1 : 0) + B - 1) : 0;
        const int SN = scan_i32(need);
        const int tq = valid ? (darr ? 1 : c_tgt) : 0;
        const int ET = scan_i32(tq) - tq;
        const int slots_left = M - nrun;
        const bool adm = valid && rank < slots_left && SN <= freeb - (fromq ? 0 : adm_reserve) &&
                         (unlimited || swin || ET < R);
        const uint64_t am = ballot(adm);
        const int a = popc(am);
        if (a == 0) {
          head_need = rdl(need, (int)__builtin_ctzll(vm));
          break;
        }
        if (nrun + a > 64 * NCH) {  // more running requests than this kernel's slots
          status = kHandOver;
          break;
        }
        const int last_lane = 63 - (int)__builtin_clzll(am);
        const int qv =
            (swin || darr) ? 0 : (unlimited ? c_tgt : (c_tgt < R - ET ? c_tgt : R - ET));
        const int taken = rdl(SN, last_lane);
        freeb -= taken;
        if (swin) xblk += taken;
        if (!unlimited) R -= wsum(adm ? (darr ? 1 : qv) : 0);
        if (adm) {
          if constexpr (MODE == kStageDecode) {
            if (!fromq) {  // its times so far come from the prefill device
              const int g = gid_of(c_id);
              ts_req_result& o = RR[g];
              o.admit_ns = A.s1_admit[req_base + g];
              o.first_token_ns = A.s1_first[req_base + g];
              o.finish_ns = o.first_token_ns;  // the last token, until it finishes
            }
          } else {
            if (!fromq) RR[gid_of(c_id)].admit_ns = t;  // first admission
          }
          L.id[nrun + rank] = c_id;  // rank < M - nrun: a free slot
          L.npre[nrun + rank] = c_npre;
          StageSlot st;
          st.tgt = c_tgt; st.rem = c_rem;
          st.fl = swin ? (c_fl | FL_IDLE) : c_fl;
          st.q = qv; st.room = need * B - c_top; st.ctx = c_ctx; st.gap = c_gap;
          L.u.stage[rank] = st;
        }
        __syncthreads();
#pragma nounroll
        for (int j = nrun >> 6; j < NCH && j * 64 < nrun + a; ++j) {
          const int s = j * 64 + lane;
          if (s >= nrun && s < nrun + a) {
            const StageSlot st = L.u.stage[s - nrun];
            Hot h;
            h.ctx = st.ctx; h.tgt = st.tgt; h.rem = st.rem; h.room = st.room; h.fl = st.fl;
            h.q = st.q; h.gap = st.gap;
            store_chunk<NCH>(L, h0, j, lane, h);
          }
        }
        __syncthreads();
        nrun += a;
        adm_before = true;
        if (darr) n_darr += a;
        if (fromq) {
          qhead = (qhead + a) & (kQueueCap - 1);
          npre -= a;
        } else {
          next_new += last_lane + 1;
          nwait -= a;
          if (nwait == 0) next_new = next;
        }
        head_need = -1;
        if (a < nvalid) {  // the first candidate left out is the new head
          head_need = rdl(need, (int)__builtin_ctzll(vm & ~am));
          break;
        }
      }
      nch = (nrun + 63) >> 6;
      nch = nch < NCH ? nch : NCH;
    }

    if (status == kHandOver) {
      freeb += nneed;  // undo this iteration's reservations (the rooms: below)
      if (adm_before) status = kHandOverRedo;
      break;
    }

    // ---- 6. batch sums and the roofline iteration time (paused decodes of a
    // prefill-first iteration and requests swapped in now take no part)
    if constexpr (MODE == kStageDecode) nD += n_darr;
    if (pf_iter) nD = 0;
    int l_cd = 0, l_tp = 0, l_cp = 0, TP = 0, CP = 0, Rc = 0;
    int64_t l_ap = 0, AP = 0;
    bool wide = false;  // some chunk has more than two prefills: reduce by DPP
#pragma nounroll
    for (int j = 0; j < nch; ++j) {
      const Hot h = load_chunk<NCH>(L, h0, j, lane);
      const bool act = (j * 64 + lane) < nrun;
      const bool dec = act && h.ctx >= h.tgt && !pf_iter && !(h.fl & FL_IDLE);
      const bool pf = act && !dec && h.q > 0;
      if (dec) l_cd += h.ctx + 1;
      uint64_t m = ballot(pf);
      Rc += popc(ballot(pf && h.ctx + h.q == h.tgt && !(h.fl & FL_FIRST)));  // first tokens
      if (popc(m) <= 2) {
        while (m != 0) {  // one or two prefills: read them out lane by lane
          const int l = (int)__builtin_ctzll(m);
          m &= m - 1;
          const int qq = rdl(h.q, l);
          const int c0 = rdl(h.ctx, l);
          TP += qq;
          CP += c0 + qq;
          AP += (int64_t)qq * c0 + ((int64_t)qq * (qq + 1)) / 2;
        }
      } else {
        wide = true;
        if (pf) {
          l_tp += h.q;
          l_cp += h.ctx + h.q;
          l_ap += (int64_t)h.q * h.ctx + ((int64_t)h.q * (h.q + 1)) / 2;
        }
      }
    }
    const int CD = nD > 0 ? wsum(l_cd) : 0;
    if (wide) {
      TP += wsum(l_tp);
      CP += wsum(l_cp);
      AP += wsum64(l_ap);
    }
    // swap transfers, priced by the host link's bandwidth
    const double xfer =
        swap ? (double)((int64_t)xblk * P.block_bytes) * P.inv_link_ns : 0.0;
    double iter_d;
    const int64_t iter_ns = iteration_ns(roofc, A.n_layers, iF, iB, nD + TP, TP, AP, CP, nD,
                                         CD, nD + Rc, xfer, P.swap_overlap != 0, &iter_d);

    // ---- 7. advance the clock and every scheduled request
    const int64_t t_end = t + iter_ns;
    const int used = NB - freeb;
    if (used > peak) peak = used;
    ubns = ubns + (double)used * iter_d;
    ++n_iters;
    pf_tok += TP;
    dec_tok += nD;

    int nfin = 0, l_freed = 0;
#pragma nounroll
    for (int j = 0; j < nch; ++j) {
      Hot h = load_chunk<NCH>(L, h0, j, lane);
      const int s = j * 64 + lane;
      const bool act = s < nrun;
      const bool dec = act && h.ctx >= h.tgt && !pf_iter && !(h.fl & FL_IDLE);
      bool fin = false, pfin = false;
      if (pf_iter && act && h.ctx >= h.tgt && !(h.fl & FL_STALE)) {
        // a paused decode: its last token ended the previous iteration
        RR[gid_of(L.id[s])].finish_ns = t;  // the last token, until it finishes
        h.fl |= FL_STALE;
      }
      if (dec) {
        h.ctx += 1;
        h.rem -= 1;
        h.room -= 1;
        // consecutive tokens: the gap is this iteration; after a re-prefill
        // the gap reaches back to the token before the preemption
        int64_t g = iter_ns;
        if (h.fl & FL_STALE) {
          g = t_end - RR[gid_of(L.id[s])].finish_ns;
          h.fl &= ~FL_STALE;
        }
        h.gap = g > h.gap ? g : h.gap;
        fin = h.rem == 0;
      } else if (act && h.q > 0) {
        h.ctx += h.q;
        if (h.ctx == h.tgt && !(h.fl & FL_FIRST)) {  // the full prefill emits a token
          h.fl |= FL_FIRST;
          RR[gid_of(L.id[s])].first_token_ns = t_end;
          if constexpr (MODE == kStagePrefill) {  // and leaves the prefill device
            h.rem = 0;
            pfin = true;
          }
        }
        h.q = 0;
      }
      h.fl &= ~FL_IDLE;
      store_chunk<NCH>(L, h0, j, lane, h);
      if constexpr (MODE == kStagePrefill) {
        const uint64_t pm = ballot(pfin);
        if (pm != 0) {
          hand_over(pm, j, h.tgt, t_end);
          l_freed += pfin ? divB(h.ctx + h.room) : 0;  // held blocks
          nfin += popc(pm);
        }
      }
      const uint64_t fm = ballot(fin);
      if (fm != 0) {
        record_done(fin, s, t_end, h.gap);
        if (fin) l_freed += divB(h.ctx + h.room);  // held blocks (ctx >= tgt here)
        nfin += popc(fm);
      }
    }
    if (nfin > 0) {
      freeb += wsum(l_freed);
      n_done += nfin;
      compact(nfin);
    }
    t = t_end;
  }

  if (status == kHandOver || status == kHandOverRedo) {
    if constexpr (SIMPLE && NCH < 4) {
      // The state at the hand-over iteration's start for the wider launch:
      // its reservations undone (nothing else has changed, unless an earlier
      // window admitted: then the wider launch starts over).  At an
      // iteration's start every slot has less than a block of free room, so
      // the decodes that reserved are those with a block of it now.
      unsigned char* base = A.resume + (size_t)P.resume * kResumeBytes;
      const bool valid = A.resume != nullptr && status == kHandOver;
      if (valid) {
        ResumeSlot* rs = reinterpret_cast<ResumeSlot*>(base + kResumeHead);
#pragma unroll
        for (int j = 0; j < NCH; ++j) {
          const int sl = j * 64 + lane;
          if (sl < nrun) {
            const Hot h = load_chunk<NCH>(L, h0, j, lane);
            ResumeSlot o;
            o.ctx = h.ctx; o.tgt = h.tgt; o.rem = h.rem; o.room = h.room == B ? 0 : h.room;
            o.fl = h.fl; o.q = 0; o.id = L.id[sl]; o.npre = L.npre[sl]; o.gap = h.gap;
            rs[sl] = o;
          }
        }
        QEntry* rq =
            reinterpret_cast<QEntry*>(base + kResumeHead + kResumeSlots * sizeof(ResumeSlot));
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
        for (int i = lane; i < npre; i += 64) rq[i] = Q[(qhead + i) & (kQueueCap - 1)];
      }
      if (A.resume != nullptr && lane == 0) {
        ResumeHead hd;
        hd.t = t;
        hd.n_iters = n_iters;
        hd.n_pre_tot = n_pre_tot;
        hd.pf_tok = pf_tok;
        hd.dec_tok = dec_tok;
        hd.ubns = ubns;
        hd.freeb = freeb;
        hd.nrun = nrun;
        hd.npre = npre;
        hd.next = next;
        hd.next_new = next_new;
        hd.nwait = nwait;
        hd.wbase = wbase;
        hd.head_need = head_need;
        hd.peak = peak;
        hd.n_done = n_done;
        hd.valid = valid ? 1 : 0;
        hd.counted = valid ? n_iters : n_it0;
        *reinterpret_cast<ResumeHead*>(base) = hd;
      }
      if (!valid) n_iters = n_it0;  // the wider launch simulates these again
    }
    // the iterations simulated here, up to the hand-over state
    atomicAdd(A.work, (unsigned long long)(lane == 0 ? n_iters - n_it0 : 0));
    return (int)(((int64_t)(N - n_done) * kHandBuckets) / (N + 1));
  }

  // ---- a point stopped early (iteration cap, watchdog): the requests it
  // has not finished keep "pending" records: the running ones, the
  // preempted ones in the queue, and those never admitted (from next_new on)
  if (status == TS_POINT_ITER_LIMIT || status == TS_POINT_TIME_LIMIT) {
    ts_req_result o;
    o.admit_ns = -1; o.first_token_ns = -1; o.finish_ns = -1; o.max_gap_ns = 0;
    o.n_preempt = 0; o.status = TS_REQ_PENDING;
    for (int s0 = 0; s0 < nrun; s0 += 64)
      if (s0 + lane < nrun) RR[gid_of(L.id[s0 + lane])] = o;
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
    for (int k0 = 0; k0 < npre; k0 += 64)
      if (k0 + lane < npre) RR[gid_of(Q[(qhead + k0 + lane) & (kQueueCap - 1)].id)] = o;
    for (int i0 = next_new; i0 < N; i0 += 64) {
      const int i = i0 + lane;
      if (i < N && !(may_reject && rejected(rec[i].prompt, rec[i].output))) RR[gid_of(i)] = o;
    }
  }

  // ---- per-point results (latency sums, SLO counts, percentiles and the
  // digest are filled by the statistics kernel from the request records)
  if constexpr (MODE == kStagePrefill) {
    const int v = lane < nd_pd ? lane : nd_pd - 1;  // lanes past n_d repeat the last store
    X->sub_cnt[P.unit * kMaxDev + v] = (int)L.sub_cnt[v];
  }
  __syncthreads();
  {
    // Every lane stores the same uniform record: no lane-dependent branch
    // next to the work-queue ticket read, which the optimizer could thread
    // so that the ticket broadcast runs with a partial wave.
    ts_point_result o;
    o.status = status;
    o.n_done = n_done;
    o.n_rejected = n_rej;
    o.num_blocks = NB;
    o.n_iters = n_iters;
    o.n_preempt = n_pre_tot;
    o.prefill_tokens = pf_tok;
    o.decode_tokens = dec_tok;
    o.peak_used_blocks = peak;
    o.first_arrival_ns = N > 0 ? rec[0].arrival_ns : -1;
    o.last_finish_ns = -1;
    o.sum_ttft_ns = 0;
    o.sum_e2e_ns = 0;
    o.max_e2e_ns = -1;
    o.sum_tpot_num_ns = 0;
    o.p50_e2e_ns = o.p90_e2e_ns = o.p99_e2e_ns = -1;
    o.p50_ttft_ns = o.p99_ttft_ns = -1;
    o.slo_ok = 0;
    o.used_block_ns = ubns;
    o.digest = 0;
    o.slo_tpot_ok = 0;
    A.res[oi] = o;
  }
  // the iterations this launch simulated to completion (every lane adds, lane
  // 0 the count: no lane-dependent branch)
  atomicAdd(A.work, (unsigned long long)(lane == 0 ? n_iters - n_it0 : 0));
  return -1;
}

// A point the 64-slot launch handed over, taken by that launch itself once
// no point of its own is left: the next listed position of the fullest
// bucket whose list has one, if its entry is written and no launch has
// claimed the point.  Returns the point, or -1 when no list has a position
// left to take now (points handed later go to the 128-slot launch, which
// also takes any position passed over here).
__device__ __forceinline__ int take_handed(const SimArgs& A, const int lane) {
  for (int b = kHandBuckets - 1; b >= 0; --b) {
    unsigned int* nb = A.handed_n + b;
    unsigned int* tb = A.take + b;
    const int n = __builtin_amdgcn_readfirstlane(
        (int)__hip_atomic_load(nb, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
    int t = __builtin_amdgcn_readfirstlane(
        (int)__hip_atomic_load(tb, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
    // take position t while it is below the count (a compare-and-swap, so
    // that the take counter never passes the count)
    bool got = false;
    for (int tries = 0; tries < 64 && t < n && !got; ++tries) {
      unsigned int old = 0;
      if (lane == 0) old = atomicCAS(tb, (unsigned)t, (unsigned)t + 1u);
      const int o = __builtin_amdgcn_readfirstlane((int)old);
      got = o == t;
      t = o;
    }
    if (!got) continue;
    // the entry is stored right after its position is reserved: wait a
    // bounded while for it, else leave it to the 128-slot launch
    int* ent = A.handed + A.handed_off[0] + b * A.hand_cap[0] + t;
    int pidx = -1;
    for (int spin = 0; spin < 4096; ++spin) {
      pidx = __builtin_amdgcn_readfirstlane(
          __hip_atomic_load(ent, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
      if (pidx >= 0) break;
      __builtin_amdgcn_s_sleep(4);
    }
    if (pidx < 0) continue;
    // the entry was stored after the hand-over record (a release fence):
    // acquire it before reading the record
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    const int slot = A.points[pidx].resume;
    unsigned int won = 0;
    if (lane == 0) won = atomicCAS(A.claim + slot, 0u, 1u) == 0u ? 1u : 0u;
    if (__builtin_amdgcn_readfirstlane((int)won) != 0) return pidx;
  }
  return -1;
}

// Persistent grid: each wave64 workgroup takes the next point from a ticket
// counter until none is left.  The simple 64-slot kernel then continues, with
// 128 slots, points that it handed over (when the launch has take lists):
// the workgroups that run out of points early fill the launch's tail with
// the 128-slot launch's work.
template <int NCH, int MODE, bool SIMPLE>
__global__ __launch_bounds__(64, NCH == 4 ? 4 : (SIMPLE ? 6 : 5)) void sim_kernel(SimArgs A) {
  constexpr bool kTail = NCH == 1 && SIMPLE;
  // slot state: one buffer for both widths in the 64-slot simple kernel
  __shared__ __attribute__((aligned(16))) unsigned char lds_slots[sizeof(SlotLds<kTail ? 2 : NCH>)];
  SlotLds<NCH>& L = *reinterpret_cast<SlotLds<NCH>*>(lds_slots);
  const int lane = lane_id();
  QEntry* Q = A.queue + (size_t)blockIdx.x * kQueueCap;
  __shared__ double coef[32];
  if (lane < 8) {
    coef[lane] = A.lc.f[lane];
    coef[8 + lane] = A.lc.b0[lane];
    coef[16 + lane] = A.lc.b1[lane];
    coef[24 + lane] = A.lc.b2[lane];
  }
  __syncthreads();
  LaneRoof roofc;
  roofc.tab = (LdsDoubles)coef;
  roofc.cl = lane < 8 ? lane : 7;
  roofc.is_attp = lane == 1;
  roofc.is_attd = lane == 2;
  roofc.is_lm = lane == 6;
  // hand a point to the launch with twice the slots, in its bucket's list
  // (every lane stores the same index)
  auto hand_on = [&](const int pidx, const int bucket, const int wc) {
    const bool live = wc == 0 && A.take != nullptr;  // read while it is written
    if (live) __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");  // the record first
    const unsigned slot = atomicAdd(A.handed_n + wc * kHandBuckets + bucket,
                                    lane == 0 ? 1u : 0u);
    int* ent = A.handed + A.handed_off[wc] + bucket * A.hand_cap[wc] +
               __builtin_amdgcn_readfirstlane((int)slot);
    if (live)
      __hip_atomic_store(ent, pidx, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else
      *ent = pidx;
  };
  // the points of this launch: a host-side count, or the points a narrow
  // launch handed over (its bucket counts were written before this launch
  // started), taken bucket by bucket, the most remaining work first
  int n_order = A.n_order;
  if (A.n_dev != nullptr) {
    n_order = 0;
    for (int k = 0; k < kHandBuckets; ++k)
      n_order += __builtin_amdgcn_readfirstlane((int)A.n_dev[k]);
  }
  // A workgroup never needs more tickets than there are points.
  for (int taken = 0; taken <= n_order; ++taken) {
    // All lanes take part (lane 0 adds 1, the others 0) so the ticket is
    // read by the whole wave without a lane-dependent branch.
    const unsigned old = atomicAdd(A.counter, lane == 0 ? 1u : 0u);
    const int tk = __builtin_amdgcn_readfirstlane((int)old);
    if (tk >= n_order) break;
    int pos = tk;
    if (A.n_dev != nullptr) {  // bucket kHandBuckets - 1 first
      int k = kHandBuckets - 1;
      for (; k > 0; --k) {
        const int c = __builtin_amdgcn_readfirstlane((int)A.n_dev[k]);
        if (pos < c) break;
        pos -= c;
      }
      pos += k * A.hand_cap_in;
    }
    const int pidx = A.order[pos];
    if (A.claim != nullptr && NCH > 1) {  // the 64-slot launch may have taken it
      unsigned int won = 0;
      if (lane == 0) won = atomicCAS(A.claim + A.points[pidx].resume, 0u, 1u) == 0u ? 1u : 0u;
      if (__builtin_amdgcn_readfirstlane((int)won) == 0) continue;
    }
    const int bucket =
        simulate_point<NCH, MODE, SIMPLE>(A, pidx, L, Q, lane, roofc, A.n_dev != nullptr);
    if (bucket >= 0) hand_on(pidx, bucket, NCH == 1 ? 0 : 1);
  }
  if constexpr (kTail) {
    if (A.take != nullptr) {
      SlotLds<2>& L2 = *reinterpret_cast<SlotLds<2>*>(lds_slots);
      // at most every point once: each take claims a different point
      for (int guard = 0; guard <= A.hand_cap[0]; ++guard) {
        const int pidx = take_handed(A, lane);
        if (pidx < 0) break;
        const int bucket = simulate_point<2, MODE, true>(A, pidx, L2, Q, lane, roofc, true);
        if (bucket >= 0) hand_on(pidx, bucket, 1);
      }
    }
  }
}

template __global__ void sim_kernel<1, kStageOne, false>(SimArgs);
template __global__ void sim_kernel<2, kStageOne, false>(SimArgs);
template __global__ void sim_kernel<4, kStageOne, false>(SimArgs);
template __global__ void sim_kernel<1, kStageOne, true>(SimArgs);
template __global__ void sim_kernel<2, kStageOne, true>(SimArgs);
template __global__ void sim_kernel<4, kStageOne, true>(SimArgs);
template __global__ void sim_kernel<1, kStagePrefill, false>(SimArgs);
template __global__ void sim_kernel<2, kStagePrefill, false>(SimArgs);
template __global__ void sim_kernel<4, kStagePrefill, false>(SimArgs);
template __global__ void sim_kernel<1, kStageDecode, false>(SimArgs);
template __global__ void sim_kernel<2, kStageDecode, false>(SimArgs);
template __global__ void sim_kernel<4, kStageDecode, false>(SimArgs);

// ------------------------------------------------------------ statistics
// Nearest-rank percentiles of the finished requests' latencies: the k-th
// smallest values by most-significant-digit radix select (8-bit digits),
// several ranks at once (one LDS histogram each, one pass over the values per
// digit), starting at the highest digit any value uses.  One 256-thread
// workgroup per point.
template <int NK>
__device__ void select_ranks(const int64_t* v, int n, const int* ks, int top_shift,
                             int64_t* out, int* hist, int* sh) {
  uint64_t prefix[NK];
  int k[NK];
#pragma unroll
  for (int r = 0; r < NK; ++r) {
    prefix[r] = 0;
    k[r] = ks[r];
  }
  for (int shift = top_shift; shift >= 0; shift -= 8) {
    const uint64_t hi_mask = shift >= 56 ? 0ull : (~0ull << (shift + 8));
#pragma unroll
    for (int r = 0; r < NK; ++r) hist[r * 256 + threadIdx.x] = 0;
    __syncthreads();
    for (int i = threadIdx.x; i < n; i += 256) {
      const uint64_t x = (uint64_t)v[i];
      const int d = (int)((x >> shift) & 255u);
#pragma unroll
      for (int r = 0; r < NK; ++r)
        if (((x ^ prefix[r]) & hi_mask) == 0) atomicAdd(&hist[r * 256 + d], 1);
    }
    __syncthreads();
    if (threadIdx.x < NK) {
      const int r = threadIdx.x;
      int acc = 0, d = 0;
      for (; d < 255; ++d) {
        if (acc + hist[r * 256 + d] > sh[2 * NK + r]) break;
        acc += hist[r * 256 + d];
      }
      sh[2 * r] = d;
      sh[2 * r + 1] = sh[2 * NK + r] - acc;
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < NK; ++r) {
      prefix[r] |= (uint64_t)sh[2 * r] << shift;
      k[r] = sh[2 * r + 1];
    }
    __syncthreads();
    if (threadIdx.x < NK) sh[2 * NK + threadIdx.x] = k[threadIdx.x];
    __syncthreads();
  }
#pragma unroll
  for (int r = 0; r < NK; ++r) out[r] = (int64_t)prefix[r];
}

__device__ __forceinline__ int nearest_rank_index(int pct, int n) {
  return (int)(((int64_t)pct * n + 99) / 100) - 1;
}

// Latency buckets for the percentile search: 2^kSubBits per octave,
// monotone in the value (values below 2^kSubBits are their own bucket; a
// value of bit length bl > kSubBits goes to 2^kSubBits * bl + its next
// kSubBits bits below the leading one).
constexpr int kSubBits = 5;
constexpr int kSub = 1 << kSubBits;
constexpr int kBuckets = kSub * 65;
constexpr int kPerThread = (kBuckets + 255) / 256;  // buckets per thread in the prefix sum
constexpr int kCandCap = 512;    // a rank's candidates kept in LDS
__device__ __forceinline__ int lat_bucket(uint64_t v) {
  if (v < (uint64_t)kSub) return (int)v;
  const int bl = 64 - __builtin_clzll(v);
  return (bl << kSubBits) | (int)((v >> (bl - 1 - kSubBits)) & (uint64_t)(kSub - 1));
}

// For each of NR ranks (0-based, below the count), the bucket holding the
// rank-th smallest value and the rank within that bucket, from a bucket
// histogram: a block-wide prefix sum over kPerThread buckets per thread.
template <int NR>
__device__ void locate_ranks(const int* hist, const int* ks, int* wsum_sh, int* out_b,
                             int* out_k) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  int loc[kPerThread];
  int tot = 0;
#pragma unroll
  for (int i = 0; i < kPerThread; ++i) {
    const int b = tid * kPerThread + i;
    loc[i] = b < kBuckets ? hist[b] : 0;
    tot += loc[i];
  }
  const int inc = scan_i32(tot);
  if (lane == 63) wsum_sh[w] = inc;
  __syncthreads();
  int before = inc - tot;
  for (int v = 0; v < w; ++v) before += wsum_sh[v];
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    const int k = ks[r];
    if (k >= before && k < before + tot) {
      int acc = before, bsel = -1, ksel = 0;
#pragma unroll
      for (int i = 0; i < kPerThread; ++i) {
        if (bsel < 0 && k < acc + loc[i]) {
          bsel = i;
          ksel = k - acc;
        }
        acc += loc[i];
      }
      out_b[r] = tid * kPerThread + bsel;
      out_k[r] = ksel;
    }
  }
  __syncthreads();
}

// The k-th smallest (0-based) of a rank's cnt <= kCandCap candidates c[] in
// LDS, found by one wave: the candidates stay in registers, and each pass
// takes the next 8-bit digit from bit `shift` down by a 256-bin histogram
// of the candidates still in the race (the wave's own bins wh[]) and a wave
// prefix sum over the bins.  `known` holds the bits every candidate shares
// (the bucket's leading bits); shift is the top unknown bit's digit.
__device__ int64_t wave_select(const int64_t* c, int cnt, int k, uint64_t known, int shift,
                               int* wh) {
  constexpr int kPer = kCandCap / 64;
  const int lane = threadIdx.x & 63;
  uint64_t v[kPer];
  uint32_t live = 0;
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int i = u * 64 + lane;
    v[u] = i < cnt ? (uint64_t)c[i] : 0ull;
    live |= i < cnt ? 1u << u : 0u;
  }
  uint64_t prefix = known;
  for (; shift >= 0; shift -= 8) {
    *reinterpret_cast<int4*>(&wh[lane * 4]) = make_int4(0, 0, 0, 0);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int u = 0; u < kPer; ++u)
      if ((live >> u) & 1u) atomicAdd(&wh[(int)((v[u] >> shift) & 255u)], 1);
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "workgroup");
    __builtin_amdgcn_wave_barrier();
    const int4 h = *reinterpret_cast<const int4*>(&wh[lane * 4]);
    const int sum = (h.x + h.y) + (h.z + h.w);
    const int inc = scan_i32(sum);
    const int before = inc - sum;
    // the one lane whose four bins hold the k-th live candidate
    const uint64_t m = ballot(k >= before && k < inc);
    const int L = m != 0 ? (int)__builtin_ctzll(m) : 0;
    int kk = k - before, d = lane * 4;
    if (kk >= h.x) {
      kk -= h.x;
      ++d;
      if (kk >= h.y) {
        kk -= h.y;
        ++d;
        if (kk >= h.z) {
          kk -= h.z;
          ++d;
        }
      }
    }
    d = rdl(d, L);
    k = rdl(kk, L);
    prefix |= (uint64_t)d << shift;
#pragma unroll
    for (int u = 0; u < kPer; ++u)
      if ((int)((v[u] >> shift) & 255u) != d) live &= ~(1u << u);
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "workgroup");
    __builtin_amdgcn_wave_barrier();
  }
  return (int64_t)prefix;
}

// The point's request statistics from its request records, one 256-thread
// workgroup per point: latency sums (TTFT = first token - arrival, E2E =
// finish - arrival, TPOT numerator = finish - first token), the largest E2E,
// the last finish, the SLO counts (Sec. IV-B), the digest over finished and
// rejected records, then nearest-rank percentiles of the finished requests'
// latencies.  The record pass (two records per thread in flight) also
// builds a bucket histogram of each latency and copies the latencies
// densely to HBM; the buckets of the ranks are located, one pass over the
// dense copy gathers each rank's bucket into LDS (over the histograms,
// which are done by then), and one wave per rank selects the exact value
// there (a bucket too full for LDS is selected by the whole workgroup in
// radix passes over the dense copy instead).  With pad_pending (per-request
// output) the row's entries past the trace also get "pending" records.
constexpr int kStatsBatch = 2;  // records per thread in flight (5 waves per SIMD: 96 VGPRs)
constexpr int kStatsUnion =
    (2 * kBuckets * 4 > 5 * kCandCap * 8) ? 2 * kBuckets * 4 : 5 * kCandCap * 8;
__global__ __launch_bounds__(256, 5) void stats_kernel(ts_req_result* rec, const TraceRec* recs,
                                                    const PointInfo* pinfo,
                                                    ts_point_result* res, int64_t* e2e,
                                                    int64_t* ttft, int max_n, int n_points,
                                                    int64_t slo_ttft_ns, int64_t slo_tpot_ns,
                                                    int pad_pending) {
  // the latency histograms (E2E buckets, then TTFT buckets) until the ranks'
  // buckets are located, then the 5 ranks' candidates
  __shared__ __attribute__((aligned(16))) unsigned char ubuf[kStatsUnion];
  int* const hist = reinterpret_cast<int*>(ubuf);
  int64_t(*const cand)[kCandCap] = reinterpret_cast<int64_t(*)[kCandCap]>(ubuf);
  __shared__ __attribute__((aligned(16))) int whist[4][256];  // select bins, per wave
  __shared__ int sh[16];
  __shared__ int rb[5], rk[5];                 // rank bucket, rank within it
  __shared__ int ks[5];                        // the ranks (0-based)
  __shared__ int64_t r5[5];                    // the percentiles
  __shared__ unsigned int ccount[5];
  __shared__ unsigned long long acc_sum[4];  // TTFT, E2E, TPOT numerator, digest
  __shared__ long long acc_max[2];           // largest E2E, last finish
  __shared__ unsigned int acc_cnt[3];        // finished (dense index), slo_ok, slo_tpot_ok
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  for (int p = blockIdx.x; p < n_points; p += gridDim.x) {
    const PointInfo pi = pinfo[p];
    ts_req_result* R = rec + (size_t)p * (size_t)max_n;
    int64_t* ve = e2e + (size_t)p * (size_t)max_n;
    int64_t* vt = ttft + (size_t)p * (size_t)max_n;
    if (tid < 4) acc_sum[tid] = 0;
    if (tid < 2) acc_max[tid] = -1;
    if (tid < 3) acc_cnt[tid] = 0;
    if (tid < 5) ccount[tid] = 0;
    for (int b = tid; b < 2 * kBuckets; b += 256) hist[b] = 0;
    __syncthreads();
    uint64_t s_tt = 0, s_ee = 0, s_tp = 0, dig = 0;
    int64_t mx = -1, lf = -1;
    unsigned int n_slo = 0, n_slo_tpot = 0;
    for (int g0 = 0; g0 < pi.n; g0 += 256 * kStatsBatch) {
      // whole waves, so the ballots see every lane
      ts_req_result rr[kStatsBatch];
      int64_t arr[kStatsBatch];
#pragma unroll
      for (int u = 0; u < kStatsBatch; ++u) {
        const int g = g0 + u * 256 + tid;
        if (g < pi.n) {
          rr[u] = R[g];
          arr[u] = recs[pi.trace_off + g].arrival_ns;
        } else {
          rr[u].admit_ns = -1; rr[u].first_token_ns = -1; rr[u].finish_ns = -1;
          rr[u].max_gap_ns = 0; rr[u].n_preempt = 0; rr[u].status = TS_REQ_PENDING;
          arr[u] = 0;
        }
      }
#pragma unroll
      for (int u = 0; u < kStatsBatch; ++u) {
        const ts_req_result& r = rr[u];
        const int g = g0 + u * 256 + tid;
        const bool done = r.status == TS_REQ_DONE;
        int64_t tt = 0, ee = 0;
        if (done) {
          tt = r.first_token_ns - arr[u];
          ee = r.finish_ns - arr[u];
          s_tt += (uint64_t)tt;
          s_ee += (uint64_t)ee;
          s_tp += (uint64_t)(r.finish_ns - r.first_token_ns);
          mx = ee > mx ? ee : mx;
          lf = r.finish_ns > lf ? r.finish_ns : lf;
          n_slo += (tt <= slo_ttft_ns && r.max_gap_ns <= slo_tpot_ns) ? 1u : 0u;
          n_slo_tpot += r.max_gap_ns <= slo_tpot_ns ? 1u : 0u;
          atomicAdd(&hist[lat_bucket((uint64_t)ee)], 1);
          atomicAdd(&hist[kBuckets + lat_bucket((uint64_t)tt)], 1);
        }
        // dense positions: one counter update per wave
        const uint64_t dm = ballot(done);
        unsigned int base = 0;
        if (lane == 0 && dm != 0) base = atomicAdd(&acc_cnt[0], (unsigned int)popc(dm));
        base = (unsigned int)__builtin_amdgcn_readfirstlane((int)base);
        if (done) {
          const unsigned int pos = base + (unsigned int)rank_below(dm);
          ve[pos] = ee;
          vt[pos] = tt;
        }
        if (done || r.status == TS_REQ_REJECTED)
          dig += record_hash(g, r.admit_ns, r.first_token_ns, r.finish_ns, r.max_gap_ns,
                             r.n_preempt, r.status);
      }
    }
    if (pad_pending) {
      ts_req_result o;
      o.admit_ns = -1; o.first_token_ns = -1; o.finish_ns = -1; o.max_gap_ns = 0;
      o.n_preempt = 0; o.status = TS_REQ_PENDING;
      for (int g = pi.n + tid; g < max_n; g += 256) R[g] = o;
    }
    atomicAdd(&acc_sum[0], (unsigned long long)s_tt);
    atomicAdd(&acc_sum[1], (unsigned long long)s_ee);
    atomicAdd(&acc_sum[2], (unsigned long long)s_tp);
    atomicAdd(&acc_sum[3], (unsigned long long)dig);
    atomicMax(&acc_max[0], (long long)mx);
    atomicMax(&acc_max[1], (long long)lf);
    atomicAdd(&acc_cnt[1], n_slo);
    atomicAdd(&acc_cnt[2], n_slo_tpot);
    __syncthreads();
    const int n = (int)acc_cnt[0];
    const int64_t max_e2e = acc_max[0];
    if (tid < 5) r5[tid] = -1;
    if (n > 0) {
      // ranks: p50, p90, p99 of E2E, then p50, p99 of TTFT
      if (tid < 5) ks[tid] = nearest_rank_index(tid == 0 || tid == 3 ? 50 : (tid == 1 ? 90 : 99), n);
      __syncthreads();
      locate_ranks<3>(hist, ks, sh, rb, rk);
      locate_ranks<2>(hist + kBuckets, ks + 3, sh, rb + 3, rk + 3);
      // (the histograms are dead from here: their LDS takes the candidates)
      // gather each rank's bucket
      for (int i0 = 0; i0 < n; i0 += 256 * kStatsBatch) {
        int64_t ev[kStatsBatch], tv[kStatsBatch];
#pragma unroll
        for (int u = 0; u < kStatsBatch; ++u) {
          const int i = i0 + u * 256 + tid;
          ev[u] = i < n ? ve[i] : -1;
          tv[u] = i < n ? vt[i] : -1;
        }
#pragma unroll
        for (int u = 0; u < kStatsBatch; ++u) {
          if (ev[u] < 0) continue;  // past the count (latencies are >= 0)
          const int be = lat_bucket((uint64_t)ev[u]), bt = lat_bucket((uint64_t)tv[u]);
#pragma unroll
          for (int r = 0; r < 5; ++r) {
            if ((r < 3 ? be : bt) == rb[r]) {
              const unsigned int c = atomicAdd(&ccount[r], 1u);
              if (c < (unsigned int)kCandCap) cand[r][c] = r < 3 ? ev[u] : tv[u];
            }
          }
        }
      }
      __syncthreads();
      // one wave per rank whose bucket fits in LDS (wave 0 also takes rank 4)
      for (int r = wv; r < 5; r += 4) {
        const int cnt = (int)ccount[r];
        const int b = rb[r];
        if (b < kSub) {  // a bucket of one value
          if (lane == 0) r5[r] = b;
          continue;
        }
        if (cnt > kCandCap) continue;
        // values of bit length bl whose leading 1 + kSubBits bits are the
        // bucket's: bl - 1 - kSubBits bits below them are unknown
        const int bl = b >> kSubBits;
        const int unk = bl - 1 - kSubBits;
        const uint64_t known = (uint64_t)(kSub | (b & (kSub - 1))) << unk;
        const int64_t v = unk > 0 ? wave_select(cand[r], cnt, rk[r], known, ((unk - 1) / 8) * 8,
                                                whist[wv])
                                  : (int64_t)known;
        if (lane == 0) r5[r] = v;
      }
      __syncthreads();
      // every latency lies in [0, max_e2e] (a first token never comes after
      // the finish): digits above the top one are zero for all of them
      const uint64_t m = (uint64_t)max_e2e;
      const int bits = m == 0 ? 1 : 64 - __builtin_clzll(m);
      const int top_all = ((bits - 1) / 8) * 8;
#pragma unroll 1
      for (int r = 0; r < 5; ++r) {
        if (rb[r] < kSub || (int)ccount[r] <= kCandCap) continue;
        if (tid == 0) sh[2] = ks[r];
        __syncthreads();
        const int kk = ks[r];
        int64_t v;
        select_ranks<1>(r < 3 ? ve : vt, n, &kk, top_all, &v, &whist[0][0], sh);
        if (tid == 0) r5[r] = v;
      }
    }
    __syncthreads();
    if (tid == 0) {
      ts_point_result& o = res[p];
      o.sum_ttft_ns = (int64_t)acc_sum[0];
      o.sum_e2e_ns = (int64_t)acc_sum[1];
      o.sum_tpot_num_ns = (int64_t)acc_sum[2];
      o.digest = acc_sum[3];
      o.max_e2e_ns = max_e2e;
      o.last_finish_ns = acc_max[1];
      o.slo_ok = (int64_t)acc_cnt[1];
      o.slo_tpot_ok = (int64_t)acc_cnt[2];
      o.p50_e2e_ns = r5[0];
      o.p90_e2e_ns = r5[1];
      o.p99_e2e_ns = r5[2];
      o.p50_ttft_ns = r5[3];
      o.p99_ttft_ns = r5[4];
    }
    __syncthreads();
  }
}

// ------------------------------------------------------------ disaggregated points
// Decode device v of a point receives its requests in (arrival of the KV,
// request index) order.  Each prefill device's sub-list (w, v) is already in
// that order (a prefill device completes prefills in admission order and its
// link delivers them in that order), so a request's place is its index in its
// own sub-list plus, for every other sub-list, how many entries come before
// it there (a binary search).  One 256-thread workgroup per (point, decode
// device); it also sets the decode device's request count.
__global__ __launch_bounds__(256) void pd_merge_kernel(const PdAux* aux, int n_aux,
                                                       const int64_t* sub_a2,
                                                       const int32_t* sub_gid, TraceRec* recs,
                                                       int32_t* gids, DevPoint* units) {
  for (int b = blockIdx.x; b < n_aux * kMaxDev; b += gridDim.x) {
    const PdAux& X = aux[b / kMaxDev];
    const int v = b % kMaxDev;
    if (v >= X.n_d) continue;
    int total = 0;
    for (int w = 0; w < X.n_p; ++w) {
      const int cnt = X.sub_cnt[w * kMaxDev + v], off = X.sub_off[w * kMaxDev + v];
      total += cnt;
      for (int k = threadIdx.x; k < cnt; k += blockDim.x) {
        const int64_t a = sub_a2[off + k];
        const int g = sub_gid[off + k];
        int rank = k;
        for (int u = 0; u < X.n_p; ++u) {
          if (u == w) continue;
          const int uo = X.sub_off[u * kMaxDev + v];
          int lo = 0, hi = X.sub_cnt[u * kMaxDev + v];
          while (lo < hi) {  // entries of sub-list u before (a, g)
            const int mid = (lo + hi) >> 1;
            const int64_t am = sub_a2[uo + mid];
            if (am < a || (am == a && sub_gid[uo + mid] < g)) lo = mid + 1;
            else hi = mid;
          }
          rank += lo;
        }
        const TraceRec o = recs[X.trace_off + g];
        TraceRec r;
        r.arrival_ns = a;
        r.prompt = o.prompt;
        r.output = o.output;
        recs[X.dec_off[v] + rank] = r;
        gids[X.dec_off[v] + rank] = g;
      }
    }
    if (threadIdx.x == 0) units[X.dec_unit0 + v].n = total;
  }
}

// A disaggregated point's record from its devices' records: finished
// requests from the decode devices, rejections from the prefill devices,
// iterations, tokens and the used-block integral (prefill devices first,
// then decode devices, in index order) over all devices, the block peak of
// the busiest decode device.  The latency sums, SLO counts, percentiles and
// digest come after, from the point's request records.  One thread per point.
__global__ __launch_bounds__(256) void pd_combine_kernel(const PdAux* aux, int n_aux,
                                                         ts_point_result* res,
                                                         const TraceRec* recs) {
  for (int b = blockIdx.x * blockDim.x + threadIdx.x; b < n_aux; b += gridDim.x * blockDim.x) {
    const PdAux& X = aux[b];
    ts_point_result o;
    const int nu = X.n_p + X.n_d;
    o.status = TS_POINT_OK;
    o.n_done = 0; o.n_rejected = 0; o.num_blocks = X.num_blocks_d;
    o.n_iters = 0; o.n_preempt = 0; o.prefill_tokens = 0; o.decode_tokens = 0;
    o.peak_used_blocks = 0;
    o.first_arrival_ns = X.n > 0 ? recs[X.trace_off].arrival_ns : -1;
    o.last_finish_ns = -1;
    o.sum_ttft_ns = 0; o.sum_e2e_ns = 0; o.max_e2e_ns = -1; o.sum_tpot_num_ns = 0;
    o.p50_e2e_ns = o.p90_e2e_ns = o.p99_e2e_ns = -1;
    o.p50_ttft_ns = o.p99_ttft_ns = -1;
    o.slo_ok = 0; o.slo_tpot_ok = 0;
    o.used_block_ns = 0.0;
    o.digest = 0;
    for (int u = 0; u < nu; ++u) {
      const ts_point_result& r = res[X.res0 + u];
      const bool dec = u >= X.n_p;
      o.status = r.status > o.status ? r.status : o.status;
      o.n_iters += r.n_iters;
      o.n_preempt += r.n_preempt;
      o.prefill_tokens += r.prefill_tokens;
      o.decode_tokens += r.decode_tokens;
      o.used_block_ns = o.used_block_ns + r.used_block_ns;
      if (dec) {
        o.n_done += r.n_done;
        o.peak_used_blocks = r.peak_used_blocks > o.peak_used_blocks ? r.peak_used_blocks
                                                                      : o.peak_used_blocks;
      } else {
        o.n_rejected += r.n_rejected;
      }
    }
    if (X.no_kv) o.status = TS_POINT_NO_KV;
    res[X.point] = o;
  }
}

// Work-queue counters are cleared by a kernel (no memset node in a captured
// stream).
__global__ void reset_counters_kernel(unsigned int* c, int n, unsigned long long* w, int nw) {
  if ((int)threadIdx.x < n) c[threadIdx.x] = 0u;
  if ((int)threadIdx.x < nw) w[threadIdx.x] = 0ull;
}

__global__ void fill_kernel(int32_t* p, int n, int32_t v) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = v;
}

}  // namespace tsw
