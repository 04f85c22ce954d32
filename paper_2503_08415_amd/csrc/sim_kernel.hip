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
//     compaction through LDS.
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

// DPP move with zero for lanes whose source is outside the row / not selected.
template <int CTRL, int ROWS>
__device__ __forceinline__ int dpp0(int v) {
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
  v += dpp0<0x111, 0xf>(v);
  v += dpp0<0x112, 0xf>(v);
  v += dpp0<0x114, 0xf>(v);
  v += dpp0<0x118, 0xf>(v);
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
// MurmurHash3's 64-bit finaliser chained over a request record.
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
  uint64_t h = fmix64((uint64_t)idx + 0x9e3779b97f4a7c15ULL);
  h = fmix64(h ^ (uint64_t)admit);
  h = fmix64(h ^ (uint64_t)first);
  h = fmix64(h ^ (uint64_t)finish);
  h = fmix64(h ^ (uint64_t)gap);
  h = fmix64(h ^ (((uint64_t)(uint32_t)npre << 32) | (uint32_t)status));
  return h;
}

// ------------------------------------------------------------ roofline
// Per operator: max(FLOPs / peak, bytes / bandwidth) in ns; both counts are
// exact integers below 2^53, so the int64 -> double conversion is exact.
__device__ __forceinline__ double roof(int64_t flops, int64_t bytes, double iF, double iB) {
  const double tf = (double)flops * iF;
  const double tb = (double)bytes * iB;
  return tf > tb ? tf : tb;
}

__device__ __forceinline__ int64_t iteration_ns(const CostCoef& C, double iF, double iB,
                                                int64_t T, int64_t TP, int64_t AP, int64_t CP,
                                                int64_t nD, int64_t CD, int64_t R) {
  const double t1 = roof(C.f_qkv * T, C.b_qkv0 + C.b_qkv * T, iF, iB);
  const double t2 = roof(C.f_attp * AP, C.b_attp_c * CP + C.b_attp_t * TP, iF, iB);
  const double t3 = roof(C.f_attd * CD, C.b_attd_c * CD + C.b_attd_n * nD, iF, iB);
  const double t4 = roof(C.f_out * T, C.b_out0 + C.b_out * T, iF, iB);
  const double t5 = roof(C.f_up * T, C.b_up0 + C.b_up * T, iF, iB);
  const double t6 = roof(C.f_dn * T, C.b_dn0 + C.b_dn * T, iF, iB);
  const double t7 = R > 0 ? roof(C.f_lm * R, C.b_lm0 + C.b_lm * R, iF, iB) : 0.0;
  double layer = t1;
  layer = layer + t2;
  layer = layer + t3;
  layer = layer + t4;
  layer = layer + t5;
  layer = layer + t6;
  double total = C.n_layers * layer;
  total = total + t7;
  const int64_t ns = (int64_t)ceil(total);
  return ns < 1 ? 1 : ns;
}

// Admission staging: one entry per admitted candidate of a window.
struct StageSlot {
  int32_t id, tgt, rem, npre, q, alloc, room, pad;
  int64_t admit, first, last, gap;
};

// Stable compaction of one per-slot field through LDS scratch.
template <int NCH, typename Tv>
__device__ __forceinline__ void compact_field(Tv (&f)[NCH], const bool (&keep)[NCH],
                                              const int (&pos)[NCH], Tv* scratch, int lane) {
#pragma unroll
  for (int j = 0; j < NCH; ++j)
    if (keep[j]) scratch[pos[j]] = f[j];
  __syncthreads();
#pragma unroll
  for (int j = 0; j < NCH; ++j) f[j] = scratch[j * 64 + lane];
  __syncthreads();
}

// ------------------------------------------------------------ one point
template <int NCH>
__device__ __forceinline__ void simulate_point(const SimArgs& A, const int pidx,
                                               StageSlot* stage, int64_t* scratch,
                                               QEntry* Q, const int lane) {
  const DevPoint P = A.points[pidx];
  const TraceRec* __restrict__ rec = A.recs + P.trace_off;
  const int N = P.n, NB = P.num_blocks, B = P.block, M = P.max_batch, K = P.chunk;
  const bool unlimited = (K == 0);
  const int64_t cap_tok = P.cap_tokens;
  const double iF = P.inv_flops_ns, iB = P.inv_bw_ns;
  const int oi = P.out_index;
  ts_req_result* RR = A.req ? A.req + (size_t)oi * (size_t)A.max_n : nullptr;
  int64_t* E2E = A.e2e + (size_t)oi * (size_t)A.max_n;
  int64_t* TTFT = A.ttft + (size_t)oi * (size_t)A.max_n;

  // per-lane accumulators of finished / rejected requests
  int64_t acc_ttft = 0, acc_e2e = 0, acc_tpot = 0, acc_maxe2e = 0, acc_last = 0;
  int64_t acc_slo = 0;
  uint64_t acc_dig = 0;
  int n_rej = 0;

  // Requests that could never fit are rejected up front.
  if (P.may_reject) {
    for (int base = 0; base < N; base += 64) {
      const int i = base + lane;
      bool rj = false;
      if (i < N) {
        const TraceRec r = rec[i];
        rj = (int64_t)r.prompt + (int64_t)r.output > cap_tok;
      }
      if (rj) {
        acc_dig += record_hash(i, -1, -1, -1, 0, 0, TS_REQ_REJECTED);
        if (RR) {
          ts_req_result o;
          o.admit_ns = -1; o.first_token_ns = -1; o.finish_ns = -1; o.max_gap_ns = 0;
          o.n_preempt = 0; o.status = TS_REQ_REJECTED;
          RR[i] = o;
        }
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
  int w_p = 0, w_o = 0;
  if (lane < N) {
    const TraceRec r = rec[lane];
    w_arr = r.arrival_ns; w_p = r.prompt; w_o = r.output;
  }

  int s_ctx[NCH], s_tgt[NCH], s_rem[NCH], s_room[NCH], s_alloc[NCH], s_id[NCH], s_npre[NCH];
  int64_t s_admit[NCH], s_first[NCH], s_last[NCH], s_gap[NCH];
  int q[NCH];
  bool act[NCH], dec[NCH];
#pragma unroll
  for (int j = 0; j < NCH; ++j) {
    s_ctx[j] = s_tgt[j] = s_rem[j] = s_room[j] = s_alloc[j] = s_id[j] = s_npre[j] = 0;
    s_admit[j] = s_first[j] = s_last[j] = s_gap[j] = 0;
    q[j] = 0;
    act[j] = dec[j] = false;
  }

  const uint64_t clock0 = A.time_limit_ticks ? __builtin_amdgcn_s_memrealtime() : 0;
  while (status == TS_POINT_OK) {
    // watchdog: a point running longer than the wall-clock limit stops
    if (A.time_limit_ticks != 0 && (n_iters & 255) == 0 &&
        __builtin_amdgcn_s_memrealtime() - clock0 > A.time_limit_ticks) {
      status = TS_POINT_TIME_LIMIT;
      break;
    }
    // ---- 1. intake: every request with arrival <= t joins the waiting set
    int guard = N / 64 + 2;  // window passes are bounded by the trace length
    while (next < N && --guard >= 0) {
      const uint64_t m = ballot(w_arr <= t);  // arrivals are sorted: a lane prefix
      const int cnt = popc(m);
      const int nn = wbase + cnt;
      if (nn > next) {
        int add = nn - next;
        if (P.may_reject) {
          const bool rj = lane >= next - wbase && lane < cnt &&
                          (int64_t)w_p + (int64_t)w_o > cap_tok;
          add -= popc(ballot(rj));
        }
        if (npre == 0 && nwait == 0) head_need = -1;
        nwait += add;
        next = nn;
      }
      if (cnt == 64 && nn < N) {
        wbase = nn;
        w_arr = INT64_MAX; w_p = 0; w_o = 0;
        if (wbase + lane < N) {
          const TraceRec r = rec[wbase + lane];
          w_arr = r.arrival_ns; w_p = r.prompt; w_o = r.output;
        }
        continue;
      }
      break;
    }
    if (nwait == 0) next_new = next;

    // ---- 2. idle: jump to the next arrival, or finish
    if (nrun == 0 && npre == 0 && nwait == 0) {
      if (next >= N) break;
      t = rdl64(w_arr, next - wbase);
      continue;
    }
    if (n_iters >= A.iter_cap) {
      status = TS_POINT_ITER_LIMIT;
      break;
    }

    // ---- 3. reserve a block for decodes crossing a block boundary
    int nneed = 0;
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
      act[j] = (j * 64 + lane) < nrun;
      dec[j] = act[j] && s_ctx[j] >= s_tgt[j];
      nneed += popc(ballot(dec[j] && s_room[j] == 0));
    }
    bool preempted = false;
    if (nneed <= freeb) {
      freeb -= nneed;
#pragma unroll
      for (int j = 0; j < NCH; ++j)
        if (dec[j] && s_room[j] == 0) { s_alloc[j] += 1; s_room[j] += B; }
    } else {
      // Recompute preemption from the tail: keep the longest prefix of slots
      // whose held + needed blocks fit in the whole budget.
      int carry = 0, k = 0, kept = 0;
      bool keep[NCH];
#pragma unroll
      for (int j = 0; j < NCH; ++j) {
        const int need = (dec[j] && s_room[j] == 0) ? 1 : 0;
        const int v = act[j] ? s_alloc[j] + need : 0;
        const int S = scan_i32(v) + carry;
        keep[j] = act[j] && S <= NB;
        k += popc(ballot(keep[j]));
        kept += wsum(keep[j] ? v : 0);
        carry = rdl(S, 63);
      }
      freeb = NB - kept;
      const int nv = nrun - k;
      qhead = (qhead - nv) & (kQueueCap - 1);
#pragma unroll
      for (int j = 0; j < NCH; ++j) {
        const int s = j * 64 + lane;
        if (keep[j]) {
          if (dec[j] && s_room[j] == 0) { s_alloc[j] += 1; s_room[j] += B; }
        } else if (act[j]) {
          // victims keep admission order at the front of the waiting queue:
          // they are older than every request still waiting
          QEntry e;
          e.id = s_id[j];
          e.target = s_ctx[j] > s_tgt[j] ? s_ctx[j] : s_tgt[j];  // prompt + tokens decoded
          e.rem = s_rem[j];
          e.n_pre = s_npre[j] + 1;
          e.admit = s_admit[j];
          e.first = s_first[j];
          e.last = s_last[j];
          e.gap = s_gap[j];
          Q[(qhead + s - k) & (kQueueCap - 1)] = e;
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
      npre += nv;
      n_pre_tot += nv;
      nrun = k;
      preempted = true;
      head_need = -1;
    }

    // ---- 4. token budget: decodes one token, running prefills share the rest
    int R = 0;
    {
      int ndec = 0;
#pragma unroll
      for (int j = 0; j < NCH; ++j) {
        act[j] = (j * 64 + lane) < nrun;
        dec[j] = act[j] && s_ctx[j] >= s_tgt[j];
        ndec += popc(ballot(dec[j]));
      }
      if (!unlimited) {
        R = K - ndec;
        int carry = 0;
#pragma unroll
        for (int j = 0; j < NCH; ++j) {
          const bool pf = act[j] && !dec[j];
          const int left = pf ? s_tgt[j] - s_ctx[j] : 0;
          const int S = scan_i32(left);
          int avail = R - (S - left + carry);
          avail = avail < 0 ? 0 : avail;
          q[j] = dec[j] ? 1 : (pf ? (left < avail ? left : avail) : 0);
          carry += rdl(S, 63);
        }
        R = R - carry;
        if (R < 0) R = 0;
      } else {
#pragma unroll
        for (int j = 0; j < NCH; ++j)
          q[j] = dec[j] ? 1 : (act[j] ? s_tgt[j] - s_ctx[j] : 0);
      }
    }

    // ---- 5. FCFS admission over 64-candidate windows (none after preemption)
    if (!preempted) {
      int guard = M + N / 64 + 4;  // each pass admits or advances a window
      while (nrun < M && (unlimited || R > 0) && (npre > 0 || nwait > 0) && --guard >= 0) {
        if (head_need >= 0 && head_need > freeb) break;
        const bool fromq = npre > 0;
        bool valid;
        int c_id, c_tgt, c_rem, c_npre;
        int64_t c_admit, c_first, c_last, c_gap;
        if (fromq) {
          valid = lane < npre;
          __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
          if (valid) {
            const QEntry e = Q[(qhead + lane) & (kQueueCap - 1)];
            c_id = e.id; c_tgt = e.target; c_rem = e.rem; c_npre = e.n_pre;
            c_admit = e.admit; c_first = e.first; c_last = e.last; c_gap = e.gap;
          } else {
            c_id = 0; c_tgt = 1; c_rem = 1; c_npre = 0;
            c_admit = -1; c_first = -1; c_last = -1; c_gap = 0;
          }
        } else {
          const int idx = next_new + lane;
          valid = idx < next;
          c_id = idx; c_npre = 0; c_admit = -1; c_first = -1; c_last = -1; c_gap = 0;
          c_tgt = 1; c_rem = 1;
          if (valid) {
            const TraceRec r = rec[idx];
            c_tgt = r.prompt;
            c_rem = r.output;
            if (P.may_reject && (int64_t)r.prompt + (int64_t)r.output > cap_tok) valid = false;
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
        const int need = valid ? (c_tgt + B - 1) / B : 0;
        const int SN = scan_i32(need);
        const int tq = valid ? c_tgt : 0;
        const int ET = scan_i32(tq) - tq;
        const int slots_left = M - nrun;
        const bool adm = valid && rank < slots_left && SN <= freeb && (unlimited || ET < R);
        const uint64_t am = ballot(adm);
        const int a = popc(am);
        if (a == 0) {
          head_need = rdl(need, (int)__builtin_ctzll(vm));
          break;
        }
        const int last_lane = 63 - (int)__builtin_clzll(am);
        const int qv = unlimited ? c_tgt : (c_tgt < R - ET ? c_tgt : R - ET);
        freeb -= rdl(SN, last_lane);
        if (!unlimited) R -= wsum(adm ? qv : 0);
        if (adm) {
          StageSlot st;
          st.id = c_id; st.tgt = c_tgt; st.rem = c_rem; st.npre = c_npre; st.q = qv;
          st.alloc = need; st.room = need * B - c_tgt; st.pad = 0;
          st.admit = c_admit < 0 ? t : c_admit;
          st.first = c_first; st.last = c_last; st.gap = c_gap;
          stage[rank] = st;
        }
        __syncthreads();
#pragma unroll
        for (int j = 0; j < NCH; ++j) {
          const int s = j * 64 + lane;
          if (s >= nrun && s < nrun + a) {
            const StageSlot st = stage[s - nrun];
            s_id[j] = st.id; s_ctx[j] = 0; s_tgt[j] = st.tgt; s_rem[j] = st.rem;
            s_npre[j] = st.npre; q[j] = st.q; s_alloc[j] = st.alloc; s_room[j] = st.room;
            s_admit[j] = st.admit; s_first[j] = st.first; s_last[j] = st.last;
            s_gap[j] = st.gap;
          }
        }
        __syncthreads();
        nrun += a;
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
    }

    // ---- 6. batch sums (wave reductions) and the roofline iteration time
    int l_nd = 0, l_cd = 0, l_r = 0, l_tp = 0, l_cp = 0;
    int64_t l_ap = 0;
    bool l_pf = false;
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
      act[j] = (j * 64 + lane) < nrun;
      dec[j] = act[j] && s_ctx[j] >= s_tgt[j];
      const int c0 = s_ctx[j];
      if (dec[j]) {
        l_nd += 1;
        l_cd += c0 + 1;
        l_r += 1;
      } else if (act[j] && q[j] > 0) {
        const int qq = q[j];
        l_tp += qq;
        l_ap += (int64_t)qq * c0 + ((int64_t)qq * (qq + 1)) / 2;
        l_cp += c0 + qq;
        if (c0 + qq == s_tgt[j] && s_first[j] < 0) l_r += 1;  // emits its first token
        l_pf = true;
      }
    }
    const int nD = wsum(l_nd);
    const int CD = wsum(l_cd);
    const int Rl = wsum(l_r);
    int TP = 0, CP = 0;
    int64_t AP = 0;
    if (ballot(l_pf) != 0) {
      TP = wsum(l_tp);
      CP = wsum(l_cp);
      AP = wsum64(l_ap);
    }
    const int64_t iter_ns = iteration_ns(A.coef, iF, iB, (int64_t)nD + TP, TP, AP, CP, nD, CD, Rl);

    // ---- 7. advance the clock and every scheduled request
    const int64_t t_end = t + iter_ns;
    const int used = NB - freeb;
    if (used > peak) peak = used;
    ubns = ubns + (double)used * (double)iter_ns;
    ++n_iters;
    pf_tok += TP;
    dec_tok += nD;

    bool fin[NCH];
    uint64_t fm[NCH];
    int nfin = 0;
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
      fin[j] = false;
      if (dec[j]) {
        s_ctx[j] += 1;
        s_rem[j] -= 1;
        s_room[j] -= 1;
        const int64_t g = t_end - s_last[j];
        if (g > s_gap[j]) s_gap[j] = g;
        s_last[j] = t_end;
        fin[j] = s_rem[j] == 0;
      } else if (act[j] && q[j] > 0) {
        s_ctx[j] += q[j];
        if (s_ctx[j] == s_tgt[j] && s_first[j] < 0) {  // the full prefill emits a token
          s_first[j] = t_end;
          s_last[j] = t_end;
        }
      }
      fm[j] = ballot(fin[j]);
      nfin += popc(fm[j]);
    }
    if (nfin > 0) {
      int base = n_done;
      int l_freed = 0;
#pragma unroll
      for (int j = 0; j < NCH; ++j) {
        if (fin[j]) {
          const int id = s_id[j];
          const int64_t arr = rec[id].arrival_ns;
          const int64_t tt = s_first[j] - arr;
          const int64_t ee = t_end - arr;
          acc_ttft += tt;
          acc_e2e += ee;
          acc_tpot += t_end - s_first[j];
          acc_maxe2e = ee > acc_maxe2e ? ee : acc_maxe2e;
          acc_last = t_end;
          if (tt <= A.slo_ttft_ns && s_gap[j] <= A.slo_tpot_ns) acc_slo += 1;
          acc_dig += record_hash(id, s_admit[j], s_first[j], t_end, s_gap[j], s_npre[j],
                                 TS_REQ_DONE);
          if (RR) {
            ts_req_result o;
            o.admit_ns = s_admit[j]; o.first_token_ns = s_first[j]; o.finish_ns = t_end;
            o.max_gap_ns = s_gap[j]; o.n_preempt = s_npre[j]; o.status = TS_REQ_DONE;
            RR[id] = o;
          }
          const int pos = base + rank_below(fm[j]);
          E2E[pos] = ee;
          TTFT[pos] = tt;
          l_freed += s_alloc[j];
        }
        base += popc(fm[j]);
      }
      freeb += wsum(l_freed);
      n_done += nfin;
      // stable compaction of the survivors
      bool keep[NCH];
      int pos[NCH];
      int off = 0;
#pragma unroll
      for (int j = 0; j < NCH; ++j) {
        keep[j] = act[j] && !fin[j];
        const uint64_t km = ballot(keep[j]);
        pos[j] = off + rank_below(km);
        off += popc(km);
      }
      int* s32 = reinterpret_cast<int*>(scratch);
      compact_field<NCH, int>(s_ctx, keep, pos, s32, lane);
      compact_field<NCH, int>(s_tgt, keep, pos, s32, lane);
      compact_field<NCH, int>(s_rem, keep, pos, s32, lane);
      compact_field<NCH, int>(s_room, keep, pos, s32, lane);
      compact_field<NCH, int>(s_alloc, keep, pos, s32, lane);
      compact_field<NCH, int>(s_id, keep, pos, s32, lane);
      compact_field<NCH, int>(s_npre, keep, pos, s32, lane);
      compact_field<NCH, int64_t>(s_admit, keep, pos, scratch, lane);
      compact_field<NCH, int64_t>(s_first, keep, pos, scratch, lane);
      compact_field<NCH, int64_t>(s_last, keep, pos, scratch, lane);
      compact_field<NCH, int64_t>(s_gap, keep, pos, scratch, lane);
      nrun -= nfin;
    }
    t = t_end;
  }

  // ---- per-point results (percentiles are filled by the statistics kernel)
  const int64_t sum_ttft = wsum64(acc_ttft);
  const int64_t sum_e2e = wsum64(acc_e2e);
  const int64_t sum_tpot = wsum64(acc_tpot);
  const int64_t slo_ok = wsum64(acc_slo);
  const int64_t max_e2e = wmax64_nonneg(acc_maxe2e);
  const int64_t last_fin = wmax64_nonneg(acc_last);
  const uint64_t digest = wsum_u64(acc_dig);
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
    o.last_finish_ns = n_done > 0 ? last_fin : -1;
    o.sum_ttft_ns = sum_ttft;
    o.sum_e2e_ns = sum_e2e;
    o.max_e2e_ns = n_done > 0 ? max_e2e : -1;
    o.sum_tpot_num_ns = sum_tpot;
    o.p50_e2e_ns = o.p90_e2e_ns = o.p99_e2e_ns = -1;
    o.p50_ttft_ns = o.p99_ttft_ns = -1;
    o.slo_ok = slo_ok;
    o.used_block_ns = ubns;
    o.digest = digest;
    A.res[oi] = o;
  }
}

// Persistent grid: each wave64 workgroup takes the next point from a ticket
// counter until none is left.
template <int NCH>
__global__ __launch_bounds__(64) void sim_kernel(SimArgs A) {
  __shared__ StageSlot stage[64];
  __shared__ int64_t scratch[64 * NCH];
  const int lane = lane_id();
  QEntry* Q = A.queue + (size_t)blockIdx.x * kQueueCap;
  // A workgroup never needs more tickets than there are points.
  for (int taken = 0; taken <= A.n_order; ++taken) {
    // All lanes take part (lane 0 adds 1, the others 0) so the ticket is
    // read by the whole wave without a lane-dependent branch.
    const unsigned old = atomicAdd(A.counter, lane == 0 ? 1u : 0u);
    const int tk = __builtin_amdgcn_readfirstlane((int)old);
    if (tk >= A.n_order) break;
    simulate_point<NCH>(A, A.order[tk], stage, scratch, Q, lane);
  }
}

template __global__ void sim_kernel<1>(SimArgs);
template __global__ void sim_kernel<2>(SimArgs);
template __global__ void sim_kernel<4>(SimArgs);

// ------------------------------------------------------------ statistics
// Nearest-rank percentiles of the finished requests' latencies: k-th
// smallest by most-significant-digit radix select (8-bit digits) with an
// LDS histogram.  One 256-thread workgroup per point.
__device__ int64_t select_kth(const int64_t* v, int n, int k, int* hist, int* sh) {
  uint64_t prefix = 0;
  for (int shift = 56; shift >= 0; shift -= 8) {
    const uint64_t hi_mask = shift == 56 ? 0ull : (~0ull << (shift + 8));
    hist[threadIdx.x] = 0;
    __syncthreads();
    for (int i = threadIdx.x; i < n; i += 256) {
      const uint64_t x = (uint64_t)v[i];
      if (((x ^ prefix) & hi_mask) == 0) atomicAdd(&hist[(x >> shift) & 255u], 1);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      int acc = 0, d = 0;
      for (; d < 255; ++d) {
        if (acc + hist[d] > k) break;
        acc += hist[d];
      }
      sh[0] = d;
      sh[1] = k - acc;
    }
    __syncthreads();
    prefix |= (uint64_t)sh[0] << shift;
    k = sh[1];
    __syncthreads();
  }
  return (int64_t)prefix;
}

__device__ __forceinline__ int nearest_rank_index(int pct, int n) {
  return (int)(((int64_t)pct * n + 99) / 100) - 1;
}

__global__ __launch_bounds__(256) void stats_kernel(const int64_t* e2e, const int64_t* ttft,
                                                    ts_point_result* res, int max_n,
                                                    int n_points) {
  __shared__ int hist[256];
  __shared__ int sh[2];
  for (int p = blockIdx.x; p < n_points; p += gridDim.x) {
    const int n = res[p].n_done;
    int64_t r[5] = {-1, -1, -1, -1, -1};
    if (n > 0) {
      const int64_t* ve = e2e + (size_t)p * (size_t)max_n;
      const int64_t* vt = ttft + (size_t)p * (size_t)max_n;
      r[0] = select_kth(ve, n, nearest_rank_index(50, n), hist, sh);
      r[1] = select_kth(ve, n, nearest_rank_index(90, n), hist, sh);
      r[2] = select_kth(ve, n, nearest_rank_index(99, n), hist, sh);
      r[3] = select_kth(vt, n, nearest_rank_index(50, n), hist, sh);
      r[4] = select_kth(vt, n, nearest_rank_index(99, n), hist, sh);
    }
    if (threadIdx.x == 0) {
      res[p].p50_e2e_ns = r[0];
      res[p].p90_e2e_ns = r[1];
      res[p].p99_e2e_ns = r[2];
      res[p].p50_ttft_ns = r[3];
      res[p].p99_ttft_ns = r[4];
    }
    __syncthreads();
  }
}

// Per-request records start as "pending" (kept by requests never finished).
__global__ void fill_pending_kernel(ts_req_result* r, size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x) {
    ts_req_result o;
    o.admit_ns = -1; o.first_token_ns = -1; o.finish_ns = -1; o.max_gap_ns = 0;
    o.n_preempt = 0; o.status = TS_REQ_PENDING;
    r[i] = o;
  }
}

// Work-queue counters are cleared by a kernel (no memset node in a captured
// stream).
__global__ void reset_counters_kernel(unsigned int* c, int n) {
  if ((int)threadIdx.x < n) c[threadIdx.x] = 0u;
}

}  // namespace tsw
