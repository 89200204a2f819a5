// Step 2 — Algorithm 1 of the paper on the device: SolveReplication (the
// threshold bisection with greedy feasibility probes of Sec. 5.1) and
// SolveReroute (locality-first proportional split of Sec. 5.2).
//
// Feasibility is not monotone in tau (the u_min floor), so the probes must be
// exactly those of the printed sequential bisection.  They are evaluated
// speculatively across the whole chip:
//   k_plan_prep   one workgroup: lambda_e, ell_r, the rank visiting order
//                 (descending excess at any threshold is descending ell), each
//                 rank's experts by descending load, tau_lo0 and tau_hi0.
//   k_plan_round  x2 launches of 1023 one-wave workgroups.  Each workgroup
//                 replays the walk of the earlier round from its stored
//                 outcome bits, then runs the probe of its node of the next
//                 depth-10 subtree of the bisection (one probe per wave on its
//                 own SIMD, so the 1023 probes of a round run at single-probe
//                 latency).  Two rounds cover threshold ranges below 2^20,
//                 which holds for every workload here; a longer bisection
//                 ends with its remaining probes run one after another in
//                 k_plan_emit.  A probe keeps the admissible targets as a
//                 sorted list across the lanes and takes the targets an
//                 expert drains whole with one ballot over the prefix sums of
//                 their slacks; a feasible probe stores its transfers.
//   k_plan_emit   one wave per expert: walks the last round to tau* and the
//                 last feasible probe, and materialises that probe's record
//                 into its expert's row of U, its CSR host list and its rank's
//                 row of X (SolveReplication ends here).
//   k_plan_reroute one wave per expert: SolveReroute, locality first, then the
//                 sources in ascending rank order split their residual demand
//                 over the residual quotas by largest remainder.  It is a
//                 separate entry point so that callers can run it alongside
//                 the weight distribution, as the paper's forward pipeline
//                 does (Eq. 1).
#include "common.hpp"
#include "kernels.hpp"
#include "pack_core.hpp"

namespace uep {

constexpr int kMaxE = 1024;
constexpr int kMaxR = 64;
constexpr int kMaxRec = 256;               // R * n_slot: one transfer per slot at most
constexpr int kDepth = 10;                 // bisection levels per round
constexpr int kNodes = (1 << kDepth) - 1;  // probes per round
constexpr int kRounds = 2;                 // 20 levels, the rest in k_plan_emit
constexpr int64_t kMaxLoad = int64_t(1) << 30;
constexpr int kNotReached = INT32_MIN;
constexpr int kPrepThreads = 1024;
constexpr int kHdr = 4 + 4 * kRounds;  // int64 header words
constexpr int kHdrSpan = 16;           // the header's share of the workspace: one 128-byte line
constexpr int kBitWords = (kNodes + 63) / 64;  // outcome bits per round
// Copies of each round's outcome words, one 128-byte line each: probe b sets
// its bit in copy b % kCopies, which spreads the round's atomics over
// kCopies lines instead of one.
constexpr int kCopies = 8;
static_assert(kHdr <= kHdrSpan && kBitWords * 8 == 128, "outcome copies are whole lines");

struct PlanWs {
  int64_t *hdr;        // [4] tau_lo0, tau_hi0, L, status, then per round j the
                       // bisection state after rounds 0..j: lo, hi, best, probes
  uint64_t *bits;      // [kRounds][kCopies][kBitWords] feasible probes, one bit per node
  int32_t *ell;        // [R]
  int32_t *rank_desc;  // [R] ranks by descending load (visiting order)
  int32_t *rank_asc;   // [R] ranks by ascending load (target order)
  int32_t *eorder;     // [E] experts of each rank, descending load
  int32_t *elam;       // [E] their loads
  int32_t *lam;        // [E] lambda_e
  int32_t *res;        // [kRounds][kNodes] probe outcome
  uint32_t *rec;       // [kRounds][kNodes][2 * RS] (e | t << 16, delta) pairs
};

size_t plan_ws_bytes(int32_t R, int32_t E, int32_t NS) {
  const int64_t RS = static_cast<int64_t>(R) * NS;
  const int64_t ints = 3 * R + 3 * E + int64_t(kRounds) * kNodes * (1 + 2 * RS);
  return static_cast<size_t>(kHdrSpan * 8 + kRounds * kCopies * kBitWords * 8 +
                             (ints * 4 + 255) / 256 * 256);
}

static PlanWs carve(void *ws, int32_t R, int32_t E, int32_t NS) {
  (void)NS;
  PlanWs w;
  w.hdr = static_cast<int64_t *>(ws);
  w.bits = reinterpret_cast<uint64_t *>(w.hdr + kHdrSpan);
  int32_t *p = reinterpret_cast<int32_t *>(w.bits + kRounds * kCopies * kBitWords);
  w.ell = p;
  p += R;
  w.rank_desc = p;
  p += R;
  w.rank_asc = p;
  p += R;
  w.eorder = p;
  p += E;
  w.elam = p;
  p += E;
  w.lam = p;
  p += E;
  w.res = p;
  p += kRounds * kNodes;
  w.rec = reinterpret_cast<uint32_t *>(p);
  return w;
}

struct PlanArgs {
  const int32_t *load;
  int32_t R, E, NS, nm, ncol;
  int32_t u_min;  // clamped to int32 range
  int64_t beta_num, beta_den;
  int32_t *X, *U, *hp, *hr, *hs, *q;
  int64_t *stats;
  PlanWs ws;
};

__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }

__device__ __forceinline__ double readlane_d(double v, int l) {
  const long long b = __double_as_longlong(v);
  const int lo = readlane(static_cast<int>(b), l), hi = readlane(static_cast<int>(b >> 32), l);
  return __longlong_as_double((static_cast<long long>(hi) << 32) | static_cast<uint32_t>(lo));
}

// ---------------------------------------------------------------- prep

__global__ void __launch_bounds__(kPrepThreads) k_plan_prep(PlanArgs a) {
  __shared__ int32_t s_lam[kMaxE];
  __shared__ int32_t s_ell[kMaxR];
  __shared__ int64_t s_part[kPrepThreads];
  __shared__ unsigned long long s_L;
  __shared__ int32_t s_bad;
  const int tid = threadIdx.x, lane = lane_id();
  const int R = a.R, E = a.E, nm = a.nm;
  if (tid == 0) {
    s_L = 0;
    s_bad = 0;
  }
  if (tid < kRounds * kCopies * kBitWords) a.ws.bits[tid] = 0;
  __syncthreads();
  // lambda_e: thread (part, e) sums rows part, part + parts, ... with up to
  // 16 loads in flight, the parts are then combined in LDS
  const int parts = max(1, kPrepThreads / E);
  const int pe = tid % E, part = tid / E;
  int64_t psum = 0;
  bool neg = false;
  if (part < parts) {
    for (int r0 = part; r0 < R; r0 += 16 * parts) {
      int v[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int r = r0 + u * parts;
        v[u] = r < R ? a.load[static_cast<int64_t>(r) * E + pe] : 0;
      }
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        neg |= v[u] < 0;
        psum += v[u];
      }
    }
  }
  if (neg) atomicOr(&s_bad, 1);
  s_part[tid] = psum;
  {
    const int64_t w = wave_sum64(psum);
    if (lane == 0) atomicAdd(&s_L, static_cast<unsigned long long>(w));
  }
  __syncthreads();
  if (tid < E) {
    int64_t lam = 0;
    for (int p = 0; p < parts; ++p) lam += s_part[p * E + tid];
    if (lam > kMaxLoad) atomicOr(&s_bad, 1);
    s_lam[tid] = static_cast<int32_t>(min(lam, kMaxLoad));
    a.ws.lam[tid] = static_cast<int32_t>(min(lam, kMaxLoad));
  }
  __syncthreads();
  const int64_t L = static_cast<int64_t>(s_L);
  if (s_bad || L > kMaxLoad) {
    if (tid == 0) {
      a.ws.hdr[2] = L;
      a.ws.hdr[3] = ULTRAEP_EDATA;
    }
    return;
  }
  if (tid < R) {
    int s = 0;
    for (int j = 0; j < nm; ++j) s += s_lam[tid * nm + j];
    s_ell[tid] = s;
    a.ws.ell[tid] = s;
  }
  if (tid < E) {  // each rank's main experts by descending load (ties: lower id)
    const int r = tid / nm, l = s_lam[tid];
    int pos = 0;
    for (int j = r * nm; j < r * nm + nm; ++j) {
      const int lj = s_lam[j];
      pos += (lj > l) || (lj == l && j < tid);
    }
    a.ws.eorder[r * nm + pos] = tid;
    a.ws.elam[r * nm + pos] = l;
  }
  __syncthreads();
  {  // ranks by descending and by ascending load (ties: lower rank): 16
     // threads per rank each compare it with 4 others, then a DPP row sum
    const int i = tid >> 4, part = tid & 15;
    int cnt = 0;  // ranks ahead in descending order << 16 | ahead in ascending
    if (i < R) {
      const int li = s_ell[i];
#pragma unroll
      for (int k = 0; k < kMaxR / 16; ++k) {
        const int r = part * (kMaxR / 16) + k;
        if (r < R) {
          const int lr = s_ell[r];
          const bool tie = lr == li && r < i;
          cnt += ((lr > li || tie) ? (1 << 16) : 0) + ((lr < li || tie) ? 1 : 0);
        }
      }
    }
    cnt = row_sum(cnt);
    if (i < R && part == 0) {
      a.ws.rank_desc[cnt >> 16] = i;
      a.ws.rank_asc[cnt & 0xFFFF] = i;
    }
  }
  if (tid < kWave) {
    const int hi = wave_max(tid < R ? s_ell[tid] : -1);
    if (tid == 0) {
      const int64_t m = (L + R - 1) / R;
      const int64_t lo = (a.beta_num * m + a.beta_den - 1) / a.beta_den;
      a.ws.hdr[0] = lo;
      a.ws.hdr[1] = hi;
      a.ws.hdr[2] = L;
      a.ws.hdr[3] = 0;
    }
  }
}

// ---------------------------------------------------------------- rounds

// DPP wave_shl:1 - lane i receives lane i+1 (lane 63 keeps its value)
__device__ __forceinline__ int wave_shl1(int v) {
  return __builtin_amdgcn_update_dpp(v, v, 0x130, 0xF, 0xF, false);
}

// Greedy feasibility probes of SolveReplication at threshold tau (Sec. 5.1),
// one wave each.  Lane i holds the i-th rank of the visiting order (rk_r,
// rank, and rk_l, its load: descending load, ties to the lower rank) and
// the i-th rank of ascending load (as_r, as_l).  A probe returns the number
// of accepted transfers, recorded in s_re / s_rd as (e | t << 16, delta) in
// acceptance order, or -1 if the threshold is infeasible.
//
// The admissible targets (slack > 0, a free slot) form a list sorted by
// slack descending, rank ascending, one per lane from the head h on.  It
// starts as the ranks of load below tau in ascending load order.  With the
// slacks m in lanes and their inclusive prefix P (B = P before the head),
// an expert that has to shed need = min(excess, its load) takes whole every
// target from the head whose running slack stays below need (one ballot),
// then the rest d from the next target.  A whole transfer is bound by the
// target's slack, so one below u_min makes the probe infeasible, and the
// target leaves the list, exactly as transfer-by-transfer evaluation finds.
// The experts are visited in one flat loop (rank by rank, experts by
// descending load) with scalar loop state.

// Loads experts [j0, j0 + 64) of rank r's visiting order into lanes.
// Lanes past the rank's last expert read that expert and hold zeros: no
// divergent branch in the probes' loops.
__device__ __forceinline__ void load_experts(const PlanArgs &a, int r, int j0, int lane,
                                             const int32_t *s_eorder, const int32_t *s_elam,
                                             int &ev, int &lv) {
  const int jl = j0 + lane;
  const int i = r * a.nm + min(jl, a.nm - 1);
  const int v = s_eorder[i], l = s_elam[i];
  ev = jl < a.nm ? v : 0;
  lv = jl < a.nm ? l : 0;
}

// One redundant slot per rank: every transfer uses up its target, so
// transfer k goes to the k-th listed target and its record stays in lane k.
// The slacks never change, so P is the fixed inclusive prefix of the list
// and the lanes with P - B < need are the prefix [0, hh) (lanes before the
// head have P <= B): the whole targets are [h, hh).
template <int kSite>
__device__ __forceinline__ int probe_one_slot(const PlanArgs &a, int tau, int lane, int rk_r, int rk_l,
                              int as_r, int as_l, const int32_t *s_eorder,
                              const int32_t *s_elam, uint32_t *s_re, int32_t *s_rd) {
  const int R = a.R, nm = a.nm, u_min = a.u_min;
  const bool tv = lane < R && as_l < tau;
  const int m = tv ? tau - as_l : 0;
  const uint64_t tmask = ballot(tv);  // a prefix of the lanes
  // inclusive prefix of the slacks: each is below 2^25, the sum below 2^31
  int P = m;
  for (int o = 1; o < kWave; o <<= 1) {
    const int t = __shfl_up(P, o);
    if (lane >= o) P += t;
  }
  const uint64_t low_umin = ballot(tv && m < u_min);
  int x = readlane(rk_l, 0) - tau;
  if (x <= 0) return 0;  // nothing to shed
  int r = readlane(rk_r, 0);
  int ev, lv;
  load_experts(a, r, 0, lane, s_eorder, s_elam, ev, lv);
  int rec_e = 0, rec_d = 0;
  int h = 0, B = 0, oi = 0, j = 0;  // head, slack before it, rank, expert
  bool fail = false;
  for (;;) {
    const int c = readlane(lv, j & (kWave - 1));
    const int e = readlane(ev, j & (kWave - 1));
    const int need = min(x, c);
    const uint64_t wm = ballot(P - B < need) & tmask;
    const int hh = __popcll(wm);
    const int Ph = readlane(P, hh & (kWave - 1)), mh = readlane(m, hh & (kWave - 1));
    const int taken = Ph - mh - B;  // slack of the whole targets
    const int d = need - taken;     // the rest, at most mh
    x -= taken;
    const int take = d >= u_min ? 1 : 0;
    // an expert with no load left, no target for the rest (every target
    // whole), a whole target below u_min, or a rest below u_min that is not
    // only this expert's shortfall (max(d, min(x, mh)) < u_min)
    fail = c <= 0 || wm == tmask || ((wm & low_umin) >> (h & (kWave - 1))) != 0 ||
           max(d, min(x, mh)) < u_min;
    if (fail) break;
    // the whole targets and, when the rest is taken, target hh
    const bool mine = static_cast<uint32_t>(lane - h) < static_cast<uint32_t>(hh - h + take);
    rec_e = mine ? e : rec_e;
    rec_d = mine ? (lane == hh ? d : m) : rec_d;
    x -= take ? d : 0;
    B = take ? Ph : Ph - mh;
    h = hh + take;
    if (x > 0) {
      if (++j < nm) {  // next expert of this rank
        if ((j & (kWave - 1)) == 0) load_experts(a, r, j, lane, s_eorder, s_elam, ev, lv);
        continue;
      }
      fail = true;  // the rank's experts ran out
      break;
    }
    if (++oi >= R) break;
    x = readlane(rk_l, oi) - tau;
    if (x <= 0) break;  // the remaining ranks are not overloaded
    r = readlane(rk_r, oi);
    load_experts(a, r, 0, lane, s_eorder, s_elam, ev, lv);
    j = 0;
  }
  if (fail) return -1;
  if (lane < h) {
    s_re[lane] = static_cast<uint32_t>(rec_e) | (static_cast<uint32_t>(as_r) << 16);
    s_rd[lane] = rec_d;
  }
  return h;
}

// Several redundant slots per rank: a target that keeps slack and a free
// slot after an expert's last (partial) transfer moves back to its place in
// the list; the lanes it passes shift down by one (DPP) and P is patched.
// The list entries are packed keys (slack << 6) | (63 - rank).  P is
// nondecreasing over the live lanes, and every lane before the head has
// P <= B, so the lanes with P - B < need are the prefix [0, hh): hh is the
// population count of one ballot, and the whole targets are [h, hh).  In
// the loop a record is (e, key of the transfer: amount << 6 | 63 - rank),
// written by the lanes of the targets themselves; the records are put into
// the common (e | rank << 16, amount) form once the probe has succeeded.
template <int kSite>
__device__ __forceinline__ int probe_multi(const PlanArgs &a, int tau, int lane, int rk_r, int rk_l,
                           int as_r, int as_l, const int32_t *s_eorder,
                           const int32_t *s_elam, uint32_t *s_re, int32_t *s_rd) {
  const int R = a.R, nm = a.nm, NS = a.NS, u_min = a.u_min;
  const bool tv = lane < R && as_l < tau && NS > 0;
  int key = tv ? ((tau - as_l) << 6) | (kWave - 1 - as_r) : 0;
  int used = 0;
  const uint64_t live = ballot(tv);  // a prefix of the lanes; its length never changes
  int P = key >> 6;
  for (int o = 1; o < kWave; o <<= 1) {
    const int t = __shfl_up(P, o);
    if (lane >= o) P += t;
  }
  // live lanes whose slack is below u_min (refreshed when a key moves)
  uint64_t low = ballot((key >> 6) < u_min);
  int x = readlane(rk_l, 0) - tau;
  if (x <= 0) return 0;
  int r = readlane(rk_r, 0);
  int ev, lv;
  load_experts(a, r, 0, lane, s_eorder, s_elam, ev, lv);
  int h = 0, B = 0, n = 0, oi = 0, j = 0;
  bool fail = false;
  for (;;) {
    const int c = readlane(lv, j & (kWave - 1));
    const int e = readlane(ev, j & (kWave - 1));
    const int need = min(x, c);
    const uint64_t wm = ballot(P - B < need) & live;
    const int hh = __popcll(wm);
    const int Ph = readlane(P, hh & (kWave - 1)), kh = readlane(key, hh & (kWave - 1));
    const int mh = kh >> 6;
    const int taken = Ph - mh - B;  // slack of the whole targets
    const int d = need - taken;     // the rest, at most mh
    x -= taken;
    const int take = d >= u_min ? 1 : 0;
    // an expert with no load left, no target for the rest (every live lane
    // whole), a whole target below u_min, or a rest below u_min that is not
    // only this expert's shortfall (max(d, min(x, mh)) < u_min)
    fail = c <= 0 || wm == live || ((wm & low) >> (h & (kWave - 1))) != 0 ||
           max(d, min(x, mh)) < u_min;
    if (fail) break;
    const int nw = hh - h + take;
    {  // the other lanes write a spare area past the records
      const int at = static_cast<uint32_t>(lane - h) < static_cast<uint32_t>(nw) ? n + lane - h
                                                                             : kMaxRec + lane;
      s_re[at] = static_cast<uint32_t>(e);
      s_rd[at] = lane == hh ? ((d << 6) | (key & (kWave - 1))) : key;
    }
    n += nw;
    B = Ph - mh;
    h = hh;
    if (take) {
      x -= d;
      const int uh = readlane(used, hh) + 1;
      if (mh == d || uh >= NS) {  // out of slack or slots: leaves the list
        B = Ph;
        h = hh + 1;
      } else {  // back to its place: after every key still larger
        const int nk = ((mh - d) << 6) | (kh & (kWave - 1));
        const int p = hh + __popcll(ballot(key > nk) & (~uint64_t(1) << hh) & live);
        const bool mv = static_cast<uint32_t>(lane - hh) < static_cast<uint32_t>(p - hh);
        const int ks = wave_shl1(key), us = wave_shl1(used), ps = wave_shl1(P);
        key = mv ? ks : (lane == p ? nk : key);
        used = mv ? us : (lane == p ? uh : used);
        P = mv ? ps - mh : (lane >= p ? P - d : P);
        low = ballot((key >> 6) < u_min);
      }
    }
    if (x > 0) {
      if (++j < nm) {  // next expert of this rank
        if ((j & (kWave - 1)) == 0) load_experts(a, r, j, lane, s_eorder, s_elam, ev, lv);
        continue;
      }
      fail = true;  // the rank's experts ran out
      break;
    }
    if (++oi >= R) break;
    x = readlane(rk_l, oi) - tau;
    if (x <= 0) break;  // the remaining ranks are not overloaded
    r = readlane(rk_r, oi);
    load_experts(a, r, 0, lane, s_eorder, s_elam, ev, lv);
    j = 0;
  }
  if (fail) return -1;
  __syncthreads();
  for (int i = lane; i < n; i += kWave) {
    const int k = s_rd[i];
    s_re[i] |= static_cast<uint32_t>(kWave - 1 - (k & (kWave - 1))) << 16;
    s_rd[i] = k >> 6;
  }
  return n;
}

// The same probe for slacks of 25 bits or more: lane t holds rank t's slack
// and slot count, and the target is a wave max plus a ballot for the lowest
// rank among ties.
template <int kSite>
__device__ __forceinline__ int probe_wide(const PlanArgs &a, int tau, int lane, int rk_r, int rk_l,
                          int ell_lane, const int32_t *s_eorder, const int32_t *s_elam,
                          uint32_t *s_re, int32_t *s_rd) {
  int slk = lane < a.R ? max(tau - ell_lane, 0) : 0;
  int used = 0;
  int n = 0;
  for (int oi = 0; oi < a.R; ++oi) {
    int exc = readlane(rk_l, oi) - tau;
    if (exc <= 0) break;
    const int r = readlane(rk_r, oi);
    for (int j0 = 0; j0 < a.nm && exc > 0; j0 += kWave) {
      const int jl = j0 + lane;
      const int ev = jl < a.nm ? s_eorder[r * a.nm + jl] : 0;
      const int lv = jl < a.nm ? s_elam[r * a.nm + jl] : 0;
      const int jn = min(kWave, a.nm - j0);
      for (int j = 0; j < jn && exc > 0; ++j) {
        const int e = readlane(ev, j);
        int cap = readlane(lv, j);
        while (exc > 0 && cap > 0) {
          const bool ok = slk > 0 && used < a.NS;
          const int v = ok ? slk : 0;
          const int m = wave_max(v);
          if (m == 0) return -1;
          const int ts = uni(__ffsll(static_cast<unsigned long long>(ballot(v == m && ok))) - 1);
          const int d = min(min(exc, m), cap);
          if (d < a.u_min) {
            if (min(exc, m) < a.u_min) return -1;
            break;
          }
          if (lane == ts) {
            slk -= d;
            ++used;
          }
          if (lane == 0) {
            s_re[n] = static_cast<uint32_t>(e) | (static_cast<uint32_t>(ts) << 16);
            s_rd[n] = d;
          }
          ++n;
          exc -= d;
          cap -= d;
        }
      }
    }
    if (exc > 0) return -1;
  }
  return n;
}

// One probe at tau with the variant the thresholds and slots allow.  kSite
// gives every call site its own copy: shared by two kernels, the compiler
// loses sight of the probes' scalar loop state.
template <int kSite>
__device__ __forceinline__ int run_probe(const PlanArgs &a, bool packed, int tau, int lane,
                                         int rk_r, int rk_l, int as_r, int as_l, int ell_lane,
                                         const int32_t *s_eorder, const int32_t *s_elam,
                                         uint32_t *s_re, int32_t *s_rd) {
  if (!packed) return probe_wide<kSite>(a, tau, lane, rk_r, rk_l, ell_lane, s_eorder, s_elam, s_re, s_rd);
  if (a.NS == 1)
    return probe_one_slot<kSite>(a, tau, lane, rk_r, rk_l, as_r, as_l, s_eorder, s_elam, s_re, s_rd);
  return probe_multi<kSite>(a, tau, lane, rk_r, rk_l, as_r, as_l, s_eorder, s_elam, s_re, s_rd);
}

// Bisection state before round rd: the initial interval, or the state
// after round rd - 1 that round rd's first workgroup published.
struct BisState {
  int64_t lo, hi;
  int best;   // last feasible probe: round * kNodes + node, or -1
  int probes; // probes of the sequential bisection so far
};

// One pointer and four loads whatever rd is (no branch that would make the
// loads wait for each other).
__device__ __forceinline__ BisState state_before(const PlanArgs &a, int rd) {
  const int64_t *h = a.ws.hdr + (rd == 0 ? 0 : 4 + 4 * (rd - 1));
  const int64_t lo = h[0], hi = h[1], best = h[2], probes = h[3];
  return {lo, hi, rd == 0 ? -1 : static_cast<int>(best), rd == 0 ? 0 : static_cast<int>(probes)};
}

__device__ __forceinline__ uint64_t readlane64(uint64_t v, int l) {
  const uint32_t lo = static_cast<uint32_t>(readlane(static_cast<int>(v), l));
  const uint32_t hi = static_cast<uint32_t>(readlane(static_cast<int>(v >> 32), l));
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

// Round rd's outcome words: the kCopies copies of word w into lane w (the
// lanes past the last word read it too).  No branch between the loads, so
// that they stay in flight together with the kernel's other inputs.
__device__ __forceinline__ void outcome_load(const PlanArgs &a, int rd, uint64_t (&v)[kCopies]) {
  const int w = min(lane_id(), kBitWords - 1);
#pragma unroll
  for (int c = 0; c < kCopies; ++c) v[c] = a.ws.bits[(rd * kCopies + c) * kBitWords + w];
}

// The OR of the copies: word w in lane w, zero past the last word.
__device__ __forceinline__ uint64_t outcome_or(const uint64_t (&v)[kCopies]) {
  uint64_t bw = 0;
#pragma unroll
  for (int c = 0; c < kCopies; ++c) bw |= v[c];
  return lane_id() < kBitWords ? bw : 0;
}

// The sequential bisection through round rd's depth-kDepth subtree, from
// state st, over the round's outcome bits (word w in lane w).
__device__ __forceinline__ void walk_bits(uint64_t bw, int rd, BisState &st) {
  int node = 0;
  for (int d = 0; d < kDepth && st.lo < st.hi; ++d) {
    const int64_t mid = (st.lo + st.hi) / 2;
    ++st.probes;
    const uint64_t w = readlane64(bw, node >> 6);
    if ((w >> (node & 63)) & 1) {
      st.hi = mid;
      st.best = rd * kNodes + node;
      node = 2 * node + 1;
    } else {
      st.lo = mid + 1;
      node = 2 * node + 2;
    }
  }
}

__global__ void __launch_bounds__(kWave) k_plan_round(PlanArgs a, int round) {
  __shared__ int32_t s_eorder[kMaxE];
  __shared__ int32_t s_elam[kMaxE];
  __shared__ uint32_t s_re[kMaxRec + kWave];
  __shared__ int32_t s_rd[kMaxRec + kWave];
  const int lane = threadIdx.x, b = blockIdx.x;
  const int R = a.R, E = a.E, RS = R * a.NS;
  // every input is requested up front, with no branch between the loads
  // (indices clamped into range, values masked afterwards), so the round
  // waits for memory once: the state before the previous round and that
  // round's outcome bits (round 0 reads the last round's words, which
  // nothing writes before that round), the per-rank expert orders and the
  // rank orders
  const int64_t status = a.ws.hdr[3];
  const bool packed = a.ws.hdr[1] < (int64_t(1) << 25);
  BisState st = state_before(a, round > 0 ? round - 1 : 0);
  uint64_t bv[kCopies];
  outcome_load(a, round > 0 ? round - 1 : kRounds - 1, bv);
  int ve[kMaxE / kWave], vl[kMaxE / kWave];
#pragma unroll
  for (int u = 0; u < kMaxE / kWave; ++u) {
    if (u * kWave < E) {
      const int i = min(u * kWave + lane, E - 1);  // stored to LDS only below E
      ve[u] = a.ws.eorder[i];
      vl[u] = a.ws.elam[i];
    }
  }
  const int lr = min(lane, R - 1);
  const int rk_v = a.ws.rank_desc[lr], as_v = a.ws.rank_asc[lr], ell_v = a.ws.ell[lr];
  // the loads above are issued before the status test (which the compiler
  // would otherwise move ahead of them, waiting for the header first)
  asm volatile("" ::: "memory");
  const int rk_r = lane < R ? rk_v : 0;
  const int as_r = lane < R ? as_v : 0;
  const int ell_lane = lane < R ? ell_v : 0;
  if (status != 0) return;
  if (round > 0) {  // every workgroup walks the previous round; the first publishes it
    walk_bits(outcome_or(bv), round - 1, st);
    if (b == 0 && lane == 0) {
      int64_t *h = a.ws.hdr + 4 + 4 * (round - 1);
      h[0] = st.lo;
      h[1] = st.hi;
      h[2] = st.best;
      h[3] = st.probes;
    }
  }
  int64_t lo = st.lo, hi = st.hi;
  if (lo >= hi) return;  // the bisection has ended
  // this workgroup's node of the round's subtree
  const int id = b + 1, depth = 31 - __clz(id);
  bool reached = true;
  for (int bit = depth - 1; bit >= 0 && reached; --bit) {
    const int64_t mid = (lo + hi) / 2;
    if ((id >> bit) & 1) lo = mid + 1;  // right child: that probe failed
    else hi = mid;                      // left child: that probe succeeded
    reached = lo < hi;
  }
  int n = kNotReached;
  if (reached) {
    const int tau = static_cast<int>((lo + hi) / 2);
#pragma unroll
    for (int u = 0; u < kMaxE / kWave; ++u) {
      const int i = u * kWave + lane;
      if (i < E) {
        s_eorder[i] = ve[u];
        s_elam[i] = vl[u];
      }
    }
    const int rk_l = __shfl(ell_lane, rk_r);
    const int as_l = __shfl(ell_lane, as_r);
    __syncthreads();
    n = run_probe<0>(a, packed, tau, lane, rk_r, rk_l, as_r, as_l, ell_lane, s_eorder, s_elam,
                  s_re, s_rd);
    if (n > 0) {
      __syncthreads();
      uint32_t *rec = a.ws.rec + (static_cast<int64_t>(round) * kNodes + b) * 2 * RS;
      for (int i = lane; i < n; i += kWave) {
        rec[2 * i] = s_re[i];
        rec[2 * i + 1] = static_cast<uint32_t>(s_rd[i]);
      }
    }
  }
  if (lane == 0) {
    a.ws.res[round * kNodes + b] = n;
    if (n >= 0)
      atomicOr(a.ws.bits + (round * kCopies + (b % kCopies)) * kBitWords + (b >> 6),
               uint64_t(1) << (b & 63));
  }
}

// ---------------------------------------------------------------- reroute

// DPP wave_shr:1 - lane i receives lane i-1 (lane 0 keeps its value)
__device__ __forceinline__ int wave_shr1(int v) {
  return __builtin_amdgcn_update_dpp(v, v, 0x138, 0xF, 0xF, false);
}

// Two hosts (home first, one replica): with residual quotas (u0, u1) and
// residual demand D = u0 + u1, a source with demand lh gives host 0
// b0 = floor(lh * u0 / D) plus the one leftover unit when its remainder is
// at least the other host's (ties go to the earlier host), i.e.
// q0 = floor((lh * u0 + D / 2) / D).  The sources run in ascending order with
// the state u0 carried from lane r to lane r + 1 by a DPP shift, so the chain
// has no scalar round trip and no branch.  Lane r returns q0 of source r.
//   kExact: lh * u0 + D / 2 < 2^52 (total load below 2^26), so the fp64
//   numerator is exact and one correction of the reciprocal estimate
//   gives the floor; otherwise the same in int64.
template <bool kExact>
__device__ __forceinline__ int split_two(int lamhat, int Dr, int u0_init, int R) {
  const bool act = lamhat > 0;
  const double lhd = static_cast<double>(lamhat);
  const double Dd = act ? static_cast<double>(Dr) : 1.0;
  const double rD = 1.0 / Dd;
  const double half = 0.5 * Dd;
  int u0 = u0_init, qout = 0;
  const int lane = lane_id();
  for (int r = 0; r < R; ++r) {
    int q;
    if (kExact) {
      const double N = __builtin_fma(lhd, static_cast<double>(u0), half);
      const double t = __builtin_trunc(N * rD);
      const double rr = __builtin_fma(-t, Dd, N);
      q = static_cast<int>(t) + (rr >= Dd ? 1 : 0) - (rr < 0.0 ? 1 : 0);
    } else {
      const int64_t D = act ? Dr : 1;
      const int64_t N = 2 * static_cast<int64_t>(lamhat) * u0 + D;
      int64_t t = static_cast<int64_t>(static_cast<double>(N) * (0.5 * rD));
      const int64_t rr = N - t * 2 * D;
      t += (rr >= 2 * D ? 1 : 0) - (rr < 0 ? 1 : 0);
      q = static_cast<int>(t);
    }
    qout = lane == r ? q : qout;
    u0 = wave_shr1(u0 - q);
  }
  return qout;
}

// LDS of one expert's SolveReroute: its hosts' ranks (kWave), then the
// shares of the lane-mirrored split (8 hosts x kMaxR sources, and a spare
// area for the lanes that are not host slots)
constexpr int kRrLds = kWave + 8 * kMaxR + kWave;

// DPP row_ror:k - within each row of 16 lanes, a rotation by k lanes (every
// lane has a source, so no old value is needed and the move folds into the
// instruction that consumes it)
template <int K>
__device__ __forceinline__ int row_ror(int v) {
  return __builtin_amdgcn_mov_dpp(v, 0x120 + K, 0xF, 0xF, true);
}

// 1 when the host k rotations away has the larger key (its key minus ours
// is positive; keys are below 2^29, so the difference cannot wrap)
template <int K>
__device__ __forceinline__ int ahead(int key) {
  return static_cast<int>(static_cast<uint32_t>(key - row_ror<K>(key)) >> 31);
}

// Sum over the kH host slots of a row that repeats them with period kH.
template <int kH>
__device__ __forceinline__ int host_sum(int b) {
  int sb = kH == 8 ? b + row_ror<4>(b) : b;
  sb += row_ror<2>(sb);
  return sb + row_ror<1>(sb);
}

// Number of the kH - 1 other host slots whose key is larger.
template <int kH>
__device__ __forceinline__ int rank_of(int key) {
  if (kH == 4) return (ahead<1>(key) + ahead<2>(key)) + ahead<3>(key);
  return (ahead<1>(key) + ahead<2>(key)) + (ahead<3>(key) + ahead<4>(key)) +
         ((ahead<5>(key) + ahead<6>(key)) + ahead<7>(key));
}

// Three to eight hosts, total load below 2^26: host i sits in lane i and in
// its mirror lane i + 8, so that rotations by 1 .. 7 within the 16 lanes of
// row 0 bring every other host's value to every host lane with no scalar
// round trip.  Lanes of host slots i >= nh, and every lane past 15, hold a
// zero residual quota (so a zero share and a zero remainder).  Per source
// with residual demand, in ascending order:
//   b_i = floor(lh * u_i / D) and rem_i exactly: the estimate
//         trunc((lh / D) * u_i) in fp64 is within one of the floor (the
//         quotient is below 2^26), and the remainder for the estimate lies
//         in (-D, 2D), so wrapping 32-bit arithmetic gives it exactly and
//         one correction gives both,
//   left = lh - sum_i b_i, the sum taken by three rotations (4, 2, 1),
//   host i gets one of the left units iff fewer than `left` hosts are ahead
//   of it in (remainder descending, host ascending): the keys rem * 8 +
//   (7 - i) order exactly so, and a zero-quota slot i >= nh is never ahead
//   of a host (its key 7 - i is below every host's),
// then u_i -= q_i.  The shares go to s_q[r * 8 + i] (lanes past 7 write a
// spare area); afterwards lane r writes source r's row of Q, adding the
// locality share of the host that is r itself.  s_hosts lists the hosts'
// ranks, s_q holds kRrLds - kWave ints.  kSmall (the expert's residual
// demand below 2^19): the same with an fp32 estimate and 24-bit products.
// kH = 4 (at most four hosts): the slots repeat with period 4 in row 0
// (lanes i, i + 4, i + 8, i + 12), so three rotations rank the keys
// rem * 4 + (3 - i) and two sum the floors.
template <int kH, bool kSmall>
__device__ __forceinline__ void split_lanes(int lane, int nh, int lamhat_r, int Dr, int loc_r,
                                            int R, int64_t ncol, int32_t *qbase,
                                            const int32_t *s_hosts, int32_t *s_q,
                                            int ures_r) {
  static_assert(kH == 4 || kH == 8, "host slots mirror with period 4 or 8 in a row");
  const int hidx = lane & (kH - 1);
  const bool slot = lane < 16 && hidx < nh;
  int ures = __shfl(ures_r, slot ? s_hosts[hidx] : 0);
  ures = slot ? ures : 0;
  const int qstep = lane < kH ? 8 : 0;
  const int qoff = lane < kH ? lane : 8 * kMaxR + lane;
  uint64_t act = ballot(lane < R && lamhat_r > 0);
  const int key_lo = kH - 1 - hidx;
  if (kSmall) {
    // Residual demand below 2^19: c = (lh / D)(1 - 2^-20) rounded to fp32
    // makes y = fl(c * u) fall strictly below x = lh * u / D and above
    // x - 1 (relative errors below 2^-20 + 2^-23 on x < 2^19), so trunc(y)
    // is floor(x) or floor(x) - 1, and the remainder lh * u - trunc(y) * D
    // lies in [0, 2D): 24-bit products wrapped to 32 bits give it exactly,
    // and one subtraction with a min gives the floor's remainder
    const float c_r = lamhat_r > 0 ? static_cast<float>(static_cast<double>(lamhat_r) *
                                                        (1.0 - 0x1p-20) / static_cast<double>(Dr))
                                   : 0.0f;
    const int nD_r = -Dr;
    while (act) {
      const int r = __ffsll(static_cast<unsigned long long>(act)) - 1;
      act &= act - 1;
      const int lh = readlane(lamhat_r, r);
      const int nD = readlane(nD_r, r);
      const float c = __int_as_float(readlane(__float_as_int(c_r), r));
      const int be = static_cast<int>(c * static_cast<float>(ures));
      const int re = static_cast<int>(static_cast<uint32_t>(__mul24(be, nD)) +
                                      __umul24(lh, static_cast<uint32_t>(ures)));
      const int t = re + nD;  // re - D, in [-D, D)
      const int rem = static_cast<int>(min(static_cast<uint32_t>(re), static_cast<uint32_t>(t)));
      const int b = be + 1 + (t >> 31);
      const int left = lh - host_sum<kH>(b);
      const int rk = rank_of<kH>((rem << (kH == 8 ? 3 : 2)) | key_lo);
      const int qi = b + ((slot && rk < left) ? 1 : 0);
      ures -= qi;
      s_q[r * qstep + qoff] = qi;
    }
  } else {
    // lh / D of source `lane`
    const double c_r = lamhat_r > 0 ? static_cast<double>(lamhat_r) / static_cast<double>(Dr) : 0.0;
    while (act) {
      const int r = __ffsll(static_cast<unsigned long long>(act)) - 1;
      act &= act - 1;
      const int lh = readlane(lamhat_r, r);
      const int D = readlane(Dr, r);
      const double c = readlane_d(c_r, r);
      const int be = static_cast<int>(c * static_cast<double>(ures));
      const int re = static_cast<int>(static_cast<uint32_t>(lh) * static_cast<uint32_t>(ures) -
                                      static_cast<uint32_t>(be) * static_cast<uint32_t>(D));
      const bool lo = re < 0, hi = re >= D;
      const int b = lo ? be - 1 : (hi ? be + 1 : be);
      const int rem = lo ? re + D : (hi ? re - D : re);
      const int left = lh - host_sum<kH>(b);
      const int rk = rank_of<kH>((rem << (kH == 8 ? 3 : 2)) | key_lo);
      const int qi = b + ((slot && rk < left) ? 1 : 0);
      ures -= qi;
      s_q[r * qstep + qoff] = qi;
    }
  }
  if (lane < R) {
    const bool dem = lamhat_r > 0;
    int32_t *qrow = qbase + static_cast<int64_t>(lane) * ncol;
    for (int i = 0; i < nh; ++i)
      qrow[i] = (dem ? s_q[lane * 8 + i] : 0) + (s_hosts[i] == lane ? loc_r : 0);
  }
}

// Any number of hosts: lane i is host i (home first, then replicas by
// ascending rank) with residual quota ures; the sources run in ascending
// order, each splitting its residual demand by largest remainder.  Writes
// q of source r, host `lane` to qcol[r * ncol].  Used above eight hosts or
// when the total load reaches 2^26.
template <bool kExact, bool kOneRow>
__device__ __forceinline__ void split_many(int lane, int nh, int lamhat_r, int Dr, int ures, int R,
                           int64_t ncol, int32_t *qcol, int t_i, int qloc_i) {
  const double rDr = lamhat_r > 0 ? 1.0 / static_cast<double>(Dr) : 0.0;
  const bool host = lane < nh;
  for (int r = 0; r < R; ++r) {
    const int lh = readlane(lamhat_r, r);
    int qi = 0;
    if (lh > 0) {
      const int D = readlane(Dr, r);
      const double rD = readlane_d(rDr, r);
      // floor(lh * ures / D) and its remainder, exact after one correction
      int b, rem;
      if (kExact) {  // lh * ures < 2^52
        const double Dd = static_cast<double>(D);
        const double pr = static_cast<double>(lh) * static_cast<double>(ures);
        const double bq = __builtin_trunc(pr * rD);
        const double rd = __builtin_fma(-bq, Dd, pr);
        const int lo = rd < 0.0 ? 1 : 0, hi = rd >= Dd ? 1 : 0;
        b = static_cast<int>(bq) + hi - lo;
        rem = static_cast<int>(rd) + (lo ? D : 0) - (hi ? D : 0);
      } else {
        b = static_cast<int>(static_cast<double>(lh) * static_cast<double>(ures) * rD);
        int64_t rm = static_cast<int64_t>(lh) * ures - static_cast<int64_t>(b) * D;
        const bool lo = rm < 0, hi = rm >= D;
        b += lo ? -1 : (hi ? 1 : 0);
        rm += lo ? D : (hi ? -D : 0);
        rem = static_cast<int>(rm);
      }
      const int left = lh - (kOneRow ? readlane(row_sum(b), 0) : wave_sum(b));
      // the `left` hosts with the largest remainders (ties: earlier host)
      int rk = 0;
      for (int j = 0; j < nh; ++j) {
        const int rj = readlane(rem, j);
        rk += (rj > rem) || (rj == rem && j < lane);
      }
      qi = b + ((host && rk < left) ? 1 : 0);
      ures -= qi;
    }
    if (host) qcol[r * ncol] = qi + (t_i == r ? qloc_i : 0);
  }
}

// SolveReroute for expert e, run by one wave.  The hosts of e are its home
// and every other rank with a positive quota (a replica's quota is at least
// u_min), so the expert's row of U (u_r: its quota on rank `lane`), its load
// column (lam_r), its first CSR column j0 and the number of CSR entries are
// all the inputs.  Locality first: a host consumes its own tokens up to its
// quota; the residual demands are then split over the residual quotas.
__device__ __forceinline__ void reroute_expert(const PlanArgs &a, int e, int j0, int total, int lam_r,
                               int u_r, int64_t L, int32_t *s_t) {
  const int lane = lane_id();
  const int R = a.R, E = a.E;
  const int64_t ncol = a.ncol;
  const int h = e / a.nm;
  const uint64_t rep = ballot(lane < R && lane != h && u_r > 0);
  const int nh = 1 + __popcll(rep);
  if (j0 < e || j0 + nh > total || total > ncol) {  // not a plan of this group
    if (lane == 0) a.stats[6] = ULTRAEP_EDATA;
    return;
  }
  const int loc_r = min(lam_r, u_r);  // 0 on ranks that do not host e
  const int lamhat_r = lam_r - loc_r;
  const int ures_r = u_r - loc_r;
  // residual demand still to place when source r comes: D0 minus the
  // demand of the sources before it
  const int incl = wave_scan_incl(lamhat_r);
  const int D0 = readlane(incl, kWave - 1);
  const int Dr = D0 - (incl - lamhat_r);
  const bool exact = L < (int64_t(1) << 26);
  int32_t *qrow = a.q + static_cast<int64_t>(lane) * ncol;
  if (nh == 1) {
    if (lane < R) qrow[j0] = lam_r;
  } else if (nh == 2) {
    const int t = __ffsll(static_cast<unsigned long long>(rep)) - 1;
    const int u0 = readlane(ures_r, h);
    const int q0 = exact ? split_two<true>(lamhat_r, Dr, u0, R)
                         : split_two<false>(lamhat_r, Dr, u0, R);
    if (lane < R) {
      qrow[j0] = q0 + (lane == h ? loc_r : 0);
      qrow[j0 + 1] = lamhat_r - q0 + (lane == t ? loc_r : 0);
    }
  } else {
    if (lane == h) s_t[0] = h;
    if ((rep >> lane) & 1) s_t[1 + popc_below(rep)] = lane;
    __syncthreads();
    if (exact && nh <= 8) {
      int32_t *qb = a.q + j0, *s_q = s_t + kWave;
      if (D0 < (1 << 19)) {
        if (nh <= 4)
          split_lanes<4, true>(lane, nh, lamhat_r, Dr, loc_r, R, ncol, qb, s_t, s_q, ures_r);
        else
          split_lanes<8, true>(lane, nh, lamhat_r, Dr, loc_r, R, ncol, qb, s_t, s_q, ures_r);
      } else {
        split_lanes<8, false>(lane, nh, lamhat_r, Dr, loc_r, R, ncol, qb, s_t, s_q, ures_r);
      }
      for (int j = total + e; j < ncol; j += E)
        if (lane < R) qrow[j] = 0;
      return;
    }
    const int t_i = lane < nh ? s_t[lane] : 0;
    // every lane takes part in the shuffles: a lane reads only from lanes
    // that execute the same shuffle
    const int ures_t = __shfl(ures_r, t_i);
    const int qloc_i = __shfl(loc_r, t_i);
    const int ures_i = lane < nh ? ures_t : 0;
    int32_t *qcol = a.q + j0 + lane;
    if (exact && nh <= 16)
      split_many<true, true>(lane, nh, lamhat_r, Dr, ures_i, R, ncol, qcol, t_i, qloc_i);
    else if (exact)
      split_many<true, false>(lane, nh, lamhat_r, Dr, ures_i, R, ncol, qcol, t_i, qloc_i);
    else if (nh <= 16)
      split_many<false, true>(lane, nh, lamhat_r, Dr, ures_i, R, ncol, qcol, t_i, qloc_i);
    else
      split_many<false, false>(lane, nh, lamhat_r, Dr, ures_i, R, ncol, qcol, t_i, qloc_i);
  }
  // CSR padding columns of Q
  for (int j = total + e; j < ncol; j += E)
    if (lane < R) qrow[j] = 0;
}

// ---------------------------------------------------------------- emit

// kReroute: the same workgroup then runs SolveReroute for its expert from
// the values it has just produced (ultraep_plan's single-launch ending).
template <bool kReroute>
__global__ void __launch_bounds__(kWave) k_plan_emit(PlanArgs a) {
  __shared__ int32_t s_t[kRrLds];
  __shared__ uint32_t s_et[kMaxRec];
  __shared__ int32_t s_d[kMaxRec];
  __shared__ int32_t s_ht[kMaxR];  // hosts of this expert: rank
  __shared__ int32_t s_hu[kMaxR];  //                       quota
  __shared__ int32_t s_fan[kMaxE];
  const int e = blockIdx.x, lane = threadIdx.x;
  const int R = a.R, E = a.E, NS = a.NS, nm = a.nm, ncol = a.ncol, RS = R * NS;
  const int64_t status = a.ws.hdr[3], L = a.ws.hdr[2];
  const int64_t lo0 = a.ws.hdr[0], hi0 = a.ws.hdr[1];
  BisState fin = state_before(a, kRounds - 1);
  uint64_t bv[kCopies];
  outcome_load(a, kRounds - 1, bv);
  const int lam_e = a.ws.lam[e];
  const int lam_v = kReroute ? a.load[static_cast<int64_t>(min(lane, R - 1)) * E + e] : 0;
  asm volatile("" ::: "memory");  // the loads above go out before the status test
  const int lam_r = lane < R ? lam_v : 0;
  if (status != 0) {
    if (e == 0 && lane < 8) a.stats[lane] = lane == 6 ? ULTRAEP_EDATA : (lane == 7 ? L : 0);
    return;
  }
  walk_bits(outcome_or(bv), kRounds - 1, fin);
  int nb = 0;  // transfers of the last feasible probe, read into s_et / s_d
  if (fin.lo < fin.hi) {
    // a bisection longer than the rounds: the remaining probes run here, one
    // after another, the same ones in every workgroup
    __shared__ int32_t s_eorder[kMaxE];
    __shared__ int32_t s_elam[kMaxE];
    __shared__ uint32_t s_re[kMaxRec + kWave];
    __shared__ int32_t s_rd[kMaxRec + kWave];
    for (int i = lane; i < E; i += kWave) {
      s_eorder[i] = a.ws.eorder[i];
      s_elam[i] = a.ws.elam[i];
    }
    const int rk_r = lane < R ? a.ws.rank_desc[lane] : 0;
    const int as_r = lane < R ? a.ws.rank_asc[lane] : 0;
    const int ell_lane = lane < R ? a.ws.ell[lane] : 0;
    const int rk_l = __shfl(ell_lane, rk_r);
    const int as_l = __shfl(ell_lane, as_r);
    const bool packed = hi0 < (int64_t(1) << 25);
    bool local = false;
    __syncthreads();
    while (fin.lo < fin.hi) {
      const int64_t mid = (fin.lo + fin.hi) / 2;
      ++fin.probes;
      const int n = run_probe<1>(a, packed, static_cast<int>(mid), lane, rk_r, rk_l, as_r, as_l,
                              ell_lane, s_eorder, s_elam, s_re, s_rd);
      __syncthreads();
      if (n >= 0) {
        fin.hi = mid;
        local = true;
        nb = n;
        for (int i = lane; i < n; i += kWave) {
          s_et[i] = s_re[i];
          s_d[i] = s_rd[i];
        }
      } else {
        fin.lo = mid + 1;
      }
      __syncthreads();
    }
    if (local) fin.best = -2;  // records already in s_et / s_d
  }
  const int64_t hi = fin.hi;
  const int n_probe = fin.probes;
  const int best = fin.best;
  if (best >= 0) {
    // the count and the node's records are requested together: every slot's
    // record is read (at most RS), the ones past the count are dropped
    const uint32_t *rec = a.ws.rec + static_cast<int64_t>(best) * 2 * RS;
    uint32_t rv_e[kMaxRec / kWave], rv_d[kMaxRec / kWave];
#pragma unroll
    for (int u = 0; u < kMaxRec / kWave; ++u) {
      if (u * kWave < RS) {
        const int i = min(u * kWave + lane, RS - 1);
        rv_e[u] = rec[2 * i];
        rv_d[u] = rec[2 * i + 1];
      }
    }
    nb = a.ws.res[best];
#pragma unroll
    for (int u = 0; u < kMaxRec / kWave; ++u) {
      const int i = u * kWave + lane;
      if (u * kWave < RS && i < nb) {
        s_et[i] = rv_e[u];
        s_d[i] = static_cast<int32_t>(rv_d[u]);
      }
    }
  }
  __syncthreads();
  const int h = e / nm;

  // CSR row pointer: every expert has 1 + (its replicas) entries
  int before = 0, shed = 0;
  for (int i = lane; i < nb; i += kWave) {
    const int ei = static_cast<int>(s_et[i] & 0xFFFFu);
    before += ei < e;
    if (ei == e) shed += s_d[i];
  }
  before = wave_sum(before);
  shed = wave_sum(shed);
  const int hp_e = e + before;
  // this expert's replicas: position among them = replicas on lower ranks
  // (an expert's transfers go to distinct ranks, so a mask of them gives
  // it); slot on the host = earlier accepted transfers to the same rank,
  // from a match of equal ranks within 64 records and per-rank counts of
  // the records before them
  uint64_t tmask = 0;
  for (int i0 = 0; i0 < nb; i0 += kWave) {
    const int i = i0 + lane;
    const uint32_t x = i < nb ? s_et[i] : 0xFFFFFFFFu;  // expert field 0xFFFF: no expert
    uint64_t mb = ballot(static_cast<int>(x & 0xFFFFu) == e);
    while (mb) {
      const int l = __ffsll(static_cast<unsigned long long>(mb)) - 1;
      mb &= mb - 1;
      tmask |= uint64_t(1) << readlane(static_cast<int>(x >> 16), l);
    }
  }
  const int fan = __popcll(tmask);
  if (fan > 0) {
    const int tb = bits_for(R);
    for (int i = lane; i < kMaxR; i += kWave) s_fan[i] = 0;  // records per rank so far
    __syncthreads();
    for (int i0 = 0; i0 < nb; i0 += kWave) {
      const int i = i0 + lane;
      const bool valid = i < nb;
      const uint32_t x = valid ? s_et[i] : 0;
      const int t = static_cast<int>(x >> 16);
      const uint64_t same = match_any(static_cast<uint32_t>(t), tb, ballot(valid));
      const int before_t = valid ? s_fan[t] : 0;
      if (valid && static_cast<int>(x & 0xFFFFu) == e) {
        const int pos = __popcll(tmask & ((uint64_t(1) << t) - 1));
        const int slot = before_t + popc_below(same);
        s_ht[1 + pos] = t;
        s_hu[1 + pos] = s_d[i];
        a.hr[hp_e + 1 + pos] = t;
        a.hs[hp_e + 1 + pos] = nm + slot;
      }
      __syncthreads();
      if (valid && popc_below(same) == 0) s_fan[t] = before_t + __popcll(same);
      __syncthreads();
    }
  }
  const int nh = 1 + fan;
  if (lane == 0) {
    s_ht[0] = h;
    s_hu[0] = lam_e - shed;
    a.hp[e] = hp_e;
    a.hr[hp_e] = h;
    a.hs[hp_e] = e - h * nm;
    if (e == E - 1) a.hp[E] = E + nb;
  }
  for (int j = E + nb + e; j < ncol; j += E) {  // CSR padding
    if (lane == 0) {
      a.hr[j] = -1;
      a.hs[j] = -1;
    }
  }
  // row e of U
  __syncthreads();
  int u_r = 0;  // quota of this expert on rank `lane`
  for (int i = 0; i < nh; ++i)
    if (s_ht[i] == lane) u_r = s_hu[i];
  if (lane < R) a.U[static_cast<int64_t>(e) * R + lane] = u_r;
  (void)ncol;
  // row t = e of X (one workgroup per rank): slots in acceptance order
  if (e < R && NS > 0) {
    int cnt = 0;
    for (int i0 = 0; i0 < nb; i0 += kWave) {
      const int i = i0 + lane;
      const bool to_me = i < nb && static_cast<int>(s_et[i] >> 16) == e;
      const uint64_t mb = ballot(to_me);
      if (to_me) a.X[e * NS + cnt + popc_below(mb)] = static_cast<int>(s_et[i] & 0xFFFFu);
      cnt += __popcll(mb);
    }
    for (int s = cnt + lane; s < NS; s += kWave) a.X[e * NS + s] = -1;
  }
  if (e == 0) {  // stats
    for (int i = lane; i < E; i += kWave) s_fan[i] = 0;
    __syncthreads();
    for (int i = lane; i < nb; i += kWave) atomicAdd(&s_fan[s_et[i] & 0xFFFFu], 1);
    __syncthreads();
    int mf = 0;
    for (int i = lane; i < E; i += kWave) mf = max(mf, s_fan[i]);
    mf = wave_max(mf);
    if (lane == 0) {
      a.stats[0] = hi;
      a.stats[1] = lo0;
      a.stats[2] = hi0;
      a.stats[3] = n_probe;
      a.stats[4] = nb;
      a.stats[5] = 1 + mf;
      a.stats[6] = 0;
      a.stats[7] = L;
    }
  }
  if (kReroute) reroute_expert(a, e, hp_e, E + nb, lam_r, u_r, L, s_t);
}

__global__ void __launch_bounds__(kWave) k_plan_reroute(PlanArgs a) {
  __shared__ int32_t s_t[kRrLds];
  const int e = blockIdx.x, lane = threadIdx.x;
  const int R = a.R, E = a.E;
  const int64_t status = a.stats[6], L = a.stats[7];
  const int j0 = a.hp[e], total = a.hp[E];
  const int lam_r = lane < R ? a.load[static_cast<int64_t>(lane) * E + e] : 0;
  const int u_r = lane < R ? a.U[static_cast<int64_t>(e) * R + lane] : 0;
  if (status != 0) return;
  reroute_expert(a, e, j0, total, lam_r, u_r, L, s_t);
}

// SolveReroute and the local weight packing in one launch, as the forward
// pipeline overlaps them (Eq. 1): workgroup e < E runs expert e's split on
// its first wave, the others pack tiles.  Packing needs only the replica
// placement, which SolveReplication has already written.  The reroute
// workgroups come first so they are placed before the packing fills the
// chip.
__global__ void __launch_bounds__(kPkThreads) k_reroute_pack(PlanArgs a, PkArgs p) {
  __shared__ int32_t s_t[kRrLds];
  const int b = blockIdx.x;
  if (b < a.E) {
    if (threadIdx.x >= kWave) return;
    const int e = b, lane = threadIdx.x;
    const int R = a.R, E = a.E;
    const int64_t status = a.stats[6], L = a.stats[7];
    const int j0 = a.hp[e], total = a.hp[E];
    const int lam_r = lane < R ? a.load[static_cast<int64_t>(lane) * E + e] : 0;
    const int u_r = lane < R ? a.U[static_cast<int64_t>(e) * R + lane] : 0;
    if (status != 0) return;
    reroute_expert(a, e, j0, total, lam_r, u_r, L, s_t);
    return;
  }
  pack_block(p, b - a.E, static_cast<int64_t>(gridDim.x) - a.E, b == a.E);
}

static PlanArgs plan_args(const int32_t *load, const ultraep_group &g,
                          const ultraep_plan_buf &out, void *ws) {
  PlanArgs a{};
  a.load = load;
  a.R = g.R;
  a.E = g.E;
  a.NS = g.n_slot;
  a.nm = g.E / g.R;
  a.ncol = g.E + g.R * g.n_slot;
  a.u_min = static_cast<int32_t>(g.u_min > INT32_MAX ? INT32_MAX : g.u_min);
  a.beta_num = g.beta_num;
  a.beta_den = g.beta_den;
  a.X = out.slot_expert;
  a.U = out.quota;
  a.hp = out.host_ptr;
  a.hr = out.host_rank;
  a.hs = out.host_pslot;
  a.q = out.reroute;
  a.stats = out.stats;
  if (ws) a.ws = carve(ws, g.R, g.E, g.n_slot);
  return a;
}

hipError_t launch_plan_replicate(const int32_t *load, const ultraep_group &g,
                                 const ultraep_plan_buf &out, void *ws, hipStream_t stream) {
  const PlanArgs a = plan_args(load, g, out, ws);
  hipLaunchKernelGGL(k_plan_prep, dim3(1), dim3(kPrepThreads), 0, stream, a);
  hipError_t err = hipGetLastError();
  for (int round = 0; round < kRounds && err == hipSuccess; ++round) {
    hipLaunchKernelGGL(k_plan_round, dim3(kNodes), dim3(kWave), 0, stream, a, round);
    err = hipGetLastError();
  }
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(k_plan_emit<false>, dim3(g.E), dim3(kWave), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_plan(const int32_t *load, const ultraep_group &g,
                       const ultraep_plan_buf &out, void *ws, hipStream_t stream) {
  const PlanArgs a = plan_args(load, g, out, ws);
  hipLaunchKernelGGL(k_plan_prep, dim3(1), dim3(kPrepThreads), 0, stream, a);
  hipError_t err = hipGetLastError();
  for (int round = 0; round < kRounds && err == hipSuccess; ++round) {
    hipLaunchKernelGGL(k_plan_round, dim3(kNodes), dim3(kWave), 0, stream, a, round);
    err = hipGetLastError();
  }
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(k_plan_emit<true>, dim3(g.E), dim3(kWave), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_reroute_pack(const int32_t *load, const ultraep_group &g,
                               const ultraep_plan_buf &out, const uint16_t *w_main, int64_t W,
                               int32_t rank, uint16_t *staging, int64_t cap, int64_t *dest_off,
                               int32_t *status, hipStream_t stream) {
  const PlanArgs a = plan_args(load, g, out, nullptr);
  const PkArgs p = pack_args(w_main, W, rank, g, out, staging, cap, dest_off, status);
  hipLaunchKernelGGL(k_reroute_pack, dim3(g.E + kPkGrid), dim3(kPkThreads), 0, stream, a, p);
  return hipGetLastError();
}

hipError_t launch_plan_reroute(const int32_t *load, const ultraep_group &g,
                               const ultraep_plan_buf &out, hipStream_t stream) {
  const PlanArgs a = plan_args(load, g, out, nullptr);
  hipLaunchKernelGGL(k_plan_reroute, dim3(g.E), dim3(kWave), 0, stream, a);
  return hipGetLastError();
}

}  // namespace uep
