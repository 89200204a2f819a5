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
//   k_plan_round  x3 launches of 1023 one-wave workgroups.  Each workgroup
//                 replays the walk of the earlier rounds from their stored
//                 outcomes, then runs the probe of its node of the next depth-10
//                 subtree of the bisection (one probe per wave on its own SIMD,
//                 so the 1023 probes of a round run at single-probe latency).
//                 Three depth-10 rounds cover any range below 2^30.  In a probe
//                 lane t holds rank t's slack and slot count; the target of
//                 largest slack (ties: lower rank) is one DPP wave max over a
//                 packed (slack, rank) key; the accepted transfers are kept in
//                 LDS and stored once at the end if the probe is feasible.
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

namespace uep {

constexpr int kMaxE = 1024;
constexpr int kMaxR = 64;
constexpr int kMaxRec = 256;               // R * n_slot: one transfer per slot at most
constexpr int kDepth = 10;                 // bisection levels per round
constexpr int kNodes = (1 << kDepth) - 1;  // probes per round
constexpr int kRounds = 3;                 // 30 levels
constexpr int64_t kMaxLoad = int64_t(1) << 30;
constexpr int kNotReached = INT32_MIN;
constexpr int kPrepThreads = 1024;
constexpr int kHdr = 4 + 4 * kRounds;  // int64 header words

struct PlanWs {
  int64_t *hdr;        // [4] tau_lo0, tau_hi0, L, status, then per round j the
                       // bisection state after rounds 0..j: lo, hi, best, probes
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
  return static_cast<size_t>(kHdr * 8 + (ints * 4 + 255) / 256 * 256);
}

static PlanWs carve(void *ws, int32_t R, int32_t E, int32_t NS) {
  (void)NS;
  PlanWs w;
  w.hdr = static_cast<int64_t *>(ws);
  int32_t *p = reinterpret_cast<int32_t *>(w.hdr + kHdr);
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
  if (tid < kWave) {  // ranks by descending load (ties: lower rank); R <= 64
    const int l = tid < R ? s_ell[tid] : -1;
    if (tid < R) {
      int pos = 0;
      for (int r = 0; r < R; ++r) {
        const int lr = s_ell[r];
        pos += (lr > l) || (lr == l && r < tid);
      }
      a.ws.rank_desc[pos] = tid;
      int apos = 0;  // ascending load, ties: lower rank
      for (int r = 0; r < R; ++r) {
        const int lr = s_ell[r];
        apos += (lr < l) || (lr == l && r < tid);
      }
      a.ws.rank_asc[apos] = tid;
    }
    const int hi = wave_max(l);
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

// Walks the depth-kDepth subtree of one round over its stored outcomes
// (s_res), from [lo, hi): updates the interval, the last feasible node and
// the number of probes of the sequential bisection.
__device__ void walk_round(const int32_t *s_res, int64_t &lo, int64_t &hi, int &best,
                           int &n_probe) {
  int node = 0;
  for (int d = 0; d < kDepth && lo < hi; ++d) {
    const int64_t mid = (lo + hi) / 2;
    ++n_probe;
    if (uni(s_res[node]) >= 0) {
      hi = mid;
      best = node;
      node = 2 * node + 1;
    } else {
      lo = mid + 1;
      node = 2 * node + 2;
    }
  }
}

// All kNodes outcomes of one round into LDS: 16 independent loads per lane.
__device__ void load_round(const int32_t *res, int32_t *s_res, int lane) {
  int v[16];
#pragma unroll
  for (int u = 0; u < 16; ++u) {
    const int i = u * kWave + lane;
    v[u] = i < kNodes ? __builtin_nontemporal_load(res + i) : 0;
  }
#pragma unroll
  for (int u = 0; u < 16; ++u) {
    const int i = u * kWave + lane;
    if (i < kNodes) s_res[i] = v[u];
  }
}

// DPP wave_shl:1 - lane i receives lane i+1 (lane 63 keeps its value)
__device__ __forceinline__ int wave_shl1(int v) {
  return __builtin_amdgcn_update_dpp(v, v, 0x130, 0xF, 0xF, false);
}

// One greedy feasibility probe at threshold tau, run by one wave.  Lane i
// holds the i-th rank of the visiting order (rk_r) and its load (rk_l).
// Returns the number of transfers (recorded in s_re / s_rd) if feasible,
// else a negative value.
//
// Admissible targets (slack > 0, a free slot) are kept as a list sorted by
// (slack descending, rank ascending) across the lanes from the head `h`
// on, each as a packed key (slack << 6) | (63 - rank) (slacks < 2^25) with
// its used-slot count beside it.  The list starts as the ranks in ascending
// load order (the same order at every threshold) cut at load < tau.  A
// transfer reads the head; a target whose slack or slots run out leaves the
// list by advancing h (always, with one slot per rank), otherwise it moves
// back to its place in the order.  Transfer n is kept in lane n % 64 of two
// registers, written to LDS every 64 transfers.
template <bool kOneSlot>
__device__ int probe_sorted(const PlanArgs &a, int tau, int lane, int rk_r, int rk_l,
                            int as_r, int as_l, const int32_t *s_eorder,
                            const int32_t *s_elam, uint32_t *s_re, int32_t *s_rd) {
  int key = (lane < a.R && as_l < tau && a.NS > 0) ? ((tau - as_l) << 6) | (kWave - 1 - as_r) : 0;
  int used = 0;
  int h = 0, n = 0;
  uint32_t cur_et = 0;
  int cur_d = 0;
  for (int oi = 0; oi < a.R; ++oi) {
    int exc = readlane(rk_l, oi) - tau;
    if (exc <= 0) break;  // the remaining ranks are not overloaded
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
          // no admissible rank: the same holds for every later expert of r
          if (h >= kWave) return -1;
          const int kh = readlane(key, h);
          if (kh == 0) return -1;
          const int m = kh >> 6;
          const int d = min(min(exc, m), cap);
          if (d < a.u_min) {
            // bounded by the excess or the slack: every later expert of r
            // meets the same bound, so r keeps its excess
            if (min(exc, m) < a.u_min) return -1;
            break;  // bounded by this expert's remaining load: next expert
          }
          if (kOneSlot) {
            ++h;
          } else {
            const int uh = readlane(used, h) + 1;
            if (m == d || uh >= a.NS) {
              ++h;  // out of slack or slots
            } else {
              const int nk = ((m - d) << 6) | (kh & (kWave - 1));
              // new place p: after every listed key still larger than nk
              const int p = h + __popcll(ballot(lane > h && key > nk));
              const int ks = wave_shl1(key), us = wave_shl1(used);
              const bool mv = lane >= h && lane < p;
              key = mv ? ks : (lane == p ? nk : key);
              used = mv ? us : (lane == p ? uh : used);
            }
          }
          const bool me = lane == (n & (kWave - 1));
          cur_et = me ? (static_cast<uint32_t>(e) | (static_cast<uint32_t>(kWave - 1 - (kh & (kWave - 1))) << 16)) : cur_et;
          cur_d = me ? d : cur_d;
          ++n;
          if ((n & (kWave - 1)) == 0) {
            s_re[n - kWave + lane] = cur_et;
            s_rd[n - kWave + lane] = cur_d;
          }
          exc -= d;
          cap -= d;
        }
      }
    }
    if (exc > 0) return -1;
  }
  const int base = n & ~(kWave - 1);
  if (lane < (n & (kWave - 1))) {
    s_re[base + lane] = cur_et;
    s_rd[base + lane] = cur_d;
  }
  return n;
}

// The same probe for slacks of 25 bits or more: lane t holds rank t's slack
// and slot count, and the target is a wave max plus a ballot for the lowest
// rank among ties.
__device__ int probe_wide(const PlanArgs &a, int tau, int lane, int rk_r, int rk_l,
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

// Bisection state after rounds 0 .. upto: the state after the round before
// (header slot, or the initial interval), then a walk of round `upto` over
// its stored outcomes.
struct BisState {
  int64_t lo, hi;
  int best;   // last feasible probe: round * kNodes + node, or -1
  int probes; // probes of the sequential bisection so far
};

__device__ BisState state_after(const PlanArgs &a, int upto, int32_t *s_res, int lane) {
  BisState st;
  if (upto == 0) {
    st = {a.ws.hdr[0], a.ws.hdr[1], -1, 0};
  } else {
    const int64_t *h = a.ws.hdr + 4 + 4 * (upto - 1);
    st = {h[0], h[1], static_cast<int>(h[2]), static_cast<int>(h[3])};
  }
  if (st.lo < st.hi) {
    load_round(a.ws.res + upto * kNodes, s_res, lane);
    __syncthreads();
    int best = -1;
    walk_round(s_res, st.lo, st.hi, best, st.probes);
    if (best >= 0) st.best = upto * kNodes + best;
  }
  return st;
}

__global__ void __launch_bounds__(kWave) k_plan_round(PlanArgs a, int round) {
  __shared__ int32_t s_res[kNodes];
  __shared__ int32_t s_eorder[kMaxE];
  __shared__ int32_t s_elam[kMaxE];
  __shared__ uint32_t s_re[kMaxRec];
  __shared__ int32_t s_rd[kMaxRec];
  const int lane = threadIdx.x, b = blockIdx.x;
  const int RS = a.R * a.NS;
  if (a.ws.hdr[3] != 0) return;
  int64_t lo, hi;
  if (round == 0) {
    lo = a.ws.hdr[0];
    hi = a.ws.hdr[1];
  } else {
    // every workgroup walks the previous round; workgroup 0 publishes it
    const BisState st = state_after(a, round - 1, s_res, lane);
    if (b == 0 && lane == 0) {
      int64_t *h = a.ws.hdr + 4 + 4 * (round - 1);
      h[0] = st.lo;
      h[1] = st.hi;
      h[2] = st.best;
      h[3] = st.probes;
    }
    lo = st.lo;
    hi = st.hi;
  }
  if (lo >= hi) return;  // the bisection has ended
  const bool packed = a.ws.hdr[1] < (int64_t(1) << 25);
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
    {  // stage the per-rank expert orders: up to 16 loads per lane in flight
      for (int i0 = 0; i0 < a.E; i0 += 16 * kWave) {
        int ve[16], vl[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) {
          const int i = i0 + u * kWave + lane;
          ve[u] = i < a.E ? a.ws.eorder[i] : 0;
          vl[u] = i < a.E ? a.ws.elam[i] : 0;
        }
#pragma unroll
        for (int u = 0; u < 16; ++u) {
          const int i = i0 + u * kWave + lane;
          if (i < a.E) {
            s_eorder[i] = ve[u];
            s_elam[i] = vl[u];
          }
        }
      }
    }
    const int rk_r = lane < a.R ? a.ws.rank_desc[lane] : 0;
    const int as_r = lane < a.R ? a.ws.rank_asc[lane] : 0;
    const int ell_lane = lane < a.R ? a.ws.ell[lane] : 0;
    const int rk_l = __shfl(ell_lane, rk_r);
    const int as_l = __shfl(ell_lane, as_r);
    __syncthreads();
    if (!packed)
      n = probe_wide(a, tau, lane, rk_r, rk_l, ell_lane, s_eorder, s_elam, s_re, s_rd);
    else if (a.NS == 1)
      n = probe_sorted<true>(a, tau, lane, rk_r, rk_l, as_r, as_l, s_eorder, s_elam, s_re, s_rd);
    else
      n = probe_sorted<false>(a, tau, lane, rk_r, rk_l, as_r, as_l, s_eorder, s_elam, s_re, s_rd);
    if (n > 0) {
      __syncthreads();
      uint32_t *rec = a.ws.rec + (static_cast<int64_t>(round) * kNodes + b) * 2 * RS;
      for (int i = lane; i < n; i += kWave) {
        rec[2 * i] = s_re[i];
        rec[2 * i + 1] = static_cast<uint32_t>(s_rd[i]);
      }
    }
  }
  if (lane == 0) a.ws.res[round * kNodes + b] = n;
}

// ---------------------------------------------------------------- emit

__global__ void __launch_bounds__(kWave) k_plan_emit(PlanArgs a) {
  __shared__ int32_t s_res[kNodes];
  __shared__ uint32_t s_et[kMaxRec];
  __shared__ int32_t s_d[kMaxRec];
  __shared__ int32_t s_ht[kMaxR];  // hosts of this expert: rank
  __shared__ int32_t s_hu[kMaxR];  //                       quota
  __shared__ int32_t s_fan[kMaxE];
  const int e = blockIdx.x, lane = threadIdx.x;
  const int R = a.R, E = a.E, NS = a.NS, nm = a.nm, ncol = a.ncol, RS = R * NS;
  if (a.ws.hdr[3] != 0) {
    if (e == 0 && lane < 8) a.stats[lane] = lane == 6 ? ULTRAEP_EDATA : (lane == 7 ? a.ws.hdr[2] : 0);
    return;
  }
  const int64_t lo0 = a.ws.hdr[0], hi0 = a.ws.hdr[1];
  const BisState fin = state_after(a, kRounds - 1, s_res, lane);
  const int64_t hi = fin.hi;
  const int n_probe = fin.probes;
  const int best = fin.best;
  const int nb = best >= 0 ? a.ws.res[best] : 0;
  if (best >= 0) {
    const uint32_t *rec = a.ws.rec + static_cast<int64_t>(best) * 2 * RS;
    for (int i = lane; i < nb; i += kWave) {
      s_et[i] = rec[2 * i];
      s_d[i] = static_cast<int32_t>(rec[2 * i + 1]);
    }
  }
  __syncthreads();
  const int h = e / nm;
  const int lam_e = a.ws.lam[e];

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
  // this expert's replicas: position among them = replicas on lower ranks;
  // slot on the host = earlier accepted transfers to the same rank
  int fan = 0;
  for (int i0 = 0; i0 < nb; i0 += kWave) {
    const int i = i0 + lane;
    const bool mine = i < nb && static_cast<int>(s_et[i] & 0xFFFFu) == e;
    const uint64_t mb = ballot(mine);
    if (mine) {
      const int t = static_cast<int>(s_et[i] >> 16);
      int pos = 0, slot = 0;
      for (int j = 0; j < nb; ++j) {
        const uint32_t x = s_et[j];
        pos += static_cast<int>(x & 0xFFFFu) == e && static_cast<int>(x >> 16) < t;
        slot += j < i && static_cast<int>(x >> 16) == t;
      }
      s_ht[1 + pos] = t;
      s_hu[1 + pos] = s_d[i];
      a.hr[hp_e + 1 + pos] = t;
      a.hs[hp_e + 1 + pos] = nm + slot;
    }
    fan += __popcll(mb);
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
      a.stats[7] = a.ws.hdr[2];
    }
  }
}

// ---------------------------------------------------------------- reroute

// SolveReroute for expert blockIdx.x: hosts and quotas from the CSR lists
// and U written by k_plan_emit, the expert's column of the load matrix.
template <bool kExact, bool kOneRow>
__device__ void split_expert(const PlanArgs &a, int e, int lane, int j0, int nh, int lam_r,
                             int u_r, int t_i, int u_i) {
  const int R = a.R, ncol = a.ncol;
  // locality: a source that hosts e first consumes its own quota
  const int loc_r = min(lam_r, u_r);
  const int lamhat_r = lam_r - loc_r;
  const int qloc_i = __shfl(loc_r, t_i);
  int ures = lane < nh ? u_i - qloc_i : 0;
  // residual quota total seen by source r: D_0 minus the demand of the
  // sources before it; its reciprocal, all computed lane-parallel up front
  int incl = lamhat_r;
  for (int o = 1; o < kWave; o <<= 1) {
    const int t = __shfl_up(incl, o);
    if (lane >= o) incl += t;
  }
  const int D0 = wave_sum(ures);
  const int Dr = D0 - (incl - lamhat_r);
  const double rDr = lamhat_r > 0 ? 1.0 / static_cast<double>(Dr) : 0.0;
  int32_t *qcol = a.q + j0 + lane;
  for (int r = 0; r < R; ++r) {
    const int lh = readlane(lamhat_r, r);
    int qi = 0;
    if (lh > 0) {
      const int D = readlane(Dr, r);
      const double rD = readlane_d(rDr, r);
      // floor(lh * ures / D): fp64 estimate (far below one unit off since
      // the quotient is < 2^30), made exact by one correction
      int b, rem;
      if (kExact) {  // all operands below 2^26: products below 2^52, exact
        const double Dd = static_cast<double>(D);
        const double pr = static_cast<double>(lh) * static_cast<double>(ures);
        double bq = __builtin_trunc(pr * rD);
        double rd = __builtin_fma(-bq, Dd, pr);
        const bool lo = rd < 0.0, hi = rd >= Dd;
        bq += lo ? -1.0 : (hi ? 1.0 : 0.0);
        rd += lo ? Dd : (hi ? -Dd : 0.0);
        b = static_cast<int>(bq);
        rem = static_cast<int>(rd);
      } else {
        b = static_cast<int>(static_cast<double>(lh) * static_cast<double>(ures) * rD);
        int64_t rm = static_cast<int64_t>(lh) * ures - static_cast<int64_t>(b) * D;
        const bool lo = rm < 0, hi = rm >= D;
        b += lo ? -1 : (hi ? 1 : 0);
        rm += lo ? D : (hi ? -D : 0);
        rem = static_cast<int>(rm);
      }
      const int left = lh - (kOneRow ? readlane(row_sum(b), 0) : wave_sum(b));
      int extra = 0;
      if (left > 0) {  // the `left` hosts with the largest remainders
        int rk = 0;
        for (int j = 0; j < nh; ++j) {
          const int rj = readlane(rem, j);
          rk += (rj > rem) || (rj == rem && j < lane);
        }
        extra = (lane < nh && rk < left) ? 1 : 0;
      }
      qi = b + extra;
      ures -= qi;
    }
    if (lane < nh) qcol[static_cast<int64_t>(r) * ncol] = qi + (t_i == r ? qloc_i : 0);
  }
}

__global__ void __launch_bounds__(kWave) k_plan_reroute(PlanArgs a) {
  const int e = blockIdx.x, lane = threadIdx.x;
  const int R = a.R, E = a.E, ncol = a.ncol;
  if (a.stats[6] != 0) return;
  const int j0 = a.hp[e], nh = a.hp[e + 1] - j0, total = a.hp[E];
  const int lam_r = lane < R ? a.load[static_cast<int64_t>(lane) * E + e] : 0;
  if (nh == 1) {
    if (lane < R) a.q[static_cast<int64_t>(lane) * ncol + j0] = lam_r;
  } else {
    const int u_r = lane < R ? a.U[static_cast<int64_t>(e) * R + lane] : 0;
    const int t_i = lane < nh ? a.hr[j0 + lane] : 0;
    const int u_i = __shfl(u_r, t_i);
    const bool exact = a.stats[7] < (int64_t(1) << 26);
    if (exact && nh <= 16) split_expert<true, true>(a, e, lane, j0, nh, lam_r, u_r, t_i, u_i);
    else if (exact) split_expert<true, false>(a, e, lane, j0, nh, lam_r, u_r, t_i, u_i);
    else if (nh <= 16) split_expert<false, true>(a, e, lane, j0, nh, lam_r, u_r, t_i, u_i);
    else split_expert<false, false>(a, e, lane, j0, nh, lam_r, u_r, t_i, u_i);
  }
  // CSR padding columns of Q
  for (int j = total + e; j < ncol; j += E)
    for (int r = lane; r < R; r += kWave) a.q[static_cast<int64_t>(r) * ncol + j] = 0;
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
  hipLaunchKernelGGL(k_plan_emit, dim3(g.E), dim3(kWave), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_plan_reroute(const int32_t *load, const ultraep_group &g,
                               const ultraep_plan_buf &out, hipStream_t stream) {
  const PlanArgs a = plan_args(load, g, out, nullptr);
  hipLaunchKernelGGL(k_plan_reroute, dim3(g.E), dim3(kWave), 0, stream, a);
  return hipGetLastError();
}

}  // namespace uep
