// Step 2 — Algorithm 1 of the paper on the device: SolveReplication (the
// threshold bisection with greedy feasibility probes of Sec. 5.1) and
// SolveReroute (locality-first proportional split of Sec. 5.2).
//
// k_plan_solve: ONE workgroup of 1024 threads (16 wave64s) on one CU.
//   - lambda_e, ell_r, the rank visiting order (descending excess is
//     descending ell for every threshold) and each rank's expert order
//     (descending lambda_e) are computed once and kept in LDS.
//   - Feasibility is not monotone in tau (the u_min floor), so the probes
//     must be exactly those of the printed sequential bisection.  Each round
//     evaluates the whole depth-4 subtree of the bisection below the current
//     [lo, hi): 15 probes, one per wave.  One thread then walks the subtree
//     with the 15 outcomes, which reproduces the sequential probe sequence,
//     and keeps the transfer record of the last feasible probe.
//   - In a probe, lane t holds rank t's slack and used-slot count; the
//     target of largest slack is a DPP wave max plus a ballot for the lowest
//     rank among ties, and all control values stay wave-uniform.
//   - The kept record is materialised into X, U and the CSR host lists.
// k_plan_reroute: one wave per expert; lanes are sources for the locality
//   pass and hosts for the proportional split, which walks the sources in
//   ascending rank order (largest remainder against the residual quotas).
#include "common.hpp"
#include "kernels.hpp"

namespace uep {

constexpr int kPlanThreads = 1024;
constexpr int kPlanWaves = kPlanThreads / kWave;
constexpr int kSpecNodes = 15;  // depth-4 bisection subtree per round
constexpr int kSpecDepth = 4;
constexpr int kMaxE = 1024;
constexpr int kMaxR = 64;
constexpr int kMaxRec = 256;  // R * n_slot: at most one transfer per slot
constexpr int64_t kMaxLoad = int64_t(1) << 30;

struct PlanArgs {
  const int32_t *load;
  int32_t R, E, NS, nm, ncol;
  int32_t u_min;  // clamped to int32 range
  int64_t beta_num, beta_den;
  int32_t *X, *U, *hp, *hr, *hs, *q;
  int64_t *stats;
};

__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }

// One greedy feasibility probe at threshold tau, run by a whole wave.
// Returns (feasible ? n : -1 - n) with n transfers recorded.
__device__ int probe_wave(const PlanArgs &a, int tau, int lane,
                          const int32_t *s_lam, const int32_t *s_ell,
                          const int32_t *s_rank_desc, const int32_t *s_eorder,
                          uint32_t *rec_et, int32_t *rec_d) {
  int slk = lane < a.R ? max(tau - s_ell[lane], 0) : 0;
  int used = 0;
  int n = 0;
  for (int oi = 0; oi < a.R; ++oi) {
    const int r = uni(s_rank_desc[oi]);
    int exc = uni(s_ell[r]) - tau;
    if (exc <= 0) break;  // the remaining ranks are not overloaded
    for (int j = 0; j < a.nm && exc > 0; ++j) {
      const int e = uni(s_eorder[r * a.nm + j]);
      int cap = uni(s_lam[e]);
      while (exc > 0 && cap > 0) {
        const int v = (slk > 0 && used < a.NS) ? slk : 0;
        const int m = wave_max(v);
        if (m == 0) break;  // no admissible rank
        const int ts = uni(__ffsll(static_cast<unsigned long long>(ballot(v == m))) - 1);
        const int d = min(min(exc, m), cap);
        if (d < a.u_min) break;
        if (lane == ts) {
          slk -= d;
          ++used;
        }
        if (lane == 0) {
          rec_et[n] = static_cast<uint32_t>(e) | (static_cast<uint32_t>(ts) << 16);
          rec_d[n] = d;
        }
        ++n;
        exc -= d;
        cap -= d;
      }
    }
    if (exc > 0) return -1 - n;
  }
  return n;
}

__device__ int block_exclusive_scan(int v, int *s_tmp, int *total) {
  // s_tmp: kPlanWaves + 1 ints
  const int lane = lane_id(), wave = threadIdx.x / kWave;
  int incl = v;
  for (int o = 1; o < kWave; o <<= 1) {
    int t = __shfl_up(incl, o);
    if (lane >= o) incl += t;
  }
  if (lane == kWave - 1) s_tmp[wave] = incl;
  __syncthreads();
  if (threadIdx.x == 0) {
    int run = 0;
    for (int w = 0; w < kPlanWaves; ++w) {
      int t = s_tmp[w];
      s_tmp[w] = run;
      run += t;
    }
    s_tmp[kPlanWaves] = run;
  }
  __syncthreads();
  int ex = s_tmp[wave] + incl - v;
  *total = s_tmp[kPlanWaves];
  __syncthreads();
  return ex;
}

__global__ void __launch_bounds__(kPlanThreads) k_plan_solve(PlanArgs a) {
  __shared__ int32_t s_lam[kMaxE];
  __shared__ int32_t s_eorder[kMaxE];
  __shared__ int32_t s_fan[kMaxE];
  __shared__ int32_t s_shed[kMaxE];
  __shared__ int32_t s_hp[kMaxE + 1];
  __shared__ int32_t s_ell[kMaxR];
  __shared__ int32_t s_rank_desc[kMaxR];
  __shared__ uint32_t s_rec_et[kSpecNodes][kMaxRec];
  __shared__ int32_t s_rec_d[kSpecNodes][kMaxRec];
  __shared__ uint32_t s_best_et[kMaxRec];
  __shared__ int32_t s_best_d[kMaxRec];
  __shared__ int32_t s_X[kMaxRec];
  __shared__ int32_t s_Xd[kMaxRec];
  __shared__ int32_t s_res[kSpecNodes];
  __shared__ int32_t s_tmp[kPlanWaves + 1];
  __shared__ int64_t s_lo, s_hi, s_lo0, s_hi0;
  __shared__ unsigned long long s_L;
  __shared__ int32_t s_bad, s_best_node, s_nbest, s_nprobe;

  const int tid = threadIdx.x, lane = lane_id(), wave = tid / kWave;
  const int R = a.R, E = a.E, NS = a.NS, nm = a.nm, RS = R * NS;

  if (tid == 0) {
    s_L = 0;
    s_bad = 0;
    s_nbest = 0;
    s_nprobe = 0;
  }
  __syncthreads();

  // lambda_e = sum_r lambda_{r,e}
  int64_t lam = 0;
  if (tid < E) {
    bool neg = false;
    for (int r = 0; r < R; ++r) {
      int v = a.load[static_cast<int64_t>(r) * E + tid];
      neg |= v < 0;
      lam += v;
    }
    if (neg || lam > kMaxLoad) atomicOr(&s_bad, 1);
    s_lam[tid] = static_cast<int32_t>(min(lam, kMaxLoad));
  }
  {
    int64_t ws = wave_sum64(lam);
    if (lane == 0) atomicAdd(&s_L, static_cast<unsigned long long>(ws));
  }
  __syncthreads();
  const int64_t L = static_cast<int64_t>(s_L);
  if (s_bad || L > kMaxLoad) {
    if (tid < 8) a.stats[tid] = tid == 6 ? ULTRAEP_EDATA : (tid == 7 ? L : 0);
    return;
  }
  // ell_r = sum of the loads of rank r's main experts
  if (tid < R) {
    int s = 0;
    for (int j = 0; j < nm; ++j) s += s_lam[tid * nm + j];
    s_ell[tid] = s;
  }
  // each rank's main experts by descending load (ties: lower id)
  if (tid < E) {
    const int r = tid / nm, l = s_lam[tid];
    int pos = 0;
    for (int j = r * nm; j < r * nm + nm; ++j) {
      int lj = s_lam[j];
      pos += (lj > l) || (lj == l && j < tid);
    }
    s_eorder[r * nm + pos] = tid;
  }
  __syncthreads();
  // ranks by descending load = descending excess at any threshold
  if (tid < R) {
    const int l = s_ell[tid];
    int pos = 0;
    for (int r = 0; r < R; ++r) {
      int lr = s_ell[r];
      pos += (lr > l) || (lr == l && r < tid);
    }
    s_rank_desc[pos] = tid;
  }
  if (tid == 0) {
    const int64_t m = (L + R - 1) / R;
    const int64_t lo = (a.beta_num * m + a.beta_den - 1) / a.beta_den;
    int64_t hi = 0;
    for (int r = 0; r < R; ++r) hi = max(hi, static_cast<int64_t>(s_ell[r]));
    s_lo = s_lo0 = lo;
    s_hi = s_hi0 = hi;
  }

  // ---- SolveReplication: speculative exact bisection -------------------
  for (;;) {
    __syncthreads();
    const int64_t lo = s_lo, hi = s_hi;
    if (lo >= hi) break;
    if (wave < kSpecNodes) {
      const int id = wave + 1;
      const int depth = 31 - __clz(id);
      int64_t l = lo, h = hi;
      bool ok = true;
      for (int b = depth - 1; b >= 0; --b) {
        if (l >= h) {
          ok = false;
          break;
        }
        const int64_t mid = (l + h) / 2;
        if ((id >> b) & 1) l = mid + 1;  // right child: the probe failed
        else h = mid;                    // left child: the probe succeeded
      }
      int res = INT32_MIN;  // node not reached
      if (ok && l < h)
        res = probe_wave(a, static_cast<int>((l + h) / 2), lane, s_lam, s_ell,
                         s_rank_desc, s_eorder, s_rec_et[wave], s_rec_d[wave]);
      if (lane == 0) s_res[wave] = res;
    }
    __syncthreads();
    if (tid == 0) {
      int64_t l = lo, h = hi;
      int node = 0, best = -1, np = 0;
      for (int d = 0; d < kSpecDepth && l < h; ++d) {
        const int64_t mid = (l + h) / 2;
        ++np;
        if (s_res[node] >= 0) {
          h = mid;
          best = node;
          node = 2 * node + 1;
        } else {
          l = mid + 1;
          node = 2 * node + 2;
        }
      }
      s_lo = l;
      s_hi = h;
      s_nprobe += np;
      s_best_node = best;
      if (best >= 0) s_nbest = s_res[best];
    }
    __syncthreads();
    const int best = s_best_node;
    if (best >= 0)
      for (int i = tid; i < s_nbest; i += kPlanThreads) {
        s_best_et[i] = s_rec_et[best][i];
        s_best_d[i] = s_rec_d[best][i];
      }
  }

  // ---- materialise X, U and the host lists ------------------------------
  const int nb = s_nbest;  // zero when no probe succeeded: identity plan
  for (int i = tid; i < RS; i += kPlanThreads) {
    s_X[i] = -1;
    s_Xd[i] = 0;
  }
  __syncthreads();
  if (tid < nb) {
    const uint32_t et = s_best_et[tid];
    const int t = static_cast<int>(et >> 16);
    int slot = 0;
    for (int j = 0; j < tid; ++j) slot += static_cast<int>(s_best_et[j] >> 16) == t;
    s_X[t * NS + slot] = static_cast<int>(et & 0xFFFFu);
    s_Xd[t * NS + slot] = s_best_d[tid];
  }
  __syncthreads();
  for (int i = tid; i < RS; i += kPlanThreads) a.X[i] = s_X[i];
  int fan = 0;
  if (tid < E) {
    int shed = 0;
    for (int j = 0; j < RS; ++j)
      if (s_X[j] == tid) {
        ++fan;
        shed += s_Xd[j];
      }
    s_fan[tid] = fan;
    s_shed[tid] = shed;
  }
  int total;
  const int ex = block_exclusive_scan(tid < E ? 1 + fan : 0, s_tmp, &total);
  if (tid < E) {
    s_hp[tid] = ex;
    a.hp[tid] = ex;
    const int h = tid / nm;
    a.hr[ex] = h;
    a.hs[ex] = tid - h * nm;
  }
  if (tid == 0) {
    s_hp[E] = total;
    a.hp[E] = total;
  }
  __syncthreads();
  if (tid < RS && s_X[tid] >= 0) {
    const int e = s_X[tid], t = tid / NS, s = tid - t * NS;
    int pos = 1;
    for (int j = 0; j < t * NS; ++j) pos += s_X[j] == e;
    const int ent = s_hp[e] + pos;
    a.hr[ent] = t;
    a.hs[ent] = nm + s;
  }
  for (int j = total + tid; j < a.ncol; j += kPlanThreads) {
    a.hr[j] = -1;
    a.hs[j] = -1;
  }
  for (int i = tid; i < E * R; i += kPlanThreads) {
    const int e = i / R, t = i - e * R;
    int v = 0;
    if (t == e / nm) {
      v = s_lam[e] - s_shed[e];
    } else {
      for (int s = 0; s < NS; ++s)
        if (s_X[t * NS + s] == e) v = s_Xd[t * NS + s];
    }
    a.U[i] = v;
  }
  // stats
  int maxh = 0;
  if (tid < E) maxh = 1 + s_fan[tid];
  maxh = wave_max(maxh);
  if (lane == 0) s_tmp[wave] = maxh;
  __syncthreads();
  if (tid == 0) {
    int mh = 0;
    for (int w = 0; w < kPlanWaves; ++w) mh = max(mh, s_tmp[w]);
    a.stats[0] = s_hi;
    a.stats[1] = s_lo0;
    a.stats[2] = s_hi0;
    a.stats[3] = s_nprobe;
    a.stats[4] = nb;
    a.stats[5] = mh;
    a.stats[6] = 0;
    a.stats[7] = L;
  }
}

// ---- SolveReroute: one wave per expert ---------------------------------
__global__ void __launch_bounds__(kWave) k_plan_reroute(PlanArgs a) {
  const int e = blockIdx.x, lane = threadIdx.x;
  const int R = a.R, E = a.E, ncol = a.ncol;
  if (a.stats[6] != 0) return;
  const int j0 = a.hp[e], nh = a.hp[e + 1] - j0, total = a.hp[E];
  // zero the CSR padding columns (spread over the expert blocks)
  for (int j = total + e; j < ncol; j += E)
    for (int r = lane; r < R; r += kWave) a.q[static_cast<int64_t>(r) * ncol + j] = 0;

  const int lam_r = lane < R ? a.load[static_cast<int64_t>(lane) * E + e] : 0;
  if (nh == 1) {
    if (lane < R) a.q[static_cast<int64_t>(lane) * ncol + j0] = lam_r;
    return;
  }
  // locality: each source that hosts e first consumes its own quota
  const int u_r = lane < R ? a.U[static_cast<int64_t>(e) * R + lane] : 0;
  const int loc_r = min(lam_r, u_r);
  const int lamhat_r = lam_r - loc_r;
  const int t_i = lane < nh ? a.hr[j0 + lane] : 0;
  const int u_i = lane < nh ? a.U[static_cast<int64_t>(e) * R + t_i] : 0;
  const int qloc_i = __shfl(loc_r, t_i);
  int ures = lane < nh ? u_i - qloc_i : 0;
  int D = wave_sum(ures);
  for (int r = 0; r < R; ++r) {
    const int lh = readlane(lamhat_r, r);
    int qi = 0;
    if (lh > 0) {
      const uint64_t prod = static_cast<uint64_t>(lh) * static_cast<uint64_t>(ures);
      const int base = static_cast<int>(prod / static_cast<uint64_t>(D));
      const int rem = static_cast<int>(prod - static_cast<uint64_t>(base) * static_cast<uint64_t>(D));
      const int left = lh - wave_sum(base);
      int extra = 0;
      if (left > 0) {
        int rk = 0;
        for (int j = 0; j < nh; ++j) {
          const int rj = readlane(rem, j);
          rk += (rj > rem) || (rj == rem && j < lane);
        }
        extra = (lane < nh && rk < left) ? 1 : 0;
      }
      qi = base + extra;
      ures -= qi;
      D -= lh;
    }
    if (lane < nh)
      a.q[static_cast<int64_t>(r) * ncol + j0 + lane] = qi + (t_i == r ? qloc_i : 0);
  }
}

hipError_t launch_plan(const int32_t *load, const ultraep_group &g,
                       const ultraep_plan_buf &out, hipStream_t stream) {
  PlanArgs a;
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
  hipLaunchKernelGGL(k_plan_solve, dim3(1), dim3(kPlanThreads), 0, stream, a);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(k_plan_reroute, dim3(g.E), dim3(kWave), 0, stream, a);
  return hipGetLastError();
}

}  // namespace uep
