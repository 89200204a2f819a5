// Relay trees for hot-expert fan-out (Sec. 6.2, load-aware relay
// scheduling): which rank sends each redundant slot its expert's blob.
//
// The paper tracks each rank's sending volume under the replication plan
// and then, one hot expert at a time, picks first-stage relays among the
// expert's replica ranks with the smallest volume and attaches every other
// replica to the relay whose volume stays smallest after taking it; the
// source's and relays' volumes are updated before the next expert.  The
// points the text leaves open are fixed as follows, for this library and
// for its tests alike:
//   - eligible: replica count f = |H(e)| - 1 exceeds the threshold (4 in the
//     paper);
//   - relay count: the integer nearest sqrt(f) (no ties for integer f);
//   - volume unit: one expert blob; a rank starts with one blob per replica
//     of each of its main experts;
//   - hot experts by f descending, then id ascending;
//   - relays: the replica ranks of smallest volume, ties to the smaller rank;
//   - leaves: the other replicas by ascending rank, each to the relay of
//     smallest volume (ties to the smaller rank), counted at once;
//   - after the expert, the source's volume drops by f minus the relays.
//
// One workgroup.  All threads validate the plan's host lists, seed the
// slot senders and volumes in LDS and sort the hot experts (a compacted
// list, ranked by counting).  The experts then depend on each other only
// through the volumes, so one wave walks them in order: a replica per lane
// (f <= R - 1 <= 63), relays chosen by each lane counting the lanes with a
// smaller (volume, rank) key, leaves attached one after another with a wave
// minimum over the relays' keys.
#include "common.hpp"
#include "kernels.hpp"

namespace uep {

constexpr int kRlThreads = 1024;
constexpr int kRlMaxSlots = 256;   // R * n_slot

struct RlArgs {
  int32_t R, E, NS, nm, ncol, threshold;
  const int32_t *X, *hp, *hr, *hs;
  const int64_t *plan_stats;
  int32_t *slot_src, *send_vol;
  int64_t *stats;
  int32_t *status;
};

__device__ __forceinline__ int nearest_sqrt(int f) {
  int n = 0;
  while ((n + 1) * (n + 1) <= f) ++n;
  return f > n * n + n ? n + 1 : n;
}

__device__ __forceinline__ int wave_min(int v) {
  v = min(v, __builtin_amdgcn_update_dpp(v, v, 0xB1, 0xF, 0xF, false));   // quad_perm 1,0,3,2
  v = min(v, __builtin_amdgcn_update_dpp(v, v, 0x4E, 0xF, 0xF, false));   // quad_perm 2,3,0,1
  v = min(v, __builtin_amdgcn_update_dpp(v, v, 0x141, 0xF, 0xF, false));  // row_half_mirror
  v = min(v, __builtin_amdgcn_update_dpp(v, v, 0x140, 0xF, 0xF, false));  // row_mirror
  int a = readlane(v, 0), b = readlane(v, 16), c = readlane(v, 32), d = readlane(v, 48);
  return __builtin_amdgcn_readfirstlane(min(min(a, b), min(c, d)));
}

__global__ void __launch_bounds__(kRlThreads) k_relay(RlArgs a) {
  __shared__ int32_t s_src[kRlMaxSlots];
  __shared__ int32_t s_vol[kWave];
  __shared__ int32_t s_hot[kRlMaxSlots];   // hot experts, unsorted
  __shared__ int32_t s_ord[kRlMaxSlots];   // sorted
  __shared__ int32_t s_wcnt[kRlThreads / kWave];
  __shared__ int32_t s_bad, s_nhot;
  const int tid = threadIdx.x, lane = lane_id(), wave = tid / kWave;
  const int R = a.R, E = a.E, NS = a.NS, nm = a.nm, RS = R * NS;
  if (tid < kWave) s_vol[tid] = 0;
  if (tid == 0) {
    s_bad = a.plan_stats[6] != 0;
    s_nhot = 0;
  }
  __syncthreads();
  // host lists: home first, then replicas by ascending rank on the slot
  // that holds the expert
  const int total = a.hp[E];
  if (a.hp[0] != 0 || total < E || total > a.ncol) s_bad = 1;
  int f = -1;
  if (tid < E) {
    const int e = tid, h = e / nm;
    const int j0 = a.hp[e], j1 = a.hp[e + 1];
    bool ok = j0 >= 0 && j1 > j0 && j1 <= a.ncol && j1 - j0 <= R;
    if (ok) ok = a.hr[j0] == h && a.hs[j0] == e - h * nm;
    for (int j = j0 + 1; ok && j < j1; ++j) {
      const int t = a.hr[j], s = a.hs[j] - nm;
      ok = t >= 0 && t < R && t != h && s >= 0 && s < NS && a.X[t * NS + s] == e &&
           (j == j0 + 1 || t > a.hr[j - 1]);
    }
    if (!ok) s_bad = 1;
    else f = j1 - j0 - 1;
  }
  // senders start at the home ranks; volumes count one blob per replica
  if (tid < RS) {
    const int e = a.X[tid];
    const bool ok = e >= -1 && e < E;
    if (!ok) s_bad = 1;
    const int h = ok && e >= 0 ? e / nm : -1;
    s_src[tid] = h;
    if (h >= 0) atomicAdd(&s_vol[h], 1);
  }
  // compact the hot experts
  const bool hot = f > a.threshold;
  const uint64_t hb = ballot(hot);
  if (lane == 0) s_wcnt[wave] = __popcll(hb);
  __syncthreads();
  if (s_bad) {
    if (tid == 0) report(a.status, ULTRAEP_EDATA);
    return;
  }
  int pos = popc_below(hb);
  for (int w = 0; w < wave; ++w) pos += s_wcnt[w];
  if (hot) s_hot[pos] = tid;
  if (tid == kRlThreads - 1) {
    int n = 0;
    for (int w = 0; w < kRlThreads / kWave; ++w) n += s_wcnt[w];
    s_nhot = n;
  }
  __syncthreads();
  const int nhot = s_nhot;
  // order: replica count descending, then id ascending (rank by counting)
  if (tid < nhot) {
    const int e = s_hot[tid], fe = a.hp[e + 1] - a.hp[e];
    int r = 0;
    for (int i = 0; i < nhot; ++i) {
      const int o = s_hot[i], fo = a.hp[o + 1] - a.hp[o];
      r += fo > fe || (fo == fe && o < e);
    }
    s_ord[r] = e;
  }
  int vmax0 = 0;
  if (wave == 0) vmax0 = wave_max(lane < R ? s_vol[lane] : 0);
  __syncthreads();
  int n_relays = 0;
  if (wave == 0) {
    for (int hi = 0; hi < nhot; ++hi) {
      const int e = s_ord[hi];
      const int j0 = a.hp[e], fe = a.hp[e + 1] - j0 - 1;
      const int n = nearest_sqrt(fe);
      const bool act = lane < fe;
      const int t = act ? a.hr[j0 + 1 + lane] : 0;
      const int s = act ? a.hs[j0 + 1 + lane] - nm : 0;
      int v = act ? s_vol[t] : 0;
      // relays: the n lanes of smallest (volume, rank)
      const int key = act ? (v << 6) | t : INT32_MAX;
      int below = 0;
      for (int l = 0; l < fe; ++l) below += readlane(key, l) < key;
      const bool relay = act && below < n;
      // leaves, ascending rank, each to the relay of smallest (volume, rank)
      uint64_t leaves = ballot(act && !relay);
      while (leaves) {
        const int l = __builtin_ctzll(leaves);
        leaves &= leaves - 1;
        const int m = wave_min(relay ? (v << 6) | t : INT32_MAX);
        const int win = m & 63;
        if (relay && t == win) v += 1;
        if (lane == l) s_src[t * NS + s] = win;
      }
      if (relay) s_vol[t] = v;
      if (lane == 0) s_vol[e / nm] -= fe - n;
      n_relays += n;
    }
  }
  __syncthreads();
  for (int i = tid; i < RS; i += kRlThreads) a.slot_src[i] = s_src[i];
  if (tid < R) a.send_vol[tid] = s_vol[tid];
  if (wave == 0) {
    const int vmax1 = wave_max(lane < R ? s_vol[lane] : 0);
    if (lane == 0) {
      a.stats[0] = nhot;
      a.stats[1] = n_relays;
      a.stats[2] = vmax0;
      a.stats[3] = vmax1;
    }
  }
}

hipError_t launch_relay(const ultraep_group &g, const ultraep_plan_buf &plan, int32_t threshold,
                        int32_t *slot_src, int32_t *send_vol, int64_t *stats, int32_t *status,
                        hipStream_t stream) {
  RlArgs a;
  a.R = g.R;
  a.E = g.E;
  a.NS = g.n_slot;
  a.nm = g.E / g.R;
  a.ncol = g.E + g.R * g.n_slot;
  a.threshold = threshold;
  a.X = plan.slot_expert;
  a.hp = plan.host_ptr;
  a.hr = plan.host_rank;
  a.hs = plan.host_pslot;
  a.plan_stats = plan.stats;
  a.slot_src = slot_src;
  a.send_vol = send_vol;
  a.stats = stats;
  a.status = status;
  hipLaunchKernelGGL(k_relay, dim3(1), dim3(kRlThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace uep
