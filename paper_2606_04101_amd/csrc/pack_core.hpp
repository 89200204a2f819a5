// Step 4 — the local half of the forward weight distribution (Sec. 6.1): every
// redundant slot that hosts one of this rank's main experts receives a copy
// of that expert's blob, in per-destination staging ordered by destination
// rank, then slot.
//
// A grid-stride loop over (expert, 16 KiB tile) tasks.  Each
// workgroup first derives the tasks from the slot map in LDS (at most
// R * n_slot entries): a slot's staging entry is the number of this rank's
// replicas in earlier slots (a ballot prefix), and the entries are grouped
// by local expert with LDS counters (every destination of an expert gets the
// whole blob, so the order inside a group does not matter; the groups are
// numbered by ascending local expert in every workgroup).  One workgroup
// also writes dest_off.  Each tile is loaded once into registers with
// 16-byte loads and stored to every destination of its expert with 16-byte
// non-temporal stores, so every source byte is read once; the experts
// interleave so hot and cold ones spread over all workgroups.
//
// With relay trees (Sec. 6.2) a rank sends the slots whose sender it is:
// its own main experts' blobs to their relays and direct replicas, and the
// blobs it holds as a relay (its own redundant slot, filled by the first
// stage) to its leaves.  The groups are then numbered by source: main
// expert l < n_main, or the rank's redundant slot n_main + s.
//
// Used by k_pack, by the kernel that runs it alongside SolveReroute, and
// (RELAY) by k_pack_relay.
#pragma once

#include "common.hpp"
#include "kernels.hpp"

namespace uep {

constexpr int kPkThreads = 256;
constexpr int kPkWaves = kPkThreads / kWave;
constexpr int kPkUnroll = 4;                        // v4u per thread per tile
constexpr int kPkTileCh = kPkThreads * kPkUnroll;   // 1024 x 16 B = 16 KiB
constexpr int kPkMaxEnt = 256;                      // R * n_slot
constexpr int kPkMaxLocal = 1024 + 256;             // main experts + redundant slots
constexpr int kPkGrid = 4096;  // about one tile per workgroup at these sizes

struct PkArgs {
  const v4u *w;
  const v4u *relay_src;    // RELAY: this rank's redundant-slot blobs [NS][nch]
  int64_t nch;  // 16-byte chunks per expert blob
  int32_t rank, R, NS, nm;
  const int32_t *X;
  const int32_t *slot_src;  // RELAY: sender rank of every redundant slot
  v4u *staging;
  int64_t cap;
  int64_t *dest_off;
  int32_t *status;
};

// Workgroup wg of n_wg runs its share of the tasks; the one with writes_meta
// also writes dest_off and reports a capacity overflow (and, RELAY, a slot
// this rank should relay without hosting its expert).
template <bool RELAY = false>
__device__ __forceinline__ void pack_block(const PkArgs &a, int64_t wg, int64_t n_wg,
                                           bool writes_meta) {
  __shared__ int32_t s_dst[kPkMaxEnt];         // destination entries, grouped by expert
  __shared__ int32_t s_cnt[kPkMaxLocal];       // per local expert: destinations
  __shared__ int32_t s_gstart[kPkMaxLocal];    //                   first s_dst index
  __shared__ int32_t s_gli[kPkMaxEnt];         // per group: local expert
  __shared__ int32_t s_wcnt[kPkWaves];
  __shared__ int32_t s_off;

  const int tid = threadIdx.x, lane = lane_id(), wave = tid / kWave;
  const int RS = a.R * a.NS;
  const int nsrc = RELAY ? a.nm + a.NS : a.nm;  // source blobs
  for (int l = tid; l < nsrc; l += kPkThreads) s_cnt[l] = 0;
  int li = -1;
  bool orphan = false;
  if (tid < RS) {
    const int e = a.X[tid];
    if (!RELAY) {
      if (e >= 0 && e / a.nm == a.rank) li = e - a.rank * a.nm;
    } else if (e >= 0 && a.slot_src[tid] == a.rank) {
      if (e / a.nm == a.rank) {
        li = e - a.rank * a.nm;
      } else {  // relayed: the first stage filled this rank's slot holding e
        for (int s2 = 0; s2 < a.NS; ++s2)
          if (a.X[a.rank * a.NS + s2] == e) li = a.nm + s2;
        orphan = li < 0;
      }
    }
  }
  if (RELAY && orphan && writes_meta) report(a.status, ULTRAEP_EDATA);
  const bool valid = li >= 0;
  const uint64_t bv = ballot(valid);
  if (lane == 0) s_wcnt[wave] = __popcll(bv);
  if (tid == 0) s_off = 0;
  __syncthreads();
  // staging entry of this slot: valid slots before it (destination rank
  // ascending, then slot)
  int entry = popc_below(bv), n_out = 0;
  for (int w = 0; w < kPkWaves; ++w) {
    entry += w < wave ? s_wcnt[w] : 0;
    n_out += s_wcnt[w];
  }
  if (writes_meta) {
    if (a.NS == 0) {
      for (int t = tid; t <= a.R; t += kPkThreads) a.dest_off[t] = 0;
    } else {
      if (tid < RS && tid % a.NS == 0) a.dest_off[tid / a.NS] = entry;
      if (tid == 0) a.dest_off[a.R] = n_out;
    }
  }
  if (n_out > a.cap) {
    if (writes_meta && tid == 0) report(a.status, ULTRAEP_ENOSPC);
    return;
  }
  if (n_out == 0) return;
  // group the entries by local expert: every destination of an expert gets
  // the whole blob, so the order inside a group is free
  const int fidx = valid ? atomicAdd(&s_cnt[li], 1) : -1;
  __syncthreads();
  if (fidx == 0) s_gstart[li] = atomicAdd(&s_off, s_cnt[li]);
  // the groups themselves in ascending local-expert order, the same in
  // every workgroup, since tasks are numbered by group; every thread keeps
  // the running group count in a register (the pass totals are read from
  // LDS by all threads between the same two barriers)
  int ngrp = 0;
  for (int l0 = 0; l0 < nsrc; l0 += kPkThreads) {
    const int l = l0 + tid;
    const bool has = l < nsrc && s_cnt[l] > 0;
    const uint64_t hb = ballot(has);
    int gi = ngrp + popc_below(hb);
    __syncthreads();  // the previous pass has read s_wcnt
    if (lane == 0) s_wcnt[wave] = __popcll(hb);
    __syncthreads();
    int tot = 0;
    for (int w = 0; w < kPkWaves; ++w) {
      gi += w < wave ? s_wcnt[w] : 0;
      tot += s_wcnt[w];
    }
    if (has) s_gli[gi] = l;
    ngrp += tot;
  }
  if (valid) s_dst[s_gstart[li] + fidx] = entry;
  __syncthreads();
  const int64_t ntile = (a.nch + kPkTileCh - 1) / kPkTileCh;
  const int64_t ntask = ntile * ngrp;
  for (int64_t task = wg; task < ntask; task += n_wg) {
    const int l = s_gli[static_cast<int>(task % ngrp)];
    const int64_t c0 = (task / ngrp) * kPkTileCh;
    const v4u *src = !RELAY || l < a.nm ? a.w + static_cast<int64_t>(l) * a.nch
                                        : a.relay_src + static_cast<int64_t>(l - a.nm) * a.nch;
    v4u v[kPkUnroll];
#pragma unroll
    for (int u = 0; u < kPkUnroll; ++u) {
      const int64_t c = c0 + u * kPkThreads + tid;
      if (c < a.nch) v[u] = __builtin_nontemporal_load(src + c);
    }
    const int fan = s_cnt[l], st = s_gstart[l];
    for (int f = 0; f < fan; ++f) {
      v4u *dst = a.staging + static_cast<int64_t>(s_dst[st + f]) * a.nch;
#pragma unroll
      for (int u = 0; u < kPkUnroll; ++u) {
        const int64_t c = c0 + u * kPkThreads + tid;
        if (c < a.nch) __builtin_nontemporal_store(v[u], dst + c);
      }
    }
  }
}

inline PkArgs pack_args(const uint16_t *w_main, int64_t W, int32_t rank,
                        const ultraep_group &g, const ultraep_plan_buf &plan,
                        uint16_t *staging, int64_t cap, int64_t *dest_off, int32_t *status) {
  PkArgs a;
  a.w = reinterpret_cast<const v4u *>(w_main);
  a.relay_src = nullptr;
  a.slot_src = nullptr;
  a.nch = W / 8;
  a.rank = rank;
  a.R = g.R;
  a.NS = g.n_slot;
  a.nm = g.E / g.R;
  a.X = plan.slot_expert;
  a.staging = reinterpret_cast<v4u *>(staging);
  a.cap = cap;
  a.dest_off = dest_off;
  a.status = status;
  return a;
}

}  // namespace uep
