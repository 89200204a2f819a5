// Step 4 — local half of the forward weight distribution (Sec. 6.1): every
// redundant slot that hosts one of this rank's main experts receives a copy
// of that expert's blob, in per-destination staging ordered by destination
// rank, then slot.
//
// One kernel with a persistent grid.  Each workgroup first derives the task
// list from the slot map in LDS (at most R * n_slot entries): the entry index
// of every destination, the replicated local experts and, per expert, its
// destination entries.  Workgroup 0 also writes dest_off.  The copy then
// walks tasks (expert, 32 KiB tile) with a grid stride, experts interleaved
// so hot and cold experts spread over all workgroups: each tile is loaded
// once into registers with 16-byte loads and stored to every destination
// with 16-byte non-temporal stores, so every source byte is read once.
#include "common.hpp"
#include "kernels.hpp"

namespace uep {

constexpr int kPkThreads = 256;
constexpr int kPkWaves = kPkThreads / kWave;
constexpr int kPkUnroll = 8;                        // v4u per thread per tile
constexpr int kPkTileCh = kPkThreads * kPkUnroll;   // 2048 x 16 B = 32 KiB
constexpr int kPkMaxEnt = 256;                      // R * n_slot
constexpr int kPkGrid = 2048;

struct PkArgs {
  const v4u *w;
  int64_t nch;  // 16-byte chunks per expert blob
  int32_t rank, R, NS, nm;
  const int32_t *X;
  v4u *staging;
  int64_t cap;
  int64_t *dest_off;
  int32_t *status;
};

__global__ void __launch_bounds__(kPkThreads) k_pack(PkArgs a) {
  __shared__ int32_t s_li[kPkMaxEnt];     // local expert of slot j, or -1
  __shared__ int32_t s_sorted[kPkMaxEnt]; // entries grouped by local expert
  __shared__ int32_t s_gli[kPkMaxEnt], s_gstart[kPkMaxEnt], s_gfan[kPkMaxEnt];
  __shared__ int32_t s_first[kPkMaxEnt];
  __shared__ int32_t s_wcnt[kPkWaves + 1];
  __shared__ int32_t s_ngrp;

  const int tid = threadIdx.x, lane = lane_id(), wave = tid / kWave;
  const int RS = a.R * a.NS;
  int li = -1;
  if (tid < RS) {
    const int e = a.X[tid];
    if (e >= 0 && e / a.nm == a.rank) li = e - a.rank * a.nm;
  }
  const bool valid = li >= 0;
  const uint64_t bv = ballot(valid);
  if (lane == 0) s_wcnt[wave] = __popcll(bv);
  s_li[tid] = li;
  if (tid == 0) s_ngrp = 0;
  __syncthreads();
  int before = popc_below(bv);
  for (int w = 0; w < wave; ++w) before += s_wcnt[w];
  int n_out = 0;
  for (int w = 0; w < kPkWaves; ++w) n_out += s_wcnt[w];

  if (blockIdx.x == 0) {
    for (int t = tid; t <= a.R; t += kPkThreads) {
      int c = 0;
      for (int j = 0; j < t * a.NS; ++j) c += s_li[j] >= 0;
      a.dest_off[t] = c;
    }
  }
  if (n_out > a.cap) {
    if (blockIdx.x == 0 && tid == 0) report(a.status, ULTRAEP_ENOSPC);
    return;
  }
  if (n_out == 0) return;
  int fidx = 0, smaller = 0, fan = 0;
  if (valid) {
    for (int j = 0; j < RS; ++j) {
      const int lj = s_li[j];
      if (lj < 0) continue;
      fidx += (lj == li) && (j < tid);
      fan += lj == li;
      smaller += lj < li;
    }
    s_sorted[smaller + fidx] = before;
  }
  s_first[tid] = valid && fidx == 0;
  __syncthreads();
  if (valid && fidx == 0) {
    int grp = 0;  // replicated local experts with a smaller index
    for (int j = 0; j < RS; ++j) grp += s_first[j] && s_li[j] < li;
    s_gli[grp] = li;
    s_gstart[grp] = smaller;
    s_gfan[grp] = fan;
    atomicAdd(&s_ngrp, 1);
  }
  __syncthreads();
  const int ngrp = s_ngrp;
  const int64_t ntile = (a.nch + kPkTileCh - 1) / kPkTileCh;
  const int64_t ntask = ntile * ngrp;
  for (int64_t task = blockIdx.x; task < ntask; task += gridDim.x) {
    const int g = static_cast<int>(task % ngrp);
    const int64_t c0 = (task / ngrp) * kPkTileCh;
    const v4u *src = a.w + static_cast<int64_t>(s_gli[g]) * a.nch;
    v4u v[kPkUnroll];
#pragma unroll
    for (int u = 0; u < kPkUnroll; ++u) {
      const int64_t c = c0 + u * kPkThreads + tid;
      if (c < a.nch) v[u] = __builtin_nontemporal_load(src + c);
    }
    const int fan = s_gfan[g], st = s_gstart[g];
    for (int f = 0; f < fan; ++f) {
      v4u *dst = a.staging + static_cast<int64_t>(s_sorted[st + f]) * a.nch;
#pragma unroll
      for (int u = 0; u < kPkUnroll; ++u) {
        const int64_t c = c0 + u * kPkThreads + tid;
        if (c < a.nch) __builtin_nontemporal_store(v[u], dst + c);
      }
    }
  }
}

hipError_t launch_pack(const uint16_t *w_main, int64_t W, int32_t rank,
                       const ultraep_group &g, const ultraep_plan_buf &plan,
                       uint16_t *staging, int64_t cap, int64_t *dest_off,
                       int32_t *status, hipStream_t stream) {
  PkArgs a;
  a.w = reinterpret_cast<const v4u *>(w_main);
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
  hipLaunchKernelGGL(k_pack, dim3(kPkGrid), dim3(kPkThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace uep
