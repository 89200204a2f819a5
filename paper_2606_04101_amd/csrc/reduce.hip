// Gradient reduction, local half (Sec. 4.2 backward pass; the tile
// streaming of Sec. 6.1): the fp32 gradients of this rank's replicated main
// experts come back from their replicas and are accumulated into the main
// gradients; the replica buffers are then cleared in place, since the next
// layer reuses them.
//
// Arithmetic (read from the paper's fp32 gradient buffers; binding for this
// library and its tests): each main gradient element is summed in fp32
// starting from its own value and adding its replicas' elements in staging
// order (destination rank ascending, then slot), the order in which the
// forward packing laid the replicas out; every replica entry is zeroed.
//
// Bandwidth bound: a grid-stride loop over (expert, 8 KiB tile) tasks.  Each
// workgroup first lists, per replicated local expert, its staging entries in
// ascending order (a slot's entry is a ballot prefix over the slot map; its
// place inside the expert's list counts the earlier slots of that expert).
// A task loads the main tile, adds the replica tiles in that order, stores
// the sum and zeroes the replica tiles, all with 16-byte non-temporal
// accesses.
#include "common.hpp"
#include "kernels.hpp"

#pragma clang fp contract(off)

namespace uep {

constexpr int kRdThreads = 256;
constexpr int kRdWaves = kRdThreads / kWave;
constexpr int kRdUnroll = 2;                        // 16-byte chunks per thread per tile
constexpr int kRdTileCh = kRdThreads * kRdUnroll;   // 512 x 16 B = 8 KiB
constexpr int kRdMaxEnt = 256;                      // R * n_slot
constexpr int kRdMaxLocal = 1024;                   // main experts per rank
constexpr int kRdGrid = 1024;

struct RdArgs {
  v4u *main_grad;  // [nm][nch] fp32 as 16-byte chunks
  v4u *rgrad;      // [cap][nch]
  int64_t nch;
  int32_t rank, R, NS, nm;
  const int32_t *X;
  int64_t cap;
  int32_t *status;
};

__device__ __forceinline__ v4u add4(v4u a, v4u b) {
  v4u o;
  o.x = __float_as_uint(__fadd_rn(__uint_as_float(a.x), __uint_as_float(b.x)));
  o.y = __float_as_uint(__fadd_rn(__uint_as_float(a.y), __uint_as_float(b.y)));
  o.z = __float_as_uint(__fadd_rn(__uint_as_float(a.z), __uint_as_float(b.z)));
  o.w = __float_as_uint(__fadd_rn(__uint_as_float(a.w), __uint_as_float(b.w)));
  return o;
}

__global__ void __launch_bounds__(kRdThreads) k_grad_reduce(RdArgs a) {
  __shared__ int32_t s_li[kRdMaxEnt];        // local expert of each slot, -1
  __shared__ int32_t s_dst[kRdMaxEnt];       // entries grouped by expert, ascending
  __shared__ int32_t s_cnt[kRdMaxLocal];     // per local expert: replicas
  __shared__ int32_t s_gstart[kRdMaxLocal];  //                   first s_dst index
  __shared__ int32_t s_gli[kRdMaxEnt];       // per group: local expert
  __shared__ int32_t s_wcnt[kRdWaves];
  __shared__ int32_t s_off;
  const int tid = threadIdx.x, lane = lane_id(), wave = tid / kWave;
  const int RS = a.R * a.NS;
  for (int l = tid; l < a.nm; l += kRdThreads) s_cnt[l] = 0;
  int li = -1;
  if (tid < RS) {
    const int e = a.X[tid];
    if (e >= 0 && e / a.nm == a.rank) li = e - a.rank * a.nm;
  }
  const bool valid = li >= 0;
  const uint64_t bv = ballot(valid);
  if (lane == 0) s_wcnt[wave] = __popcll(bv);
  if (tid < kRdMaxEnt) s_li[tid] = li;
  if (tid == 0) s_off = 0;
  __syncthreads();
  // staging entry of this slot (destination rank, then slot) and the number
  // of replicas in all
  int entry = popc_below(bv), n_out = 0;
  for (int w = 0; w < kRdWaves; ++w) {
    entry += w < wave ? s_wcnt[w] : 0;
    n_out += s_wcnt[w];
  }
  if (n_out > a.cap) {
    if (blockIdx.x == 0 && tid == 0) report(a.status, ULTRAEP_ENOSPC);
    return;
  }
  if (n_out == 0) return;
  // place of this slot in its expert's list: earlier slots of the expert
  int pos = 0;
  if (valid)
    for (int j = 0; j < tid; ++j) pos += s_li[j] == li;
  if (valid) atomicAdd(&s_cnt[li], 1);
  __syncthreads();
  if (valid && pos == 0) s_gstart[li] = atomicAdd(&s_off, s_cnt[li]);
  // groups in ascending local-expert order, the same in every workgroup;
  // every thread keeps the running group count in a register
  int ngrp = 0;
  for (int l0 = 0; l0 < a.nm; l0 += kRdThreads) {
    const int l = l0 + tid;
    const bool has = l < a.nm && s_cnt[l] > 0;
    const uint64_t hb = ballot(has);
    int gi = ngrp + popc_below(hb);
    __syncthreads();  // the previous pass has read s_wcnt
    if (lane == 0) s_wcnt[wave] = __popcll(hb);
    __syncthreads();
    int tot = 0;
    for (int w = 0; w < kRdWaves; ++w) {
      gi += w < wave ? s_wcnt[w] : 0;
      tot += s_wcnt[w];
    }
    if (has) s_gli[gi] = l;
    ngrp += tot;
  }
  if (valid) s_dst[s_gstart[li] + pos] = entry;
  __syncthreads();
  const int64_t ntile = (a.nch + kRdTileCh - 1) / kRdTileCh;
  const int64_t ntask = ntile * ngrp;
  const v4u z = v4u{0u, 0u, 0u, 0u};
  for (int64_t task = blockIdx.x; task < ntask; task += gridDim.x) {
    const int l = s_gli[static_cast<int>(task % ngrp)];
    const int64_t c0 = (task / ngrp) * kRdTileCh;
    v4u *mg = a.main_grad + static_cast<int64_t>(l) * a.nch;
    v4u acc[kRdUnroll];
#pragma unroll
    for (int u = 0; u < kRdUnroll; ++u) {
      const int64_t c = c0 + u * kRdThreads + tid;
      if (c < a.nch) acc[u] = __builtin_nontemporal_load(mg + c);
    }
    const int fan = s_cnt[l], st = s_gstart[l];
#pragma unroll 4
    for (int f = 0; f < fan; ++f) {
      const v4u *rg = a.rgrad + static_cast<int64_t>(s_dst[st + f]) * a.nch;
#pragma unroll
      for (int u = 0; u < kRdUnroll; ++u) {
        const int64_t c = c0 + u * kRdThreads + tid;
        if (c < a.nch) acc[u] = add4(acc[u], __builtin_nontemporal_load(rg + c));
      }
    }
#pragma unroll
    for (int u = 0; u < kRdUnroll; ++u) {
      const int64_t c = c0 + u * kRdThreads + tid;
      if (c < a.nch) __builtin_nontemporal_store(acc[u], mg + c);
    }
    for (int f = 0; f < fan; ++f) {
      v4u *rg = a.rgrad + static_cast<int64_t>(s_dst[st + f]) * a.nch;
#pragma unroll
      for (int u = 0; u < kRdUnroll; ++u) {
        const int64_t c = c0 + u * kRdThreads + tid;
        if (c < a.nch) __builtin_nontemporal_store(z, rg + c);
      }
    }
  }
}

hipError_t launch_grad_reduce(float *main_grad, float *rgrad, int64_t W, int32_t rank,
                              const ultraep_group &g, const ultraep_plan_buf &plan, int64_t cap,
                              int32_t *status, hipStream_t stream) {
  RdArgs a;
  a.main_grad = reinterpret_cast<v4u *>(main_grad);
  a.rgrad = reinterpret_cast<v4u *>(rgrad);
  a.nch = W / 4;
  a.rank = rank;
  a.R = g.R;
  a.NS = g.n_slot;
  a.nm = g.E / g.R;
  a.X = plan.slot_expert;
  a.cap = cap;
  a.status = status;
  hipLaunchKernelGGL(k_grad_reduce, dim3(kRdGrid), dim3(kRdThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace uep
