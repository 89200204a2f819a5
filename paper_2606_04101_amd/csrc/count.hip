// Step 1 — exact per-expert loads lambda_{r,e} from top-k routing ids
// (Table 1; gathered after gating in the forward pipeline of Sec. 4.2).
//
// Up to kSplitIds ids per block: one workgroup of 1024 threads per block of
// T*k ids.  Every thread issues all of its 16-byte loads of a batch before
// using any (one memory latency per batch instead of one per id), then adds
// each id into its wave's private LDS histogram with an LDS atomic: a
// histogram needs no order, so the per-wave privatisation bounds contention
// to the 64 lanes of one wave.  The 16 wave histograms are summed at the end
// and every count is written (no global atomics, no zero-fill).
// Larger blocks: one workgroup's LDS atomics become the limit (hot experts
// make the lanes of an atomic collide), so a fill kernel zeroes the counts
// and a grid of 256-thread workgroups, each counting 2048 or 4096 ids into
// per-wave LDS histograms, adds its non-zero bins with global atomics.
// (Aggregating equal ids within a wave first, with bit-sliced ballot
// matches and one LDS add per distinct id, measured five times slower: the
// ballots cost far more than the collisions they save.)
#include "common.hpp"
#include "kernels.hpp"

namespace uep {

constexpr int kCountThreads = 1024;
constexpr int kCountWaves = kCountThreads / kWave;
constexpr int kCountBatch = 8;  // int4 loads in flight per thread

__device__ __forceinline__ bool count_one(int32_t e, int32_t E, int32_t *wh) {
  if (e >= 0 && e < E) atomicAdd(wh + e, 1);
  return e < -1 || e >= E;
}

__global__ void __launch_bounds__(kCountThreads)
k_count(const int32_t *__restrict__ topk, int64_t V, int32_t E,
        int32_t *__restrict__ counts, int32_t *status) {
  extern __shared__ int32_t hist[];  // [kCountWaves][E]
  const int wave = threadIdx.x / kWave;
  for (int i = threadIdx.x; i < kCountWaves * E; i += kCountThreads) hist[i] = 0;
  __syncthreads();

  const int32_t *src = topk + static_cast<int64_t>(blockIdx.x) * V;
  int32_t *wh = hist + wave * E;
  bool bad = false;
  // the block's rows are 4-aligned only if V is: otherwise use scalar loads
  const bool vec = (V % 4 == 0) && ((reinterpret_cast<uintptr_t>(src) & 15u) == 0);
  if (vec) {
    const v4i *s4 = reinterpret_cast<const v4i *>(src);
    const int64_t n4 = V / 4;
    for (int64_t b = 0; b < n4; b += int64_t(kCountThreads) * kCountBatch) {
      v4i v[kCountBatch];
#pragma unroll
      for (int u = 0; u < kCountBatch; ++u) {
        const int64_t i = b + u * kCountThreads + threadIdx.x;
        v[u] = i < n4 ? __builtin_nontemporal_load(s4 + i) : v4i{-1, -1, -1, -1};
      }
#pragma unroll
      for (int u = 0; u < kCountBatch; ++u) {
        bad |= count_one(v[u].x, E, wh);
        bad |= count_one(v[u].y, E, wh);
        bad |= count_one(v[u].z, E, wh);
        bad |= count_one(v[u].w, E, wh);
      }
    }
  } else {
    for (int64_t i = threadIdx.x; i < V; i += kCountThreads) bad |= count_one(src[i], E, wh);
  }
  if (bad) report(status, ULTRAEP_EDATA);
  __syncthreads();
  int32_t *dst = counts + static_cast<int64_t>(blockIdx.x) * E;
  for (int e = threadIdx.x; e < E; e += kCountThreads) {
    int s = 0;
#pragma unroll
    for (int w = 0; w < kCountWaves; ++w) s += hist[w * E + e];
    dst[e] = s;
  }
}

// Above kSplitIds ids per block the split path runs; its workgroups take
// 2048 ids each up to kSplitSmall ids per block, 4096 above (measured on one
// rank's block of the workloads here: 32768 ids count in 4.1 us split
// against 5.6 us in one workgroup, 131072 ids in 4.8 us with 4096 per
// workgroup against 5.0 us with 2048).
constexpr int64_t kSplitIds = 16384;
constexpr int64_t kSplitSmall = 65536;
constexpr int kSplitThreads = 256;
constexpr int kSplitWaves = kSplitThreads / kWave;

__global__ void __launch_bounds__(kSplitThreads)
k_count_zero(int32_t *__restrict__ counts, int64_t n) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * kSplitThreads + threadIdx.x;
  if (i < n) counts[i] = 0;
}

// blockIdx.y = block of ids, blockIdx.x = its part of kPerWg ids
template <int kPerWg>
__global__ void __launch_bounds__(kSplitThreads)
k_count_split(const int32_t *__restrict__ topk, int64_t V, int32_t E,
              int32_t *__restrict__ counts, int32_t *status) {
  constexpr int kSplitPerWg = kPerWg;
  extern __shared__ int32_t hist[];  // [kSplitWaves][E]
  const int wave = threadIdx.x / kWave;
  for (int i = threadIdx.x; i < kSplitWaves * E; i += kSplitThreads) hist[i] = 0;
  __syncthreads();
  const int32_t *src = topk + static_cast<int64_t>(blockIdx.y) * V;
  const int64_t b0 = static_cast<int64_t>(blockIdx.x) * kSplitPerWg;
  int32_t *wh = hist + wave * E;
  bool bad = false;
  const bool vec = (V % 4 == 0) && ((reinterpret_cast<uintptr_t>(src) & 15u) == 0);
  if (vec) {
    const v4i *s4 = reinterpret_cast<const v4i *>(src + b0);
    const int64_t n4 = (min(V - b0, static_cast<int64_t>(kSplitPerWg)) + 3) / 4;
    v4i v[kSplitPerWg / 4 / kSplitThreads];
#pragma unroll
    for (int u = 0; u < kSplitPerWg / 4 / kSplitThreads; ++u) {
      const int64_t i = u * kSplitThreads + threadIdx.x;
      v[u] = i < n4 ? __builtin_nontemporal_load(s4 + i) : v4i{-1, -1, -1, -1};
    }
#pragma unroll
    for (int u = 0; u < kSplitPerWg / 4 / kSplitThreads; ++u) {
      bad |= count_one(v[u].x, E, wh);
      bad |= count_one(v[u].y, E, wh);
      bad |= count_one(v[u].z, E, wh);
      bad |= count_one(v[u].w, E, wh);
    }
  } else {
    const int64_t end = min(V, b0 + kSplitPerWg);
    for (int64_t i = b0 + threadIdx.x; i < end; i += kSplitThreads) bad |= count_one(src[i], E, wh);
  }
  if (bad) report(status, ULTRAEP_EDATA);
  __syncthreads();
  int32_t *dst = counts + static_cast<int64_t>(blockIdx.y) * E;
  for (int e = threadIdx.x; e < E; e += kSplitThreads) {
    int s = 0;
#pragma unroll
    for (int w = 0; w < kSplitWaves; ++w) s += hist[w * E + e];
    if (s) atomicAdd(dst + e, s);
  }
}

hipError_t launch_count(const int32_t *topk, int64_t T, int32_t k, int32_t E,
                        int32_t n_groups, int32_t *counts, int32_t *status,
                        hipStream_t stream) {
  const int64_t V = T * k;
  if (V <= kSplitIds) {
    const size_t lds = sizeof(int32_t) * kCountWaves * E;
    hipLaunchKernelGGL(k_count, dim3(n_groups), dim3(kCountThreads), lds, stream,
                       topk, V, E, counts, status);
    return hipGetLastError();
  }
  const int64_t n = static_cast<int64_t>(n_groups) * E;
  hipLaunchKernelGGL(k_count_zero, dim3(static_cast<unsigned>((n + kSplitThreads - 1) / kSplitThreads)),
                     dim3(kSplitThreads), 0, stream, counts, n);
  const size_t lds = sizeof(int32_t) * kSplitWaves * E;
  if (V <= kSplitSmall) {
    constexpr int per = kSplitThreads * 8;
    const unsigned parts = static_cast<unsigned>((V + per - 1) / per);
    hipLaunchKernelGGL(k_count_split<per>, dim3(parts, n_groups), dim3(kSplitThreads), lds, stream,
                       topk, V, E, counts, status);
  } else {
    constexpr int per = kSplitThreads * 16;
    const unsigned parts = static_cast<unsigned>((V + per - 1) / per);
    hipLaunchKernelGGL(k_count_split<per>, dim3(parts, n_groups), dim3(kSplitThreads), lds, stream,
                       topk, V, E, counts, status);
  }
  return hipGetLastError();
}

}  // namespace uep
