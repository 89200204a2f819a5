// Step 1 — exact per-expert loads lambda_{r,e} from top-k routing ids
// (Table 1; gathered after gating in the forward pipeline of Sec. 4.2).
//
// One workgroup of 1024 threads per block of T*k ids.  Every thread issues
// all of its 16-byte loads of a batch before using any (one memory latency
// per batch instead of one per id), then adds each id into its wave's
// private LDS histogram with an LDS atomic: a histogram needs no order, so
// the per-wave privatisation bounds contention to the 64 lanes of one wave
// (at most k lanes per token share a hot expert).  The 16 wave histograms
// are summed at the end and every count is written (no global atomics, no
// zero-fill, no memset).
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

hipError_t launch_count(const int32_t *topk, int64_t T, int32_t k, int32_t E,
                        int32_t n_groups, int32_t *counts, int32_t *status,
                        hipStream_t stream) {
  const size_t lds = sizeof(int32_t) * kCountWaves * E;
  hipLaunchKernelGGL(k_count, dim3(n_groups), dim3(kCountThreads), lds, stream,
                     topk, T * k, E, counts, status);
  return hipGetLastError();
}

}  // namespace uep
