// Step 1 — exact per-expert loads lambda_{r,e} from top-k routing ids
// (Table 1; gathered after gating in the forward pipeline of Sec. 4.2).
//
// One workgroup of 1024 threads per block of T*k ids.  Each wave keeps a
// private LDS histogram; a wave aggregates equal ids with a ballot match
// (log2(E) ballots), so one leader lane adds the whole group with a single
// LDS update and hot experts never serialise on one bank.  The wave
// histograms are summed at the end and every count is written (no global
// atomics, hence no zero-fill and no memset).
#include "common.hpp"
#include "kernels.hpp"

namespace uep {

constexpr int kCountThreads = 1024;
constexpr int kCountWaves = kCountThreads / kWave;

__global__ void __launch_bounds__(kCountThreads)
k_count(const int32_t *__restrict__ topk, int64_t V, int32_t E, int nbits,
        int32_t *__restrict__ counts, int32_t *status) {
  extern __shared__ int32_t hist[];  // [kCountWaves][E]
  const int wave = threadIdx.x / kWave;
  for (int i = threadIdx.x; i < kCountWaves * E; i += kCountThreads) hist[i] = 0;
  __syncthreads();

  const int32_t *src = topk + static_cast<int64_t>(blockIdx.x) * V;
  int32_t *wh = hist + wave * E;
  bool bad = false;
  for (int64_t base = 0; base < V; base += kCountThreads) {
    const int64_t i = base + threadIdx.x;
    const int32_t e = i < V ? __builtin_nontemporal_load(src + i) : -1;
    const bool valid = e >= 0 && e < E;
    bad |= (i < V) && (e < -1 || e >= E);
    const uint64_t act = ballot(valid);
    if (act == 0) continue;  // wave-uniform
    const uint64_t m = match_any(static_cast<uint32_t>(valid ? e : 0), nbits, act);
    if (valid && popc_below(m) == 0) wh[e] += __popcll(m);
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
                     topk, T * k, E, bits_for(E), counts, status);
  return hipGetLastError();
}

}  // namespace uep
