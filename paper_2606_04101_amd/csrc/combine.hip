// Reverse reroute: the combine gather.  After the experts have run, each
// source rank gets its rows back in the dispatch layout; token t's output
// is the gate-weighted sum of the rows its k slots were sent to (the
// scatter-to-gather inversion of the forward token assignment, Sec. 4.2).
//
// Arithmetic (the paper fixes bf16 activations only; this library and its
// tests read it so): every product gate * row and every partial sum is an
// fp32 value (no fused multiply-add), the sum runs over k ascending from
// +0, masked slots (row -1) add nothing, and the fp32 result is rounded to
// bf16 to nearest-even, every NaN to 0x7FC0.
//
// Bandwidth bound: each routed row is read once, each output row written
// once.  A wave takes a work unit of two 16-byte chunks (8 bf16 each) per
// lane of one token's row, issues the k rows' loads of both chunks together
// (16 loads in flight for k = 8), accumulates and stores.  Many short waves
// keep the most row reads in flight: on the DeepSeek-V3-shaped layer this
// measured 90 us against 99-121 us for persistent waves that walk whole
// rows, and against 92-105 us for units of 1, 3 or 4 chunks per lane.
#include "common.hpp"
#include "kernels.hpp"

#pragma clang fp contract(off)

namespace uep {

constexpr int kCbThreads = 256;
constexpr int kCbWaves = kCbThreads / kWave;
constexpr int kCbGrid = 65535;
constexpr int kCbMaxK = 8;  // rows loaded together per chunk
constexpr int kCbChunks = 2;       // 16-byte chunks per lane per step
constexpr int kCbLaneChunks = 2;   // 16-byte chunks per lane per work unit

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// fp32 -> bf16, round to nearest-even by adding 0x7FFF plus the kept
// part's lowest bit before dropping 16 bits; NaN -> 0x7FC0
__device__ __forceinline__ uint32_t to_bf16(float f) {
  const uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0u;
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ void acc_chunk(float (&acc)[8], float g, v4u v) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    acc[2 * i] = __fadd_rn(acc[2 * i], __fmul_rn(g, bf16_lo(w[i])));
    acc[2 * i + 1] = __fadd_rn(acc[2 * i + 1], __fmul_rn(g, bf16_hi(w[i])));
  }
}

__device__ __forceinline__ v4u pack_chunk(const float (&acc)[8]) {
  v4u o;
  o.x = to_bf16(acc[0]) | (to_bf16(acc[1]) << 16);
  o.y = to_bf16(acc[2]) | (to_bf16(acc[3]) << 16);
  o.z = to_bf16(acc[4]) | (to_bf16(acc[5]) << 16);
  o.w = to_bf16(acc[6]) | (to_bf16(acc[7]) << 16);
  return o;
}

// rows of token t for this lane (lane < k); -1 = masked; out-of-range rows
// are reported and treated as masked
__device__ __forceinline__ void token_rows(const int32_t *row_of_slot, const float *gate,
                                           int64_t t, int k, int lane, int64_t n_rows,
                                           int32_t *status, int &row, float &g) {
  row = -1;
  g = 0.f;
  if (lane < k) {
    row = row_of_slot[t * k + lane];
    g = gate[t * k + lane];
    if (row < -1 || row >= n_rows) {
      report(status, ULTRAEP_EDATA);
      row = -1;
    }
  }
}

// k <= kCbMaxK.  Work unit: kCbLaneChunks 16-byte chunks per lane of one
// token's row; the k rows' loads of kCbChunks chunks are in flight together.
__global__ void __launch_bounds__(kCbThreads)
k_combine(const v4u *__restrict__ y, int64_t n_rows, const float *__restrict__ gate,
          const int32_t *__restrict__ row_of_slot, int64_t T, int32_t k, int32_t nch,
          v4u *__restrict__ out, int32_t *status) {
  const int lane = lane_id();
  const int nblk = (nch + kCbLaneChunks * kWave - 1) / (kCbLaneChunks * kWave);
  const int64_t n_units = T * nblk;
  const int64_t nw = static_cast<int64_t>(gridDim.x) * kCbWaves;
  for (int64_t unit = static_cast<int64_t>(blockIdx.x) * kCbWaves + threadIdx.x / kWave;
       unit < n_units; unit += nw) {
    const int64_t t = unit / nblk;
    const int b = static_cast<int>(unit - t * nblk);
    int row;
    float g;
    token_rows(row_of_slot, gate, t, k, lane, n_rows, status, row, g);
    const int c_end = min(nch, (b + 1) * kCbLaneChunks * kWave);
    for (int c0 = b * kCbLaneChunks * kWave + lane; c0 < c_end; c0 += kCbChunks * kWave) {
      v4u v[kCbChunks][kCbMaxK];
#pragma unroll
      for (int kk = 0; kk < kCbMaxK; ++kk) {
        const int r = kk < k ? readlane(row, kk) : -1;
#pragma unroll
        for (int u = 0; u < kCbChunks; ++u) {
          const int cc = c0 + u * kWave;
          if (r >= 0 && cc < c_end)
            v[u][kk] = __builtin_nontemporal_load(y + static_cast<int64_t>(r) * nch + cc);
        }
      }
#pragma unroll
      for (int u = 0; u < kCbChunks; ++u) {
        const int cc = c0 + u * kWave;
        float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < kCbMaxK; ++kk) {
          const int r = kk < k ? readlane(row, kk) : -1;
          if (r >= 0 && cc < c_end)
            acc_chunk(acc, __int_as_float(readlane(__float_as_int(g), kk)), v[u][kk]);
        }
        if (cc < c_end) __builtin_nontemporal_store(pack_chunk(acc), out + t * nch + cc);
      }
    }
  }
}

// any k: one row at a time
__global__ void __launch_bounds__(kCbThreads)
k_combine_wide(const v4u *__restrict__ y, int64_t n_rows, const float *__restrict__ gate,
               const int32_t *__restrict__ row_of_slot, int64_t T, int32_t k, int32_t nch,
               v4u *__restrict__ out, int32_t *status) {
  const int lane = lane_id();
  const int64_t nw = static_cast<int64_t>(gridDim.x) * kCbWaves;
  for (int64_t t = static_cast<int64_t>(blockIdx.x) * kCbWaves + threadIdx.x / kWave; t < T;
       t += nw) {
    int row;
    float g;
    token_rows(row_of_slot, gate, t, k, lane, n_rows, status, row, g);
    for (int cc = lane; cc < nch; cc += kWave) {
      float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      for (int kk = 0; kk < k; ++kk) {
        const int r = readlane(row, kk);
        if (r >= 0)
          acc_chunk(acc, __int_as_float(readlane(__float_as_int(g), kk)),
                    y[static_cast<int64_t>(r) * nch + cc]);
      }
      out[t * nch + cc] = pack_chunk(acc);
    }
  }
}

hipError_t launch_combine(const uint16_t *y, int64_t n_rows, const float *gate,
                          const int32_t *row_of_slot, int64_t T, int32_t k, int32_t H,
                          uint16_t *out, int32_t *status, hipStream_t stream) {
  const int32_t nch = H / 8;
  const int64_t units = T * ((nch + kCbLaneChunks * kWave - 1) / (kCbLaneChunks * kWave));
  const int64_t need = (units + kCbWaves - 1) / kCbWaves;
  const dim3 grid(static_cast<unsigned>(need < kCbGrid ? need : kCbGrid));
  const v4u *ys = reinterpret_cast<const v4u *>(y);
  v4u *os = reinterpret_cast<v4u *>(out);
  if (k <= kCbMaxK)
    hipLaunchKernelGGL(k_combine, grid, dim3(kCbThreads), 0, stream, ys, n_rows, gate,
                       row_of_slot, T, k, nch, os, status);
  else
    hipLaunchKernelGGL(k_combine_wide, grid, dim3(kCbThreads), 0, stream, ys, n_rows, gate,
                       row_of_slot, T, k, nch, os, status);
  return hipGetLastError();
}

}  // namespace uep
