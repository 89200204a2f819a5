// Wave-level helpers for gfx950 (CDNA4, wave64) shared by the kernels of the
// UltraEP balancing library.  Internal header.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/ultraep.h"

namespace uep {

constexpr int kWave = 64;

// 16-byte vector moved by one lane (global_load/store_dwordx4)
typedef uint32_t v4u __attribute__((ext_vector_type(4)));
typedef int32_t v4i __attribute__((ext_vector_type(4)));

__device__ __forceinline__ int lane_id() {
  return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0));
}

// number of set bits of m strictly below this lane
__device__ __forceinline__ int popc_below(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(m >> 32),
                                   __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(m), 0));
}

__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }

__device__ __forceinline__ int readlane(int v, int l) {
  return __builtin_amdgcn_readlane(v, l);
}

// Row (16-lane) reductions with DPP mirrors, then the four row results are
// combined through scalar registers.  Every lane must be active.
__device__ __forceinline__ int row_max(int v) {
  v = max(v, __builtin_amdgcn_update_dpp(v, v, 0xB1, 0xF, 0xF, false));   // quad_perm 1,0,3,2
  v = max(v, __builtin_amdgcn_update_dpp(v, v, 0x4E, 0xF, 0xF, false));   // quad_perm 2,3,0,1
  v = max(v, __builtin_amdgcn_update_dpp(v, v, 0x141, 0xF, 0xF, false));  // row_half_mirror
  v = max(v, __builtin_amdgcn_update_dpp(v, v, 0x140, 0xF, 0xF, false));  // row_mirror
  return v;
}

// Results are wave-uniform; readfirstlane makes that visible to the compiler
// so the branches that depend on them stay scalar.
__device__ __forceinline__ int wave_max(int v) {
  v = row_max(v);
  int a = readlane(v, 0), b = readlane(v, 16), c = readlane(v, 32), d = readlane(v, 48);
  return __builtin_amdgcn_readfirstlane(max(max(a, b), max(c, d)));
}

__device__ __forceinline__ int row_sum(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x140, 0xF, 0xF, false);
  return v;
}

__device__ __forceinline__ int wave_sum(int v) {
  v = row_sum(v);
  return __builtin_amdgcn_readfirstlane(readlane(v, 0) + readlane(v, 16) +
                                        readlane(v, 32) + readlane(v, 48));
}

// Inclusive prefix sum over the 64 lanes: a Hillis-Steele scan inside each
// row of 16 lanes with DPP row shifts (a lane without a source adds 0),
// then each row adds the totals of the rows before it.  Every lane must be
// active.
__device__ __forceinline__ int wave_scan_incl(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, false);  // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, false);  // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, false);  // row_shr:4
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, false);  // row_shr:8
  const int t0 = readlane(v, 15), t1 = readlane(v, 31), t2 = readlane(v, 47);
  const int lane = lane_id();
  return v + (lane >= 16 ? t0 : 0) + (lane >= 32 ? t1 : 0) + (lane >= 48 ? t2 : 0);
}

__device__ __forceinline__ int64_t wave_sum64(int64_t v) {
  int lo = static_cast<int>(static_cast<uint32_t>(v));
  int hi = static_cast<int>(v >> 32);
  // sum the low halves as unsigned with carries tracked in the high halves:
  // split each 32-bit half into 16-bit pieces so no piece overflows
  int l0 = lo & 0xFFFF, l1 = (lo >> 16) & 0xFFFF;
  int64_t s0 = wave_sum(l0), s1 = wave_sum(l1), sh = wave_sum(hi);
  return s0 + (s1 << 16) + (sh << 32);
}

// Lanes of the wave holding the same key (bits [0, nbits) of key), among the
// lanes set in `active`.  Every lane must execute this.
__device__ __forceinline__ uint64_t match_any(uint32_t key, int nbits, uint64_t active) {
  uint64_t m = active;
  for (int b = 0; b < nbits; ++b) {
    bool bit = (key >> b) & 1u;
    uint64_t bb = ballot(bit);
    m &= bit ? bb : ~bb;
  }
  return m;
}

__device__ __forceinline__ void report(int32_t *status, int code) {
  if (status) atomicCAS(status, 0, code);
}

// bits needed to hold values 0 .. n-1
__host__ __device__ __forceinline__ int bits_for(int n) {
  int b = 0;
  while ((1 << b) < n) ++b;
  return b;
}

}  // namespace uep
