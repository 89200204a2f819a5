// Step 4 — local half of the forward weight distribution (Sec. 6.1) as a
// kernel of its own, without and with relay trees (Sec. 6.2); the work
// itself is in pack_core.hpp.
#include "pack_core.hpp"

namespace uep {

__global__ void __launch_bounds__(kPkThreads) k_pack(PkArgs a) {
  pack_block(a, blockIdx.x, gridDim.x, blockIdx.x == 0);
}

// With relay trees: the slots whose sender is this rank (Sec. 6.2).
__global__ void __launch_bounds__(kPkThreads) k_pack_relay(PkArgs a) {
  pack_block<true>(a, blockIdx.x, gridDim.x, blockIdx.x == 0);
}

hipError_t launch_pack_relay(const uint16_t *w_main, const uint16_t *relay_src, int64_t W,
                             int32_t rank, const ultraep_group &g, const ultraep_plan_buf &plan,
                             const int32_t *slot_src, uint16_t *staging, int64_t cap,
                             int64_t *dest_off, int32_t *status, hipStream_t stream) {
  PkArgs a = pack_args(w_main, W, rank, g, plan, staging, cap, dest_off, status);
  a.relay_src = reinterpret_cast<const v4u *>(relay_src);
  a.slot_src = slot_src;
  hipLaunchKernelGGL(k_pack_relay, dim3(kPkGrid), dim3(kPkThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_pack(const uint16_t *w_main, int64_t W, int32_t rank,
                       const ultraep_group &g, const ultraep_plan_buf &plan,
                       uint16_t *staging, int64_t cap, int64_t *dest_off,
                       int32_t *status, hipStream_t stream) {
  const PkArgs a = pack_args(w_main, W, rank, g, plan, staging, cap, dest_off, status);
  hipLaunchKernelGGL(k_pack, dim3(kPkGrid), dim3(kPkThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace uep
