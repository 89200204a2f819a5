// Internal launchers of the UltraEP balancing kernels (one per translation
// unit); the C ABI in abi.hip validates arguments and calls these.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/ultraep.h"

namespace uep {

hipError_t launch_count(const int32_t *topk, int64_t T, int32_t k, int32_t E,
                        int32_t n_groups, int32_t *counts, int32_t *status,
                        hipStream_t stream);

size_t plan_ws_bytes(int32_t R, int32_t E, int32_t NS);
hipError_t launch_plan_replicate(const int32_t *load, const ultraep_group &g,
                                 const ultraep_plan_buf &out, void *ws, hipStream_t stream);
hipError_t launch_plan_reroute(const int32_t *load, const ultraep_group &g,
                               const ultraep_plan_buf &out, hipStream_t stream);
// SolveReroute and the local weight packing in one launch
hipError_t launch_reroute_pack(const int32_t *load, const ultraep_group &g,
                               const ultraep_plan_buf &out, const uint16_t *w_main, int64_t W,
                               int32_t rank, uint16_t *staging, int64_t cap, int64_t *dest_off,
                               int32_t *status, hipStream_t stream);
// both halves, the reroute fused into the last kernel of the replication
hipError_t launch_plan(const int32_t *load, const ultraep_group &g,
                       const ultraep_plan_buf &out, void *ws, hipStream_t stream);

// dispatch workspace carve-up
struct DispatchWs {
  int32_t *hist;      // [n_chunks][E] per-chunk expert histograms
  int32_t *ent_cum;   // [ncol] cumulative quota at the end of each CSR entry
  int32_t *ent_base;  // [ncol] first send row of the entry minus its start ordinal
  int32_t *exp_tot;   // [E]   planned routed slots per expert for this rank
  int64_t n_chunks;
};
constexpr int kDispatchChunk = 2048;  // slots per layout workgroup
size_t dispatch_ws_bytes(int64_t V, int32_t E, int32_t ncol);
DispatchWs dispatch_ws(void *ws, int64_t V, int32_t E, int32_t ncol);

hipError_t launch_dispatch_layout(const int32_t *topk, int64_t V, int32_t rank,
                                  const ultraep_group &g,
                                  const ultraep_plan_buf &plan,
                                  int32_t *row_of_slot, int64_t *block_off,
                                  const DispatchWs &ws, int32_t *status,
                                  hipStream_t stream);

hipError_t launch_dispatch_scatter(const uint16_t *x, int64_t T, int32_t k,
                                   int32_t H, const int32_t *row_of_slot,
                                   const int64_t *n_routed, uint16_t *send,
                                   hipStream_t stream);

hipError_t launch_pack(const uint16_t *w_main, int64_t W, int32_t rank,
                       const ultraep_group &g, const ultraep_plan_buf &plan,
                       uint16_t *staging, int64_t cap, int64_t *dest_off,
                       int32_t *status, hipStream_t stream);

hipError_t launch_pack_relay(const uint16_t *w_main, const uint16_t *relay_src, int64_t W,
                             int32_t rank, const ultraep_group &g, const ultraep_plan_buf &plan,
                             const int32_t *slot_src, uint16_t *staging, int64_t cap,
                             int64_t *dest_off, int32_t *status, hipStream_t stream);

// relay trees of the hot experts (one workgroup)
hipError_t launch_relay(const ultraep_group &g, const ultraep_plan_buf &plan, int32_t threshold,
                        int32_t *slot_src, int32_t *send_vol, int64_t *stats, int32_t *status,
                        hipStream_t stream);

// combine gather (reverse reroute) and the local gradient reduction
hipError_t launch_combine(const uint16_t *y, int64_t n_rows, const float *gate,
                          const int32_t *row_of_slot, int64_t T, int32_t k, int32_t H,
                          uint16_t *out, int32_t *status, hipStream_t stream);
hipError_t launch_grad_reduce(float *main_grad, float *rgrad, int64_t W, int32_t rank,
                              const ultraep_group &g, const ultraep_plan_buf &plan, int64_t cap,
                              int32_t *status, hipStream_t stream);

}  // namespace uep
