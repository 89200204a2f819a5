// C ABI of the UltraEP balancing library (see include/ultraep.h): argument
// validation on the host, then stream-ordered kernel launches.  No
// allocation, no host synchronisation, no memset.  The one piece of library
// state is the fixed planner workspace of ultraep_plan_noalloc.
#include <stdint.h>

#include <atomic>
#include <mutex>

#include "common.hpp"
#include "kernels.hpp"

// Planner workspace of ultraep_plan_noalloc: one copy per device, resident
// for the life of the process.  Host code never uses this name as an
// address: a device's copy is reached only through the pointer that
// hipGetSymbolAddress returns for it.
static __device__ __align__(256) uint8_t scratch[ULTRAEP_PLAN_STATIC_WS_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::atomic<void *> g_scratch_ptr[kMaxDevices];
std::mutex g_scratch_mu;

// Device address of the current device's copy of `scratch`, looked up once
// per device (nullptr on failure).
void *scratch_of_current_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  void *p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (p) return p;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
  if (!p) {
    void *q = nullptr;
    if (hipGetSymbolAddress(&q, HIP_SYMBOL(scratch)) != hipSuccess || !q) return nullptr;
    g_scratch_ptr[dev].store(q, std::memory_order_release);
    p = q;
  }
  return p;
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool group_ok(const ultraep_group *g) {
  if (!g) return false;
  if (g->R < 1 || g->R > 64 || g->E < 1 || g->E > 1024 || g->E % g->R != 0) return false;
  if (g->n_slot < 0 || static_cast<int64_t>(g->R) * g->n_slot > 256) return false;
  if (g->u_min < 1) return false;
  if (g->beta_den < 1 || g->beta_num < g->beta_den || g->beta_num > (1 << 20)) return false;
  return true;
}

int32_t ncol_of(const ultraep_group *g) { return g->E + g->R * g->n_slot; }

bool plan_ok(const ultraep_group *g, const ultraep_plan_buf *p) {
  if (!p) return false;
  if (g->n_slot > 0 && !p->slot_expert) return false;
  return p->quota && p->host_ptr && p->host_rank && p->host_pslot && p->reroute && p->stats;
}

bool routing_ok(int64_t T, int32_t k, int32_t E) {
  return T >= 0 && k >= 1 && k <= E && k <= 64 && T * static_cast<int64_t>(k) < (int64_t(1) << 31);
}

int rc(hipError_t e) { return e == hipSuccess ? ULTRAEP_OK : ULTRAEP_EDEVICE; }

}  // namespace

extern "C" {

int ultraep_plan_sizes(const ultraep_group *g, size_t counts_out[7]) {
  if (!group_ok(g) || !counts_out) return ULTRAEP_EINVAL;
  const size_t R = g->R, E = g->E, nc = ncol_of(g);
  counts_out[0] = R * g->n_slot;
  counts_out[1] = E * R;
  counts_out[2] = E + 1;
  counts_out[3] = nc;
  counts_out[4] = nc;
  counts_out[5] = R * nc;
  counts_out[6] = 8;
  return ULTRAEP_OK;
}

int ultraep_count(const int32_t *topk, int64_t T, int32_t k, int32_t E,
                  int32_t n_groups, int32_t *counts, int32_t *status,
                  hipStream_t stream) {
  if (E < 1 || E > 1024 || n_groups < 1 || n_groups > 65535 || !routing_ok(T, k, E) || !counts ||
      !status)
    return ULTRAEP_EINVAL;
  if (T > 0 && !topk) return ULTRAEP_EINVAL;
  return rc(uep::launch_count(topk, T, k, E, n_groups, counts, status, stream));
}

size_t ultraep_plan_ws_bytes(const ultraep_group *g) {
  if (!group_ok(g)) return 0;
  return uep::plan_ws_bytes(g->R, g->E, g->n_slot);
}

int ultraep_plan_replicate(const int32_t *load, const ultraep_group *g,
                           const ultraep_plan_buf *out, void *ws, size_t ws_bytes,
                           hipStream_t stream) {
  if (!load || !group_ok(g) || !plan_ok(g, out) || !ws) return ULTRAEP_EINVAL;
  if (ws_bytes < uep::plan_ws_bytes(g->R, g->E, g->n_slot)) return ULTRAEP_EINVAL;
  return rc(uep::launch_plan_replicate(load, *g, *out, ws, stream));
}

int ultraep_plan_reroute(const int32_t *load, const ultraep_group *g,
                         const ultraep_plan_buf *out, hipStream_t stream) {
  if (!load || !group_ok(g) || !plan_ok(g, out)) return ULTRAEP_EINVAL;
  return rc(uep::launch_plan_reroute(load, *g, *out, stream));
}

int ultraep_plan(const int32_t *load, const ultraep_group *g,
                 const ultraep_plan_buf *out, void *ws, size_t ws_bytes,
                 hipStream_t stream) {
  if (!load || !group_ok(g) || !plan_ok(g, out) || !ws) return ULTRAEP_EINVAL;
  if (ws_bytes < uep::plan_ws_bytes(g->R, g->E, g->n_slot)) return ULTRAEP_EINVAL;
  return rc(uep::launch_plan(load, *g, *out, ws, stream));
}

int ultraep_plan_noalloc(const int32_t *load, const ultraep_group *g,
                         const ultraep_plan_buf *out, hipStream_t stream) {
  if (!load || !group_ok(g) || !plan_ok(g, out)) return ULTRAEP_EINVAL;
  if (uep::plan_ws_bytes(g->R, g->E, g->n_slot) > ULTRAEP_PLAN_STATIC_WS_BYTES)
    return ULTRAEP_EINVAL;
  void *ws = scratch_of_current_device();
  if (!ws) return ULTRAEP_EDEVICE;
  return rc(uep::launch_plan(load, *g, *out, ws, stream));
}

size_t ultraep_dispatch_ws_bytes(int64_t T, int32_t k, const ultraep_group *g) {
  if (!group_ok(g) || !routing_ok(T, k, g->E)) return 0;
  return uep::dispatch_ws_bytes(T * k, g->E, ncol_of(g));
}

int ultraep_dispatch_layout(const int32_t *topk, int64_t T, int32_t k,
                            int32_t rank, const ultraep_group *g,
                            const ultraep_plan_buf *plan, int32_t *row_of_slot,
                            int64_t *block_off, void *ws, size_t ws_bytes,
                            int32_t *status, hipStream_t stream) {
  if (!group_ok(g) || !plan_ok(g, plan) || !routing_ok(T, k, g->E)) return ULTRAEP_EINVAL;
  if (rank < 0 || rank >= g->R || !block_off || !ws || !status) return ULTRAEP_EINVAL;
  if (T > 0 && (!topk || !row_of_slot)) return ULTRAEP_EINVAL;
  if (ws_bytes < uep::dispatch_ws_bytes(T * k, g->E, ncol_of(g))) return ULTRAEP_EINVAL;
  const uep::DispatchWs w = uep::dispatch_ws(ws, T * k, g->E, ncol_of(g));
  return rc(uep::launch_dispatch_layout(topk, T * k, rank, *g, *plan, row_of_slot,
                                        block_off, w, status, stream));
}

int ultraep_dispatch_scatter(const uint16_t *x, int64_t T, int32_t k,
                             int32_t H, const int32_t *row_of_slot,
                             const int64_t *n_routed, uint16_t *send,
                             hipStream_t stream) {
  if (T < 0 || k < 1 || k > 64 || H < 8 || H % 8 != 0 || !n_routed) return ULTRAEP_EINVAL;
  if (T * static_cast<int64_t>(k) >= (int64_t(1) << 31)) return ULTRAEP_EINVAL;
  if (T == 0) return ULTRAEP_OK;
  if (!x || !row_of_slot || !send || !aligned16(x) || !aligned16(send)) return ULTRAEP_EINVAL;
  return rc(uep::launch_dispatch_scatter(x, T, k, H, row_of_slot, n_routed, send, stream));
}

int ultraep_dispatch(const uint16_t *x, const int32_t *topk, int64_t T,
                     int32_t k, int32_t H, int32_t rank,
                     const ultraep_group *g, const ultraep_plan_buf *plan,
                     uint16_t *send, int32_t *row_of_slot, int64_t *block_off,
                     void *ws, size_t ws_bytes, int32_t *status,
                     hipStream_t stream) {
  if (!group_ok(g) || H < 8 || H % 8 != 0) return ULTRAEP_EINVAL;
  if (T > 0 && (!x || !send || !aligned16(x) || !aligned16(send))) return ULTRAEP_EINVAL;
  int r = ultraep_dispatch_layout(topk, T, k, rank, g, plan, row_of_slot, block_off, ws,
                                  ws_bytes, status, stream);
  if (r != ULTRAEP_OK) return r;
  const int64_t nblk = static_cast<int64_t>(g->R) * (g->E / g->R + g->n_slot);
  return ultraep_dispatch_scatter(x, T, k, H, row_of_slot, block_off + nblk, send, stream);
}

int ultraep_pack_replicas(const uint16_t *w_main, int64_t W, int32_t rank,
                          const ultraep_group *g, const ultraep_plan_buf *plan,
                          uint16_t *staging, int64_t cap, int64_t *dest_off,
                          int32_t *status, hipStream_t stream) {
  if (!group_ok(g) || !plan_ok(g, plan) || rank < 0 || rank >= g->R) return ULTRAEP_EINVAL;
  if (W < 8 || W % 8 != 0 || cap < 0 || !dest_off || !status || !w_main) return ULTRAEP_EINVAL;
  if (!aligned16(w_main) || (cap > 0 && (!staging || !aligned16(staging)))) return ULTRAEP_EINVAL;
  return rc(uep::launch_pack(w_main, W, rank, *g, *plan, staging, cap, dest_off, status, stream));
}

int ultraep_reroute_and_pack(const int32_t *load, const ultraep_group *g,
                             const ultraep_plan_buf *plan, const uint16_t *w_main, int64_t W,
                             int32_t rank, uint16_t *staging, int64_t cap, int64_t *dest_off,
                             int32_t *status, hipStream_t stream) {
  if (!load || !group_ok(g) || !plan_ok(g, plan) || rank < 0 || rank >= g->R) return ULTRAEP_EINVAL;
  if (W < 8 || W % 8 != 0 || cap < 0 || !dest_off || !status || !w_main) return ULTRAEP_EINVAL;
  if (!aligned16(w_main) || (cap > 0 && (!staging || !aligned16(staging)))) return ULTRAEP_EINVAL;
  return rc(uep::launch_reroute_pack(load, *g, *plan, w_main, W, rank, staging, cap, dest_off,
                                     status, stream));
}

int ultraep_relay_plan(const ultraep_group *g, const ultraep_plan_buf *plan, int32_t threshold,
                       int32_t *slot_src, int32_t *send_vol, int64_t *relay_stats,
                       int32_t *status, hipStream_t stream) {
  if (!group_ok(g) || !plan_ok(g, plan) || threshold < 0) return ULTRAEP_EINVAL;
  if (!send_vol || !relay_stats || !status || (g->n_slot > 0 && !slot_src)) return ULTRAEP_EINVAL;
  return rc(uep::launch_relay(*g, *plan, threshold, slot_src, send_vol, relay_stats, status,
                              stream));
}

int ultraep_pack_relay(const uint16_t *w_main, const uint16_t *relay_src, int64_t W, int32_t rank,
                       const ultraep_group *g, const ultraep_plan_buf *plan,
                       const int32_t *slot_src, uint16_t *staging, int64_t cap,
                       int64_t *dest_off, int32_t *status, hipStream_t stream) {
  if (!group_ok(g) || !plan_ok(g, plan) || rank < 0 || rank >= g->R) return ULTRAEP_EINVAL;
  if (W < 8 || W % 8 != 0 || cap < 0 || !dest_off || !status || !w_main) return ULTRAEP_EINVAL;
  if (g->n_slot > 0 && (!slot_src || !relay_src || !aligned16(relay_src))) return ULTRAEP_EINVAL;
  if (!aligned16(w_main) || (cap > 0 && (!staging || !aligned16(staging)))) return ULTRAEP_EINVAL;
  return rc(uep::launch_pack_relay(w_main, relay_src, W, rank, *g, *plan, slot_src, staging, cap,
                                   dest_off, status, stream));
}

int ultraep_combine(const uint16_t *y, int64_t n_rows, const float *gate,
                    const int32_t *row_of_slot, int64_t T, int32_t k, int32_t H, uint16_t *out,
                    int32_t *status, hipStream_t stream) {
  if (T < 0 || k < 1 || k > 64 || H < 8 || H % 8 != 0 || n_rows < 0 || !status)
    return ULTRAEP_EINVAL;
  if (T * static_cast<int64_t>(k) >= (int64_t(1) << 31) || n_rows >= (int64_t(1) << 31))
    return ULTRAEP_EINVAL;
  if (T == 0) return ULTRAEP_OK;
  if (!gate || !row_of_slot || !out || !aligned16(out)) return ULTRAEP_EINVAL;
  if (n_rows > 0 && (!y || !aligned16(y))) return ULTRAEP_EINVAL;
  return rc(uep::launch_combine(y, n_rows, gate, row_of_slot, T, k, H, out, status, stream));
}

int ultraep_grad_reduce(float *main_grad, float *rgrad, int64_t W, int32_t rank,
                        const ultraep_group *g, const ultraep_plan_buf *plan, int64_t cap,
                        int32_t *status, hipStream_t stream) {
  if (!group_ok(g) || !plan_ok(g, plan) || rank < 0 || rank >= g->R) return ULTRAEP_EINVAL;
  if (W < 4 || W % 4 != 0 || cap < 0 || !status || !main_grad || !aligned16(main_grad))
    return ULTRAEP_EINVAL;
  if (cap > 0 && (!rgrad || !aligned16(rgrad))) return ULTRAEP_EINVAL;
  return rc(uep::launch_grad_reduce(main_grad, rgrad, W, rank, *g, *plan, cap, status, stream));
}

const char *ultraep_strerror(int code) {
  switch (code) {
    case ULTRAEP_OK: return "ok";
    case ULTRAEP_EINVAL: return "invalid argument";
    case ULTRAEP_ENOSPC: return "staging capacity too small";
    case ULTRAEP_EDEVICE: return "kernel launch failed";
    case ULTRAEP_EDATA: return "inconsistent device data";
    default: return "unknown status";
  }
}

}  // extern "C"
