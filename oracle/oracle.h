/*
 * UltraEP reference oracle — TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.
 *
 * A plain, slow, single-threaded C11 implementation of the per-microbatch,
 * per-layer balancing path of "UltraEP: Unleash MoE Training and Inference on
 * Rack-Scale Nodes with Near-Optimal Load Balancing" (arXiv 2606.04101).
 * Only the test-suite, the smoke check and the benchmark's CPU-baseline leg
 * may load it.  It shares no source, header, table or helper with the HIP
 * library; the buffer layouts below are restated here on purpose so that the
 * two sides can be compared byte for byte.
 *
 * Arithmetic: int64 everywhere; fp32 with a fixed order in the combine
 * gather and the gradient reduction only.
 *
 * Layouts (all row-major, caller-owned host memory):
 *   R ranks, E logical experts, n_main = E / R main experts per rank,
 *   home rank h(e) = e / n_main, n_slot redundant slots per rank,
 *   S = n_main + n_slot physical slots per rank, ncol = E + R * n_slot.
 *   slot_expert [R][n_slot]   X: expert in redundant slot s of rank t, -1 = empty
 *   quota       [E][R]        U: u_{e,t}
 *   host_ptr    [E+1]         CSR row pointers over H(e)
 *   host_rank   [ncol]        H(e) = home first, then replica ranks ascending; -1 pad
 *   host_pslot  [ncol]        physical slot on that rank (e - h(e)*n_main for the
 *                             home, n_main + s for redundant slot s); -1 pad
 *   reroute     [R][ncol]     q_{r,e,t} aligned with the CSR entries; 0 pad
 *   stats       [8]           tau*, tau_lo0, tau_hi0, n_probes, n_replicas,
 *                             max |H(e)|, status, total load L
 */
#ifndef ULTRAEP_ORACLE_H
#define ULTRAEP_ORACLE_H
#include <stdint.h>

#define ORC_OK 0
#define ORC_EINVAL (-1)
#define ORC_ENOSPC (-2)
#define ORC_EDATA (-4)
#define ORC_ELEMMA (-6) /* the no-duplicate test excluded a rank: see probe() */

typedef struct {
  int32_t R, E, n_slot;
  int64_t u_min;
  int32_t beta_num, beta_den;
} orc_group;

/* Histogram of routed slots: counts[g*E+e] over n_groups blocks of T*k ids. */
int orc_count(const int32_t *topk, int64_t T, int32_t k, int32_t E,
              int32_t n_groups, int32_t *counts);

/* One greedy feasibility probe of SolveReplication at threshold tau.
 * Writes the temporary quota table Ut[E][R] and slot map X[R][n_slot] when
 * the pointers are non-null; *feasible = 1 iff all excess drained. */
int orc_probe(const int32_t *load, const orc_group *g, int64_t tau,
              int32_t *feasible, int64_t *Ut, int32_t *X);

/* Full plan (SolveReplication then SolveReroute).  locality = 1 is the
 * paper's method; 0 skips the local-consumption pass (diagnostics only). */
int orc_plan(const int32_t *load, const orc_group *g, int32_t locality,
             int32_t *slot_expert, int32_t *quota, int32_t *host_ptr,
             int32_t *host_rank, int32_t *host_pslot, int32_t *reroute,
             int64_t *stats);

/* Sequence of bisection thresholds probed and their outcomes (for tests).
 * Returns the number of probes written (at most cap). */
int orc_bisect_trace(const int32_t *load, const orc_group *g, int64_t *taus,
                     int32_t *feasible, int32_t cap);

/* One largest-remainder step of the proportional split: apportions demand
 * over nh residual quotas ures (sum D > 0) into out[nh]. */
int orc_apportion(int64_t demand, const int64_t *ures, int32_t nh,
                  int64_t *out);

/* Dispatch for one source rank: per-slot destination rows, block offsets and
 * the bf16 row scatter (bit copy of H uint16 per row). */
int orc_dispatch(const uint16_t *x, const int32_t *topk, int64_t T, int32_t k,
                 int32_t H, int32_t rank, const orc_group *g,
                 const int32_t *slot_expert, const int32_t *host_ptr,
                 const int32_t *host_rank, const int32_t *host_pslot,
                 const int32_t *reroute, uint16_t *send, int32_t *row_of_slot,
                 int64_t *block_off);

/* Pack the main-expert blobs this rank must replicate into per-destination
 * staging.  Returns ORC_ENOSPC (and copies nothing) if n_out > cap. */
int orc_pack(const uint16_t *w_main, int64_t W, int32_t rank,
             const orc_group *g, const int32_t *slot_expert,
             uint16_t *staging, int64_t cap, int64_t *dest_off,
             int64_t *n_out);

/* Relay trees for experts with more than `threshold` replicas (Sec. 6.2):
 * slot_src[R][n_slot] = the rank sending each redundant slot's blob (-1:
 * empty slot), send_vol[R] = blobs each rank sends, relay_stats[4] = relay
 * experts, relays, max volume before, max volume after. */
int orc_relay(const orc_group *g, const int32_t *slot_expert,
              const int32_t *host_ptr, const int32_t *host_rank,
              const int32_t *host_pslot, int32_t threshold, int32_t *slot_src,
              int32_t *send_vol, int64_t *relay_stats);

/* Pack with relay trees: one copy per redundant slot whose sender is `rank`;
 * relayed blobs come from relay_src[n_slot][W] (this rank's own slots). */
int orc_pack_relay(const uint16_t *w_main, const uint16_t *relay_src, int64_t W,
                   int32_t rank, const orc_group *g, const int32_t *slot_expert,
                   const int32_t *slot_src, uint16_t *staging, int64_t cap,
                   int64_t *dest_off, int64_t *n_out);

/* Combine gather: out[t] = bf16(sum_k fp32(gate[t][k] * y[row_of_slot[t][k]]))
 * accumulated in fp32 in k order from +0 (no fused multiply-add); rows -1
 * skipped.  y [n_rows][H] bf16, gate [T][k] fp32, out [T][H] bf16. */
int orc_combine(const uint16_t *y, const float *gate, const int32_t *row_of_slot,
                int64_t T, int32_t k, int32_t H, int64_t n_rows, uint16_t *out);

/* Gradient reduction of this rank's replicated main experts: main_grad
 * [n_main][W] fp32 += the rgrad entries [n_out][W] fp32 of each expert, in
 * staging order (destination rank, then slot), sequentially in fp32; rgrad
 * entries are then zeroed. */
int orc_grad_reduce(float *main_grad, float *rgrad, int64_t W, int32_t rank,
                    const orc_group *g, const int32_t *slot_expert, int64_t cap,
                    int64_t *n_out);

/* Diagnostics of a plan: out[0..5] = max rank load before, mean load (x1),
 * max rank load after, n_replicas, max |H(e)|, remote (in-flight) tokens. */
int orc_metrics(const int32_t *load, const orc_group *g,
                const int32_t *quota, const int32_t *host_ptr,
                const int32_t *host_rank, const int32_t *reroute,
                int64_t *out);

#endif
