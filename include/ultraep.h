/*
 * ultraep.h — C ABI of the MI355X (gfx950) library for UltraEP's
 * per-microbatch, per-layer balancing path (arXiv 2606.04101):
 *
 *   1. ultraep_count          exact per-expert loads from top-k routing ids
 *   2. ultraep_plan           quota-driven replication (SolveReplication) and
 *                             reroute split (SolveReroute), Algorithm 1
 *   3. ultraep_dispatch       token-to-replica assignment and bf16 row scatter
 *                             into per-destination, per-replica blocks
 *   4. ultraep_pack_replicas  local half of weight distribution: the blobs of
 *                             this rank's replicated main experts copied into
 *                             per-destination staging
 *      ultraep_relay_plan     relay trees for hot-expert fan-out, and
 *      ultraep_pack_relay     the packing that follows them
 *   5. ultraep_combine        reverse reroute: gate-weighted gather of the
 *                             experts' output rows back to token order
 *   6. ultraep_grad_reduce    local half of the gradient reduction: replica
 *                             gradients accumulated into main gradients
 *
 * Conventions for every call:
 *   - Buffer pointers are DEVICE pointers unless marked "host".  The caller
 *     owns and allocates every buffer; the library never allocates, never
 *     frees, never synchronises the host, keeps no state between calls and
 *     issues no memset, so every call can be captured into a HIP graph.
 *     (ultraep_plan_noalloc takes its workspace from a fixed array in the
 *     library's device memory instead of a caller buffer; see there.)
 *   - Work is enqueued on `stream` in order; results are ready when the
 *     stream reaches that point.  Calls on different streams must use
 *     distinct output and workspace buffers.
 *   - Return value: ULTRAEP_OK, or ULTRAEP_EINVAL for an argument problem
 *     that the host can see (nothing is launched), or ULTRAEP_EDEVICE when a
 *     launch fails.
 *   - Problems visible only in device data are reported through a device
 *     status word: the first failing kernel stores its (negative) code into
 *     *status if it still holds 0.  The caller zeroes the word before a
 *     sequence of calls and reads it after its own synchronisation.  When
 *     the status is nonzero the outputs of the failing call are undefined.
 *   - Layouts are row-major.  With n_main = E / R main experts per rank,
 *     home rank h(e) = e / n_main (main experts in contiguous blocks),
 *     S = n_main + n_slot physical slots per rank (slot p < n_main is main
 *     expert r*n_main + p, slot n_main + s is redundant slot s) and
 *     ncol = E + R * n_slot CSR entries at most.
 *   - bf16 data are moved as raw 16-bit patterns (never converted).
 *
 * Supported sizes (else ULTRAEP_EINVAL): 1 <= R <= 64, E % R == 0,
 * E <= 1024, 0 <= n_slot, R * n_slot <= 256, u_min >= 1,
 * 1 <= beta_den <= beta_num <= 2^20, 1 <= k <= min(E, 64), T >= 0,
 * T * k < 2^31, H % 8 == 0, W % 8 == 0, 16-byte aligned x / send / w_main /
 * staging.  The total load of a plan must not exceed 2^30 tokens (device
 * status ULTRAEP_EDATA otherwise).
 */
#ifndef ULTRAEP_H
#define ULTRAEP_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  ULTRAEP_OK = 0,
  ULTRAEP_EINVAL = -1,  /* bad argument (host-visible); nothing launched */
  ULTRAEP_ENOSPC = -2,  /* device: staging capacity too small */
  ULTRAEP_EDEVICE = -3, /* a kernel launch failed */
  ULTRAEP_EDATA = -4    /* device: ids out of range, negative or oversized
                           loads, or a load row that disagrees with topk */
};

/* EP group metadata and the planner's constants (host struct).
 * Table 1 of the paper: R ranks, E logical experts, N_slot redundant slots per
 * rank, quota floor u_min (1024 in the paper) and balancing target
 * beta = beta_num / beta_den (1.01 in the paper, i.e. 101/100). */
typedef struct {
  int32_t R;
  int32_t E;
  int32_t n_slot;
  int64_t u_min;
  int32_t beta_num;
  int32_t beta_den;
} ultraep_group;

/* Plan outputs (device buffers; element counts from ultraep_plan_sizes).
 *   slot_expert [R * n_slot]   X (Table 1): x_{t,s} = expert hosted by
 *                              redundant slot s of rank t, -1 when empty;
 *                              slots fill in the order replicas are accepted.
 *   quota       [E * R]        U (Table 1): u_{e,t} at e * R + t.
 *   host_ptr    [E + 1]        CSR row pointers over the hosts H(e).
 *   host_rank   [ncol]         H(e) in order: home first, then replica ranks
 *                              ascending; -1 padding after host_ptr[E].
 *   host_pslot  [ncol]         physical slot of that instance on its rank;
 *                              -1 padding.
 *   reroute     [R * ncol]     Q (Table 1): q_{r,e,t} at r * ncol + j where j
 *                              is the CSR entry of (e, t); 0 padding.
 *   stats       [8] int64      tau*, tau_lo0, tau_hi0, number of bisection
 *                              probes, number of replicas, max |H(e)|,
 *                              status (0 or ULTRAEP_EDATA), total load L. */
typedef struct {
  int32_t *slot_expert;
  int32_t *quota;
  int32_t *host_ptr;
  int32_t *host_rank;
  int32_t *host_pslot;
  int32_t *reroute;
  int64_t *stats;
} ultraep_plan_buf;

/* Host only.  Element counts of the seven plan buffers, in struct order, for
 * group *g (host pointer).  Returns ULTRAEP_EINVAL for an unsupported group. */
int ultraep_plan_sizes(const ultraep_group *g, size_t counts_out[7]);

/* Step 1 — exact load acquisition (Sec. 4.2 forward pipeline; lambda_{r,e} of
 * Table 1): counts[b * E + e] = number of (token, k) slots of block b routed
 * to expert e, for n_groups blocks of T * k ids stored back to back in topk
 * ([n_groups][T][k] int32).  Id -1 means "not routed" and is skipped; ids
 * outside [-1, E) are skipped and raise ULTRAEP_EDATA in *status.  One count
 * per routed slot (no per-token deduplication).  counts is fully written.
 * 1 <= n_groups <= 65535, 1 <= k <= min(E, 64), E <= 1024, T * k < 2^31. */
int ultraep_count(const int32_t *topk, int64_t T, int32_t k, int32_t E,
                  int32_t n_groups, int32_t *counts, int32_t *status,
                  hipStream_t stream);

/* Step 2 — Algorithm 1 on the load matrix (device, [R][E] int32, row r =
 * lambda_{r,.}).  SolveReplication binary-searches the integer threshold tau
 * from tau_lo = ceil(beta * ceil(L / R)) to tau_hi = max_r ell_r with
 * tau = floor((lo + hi) / 2), running the greedy probe of Sec. 5.1 at each
 * step (overloaded ranks by descending excess, their main experts by
 * descending load, transfers of min(excess, slack, remaining load) to the
 * admissible rank of largest slack, a transfer below u_min ends the expert;
 * all ties go to the lower id).  The last feasible probe gives X and U; with
 * no feasible probe every expert stays on its home.  SolveReroute (Sec. 5.2)
 * lets each host's own tokens consume its quota first, then splits every
 * source's residual demand over the residual quotas in proportion, sources
 * in ascending rank order, by largest remainder against the quotas still
 * unconsumed (ties to the earlier host), which keeps both margins of Q
 * exact.  Every output buffer is fully written (padding included).  Data
 * errors (negative loads, L > 2^30) set stats[6] = ULTRAEP_EDATA.
 *   ws  device workspace of ws_bytes >= ultraep_plan_ws_bytes(g); its
 *       contents on entry do not matter. */
int ultraep_plan(const int32_t *load, const ultraep_group *g,
                 const ultraep_plan_buf *out, void *ws, size_t ws_bytes,
                 hipStream_t stream);

/* ultraep_plan for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same kernels and outputs as ultraep_plan, with the planner workspace
 * taken from a fixed array in the library's device memory instead of a
 * caller buffer.  The array holds ULTRAEP_PLAN_STATIC_WS_BYTES (4.25 MiB),
 * enough for every supported group (R <= 64, E <= 1024, R * n_slot <= 256);
 * a group that would need more is rejected with ULTRAEP_EINVAL before any
 * launch.  Each device the library runs on holds its own copy from the
 * first call on that device (made with that device current) until the
 * process ends.  The call allocates nothing and launches the planner's
 * kernels only; the first kernel clears the part of the array that must
 * start at zero.  Every call on one device shares that device's array:
 * calls that overlap in time on one device (on different streams without
 * an ordering between them, or from several host threads) race on it, so
 * the caller serialises them.  ULTRAEP_EDEVICE if the array's device
 * address cannot be obtained or a launch fails. */
#define ULTRAEP_PLAN_STATIC_WS_BYTES ((size_t)17 << 18)
int ultraep_plan_noalloc(const int32_t *load, const ultraep_group *g,
                         const ultraep_plan_buf *out, hipStream_t stream);

/* The two halves of ultraep_plan, in this order on one stream (or with the
 * second made to wait for the first): SolveReplication writes slot_expert,
 * quota, host_ptr, host_rank, host_pslot and stats; SolveReroute then writes
 * reroute from the load matrix and those buffers.  They are separate so a
 * caller can run the reroute alongside the weight distribution
 * (ultraep_pack_replicas needs only slot_expert), as in the forward pipeline
 * of Sec. 4.2 and Eq. (1). */
int ultraep_plan_replicate(const int32_t *load, const ultraep_group *g,
                           const ultraep_plan_buf *out, void *ws, size_t ws_bytes,
                           hipStream_t stream);
int ultraep_plan_reroute(const int32_t *load, const ultraep_group *g,
                         const ultraep_plan_buf *out, hipStream_t stream);

/* Bytes of device workspace ultraep_plan needs for group *g (host only; 0
 * for an unsupported group): per-expert orders and the outcome and transfer
 * record of every speculatively evaluated bisection probe. */
size_t ultraep_plan_ws_bytes(const ultraep_group *g);

/* Bytes of device workspace ultraep_dispatch / ultraep_dispatch_layout need
 * (host only; 0 for unsupported arguments). */
size_t ultraep_dispatch_ws_bytes(int64_t T, int32_t k, const ultraep_group *g);

/* Step 3 — token assignment and dispatch permutation of source rank `rank`
 * (Sec. 5.2 Token Assignment).  The j-th local slot routed to expert e
 * (counted over the (token, k) slots in token-major order) goes to the first
 * instance of H(e) whose cumulative quota q_{rank,e,.} exceeds j.  The send
 * buffer holds one block per (destination rank t, physical slot p) in
 * (t, p) order, block (t, p) holding q_{rank, e(t,p), t} rows in ascending
 * token order.
 *   x            [T][H] bf16 token rows of this rank
 *   topk         [T][k] int32 expert ids (-1 = not routed)
 *   plan         outputs of ultraep_plan (device buffers)
 *   send         [T*k][H] bf16: routed rows at their positions, rows from
 *                block_off[R*S] to T*k - 1 zero-filled
 *   row_of_slot  [T*k] int32 row of send for each slot, -1 if not routed
 *   block_off    [R*S + 1] int64 first row of each block, last = routed rows
 *   ws           device workspace of ws_bytes >= ultraep_dispatch_ws_bytes
 * A plan row that does not describe exactly the routed ids of topk raises
 * ULTRAEP_EDATA. */
int ultraep_dispatch(const uint16_t *x, const int32_t *topk, int64_t T,
                     int32_t k, int32_t H, int32_t rank,
                     const ultraep_group *g, const ultraep_plan_buf *plan,
                     uint16_t *send, int32_t *row_of_slot, int64_t *block_off,
                     void *ws, size_t ws_bytes, int32_t *status,
                     hipStream_t stream);

/* The two halves of ultraep_dispatch, for callers that move the rows
 * themselves or time them apart: the layout (row_of_slot, block_off) and the
 * scatter (send rows; n_routed = block_off + R * S, the routed row count,
 * read on the device: rows n_routed .. T*k - 1 are zero-filled, none when
 * the count lies outside [0, T*k]). */
int ultraep_dispatch_layout(const int32_t *topk, int64_t T, int32_t k,
                            int32_t rank, const ultraep_group *g,
                            const ultraep_plan_buf *plan, int32_t *row_of_slot,
                            int64_t *block_off, void *ws, size_t ws_bytes,
                            int32_t *status, hipStream_t stream);
int ultraep_dispatch_scatter(const uint16_t *x, int64_t T, int32_t k,
                             int32_t H, const int32_t *row_of_slot,
                             const int64_t *n_routed, uint16_t *send,
                             hipStream_t stream);

/* Step 4 — local half of the forward weight distribution (Sec. 6.1; the
 * remote peer stores are not part of this library).  Every redundant slot
 * (t, s) whose expert e has home `rank` receives a bit copy of
 * w_main[e - rank * n_main]; entries are ordered by destination rank t, then
 * slot s.
 *   w_main    [n_main][W] bf16 blobs of this rank's main experts (W elements
 *             each; an expert's gate, up and down matrices as stored)
 *   staging   [cap][W] bf16; entries 0 .. n_out-1 written, the rest untouched
 *   dest_off  [R + 1] int64 first entry of each destination rank, last = n_out
 * If n_out > cap, ULTRAEP_ENOSPC is raised, dest_off is still written and no
 * entry is copied. */
int ultraep_pack_replicas(const uint16_t *w_main, int64_t W, int32_t rank,
                          const ultraep_group *g, const ultraep_plan_buf *plan,
                          uint16_t *staging, int64_t cap, int64_t *dest_off,
                          int32_t *status, hipStream_t stream);

/* SolveReroute of ultraep_plan_reroute and the packing of
 * ultraep_pack_replicas in one launch, overlapped as the forward pipeline of
 * Sec. 4.2 overlaps the reroute with the weight distribution (Eq. (1)): the
 * same results as the two calls.  Needs the buffers ultraep_plan_replicate
 * wrote; arguments and errors as for the two calls. */
int ultraep_reroute_and_pack(const int32_t *load, const ultraep_group *g,
                             const ultraep_plan_buf *plan, const uint16_t *w_main, int64_t W,
                             int32_t rank, uint16_t *staging, int64_t cap, int64_t *dest_off,
                             int32_t *status, hipStream_t stream);

/* Relay trees for hot-expert fan-out (Sec. 6.2, load-aware relay
 * scheduling), from a plan (slot_expert and the host lists).  Each rank's
 * sending volume starts at one expert blob per replica of its main experts.
 * Every expert with more than `threshold` replicas (the paper uses 4), by
 * replica count descending then id ascending, gets the integer nearest
 * sqrt(replicas) first-stage relays: its replica ranks of smallest volume;
 * each other replica, by ascending rank, is served by the relay whose
 * volume is smallest (one blob added at once); the source's volume then
 * drops to one blob per relay.  Ties go to the smaller rank.
 *   threshold    >= 0
 *   slot_src     [R * n_slot] int32: the rank that sends redundant slot
 *                (t, s) its blob (the expert's home rank or a relay), -1 for
 *                an empty slot
 *   send_vol     [R] int32: blobs each rank sends under the trees
 *   relay_stats  [4] int64: experts with relays, relays in total, largest
 *                sending volume before and after
 * A plan whose host lists do not match its slot map, or whose stats[6] is
 * nonzero, raises ULTRAEP_EDATA (outputs undefined).  Every output element
 * is written otherwise. */
int ultraep_relay_plan(const ultraep_group *g, const ultraep_plan_buf *plan, int32_t threshold,
                       int32_t *slot_src, int32_t *send_vol, int64_t *relay_stats,
                       int32_t *status, hipStream_t stream);

/* Local half of the weight distribution with relay trees (Sec. 6.1 tile
 * copy, Sec. 6.2 trees): every redundant slot (t, s) whose sender
 * slot_src[t * n_slot + s] is `rank` receives a bit copy of its expert's
 * blob, entries ordered by destination rank t, then slot s.  The blob of a
 * main expert of `rank` comes from w_main; the blob of an expert that
 * `rank` relays comes from relay_src[s'], this rank's own redundant slot s'
 * holding that expert (the buffer the first stage fills).
 *   relay_src  [n_slot][W] bf16 (needed when n_slot > 0)
 *   staging, dest_off, cap as for ultraep_pack_replicas.
 * A slot this rank should relay without hosting its expert raises
 * ULTRAEP_EDATA; n_out > cap raises ULTRAEP_ENOSPC. */
int ultraep_pack_relay(const uint16_t *w_main, const uint16_t *relay_src, int64_t W, int32_t rank,
                       const ultraep_group *g, const ultraep_plan_buf *plan,
                       const int32_t *slot_src, uint16_t *staging, int64_t cap,
                       int64_t *dest_off, int32_t *status, hipStream_t stream);

/* Reverse reroute: the combine gather (Sec. 4.2, the scatter-to-gather
 * inversion of the token assignment).  Token t's output row is the sum of
 * its routed slots' rows weighted by their gates:
 *   out[t] = bf16( sum_{kk ascending, row_of_slot[t*k+kk] >= 0}
 *                  gate[t*k+kk] * y[row_of_slot[t*k+kk]] )
 * in fp32: every product and every partial sum rounded to fp32 (no fused
 * multiply-add), from +0; the result rounded to bf16 to nearest-even, every
 * NaN to 0x7FC0.  The paper fixes bf16 activations only; this order and
 * precision are the library's reading.
 *   y            [n_rows][H] bf16: rows in the dispatch layout (the experts'
 *                outputs for the rows ultraep_dispatch sent)
 *   gate         [T][k] fp32 top-k gate weights
 *   row_of_slot  [T*k] int32 from ultraep_dispatch (-1 = not routed)
 *   out          [T][H] bf16, fully written
 * A row outside [-1, n_rows) raises ULTRAEP_EDATA (that slot is skipped).
 * 1 <= k <= 64, H % 8 == 0, 16-byte aligned y and out. */
int ultraep_combine(const uint16_t *y, int64_t n_rows, const float *gate,
                    const int32_t *row_of_slot, int64_t T, int32_t k, int32_t H, uint16_t *out,
                    int32_t *status, hipStream_t stream);

/* Gradient reduction, local half (Sec. 4.2 backward pass, tile streaming of
 * Sec. 6.1): every replica of a main expert of `rank` returns an fp32
 * gradient blob, laid out like the forward staging (one [W] entry per
 * redundant slot (t, s) whose expert has home `rank`, destination rank
 * ascending, then slot).  Each main gradient is updated in place to
 *   main_grad[l] = (...(main_grad[l] + r_0) + r_1 ...) + r_{f-1}
 * element by element in fp32, its replicas' entries taken in that staging
 * order, and every replica entry is then zeroed for reuse by the next layer.
 *   main_grad  [n_main][W] fp32, read and written
 *   rgrad      [cap][W] fp32, entries 0 .. n_out-1 read and zeroed
 * n_out > cap raises ULTRAEP_ENOSPC and changes nothing.  W % 4 == 0,
 * 16-byte aligned buffers. */
int ultraep_grad_reduce(float *main_grad, float *rgrad, int64_t W, int32_t rank,
                        const ultraep_group *g, const ultraep_plan_buf *plan, int64_t cap,
                        int32_t *status, hipStream_t stream);

/* Host only.  Static description of a status code. */
const char *ultraep_strerror(int code);

#ifdef __cplusplus
}
#endif

#endif /* ULTRAEP_H */
