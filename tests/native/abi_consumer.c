/*
 * A plain C11 caller of libultraep's C ABI (test infrastructure): no torch,
 * no C++, device memory from hipMalloc, the null stream.  It runs the
 * balancing path of one rank -- ultraep_count over every rank's routing,
 * ultraep_plan, ultraep_dispatch and ultraep_pack_replicas -- on inputs read
 * from a file and writes every output to another file, which the GPU test
 * compares with the oracle.
 *
 * usage: abi_consumer IN OUT
 *   IN   int64 header {R, E, n_slot, T, k, H, W, rank, u_min, beta_num,
 *        beta_den}, then int32 topk [R][T][k], uint16 x [T][H],
 *        uint16 w_main [E/R][W]
 *   OUT  int32 status, int32 load [R][E], the seven plan buffers in
 *        ultraep_plan_buf order, uint16 send [T*k][H], int32 row_of_slot
 *        [T*k], int64 block_off [R*S+1], int64 dest_off [R+1], int64 n_out,
 *        uint16 staging [n_out][W]
 * Exit status 0 when every call returned ULTRAEP_OK, 1 on a bad input file,
 * 2 on a failed call (its name and code on stderr).
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "ultraep.h"

static int fail(const char *what, int code) {
  fprintf(stderr, "%s: %d\n", what, code);
  return 2;
}

#define CALL(expr)                                   \
  do {                                               \
    const int rc_ = (int)(expr);                     \
    if (rc_ != 0) return fail(#expr, rc_);           \
  } while (0)

static void *dev_alloc(size_t bytes, int *ok) {
  void *p = NULL;
  if (hipMalloc(&p, bytes ? bytes : 16) != hipSuccess) *ok = 0;
  return p;
}

static int read_all(FILE *f, void *dst, size_t bytes) {
  return fread(dst, 1, bytes, f) == bytes;
}

int main(int argc, char **argv) {
  if (argc != 3) return 1;
  FILE *in = fopen(argv[1], "rb");
  if (!in) return 1;
  int64_t h[11];
  if (!read_all(in, h, sizeof h)) return 1;
  ultraep_group g;
  g.R = (int32_t)h[0];
  g.E = (int32_t)h[1];
  g.n_slot = (int32_t)h[2];
  const int64_t T = h[3];
  const int32_t k = (int32_t)h[4], H = (int32_t)h[5];
  const int64_t W = h[6];
  const int32_t rank = (int32_t)h[7];
  g.u_min = h[8];
  g.beta_num = (int32_t)h[9];
  g.beta_den = (int32_t)h[10];
  if (g.R < 1 || g.E < g.R || g.n_slot < 0 || T < 1 || k < 1 || H < 8 || W < 8) return 1;
  const int64_t R = g.R, E = g.E, nm = E / R, V = T * k;
  const int64_t S = nm + g.n_slot, ncol = E + R * g.n_slot, cap = R * g.n_slot;

  size_t sizes[7];
  CALL(ultraep_plan_sizes(&g, sizes));
  const size_t bytes_topk = sizeof(int32_t) * R * V, bytes_x = 2 * (size_t)(T * H);
  const size_t bytes_w = 2 * (size_t)(nm * W);
  int32_t *topk = malloc(bytes_topk);
  uint16_t *x = malloc(bytes_x), *w = malloc(bytes_w);
  if (!topk || !x || !w) return 1;
  if (!read_all(in, topk, bytes_topk) || !read_all(in, x, bytes_x) || !read_all(in, w, bytes_w))
    return 1;
  fclose(in);

  int ok = 1;
  int32_t *d_topk = dev_alloc(bytes_topk, &ok), *d_load = dev_alloc(4 * R * E, &ok);
  int32_t *d_status = dev_alloc(4, &ok);
  uint16_t *d_x = dev_alloc(bytes_x, &ok), *d_w = dev_alloc(bytes_w, &ok);
  ultraep_plan_buf plan;
  plan.slot_expert = dev_alloc(4 * sizes[0], &ok);
  plan.quota = dev_alloc(4 * sizes[1], &ok);
  plan.host_ptr = dev_alloc(4 * sizes[2], &ok);
  plan.host_rank = dev_alloc(4 * sizes[3], &ok);
  plan.host_pslot = dev_alloc(4 * sizes[4], &ok);
  plan.reroute = dev_alloc(4 * sizes[5], &ok);
  plan.stats = dev_alloc(8 * sizes[6], &ok);
  const size_t plan_ws = ultraep_plan_ws_bytes(&g), disp_ws = ultraep_dispatch_ws_bytes(T, k, &g);
  void *d_pws = dev_alloc(plan_ws, &ok), *d_dws = dev_alloc(disp_ws, &ok);
  uint16_t *d_send = dev_alloc(2 * (size_t)(V * H), &ok);
  int32_t *d_ros = dev_alloc(4 * (size_t)V, &ok);
  int64_t *d_boff = dev_alloc(8 * (size_t)(R * S + 1), &ok), *d_doff = dev_alloc(8 * (R + 1), &ok);
  uint16_t *d_stg = dev_alloc(2 * (size_t)(cap * W), &ok);
  if (!ok || plan_ws == 0 || disp_ws == 0) return fail("allocation", 0);
  CALL(hipMemcpy(d_topk, topk, bytes_topk, hipMemcpyHostToDevice));
  CALL(hipMemcpy(d_x, x, bytes_x, hipMemcpyHostToDevice));
  CALL(hipMemcpy(d_w, w, bytes_w, hipMemcpyHostToDevice));
  CALL(hipMemset(d_status, 0, 4));

  CALL(ultraep_count(d_topk, T, k, g.E, g.R, d_load, d_status, 0));
  CALL(ultraep_plan(d_load, &g, &plan, d_pws, plan_ws, 0));
  CALL(ultraep_dispatch(d_x, d_topk + rank * V, T, k, H, rank, &g, &plan, d_send, d_ros, d_boff,
                        d_dws, disp_ws, d_status, 0));
  CALL(ultraep_pack_replicas(d_w, W, rank, &g, &plan, d_stg, cap, d_doff, d_status, 0));
  CALL(hipDeviceSynchronize());

  FILE *out = fopen(argv[2], "wb");
  if (!out) return 1;
  const struct {
    const void *p;
    size_t bytes;
  } parts[] = {{d_status, 4},
               {d_load, 4 * (size_t)(R * E)},
               {plan.slot_expert, 4 * sizes[0]},
               {plan.quota, 4 * sizes[1]},
               {plan.host_ptr, 4 * sizes[2]},
               {plan.host_rank, 4 * sizes[3]},
               {plan.host_pslot, 4 * sizes[4]},
               {plan.reroute, 4 * sizes[5]},
               {plan.stats, 8 * sizes[6]},
               {d_send, 2 * (size_t)(V * H)},
               {d_ros, 4 * (size_t)V},
               {d_boff, 8 * (size_t)(R * S + 1)},
               {d_doff, 8 * (size_t)(R + 1)}};
  int64_t n_out = 0;
  for (size_t i = 0; i < sizeof parts / sizeof parts[0]; ++i) {
    void *hbuf = malloc(parts[i].bytes ? parts[i].bytes : 1);
    if (!hbuf) return 1;
    CALL(hipMemcpy(hbuf, parts[i].p, parts[i].bytes, hipMemcpyDeviceToHost));
    fwrite(hbuf, 1, parts[i].bytes, out);
    if (parts[i].p == d_doff) n_out = ((const int64_t *)hbuf)[R];
    free(hbuf);
  }
  if (n_out < 0 || n_out > cap) return fail("dest_off", (int)n_out);
  fwrite(&n_out, sizeof n_out, 1, out);
  if (n_out > 0) {
    const size_t sb = 2 * (size_t)(n_out * W);
    void *hbuf = malloc(sb);
    if (!hbuf) return 1;
    CALL(hipMemcpy(hbuf, d_stg, sb, hipMemcpyDeviceToHost));
    fwrite(hbuf, 1, sb, out);
    free(hbuf);
  }
  fclose(out);
  (void)ncol;
  return 0;
}
