/*
 * UltraEP reference oracle — TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.
 *
 * Plain, slow, single-threaded C11 restatement of the balancing path of
 * UltraEP (arXiv 2606.04101).  Each function cites the passage it follows:
 *   - Table 1 (notation: Lambda, U, X, Q, h, H(e), E_r, u_min, beta)
 *   - Sec. 5.1 "Threshold Formulation" / Eq. (6) and "Quota Construction"
 *   - Algorithm 1 (SolveReplication, SolveReroute)
 *   - Sec. 5.2 "Quota Decomposition with Locality" and "Token Assignment"
 *   - Sec. 4.1 (main / redundant slot layout) and Sec. 6.1 (weight tiles)
 *   - Eqs. (3)-(5) and Table 3 (diagnostic metrics)
 * Where the paper is silent the reading used is stated inline; the same
 * readings bind the HIP library.  Floating point appears only in the
 * combine gather and the gradient reduction, in fp32 with a fixed order.  Only the test-suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this code.
 */
#include "oracle.h"

#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------ */
/* helpers                                                            */
/* ------------------------------------------------------------------ */

static int64_t max64(int64_t a, int64_t b) { return a > b ? a : b; }
static int64_t min64(int64_t a, int64_t b) { return a < b ? a : b; }

static int group_ok(const orc_group *g) {
  if (!g) return 0;
  if (g->R < 1 || g->E < 1 || g->n_slot < 0) return 0;
  if (g->E % g->R != 0) return 0;
  if (g->u_min < 1) return 0;
  if (g->beta_den < 1 || g->beta_num < g->beta_den) return 0; /* beta >= 1 */
  return 1;
}

/* home rank h(e): main experts sit in contiguous blocks of n_main per rank
 * (reading: the layout figure of Sec. 4.1 is not in the text). */
static int32_t home(const orc_group *g, int32_t e) { return e / (g->E / g->R); }

/* ------------------------------------------------------------------ */
/* Step 1 — exact load acquisition: lambda_{r,e} (Table 1)            */
/* One count per routed (token, k) slot; id -1 is "not routed".      */
/* ------------------------------------------------------------------ */

int orc_count(const int32_t *topk, int64_t T, int32_t k, int32_t E,
              int32_t n_groups, int32_t *counts) {
  if ((!topk && T * k > 0) || !counts || T < 0 || k < 1 || E < 1 || k > E ||
      n_groups < 1)
    return ORC_EINVAL;
  int status = ORC_OK;
  for (int32_t gi = 0; gi < n_groups; gi++) {
    int32_t *c = counts + (int64_t)gi * E;
    for (int32_t e = 0; e < E; e++) c[e] = 0;
    const int32_t *tk = topk + (int64_t)gi * T * k;
    for (int64_t i = 0; i < T * k; i++) {
      int32_t e = tk[i];
      if (e == -1) continue;
      if (e < -1 || e >= E) { status = ORC_EDATA; continue; }
      c[e] += 1;
    }
  }
  return status;
}

/* ------------------------------------------------------------------ */
/* Step 2a — SolveReplication (Sec. 5.1, Eq. (6), Algorithm 1)        */
/* ------------------------------------------------------------------ */

typedef struct {
  const orc_group *g;
  int32_t n_main;
  int64_t *lam_e; /* lambda_e = sum_r lambda_{r,e} */
  int64_t *ell;   /* ell_r = sum_{e in E_r} lambda_e */
  int64_t L;      /* total load */
} ctx_t;

static int ctx_init(ctx_t *c, const int32_t *load, const orc_group *g) {
  c->g = g;
  c->n_main = g->E / g->R;
  c->lam_e = calloc((size_t)g->E, sizeof(int64_t));
  c->ell = calloc((size_t)g->R, sizeof(int64_t));
  if (!c->lam_e || !c->ell) return ORC_EINVAL;
  c->L = 0;
  int bad = 0;
  for (int32_t r = 0; r < g->R; r++)
    for (int32_t e = 0; e < g->E; e++) {
      int32_t v = load[(int64_t)r * g->E + e];
      if (v < 0) bad = 1;
      c->lam_e[e] += v;
    }
  for (int32_t e = 0; e < g->E; e++) {
    c->ell[home(g, e)] += c->lam_e[e];
    c->L += c->lam_e[e];
  }
  /* Loads must stay far from int32 range on the device side as well. */
  if (bad || c->L > ((int64_t)1 << 30)) return ORC_EDATA;
  return ORC_OK;
}

static void ctx_free(ctx_t *c) {
  free(c->lam_e);
  free(c->ell);
}

/* sort keys for the two visiting orders of the probe */
typedef struct {
  int64_t key;
  int32_t id;
} kv_t;

/* descending key, ascending id on ties */
static int cmp_desc(const void *a, const void *b) {
  const kv_t *x = a, *y = b;
  if (x->key != y->key) return x->key > y->key ? -1 : 1;
  return x->id < y->id ? -1 : (x->id > y->id);
}

/* One greedy feasibility probe (the inner body of SolveReplication).
 *   exc_r = max(ell_r - tau, 0), slk_r = max(tau - ell_r, 0)      (Eq. 6)
 *   visit overloaded ranks by descending excess (ties: lower rank), and
 *   within a rank its main experts by descending lambda_e (ties: lower id);
 *   cap_e starts at lambda_e and shrinks with each accepted transfer;
 *   repeatedly move delta = min(exc_r, slk_t*, cap_e) to the admissible rank
 *   t* of largest slack (ties: lower rank); stop the expert when no rank is
 *   admissible or delta < u_min.  Feasible iff all excess drained.
 * The no-duplicate rule is tested literally (t must not already host e, the
 * home counting as a host).  Within one probe it can never be the deciding
 * test (the home is overloaded, so has no slack; and after a transfer either
 * the rank's excess, the expert's cap or the target's slack is exhausted);
 * if it ever were, *lemma is cleared so the tests can flag it. */
static int probe(const ctx_t *c, int64_t tau, int64_t *Ut, int32_t *X,
                 int *lemma) {
  const orc_group *g = c->g;
  const int32_t R = g->R, E = g->E, NS = g->n_slot, nm = c->n_main;
  int64_t *exc = calloc((size_t)R, sizeof(int64_t));
  int64_t *slk = calloc((size_t)R, sizeof(int64_t));
  int32_t *used = calloc((size_t)R, sizeof(int32_t));
  int32_t *slots = malloc(sizeof(int32_t) * (size_t)(R * (NS > 0 ? NS : 1)));
  kv_t *order = malloc(sizeof(kv_t) * (size_t)(R > nm ? R : nm));
  kv_t *eorder = malloc(sizeof(kv_t) * (size_t)nm);

  for (int32_t r = 0; r < R; r++) {
    exc[r] = max64(c->ell[r] - tau, 0);
    slk[r] = max64(tau - c->ell[r], 0);
  }
  for (int64_t i = 0; i < (int64_t)R * NS; i++) slots[i] = -1;
  if (Ut) {
    memset(Ut, 0, sizeof(int64_t) * (size_t)E * R);
    for (int32_t e = 0; e < E; e++) Ut[(int64_t)e * R + home(g, e)] = c->lam_e[e];
  }

  /* overloaded ranks in descending excess (static: only the rank being
   * processed ever loses excess and overloaded ranks never gain load) */
  int32_t n_over = 0;
  for (int32_t r = 0; r < R; r++)
    if (exc[r] > 0) { order[n_over].key = exc[r]; order[n_over].id = r; n_over++; }
  qsort(order, (size_t)n_over, sizeof(kv_t), cmp_desc);

  for (int32_t oi = 0; oi < n_over; oi++) {
    int32_t r = order[oi].id;
    for (int32_t j = 0; j < nm; j++) {
      eorder[j].id = r * nm + j;
      eorder[j].key = c->lam_e[r * nm + j];
    }
    qsort(eorder, (size_t)nm, sizeof(kv_t), cmp_desc);
    for (int32_t j = 0; j < nm; j++) {
      int32_t e = eorder[j].id;
      int64_t cap = c->lam_e[e]; /* remaining transferable load of e */
      while (exc[r] > 0 && cap > 0) {
        int32_t best = -1;
        for (int32_t t = 0; t < R; t++) {
          int slack_ok = slk[t] > 0;
          int slot_ok = used[t] < NS;
          int dup = (t == home(g, e));
          for (int32_t s = 0; s < used[t]; s++)
            if (slots[(int64_t)t * NS + s] == e) dup = 1;
          if (slack_ok && slot_ok && dup) *lemma = 0;
          if (!(slack_ok && slot_ok && !dup)) continue;
          if (best < 0 || slk[t] > slk[best]) best = t;
        }
        if (best < 0) break;
        int64_t delta = min64(min64(exc[r], slk[best]), cap);
        if (delta < g->u_min) break;
        if (Ut) {
          Ut[(int64_t)e * R + home(g, e)] -= delta;
          Ut[(int64_t)e * R + best] += delta;
        }
        slots[(int64_t)best * NS + used[best]] = e;
        used[best] += 1;
        exc[r] -= delta;
        slk[best] -= delta;
        cap -= delta;
      }
    }
  }
  int64_t rest = 0;
  for (int32_t r = 0; r < R; r++) rest += exc[r];
  if (X) memcpy(X, slots, sizeof(int32_t) * (size_t)R * NS);
  free(exc); free(slk); free(used); free(slots); free(order); free(eorder);
  return rest == 0;
}

/* tau_lo = beta * ceil(L / R), tau_hi = max_r ell_r (Algorithm 1).
 * Reading: tau is an integer load bound, so tau_lo is rounded up with beta
 * taken as the exact rational beta_num / beta_den. */
static void bounds(const ctx_t *c, int64_t *lo, int64_t *hi) {
  const orc_group *g = c->g;
  int64_t m = (c->L + g->R - 1) / g->R;
  *lo = (g->beta_num * m + g->beta_den - 1) / g->beta_den;
  int64_t mx = 0;
  for (int32_t r = 0; r < g->R; r++) mx = max64(mx, c->ell[r]);
  *hi = mx;
}

int orc_probe(const int32_t *load, const orc_group *g, int64_t tau,
              int32_t *feasible, int64_t *Ut, int32_t *X) {
  if (!load || !group_ok(g) || !feasible || tau < 0) return ORC_EINVAL;
  ctx_t c;
  int st = ctx_init(&c, load, g);
  if (st != ORC_OK) { ctx_free(&c); return st; }
  int lemma = 1;
  *feasible = probe(&c, tau, Ut, X, &lemma);
  ctx_free(&c);
  return lemma ? ORC_OK : ORC_ELEMMA;
}

/* Binary search of Algorithm 1: lo/hi move exactly as printed, with
 * tau = floor((lo + hi) / 2).  Feasibility is not monotone in tau (the
 * u_min floor), so the sequence of probes is part of the definition. */
typedef struct {
  int64_t tau_star, tau_lo0, tau_hi0;
  int32_t n_probes;
  int32_t have; /* a probe succeeded: U, X come from the last one */
} bis_t;

static int bisect(const ctx_t *c, int64_t *U, int32_t *X, bis_t *b,
                  int64_t *taus, int32_t *feas, int32_t cap) {
  const orc_group *g = c->g;
  int64_t lo, hi;
  bounds(c, &lo, &hi);
  b->tau_lo0 = lo;
  b->tau_hi0 = hi;
  b->n_probes = 0;
  b->have = 0;
  int lemma = 1;
  int64_t *Ut = U ? malloc(sizeof(int64_t) * (size_t)g->E * g->R) : NULL;
  int32_t *Xt = X ? malloc(sizeof(int32_t) * (size_t)(g->R * (g->n_slot > 0 ? g->n_slot : 1))) : NULL;
  while (lo < hi) {
    int64_t tau = (lo + hi) / 2;
    int ok = probe(c, tau, Ut, Xt, &lemma);
    if (taus && b->n_probes < cap) { taus[b->n_probes] = tau; feas[b->n_probes] = ok; }
    b->n_probes++;
    if (ok) {
      hi = tau;
      b->have = 1;
      if (U) memcpy(U, Ut, sizeof(int64_t) * (size_t)g->E * g->R);
      if (X) memcpy(X, Xt, sizeof(int32_t) * (size_t)g->R * g->n_slot);
    } else {
      lo = tau + 1;
    }
  }
  b->tau_star = hi;
  free(Ut);
  free(Xt);
  return lemma ? ORC_OK : ORC_ELEMMA;
}

int orc_bisect_trace(const int32_t *load, const orc_group *g, int64_t *taus,
                     int32_t *feasible, int32_t cap) {
  if (!load || !group_ok(g) || !taus || !feasible) return ORC_EINVAL;
  ctx_t c;
  int st = ctx_init(&c, load, g);
  if (st != ORC_OK) { ctx_free(&c); return st; }
  bis_t b;
  bisect(&c, NULL, NULL, &b, taus, feasible, cap);
  ctx_free(&c);
  return b.n_probes;
}

/* ------------------------------------------------------------------ */
/* Step 2b — SolveReroute (Sec. 5.2, Algorithm 1)                     */
/* ------------------------------------------------------------------ */

/* Largest-remainder (Hamilton) apportionment of `demand` over residual
 * quotas ures[] with D = sum(ures) >= demand.  Reading of the "deterministic
 * rounding" that must keep both margins: floor(demand * u_i / D) to every
 * host, then the leftover units one each to the hosts with the largest
 * remainders, ties to the earlier host of H(e). */
int orc_apportion(int64_t demand, const int64_t *ures, int32_t nh,
                  int64_t *out) {
  if (!ures || !out || nh < 1 || demand < 0) return ORC_EINVAL;
  int64_t D = 0;
  for (int32_t i = 0; i < nh; i++) {
    if (ures[i] < 0) return ORC_EINVAL;
    D += ures[i];
  }
  if (demand > D) return ORC_EINVAL;
  if (demand == 0) {
    for (int32_t i = 0; i < nh; i++) out[i] = 0;
    return ORC_OK;
  }
  int64_t *rem = malloc(sizeof(int64_t) * (size_t)nh);
  char *taken = calloc((size_t)nh, 1);
  int64_t given = 0;
  for (int32_t i = 0; i < nh; i++) {
    int64_t p = demand * ures[i];
    out[i] = p / D;
    rem[i] = p % D;
    given += out[i];
  }
  for (int64_t left = demand - given; left > 0; left--) {
    int32_t best = -1;
    for (int32_t i = 0; i < nh; i++)
      if (!taken[i] && (best < 0 || rem[i] > rem[best])) best = i;
    taken[best] = 1;
    out[best] += 1;
  }
  free(rem);
  free(taken);
  return ORC_OK;
}

/* ------------------------------------------------------------------ */
/* The plan: SolveReplication, then SolveReroute, then the layouts.   */
/* ------------------------------------------------------------------ */

int orc_plan(const int32_t *load, const orc_group *g, int32_t locality,
             int32_t *slot_expert, int32_t *quota, int32_t *host_ptr,
             int32_t *host_rank, int32_t *host_pslot, int32_t *reroute,
             int64_t *stats) {
  if (!load || !group_ok(g) || !slot_expert || !quota || !host_ptr ||
      !host_rank || !host_pslot || !reroute || !stats)
    return ORC_EINVAL;
  const int32_t R = g->R, E = g->E, NS = g->n_slot;
  const int32_t nm = E / R;
  const int64_t ncol = (int64_t)E + (int64_t)R * NS;
  ctx_t c;
  for (int i = 0; i < 8; i++) stats[i] = 0;
  int st = ctx_init(&c, load, g);
  if (st != ORC_OK) {
    ctx_free(&c);
    stats[6] = st;
    return st;
  }

  /* SolveReplication */
  int64_t *U = malloc(sizeof(int64_t) * (size_t)E * R);
  int32_t *X = malloc(sizeof(int32_t) * (size_t)(R * (NS > 0 ? NS : 1)));
  bis_t b;
  int lemma_st = bisect(&c, U, X, &b, NULL, NULL, 0);
  if (!b.have) {
    /* No probe succeeded (or the loop never ran because the loads are
     * already within tau_lo): keep every expert on its main instance. */
    memset(U, 0, sizeof(int64_t) * (size_t)E * R);
    for (int32_t e = 0; e < E; e++) U[(int64_t)e * R + home(g, e)] = c.lam_e[e];
    for (int64_t i = 0; i < (int64_t)R * NS; i++) X[i] = -1;
  }

  /* H(e): the home first, then replica ranks in ascending rank order. */
  int32_t *nh = calloc((size_t)E, sizeof(int32_t));
  for (int32_t e = 0; e < E; e++) nh[e] = 1;
  for (int64_t i = 0; i < (int64_t)R * NS; i++)
    if (X[i] >= 0) nh[X[i]] += 1;
  host_ptr[0] = 0;
  for (int32_t e = 0; e < E; e++) host_ptr[e + 1] = host_ptr[e] + nh[e];
  for (int64_t j = 0; j < ncol; j++) { host_rank[j] = -1; host_pslot[j] = -1; }
  for (int32_t e = 0; e < E; e++) {
    int32_t j = host_ptr[e];
    host_rank[j] = home(g, e);
    host_pslot[j] = e - home(g, e) * nm;
    j++;
    for (int32_t t = 0; t < R; t++)
      for (int32_t s = 0; s < NS; s++)
        if (X[(int64_t)t * NS + s] == e) {
          host_rank[j] = t;
          host_pslot[j] = nm + s;
          j++;
        }
  }

  /* SolveReroute: for each expert, local sources first consume their own
   * host's quota, then the residual demand of each source (ascending rank)
   * is apportioned over the residual quotas that are still unconsumed. */
  memset(reroute, 0, sizeof(int32_t) * (size_t)(R * ncol));
  int64_t *lamhat = malloc(sizeof(int64_t) * (size_t)R);
  int64_t *uhat = malloc(sizeof(int64_t) * (size_t)(R + 1));
  int64_t *qv = malloc(sizeof(int64_t) * (size_t)(R + 1));
  for (int32_t e = 0; e < E; e++) {
    int32_t j0 = host_ptr[e], n = nh[e];
    for (int32_t r = 0; r < R; r++) lamhat[r] = load[(int64_t)r * E + e];
    for (int32_t i = 0; i < n; i++) {
      int32_t t = host_rank[j0 + i];
      int64_t u = U[(int64_t)e * R + t];
      int64_t q = locality ? min64(lamhat[t], u) : 0; /* consume local quota */
      reroute[(int64_t)t * ncol + j0 + i] += (int32_t)q;
      lamhat[t] -= q; /* residual demand */
      uhat[i] = u - q; /* residual quota */
    }
    for (int32_t r = 0; r < R; r++) {
      if (lamhat[r] == 0) continue;
      orc_apportion(lamhat[r], uhat, n, qv);
      for (int32_t i = 0; i < n; i++) {
        reroute[(int64_t)r * ncol + j0 + i] += (int32_t)qv[i];
        uhat[i] -= qv[i];
      }
    }
  }

  /* quotas and slot map */
  for (int64_t i = 0; i < (int64_t)E * R; i++) quota[i] = (int32_t)U[i];
  memcpy(slot_expert, X, sizeof(int32_t) * (size_t)R * NS);

  int32_t n_rep = 0, max_h = 0;
  for (int32_t e = 0; e < E; e++) {
    n_rep += nh[e] - 1;
    if (nh[e] > max_h) max_h = nh[e];
  }
  stats[0] = b.tau_star;
  stats[1] = b.tau_lo0;
  stats[2] = b.tau_hi0;
  stats[3] = b.n_probes;
  stats[4] = n_rep;
  stats[5] = max_h;
  stats[6] = ORC_OK;
  stats[7] = c.L;

  free(U); free(X); free(nh); free(lamhat); free(uhat); free(qv);
  ctx_free(&c);
  return lemma_st;
}

/* ------------------------------------------------------------------ */
/* Step 3 — token assignment and dispatch layout (Sec. 5.2)           */
/* ------------------------------------------------------------------ */

/* The j-th local token of (rank, e) (j counted in flat token-major order of
 * the (token, k) slots) goes to the first instance of H(e) whose cumulative
 * quota q_{rank,e,.} exceeds j.  The send buffer holds one block per
 * (destination rank t, physical slot p), blocks in (t, p) order, tokens
 * ascending inside a block; block sizes are q_{rank, e(t,p), t}. */
int orc_dispatch(const uint16_t *x, const int32_t *topk, int64_t T, int32_t k,
                 int32_t H, int32_t rank, const orc_group *g,
                 const int32_t *slot_expert, const int32_t *host_ptr,
                 const int32_t *host_rank, const int32_t *host_pslot,
                 const int32_t *reroute, uint16_t *send, int32_t *row_of_slot,
                 int64_t *block_off) {
  if (!group_ok(g) || T < 0 || k < 1 || k > g->E || H < 1 || rank < 0 ||
      rank >= g->R || !slot_expert || !host_ptr || !host_rank || !host_pslot ||
      !reroute || !block_off)
    return ORC_EINVAL;
  if (T * k > 0 && (!x || !topk || !send || !row_of_slot)) return ORC_EINVAL;
  (void)slot_expert;
  const int32_t R = g->R, E = g->E, NS = g->n_slot, nm = E / R, S = nm + NS;
  const int64_t ncol = (int64_t)E + (int64_t)R * NS, V = T * k;
  const int32_t *q = reroute + (int64_t)rank * ncol;

  /* block sizes and their exclusive prefix */
  int64_t *cnt = calloc((size_t)R * S, sizeof(int64_t));
  for (int32_t e = 0; e < E; e++)
    for (int32_t j = host_ptr[e]; j < host_ptr[e + 1]; j++)
      cnt[(int64_t)host_rank[j] * S + host_pslot[j]] = q[j];
  block_off[0] = 0;
  for (int64_t b = 0; b < (int64_t)R * S; b++) block_off[b + 1] = block_off[b] + cnt[b];
  int64_t v_valid = block_off[(int64_t)R * S];

  /* ordinal of every slot within its expert, and the per-expert totals */
  int64_t *seen = calloc((size_t)E, sizeof(int64_t));
  int status = ORC_OK;
  for (int64_t i = 0; i < V; i++) {
    int32_t e = topk[i];
    if (e == -1) { row_of_slot[i] = -1; continue; }
    if (e < -1 || e >= E) { row_of_slot[i] = -1; status = ORC_EDATA; continue; }
    int64_t j = seen[e]++;
    int64_t C = 0;
    int64_t row = -1;
    for (int32_t jj = host_ptr[e]; jj < host_ptr[e + 1]; jj++) {
      int64_t qi = q[jj];
      if (j < C + qi) {
        row = block_off[(int64_t)host_rank[jj] * S + host_pslot[jj]] + (j - C);
        break;
      }
      C += qi;
    }
    if (row < 0) status = ORC_EDATA;
    row_of_slot[i] = (int32_t)row;
  }
  /* the plan's row of this rank must describe exactly these tokens */
  for (int32_t e = 0; e < E; e++) {
    int64_t tot = 0;
    for (int32_t jj = host_ptr[e]; jj < host_ptr[e + 1]; jj++) tot += q[jj];
    if (tot != seen[e]) status = ORC_EDATA;
  }
  if (status == ORC_OK) {
    for (int64_t i = 0; i < V; i++)
      if (row_of_slot[i] >= 0)
        memcpy(send + (int64_t)row_of_slot[i] * H, x + (i / k) * H,
               sizeof(uint16_t) * (size_t)H);
    /* rows beyond the routed ones (masked slots) are zero */
    if (V > v_valid)
      memset(send + v_valid * H, 0, sizeof(uint16_t) * (size_t)((V - v_valid) * H));
  }
  free(cnt);
  free(seen);
  return status;
}

/* ------------------------------------------------------------------ */
/* Step 4 — local half of weight distribution (Sec. 6.1)              */
/* ------------------------------------------------------------------ */

/* Every redundant slot (t, s) that hosts a main expert of `rank` receives
 * a bit copy of that expert's blob; entries are ordered by destination rank,
 * then by the destination's slot index. */
int orc_pack(const uint16_t *w_main, int64_t W, int32_t rank,
             const orc_group *g, const int32_t *slot_expert,
             uint16_t *staging, int64_t cap, int64_t *dest_off,
             int64_t *n_out) {
  if (!group_ok(g) || W < 1 || rank < 0 || rank >= g->R || !slot_expert ||
      !dest_off || !n_out || cap < 0 || !w_main)
    return ORC_EINVAL;
  const int32_t R = g->R, NS = g->n_slot, nm = g->E / g->R;
  int64_t n = 0;
  for (int32_t t = 0; t < R; t++) {
    dest_off[t] = n;
    for (int32_t s = 0; s < NS; s++) {
      int32_t e = slot_expert[(int64_t)t * NS + s];
      if (e >= 0 && home(g, e) == rank) n++;
    }
  }
  dest_off[R] = n;
  *n_out = n;
  if (n > cap) return ORC_ENOSPC;
  if (n > 0 && !staging) return ORC_EINVAL;
  n = 0;
  for (int32_t t = 0; t < R; t++)
    for (int32_t s = 0; s < NS; s++) {
      int32_t e = slot_expert[(int64_t)t * NS + s];
      if (e >= 0 && home(g, e) == rank) {
        memcpy(staging + n * W, w_main + (int64_t)(e - rank * nm) * W,
               sizeof(uint16_t) * (size_t)W);
        n++;
      }
    }
  return ORC_OK;
}

/* ------------------------------------------------------------------ */
/* Relay trees for hot-expert fan-out (Sec. 6.2, "Load-Aware Relay    */
/* Scheduling")                                                       */
/* ------------------------------------------------------------------ */

/* Integer nearest to sqrt(f) for f >= 0.  For an integer f, sqrt(f) is never
 * a half-integer, so the rounding has no ties: with n = floor(sqrt(f)),
 * round up iff f > n^2 + n (that is, f >= (n + 1/2)^2). */
static int64_t nearest_sqrt(int64_t f) {
  int64_t n = 0;
  while ((n + 1) * (n + 1) <= f) n++;
  return f > n * n + n ? n + 1 : n;
}

/* The paper tracks each rank's sending volume under the replication plan,
 * then, one hot expert at a time, picks first-stage relays among the
 * expert's replica ranks with the smallest volume and hangs every other
 * replica under the relay whose volume stays smallest after taking it; the
 * source's and relays' volumes are updated before the next expert.
 * Readings where the text is open:
 *   - eligible: replica count f_e = |H(e)| - 1 exceeds `threshold` (4 in
 *     the paper);
 *   - frontier: n_e = the integer nearest sqrt(f_e);
 *   - volume unit: one expert blob (all experts of a layer have the same
 *     size); rank r starts with one blob per replica of each main expert;
 *   - hot experts in order of f_e descending, then e ascending;
 *   - relays: the n_e replica ranks of smallest volume, ties to the smaller
 *     rank;
 *   - leaves: the other replicas by ascending rank, each under the relay of
 *     smallest volume (ties to the smaller rank), whose volume grows by one
 *     at once;
 *   - after the expert's leaves, the source's volume drops by f_e - n_e.
 * Output: slot_src[t*n_slot + s] = the rank that sends the blob of redundant
 * slot (t, s) (the home rank or a relay), -1 for an empty slot; send_vol[r];
 * relay_stats = {relay experts, sum of n_e, max volume before, max volume
 * after}. */
int orc_relay(const orc_group *g, const int32_t *slot_expert,
              const int32_t *host_ptr, const int32_t *host_rank,
              const int32_t *host_pslot, int32_t threshold, int32_t *slot_src,
              int32_t *send_vol, int64_t *relay_stats) {
  if (!group_ok(g) || !host_ptr || !host_rank || !host_pslot || threshold < 0 ||
      !send_vol || !relay_stats || (g->n_slot > 0 && (!slot_expert || !slot_src)))
    return ORC_EINVAL;
  const int32_t R = g->R, E = g->E, NS = g->n_slot, nm = E / R;
  const int64_t ncol = (int64_t)E + (int64_t)R * NS;
  /* the CSR must describe the slot map: home first, then replicas by
   * ascending rank, each on the slot that holds the expert */
  if (host_ptr[0] != 0 || host_ptr[E] < E || host_ptr[E] > ncol) return ORC_EDATA;
  for (int32_t e = 0; e < E; e++) {
    int32_t j0 = host_ptr[e], j1 = host_ptr[e + 1];
    if (j1 <= j0 || host_rank[j0] != home(g, e) || host_pslot[j0] != e - home(g, e) * nm)
      return ORC_EDATA;
    for (int32_t j = j0 + 1; j < j1; j++) {
      int32_t t = host_rank[j], s = host_pslot[j] - nm;
      if (t < 0 || t >= R || s < 0 || s >= NS || slot_expert[(int64_t)t * NS + s] != e ||
          (j > j0 + 1 && t <= host_rank[j - 1]) || t == home(g, e))
        return ORC_EDATA;
    }
  }
  int64_t *vol = calloc((size_t)R, sizeof(int64_t));
  for (int32_t t = 0; t < R; t++)
    for (int32_t s = 0; s < NS; s++) {
      int32_t e = slot_expert[(int64_t)t * NS + s];
      slot_src[(int64_t)t * NS + s] = e >= 0 ? home(g, e) : -1;
      if (e >= 0) vol[home(g, e)] += 1;
    }
  int64_t vmax0 = 0;
  for (int32_t r = 0; r < R; r++) vmax0 = max64(vmax0, vol[r]);

  /* hot experts, by replica count descending, then id ascending */
  int32_t *hot = malloc(sizeof(int32_t) * (size_t)E);
  int32_t nhot = 0;
  for (int32_t e = 0; e < E; e++)
    if (host_ptr[e + 1] - host_ptr[e] - 1 > threshold) hot[nhot++] = e;
  for (int32_t a = 1; a < nhot; a++) { /* insertion sort */
    int32_t e = hot[a], fe = host_ptr[e + 1] - host_ptr[e] - 1, b = a;
    while (b > 0) {
      int32_t p = hot[b - 1], fp = host_ptr[p + 1] - host_ptr[p] - 1;
      if (fp > fe || (fp == fe && p < e)) break;
      hot[b] = p;
      b--;
    }
    hot[b] = e;
  }

  int64_t n_relays = 0;
  int32_t *is_relay = calloc((size_t)R, sizeof(int32_t));
  for (int32_t h = 0; h < nhot; h++) {
    int32_t e = hot[h], j0 = host_ptr[e], j1 = host_ptr[e + 1];
    int64_t f = j1 - j0 - 1, n = nearest_sqrt(f);
    for (int32_t r = 0; r < R; r++) is_relay[r] = 0;
    /* first-stage relays: smallest volume, ties to the smaller rank */
    for (int64_t i = 0; i < n; i++) {
      int32_t best = -1;
      for (int32_t j = j0 + 1; j < j1; j++) {
        int32_t t = host_rank[j];
        if (is_relay[t]) continue;
        if (best < 0 || vol[t] < vol[best] || (vol[t] == vol[best] && t < best)) best = t;
      }
      is_relay[best] = 1;
    }
    /* leaves, ascending rank: the relay whose volume stays smallest */
    for (int32_t j = j0 + 1; j < j1; j++) {
      int32_t t = host_rank[j];
      if (is_relay[t]) continue;
      int32_t best = -1;
      for (int32_t jr = j0 + 1; jr < j1; jr++) {
        int32_t u = host_rank[jr];
        if (!is_relay[u]) continue;
        if (best < 0 || vol[u] + 1 < vol[best] + 1 || (vol[u] == vol[best] && u < best)) best = u;
      }
      vol[best] += 1;
      slot_src[(int64_t)t * NS + (host_pslot[j] - nm)] = best;
    }
    vol[home(g, e)] -= f - n; /* the source now sends to its relays only */
    n_relays += n;
  }
  int64_t vmax1 = 0;
  for (int32_t r = 0; r < R; r++) {
    vmax1 = max64(vmax1, vol[r]);
    send_vol[r] = (int32_t)vol[r];
  }
  relay_stats[0] = nhot;
  relay_stats[1] = n_relays;
  relay_stats[2] = vmax0;
  relay_stats[3] = vmax1;
  free(vol);
  free(hot);
  free(is_relay);
  return ORC_OK;
}

/* Local half of the weight distribution with relay trees: rank `rank`
 * stages one copy for every redundant slot whose sender (slot_src) it is,
 * destination ascending then slot ascending.  The blob of its own main
 * expert comes from w_main; the blob of an expert it relays comes from its
 * own redundant slot holding that expert (relay_src[s], the buffer the
 * first stage fills). */
int orc_pack_relay(const uint16_t *w_main, const uint16_t *relay_src, int64_t W,
                   int32_t rank, const orc_group *g, const int32_t *slot_expert,
                   const int32_t *slot_src, uint16_t *staging, int64_t cap,
                   int64_t *dest_off, int64_t *n_out) {
  if (!group_ok(g) || W < 1 || rank < 0 || rank >= g->R || !dest_off || !n_out ||
      cap < 0 || !w_main || (g->n_slot > 0 && (!slot_expert || !slot_src)))
    return ORC_EINVAL;
  const int32_t R = g->R, NS = g->n_slot, nm = g->E / g->R;
  int64_t n = 0;
  for (int32_t t = 0; t < R; t++) {
    dest_off[t] = n;
    for (int32_t s = 0; s < NS; s++)
      if (slot_expert[(int64_t)t * NS + s] >= 0 && slot_src[(int64_t)t * NS + s] == rank) n++;
  }
  dest_off[R] = n;
  *n_out = n;
  if (n > cap) return ORC_ENOSPC;
  if (n > 0 && !staging) return ORC_EINVAL;
  n = 0;
  for (int32_t t = 0; t < R; t++)
    for (int32_t s = 0; s < NS; s++) {
      int32_t e = slot_expert[(int64_t)t * NS + s];
      if (e < 0 || slot_src[(int64_t)t * NS + s] != rank) continue;
      const uint16_t *src = NULL;
      if (home(g, e) == rank) {
        src = w_main + (int64_t)(e - rank * nm) * W;
      } else {
        for (int32_t s2 = 0; s2 < NS; s2++)
          if (slot_expert[(int64_t)rank * NS + s2] == e) src = relay_src + (int64_t)s2 * W;
        if (!src || !relay_src) return ORC_EDATA; /* relays an expert it does not host */
      }
      memcpy(staging + n * W, src, sizeof(uint16_t) * (size_t)W);
      n++;
    }
  return ORC_OK;
}

/* ------------------------------------------------------------------ */
/* Reverse reroute: combine gather (Sec. 4.2 backward / the inverse   */
/* of the token assignment).  The ONLY floating point in the oracle.  */
/* ------------------------------------------------------------------ */

/* bf16 <-> fp32.  A bf16 pattern is the upper half of an fp32 pattern, so
 * widening is exact.  Narrowing rounds to nearest, ties to even: keep the
 * upper 16 bits, and add one unit of the kept part when the dropped 16 bits
 * exceed half a unit, or equal half a unit with an odd kept part.  Every
 * NaN becomes the quiet NaN 0x7FC0 (the sign of a NaN that an invalid
 * operation produces differs between processors). */
static float bf16_to_f32(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

static uint16_t f32_to_bf16(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  uint32_t mag = u & 0x7FFFFFFFu;
  if (mag > 0x7F800000u) return (uint16_t)0x7FC0u; /* NaN */
  uint32_t kept = u >> 16, dropped = u & 0xFFFFu;
  if (dropped > 0x8000u || (dropped == 0x8000u && (kept & 1u))) kept += 1; /* may carry into the exponent: correct, up to inf */
  return (uint16_t)kept;
}

/* Reading of the combine's arithmetic (the paper fixes bf16 activations
 * only): out[t] = bf16( sum over k ascending of fp32(gate[t][kk] * y[row]) )
 * with the sum accumulated in fp32 from +0, each product and each partial
 * sum rounded to fp32 (no fused multiply-add), masked slots (row -1)
 * skipped.  y is [n_rows][H] bf16 in the dispatch layout (row_of_slot),
 * gate [T][k] fp32, out [T][H] bf16.  A row outside [0, n_rows) is
 * ORC_EDATA. */
int orc_combine(const uint16_t *y, const float *gate, const int32_t *row_of_slot,
                int64_t T, int32_t k, int32_t H, int64_t n_rows, uint16_t *out) {
  if (T < 0 || k < 1 || H < 1 || n_rows < 0) return ORC_EINVAL;
  if (T > 0 && (!gate || !row_of_slot || !out)) return ORC_EINVAL;
  if (n_rows > 0 && !y) return ORC_EINVAL;
  for (int64_t i = 0; i < T * k; i++)
    if (row_of_slot[i] < -1 || row_of_slot[i] >= n_rows) return ORC_EDATA;
  for (int64_t t = 0; t < T; t++)
    for (int32_t h = 0; h < H; h++) {
      volatile float acc = 0.0f; /* volatile: every partial sum is an fp32 value */
      for (int32_t kk = 0; kk < k; kk++) {
        int32_t row = row_of_slot[t * k + kk];
        if (row < 0) continue;
        volatile float prod = gate[t * k + kk] * bf16_to_f32(y[(int64_t)row * H + h]);
        acc = acc + prod;
      }
      out[t * H + h] = f32_to_bf16(acc);
    }
  return ORC_OK;
}

/* ------------------------------------------------------------------ */
/* Gradient reduction, local half (Sec. 4.2 backward, Sec. 6.1)       */
/* ------------------------------------------------------------------ */

/* The gradients of this rank's replicated main experts come back from
 * their replicas and are accumulated into the main gradients, then the
 * replica buffers are cleared for the next layer.  Gradients are fp32 (the
 * paper's redundant-slot gradient is twice its bf16 weight).  Readings:
 * rgrad holds one [W] fp32 blob per replica, in the staging order of the
 * forward packing (destination rank ascending, then slot); each main
 * gradient is summed in fp32 starting from its own value and adding its
 * replicas in that order; every rgrad entry is zeroed afterwards.
 * ORC_ENOSPC if this rank has more replicas than cap (nothing changes). */
int orc_grad_reduce(float *main_grad, float *rgrad, int64_t W, int32_t rank,
                    const orc_group *g, const int32_t *slot_expert, int64_t cap,
                    int64_t *n_out) {
  if (!group_ok(g) || W < 1 || rank < 0 || rank >= g->R || !main_grad || !n_out || cap < 0 ||
      (g->n_slot > 0 && !slot_expert))
    return ORC_EINVAL;
  const int32_t R = g->R, NS = g->n_slot, nm = g->E / g->R;
  int64_t n = 0;
  for (int32_t t = 0; t < R; t++)
    for (int32_t s = 0; s < NS; s++) {
      int32_t e = slot_expert[(int64_t)t * NS + s];
      if (e >= 0 && home(g, e) == rank) n++;
    }
  *n_out = n;
  if (n > cap) return ORC_ENOSPC;
  if (n > 0 && !rgrad) return ORC_EINVAL;
  n = 0;
  for (int32_t t = 0; t < R; t++)
    for (int32_t s = 0; s < NS; s++) {
      int32_t e = slot_expert[(int64_t)t * NS + s];
      if (e < 0 || home(g, e) != rank) continue;
      float *mg = main_grad + (int64_t)(e - rank * nm) * W;
      float *rg = rgrad + n * W;
      for (int64_t i = 0; i < W; i++) {
        volatile float sum = mg[i] + rg[i];
        mg[i] = sum;
        rg[i] = 0.0f;
      }
      n++;
    }
  return ORC_OK;
}

/* ------------------------------------------------------------------ */
/* Diagnostics — Eqs. (3)-(5) and Table 3                             */
/* ------------------------------------------------------------------ */

int orc_metrics(const int32_t *load, const orc_group *g,
                const int32_t *quota, const int32_t *host_ptr,
                const int32_t *host_rank, const int32_t *reroute,
                int64_t *out) {
  if (!load || !group_ok(g) || !quota || !host_ptr || !host_rank ||
      !reroute || !out)
    return ORC_EINVAL;
  const int32_t R = g->R, E = g->E;
  const int64_t ncol = (int64_t)E + (int64_t)R * g->n_slot;
  ctx_t c;
  int st = ctx_init(&c, load, g);
  if (st != ORC_OK) { ctx_free(&c); return st; }
  int64_t before = 0, after = 0;
  for (int32_t r = 0; r < R; r++) before = max64(before, c.ell[r]);
  for (int32_t t = 0; t < R; t++) {
    int64_t s = 0;
    for (int32_t e = 0; e < E; e++) s += quota[(int64_t)e * R + t];
    after = max64(after, s);
  }
  int64_t n_rep = 0, max_h = 0, remote = 0;
  for (int32_t e = 0; e < E; e++) {
    int64_t n = host_ptr[e + 1] - host_ptr[e];
    n_rep += n - 1;
    max_h = max64(max_h, n);
    for (int32_t j = host_ptr[e]; j < host_ptr[e + 1]; j++)
      for (int32_t r = 0; r < R; r++)
        if (r != host_rank[j]) remote += reroute[(int64_t)r * ncol + j];
  }
  out[0] = before;
  out[1] = c.L;
  out[2] = after;
  out[3] = n_rep;
  out[4] = max_h;
  out[5] = remote;
  ctx_free(&c);
  return ORC_OK;
}
