/*
 * Brute-force optimum of the replication problem on tiny groups (test pin).
 *
 * For every full placement (each rank fills all of its n_slot redundant
 * slots with distinct experts that it does not already host), the smallest
 * achievable max rank load with integer splits is, by Hall's theorem and the
 * integrality of max-flow, max over non-empty rank subsets T of
 *     ceil( sum_{e : H(e) subset of T} lambda_e / |T| ).
 * The optimum is the minimum of that over all placements.  With u_min = 1
 * adding a replica never hurts, so full placements suffice.  Placements that
 * leave slots empty are also enumerated when fewer candidates than slots
 * exist.  R <= 6, E <= 16.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

static int R, E, NS, nm;
static int64_t lam[64];
static int nchoice;
static uint32_t choices[16384]; /* bitmask of experts chosen by one rank */
static int rank_choice_ok[8][16384];
static int cur[8];
static int64_t best = -1;

static int popc(uint32_t x) { return __builtin_popcount(x); }

static void eval(void) {
  uint32_t hm[64];
  for (int e = 0; e < E; e++) hm[e] = 1u << (e / nm);
  for (int r = 0; r < R; r++) {
    uint32_t m = choices[cur[r]];
    for (int e = 0; e < E; e++)
      if (m >> e & 1u) hm[e] |= 1u << r;
  }
  int64_t by_mask[256] = {0};
  for (int e = 0; e < E; e++) by_mask[hm[e]] += lam[e];
  /* subset-sum (zeta) transform: f[T] = sum over masks inside T */
  for (int b = 0; b < R; b++)
    for (int m = 0; m < (1 << R); m++)
      if (m >> b & 1) by_mask[m] += by_mask[m ^ (1 << b)];
  int64_t opt = 0;
  for (int T = 1; T < (1 << R); T++) {
    int64_t n = popc((uint32_t)T);
    int64_t v = (by_mask[T] + n - 1) / n;
    if (v > opt) opt = v;
  }
  if (best < 0 || opt < best) best = opt;
}

static void rec(int r) {
  if (r == R) { eval(); return; }
  for (int c = 0; c < nchoice; c++)
    if (rank_choice_ok[r][c]) { cur[r] = c; rec(r + 1); }
}

int main(int argc, char **argv) {
  /* usage: bruteforce R E n_slot lam_0 ... lam_{E-1} */
  if (argc < 4) return 2;
  R = atoi(argv[1]); E = atoi(argv[2]); NS = atoi(argv[3]);
  if (R < 1 || R > 6 || E < 1 || E > 16 || E % R || argc != 4 + E) return 2;
  nm = E / R;
  for (int e = 0; e < E; e++) lam[e] = atoll(argv[4 + e]);
  /* all subsets of experts of size min(NS, E - nm) */
  int want = NS < E - nm ? NS : E - nm;
  nchoice = 0;
  for (uint32_t m = 0; m < (1u << E); m++)
    if (popc(m) == want) choices[nchoice++] = m;
  for (int r = 0; r < R; r++)
    for (int c = 0; c < nchoice; c++) {
      uint32_t home = ((1u << nm) - 1) << (r * nm);
      rank_choice_ok[r][c] = (choices[c] & home) == 0;
    }
  rec(0);
  printf("%lld\n", (long long)best);
  return 0;
}
