/*
 * Seeded synthetic MoE routing / activation / weight generator.
 *
 * Shared input source for the test-suite and the benchmark.  It holds none of
 * the balancing method's arithmetic: it only draws router logits, selects the
 * top-k experts per token the way the evaluated MoE routers do, and fills
 * activation and weight buffers.
 *
 * Random numbers: counter-based splitmix64 (Steele, Lea, Flood, "Fast
 * splittable pseudorandom number generators", OOPSLA 2014).  Draw i of a
 * stream with key K is mix64(K + (i + 1) * 0x9E3779B97F4A7C15), so any slice
 * of any stream can be produced independently and the output does not depend
 * on the number of threads.  Normals use the Box-Muller transform (cosine
 * branch only); bf16 values are rounded to nearest-even from fp32.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define GOLDEN 0x9E3779B97F4A7C15ULL

static inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

static inline uint64_t draw(uint64_t key, uint64_t i) {
  return mix64(key + (i + 1) * GOLDEN);
}

/* uniform in (0, 1] with 53 random bits */
static inline double unif(uint64_t key, uint64_t i) {
  return ((double)(draw(key, i) >> 11) + 1.0) * (1.0 / 9007199254740992.0);
}

static inline double normal(uint64_t key, uint64_t i) {
  double u1 = unif(key, 2 * i), u2 = unif(key, 2 * i + 1);
  return sqrt(-2.0 * log(u1)) * cos(6.283185307179586 * u2);
}

/* Stream key from a seed and four labels. */
uint64_t gen_key(uint64_t seed, uint64_t a, uint64_t b, uint64_t c, uint64_t d) {
  uint64_t h = mix64(seed + GOLDEN);
  h = mix64(h ^ (a + GOLDEN));
  h = mix64(h ^ (b + 2 * GOLDEN));
  h = mix64(h ^ (c + 3 * GOLDEN));
  h = mix64(h ^ (d + 4 * GOLDEN));
  return h;
}

void gen_normals(uint64_t key, int64_t n, double *out) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; i++) out[i] = normal(key, (uint64_t)i);
}

static inline uint16_t f32_to_bf16_rne(float f) {
  uint32_t b;
  memcpy(&b, &f, 4);
  uint32_t lsb = (b >> 16) & 1u;
  b += 0x7FFFu + lsb;
  return (uint16_t)(b >> 16);
}

/* bf16 N(0,1) activations, n values */
void gen_bf16_normals(uint64_t key, int64_t n, uint16_t *out) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; i++) out[i] = f32_to_bf16_rne((float)normal(key, (uint64_t)i));
}

/* arbitrary 16-bit patterns (every bf16 encoding, NaN and Inf included) */
void gen_bits16(uint64_t key, int64_t n, uint16_t *out) {
  int64_t nw = (n + 3) / 4;
#pragma omp parallel for schedule(static)
  for (int64_t w = 0; w < nw; w++) {
    uint64_t v = draw(key, (uint64_t)w);
    for (int j = 0; j < 4; j++) {
      int64_t i = 4 * w + j;
      if (i < n) out[i] = (uint16_t)(v >> (16 * j));
    }
  }
}

/* Seeded permutation of 0..n-1 (Fisher-Yates). */
void gen_perm(uint64_t key, int32_t n, int32_t *out) {
  for (int32_t i = 0; i < n; i++) out[i] = i;
  for (int32_t i = n - 1; i > 0; i--) {
    int32_t j = (int32_t)(draw(key, (uint64_t)i) % (uint64_t)(i + 1));
    int32_t t = out[i];
    out[i] = out[j];
    out[j] = t;
  }
}

/* is (va, a) ranked before (vb, b): larger value first, smaller index on ties */
static inline int before(double va, int32_t a, double vb, int32_t b) {
  return va > vb || (va == vb && a < b);
}

/*
 * Router: for each of n_tok tokens (global token ids tok0 .. tok0+n_tok-1 of
 * the logit stream `key`), logits z_e = N(0,1) + bias[e]; returns the k
 * experts with the largest logits in descending order (ties: smaller id).
 * With n_group > 0 the experts are split into n_group contiguous groups, a
 * group scores the sum of its two largest logits, only the top_group best
 * groups (ties: smaller group) stay eligible, and the k experts are taken
 * among them (DeepSeek-V3 style node-limited routing).
 */
int gen_router_topk(uint64_t key, int64_t tok0, int64_t n_tok, int32_t E,
                    int32_t k, const double *bias, int32_t n_group,
                    int32_t top_group, int32_t *topk) {
  if (E < 1 || k < 1 || k > E || E > 4096) return -1;
  if (n_group > 0 && (E % n_group != 0 || top_group < 1 || top_group > n_group ||
                      k > top_group * (E / n_group) || E / n_group < 2 || n_group > 64))
    return -1;
#pragma omp parallel
  {
    double z[4096];
    double gs[64];
    int32_t gsel[64];
#pragma omp for schedule(static)
    for (int64_t t = 0; t < n_tok; t++) {
      uint64_t base = (uint64_t)(tok0 + t) * (uint64_t)E;
      for (int32_t e = 0; e < E; e++) z[e] = normal(key, base + (uint64_t)e) + bias[e];
      int32_t *out = topk + t * k;
      if (n_group > 0) {
        int32_t gsz = E / n_group;
        for (int32_t gi = 0; gi < n_group; gi++) {
          double m1 = -INFINITY, m2 = -INFINITY;
          for (int32_t j = 0; j < gsz; j++) {
            double v = z[gi * gsz + j];
            if (v > m1) { m2 = m1; m1 = v; }
            else if (v > m2) { m2 = v; }
          }
          gs[gi] = m1 + m2;
          gsel[gi] = 0;
        }
        for (int32_t s = 0; s < top_group; s++) {
          int32_t b = -1;
          for (int32_t gi = 0; gi < n_group; gi++)
            if (!gsel[gi] && (b < 0 || before(gs[gi], gi, gs[b], b))) b = gi;
          gsel[b] = 1;
        }
        for (int32_t gi = 0; gi < n_group; gi++)
          if (!gsel[gi])
            for (int32_t j = 0; j < gsz; j++) z[gi * gsz + j] = -INFINITY;
      }
      /* insertion into a descending list of length k */
      int32_t cnt = 0;
      for (int32_t e = 0; e < E; e++) {
        double v = z[e];
        if (v == -INFINITY) continue;
        if (cnt == k && !before(v, e, z[out[k - 1]], out[k - 1])) continue;
        int32_t p = cnt < k ? cnt : k - 1;
        while (p > 0 && before(v, e, z[out[p - 1]], out[p - 1])) {
          out[p] = out[p - 1];
          p--;
        }
        out[p] = e;
        if (cnt < k) cnt++;
      }
    }
  }
  return 0;
}
