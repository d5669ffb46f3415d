/*
 * Seeded candidate-placement generator (input synthesis only).
 *
 * This file draws the batch of candidate placements that the what-if
 * simulator evaluates (the "CandidatePartitions" loop of the incremental
 * simulation-based scheduling algorithm, Alg. 1 / Sec. 3.4.2).  It holds no
 * part of the simulator's arithmetic: it only produces device ids.
 *
 * Random numbers come from SplitMix64 (Steele, Lea & Flood, "Fast splittable
 * pseudorandom number generators", OOPSLA 2014) used as a counter-based
 * generator: the n-th output under key k is mix(k + (n + 1) * gamma).  The
 * Python side of the generator uses the same definition for every other
 * seeded quantity, so a candidate is a pure function of (root key, index).
 *
 * Candidate b (row-major output, one byte per operator):
 *   key_b  = draw(root, b)
 *   mode   = (b odd) ? mode_odd : mode_even
 *   mode 0 (uniform):  p[v] = below(draw(key_b, v), D)
 *   mode 1 (perturb):  p = base; k = kmin + below(draw(key_b, 0), kmax-kmin+1);
 *                      for j = 1..k: v = below(draw(key_b, 2j-1), N);
 *                        distinct: r = below(draw(key_b, 2j), D-1); p[v] = r + (r >= p[v])
 *                        else:     p[v] = below(draw(key_b, 2j), D)
 * where below(x, n) = floor(x * n / 2^64) (Lemire's multiply-shift).
 */
#include <pthread.h>
#include <stdint.h>
#include <string.h>

#define SYN_GAMMA 0x9E3779B97F4A7C15ULL

static inline uint64_t syn_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

static inline uint64_t syn_draw(uint64_t key, uint64_t n) {
  return syn_mix(key + (n + 1) * SYN_GAMMA);
}

static inline uint64_t syn_below(uint64_t x, uint64_t n) {
  return (uint64_t)(((unsigned __int128)x * n) >> 64);
}

typedef struct {
  uint64_t root;
  int64_t n_ops;
  int32_t n_dev;
  int32_t mode_even, mode_odd;
  int32_t kmin, kmax, distinct;
  const uint8_t *base;
} syn_recipe;

uint64_t synth_draw(uint64_t key, uint64_t n) { return syn_draw(key, n); }

static void syn_one(const syn_recipe *r, int64_t b, uint8_t *row) {
  const uint64_t kb = syn_draw(r->root, (uint64_t)b);
  const int mode = (b & 1) ? r->mode_odd : r->mode_even;
  const int64_t N = r->n_ops;
  const uint64_t D = (uint64_t)r->n_dev;
  if (mode == 0) {
    for (int64_t v = 0; v < N; ++v) row[v] = (uint8_t)syn_below(syn_draw(kb, (uint64_t)v), D);
    return;
  }
  memcpy(row, r->base, (size_t)N);
  if (N == 0) return;
  const uint64_t span = (uint64_t)(r->kmax - r->kmin + 1);
  const int64_t k = r->kmin + (int64_t)syn_below(syn_draw(kb, 0), span);
  for (int64_t j = 1; j <= k; ++j) {
    const int64_t v = (int64_t)syn_below(syn_draw(kb, (uint64_t)(2 * j - 1)), (uint64_t)N);
    const uint64_t x = syn_draw(kb, (uint64_t)(2 * j));
    if (r->distinct && D > 1) {
      const uint64_t t = syn_below(x, D - 1);
      row[v] = (uint8_t)(t + (t >= row[v] ? 1 : 0));
    } else {
      row[v] = (uint8_t)syn_below(x, D);
    }
  }
}

typedef struct {
  const syn_recipe *r;
  int64_t b_lo, b_hi;
  uint8_t *out;
  int64_t b0;
} syn_job;

static void *syn_worker(void *arg) {
  const syn_job *j = (const syn_job *)arg;
  for (int64_t b = j->b_lo; b < j->b_hi; ++b)
    syn_one(j->r, b, j->out + (b - j->b0) * j->r->n_ops);
  return 0;
}

/* Fill out[nb][n_ops] with candidates b0 .. b0+nb-1.  Returns 0 on success. */
int synth_placements(uint64_t root, int64_t n_ops, int32_t n_dev, int32_t mode_even, int32_t mode_odd,
                     int32_t kmin, int32_t kmax, int32_t distinct, const uint8_t *base, int64_t b0,
                     int64_t nb, uint8_t *out, int32_t n_threads) {
  if (n_ops < 0 || n_dev < 1 || n_dev > 256 || nb < 0 || kmin < 0 || kmax < kmin) return -1;
  if ((mode_even == 1 || mode_odd == 1) && base == 0) return -1;
  syn_recipe r = {root, n_ops, n_dev, mode_even, mode_odd, kmin, kmax, distinct, base};
  if (n_threads < 1) n_threads = 1;
  if (n_threads > 64) n_threads = 64;
  if (nb < 64 * (int64_t)n_threads) n_threads = (int32_t)(nb / 64 > 0 ? (nb / 64 < n_threads ? nb / 64 : n_threads) : 1);
  pthread_t th[64];
  int spawned[64];
  syn_job jobs[64];
  const int64_t per = (nb + n_threads - 1) / n_threads;
  int used = 0;
  for (int t = 0; t < n_threads; ++t) {
    int64_t lo = b0 + t * per, hi = lo + per;
    if (hi > b0 + nb) hi = b0 + nb;
    if (lo >= hi) break;
    jobs[t] = (syn_job){&r, lo, hi, out, b0};
    spawned[t] = (t < n_threads - 1) && pthread_create(&th[t], 0, syn_worker, &jobs[t]) == 0;
    if (!spawned[t]) syn_worker(&jobs[t]);
    used = t + 1;
  }
  for (int t = 0; t < used; ++t)
    if (spawned[t]) pthread_join(th[t], 0);
  return 0;
}
