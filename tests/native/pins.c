/*
 * Native loops for the oracle's pins (tests only).  Links against the
 * oracle library; each function enumerates or samples far more cases than a
 * Python loop could.
 */
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

int orc_bounded_from_word(uint32_t x, uint32_t m, uint32_t* t);
int64_t orc_sample_node(uint64_t seed, uint32_t v, uint32_t l, int64_t d, int64_t f, uint32_t* slots);

typedef struct {
  uint32_t m; uint64_t lo, hi;
  uint64_t* counts; uint64_t rejects; int bad;
} bnd_job;

static void* bnd_run(void* p) {
  bnd_job* j = (bnd_job*)p;
  for (uint64_t x = j->lo; x < j->hi; ++x) {
    uint32_t t;
    if (orc_bounded_from_word((uint32_t)x, j->m, &t)) {
      if (t >= j->m) { j->bad = 1; continue; }
      j->counts[t]++;
    } else {
      j->rejects++;
    }
  }
  return NULL;
}

/* For every 32-bit word: accepted values counted in counts[m], rejected
 * words in *rejects.  Returns 1 if any accepted value fell outside [0, m). */
int pin_bounded_exhaustive(uint32_t m, uint64_t* counts, uint64_t* rejects, int nth) {
  if (nth < 1) nth = 1;
  if (nth > 32) nth = 32;
  pthread_t th[32];
  bnd_job jobs[32];
  uint64_t total = 1ULL << 32, chunk = (total + nth - 1) / nth;
  for (int t = 0; t < nth; ++t) {
    jobs[t].m = m;
    jobs[t].lo = chunk * t;
    jobs[t].hi = chunk * (t + 1) < total ? chunk * (t + 1) : total;
    jobs[t].counts = (uint64_t*)calloc(m, sizeof(uint64_t));
    jobs[t].rejects = 0;
    jobs[t].bad = 0;
    pthread_create(&th[t], NULL, bnd_run, &jobs[t]);
  }
  int bad = 0;
  *rejects = 0;
  memset(counts, 0, sizeof(uint64_t) * m);
  for (int t = 0; t < nth; ++t) {
    pthread_join(th[t], NULL);
    for (uint32_t i = 0; i < m; ++i) counts[i] += jobs[t].counts[i];
    *rejects += jobs[t].rejects;
    bad |= jobs[t].bad;
    free(jobs[t].counts);
  }
  return bad;
}

/* Histogram of sampled subsets (as bitmasks over d <= 24 slots) of a node of
 * degree d with fan-out f, over keys seed0 .. seed0+n-1 for node v, layer l.
 * Returns 1 if any sample broke an invariant (wrong size, not ascending,
 * slot out of range). */
int pin_subset_hist(uint32_t d, uint32_t f, uint32_t v, uint32_t l, uint64_t seed0, uint64_t n,
                    uint64_t* hist) {
  uint32_t slots[64];
  uint32_t k = d < f ? d : f;
  for (uint64_t s = 0; s < n; ++s) {
    int64_t got = orc_sample_node(seed0 + s, v, l, d, f, slots);
    if (got != (int64_t)k) return 1;
    uint32_t mask = 0;
    for (uint32_t q = 0; q < k; ++q) {
      if (slots[q] >= d) return 1;
      if (q > 0 && slots[q] <= slots[q - 1]) return 1;
      mask |= 1u << slots[q];
    }
    hist[mask]++;
  }
  return 0;
}

/* Same, varying the node id v0 .. v0+n-1 under one key (independence of the
 * per-node streams). */
int pin_subset_hist_nodes(uint32_t d, uint32_t f, uint32_t v0, uint32_t l, uint64_t seed, uint64_t n,
                          uint64_t* hist) {
  uint32_t slots[64];
  uint32_t k = d < f ? d : f;
  for (uint64_t s = 0; s < n; ++s) {
    int64_t got = orc_sample_node(seed, v0 + (uint32_t)s, l, d, f, slots);
    if (got != (int64_t)k) return 1;
    uint32_t mask = 0;
    for (uint32_t q = 0; q < k; ++q) {
      if (slots[q] >= d) return 1;
      if (q > 0 && slots[q] <= slots[q - 1]) return 1;
      mask |= 1u << slots[q];
    }
    hist[mask]++;
  }
  return 0;
}

/* Marginal inclusion counts incl[d] of each slot for a large degree d. */
int pin_marginals(uint32_t d, uint32_t f, uint32_t v, uint32_t l, uint64_t seed0, uint64_t n,
                  uint64_t* incl) {
  uint32_t* slots = (uint32_t*)malloc(sizeof(uint32_t) * (f > 0 ? f : 1));
  uint32_t k = d < f ? d : f;
  for (uint64_t s = 0; s < n; ++s) {
    int64_t got = orc_sample_node(seed0 + s, v, l, d, f, slots);
    if (got != (int64_t)k) { free(slots); return 1; }
    for (uint32_t q = 0; q < k; ++q) {
      if (slots[q] >= d || (q > 0 && slots[q] <= slots[q - 1])) { free(slots); return 1; }
      incl[slots[q]]++;
    }
  }
  free(slots);
  return 0;
}
