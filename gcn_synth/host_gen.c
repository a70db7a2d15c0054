/* host_gen.c -- the Chung-Lu edge sampler of gcn_synth in C (libsynth_host.so).
 *
 * Draws exactly the edge set gcn_synth.chung_lu's numpy loop draws, an order of
 * magnitude faster, for graphs with tens of millions of edges.  Holds no
 * arithmetic of the GCN method: it only samples node pairs.
 *
 * The sampling rule (shared with the numpy loop): while fewer than e_und distinct
 * pairs are kept, a batch of b = trunc(1.15 need) + 1024 samples is drawn, need
 * being the pairs still missing.  Sample j of a batch that starts at stream offset
 * off takes u from output off + j and v from output off + b + j of the SplitMix64
 * sequence; each output h becomes a uniform (h >> 11) 2^-53 and the endpoint is the
 * first index whose cumulative weight exceeds it (clamped to n - 1).  Pairs with
 * u == v are skipped; the pair is keyed min * n + max; within a batch keys are kept
 * in sampling order, each the first time it appears and only if no earlier batch
 * kept it, until e_und are kept.  The next batch starts at off + 2 b.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define GAMMA 0x9E3779B97F4A7C15ull

static inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

/* first i with cdf[i] > x (numpy searchsorted side="right"), clamped to n - 1 */
static inline int64_t pick(const double* cdf, int64_t n, double x) {
  int64_t lo = 0, hi = n;
  while (lo < hi) {
    const int64_t mid = lo + ((hi - lo) >> 1);
    if (cdf[mid] > x) hi = mid; else lo = mid + 1;
  }
  return lo < n - 1 ? lo : n - 1;
}

static inline double u01(uint64_t state, uint64_t idx) {
  const uint64_t h = mix64(state + (idx + 1) * GAMMA);
  return (double)(h >> 11) * (1.0 / 9007199254740992.0);
}

/* Fills keys[0 .. e_und) with the kept pair keys (in the order they were kept).
 * Returns 0, or -1 if memory runs out. */
int synth_chung_lu_keys(int64_t n, int64_t e_und, const double* cdf, uint64_t state, int64_t* keys) {
  if (e_und <= 0) return 0;
  uint64_t cap = 1;
  while (cap < (uint64_t)e_und * 2 + 16) cap <<= 1;
  uint64_t* table = (uint64_t*)malloc(cap * sizeof(uint64_t));
  if (!table) return -1;
  memset(table, 0xff, cap * sizeof(uint64_t));
  const uint64_t empty = ~0ull, mask = cap - 1;
  const int64_t chunk = 1 << 20;
  int64_t* cand = (int64_t*)malloc(chunk * sizeof(int64_t));
  if (!cand) { free(table); return -1; }
  int64_t have = 0;
  uint64_t off = 0;
  while (have < e_und) {
    const int64_t need = e_und - have;
    const int64_t b = (int64_t)((double)need * 1.15) + 1024;
    for (int64_t j0 = 0; j0 < b && have < e_und; j0 += chunk) {
      const int64_t cnt = b - j0 < chunk ? b - j0 : chunk;
#pragma omp parallel for schedule(static)
      for (int64_t j = 0; j < cnt; ++j) {
        const int64_t u = pick(cdf, n, u01(state, off + (uint64_t)(j0 + j)));
        const int64_t v = pick(cdf, n, u01(state, off + (uint64_t)(b + j0 + j)));
        cand[j] = u == v ? -1 : (u < v ? u * n + v : v * n + u);
      }
      for (int64_t j = 0; j < cnt && have < e_und; ++j) {
        const int64_t k = cand[j];
        if (k < 0) continue;
        uint64_t slot = mix64((uint64_t)k) & mask;
        while (table[slot] != empty && table[slot] != (uint64_t)k) slot = (slot + 1) & mask;
        if (table[slot] == empty) {
          table[slot] = (uint64_t)k;
          keys[have++] = k;
        }
      }
    }
    off += 2 * (uint64_t)b;
  }
  free(cand);
  free(table);
  return 0;
}
