/*
 * Native generators for the shortest-path-distance (SPD) index matrices that
 * the synthetic graph workloads feed to biased graph attention.
 *
 * This is input construction only: the attention method takes spd as given
 * (the paper builds its structural bias on the CPU during data loading,
 * Section II-A and Section III-A-1, query-dimension bias sharding). Nothing
 * here computes any part of the attention.
 *
 * spd encoding (one byte per node pair, row-major):
 *   spd[s][v] = min(dist(s, v), clip)   if v is reachable from s
 *   spd[s][v] = clip + 1                if v is unreachable
 *   spd[s][s] = 0
 *
 * Build: gcc -O3 -fopenmp -shared -fPIC spdgen.c -o libspdgen.so
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <omp.h>

/* Clipped BFS distances from each requested source over an undirected graph
 * in CSR form, 64 sources at a time: bit b of frontier[v] / seen[v] says
 * whether source b of the block has reached node v (bit-parallel BFS).
 *   n        number of nodes
 *   indptr   [n+1] CSR row pointers, indices [indptr[n]] neighbour ids
 *   comp     [n] connected-component label of every node
 *   sources  [nsrc] source node ids; row r of out belongs to sources[r]
 *   clip     distance clip D (1..254); unreachable nodes get D+1
 *   out      nsrc rows, row r at out + r*ld_out, columns [0, n) written
 * Returns 0 on success, -1 on bad arguments, -2 on allocation failure. */
int spd_bfs_rows(int64_t n, const int64_t* indptr, const int32_t* indices,
                 const int32_t* comp, const int64_t* sources, int64_t nsrc,
                 int32_t clip, uint8_t* out, int64_t ld_out, int32_t nthreads) {
  if (n <= 0 || nsrc < 0 || clip < 1 || clip > 254 || ld_out < n) return -1;
  if (nthreads > 0) omp_set_num_threads(nthreads);
  const int64_t nblk = (nsrc + 63) / 64;
  int failed = 0;
#pragma omp parallel
  {
    uint64_t* front = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)n);
    uint64_t* next = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)n);
    uint64_t* seen = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)n);
    /* goal[v]: the sources of this block that share v's component, i.e. the
     * bits seen[v] ends with; nodes that reached it need no more work. */
    uint64_t* goal = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)n);
    int32_t ncomp = 0;
    for (int64_t v = 0; v < n; ++v) ncomp = comp[v] + 1 > ncomp ? comp[v] + 1 : ncomp;
    uint64_t* cmask = (uint64_t*)calloc((size_t)ncomp + 1, sizeof(uint64_t));
    const int ok = front && next && seen && goal && cmask;
    if (!ok) {
#pragma omp atomic write
      failed = 1;
    }
#pragma omp for schedule(dynamic, 1)
    for (int64_t blk = 0; blk < nblk; ++blk) {
      if (!ok) continue;
      const int64_t r0 = blk * 64;
      const int nb = (int)((nsrc - r0) < 64 ? (nsrc - r0) : 64);
      memset(front, 0, sizeof(uint64_t) * (size_t)n);
      memset(seen, 0, sizeof(uint64_t) * (size_t)n);
      /* Rows start as "distance >= clip": clip inside the source's component,
       * clip+1 outside it. BFS then overwrites the exact distances < clip. */
      for (int b = 0; b < nb; ++b) {
        const int64_t s = sources[r0 + b];
        uint8_t* row = out + (r0 + b) * ld_out;
        if (s < 0 || s >= n) { memset(row, 0xFF, (size_t)n); continue; }
        const int32_t cs = comp[s];
        for (int64_t v = 0; v < n; ++v)
          row[v] = (uint8_t)(comp[v] == cs ? clip : clip + 1);
        row[s] = 0;
        front[s] |= 1ull << b;
        seen[s] |= 1ull << b;
        cmask[cs] |= 1ull << b;
      }
      for (int64_t v = 0; v < n; ++v) goal[v] = cmask[comp[v]];
      for (int32_t level = 1; level < clip; ++level) {
        uint64_t any = 0;
        for (int64_t v = 0; v < n; ++v) {
          uint64_t acc = 0;
          if (seen[v] == goal[v]) { next[v] = 0; continue; }
          for (int64_t e = indptr[v]; e < indptr[v + 1]; ++e) acc |= front[indices[e]];
          acc &= ~seen[v];
          next[v] = acc;
          any |= acc;
        }
        if (!any) break;
        for (int64_t v = 0; v < n; ++v) {
          uint64_t m = next[v];
          if (!m) continue;
          seen[v] |= m;
          while (m) {
            const int b = __builtin_ctzll(m);
            m &= m - 1;
            out[(r0 + b) * ld_out + v] = (uint8_t)level;
          }
        }
        uint64_t* t = front; front = next; next = t;
      }
      for (int b = 0; b < nb; ++b) {
        const int64_t s = sources[r0 + b];
        if (s >= 0 && s < n) cmask[comp[s]] = 0;
      }
    }
    free(front); free(next); free(seen); free(goal); free(cmask);
  }
  return failed ? -2 : 0;
}

/* SplitMix64 finaliser (Steele, Lea, Flood 2014), used as a counter-based
 * generator: element (r, c) of the matrix draws from hash(seed, r*n + c). */
static inline uint64_t splitmix64(uint64_t x) {
  x += 0x9E3779B97F4A7C15ull;
  x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
  x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
  return x ^ (x >> 31);
}

/* i.i.d. bucket draws from a discrete distribution given by its CDF
 * (cdf[b] = P(bucket <= b), cdf[nb-1] == 1), diagonal forced to 0.
 * Rows [row0, row0+nrows) of an n x n matrix; row r at out + (r-row0)*ld_out. */
int spd_iid_rows(int64_t n, int64_t row0, int64_t nrows, const double* cdf,
                 int32_t nb, uint64_t seed, uint8_t* out, int64_t ld_out,
                 int32_t nthreads) {
  if (n <= 0 || row0 < 0 || nrows < 0 || nb < 1 || nb > 256 || ld_out < n) return -1;
  if (nthreads > 0) omp_set_num_threads(nthreads);
  const uint64_t key = splitmix64(seed);
#pragma omp parallel for schedule(static)
  for (int64_t rr = 0; rr < nrows; ++rr) {
    const int64_t r = row0 + rr;
    uint8_t* row = out + rr * ld_out;
    for (int64_t c = 0; c < n; ++c) {
      const uint64_t h = splitmix64(key ^ (uint64_t)(r * n + c));
      const double u = (double)(h >> 11) * (1.0 / 9007199254740992.0); /* [0,1) */
      int32_t lo = 0, hi = nb - 1;                                      /* first b with u < cdf[b] */
      while (lo < hi) {
        const int32_t mid = (lo + hi) >> 1;
        if (u < cdf[mid]) hi = mid; else lo = mid + 1;
      }
      row[c] = (uint8_t)lo;
    }
    if (r < n) row[r] = 0;
  }
  return 0;
}
