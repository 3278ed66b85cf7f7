/* Host side of the synthetic gradient generator (input plumbing only).
 * Built with gcc -O2 -fopenmp -ffp-contract=off; see gradgen.h for the
 * definition of every value. */
#include <stddef.h>
#include <stdint.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define GG_FN static inline
#include "gradgen.h"

/* out[j] = value of element x0 + j of one worker's flat gradient, j < count.
 * Segments: seg_start[s] <= x < seg_start[s+1] uses seg_scale[s]
 * (seg_start has nseg + 1 entries, seg_start[0] = 0, increasing). */
void gg_fill(float* out, int64_t count, int64_t x0, uint64_t key, int dist,
             const int64_t* seg_start, const double* seg_scale, int nseg, double zero_prob) {
  if (count <= 0) return;
#pragma omp parallel
  {
    int nt = 1, tid = 0;
#ifdef _OPENMP
    nt = omp_get_num_threads();
    tid = omp_get_thread_num();
#endif
    const int64_t lo = x0 + count * tid / nt, hi = x0 + count * (tid + 1) / nt;
    int s = 0, s_hi = nseg;          /* last segment with seg_start[s] <= lo */
    while (s_hi - s > 1) {
      int mid = (s + s_hi) / 2;
      if (seg_start[mid] <= lo) s = mid;
      else s_hi = mid;
    }
    for (int64_t x = lo; x < hi; ++x) {
      while (s + 1 < nseg && seg_start[s + 1] <= x) ++s;
      out[x - x0] = gg_value(key, (uint64_t)x, dist, seg_scale[s], zero_prob);
    }
  }
}

uint64_t gg_mix(uint64_t z) { return gg_mix64(z); }
double gg_log_host(double x) { return gg_log(x); }
