/* Device side of the synthetic gradient generator (input plumbing only).
 *
 * The same definitions as the host generator (gradgen.h), compiled for the
 * GPU with no contraction, so a slice generated here has the bits the host
 * generator gives for it.  It lets the largest workloads create their
 * per-worker gradients in HBM in milliseconds; the oracle still regenerates
 * the blocks it checks on the host. */
#include <hip/hip_runtime.h>
#include <stdint.h>

#define GG_FN __device__ static inline
#include "gradgen.h"

/* out[j] = element x0 + j of one worker's gradient, j < count; seg_start
 * (nseg + 1 entries) and seg_scale (nseg) are device arrays. */
__global__ __launch_bounds__(256) void gg_fill_kernel(float* __restrict__ out, int64_t count, int64_t x0,
                                                      uint64_t key, int dist,
                                                      const int64_t* __restrict__ seg_start,
                                                      const double* __restrict__ seg_scale, int nseg,
                                                      double zero_prob) {
  for (int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x; j < count; j += (int64_t)gridDim.x * 256) {
    const int64_t x = x0 + j;
    int lo = 0, hi = nseg;   /* last segment with seg_start[lo] <= x */
    while (hi - lo > 1) {
      const int mid = (lo + hi) / 2;
      if (seg_start[mid] <= x) lo = mid;
      else hi = mid;
    }
    out[j] = gg_value(key, (uint64_t)x, dist, seg_scale[lo], zero_prob);
  }
}

extern "C" int gg_fill_device(float* out, int64_t count, int64_t x0, uint64_t key, int dist,
                              const int64_t* seg_start, const double* seg_scale, int nseg,
                              double zero_prob, hipStream_t stream) {
  if (count <= 0) return 0;
  if (!out || !seg_start || !seg_scale || nseg < 1) return (int)hipErrorInvalidValue;
  int64_t blocks = (count + 255) / 256;
  if (blocks > 262144) blocks = 262144;
  hipLaunchKernelGGL(gg_fill_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, out, count, x0, key, dist,
                     seg_start, seg_scale, nseg, zero_prob);
  return (int)hipGetLastError();
}
