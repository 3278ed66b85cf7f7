// Device helpers shared by the kernel files of libspardl (internal).
#pragma once

#include "common.hpp"

namespace spardl {

typedef float f4v __attribute__((ext_vector_type(4)));

// Adds the non-zero bins of an LDS histogram of NB1 bins into a global one.
// Consecutive lanes take consecutive bins, so one wave's atomics fall on a
// few cache lines (a lane-strided split multiplies the L2 atomic requests).
__device__ __forceinline__ void flush_hist(const uint32_t* h, uint32_t* __restrict__ H) {
  for (int i = threadIdx.x; i < NB1; i += blockDim.x) {
    const uint32_t c = h[i];
    if (c) atomicAdd(&H[i], c);
  }
}

// Speculative candidates of the fused residual add (kernels_add.hip) and the
// floor of its level-1 histogram; the level-1 select (kernels_select.hip) and
// the lazy receipts (kernels_variants.hip) read the same words.
constexpr uint32_t SPEC_MARGIN = 2;     // level-1 bins between the previous threshold bin and the floor
constexpr uint32_t HIST_MARGIN = 32;    // further level-1 bins below the candidate floor kept in the histogram
constexpr uint32_t SPEC_NONE = 0xFFFFFFFFu;
constexpr uint32_t SPEC_DIRTY = 0x80000000u;   // set on spec_used: entries changed since the add, candidates stale

// Histogram floor (a key) for a candidate floor F (SPEC_NONE: histogram everything).
__device__ __forceinline__ uint32_t hist_floor(uint32_t F) {
  if (F == SPEC_NONE) return 0u;
  F &= ~SPEC_DIRTY;
  const uint32_t fb = F >> D1_SHIFT;
  return fb > HIST_MARGIN ? (fb - HIST_MARGIN) << D1_SHIFT : 0u;
}

// Levels 2 and 3 over the threshold-bin keys: visit(f) calls f(key) for
// every entry in bin T1.  Returns the threshold as (tge, teq, need_eq).
template <typename Visit>
__device__ __forceinline__ void resolve_low_digits(uint32_t T1, uint32_t need1, uint32_t cnt1, uint32_t* h,
                                                   uint32_t* scratch, uint32_t* err, Visit visit, uint32_t& tge,
                                                   uint32_t& teq, uint32_t& need_eq) {
  constexpr int NT = 1024;
  tge = T1 << D1_SHIFT;
  teq = 0u;
  need_eq = 0u;
  if (need1 == cnt1) return;
  __syncthreads();
  for (int i = threadIdx.x; i < NB2; i += NT) h[i] = 0u;
  __syncthreads();
  visit([&](uint32_t key) { atomicAdd(&h[(key >> D2_SHIFT) & (NB2 - 1)], 1u); });
  __syncthreads();
  uint32_t T2, above2, cnt2, ok;
  block_select_desc(h, NB2, need1, scratch, &T2, &above2, &cnt2, &ok);
  if (!ok) {
    if (threadIdx.x == 0) atomicOr(err, ERR_COUNT_L23);
    return;
  }
  const uint32_t need2 = need1 - above2;
  const uint32_t pre23 = (T1 << (D1_SHIFT - D2_SHIFT)) | T2;   // top 23 bits of the key
  tge = pre23 << D2_SHIFT;
  if (need2 == cnt2) return;
  for (int i = threadIdx.x; i < NB3; i += NT) h[i] = 0u;
  __syncthreads();
  visit([&](uint32_t key) {
    if ((key >> D2_SHIFT) == pre23) atomicAdd(&h[key & (NB3 - 1)], 1u);
  });
  __syncthreads();
  uint32_t T3, above3, cnt3;
  block_select_desc(h, NB3, need2, scratch, &T3, &above3, &cnt3, &ok);
  if (!ok) {
    if (threadIdx.x == 0) atomicOr(err, ERR_COUNT_L23);
    return;
  }
  const uint32_t need3 = need2 - above3;
  const uint32_t T = (pre23 << D2_SHIFT) | T3;
  if (need3 == cnt3) {
    tge = T;
  } else {
    tge = T + 1u;
    teq = T;
    need_eq = need3;
  }
}

// Bit x of the membership bitmap of the final index set.
__device__ __forceinline__ bool in_final(const uint32_t* __restrict__ bm, int32_t x) {
  return (bm[x >> 5] >> (x & 31)) & 1u;
}

static inline unsigned grid_for(int64_t work, int per_block, unsigned cap) {
  int64_t g = (work + per_block - 1) / per_block;
  if (g < 1) g = 1;
  return (unsigned)(g > cap ? cap : g);
}

}  // namespace spardl
