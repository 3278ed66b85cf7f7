// Device helpers shared by the kernel files of libspardl (internal).
#pragma once

#include "common.hpp"

namespace spardl {

typedef float f4v __attribute__((ext_vector_type(4)));

// Adds the non-zero bins of an LDS histogram of NB1 bins into a global one,
// by a workgroup of NT threads.  Consecutive lanes take consecutive bins
// (thread t bins t, t + NT, ...), so one wave's atomics fall on a few cache
// lines (a lane-strided split multiplies the L2 atomic requests); a thread
// issues all its LDS reads before its atomics.
template <int NT>
__device__ __forceinline__ void flush_hist(const uint32_t* h, uint32_t* __restrict__ H) {
  constexpr int PER = NB1 / NT;
  static_assert(PER * NT == NB1, "whole bins per thread");
  uint32_t c[PER];
#pragma unroll
  for (int k = 0; k < PER; ++k) c[k] = h[threadIdx.x + k * NT];
#pragma unroll
  for (int k = 0; k < PER; ++k)
    if (c[k]) atomicAdd(&H[threadIdx.x + k * NT], c[k]);
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

// Level-1 bins of a block's histogram, given the word the fused add left in
// spec_used for the block (its candidate floor F; SPEC_NONE: none).  With a
// floor the histogram counts only keys at or above FH = hist_floor(F), two
// binades lower: the keys in [FH, F) in bins of the top 12 key bits (bins 0
// .. M_MARGIN - 1), the keys from F up -- the speculative candidates, a few
// per cent of the block -- in bins of 2^FINE_SHIFT keys (1/256 binade, bins
// M_MARGIN .. NB1 - 1, the last also holding every larger key), so that a
// threshold bin among the candidates holds few entries while a tile still
// touches few bins.  Bin order is key order throughout.  Without a floor (a
// block's first step, or a histogram made without the add) every key counts
// and a bin is the top 12 key bits.  The fused add, the lazy receipts that
// keep its histograms exact and the level-1 select all bin through this map.
constexpr uint32_t M_MARGIN = HIST_MARGIN;   // 12-bit bins below the candidate floor
struct L1Map {
  uint32_t floor;   // smallest key counted (FH)
  uint32_t cand;    // the candidate floor F (fine bins from here)
  bool fine;
  __device__ __forceinline__ uint32_t bin(uint32_t key) const {
    if (!fine) return key >> D1_SHIFT;
    if (key < cand) return (key >> D1_SHIFT) - (floor >> D1_SHIFT);   // key >= floor
    return M_MARGIN + min((key >> FINE_SHIFT) - (cand >> FINE_SHIFT), (uint32_t)NB1 - 1u - M_MARGIN);
  }
  // the keys of bin T: k >> *S == *pfx; false for the last fine bin, which
  // also holds every larger key
  __device__ __forceinline__ bool bin_keys(uint32_t T, uint32_t* pfx, uint32_t* S) const {
    if (!fine) {
      *pfx = T;
      *S = D1_SHIFT;
      return true;
    }
    if (T < M_MARGIN) {
      *pfx = (floor >> D1_SHIFT) + T;
      *S = D1_SHIFT;
      return true;
    }
    *pfx = (cand >> FINE_SHIFT) + (T - M_MARGIN);
    *S = FINE_SHIFT;
    return T != (uint32_t)NB1 - 1u;
  }
};
__device__ __forceinline__ L1Map l1_map(uint32_t used) {
  L1Map m;
  m.fine = used != SPEC_NONE;
  m.cand = used & ~SPEC_DIRTY;
  m.floor = hist_floor(used);
  return m;
}
static_assert(HIST_MARGIN < (uint32_t)NB1 / 2, "the 12-bit margin bins leave most bins fine");

// Levels 2 and 3 over the keys of one level-1 bin, the keys k with
// k >> S == pfx (visit(f) calls f(key) for each of them), in two digits of
// the low S bits, the last of S == FINE_SHIFT ? 7 : 8 bits; h holds at
// least 2^(S - that) words.  Returns the threshold as (tge, teq, need_eq):
// every key >= tge is selected, and the first need_eq (by index) with key
// == teq.
template <typename Visit>
__device__ __forceinline__ void resolve_bin(uint32_t pfx, int S, uint32_t need1, uint32_t cnt1, uint32_t* h,
                                            uint32_t* scratch, uint32_t* err, Visit visit, uint32_t& tge,
                                            uint32_t& teq, uint32_t& need_eq) {
  const int D3 = S == FINE_SHIFT ? 7 : 8;
  const int nb2 = 1 << (S - D3), nb3 = 1 << D3;
  tge = pfx << S;
  teq = 0u;
  need_eq = 0u;
  if (need1 == cnt1) return;
  __syncthreads();
  for (int i = threadIdx.x; i < nb2; i += blockDim.x) h[i] = 0u;
  __syncthreads();
  visit([&](uint32_t key) { atomicAdd(&h[(key >> D3) & (uint32_t)(nb2 - 1)], 1u); });
  __syncthreads();
  uint32_t T2, above2, cnt2, ok;
  block_select_desc(h, nb2, need1, scratch, &T2, &above2, &cnt2, &ok);
  if (!ok) {
    if (threadIdx.x == 0) atomicOr(err, ERR_COUNT_L23);
    return;
  }
  const uint32_t need2 = need1 - above2;
  const uint32_t pre = (pfx << (S - D3)) | T2;   // all but the last D3 key bits
  tge = pre << D3;
  if (need2 == cnt2) return;
  for (int i = threadIdx.x; i < nb3; i += blockDim.x) h[i] = 0u;
  __syncthreads();
  visit([&](uint32_t key) {
    if ((key >> D3) == pre) atomicAdd(&h[key & (uint32_t)(nb3 - 1)], 1u);
  });
  __syncthreads();
  uint32_t T3, above3, cnt3;
  block_select_desc(h, nb3, need2, scratch, &T3, &above3, &cnt3, &ok);
  if (!ok) {
    if (threadIdx.x == 0) atomicOr(err, ERR_COUNT_L23);
    return;
  }
  const uint32_t need3 = need2 - above3;
  const uint32_t T = (pre << D3) | T3;
  if (need3 == cnt3) {
    tge = T;
  } else {
    tge = T + 1u;
    teq = T;
    need_eq = need3;
  }
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
