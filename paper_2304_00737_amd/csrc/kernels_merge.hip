// Index-sum merge of a Spar-Reduce-Scatter step (Sec. III-B "Transmission
// with sparsification"; also the R-SAG exchanges of Sec. III-D) for gfx950:
// merge-path tiles of two index-sorted sparse blocks, feeding the selection
// stages of kernels_select.hip.

#include "device.hpp"
#include "launch.hpp"

#include <algorithm>

namespace spardl {

// ============================================================================ a4: merge-path index sum
// Pair p (Pairs in common.hpp): held block + received block, e.g. for an SRS
// step held = sp[w][b], received = sp[(w - d) mod P][b], b = (w+t) mod P.
// The merged sequence orders by index with the held entry first on equal
// indices; the held entry then emits held + received and the received entry
// leaves a hole.  Tile = MERGE_TILE merged positions; its hole-free part is
// written densely into the tile's slot, and the level-1 histogram of the
// union is accumulated for the selection.
__global__ __launch_bounds__(MERGE_THREADS) void k_merge(
    const int32_t* __restrict__ sp_idx, const float* __restrict__ sp_val, Pairs PM, int32_t kb,
    int32_t tiles_per_pair, uint32_t* __restrict__ hist1,
    uint32_t* __restrict__ slot_cnt, int32_t* __restrict__ U_idx, float* __restrict__ U_val) {
  // held entries a0-1 .. a1 at [0, nh + 2), received b0 .. b1 at [nh + 2, nh + nr + 3)
  __shared__ int32_t cI[MERGE_TILE + 3];
  __shared__ float cV[MERGE_TILE + 3];
  __shared__ __align__(16) uint32_t hist[NB1];
  __shared__ uint32_t scratch[2 * (MERGE_THREADS / WAVE) + 1];
  const uint32_t pair = blockIdx.x / (uint32_t)tiles_per_pair;
  const int32_t tile = (int32_t)(blockIdx.x % (uint32_t)tiles_per_pair);
  int64_t hb, rb;
  bool both;
  PM.decode(pair, &hb, &rb, &both);
  const int32_t* __restrict__ Hi = sp_idx + hb * kb;
  const float* __restrict__ Hv = sp_val + hb * kb;
  const int32_t* __restrict__ Ri = sp_idx + rb * kb;
  const float* __restrict__ Rv = sp_val + rb * kb;
  const int32_t L2 = 2 * kb;
  for (int i = threadIdx.x; i < NB1 / 4; i += blockDim.x) reinterpret_cast<uint4*>(hist)[i] = make_uint4(0u, 0u, 0u, 0u);
  const int32_t Q0 = tile * MERGE_TILE;
  const int32_t Q1 = min(Q0 + MERGE_TILE, L2);
  // split(q) = number of held entries among the first q merged positions:
  // the first a in [max(0, q-kb), min(q, kb)) whose held entry does not go
  // before received entry q-a-1 (held goes first on equal indices).  The
  // tile's two splits are searched together.
  int32_t a0, a1;
  wg_partition_point2(max(0, Q0 - kb), min(Q0, kb), [&](int32_t a) { return Hi[a] <= Ri[Q0 - a - 1]; },
                      max(0, Q1 - kb), min(Q1, kb), [&](int32_t a) { return Hi[a] <= Ri[Q1 - a - 1]; }, scratch,
                      &a0, &a1);
  const int32_t b0 = Q0 - a0, b1 = Q1 - a1;
  const int32_t nh = a1 - a0, nr = b1 - b0;
  int32_t* hI = cI;
  float* hV = cV;
  int32_t* rI = cI + nh + 2;
  float* rV = cV + nh + 2;
  {
    // hI[i] = held[a0 - 1 + i] (outside [0, kb): -1 before, INT_MAX after), i <= nh + 1;
    // rI[i] = recv[b0 + i] (INT_MAX past the end), i <= nr.  All loads first.
    constexpr int SU = (MERGE_TILE + 3 + MERGE_THREADS - 1) / MERGE_THREADS;
    int32_t ti[SU];
    float tv[SU];
#pragma unroll
    for (int u = 0; u < SU; ++u) {
      const int i = threadIdx.x + u * MERGE_THREADS;   // position in the combined buffer
      ti[u] = INT32_MAX;
      tv[u] = 0.f;
      if (i <= nh + 1) {
        const int32_t gi = a0 - 1 + i;
        if (gi < 0) ti[u] = -1;
        else if (gi < kb) { ti[u] = Hi[gi]; tv[u] = Hv[gi]; }
      } else if (i <= nh + 2 + nr) {
        const int32_t gj = b0 + (i - nh - 2);
        if (gj < kb) { ti[u] = Ri[gj]; tv[u] = Rv[gj]; }
      }
    }
#pragma unroll
    for (int u = 0; u < SU; ++u) {
      const int i = threadIdx.x + u * MERGE_THREADS;
      if (i <= nh + 2 + nr) {
        cI[i] = ti[u];
        cV[i] = tv[u];
      }
    }
  }
  __syncthreads();
  // held(i) = hI[i - a0 + 1], recv(j) = rI[j - b0]
  int32_t ei[MERGE_PER_THREAD];
  float ev[MERGE_PER_THREAD];
  bool eok[MERGE_PER_THREAD];
  uint32_t cnt = 0;
  const int32_t q_lo = Q0 + (int32_t)threadIdx.x * MERGE_PER_THREAD;
  int32_t a = 0, bb = 0;
  if (q_lo < Q1) {
    int32_t lo = max(a0, a1 - (Q1 - q_lo)), hi = min(a1, a0 + (q_lo - Q0));
    while (lo < hi) {
      const int32_t mid = (lo + hi) >> 1;
      if (hI[mid - a0 + 1] <= rI[q_lo - mid - 1 - b0]) lo = mid + 1;
      else hi = mid;
    }
    a = lo;
    bb = q_lo - a;
  }
#pragma unroll
  for (int k = 0; k < MERGE_PER_THREAD; ++k) {
    eok[k] = false;
    ei[k] = 0;
    ev[k] = 0.f;
    if (q_lo + k < Q1) {
      a = min(a, a1);     // only reachable with unsorted input; keeps LDS reads in range
      bb = min(bb, b1);
      const int32_t hx = hI[a - a0 + 1];
      const int32_t rx = rI[bb - b0];
      if (hx <= rx) {
        float v = hV[a - a0 + 1];
        if (rx == hx) v = v + rV[bb - b0];
        ei[k] = hx;
        ev[k] = v;
        eok[k] = true;
        ++a;
      } else {
        if (hI[a - a0] != rx) {
          ei[k] = rx;
          ev[k] = rV[bb - b0];
          eok[k] = true;
        }
        ++bb;
      }
      if (eok[k]) {
        ++cnt;
        atomicAdd(&hist[mag_key(ev[k]) >> D1_SHIFT], 1u);
      }
    }
  }
  // the scan's barriers put every thread past its merge loop, so the tile is
  // staged in the (now free) input buffer and written out coalesced
  uint32_t tot;
  uint32_t pos = block_excl_scan(cnt, scratch, &tot);
  if (threadIdx.x == 0) slot_cnt[(int64_t)pair * tiles_per_pair + tile] = tot;
#pragma unroll
  for (int k = 0; k < MERGE_PER_THREAD; ++k) {
    if (eok[k]) {
      cI[pos] = ei[k];
      cV[pos] = ev[k];
      ++pos;
    }
  }
  __syncthreads();
  const int64_t ubase = (int64_t)pair * tiles_per_pair * MERGE_TILE + Q0;
  for (uint32_t k = threadIdx.x; k < tot; k += blockDim.x) {
    U_idx[ubase + k] = cI[k];
    U_val[ubase + k] = cV[k];
  }
  flush_hist(hist, hist1 + (int64_t)pair * NB1);
}

// ============================================================================ launchers
hipError_t launch_merge(const int32_t* sp_idx, const float* sp_val, const Pairs& PM, int64_t npairs, int32_t kb,
                        int32_t tiles_per_pair, uint32_t* hist1, uint32_t* slot_cnt, int32_t* U_idx,
                        float* U_val, hipStream_t s) {
  const dim3 grid((unsigned)(npairs * tiles_per_pair));
  hipLaunchKernelGGL(k_merge, grid, dim3(MERGE_THREADS), 0, s, sp_idx, sp_val, PM, kb, tiles_per_pair, hist1, slot_cnt, U_idx, U_val);
  return hipGetLastError();
}

}  // namespace spardl
