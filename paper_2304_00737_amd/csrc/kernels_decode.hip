// All-Gather decode (end of Sec. III-B) and global residual collection
// (Sec. III-C, Algorithm 1; the R-SAG drop shares of Sec. III-D) for gfx950.

#include "device.hpp"
#include "launch.hpp"

#include <algorithm>

namespace spardl {

// ============================================================================ a5: all-gather + densify
// One workgroup per tile [t0, t0 + DENSE_TILE) of the output.  The tile is
// built in LDS as an image -- zeros, then the final entries whose index falls
// in the tile (both ends found by one joint search in the index-sorted final
// blocks sp[b][b], whose loads overlap the image's zeroing) -- and written
// once with whole-line stores, so no line of the output is written twice.
// With `member`, the tile's words of the membership bitmap of the final index
// set I are written as well (bit x & 31 of word x >> 5 set iff x is in I),
// every word of [0, ceil(n/32)) exactly once.
template <int VEC>
__global__ __launch_bounds__(256) void k_densify(const int32_t* __restrict__ sp_idx,
                                                 const float* __restrict__ sp_val, Blocks B,
                                                 int32_t kb, float* __restrict__ dense,
                                                 uint32_t* __restrict__ member) {
  static_assert(DENSE_TILE % 1024 == 0, "whole float4 rounds and bitmap words");
  __shared__ __align__(16) float img[DENSE_TILE];
  __shared__ uint32_t bits[DENSE_TILE / 32];
  __shared__ uint32_t cnt[8];
  const int64_t n = B.n;
  const int64_t t0 = (int64_t)blockIdx.x * DENSE_TILE;
  const int64_t t1 = min(t0 + DENSE_TILE, n);
  for (int i = threadIdx.x; i < DENSE_TILE / 4; i += blockDim.x)
    reinterpret_cast<float4*>(img)[i] = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int i = threadIdx.x; i < DENSE_TILE / 32; i += blockDim.x) bits[i] = 0u;
  const uint32_t blo = B.of((uint32_t)t0), bhi = B.of((uint32_t)(t1 - 1));
  for (uint32_t b = blo; b <= bhi; ++b) {
    const int32_t* Fi = sp_idx + ((int64_t)b * B.P + b) * kb;
    const float* Fv = sp_val + ((int64_t)b * B.P + b) * kb;
    int32_t lo, hi;
    wg_partition_point2(
        0, kb, [&](int32_t p) { return (int64_t)Fi[p] < t0; }, 0, kb,
        [&](int32_t p) { return (int64_t)Fi[p] < t1; }, cnt, &lo, &hi);   // its barriers order the zeroing
    for (int32_t j = lo + (int32_t)threadIdx.x; j < hi; j += blockDim.x) {
      const int64_t r = (int64_t)Fi[j] - t0;
      if (r >= 0 && r < t1 - t0) {
        img[r] = Fv[j];
        atomicOr(&bits[r >> 5], 1u << (r & 31));
      }
    }
  }
  __syncthreads();
  const int64_t len = t1 - t0;
  if (VEC == 4 && len == DENSE_TILE) {
    for (int i = threadIdx.x; i < DENSE_TILE / 4; i += blockDim.x)
      __builtin_nontemporal_store(reinterpret_cast<const f4v*>(img)[i], reinterpret_cast<f4v*>(dense + t0) + i);
  } else {
    for (int i = threadIdx.x; i < len; i += blockDim.x) dense[t0 + i] = img[i];
  }
  if (member) {
    for (int i = threadIdx.x; i < DENSE_TILE / 32 && t0 + 32 * (int64_t)i < t1; i += blockDim.x)
      member[(t0 >> 5) + i] = bits[i];
  }
}

// ============================================================================ a6: residual collection
// Membership bitmap of the final index set I, one bit per index.  The
// workspace keeps it at zero between steps: one thread per final entry sets
// its bit before the residual updates and clears the word afterwards.
__global__ __launch_bounds__(256) void k_bm_mark(const int32_t* __restrict__ sp_idx, uint32_t P, uint32_t n,
                                                 uint32_t kb, uint32_t* __restrict__ bm, int set) {
  const uint32_t per_b = kb;
  for (uint32_t b = blockIdx.y; b < P; b += gridDim.y) {
    const int32_t* __restrict__ F = sp_idx + ((int64_t)b * P + b) * kb;
    for (uint32_t j = blockIdx.x * 256u + threadIdx.x; j < per_b; j += gridDim.x * 256u) {
      const int32_t x = F[j];
      if (x >= 0 && (uint32_t)x < n) {
        if (set) atomicOr(&bm[(uint32_t)x >> 5], 1u << ((uint32_t)x & 31u));
        else bm[(uint32_t)x >> 5] = 0u;
      }
    }
  }
}


// acc[w][x] = 0 where worker w selected x locally and x is a final index.
// Grid: x over the worker's P k_blk local indices, y over workers.
__global__ __launch_bounds__(256) void k_grc_zero(float* __restrict__ acc, int64_t ld_acc, uint32_t nw, uint32_t Q,
                                                  uint32_t n, uint32_t kb, const int32_t* __restrict__ local_idx,
                                                  const uint32_t* __restrict__ bm) {
  const uint32_t per_w = Q * kb;   // <= n < 2^31
  for (uint32_t w = blockIdx.y; w < nw; w += gridDim.y) {
    const int32_t* __restrict__ L = local_idx + (int64_t)w * per_w;
    float* __restrict__ A = acc + (int64_t)w * ld_acc;
    for (uint32_t i = blockIdx.x * 256u + threadIdx.x; i < per_w; i += gridDim.x * 256u) {
      const int32_t x = L[i];
      if (x >= 0 && (uint32_t)x < n && in_final(bm, x)) A[x] = 0.0f;
    }
  }
}

// acc[w][x] += v for the drops (x, v) of one step with x a final index.
// Within one step a worker drops a given index at most once.  Grid: x over a
// pair's drop list, y over pairs (w, t); pair p belongs to worker p / m.
__global__ __launch_bounds__(256) void k_grc_drops(float* __restrict__ acc, int64_t ld_acc, uint32_t n, uint32_t m,
                                                   uint32_t kb, uint32_t npairs,
                                                   const int32_t* __restrict__ drop_idx,
                                                   const float* __restrict__ drop_val,
                                                   const int32_t* __restrict__ drop_cnt,
                                                   const uint32_t* __restrict__ bm) {
  for (uint32_t pair = blockIdx.y; pair < npairs; pair += gridDim.y) {
    const int32_t c = drop_cnt[pair];
    const uint32_t cnt = c < 0 ? 0u : min((uint32_t)c, kb);
    const int32_t* __restrict__ Di = drop_idx + (int64_t)pair * kb;
    const float* __restrict__ Dv = drop_val + (int64_t)pair * kb;
    float* __restrict__ A = acc + (int64_t)(pair / m) * ld_acc;
    for (uint32_t j = blockIdx.x * 256u + threadIdx.x; j < cnt; j += gridDim.x * 256u) {
      const int32_t x = Di[j];
      if (x >= 0 && (uint32_t)x < n && in_final(bm, x)) A[x] = A[x] + Dv[j];
    }
  }
}

// The per-tile index of a fused residual collection: for every pair of the
// call's rows at SRS step i (worker w, bag block t, merging block
// b = (w + t) mod P) and every add tile g of block b with drops, the range
// [first, end) of the pair's drop list inside the tile.  A list is index
// sorted inside its block (an SRS step emits its drops in index order), so
// an entry starts its tile's range if the entry before it lies in another
// tile, and ends it if the entry after it does.  Tiles without drops keep
// the (0, 0) the caller cleared them to.  Grid: x over a list, y over the
// (step, pair) lists of the call's rows.
constexpr int DT_PER = 4;   // list entries per thread of the index build

struct DropTiles {
  AddCollect C;
  const int32_t* cnt[COLLECT_MAX_STEPS];
  uint32_t pcum[COLLECT_MAX_STEPS + 1];   // lists of the call's rows before step i
  uint32_t nw;
};

__global__ __launch_bounds__(256) void k_drop_tiles(DropTiles D, Blocks B, uint32_t* __restrict__ err) {
  const AddCollect& C = D.C;
  for (uint32_t y = blockIdx.y; y < D.pcum[C.l]; y += gridDim.y) {
    int i = 0;
    while (y >= D.pcum[i + 1]) ++i;
    const uint32_t m = C.m[i];
    const uint32_t q = y - D.pcum[i];
    const uint32_t w = C.w0 + q / m, tt = q - (q / m) * m;
    const uint32_t b = (w + tt) % B.P;
    const int64_t p = (int64_t)w * m + tt;
    const int32_t c = D.cnt[i][p];
    const uint32_t cnt = c < 0 ? 0u : min((uint32_t)c, C.kb);
    const int32_t* __restrict__ X = C.didx[i] + p * C.kb;
    uint2* __restrict__ T = const_cast<uint2*>(C.tile[i]) + p * C.G;
    const uint32_t s = B.start(b), e = B.start(b + 1u), o = block_origin(s);
    // DT_PER consecutive entries per thread, with the entries on either side
    for (uint32_t j0 = (blockIdx.x * 256u + threadIdx.x) * DT_PER; j0 < cnt; j0 += gridDim.x * 256u * DT_PER) {
      uint32_t xs[DT_PER + 2];
#pragma unroll
      for (int u = 0; u < DT_PER + 2; ++u) {
        const uint32_t j = j0 + (uint32_t)u - 1u;   // j0 - 1 wraps for j0 = 0 and fails the test
        xs[u] = j < cnt ? (uint32_t)X[j] : 0u;
      }
#pragma unroll
      for (int u = 1; u <= DT_PER; ++u) {
        const uint32_t j = j0 + (uint32_t)u - 1u;
        if (j >= cnt) break;
        const uint32_t x = xs[u];
        if (x < s || x >= e || (j > 0u && xs[u - 1] >= x)) {
          atomicOr(err, ERR_DROPS);
          continue;
        }
        const uint32_t t = (x - o) / (uint32_t)ADD_TILE;
        const bool first = j == 0u || (xs[u - 1] - o) / (uint32_t)ADD_TILE != t;
        const bool last = j + 1u == cnt || (xs[u + 1] - o) / (uint32_t)ADD_TILE != t;
        if (first) T[t].x = j;
        if (last) T[t].y = j + 1u;
      }
    }
  }
}

// acc[w][x] += share * v for the drops (x, v) of R-SAG exchange t with x a
// final index, on both workers of each pair (they made the same merge;
// share = 2^-(t+1), the product exact unless it is subnormal).  Grid: x over
// a pair's drop list, y over pairs, numbered as in the exchange.
__global__ __launch_bounds__(256) void k_grc_sag_drops(float* __restrict__ acc, int64_t ld_acc, uint32_t n,
                                                       uint32_t Q, uint32_t t, uint32_t kb, uint32_t npairs,
                                                       const int32_t* __restrict__ drop_idx,
                                                       const float* __restrict__ drop_val,
                                                       const int32_t* __restrict__ drop_cnt,
                                                       const uint32_t* __restrict__ bm, float share) {
  for (uint32_t pair = blockIdx.y; pair < npairs; pair += gridDim.y) {
    const int32_t c = drop_cnt[pair];
    const uint32_t cnt = c < 0 ? 0u : min((uint32_t)c, kb);
    const uint32_t j = pair / Q, q = pair - j * Q;
    const uint32_t lowmask = (1u << t) - 1u;
    const uint32_t X = ((j & ~lowmask) << 1) | (j & lowmask), Y = X | (1u << t);
    const int32_t* __restrict__ Di = drop_idx + (int64_t)pair * kb;
    const float* __restrict__ Dv = drop_val + (int64_t)pair * kb;
    float* __restrict__ AX = acc + (int64_t)(X * Q + q) * ld_acc;
    float* __restrict__ AY = acc + (int64_t)(Y * Q + q) * ld_acc;
    for (uint32_t j2 = blockIdx.x * 256u + threadIdx.x; j2 < cnt; j2 += gridDim.x * 256u) {
      const int32_t x = Di[j2];
      if (x >= 0 && (uint32_t)x < n && in_final(bm, x)) {
        const float v = Dv[j2] * share;
        AX[x] = AX[x] + v;
        AY[x] = AY[x] + v;
      }
    }
  }
}

// ============================================================================ launchers
hipError_t launch_densify(const int32_t* sp_idx, const float* sp_val, int32_t P, int64_t n, int32_t kb,
                          float* dense, uint32_t* member, bool vec4, hipStream_t s) {
  const dim3 grid((unsigned)((n + DENSE_TILE - 1) / DENSE_TILE));
  const Blocks B = make_blocks(n, P);
  if (vec4) hipLaunchKernelGGL(k_densify<4>, grid, dim3(256), 0, s, sp_idx, sp_val, B, kb, dense, member);
  else hipLaunchKernelGGL(k_densify<1>, grid, dim3(256), 0, s, sp_idx, sp_val, B, kb, dense, member);
  return hipGetLastError();
}

hipError_t launch_bm_mark(const int32_t* sp_idx, int32_t P, int64_t n, int32_t kb, uint32_t* bm, bool set,
                          hipStream_t s) {
  const dim3 grid(grid_for(kb, 256, 1024), (unsigned)std::min<int32_t>(P, 65535));
  hipLaunchKernelGGL(k_bm_mark, grid, dim3(256), 0, s, sp_idx, (uint32_t)P, (uint32_t)n, (uint32_t)kb, bm, set ? 1 : 0);
  return hipGetLastError();
}

hipError_t launch_grc_zero(float* acc, int64_t ld_acc, int32_t nw, int32_t Q, int64_t n, int32_t kb,
                           const int32_t* local_idx, const uint32_t* bm, hipStream_t s) {
  const dim3 grid(grid_for((int64_t)Q * kb, 256, 1024), (unsigned)std::min<int32_t>(nw, 65535));
  hipLaunchKernelGGL(k_grc_zero, grid, dim3(256), 0, s, acc, ld_acc, (uint32_t)nw, (uint32_t)Q, (uint32_t)n,
                     (uint32_t)kb, local_idx, bm);
  return hipGetLastError();
}

hipError_t launch_grc_drops(float* acc, int64_t ld_acc, int64_t n, int32_t m, int32_t kb, int32_t npairs,
                            const int32_t* drop_idx, const float* drop_val, const int32_t* drop_cnt,
                            const uint32_t* bm, hipStream_t s) {
  const dim3 grid(grid_for(kb, 256, 1024), (unsigned)std::min<int32_t>(npairs, 65535));
  hipLaunchKernelGGL(k_grc_drops, grid, dim3(256), 0, s, acc, ld_acc, (uint32_t)n, (uint32_t)m, (uint32_t)kb, (uint32_t)npairs, drop_idx, drop_val, drop_cnt, bm);
  return hipGetLastError();
}

hipError_t launch_drop_tiles(const AddCollect& C, const int32_t* const* drop_cnt, int32_t nw, int64_t n, int32_t P,
                             uint32_t* err, hipStream_t s) {
  if (C.l <= 0) return hipSuccess;
  if (C.l > COLLECT_MAX_STEPS) return hipErrorInvalidValue;
  DropTiles D;
  D.C = C;
  D.nw = (uint32_t)nw;
  D.pcum[0] = 0u;
  for (int i = 0; i < C.l; ++i) {
    D.cnt[i] = drop_cnt[i];
    D.pcum[i + 1] = D.pcum[i] + (uint32_t)nw * C.m[i];
  }
  const dim3 grid(grid_for(((int64_t)C.kb + DT_PER - 1) / DT_PER, 256, 1024), (unsigned)std::min<uint32_t>(D.pcum[C.l], 65535u));
  hipLaunchKernelGGL(k_drop_tiles, grid, dim3(256), 0, s, D, make_blocks(n, P), err);
  return hipGetLastError();
}

hipError_t launch_grc_sag_drops(float* acc, int64_t ld_acc, int64_t n, int32_t Q, int32_t t, int32_t kb,
                                int32_t npairs, const int32_t* drop_idx, const float* drop_val,
                                const int32_t* drop_cnt, const uint32_t* bm, hipStream_t s) {
  const dim3 grid(grid_for(kb, 256, 1024), (unsigned)std::min<int32_t>(npairs, 65535));
  hipLaunchKernelGGL(k_grc_sag_drops, grid, dim3(256), 0, s, acc, ld_acc, (uint32_t)n, (uint32_t)Q, (uint32_t)t,
                     (uint32_t)kb, (uint32_t)npairs, drop_idx, drop_val, drop_cnt, bm, 1.0f / (float)(2 << t));
  return hipGetLastError();
}

}  // namespace spardl
