// Residual add of the SparDL per-worker hot path for gfx950 (CDNA4, wave64):
// A = G + xi (Sec. III-B, Algorithm 1), fused with the level-1 histogram and
// the speculative candidates of the block top-k that follows; the level-1
// histogram alone for selections without a fused add; the workspace fill.

#include "device.hpp"
#include "launch.hpp"

#include <algorithm>

namespace spardl {

// ============================================================================ fill
// Zero up to FILL_MAX word ranges in one launch (counters, histograms and
// look-back status words are cleared this way; no memset nodes are used).
__global__ __launch_bounds__(256) void k_fill(FillRanges r) {
  int64_t total = 0;
  for (int k = 0; k < r.count; ++k) total += r.len[k];
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
    int64_t j = i;
    int k = 0;
    while (j >= r.len[k]) {
      j -= r.len[k];
      ++k;
    }
    r.ptr[k][j] = 0u;
  }
}

// ============================================================================ a1: residual add
// One workgroup = one tile of ADD_TILE elements of one block of one row.
// With HIST, every sum's level-1 digit is counted in an LDS histogram that is
// flushed (non-zero bins only) into the block's global one.  The gradient is
// read once, so it is loaded non-temporally.
//
// The float4 path with HIST also writes speculative candidates for the block
// top-k that follows: every sum whose key is at or above a floor two level-1
// bins below the block's previous threshold bin (nothing on a block's first
// step), in index order at the tile's own span of the candidate arrays, with
// the count per tile.  The exact threshold bin found from this pass's
// histogram decides whether the floor was low enough; if not, the top-k reads
// the block again.  Thread t owns the 8 consecutive elements at 8 t.
//
// From a block's second step on, the histogram counts only keys at or above
// a lower floor (two binades further down): the threshold lies there unless it
// fell by more than that since the previous step, and then the level-1 select
// rebuilds the block's full histogram itself.
constexpr int ADD_STAGE = 512;          // speculative candidates staged in LDS per tile


template <int VEC, bool HIST>
__global__ __launch_bounds__(256) void k_residual_add(float* __restrict__ acc, int64_t ld_acc,
                                                      const float* __restrict__ grad, int64_t ld_grad,
                                                      Blocks B, uint32_t G, AddSpec sp) {
  constexpr bool SPEC = HIST && VEC == 4;
  __shared__ __align__(16) uint32_t h[HIST ? NB1 : 4];
  __shared__ int32_t s_idx[SPEC ? ADD_STAGE : 1];
  __shared__ float s_val[SPEC ? ADD_STAGE : 1];
  __shared__ uint32_t wtot[4];
  const uint32_t g = blockIdx.x % G;
  const uint32_t wb = blockIdx.x / G;
  const uint32_t b = wb % B.P, w = wb / B.P;
  const uint32_t s = B.start(b), e = B.start(b + 1u);
  const uint32_t t0 = s + g * (uint32_t)ADD_TILE;
  if (t0 >= e) return;
  if (HIST) {
    for (int i = threadIdx.x; i < NB1 / 4; i += 256) reinterpret_cast<uint4*>(h)[i] = make_uint4(0u, 0u, 0u, 0u);
    __syncthreads();
  }
  float* __restrict__ A = acc + (int64_t)w * ld_acc;
  const float* __restrict__ Gr = grad + (int64_t)w * ld_grad;
  if (VEC == 4) {
    static_assert(ADD_TILE == 256 * 8, "eight elements per thread");
    const uint32_t my0 = t0 + threadIdx.x * 8u;
    f4v a[2], gg[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      if (my0 + 4u * j < e) {
        a[j] = *reinterpret_cast<const f4v*>(A + my0 + 4u * j);
        gg[j] = __builtin_nontemporal_load(reinterpret_cast<const f4v*>(Gr + my0 + 4u * j));
      }
    }
    uint32_t F = SPEC_NONE;
    if (SPEC) {
      const uint32_t sw = sp.spec_t1[wb];
      if (sw != 0u) {
        const uint32_t T1p = sw - 1u;
        F = T1p > SPEC_MARGIN ? (T1p - SPEC_MARGIN) << D1_SHIFT : 0u;
      }
      if (g == 0u && threadIdx.x == 0) sp.spec_used[wb] = F;
    }
    const uint32_t FH = hist_floor(F);
    float r[8];
    uint32_t nc = 0;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      if (my0 + 4u * j < e) {
        f4v q;
        q.x = a[j].x + gg[j].x;
        q.y = a[j].y + gg[j].y;
        q.z = a[j].z + gg[j].z;
        q.w = a[j].w + gg[j].w;
        __builtin_nontemporal_store(q, reinterpret_cast<f4v*>(A + my0 + 4u * j));   // re-read only next step
        r[4 * j + 0] = q.x;
        r[4 * j + 1] = q.y;
        r[4 * j + 2] = q.z;
        r[4 * j + 3] = q.w;
        if (HIST) {
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            const uint32_t key = mag_key(r[4 * j + c]);
            if (key >= FH) atomicAdd(&h[key >> D1_SHIFT], 1u);
            nc += key >= F ? 1u : 0u;
          }
        }
      } else {
#pragma unroll
        for (int c = 0; c < 4; ++c) r[4 * j + c] = 0.f;
      }
    }
    if (SPEC) {
      // index-ordered compaction of the candidates (keys >= F) of the tile
      const int lane = lane_id(), wv = wave_id();
      const uint32_t incl = wave_incl_scan(nc);
      if (lane == WAVE - 1) wtot[wv] = incl;
      __syncthreads();
      uint32_t base = 0, tot = 0;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const uint32_t x = wtot[k];
        base += k < wv ? x : 0u;
        tot += x;
      }
      const bool staged = tot <= (uint32_t)ADD_STAGE;   // uniform
      int32_t* __restrict__ CI = sp.cand_idx + (int64_t)w * B.n + t0;
      float* __restrict__ CV = sp.cand_val + (int64_t)w * B.n + t0;
      int32_t* __restrict__ oI = staged ? s_idx : CI;
      float* __restrict__ oV = staged ? s_val : CV;
      uint32_t pos = base + incl - nc;
      if (nc != 0u) {
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          if (my0 + (uint32_t)k < e && mag_key(r[k]) >= F) {
            oI[pos] = (int32_t)(my0 + k);
            oV[pos] = r[k];
            ++pos;
          }
        }
      }
      if (threadIdx.x == 0) sp.spec_cnt[(int64_t)wb * G + g] = tot;
      if (staged) {
        __syncthreads();
        for (uint32_t k = threadIdx.x; k < tot; k += 256) {
          CI[k] = s_idx[k];
          CV[k] = s_val[k];
        }
      }
    }
  } else {
#pragma unroll
    for (int j = 0; j < ADD_F4 * 4; ++j) {
      const uint32_t off = t0 + j * 256u + threadIdx.x;
      if (off < e) {
        const float r = A[off] + Gr[off];
        A[off] = r;
        if (HIST) atomicAdd(&h[mag_key(r) >> D1_SHIFT], 1u);
      }
    }
    if (HIST && g == 0u && threadIdx.x == 0) sp.spec_used[wb] = SPEC_NONE;   // no candidates on this path
  }
  if (HIST) {
    __syncthreads();
    uint32_t* __restrict__ H = sp.hist1 + ((int64_t)wb * HCOPIES + blockIdx.x % HCOPIES) * NB1;
    flush_hist(h, H);
  }
}

// Level-1 histogram only (block_topk without a fused residual add).
template <int VEC>
__global__ __launch_bounds__(256) void k_hist1(const float* __restrict__ acc, int64_t ld_acc, Blocks B, Units U,
                                               uint32_t G, uint32_t* __restrict__ hist1) {
  __shared__ __align__(16) uint32_t h[NB1];
  const uint32_t g = blockIdx.x % G;
  uint32_t w, b;
  U.decode(blockIdx.x / G, B.P, &w, &b);
  const uint32_t wb = w * B.P + b;   // the block's histogram
  const uint32_t s = B.start(b), e = B.start(b + 1u);
  const uint32_t t0 = s + g * (uint32_t)ADD_TILE;
  if (t0 >= e) return;
  for (int i = threadIdx.x; i < NB1 / 4; i += 256) reinterpret_cast<uint4*>(h)[i] = make_uint4(0u, 0u, 0u, 0u);
  __syncthreads();
  const float* __restrict__ A = acc + (int64_t)w * ld_acc;
  if (VEC == 4) {
#pragma unroll
    for (int j = 0; j < ADD_F4; ++j) {
      const uint32_t off = t0 + (j * 256u + threadIdx.x) * 4u;
      if (off < e) {
        const f4v a = *reinterpret_cast<const f4v*>(A + off);
        atomicAdd(&h[mag_key(a.x) >> D1_SHIFT], 1u);
        atomicAdd(&h[mag_key(a.y) >> D1_SHIFT], 1u);
        atomicAdd(&h[mag_key(a.z) >> D1_SHIFT], 1u);
        atomicAdd(&h[mag_key(a.w) >> D1_SHIFT], 1u);
      }
    }
  } else {
#pragma unroll
    for (int j = 0; j < ADD_F4 * 4; ++j) {
      const uint32_t off = t0 + j * 256u + threadIdx.x;
      if (off < e) atomicAdd(&h[mag_key(A[off]) >> D1_SHIFT], 1u);
    }
  }
  __syncthreads();
  uint32_t* __restrict__ H = hist1 + ((int64_t)wb * HCOPIES + blockIdx.x % HCOPIES) * NB1;
  flush_hist(h, H);
}

// ============================================================================ launchers
hipError_t launch_fill(const FillRanges& r, hipStream_t s) {
  int64_t total = 0;
  for (int k = 0; k < r.count; ++k) total += r.len[k];
  if (total <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_fill, dim3(grid_for(total, 256, 4096)), dim3(256), 0, s, r);
  return hipGetLastError();
}

hipError_t launch_residual_add(float* acc, int64_t ld_acc, const float* grad, int64_t ld_grad,
                               int32_t nworkers, int64_t n, int32_t P, bool vec4, const AddSpec& sp,
                               hipStream_t s) {
  const bool hist = sp.hist1 != nullptr;
  const int32_t PP = hist ? P : 1;
  const int64_t maxlen = (n + PP - 1) / PP;
  const int32_t G = (int32_t)((maxlen + ADD_TILE - 1) / ADD_TILE);
  const dim3 grid((unsigned)((int64_t)nworkers * PP * G));
  const Blocks B = make_blocks(n, PP);
  const uint32_t uG = (uint32_t)G;
  if (hist) {
    if (vec4) hipLaunchKernelGGL((k_residual_add<4, true>), grid, dim3(256), 0, s, acc, ld_acc, grad, ld_grad, B, uG, sp);
    else hipLaunchKernelGGL((k_residual_add<1, true>), grid, dim3(256), 0, s, acc, ld_acc, grad, ld_grad, B, uG, sp);
  } else {
    if (vec4) hipLaunchKernelGGL((k_residual_add<4, false>), grid, dim3(256), 0, s, acc, ld_acc, grad, ld_grad, B, uG, sp);
    else hipLaunchKernelGGL((k_residual_add<1, false>), grid, dim3(256), 0, s, acc, ld_acc, grad, ld_grad, B, uG, sp);
  }
  return hipGetLastError();
}

hipError_t launch_hist1(const float* acc, int64_t ld_acc, int64_t nunits, const Units& U, int64_t n, int32_t P,
                        bool vec4, uint32_t* hist1, hipStream_t s) {
  const int64_t maxlen = (n + P - 1) / P;
  const int32_t G = (int32_t)((maxlen + ADD_TILE - 1) / ADD_TILE);
  const dim3 grid((unsigned)(nunits * G));
  const Blocks B = make_blocks(n, P);
  if (vec4) hipLaunchKernelGGL(k_hist1<4>, grid, dim3(256), 0, s, acc, ld_acc, B, U, (uint32_t)G, hist1);
  else hipLaunchKernelGGL(k_hist1<1>, grid, dim3(256), 0, s, acc, ld_acc, B, U, (uint32_t)G, hist1);
  return hipGetLastError();
}

}  // namespace spardl
