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

// A relaxed atomic load: an ordinary load to the hardware, which the compiler
// keeps where it is written relative to a compiler fence (no wait follows it).
template <typename T>
__device__ __forceinline__ T early_load(const T* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ============================================================================ a1: residual add
// Tiles of ADD_TILE elements start at the block's aligned origin (its start
// rounded down to 32 elements), so every tile after a block's first begins on
// a 128-byte boundary of the row; tile g of block b is
// [origin + g ADD_TILE, origin + (g+1) ADD_TILE) clipped to the block.
// One workgroup per tile; chunk j of the tile is the 1024 elements at
// 1024 j, thread t holding elements 4t .. 4t+3 of each chunk, so each wave's
// float4 access covers 1 KB of whole lines.  The gradient is read once, so it
// is loaded non-temporally; A is re-read only by a fallback, so it is stored
// non-temporally.
//
// With HIST, every sum's level-1 bin (L1Map in device.hpp) is counted in an
// LDS histogram that is flushed (non-zero bins only) into one of the block's
// global copies, and the
// speculative candidates of the block top-k that follows are written: every
// sum whose key is at or above a floor two level-1 bins below the block's
// previous threshold bin (nothing on a block's first step), in index order at
// the tile's own span of the candidate arrays, with the count per tile.  The
// run is staged in LDS and written as whole 128-byte lines (padded past the
// count inside the tile's span, non-temporal): small partial-line writes
// into the candidate arrays cost far more than their bytes.  The exact
// threshold bin found from this pass's histogram decides whether the floor
// was low enough; if not, the top-k reads the block again.
//
// From a block's second step on, the histogram counts only keys at or above
// a lower floor (two binades further down): the threshold lies there unless it
// fell by more than that since the previous step, and then the level-1 select
// rebuilds the block's full histogram itself.  The previous threshold is the
// larger of the worker's own from its previous step and the same block's
// latest at the preceding worker.
//
// With COLL, the previous step's global residual collection (Sec. III-C) is
// applied to the tile before the gradient is added, in the order of the
// separate collection: the worker's own selections that became final are
// zeroed -- the block top-k's rule (KEEP_WORDS) recomputed on the values it
// selected from, which nothing changed since -- and then, SRS step by step,
// its final drops are added back.  The drops of one step are distinct
// indices, so a step's additions run in parallel on an LDS image of the tile.
// The separate collection's scattered writes leave a partly written line in
// the caches for every index they touch, which the next add's stream then
// writes back; here every line of acc is written once, whole.
constexpr int ADD_STAGE = 512;          // speculative candidates (or drops) staged in LDS per tile

template <bool HIST, bool COLL>
__global__ __launch_bounds__(256) void k_residual_add4(float* __restrict__ acc, int64_t ld_acc,
                                                       const float* __restrict__ grad, int64_t ld_grad, Blocks B,
                                                       uint32_t G, AddSpec sp, AddCollect C) {
  static_assert(ADD_TILE == 2 * 1024, "two 1024-element chunks per tile");
  static_assert(!COLL || HIST, "the fused collection runs in the fused add");
  __shared__ __align__(16) uint32_t h[HIST ? NB1 : 4];
  __shared__ int32_t s_idx[HIST ? ADD_STAGE : 1];
  __shared__ float s_val[HIST ? ADD_STAGE : 1];
  __shared__ uint32_t wtot[4];
  // COLL: the tile image (in the histogram's space: each thread clears its
  // words of it again after the collection), the tile's final-index bitmap
  // words, and per SRS step the range of the worker's drops inside the tile
  // with their arrays
  static_assert(NB1 >= ADD_TILE, "the tile image fits in the histogram's space");
  float* cimg = reinterpret_cast<float*>(h);
  __shared__ uint32_t cmw[COLL ? ADD_TILE / 32 : 1];
  __shared__ uint32_t c_lo[COLL ? COLLECT_MAX_STEPS : 1], c_hi[COLL ? COLLECT_MAX_STEPS : 1];
  __shared__ uint32_t c_cum[COLL ? COLLECT_MAX_STEPS + 1 : 1];
  __shared__ const int32_t* c_di[COLL ? COLLECT_MAX_STEPS : 1];
  __shared__ const float* c_dv[COLL ? COLLECT_MAX_STEPS : 1];
  // grid: x = tile of the block, y = block, z = row (no division decodes it)
  const uint32_t g = blockIdx.x;
  const uint32_t b = blockIdx.y, w = blockIdx.z;
  const uint32_t wb = w * B.P + b;
  const uint32_t s = B.start(b), e = B.start(b + 1u);
  const uint32_t ta = block_origin(s) + g * (uint32_t)ADD_TILE;
  if (ta >= e) return;
  float* __restrict__ A = acc + (int64_t)w * ld_acc;
  const float* __restrict__ Gr = grad + (int64_t)w * ld_grad;
  const uint32_t x0 = ta + threadIdx.x * 4u;
  // The workgroup's own words are loaded before the tile's stream: a wave's
  // loads complete in order, so a word loaded after the stream could only be
  // used once the whole stream had arrived.  HIST: the previous threshold
  // hints (every wave); COLL: the drop-tile ranges of the SRS steps (thread
  // 0; steps past RR_EARLY, only for P > 256, are loaded later).  They are
  // relaxed atomic loads behind a compiler-only fence, which the compiler
  // neither sinks below the stream nor waits for at once.
  const uint32_t wa = C.w0 + w;   // COLL: the absolute worker
  const uint32_t tt = (b + B.P - wa % B.P) % B.P;   // COLL: this block's place in the worker's bags
  constexpr int RR_EARLY = 8;
  uint2 rr[RR_EARLY];
  int32_t rc[RR_EARLY];   // COLL: the pair's drop count of each step
  if constexpr (COLL) {
    if (threadIdx.x == 0) {
#pragma unroll
      for (int i = 0; i < RR_EARLY; ++i) {
        rr[i] = make_uint2(0u, 0u);
        rc[i] = 0;
        if (i < C.l && tt < C.m[i]) {
          const int64_t p = (int64_t)wa * C.m[i] + tt;
          const uint64_t v = early_load(reinterpret_cast<const uint64_t*>(C.tile[i] + p * C.G + g));
          rr[i] = make_uint2((uint32_t)v, (uint32_t)(v >> 32));
          rc[i] = early_load(C.dcnt[i] + p);
        }
      }
    }
  }
  uint32_t sw = 0u, pw = 0u;
  if constexpr (HIST) {
    // a zero the compiler cannot see through keeps the hints in vector
    // registers (a uniform value would be moved to a scalar one at once,
    // which waits for the load)
    uint32_t z;
    asm volatile("v_mov_b32 %0, 0" : "=v"(z));
    sw = early_load(sp.spec_t1 + wb + z);
    // the same block's latest hint at the preceding worker: when workers run a few at
    // a time it is this step's, a closer estimate while the residual is still growing
    // (a threshold from the step before can lie several bins lower then); the larger
    // of the two is used (without that hint, the worker's own again)
    const uint32_t* pa = !sp.spec_prev ? sp.spec_t1 + wb : w == 0u ? sp.spec_prev + b : sp.spec_t1 + (wb - B.P);
    pw = early_load(pa + z);
  }
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
  // block starts and ends are multiples of 4 here, so a float4 lies wholly
  // inside or outside the block; one outside loads the block's first float4
  // instead (unused), so that the loads need no branch
  bool in[2];
  f4v a[2], gg[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const uint32_t x = x0 + 1024u * j;
    in[j] = x >= s && x < e;
    const uint32_t xl = in[j] ? x : s;
    a[j] = *reinterpret_cast<const f4v*>(A + xl);
    gg[j] = __builtin_nontemporal_load(reinterpret_cast<const f4v*>(Gr + xl));
  }
  // COLL: the final-index bitmap words of this thread's two float4 (the four
  // elements share a word: tiles start on 32-element boundaries)
  uint32_t mw[2] = {0u, 0u};
  uint32_t k_tge = 0, k_teq = 0, k_need = 0, k_cut = 0;   // COLL: the block top-k's selection rule
  if constexpr (COLL) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const uint32_t x = x0 + 1024u * j;
      if (x < B.n) mw[j] = C.member[x >> 5];
    }
    const uint32_t* __restrict__ kp = C.keep + ((int64_t)(C.w0 + w) * B.P + b) * KEEP_WORDS;
    k_tge = kp[KEEP_TGE];
    k_teq = kp[KEEP_TEQ];
    k_need = kp[KEEP_NEEDEQ];
    k_cut = kp[KEEP_CUT];
  }
  if (!HIST) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      if (in[j]) {
        f4v q;
        q.x = a[j].x + gg[j].x;
        q.y = a[j].y + gg[j].y;
        q.z = a[j].z + gg[j].z;
        q.w = a[j].w + gg[j].w;
        __builtin_nontemporal_store(q, reinterpret_cast<f4v*>(A + x0 + 1024u * j));
      }
    }
    return;
  }
  // the histogram is cleared while the loads are in flight (with COLL, a tile
  // with drops clears its image's words again after the collection)
  for (int i = threadIdx.x; i < NB1 / 4; i += 256) reinterpret_cast<uint4*>(h)[i] = make_uint4(0u, 0u, 0u, 0u);
  uint32_t F = SPEC_NONE;
  sw = max(sw, pw);
  if (sw != 0u) {
    const uint32_t T1p = sw - 1u;
    F = T1p > SPEC_MARGIN ? (T1p - SPEC_MARGIN) << D1_SHIFT : 0u;
  }
  if (g == 0u && threadIdx.x == 0) sp.spec_used[wb] = F;
  const L1Map M = l1_map(F);
  const uint32_t FH = M.floor;
  if constexpr (COLL) {
    // one thread turns the ranges into the tile's drop runs
    if (threadIdx.x == 0) {
      uint32_t cum = 0;
#pragma unroll
      for (int i = 0; i < COLLECT_MAX_STEPS; ++i) {
        if (i < C.l) {
          uint2 ri = make_uint2(0u, 0u);
          int32_t ci = 0;
          if (i < RR_EARLY) {
            ri = rr[i];
            ci = rc[i];
          } else if (tt < C.m[i]) {
            const int64_t p = (int64_t)wa * C.m[i] + tt;
            ri = C.tile[i][p * C.G + g];
            ci = C.dcnt[i][p];
          }
          // a tile without drops this step may hold an older range: within
          // this step's count its entries lie in other tiles and are skipped
          const uint32_t cap = min((uint32_t)max(ci, 0), C.kb);
          const uint32_t lo = min(ri.x, cap), hi = min(max(ri.y, lo), cap);
          if (hi > lo) {
            const int64_t p = (int64_t)wa * C.m[i] + tt;
            c_di[i] = C.didx[i] + p * C.kb;
            c_dv[i] = C.dval[i] + p * C.kb;
          }
          c_lo[i] = lo;
          c_hi[i] = hi;
          c_cum[i] = cum;
          cum += hi - lo;
        }
      }
      c_cum[C.l] = cum;
    }
  }
  __syncthreads();
  if constexpr (COLL) {
    // the worker's selections of this block that became final -> 0
    const uint32_t tge = k_tge, teq = k_teq, need_eq = k_need, xcut = k_cut;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      if (in[j]) {
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const uint32_t x = x0 + 1024u * j + (uint32_t)c;
          const uint32_t key = mag_key(a[j][c]);
          const bool sel = key >= tge || (need_eq != 0u && key == teq && x <= xcut);
          if (sel && ((mw[j] >> (x & 31u)) & 1u)) a[j][c] = 0.0f;
        }
      }
    }
    const uint32_t ndrop = c_cum[C.l];   // uniform
    if (ndrop != 0u) {
      // the final drops of SRS steps 1..l, in order, on the tile image
#pragma unroll
      for (int j = 0; j < 2; ++j)
        if (in[j]) *reinterpret_cast<f4v*>(cimg + threadIdx.x * 4u + 1024u * j) = a[j];
      if ((threadIdx.x & 7u) == 0u) {
        cmw[threadIdx.x >> 3] = mw[0];
        cmw[32u + (threadIdx.x >> 3)] = mw[1];
      }
      const bool staged = ndrop <= (uint32_t)ADD_STAGE;   // uniform: every step's drops in one round of loads
      if (staged) {
        for (uint32_t f = threadIdx.x; f < ndrop; f += 256u) {
          int i = 0;
          while (f >= c_cum[i + 1]) ++i;
          const uint32_t jj = c_lo[i] + (f - c_cum[i]);
          s_idx[f] = c_di[i][jj];
          s_val[f] = c_dv[i][jj];
        }
      }
      __syncthreads();
      for (int i = 0; i < C.l; ++i) {
        const uint32_t lo = c_lo[i], hi = c_hi[i];
        if (hi == lo) continue;   // uniform
        for (uint32_t jj = lo + threadIdx.x; jj < hi; jj += 256u) {
          const uint32_t f = c_cum[i] + (jj - lo);
          const int32_t x = staged ? s_idx[f] : c_di[i][jj];
          const float v = staged ? s_val[f] : c_dv[i][jj];
          const uint32_t o = (uint32_t)x - ta;
          if (o < (uint32_t)ADD_TILE && (uint32_t)x >= s && (uint32_t)x < e && ((cmw[o >> 5] >> (o & 31u)) & 1u))
            cimg[o] = cimg[o] + v;
        }
        __syncthreads();
      }
      // each thread reads back its own words of the image and clears them for the
      // histogram; the barrier orders every clear before any histogram update
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        f4v* q = reinterpret_cast<f4v*>(cimg + threadIdx.x * 4u + 1024u * j);
        if (in[j]) a[j] = *q;
        *q = f4v{0.f, 0.f, 0.f, 0.f};
      }
      __syncthreads();
    }
  }
  float r[8];
  uint32_t packed = 0;   // candidates of chunk 0 | chunk 1 << 16 (at most 1024 each)
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    if (in[j]) {
      f4v q;
      q.x = a[j].x + gg[j].x;
      q.y = a[j].y + gg[j].y;
      q.z = a[j].z + gg[j].z;
      q.w = a[j].w + gg[j].w;
      __builtin_nontemporal_store(q, reinterpret_cast<f4v*>(A + x0 + 1024u * j));
      r[4 * j + 0] = q.x;
      r[4 * j + 1] = q.y;
      r[4 * j + 2] = q.z;
      r[4 * j + 3] = q.w;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const uint32_t key = mag_key(r[4 * j + c]);
        if (key >= FH) atomicAdd(&h[M.bin(key)], 1u);
        packed += key >= F ? (1u << (16 * j)) : 0u;
      }
    } else {
#pragma unroll
      for (int c = 0; c < 4; ++c) r[4 * j + c] = 0.f;
    }
  }
  // index-ordered compaction of the tile's candidates (keys >= F): chunk 0, then chunk 1
  const int lane = lane_id(), wv = wave_id();
  const uint32_t incl = wave_incl_scan(packed);
  if (lane == WAVE - 1) wtot[wv] = incl;
  __syncthreads();   // also ends the histogram's updates
  uint32_t base = 0, tot = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const uint32_t x = wtot[k];
    base += k < wv ? x : 0u;
    tot += x;
  }
  {
    uint32_t* __restrict__ H = sp.hist1 + ((int64_t)wb * sp.hcopies + (g & (sp.hcopies - 1u))) * NB1;   // a power of 2
    flush_hist<256>(h, H);
  }
  const uint32_t tot0 = tot & 0xFFFFu, all = tot0 + (tot >> 16);
  const uint32_t ex = base + incl - packed;
  const uint32_t t0 = ta > s ? ta : s;   // the tile's first element: its candidate run starts there
  const bool staged = all <= (uint32_t)ADD_STAGE;   // uniform
  int32_t* __restrict__ CI = sp.cand_idx + (int64_t)w * B.n + t0;
  float* __restrict__ CV = sp.cand_val + (int64_t)w * B.n + t0;
  int32_t* __restrict__ oI = staged ? s_idx : CI;
  float* __restrict__ oV = staged ? s_val : CV;
  if (packed != 0u) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      uint32_t pos = j == 0 ? (ex & 0xFFFFu) : tot0 + (ex >> 16);
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        if (in[j] && mag_key(r[4 * j + c]) >= F) {
          oI[pos] = (int32_t)(x0 + 1024u * j + (uint32_t)c);
          oV[pos] = r[4 * j + c];
          ++pos;
        }
      }
    }
  }
  if (threadIdx.x == 0) sp.spec_cnt[(int64_t)wb * G + g] = all;
  if (staged) {
    __syncthreads();
    // whole lines: pad the run to a multiple of 32 entries, inside the tile's span
    const uint32_t span = min(e, ta + (uint32_t)ADD_TILE) - t0;
    const uint32_t padded = min((all + 31u) & ~31u, span);
    for (uint32_t k = threadIdx.x; k < padded; k += 256) {
      __builtin_nontemporal_store(s_idx[k], CI + k);
      __builtin_nontemporal_store(s_val[k], CV + k);
    }
  }
}

// Rows that are not float4-aligned: one element per thread and step, ADD_F4 * 4
// steps per tile (tiles from the block start); histogram only, no candidates.
template <bool HIST>
__global__ __launch_bounds__(256) void k_residual_add1(float* __restrict__ acc, int64_t ld_acc,
                                                       const float* __restrict__ grad, int64_t ld_grad, Blocks B,
                                                       uint32_t G, AddSpec sp) {
  __shared__ __align__(16) uint32_t h[HIST ? NB1 : 4];
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
#pragma unroll
  for (int j = 0; j < ADD_F4 * 4; ++j) {
    const uint32_t off = t0 + j * 256u + threadIdx.x;
    if (off < e) {
      const float r = A[off] + Gr[off];
      A[off] = r;
      if (HIST) atomicAdd(&h[mag_key(r) >> D1_SHIFT], 1u);
    }
  }
  if (HIST) {
    if (g == 0u && threadIdx.x == 0) sp.spec_used[wb] = SPEC_NONE;   // no candidates on this path
    __syncthreads();
    uint32_t* __restrict__ H = sp.hist1 + ((int64_t)wb * sp.hcopies + blockIdx.x % HCOPIES_MIN) * NB1;
    flush_hist<256>(h, H);
  }
}

// Level-1 histogram only (block_topk without a fused residual add).
template <int VEC>
__global__ __launch_bounds__(256) void k_hist1(const float* __restrict__ acc, int64_t ld_acc, Blocks B, Units U,
                                               uint32_t G, uint32_t hc, uint32_t* __restrict__ hist1) {
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
  uint32_t* __restrict__ H = hist1 + ((int64_t)wb * hc + blockIdx.x % HCOPIES_MIN) * NB1;
  flush_hist<256>(h, H);
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
                               hipStream_t s, const AddCollect& C) {
  const bool hist = sp.hist1 != nullptr;
  AddSpec spc = sp;
  spc.hcopies = hist_copies_for(n, P);
  if (C.member && !(hist && vec4)) return hipErrorInvalidValue;   // the fused collection needs the fused float4 add
  const int32_t PP = hist ? P : 1;
  const int64_t maxlen = (n + PP - 1) / PP;
  const Blocks B = make_blocks(n, PP);
  if (vec4) {
    // tiles from each block's aligned origin: up to 31 more elements per block
    const uint32_t G = (uint32_t)add_tiles_per_block(maxlen);
    const dim3 grid(G, (unsigned)PP, (unsigned)nworkers);
    if (C.member)
      hipLaunchKernelGGL((k_residual_add4<true, true>), grid, dim3(256), 0, s, acc, ld_acc, grad, ld_grad, B, G, spc, C);
    else if (hist)
      hipLaunchKernelGGL((k_residual_add4<true, false>), grid, dim3(256), 0, s, acc, ld_acc, grad, ld_grad, B, G, spc, C);
    else
      hipLaunchKernelGGL((k_residual_add4<false, false>), grid, dim3(256), 0, s, acc, ld_acc, grad, ld_grad, B, G, spc, C);
  } else {
    const uint32_t G = (uint32_t)((maxlen + ADD_TILE - 1) / ADD_TILE);
    const dim3 grid((unsigned)((int64_t)nworkers * PP * G));
    if (hist) hipLaunchKernelGGL(k_residual_add1<true>, grid, dim3(256), 0, s, acc, ld_acc, grad, ld_grad, B, G, spc);
    else hipLaunchKernelGGL(k_residual_add1<false>, grid, dim3(256), 0, s, acc, ld_acc, grad, ld_grad, B, G, sp);
  }
  return hipGetLastError();
}

hipError_t launch_hist1(const float* acc, int64_t ld_acc, int64_t nunits, const Units& U, int64_t n, int32_t P,
                        bool vec4, uint32_t* hist1, hipStream_t s) {
  const int64_t maxlen = (n + P - 1) / P;
  const int32_t G = (int32_t)((maxlen + ADD_TILE - 1) / ADD_TILE);
  const dim3 grid((unsigned)(nunits * G));
  const Blocks B = make_blocks(n, P);
  const uint32_t hc = hist_copies_for(n, P);
  if (vec4) hipLaunchKernelGGL(k_hist1<4>, grid, dim3(256), 0, s, acc, ld_acc, B, U, (uint32_t)G, hc, hist1);
  else hipLaunchKernelGGL(k_hist1<1>, grid, dim3(256), 0, s, acc, ld_acc, B, U, (uint32_t)G, hc, hist1);
  return hipGetLastError();
}

}  // namespace spardl
