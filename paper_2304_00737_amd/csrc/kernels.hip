// SparDL per-worker hot path kernels for gfx950 (CDNA4, wave64).
//
// Paper: SparDL (arXiv 2304.00737).  Residual add: Sec. III-B / Algorithm 1.
// Block top-k: Sec. III-B with top-k of Sec. II.  Spar-Reduce-Scatter step:
// Sec. III-B "Transmission with sparsification".  All-Gather + decode: end of
// Sec. III-B.  Global residual collection: Sec. III-C / Algorithm 1.
//
// Exact top-k is a radix select on the 31-bit magnitude key in three digits
// (12/11/8 bits).  Dense blocks: the level-1 histogram is built while
// streaming (fused with the residual add), one more streaming pass keeps the
// entries at or above the level-1 threshold bin as index-ordered candidates,
// and the remaining digits are resolved on those candidates only.  Merges of
// two sorted sparse blocks use merge-path tiles; their union is treated like
// the candidates of a dense block.  Ordered compaction across workgroups uses
// a bounded decoupled look-back.  No floating-point atomics are used anywhere,
// so every result is bit-reproducible.

#include "common.hpp"
#include "launch.hpp"

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
// One workgroup = STREAM_WAVES waves; each wave streams one UNIT of one block
// of one row.  With HIST, every sum's level-1 digit is counted in an LDS
// histogram that is flushed (non-zero bins only) into the block's global one.
template <int VEC, bool HIST>
__global__ __launch_bounds__(256) void k_residual_add(float* __restrict__ acc, int64_t ld_acc,
                                                      const float* __restrict__ grad, int64_t ld_grad,
                                                      int64_t n, int32_t P, int32_t G,
                                                      uint32_t* __restrict__ hist1) {
  __shared__ uint32_t h[HIST ? NB1 : 1];
  const int g = blockIdx.x % G;
  const int64_t wb = blockIdx.x / G;
  const int64_t b = wb % P, w = wb / P;
  const int64_t s = blk_start(b, n, P), e = blk_start(b + 1, n, P);
  const int lane = lane_id();
  if (HIST) {
    for (int i = threadIdx.x; i < NB1; i += blockDim.x) h[i] = 0u;
    __syncthreads();
  }
  const int64_t u0 = s + ((int64_t)g * STREAM_WAVES + wave_id()) * UNIT;
  float* __restrict__ A = acc + w * ld_acc;
  const float* __restrict__ Gr = grad + w * ld_grad;
  if (u0 < e) {
    if (VEC == 4) {
      float4 a[16], gg[16];
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int64_t off = u0 + j * 256 + lane * 4;
        if (off < e) {
          a[j] = *reinterpret_cast<const float4*>(A + off);
          gg[j] = *reinterpret_cast<const float4*>(Gr + off);
        }
      }
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int64_t off = u0 + j * 256 + lane * 4;
        if (off < e) {
          float4 r;
          r.x = a[j].x + gg[j].x;
          r.y = a[j].y + gg[j].y;
          r.z = a[j].z + gg[j].z;
          r.w = a[j].w + gg[j].w;
          *reinterpret_cast<float4*>(A + off) = r;
          if (HIST) {
            atomicAdd(&h[mag_key(r.x) >> D1_SHIFT], 1u);
            atomicAdd(&h[mag_key(r.y) >> D1_SHIFT], 1u);
            atomicAdd(&h[mag_key(r.z) >> D1_SHIFT], 1u);
            atomicAdd(&h[mag_key(r.w) >> D1_SHIFT], 1u);
          }
        }
      }
    } else {
#pragma unroll 16
      for (int j = 0; j < 64; ++j) {
        const int64_t off = u0 + j * 64 + lane;
        if (off < e) {
          const float r = A[off] + Gr[off];
          A[off] = r;
          if (HIST) atomicAdd(&h[mag_key(r) >> D1_SHIFT], 1u);
        }
      }
    }
  }
  if (HIST) {
    __syncthreads();
    uint32_t* __restrict__ H = hist1 + wb * NB1;
    for (int i = threadIdx.x; i < NB1; i += blockDim.x) {
      const uint32_t c = h[i];
      if (c) atomicAdd(&H[i], c);
    }
  }
}

// Level-1 histogram only (block_topk without a fused residual add).
template <int VEC>
__global__ __launch_bounds__(256) void k_hist1(const float* __restrict__ acc, int64_t ld_acc, int64_t n,
                                               int32_t P, int32_t G, uint32_t* __restrict__ hist1) {
  __shared__ uint32_t h[NB1];
  const int g = blockIdx.x % G;
  const int64_t wb = blockIdx.x / G;
  const int64_t b = wb % P, w = wb / P;
  const int64_t s = blk_start(b, n, P), e = blk_start(b + 1, n, P);
  const int lane = lane_id();
  for (int i = threadIdx.x; i < NB1; i += blockDim.x) h[i] = 0u;
  __syncthreads();
  const int64_t u0 = s + ((int64_t)g * STREAM_WAVES + wave_id()) * UNIT;
  const float* __restrict__ A = acc + w * ld_acc;
  if (u0 < e) {
    if (VEC == 4) {
      float4 a[16];
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int64_t off = u0 + j * 256 + lane * 4;
        if (off < e) a[j] = *reinterpret_cast<const float4*>(A + off);
      }
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int64_t off = u0 + j * 256 + lane * 4;
        if (off < e) {
          atomicAdd(&h[mag_key(a[j].x) >> D1_SHIFT], 1u);
          atomicAdd(&h[mag_key(a[j].y) >> D1_SHIFT], 1u);
          atomicAdd(&h[mag_key(a[j].z) >> D1_SHIFT], 1u);
          atomicAdd(&h[mag_key(a[j].w) >> D1_SHIFT], 1u);
        }
      }
    } else {
#pragma unroll 16
      for (int j = 0; j < 64; ++j) {
        const int64_t off = u0 + j * 64 + lane;
        if (off < e) atomicAdd(&h[mag_key(A[off]) >> D1_SHIFT], 1u);
      }
    }
  }
  __syncthreads();
  uint32_t* __restrict__ H = hist1 + wb * NB1;
  for (int i = threadIdx.x; i < NB1; i += blockDim.x) {
    const uint32_t c = h[i];
    if (c) atomicAdd(&H[i], c);
  }
}

// ============================================================================ level-1 select
__global__ __launch_bounds__(256) void k_select1(const uint32_t* __restrict__ hist1,
                                                 uint32_t* __restrict__ state, uint32_t need,
                                                 uint32_t* __restrict__ err) {
  __shared__ uint32_t h[NB1];
  __shared__ uint32_t scratch[16];
  const int64_t u = blockIdx.x;
  const uint32_t* __restrict__ H = hist1 + u * NB1;
  for (int i = threadIdx.x; i < NB1; i += blockDim.x) h[i] = H[i];
  __syncthreads();
  uint32_t T, above, cnt, ok;
  block_select_desc(h, NB1, need, scratch, &T, &above, &cnt, &ok);
  if (threadIdx.x == 0) {
    uint32_t* st = state + u * ST_WORDS;
    if (!ok) atomicOr(err, ERR_COUNT);
    st[ST_T1] = T;
    st[ST_ABOVE1] = above;
    st[ST_NEED1] = ok ? need - above : 0u;
    st[ST_CNT1] = cnt;
  }
}

// ============================================================================ a3: ordered candidates
// Each wave holds 64 values per lane in registers, counts the entries whose
// key lies at or above the level-1 threshold bin, the workgroup gets its
// output offset from the look-back, and the wave writes its candidates in
// index order: (register j, lane, component c) is ascending index.
template <int VEC>
__global__ __launch_bounds__(256) void k_collect(const float* __restrict__ acc, int64_t ld_acc,
                                                 int64_t n, int32_t P, int32_t tiles_per_unit,
                                                 uint32_t* __restrict__ state, uint32_t* __restrict__ tickets,
                                                 uint64_t* __restrict__ status,
                                                 int32_t* __restrict__ cand_idx, float* __restrict__ cand_val,
                                                 uint32_t* __restrict__ err) {
  __shared__ uint32_t sh[16];
  const int64_t unit = blockIdx.x / tiles_per_unit;
  const int64_t b = unit % P, w = unit / P;
  const int64_t s = blk_start(b, n, P), e = blk_start(b + 1, n, P);
  const int64_t len = e - s;
  const uint32_t ntiles = (uint32_t)((len + STREAM_TILE - 1) / STREAM_TILE);
  if (threadIdx.x == 0) sh[0] = atomicAdd(&tickets[unit], 1u);
  __syncthreads();
  const uint32_t tile = sh[0];
  if (tile >= ntiles) return;
  const uint32_t tlo = state[unit * ST_WORDS + ST_T1] << D1_SHIFT;
  const int lane = lane_id(), wv = wave_id();
  const int64_t u0 = s + (int64_t)tile * STREAM_TILE + (int64_t)wv * UNIT;
  const float* __restrict__ A = acc + w * ld_acc;
  const uint64_t lt = __lanemask_lt();

  float v[64];
  if (VEC == 4) {
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int64_t off = u0 + j * 256 + lane * 4;
      float4 q = make_float4(0.f, 0.f, 0.f, 0.f);
      if (off < e) q = *reinterpret_cast<const float4*>(A + off);
      v[4 * j + 0] = q.x;
      v[4 * j + 1] = q.y;
      v[4 * j + 2] = q.z;
      v[4 * j + 3] = q.w;
    }
  } else {
#pragma unroll
    for (int j = 0; j < 64; ++j) {
      const int64_t off = u0 + j * 64 + lane;
      v[j] = off < e ? A[off] : 0.f;
    }
  }
  // element position of register r of this lane
  auto pos_of = [&](int r) -> int64_t {
    return VEC == 4 ? u0 + (r >> 2) * 256 + lane * 4 + (r & 3) : u0 + r * 64 + lane;
  };
  uint32_t wcount = 0;
#pragma unroll
  for (int r = 0; r < 64; ++r) {
    const bool p = pos_of(r) < e && mag_key(v[r]) >= tlo;
    wcount += popc64(__ballot(p));
  }
  if (lane == 0) sh[1 + wv] = wcount;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t run = 0;
    for (int i = 0; i < STREAM_WAVES; ++i) {
      const uint32_t c = sh[1 + i];
      sh[1 + i] = run;
      run += c;
    }
    uint32_t ex, exb;
    lookback(status + unit * tiles_per_unit, tile, run, 0u, &ex, &exb, err);
    sh[8] = ex;
    if (tile == ntiles - 1) state[unit * ST_WORDS + ST_COUNT] = ex + run;
  }
  __syncthreads();
  const int64_t cbase = w * n + s;
  uint32_t run = sh[8] + sh[1 + wv];
  if (VEC == 4) {
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      bool p[4];
      uint64_t m[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        p[c] = pos_of(4 * j + c) < e && mag_key(v[4 * j + c]) >= tlo;
        m[c] = __ballot(p[c]);
      }
      uint32_t before = popc64(m[0] & lt) + popc64(m[1] & lt) + popc64(m[2] & lt) + popc64(m[3] & lt);
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        if (p[c]) {
          const uint32_t pos = run + before;
          if ((int64_t)pos < len) {
            cand_idx[cbase + pos] = (int32_t)pos_of(4 * j + c);
            cand_val[cbase + pos] = v[4 * j + c];
          } else {
            atomicOr(err, ERR_COUNT);
          }
          ++before;
        }
      }
      run += popc64(m[0]) + popc64(m[1]) + popc64(m[2]) + popc64(m[3]);
    }
  } else {
#pragma unroll
    for (int r = 0; r < 64; ++r) {
      const bool p = pos_of(r) < e && mag_key(v[r]) >= tlo;
      const uint64_t m = __ballot(p);
      if (p) {
        const uint32_t pos = run + popc64(m & lt);
        if ((int64_t)pos < len) {
          cand_idx[cbase + pos] = (int32_t)pos_of(r);
          cand_val[cbase + pos] = v[r];
        } else {
          atomicOr(err, ERR_COUNT);
        }
      }
      run += popc64(m);
    }
  }
}

// Start of a unit's candidate region.  Top-k: unit = (w, b), region = the
// block's own span of a row-sized buffer.  Merge: unit = pair, 2 k_blk slots.
__device__ __forceinline__ int64_t cand_base(int mode, int64_t unit, int64_t n, int64_t P, int64_t kb) {
  if (mode == 0) {
    const int64_t b = unit % P, w = unit / P;
    return w * n + blk_start(b, n, P);
  }
  return unit * 2 * kb;
}

// Capacity of a unit's candidate region (the block length, or 2 k_blk).
__device__ __forceinline__ int64_t cand_cap(int mode, int64_t unit, int64_t n, int64_t P, int64_t kb) {
  if (mode == 0) {
    const int64_t b = unit % P;
    return blk_start(b + 1, n, P) - blk_start(b, n, P);
  }
  return 2 * kb;
}

// ============================================================================ levels 2 and 3
// One workgroup per unit resolves the exact threshold on its candidates:
// select keys >= ST_TGE, plus the first ST_NEEDEQ (by index) with key ST_TEQ.
__global__ __launch_bounds__(1024) void k_thresh(const float* __restrict__ cand_val, int mode, int64_t n,
                                                 int32_t P, int32_t kb, uint32_t* __restrict__ state,
                                                 uint32_t* __restrict__ err) {
  __shared__ uint32_t h[NB2];
  __shared__ uint32_t scratch[24];
  const int64_t unit = blockIdx.x;
  uint32_t* st = state + unit * ST_WORDS;
  const uint32_t T1 = st[ST_T1], need1 = st[ST_NEED1], cnt1 = st[ST_CNT1];
  const uint32_t C = min(st[ST_COUNT], (uint32_t)cand_cap(mode, unit, n, P, kb));
  if (need1 == cnt1) {
    if (threadIdx.x == 0) {
      st[ST_TGE] = T1 << D1_SHIFT;
      st[ST_TEQ] = 0u;
      st[ST_NEEDEQ] = 0u;
    }
    return;
  }
  const float* __restrict__ V = cand_val + cand_base(mode, unit, n, P, kb);
  for (int i = threadIdx.x; i < NB2; i += blockDim.x) h[i] = 0u;
  __syncthreads();
  for (uint32_t p = threadIdx.x; p < C; p += blockDim.x) {
    const uint32_t key = mag_key(V[p]);
    if ((key >> D1_SHIFT) == T1) atomicAdd(&h[(key >> D2_SHIFT) & (NB2 - 1)], 1u);
  }
  __syncthreads();
  uint32_t T2, above2, cnt2, ok;
  block_select_desc(h, NB2, need1, scratch, &T2, &above2, &cnt2, &ok);
  const uint32_t need2 = need1 - above2;
  const uint32_t pre = (T1 << (D1_SHIFT - D2_SHIFT)) | T2;   // top 23 bits of the key
  if (!ok || need2 == cnt2) {
    if (threadIdx.x == 0) {
      if (!ok) atomicOr(err, ERR_COUNT);
      st[ST_TGE] = pre << D2_SHIFT;
      st[ST_TEQ] = 0u;
      st[ST_NEEDEQ] = 0u;
    }
    return;
  }
  for (int i = threadIdx.x; i < NB3; i += blockDim.x) h[i] = 0u;
  __syncthreads();
  for (uint32_t p = threadIdx.x; p < C; p += blockDim.x) {
    const uint32_t key = mag_key(V[p]);
    if ((key >> D2_SHIFT) == pre) atomicAdd(&h[key & (NB3 - 1)], 1u);
  }
  __syncthreads();
  uint32_t T3, above3, cnt3;
  block_select_desc(h, NB3, need2, scratch, &T3, &above3, &cnt3, &ok);
  if (threadIdx.x == 0) {
    if (!ok) atomicOr(err, ERR_COUNT);
    const uint32_t need3 = need2 - above3;
    const uint32_t T = (pre << D2_SHIFT) | T3;
    if (need3 == cnt3) {
      st[ST_TGE] = T;
      st[ST_TEQ] = 0u;
      st[ST_NEEDEQ] = 0u;
    } else {
      st[ST_TGE] = T + 1u;
      st[ST_TEQ] = T;
      st[ST_NEEDEQ] = need3;
    }
  }
}

// ============================================================================ ordered emit
// Candidates are dense and index-ordered.  An entry is selected if its key is
// >= TGE, or equals TEQ and fewer than NEEDEQ equal keys precede it.  The
// number of selected entries before position p is
//   (#ge before p) + min(#eq before p, NEEDEQ),
// so a tile only needs the two counts of everything before it (look-back).
// MODE 0 (block top-k): selected -> sp (and local_idx).  MODE 1 (merge):
// selected -> sp[w][b] in place, the rest -> the step's drop lists.
template <int MODE>
__global__ __launch_bounds__(EMIT_THREADS) void k_emit(
    const int32_t* __restrict__ cand_idx, const float* __restrict__ cand_val, int64_t n, int32_t P,
    int32_t kb, int32_t m, const uint32_t* __restrict__ state, uint32_t* __restrict__ tickets,
    uint64_t* __restrict__ status, int32_t tiles_per_unit, int32_t* __restrict__ out_idx,
    float* __restrict__ out_val, int32_t* __restrict__ local_idx, int32_t* __restrict__ drop_idx,
    float* __restrict__ drop_val, int32_t* __restrict__ drop_cnt, uint32_t* __restrict__ err) {
  constexpr int NWV = EMIT_THREADS / WAVE;
  constexpr int NJ = EMIT_PER_THREAD;
  __shared__ uint32_t cge[NJ * NWV], ceq[NJ * NWV];
  __shared__ uint32_t sh[8];
  const int64_t unit = blockIdx.x / EMIT_WGS_PER_UNIT;
  const uint32_t* st = state + unit * ST_WORDS;
  const uint32_t C = min(st[ST_COUNT], (uint32_t)cand_cap(MODE, unit, n, P, kb));
  const uint32_t tge = st[ST_TGE], teq = st[ST_TEQ], need_eq = st[ST_NEEDEQ];
  const uint32_t ntiles = (C + EMIT_TILE - 1) / EMIT_TILE;
  const int64_t base = cand_base(MODE, unit, n, P, kb);
  int64_t o;
  if (MODE == 0) {
    o = unit * kb;
  } else {
    const int64_t w = unit / m, t = unit % m, b = (w + t) % P;
    o = (w * P + b) * kb;
  }
  const int lane = lane_id(), wv = wave_id();
  const uint64_t lt = __lanemask_lt();
  for (;;) {
    if (threadIdx.x == 0) sh[0] = atomicAdd(&tickets[unit], 1u);
    __syncthreads();
    const uint32_t tile = sh[0];
    if (tile >= ntiles) break;
    const uint32_t p0 = tile * EMIT_TILE;
    int32_t ix[NJ];
    float vx[NJ];
    uint64_t mg[NJ], me[NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const uint32_t p = p0 + j * EMIT_THREADS + threadIdx.x;
      ix[j] = -1;
      vx[j] = 0.f;
      if (p < C) {
        ix[j] = cand_idx[base + p];
        vx[j] = cand_val[base + p];
      }
    }
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const uint32_t p = p0 + j * EMIT_THREADS + threadIdx.x;
      const uint32_t key = mag_key(vx[j]);
      const bool valid = p < C;
      mg[j] = __ballot(valid && key >= tge);
      me[j] = __ballot(valid && need_eq != 0u && key == teq);
      if (lane == 0) {
        cge[j * NWV + wv] = popc64(mg[j]);
        ceq[j * NWV + wv] = popc64(me[j]);
      }
    }
    __syncthreads();
    if (wv == 0) {
      // exclusive scan over (j, wave) in j-major order: 2 entries per lane
      const uint32_t g0 = cge[2 * lane], g1 = cge[2 * lane + 1];
      const uint32_t e0 = ceq[2 * lane], e1 = ceq[2 * lane + 1];
      const uint32_t gi = wave_incl_scan(g0 + g1), ei = wave_incl_scan(e0 + e1);
      cge[2 * lane] = gi - g0 - g1;
      cge[2 * lane + 1] = gi - g1;
      ceq[2 * lane] = ei - e0 - e1;
      ceq[2 * lane + 1] = ei - e1;
      if (lane == WAVE - 1) {
        sh[1] = gi;
        sh[2] = ei;
      }
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      uint32_t exg, exe;
      lookback(status + unit * tiles_per_unit, tile, sh[1], sh[2], &exg, &exe, err);
      sh[3] = exg;
      sh[4] = exe;
      if (tile == ntiles - 1) {
        const uint32_t tot_eq = exe + sh[2];
        const uint32_t sel = exg + sh[1] + (tot_eq < need_eq ? tot_eq : need_eq);
        if (sel != (uint32_t)kb) atomicOr(err, ERR_COUNT);
        if (MODE == 1) drop_cnt[unit] = (int32_t)(C - (uint32_t)kb);
      }
    }
    __syncthreads();
    const uint32_t exg = sh[3], exe = sh[4];
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const uint32_t p = p0 + j * EMIT_THREADS + threadIdx.x;
      if (p < C) {
        const uint32_t ge_pre = exg + cge[j * NWV + wv] + popc64(mg[j] & lt);
        const uint32_t eq_pre = exe + ceq[j * NWV + wv] + popc64(me[j] & lt);
        const bool is_ge = (mg[j] >> lane) & 1ull;
        const bool is_eq = (me[j] >> lane) & 1ull;
        const uint32_t sel_before = ge_pre + (eq_pre < need_eq ? eq_pre : need_eq);
        const bool sel = is_ge || (is_eq && eq_pre < need_eq);
        if (sel) {
          if (sel_before < (uint32_t)kb) {
            out_idx[o + sel_before] = ix[j];
            out_val[o + sel_before] = vx[j];
            if (MODE == 0 && local_idx) local_idx[o + sel_before] = ix[j];
          } else {
            atomicOr(err, ERR_COUNT);
          }
        } else if (MODE == 1) {
          const uint32_t dpos = p - sel_before;
          if (dpos < (uint32_t)kb) {
            drop_idx[unit * kb + dpos] = ix[j];
            drop_val[unit * kb + dpos] = vx[j];
          } else {
            atomicOr(err, ERR_COUNT);
          }
        }
      }
    }
    __syncthreads();
  }
}

// ============================================================================ a4: merge-path index sum
// Pair (w, t): held = sp[w][b], received = sp[(w - d) mod P][b], b = (w+t) mod P.
// The merged sequence orders by index with the held entry first on equal
// indices; the held entry then emits held + received and the received entry
// leaves a hole.  Tile = MERGE_TILE merged positions; the emitted (hole-free)
// union is written densely in index order via the look-back, and its level-1
// histogram is accumulated for the selection.
__global__ __launch_bounds__(MERGE_THREADS) void k_merge(
    const int32_t* __restrict__ sp_idx, const float* __restrict__ sp_val, int32_t P, int32_t kb,
    int32_t d, int32_t m, int32_t tiles_per_pair, uint32_t* __restrict__ tickets,
    uint64_t* __restrict__ status, uint32_t* __restrict__ hist1, uint32_t* __restrict__ state,
    int32_t* __restrict__ U_idx, float* __restrict__ U_val, uint32_t* __restrict__ err) {
  // held entries a0-1 .. a1 at [0, nh + 2), received b0 .. b1 at [nh + 2, nh + nr + 3)
  __shared__ int32_t cI[MERGE_TILE + 3];
  __shared__ float cV[MERGE_TILE + 3];
  __shared__ uint32_t hist[NB1];
  __shared__ uint32_t scratch[16];
  __shared__ uint32_t sh[8];
  const int64_t pair = blockIdx.x / tiles_per_pair;
  const int64_t w = pair / m, t = pair % m, b = (w + t) % P, src = (w - d + P) % P;
  const int32_t* __restrict__ Hi = sp_idx + (w * P + b) * kb;
  const float* __restrict__ Hv = sp_val + (w * P + b) * kb;
  const int32_t* __restrict__ Ri = sp_idx + (src * P + b) * kb;
  const float* __restrict__ Rv = sp_val + (src * P + b) * kb;
  const uint32_t L2 = 2u * (uint32_t)kb;
  const uint32_t ntiles = (L2 + MERGE_TILE - 1) / MERGE_TILE;
  if (threadIdx.x == 0) sh[0] = atomicAdd(&tickets[pair], 1u);
  for (int i = threadIdx.x; i < NB1; i += blockDim.x) hist[i] = 0u;
  __syncthreads();
  const uint32_t tile = sh[0];
  if (tile >= ntiles) return;
  const int32_t Q0 = (int32_t)(tile * MERGE_TILE);
  const int32_t Q1 = (int32_t)min(tile * MERGE_TILE + MERGE_TILE, L2);
  // split(q) = number of held entries among the first q merged positions
  if (threadIdx.x < 2) {
    const int32_t q = threadIdx.x == 0 ? Q0 : Q1;
    int32_t lo = max(0, q - kb), hi = min(q, kb);
    while (lo < hi) {
      const int32_t mid = (lo + hi) >> 1;
      if (Hi[mid] <= Ri[q - mid - 1]) lo = mid + 1;
      else hi = mid;
    }
    sh[1 + threadIdx.x] = (uint32_t)lo;
  }
  __syncthreads();
  const int32_t a0 = (int32_t)sh[1], a1 = (int32_t)sh[2];
  const int32_t b0 = Q0 - a0, b1 = Q1 - a1;
  const int32_t nh = a1 - a0, nr = b1 - b0;
  int32_t* hI = cI;
  float* hV = cV;
  int32_t* rI = cI + nh + 2;
  float* rV = cV + nh + 2;
  for (int i = threadIdx.x; i <= nh + 1; i += blockDim.x) {
    // hI[i] = held[a0 - 1 + i]; outside [0, kb): -1 before, INT_MAX after
    const int32_t gi = a0 - 1 + i;
    if (gi < 0) {
      hI[i] = -1;
      hV[i] = 0.f;
    } else if (gi >= kb) {
      hI[i] = INT32_MAX;
      hV[i] = 0.f;
    } else {
      hI[i] = Hi[gi];
      hV[i] = Hv[gi];
    }
  }
  for (int i = threadIdx.x; i <= nr; i += blockDim.x) {
    const int32_t gj = b0 + i;
    if (gj >= kb) {
      rI[i] = INT32_MAX;
      rV[i] = 0.f;
    } else {
      rI[i] = Ri[gj];
      rV[i] = Rv[gj];
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
  uint32_t tot;
  const uint32_t excl = block_excl_scan(cnt, scratch, &tot);
  if (threadIdx.x == 0) {
    uint32_t ex, exb;
    lookback(status + pair * tiles_per_pair, tile, tot, 0u, &ex, &exb, err);
    sh[3] = ex;
    if (tile == ntiles - 1) state[pair * ST_WORDS + ST_COUNT] = ex + tot;
  }
  __syncthreads();
  uint32_t pos = sh[3] + excl;
  const int64_t ubase = pair * (int64_t)L2;
#pragma unroll
  for (int k = 0; k < MERGE_PER_THREAD; ++k) {
    if (eok[k]) {
      if (pos < L2) {
        U_idx[ubase + pos] = ei[k];
        U_val[ubase + pos] = ev[k];
      } else {
        atomicOr(err, ERR_COUNT);
      }
      ++pos;
    }
  }
  uint32_t* __restrict__ H = hist1 + pair * NB1;
  for (int i = threadIdx.x; i < NB1; i += blockDim.x) {
    const uint32_t c = hist[i];
    if (c) atomicAdd(&H[i], c);
  }
}

// ============================================================================ a5: all-gather + densify
// Tile [t0, t0 + DENSE_TILE) of the output is assembled in LDS: zeros, then
// the final entries whose index falls in the tile (found by binary search in
// the index-sorted final blocks sp[b][b]), then streamed out.
__device__ __forceinline__ int32_t lower_bound_i32(const int32_t* __restrict__ a, int32_t len, int64_t x) {
  int32_t lo = 0, hi = len;
  while (lo < hi) {
    const int32_t mid = (lo + hi) >> 1;
    if ((int64_t)a[mid] < x) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

template <int VEC>
__global__ __launch_bounds__(256) void k_densify(const int32_t* __restrict__ sp_idx,
                                                 const float* __restrict__ sp_val, int32_t P, int64_t n,
                                                 int32_t kb, float* __restrict__ dense) {
  __shared__ float tileb[DENSE_TILE];
  __shared__ int32_t rng[2];
  const int64_t t0 = (int64_t)blockIdx.x * DENSE_TILE;
  const int64_t t1 = min(t0 + DENSE_TILE, n);
  for (int i = threadIdx.x; i < DENSE_TILE; i += blockDim.x) tileb[i] = 0.f;
  const int64_t blo = block_of(t0, n, P), bhi = block_of(t1 - 1, n, P);
  for (int64_t b = blo; b <= bhi; ++b) {
    const int32_t* Fi = sp_idx + (b * P + b) * kb;
    const float* Fv = sp_val + (b * P + b) * kb;
    __syncthreads();
    if (threadIdx.x == 0) {
      rng[0] = lower_bound_i32(Fi, kb, t0);
      rng[1] = lower_bound_i32(Fi, kb, t1);
    }
    __syncthreads();
    for (int32_t j = rng[0] + (int32_t)threadIdx.x; j < rng[1]; j += blockDim.x) {
      const int64_t r = (int64_t)Fi[j] - t0;
      if (r >= 0 && r < DENSE_TILE) tileb[r] = Fv[j];
    }
  }
  __syncthreads();
  if (VEC == 4) {
    for (int i = threadIdx.x * 4; i < DENSE_TILE; i += blockDim.x * 4) {
      const int64_t x = t0 + i;
      if (x + 3 < t1) {
        *reinterpret_cast<float4*>(dense + x) = make_float4(tileb[i], tileb[i + 1], tileb[i + 2], tileb[i + 3]);
      } else {
        for (int c = 0; c < 4; ++c)
          if (x + c < t1) dense[x + c] = tileb[i + c];
      }
    }
  } else {
    for (int i = threadIdx.x; i < DENSE_TILE; i += blockDim.x)
      if (t0 + i < t1) dense[t0 + i] = tileb[i];
  }
}

// ============================================================================ a6: residual collection
// Membership bitmap of the final index set I, one 32-bit word per 32 indices,
// built tile by tile without atomics on global memory.
__global__ __launch_bounds__(256) void k_bitmap(const int32_t* __restrict__ sp_idx, int32_t P, int64_t n,
                                                int32_t kb, uint32_t* __restrict__ bm) {
  constexpr int WORDS = DENSE_TILE / 32;
  __shared__ uint32_t words[WORDS];
  __shared__ int32_t rng[2];
  const int64_t t0 = (int64_t)blockIdx.x * DENSE_TILE;
  const int64_t t1 = min(t0 + DENSE_TILE, n);
  for (int i = threadIdx.x; i < WORDS; i += blockDim.x) words[i] = 0u;
  const int64_t blo = block_of(t0, n, P), bhi = block_of(t1 - 1, n, P);
  for (int64_t b = blo; b <= bhi; ++b) {
    const int32_t* Fi = sp_idx + (b * P + b) * kb;
    __syncthreads();
    if (threadIdx.x == 0) {
      rng[0] = lower_bound_i32(Fi, kb, t0);
      rng[1] = lower_bound_i32(Fi, kb, t1);
    }
    __syncthreads();
    for (int32_t j = rng[0] + (int32_t)threadIdx.x; j < rng[1]; j += blockDim.x) {
      const int64_t r = (int64_t)Fi[j] - t0;
      if (r >= 0 && r < DENSE_TILE) atomicOr(&words[r >> 5], 1u << (r & 31));
    }
  }
  __syncthreads();
  const int64_t nw = (n + 31) / 32;
  for (int i = threadIdx.x; i < WORDS; i += blockDim.x) {
    const int64_t wi = t0 / 32 + i;
    if (wi < nw) bm[wi] = words[i];
  }
}

__device__ __forceinline__ bool in_final(const uint32_t* __restrict__ bm, int32_t x) {
  return (bm[x >> 5] >> (x & 31)) & 1u;
}

// acc[w][x] = 0 where worker w selected x locally and x is a final index.
__global__ __launch_bounds__(256) void k_grc_zero(float* __restrict__ acc, int64_t ld_acc, int32_t P,
                                                  int64_t n, int32_t kb, const int32_t* __restrict__ local_idx,
                                                  const uint32_t* __restrict__ bm) {
  const int64_t total = (int64_t)P * P * kb;
  const int64_t per_w = (int64_t)P * kb;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int32_t x = local_idx[i];
    if (x >= 0 && x < n && in_final(bm, x)) acc[(i / per_w) * ld_acc + x] = 0.0f;
  }
}

// acc[w][x] += v for the drops (x, v) of one step with x a final index.
// Within one step a worker drops a given index at most once.
__global__ __launch_bounds__(256) void k_grc_drops(float* __restrict__ acc, int64_t ld_acc, int64_t n, int32_t m,
                                                   int32_t kb, int32_t npairs,
                                                   const int32_t* __restrict__ drop_idx,
                                                   const float* __restrict__ drop_val,
                                                   const int32_t* __restrict__ drop_cnt,
                                                   const uint32_t* __restrict__ bm) {
  const int64_t total = (int64_t)npairs * kb;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t pair = i / kb, j = i % kb;
    if (j >= drop_cnt[pair]) continue;
    const int32_t x = drop_idx[i];
    if (x >= 0 && x < n && in_final(bm, x)) {
      float* p = acc + (pair / m) * ld_acc + x;
      *p = *p + drop_val[i];
    }
  }
}

// ============================================================================ launchers
static inline unsigned grid_for(int64_t work, int per_block, unsigned cap) {
  int64_t g = (work + per_block - 1) / per_block;
  if (g < 1) g = 1;
  return (unsigned)(g > cap ? cap : g);
}

hipError_t launch_fill(const FillRanges& r, hipStream_t s) {
  int64_t total = 0;
  for (int k = 0; k < r.count; ++k) total += r.len[k];
  if (total <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_fill, dim3(grid_for(total, 256, 4096)), dim3(256), 0, s, r);
  return hipGetLastError();
}

hipError_t launch_residual_add(float* acc, int64_t ld_acc, const float* grad, int64_t ld_grad,
                               int32_t nworkers, int64_t n, int32_t P, bool vec4, uint32_t* hist1,
                               hipStream_t s) {
  const int32_t PP = hist1 ? P : 1;
  const int64_t maxlen = (n + PP - 1) / PP;
  const int64_t units = (maxlen + UNIT - 1) / UNIT;
  const int32_t G = (int32_t)((units + STREAM_WAVES - 1) / STREAM_WAVES);
  const dim3 grid((unsigned)((int64_t)nworkers * PP * G));
  if (hist1) {
    if (vec4) hipLaunchKernelGGL((k_residual_add<4, true>), grid, dim3(256), 0, s, acc, ld_acc, grad, ld_grad, n, PP, G, hist1);
    else hipLaunchKernelGGL((k_residual_add<1, true>), grid, dim3(256), 0, s, acc, ld_acc, grad, ld_grad, n, PP, G, hist1);
  } else {
    if (vec4) hipLaunchKernelGGL((k_residual_add<4, false>), grid, dim3(256), 0, s, acc, ld_acc, grad, ld_grad, n, PP, G, hist1);
    else hipLaunchKernelGGL((k_residual_add<1, false>), grid, dim3(256), 0, s, acc, ld_acc, grad, ld_grad, n, PP, G, hist1);
  }
  return hipGetLastError();
}

hipError_t launch_hist1(const float* acc, int64_t ld_acc, int32_t nworkers, int64_t n, int32_t P,
                        bool vec4, uint32_t* hist1, hipStream_t s) {
  const int64_t maxlen = (n + P - 1) / P;
  const int64_t units = (maxlen + UNIT - 1) / UNIT;
  const int32_t G = (int32_t)((units + STREAM_WAVES - 1) / STREAM_WAVES);
  const dim3 grid((unsigned)((int64_t)nworkers * P * G));
  if (vec4) hipLaunchKernelGGL(k_hist1<4>, grid, dim3(256), 0, s, acc, ld_acc, n, P, G, hist1);
  else hipLaunchKernelGGL(k_hist1<1>, grid, dim3(256), 0, s, acc, ld_acc, n, P, G, hist1);
  return hipGetLastError();
}

hipError_t launch_select1(const uint32_t* hist1, uint32_t* state, int64_t nunits, uint32_t need,
                          uint32_t* err, hipStream_t s) {
  hipLaunchKernelGGL(k_select1, dim3((unsigned)nunits), dim3(256), 0, s, hist1, state, need, err);
  return hipGetLastError();
}

hipError_t launch_collect(const float* acc, int64_t ld_acc, int32_t nworkers, int64_t n, int32_t P,
                          bool vec4, int32_t tiles_per_unit, uint32_t* state, uint32_t* tickets,
                          uint64_t* status, int32_t* cand_idx, float* cand_val, uint32_t* err,
                          hipStream_t s) {
  const dim3 grid((unsigned)((int64_t)nworkers * P * tiles_per_unit));
  if (vec4) hipLaunchKernelGGL(k_collect<4>, grid, dim3(256), 0, s, acc, ld_acc, n, P, tiles_per_unit, state, tickets, status, cand_idx, cand_val, err);
  else hipLaunchKernelGGL(k_collect<1>, grid, dim3(256), 0, s, acc, ld_acc, n, P, tiles_per_unit, state, tickets, status, cand_idx, cand_val, err);
  return hipGetLastError();
}

hipError_t launch_thresh(const float* cand_val, int mode, int64_t nunits, int64_t n, int32_t P,
                         int32_t kb, uint32_t* state, uint32_t* err, hipStream_t s) {
  hipLaunchKernelGGL(k_thresh, dim3((unsigned)nunits), dim3(THRESH_THREADS), 0, s, cand_val, mode, n, P, kb, state, err);
  return hipGetLastError();
}

hipError_t launch_emit(int mode, const int32_t* cand_idx, const float* cand_val, int64_t nunits,
                       int64_t n, int32_t P, int32_t kb, int32_t m, const uint32_t* state,
                       uint32_t* tickets, uint64_t* status, int32_t tiles_per_unit, int32_t* out_idx,
                       float* out_val, int32_t* local_idx, int32_t* drop_idx, float* drop_val,
                       int32_t* drop_cnt, uint32_t* err, hipStream_t s) {
  const dim3 grid((unsigned)(nunits * EMIT_WGS_PER_UNIT));
  if (mode == 0)
    hipLaunchKernelGGL(k_emit<0>, grid, dim3(EMIT_THREADS), 0, s, cand_idx, cand_val, n, P, kb, m, state, tickets, status, tiles_per_unit, out_idx, out_val, local_idx, drop_idx, drop_val, drop_cnt, err);
  else
    hipLaunchKernelGGL(k_emit<1>, grid, dim3(EMIT_THREADS), 0, s, cand_idx, cand_val, n, P, kb, m, state, tickets, status, tiles_per_unit, out_idx, out_val, local_idx, drop_idx, drop_val, drop_cnt, err);
  return hipGetLastError();
}

hipError_t launch_merge(const int32_t* sp_idx, const float* sp_val, int32_t P, int32_t kb, int32_t d,
                        int32_t m, int32_t tiles_per_pair, uint32_t* tickets, uint64_t* status,
                        uint32_t* hist1, uint32_t* state, int32_t* U_idx, float* U_val, uint32_t* err,
                        hipStream_t s) {
  const dim3 grid((unsigned)((int64_t)P * m * tiles_per_pair));
  hipLaunchKernelGGL(k_merge, grid, dim3(MERGE_THREADS), 0, s, sp_idx, sp_val, P, kb, d, m, tiles_per_pair, tickets, status, hist1, state, U_idx, U_val, err);
  return hipGetLastError();
}

hipError_t launch_densify(const int32_t* sp_idx, const float* sp_val, int32_t P, int64_t n, int32_t kb,
                          float* dense, bool vec4, hipStream_t s) {
  const dim3 grid((unsigned)((n + DENSE_TILE - 1) / DENSE_TILE));
  if (vec4) hipLaunchKernelGGL(k_densify<4>, grid, dim3(256), 0, s, sp_idx, sp_val, P, n, kb, dense);
  else hipLaunchKernelGGL(k_densify<1>, grid, dim3(256), 0, s, sp_idx, sp_val, P, n, kb, dense);
  return hipGetLastError();
}

hipError_t launch_bitmap(const int32_t* sp_idx, int32_t P, int64_t n, int32_t kb, uint32_t* bm,
                         hipStream_t s) {
  const dim3 grid((unsigned)((n + DENSE_TILE - 1) / DENSE_TILE));
  hipLaunchKernelGGL(k_bitmap, grid, dim3(256), 0, s, sp_idx, P, n, kb, bm);
  return hipGetLastError();
}

hipError_t launch_grc_zero(float* acc, int64_t ld_acc, int32_t P, int64_t n, int32_t kb, const int32_t* local_idx,
                           const uint32_t* bm, hipStream_t s) {
  hipLaunchKernelGGL(k_grc_zero, dim3(grid_for((int64_t)P * P * kb, 256, 8192)), dim3(256), 0, s, acc, ld_acc, P, n, kb, local_idx, bm);
  return hipGetLastError();
}

hipError_t launch_grc_drops(float* acc, int64_t ld_acc, int64_t n, int32_t m, int32_t kb, int32_t npairs,
                            const int32_t* drop_idx, const float* drop_val, const int32_t* drop_cnt,
                            const uint32_t* bm, hipStream_t s) {
  hipLaunchKernelGGL(k_grc_drops, dim3(grid_for((int64_t)npairs * kb, 256, 8192)), dim3(256), 0, s, acc, ld_acc, n, m, kb, npairs, drop_idx, drop_val, drop_cnt, bm);
  return hipGetLastError();
}

}  // namespace spardl
