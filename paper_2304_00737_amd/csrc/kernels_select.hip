// Exact top-k selection of the SparDL per-worker hot path for gfx950 (CDNA4,
// wave64): block top-k (Sec. III-B, top-k of Sec. II) and the selection of a
// Spar-Reduce-Scatter merge (Sec. III-B "Transmission with sparsification").
//
// Exact top-k is a radix select on the 31-bit magnitude key in three digits
// (12/11/8 bits).  Dense blocks: the level-1 histogram is built while
// streaming (fused with the residual add); one more streaming pass keeps the
// entries at or above the level-1 threshold bin as candidates in per-tile
// slots (index order inside a slot) and the threshold-bin keys beside them;
// the last two digits are resolved on those keys only; an ordered emit writes
// the selection.  Merges feed the same threshold and emit stages.  No
// workgroup ever waits on another, and no floating-point atomics are used, so
// every result is bit-reproducible.

#include "device.hpp"
#include "launch.hpp"

#include <algorithm>

namespace spardl {

// ============================================================================ level-1 select
// The block's histogram is the sum of its hc copies (hist_copies_for);
// four copies' loads are in flight at a time.  The copies are cleared once read (the
// workspace keeps its histograms at zero between steps).  A histogram of the
// fused add covers keys at or above hist_floor(its candidate floor) in fine
// bins (L1Map in device.hpp), which decides the select exactly whenever the
// threshold bin lies inside that window; otherwise the workgroup rebuilds the
// block's full histogram of the top 12 key bits from acc.  A full histogram
// must hold exactly the block's entries.  The threshold bin goes to the state
// as a key prefix and its shift (ST_T1, ST_SHIFT).
__global__ __launch_bounds__(1024) void k_select1(uint32_t* __restrict__ hist1, uint32_t* __restrict__ state,
                                                  Blocks B, Units U, uint32_t need, uint32_t* __restrict__ spec_t1,
                                                  const uint32_t* __restrict__ spec_used, int spec,
                                                  const float* __restrict__ acc, int64_t ld_acc, int vec4,
                                                  uint32_t hc, uint32_t* __restrict__ err) {
  constexpr int NT = 1024, PER = NB1 / NT;
  static_assert(HCOPIES_MIN == 4, "copies are summed four at a time");
  __shared__ uint32_t h[NB1];
  __shared__ uint32_t scratch[24];
  uint32_t w, b;
  U.decode(blockIdx.x, B.P, &w, &b);
  const int64_t u = (int64_t)w * B.P + b;   // the block's arrays
  uint32_t* __restrict__ H = hist1 + u * hc * NB1;
  uint32_t c[PER];
#pragma unroll
  for (int q = 0; q < PER; ++q) c[q] = 0u;
  for (uint32_t k0 = 0; k0 < hc; k0 += HCOPIES_MIN) {
    uint32_t r[PER][HCOPIES_MIN];
#pragma unroll
    for (int q = 0; q < PER; ++q)
#pragma unroll
      for (uint32_t k = 0; k < HCOPIES_MIN; ++k) r[q][k] = H[(k0 + k) * NB1 + q * NT + threadIdx.x];
#pragma unroll
    for (int q = 0; q < PER; ++q)
#pragma unroll
      for (uint32_t k = 0; k < HCOPIES_MIN; ++k) {
        c[q] += r[q][k];
        H[(k0 + k) * NB1 + q * NT + threadIdx.x] = 0u;
      }
  }
#pragma unroll
  for (int q = 0; q < PER; ++q) h[q * NT + threadIdx.x] = c[q];
  const uint32_t used = spec ? spec_used[u] : SPEC_NONE;
  const L1Map M = l1_map(used);
  __syncthreads();
  uint32_t T, above, cnt, ok, total;
  block_select_desc(h, NB1, need, scratch, &T, &above, &cnt, &ok, &total);
  const uint32_t s = B.start(b), e = B.start(b + 1u);
  bool full = !M.fine;   // the top-12-bit histogram of every key
  uint32_t pfx = T, S = D1_SHIFT;   // the threshold bin: the keys k with k >> S == pfx
  // the threshold fell below the histogram's floor, or above its fine window:
  // count the whole block by its top 12 key bits
  if (!full && (!ok || !M.bin_keys(T, &pfx, &S))) {
    for (int i = threadIdx.x; i < NB1; i += NT) h[i] = 0u;
    __syncthreads();
    const float* __restrict__ A = acc + (int64_t)w * ld_acc;
    if (vec4) {
      for (uint32_t x0 = s + threadIdx.x * 4u; x0 < e; x0 += NT * 4u * 4u) {
        f4v v[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const uint32_t x = x0 + (uint32_t)k * NT * 4u;
          if (x < e) v[k] = *reinterpret_cast<const f4v*>(A + x);
        }
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const uint32_t x = x0 + (uint32_t)k * NT * 4u;
          if (x < e) {
            atomicAdd(&h[mag_key(v[k].x) >> D1_SHIFT], 1u);
            atomicAdd(&h[mag_key(v[k].y) >> D1_SHIFT], 1u);
            atomicAdd(&h[mag_key(v[k].z) >> D1_SHIFT], 1u);
            atomicAdd(&h[mag_key(v[k].w) >> D1_SHIFT], 1u);
          }
        }
      }
    } else {
      for (uint32_t x = s + threadIdx.x; x < e; x += NT) atomicAdd(&h[mag_key(A[x]) >> D1_SHIFT], 1u);
    }
    __syncthreads();
    block_select_desc(h, NB1, need, scratch, &T, &above, &cnt, &ok, &total);
    full = true;
    pfx = T;
    S = D1_SHIFT;
  }
  if (threadIdx.x == 0) {
    uint32_t* st = state + u * ST_WORDS;
    const uint32_t len = e - s;
    if (!ok || (full ? total != len : total > len)) atomicOr(err, ERR_COUNT);
    // the fused add's speculative candidates hold every key >= its floor, so
    // they are usable when the floor is at or below the threshold bin
    st[ST_SPECOK] = (spec && ok && used <= (pfx << S)) ? 1u : 0u;
    if (spec_t1) spec_t1[u] = ok ? ((pfx << S) >> D1_SHIFT) + 1u : 0u;   // the next add's floor: 12-bit bins
    st[ST_T1] = pfx;
    st[ST_SHIFT] = S;
    st[ST_ABOVE1] = above;
    st[ST_NEED1] = ok ? need - above : 0u;
    st[ST_CNT1] = cnt;
  }
}

// ============================================================================ candidate slots
// Candidates of a selection unit live in fixed slots, one per producer
// workgroup, each holding its entries densely and in index order from the
// slot start; the keys of its threshold-bin entries sit at the same offsets
// of a parallel array.
//  mode 0 (block top-k): unit (w, b), region = the block's span of a
//          row-sized buffer, slot = SLOT elements of the block;
//  mode 1 (merge):       unit = pair, region = 2 k_blk merged positions
//          rounded up to whole slots of MERGE_TILE positions.
struct SlotGeom {
  int64_t base;    // first entry of the unit's region
  int64_t len;     // length of the unit's region
  int32_t ss;      // slot size
  int32_t lead;    // slot 0 is short by this much (mode 0: slots start at the block's aligned origin)
  int32_t nslots;  // slots of this unit
  // first entry of slot s in the region, and the entries the slot spans
  __device__ __forceinline__ int64_t off(int32_t s) const { return s == 0 ? 0 : (int64_t)s * ss - lead; }
  __device__ __forceinline__ int64_t cap(int32_t s) const {
    const int64_t hi = (int64_t)(s + 1) * ss - lead;
    return (hi < len ? hi : len) - off(s);
  }
};

__device__ __forceinline__ SlotGeom slot_geom(int mode, uint32_t unit, const Blocks& B, const Units& U,
                                              int64_t kb) {
  SlotGeom g;
  if (mode == 0) {
    uint32_t w, b;   // w: the unit's row within the call
    U.decode(unit, B.P, &w, &b);
    const uint32_t s = B.start(b), e = B.start(b + 1u);
    g.base = (int64_t)w * B.n + s;
    g.len = e - s;
    g.ss = SLOT;
    g.lead = (int32_t)block_lead(s);
    g.nslots = (int32_t)((e - s + g.lead + SLOT - 1) / SLOT);
  } else {
    g.nslots = (int32_t)((2 * kb + MERGE_TILE - 1) / MERGE_TILE);
    g.base = (int64_t)unit * g.nslots * MERGE_TILE;   // whole slots per unit: float4-aligned, full last slot
    g.len = 2 * kb;
    g.ss = MERGE_TILE;
    g.lead = 0;
  }
  return g;
}

// ============================================================================ a3: candidates
// One workgroup per slot of SLOT elements: keeps the entries whose key lies
// at or above the level-1 threshold bin, in index order, and the keys of the
// entries inside the threshold bin.  Thread t owns the SLOT/256 consecutive
// elements starting at SLOT/256 * t, so index order is thread order: one
// wave scan of the packed per-thread counts (candidates | bin entries << 16)
// and one barrier give every thread its write offsets.  No atomics and no
// waiting on other workgroups.
// Candidates of a slot are staged in LDS and written out with coalesced
// stores when they fit COLLECT_STAGE entries (the usual case: about 1 % of a
// slot); a slot with more writes them directly.
constexpr int COLLECT_STAGE = 1024;

struct CollectSmem {
  int32_t si[COLLECT_STAGE];
  float sv[COLLECT_STAGE];
  uint32_t sk[COLLECT_STAGE];
  uint32_t wtot[4];
  uint32_t ck[SLOT / 256 * 4 + 1];   // speculative path: kept entries per (register, wave), then their prefix
  uint32_t cb[SLOT / 256 * 4 + 1];   // ... and threshold-bin entries
};

template <int VEC, bool FULL>
__device__ __forceinline__ void collect_slot(const float* __restrict__ A, uint32_t nvalid, int32_t pos0,
                                             const uint32_t* __restrict__ st, CollectSmem& L,
                                             uint32_t* cnt_out, uint32_t* nbin_out, int32_t* __restrict__ CI,
                                             float* __restrict__ CV, uint32_t* __restrict__ BK) {
  constexpr int PT = SLOT / 256;
  const int lane = lane_id(), wv = wave_id();
  const uint32_t my0 = threadIdx.x * PT;
  float v[PT];
  if (VEC == 4) {
#pragma unroll
    for (int q = 0; q < PT / 4; ++q) {
      f4v x = {0.f, 0.f, 0.f, 0.f};
      if (FULL || my0 + 4 * q < nvalid) x = *reinterpret_cast<const f4v*>(A + my0 + 4 * q);
      v[4 * q + 0] = x.x;
      v[4 * q + 1] = x.y;
      v[4 * q + 2] = x.z;
      v[4 * q + 3] = x.w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < PT; ++i) v[i] = (FULL || my0 + i < nvalid) ? A[my0 + i] : 0.f;
  }
  // the threshold bin is read only now, so its latency overlaps the data loads
  __builtin_amdgcn_sched_barrier(0);
  const uint32_t S = st[ST_SHIFT];
  const uint32_t tlo = st[ST_T1] << S;
  const uint32_t thi = tlo + (1u << S);   // the bin's keys are below 2^31, so this fits in 32 bits
  uint32_t tc = 0, tb = 0;
#pragma unroll
  for (int i = 0; i < PT; ++i) {
    const uint32_t key = mag_key(v[i]);
    const bool c = (FULL || my0 + i < nvalid) && key >= tlo;
    tc += c ? 1u : 0u;
    tb += (c && key < thi) ? 1u : 0u;
  }
  const uint32_t packed = tc | (tb << 16);   // a slot holds at most SLOT < 2^16 of each
  const uint32_t incl = wave_incl_scan(packed);
  if (lane == WAVE - 1) L.wtot[wv] = incl;
  __syncthreads();
  uint32_t base = 0, tot = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const uint32_t x = L.wtot[k];
    base += k < wv ? x : 0u;
    tot += x;
  }
  const uint32_t ncand = tot & 0xFFFFu, nbin = tot >> 16;
  if (threadIdx.x == 255) {
    *cnt_out = ncand;
    *nbin_out = nbin;
  }
  const uint32_t ex = base + incl - packed;
  uint32_t pc = ex & 0xFFFFu, pb = ex >> 16;
  const bool staged = ncand <= (uint32_t)COLLECT_STAGE;   // uniform
  int32_t* __restrict__ oI = staged ? L.si : CI;
  float* __restrict__ oV = staged ? L.sv : CV;
  uint32_t* __restrict__ oK = staged ? L.sk : BK;
  if (tc != 0u) {
#pragma unroll
    for (int i = 0; i < PT; ++i) {
      const uint32_t key = mag_key(v[i]);
      if ((FULL || my0 + i < nvalid) && key >= tlo) {
        oI[pc] = pos0 + (int32_t)(my0 + i);
        oV[pc] = v[i];
        ++pc;
        if (key < thi) {
          oK[pb] = key;
          ++pb;
        }
      }
    }
  }
  if (staged) {
    __syncthreads();
    for (uint32_t j = threadIdx.x; j < ncand; j += 256) {
      CI[j] = L.si[j];
      CV[j] = L.sv[j];
    }
    for (uint32_t j = threadIdx.x; j < nbin; j += 256) BK[j] = L.sk[j];
  }
}

// A slot whose candidates the fused residual add already wrote (every key at
// or above its floor; per add tile, in index order at the tile's span: the
// second tile's list starts off1 entries after the slot's first) is
// filtered by one wave: the entries at or above the level-1 threshold bin are
// compacted in place in index order (the first tile's list, then the
// second's) and the bin keys stored.  Each chunk is loaded into registers
// before any of its writes, and a compacted position never exceeds the
// storage position of an entry not yet read, so no barrier is needed.
static_assert(SLOT == 2 * ADD_TILE, "a slot holds two residual-add tiles");
constexpr int RC_R = 16;  // entries per lane per chunk (a crowded slot holds up to 4096)
__device__ __forceinline__ void recollect_wave(uint32_t c0, uint32_t c1, uint32_t off1, uint32_t tlo, uint32_t thi,
                                               uint32_t* cnt_out, uint32_t* nbin_out, int32_t* __restrict__ CI,
                                               float* __restrict__ CV, uint32_t* __restrict__ BK) {
  const int lane = lane_id();
  const uint64_t lt = __lanemask_lt();
  const uint32_t tot = c0 + c1;
  uint32_t kept = 0, nbin = 0;
  for (uint32_t e0 = 0; e0 < tot; e0 += WAVE * RC_R) {
    int32_t ix[RC_R];
    float vx[RC_R];
#pragma unroll
    for (int r = 0; r < RC_R; ++r) {
      const uint32_t e = e0 + r * WAVE + lane;
      ix[r] = 0;
      vx[r] = 0.f;
      if (e < tot) {
        const uint32_t src = e < c0 ? e : off1 + (e - c0);
        ix[r] = CI[src];
        vx[r] = CV[src];
      }
    }
#pragma unroll
    for (int r = 0; r < RC_R; ++r) {
      const uint32_t e = e0 + r * WAVE + lane;
      const uint32_t key = mag_key(vx[r]);
      const bool k = e < tot && key >= tlo;
      const bool bk = k && key < thi;
      const uint64_t mk = __ballot(k), mb = __ballot(bk);
      if (k) {
        const uint32_t pos = kept + popc64(mk & lt);
        CI[pos] = ix[r];
        CV[pos] = vx[r];
      }
      if (bk) BK[nbin + popc64(mb & lt)] = key;
      kept += popc64(mk);
      nbin += popc64(mb);
    }
  }
  if (lane == 0) {
    *cnt_out = kept;
    *nbin_out = nbin;
  }
}

// The same for a slot whose first R1 WAVE entries the caller loaded into
// ix1 / vx1 (lane l holds entries r WAVE + l), so that the loads of several
// slots are in flight together; later chunks of RC_R2 per lane.
constexpr int RC_R2 = 8;
template <int R1>
__device__ __forceinline__ void recollect_wave_pre(uint32_t c0, uint32_t c1, uint32_t off1, uint32_t tlo, uint32_t thi,
                                                   uint32_t* cnt_out, uint32_t* nbin_out, int32_t* __restrict__ CI,
                                                   float* __restrict__ CV, uint32_t* __restrict__ BK,
                                                   const int32_t (&ix1)[R1], const float (&vx1)[R1]) {
  const int lane = lane_id();
  const uint64_t lt = __lanemask_lt();
  const uint32_t tot = c0 + c1;
  uint32_t kept = 0, nbin = 0;
  auto put = [&](uint32_t e, int32_t ix, float vx) {
    const uint32_t key = mag_key(vx);
    const bool k = e < tot && key >= tlo;
    const bool bk = k && key < thi;
    const uint64_t mk = __ballot(k), mb = __ballot(bk);
    if (k) {
      const uint32_t pos = kept + popc64(mk & lt);
      CI[pos] = ix;
      CV[pos] = vx;
    }
    if (bk) BK[nbin + popc64(mb & lt)] = key;
    kept += popc64(mk);
    nbin += popc64(mb);
  };
#pragma unroll
  for (int r = 0; r < R1; ++r)
    if ((uint32_t)(r * WAVE) < tot) put((uint32_t)(r * WAVE + lane), ix1[r], vx1[r]);
  for (uint32_t e0 = (uint32_t)(R1 * WAVE); e0 < tot; e0 += WAVE * RC_R2) {
    int32_t ix[RC_R2];
    float vx[RC_R2];
#pragma unroll
    for (int r = 0; r < RC_R2; ++r) {
      const uint32_t e = e0 + r * WAVE + lane;
      ix[r] = 0;
      vx[r] = 0.f;
      if (e < tot) {
        const uint32_t src = e < c0 ? e : off1 + (e - c0);
        ix[r] = CI[src];
        vx[r] = CV[src];
      }
    }
#pragma unroll
    for (int r = 0; r < RC_R2; ++r) put(e0 + r * WAVE + lane, ix[r], vx[r]);
  }
  if (lane == 0) {
    *cnt_out = kept;
    *nbin_out = nbin;
  }
}

// One workgroup per 4 SPW consecutive slots of one (worker, block).  With
// the fused add's candidates usable, each wave filters SPW consecutive slots,
// the counts and first entries of all of them loaded before any is filtered
// (when a call has many sparse slots, one slot per wave leaves the wave
// waiting on memory most of the time); otherwise the workgroup collects the
// group's slots from acc one by one.  64 registers let 8 waves share a SIMD
// (the 8-slot form, holding 8 slots' loads, takes up to 96 and 5 waves).
// Slots per call from which the block top-k's collect and emit give each wave
// 2 slots and its staged threshold takes 256 slots per workgroup.
constexpr int64_t MULTI_SLOT_MIN = 1 << 17;
// Slots per wave of the block top-k's collect and emit: 1; 2 from
// MULTI_SLOT_MIN slots per call; 8 when, besides, a block keeps fewer than 8
// entries per slot (its slots hold a few candidates each, so the loads of 8
// slots are in flight for the cost of one).
static inline int topk_slots_per_wave(int64_t nunits, int32_t smax, int32_t kb) {
  if (nunits * smax < MULTI_SLOT_MIN) return 1;
  return (int64_t)kb < 8ll * smax ? 8 : 2;
}
template <int VEC, int SPW>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(SPW >= 8 ? 5 : 8, 8))) void k_collect(const float* __restrict__ acc, int64_t ld_acc, Blocks B, Units U,
                                                 uint32_t smax, uint32_t gq, const uint32_t* __restrict__ state,
                                                 const uint32_t* __restrict__ spec_cnt, uint32_t add_tiles,
                                                 uint32_t* __restrict__ slot_cnt, uint32_t* __restrict__ slot_nbin,
                                                 int32_t* __restrict__ cand_idx, float* __restrict__ cand_val,
                                                 uint32_t* __restrict__ bin_key) {
  constexpr int COLLECT_GROUP = 4 * SPW;     // slots per workgroup
  __shared__ CollectSmem L;
  const uint32_t slot0 = (blockIdx.x % gq) * (uint32_t)COLLECT_GROUP;
  uint32_t w, b;
  U.decode(blockIdx.x / gq, B.P, &w, &b);
  const uint32_t unit = w * B.P + b;   // the block's arrays
  const uint32_t s = B.start(b), e = B.start(b + 1u);
  // slot i spans [o + i SLOT, o + (i+1) SLOT) clipped to the block, o its aligned origin; its two add
  // tiles' candidate lists start at the slot's first element and at o + i SLOT + ADD_TILE
  const uint32_t o = block_origin(s);
  if (o + slot0 * (uint32_t)SLOT >= e) return;
  const uint32_t* st = state + (int64_t)unit * ST_WORDS;
  // counts are clamped to the tiles' lengths inside the block, so reads stay in the slot
  auto tiles = [&](uint32_t slot, uint32_t* t0, uint32_t* len0, uint32_t* len1) {
    const uint32_t sa = o + slot * (uint32_t)SLOT;
    *t0 = sa > s ? sa : s;
    const uint32_t m = sa + (uint32_t)ADD_TILE;
    *len0 = (m < e ? m : e) - *t0;
    *len1 = m < e ? min(e - m, (uint32_t)ADD_TILE) : 0u;
  };
  if constexpr (SPW == 1) {
    const uint32_t specok = st[ST_SPECOK];
    if (specok != 0u) {
      const uint32_t tlo = st[ST_T1] << st[ST_SHIFT], thi = tlo + (1u << st[ST_SHIFT]);
      const uint32_t slot = slot0 + (uint32_t)wave_id();
      if (slot >= smax || o + slot * (uint32_t)SLOT >= e) return;
      uint32_t t0, len0, len1;
      tiles(slot, &t0, &len0, &len1);
      const int64_t tile0 = (int64_t)unit * add_tiles + (int64_t)slot * (SLOT / ADD_TILE);
      const uint32_t c0 = min(spec_cnt[tile0], len0);
      const uint32_t c1 = len1 != 0u ? min(spec_cnt[tile0 + 1], len1) : 0u;
      const int64_t cbase = (int64_t)w * B.n + t0;
      const int64_t si = (int64_t)unit * smax + slot;
      recollect_wave(c0, c1, len0, tlo, thi, slot_cnt + si, slot_nbin + si, cand_idx + cbase, cand_val + cbase,
                     bin_key + cbase);
      return;
    }
  } else {
    // this wave's slots: their candidate counts are loaded beside the unit's
    // state words (in bounds for any live slot)
    constexpr int R1 = SPW >= 8 ? 1 : 4;   // first entries per lane of each slot
    const uint32_t sw = slot0 + (uint32_t)wave_id() * (uint32_t)SPW;
    uint32_t c0[SPW], c1[SPW], off1[SPW];
#pragma unroll
    for (int j = 0; j < SPW; ++j) {
      const uint32_t slot = sw + (uint32_t)j;
      c0[j] = 0u;
      c1[j] = 0u;
      off1[j] = 0u;
      if (slot < smax && o + slot * (uint32_t)SLOT < e) {
        uint32_t t0, len0, len1;
        tiles(slot, &t0, &len0, &len1);
        const int64_t tile0 = (int64_t)unit * add_tiles + (int64_t)slot * (SLOT / ADD_TILE);
        c0[j] = min(spec_cnt[tile0], len0);
        c1[j] = len1 != 0u ? min(spec_cnt[tile0 + 1], len1) : 0u;
        off1[j] = len0;
      }
    }
    const uint32_t specok = st[ST_SPECOK];
    const uint32_t pfx = st[ST_T1], S = st[ST_SHIFT];
    if (specok != 0u) {
      const uint32_t tlo = pfx << S, thi = tlo + (1u << S);
      const int lane = lane_id();
      int32_t ix[SPW][R1];
      float vx[SPW][R1];
#pragma unroll
      for (int j = 0; j < SPW; ++j) {
        const uint32_t tot = c0[j] + c1[j];
        const uint32_t sa = o + (sw + (uint32_t)j) * (uint32_t)SLOT;
        const int64_t cbase = (int64_t)w * B.n + (sa > s ? sa : s);
#pragma unroll
        for (int r = 0; r < R1; ++r) {
          const uint32_t q = (uint32_t)(r * WAVE + lane);
          ix[j][r] = 0;
          vx[j][r] = 0.f;
          if (q < tot) {
            const uint32_t src = q < c0[j] ? q : off1[j] + (q - c0[j]);
            ix[j][r] = cand_idx[cbase + src];
            vx[j][r] = cand_val[cbase + src];
          }
        }
      }
#pragma unroll
      for (int j = 0; j < SPW; ++j) {
        const uint32_t slot = sw + (uint32_t)j;
        if (slot >= smax || o + slot * (uint32_t)SLOT >= e) break;   // wave-uniform; later slots are past the block too
        const uint32_t sa = o + slot * (uint32_t)SLOT;
        const int64_t cbase = (int64_t)w * B.n + (sa > s ? sa : s);
        const int64_t si = (int64_t)unit * smax + slot;
        recollect_wave_pre<R1>(c0[j], c1[j], off1[j], tlo, thi, slot_cnt + si, slot_nbin + si, cand_idx + cbase,
                               cand_val + cbase, bin_key + cbase, ix[j], vx[j]);
      }
      return;
    }
  }
  for (int k = 0; k < COLLECT_GROUP; ++k) {
    const uint32_t slot = slot0 + (uint32_t)k;
    if (slot >= smax || o + slot * (uint32_t)SLOT >= e) break;   // uniform
    if (k > 0) __syncthreads();           // LDS reuse
    const uint32_t sa = o + slot * (uint32_t)SLOT;
    const uint32_t t0 = sa > s ? sa : s;
    const uint32_t hi = sa + (uint32_t)SLOT;
    const uint32_t nvalid = (hi < e ? hi : e) - t0;   // entries of this slot inside the block
    const float* __restrict__ A = acc + (int64_t)w * ld_acc + t0;
    const int64_t cbase = (int64_t)w * B.n + t0;
    const int64_t si = (int64_t)unit * smax + slot;
    if (nvalid == (uint32_t)SLOT)
      collect_slot<VEC, true>(A, nvalid, (int32_t)t0, st, L, slot_cnt + si, slot_nbin + si,
                              cand_idx + cbase, cand_val + cbase, bin_key + cbase);
    else
      collect_slot<VEC, false>(A, nvalid, (int32_t)t0, st, L, slot_cnt + si, slot_nbin + si,
                               cand_idx + cbase, cand_val + cbase, bin_key + cbase);
  }
}

// ============================================================================ exact threshold
// One workgroup per unit.  Resolves the exact threshold -- select every key
// >= TGE, plus the first NEEDEQ (by index) with key TEQ -- and turns per-slot
// counts into exclusive prefixes in index order for the emitter.
//
// Only the entries of the level-1 threshold bin need levels 2 and 3.  For a
// dense block they were stored per slot by k_collect (k_thresh below); for a
// merge they are picked out of the union after the level-1 select on the
// union's histogram (k_mthresh).  Units too long for these one-workgroup
// kernels take the staged threshold over slot groups further below, which
// writes the same results (launch_thresh chooses).

// ---- resident fast path (block top-k)
// When a unit's threshold-bin entries fit in registers -- 32 entries per
// thread -- they are loaded once, with every load in flight together, and
// levels 2, 3 and the per-slot counts run on registers and LDS only.
constexpr int FAST_SLOTS = 8192;                 // block top-k: slots per unit
constexpr int FAST_R0 = 32;                      // block top-k: consecutive bin entries per thread
constexpr int FAST_CAP0 = 1024 * FAST_R0;        // block top-k: bin entries per register-resident chunk
constexpr uint32_t KEY_NONE = 0xFFFFFFFFu;       // marks a register that holds no entry (keys are 31-bit)

// The slot map of chunk 0 holds two 16-bit slot ids per word, with one pad
// word after every 16 so that a thread walking its 16 consecutive words hits
// 16 different banks as its neighbours do.
__device__ __forceinline__ uint32_t map_word(uint32_t w) { return w + (w >> 4); }
__device__ __forceinline__ uint32_t map_half(uint32_t f) { return 2u * map_word(f >> 1) + (f & 1u); }

struct FastSmem {
  uint32_t pref[FAST_SLOTS + 1];   // exclusive prefix of bin entries per slot
  union {
    uint16_t slotid[FAST_CAP0 + FAST_CAP0 / 16];   // block top-k: slot of each entry of chunk 0, padded
    struct {
      uint32_t h[NB1];
      uint32_t cg[FAST_SLOTS];     // per-slot count of selected-by-key (>= TGE) bin entries
      uint32_t ce[FAST_SLOTS];     // per-slot count of key == TEQ
    } c;
  } u;
  uint32_t scratch[48];
};

__device__ __forceinline__ void finish_unit(uint32_t* st, uint32_t T1, uint32_t tge, uint32_t teq, uint32_t need_eq,
                                            uint32_t tot_all, uint32_t tot_ge, uint32_t tot_eq, int32_t kb,
                                            int32_t* drop_cnt, int64_t unit, uint32_t* err, uint32_t hist_total) {
  if (tot_ge + (tot_eq < need_eq ? tot_eq : need_eq) != (uint32_t)kb) atomicOr(err, ERR_COUNT_SUM);
  if (drop_cnt && tot_all != hist_total) atomicOr(err, ERR_COUNT);
  st[ST_T1] = T1;
  st[ST_TGE] = tge;
  st[ST_TEQ] = teq;
  st[ST_NEEDEQ] = need_eq;
  if (drop_cnt) drop_cnt[unit] = (int32_t)(tot_all - (uint32_t)kb);
}

// Block top-k unit with at most FAST_SLOTS slots.  Its threshold-bin entries
// are numbered in slot order, f = 0 .. total-1 (pref[s] = first entry of slot
// s, pref[ns] = total), and taken in chunks of FAST_CAP0 entries, entry
// chunk + r 1024 + t in register r of thread t (coalesced loads).  Chunk 0
// stays in registers; the entry -> slot map of chunk 0 is built in LDS (each
// non-empty slot marks its first entry, then a max-scan fills the gaps).  A
// bin larger than one chunk re-reads the other chunks per pass, finding each
// entry's slot by binary search.

// The largest s in [0, ns) with pref[s] <= f (f < pref[ns]).
__device__ __forceinline__ int slot_of_entry(const uint32_t* pref, int ns, uint32_t f) {
  int lo = 0, hi = ns;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (pref[mid] <= f) lo = mid;
    else hi = mid;
  }
  return lo;
}

// Exclusive prefix maximum of one value per thread over the workgroup
// (0 for thread 0).  `scratch` needs blockDim/64 + 1 words.  Contains barriers.
__device__ __forceinline__ uint32_t block_excl_max(uint32_t v, uint32_t* scratch) {
  const int nw = blockDim.x / WAVE, lane = lane_id(), w = wave_id();
  const uint32_t incl = wave_incl_max(v);
  uint32_t excl = __shfl_up(incl, 1, WAVE);
  if (lane == 0) excl = 0u;
  if (lane == WAVE - 1) scratch[w] = incl;
  __syncthreads();
  // the waves before this one: every wave scans the wave maxima itself
  const uint32_t xi = wave_incl_max(lane < nw ? scratch[lane] : 0u);
  const uint32_t carry = w == 0 ? 0u : (uint32_t)__builtin_amdgcn_readlane((int)xi, w - 1);
  __syncthreads();
  return max(carry, excl);
}

// Entries of chunks after the first: fn(key, slot) for entries
// c0 + r 1024 + t, r < FAST_R0, in batches of 8 loads in flight; the slot of
// each entry by binary search.
template <typename F>
__device__ __forceinline__ void visit_bin_chunk(const uint32_t* __restrict__ K, const uint32_t* pref, int ns,
                                                const SlotGeom& g, uint32_t c0, uint32_t total, F fn) {
  constexpr int B = 8;
  for (int r0 = 0; r0 < FAST_R0; r0 += B) {
    uint32_t key[B], sl[B];
#pragma unroll
    for (int r = 0; r < B; ++r) {
      const uint32_t f = c0 + (uint32_t)((r0 + r) * 1024) + threadIdx.x;
      key[r] = KEY_NONE;
      sl[r] = 0u;
      if (f < total) {
        sl[r] = (uint32_t)slot_of_entry(pref, ns, f);
        key[r] = K[g.off((int32_t)sl[r]) + (f - pref[sl[r]])];
      }
    }
#pragma unroll
    for (int r = 0; r < B; ++r)
      if (key[r] != KEY_NONE) fn(key[r], sl[r]);
  }
}

__device__ __forceinline__ void thresh_fast_topk(FastSmem& L, int64_t unit, const SlotGeom& g, int32_t kb,
                                                 int32_t smax, const uint32_t* __restrict__ K,
                                                 const uint32_t* __restrict__ cnt, const uint32_t* __restrict__ nbn,
                                                 uint32_t T1, uint32_t S, uint32_t need1, uint32_t cnt1, uint32_t* st,
                                                 uint32_t* __restrict__ pre_all, uint32_t* __restrict__ pre_ge,
                                                 uint32_t* __restrict__ pre_eq, uint32_t* err) {
  constexpr int NT = 1024, PS = FAST_SLOTS / NT;   // thread t owns slots PS t .. PS t + PS - 1
  constexpr int MW = FAST_CAP0 / 2 / NT;           // slot-map words (two 16-bit ids) per thread
  static_assert(FAST_SLOTS <= 65536, "slot ids are 16-bit");
  const int t = threadIdx.x;
  const int ns = g.nslots;
  // per owned slot: its entries (clamped to the slot's span) and its bin entries
  uint32_t nb[PS], ca[PS];
#pragma unroll
  for (int u = 0; u < PS; ++u) {
    const int s = PS * t + u;
    ca[u] = 0u;
    nb[u] = 0u;
    if (s < ns) {
      ca[u] = cnt[s];
      nb[u] = nbn[s];
    }
  }
#pragma unroll
  for (int u = 0; u < PS; ++u) {
    const int s = PS * t + u;
    const uint32_t cap = s < ns ? (uint32_t)g.cap(s) : 0u;
    ca[u] = min(ca[u], cap);
    nb[u] = min(nb[u], ca[u]);
  }
  uint32_t sb = 0;
#pragma unroll
  for (int u = 0; u < PS; ++u) sb += nb[u];
  // zero the slot map of chunk 0 while the scan runs
  uint32_t* smw = reinterpret_cast<uint32_t*>(L.u.slotid);
#pragma unroll
  for (int q = 0; q < MW; ++q) smw[map_word(q * NT + t)] = 0u;
  uint32_t total;
  uint32_t run = block_excl_scan(sb, L.scratch, &total);   // has barriers: the map is zero after it
  if (total != cnt1 && t == 0) atomicOr(err, ERR_COUNT);
  const uint32_t m = min(total, (uint32_t)FAST_CAP0);
#pragma unroll
  for (int u = 0; u < PS; ++u) {
    const int s = PS * t + u;
    if (s < ns) {
      L.pref[s] = run;
      if (nb[u] != 0u && run < m) L.u.slotid[map_half(run)] = (uint16_t)s;   // first entry of a non-empty slot
    }
    run += nb[u];
  }
  if (t == 0) L.pref[ns] = total;
  __syncthreads();
  // fill forward: slot of entry f = the last slot head at or before f
  {
    uint32_t wv[MW / 2 * 2];
    uint32_t mx = 0u;
#pragma unroll
    for (int q = 0; q < MW; ++q) {
      wv[q] = smw[map_word(MW * t + q)];
      mx = max(mx, max(wv[q] & 0xFFFFu, wv[q] >> 16));
    }
    uint32_t run_max = block_excl_max(mx, L.scratch);
#pragma unroll
    for (int q = 0; q < MW; ++q) {
      const uint32_t lo = max(run_max, wv[q] & 0xFFFFu);
      const uint32_t hi = max(lo, wv[q] >> 16);
      run_max = hi;
      smw[map_word(MW * t + q)] = lo | (hi << 16);
    }
  }
  __syncthreads();
  const uint32_t nchunks = (total + FAST_CAP0 - 1) / FAST_CAP0;
  uint32_t rk[FAST_R0], rs[FAST_R0 / 2];
#pragma unroll
  for (int r = 0; r < FAST_R0; ++r) {
    const uint32_t f = (uint32_t)(r * NT + t);
    uint32_t key = KEY_NONE, sl = 0u;
    if (f < m) {
      sl = L.u.slotid[map_half(f)];
      key = K[g.off((int32_t)sl) + (f - L.pref[sl])];
    }
    rk[r] = key;
    if (r & 1) rs[r / 2] |= sl << 16;
    else rs[r / 2] = sl;
  }
  __syncthreads();   // the slot map is dead from here (its LDS holds the histograms next)
  auto visit = [&](auto fn) {
#pragma unroll
    for (int r = 0; r < FAST_R0; ++r)
      if ((rk[r] >> S) == T1) fn(rk[r]);
    for (uint32_t c = 1; c < nchunks; ++c)
      visit_bin_chunk(K, L.pref, ns, g, c * FAST_CAP0, total, [&](uint32_t key, uint32_t) {
        if ((key >> S) == T1) fn(key);
      });
  };
  uint32_t tge, teq, need_eq;
  resolve_bin(T1, (int)S, need1, cnt1, L.u.c.h, L.scratch, err, visit, tge, teq, need_eq);
  for (int i = t; i < ns; i += NT) {
    L.u.c.cg[i] = 0u;
    L.u.c.ce[i] = 0u;
  }
  __syncthreads();
  auto count1 = [&](uint32_t key, uint32_t si) {
    if (key >= tge) atomicAdd(&L.u.c.cg[si], 1u);
    else if (need_eq != 0u && key == teq) atomicAdd(&L.u.c.ce[si], 1u);
  };
#pragma unroll
  for (int r = 0; r < FAST_R0; ++r)
    if (rk[r] != KEY_NONE) count1(rk[r], (r & 1) ? (rs[r / 2] >> 16) : (rs[r / 2] & 0xFFFFu));
  for (uint32_t c = 1; c < nchunks; ++c) visit_bin_chunk(K, L.pref, ns, g, c * FAST_CAP0, total, count1);
  __syncthreads();
  uint32_t sa = 0, sg = 0, se = 0, gq[PS], eq[PS];
#pragma unroll
  for (int u = 0; u < PS; ++u) {
    const int s = PS * t + u;
    const uint32_t nbu = s < ns ? L.pref[s + 1] - L.pref[s] : 0u;   // bin entries of the slot (<= ca)
    gq[u] = s < ns ? ca[u] - nbu + L.u.c.cg[s] : 0u;                 // entries above the bin are all selected
    eq[u] = s < ns ? L.u.c.ce[s] : 0u;
    sa += ca[u];
    sg += gq[u];
    se += eq[u];
  }
  uint32_t x3[3] = {sa, sg, se}, t3[3];
  block_excl_scan3(x3, L.scratch, t3);
  uint32_t xa = x3[0], xg = x3[1], xe = x3[2];
  const uint32_t ta = t3[0], tg = t3[1], te = t3[2];
  const int64_t o = unit * smax;
#pragma unroll
  for (int u = 0; u < PS; ++u) {
    const int s = PS * t + u;
    if (s < ns) {
      pre_all[o + s] = xa;
      pre_ge[o + s] = xg;
      pre_eq[o + s] = xe;
    }
    xa += ca[u];
    xg += gq[u];
    xe += eq[u];
  }
  if (t == 0) finish_unit(st, T1, tge, teq, need_eq, ta, tg, te, kb, nullptr, unit, err, 0u);
}

__global__ __launch_bounds__(1024) void k_thresh(Blocks B, Units U, int32_t kb, int32_t smax,
                                                 uint32_t* __restrict__ state, const uint32_t* __restrict__ slot_cnt,
                                                 const uint32_t* __restrict__ slot_nbin,
                                                 const uint32_t* __restrict__ bin_key,
                                                 uint32_t* __restrict__ pre_all, uint32_t* __restrict__ pre_ge,
                                                 uint32_t* __restrict__ pre_eq, uint32_t* __restrict__ err) {
  __shared__ FastSmem S;
  const int64_t cunit = blockIdx.x;
  const SlotGeom g = slot_geom(0, (uint32_t)cunit, B, U, kb);
  const int64_t unit = (int64_t)U.canon((uint32_t)cunit, B.P);   // the unit's arrays
  uint32_t* st = state + unit * ST_WORDS;
  // level 1 was resolved by the level-1 select
  const uint32_t T1 = st[ST_T1], S1 = st[ST_SHIFT], need1 = st[ST_NEED1], cnt1 = st[ST_CNT1];
  if (g.nslots <= FAST_SLOTS) {
    thresh_fast_topk(S, unit, g, kb, smax, bin_key + g.base, slot_cnt + unit * smax, slot_nbin + unit * smax, T1,
                     S1, need1, cnt1, st, pre_all, pre_ge, pre_eq, err);
    return;
  }
  if (threadIdx.x == 0) atomicOr(err, ERR_COUNT);   // longer units are routed to the staged threshold
}

// ---- merge threshold
// One workgroup per merge unit (a union of up to MT_SLOTS slots of
// MERGE_TILE positions).  The union's level-1 histogram, summed by k_merge
// over the fine window (merge_fine in common.hpp), gives the threshold bin:
// the keys k with k >> S == pfx, S = FINE_SHIFT.  k_merge also left, per
// slot, its keys' low bits in bin order and the bins' prefix, so the bin's
// entries of every slot are one contiguous run there: two prefix words per
// slot give the run (and the entries above the bin), and one round of loads
// gathers the runs into a list in LDS -- a few hundred or thousand entries --
// over which the last S key bits (two digits) and the per-slot counts of
// selected and tied keys are resolved.  If the threshold fell in one of the
// window's two clamped bins, a pass over the union builds the histogram of
// the top 12 key bits and a second one counts and lists the bin's entries
// (S = D1_SHIFT).  A bin too large for the list is visited from the union
// again instead (the same results, more passes).
constexpr int MT_THREADS = 1024;
constexpr int MT_LIST = 16384;    // threshold-bin entries held in LDS
static_assert(MERGE_TILE == 4 * MT_THREADS, "a merge slot is one float4 per thread of the merge threshold");
static_assert(MT_SLOTS <= MT_THREADS, "one slot per thread in the per-slot scans");
static_assert((MT_SLOTS - 1) < (1 << (32 - D1_SHIFT)), "slot and low key bits share a list word");

struct MThreshSmem {
  uint32_t h[NB1];
  uint32_t list[MT_LIST];
  uint32_t above[MT_SLOTS];   // per slot: entries above the threshold bin
  uint32_t cg[MT_SLOTS];      // per slot: bin entries with key >= TGE
  uint32_t ce[MT_SLOTS];      // per slot: bin entries with key == TEQ
  uint32_t roff[MT_SLOTS];    // per slot: the run's first position in the list
  uint32_t rlo[MT_SLOTS];     // per slot: the run's first position among the slot's keys
  uint32_t nlist;
  uint32_t scratch[40];
};

// f(key, slot) for every union entry of a unit, read in chunks of 4 slots
// (slot s0 + r, positions 4t .. 4t+3 of it in thread t).
template <typename F>
__device__ __forceinline__ void mt_each(const f4v* __restrict__ V4, const uint32_t* __restrict__ cnt, int32_t ns,
                                        uint32_t cap_last, F f) {
  for (int32_t s0 = 0; s0 < ns; s0 += 4) {
    uint32_t c[4];
    f4v v[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int32_t s = s0 + r;
      c[r] = 0u;
      v[r] = f4v{0.f, 0.f, 0.f, 0.f};
      if (s < ns) {
        c[r] = min(cnt[s], s == ns - 1 ? cap_last : (uint32_t)MERGE_TILE);
        v[r] = V4[(int64_t)s * (MERGE_TILE / 4) + threadIdx.x];
      }
    }
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if ((uint32_t)(4 * threadIdx.x + q) < c[r]) f(mag_key(v[r][q]), (uint32_t)(s0 + r));
  }
}

// Exclusive prefix over the unit's slots of one value per thread (slot t):
// one wave when the unit has at most WAVE slots, else the whole workgroup.
// *total gets the sum.  Uniform over the workgroup; may contain barriers.
__device__ __forceinline__ uint32_t slot_excl_scan(uint32_t v, int32_t ns, uint32_t* scratch, uint32_t* total) {
  if (ns <= WAVE) {
    const uint32_t incl = wave_incl_scan(v);   // every wave scans lanes 0..63 alike; wave 0 holds the slots
    *total = __shfl(incl, WAVE - 1, WAVE);
    return incl - v;
  }
  return block_excl_scan(v, scratch, total);
}

__global__ __launch_bounds__(MT_THREADS) void k_mthresh(int32_t kb, int32_t smax, uint32_t* __restrict__ hist1,
                                                        const float* __restrict__ U_val,
                                                        const uint32_t* __restrict__ U_key,
                                                        uint32_t* __restrict__ state,
                                                        const uint32_t* __restrict__ slot_cnt,
                                                        uint32_t* __restrict__ pre_all, uint32_t* __restrict__ pre_ge,
                                                        uint32_t* __restrict__ pre_eq, int32_t* __restrict__ drop_cnt,
                                                        uint32_t* __restrict__ err) {
  __shared__ MThreshSmem L;
  const int t = threadIdx.x;
  const int64_t unit = blockIdx.x;
  const int32_t ns = (int32_t)((2ll * kb + MERGE_TILE - 1) / MERGE_TILE);   // the merge's slots of this unit
  const uint32_t cap_last = (uint32_t)(2ll * kb - (int64_t)(ns - 1) * MERGE_TILE);
  const int64_t ubase = unit * ns * (int64_t)MERGE_TILE;
  const f4v* __restrict__ V4 = reinterpret_cast<const f4v*>(U_val + ubase);
  const uint32_t* __restrict__ cnt = slot_cnt + unit * smax;
  uint32_t* st = state + unit * ST_WORDS;
  const uint32_t wbase = st[ST_WBASE];
  // the slot's entry count (its own thread), loaded with the histogram
  const uint32_t my_c = t < ns ? min(cnt[t], t == ns - 1 ? cap_last : (uint32_t)MERGE_TILE) : 0u;

  // ---- level 1 on the union's fine histogram (which is left at zero for the next merge)
  uint32_t* __restrict__ H = hist1 + unit * NB1;
  g2lds<NB1 / MT_THREADS>(L.h, H, NB1);
#pragma unroll
  for (int q = 0; q < NB1 / MT_THREADS; ++q) H[q * MT_THREADS + t] = 0u;
  if (t < ns) {
    L.above[t] = 0u;
    L.cg[t] = 0u;
    L.ce[t] = 0u;
  }
  if (t == 0) L.nlist = 0u;
  __syncthreads();
  uint32_t T1, above1, cnt1, ok, hist_total;
  block_select_desc(L.h, NB1, (uint32_t)kb, L.scratch, &T1, &above1, &cnt1, &ok, &hist_total);
  const bool fine = ok && T1 != 0u && T1 != (uint32_t)NB1 - 1u;   // uniform: inside the window
  int S = FINE_SHIFT;
  uint32_t pfx = wbase + T1;
  if (!fine) {
    // the histogram of the top 12 key bits, from the union itself
    __syncthreads();
    for (int i = t; i < NB1; i += MT_THREADS) L.h[i] = 0u;
    __syncthreads();
    mt_each(V4, cnt, ns, cap_last, [&](uint32_t key, uint32_t) { atomicAdd(&L.h[key >> D1_SHIFT], 1u); });
    __syncthreads();
    uint32_t tot2;
    block_select_desc(L.h, NB1, (uint32_t)kb, L.scratch, &T1, &above1, &cnt1, &ok, &tot2);
    S = D1_SHIFT;
    pfx = T1;
  }
  if (!ok && t == 0) atomicOr(err, ERR_COUNT);
  const uint32_t need1 = ok ? (uint32_t)kb - above1 : 0u;
  const uint32_t lowm = (1u << S) - 1u;
  const bool listed = cnt1 <= (uint32_t)MT_LIST;   // uniform

  if (fine) {
    // ---- the bin's run in every slot: [p0, p1) among the slot's keys in bin order
    uint32_t p0 = 0, p1 = 0;
    if (t < ns) {
      const uint16_t* PRE = reinterpret_cast<const uint16_t*>(U_key + ubase + (int64_t)t * MERGE_TILE) + MERGE_TILE;
      p0 = min((uint32_t)PRE[T1], my_c);
      p1 = min(max((uint32_t)PRE[T1 + 1u], p0), my_c);
      L.above[t] = my_c - p1;
      L.rlo[t] = p0;
    }
    uint32_t run_total;
    const uint32_t roff = slot_excl_scan(p1 - p0, ns, L.scratch, &run_total);
    if (t < ns) L.roff[t] = roff;
    if (t == 0) L.nlist = run_total;
    if (run_total != cnt1 && t == 0) atomicOr(err, ERR_COUNT);
    __syncthreads();
    if (listed) {
      // gather: list entry i belongs to the last slot whose run starts at or before it
      constexpr int GR = 4;   // loads in flight per thread
      const uint32_t n = min(L.nlist, (uint32_t)MT_LIST);   // the total, from the scan's wave
      for (uint32_t i0 = 0; i0 < n; i0 += GR * MT_THREADS) {
        uint32_t low[GR], sl[GR];
#pragma unroll
        for (int g = 0; g < GR; ++g) {
          const uint32_t i = i0 + (uint32_t)(g * MT_THREADS + t);
          sl[g] = 0u;
          low[g] = 0u;
          if (i < n) {
            int32_t lo = 0, hi = ns;
            while (hi - lo > 1) {
              const int32_t mid = (lo + hi) >> 1;
              if (L.roff[mid] <= i) lo = mid;
              else hi = mid;
            }
            sl[g] = (uint32_t)lo;
            const uint16_t* SK = reinterpret_cast<const uint16_t*>(U_key + ubase + (int64_t)lo * MERGE_TILE);
            low[g] = SK[L.rlo[lo] + (i - L.roff[lo])];
          }
        }
#pragma unroll
        for (int g = 0; g < GR; ++g) {
          const uint32_t i = i0 + (uint32_t)(g * MT_THREADS + t);
          if (i < n) L.list[i] = (sl[g] << S) | (low[g] & lowm);
        }
      }
    }
  } else {
    // ---- a pass over the union: per-slot counts above the bin, the bin's entries into the list
    mt_each(V4, cnt, ns, cap_last, [&](uint32_t key, uint32_t s) {
      const uint32_t k = key >> S;
      if (k > pfx) atomicAdd(&L.above[s], 1u);
      else if (k == pfx && listed) {
        const uint32_t pos = atomicAdd(&L.nlist, 1u);
        if (pos < (uint32_t)MT_LIST) L.list[pos] = (s << S) | (key & lowm);
      }
    });
  }
  __syncthreads();
  const uint32_t nl = min(L.nlist, (uint32_t)MT_LIST);
  if (listed && nl != cnt1 && t == 0) atomicOr(err, ERR_COUNT);
  // f(key, slot) for every entry of the threshold bin: from the list, or from the union again
  auto each_bin_entry = [&](auto f) {
    if (listed) {
      for (uint32_t i = t; i < nl; i += MT_THREADS) {
        const uint32_t w = L.list[i];
        f((pfx << S) | (w & lowm), w >> S);
      }
    } else {
      mt_each(V4, cnt, ns, cap_last, [&](uint32_t key, uint32_t s) {
        if ((key >> S) == pfx) f(key, s);
      });
    }
  };
  uint32_t tge, teq, need_eq;
  resolve_bin(pfx, S, need1, cnt1, L.h, L.scratch, err,
              [&](auto f) { each_bin_entry([&](uint32_t key, uint32_t) { f(key); }); }, tge, teq, need_eq);
  __syncthreads();
  each_bin_entry([&](uint32_t key, uint32_t s) {
    if (key >= tge) atomicAdd(&L.cg[s], 1u);
    else if (need_eq != 0u && key == teq) atomicAdd(&L.ce[s], 1u);
  });
  __syncthreads();
  // ---- per-slot exclusive prefixes (slot t)
  const uint32_t gq = t < ns ? L.above[t] + L.cg[t] : 0u;
  const uint32_t eq = t < ns ? L.ce[t] : 0u;
  uint32_t ta, tg, te;
  const uint32_t xa = slot_excl_scan(my_c, ns, L.scratch, &ta);
  const uint32_t xg = slot_excl_scan(gq, ns, L.scratch, &tg);
  const uint32_t xe = slot_excl_scan(eq, ns, L.scratch, &te);
  if (t < ns) {
    const int64_t o = unit * smax + t;
    pre_all[o] = xa;
    pre_ge[o] = xg;
    pre_eq[o] = xe;
  }
  if (t == 0) finish_unit(st, pfx, tge, teq, need_eq, ta, tg, te, kb, drop_cnt, unit, err, hist_total);
}

// ============================================================================ exact threshold, large units
// When units are few and long (a worker's blocks of a very long gradient, a
// team's blocks, unions larger than the register-resident merge path holds),
// one workgroup per unit leaves most of the GPU idle.  These kernels resolve
// the same threshold in stages spread over slot groups:
//   merge only: level-1 select on the union histogram (one workgroup per unit);
//   level-2 histogram of the threshold bin's keys (slot groups; LDS, then
//   atomics into the unit's level-1 histogram space, already cleared);
//   level-2 select (one workgroup per unit); level-3 histogram; level-3 select;
//   per-slot counts of selected-by-key and tied keys (slot groups);
//   per-unit exclusive scans into pre_all / pre_ge / pre_eq.
// They write exactly what k_thresh writes.
constexpr int BIG_THREADS = 256;  // threads of the slot-group kernels
constexpr int BIG_R0 = 4;         // block top-k: bin entries per thread in flight
constexpr int BIG_R1 = MERGE_TILE / BIG_THREADS;   // merge: union entries per thread in flight (a slot)
// block top-k: slots per workgroup: 64, a wave per slot in turn, or, when the
// call has at least MULTI_SLOT_MIN slots (sparse bins), 256, one per thread,
// their bin entries walked as one flattened list
constexpr int BIG_GROUP0 = 64;
constexpr int BIG_GROUP0_MANY = BIG_THREADS;

// The bin entries of the block top-k slots s0 .. s0 + group - 1 (one per
// thread; my_nb: the thread's slot's count, 0 for threads past them) taken as
// one flattened list, so that every load of the group is in flight at once
// instead of one slot's after another's: f(key, slot - s0) for each.  The
// slot of entry e is the last one whose exclusive prefix is at most e.
// Workgroups of BIG_THREADS threads; `pref` holds BIG_THREADS words of LDS,
// `scratch` 5.  Contains barriers.
template <typename F>
__device__ __forceinline__ void visit_bin_group(const SlotGeom& g, int32_t s0, int32_t group,
                                                const uint32_t* __restrict__ K, uint32_t my_nb, uint32_t* pref,
                                                uint32_t* scratch, F f) {
  uint32_t total;
  pref[threadIdx.x] = block_excl_scan(my_nb, scratch, &total);
  __syncthreads();
  for (uint32_t e0 = 0; e0 < total; e0 += (uint32_t)(BIG_THREADS * BIG_R0)) {
    uint32_t key[BIG_R0];
    int32_t sl[BIG_R0];
#pragma unroll
    for (int r = 0; r < BIG_R0; ++r) {
      const uint32_t e = e0 + (uint32_t)(r * BIG_THREADS) + threadIdx.x;
      sl[r] = -1;
      key[r] = 0u;
      if (e < total) {
        int32_t lo = 0, hi = group;   // threads past the group hold no entries
        while (hi - lo > 1) {
          const int32_t mid = (lo + hi) >> 1;
          if (pref[mid] <= e) lo = mid;
          else hi = mid;
        }
        sl[r] = lo;
        key[r] = K[g.off(s0 + lo) + (e - pref[lo])];
      }
    }
#pragma unroll
    for (int r = 0; r < BIG_R0; ++r)
      if (sl[r] >= 0) f(key[r], sl[r]);
  }
}

// f(key, slot) for every threshold-bin entry of the block top-k slots
// [s0, s1), a wave per slot in turn (groups of BIG_GROUP0 slots, whose bins
// are fuller: the flattened walk's searches cost more than they save there).
template <typename F>
__device__ __forceinline__ void visit_bin_slots_topk(const SlotGeom& g, int32_t s0, int32_t s1,
                                                     const uint32_t* __restrict__ K,
                                                     const uint32_t* __restrict__ nbn, F f) {
  const int nw = blockDim.x / WAVE;
  for (int32_t slot = s0 + wave_id(); slot < s1; slot += nw) {
    const uint32_t nb = (uint32_t)min((int64_t)nbn[slot], g.cap(slot));   // within the slot's span
    const uint32_t* __restrict__ Ks = K + g.off(slot);
    for (uint32_t j = lane_id(); j < nb; j += WAVE) f(Ks[j], slot);
  }
}

// f(key, slot) for every threshold-bin entry of the merge slots [s0, s1):
// the union entries whose key is in bin T1, the whole workgroup per slot.
template <typename F>
__device__ __forceinline__ void visit_bin_slots_merge(const SlotGeom& g, int32_t s0, int32_t s1,
                                                      const float* __restrict__ V, const uint32_t* __restrict__ cnt,
                                                      uint32_t T1, uint32_t S, F f) {
  for (int32_t slot = s0; slot < s1; ++slot) {
    const uint32_t c = min(cnt[slot], (uint32_t)g.ss);
    const float* __restrict__ Vs = V + g.off(slot);
    for (uint32_t j0 = 0; j0 < c; j0 += BIG_THREADS * BIG_R1) {   // a merge slot is one chunk
      float v[BIG_R1];
#pragma unroll
      for (int r = 0; r < BIG_R1; ++r) {
        const uint32_t j = j0 + (uint32_t)(r * BIG_THREADS) + threadIdx.x;
        v[r] = j < c ? Vs[j] : 0.f;
      }
#pragma unroll
      for (int r = 0; r < BIG_R1; ++r) {
        const uint32_t key = mag_key(v[r]);
        if (j0 + (uint32_t)(r * BIG_THREADS) + threadIdx.x < c && (key >> S) == T1) f(key, slot);
      }
    }
  }
}

struct BigArgs {
  Blocks B;
  Units U;
  int mode;
  int32_t kb, smax, group;   // group: slots per workgroup of the slot-group kernels
  int64_t hstride;           // words of level-1 histogram space per unit
  uint32_t* hist1;
  const float* U_val;
  uint32_t* state;
  const uint32_t *slot_cnt, *slot_nbin, *bin_key;
  uint32_t *pre_all, *pre_ge, *pre_eq;
  int32_t* drop_cnt;
  uint32_t* err;
};

// where a unit's arrays live: block top-k units at row * P + block (as for
// k_thresh), merge pairs at their own number
__device__ __forceinline__ int64_t big_unit(const BigArgs& a, int64_t unit) {
  return a.mode == 0 ? (int64_t)a.U.canon((uint32_t)unit, a.B.P) : unit;
}

__global__ __launch_bounds__(1024) void k_big_level1(BigArgs a) {
  __shared__ uint32_t h[NB1];
  __shared__ uint32_t scratch[32];
  constexpr int NT = 1024;
  const int64_t unit = blockIdx.x;
  const int64_t ua = big_unit(a, unit);
  uint32_t* H = a.hist1 + ua * a.hstride;
  for (int i = threadIdx.x; i < NB1; i += NT) {
    h[i] = H[i];
    H[i] = 0u;   // histograms rest at zero
  }
  __syncthreads();
  uint32_t T1, above1, cnt1, ok, total;
  block_select_desc(h, NB1, (uint32_t)a.kb, scratch, &T1, &above1, &cnt1, &ok, &total);
  if (threadIdx.x == 0) {
    uint32_t* st = a.state + ua * ST_WORDS;
    if (!ok) atomicOr(a.err, ERR_COUNT);
    st[ST_T1] = T1;
    st[ST_SHIFT] = D1_SHIFT;
    st[ST_NEED1] = ok ? (uint32_t)a.kb - above1 : 0u;
    st[ST_CNT1] = cnt1;
    st[ST_HTOT] = total;
  }
}

// The level-1 bin is the keys k with k >> S == ST_T1 (S = ST_SHIFT); its last
// S bits are resolved in two digits, the last of D3 = (S == FINE_SHIFT ? 7 : 8)
// bits.  LEVEL 2: histogram of the first digit of the bin's keys; LEVEL 3: of
// the last digit of the keys whose other bits are ST_PRE23.
__device__ __forceinline__ int digit3_bits(uint32_t S) { return S == (uint32_t)FINE_SHIFT ? 7 : 8; }
template <int mode, int LEVEL>
__global__ __launch_bounds__(256) void k_big_hist(BigArgs a, uint32_t ngroups) {
  constexpr int NB = LEVEL == 2 ? NB2 : NB3;   // the most bins either digit has
  __shared__ uint32_t h[NB];
  const int64_t unit = blockIdx.x / ngroups;
  const int64_t ua = big_unit(a, unit);
  const int32_t grp = (int32_t)(blockIdx.x % ngroups);
  const uint32_t* st = a.state + ua * ST_WORDS;
  const uint32_t T1 = st[ST_T1], S = st[ST_SHIFT];
  const int D3 = digit3_bits(S);
  const uint32_t m2 = (1u << (S - (uint32_t)D3)) - 1u, m3 = (1u << D3) - 1u;
  if (LEVEL == 2 ? st[ST_NEED1] == st[ST_CNT1] : st[ST_STAGE] != 2u) return;   // uniform: resolved already
  const uint32_t pre23 = st[ST_PRE23];
  const SlotGeom g = slot_geom(mode, (uint32_t)unit, a.B, a.U, a.kb);
  const int32_t s0 = grp * a.group, s1 = min(g.nslots, s0 + a.group);
  if (s0 >= s1) return;
  for (int i = threadIdx.x; i < NB; i += blockDim.x) h[i] = 0u;
  auto bump = [&](uint32_t key, int32_t) {
    if (LEVEL == 2) atomicAdd(&h[(key >> D3) & m2], 1u);
    else if ((key >> D3) == pre23) atomicAdd(&h[key & m3], 1u);
  };
  if (mode == 0 && a.group == BIG_GROUP0_MANY) {
    __shared__ uint32_t pref[BIG_THREADS];
    __shared__ uint32_t scratch[8];
    const int32_t slot = s0 + (int32_t)threadIdx.x;
    uint32_t nb = 0u;
    if (slot < s1) {
      nb = (uint32_t)min((int64_t)a.slot_nbin[ua * a.smax + slot], g.cap(slot));   // within the slot's span
    }
    visit_bin_group(g, s0, a.group, a.bin_key + g.base, nb, pref, scratch, bump);   // its first barrier orders the zeroing
  } else if (mode == 0) {
    __syncthreads();
    visit_bin_slots_topk(g, s0, s1, a.bin_key + g.base, a.slot_nbin + ua * a.smax, bump);
  } else {
    __syncthreads();
    visit_bin_slots_merge(g, s0, s1, a.U_val + g.base, a.slot_cnt + ua * a.smax, T1, S, bump);
  }
  __syncthreads();
  uint32_t* H = a.hist1 + ua * a.hstride + (LEVEL == 2 ? 0 : NB2);
  for (int i = threadIdx.x; i < NB; i += blockDim.x) {
    const uint32_t c = h[i];
    if (c) atomicAdd(&H[i], c);
  }
}

template <int LEVEL>
__global__ __launch_bounds__(1024) void k_big_select(BigArgs a) {
  constexpr int NB = LEVEL == 2 ? NB2 : NB3;
  __shared__ uint32_t h[NB];
  __shared__ uint32_t scratch[32];
  const int64_t unit = blockIdx.x;
  const int64_t ua = big_unit(a, unit);
  uint32_t* st = a.state + ua * ST_WORDS;
  const uint32_t T1 = st[ST_T1], S = st[ST_SHIFT], need1 = st[ST_NEED1], cnt1 = st[ST_CNT1];
  const int D3 = digit3_bits(S);
  const int nb = LEVEL == 2 ? 1 << (S - (uint32_t)D3) : 1 << D3;
  if (LEVEL == 2 && need1 == cnt1) {   // the whole bin is selected
    if (threadIdx.x == 0) {
      st[ST_TGE] = T1 << S;
      st[ST_TEQ] = 0u;
      st[ST_NEEDEQ] = 0u;
      st[ST_STAGE] = 0u;
    }
    return;
  }
  if (LEVEL == 3 && st[ST_STAGE] != 2u) return;
  uint32_t* H = a.hist1 + ua * a.hstride + (LEVEL == 2 ? 0 : NB2);
  for (int i = threadIdx.x; i < NB; i += blockDim.x) {
    h[i] = H[i];
    H[i] = 0u;
  }
  __syncthreads();
  const uint32_t need = LEVEL == 2 ? need1 : st[ST_NEED2];
  uint32_t T, above, cnt, ok;
  block_select_desc(h, nb, need, scratch, &T, &above, &cnt, &ok);
  if (threadIdx.x != 0) return;
  if (!ok) atomicOr(a.err, ERR_COUNT_L23);
  const uint32_t rest = need - above;
  if (LEVEL == 2) {
    const uint32_t pre23 = (T1 << (S - (uint32_t)D3)) | T;
    st[ST_TGE] = pre23 << D3;
    st[ST_TEQ] = 0u;
    st[ST_NEEDEQ] = 0u;
    st[ST_PRE23] = pre23;
    st[ST_NEED2] = rest;
    st[ST_STAGE] = (ok && rest != cnt) ? 2u : 0u;
  } else {
    const uint32_t key = (st[ST_PRE23] << D3) | T;
    if (rest == cnt) {
      st[ST_TGE] = key;
    } else {
      st[ST_TGE] = key + 1u;
      st[ST_TEQ] = key;
      st[ST_NEEDEQ] = rest;
    }
    st[ST_STAGE] = 0u;
  }
}

// per slot: entries selected by key (>= TGE) into pre_ge, tied (== TEQ) into pre_eq
template <int mode>
__global__ __launch_bounds__(256) void k_big_count(BigArgs a, uint32_t ngroups) {
  __shared__ uint32_t part[2 * 4];
  const int64_t unit = blockIdx.x / ngroups;
  const int64_t ua = big_unit(a, unit);
  const int32_t grp = (int32_t)(blockIdx.x % ngroups);
  const uint32_t* st = a.state + ua * ST_WORDS;
  const uint32_t T1 = st[ST_T1], tge = st[ST_TGE], teq = st[ST_TEQ], need_eq = st[ST_NEEDEQ];
  const SlotGeom g = slot_geom(mode, (uint32_t)unit, a.B, a.U, a.kb);
  const int32_t s0 = grp * a.group, s1 = min(g.nslots, s0 + a.group);
  const uint32_t* __restrict__ cnt = a.slot_cnt + ua * a.smax;
  const uint32_t* __restrict__ nbn = a.slot_nbin + ua * a.smax;
  const int64_t o = ua * a.smax;
  if (mode == 0 && a.group != BIG_GROUP0_MANY) {
    // a wave per slot: the entries above the bin are selected; count the bin's keys
    const int nw = blockDim.x / WAVE;
    for (int32_t slot = s0 + wave_id(); slot < s1; slot += nw) {
      const uint32_t c = (uint32_t)min((int64_t)cnt[slot], g.cap(slot));
      const uint32_t nb = min(nbn[slot], c);
      const uint32_t* __restrict__ Ks = a.bin_key + g.base + g.off(slot);
      uint32_t ge = 0, eq = 0;
      for (uint32_t j = lane_id(); j < nb; j += WAVE) {
        const uint32_t key = Ks[j];
        ge += key >= tge;
        eq += need_eq != 0u && key == teq;
      }
      ge = wave_sum(ge);
      eq = wave_sum(eq);
      if (lane_id() == 0) {
        a.pre_ge[o + slot] = (c - nb) + ge;
        a.pre_eq[o + slot] = eq;
      }
    }
  } else if (mode == 0) {
    // a thread per slot: the entries above the bin are selected; the bin's
    // keys, flattened over the group, are counted into LDS per slot
    __shared__ uint32_t pref[BIG_THREADS], sge[BIG_THREADS], seq[BIG_THREADS];
    __shared__ uint32_t scratch[8];
    if (s0 >= s1) return;   // uniform
    const int32_t slot = s0 + (int32_t)threadIdx.x;
    uint32_t c = 0u, nb = 0u;
    if (slot < s1) {
      c = (uint32_t)min((int64_t)cnt[slot], g.cap(slot));
      nb = min(nbn[slot], c);
    }
    sge[threadIdx.x] = 0u;
    seq[threadIdx.x] = 0u;   // ordered before the visits by the scan's barriers
    visit_bin_group(g, s0, a.group, a.bin_key + g.base, nb, pref, scratch, [&](uint32_t key, int32_t ls) {
      if (key >= tge) atomicAdd(&sge[ls], 1u);
      else if (need_eq != 0u && key == teq) atomicAdd(&seq[ls], 1u);
    });
    __syncthreads();
    if (slot < s1) {
      a.pre_ge[o + slot] = (c - nb) + sge[threadIdx.x];
      a.pre_eq[o + slot] = seq[threadIdx.x];
    }
  } else {
    (void)T1;
    for (int32_t slot = s0; slot < s1; ++slot) {
      const uint32_t c = min(cnt[slot], (uint32_t)g.ss);
      const float* __restrict__ Vs = a.U_val + g.base + g.off(slot);
      uint32_t ge = 0, eq = 0;
      for (uint32_t j0 = 0; j0 < c; j0 += BIG_THREADS * BIG_R1) {   // a merge slot is one chunk
        float v[BIG_R1];
#pragma unroll
        for (int r = 0; r < BIG_R1; ++r) {
          const uint32_t j = j0 + (uint32_t)(r * BIG_THREADS) + threadIdx.x;
          v[r] = j < c ? Vs[j] : 0.f;
        }
#pragma unroll
        for (int r = 0; r < BIG_R1; ++r) {
          const uint32_t key = mag_key(v[r]);
          const bool in = j0 + (uint32_t)(r * BIG_THREADS) + threadIdx.x < c;
          ge += in && key >= tge;
          eq += in && need_eq != 0u && key == teq;
        }
      }
      ge = wave_sum(ge);
      eq = wave_sum(eq);
      if (lane_id() == 0) {
        part[2 * wave_id()] = ge;
        part[2 * wave_id() + 1] = eq;
      }
      __syncthreads();
      if (threadIdx.x == 0) {
        uint32_t tg = 0, te = 0;
        for (int w = 0; w < (int)(blockDim.x / WAVE); ++w) {
          tg += part[2 * w];
          te += part[2 * w + 1];
        }
        a.pre_ge[o + slot] = tg;
        a.pre_eq[o + slot] = te;
      }
      __syncthreads();
    }
  }
}

// per unit: exclusive prefixes in slot order (in place over the counts), the
// consistency checks and the merge's drop count
constexpr int SCAN_R = 16;   // slots per thread the scan holds in registers (units of up to 16384 slots)
template <int mode>
__global__ __launch_bounds__(1024) void k_big_scan(BigArgs a) {
  __shared__ uint32_t scratch[32];
  constexpr uint32_t NT = 1024;
  const int64_t unit = blockIdx.x;
  const int64_t ua = big_unit(a, unit);
  uint32_t* st = a.state + ua * ST_WORDS;
  const SlotGeom g = slot_geom(mode, (uint32_t)unit, a.B, a.U, a.kb);
  const uint32_t ns = (uint32_t)g.nslots;
  const uint32_t per = (ns + NT - 1) / NT;
  const uint32_t i0 = min(ns, threadIdx.x * per), i1 = min(ns, i0 + per);
  const int64_t o = ua * a.smax;
  const uint32_t* __restrict__ cnt = a.slot_cnt + o;
  uint32_t sa = 0, sg = 0, se = 0;
  uint32_t ta, tg, te;
  if (per <= (uint32_t)SCAN_R) {   // uniform
    // the three arrays loaded coalesced (slot r NT + t in register r of
    // thread t), all loads in flight; each array then goes through LDS so
    // that thread t scans its contiguous slots [i0, i1) and the prefixes
    // are stored coalesced again
    __shared__ uint32_t buf[SCAN_R * NT];
    uint32_t v[3][SCAN_R];
#pragma unroll
    for (int r = 0; r < SCAN_R; ++r) {
      const uint32_t i = (uint32_t)r * NT + threadIdx.x;
      v[0][r] = i < ns ? (uint32_t)min((int64_t)cnt[i], g.cap((int32_t)i)) : 0u;
      v[1][r] = i < ns ? a.pre_ge[o + i] : 0u;
      v[2][r] = i < ns ? a.pre_eq[o + i] : 0u;
    }
    uint32_t* const outs[3] = {a.pre_all + o, a.pre_ge + o, a.pre_eq + o};
    uint32_t tots[3];
#pragma unroll
    for (int q = 0; q < 3; ++q) {
#pragma unroll
      for (int r = 0; r < SCAN_R; ++r) buf[r * NT + threadIdx.x] = v[q][r];
      __syncthreads();
      uint32_t sum = 0;
      for (uint32_t i = i0; i < i1; ++i) sum += buf[i];
      uint32_t x = block_excl_scan(sum, scratch, &tots[q]);   // its barriers order the reads above
      for (uint32_t i = i0; i < i1; ++i) {
        const uint32_t c = buf[i];
        buf[i] = x;
        x += c;
      }
      __syncthreads();
#pragma unroll
      for (int r = 0; r < SCAN_R; ++r) {
        const uint32_t i = (uint32_t)r * NT + threadIdx.x;
        if (i < ns) outs[q][i] = buf[i];
      }
      __syncthreads();   // buf is rewritten for the next array
    }
    ta = tots[0];
    tg = tots[1];
    te = tots[2];
  } else {
    for (uint32_t i = i0; i < i1; ++i) {
      sa += (uint32_t)min((int64_t)cnt[i], g.cap((int32_t)i));
      sg += a.pre_ge[o + i];
      se += a.pre_eq[o + i];
    }
    uint32_t xa = block_excl_scan(sa, scratch, &ta);
    uint32_t xg = block_excl_scan(sg, scratch, &tg);
    uint32_t xe = block_excl_scan(se, scratch, &te);
    for (uint32_t i = i0; i < i1; ++i) {
      const uint32_t ca = (uint32_t)min((int64_t)cnt[i], g.cap((int32_t)i)), cg = a.pre_ge[o + i], ce = a.pre_eq[o + i];
      a.pre_all[o + i] = xa;
      a.pre_ge[o + i] = xg;
      a.pre_eq[o + i] = xe;
      xa += ca;
      xg += cg;
      xe += ce;
    }
  }
  if (threadIdx.x == 0) {
    const uint32_t need_eq = st[ST_NEEDEQ];
    if (tg + (te < need_eq ? te : need_eq) != (uint32_t)a.kb) atomicOr(a.err, ERR_COUNT_SUM);
    if (mode == 1) {
      a.drop_cnt[unit] = (int32_t)(ta - (uint32_t)a.kb);
      if (ta != st[ST_HTOT]) atomicOr(a.err, ERR_COUNT);
    }
  }
}

// ============================================================================ ordered emit
// An entry is selected if its key is >= TGE, or equals TEQ and fewer than
// NEEDEQ equal keys precede it, so the number of selected entries before an
// entry is
//   (#ge before it) + min(#eq before it, NEEDEQ),
// with the counts before the slot taken from the per-slot prefixes of the
// threshold stage and those inside it from wave ballots.  Unselected entries
// of a merge go to the drop list at (#entries before) - (#selected before).
// MODE 0 (block top-k): few candidates per slot, one wave per slot, or SPW
// consecutive slots per wave when the call has many slots (as the collect),
// with the counts, prefixes and first entries of all of them loaded before
// any is emitted; no LDS and no barrier; selected -> sp (and local_idx).
// MODE 1 (merge): slots are full merge tiles, so a workgroup takes one slot
// and each wave a quarter of it, the counts of the quarters before it
// exchanged through LDS; selected -> sp[w][b] in place, the rest -> the
// step's drop lists.
constexpr int EMIT_R = 16;    // entries per lane per chunk (a crowded slot holds up to 4096)
constexpr int EMIT_R1 = 4;    // block top-k, several slots per wave: first entries per lane of each slot
constexpr int EMIT_R0 = 8;    // ... entries per lane per chunk after the first

// Block top-k emit of one slot whose first R1 WAVE entries are in ix1 / vx1
// (lane l holds entries r WAVE + l); run_g / run_e: the >= and == counts of
// the unit's slots before this one.
template <int R1>
__device__ __forceinline__ void emit_topk_slot(uint32_t cnt, uint32_t run_g, uint32_t run_e, uint32_t tge,
                                               uint32_t teq, uint32_t need_eq, int32_t kb,
                                               const int32_t* __restrict__ CI, const float* __restrict__ CV,
                                               const int32_t (&ix1)[R1], const float (&vx1)[R1],
                                               int32_t* __restrict__ oI, float* __restrict__ oV,
                                               int32_t* __restrict__ oL, uint32_t* __restrict__ err,
                                               uint32_t* __restrict__ kcut) {
  const int lane = lane_id();
  const uint64_t lt = __lanemask_lt();
  auto put = [&](uint32_t p, int32_t ix, float vx) {
    const uint32_t key = mag_key(vx);
    const bool is_ge = p < cnt && key >= tge;
    const bool is_eq = p < cnt && need_eq != 0u && key == teq;
    const uint64_t mg = __ballot(is_ge), me = __ballot(is_eq);
    const uint32_t ge_pre = run_g + popc64(mg & lt);
    const uint32_t eq_pre = run_e + popc64(me & lt);
    if (kcut && is_eq && eq_pre + 1u == need_eq) *kcut = (uint32_t)ix;   // the last tie taken
    if (is_ge || (is_eq && eq_pre < need_eq)) {
      const uint32_t sel_before = ge_pre + (eq_pre < need_eq ? eq_pre : need_eq);
      if (sel_before < (uint32_t)kb) {
        oI[sel_before] = ix;
        oV[sel_before] = vx;
        if (oL) oL[sel_before] = ix;
      } else {
        atomicOr(err, ERR_COUNT_POS);
      }
    }
    run_g += popc64(mg);
    run_e += popc64(me);
  };
#pragma unroll
  for (int r = 0; r < R1; ++r)
    if ((uint32_t)(r * WAVE) < cnt) put((uint32_t)(r * WAVE + lane), ix1[r], vx1[r]);
  for (uint32_t e0 = (uint32_t)(R1 * WAVE); e0 < cnt; e0 += WAVE * EMIT_R0) {
    int32_t ix[EMIT_R0];
    float vx[EMIT_R0];
#pragma unroll
    for (int r = 0; r < EMIT_R0; ++r) {
      const uint32_t p = e0 + r * WAVE + lane;
      ix[r] = -1;
      vx[r] = 0.f;
      if (p < cnt) {
        ix[r] = CI[p];
        vx[r] = CV[p];
      }
    }
#pragma unroll
    for (int r = 0; r < EMIT_R0; ++r) put(e0 + r * WAVE + lane, ix[r], vx[r]);
  }
}

template <int MODE, int SPW = 1>
__global__ __launch_bounds__(256) void k_emit(
    const int32_t* __restrict__ cand_idx, const float* __restrict__ cand_val, Blocks B, Units U, Pairs PM,
    int32_t kb, int32_t smax, uint32_t gq, const uint32_t* __restrict__ state,
    const uint32_t* __restrict__ slot_cnt, const uint32_t* __restrict__ pre_all,
    const uint32_t* __restrict__ pre_ge, const uint32_t* __restrict__ pre_eq, int32_t* __restrict__ out_idx,
    float* __restrict__ out_val, int32_t* __restrict__ local_idx, int32_t* __restrict__ drop_idx,
    float* __restrict__ drop_val, uint32_t* __restrict__ err, uint32_t* __restrict__ keep) {
  const uint32_t unit = blockIdx.x / gq;
  const int wv = wave_id();
  if constexpr (MODE == 0 && SPW == 1) {
    const int32_t slot = (int32_t)((blockIdx.x % gq) * 4u + (uint32_t)wv);
    const SlotGeom g = slot_geom(0, unit, B, U, kb);
    if (slot >= g.nslots) return;
    const int lane = lane_id();
    const uint64_t lt = __lanemask_lt();
    const uint32_t au = U.canon(unit, B.P);   // the unit's arrays
    const int64_t si = (int64_t)au * smax + slot;
    const uint32_t* st = state + (int64_t)au * ST_WORDS;
    // independent loads: the slot's count and prefixes, the unit's threshold
    const uint32_t cnt = (uint32_t)min((int64_t)slot_cnt[si], g.cap(slot));
    uint32_t run_g = pre_ge[si], run_e = pre_eq[si];
    const uint32_t tge = st[ST_TGE], teq = st[ST_TEQ], need_eq = st[ST_NEEDEQ];
    const int64_t base = g.base + g.off(slot);
    uint32_t w, b;
    U.decode(unit, B.P, &w, &b);
    const int64_t o = ((int64_t)w * B.P + b) * kb;
    // the selection rule, kept for a residual collection fused into the next add
    uint32_t* __restrict__ kp = keep ? keep + (int64_t)au * KEEP_WORDS : nullptr;
    if (kp && slot == 0 && lane == 0) {
      kp[KEEP_TGE] = tge;
      kp[KEEP_TEQ] = teq;
      kp[KEEP_NEEDEQ] = need_eq;
    }
    for (uint32_t e0 = 0; e0 < cnt; e0 += WAVE * EMIT_R) {
      int32_t ix[EMIT_R];
      float vx[EMIT_R];
#pragma unroll
      for (int r = 0; r < EMIT_R; ++r) {
        const uint32_t p = e0 + r * WAVE + lane;
        ix[r] = -1;
        vx[r] = 0.f;
        if (p < cnt) {
          ix[r] = cand_idx[base + p];
          vx[r] = cand_val[base + p];
        }
      }
#pragma unroll
      for (int r = 0; r < EMIT_R; ++r) {
        const uint32_t p = e0 + r * WAVE + lane;
        const uint32_t key = mag_key(vx[r]);
        const bool is_ge = p < cnt && key >= tge;
        const bool is_eq = p < cnt && need_eq != 0u && key == teq;
        const uint64_t mg = __ballot(is_ge), me = __ballot(is_eq);
        if (p < cnt) {
          const uint32_t ge_pre = run_g + popc64(mg & lt);
          const uint32_t eq_pre = run_e + popc64(me & lt);
          const uint32_t sel_before = ge_pre + (eq_pre < need_eq ? eq_pre : need_eq);
          if (kp && is_eq && eq_pre + 1u == need_eq) kp[KEEP_CUT] = (uint32_t)ix[r];   // the last tie taken
          if (is_ge || (is_eq && eq_pre < need_eq)) {
            if (sel_before < (uint32_t)kb) {
              out_idx[o + sel_before] = ix[r];
              out_val[o + sel_before] = vx[r];
              if (local_idx) local_idx[o + sel_before] = ix[r];
            } else {
              atomicOr(err, ERR_COUNT_POS);
            }
          }
        }
        run_g += popc64(mg);
        run_e += popc64(me);
      }
    }
  } else if constexpr (MODE == 0) {
    constexpr int R1 = SPW >= 8 ? 1 : EMIT_R1;
    const int32_t sw = (int32_t)((blockIdx.x % gq) * (4u * SPW) + (uint32_t)wv * SPW);
    const SlotGeom g = slot_geom(0, unit, B, U, kb);
    if (sw >= g.nslots) return;
    const int lane = lane_id();
    const uint32_t au = U.canon(unit, B.P);   // the unit's arrays
    const uint32_t* st = state + (int64_t)au * ST_WORDS;
    // independent loads: every slot's count and prefixes, the unit's threshold
    uint32_t cnt[SPW], rg[SPW], re[SPW];
#pragma unroll
    for (int j = 0; j < SPW; ++j) {
      cnt[j] = 0u;
      rg[j] = 0u;
      re[j] = 0u;
      if (sw + j < g.nslots) {
        const int64_t si = (int64_t)au * smax + sw + j;
        cnt[j] = (uint32_t)min((int64_t)slot_cnt[si], g.cap(sw + j));
        rg[j] = pre_ge[si];
        re[j] = pre_eq[si];
      }
    }
    const uint32_t tge = st[ST_TGE], teq = st[ST_TEQ], need_eq = st[ST_NEEDEQ];
    int32_t ix[SPW][R1];
    float vx[SPW][R1];
#pragma unroll
    for (int j = 0; j < SPW; ++j) {
      const int64_t base = g.base + g.off(sw + j);
#pragma unroll
      for (int r = 0; r < R1; ++r) {
        const uint32_t p = (uint32_t)(r * WAVE + lane);
        ix[j][r] = -1;
        vx[j][r] = 0.f;
        if (p < cnt[j]) {
          ix[j][r] = cand_idx[base + p];
          vx[j][r] = cand_val[base + p];
        }
      }
    }
    uint32_t w, b;
    U.decode(unit, B.P, &w, &b);
    const int64_t o = ((int64_t)w * B.P + b) * kb;
    // the selection rule, kept for a residual collection fused into the next add
    uint32_t* __restrict__ kp = keep ? keep + (int64_t)au * KEEP_WORDS : nullptr;
    if (kp && sw == 0 && lane == 0) {
      kp[KEEP_TGE] = tge;
      kp[KEEP_TEQ] = teq;
      kp[KEEP_NEEDEQ] = need_eq;
    }
#pragma unroll
    for (int j = 0; j < SPW; ++j) {
      if (sw + j >= g.nslots) break;   // wave-uniform
      const int64_t base = g.base + g.off(sw + j);
      emit_topk_slot<R1>(cnt[j], rg[j], re[j], tge, teq, need_eq, kb, cand_idx + base, cand_val + base, ix[j], vx[j],
                     out_idx + o, out_val + o, local_idx ? local_idx + o : nullptr, err,
                     kp ? kp + KEEP_CUT : nullptr);
    }
  } else {
    constexpr int NPART = 4;   // waves sharing one slot
    const int32_t slot = (int32_t)(blockIdx.x % gq);
    const SlotGeom g = slot_geom(1, unit, B, U, kb);
    if (slot >= g.nslots) return;   // uniform over the workgroup
    const int lane = lane_id();
    const uint64_t lt = __lanemask_lt();
    const int64_t si = (int64_t)unit * smax + slot;
    const uint32_t* st = state + (int64_t)unit * ST_WORDS;
    // independent loads: the slot's count and prefixes, the unit's threshold
    const uint32_t cnt = min(slot_cnt[si], (uint32_t)g.ss);
    const uint32_t all_before = pre_all[si];
    uint32_t run_g = pre_ge[si], run_e = pre_eq[si];
    const uint32_t tge = st[ST_TGE], teq = st[ST_TEQ], need_eq = st[ST_NEEDEQ];
    const int64_t base = g.base + g.off(slot);
    int64_t hb, rb;
    bool both;
    PM.decode(unit, &hb, &rb, &both);
    const int64_t o = hb * kb, o2 = both ? rb * kb : -1;   // output block(s); o2: the other side of an R-SAG exchange
    // this wave's quarter of the slot, loaded once into registers (a quarter
    // is one chunk) together with the loads above: a merge slot is full but
    // for the union's last one and its holes, and its whole MERGE_TILE
    // entries lie in the union's region (entries past the count are not
    // used); the ge / eq counts of the quarters before it through LDS
    static_assert(MERGE_TILE == NPART * WAVE * EMIT_R, "a quarter of a merge slot is one chunk");
    __shared__ uint32_t part_cnt[2 * NPART];
    const uint32_t q_lo = (uint32_t)(wv * WAVE * EMIT_R);
    int32_t ix[EMIT_R];
    float vx[EMIT_R];
#pragma unroll
    for (int r = 0; r < EMIT_R; ++r) {
      const uint32_t p = q_lo + r * WAVE + lane;
      ix[r] = cand_idx[base + p];
      vx[r] = cand_val[base + p];
    }
    const uint32_t p_lo = min(cnt, q_lo);
    const uint32_t p_hi = min(cnt, q_lo + (uint32_t)(WAVE * EMIT_R));
    {
      uint32_t cg = 0, ce = 0;
#pragma unroll
      for (int r = 0; r < EMIT_R; ++r) {
        const uint32_t p = p_lo + r * WAVE + lane;
        const uint32_t key = mag_key(vx[r]);
        cg += popc64(__ballot(p < p_hi && key >= tge));
        ce += popc64(__ballot(p < p_hi && need_eq != 0u && key == teq));
      }
      if (lane == 0) {
        part_cnt[2 * wv] = cg;
        part_cnt[2 * wv + 1] = ce;
      }
      __syncthreads();
      for (int k = 0; k < wv; ++k) {
        run_g += part_cnt[2 * k];
        run_e += part_cnt[2 * k + 1];
      }
    }
    {
      const uint32_t e0 = p_lo;
#pragma unroll
      for (int r = 0; r < EMIT_R; ++r) {
        const uint32_t p = e0 + r * WAVE + lane;
        const uint32_t key = mag_key(vx[r]);
        const bool is_ge = p < p_hi && key >= tge;
        const bool is_eq = p < p_hi && need_eq != 0u && key == teq;
        const uint64_t mg = __ballot(is_ge), me = __ballot(is_eq);
        if (p < p_hi) {
          const uint32_t ge_pre = run_g + popc64(mg & lt);
          const uint32_t eq_pre = run_e + popc64(me & lt);
          const uint32_t sel_before = ge_pre + (eq_pre < need_eq ? eq_pre : need_eq);
          const bool sel = is_ge || (is_eq && eq_pre < need_eq);
          if (sel) {
            if (sel_before < (uint32_t)kb) {
              out_idx[o + sel_before] = ix[r];
              out_val[o + sel_before] = vx[r];
              if (o2 >= 0) {
                out_idx[o2 + sel_before] = ix[r];
                out_val[o2 + sel_before] = vx[r];
              }
            } else {
              atomicOr(err, ERR_COUNT_POS);
            }
          } else {
            const uint32_t dpos = all_before + p - sel_before;
            if (dpos < (uint32_t)kb) {
              drop_idx[(int64_t)unit * kb + dpos] = ix[r];
              drop_val[(int64_t)unit * kb + dpos] = vx[r];
            } else {
              atomicOr(err, ERR_COUNT_DROP);
            }
          }
        }
        run_g += popc64(mg);
        run_e += popc64(me);
      }
    }
  }
}

// ============================================================================ launchers
hipError_t launch_select1(uint32_t* hist1, uint32_t* state, int64_t nunits, const Units& U, int64_t n, int32_t P,
                          uint32_t need, uint32_t* spec_t1, const uint32_t* spec_used, bool spec, const float* acc,
                          int64_t ld_acc, bool vec4, uint32_t* err, hipStream_t s) {
  hipLaunchKernelGGL(k_select1, dim3((unsigned)nunits), dim3(1024), 0, s, hist1, state, make_blocks(n, P), U, need,
                     spec_t1, spec_used, spec ? 1 : 0, acc, ld_acc, vec4 ? 1 : 0, hist_copies_for(n, P), err);
  return hipGetLastError();
}

hipError_t launch_collect(const float* acc, int64_t ld_acc, int64_t nunits, const Units& U, int64_t n, int32_t P,
                          int32_t kb, bool vec4, int32_t smax, const uint32_t* state, const uint32_t* spec_cnt,
                          int32_t add_tiles, uint32_t* slot_cnt, uint32_t* slot_nbin, int32_t* cand_idx,
                          float* cand_val, uint32_t* bin_key, hipStream_t s) {
  // the speculative path exists for float4 rows only (the add writes no candidates otherwise)
  const int spw = vec4 ? topk_slots_per_wave(nunits, smax, kb) : 1;
  const uint32_t gq = (uint32_t)((smax + 4 * spw - 1) / (4 * spw));
  const dim3 grid((unsigned)(nunits * gq));
  const Blocks B = make_blocks(n, P);
  if (spw == 8) hipLaunchKernelGGL((k_collect<4, 8>), grid, dim3(256), 0, s, acc, ld_acc, B, U, (uint32_t)smax, gq, state, spec_cnt, (uint32_t)add_tiles, slot_cnt, slot_nbin, cand_idx, cand_val, bin_key);
  else if (spw == 2) hipLaunchKernelGGL((k_collect<4, 2>), grid, dim3(256), 0, s, acc, ld_acc, B, U, (uint32_t)smax, gq, state, spec_cnt, (uint32_t)add_tiles, slot_cnt, slot_nbin, cand_idx, cand_val, bin_key);
  else if (vec4) hipLaunchKernelGGL((k_collect<4, 1>), grid, dim3(256), 0, s, acc, ld_acc, B, U, (uint32_t)smax, gq, state, spec_cnt, (uint32_t)add_tiles, slot_cnt, slot_nbin, cand_idx, cand_val, bin_key);
  else hipLaunchKernelGGL((k_collect<1, 1>), grid, dim3(256), 0, s, acc, ld_acc, B, U, (uint32_t)smax, gq, state, spec_cnt, (uint32_t)add_tiles, slot_cnt, slot_nbin, cand_idx, cand_val, bin_key);
  return hipGetLastError();
}

hipError_t launch_thresh(int mode, int64_t nunits, const Units& U, int64_t n, int32_t P, int32_t kb, int32_t smax,
                         uint32_t* hist1, const float* U_val, uint32_t* state, const uint32_t* slot_cnt,
                         const uint32_t* slot_nbin, const uint32_t* bin_key, uint32_t* pre_all, uint32_t* pre_ge,
                         uint32_t* pre_eq, int32_t* drop_cnt, uint32_t* err, hipStream_t s) {
  // few long units: the staged threshold over slot groups (same results)
  const bool big = mode == 0 ? (smax > FAST_SLOTS || (nunits < 32 && smax > 1024)) : !merge_fine(kb);
  if (big) {
    if (!hist1) return hipErrorInvalidValue;   // the staged threshold needs the histogram space
    BigArgs a;
    a.B = make_blocks(n, P);
    a.U = U;
    a.mode = mode;
    a.kb = kb;
    a.smax = smax;
    a.group = mode == 0 ? (nunits * smax >= MULTI_SLOT_MIN ? BIG_GROUP0_MANY : BIG_GROUP0) : 1;
    a.hstride = mode == 0 ? (int64_t)hist_copies_for(n, P) * NB1 : NB1;
    a.hist1 = hist1;
    a.U_val = U_val;
    a.state = state;
    a.slot_cnt = slot_cnt;
    a.slot_nbin = slot_nbin;
    a.bin_key = bin_key;
    a.pre_all = pre_all;
    a.pre_ge = pre_ge;
    a.pre_eq = pre_eq;
    a.drop_cnt = drop_cnt;
    a.err = err;
    const uint32_t ngroups = (uint32_t)((smax + a.group - 1) / a.group);
    const dim3 gu((unsigned)nunits), gg((unsigned)(nunits * ngroups));
    if (mode == 0) {
      hipLaunchKernelGGL((k_big_hist<0, 2>), gg, dim3(256), 0, s, a, ngroups);
      hipLaunchKernelGGL(k_big_select<2>, gu, dim3(1024), 0, s, a);
      hipLaunchKernelGGL((k_big_hist<0, 3>), gg, dim3(256), 0, s, a, ngroups);
      hipLaunchKernelGGL(k_big_select<3>, gu, dim3(1024), 0, s, a);
      hipLaunchKernelGGL(k_big_count<0>, gg, dim3(256), 0, s, a, ngroups);
      hipLaunchKernelGGL(k_big_scan<0>, gu, dim3(1024), 0, s, a);
    } else {
      hipLaunchKernelGGL(k_big_level1, gu, dim3(1024), 0, s, a);
      hipLaunchKernelGGL((k_big_hist<1, 2>), gg, dim3(256), 0, s, a, ngroups);
      hipLaunchKernelGGL(k_big_select<2>, gu, dim3(1024), 0, s, a);
      hipLaunchKernelGGL((k_big_hist<1, 3>), gg, dim3(256), 0, s, a, ngroups);
      hipLaunchKernelGGL(k_big_select<3>, gu, dim3(1024), 0, s, a);
      hipLaunchKernelGGL(k_big_count<1>, gg, dim3(256), 0, s, a, ngroups);
      hipLaunchKernelGGL(k_big_scan<1>, gu, dim3(1024), 0, s, a);
    }
    return hipGetLastError();
  }
  if (mode == 0)
    hipLaunchKernelGGL(k_thresh, dim3((unsigned)nunits), dim3(1024), 0, s, make_blocks(n, P), U, kb, smax, state,
                       slot_cnt, slot_nbin, bin_key, pre_all, pre_ge, pre_eq, err);
  else
    hipLaunchKernelGGL(k_mthresh, dim3((unsigned)nunits), dim3(MT_THREADS), 0, s, kb, smax, hist1, U_val, bin_key,
                       state, slot_cnt, pre_all, pre_ge, pre_eq, drop_cnt, err);
  return hipGetLastError();
}

hipError_t launch_emit(int mode, const int32_t* cand_idx, const float* cand_val, int64_t nunits, const Units& U,
                       int64_t n, int32_t P, int32_t kb, const Pairs& PM, int32_t smax, const uint32_t* state,
                       const uint32_t* slot_cnt, const uint32_t* pre_all, const uint32_t* pre_ge,
                       const uint32_t* pre_eq, int32_t* out_idx, float* out_val, int32_t* local_idx,
                       int32_t* drop_idx, float* drop_val, uint32_t* err, hipStream_t s, uint32_t* keep) {
  // block top-k: 4 spw slots per workgroup (spw per wave); merge: one slot per workgroup
  const int spw = mode == 0 ? topk_slots_per_wave(nunits, smax, kb) : 1;
  const uint32_t gq = mode == 0 ? (uint32_t)((smax + 4 * spw - 1) / (4 * spw)) : (uint32_t)smax;
  const dim3 grid((unsigned)(nunits * gq));
  const Blocks B = make_blocks(n, P);
  if (mode == 0 && spw == 8)
    hipLaunchKernelGGL((k_emit<0, 8>), grid, dim3(256), 0, s, cand_idx, cand_val, B, U, PM, kb, smax, gq, state, slot_cnt, pre_all, pre_ge, pre_eq, out_idx, out_val, local_idx, drop_idx, drop_val, err, keep);
  else if (mode == 0 && spw == 2)
    hipLaunchKernelGGL((k_emit<0, 2>), grid, dim3(256), 0, s, cand_idx, cand_val, B, U, PM, kb, smax, gq, state, slot_cnt, pre_all, pre_ge, pre_eq, out_idx, out_val, local_idx, drop_idx, drop_val, err, keep);
  else if (mode == 0)
    hipLaunchKernelGGL(k_emit<0>, grid, dim3(256), 0, s, cand_idx, cand_val, B, U, PM, kb, smax, gq, state, slot_cnt, pre_all, pre_ge, pre_eq, out_idx, out_val, local_idx, drop_idx, drop_val, err, keep);
  else
    hipLaunchKernelGGL(k_emit<1>, grid, dim3(256), 0, s, cand_idx, cand_val, B, U, PM, kb, smax, gq, state, slot_cnt, pre_all, pre_ge, pre_eq, out_idx, out_val, local_idx, drop_idx, drop_val, err, keep);
  return hipGetLastError();
}

}  // namespace spardl
