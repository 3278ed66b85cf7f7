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
//
// The tile's two merge-path splits (held entries before its first and past
// its last position) are bracketed by one wave each, MERGE_PROBES-ary
// searches over global memory (two rounds for blocks of up to about 260 Ki
// entries; a probe per lane, no barrier), and resolved exactly in LDS after
// the tile's entries and the brackets' slack have been loaded there in one
// round of coalesced loads.  Meanwhile the other waves read the leading
// FINE_SAMPLE entries of both blocks, whose median keys place the fine
// level-1 window (FINE; see merge_fine in common.hpp); every tile of a pair
// reads the same entries, so all of them use the same window.
constexpr int MERGE_PROBES = WAVE;                 // probes per search round (a lane each)
constexpr int MERGE_BRK = 32;                      // bracket width resolved in LDS
constexpr int MERGE_WIN = MERGE_TILE + 4 * MERGE_BRK + 8;   // LDS entries: the tile, the slack and sentinels
static_assert(2 * MERGE_BRK <= MERGE_THREADS, "both brackets are tested in one pass");
static_assert(MERGE_THREADS / WAVE >= 4 && FINE_SAMPLE % WAVE == 0, "two searching and two sampling waves");

// The bracket [lo, hi] of a monotone partition point (pred true below it),
// narrowed by one wave until at most MERGE_BRK wide.
template <typename Pred>
__device__ __forceinline__ void wave_bracket(int32_t& lo, int32_t& hi, Pred pred) {
  const int lane = lane_id();
  while (hi - lo > MERGE_BRK) {   // uniform over the wave
    const int32_t S = hi - lo;
    const int32_t p = lo + (int32_t)(((int64_t)S * (lane + 1)) / (MERGE_PROBES + 1));
    const int32_t c = (int32_t)popc64(__ballot(pred(p)));
    const int32_t nlo = c == 0 ? lo : lo + (int32_t)(((int64_t)S * c) / (MERGE_PROBES + 1)) + 1;
    const int32_t nhi = c == MERGE_PROBES ? hi : lo + (int32_t)(((int64_t)S * (c + 1)) / (MERGE_PROBES + 1));
    lo = nlo;
    hi = nhi;
  }
}

// Level-1 bin of a union key: FINE, NB1 bins of 2^FINE_SHIFT keys from
// `base` (clamped to the first and last); else the top 12 key bits.
template <bool FINE>
__device__ __forceinline__ uint32_t merge_bin(uint32_t key, uint32_t base) {
  if (!FINE) return key >> D1_SHIFT;
  const int32_t b = (int32_t)(key >> FINE_SHIFT) - (int32_t)base;
  return (uint32_t)min(max(b, 0), NB1 - 1);
}

template <bool FINE>
__global__ __launch_bounds__(MERGE_THREADS) void k_merge(
    const int32_t* __restrict__ sp_idx, const float* __restrict__ sp_val, Pairs PM, int32_t kb,
    int32_t tiles_per_pair, uint32_t* __restrict__ hist1, uint32_t* __restrict__ state,
    uint32_t* __restrict__ slot_cnt, int32_t* __restrict__ U_idx, float* __restrict__ U_val,
    uint32_t* __restrict__ U_key) {
  __shared__ int32_t cI[MERGE_WIN];
  __shared__ float cV[MERGE_WIN];
  __shared__ __align__(16) uint32_t hist[NB1];
  __shared__ uint32_t scratch[2 * (MERGE_THREADS / WAVE) + 1];
  __shared__ int32_t brk[4];
  __shared__ uint32_t smin[2];   // the two blocks' median keys (reused as a flag below)
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
  // before received entry q-a-1 (held goes first on equal indices).
  const int wv = wave_id(), lane = lane_id();
  if (wv < 2) {
    const int32_t q = wv == 0 ? Q0 : Q1;
    int32_t lo = max(0, q - kb), hi = min(q, kb);
    wave_bracket(lo, hi, [&](int32_t a) { return Hi[a] <= Ri[q - a - 1]; });
    if (lane == 0) {
      brk[2 * wv] = lo;
      brk[2 * wv + 1] = hi;
    }
  } else if (FINE && wv < 4) {
    // the median key among the leading entries of the held (wave 2) or received (wave 3)
    // block to 1/8 binade: the largest multiple T of 2^FINE_CENTRE_BIT with at least
    // half of them >= T, found bit by bit
    const float* __restrict__ V = wv == 2 ? Hv : Rv;
    constexpr int U = FINE_SAMPLE / WAVE;
    uint32_t key[U];
    bool ok[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int32_t j = u * WAVE + lane;
      ok[u] = j < kb;
      key[u] = ok[u] ? mag_key(V[j]) : 0u;
    }
    const uint32_t half = ((uint32_t)min(kb, FINE_SAMPLE) + 1u) / 2u;
    uint32_t T = 0;
    for (int bit = 30; bit >= FINE_CENTRE_BIT; --bit) {
      const uint32_t c = T | (1u << bit);
      uint32_t nge = 0;
#pragma unroll
      for (int u = 0; u < U; ++u) nge += popc64(__ballot(ok[u] && key[u] >= c));
      if (nge >= half) T = c;
    }
    if (lane == 0) smin[wv - 2] = T;
  }
  __syncthreads();
  const int32_t lo0 = brk[0], hi0 = brk[1], lo1 = brk[2], hi1 = brk[3];
  uint32_t wbase = 0;
  if (FINE) {
    // the window's centre: the mean of the two median keys (the geometric mean of the values)
    const uint32_t mid = ((smin[0] >> 1) + (smin[1] >> 1)) >> FINE_SHIFT;
    wbase = mid > FINE_BELOW ? mid - FINE_BELOW : 0u;
    if (tile == 0 && threadIdx.x == 0) state[(int64_t)pair * ST_WORDS + ST_WBASE] = wbase;
  }
  // the LDS window: held [ha, hz) and received [ra, rz) cover both brackets'
  // tests and every entry the merge reads (held a0-1 .. a1, received b0 .. b1)
  const int32_t ha = lo0 - 1, hz = max(hi0, hi1) + 1;
  const int32_t ra = min(Q0 - hi0, Q1 - hi1), rz = max(Q0 - lo0, Q1 - lo1) + 1;
  const int32_t nhw = hz - ha, nrw = rz - ra;
  {
    // held(i) = cI[i - ha] (-1 before the block, INT_MAX past it), received(j) = cI[nhw + j - ra]
    // (INT_MAX past the block); all loads first
    constexpr int SU = (MERGE_WIN + MERGE_THREADS - 1) / MERGE_THREADS;
    int32_t ti[SU];
    float tv[SU];
#pragma unroll
    for (int u = 0; u < SU; ++u) {
      const int i = threadIdx.x + u * MERGE_THREADS;
      ti[u] = INT32_MAX;
      tv[u] = 0.f;
      if (i < nhw) {
        const int32_t gi = ha + i;
        if (gi < 0) ti[u] = -1;
        else if (gi < kb) { ti[u] = Hi[gi]; tv[u] = Hv[gi]; }
      } else if (i < nhw + nrw) {
        const int32_t gj = ra + (i - nhw);
        if (gj < kb) { ti[u] = Ri[gj]; tv[u] = Rv[gj]; }
      }
    }
#pragma unroll
    for (int u = 0; u < SU; ++u) {
      const int i = threadIdx.x + u * MERGE_THREADS;
      if (i < nhw + nrw && i < MERGE_WIN) {
        cI[i] = ti[u];
        cV[i] = tv[u];
      }
    }
  }
  __syncthreads();
  const int32_t* hI = cI - ha;          // hI[a]: held(a) for a in [ha, hz)
  const int32_t* rI = cI + nhw - ra;    // rI[j]: received(j) for j in [ra, rz)
  const float* hV = cV - ha;
  const float* rV = cV + nhw - ra;
  // exact splits: half the workgroup tests each bracket
  int32_t a0, a1;
  {
    const int half = MERGE_THREADS / 2;
    const bool second = (int)threadIdx.x >= half;
    const int32_t lo = second ? lo1 : lo0, hi = second ? hi1 : hi0, q = second ? Q1 : Q0;
    const int32_t a = lo + ((int)threadIdx.x - (second ? half : 0));
    const bool p = a < hi && hI[a] <= rI[q - a - 1];
    const uint32_t c = popc64(__ballot(p));
    if (lane_id() == 0) scratch[wave_id()] = c;
    __syncthreads();
    int32_t c0 = 0, c1 = 0;
    for (int i = 0; i < MERGE_THREADS / WAVE; ++i) {
      if (i < half / WAVE) c0 += (int32_t)scratch[i];
      else c1 += (int32_t)scratch[i];
    }
    a0 = lo0 + c0;
    a1 = lo1 + c1;
    __syncthreads();
  }
  const int32_t b1 = Q1 - a1;
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
      if (hI[mid] <= rI[q_lo - mid - 1]) lo = mid + 1;
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
      const int32_t hx = hI[a];
      const int32_t rx = rI[bb];
      if (hx <= rx) {
        float v = hV[a];
        if (rx == hx) v = v + rV[bb];
        ei[k] = hx;
        ev[k] = v;
        eok[k] = true;
        ++a;
      } else {
        if (hI[a - 1] != rx) {
          ei[k] = rx;
          ev[k] = rV[bb];
          eok[k] = true;
        }
        ++bb;
      }
      if (eok[k]) {
        ++cnt;
        atomicAdd(&hist[merge_bin<FINE>(mag_key(ev[k]), wbase)], 1u);
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
  flush_hist<MERGE_THREADS>(hist, hist1 + (int64_t)pair * NB1);
  if (FINE) {
    // the tile's keys ordered by fine bin (a counting sort in LDS), for the
    // threshold kernel: in the slot's MERGE_TILE words of U_key, the low
    // FINE_SHIFT bits of each key (uint16, bin order) and then the exclusive
    // prefix of the bin counts (uint16 per bin)
    constexpr int BPT = NB1 / MERGE_THREADS;   // bins per thread, one uint4 of LDS
    static_assert(BPT == 4 && FINE_SHIFT <= 16, "4 bins per thread, keys' low bits in 16 bits");
    uint16_t* __restrict__ SK = reinterpret_cast<uint16_t*>(U_key + ubase);
    uint16_t* __restrict__ PRE = SK + MERGE_TILE;
    const uint4 h4 = reinterpret_cast<const uint4*>(hist)[threadIdx.x];
    const uint32_t hc[BPT] = {h4.x, h4.y, h4.z, h4.w};
    uint32_t tot2;
    // the scan's barriers end the flush's and the write-out's reads
    uint32_t x = block_excl_scan(hc[0] + hc[1] + hc[2] + hc[3], scratch, &tot2);
    uint32_t ex[BPT];
#pragma unroll
    for (int j = 0; j < BPT; ++j) {
      ex[j] = x;
      x += hc[j];
    }
    reinterpret_cast<uint4*>(hist)[threadIdx.x] = make_uint4(ex[0], ex[1], ex[2], ex[3]);
    reinterpret_cast<uint2*>(PRE)[threadIdx.x] = make_uint2(ex[0] | (ex[1] << 16), ex[2] | (ex[3] << 16));
    __syncthreads();
    uint16_t* sk = reinterpret_cast<uint16_t*>(cI);   // the staged indices are written out already
    for (uint32_t k = threadIdx.x; k < tot; k += blockDim.x) {
      const uint32_t key = mag_key(cV[k]);
      const uint32_t pos = atomicAdd(&hist[merge_bin<true>(key, wbase)], 1u);
      sk[pos] = (uint16_t)(key & ((1u << FINE_SHIFT) - 1u));
    }
    __syncthreads();
    const uint32_t* sk2 = reinterpret_cast<const uint32_t*>(sk);
    uint32_t* SK2 = reinterpret_cast<uint32_t*>(SK);
    for (uint32_t k = threadIdx.x; 2 * k < tot; k += blockDim.x) SK2[k] = sk2[k];
  }
}

// ============================================================================ a4: small unions, one workgroup per pair
// When a pair's union fits in LDS (merge_small in common.hpp), one workgroup
// does the merge, the exact threshold and the emit of the tiled path in one
// launch: both blocks are loaded into LDS, merged by merge-path splits
// (SMALL_MP positions per thread; held first on equal indices, the held
// entry carrying held + received and the received one leaving a hole), the
// union compacted in index order over the same LDS, its threshold found on
// a fine level-1 histogram placed from the union's largest key and
// resolve_bin's levels 2 and 3, and its
// entries written in index order: the selected ones into the held block's
// place, the rest into the step's drop list.  The held block is in LDS
// before it is overwritten, and an SRS step never writes a block it
// receives.  The results are the tiled path's: the same sums, selection rule
// and orders.
constexpr int SMALL_MP = SMALL_UNION / SMALL_THREADS;   // merged positions per thread

__global__ __launch_bounds__(SMALL_THREADS) void k_merge_small(int32_t* __restrict__ sp_idx, float* __restrict__ sp_val,
                                                               Pairs PM, int32_t kb, int32_t* __restrict__ drop_idx,
                                                               float* __restrict__ drop_val,
                                                               int32_t* __restrict__ drop_cnt, uint32_t* __restrict__ err) {
  __shared__ int32_t sI[SMALL_UNION];
  __shared__ float sV[SMALL_UNION];
  __shared__ __align__(16) uint32_t h[NB1];
  __shared__ uint32_t scratch[3 * (SMALL_THREADS / WAVE) + 8];
  __shared__ uint32_t s_top;   // the union's largest key
  const uint32_t unit = blockIdx.x;
  const int t = threadIdx.x;
  int64_t hb, rb;
  bool both;
  PM.decode(unit, &hb, &rb, &both);
  const int32_t L2 = 2 * kb;   // <= SMALL_UNION
  {
    // held at [0, kb), received at [kb, 2 kb); every load first
    int32_t ti[SMALL_MP];
    float tv[SMALL_MP];
#pragma unroll
    for (int u = 0; u < SMALL_MP; ++u) {
      const int32_t i = t + u * SMALL_THREADS;
      ti[u] = 0;
      tv[u] = 0.f;
      if (i < L2) {
        const int64_t g = i < kb ? hb * kb + i : rb * kb + (i - kb);
        ti[u] = sp_idx[g];
        tv[u] = sp_val[g];
      }
    }
#pragma unroll
    for (int u = 0; u < SMALL_MP; ++u) {
      const int32_t i = t + u * SMALL_THREADS;
      if (i < L2) {
        sI[i] = ti[u];
        sV[i] = tv[u];
      }
    }
    static_assert(NB1 == 4 * SMALL_THREADS, "one uint4 of the histogram per thread");
    reinterpret_cast<uint4*>(h)[t] = make_uint4(0u, 0u, 0u, 0u);
    if (t == 0) s_top = 0u;
  }
  __syncthreads();
  // held(a) (-1 before the block, INT_MAX past it), received(b) (INT_MAX past it)
  auto hI = [&](int32_t a) { return a < 0 ? -1 : a < kb ? sI[a] : INT32_MAX; };
  auto rI = [&](int32_t b) { return b < kb ? sI[kb + b] : INT32_MAX; };
  int32_t ei[SMALL_MP];
  float ev[SMALL_MP];
  bool eok[SMALL_MP];
  uint32_t cnt = 0;
  const int32_t q_lo = t * SMALL_MP;
  int32_t a = 0, bb = 0;
  if (q_lo < L2) {
    int32_t lo = max(0, q_lo - kb), hi = min(q_lo, kb);
    while (lo < hi) {
      const int32_t mid = (lo + hi) >> 1;
      if (hI(mid) <= rI(q_lo - mid - 1)) lo = mid + 1;
      else hi = mid;
    }
    a = lo;
    bb = q_lo - a;
  }
#pragma unroll
  for (int k = 0; k < SMALL_MP; ++k) {
    eok[k] = false;
    ei[k] = 0;
    ev[k] = 0.f;
    if (q_lo + k < L2) {
      a = min(a, kb);     // only reachable with unsorted input; keeps LDS reads in range
      bb = min(bb, kb);
      const int32_t hx = hI(a), rx = rI(bb);
      if (hx <= rx) {
        float v = a < kb ? sV[a] : 0.f;
        if (rx == hx && bb < kb) v = v + sV[kb + bb];
        ei[k] = hx;
        ev[k] = v;
        eok[k] = true;
        ++a;
      } else {
        if (hI(a - 1) != rx) {
          ei[k] = rx;
          ev[k] = sV[kb + bb];
          eok[k] = true;
        }
        ++bb;
      }
      if (eok[k]) ++cnt;
    }
  }
  {
    uint32_t mk = 0;
#pragma unroll
    for (int k = 0; k < SMALL_MP; ++k) mk = eok[k] ? max(mk, mag_key(ev[k])) : mk;
    mk = wave_incl_max(mk);
    if (lane_id() == WAVE - 1) atomicMax(&s_top, mk);
  }
  // the union, compacted in index order over the blocks (the scan's barriers
  // put every thread past its reads of them)
  uint32_t tot;
  uint32_t pos = block_excl_scan(cnt, scratch, &tot);
#pragma unroll
  for (int k = 0; k < SMALL_MP; ++k) {
    if (eok[k]) {
      sI[pos] = ei[k];
      sV[pos] = ev[k];
      ++pos;
    }
  }
  __syncthreads();
  // the exact threshold: every key >= tge, and the first need_eq with key ==
  // teq.  Level 1 on NB1 fine bins of 2^FINE_SHIFT keys (1/256 binade) from
  // the union's largest key down (the union keeps its larger half, whose keys
  // crowd into a few 1/16-binade bins); keys further down share the lowest
  // bin, and a threshold there takes the 2^D1_SHIFT-key bins instead
  const uint32_t top = s_top >> FINE_SHIFT;
  auto fine_bin = [&](uint32_t key) {
    const uint32_t d = top - (key >> FINE_SHIFT);
    return d >= (uint32_t)NB1 - 1u ? 0u : (uint32_t)NB1 - 1u - d;
  };
  for (uint32_t i = (uint32_t)t; i < tot; i += SMALL_THREADS) atomicAdd(&h[fine_bin(mag_key(sV[i]))], 1u);
  __syncthreads();
  uint32_t T1, above1, cnt1, ok;
  block_select_desc(h, NB1, (uint32_t)kb, scratch, &T1, &above1, &cnt1, &ok);
  uint32_t pfx = top - ((uint32_t)NB1 - 1u - T1);
  int S = FINE_SHIFT;
  if (!ok || T1 == 0u) {   // uniform: the threshold below the window
    __syncthreads();
    reinterpret_cast<uint4*>(h)[t] = make_uint4(0u, 0u, 0u, 0u);
    __syncthreads();
    for (uint32_t i = (uint32_t)t; i < tot; i += SMALL_THREADS) atomicAdd(&h[mag_key(sV[i]) >> D1_SHIFT], 1u);
    __syncthreads();
    block_select_desc(h, NB1, (uint32_t)kb, scratch, &T1, &above1, &cnt1, &ok);
    pfx = T1;
    S = D1_SHIFT;
  }
  if (!ok && t == 0) atomicOr(err, ERR_COUNT);
  const uint32_t need1 = ok ? (uint32_t)kb - above1 : 0u;
  uint32_t tge, teq, need_eq;
  resolve_bin(pfx, S, need1, cnt1, h, scratch, err,
              [&](auto f) {
                for (uint32_t i = (uint32_t)t; i < tot; i += SMALL_THREADS) {
                  const uint32_t key = mag_key(sV[i]);
                  if ((key >> S) == pfx) f(key);
                }
              },
              tge, teq, need_eq);
  // emit: each thread's SMALL_MP consecutive union entries, in index order
  const uint32_t e0 = min((uint32_t)q_lo, tot), e1 = min(e0 + (uint32_t)SMALL_MP, tot);
  uint32_t x3[3] = {0u, 0u, 0u}, t3[3];
  for (uint32_t i = e0; i < e1; ++i) {
    const uint32_t key = mag_key(sV[i]);
    x3[0] += key >= tge ? 1u : 0u;
    x3[1] += need_eq != 0u && key == teq ? 1u : 0u;
  }
  block_excl_scan3(x3, scratch, t3);
  uint32_t run_g = x3[0], run_e = x3[1];
  const int64_t o = hb * kb, o2 = both ? rb * kb : -1;
  for (uint32_t i = e0; i < e1; ++i) {
    const int32_t ix = sI[i];
    const float vx = sV[i];
    const uint32_t key = mag_key(vx);
    const bool is_ge = key >= tge;
    const bool is_eq = need_eq != 0u && key == teq;
    const uint32_t sel_before = run_g + (run_e < need_eq ? run_e : need_eq);
    if (is_ge || (is_eq && run_e < need_eq)) {
      if (sel_before < (uint32_t)kb) {
        sp_idx[o + sel_before] = ix;
        sp_val[o + sel_before] = vx;
        if (o2 >= 0) {
          sp_idx[o2 + sel_before] = ix;
          sp_val[o2 + sel_before] = vx;
        }
      } else {
        atomicOr(err, ERR_COUNT_POS);
      }
    } else {
      const uint32_t dpos = i - sel_before;
      if (dpos < (uint32_t)kb) {
        drop_idx[(int64_t)unit * kb + dpos] = ix;
        drop_val[(int64_t)unit * kb + dpos] = vx;
      } else {
        atomicOr(err, ERR_COUNT_DROP);
      }
    }
    run_g += is_ge ? 1u : 0u;
    run_e += is_eq ? 1u : 0u;
  }
  if (t == 0) {
    if (t3[0] + (t3[1] < need_eq ? t3[1] : need_eq) != (uint32_t)kb) atomicOr(err, ERR_COUNT_SUM);
    drop_cnt[unit] = (int32_t)(tot - (uint32_t)kb);
  }
}

// ============================================================================ launchers
hipError_t launch_merge(const int32_t* sp_idx, const float* sp_val, const Pairs& PM, int64_t npairs, int32_t kb,
                        int32_t tiles_per_pair, uint32_t* hist1, uint32_t* state, uint32_t* slot_cnt, int32_t* U_idx,
                        float* U_val, uint32_t* U_key, hipStream_t s) {
  const dim3 grid((unsigned)(npairs * tiles_per_pair));
  if (merge_fine(kb))
    hipLaunchKernelGGL(k_merge<true>, grid, dim3(MERGE_THREADS), 0, s, sp_idx, sp_val, PM, kb, tiles_per_pair, hist1,
                       state, slot_cnt, U_idx, U_val, U_key);
  else
    hipLaunchKernelGGL(k_merge<false>, grid, dim3(MERGE_THREADS), 0, s, sp_idx, sp_val, PM, kb, tiles_per_pair, hist1,
                       state, slot_cnt, U_idx, U_val, U_key);
  return hipGetLastError();
}

hipError_t launch_merge_small(int32_t* sp_idx, float* sp_val, const Pairs& PM, int64_t npairs, int32_t kb,
                              int32_t* drop_idx, float* drop_val, int32_t* drop_cnt, uint32_t* err, hipStream_t s) {
  if (!merge_small(kb)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_merge_small, dim3((unsigned)npairs), dim3(SMALL_THREADS), 0, s, sp_idx, sp_val, PM, kb, drop_idx,
                     drop_val, drop_cnt, err);
  return hipGetLastError();
}

}  // namespace spardl
