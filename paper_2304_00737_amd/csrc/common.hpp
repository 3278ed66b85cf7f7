// Device helpers shared by the SparDL kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace spardl {

// ---------------------------------------------------------------- radix digits
// The 31-bit magnitude key |v| (fp32 bits without the sign) is selected on in
// three digits: bits 30..19 (4096 bins), 18..8 (2048 bins), 7..0 (256 bins).
constexpr int D1_SHIFT = 19;
constexpr int NB1 = 4096;
constexpr uint32_t LIST_CHUNK = 4096;    // list entries per workgroup of the B-SAG list selections
constexpr uint32_t UNION_TILE = 16384;   // indices per workgroup of the B-SAG union
constexpr int D2_SHIFT = 8;
constexpr int NB2 = 2048;
constexpr int NB3 = 256;

// ---------------------------------------------------------------- tiling
// Streaming kernels are one-shot workgroups over small contiguous tiles,
// dispatched in address order (this keeps DRAM pages open and beats both
// larger per-lane batches and workgroups that walk long ranges).
constexpr int WAVE = 64;
constexpr int ADD_F4 = 2;                        // float4 per lane per array in the residual add
constexpr int ADD_TILE = 256 * ADD_F4 * 4;       // elements per residual-add workgroup
constexpr int SLOT = 4096;                       // elements per candidate slot (one collect workgroup)
constexpr int MERGE_THREADS = 1024;               // a merge tile's serial steps (split search, merge,
constexpr int MERGE_PER_THREAD = 4;                // histogram flush, bin sort) shrink with the positions per thread
constexpr int MERGE_TILE = MERGE_THREADS * MERGE_PER_THREAD;   // merged positions per workgroup
constexpr int DENSE_TILE = 8192;                 // output elements per densify workgroup (an LDS image)
constexpr uint32_t HCOPIES_MIN = 4;               // level-1 histogram copies per block (spread the flush atomics)
constexpr uint32_t HCOPIES_MAX = 32;

// ---------------------------------------------------------------- merge threshold
// A merge's union (two index-sorted top-k blocks, summed on shared indices)
// keeps half its entries, whose keys crowd just above the blocks' own
// thresholds: a level-1 bin of 2^D1_SHIFT keys (1/16 binade) can hold half
// the union.  Unions of up to MT_SLOTS slots therefore take a finer level 1:
// NB1 bins of 2^FINE_SHIFT keys (1/256 binade, a window of 16 binades)
// centred on the two blocks' median keys, each the median of the block's
// leading FINE_SAMPLE entries to 1/8 binade (the union keeps its larger half,
// so its threshold lies near them; a median is not moved by a few entries
// that nearly cancelled); keys outside the window are counted in its first or
// last bin.  If the threshold falls in one of those two bins the threshold
// kernel builds the 2^D1_SHIFT-key histogram itself (exact either way, so the
// centre only needs to be close).
constexpr int MT_SLOTS = 1024;                   // merge slots per unit of the one-workgroup merge threshold
constexpr int FINE_SHIFT = 15;
constexpr uint32_t FINE_BELOW = NB1 / 2;        // fine bins from the window's first to its centre (8 binades)
constexpr int FINE_SAMPLE = 64;                  // leading entries of each block sampled for the window
constexpr int FINE_CENTRE_BIT = 20;              // the sampled medians' lowest key bit (1/8 binade)
// Pairs whose union fits in one workgroup's LDS take one launch for the
// merge, threshold and emit (k_merge_small).
constexpr int SMALL_THREADS = 1024;
constexpr int SMALL_UNION = 8192;                // union entries (both blocks) held in LDS
__host__ __device__ __forceinline__ bool merge_small(int64_t kb) { return 2 * kb <= (int64_t)SMALL_UNION; }
__host__ __device__ __forceinline__ bool merge_fine(int64_t kb) { return 2 * kb <= (int64_t)MT_SLOTS * MERGE_TILE; }

// ---------------------------------------------------------------- state words
// Per selection unit (a (worker, block) pair or a merge pair), 16 u32:
enum : int {
  ST_T1 = 0,        // level-1 threshold bin (its key prefix; see ST_SHIFT)
  ST_ABOVE1 = 1,    // entries in bins above ST_T1
  ST_NEED1 = 2,     // entries still needed from bin ST_T1
  ST_CNT1 = 3,      // entries in bin ST_T1
  ST_TGE = 4,       // every candidate with key >= ST_TGE is selected
  ST_TEQ = 5,       // ... and the first ST_NEEDEQ (by index) with key == ST_TEQ
  ST_NEEDEQ = 6,
  ST_SPECOK = 7,    // block top-k: the fused add's speculative candidates cover the threshold bin
  ST_HTOT = 8,      // large-unit threshold: entries in the merge union's histogram
  ST_PRE23 = 9,     // ... the key bits fixed by level 2 (all but the last digit's)
  ST_NEED2 = 10,    // ... entries still needed from that level-2 bin
  ST_STAGE = 11,    // ... 2 while level 3 is still needed, else 0
  ST_WBASE = 12,    // merge: first fine key bin (key >> FINE_SHIFT) of the union's level-1 histogram window
  ST_SHIFT = 14,    // block top-k and staged threshold: the level-1 bin is the keys k with k >> ST_SHIFT == ST_T1
  ST_WORDS = 16
};

constexpr uint32_t ERR_COUNT = 2u;            // a selection could not find its threshold
constexpr uint32_t ERR_COUNT_L23 = 2u | 4u;   // ... at level 2 or 3
constexpr uint32_t ERR_COUNT_POS = 2u | 8u;   // an emitted position fell outside [0, k_blk)
constexpr uint32_t ERR_COUNT_DROP = 2u | 16u; // a drop position fell outside [0, k_blk)
constexpr uint32_t ERR_COUNT_SUM = 2u | 32u;  // the emitted selection does not have k_blk entries
constexpr uint32_t ERR_DROPS = 64u;           // a drop list of the fused collection is not an index-sorted
                                              // list inside its block

// ---------------------------------------------------------------- deferred residual collection
// Per (worker, block) the block top-k keeps its selection rule for the
// residual collection that a later fused residual add applies: it selected
// every key >= KEEP_TGE and, when KEEP_NEEDEQ != 0, the keys == KEEP_TEQ
// whose index is at most KEEP_CUT (ties are taken in index order).
enum KeepWord : int { KEEP_TGE = 0, KEEP_TEQ = 1, KEEP_NEEDEQ = 2, KEEP_CUT = 3, KEEP_WORDS = 4 };
constexpr int COLLECT_MAX_STEPS = 16;   // SRS steps the fused collection takes (P <= 2^16)

__device__ __forceinline__ uint32_t mag_key(float v) { return __float_as_uint(v) & 0x7FFFFFFFu; }

__host__ __device__ __forceinline__ int64_t blk_start(int64_t b, int64_t n, int64_t P) {
  return (b * n) / P;
}

// The P blocks of a row of n < 2^31 elements, block b = [start(b), start(b+1))
// with start(b) = floor(b n / P).  With q = n / P and r = n % P supplied by the
// host, start(b) = b q + floor(b r / P) takes 32-bit arithmetic only when
// P < 2^16 (b r < P^2 < 2^32); kernels index everything in 32 bits so that no
// 64-bit division (a long scalar sequence per wave) precedes their loads.
struct Blocks {
  uint32_t n, P, q, r;
  __device__ __forceinline__ uint32_t start(uint32_t b) const {
    if (P < 65536u) return b * q + (b * r) / P;
    return (uint32_t)(((uint64_t)b * n) / P);
  }
  // block containing element x < n
  __device__ __forceinline__ uint32_t of(uint32_t x) const {
    uint32_t b = x / q;   // q >= 1; start(b) >= b q, so this never undershoots
    if (b > P - 1u) b = P - 1u;
    while (b > 0u && start(b) > x) --b;
    while (b + 1u < P && start(b + 1u) <= x) ++b;
    return b;
  }
};

inline Blocks make_blocks(int64_t n, int32_t P) {
  return Blocks{(uint32_t)n, (uint32_t)P, (uint32_t)(n / P), (uint32_t)(n % P)};
}

// Tiles of the fused residual add and slots of the block top-k start at a
// block's aligned origin, its first element rounded down to a multiple of 32
// (128 bytes): every tile and slot after a block's first then starts on a
// 128-byte boundary of a row that does, and the first is short by the lead.
__host__ __device__ __forceinline__ uint32_t block_lead(uint32_t s) { return s & 31u; }
__host__ __device__ __forceinline__ uint32_t block_origin(uint32_t s) { return s & ~31u; }
// Tiles (or slots of `len` elements) a block of up to maxlen elements spans from its origin.
__host__ __device__ __forceinline__ int64_t spans_per_block(int64_t maxlen, int64_t len) {
  return (maxlen + 31 + len - 1) / len;
}
__host__ __device__ __forceinline__ int64_t add_tiles_per_block(int64_t maxlen) {
  return spans_per_block(maxlen, ADD_TILE);
}

// Level-1 histogram copies of each of the P blocks of a row of n elements:
// every add tile flushes its histogram into copy (workgroup mod copies), and
// the flushes into one copy serialise on its words, so a block has a copy per
// ~512 of its add tiles (a power of two in [HCOPIES_MIN, HCOPIES_MAX]); the
// level-1 select sums them.  Other writers use the first HCOPIES_MIN copies.
__host__ __device__ inline uint32_t hist_copies_for(int64_t n, int64_t P) {
  const int64_t tiles = add_tiles_per_block((n + P - 1) / P);
  uint32_t c = HCOPIES_MIN;
  while (c < HCOPIES_MAX && (int64_t)c * 512 < tiles) c *= 2;
  return c;
}

// Selection units of a block top-k call over rows (workers) w0, w0 + 1, ...:
// unit u selects in row u / m the block (d + u % m + (rel ? w : 0)) mod P,
// w = w0 + u / m being the worker.  All blocks of all rows: m = P, d = 0,
// rel = 0, so unit = row * P + block.  The bag a worker sends at one SRS step:
// m = bag size, d = distance, rel = 1.
struct Units {
  uint32_t m, d, rel, w0;
  __device__ __forceinline__ void decode(uint32_t u, uint32_t P, uint32_t* row, uint32_t* b) const {
    const uint32_t r = u / m;
    *row = r;
    *b = (d + (u - r * m) + (rel ? w0 + r : 0u)) % P;
  }
  // row * P + block: where the unit's per-block arrays live (histograms,
  // speculation words, selection state, slot counts), the same place for
  // every map, so a selection finds what the fused add left for its block
  __device__ __forceinline__ uint32_t canon(uint32_t u, uint32_t P) const {
    uint32_t r, b;
    decode(u, P, &r, &b);
    return r * P + b;
  }
};

inline Units all_blocks(int32_t P) { return Units{(uint32_t)P, 0u, 0u, 0u}; }

// Pairs of one merge call.  Pair p adds the received block into the held
// block (both named by their block number row * nb + b in sp) and keeps the
// top k_blk in the held block and, if `both`, in the received one too.
//  SRS step (kind 0, nb = P workers): pair p = (w, t), held = sp[w][b],
//    received = sp[(w - dist) mod P][b], b = (w + t) mod P, t < m.
//  R-SAG exchange t (kind 1, nb = Q): pair p = (j, q); team X = j with a 0
//    bit inserted at bit t, team Y = X + 2^t; held = sp[X Q + q][q],
//    received = sp[Y Q + q][q], and both keep the result.
//  SRS step of every team at once (kind 2, nb = Q workers per team): pair
//    p = tau Q m + (w, t) is the kind-0 pair (w, t) of team tau, on the
//    team's rows tau Q .. tau Q + Q - 1.
struct Pairs {
  uint32_t kind, nb, m, dist, t;
  __device__ __forceinline__ void decode(uint32_t p, int64_t* held, int64_t* recv, bool* both) const {
    if (kind != 1u) {
      const uint32_t team = kind == 2u ? p / (nb * m) : 0u;
      p -= team * nb * m;
      const uint32_t w = p / m, tt = p - w * m;
      const uint32_t b = (w + tt) % nb, src = (w + nb - dist) % nb;
      *held = (int64_t)(team * nb + w) * nb + b;
      *recv = (int64_t)(team * nb + src) * nb + b;
      *both = false;
    } else {
      const uint32_t j = p / nb, q = p - j * nb;
      const uint32_t lowmask = (1u << t) - 1u;
      const uint32_t X = ((j & ~lowmask) << 1) | (j & lowmask), Y = X | (1u << t);
      *held = (int64_t)(X * nb + q) * nb + q;
      *recv = (int64_t)(Y * nb + q) * nb + q;
      *both = true;
    }
  }
};

inline Pairs srs_pairs(int32_t P, int32_t m, int32_t dist) {
  return Pairs{0u, (uint32_t)P, (uint32_t)m, (uint32_t)dist, 0u};
}
inline Pairs rsag_pairs(int32_t Q, int32_t t) { return Pairs{1u, (uint32_t)Q, 0u, 0u, (uint32_t)t}; }
inline Pairs team_srs_pairs(int32_t Q, int32_t m, int32_t dist) {
  return Pairs{2u, (uint32_t)Q, (uint32_t)m, (uint32_t)dist, 0u};
}

__device__ __forceinline__ int lane_id() { return threadIdx.x & (WAVE - 1); }
__device__ __forceinline__ int wave_id() { return threadIdx.x / WAVE; }

__device__ __forceinline__ uint32_t popc64(uint64_t m) { return (uint32_t)__popcll(m); }

// Inclusive prefix sum across the 64 lanes of a wave.
// Wave-wide inclusive scans in DPP: Hillis-Steele steps of 1, 2, 4 and 8
// lanes inside each row of 16 (a lane with no source in its row takes 0, the
// identity of both operations), then the totals of the rows before each row
// (v_readlane) added in.  Every lane of the wave must be active.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_shr(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}
constexpr int DPP_ROW_SHR1 = 0x111, DPP_ROW_SHR2 = 0x112, DPP_ROW_SHR4 = 0x114, DPP_ROW_SHR8 = 0x118;

__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v) {
  v += dpp_shr<DPP_ROW_SHR1>(v);
  v += dpp_shr<DPP_ROW_SHR2>(v);
  v += dpp_shr<DPP_ROW_SHR4>(v);
  v += dpp_shr<DPP_ROW_SHR8>(v);
  const uint32_t r0 = (uint32_t)__builtin_amdgcn_readlane((int)v, 15);
  const uint32_t r1 = r0 + (uint32_t)__builtin_amdgcn_readlane((int)v, 31);
  const uint32_t r2 = r1 + (uint32_t)__builtin_amdgcn_readlane((int)v, 47);
  const int row = lane_id() >> 4;
  return v + (row == 0 ? 0u : row == 1 ? r0 : row == 2 ? r1 : r2);
}

__device__ __forceinline__ uint32_t wave_incl_max(uint32_t v) {
  v = max(v, dpp_shr<DPP_ROW_SHR1>(v));
  v = max(v, dpp_shr<DPP_ROW_SHR2>(v));
  v = max(v, dpp_shr<DPP_ROW_SHR4>(v));
  v = max(v, dpp_shr<DPP_ROW_SHR8>(v));
  const uint32_t r0 = (uint32_t)__builtin_amdgcn_readlane((int)v, 15);
  const uint32_t r1 = max(r0, (uint32_t)__builtin_amdgcn_readlane((int)v, 31));
  const uint32_t r2 = max(r1, (uint32_t)__builtin_amdgcn_readlane((int)v, 47));
  const int row = lane_id() >> 4;
  return max(v, row == 0 ? 0u : row == 1 ? r0 : row == 2 ? r1 : r2);
}

__device__ __forceinline__ uint32_t wave_sum(uint32_t v) {
#pragma unroll
  for (int d = WAVE / 2; d > 0; d >>= 1) v += __shfl_xor(v, d, WAVE);
  return v;
}

// Exclusive prefix sum of one value per thread over the workgroup, in thread
// order.  `scratch` needs blockDim/64 + 1 words of LDS.  Returns the exclusive
// prefix and writes the workgroup total to *total.  Contains barriers.
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t* scratch, uint32_t* total) {
  const int nw = blockDim.x / WAVE;
  const uint32_t incl = wave_incl_scan(v);
  if (lane_id() == WAVE - 1) scratch[wave_id()] = incl;
  __syncthreads();
  // every wave scans the wave totals itself (one lane per wave, at most 16)
  const int l = lane_id();
  const uint32_t x = l < nw ? scratch[l] : 0u;
  const uint32_t xi = wave_incl_scan(x);
  const uint32_t before = (uint32_t)__builtin_amdgcn_readlane((int)(xi - x), wave_id());
  *total = (uint32_t)__builtin_amdgcn_readlane((int)xi, WAVE - 1);
  __syncthreads();   // the caller may write scratch next
  return before + incl - v;
}

// Three exclusive prefix sums at once (one set of barriers): v[q] becomes
// its prefix and total[q] the workgroup total.  `scratch` needs
// 3 blockDim/64 words of LDS.  Contains barriers.
__device__ __forceinline__ void block_excl_scan3(uint32_t (&v)[3], uint32_t* scratch, uint32_t (&total)[3]) {
  const int nw = blockDim.x / WAVE, l = lane_id(), w = wave_id();
  uint32_t incl[3];
#pragma unroll
  for (int q = 0; q < 3; ++q) {
    incl[q] = wave_incl_scan(v[q]);
    if (l == WAVE - 1) scratch[q * nw + w] = incl[q];
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < 3; ++q) {
    const uint32_t x = l < nw ? scratch[q * nw + l] : 0u;
    const uint32_t xi = wave_incl_scan(x);
    const uint32_t before = (uint32_t)__builtin_amdgcn_readlane((int)(xi - x), w);
    total[q] = (uint32_t)__builtin_amdgcn_readlane((int)xi, WAVE - 1);
    v[q] = before + incl[q] - v[q];
  }
  __syncthreads();   // the caller may write scratch next
}

// Select on a histogram in descending bin order: find bin T such that
// count(bins > T) < need <= count(bins >= T).  hist is in LDS with nb bins.
// Every thread gets the answer.  `scratch` needs blockDim/64 + 4 words of LDS.
// If the histogram holds fewer than `need` entries, *ok is 0 and T = 0.
// *total (optional) receives the number of entries in the histogram.
__device__ __forceinline__ void block_select_desc(const uint32_t* hist, int nb, uint32_t need,
                                                  uint32_t* scratch, uint32_t* T, uint32_t* above,
                                                  uint32_t* cnt, uint32_t* ok, uint32_t* total = nullptr) {
  const int nt = blockDim.x;
  const int per = (nb + nt - 1) / nt;
  // thread t owns bins [nb - per (t+1), nb - per t) (the highest bins go to thread 0)
  const int hi = nb - per * (int)threadIdx.x;
  const int lo = hi - per;
  uint32_t s = 0;
  for (int bin = hi - 1; bin >= lo && bin >= 0; --bin) s += hist[bin];
  uint32_t tot;
  uint32_t ex = block_excl_scan(s, scratch, &tot);
  if (total) *total = tot;
  const int nw = nt / WAVE;
  // exactly one thread's bins hold the crossing when the histogram holds need >= 1 entries
  *ok = need != 0u && tot >= need ? 1u : 0u;
  if (ex < need && ex + s >= need) {
    uint32_t run = ex;
    for (int bin = hi - 1; bin >= lo && bin >= 0; --bin) {
      uint32_t h = hist[bin];
      if (run + h >= need) {
        scratch[nw + 2] = (uint32_t)bin;
        scratch[nw + 3] = run;
        break;
      }
      run += h;
    }
  }
  __syncthreads();
  if (*ok) {
    *T = scratch[nw + 2];
    *above = scratch[nw + 3];
    *cnt = hist[*T];
  } else {
    *T = 0;
    *above = 0;
    *cnt = 0;
  }
  __syncthreads();
}

// Copy count words from global memory to LDS with every load issued before
// the first LDS write (one memory round trip instead of one per iteration).
// PER >= ceil(count / blockDim.x) must hold.  No barrier included.
template <int PER>
__device__ __forceinline__ void g2lds(uint32_t* lds, const uint32_t* __restrict__ g, int count) {
  uint32_t r[PER];
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int i = threadIdx.x + u * blockDim.x;
    r[u] = i < count ? g[i] : 0u;
  }
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int i = threadIdx.x + u * blockDim.x;
    if (i < count) lds[i] = r[u];
  }
}

// ---------------------------------------------------------------- cooperative searches
// Number of leading positions p in [lo, hi) for which the monotone predicate
// pred(p) holds (true ... true false ... false), found by the whole workgroup
// with a (blockDim+1)-ary search: every round tests blockDim points at once,
// so a range of 2^15 needs two rounds of loads.  `cnt` needs blockDim/64 + 1
// words of LDS.  Contains barriers; every thread gets the answer.
template <typename Pred>
__device__ __forceinline__ int32_t wg_partition_point(int32_t lo, int32_t hi, Pred pred, uint32_t* cnt) {
  const int nt = blockDim.x;
  const int nw = nt / WAVE;
  while (hi > lo) {
    const int32_t S = hi - lo;
    int32_t p;
    bool active;
    if (S <= nt) {
      p = lo + (int32_t)threadIdx.x;
      active = (int32_t)threadIdx.x < S;
    } else {
      p = lo + (int32_t)(((int64_t)S * (threadIdx.x + 1)) / (nt + 1));
      active = true;
    }
    const bool t = active && pred(p);
    const uint64_t m = __ballot(t);
    if (lane_id() == 0) cnt[wave_id()] = popc64(m);
    __syncthreads();
    int32_t c = 0;
    for (int i = 0; i < nw; ++i) c += (int32_t)cnt[i];
    __syncthreads();
    if (S <= nt) {
      lo += c;
      hi = lo;
    } else {
      const int32_t new_lo = c == 0 ? lo : lo + (int32_t)(((int64_t)S * c) / (nt + 1)) + 1;
      const int32_t new_hi = c == nt ? hi : lo + (int32_t)(((int64_t)S * (c + 1)) / (nt + 1));
      lo = new_lo;
      hi = new_hi;
    }
  }
  return lo;
}

// Two independent partition points found together: every round tests
// blockDim points of each range, so both searches share their rounds of loads
// and barriers.  `cnt` needs 2 (blockDim/64) words of LDS.
template <typename Pred0, typename Pred1>
__device__ __forceinline__ void wg_partition_point2(int32_t lo0, int32_t hi0, Pred0 pred0, int32_t lo1, int32_t hi1,
                                                    Pred1 pred1, uint32_t* cnt, int32_t* r0, int32_t* r1) {
  const int nt = blockDim.x;
  const int nw = nt / WAVE;
  auto probe = [&](int32_t lo, int32_t hi, int32_t* p, bool* active) {
    const int32_t S = hi - lo;
    if (S <= nt) {
      *p = lo + (int32_t)threadIdx.x;
      *active = (int32_t)threadIdx.x < S;
    } else {
      *p = lo + (int32_t)(((int64_t)S * (threadIdx.x + 1)) / (nt + 1));
      *active = true;
    }
  };
  auto narrow = [&](int32_t* lo, int32_t* hi, int32_t c) {
    const int32_t S = *hi - *lo;
    if (S <= nt) {
      *lo += c;
      *hi = *lo;
    } else {
      const int32_t new_lo = c == 0 ? *lo : *lo + (int32_t)(((int64_t)S * c) / (nt + 1)) + 1;
      const int32_t new_hi = c == nt ? *hi : *lo + (int32_t)(((int64_t)S * (c + 1)) / (nt + 1));
      *lo = new_lo;
      *hi = new_hi;
    }
  };
  while (hi0 > lo0 || hi1 > lo1) {
    int32_t p0 = 0, p1 = 0;
    bool a0 = false, a1 = false;
    if (hi0 > lo0) probe(lo0, hi0, &p0, &a0);
    if (hi1 > lo1) probe(lo1, hi1, &p1, &a1);
    const bool t0 = a0 && pred0(p0);
    const bool t1 = a1 && pred1(p1);
    const uint64_t m0 = __ballot(t0), m1 = __ballot(t1);
    if (lane_id() == 0) {
      cnt[wave_id()] = popc64(m0);
      cnt[nw + wave_id()] = popc64(m1);
    }
    __syncthreads();
    int32_t c0 = 0, c1 = 0;
    for (int i = 0; i < nw; ++i) {
      c0 += (int32_t)cnt[i];
      c1 += (int32_t)cnt[nw + i];
    }
    __syncthreads();
    if (hi0 > lo0) narrow(&lo0, &hi0, c0);
    if (hi1 > lo1) narrow(&lo1, &hi1, c1);
  }
  *r0 = lo0;
  *r1 = lo1;
}

// First position j in [0, len) with a[j] >= x (len if none); a sorted ascending.
__device__ __forceinline__ int32_t wg_lower_bound(const int32_t* __restrict__ a, int32_t len, int64_t x,
                                                  uint32_t* cnt) {
  return wg_partition_point(0, len, [&](int32_t p) { return (int64_t)a[p] < x; }, cnt);
}

}  // namespace spardl
