// The B-SAG exchange with its compression-ratio controller (Sec. III-D,
// Algorithm 2) and the receipts of the lazy-sparsification step (Sec. III-B
// "Optimization for SRS", Algorithm 1) for gfx950.

#include "device.hpp"
#include "launch.hpp"

#include <algorithm>

namespace spardl {

// ============================================================================ B-SAG
// Spar-All-Gather across d teams, Bruck form, and its compression-ratio
// controller (Sec. III-D, Algorithm 2).  Per block q of a team's Q blocks the
// workspace keeps the controller state (h, step, flag in double precision, the
// last union size N) and the count used at this step.

// Algorithm 2, one thread per block: update step and h from the last N, keep
// h in [L/d, L], count = floor(h + 1/2) clamped to [1, L].
__global__ __launch_bounds__(64) void k_bsag_control(uint32_t Q, uint32_t L, uint32_t d, double* __restrict__ H,
                                                     double* __restrict__ S, uint32_t* __restrict__ F,
                                                     const uint32_t* __restrict__ N, uint32_t* __restrict__ cnt) {
  for (uint32_t q = blockIdx.x * 64u + threadIdx.x; q < Q; q += gridDim.x * 64u) {
    double h = H[q], step = S[q];
    uint32_t flag = F[q];
    const bool too_many = N[q] > L;
    if (too_many != (step > 0.0)) {
      if (flag) {
        step = step * 2.0;
        flag = 0u;
      } else {
        flag = 1u;
      }
    } else {
      step = -step * 0.5;
      flag = 0u;
    }
    const double lo = (double)L / (double)d;
    h = h + step;
    h = h < lo ? lo : h;
    h = h > (double)L ? (double)L : h;
    double c = floor(h + 0.5);
    c = c < 1.0 ? 1.0 : c;
    c = c > (double)L ? (double)L : c;
    H[q] = h;
    S[q] = step;
    F[q] = flag;
    cnt[q] = (uint32_t)c;
  }
}

__global__ __launch_bounds__(64) void k_bsag_init(uint32_t Q, double h0, double step0, double* __restrict__ H,
                                                  double* __restrict__ S, uint32_t* __restrict__ F,
                                                  uint32_t* __restrict__ N) {
  for (uint32_t q = blockIdx.x * 64u + threadIdx.x; q < Q; q += gridDim.x * 64u) {
    H[q] = h0;
    S[q] = step0;
    F[q] = 0u;
    N[q] = 0u;
  }
}

// ---- top-c selection of many sparse lists (each sorted by index), spread
// over workgroups: a chunked level-1 histogram, one workgroup per list for
// the threshold (levels 2-3 scan the list for the threshold bin's keys),
// chunked counts, chunked emit in index order.  ListSel says where list i
// lives, its length, how many entries it keeps and where the kept (and then
// sentinels -- index INT32_MAX, value 0 -- up to `pad`) and dropped entries go.

struct ListDesc {
  const int32_t* ii;
  const float* iv;
  uint32_t len, c, pad;
  int32_t* ki;
  float* kv;
  int32_t* di;
  float* dv;
  int32_t* dcnt;
};

struct ListSel {
  uint32_t mode;       // 0: top-h of the held blocks, list = worker; 1: final top-L, list = block
  uint32_t Q, kb, cap;  // cap = d k_blk
  int32_t* sp_idx;
  float* sp_val;
  const uint32_t* cnt;  // top-h count per block
  const uint32_t* N;    // union size per block
  int32_t *kept_i, *drop_i, *U_i, *fd_i;
  float *kept_v, *drop_v, *U_v, *fd_v;
  int32_t *drop_cnt, *fd_cnt;
  __device__ __forceinline__ ListDesc desc(uint32_t i) const {
    ListDesc D;
    if (mode == 0u) {
      const uint32_t q = i % Q;
      const int64_t in = ((int64_t)i * Q + q) * kb, o = (int64_t)i * kb;
      D.ii = sp_idx + in;
      D.iv = sp_val + in;
      D.len = kb;
      D.c = min(cnt[q], kb);
      D.pad = 0u;
      D.ki = kept_i + o;
      D.kv = kept_v + o;
      D.di = drop_i + o;
      D.dv = drop_v + o;
      D.dcnt = drop_cnt + i;
    } else {
      const int64_t in = (int64_t)i * cap, o = ((int64_t)i * Q + i) * kb;
      D.ii = U_i + in;
      D.iv = U_v + in;
      D.len = min(N[i], cap);
      D.c = kb;
      D.pad = kb;
      D.ki = sp_idx + o;
      D.kv = sp_val + o;
      D.di = fd_i + in;
      D.dv = fd_v + in;
      D.dcnt = fd_cnt + i;
    }
    return D;
  }
};

__global__ __launch_bounds__(256) void k_lsel_hist(ListSel S, uint32_t nch, uint32_t* __restrict__ hist) {
  __shared__ __align__(16) uint32_t h[NB1];
  const uint32_t i = blockIdx.x / nch, k = blockIdx.x % nch;
  const ListDesc D = S.desc(i);
  const uint32_t j0 = k * LIST_CHUNK;
  if (D.c >= D.len || j0 >= D.len) return;   // uniform: nothing to select, or no entries here
  const uint32_t j1 = min(D.len, j0 + LIST_CHUNK);
  for (int b = threadIdx.x; b < NB1; b += 256) h[b] = 0u;
  __syncthreads();
  for (uint32_t j = j0 + threadIdx.x; j < j1; j += 256u) atomicAdd(&h[mag_key(D.iv[j]) >> D1_SHIFT], 1u);
  __syncthreads();
  flush_hist<256>(h, hist + (int64_t)i * NB1);
}

// st[4 i ..]: key bound tge, tie key teq, ties to keep need_eq, entries kept
constexpr int LSEL_R = 8;   // list entries per thread in flight in the threshold's scans
__global__ __launch_bounds__(1024) void k_lsel_level(ListSel S, uint32_t* __restrict__ hist,
                                                     uint32_t* __restrict__ st, uint32_t* __restrict__ err) {
  __shared__ uint32_t h[NB1];
  __shared__ uint32_t scratch[32];
  constexpr uint32_t NT = 1024;
  const uint32_t i = blockIdx.x;
  const ListDesc D = S.desc(i);
  uint32_t tge = 0u, teq = 0u, need_eq = 0u;   // keep everything unless a selection is needed
  if (D.c < D.len) {
    uint32_t* __restrict__ H = hist + (int64_t)i * NB1;
    for (uint32_t b = threadIdx.x; b < NB1; b += NT) {
      h[b] = H[b];
      H[b] = 0u;   // histograms rest at zero
    }
    __syncthreads();
    uint32_t T1, above1, cnt1, ok;
    block_select_desc(h, NB1, D.c, scratch, &T1, &above1, &cnt1, &ok);
    if (!ok) {
      if (threadIdx.x == 0) atomicOr(err, ERR_COUNT);
    } else {
      resolve_low_digits(T1, D.c - above1, cnt1, h, scratch, err,
                         [&](auto f) {   // LSEL_R loads per thread in flight
                           for (uint32_t j0 = 0; j0 < D.len; j0 += NT * LSEL_R) {
                             float v[LSEL_R];
#pragma unroll
                             for (int r = 0; r < LSEL_R; ++r) {
                               const uint32_t j = j0 + (uint32_t)r * NT + threadIdx.x;
                               v[r] = j < D.len ? D.iv[j] : 0.f;
                             }
#pragma unroll
                             for (int r = 0; r < LSEL_R; ++r) {
                               const uint32_t key = mag_key(v[r]);
                               if (j0 + (uint32_t)r * NT + threadIdx.x < D.len && (key >> D1_SHIFT) == T1) f(key);
                             }
                           }
                         },
                         tge, teq, need_eq);
    }
  }
  if (threadIdx.x == 0) {
    st[4 * i + 0] = tge;
    st[4 * i + 1] = teq;
    st[4 * i + 2] = need_eq;
    st[4 * i + 3] = min(D.c, D.len);
  }
}

__device__ __forceinline__ uint32_t block_sum256(uint32_t v, uint32_t* sc) {
  uint32_t tot;
  block_excl_scan(v, sc, &tot);
  return tot;
}

// per chunk: entries with key >= tge, and with key == teq (when ties are to be split)
__global__ __launch_bounds__(256) void k_lsel_count(ListSel S, uint32_t nch, const uint32_t* __restrict__ st,
                                                    uint32_t* __restrict__ ccnt) {
  __shared__ uint32_t sc[8];
  const uint32_t i = blockIdx.x / nch, k = blockIdx.x % nch;
  const ListDesc D = S.desc(i);
  const uint32_t tge = st[4 * i], teq = st[4 * i + 1], need_eq = st[4 * i + 2];
  const uint32_t j0 = k * LIST_CHUNK, j1 = min(D.len, j0 + LIST_CHUNK);
  uint32_t ng = 0, ne = 0;
  for (uint32_t j = j0 + threadIdx.x; j < j1; j += 256u) {
    const uint32_t key = mag_key(D.iv[j]);
    ng += key >= tge;
    ne += need_eq != 0u && key == teq;
  }
  ng = block_sum256(ng, sc);
  ne = block_sum256(ne, sc);
  if (threadIdx.x == 0) {
    ccnt[2 * ((int64_t)i * nch + k)] = ng;
    ccnt[2 * ((int64_t)i * nch + k) + 1] = ne;
  }
}

// per chunk: kept entries to K in index order, the rest to D; chunk 0 also
// writes the sentinels and the drop count
__global__ __launch_bounds__(256) void k_lsel_emit(ListSel S, uint32_t nch, const uint32_t* __restrict__ st,
                                                   const uint32_t* __restrict__ ccnt, uint32_t* __restrict__ err) {
  constexpr uint32_t PT = LIST_CHUNK / 256;   // consecutive entries per thread
  __shared__ uint32_t sc[8];
  const uint32_t i = blockIdx.x / nch, k = blockIdx.x % nch;
  const ListDesc D = S.desc(i);
  const uint32_t tge = st[4 * i], teq = st[4 * i + 1], need_eq = st[4 * i + 2], keep = st[4 * i + 3];
  if (k == 0) {
    for (uint32_t j = keep + threadIdx.x; j < D.pad; j += 256u) {
      D.ki[j] = INT32_MAX;
      D.kv[j] = 0.f;
    }
    if (threadIdx.x == 0) *D.dcnt = (int32_t)(D.len - keep);
  }
  const uint32_t j0 = k * LIST_CHUNK;
  if (j0 >= D.len) return;   // uniform
  // selected and tied entries of the chunks before this one
  uint32_t pg = 0, pe = 0;
  for (uint32_t k2 = threadIdx.x; k2 < k; k2 += 256u) {
    pg += ccnt[2 * ((int64_t)i * nch + k2)];
    pe += ccnt[2 * ((int64_t)i * nch + k2) + 1];
  }
  pg = block_sum256(pg, sc);
  pe = block_sum256(pe, sc);
  const uint32_t a = min(D.len, j0 + threadIdx.x * PT), b = min(D.len, a + PT);
  uint32_t ng = 0, ne = 0;
  for (uint32_t j = a; j < b; ++j) {
    const uint32_t key = mag_key(D.iv[j]);
    ng += key >= tge;
    ne += need_eq != 0u && key == teq;
  }
  uint32_t tg, te;
  uint32_t rg = pg + block_excl_scan(ng, sc, &tg);
  uint32_t re = pe + block_excl_scan(ne, sc, &te);
  const uint32_t ndrop = D.len - keep;
  for (uint32_t j = a; j < b; ++j) {
    const int32_t x = D.ii[j];
    const float v = D.iv[j];
    const uint32_t key = mag_key(v);
    const bool is_g = key >= tge, is_e = need_eq != 0u && key == teq;
    const uint32_t before = rg + min(re, need_eq);
    if (is_g || (is_e && re < need_eq)) {
      if (before < keep) {
        D.ki[before] = x;
        D.kv[before] = v;
      } else {
        atomicOr(err, ERR_COUNT_POS);
      }
    } else if (j - before < ndrop) {
      D.di[j - before] = x;
      D.dv[j - before] = v;
    } else {
      atomicOr(err, ERR_COUNT_DROP);
    }
    rg += is_g;
    re += is_e;
  }
}

// ---- the Bruck All-Gather's result summed in team order, for block q, in
// tiles of UT indices: each workgroup takes the d kept lists' entries that
// fall in its tile (found by wave searches in the index-sorted lists, all
// teams' at once), adds them in team order in LDS (first occurrence stores,
// later ones add; an LDS occupancy bitmap tells which), and either counts
// the tile's distinct indices (pass 1) or writes them in index order after
// the counts of the tiles before it (pass 2).  Tile 0 of each block also
// records N_q.
constexpr uint32_t UT = UNION_TILE;
constexpr uint32_t UNION_TEAMS = 8;   // teams whose ranges are searched together (two waves each)
static_assert(2 * UNION_TEAMS <= 1024 / WAVE, "two waves of the union workgroup per team of a batch");

// First position m in [0, len) with a[m] >= bound (len if none), a sorted
// ascending; one wave, 64 probes per round (three rounds for 64000 entries).
__device__ __forceinline__ uint32_t wave_lower_bound(const int32_t* __restrict__ a, uint32_t len, int32_t bound) {
  const uint32_t lane = (uint32_t)lane_id();
  uint32_t l = 0, h = len;   // the answer lies in [l, h]
  while (h > l) {
    const uint32_t S = h - l;
    if (S <= (uint32_t)WAVE) {
      l += (uint32_t)popc64(__ballot(lane < S && a[l + lane] < bound));
      break;
    }
    // probe k at l + S (k + 1) / (WAVE + 1) < h; the true probes are a prefix
    const uint32_t m = l + (uint32_t)(((uint64_t)S * (lane + 1u)) / (WAVE + 1u));
    const uint32_t t = (uint32_t)popc64(__ballot(a[m] < bound));
    const uint32_t nl = t == 0u ? l : l + (uint32_t)(((uint64_t)S * t) / (WAVE + 1u)) + 1u;
    const uint32_t nh = t == (uint32_t)WAVE ? h : l + (uint32_t)(((uint64_t)S * (t + 1u)) / (WAVE + 1u));
    l = nl;
    h = nh;
  }
  return l;
}

template <bool WRITE>
__global__ __launch_bounds__(1024) void k_bsag_union(const int32_t* __restrict__ kept_i,
                                                     const float* __restrict__ kept_v, Blocks B, uint32_t d,
                                                     uint32_t kb, const uint32_t* __restrict__ cnt, uint32_t ntile,
                                                     uint32_t* __restrict__ tile_cnt, int32_t* __restrict__ U_i,
                                                     float* __restrict__ U_v, uint32_t* __restrict__ N,
                                                     int32_t* __restrict__ info, uint32_t* __restrict__ err) {
  constexpr uint32_t NT = 1024;
  __shared__ float vals[WRITE ? UT : 1];
  __shared__ uint32_t bits[UT / 32];
  __shared__ uint32_t sc[24];
  __shared__ uint32_t range[2 * UNION_TEAMS];
  const uint32_t q = blockIdx.x / ntile, tile = blockIdx.x % ntile, Q = B.P;
  const uint32_t s = B.start(q), e = B.start(q + 1u);
  const uint32_t lo = s + tile * UT;
  if (lo >= e) {   // uniform: a shorter block has fewer tiles
    if (!WRITE && threadIdx.x == 0) tile_cnt[(int64_t)q * ntile + tile] = 0u;
    return;
  }
  const uint32_t hi = min(e, lo + UT);
  const uint32_t c = min(cnt[q], kb);
  for (uint32_t w = threadIdx.x; w < UT / 32; w += NT) bits[w] = 0u;
  for (uint32_t t0 = 0; t0 < d; t0 += UNION_TEAMS) {
    const uint32_t nt = min(d - t0, UNION_TEAMS);
    __syncthreads();   // the previous batch's ranges have been read
    // the tile's range in each team's list: wave 2k finds the first entry of
    // team t0 + k at or above lo, wave 2k + 1 the first at or above hi
    const uint32_t sx = (uint32_t)wave_id();
    if (sx < 2u * nt) {
      const int64_t o = ((int64_t)(t0 + sx / 2u) * Q + q) * kb;
      const uint32_t r = wave_lower_bound(kept_i + o, c, (int32_t)((sx & 1u) ? hi : lo));
      if (lane_id() == 0) range[sx] = r;
    }
    __syncthreads();   // also orders the zeroing above before the first additions
    for (uint32_t k = 0; k < nt; ++k) {
      const int64_t o = ((int64_t)(t0 + k) * Q + q) * kb;
      const uint32_t a = range[2u * k], b = range[2u * k + 1u];
      for (uint32_t j = a + threadIdx.x; j < b; j += NT) {
        const uint32_t r = (uint32_t)kept_i[o + j] - lo, bit = 1u << (r & 31u);
        const uint32_t old = atomicOr(&bits[r >> 5], bit);
        if (WRITE) {
          const float v = kept_v[o + j];
          vals[r] = (old & bit) ? vals[r] + v : v;
        }
      }
      __syncthreads();   // this team's additions before the next team's
    }
  }
  const uint32_t words = (hi - lo + 31u) >> 5;
  const uint32_t m0 = threadIdx.x < words ? bits[threadIdx.x] : 0u;   // words <= UT / 32 = 512 < NT
  uint32_t tot;
  uint32_t pos = block_excl_scan(__popc(m0), sc, &tot);
  if (!WRITE) {
    if (threadIdx.x == 0) tile_cnt[(int64_t)q * ntile + tile] = tot;
    return;
  }
  // distinct indices of the tiles before this one (and of all tiles, for tile 0)
  const uint32_t* __restrict__ tc = tile_cnt + (int64_t)q * ntile;
  uint32_t before = 0, all = 0;
  for (uint32_t t2 = threadIdx.x; t2 < ntile; t2 += NT) {
    const uint32_t v = tc[t2];
    before += t2 < tile ? v : 0u;
    all += v;
  }
  uint32_t tmp;
  block_excl_scan(before, sc, &tmp);
  before = tmp;
  block_excl_scan(all, sc, &tmp);
  all = tmp;
  const uint32_t cap = d * kb;
  pos += before;
  uint32_t m = m0;
  while (m) {
    const uint32_t bt = __ffs(m) - 1u;
    m &= m - 1u;
    const uint32_t r = 32u * threadIdx.x + bt;
    if (pos < cap) {
      U_i[(int64_t)q * cap + pos] = (int32_t)(lo + r);
      U_v[(int64_t)q * cap + pos] = vals[r];
    }
    ++pos;
  }
  if (tile == 0 && threadIdx.x == 0) {
    if (all > cap) atomicOr(err, ERR_COUNT);
    N[q] = all;
    if (info) {
      info[q] = (int32_t)c;
      info[Q + q] = (int32_t)all;
    }
  }
}

// ============================================================================ lazy summation
// One SRS step of the lazy variant (Sec. III-B "Optimization for SRS",
// Algorithm 1): worker w sent sp[w][b], b = (w + d + t) mod P for t < m, to
// worker r = (w + d) mod P.
//  restore = 0: r adds every entry into its dense row, first saving the
//               value there into saved[w][b] at the entry's position;
//  restore = 1: r puts the saved value back where the index is not a final
//               index (bm); run over the steps in reverse order, so the value
//               before the first receipt is what stays.
// Within one step each (receiver, block) has one sender whose indices are
// distinct, so no two threads touch one element.  Entries outside their block
// are skipped.  With hist1 (receive only), the receiver block's level-1
// histogram left by the fused add is kept exact -- the old key's bin loses
// the entry, the new key's bin gains it, both only at or above the add's
// histogram floor, as deltas gathered in LDS per workgroup and added bin by
// bin -- and the block is marked in spec_used, since its speculative
// candidates no longer hold its values.  Grid: x over chunks of a block's
// k_blk entries (LAZY_CHUNK per workgroup with hist1, else 256 per sweep),
// y over pairs (w, t).
constexpr uint32_t LAZY_CHUNK = 4096;
constexpr int LAZY_R = LAZY_CHUNK / 256;   // entries per thread of a receipt chunk

template <bool HIST>   // HIST: hist1 is given (receive only); the two forms get their own registers
__global__ __launch_bounds__(256) void k_lazy_step(float* __restrict__ acc, int64_t ld_acc, Blocks B, uint32_t kb,
                                                   uint32_t d, uint32_t m, const int32_t* __restrict__ sp_idx,
                                                   const float* __restrict__ sp_val, float* __restrict__ saved,
                                                   const uint32_t* __restrict__ bm, int restore,
                                                   uint32_t* __restrict__ hist1, uint32_t* __restrict__ spec_used,
                                                   uint32_t hc) {
  __shared__ uint32_t dh[HIST ? NB1 : 1];   // histogram deltas
  const uint32_t npairs = B.P * m;
  for (uint32_t pair = blockIdx.y; pair < npairs; pair += gridDim.y) {
    const uint32_t w = pair / m, t = pair - w * m;
    const uint32_t r = (w + d) % B.P, b = (w + d + t) % B.P;
    const uint32_t s = B.start(b), e = B.start(b + 1u);
    const int64_t o = ((int64_t)w * B.P + b) * kb;
    float* __restrict__ A = acc + (int64_t)r * ld_acc;
    if constexpr (HIST) {
      const int64_t cu = (int64_t)r * B.P + b;   // the receiver block's arrays
      const L1Map M = l1_map(spec_used[cu]);   // the add's bins
      const uint32_t FH = M.floor;
      const uint32_t j0 = blockIdx.x * LAZY_CHUNK;
      if (j0 >= kb) continue;
      if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(&spec_used[cu], SPEC_DIRTY);
      for (int i = threadIdx.x; i < NB1; i += 256) dh[i] = 0u;
      __syncthreads();
      // the chunk's entries, then the values they land on, all loads in flight
      // before any store (a pair's indices are distinct, so no entry's store
      // meets another's load)
      const uint32_t j1 = min(kb, j0 + LAZY_CHUNK);
      int32_t xs[LAZY_R];
      float vs[LAZY_R], olds[LAZY_R];
#pragma unroll
      for (int q = 0; q < LAZY_R; ++q) {
        const uint32_t j = j0 + (uint32_t)q * 256u + threadIdx.x;
        xs[q] = -1;
        vs[q] = 0.f;
        if (j < j1) {
          xs[q] = sp_idx[o + j];
          vs[q] = sp_val[o + j];
        }
      }
#pragma unroll
      for (int q = 0; q < LAZY_R; ++q) {
        const bool in = xs[q] >= (int32_t)s && xs[q] < (int32_t)e;   // false for an empty lane (-1)
        olds[q] = in ? A[xs[q]] : 0.f;
      }
#pragma unroll
      for (int q = 0; q < LAZY_R; ++q) {
        if (xs[q] < (int32_t)s || xs[q] >= (int32_t)e) continue;
        const uint32_t j = j0 + (uint32_t)q * 256u + threadIdx.x;
        const float old = olds[q];
        const float nv = old + vs[q];
        saved[o + j] = old;
        A[xs[q]] = nv;
        const uint32_t k0 = mag_key(old), k1 = mag_key(nv);
        if (k0 >= FH) atomicSub(&dh[M.bin(k0)], 1u);
        if (k1 >= FH) atomicAdd(&dh[M.bin(k1)], 1u);
      }
      __syncthreads();
      uint32_t* __restrict__ H = hist1 + (cu * hc + (blockIdx.x % HCOPIES_MIN)) * NB1;
      for (int i = threadIdx.x; i < NB1; i += 256) {
        const uint32_t c = dh[i];   // a signed delta, added modulo 2^32
        if (c) atomicAdd(&H[i], c);
      }
      __syncthreads();   // dh is cleared for the next pair
      continue;
    }
    for (uint32_t j = blockIdx.x * 256u + threadIdx.x; j < kb; j += gridDim.x * 256u) {
      const int32_t x = sp_idx[o + j];
      if (x < (int32_t)s || x >= (int32_t)e) continue;
      if (restore) {
        if (!in_final(bm, x)) A[x] = saved[o + j];
      } else {
        const float old = A[x];
        saved[o + j] = old;
        A[x] = old + sp_val[o + j];
      }
    }
  }
}

// ============================================================================ launchers
hipError_t launch_bsag_init(int32_t Q, double h0, double step0, double* H, double* S, uint32_t* F, uint32_t* N,
                            hipStream_t s) {
  hipLaunchKernelGGL(k_bsag_init, dim3(grid_for(Q, 64, 1024)), dim3(64), 0, s, (uint32_t)Q, h0, step0, H, S, F, N);
  return hipGetLastError();
}

hipError_t launch_bsag_exchange(const BsagArgs& a, hipStream_t s) {
  const uint32_t Q = (uint32_t)a.Q, d = (uint32_t)a.d, kb = (uint32_t)a.kb, P = Q * d, cap = d * kb;
  hipLaunchKernelGGL(k_bsag_control, dim3(grid_for(Q, 64, 1024)), dim3(64), 0, s, Q, kb, d, a.H, a.S, a.F, a.N,
                     a.cnt);
  ListSel L{};
  L.Q = Q;
  L.kb = kb;
  L.cap = cap;
  L.sp_idx = a.sp_idx;
  L.sp_val = a.sp_val;
  L.cnt = a.cnt;
  L.N = a.N;
  L.kept_i = a.kept_i;
  L.kept_v = a.kept_v;
  L.drop_i = a.drop_i;
  L.drop_v = a.drop_v;
  L.drop_cnt = a.drop_cnt;
  L.U_i = a.U_i;
  L.U_v = a.U_v;
  L.fd_i = a.fd_i;
  L.fd_v = a.fd_v;
  L.fd_cnt = a.fd_cnt;
  // top-h of every held block: P lists of k_blk entries
  L.mode = 0u;
  const uint32_t nch0 = (kb + LIST_CHUNK - 1) / LIST_CHUNK;
  hipLaunchKernelGGL(k_lsel_hist, dim3(P * nch0), dim3(256), 0, s, L, nch0, a.hist);
  hipLaunchKernelGGL(k_lsel_level, dim3(P), dim3(1024), 0, s, L, a.hist, a.lst, a.err);
  hipLaunchKernelGGL(k_lsel_count, dim3(P * nch0), dim3(256), 0, s, L, nch0, a.lst, a.ccnt);
  hipLaunchKernelGGL(k_lsel_emit, dim3(P * nch0), dim3(256), 0, s, L, nch0, a.lst, a.ccnt, a.err);
  // team-order sums, counted then written tile by tile
  const Blocks B = make_blocks(a.n, a.Q);
  hipLaunchKernelGGL(k_bsag_union<false>, dim3(Q * a.ntile), dim3(1024), 0, s, a.kept_i, a.kept_v, B, d, kb, a.cnt,
                     a.ntile, a.tile_cnt, a.U_i, a.U_v, a.N, a.info, a.err);
  hipLaunchKernelGGL(k_bsag_union<true>, dim3(Q * a.ntile), dim3(1024), 0, s, a.kept_i, a.kept_v, B, d, kb, a.cnt,
                     a.ntile, a.tile_cnt, a.U_i, a.U_v, a.N, a.info, a.err);
  // final top-L of every block: Q lists of up to d k_blk entries
  L.mode = 1u;
  const uint32_t nch1 = (cap + LIST_CHUNK - 1) / LIST_CHUNK;
  hipLaunchKernelGGL(k_lsel_hist, dim3(Q * nch1), dim3(256), 0, s, L, nch1, a.hist);
  hipLaunchKernelGGL(k_lsel_level, dim3(Q), dim3(1024), 0, s, L, a.hist, a.lst, a.err);
  hipLaunchKernelGGL(k_lsel_count, dim3(Q * nch1), dim3(256), 0, s, L, nch1, a.lst, a.ccnt);
  hipLaunchKernelGGL(k_lsel_emit, dim3(Q * nch1), dim3(256), 0, s, L, nch1, a.lst, a.ccnt, a.err);
  return hipGetLastError();
}

hipError_t launch_lazy_step(float* acc, int64_t ld_acc, int32_t P, int64_t n, int32_t kb, int32_t d, int32_t m,
                            const int32_t* sp_idx, const float* sp_val, float* saved, const uint32_t* bm,
                            bool restore, uint32_t* hist1, uint32_t* spec_used, hipStream_t s) {
  const unsigned gx = hist1 ? (unsigned)((kb + LAZY_CHUNK - 1) / LAZY_CHUNK) : grid_for(kb, 256, 1024);
  const dim3 grid(gx, (unsigned)std::min<int64_t>((int64_t)P * m, 65535));
  if (hist1)
    hipLaunchKernelGGL(k_lazy_step<true>, grid, dim3(256), 0, s, acc, ld_acc, make_blocks(n, P), (uint32_t)kb,
                       (uint32_t)d, (uint32_t)m, sp_idx, sp_val, saved, bm, restore ? 1 : 0, hist1, spec_used,
                       hist_copies_for(n, P));
  else
    hipLaunchKernelGGL(k_lazy_step<false>, grid, dim3(256), 0, s, acc, ld_acc, make_blocks(n, P), (uint32_t)kb,
                       (uint32_t)d, (uint32_t)m, sp_idx, sp_val, saved, bm, restore ? 1 : 0, hist1, spec_used,
                       hist_copies_for(n, P));
  return hipGetLastError();
}

}  // namespace spardl
