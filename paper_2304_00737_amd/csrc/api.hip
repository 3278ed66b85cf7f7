// C ABI of libspardl (declared in include/spardl.h): argument checks,
// workspace layout and kernel sequencing.  Nothing here allocates,
// synchronises or copies between host and device.

#include <stddef.h>
#include <stdint.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "../../include/spardl.h"
#include "common.hpp"
#include "launch.hpp"

using namespace spardl;

namespace {

constexpr int64_t kMaxN = (int64_t)INT32_MAX;   // indices are int32: n < 2^31

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

inline int32_t steps_of(int32_t P) {
  int32_t l = 0;
  while ((1ll << l) < P) ++l;
  return l;
}

// blocks in the bag of step i (1-based) of Spar-Reduce-Scatter
inline int32_t bag_of(int32_t P, int32_t l, int32_t i) {
  return i == 1 ? P - (1 << (l - 1)) : (1 << (l - i));
}

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Workspace layout.  Everything before the candidate region depends only on
// (P, n, k_blk), so every call finds the same offsets; the candidate region
// takes the rest of ws, split into three equal arrays (candidate index,
// candidate value, threshold-bin key).
struct Layout {
  size_t err = 0, bitmap = 0, hist1 = 0, spec_t1 = 0, spec_used = 0, spec_cnt = 0, state = 0, slot_cnt = 0,
         slot_nbin = 0, pre_all = 0, pre_ge = 0, pre_eq = 0, keep = 0, dtile = 0;
  int64_t dtile_pairs = 0;   // (pair, step) lists of all rows over the SRS steps
  uint32_t hcopies = HCOPIES_MIN;   // level-1 histogram copies per unit
  size_t fixed_end = 0;
  int64_t units = 0, tiles_tk = 0, tiles_mg = 0, slot_n = 0, pairs_max = 0, add_tiles = 0;
};

// rows: rows of acc the calls cover (P, or all d teams' rows with P = Q
// blocks per row); everything scales with rows x blocks.
Layout make_layout(int32_t P, int64_t n, int32_t kb, int32_t rows = 0) {
  Layout L;
  if (rows <= 0) rows = P;
  const int32_t l = steps_of(P);
  int64_t mmax = 0;   // largest bag over the steps (step 1 is not always the largest)
  for (int32_t i = 1; i <= l; ++i) mmax = std::max<int64_t>(mmax, bag_of(P, l, i));
  const int64_t maxlen = ceil_div(n, P);
  L.pairs_max = (int64_t)rows * mmax;
  L.units = std::max<int64_t>((int64_t)rows * P, L.pairs_max);
  L.tiles_tk = spans_per_block(maxlen, SLOT);   // slots from each block's aligned origin
  L.tiles_mg = ceil_div(2ll * kb, MERGE_TILE);
  L.slot_n = std::max<int64_t>((int64_t)rows * P * L.tiles_tk, L.pairs_max * L.tiles_mg);
  size_t off = 256;
  L.bitmap = off;
  off += align256((size_t)ceil_div(n, 32) * 4);
  L.hist1 = off;
  L.hcopies = hist_copies_for(n, P);
  off += align256((size_t)L.units * L.hcopies * NB1 * 4);
  // speculative candidates of the fused residual add: per (worker, block) the
  // previous threshold bin + 1 (0: none) and the floor used; per add tile the count
  L.add_tiles = add_tiles_per_block(maxlen);
  L.spec_t1 = off;
  off += align256((size_t)rows * P * 4);
  L.spec_used = off;
  off += align256((size_t)rows * P * 4);
  L.spec_cnt = off;   // per add tile
  off += align256((size_t)rows * P * L.add_tiles * 4);
  L.state = off;
  off += align256((size_t)L.units * ST_WORDS * 4);
  L.slot_cnt = off;
  off += align256((size_t)L.slot_n * 4);
  L.slot_nbin = off;
  off += align256((size_t)L.slot_n * 4);
  L.pre_all = off;
  off += align256((size_t)L.slot_n * 4);
  L.pre_ge = off;
  off += align256((size_t)L.slot_n * 4);
  L.pre_eq = off;
  off += align256((size_t)L.slot_n * 4);
  // a residual collection fused into the next add: per (worker, block) the
  // block top-k's selection rule; per SRS step, pair and add tile the range
  // of the pair's drops in the tile (step i's pairs after those of steps < i)
  L.keep = off;
  off += align256((size_t)rows * P * KEEP_WORDS * 4);
  for (int32_t i = 1; i <= l; ++i) L.dtile_pairs += (int64_t)rows * bag_of(P, l, i);
  L.dtile = off;
  off += align256((size_t)L.dtile_pairs * L.add_tiles * 8);
  L.fixed_end = off;
  return L;
}

inline size_t cand_bytes(int64_t entries) { return 3 * align256((size_t)entries * 4); }

// Workspace of the R-SAG exchanges (npairs merges of two k_blk blocks): the
// error word, one level-1 histogram and the selection state per pair, per-slot
// counts and prefixes, then the merged candidates.
Layout make_pair_layout(int64_t npairs, int32_t kb) {
  Layout L;
  L.pairs_max = npairs;
  L.units = npairs;
  L.tiles_mg = ceil_div(2ll * kb, MERGE_TILE);
  L.slot_n = npairs * L.tiles_mg;
  size_t off = 256;
  L.hist1 = off;
  off += align256((size_t)npairs * NB1 * 4);
  L.state = off;
  off += align256((size_t)npairs * ST_WORDS * 4);
  L.slot_cnt = off;
  off += align256((size_t)L.slot_n * 4);
  L.slot_nbin = off;
  off += align256((size_t)L.slot_n * 4);
  L.pre_all = off;
  off += align256((size_t)L.slot_n * 4);
  L.pre_ge = off;
  off += align256((size_t)L.slot_n * 4);
  L.pre_eq = off;
  off += align256((size_t)L.slot_n * 4);
  L.fixed_end = off;
  return L;
}


inline int32_t log2_exact(int32_t d) {
  int32_t t = 0;
  while ((1 << t) < d) ++t;
  return t;
}

struct Ws {
  char* base;
  uint32_t *err, *bitmap, *hist1, *spec_t1, *spec_used, *spec_cnt, *state, *slot_cnt, *slot_nbin, *pre_all, *pre_ge,
      *pre_eq, *keep;
  uint2* dtile;
  int32_t* cand_idx;
  float* cand_val;
  uint32_t* bin_key;
};

Ws carve(void* ws, size_t ws_bytes, const Layout& L) {
  Ws w;
  w.base = (char*)ws;
  auto at = [&](size_t off) { return (uint32_t*)(w.base + off); };
  w.err = at(L.err);
  w.bitmap = at(L.bitmap);
  w.hist1 = at(L.hist1);
  w.spec_t1 = at(L.spec_t1);
  w.spec_used = at(L.spec_used);
  w.spec_cnt = at(L.spec_cnt);
  w.state = at(L.state);
  w.slot_cnt = at(L.slot_cnt);
  w.slot_nbin = at(L.slot_nbin);
  w.pre_all = at(L.pre_all);
  w.pre_ge = at(L.pre_ge);
  w.pre_eq = at(L.pre_eq);
  w.keep = at(L.keep);
  w.dtile = (uint2*)at(L.dtile);
  const size_t q = ws_bytes > L.fixed_end ? ((ws_bytes - L.fixed_end) / 3) & ~(size_t)255 : 0;
  w.cand_idx = (int32_t*)(w.base + L.fixed_end);
  w.cand_val = (float*)(w.base + L.fixed_end + q);
  w.bin_key = at(L.fixed_end + 2 * q);
  return w;
}

inline bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }
inline bool ws_misaligned(const void* ws) { return ((uintptr_t)ws & 255u) != 0; }

// float4 streaming is used when every block start, the row length and the
// row strides are multiples of 4 and the base pointers are 16-byte aligned.
bool blocks_vec4(int64_t n, int32_t P) {
  if (n % 4) return false;
  for (int64_t b = 0; b <= P; ++b)
    if (blk_start(b, n, P) % 4) return false;
  return true;
}

bool sizes_ok(int32_t P, int64_t n, int32_t kb) {
  if (P < 1 || n < P || n > kMaxN) return false;
  if (kb < 1 || (int64_t)kb > n / P) return false;
  return true;
}

// d a power of two dividing P, and k_blk valid for blocks of a team of P / d
bool rsag_sizes_ok(int32_t P, int32_t d, int64_t n, int32_t kb) {
  if (P < 2 || d < 2 || (d & (d - 1)) || P % d) return false;
  return sizes_ok(P / d, n, kb);
}

// any d >= 2 dividing P, k_blk valid for blocks of a team of P / d
bool bsag_sizes_ok(int32_t P, int32_t d, int64_t n, int32_t kb) {
  if (P < 2 || d < 2 || P % d) return false;
  return sizes_ok(P / d, n, kb);
}

// Workspace of the B-SAG exchange.
struct BsagLayout {
  size_t H, S, F, N, cnt, hist, lst, ccnt, tile_cnt, kept_i, kept_v, U_i, U_v, fd_i, fd_v, fd_cnt, end;
  uint32_t ntile;
};

BsagLayout make_bsag_layout(int32_t P, int32_t d, int64_t n, int32_t kb) {
  BsagLayout L;
  const int64_t Q = P / d;
  const int64_t maxlen = (n + Q - 1) / Q;
  L.ntile = (uint32_t)ceil_div(maxlen, (int64_t)UNION_TILE);
  const int64_t cap = (int64_t)d * kb;
  const int64_t nch = ceil_div(cap, (int64_t)LIST_CHUNK);
  size_t off = 256;   // error word
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += (bytes + 255) & ~(size_t)255;
    return at;
  };
  L.H = take((size_t)Q * 8);
  L.S = take((size_t)Q * 8);
  L.F = take((size_t)Q * 4);
  L.N = take((size_t)Q * 4);
  L.cnt = take((size_t)Q * 4);
  L.hist = take((size_t)P * NB1 * 4);
  L.lst = take((size_t)P * 4 * 4);
  L.ccnt = take((size_t)P * nch * 2 * 4);
  L.tile_cnt = take((size_t)Q * L.ntile * 4);
  L.kept_i = take((size_t)P * kb * 4);
  L.kept_v = take((size_t)P * kb * 4);
  L.U_i = take((size_t)Q * cap * 4);
  L.U_v = take((size_t)Q * cap * 4);
  L.fd_i = take((size_t)Q * cap * 4);
  L.fd_v = take((size_t)Q * cap * 4);
  L.fd_cnt = take((size_t)Q * 4);
  L.end = off;
  return L;
}

struct Fill {
  FillRanges r{};
  Fill& add(void* p, int64_t words) {
    if (words > 0) {
      r.ptr[r.count] = (uint32_t*)p;
      r.len[r.count] = words;
      ++r.count;
    }
    return *this;
  }
};

#define SPARDL_TRY(expr)                      \
  do {                                        \
    if ((expr) != hipSuccess) return SPARDL_EDEVICE; \
  } while (0)

// The block top-k pipeline over `units` selection units: level-1 histogram
// (unless the fused add made it), level-1 select, candidates, exact
// threshold, emit into sp[row][b].  With `spec` the fused add's speculative
// candidates may be used; without it the previous-threshold hint is only
// kept for the all-blocks map (the fused add of the next step reads it).
int topk_units(const float* acc, int64_t ld_acc, int64_t units, const Units& U, int64_t n, int32_t P, int32_t k_blk,
               bool make_hist, bool spec, int32_t* sp_idx, float* sp_val, int32_t* local_idx, const Ws& w,
               const Layout& L, hipStream_t stream, int64_t hint_off = 0, bool keep_rule = false) {
  const bool v4 = aligned16(acc) && ld_acc % 4 == 0 && blocks_vec4(n, P);
  const int32_t smax = (int32_t)L.tiles_tk;
  if (make_hist) {
    SPARDL_TRY(launch_fill(Fill().add(w.hist1, units * L.hcopies * NB1).r, stream));
    SPARDL_TRY(launch_hist1(acc, ld_acc, units, U, n, P, v4, w.hist1, stream));
  }
  // the previous-threshold hint feeds the next fused add: kept unless this is a
  // lazy selection that did not start from a fused add; hint_off: the words of
  // the workers before the call's rows (hints are kept per absolute worker)
  uint32_t* hint = (U.rel && !spec) ? nullptr : w.spec_t1 + hint_off;
  SPARDL_TRY(launch_select1(w.hist1, w.state, units, U, n, P, (uint32_t)k_blk, hint, w.spec_used, spec, acc, ld_acc,
                            v4, w.err, stream));
  SPARDL_TRY(launch_collect(acc, ld_acc, units, U, n, P, k_blk, v4, smax, w.state, w.spec_cnt, (int32_t)L.add_tiles,
                            w.slot_cnt, w.slot_nbin, w.cand_idx, w.cand_val, w.bin_key, stream));
  // hist1: the staged threshold for long units builds its level-2/3 histograms in the units'
  // level-1 histogram space, which the select has cleared
  SPARDL_TRY(launch_thresh(0, units, U, n, P, k_blk, smax, w.hist1, w.cand_val, w.state, w.slot_cnt,
                           w.slot_nbin, w.bin_key, w.pre_all, w.pre_ge, w.pre_eq, nullptr, w.err, stream));
  SPARDL_TRY(launch_emit(0, w.cand_idx, w.cand_val, units, U, n, P, k_blk, Pairs{}, smax, w.state, w.slot_cnt,
                         w.pre_all, w.pre_ge, w.pre_eq, sp_idx, sp_val, local_idx, nullptr, nullptr, w.err, stream,
                         keep_rule ? w.keep + hint_off * KEEP_WORDS : nullptr));
  return SPARDL_OK;
}

// ---- all d teams in one call: P rows, Q = P / d blocks per row, SRS inside
// each team on its own rows (the d = 1 calls above with rows = blocks = Q
// give the same results team by team).
bool team_sizes_ok(int32_t P, int32_t d, int64_t n, int32_t kb) {
  return P >= 1 && d >= 1 && P % d == 0 && sizes_ok(P / d, n, kb);
}
size_t team_ws_bytes(int32_t P, int32_t d, int64_t n, int32_t kb) {
  const int32_t Q = P / d;
  const Layout L = make_layout(Q, n, kb, P);
  const int64_t cand = std::max<int64_t>((int64_t)P * n, L.pairs_max * L.tiles_mg * MERGE_TILE);
  return L.fixed_end + cand_bytes(cand);
}

// ---- scratch of the workspace-free SRS step (spardl_sparse_merge_topk_noalloc):
// per merge pair a level-1 histogram and the selection state, per slot the
// counts and prefixes, then the summed union (index, value).
struct NoallocLayout {
  size_t hist, state, slot_cnt, slot_nbin, pre_all, pre_ge, pre_eq, uidx, uval, ukey, end;
};

NoallocLayout make_noalloc_layout(int64_t npairs, int32_t kb) {
  NoallocLayout L;
  const int64_t slots = npairs * ceil_div(2ll * kb, MERGE_TILE);
  size_t off = 0;
  auto take = [&](int64_t bytes) {
    const size_t at = off;
    off += align256((size_t)bytes);
    return at;
  };
  L.hist = take(npairs * NB1 * 4);
  L.state = take(npairs * ST_WORDS * 4);
  L.slot_cnt = take(slots * 4);
  L.slot_nbin = take(slots * 4);
  L.pre_all = take(slots * 4);
  L.pre_ge = take(slots * 4);
  L.pre_eq = take(slots * 4);
  L.uidx = take(slots * MERGE_TILE * 4);
  L.uval = take(slots * MERGE_TILE * 4);
  L.ukey = take(slots * MERGE_TILE * 4);
  L.end = off;
  return L;
}

}  // namespace

// The scratch array of spardl_sparse_merge_topk_noalloc.  In host code its
// name is a host-side stand-in: the device address (one per GPU) comes from
// hipGetSymbolAddress and only that address is handed to kernels.
static __device__ __align__(256) unsigned char scratch[SPARDL_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxDevices];

// Device address of `scratch` on the GPU that runs `stream`: looked up once
// per GPU, with that GPU current, and kept.  Null if it cannot be obtained.
void* noalloc_scratch(hipStream_t stream) {
  int cur = -1, dev = -1;
  if (hipGetDevice(&cur) != hipSuccess) return nullptr;
  if (stream) {
    if (hipStreamGetDevice(stream, &dev) != hipSuccess) return nullptr;
  } else {
    dev = cur;
  }
  if (dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_addr[dev]) {
    if (dev != cur && hipSetDevice(dev) != hipSuccess) return nullptr;
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (dev != cur) (void)hipSetDevice(cur);
    if (e != hipSuccess || !p) return nullptr;
    g_scratch_addr[dev] = p;
  }
  return g_scratch_addr[dev];
}

// The collection arguments of the rows from w0 on: per SRS step its drop
// arrays, bag size and its part of the workspace's drop-tile index.
AddCollect add_collect_args(int32_t P, int32_t l, int32_t w0, int32_t k_blk, const uint32_t* member,
                            const int32_t* const* drop_idx, const float* const* drop_val,
                            const int32_t* const* drop_cnt, const Ws& w, const Layout& L) {
  AddCollect C;
  C.member = member;
  C.keep = w.keep;
  C.l = l;
  C.w0 = (uint32_t)w0;
  C.kb = (uint32_t)k_blk;
  C.G = (uint32_t)L.add_tiles;
  int64_t pairs_before = 0;
  for (int32_t i = 1; i <= l; ++i) {
    const int32_t m = bag_of(P, l, i);
    C.didx[i - 1] = drop_idx[i - 1];
    C.dval[i - 1] = drop_val[i - 1];
    C.dcnt[i - 1] = drop_cnt[i - 1];
    C.m[i - 1] = (uint32_t)m;
    C.tile[i - 1] = w.dtile + pairs_before * L.add_tiles;
    pairs_before += (int64_t)P * m;
  }
  return C;
}

}  // namespace

extern "C" {

const char* spardl_strerror(int status) {
  switch (status) {
    case SPARDL_OK: return "ok";
    case SPARDL_EINVAL: return "invalid argument";
    case SPARDL_ECAPACITY: return "workspace (or the library's static scratch) too small for these sizes";
    case SPARDL_EDEVICE: return "kernel launch failed";
    default: return "unknown status";
  }
}

int spardl_srs_plan(int32_t P, int32_t* distance, int32_t* bag_blocks) {
  if (P < 1) return SPARDL_EINVAL;
  const int32_t l = steps_of(P);
  for (int32_t i = 1; i <= l; ++i) {
    if (distance) distance[i - 1] = 1 << (l - i);
    if (bag_blocks) bag_blocks[i - 1] = bag_of(P, l, i);
  }
  return l;
}

size_t spardl_workspace_bytes(int32_t nworkers, int32_t P, int64_t n, int32_t k_blk) {
  if (!sizes_ok(P, n, k_blk) || nworkers < 1 || nworkers > P) return 0;
  const Layout L = make_layout(P, n, k_blk);
  const int64_t cand = std::max<int64_t>((int64_t)nworkers * n, L.pairs_max * L.tiles_mg * MERGE_TILE);
  return L.fixed_end + cand_bytes(cand);
}

int spardl_workspace_init(int32_t nworkers, int32_t P, int64_t n, int32_t k_blk, void* ws, size_t ws_bytes,
                          hipStream_t stream) {
  if (!ws || ws_misaligned(ws)) return SPARDL_EINVAL;
  const size_t need = spardl_workspace_bytes(nworkers, P, n, k_blk);
  if (need == 0) return SPARDL_EINVAL;
  if (ws_bytes < need) return SPARDL_ECAPACITY;
  const Layout L = make_layout(P, n, k_blk);
  Ws w = carve(ws, ws_bytes, L);
  SPARDL_TRY(launch_fill(Fill()
                             .add(w.err, 64)
                             .add(w.bitmap, ceil_div(n, 32))
                             .add(w.hist1, L.units * L.hcopies * NB1)
                             .add(w.spec_t1, (int64_t)P * P)
                             .add(w.keep, (int64_t)P * P * KEEP_WORDS)
                             .add((uint32_t*)w.dtile, L.dtile_pairs * L.add_tiles * 2)
                             .r,
                         stream));
  return SPARDL_OK;
}

int spardl_residual_add(float* acc, int64_t ld_acc, const float* grad, int64_t ld_grad, int32_t w0,
                        int32_t nworkers, int64_t n, int32_t P, int32_t k_blk, void* ws, size_t ws_bytes,
                        hipStream_t stream) {
  if (!acc || !grad || nworkers < 1 || n < 1 || n > kMaxN || ld_acc < n || ld_grad < n || P < 0 ||
      P > n || w0 < 0)
    return SPARDL_EINVAL;
  if (P == 0 || ws == nullptr) {
    const bool v4 = aligned16(acc) && aligned16(grad) && ld_acc % 4 == 0 && ld_grad % 4 == 0 && n % 4 == 0;
    SPARDL_TRY(launch_residual_add(acc, ld_acc, grad, ld_grad, nworkers, n, 1, v4, AddSpec{}, stream));
    return SPARDL_OK;
  }
  if (nworkers > P || w0 > P - nworkers || ws_misaligned(ws) || !sizes_ok(P, n, k_blk)) return SPARDL_EINVAL;
  const size_t need = spardl_workspace_bytes(nworkers, P, n, k_blk);
  if (need == 0) return SPARDL_EINVAL;
  if (ws_bytes < need) return SPARDL_ECAPACITY;
  const Layout L = make_layout(P, n, k_blk);
  Ws w = carve(ws, ws_bytes, L);
  const bool v4 = aligned16(acc) && aligned16(grad) && ld_acc % 4 == 0 && ld_grad % 4 == 0 && blocks_vec4(n, P);
  AddSpec sp;
  sp.hist1 = w.hist1;
  sp.spec_t1 = w.spec_t1 + (int64_t)w0 * P;   // the hints of workers w0 .. w0 + nworkers - 1
  if (P > 1) sp.spec_prev = w.spec_t1 + (int64_t)((w0 + P - 1) % P) * P;
  sp.spec_used = w.spec_used;
  sp.spec_cnt = w.spec_cnt;
  sp.cand_idx = w.cand_idx;
  sp.cand_val = w.cand_val;
  SPARDL_TRY(launch_residual_add(acc, ld_acc, grad, ld_grad, nworkers, n, P, v4, sp, stream));
  return SPARDL_OK;
}

int spardl_residual_add_collect(float* acc, int64_t ld_acc, const float* grad, int64_t ld_grad, int32_t w0,
                                int32_t nworkers, int64_t n, int32_t P, int32_t k_blk, const int32_t* local_idx,
                                const uint32_t* member, const int32_t* const* drop_idx,
                                const float* const* drop_val, const int32_t* const* drop_cnt, void* ws,
                                size_t ws_bytes, hipStream_t stream) {
  if (!acc || !grad || !local_idx || !member || (reinterpret_cast<uintptr_t>(member) & 3u) || !ws ||
      ws_misaligned(ws) || nworkers < 1 || nworkers > P || w0 < 0 || w0 > P - nworkers || !sizes_ok(P, n, k_blk) ||
      ld_acc < n || ld_grad < n)
    return SPARDL_EINVAL;
  const int32_t l = steps_of(P);
  if (l > 0 && (!drop_idx || !drop_val || !drop_cnt)) return SPARDL_EINVAL;
  for (int32_t i = 0; i < l; ++i)
    if (!drop_idx[i] || !drop_val[i] || !drop_cnt[i]) return SPARDL_EINVAL;
  const size_t need = spardl_workspace_bytes(nworkers, P, n, k_blk);
  if (need == 0) return SPARDL_EINVAL;
  if (ws_bytes < need) return SPARDL_ECAPACITY;
  const Layout L = make_layout(P, n, k_blk);
  Ws w = carve(ws, ws_bytes, L);
  const bool v4 = aligned16(acc) && aligned16(grad) && ld_acc % 4 == 0 && ld_grad % 4 == 0 && blocks_vec4(n, P);
  AddSpec sp;
  sp.hist1 = w.hist1;
  sp.spec_t1 = w.spec_t1 + (int64_t)w0 * P;
  if (P > 1) sp.spec_prev = w.spec_t1 + (int64_t)((w0 + P - 1) % P) * P;
  sp.spec_used = w.spec_used;
  sp.spec_cnt = w.spec_cnt;
  sp.cand_idx = w.cand_idx;
  sp.cand_val = w.cand_val;
  if (!v4 || l > COLLECT_MAX_STEPS) {
    // rows the float4 add does not take: the separate collection of these rows, then the add
    SPARDL_TRY(launch_grc_zero(acc, ld_acc, nworkers, P, n, k_blk, local_idx, member, stream));
    for (int32_t i = 1; i <= l; ++i) {
      const int32_t m = bag_of(P, l, i);
      const int64_t skip = (int64_t)w0 * m;   // the pairs of the rows before w0
      SPARDL_TRY(launch_grc_drops(acc, ld_acc, n, m, k_blk, nworkers * m, drop_idx[i - 1] + skip * k_blk,
                                  drop_val[i - 1] + skip * k_blk, drop_cnt[i - 1] + skip, member, stream));
    }
    SPARDL_TRY(launch_residual_add(acc, ld_acc, grad, ld_grad, nworkers, n, P, v4, sp, stream));
    return SPARDL_OK;
  }
  const AddCollect C = add_collect_args(P, l, w0, k_blk, member, drop_idx, drop_val, drop_cnt, w, L);
  SPARDL_TRY(launch_residual_add(acc, ld_acc, grad, ld_grad, nworkers, n, P, v4, sp, stream, C));
  return SPARDL_OK;
}

int spardl_residual_collect_index(int32_t w0, int32_t nworkers, int64_t n, int32_t P, int32_t k_blk,
                                  const int32_t* const* drop_idx, const int32_t* const* drop_cnt, void* ws,
                                  size_t ws_bytes, hipStream_t stream) {
  if (!ws || ws_misaligned(ws) || nworkers < 1 || nworkers > P || w0 < 0 || w0 > P - nworkers ||
      !sizes_ok(P, n, k_blk))
    return SPARDL_EINVAL;
  const int32_t l = steps_of(P);
  if (l > 0 && (!drop_idx || !drop_cnt)) return SPARDL_EINVAL;
  for (int32_t i = 0; i < l; ++i)
    if (!drop_idx[i] || !drop_cnt[i]) return SPARDL_EINVAL;
  // the index lives in the part of every workspace for these sizes that does not grow with its rows
  const size_t need = spardl_workspace_bytes(1, P, n, k_blk);
  if (need == 0) return SPARDL_EINVAL;
  if (ws_bytes < need) return SPARDL_ECAPACITY;
  if (l == 0 || l > COLLECT_MAX_STEPS || !blocks_vec4(n, P)) return SPARDL_OK;   // the add collects without an index
  const Layout L = make_layout(P, n, k_blk);
  Ws w = carve(ws, ws_bytes, L);
  std::vector<const float*> no_val(l, nullptr);
  const AddCollect C = add_collect_args(P, l, w0, k_blk, nullptr, drop_idx, no_val.data(), drop_cnt, w, L);
  // only tiles with drops are written: the add clamps every range to the
  // pair's drop count and takes only entries inside its tile, so a range a
  // tile kept from an earlier step adds nothing
  SPARDL_TRY(launch_drop_tiles(C, drop_cnt, nworkers, n, P, w.err, stream));
  return SPARDL_OK;
}

int spardl_block_topk(const float* acc, int64_t ld_acc, int32_t w0, int32_t nworkers, int64_t n, int32_t P,
                      int32_t k_blk, int32_t flags, int32_t* sp_idx, float* sp_val, int32_t* local_idx,
                      void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!acc || !sp_idx || !sp_val || !ws || nworkers < 1 || nworkers > P || w0 < 0 || w0 > P - nworkers ||
      !sizes_ok(P, n, k_blk) || ld_acc < n || (flags & ~SPARDL_TOPK_HIST_READY) || ws_misaligned(ws))
    return SPARDL_EINVAL;
  const size_t need = spardl_workspace_bytes(nworkers, P, n, k_blk);
  if (need == 0) return SPARDL_EINVAL;
  if (ws_bytes < need) return SPARDL_ECAPACITY;
  const Layout L = make_layout(P, n, k_blk);
  Ws w = carve(ws, ws_bytes, L);
  const bool spec = (flags & SPARDL_TOPK_HIST_READY) != 0;   // candidates of the fused add may be used
  return topk_units(acc, ld_acc, (int64_t)nworkers * P, all_blocks(P), n, P, k_blk, !spec, spec, sp_idx, sp_val,
                    local_idx, w, L, stream, (int64_t)w0 * P, true);
}

int spardl_sparse_merge_topk(int32_t* sp_idx, float* sp_val, int32_t P, int64_t n, int32_t k_blk,
                             int32_t round, int32_t* drop_idx, float* drop_val, int32_t* drop_cnt,
                             void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!sp_idx || !sp_val || !drop_idx || !drop_val || !drop_cnt || !ws || ws_misaligned(ws) || P < 2 ||
      !sizes_ok(P, n, k_blk))
    return SPARDL_EINVAL;
  const int32_t l = steps_of(P);
  if (round < 1 || round > l) return SPARDL_EINVAL;
  const Layout L = make_layout(P, n, k_blk);
  if (ws_bytes < L.fixed_end + cand_bytes(L.pairs_max * L.tiles_mg * MERGE_TILE)) return SPARDL_ECAPACITY;
  Ws w = carve(ws, ws_bytes, L);
  const int32_t d = 1 << (l - round);
  const int32_t m = bag_of(P, l, round);
  const int64_t pairs = (int64_t)P * m;
  const int32_t smax = (int32_t)L.tiles_mg;
  const Pairs PM = srs_pairs(P, m, d);
  if (merge_small(k_blk)) {
    SPARDL_TRY(launch_merge_small(sp_idx, sp_val, PM, pairs, k_blk, drop_idx, drop_val, drop_cnt, w.err, stream));
    return SPARDL_OK;
  }
  SPARDL_TRY(launch_merge(sp_idx, sp_val, PM, pairs, k_blk, smax, w.hist1, w.state, w.slot_cnt, w.cand_idx, w.cand_val,
                          w.bin_key, stream));
  SPARDL_TRY(launch_thresh(1, pairs, all_blocks(P), n, P, k_blk, smax, w.hist1, w.cand_val, w.state, w.slot_cnt, w.slot_nbin,
                           w.bin_key, w.pre_all, w.pre_ge, w.pre_eq, drop_cnt, w.err, stream));
  SPARDL_TRY(launch_emit(1, w.cand_idx, w.cand_val, pairs, all_blocks(P), n, P, k_blk, PM, smax, w.state, w.slot_cnt, w.pre_all,
                         w.pre_ge, w.pre_eq, sp_idx, sp_val, nullptr, drop_idx, drop_val, w.err, stream));
  return SPARDL_OK;
}

int spardl_sparse_merge_topk_noalloc(int32_t* sp_idx, float* sp_val, int32_t P, int64_t n, int32_t k_blk,
                                     int32_t round, int32_t* drop_idx, float* drop_val, int32_t* drop_cnt,
                                     uint32_t* err, hipStream_t stream) {
  if (!sp_idx || !sp_val || !drop_idx || !drop_val || !drop_cnt || !err || P < 2 || !sizes_ok(P, n, k_blk))
    return SPARDL_EINVAL;
  const int32_t l = steps_of(P);
  if (round < 1 || round > l) return SPARDL_EINVAL;
  const int32_t d = 1 << (l - round);
  const int32_t m = bag_of(P, l, round);
  const int64_t pairs = (int64_t)P * m;
  const NoallocLayout L = make_noalloc_layout(pairs, k_blk);
  if (L.end > (size_t)SPARDL_NOALLOC_SCRATCH_BYTES) return SPARDL_ECAPACITY;
  char* base = (char*)noalloc_scratch(stream);
  if (!base) return SPARDL_EDEVICE;
  auto at = [&](size_t off) { return (uint32_t*)(base + off); };
  uint32_t* hist = at(L.hist);
  uint32_t* state = at(L.state);
  uint32_t *slot_cnt = at(L.slot_cnt), *slot_nbin = at(L.slot_nbin);
  uint32_t *pre_all = at(L.pre_all), *pre_ge = at(L.pre_ge), *pre_eq = at(L.pre_eq);
  int32_t* uidx = (int32_t*)(base + L.uidx);
  float* uval = (float*)(base + L.uval);
  uint32_t* ukey = at(L.ukey);
  const int32_t smax = (int32_t)ceil_div(2ll * k_blk, MERGE_TILE);
  const Pairs PM = srs_pairs(P, m, d);
  // the scratch keeps the previous call's contents: the histograms the merge
  // accumulates into start from zero, and so does the caller's error word
  if (merge_small(k_blk)) {
    SPARDL_TRY(launch_fill(Fill().add(err, 1).r, stream));
    SPARDL_TRY(launch_merge_small(sp_idx, sp_val, PM, pairs, k_blk, drop_idx, drop_val, drop_cnt, err, stream));
    return SPARDL_OK;
  }
  SPARDL_TRY(launch_fill(Fill().add(hist, pairs * NB1).add(err, 1).r, stream));
  SPARDL_TRY(launch_merge(sp_idx, sp_val, PM, pairs, k_blk, smax, hist, state, slot_cnt, uidx, uval, ukey, stream));
  SPARDL_TRY(launch_thresh(1, pairs, all_blocks(P), n, P, k_blk, smax, hist, uval, state, slot_cnt, slot_nbin, ukey,
                           pre_all, pre_ge, pre_eq, drop_cnt, err, stream));
  SPARDL_TRY(launch_emit(1, uidx, uval, pairs, all_blocks(P), n, P, k_blk, PM, smax, state, slot_cnt, pre_all,
                         pre_ge, pre_eq, sp_idx, sp_val, nullptr, drop_idx, drop_val, err, stream));
  return SPARDL_OK;
}

int spardl_allgather_densify(const int32_t* sp_idx, const float* sp_val, int32_t P, int64_t n,
                             int32_t k_blk, float* dense, uint32_t* member, hipStream_t stream) {
  if (!sp_idx || !sp_val || !dense || !sizes_ok(P, n, k_blk)) return SPARDL_EINVAL;
  if (member && (reinterpret_cast<uintptr_t>(member) & 3u)) return SPARDL_EINVAL;
  SPARDL_TRY(launch_densify(sp_idx, sp_val, P, n, k_blk, dense, member, aligned16(dense), stream));
  return SPARDL_OK;
}

int spardl_residual_collect(float* acc, int64_t ld_acc, int32_t P, int64_t n, int32_t k_blk,
                            const int32_t* local_idx, const int32_t* sp_idx, const uint32_t* member,
                            const int32_t* const* drop_idx, const float* const* drop_val,
                            const int32_t* const* drop_cnt, void* ws, size_t ws_bytes,
                            hipStream_t stream) {
  if (!acc || !local_idx || !sizes_ok(P, n, k_blk) || ld_acc < n) return SPARDL_EINVAL;
  if (member ? (reinterpret_cast<uintptr_t>(member) & 3u) != 0u : (!sp_idx || !ws || ws_misaligned(ws)))
    return SPARDL_EINVAL;
  const int32_t l = steps_of(P);
  if (l > 0 && (!drop_idx || !drop_val || !drop_cnt)) return SPARDL_EINVAL;
  for (int32_t i = 0; i < l; ++i)
    if (!drop_idx[i] || !drop_val[i] || !drop_cnt[i]) return SPARDL_EINVAL;
  uint32_t* bm = nullptr;
  if (!member) {
    const Layout L = make_layout(P, n, k_blk);
    if (ws_bytes < L.hist1) return SPARDL_ECAPACITY;
    bm = carve(ws, ws_bytes, L).bitmap;
    // the workspace bitmap rests at zero between calls: mark I, update, clear
    SPARDL_TRY(launch_bm_mark(sp_idx, P, n, k_blk, bm, true, stream));
  }
  const uint32_t* in_I = member ? member : bm;
  SPARDL_TRY(launch_grc_zero(acc, ld_acc, P, P, n, k_blk, local_idx, in_I, stream));
  for (int32_t i = 1; i <= l; ++i) {
    const int32_t m = bag_of(P, l, i);
    SPARDL_TRY(launch_grc_drops(acc, ld_acc, n, m, k_blk, P * m, drop_idx[i - 1], drop_val[i - 1],
                                drop_cnt[i - 1], in_I, stream));
  }
  if (!member) SPARDL_TRY(launch_bm_mark(sp_idx, P, n, k_blk, bm, false, stream));
  return SPARDL_OK;
}

int spardl_lazy_topk(const float* acc, int64_t ld_acc, int32_t w0, int32_t nworkers, int64_t n, int32_t P,
                     int32_t k_blk, int32_t round, int32_t flags, int32_t* sp_idx, float* sp_val, void* ws,
                     size_t ws_bytes, hipStream_t stream) {
  if (!acc || !sp_idx || !sp_val || !ws || ws_misaligned(ws) || nworkers < 1 || w0 < 0 || w0 > P - nworkers ||
      !sizes_ok(P, n, k_blk) || ld_acc < n || (flags & ~SPARDL_TOPK_HIST_READY))
    return SPARDL_EINVAL;
  const bool fused = (flags & SPARDL_TOPK_HIST_READY) != 0;
  if (fused && (w0 != 0 || nworkers != P)) return SPARDL_EINVAL;   // the fused add's arrays cover all P rows
  const int32_t l = steps_of(P);
  if (round < 0 || round > l) return SPARDL_EINVAL;
  const size_t need = spardl_workspace_bytes(nworkers, P, n, k_blk);
  if (need == 0) return SPARDL_EINVAL;
  if (ws_bytes < need) return SPARDL_ECAPACITY;
  const Layout L = make_layout(P, n, k_blk);
  Ws w = carve(ws, ws_bytes, L);
  // round r >= 1: the bag sent at step r, blocks (w + 2^(l-r) + t) mod P, t < m_r; round 0: block w
  const Units U{round ? (uint32_t)bag_of(P, l, round) : 1u, round ? (uint32_t)(1 << (l - round)) : 0u, 1u,
                (uint32_t)w0};
  return topk_units(acc, ld_acc, (int64_t)nworkers * U.m, U, n, P, k_blk, !fused, fused, sp_idx, sp_val, nullptr, w,
                    L, stream);
}

int spardl_lazy_receive(float* acc, int64_t ld_acc, int32_t P, int64_t n, int32_t k_blk, int32_t round,
                        const int32_t* sp_idx, const float* sp_val, float* saved, void* ws, size_t ws_bytes,
                        hipStream_t stream) {
  if (!acc || !sp_idx || !sp_val || !saved || !sizes_ok(P, n, k_blk) || ld_acc < n) return SPARDL_EINVAL;
  const int32_t l = steps_of(P);
  if (round < 1 || round > l) return SPARDL_EINVAL;
  uint32_t *hist1 = nullptr, *spec_used = nullptr;
  if (ws) {   // keep the fused add's histograms exact through the receipts
    if (ws_misaligned(ws)) return SPARDL_EINVAL;
    const size_t need = spardl_workspace_bytes(P, P, n, k_blk);
    if (ws_bytes < need) return SPARDL_ECAPACITY;
    const Layout L = make_layout(P, n, k_blk);
    Ws w = carve(ws, ws_bytes, L);
    hist1 = w.hist1;
    spec_used = w.spec_used;
  }
  SPARDL_TRY(launch_lazy_step(acc, ld_acc, P, n, k_blk, 1 << (l - round), bag_of(P, l, round), sp_idx, sp_val, saved,
                              nullptr, false, hist1, spec_used, stream));
  return SPARDL_OK;
}

int spardl_lazy_residual_collect(float* acc, int64_t ld_acc, int32_t P, int64_t n, int32_t k_blk,
                                 const int32_t* sp_idx, const uint32_t* member, const float* saved,
                                 hipStream_t stream) {
  if (!acc || !sp_idx || !member || (reinterpret_cast<uintptr_t>(member) & 3u) || !sizes_ok(P, n, k_blk) ||
      ld_acc < n)
    return SPARDL_EINVAL;
  const int32_t l = steps_of(P);
  if (l > 0 && !saved) return SPARDL_EINVAL;
  // selected and final -> 0 (every (w, b) pair of sp is a selection of worker w)
  SPARDL_TRY(launch_grc_zero(acc, ld_acc, P, P, n, k_blk, sp_idx, member, stream));
  // received and not final -> the value before the first receipt
  for (int32_t i = l; i >= 1; --i)
    SPARDL_TRY(launch_lazy_step(acc, ld_acc, P, n, k_blk, 1 << (l - i), bag_of(P, l, i), sp_idx, nullptr,
                                const_cast<float*>(saved), member, true, nullptr, nullptr, stream));
  return SPARDL_OK;
}

size_t spardl_rsag_workspace_bytes(int32_t P, int32_t d, int64_t n, int32_t k_blk) {
  if (!rsag_sizes_ok(P, d, n, k_blk)) return 0;
  const int64_t npairs = (int64_t)(d / 2) * (P / d);
  const Layout L = make_pair_layout(npairs, k_blk);
  return L.fixed_end + cand_bytes(npairs * L.tiles_mg * MERGE_TILE);
}

int spardl_rsag_workspace_init(int32_t P, int32_t d, int64_t n, int32_t k_blk, void* ws, size_t ws_bytes,
                               hipStream_t stream) {
  if (!ws || ws_misaligned(ws)) return SPARDL_EINVAL;
  const size_t need = spardl_rsag_workspace_bytes(P, d, n, k_blk);
  if (need == 0) return SPARDL_EINVAL;
  if (ws_bytes < need) return SPARDL_ECAPACITY;
  const int64_t npairs = (int64_t)(d / 2) * (P / d);
  const Layout L = make_pair_layout(npairs, k_blk);
  Ws w = carve(ws, ws_bytes, L);
  SPARDL_TRY(launch_fill(Fill().add(w.err, 64).add(w.hist1, npairs * NB1).r, stream));
  return SPARDL_OK;
}

int spardl_rsag_merge_topk(int32_t* sp_idx, float* sp_val, int32_t P, int32_t d, int64_t n, int32_t k_blk,
                           int32_t t, int32_t* drop_idx, float* drop_val, int32_t* drop_cnt, void* ws,
                           size_t ws_bytes, hipStream_t stream) {
  if (!sp_idx || !sp_val || !drop_idx || !drop_val || !drop_cnt || !ws || ws_misaligned(ws) ||
      !rsag_sizes_ok(P, d, n, k_blk))
    return SPARDL_EINVAL;
  if (t < 0 || t >= log2_exact(d)) return SPARDL_EINVAL;
  const int32_t Q = P / d;
  const int64_t npairs = (int64_t)(d / 2) * Q;
  const Layout L = make_pair_layout(npairs, k_blk);
  if (ws_bytes < spardl_rsag_workspace_bytes(P, d, n, k_blk)) return SPARDL_ECAPACITY;
  Ws w = carve(ws, ws_bytes, L);
  const Pairs PM = rsag_pairs(Q, t);
  const int32_t smax = (int32_t)L.tiles_mg;
  SPARDL_TRY(launch_merge(sp_idx, sp_val, PM, npairs, k_blk, smax, w.hist1, w.state, w.slot_cnt, w.cand_idx, w.cand_val,
                          w.bin_key, stream));
  SPARDL_TRY(launch_thresh(1, npairs, all_blocks(Q), n, Q, k_blk, smax, w.hist1, w.cand_val, w.state,
                           w.slot_cnt, w.slot_nbin, w.bin_key, w.pre_all, w.pre_ge, w.pre_eq, drop_cnt, w.err,
                           stream));
  SPARDL_TRY(launch_emit(1, w.cand_idx, w.cand_val, npairs, all_blocks(Q), n, Q, k_blk, PM, smax, w.state,
                         w.slot_cnt, w.pre_all, w.pre_ge, w.pre_eq, sp_idx, sp_val, nullptr, drop_idx, drop_val,
                         w.err, stream));
  return SPARDL_OK;
}

int spardl_rsag_residual(float* acc, int64_t ld_acc, int32_t P, int32_t d, int64_t n, int32_t k_blk,
                         const uint32_t* member, const int32_t* const* drop_idx, const float* const* drop_val,
                         const int32_t* const* drop_cnt, hipStream_t stream) {
  if (!acc || !member || (reinterpret_cast<uintptr_t>(member) & 3u) || !rsag_sizes_ok(P, d, n, k_blk) ||
      ld_acc < n || !drop_idx || !drop_val || !drop_cnt)
    return SPARDL_EINVAL;
  const int32_t steps = log2_exact(d);
  for (int32_t t = 0; t < steps; ++t)
    if (!drop_idx[t] || !drop_val[t] || !drop_cnt[t]) return SPARDL_EINVAL;
  const int32_t Q = P / d;
  for (int32_t t = 0; t < steps; ++t)
    SPARDL_TRY(launch_grc_sag_drops(acc, ld_acc, n, Q, t, k_blk, (d / 2) * Q, drop_idx[t], drop_val[t], drop_cnt[t],
                                    member, stream));
  return SPARDL_OK;
}

size_t spardl_bsag_workspace_bytes(int32_t P, int32_t d, int64_t n, int32_t k_blk) {
  if (!bsag_sizes_ok(P, d, n, k_blk)) return 0;
  return make_bsag_layout(P, d, n, k_blk).end;
}

int spardl_bsag_workspace_init(int32_t P, int32_t d, int64_t n, int32_t k_blk, void* ws, size_t ws_bytes,
                               hipStream_t stream) {
  if (!ws || ws_misaligned(ws)) return SPARDL_EINVAL;
  const size_t need = spardl_bsag_workspace_bytes(P, d, n, k_blk);
  if (need == 0) return SPARDL_EINVAL;
  if (ws_bytes < need) return SPARDL_ECAPACITY;
  const BsagLayout L = make_bsag_layout(P, d, n, k_blk);
  char* base = (char*)ws;
  const int32_t Q = P / d;
  SPARDL_TRY(launch_fill(Fill().add(base, 64).add(base + L.hist, (int64_t)P * NB1).r, stream));
  // Algorithm 2's initial state: h = k/P = L/d, step = 0.01 (d - 1) L / d, flag false, N = 0
  const double h0 = (double)k_blk / (double)d;
  const double step0 = 0.01 * (d - 1) * k_blk / d;
  SPARDL_TRY(launch_bsag_init(Q, h0, step0, (double*)(base + L.H), (double*)(base + L.S), (uint32_t*)(base + L.F),
                              (uint32_t*)(base + L.N), stream));
  return SPARDL_OK;
}

int spardl_bsag_exchange(int32_t* sp_idx, float* sp_val, int32_t P, int32_t d, int64_t n, int32_t k_blk,
                         int32_t* drop_idx, float* drop_val, int32_t* drop_cnt, int32_t* info, void* ws,
                         size_t ws_bytes, hipStream_t stream) {
  if (!sp_idx || !sp_val || !drop_idx || !drop_val || !drop_cnt || !ws || ws_misaligned(ws) ||
      !bsag_sizes_ok(P, d, n, k_blk))
    return SPARDL_EINVAL;
  if (ws_bytes < spardl_bsag_workspace_bytes(P, d, n, k_blk)) return SPARDL_ECAPACITY;
  const BsagLayout L = make_bsag_layout(P, d, n, k_blk);
  char* base = (char*)ws;
  BsagArgs a;
  a.sp_idx = sp_idx;
  a.sp_val = sp_val;
  a.Q = P / d;
  a.d = d;
  a.kb = k_blk;
  a.n = n;
  a.H = (double*)(base + L.H);
  a.S = (double*)(base + L.S);
  a.F = (uint32_t*)(base + L.F);
  a.N = (uint32_t*)(base + L.N);
  a.cnt = (uint32_t*)(base + L.cnt);
  a.kept_i = (int32_t*)(base + L.kept_i);
  a.kept_v = (float*)(base + L.kept_v);
  a.drop_i = drop_idx;
  a.drop_v = drop_val;
  a.drop_cnt = drop_cnt;
  a.hist = (uint32_t*)(base + L.hist);
  a.lst = (uint32_t*)(base + L.lst);
  a.ccnt = (uint32_t*)(base + L.ccnt);
  a.tile_cnt = (uint32_t*)(base + L.tile_cnt);
  a.ntile = L.ntile;
  a.U_i = (int32_t*)(base + L.U_i);
  a.U_v = (float*)(base + L.U_v);
  a.fd_i = (int32_t*)(base + L.fd_i);
  a.fd_v = (float*)(base + L.fd_v);
  a.fd_cnt = (int32_t*)(base + L.fd_cnt);
  a.info = info;
  a.err = (uint32_t*)base;
  SPARDL_TRY(launch_bsag_exchange(a, stream));
  return SPARDL_OK;
}

int spardl_bsag_residual(float* acc, int64_t ld_acc, int32_t P, int32_t d, int64_t n, int32_t k_blk,
                         const uint32_t* member, const int32_t* drop_idx, const float* drop_val,
                         const int32_t* drop_cnt, hipStream_t stream) {
  if (!acc || !member || (reinterpret_cast<uintptr_t>(member) & 3u) || !bsag_sizes_ok(P, d, n, k_blk) ||
      ld_acc < n || !drop_idx || !drop_val || !drop_cnt)
    return SPARDL_EINVAL;
  // worker w's top-h drops: pairs of one entry each (m = 1), pair w = row w
  SPARDL_TRY(launch_grc_drops(acc, ld_acc, n, 1, k_blk, P, drop_idx, drop_val, drop_cnt, member, stream));
  return SPARDL_OK;
}

size_t spardl_team_workspace_bytes(int32_t P, int32_t d, int64_t n, int32_t k_blk) {
  if (!team_sizes_ok(P, d, n, k_blk)) return 0;
  return team_ws_bytes(P, d, n, k_blk);
}

int spardl_team_workspace_init(int32_t P, int32_t d, int64_t n, int32_t k_blk, void* ws, size_t ws_bytes,
                               hipStream_t stream) {
  if (!ws || ws_misaligned(ws) || !team_sizes_ok(P, d, n, k_blk)) return SPARDL_EINVAL;
  if (ws_bytes < team_ws_bytes(P, d, n, k_blk)) return SPARDL_ECAPACITY;
  const int32_t Q = P / d;
  const Layout L = make_layout(Q, n, k_blk, P);
  Ws w = carve(ws, ws_bytes, L);
  SPARDL_TRY(launch_fill(Fill()
                             .add(w.err, 64)
                             .add(w.bitmap, ceil_div(n, 32))
                             .add(w.hist1, L.units * L.hcopies * NB1)
                             .add(w.spec_t1, (int64_t)P * Q)
                             .r,
                         stream));
  return SPARDL_OK;
}

int spardl_team_residual_add(float* acc, int64_t ld_acc, const float* grad, int64_t ld_grad, int32_t P, int32_t d,
                             int64_t n, int32_t k_blk, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!acc || !grad || !ws || ws_misaligned(ws) || !team_sizes_ok(P, d, n, k_blk) || ld_acc < n || ld_grad < n)
    return SPARDL_EINVAL;
  if (ws_bytes < team_ws_bytes(P, d, n, k_blk)) return SPARDL_ECAPACITY;
  const int32_t Q = P / d;
  const Layout L = make_layout(Q, n, k_blk, P);
  Ws w = carve(ws, ws_bytes, L);
  const bool v4 = aligned16(acc) && aligned16(grad) && ld_acc % 4 == 0 && ld_grad % 4 == 0 && blocks_vec4(n, Q);
  AddSpec sp;
  sp.hist1 = w.hist1;
  sp.spec_t1 = w.spec_t1;
  sp.spec_used = w.spec_used;
  sp.spec_cnt = w.spec_cnt;
  sp.cand_idx = w.cand_idx;
  sp.cand_val = w.cand_val;
  SPARDL_TRY(launch_residual_add(acc, ld_acc, grad, ld_grad, P, n, Q, v4, sp, stream));
  return SPARDL_OK;
}

int spardl_team_block_topk(const float* acc, int64_t ld_acc, int32_t P, int32_t d, int64_t n, int32_t k_blk,
                           int32_t flags, int32_t* sp_idx, float* sp_val, int32_t* local_idx, void* ws,
                           size_t ws_bytes, hipStream_t stream) {
  if (!acc || !sp_idx || !sp_val || !ws || ws_misaligned(ws) || !team_sizes_ok(P, d, n, k_blk) || ld_acc < n ||
      (flags & ~SPARDL_TOPK_HIST_READY))
    return SPARDL_EINVAL;
  if (ws_bytes < team_ws_bytes(P, d, n, k_blk)) return SPARDL_ECAPACITY;
  const int32_t Q = P / d;
  const Layout L = make_layout(Q, n, k_blk, P);
  Ws w = carve(ws, ws_bytes, L);
  const bool spec = (flags & SPARDL_TOPK_HIST_READY) != 0;
  return topk_units(acc, ld_acc, (int64_t)P * Q, all_blocks(Q), n, Q, k_blk, !spec, spec, sp_idx, sp_val, local_idx,
                    w, L, stream);
}

int spardl_team_merge_topk(int32_t* sp_idx, float* sp_val, int32_t P, int32_t d, int64_t n, int32_t k_blk,
                           int32_t round, int32_t* drop_idx, float* drop_val, int32_t* drop_cnt, void* ws,
                           size_t ws_bytes, hipStream_t stream) {
  if (!sp_idx || !sp_val || !drop_idx || !drop_val || !drop_cnt || !ws || ws_misaligned(ws) ||
      !team_sizes_ok(P, d, n, k_blk))
    return SPARDL_EINVAL;
  const int32_t Q = P / d;
  const int32_t l = steps_of(Q);
  if (round < 1 || round > l) return SPARDL_EINVAL;
  if (ws_bytes < team_ws_bytes(P, d, n, k_blk)) return SPARDL_ECAPACITY;
  const Layout L = make_layout(Q, n, k_blk, P);
  Ws w = carve(ws, ws_bytes, L);
  const int32_t dist = 1 << (l - round);
  const int32_t m = bag_of(Q, l, round);
  const int64_t pairs = (int64_t)P * m;
  const int32_t smax = (int32_t)L.tiles_mg;
  const Pairs PM = team_srs_pairs(Q, m, dist);
  SPARDL_TRY(launch_merge(sp_idx, sp_val, PM, pairs, k_blk, smax, w.hist1, w.state, w.slot_cnt, w.cand_idx, w.cand_val,
                          w.bin_key, stream));
  SPARDL_TRY(launch_thresh(1, pairs, all_blocks(Q), n, Q, k_blk, smax, w.hist1, w.cand_val, w.state, w.slot_cnt,
                           w.slot_nbin, w.bin_key, w.pre_all, w.pre_ge, w.pre_eq, drop_cnt, w.err, stream));
  SPARDL_TRY(launch_emit(1, w.cand_idx, w.cand_val, pairs, all_blocks(Q), n, Q, k_blk, PM, smax, w.state,
                         w.slot_cnt, w.pre_all, w.pre_ge, w.pre_eq, sp_idx, sp_val, nullptr, drop_idx, drop_val,
                         w.err, stream));
  return SPARDL_OK;
}

int spardl_team_residual_collect(float* acc, int64_t ld_acc, int32_t P, int32_t d, int64_t n, int32_t k_blk,
                                 const int32_t* local_idx, const uint32_t* member, const int32_t* const* drop_idx,
                                 const float* const* drop_val, const int32_t* const* drop_cnt, hipStream_t stream) {
  if (!acc || !local_idx || !member || (reinterpret_cast<uintptr_t>(member) & 3u) || !team_sizes_ok(P, d, n, k_blk) ||
      ld_acc < n)
    return SPARDL_EINVAL;
  const int32_t Q = P / d;
  const int32_t l = steps_of(Q);
  if (l > 0 && (!drop_idx || !drop_val || !drop_cnt)) return SPARDL_EINVAL;
  for (int32_t i = 0; i < l; ++i)
    if (!drop_idx[i] || !drop_val[i] || !drop_cnt[i]) return SPARDL_EINVAL;
  SPARDL_TRY(launch_grc_zero(acc, ld_acc, P, Q, n, k_blk, local_idx, member, stream));
  for (int32_t i = 1; i <= l; ++i) {
    const int32_t m = bag_of(Q, l, i);
    SPARDL_TRY(launch_grc_drops(acc, ld_acc, n, m, k_blk, P * m, drop_idx[i - 1], drop_val[i - 1], drop_cnt[i - 1],
                                member, stream));
  }
  return SPARDL_OK;
}

}  // extern "C"
