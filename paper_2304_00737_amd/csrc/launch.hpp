// Host-side launchers of the kernels in kernels_*.hip (internal to libspardl).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.hpp"

namespace spardl {

constexpr int FILL_MAX = 8;
struct FillRanges {
  uint32_t* ptr[FILL_MAX];
  int64_t len[FILL_MAX];
  int count;
};

// Workspace arrays of the fused residual add (all null: plain add).
struct AddSpec {
  uint32_t* hist1 = nullptr;       // level-1 histograms, hist_copies_for(n, P) per (worker, block)
  const uint32_t* spec_t1 = nullptr;  // previous threshold bin + 1 per (worker, block), 0 = none
  const uint32_t* spec_prev = nullptr;   // the hints of the worker before row 0 (null: only each row's own)
  uint32_t* spec_used = nullptr;   // floor used for the speculative candidates per (worker, block)
  uint32_t* spec_cnt = nullptr;    // speculative candidates per add tile
  int32_t* cand_idx = nullptr;     // candidate index / value arrays (row-sized)
  float* cand_val = nullptr;
  uint32_t hcopies = HCOPIES_MIN;  // histogram copies per (worker, block) (set by the launcher)
};

// The previous step's global residual collection, applied by the fused
// residual add to each tile before it adds the gradient (member null: none).
struct AddCollect {
  const uint32_t* member = nullptr;              // bitmap of the final indices
  const uint32_t* keep = nullptr;                // per absolute (worker, block): the top-k's KEEP_WORDS
  const int32_t* didx[COLLECT_MAX_STEPS] = {};   // per SRS step: the drops, [pair][k_blk]
  const float* dval[COLLECT_MAX_STEPS] = {};
  const int32_t* dcnt[COLLECT_MAX_STEPS] = {};   // per step: the drop count of every pair
  const uint2* tile[COLLECT_MAX_STEPS] = {};     // per step: [pair][add tile] -> (first, end) of its drops there
                                                 // (tiles without drops this step may hold an older range)
  uint32_t m[COLLECT_MAX_STEPS] = {};            // per step: blocks per bag
  int32_t l = 0;
  uint32_t w0 = 0, kb = 0, G = 0;                // first worker of the call's rows; add tiles per block
};

hipError_t launch_fill(const FillRanges& r, hipStream_t s);
hipError_t launch_residual_add(float* acc, int64_t ld_acc, const float* grad, int64_t ld_grad,
                               int32_t nworkers, int64_t n, int32_t P, bool vec4, const AddSpec& sp,
                               hipStream_t s, const AddCollect& C = AddCollect{});
// The per-tile ranges of the drops of the call's rows (C.w0 .. C.w0 + nw - 1)
// for a fused collection, into the index C.tile.  Only tiles with drops are
// written; the others keep whatever range they held, which the add reads
// harmlessly (it clamps a range to the pair's drop count and adds only
// entries inside its tile).
hipError_t launch_drop_tiles(const AddCollect& C, const int32_t* const* drop_cnt, int32_t nw, int64_t n, int32_t P,
                             uint32_t* err, hipStream_t s);
// Block top-k stages over nunits selection units (Units in common.hpp).
hipError_t launch_hist1(const float* acc, int64_t ld_acc, int64_t nunits, const Units& U, int64_t n, int32_t P,
                        bool vec4, uint32_t* hist1, hipStream_t s);
hipError_t launch_select1(uint32_t* hist1, uint32_t* state, int64_t nunits, const Units& U, int64_t n, int32_t P,
                          uint32_t need, uint32_t* spec_t1, const uint32_t* spec_used, bool spec, const float* acc,
                          int64_t ld_acc, bool vec4, uint32_t* err, hipStream_t s);
hipError_t launch_collect(const float* acc, int64_t ld_acc, int64_t nunits, const Units& U, int64_t n, int32_t P,
                          int32_t kb, bool vec4, int32_t smax, const uint32_t* state, const uint32_t* spec_cnt,
                          int32_t add_tiles, uint32_t* slot_cnt, uint32_t* slot_nbin, int32_t* cand_idx,
                          float* cand_val, uint32_t* bin_key, hipStream_t s);
hipError_t launch_thresh(int mode, int64_t nunits, const Units& U, int64_t n, int32_t P, int32_t kb, int32_t smax,
                         uint32_t* hist1, const float* U_val, uint32_t* state, const uint32_t* slot_cnt,
                         const uint32_t* slot_nbin, const uint32_t* bin_key, uint32_t* pre_all, uint32_t* pre_ge,
                         uint32_t* pre_eq, int32_t* drop_cnt, uint32_t* err, hipStream_t s);
hipError_t launch_emit(int mode, const int32_t* cand_idx, const float* cand_val, int64_t nunits, const Units& U,
                       int64_t n, int32_t P, int32_t kb, const Pairs& PM, int32_t smax, const uint32_t* state,
                       const uint32_t* slot_cnt, const uint32_t* pre_all, const uint32_t* pre_ge,
                       const uint32_t* pre_eq, int32_t* out_idx, float* out_val, int32_t* local_idx,
                       int32_t* drop_idx, float* drop_val, uint32_t* err, hipStream_t s, uint32_t* keep = nullptr);
// Union tiles and their level-1 histogram; with merge_fine(kb) the fine window
// (its first bin in the pairs' state word ST_WBASE) and, per slot, the keys'
// low bits in bin order and the bins' prefix in the slot's words of U_key.
hipError_t launch_merge(const int32_t* sp_idx, const float* sp_val, const Pairs& PM, int64_t npairs, int32_t kb,
                        int32_t tiles_per_pair, uint32_t* hist1, uint32_t* state, uint32_t* slot_cnt, int32_t* U_idx,
                        float* U_val, uint32_t* U_key, hipStream_t s);
// One SRS step for unions of up to SMALL_UNION entries: merge, threshold
// and emit in one launch (the same results as launch_merge + launch_thresh +
// launch_emit).
hipError_t launch_merge_small(int32_t* sp_idx, float* sp_val, const Pairs& PM, int64_t npairs, int32_t kb,
                              int32_t* drop_idx, float* drop_val, int32_t* drop_cnt, uint32_t* err, hipStream_t s);
hipError_t launch_densify(const int32_t* sp_idx, const float* sp_val, int32_t P, int64_t n, int32_t kb,
                          float* dense, uint32_t* member, bool vec4, hipStream_t s);
hipError_t launch_bm_mark(const int32_t* sp_idx, int32_t P, int64_t n, int32_t kb, uint32_t* bm, bool set,
                          hipStream_t s);
hipError_t launch_grc_zero(float* acc, int64_t ld_acc, int32_t nw, int32_t Q, int64_t n, int32_t kb,
                           const int32_t* local_idx, const uint32_t* bm, hipStream_t s);
hipError_t launch_grc_sag_drops(float* acc, int64_t ld_acc, int64_t n, int32_t Q, int32_t t, int32_t kb,
                                int32_t npairs, const int32_t* drop_idx, const float* drop_val,
                                const int32_t* drop_cnt, const uint32_t* bm, hipStream_t s);
// Device arrays of one B-SAG exchange (kernels_variants.hip).
struct BsagArgs {
  int32_t* sp_idx;
  float* sp_val;
  int32_t Q, d, kb;
  int64_t n;
  double *H, *S;            // controller h and step per block
  uint32_t *F, *N, *cnt;    // controller flag, last union size, count in use
  int32_t* kept_i;          // top-h of every worker's held block (P x kb)
  float* kept_v;
  int32_t* drop_i;          // the rest (caller's arrays, P x kb, counts P)
  float* drop_v;
  int32_t* drop_cnt;
  uint32_t* hist;           // level-1 histograms of the list selections (P x 4096, at zero between calls)
  uint32_t* lst;            // per list: threshold words (P x 4)
  uint32_t* ccnt;           // per list chunk: selected and tied counts
  uint32_t* tile_cnt;       // per block tile of the union: distinct indices
  uint32_t ntile;           // union tiles per block
  int32_t* U_i;             // team-order sums (Q x d kb)
  float* U_v;
  int32_t* fd_i;            // final drops (Q x d kb, counts Q)
  float* fd_v;
  int32_t* fd_cnt;
  int32_t* info;            // optional: count used and union size per block
  uint32_t* err;
};
hipError_t launch_bsag_init(int32_t Q, double h0, double step0, double* H, double* S, uint32_t* F, uint32_t* N,
                            hipStream_t s);
hipError_t launch_bsag_exchange(const BsagArgs& a, hipStream_t s);
hipError_t launch_lazy_step(float* acc, int64_t ld_acc, int32_t P, int64_t n, int32_t kb, int32_t d, int32_t m,
                            const int32_t* sp_idx, const float* sp_val, float* saved, const uint32_t* bm,
                            bool restore, uint32_t* hist1, uint32_t* spec_used, hipStream_t s);
hipError_t launch_grc_drops(float* acc, int64_t ld_acc, int64_t n, int32_t m, int32_t kb, int32_t npairs,
                            const int32_t* drop_idx, const float* drop_val, const int32_t* drop_cnt,
                            const uint32_t* bm, hipStream_t s);

}  // namespace spardl
