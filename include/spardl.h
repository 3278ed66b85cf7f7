/* spardl.h -- C ABI of libspardl.so: the per-worker compute path of SparDL's
 * sparse gradient synchronisation with one team (d = 1), for AMD Instinct
 * MI355X (gfx950).
 *
 * Paper: M. Zhao et al., "SparDL: Distributed Deep Learning Training with
 * Efficient Sparse Communication", arXiv 2304.00737.  Section numbers below
 * refer to it.
 *
 * Model.  P data-parallel workers each hold a flat fp32 gradient of n values
 * and a residual of the same size.  The gradient is split into P contiguous
 * blocks, block b = [floor(b n / P), floor((b+1) n / P)).  A sparse block is
 * exactly k_blk (index, value) pairs sorted by ascending index; indices are
 * int32 offsets into the worker's flat gradient (so n < 2^31).  Several
 * workers' rows may live in one allocation with a row stride ("ld", in
 * elements).  "Top-k" always means: larger |v| first, where |v| is compared
 * as the fp32 bit pattern with the sign bit cleared; equal |v| -> lower index
 * first.  All value arithmetic is IEEE fp32 round-to-nearest-even addition;
 * results are deterministic (bit-identical run to run).  Non-finite values are
 * allowed: +-Inf ranks above every finite |v| and NaN above +-Inf (by its
 * bits), -0 ties with +0, subnormals are kept (no flush to zero), and sums
 * overflow to +-Inf.  A NaN that an addition creates or propagates has the
 * sign and payload the hardware gives it (IEEE 754 leaves them open), so
 * another implementation may hold different NaN bits at the same positions.
 *
 * Sparse state layout used by the SRS calls: sp_idx/sp_val[w][b][k_blk] for
 * worker w and block b (row-major, P * P * k_blk entries each).
 *
 * Conventions for every call below.
 *  - Pointers named acc, grad, sp_*, local_idx, drop_*, dense and ws are
 *    DEVICE pointers owned by the caller.  The library allocates nothing,
 *    keeps no state between calls, never synchronises and never copies
 *    between host and device.
 *  - Arguments are validated on the host first; on error nothing is enqueued
 *    and a negative status is returned.  Otherwise kernels are enqueued on
 *    `stream` and SPARDL_OK is returned; results are valid once the stream
 *    reaches that point.
 *  - ws is scratch device memory of at least spardl_workspace_bytes(...)
 *    bytes, 256-byte aligned (EINVAL otherwise), prepared once by
 *    spardl_workspace_init before its first use.  Between calls it keeps its
 *    level-1 histograms and the final-index bitmap at zero (the call that
 *    uses one clears it again), so no call spends a memset on them.  The first 4 bytes of ws hold an
 *    error word that spardl_workspace_init clears and that kernels OR bits
 *    into if an internal check fails (see SPARDL_WS_ERR_*); it stays set until
 *    the next spardl_workspace_init.  Read it after the stream completes.
 *    After an error, prepare the workspace again before reusing it.
 *  - Calls on different streams must use different ws and disjoint outputs.
 */
#ifndef SPARDL_H
#define SPARDL_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  SPARDL_OK = 0,
  SPARDL_EINVAL = -1,    /* an argument is NULL, out of range or misaligned */
  SPARDL_ECAPACITY = -2, /* ws_bytes is below spardl_workspace_bytes(...) */
  SPARDL_EDEVICE = -3    /* a kernel launch failed (hipGetLastError) */
};

/* Bits of the error word at the start of ws (set by kernels, cleared by
 * spardl_workspace_init).  Bit 1 is set whenever a selection's counts are
 * inconsistent (a histogram whose total is not the number of entries it
 * covers, no threshold found, an output position outside [0, k_blk), or a
 * selection without exactly k_blk entries); bits 2-5 tell which check. */
#define SPARDL_WS_ERR_LOOKBACK 1u  /* reserved (no kernel waits on another workgroup) */
#define SPARDL_WS_ERR_COUNT 2u     /* a selection's counts are inconsistent */
#define SPARDL_WS_ERR_DROPS 64u    /* spardl_residual_collect_index: a drop list not sorted inside its block */

/* Flag for spardl_block_topk: the level-1 |v| histograms (and speculative
 * candidates) of acc are already in ws, written by the immediately preceding
 * spardl_residual_add call with the same acc, ld_acc, nworkers, n, P, k_blk,
 * ws and ws_bytes (fused pass; saves one or two reads of acc). */
#define SPARDL_TOPK_HIST_READY 1

/* Static text for a status code. */
const char* spardl_strerror(int status);

/* Spar-Reduce-Scatter schedule (Sec. III-B "Partitioning" and "Transmission
 * with sparsification", Examples 1-2, Theorem 1).  Host only; no GPU needed.
 * Returns l = ceil(log2 P) (0 for P = 1), or SPARDL_EINVAL for P < 1.  If the
 * arrays are non-NULL they receive, for steps i = 1..l at position i-1:
 * distance[i-1] = 2^(l-i) (worker w sends to w + distance and receives from
 * w - distance, mod P) and bag_blocks[i-1] = number of blocks in the bag sent
 * and received at step i (P - 2^(l-1) at step 1, 2^(l-i) afterwards).  At
 * step i worker w receives blocks (w + t) mod P for t < bag_blocks[i-1].
 * Arrays must hold at least 32 entries. */
int spardl_srs_plan(int32_t P, int32_t* distance, int32_t* bag_blocks);

/* Bytes of ws that every call below needs for these sizes (nworkers = rows
 * passed to spardl_block_topk / spardl_residual_add).  0 on invalid sizes. */
size_t spardl_workspace_bytes(int32_t nworkers, int32_t P, int64_t n, int32_t k_blk);

/* Prepares ws for calls with these sizes: clears the error word, the
 * level-1 histograms, the final-index bitmap and the record of previous
 * thresholds (one fill kernel on `stream`).  Call it once after
 * allocating ws, and again after any call left an error bit set.
 * Errors: EINVAL for NULL or misaligned ws or invalid sizes (as
 * spardl_workspace_bytes); ECAPACITY if ws_bytes is below
 * spardl_workspace_bytes(nworkers, P, n, k_blk). */
int spardl_workspace_init(int32_t nworkers, int32_t P, int64_t n, int32_t k_blk, void* ws, size_t ws_bytes,
                          hipStream_t stream);

/* Residual add (Sec. III-B "Partitioning": each worker adds its residual
 * xi^{t-1} to its new gradient; first step of Algorithm 1):
 *   acc[w*ld_acc + x] = acc[w*ld_acc + x] + grad[w*ld_grad + x]
 * for w < nworkers, x < n, in place.  acc then holds A = G + xi, which also
 * serves as the copy that Algorithm 1 keeps for residual collection.
 * If P > 0 and ws != NULL, the same pass also prepares the block top-k that
 * must follow with the same acc, nworkers, n, P, k_blk, ws and ws_bytes and
 * SPARDL_TOPK_HIST_READY: it records each block's level-1 |v| histogram
 * (that call consumes and clears it) and, from a block's second step on, the
 * entries at or above a floor just below the block's previous threshold, so
 * that the top-k need not read acc again when the floor held.  P = 0 (k_blk
 * and ws ignored) is a plain add.
 * w0: the worker that row 0 of acc and grad belongs to, when a call covers
 * workers w0 .. w0 + nworkers - 1 of the P (a workspace for fewer rows than
 * P, the workers taken a few at a time).  The floor of each block comes from
 * the larger of two thresholds kept in ws per worker and block: the worker's
 * own from its previous top-k and the same block's latest at the preceding
 * worker (w - 1, or P - 1 for worker 0) -- this step's when that worker was
 * selected earlier in it, a closer estimate while the residual grows.  The
 * floor only decides how much the top-k reads; its results never depend on
 * it.  0 when the call covers all workers; ignored for the plain add.
 * Errors: EINVAL for NULL acc/grad, nworkers < 1, n < 1 or n >= 2^31,
 * ld < n, P < 0, P > n, w0 < 0, and with ws: nworkers > P,
 * w0 + nworkers > P, misaligned ws or k_blk out of [1, floor(n / P)];
 * ECAPACITY if ws is smaller than spardl_workspace_bytes(nworkers, P, n,
 * k_blk). */
int spardl_residual_add(float* acc, int64_t ld_acc, const float* grad, int64_t ld_grad, int32_t w0,
                        int32_t nworkers, int64_t n, int32_t P, int32_t k_blk, void* ws, size_t ws_bytes,
                        hipStream_t stream);

/* The previous step's global residual collection (Sec. III-C) and this
 * step's residual add (Algorithm 1, G + xi) in one pass over acc: the same
 * acc, bit for bit, as spardl_residual_collect(..., member) followed by
 * spardl_residual_add with ws, and the same histograms and candidates for
 * spardl_block_topk(SPARDL_TOPK_HIST_READY) after it.  Each tile of acc is
 * read once and written once, whole; the separate collection writes single
 * words all over acc instead.
 * The zeroing half finds a worker's selections from the values themselves:
 * the previous step's spardl_block_topk on these rows, with this ws, keeps
 * each block's selection rule in ws, so acc must be unchanged since that
 * call.  member, drop_idx, drop_val, drop_cnt: as the previous step left
 * them and as for spardl_residual_collect (the decode's bitmap; HOST arrays
 * of l DEVICE pointers, element i-1 the buffers of SRS step i for all P
 * workers; they may be NULL when P = 1).  acc, grad, local_idx: the rows
 * w0 .. w0 + nworkers - 1 (local_idx as spardl_block_topk wrote it; read
 * only for rows the float4 add does not take, which are collected by the
 * separate kernels before the add).  The drops are read through a per-tile
 * index that spardl_residual_collect_index must have built in ws after the
 * previous step's SRS steps, for these rows and these drop lists.
 * Errors: as for spardl_residual_add with ws, plus EINVAL for NULL
 * local_idx, member or ws, a misaligned member, or a NULL drop pointer. */
int spardl_residual_add_collect(float* acc, int64_t ld_acc, const float* grad, int64_t ld_grad, int32_t w0,
                                int32_t nworkers, int64_t n, int32_t P, int32_t k_blk, const int32_t* local_idx,
                                const uint32_t* member, const int32_t* const* drop_idx,
                                const float* const* drop_val, const int32_t* const* drop_cnt, void* ws,
                                size_t ws_bytes, hipStream_t stream);

/* The first half of a residual collection left to the next add: for the
 * rows w0 .. w0 + nworkers - 1, every SRS step and every add tile, the range
 * of the row's drops inside the tile, written into ws (the drop lists are
 * index-sorted inside their blocks, as spardl_sparse_merge_topk writes them).
 * Call it once after a step's SRS steps, before the next step's
 * spardl_residual_add_collect of the same rows.  Only tiles that hold drops
 * are written; the add bounds every range by the pair's drop count (it reads
 * drop_cnt too) and adds only entries inside its tile, so a range a tile
 * kept from an earlier step adds nothing.  drop_idx / drop_cnt: HOST
 * arrays of l DEVICE pointers, as for spardl_residual_collect.  Nothing is
 * enqueued where the add collects without an index (P = 1, P > 256, or
 * blocks not float4-aligned).
 * The index lives in the part of the workspace that does not grow with its
 * rows, so any workspace for these sizes holds it (a workspace for fewer
 * rows than P included).
 * Errors: EINVAL for NULL or misaligned ws, rows outside [0, P), invalid
 * sizes, a NULL drop pointer; ECAPACITY if ws is smaller than
 * spardl_workspace_bytes(1, P, n, k_blk).  The error word
 * gets SPARDL_WS_ERR_DROPS if a drop list is not sorted by index inside its
 * block. */
int spardl_residual_collect_index(int32_t w0, int32_t nworkers, int64_t n, int32_t P, int32_t k_blk,
                                  const int32_t* const* drop_idx, const int32_t* const* drop_cnt, void* ws,
                                  size_t ws_bytes, hipStream_t stream);

/* Block-wise top-k (Sec. III-B: every worker sparsifies each of its P blocks
 * to its top k/P values; top-k as in Sec. II).  For w < nworkers, b < P:
 *   sp_idx/sp_val[(w*P + b)*k_blk + j], j < k_blk = the top-k_blk entries of
 *   block b of row w of acc, sorted by ascending index.
 * local_idx (optional, may be NULL) receives a second copy of the indices;
 * spardl_residual_collect needs it after the SRS steps have overwritten sp.
 * flags: 0 or SPARDL_TOPK_HIST_READY.  w0: as for spardl_residual_add (the
 * worker of row 0; the call records each block's threshold for that
 * worker's next residual add).
 * Errors: EINVAL for NULL acc/sp/ws, nworkers < 1, w0 < 0,
 * w0 + nworkers > P, P < 1, n < P, n >= 2^31, ld_acc < n, k_blk < 1 or
 * k_blk > floor(n / P); ECAPACITY if ws is small. */
int spardl_block_topk(const float* acc, int64_t ld_acc, int32_t w0, int32_t nworkers, int64_t n, int32_t P,
                      int32_t k_blk, int32_t flags, int32_t* sp_idx, float* sp_val,
                      int32_t* local_idx, void* ws, size_t ws_bytes, hipStream_t stream);

/* One Spar-Reduce-Scatter step `round` in [1, l] for all P workers at once
 * (Sec. III-B "Transmission with sparsification").  With d = 2^(l-round) and
 * m = bag_blocks of that step (see spardl_srs_plan), for every worker w and
 * t < m, block b = (w + t) mod P of worker w receives block b of worker
 * (w - d) mod P: the two sparse blocks are summed by index (held + received
 * where both have an index), the top k_blk of the union are kept in
 * sp[w][b] (sorted by index, in place), and the rest -- this worker's
 * in-procedure residual for the block at this step (Sec. III-C) -- go to
 *   drop_idx/drop_val[(w*m + t)*k_blk + j], j < drop_cnt[w*m + t]
 * sorted by index (the union has between k_blk and 2 k_blk entries, so
 * 0 <= drop_cnt <= k_blk).  Steps must be run in order 1..l.
 * Errors: EINVAL for NULL pointers, P < 2, n < P, n >= 2^31, k_blk out of
 * [1, floor(n/P)], round outside [1, l]; ECAPACITY if ws is too small. */
int spardl_sparse_merge_topk(int32_t* sp_idx, float* sp_val, int32_t P, int64_t n, int32_t k_blk,
                             int32_t round, int32_t* drop_idx, float* drop_val, int32_t* drop_cnt,
                             void* ws, size_t ws_bytes, hipStream_t stream);

/* The same SRS step without a workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, hosts
 * that forbid hipMalloc).  Its scratch (per merge pair: the level-1
 * histogram, selection state, slot counts, the summed union and its sorted
 * key bits) lives in one
 * array of SPARDL_NOALLOC_SCRATCH_BYTES inside the library, which every GPU
 * the library runs on holds from its first such call until the process ends;
 * the call allocates nothing, and it neither synchronises nor copies.
 * Results are bit-identical to spardl_sparse_merge_topk with the same
 * arguments.  err (device, 4 bytes, caller owned) is an output: the call
 * clears it and its kernels OR in SPARDL_WS_ERR_* bits if an internal check
 * fails.  The scratch is shared by every call on one GPU and keeps the last
 * call's contents (each call clears what it needs zeroed), so calls that
 * overlap on one GPU (different streams, or different host threads) race and
 * must not be issued.
 * Errors: as spardl_sparse_merge_topk (EINVAL also for NULL err);
 * ECAPACITY when the step needs more than SPARDL_NOALLOC_SCRATCH_BYTES of
 * scratch, checked before any GPU call: each of the P m merge pairs of the
 * step (m = its bag_blocks) takes 16 KiB + 64 bytes, plus 48 KiB + 20 bytes
 * per slot of 4096 merged positions (ceil(2 k_blk / 4096) slots), each
 * array rounded up to 256 bytes (the ResNet-50-sized step 1: 32 pairs,
 * 16 slots each, 24.5 MiB); EDEVICE if the scratch's device address cannot
 * be obtained. */
#define SPARDL_NOALLOC_SCRATCH_BYTES (64u << 20)
int spardl_sparse_merge_topk_noalloc(int32_t* sp_idx, float* sp_val, int32_t P, int64_t n, int32_t k_blk,
                                     int32_t round, int32_t* drop_idx, float* drop_val, int32_t* drop_cnt,
                                     uint32_t* err, hipStream_t stream);

/* Final All-Gather and decode (end of Sec. III-B; Algorithm 1 "All-Gather all
 * blocks from all workers").  After step l, worker b holds the reduced block
 * b in sp[b][b]; the All-Gather gives every worker all P of them, which on
 * one device is the identity.  Writes the dense update once:
 *   dense[x] = value of x in the final block containing x, if x is there;
 *   dense[x] = +0.0f otherwise;     for x < n.
 * member (optional, may be NULL; 4-byte aligned, ceil(n/32) words, caller
 * owned) receives the membership bitmap of the final index set I: bit
 * (x & 31) of word (x >> 5) is 1 iff x is in I; every word is written, bits
 * at or above n are 0.  spardl_residual_collect can take it in place of
 * building I itself.
 * Errors: EINVAL for NULL sp/dense, misaligned member, P < 1, n < P,
 * n >= 2^31, k_blk out of [1, floor(n/P)]. */
int spardl_allgather_densify(const int32_t* sp_idx, const float* sp_val, int32_t P, int64_t n,
                             int32_t k_blk, float* dense, uint32_t* member, hipStream_t stream);

/* Global residual collection (Sec. III-C, Algorithm 1).  Let I be the set of
 * indices in the final blocks sp[b][b], b < P.  For every worker w < P (row w
 * of acc holds A_w = G + xi from spardl_residual_add):
 *   acc[w][x] = 0.0f           for x in I that w selected locally
 *                              (local_idx[w][*][*] from spardl_block_topk);
 *   acc[w][x] = acc[w][x] + v  for every in-procedure drop (x, v) of w with
 *                              x in I, steps 1..l in that order;
 *   other entries keep A_w    (local and end-procedure residuals).
 * The result is xi^t_w, the residual for the next iteration.
 * I is read from member when it is given (the bitmap spardl_allgather_densify
 * wrote for the same final blocks; sp_idx and ws are then unused and may be
 * NULL), else built from sp_idx in the workspace's bitmap, which is left at
 * zero again.
 * drop_idx/drop_val/drop_cnt are HOST arrays of l DEVICE pointers (element
 * i-1 = the buffers passed to spardl_sparse_merge_topk for step i); they may
 * be NULL when P = 1.
 * Errors: EINVAL for NULL acc/local_idx, NULL sp_idx or ws (or a ws not
 * 256-byte aligned) without member, misaligned member, P < 1, n < P,
 * n >= 2^31, ld_acc < n, k_blk out of [1, floor(n/P)]; ECAPACITY if ws is
 * too small. */
int spardl_residual_collect(float* acc, int64_t ld_acc, int32_t P, int64_t n, int32_t k_blk,
                            const int32_t* local_idx, const int32_t* sp_idx, const uint32_t* member,
                            const int32_t* const* drop_idx, const float* const* drop_val,
                            const int32_t* const* drop_cnt, void* ws, size_t ws_bytes,
                            hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Lazy sparsification (Sec. III-B "Optimization for SRS"; Algorithm 1).
 * Held blocks stay dense: a worker sparsifies a block only right before it
 * sends it (and its reserved block after the last step), and a receiver adds
 * the received entries into its dense row.  One step, for P workers whose
 * rows are acc[w*ld_acc ...] (A_w after spardl_residual_add), is:
 *   for round = 1..l: spardl_lazy_topk(round) on every worker, then
 *                     spardl_lazy_receive(round);
 *   spardl_lazy_topk(0) on every worker;
 *   spardl_allgather_densify(sp, ..., member);      (final block b = sp[b][b])
 *   spardl_lazy_residual_collect(..., member, saved).
 * Every worker selects every block once, so sp[w][b] (layout as for
 * spardl_block_topk) ends holding all P x P selections.
 * Fused form (all P rows in one workspace): the residual add with the
 * workspace (as for spardl_block_topk), every spardl_lazy_topk with
 * SPARDL_TOPK_HIST_READY and every spardl_lazy_receive with the workspace,
 * which keeps the add's histograms exact through the receipts; a selection
 * then reads its block at most once, not at all while it is unchanged since
 * the add.  Plain form: a plain add, flags 0, receipts without a workspace.
 * ------------------------------------------------------------------------- */

/* Block top-k of the blocks that workers w0 .. w0 + nworkers - 1 sparsify at
 * SRS step `round`: for round in [1, l] the bag they send at that step,
 * blocks b = (w + 2^(l-round) + t) mod P for t < bag_blocks of the step (see
 * spardl_srs_plan); for round 0 the reserved block b = w.  acc points at row
 * w0 (row w is acc + (w - w0)*ld_acc) and sp_idx/sp_val at sp[w0]:
 *   sp_idx/sp_val[((w - w0)*P + b)*k_blk + j], j < k_blk = the top-k_blk
 *   entries of block b of row w, sorted by ascending index (order as for
 *   spardl_block_topk).
 * Other blocks of sp are not written.  ws: a workspace for nworkers rows
 * (spardl_workspace_bytes(nworkers, P, n, k_blk)), prepared once.
 * flags: 0, or SPARDL_TOPK_HIST_READY in the fused form (then w0 = 0 and
 * nworkers = P).
 * Errors: EINVAL for NULL acc/sp/ws, misaligned ws, nworkers < 1, w0 < 0,
 * w0 + nworkers > P, P < 1, n < P, n >= 2^31, ld_acc < n, k_blk outside
 * [1, floor(n/P)], round outside [0, l], unknown flags, HIST_READY with a
 * row subset; ECAPACITY if ws is too small. */
int spardl_lazy_topk(const float* acc, int64_t ld_acc, int32_t w0, int32_t nworkers, int64_t n, int32_t P,
                     int32_t k_blk, int32_t round, int32_t flags, int32_t* sp_idx, float* sp_val, void* ws,
                     size_t ws_bytes, hipStream_t stream);

/* Transmission and summation of SRS step `round` in [1, l] (Algorithm 1),
 * all P workers at once.  With d = 2^(l-round) and m = bag_blocks of the
 * step, worker w sent sp[w][b], b = (w + d + t) mod P, t < m, to worker
 * r = (w + d) mod P, which adds each entry into its dense row:
 *   saved[(w*P + b)*k_blk + j] = acc[r][x];  acc[r][x] = acc[r][x] + v
 * for (x, v) = entry j of sp[w][b].  saved (device, P*P*k_blk floats, caller
 * owned, same layout as sp) keeps what was overwritten for
 * spardl_lazy_residual_collect; each (w, b) is sent at exactly one step, so
 * one buffer serves all steps.  Entries whose index lies outside block b are
 * skipped.  Steps must run in order 1..l, each after spardl_lazy_topk of the
 * same round on every worker.  ws (optional): the fused form's workspace for
 * all P rows; the receipt then updates the receiving block's histogram and
 * marks the block as changed since the add.
 * Errors: EINVAL for NULL pointers, P < 2 (no steps), n < P, n >= 2^31,
 * ld_acc < n, k_blk outside [1, floor(n/P)], round outside [1, l], a
 * misaligned ws; ECAPACITY if ws is smaller than
 * spardl_workspace_bytes(P, P, n, k_blk). */
int spardl_lazy_receive(float* acc, int64_t ld_acc, int32_t P, int64_t n, int32_t k_blk, int32_t round,
                        const int32_t* sp_idx, const float* sp_val, float* saved, void* ws, size_t ws_bytes,
                        hipStream_t stream);

/* Residual collection of the lazy step (Algorithm 1: "Replace part of
 * G_copy at indexes I_i with xi_i").  With I the final index set given by
 * member (the bitmap spardl_allgather_densify wrote), for every worker w:
 *   acc[w][x] = 0.0f       for x in I that w selected (x in sp[w][b], any b);
 *   acc[w][x] = A_w[x]     for x not in I that w received at some step (the
 *                          value saved before the first receipt);
 *   other entries keep acc: A_w off I, and on I what w held but did not send.
 * The result is xi^t_w.  saved: the buffer spardl_lazy_receive filled (may
 * be NULL when P = 1).
 * Errors: EINVAL for NULL acc/sp_idx/member, misaligned member, NULL saved
 * with P > 1, P < 1, n < P, n >= 2^31, ld_acc < n, k_blk outside
 * [1, floor(n/P)]. */
int spardl_lazy_residual_collect(float* acc, int64_t ld_acc, int32_t P, int64_t n, int32_t k_blk,
                                 const int32_t* sp_idx, const uint32_t* member, const float* saved,
                                 hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Spar-All-Gather across d teams, recursive form (R-SAG; Sec. III-D, d a
 * power of 2).  P workers form d teams of Q = P / d consecutive workers
 * (team tau = workers tau*Q .. tau*Q + Q - 1).  Each team runs the d = 1
 * calls above on its own rows with Q in place of P and k_blk = L(k, d, P) =
 * d k / P: its rows of acc, its Q x Q x k_blk slice of sp (rows tau*Q ..),
 * its own workspace.  After the team's SRS the worker at position q holds
 * block q in sp[tau*Q + q][q].  Then, for t = 0 .. log2(d) - 1:
 *   spardl_rsag_merge_topk(t);
 * then the final blocks are sp[q][q], q < Q (any team): decode them with
 * spardl_allgather_densify(sp, P = Q, ..., member) and collect residuals per
 * team with spardl_residual_collect(..., member) (or all teams at once with
 * spardl_team_residual_collect), then
 * spardl_rsag_residual(..., member).  sp below is the whole P x Q x k_blk
 * array (row w = worker w, Q blocks per row).
 * ------------------------------------------------------------------------- */

/* All d teams in one call (the same results as the calls above team by team,
 * with fewer and larger launches): a workspace for P rows of Q = P / d blocks,
 * 256-byte aligned, spardl_team_workspace_bytes(P, d, n, k_blk) bytes,
 * prepared once by spardl_team_workspace_init.  0 on invalid sizes: P < 1,
 * d < 1, d not dividing P, n < Q, n >= 2^31, k_blk outside [1, floor(n/Q)]. */
size_t spardl_team_workspace_bytes(int32_t P, int32_t d, int64_t n, int32_t k_blk);
int spardl_team_workspace_init(int32_t P, int32_t d, int64_t n, int32_t k_blk, void* ws, size_t ws_bytes,
                               hipStream_t stream);

/* spardl_residual_add (with the workspace) for all P rows, blocks of the
 * team's Q-block partition.  Errors: EINVAL for NULL pointers, misaligned
 * ws, invalid sizes, ld < n; ECAPACITY if ws is too small. */
int spardl_team_residual_add(float* acc, int64_t ld_acc, const float* grad, int64_t ld_grad, int32_t P, int32_t d,
                             int64_t n, int32_t k_blk, void* ws, size_t ws_bytes, hipStream_t stream);

/* spardl_block_topk for all P rows, Q blocks each: sp_idx/sp_val/local_idx
 * [(w*Q + b)*k_blk + j].  flags: 0 or SPARDL_TOPK_HIST_READY (after
 * spardl_team_residual_add with the same workspace).  Errors as for
 * spardl_team_residual_add, plus unknown flags. */
int spardl_team_block_topk(const float* acc, int64_t ld_acc, int32_t P, int32_t d, int64_t n, int32_t k_blk,
                           int32_t flags, int32_t* sp_idx, float* sp_val, int32_t* local_idx, void* ws,
                           size_t ws_bytes, hipStream_t stream);

/* spardl_sparse_merge_topk step `round` in [1, ceil(log2 Q)] inside every
 * team at once: pair (tau Q + w)*m + t merges block (w + t) mod Q of row
 * tau Q + w with that block of row tau Q + (w - 2^(l-round)) mod Q; drops at
 * drop_idx/drop_val[((tau Q + w)*m + t)*k_blk + j], j < drop_cnt[...].
 * Errors as for spardl_team_residual_add, plus round out of range. */
int spardl_team_merge_topk(int32_t* sp_idx, float* sp_val, int32_t P, int32_t d, int64_t n, int32_t k_blk,
                           int32_t round, int32_t* drop_idx, float* drop_val, int32_t* drop_cnt, void* ws,
                           size_t ws_bytes, hipStream_t stream);

/* spardl_residual_collect(..., member) for all P rows at once (Sec. III-C,
 * global residual collection inside every team): worker w's residual keeps
 * what it selected or dropped at the team's SRS steps minus the final
 * indices.  local_idx as written by spardl_team_block_topk; member the
 * bitmap spardl_allgather_densify wrote (required); drop_idx / drop_val /
 * drop_cnt HOST arrays of ceil(log2 Q) DEVICE pointers, element i-1 = the
 * buffers of spardl_team_merge_topk round i (may be NULL when Q = 1).  No
 * workspace.  Errors: EINVAL for NULL acc/local_idx/member or a NULL drop
 * pointer, misaligned member, invalid sizes (as for the team workspace),
 * ld_acc < n. */
int spardl_team_residual_collect(float* acc, int64_t ld_acc, int32_t P, int32_t d, int64_t n, int32_t k_blk,
                                 const int32_t* local_idx, const uint32_t* member, const int32_t* const* drop_idx,
                                 const float* const* drop_val, const int32_t* const* drop_cnt, hipStream_t stream);

/* Workspace of spardl_rsag_merge_topk (separate from the teams' workspaces):
 * 256-byte aligned device memory of this many bytes, prepared once by
 * spardl_rsag_workspace_init (it rests at zero between calls, except the
 * error word).  0 on invalid sizes: P < 2, d < 2, d not a power of 2, d not
 * dividing P, n < Q, n >= 2^31, k_blk outside [1, floor(n / Q)]. */
size_t spardl_rsag_workspace_bytes(int32_t P, int32_t d, int64_t n, int32_t k_blk);
int spardl_rsag_workspace_init(int32_t P, int32_t d, int64_t n, int32_t k_blk, void* ws, size_t ws_bytes,
                               hipStream_t stream);

/* R-SAG exchange t in [0, log2 d) (Sec. III-D): team X and team X xor 2^t
 * exchange, for every position q < Q, the block q their workers hold; both
 * add the other's entries by index (held + received) and keep the top k_blk,
 * so both hold the same block.  Pair p < (d/2)*Q is (j, q) = (p / Q, p % Q),
 * X = j with a 0 bit inserted at bit t, Y = X + 2^t:
 *   sp[X*Q + q][q] and sp[Y*Q + q][q] <- the kept entries (sorted by index);
 *   drop_idx/drop_val[p*k_blk + j], j < drop_cnt[p] <- the dropped ones.
 * Errors: EINVAL for NULL pointers, misaligned ws, invalid sizes (see
 * spardl_rsag_workspace_bytes), t outside [0, log2 d); ECAPACITY if ws is
 * smaller than spardl_rsag_workspace_bytes. */
int spardl_rsag_merge_topk(int32_t* sp_idx, float* sp_val, int32_t P, int32_t d, int64_t n, int32_t k_blk,
                           int32_t t, int32_t* drop_idx, float* drop_val, int32_t* drop_cnt, void* ws,
                           size_t ws_bytes, hipStream_t stream);

/* Residual share of the R-SAG drops (Sec. III-D): 2^(t+1) workers made the
 * identical merge at exchange t, so each adds 2^-(t+1) of every value its
 * pair dropped, at final indices only:
 *   acc[w][x] = acc[w][x] + 2^-(t+1) * v   for w in {X*Q + q, Y*Q + q} of
 *   pair p, every drop (x, v) of p with x in I (member), t = 0, 1, ... in
 *   that order.
 * Run after the teams' spardl_residual_collect.  drop_idx/drop_val/drop_cnt
 * are HOST arrays of log2(d) DEVICE pointers (element t = the buffers of
 * exchange t).
 * Errors: EINVAL for NULL pointers, misaligned member, invalid sizes,
 * ld_acc < n. */
int spardl_rsag_residual(float* acc, int64_t ld_acc, int32_t P, int32_t d, int64_t n, int32_t k_blk,
                         const uint32_t* member, const int32_t* const* drop_idx, const float* const* drop_val,
                         const int32_t* const* drop_cnt, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Spar-All-Gather across d teams, Bruck form (B-SAG; Sec. III-D, any d >= 2
 * dividing P) with the compression-ratio controller of Algorithm 2.  Teams,
 * their SRS and sp (P x Q x k_blk, k_blk = L = d k / P) as for R-SAG.  After
 * the teams' SRS:
 *   spardl_bsag_exchange(...);   final block q in sp[q][q], padded
 *   spardl_allgather_densify(sp, P = Q, ..., member);
 *   spardl_residual_collect(...) per team (with member), then
 *   spardl_bsag_residual(..., member).
 * ------------------------------------------------------------------------- */

/* Workspace of spardl_bsag_exchange: 256-byte aligned, this many bytes,
 * prepared once by spardl_bsag_workspace_init, which also sets Algorithm 2's
 * initial state for every block (h = L/d, step = 0.01 (d-1) L / d, flag
 * false, no previous count).  The workspace carries that state from step to
 * step.  0 on invalid sizes: P < 2, d < 2, d not dividing P, n < Q,
 * n >= 2^31, k_blk outside [1, floor(n / Q)]. */
size_t spardl_bsag_workspace_bytes(int32_t P, int32_t d, int64_t n, int32_t k_blk);
int spardl_bsag_workspace_init(int32_t P, int32_t d, int64_t n, int32_t k_blk, void* ws, size_t ws_bytes,
                               hipStream_t stream);

/* One B-SAG exchange (Sec. III-D; Algorithm 2), for every block q < Q:
 *  1. Algorithm 2 updates block q's state from the previous union size and
 *     gives the count h_q (in [1, k_blk]);
 *  2. every holder w = tau*Q + q keeps the top h_q of sp[w][q]; the other
 *     k_blk - h_q entries go to drop_idx/drop_val[w*k_blk + j],
 *     j < drop_cnt[w], sorted by index (its own residual);
 *  3. the d kept lists are summed by index in team order (the result of the
 *     Bruck All-Gather, the same on every holder); N_q = its size;
 *  4. sp[q][q] (team 0's holder) <- the top k_blk of that sum, or all of it
 *     when N_q <= k_blk, sorted by index and padded to k_blk entries with
 *     index INT32_MAX, value 0 (spardl_allgather_densify and the residual
 *     calls skip such entries).
 * info (optional, device, 2*Q int32): info[q] = h_q, info[Q + q] = N_q.
 * Errors: EINVAL for NULL pointers, misaligned ws, invalid sizes (see
 * spardl_bsag_workspace_bytes); ECAPACITY if ws is too small. */
int spardl_bsag_exchange(int32_t* sp_idx, float* sp_val, int32_t P, int32_t d, int64_t n, int32_t k_blk,
                         int32_t* drop_idx, float* drop_val, int32_t* drop_cnt, int32_t* info, void* ws,
                         size_t ws_bytes, hipStream_t stream);

/* Residual share of the top-h drops: every worker w adds its own drops
 * (drop_idx/drop_val/drop_cnt of spardl_bsag_exchange) at final indices:
 *   acc[w][x] = acc[w][x] + v   for every drop (x, v) of w with x in I.
 * Run after the teams' spardl_residual_collect.  The final selection's drops
 * need no share: none of their indices is final, and off I every worker
 * keeps its own A.
 * Errors: EINVAL for NULL pointers, misaligned member, invalid sizes,
 * ld_acc < n. */
int spardl_bsag_residual(float* acc, int64_t ld_acc, int32_t P, int32_t d, int64_t n, int32_t k_blk,
                         const uint32_t* member, const int32_t* drop_idx, const float* drop_val,
                         const int32_t* drop_cnt, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* SPARDL_H */
