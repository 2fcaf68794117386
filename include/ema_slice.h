/*
 * ema_slice.h -- C ABI of the memory-slice hot path on one MI355X (gfx950).
 *
 * The method is EMA's memory slice ("Elastic and Performance Transparent Memory
 * Across GPUs"): a borrower keeps part of its paged KV cache in memory lent by
 * a peer, prefetches it into local memory before use so remote and local
 * blocks perform alike (local-remote symmetry, section 3), and the lender can
 * reclaim what it lent at any time (static-dynamic symmetry, sections 3 and
 * 4.1). Here the slice is a second, separately allocated HBM region of the
 * same GPU standing in for the peer's share.
 *
 * Objects
 *   layer-block   K and V of `block_size` consecutive tokens, all KV heads,
 *                 one layer; 2*block_size*num_kv_heads*head_dim*2 bytes.
 *   local pool    n_local layer-blocks; always in EMA_LAYOUT_ATTN.
 *   slice pool    n_slice layer-blocks in the shape's slice_layout; slots at
 *                 or above `lim` are held by the lender.
 *   unified id    u < n_local: local block u; u >= n_local: slice slot
 *                 u - n_local; -1: padding. Ids of different layers are
 *                 different blocks (the pools are flat).
 *   owner tag     >= 0: a sequence; EMA_FREE; EMA_STAGING (a local block that
 *                 holds a prefetched copy); EMA_LENDER (slice slot at/above lim).
 *
 * Layouts of one layer-block (16-bit elements, K half first, then V half):
 *   EMA_LAYOUT_ATTN  K[kv_head][token][channel], V[kv_head][channel][token]
 *   EMA_LAYOUT_NHD   K[token][kv_head][channel], V[token][kv_head][channel]
 *
 * Conventions
 *   Return value: EMA_OK or a negative EMA_ERR_*; ema_last_error() gives a
 *   message (thread-local). No C++ exception leaves the library. Host
 *   bookkeeping is all-or-nothing: on error no state changes, except that a
 *   HIP error raised after a call's bookkeeping took effect (reclaim; see
 *   there) leaves that bookkeeping in place.
 *   Pointers marked "device" are HIP device pointers owned by the caller;
 *   "host" pointers are ordinary memory. The library owns both pools.
 *   Entry points make the handle's device current while they run and give
 *   the caller's current device back before returning.
 *   `stream` is a hipStream_t (NULL = the null stream). Kernels are enqueued
 *   asynchronously; host bookkeeping changes at call time. Ordering across
 *   streams is the caller's job (events).
 *   A handle is not thread-safe. Attention calls on one handle share its
 *   split-K workspace: do not run two of them concurrently on different
 *   streams. Reclaim and run prefetches share the handle's plan upload area
 *   and order themselves on the device (a later call's stream waits for the
 *   earlier call's kernels), so they may be issued on different streams.
 *   Device paths support head_dim 128 and block_size in {16,32,64,128,256}.
 *   Device id arrays are validated on the host only when the slice was
 *   created with EMA_CREATE_CHECKED (it costs a device-to-host copy). Without
 *   it, kernels skip out-of-range ids and count them; read the count with
 *   ema_slice_device_errors().
 */
#ifndef EMA_SLICE_H
#define EMA_SLICE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define EMA_OK 0
#define EMA_ERR_INVAL (-1)   /* bad argument, range, duplicate, wrong tag  */
#define EMA_ERR_NOMEM (-2)   /* not enough free blocks (slice: below lim),
                                or host memory exhausted                   */
#define EMA_ERR_OWNER (-3)   /* freeing a block that is not allocated      */
#define EMA_ERR_HIP (-4)     /* a HIP runtime call failed                  */

#define EMA_F16 0
#define EMA_BF16 1
#define EMA_F32 2    /* attention output only */

#define EMA_LAYOUT_ATTN 0
#define EMA_LAYOUT_NHD 1

#define EMA_POOL_LOCAL 0
#define EMA_POOL_SLICE 1

#define EMA_FREE (-1)
#define EMA_STAGING (-2)
#define EMA_LENDER (-3)

#define EMA_CREATE_HOST_ONLY 1u  /* bookkeeping only: no device memory, no kernels */
#define EMA_CREATE_CHECKED 2u    /* validate device id arrays on the host          */
#define EMA_CREATE_ATTN_GRID 4u  /* attention always in the grid form (see there)  */

typedef struct ema_slice* ema_slice_t;

typedef struct {
  int32_t num_kv_heads;
  int32_t head_dim;
  int32_t block_size;     /* tokens per block */
  int32_t dtype;          /* EMA_F16 or EMA_BF16 */
  int32_t slice_layout;   /* EMA_LAYOUT_ATTN or EMA_LAYOUT_NHD */
} ema_kv_shape;

typedef struct {
  int64_t block_bytes;
  int32_t n_local;
  int32_t n_slice;
  int32_t lim;            /* slice slots currently lent */
  int32_t free_local;
  int32_t free_slice;     /* FREE slots below lim */
  int32_t device;         /* HIP device of the pools, -1 when host-only */
  void* local_base;       /* device, library-owned, n_local*block_bytes */
  void* slice_base;       /* device, library-owned, n_slice*block_bytes */
} ema_slice_info;

typedef struct {
  int32_t reclaimed;      /* slots returned to the lender: min(n, lim) */
  int32_t moved;          /* borrowed blocks copied out of the returned range */
  int32_t written_back;   /* of those, copied into the local pool */
  int32_t n_victims;      /* sequences preempted */
  int32_t lim;            /* lent slots after the call */
} ema_reclaim_result;

/*
 * slice_create -- a memory slice and the local paged cache (section 4: a slice
 * is reserved jointly and its segments are assigned one user at a time).
 * Allocates two separate device regions on the current HIP device:
 * floor(local_bytes/block_bytes) local blocks and floor(lent_bytes/block_bytes)
 * slice slots, all FREE, lim = n_slice (everything lent), plus the plan
 * upload area of reclaim and run prefetches (16 bytes per block, pinned host
 * and device) and the stream-K attention workspace (partials of one
 * workgroup per compute unit, combine records for 4096 sequences), so that
 * neither reclaim nor stream-K attention ever allocates.
 * flags: EMA_CREATE_HOST_ONLY (no device memory; copy and attention entry
 * points then take host id arrays, validate them and launch nothing),
 * EMA_CREATE_CHECKED, EMA_CREATE_ATTN_GRID.
 * Errors: INVAL (shape out of the supported range, NULL out), HIP (device
 * allocation failed; nothing is leaked).
 */
int ema_slice_create(const ema_kv_shape* shape, size_t local_bytes, size_t lent_bytes,
                     uint32_t flags, ema_slice_t* out);

/* Frees both pools and all library scratch; synchronizes the device first. */
int ema_slice_destroy(ema_slice_t h);

/* Sizes, counts and pool base addresses. */
int ema_slice_get_info(ema_slice_t h, ema_slice_info* out);

/* Copies the owner tags: own_local[n_local], own_slice[n_slice] (host). */
int ema_slice_owners(ema_slice_t h, int32_t* own_local, int32_t* own_slice);

/*
 * slice_alloc_blocks -- allocation first tries free memory (section 4.1).
 * Takes the n lowest-index FREE blocks of `pool` (slice: below lim); the i-th
 * gets owner owners[i] (>= 0, or EMA_STAGING in the local pool). Writes their
 * unified ids to out_ids[n] (host). All or nothing.
 * Errors: INVAL (bad pool, owner, n < 0), NOMEM (fewer than n free).
 */
int ema_slice_alloc_blocks(ema_slice_t h, int32_t pool, int32_t n, const int32_t* owners,
                           int32_t* out_ids);

/*
 * Returns blocks to FREE (a finished request frees its memory, section 4.2.1).
 * ids: host [n] unified ids. Errors: INVAL (range, duplicate), OWNER (a block
 * that is FREE or the lender's).
 */
int ema_slice_free_blocks(ema_slice_t h, const int32_t* ids, int32_t n);

/*
 * The lender contributes slots again (section 6.6: an underused GPU lends its
 * free memory): lim <- min(n_slice, lim + n_blocks); the slots become FREE.
 * *added (host, may be NULL) receives the number added. Errors: INVAL (n < 0).
 */
int ema_slice_lend(ema_slice_t h, int32_t n_blocks, int32_t* added);

/*
 * slice_prefetch -- the slice process prefetches data to the accessing GPU
 * ahead of use (section 5.1), in large transfers (section 4.2). For i < n:
 * local block dst_block_table[i] <- slice block block_ids[i], re-laid from the
 * slice layout into EMA_LAYOUT_ATTN. block_ids: device [n] unified ids of
 * owned slice slots; dst_block_table: device [n] unified ids of EMA_STAGING
 * local blocks, no duplicates. Canonical placement does not change: the
 * destination holds a copy. Async on `stream`.
 * Errors (checked mode or host-only): INVAL for any violation above.
 */
int ema_slice_prefetch(ema_slice_t h, const int32_t* block_ids, const int32_t* dst_block_table,
                       int32_t n, void* stream);

#define EMA_ENGINE_KERNEL 0  /* copy runs with the gather kernel (compute units)      */
#define EMA_ENGINE_DMA 1     /* copy runs with the copy engines, one transfer per run */

/*
 * slice_prefetch_runs -- prefetch of contiguous runs (section 4.2: the slab and
 * layer-group layouts keep a user's data physically contiguous so that a swap
 * is a few large transfers). For r < n_runs: the run_blocks[r] local blocks
 * from dst_first[r] <- the slice blocks from src_first[r], i.e. block
 * dst_first[r] + k <- block src_first[r] + k for k < run_blocks[r] (unified
 * ids; host arrays, so the call can issue one transfer per run). Sources must
 * be owned slice blocks, destinations EMA_STAGING local blocks, no block named
 * twice. engine EMA_ENGINE_KERNEL expands the runs into one block list for the
 * gather kernel (any slice layout); EMA_ENGINE_DMA issues one device-to-device
 * transfer per run on the copy engines, leaving the compute units free (slice
 * in EMA_LAYOUT_ATTN only: the engines copy bytes as they are). The list
 * upload uses the handle's plan upload area (see the conventions above).
 * Async on `stream`. Errors: INVAL (validated on the host in every mode),
 * HIP.
 */
int ema_slice_prefetch_runs(ema_slice_t h, const int32_t* src_first, const int32_t* dst_first,
                            const int32_t* run_blocks, int32_t n_runs, int32_t engine,
                            void* stream);

/*
 * slice_migrate -- moves logical blocks between pools, the borrower-side step of
 * dynamic sharing (section 4: each segment of the slice serves one user at a
 * time, is handed out when needed and can change hands later; section 4.1:
 * allocation first tries free memory, so a block placed locally can later
 * move into a lent slot and back). Block dst_ids[i] <- block src_ids[i]
 * (device [n] unified ids; each destination already allocated to the
 * source's owner; no duplicate destinations; sources and destinations
 * disjoint), re-laid into the destination pool's layout. The caller then
 * frees the sources and updates its tables. Async on `stream`.
 * Errors (checked mode or host-only): INVAL.
 */
int ema_slice_migrate(ema_slice_t h, const int32_t* src_ids, const int32_t* dst_ids, int32_t n,
                      void* stream);

/*
 * slice_writeback -- swap-out of modified staged copies (section 4: data swapped
 * in must be matched by data swapped out; since a prefetch leaves the slice
 * block in place, only blocks written since their prefetch need to travel).
 * For i < n: slice block slice_ids[i] <- local block staging_ids[i], re-laid
 * from EMA_LAYOUT_ATTN into the slice layout. staging_ids: device [n] unified
 * ids of EMA_STAGING local blocks; slice_ids: device [n] unified ids of owned
 * slice slots, no duplicates. Async on `stream`.
 * Errors (checked mode or host-only): INVAL for any violation above.
 */
int ema_slice_writeback(ema_slice_t h, const int32_t* staging_ids, const int32_t* slice_ids,
                        int32_t n, void* stream);

/*
 * kv_append -- a decode step stores each sequence's new token before attention
 * reads it (section 2.3 and 4.2.2: decode appends to the KV cache every step,
 * and data swapped in through the swap buffer must later be swapped out; the
 * append lands in the staged copy that the swap-out returns): for sequence b
 * with seq_lens[b] > 0 (lengths already counting the new token), the token at
 * position p = seq_lens[b] - 1 gets K = k_new[b] and V = v_new[b] in row p %
 * block_size of local block block_table[b][p / block_size]. block_table is an
 * attention table (device [batch][max_blocks] local ids): a slice-resident
 * block is named by its staged copy, which the caller then writes back with
 * ema_slice_writeback. k_new, v_new: device [batch][num_kv_heads][head_dim] in
 * the slice's dtype. Async on `stream`. Rows whose block index is >= max_blocks
 * or whose id is not a local block are skipped and counted
 * (ema_slice_device_errors); checked mode rejects them on the host first
 * (INVAL), and host-only mode validates host arrays.
 */
int ema_kv_append(ema_slice_t h, const void* k_new, const void* v_new, const int32_t* block_table,
                  const int32_t* seq_lens, int32_t batch, int32_t max_blocks, void* stream);

/*
 * slice_reclaim -- the lender takes back n_blocks lent slots (section 4.1:
 * reclamation works on logical ownership and preempts the borrower's requests
 * until the allocation is satisfied; a preempted request releases its local
 * and remote blocks together, the dependency chain of section 4.1).
 *   1. n' = min(n_blocks, lim); the top range [lim - n', lim) is returned.
 *   2. movers: slots in that range owned by a sequence, ascending.
 *   3. destinations: FREE slice slots below the range ascending, then FREE
 *      local blocks ascending.
 *   4. while movers outnumber destinations, the owner with the most movers
 *      (ties: larger id) is preempted and every block it holds becomes FREE.
 *   5. mover i is copied to destination i on `stream` (written-back blocks
 *      are re-laid into EMA_LAYOUT_ATTN) and takes its owner.
 *   6. the range becomes EMA_LENDER, lim drops by n', and every entry t of
 *      canon_tables (device int32 [n_entries], rewritten in place on
 *      `stream`) becomes: the destination if t was a mover, -1 if t was a
 *      preempted sequence's block, else t.
 * result (host, required), victims (host [victims_cap], may be NULL): the
 * preempted owners in order; moves_src/moves_dst (host [moves_cap], may be
 * NULL): the copies made. Counts beyond a cap are still reported in result.
 * In host-only mode canon_tables must be NULL with n_entries 0.
 * Device work: when nothing is preempted and the movers form at most 24
 * contiguous runs, one launch with the runs in its arguments (no upload);
 * otherwise one upload of the plan (4 bytes per mover twice, per slot of the
 * returned range, and a bitmap over the span of the released blocks outside
 * it) from the handle's pinned buffer, then one launch that copies the movers
 * and, in its first workgroups, rewrites the tables. The upload area is shared with run
 * prefetches (see the conventions above): before overwriting it, a reclaim
 * waits on the host for the previous upload to leave the pinned buffer and
 * makes `stream` wait for the kernels that read the previous plan.
 * Errors: INVAL (n_blocks < 0, n_entries < 0, bad table pointer), HIP. The
 * bookkeeping changes before the copies are enqueued: after a HIP error the
 * ownership and lim already reflect the plan, while the copies and the table
 * rewrite may not have run.
 */
int ema_slice_reclaim(ema_slice_t h, int32_t n_blocks, int32_t* canon_tables, int64_t n_entries,
                      void* stream, ema_reclaim_result* result, int32_t* victims,
                      int32_t victims_cap, int32_t* moves_src, int32_t* moves_dst,
                      int32_t moves_cap);

/*
 * paged_decode_attention -- one decode token per sequence over its paged KV
 * cache in the local pool (the per-token compute whose latency must not
 * depend on where a block started, section 6.4). For sequence b and query
 * head hq, with kv head g = hq / (num_q_heads / num_kv_heads):
 *   out[b][hq] = sum_t softmax_t(scale * q[b][hq] . K_t) V_t, t < seq_lens[b],
 * token t read from row t % block_size of local block block_table[b][t / bs].
 * q: device [batch][num_q_heads][head_dim] in the slice's dtype.
 * block_table: device int32 [batch][max_blocks] local ids (slice ids are an
 * error; read the prefetched staging copies instead). seq_lens: device int32
 * [batch], each <= max_blocks*block_size; 0 gives zeros. scale <= 0 means
 * 1/sqrt(head_dim). out: device [batch][num_q_heads][head_dim] of out_dtype:
 * EMA_F32 (fp32 accumulation stored as is), or EMA_BF16 / EMA_F16 (the same
 * fp32 result rounded to nearest even).
 * The result does not depend on which local blocks hold the tokens, bit for
 * bit. Async on `stream`.
 * Scheduling: stream-K over all (sequence, KV head) pairs when batch <= 4096
 * (2048 at 16 query heads per KV head), in the workspace allocated at create;
 * otherwise, or with EMA_CREATE_ATTN_GRID, a grid of 1024-token chunks whose
 * split-K workspace grows on first use (which synchronizes the device, frees
 * the smaller workspace -- graphs captured earlier with grid-form calls must
 * not be replayed afterwards -- and is refused while `stream` is capturing).
 * Errors: INVAL (num_q_heads not a multiple of num_kv_heads or group > 16,
 * batch/max_blocks < 0, unsupported shape or out_dtype, workspace growth
 * during capture), HIP.
 */
int ema_paged_decode_attention(ema_slice_t h, const void* q, const int32_t* block_table,
                               const int32_t* seq_lens, int32_t batch, int32_t num_q_heads,
                               int32_t max_blocks, float scale, void* out, int32_t out_dtype,
                               void* stream);

/*
 * paged_decode_attention_noalloc -- for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): the same computation, arguments and result as
 * ema_paged_decode_attention, always in the stream-K form, with its partials
 * and combine records in a fixed per-GPU workspace (a file-scope device array
 * of about 8.9 MB, held by each GPU the library runs on until the process
 * ends) instead of the handle's. The call allocates nothing, on the device or
 * on the host, and never reads device arrays back (on a checked handle it
 * validates nothing on the host; kernels still skip and count invalid ids).
 * All calls on one GPU share that workspace: calls that may overlap on one
 * GPU (different streams, or concurrent host threads) race on it and must be
 * ordered by the caller. Nothing in it needs clearing: each call writes every
 * record it reads.
 * Limits: batch <= 4096 (2048 at 16 query heads per KV head),
 * batch * num_kv_heads <= 32768, at most 512 compute units; beyond them the
 * call returns INVAL and does nothing. Other errors as for
 * ema_paged_decode_attention.
 */
int ema_paged_decode_attention_noalloc(ema_slice_t h, const void* q, const int32_t* block_table,
                                       const int32_t* seq_lens, int32_t batch,
                                       int32_t num_q_heads, int32_t max_blocks, float scale,
                                       void* out, int32_t out_dtype, void* stream);

/*
 * Error accounting of the unchecked mode (no passage: a property of this
 * library). Synchronizes the device, then reads and clears the number of ids
 * the kernels skipped as out of range since the last call (0 when all were
 * valid).
 */
int ema_slice_device_errors(ema_slice_t h, int32_t* count);

/*
 * ---- Slab management of the slice (sections 4.2.1-4.2.3) ----
 *
 * A slab is `slab_blocks` (S) block positions, the same positions in every
 * one of `layers` (L) layers, so one slab spans L*S slice slots; a slab
 * belongs to one user at a time: the lender, nobody (lent, free) or the
 * borrower. A borrowed slab's positions each hold one logical block of one
 * sequence, in all L layers at once, or are free. Placement of (slab i,
 * layer l, position p) among the slice slots, n slabs, k = group:
 *   EMA_SLAB_LAYER_MAJOR  (l*n + i)*S + p                  (section 4.2.1)
 *   EMA_SLAB_SLAB_MAJOR   (i*L + l)*S + p                  (section 4.2.2)
 *   EMA_SLAB_GROUP_MAJOR  ((l/k*n + i)*k + l%k)*S + p      (section 4.2.3)
 * In slab mode the slice's blocks are allocated, freed and reclaimed only by
 * the ema_slab_* calls (ema_slice_alloc_blocks on the slice pool,
 * ema_slice_free_blocks of slice ids and ema_slice_reclaim return INVAL);
 * ema_slice_lend lends slabs (the lowest-indexed of the lender's); the local
 * pool, migrate, prefetch, write-back, append and attention work as before,
 * a slab position's owner being the owner of its L slots.
 */
#define EMA_SLAB_LAYER_MAJOR 0
#define EMA_SLAB_SLAB_MAJOR 1
#define EMA_SLAB_GROUP_MAJOR 2
#define EMA_BORROWED (-4)   /* slab tag: the borrower's */

typedef struct {
  int32_t layers;        /* L: layers of the cache, every slab spans all of them */
  int32_t slab_blocks;   /* S: block positions per slab */
  int32_t group;         /* k: layers per layer group (divides L) */
  int32_t layout;        /* EMA_SLAB_* */
} ema_slab_cfg;

typedef struct {
  int32_t n_slabs;       /* floor(n_slice / (L*S)); slots past them stay the lender's */
  int32_t layers, slab_blocks, group, layout;
  int32_t borrowed;      /* slabs the borrower holds */
} ema_slab_info;

typedef struct {
  int32_t reclaimed;     /* slabs returned to the lender: min(n, slabs lent) */
  int32_t n_victims;     /* sequences preempted */
  int32_t released;      /* blocks those sequences held (local and slab) */
} ema_slab_reclaim_result;

/*
 * slab_init -- manage an untouched slice (every slot lent and free, as after
 * create) in slabs: all slabs FREE (lent, unused). Device: allocates the
 * lists the layer-group swaps copy from (4 bytes per slice slot, device and
 * pinned host). Errors: INVAL (already in slabs, slice touched, layers, S or
 * group < 1, group not dividing layers, bad layout, no whole slab), HIP.
 */
int ema_slab_init(ema_slice_t h, const ema_slab_cfg* cfg);

/* Slab shape and state; slab_tag[n_slabs] (EMA_LENDER, EMA_FREE or
 * EMA_BORROWED) and pos_owner[n_slabs*S] (owner or EMA_FREE) may be NULL. */
int ema_slab_get_info(ema_slice_t h, ema_slab_info* out, int32_t* slab_tag, int32_t* pos_owner);

/*
 * slab_alloc -- a task that exhausts its memory requests more slabs (section
 * 4.2.1). One position per owners[i] (a sequence, >= 0), in order: the lowest
 * free position of the borrowed slabs (slab index order), and when those are
 * full the lowest-indexed free slab is borrowed. out_pos[n] (host) gets the
 * positions i*S + p. All or nothing. Errors: INVAL, NOMEM.
 */
int ema_slab_alloc(ema_slice_t h, int32_t n, const int32_t* owners, int32_t* out_pos);

/*
 * slab_free -- positions back to free; a borrowed slab left without a block
 * returns to the slice for either user (section 4.2.1). Errors: INVAL (range,
 * duplicate), OWNER (a free position).
 */
int ema_slab_free(ema_slice_t h, const int32_t* pos, int32_t n);

/*
 * Where a slab position's blocks live (sections 4.2.1-4.2.3: the placement
 * maps a slab, layer and position to a slice slot; section 4.2.2: a swapped
 * group is read from its copy in the swap buffer).
 * The unified ids of layer `layer`'s blocks at slab positions pos[n] (host):
 * with staging_first < 0 the slice blocks; otherwise the blocks the swap of
 * that layer's group puts them in, in the staging image that starts at local
 * block staging_first (their slabs must be borrowed). Errors: INVAL.
 */
int ema_slab_block_ids(ema_slice_t h, const int32_t* pos, int32_t n, int32_t layer,
                       int32_t staging_first, int32_t* out_ids);

/*
 * The swap of a layer group as transfers (section 4.2.2: a group is swapped
 * at once; sections 4.2.1-4.2.3 give each placement's transfer sizes).
 * The swap of layer group `group` as runs (host arrays of cap entries; any
 * may be NULL): every borrowed slab's blocks of the group's layers, used and
 * unused positions alike, into a staging image at staging_first that keeps
 * the slice layout's order -- (j*m + r)*S + p for layer-major, (r*k + j)*S + p
 * otherwise (r: rank among the m borrowed slabs, j: layer within the group).
 * Runs are maximal ranges contiguous on both sides, in staging order, so their
 * sizes are S..mS (layer-major), kS (slab-major), kS..mkS (layer-group-major).
 * *n_runs receives the total even past cap. Errors: INVAL.
 */
int ema_slab_group_runs(ema_slice_t h, int32_t group, int32_t staging_first, int32_t* src_first,
                        int32_t* dst_first, int32_t* run_blocks, int32_t cap, int32_t* n_runs);

/*
 * slab_prefetch_group -- at a layer-group boundary the group's swap is issued
 * (section 4.2.2): local blocks staging_first + t <- the t-th block of the
 * group's swap (as above), m*k*S blocks, all of which must be EMA_STAGING
 * local blocks. engine EMA_ENGINE_KERNEL: the gather kernel over a source list
 * kept on the device (rebuilt, with one upload, only when the set of borrowed
 * slabs changed); EMA_ENGINE_DMA: one copy-engine transfer per run (slice in
 * EMA_LAYOUT_ATTN only). Async on `stream`. Errors: INVAL, HIP.
 */
int ema_slab_prefetch_group(ema_slice_t h, int32_t group, int32_t staging_first, int32_t engine,
                            void* stream);

/*
 * slab_reclaim -- the lender takes back n_slabs slabs (section 4.2.1: the
 * allocator selects the borrower's slab with the fewest active requests;
 * section 4.1: reclamation preempts requests, each releasing its whole
 * dependency chain). For each slab: the highest-indexed free slab if there is
 * one; else the borrowed slab with the fewest distinct sequences (ties: the
 * highest index), whose sequences are preempted in ascending order -- every
 * block each holds, local or in any slab, becomes free, slabs left empty
 * return to the slice -- and the slab goes to the lender. Every entry of
 * canon_tables (device int32 [n_entries], rewritten in place on `stream`)
 * naming a released block becomes -1; no data moves. slabs[slabs_cap] and
 * victims[victims_cap] (host, may be NULL) get the slabs taken and the
 * preempted sequences in order. In host-only mode canon_tables must be NULL.
 * The released blocks travel as a bitmap over their span, through the
 * handle's plan upload area (see the conventions).
 * Errors: INVAL, HIP (after the bookkeeping took effect, as for reclaim).
 */
int ema_slab_reclaim(ema_slice_t h, int32_t n_slabs, int32_t* canon_tables, int64_t n_entries,
                     void* stream, ema_slab_reclaim_result* result, int32_t* slabs,
                     int32_t slabs_cap, int32_t* victims, int32_t victims_cap);

/*
 * Slice scheduling across GPUs (section 5.2, Appendix C) and bursty
 * preemption control (section 5.3) -- host policy, no device work.
 *
 * n_gpus GPUs share one slice per unordered pair {i, j}, each of slice_units
 * units. A request owned by GPU i places its units one at a time on a slice
 * {i, j}, j != i, by Greedy-Least-Loaded: the incident slice with the lowest
 * total use (both users' units; ties: the lowest j) among those with a free
 * unit and, if GPU i is capped on it, below its cap. Releases free the
 * request's most recently placed units first. A preemption of GPU i on slice
 * {i, j} recorded while i holds more than half of the slice caps i's units
 * there at that level for cap_window ticks; another such preemption within
 * the window restarts it and lowers the cap if its level is lower; the cap
 * lifts when a window passes without one. cap_window 0 disables caps.
 * Handles are not thread-safe. Errors: INVAL (ranges, unknown request, more
 * units released than held), NOMEM (host memory).
 */
typedef struct ema_sched* ema_sched_t;
int ema_sched_create(int32_t n_gpus, int32_t slice_units, int64_t cap_window, ema_sched_t* out);
int ema_sched_destroy(ema_sched_t s);
/* Places n units of request `req` (any id >= 0) of GPU `gpu` at tick t:
 * out_peer[n] (host) gets the peer j of each unit's slice, or -1 when no
 * incident slice can take it; *placed (host, may be NULL) the number placed. */
int ema_sched_place(ema_sched_t s, int32_t gpu, int32_t req, int32_t n, int64_t t,
                    int32_t* out_peer, int32_t* placed);
/* Releases n units of request `req` of GPU `gpu`, most recent first. */
int ema_sched_release(ema_sched_t s, int32_t gpu, int32_t req, int32_t n);
/* Records a preemption of GPU `gpu` on slice {gpu, peer} at tick t. */
int ema_sched_preempted(ema_sched_t s, int32_t gpu, int32_t peer, int64_t t);
/* use[n_gpus * n_gpus] (host): use[i * n_gpus + j] = units GPU i holds on
 * slice {i, j}; cap[n_gpus * n_gpus] (host, may be NULL): GPU i's cap on that
 * slice at tick t, or -1 when none is active. */
int ema_sched_usage(ema_sched_t s, int64_t t, int32_t* use, int32_t* cap);

/* Message of the last failed call on this thread ("" if none). */
const char* ema_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* EMA_SLICE_H */
