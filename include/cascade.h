/*
 * cascade.h -- C ABI of the MI355X (gfx950) Cascade scheduling step.
 *
 * Cascade (arXiv 2608.06557) gives every request a latency budget: its
 * class TTFT target minus the predicted remaining service time (Section 4.2,
 * eq:est_latency and eq:budget_eq), reduced by the time it has waited
 * (eq:rem_budget_eq).  One scheduling iteration (Algorithm 1, Phase 2, and the
 * memory management of Section 4.4) is computed here in one call:
 *
 *   1. budget of every queued / running request, its Tier-1 / Tier-2 queue,
 *   2. its memory action: retain in HBM, restore or prefetch a prefix from
 *      DRAM / NVMe (eq:restore_time, eq:max_restorable), recompute, or be
 *      preempted with a spill to DRAM or a drop (Section 4.4),
 *   3. least-remaining-budget-first order and admission under the batch token
 *      cap (chunked prefill) and the HBM KV-block capacity,
 *   4. the KV block moves, executed by cascade_pack / cascade_unpack (or both
 *      in one launch by cascade_pack_unpack) between the paged HBM pool and
 *      contiguous staging buffers.
 *
 * Conventions for every entry point:
 *   - Pointers named *_dev and every array in the structs below are DEVICE
 *     pointers (hipMalloc / torch CUDA memory) owned by the caller; structs
 *     themselves are passed by host pointer and read during the call only.
 *   - Work is enqueued on `stream` (a hipStream_t, NULL = default stream) and
 *     runs asynchronously; outputs are valid once the stream has completed
 *     and info[CASCADE_INFO_STATUS] == CASCADE_OK.
 *   - The library never allocates memory, never synchronises the stream and
 *     never throws across the ABI.  Errors that the host can see (NULL
 *     pointers, parameters out of domain, sizes) are returned at once and
 *     nothing is enqueued.  Errors in device data are written to
 *     info[CASCADE_INFO_STATUS]; all outputs are unspecified then.
 *   - Calls that share a workspace must not overlap in time.
 */
#ifndef CASCADE_H
#define CASCADE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Return codes and device status values. */
#define CASCADE_OK 0
#define CASCADE_EINVAL (-1)   /* parameter or request data outside the domain */
#define CASCADE_ENOSPC (-2)   /* workspace or an output list too small */
#define CASCADE_EHIP (-3)     /* a HIP launch failed */
#define CASCADE_ETIMEOUT (-4) /* a cross-workgroup wait exceeded its bound */
#define CASCADE_EINTERNAL (-5) /* an internal consistency check failed */

/* Request state. */
#define CASCADE_QUEUED 0
#define CASCADE_RUNNING_PREFILL 1 /* some prompt tokens computed, KV rows held */
#define CASCADE_DECODE 2
/* Queue tier (Section 4 overview: Tier-1 priority queue, Tier-2 best effort). */
#define CASCADE_QT_NEW 0
#define CASCADE_QT_TIER1 1
#define CASCADE_QT_TIER2 2
/* Residency of a request's matched prefix (Section 4.1: tiers 0, 1, 2). */
#define CASCADE_KV_HBM 0
#define CASCADE_KV_DRAM 1
#define CASCADE_KV_NVME 2
#define CASCADE_KV_NONE 3
/* Memory actions (Section 1, Section 4.3, Section 4.4). */
#define CASCADE_ACT_RETAIN 1          /* KV stays (or is shared) in HBM */
#define CASCADE_ACT_RESTORE 2         /* admitted: restore_blocks prefix blocks now */
#define CASCADE_ACT_PREFETCH 3        /* not admitted: start the restore, no HBM yet */
#define CASCADE_ACT_RECOMPUTE 4       /* recompute the prefix on the GPU */
#define CASCADE_ACT_PREEMPT_OFFLOAD 5 /* preempted, blocks spilled to DRAM */
#define CASCADE_ACT_PREEMPT_DROP 6    /* preempted, blocks dropped */
#define CASCADE_ACT_SHARE 7           /* references the prefix blocks another request
                                         of its prefix group restores this step */

/* Indices into the device info array of cascade_outputs_t. */
#define CASCADE_INFO_STATUS 0
#define CASCADE_INFO_N_ADMITTED 1
#define CASCADE_INFO_N_SLOT_LIST 2
#define CASCADE_INFO_N_UNPACK 3
#define CASCADE_INFO_N_PACK 4
#define CASCADE_INFO_LEN 8

/* Per-request metadata (Section 4.4, "Per-request state"), structure of
   arrays with n entries each.  Request i's position in these arrays is its
   tie-break: ids must be strictly increasing, so equal budgets keep id order.
     slo_class   < num_classes; the class's TTFT target is params.slo_ns[c]
     state       CASCADE_QUEUED / _RUNNING_PREFILL / _DECODE
     queue_tier  tier from the previous step (CASCADE_QT_*)
     prefix_tier deepest tier holding the matched prefix (CASCADE_KV_*)
     arrival_ns  0 <= arrival <= params.t_now_ns
     n_in        prompt tokens, 1 .. 2^17
     n_out_pred  predicted output tokens, 0 .. 2^17
     n_prefix    matched prefix tokens, multiple of block_tokens, <= n_in - 1;
                 for a queued request 0 exactly when prefix_tier is NONE
     n_progress  QUEUED: 0; RUNNING_PREFILL: prompt tokens computed
                 (1 .. n_in-1); DECODE: tokens generated (0 .. 2^17)
     prefix_group optional (NULL = none): -1, or an id in [0, n) shared by
                 requests whose matched prefixes begin with the same blocks
                 (e.g. one shared system prompt or document).  Within a step,
                 a prefix in DRAM or NVMe is then restored once per group and
                 priority group (Section 4.4 prefix hit detection; the
                 paper leaves within-step sharing open): the first queued
                 DRAM/NVMe member in priority order with a positive restore
                 want restores it as usual, and every later such member of
                 the same group and priority group (decodes with Tier-1, or
                 Tier-2) takes nothing from the link cap and references the
                 first min(leader's restore blocks, own prefix blocks) blocks
                 of that restore like an HBM prefix: action
                 CASCADE_ACT_SHARE, restore_blocks = those blocks,
                 share_leader = the leader (a plain RECOMPUTE when that is 0
                 blocks).  Other requests ignore their group. */
typedef struct {
  int32_t n; /* 0 .. 2^20 */
  const uint64_t *id;
  const uint8_t *slo_class, *state, *queue_tier, *prefix_tier;
  const int64_t *arrival_ns;
  const int32_t *n_in, *n_out_pred, *n_prefix, *n_progress;
  const int32_t *prefix_group;
} cascade_requests_t;

/* Paged KV block table (CSR): request i holds HBM pool slots
   slots[row_offsets[i] .. row_offsets[i+1]).  row_offsets[0] = 0; the row of
   a queued request is empty, a running prefill holds ceil(n_progress/bt)
   blocks and a decode ceil((n_in + n_progress)/bt). */
typedef struct {
  const int32_t *row_offsets; /* n + 1 entries */
  const int32_t *slots;       /* row_offsets[n] entries, each in [0, num_blocks) */
} cascade_block_table_t;

/* HBM pool state: num_blocks slots, n_free of them listed in free_slots,
   taken in list order. */
typedef struct {
  int32_t num_blocks;
  int32_t n_free; /* 0 .. num_blocks */
  const int32_t *free_slots;
} cascade_tier_state_t;

/* Scheduling parameters (host struct, passed by value to the kernels).
   Latency estimate (Section 4.2): computing n prompt tokens that start at
   position s with dd co-scheduled decodes takes, in picoseconds,
     ceil(n/chunk_tokens)*(c_iter_ps + dd*c_decode_ps) + n*c_token_ps
       + c_attn_ps * n*(2s+n+1)/2
   under the actual load dd = load_decodes and the maximum load
   dd = max_batch - 1.  Links (eq:restore_time): [0] DRAM->HBM, [1]
   NVMe->DRAM, each a fixed overhead in ns and a time per KV block in ns.
   Domain: 0 <= t_now < 2^62; 1 <= num_classes <= 16; 0 <= slo_ns <= 2^50;
   1 <= block_tokens <= 2^16; 16 <= chunk_tokens <= 2^20; 1 <= max_batch <=
   4096; 0 <= load_decodes < max_batch; 2^16 <= gamma_q16 <= 2^20 (gamma in
   Q16, >= 1); c_iter, c_decode >= 0 and c_iter + max_batch*c_decode <= 2^36;
   0 <= c_token <= 2^28; 0 <= c_attn <= 2^16; 0 <= link_delta <= 2^40;
   1 <= link_blk <= 2^32; 1 <= token_cap <= 2^24; 0 <= tier2_reserve_q16 <=
   65536 (share of the token cap kept for Tier-2 when Tier-2 is non-empty);
   max_move_blocks >= 0 (restore + prefetch blocks per step, the link
   constraint of eq:opt_goal_compact). */
typedef struct {
  int64_t t_now_ns;
  int32_t num_classes;
  int64_t slo_ns[16];
  int32_t block_tokens, chunk_tokens, load_decodes, max_batch;
  int32_t gamma_q16;
  int64_t c_iter_ps, c_decode_ps, c_token_ps, c_attn_ps;
  int64_t link_delta_ns[2];
  int64_t link_blk_ns[2];
  int32_t token_cap, tier2_reserve_q16, max_move_blocks;
} cascade_params_t;

/* One KV block move: request, block index within that request, HBM pool slot
   and staging slot. */
typedef struct { int32_t req, blk, pool_slot, staging_slot; } cascade_move_t;

/* Outputs (device arrays of n entries unless stated, written by the step).
     budget_ns       remaining budget B_rem (eq:rem_budget_eq)
     action          CASCADE_ACT_*
     queue_tier_out  tier after this step
     tokens_granted  prompt / decode tokens scheduled this step (0 if not
                     admitted)
     restore_blocks  prefix blocks restored (RESTORE) or prefetched
                     (PREFETCH), or taken from another request's restore
                     (SHARE), 0 otherwise
     order           request index at each priority position
     alloc_begin     first slot_list index of the request's new HBM blocks,
                     -1 if not admitted; its first restore_blocks entries
                     receive the restored prefix
     alloc_count     number of new HBM blocks (0 if not admitted)
     admitted        admitted request indices in priority order
                     (info[N_ADMITTED] entries)
     slot_list       free slots, then the preempted requests' slots (back of
                     the order first, each row in order); capacity entries
     unpack_moves    one per restored block, admitted order
     pack_moves      one per block of each request preempted with a spill
     unpack_hazard   per unpack move: index of the pack move that reads the
                     pool slot this move overwrites (a preempted request's
                     slot handed to a restore), else -1; unpack_capacity
                     entries
     pack_hazard     per pack move: index of the unpack move that later
                     overwrites the slot it reads, else -1; pack_capacity
                     entries.  Both NULL (not written) or both set; they are
                     meaningful when the step ends with status CASCADE_OK.
     info            device int32[CASCADE_INFO_LEN]: status and counts.  The
                     counts are the required sizes even when a list did not
                     fit its capacity (status CASCADE_ENOSPC).
     share_leader    with a prefix_group input (required then, else not
                     written): the request whose restore a SHARE request
                     references, -1 for every other request.  The shared
                     blocks are the first restore_blocks entries of the
                     leader's allocation (alloc_begin) when both are in the
                     batch; a SHARE request outside the batch waits on its
                     leader's prefetch. */
typedef struct {
  int64_t *budget_ns;
  uint8_t *action, *queue_tier_out;
  int32_t *tokens_granted, *restore_blocks, *order, *alloc_begin, *alloc_count, *admitted;
  int32_t *slot_list;
  cascade_move_t *unpack_moves, *pack_moves;
  int32_t slot_list_capacity, unpack_capacity, pack_capacity;
  int32_t *info;
  int32_t *unpack_hazard, *pack_hazard;
  int32_t *share_leader;
} cascade_outputs_t;

/* Paged KV pool: chunk (slot, layer l, kv in {0: K, 1: V}) of chunk_bytes
   starts at base + l*layer_stride + kv*kv_stride + slot*slot_stride, for
   slot in [0, num_slots).  Staging slot j holds its 2*num_layers chunks back
   to back: chunk (j, l, kv) at ((j*num_layers + l)*2 + kv)*chunk_bytes.
   base, staging, chunk_bytes and the strides must be multiples of 16. */
typedef struct {
  void *base;
  int32_t num_layers;
  int32_t num_slots;
  int64_t chunk_bytes, layer_stride, kv_stride, slot_stride;
} cascade_kv_pool_t;

/* Workspace size in bytes needed by cascade_step for n requests.  The caller
   allocates it once (device memory, 256-byte aligned) and may reuse it for
   every step of at most n requests. */
size_t cascade_step_workspace_bytes(int32_t n);

/* One scheduling step (Algorithm 1, Phase 2 over the whole queue, with the
   estimator and budget engine of Section 4.2 and the preemption of Section
   4.4).  Returns CASCADE_OK once enqueued, CASCADE_EINVAL for NULL pointers
   (or exactly one hazard array, or a prefix_group input without a
   share_leader output), parameters out of domain or negative capacities,
   CASCADE_ENOSPC when
   workspace_bytes < cascade_step_workspace_bytes(n), CASCADE_EHIP when a
   launch fails.  Request data, block-table and free-list errors set
   info[STATUS] = CASCADE_EINVAL; lists longer than their capacity set
   CASCADE_ENOSPC. */
int cascade_step(const cascade_requests_t *requests, const cascade_block_table_t *table,
                 const cascade_tier_state_t *tier, const cascade_params_t *params,
                 const cascade_outputs_t *out, void *workspace, size_t workspace_bytes,
                 void *stream);

/* cascade_step for callers that cannot allocate device memory: code under
   HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
   The same step, on the same kernels, with the same results; the workspace
   is a fixed array inside the library instead of an argument, one per GPU,
   sized for CASCADE_NOALLOC_MAX_REQUESTS requests (about 45 MB) and held
   until the process ends.  The call allocates nothing.  Its first call on a
   device looks up that device's array (the calling thread's current
   device, which must be the stream's), so make that first call outside
   graph capture.  Every call on one GPU shares that GPU's array: calls that
   overlap in time on one GPU (streams not ordered against each other, or
   host threads) race and give undefined results.  Returns CASCADE_ENOSPC
   when requests->n exceeds CASCADE_NOALLOC_MAX_REQUESTS (nothing is
   enqueued), CASCADE_EHIP when the array cannot be located, and otherwise
   what cascade_step returns. */
#define CASCADE_NOALLOC_MAX_REQUESTS 262144
int cascade_step_noalloc(const cascade_requests_t *requests, const cascade_block_table_t *table,
                         const cascade_tier_state_t *tier, const cascade_params_t *params,
                         const cascade_outputs_t *out, void *stream);

/* KV block gather (Section 4.4 preemption spill): for each of the first
   min(*n_moves_dev, max_moves) moves, copy every (layer, K/V) chunk of HBM
   pool slot moves[m].pool_slot to staging slot moves[m].staging_slot of a
   staging buffer of staging_slots slots.  A move whose pool slot is outside
   [0, num_slots) or staging slot outside [0, staging_slots) is skipped and
   sets *status_dev = CASCADE_EINVAL (status_dev may be NULL).  Enqueue
   before cascade_unpack of the same step: a preempted request's slots may be
   restore destinations.  Returns CASCADE_EINVAL for NULL pointers,
   misalignment or a bad geometry, CASCADE_EHIP on launch failure. */
int cascade_pack(const cascade_kv_pool_t *pool, void *staging, int32_t staging_slots,
                 const cascade_move_t *moves, const int32_t *n_moves_dev, int32_t max_moves,
                 int32_t *status_dev, void *stream);

/* KV block scatter (Section 4.3 restore, final DRAM->HBM hop, Section 4.4):
   the inverse copy, staging slot -> pool slot, same rules. */
int cascade_unpack(const cascade_kv_pool_t *pool, const void *staging, int32_t staging_slots,
                   const cascade_move_t *moves, const int32_t *n_moves_dev, int32_t max_moves,
                   int32_t *status_dev, void *stream);

/* Both copies of one step in a single launch (Section 4.4: spill of the
   preempted prefills and the final DRAM->HBM hop of the restores).  The
   result equals cascade_pack(pack list) followed by cascade_unpack(unpack
   list): chunks of the two lists are interleaved over the GPU, and an unpack
   move m paired with a pack move j (unpack_hazard[m] == j and
   pack_hazard[j] == m, as cascade_step writes them) is copied by the thread
   that has just read the same chunk for pack move j, so the slot is read
   before it is overwritten.  Every unpack move is performed exactly once
   whatever the hazard arrays hold; the pack-before-unpack order is
   guaranteed for the pairs they declare, which must cover every pool slot
   that is both a pack source and an unpack destination.  Move, count and
   staging rules as for cascade_pack / cascade_unpack, each list with its own
   staging buffer; a bad move sets *status_dev = CASCADE_EINVAL and is
   skipped.  The hazard arrays hold max_pack / max_unpack entries (device).
   Returns CASCADE_EINVAL for NULL pointers, misalignment or a bad geometry,
   CASCADE_EHIP on launch failure. */
int cascade_pack_unpack(const cascade_kv_pool_t *pool, void *pack_staging,
                        int32_t pack_staging_slots, const cascade_move_t *pack_moves,
                        const int32_t *n_pack_dev, int32_t max_pack, const int32_t *pack_hazard,
                        const void *unpack_staging, int32_t unpack_staging_slots,
                        const cascade_move_t *unpack_moves, const int32_t *n_unpack_dev,
                        int32_t max_unpack, const int32_t *unpack_hazard, int32_t *status_dev,
                        void *stream);

/* The DRAM tier's side of a restore and of a spill (Section 4.4: HBM is
   allocated only at the final DRAM->HBM hop, eq:restore_time's DRAM link;
   preempted prefills are spilled to DRAM).  host_blocks is pinned host memory
   (hipHostMalloc) owned by the caller; move m's block lives at byte
   host_offsets[m] of it (host array of n_moves entries, 2*num_layers*
   chunk_bytes bytes per block, in the staging order of one block), and the
   moves must use staging slot m for move m, as cascade_step's lists do.
   cascade_restore_from_host first makes copy_stream wait for the work
   enqueued so far on compute_stream (an event recorded there), then copies
   each batch of batch_moves blocks host -> staging on copy_stream, records
   events[k % n_events] there, makes compute_stream wait on it and unpacks
   the batch on compute_stream, so the host link of batch k+1 overlaps the
   unpack of batch k.  cascade_spill_to_host packs each batch on
   compute_stream, then copies it staging -> host on copy_stream after an
   event.  n_moves is the host-known move count (e.g.
   info[CASCADE_INFO_N_UNPACK] read back) and sets the host-link copies;
   n_moves_dev is the step's device count, and moves at or past it are
   neither unpacked nor packed.  streams and events (hipEvent_t) are the
   caller's; any work before the call on compute_stream (the step) is
   ordered before the copies of both directions, and the caller
   synchronises copy_stream (spill) or compute_stream (restore) before using
   the results.  Returns CASCADE_EINVAL
   for NULL pointers or bad sizes, CASCADE_ENOSPC when n_moves exceeds
   staging_slots, CASCADE_EHIP when a copy or launch fails. */
int cascade_restore_from_host(const cascade_kv_pool_t *pool, void *staging,
                              int32_t staging_slots, const void *host_blocks,
                              const int64_t *host_offsets, const cascade_move_t *moves_dev,
                              const int32_t *n_moves_dev, int32_t n_moves, int32_t batch_moves,
                              int32_t *status_dev, void *copy_stream, void *compute_stream,
                              void *const *events, int32_t n_events);
int cascade_spill_to_host(const cascade_kv_pool_t *pool, void *staging, int32_t staging_slots,
                          void *host_blocks, const int64_t *host_offsets,
                          const cascade_move_t *moves_dev, const int32_t *n_moves_dev,
                          int32_t n_moves, int32_t batch_moves, int32_t *status_dev,
                          void *copy_stream, void *compute_stream, void *const *events,
                          int32_t n_events);

/* Prefix hit detection (Section 4.4): an index that records, for every
   cached KV block (keyed by its nonzero 64-bit prefix hash), the set of
   tiers holding it; the lookup reads its deepest tier (CASCADE_KV_HBM <
   DRAM < NVME), and a block whose set has become empty (every copy
   reclaimed, cascade_tier_reclaim) counts as not cached.  A request's
   matched prefix is the longest run of its leading prompt blocks that are
   all cached, capped at floor((n_in - 1) / block_tokens) blocks so that at
   least one prompt token is computed; its tier is the deepest over that run.
   The results are the n_prefix / prefix_tier inputs of cascade_step.

   The index is caller-owned device memory of cascade_prefix_index_bytes()
   bytes (16-byte aligned), an open-addressing table of `capacity` slots
   (a power of two in [64, 2^30]; keep it at least twice the number of
   distinct cached blocks).  cascade_prefix_index_clear empties it (a fill
   kernel, so it may be captured in a graph).  cascade_prefix_index_insert
   adds n (hash, tier) facts, each adding the tier to the block's set;
   inserts may run concurrently with each other but not with a probe or a
   reclamation.  Hash 0 or a tier above CASCADE_KV_NVME sets *status_dev =
   CASCADE_EINVAL and is skipped; a full table sets CASCADE_ENOSPC.
   cascade_prefix_probe looks up request i's block hashes
   block_hashes[block_offsets[i] .. block_offsets[i+1]) (device CSR, offsets
   starting at 0) and writes n_prefix_out[i] (tokens, a multiple of
   block_tokens) and prefix_tier_out[i] (CASCADE_KV_NONE when nothing
   matches).  Decreasing offsets, n_in < 1 or a zero hash set
   CASCADE_EINVAL.  status_dev may be NULL.  All return CASCADE_EINVAL for
   NULL pointers, a bad capacity or misalignment, CASCADE_EHIP on a failed
   launch. */
#define CASCADE_INDEX_SLOT_BYTES 16
size_t cascade_prefix_index_bytes(int32_t capacity);
int cascade_prefix_index_clear(void *index, int32_t capacity, void *stream);
int cascade_prefix_index_insert(void *index, int32_t capacity, const uint64_t *hashes,
                                const uint8_t *tiers, int32_t n, int32_t *status_dev,
                                void *stream);
int cascade_prefix_probe(const void *index, int32_t capacity, int32_t n,
                         const int32_t *block_offsets, const uint64_t *block_hashes,
                         const int32_t *n_in, int32_t block_tokens, int32_t *n_prefix_out,
                         uint8_t *prefix_tier_out, int32_t *status_dev, void *stream);

/* Per-tier LRU reclamation (Section 4.4, prefix hit detection: free blocks
   are reclaimed least-recently-used within each tier, so hot prefixes stay
   in the fast tiers and cold ones spill deeper).  One call frees
   need + n_incoming slots of one tier (0 HBM, 1 DRAM, 2 NVMe), all device
   memory:
     - candidates are the slots with held[s] == 0: empty slots (hash 0)
       first, then cached blocks by ascending last_use_ns, ties by the lower
       slot; the first need + n_incoming are reclaimed;
     - the reclaimed slots in ascending order give the caller freed[0 ..
       need) and receive incoming[j] (blocks the tier above demoted) in
       placed[j], j < n_incoming;
     - a reclaimed cached block of tier 0 or 1 is demoted, appended to
       outgoing in slot order, unless the index (as it was when the call
       began) has it in a deeper tier; a hash absent from the index, or no
       index, counts as held nowhere deeper.  Tier 2 drops what it reclaims.
       The caller copies each demoted block from slot src_slot of this tier
       before anything is written into that slot (for the HBM tier:
       cascade_pack / cascade_spill_to_host before the step's restores);
     - the index loses this tier for every reclaimed cached block and gains
       tier + 1 for every demoted one (hashes absent from it are skipped);
     - the slot table is updated in place: freed slots become empty (hash 0,
       last use 0), placed slots take their block's hash and last use.
   A chain HBM -> DRAM -> NVMe passes each call's outgoing / n_outgoing_dev
   as the next call's incoming / n_incoming_dev, with one status word.
   Hashes are assumed unique within a tier (one copy of a block per tier).

   table        the tier's slot table (n_slots in [0, 2^30]).
   need         slots for the caller (>= 0).
   incoming     blocks demoted into this tier, *n_incoming_dev of them
                (<= max_incoming); NULL with max_incoming 0 for none.
   outgoing     demoted blocks; max_outgoing >= need + max_incoming on tiers
                0 and 1; *n_outgoing_dev receives their count (tier 2: 0,
                outgoing may be NULL).
   freed        device int32[need]; placed device int32[max_incoming].
   index        the prefix index (NULL = none) and its capacity.
   workspace    device memory of cascade_reclaim_workspace_bytes(n_slots)
                bytes (about 24 bytes per slot: the call lists the slots it
                may reclaim), 256-byte aligned, zero-filled once before its
                first use; every call leaves its counters and histograms at
                zero again (the rest is rewritten before it is read).  A
                workspace sized for n slots serves every table of at most n
                slots.  One call at a time per workspace.
   status_dev   device int32, cleared by the caller before the first call of
                a chain.  A call that finds it nonzero does nothing.  A call
                sets CASCADE_EINVAL for a negative last use, an incoming
                hash 0 or *n_incoming_dev outside [0, max_incoming], and
                CASCADE_ENOSPC when fewer than need + n_incoming slots are
                free; then it writes nothing else.  CASCADE_ETIMEOUT or
                CASCADE_EINTERNAL report a failed cross-workgroup wait or
                consistency check.
   Alignment: block_hash and last_use_ns 16 bytes, held 2 bytes.
   Returns CASCADE_EINVAL for bad host arguments, CASCADE_EHIP on a failed
   launch.  Asynchronous on `stream`. */
typedef struct {
  int32_t n_slots;
  uint64_t *block_hash;   /* [n_slots] block in the slot, 0 = empty */
  int64_t *last_use_ns;   /* [n_slots] last access, >= 0 */
  const uint8_t *held;    /* [n_slots] nonzero = in use, never reclaimed */
} cascade_tier_table_t;

/* one demoted block: its hash, last use, and slot in the tier it leaves */
typedef struct {
  uint64_t hash;
  int64_t last_use_ns;
  int32_t src_slot, pad;
} cascade_demotion_t;

size_t cascade_reclaim_workspace_bytes(int32_t n_slots);
int cascade_tier_reclaim(int32_t tier, const cascade_tier_table_t *table, int32_t need,
                         const cascade_demotion_t *incoming, const int32_t *n_incoming_dev,
                         int32_t max_incoming, cascade_demotion_t *outgoing,
                         int32_t *n_outgoing_dev, int32_t max_outgoing, int32_t *freed,
                         int32_t *placed, void *index, int32_t index_capacity, void *workspace,
                         size_t workspace_bytes, int32_t *status_dev, void *stream);

/* The whole chain HBM -> DRAM -> NVMe of per-tier LRU reclamation (Section
   4.4, prefix hit detection) in one call: the same results, status word and
   index updates as cascade_tier_reclaim on tiers 0, 1 and 2 in turn, each
   tier's outgoing blocks passed as the next tier's incoming ones.  Neither
   the counting pass nor the histogram pass of a table depends on the tier
   above, so the call runs each of them once for all three tables, and the
   deeper tiers' full-table reads overlap the shallower tiers' work (11
   launches instead of 15).  The demotions it passes between tiers are its
   own, so it does not check their hashes.

   chain      per tier t: table[t], need[t], freed[t] (device int32[need[t]]);
              outgoing[t], n_outgoing_dev[t], max_outgoing[t] for t = 0, 1
              (max_outgoing[0] >= need[0], max_outgoing[1] >= need[1] +
              max_outgoing[0]); placed[t] for t = 1, 2 (device
              int32[max_outgoing[t - 1]]), placed[0] unused.  The arguments
              of each tier follow cascade_tier_reclaim.
   index      the prefix index (NULL = none) and its capacity.
   workspace  device memory of cascade_tier_chain_workspace_bytes(n) bytes
              (n = the three tables' slot counts: the three tiers' workspaces,
              their fixed-size parts first), 256-byte aligned, zero-filled
              once before its first use; every call leaves it ready for the
              next.  A workspace sized for n serves every chain whose tables
              hold at most n[t] slots.  One call at a time per workspace.
   status_dev as for cascade_tier_reclaim, one word for the chain.
   Returns CASCADE_EINVAL for bad host arguments (of any tier), CASCADE_EHIP
   on a failed launch.  Asynchronous on `stream`. */
typedef struct {
  cascade_tier_table_t table[3];
  int32_t need[3];
  cascade_demotion_t *outgoing[2];
  int32_t *n_outgoing_dev[2];
  int32_t max_outgoing[2];
  int32_t *freed[3];
  int32_t *placed[3];
} cascade_tier_chain_t;

size_t cascade_tier_chain_workspace_bytes(const int32_t *n_slots);
int cascade_tier_reclaim_chain(const cascade_tier_chain_t *chain, void *index,
                               int32_t index_capacity, void *workspace, size_t workspace_bytes,
                               int32_t *status_dev, void *stream);

/* Short English text for a return code or status value. */
const char *cascade_strerror(int code);

#ifdef __cplusplus
}
#endif
#endif
