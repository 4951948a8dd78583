/*
 * cascade_ref.h -- CPU oracle of Cascade's per-iteration scheduling step.
 *
 * TEST INFRASTRUCTURE ONLY.  This oracle exists to check the GPU library
 * bit for bit.  Only the tests, the smoke check and the benchmark's CPU
 * baseline may load it; the product path never does.  It shares no code,
 * header, table or helper with the GPU library: every type below is
 * declared here again on purpose.
 *
 * Paper: "Cascade" (arXiv 2608.06557).  What each part follows:
 *   - Section 4.2: TTFT estimator regimes, eq:est_latency, eq:budget_eq,
 *     the Tier-1 / Tier-2 split.
 *   - Section 4.3: eq:rem_budget_eq, eq:restore_time, eq:max_restorable,
 *     budget-aware preemption, Algorithm 1 (Phase 2 loop).
 *   - Section 4.4: chunked prefill co-scheduled with decodes, HBM allocated
 *     only at the final DRAM->HBM hop, preemption of the resident
 *     prefill-stage request with the largest remaining budget.
 * All arithmetic is 64-bit integer (the gamma product uses a 128-bit
 * intermediate), so the GPU must agree exactly.
 */
#ifndef CASCADE_REF_H
#define CASCADE_REF_H
#include <stdint.h>

#define CREF_OK 0
#define CREF_EINVAL (-1)
#define CREF_ENOSPC (-2)

/* request state */
#define CREF_QUEUED 0
#define CREF_RUNNING_PREFILL 1
#define CREF_DECODE 2
/* queue tier */
#define CREF_QT_NEW 0
#define CREF_QT_TIER1 1
#define CREF_QT_TIER2 2
/* KV residency tier of the matched prefix (Section 4.1: tiers 0,1,2) */
#define CREF_KV_HBM 0
#define CREF_KV_DRAM 1
#define CREF_KV_NVME 2
#define CREF_KV_NONE 3
/* memory actions */
#define CREF_ACT_RETAIN 1
#define CREF_ACT_RESTORE 2
#define CREF_ACT_PREFETCH 3
#define CREF_ACT_RECOMPUTE 4
#define CREF_ACT_PREEMPT_OFFLOAD 5
#define CREF_ACT_PREEMPT_DROP 6
#define CREF_ACT_SHARE 7          /* references a prefix another request restores */

typedef struct {
  int64_t t_now_ns;
  int32_t num_classes;
  int64_t slo_ns[16];           /* TTFT target per class */
  int32_t block_tokens;         /* tokens per KV block */
  int32_t chunk_tokens;         /* chunked-prefill chunk of the estimator */
  int32_t load_decodes;         /* d: active decodes (actual load) */
  int32_t max_batch;            /* B_max; maximum load is B_max - 1 decodes */
  int32_t gamma_q16;            /* guardband gamma * 65536 */
  int64_t c_iter_ps, c_decode_ps, c_token_ps, c_attn_ps;
  int64_t link_delta_ns[2];     /* [0] DRAM->HBM, [1] NVMe->DRAM */
  int64_t link_blk_ns[2];       /* ns to move one KV block over the link */
  int32_t token_cap;            /* prefill+decode tokens per iteration */
  int32_t tier2_reserve_q16;    /* Tier-2 reserved fraction * 65536 */
  int32_t max_move_blocks;      /* U: restore/prefetch blocks per step */
  int32_t num_blocks;           /* HBM pool blocks */
} cref_params;

typedef struct { int32_t req, blk, pool_slot, staging_slot; } cref_move;

typedef struct {
  int64_t *budget_ns;           /* [n] remaining budget B_rem */
  uint8_t *action;              /* [n] */
  uint8_t *queue_tier_out;      /* [n] */
  int32_t *tokens_granted;      /* [n] */
  int32_t *restore_blocks;      /* [n] */
  int32_t *order;               /* [n] request index at each priority position */
  int32_t *alloc_begin;         /* [n] index into slot_list, -1 if not admitted */
  int32_t *alloc_count;         /* [n] new HBM blocks, 0 if not admitted */
  int32_t *admitted;            /* [n] admitted request indices in priority order */
  int32_t n_admitted;
  int32_t *slot_list; int32_t slot_list_capacity; int32_t n_slot_list;
  cref_move *unpack_moves; int32_t unpack_capacity; int32_t n_unpack;
  cref_move *pack_moves;   int32_t pack_capacity;   int32_t n_pack;
  /* Copy-order hazards (written only when the step returns CREF_OK; either
     pointer may be NULL): unpack_hazard[m] = the pack move reading the pool
     slot that unpack move m writes, pack_hazard[j] = the unpack move writing
     the slot that pack move j reads, -1 where there is none. */
  int32_t *unpack_hazard;
  int32_t *pack_hazard;
  /* Shared-prefix restores (only with a prefix_group input; may be NULL):
     for a request that shares another request's restore (action SHARE),
     that request's index, else -1. */
  int32_t *share_leader;
} cref_outputs;

/* Intermediate values of the per-request evaluation, exposed for pinning. */
typedef struct {
  int64_t l_actual_ns, l_max_ns, l_ns, budget0_ns, budget_rem_ns;
  int32_t tier_out, group, want_blocks;
  uint64_t key;
} cref_eval_out;

/* Latency of computing n prompt tokens that start at position s while dd
   decodes share each iteration, in picoseconds. */
int64_t cref_compute_ps(const cref_params *p, int64_t n, int64_t s, int64_t dd);
/* eq:restore_time in blocks: time to restore x blocks from tier k (1 or 2). */
int64_t cref_restore_time_ns(const cref_params *p, int32_t tier, int64_t x);
/* 0 if the parameters are in the domain, else CREF_EINVAL. */
int32_t cref_check_params(const cref_params *p, int32_t n, int32_t n_free);
/* Evaluation of one request (no validation). */
void cref_eval(const cref_params *p, uint8_t slo_class, uint8_t state, uint8_t queue_tier,
               uint8_t prefix_tier, int64_t arrival_ns, int32_t n_in, int32_t n_out_pred,
               int32_t n_prefix, int32_t n_progress, cref_eval_out *o);

/* One step.  prefix_group (NULL = none) turns on shared-prefix restores
   within the step (Section 4.4 prefix hit detection; the paper leaves
   within-step sharing open, the reading is this oracle's): requests with
   the same group id g >= 0 share the leading blocks of their matched
   prefixes.  It matters for queued requests whose prefix is in DRAM or NVMe
   ("deep members").  Within each priority group (Tier-1 with decodes,
   Tier-2) the first deep member in priority order with a positive restore
   want is the group's leader: it restores under the link cap as any
   request does.  Every later deep member of the same group and tier is a
   follower: it takes nothing from the link cap and references the first
   min(leader's restore blocks, its own prefix blocks) blocks of the
   leader's restore, like an HBM prefix (need and new blocks shrink
   accordingly); action SHARE, restore_blocks = those blocks, share_leader
   = the leader (RECOMPUTE and -1 when that is 0 blocks).  Group ids must
   lie in [-1, n). */
int32_t cref_step(int32_t n, const uint64_t *id, const uint8_t *slo_class, const uint8_t *state,
                  const uint8_t *queue_tier, const uint8_t *prefix_tier,
                  const int64_t *arrival_ns, const int32_t *n_in, const int32_t *n_out_pred,
                  const int32_t *n_prefix, const int32_t *n_progress,
                  const int32_t *row_offsets, const int32_t *slots,
                  int32_t n_free, const int32_t *free_slots, const int32_t *prefix_group,
                  const cref_params *p, cref_outputs *out);

/* Paged-KV block copies, one chunk_bytes memcpy per (move, layer, K/V). */
typedef struct {
  uint8_t *base; int32_t num_layers;
  int64_t chunk_bytes, layer_stride, kv_stride, slot_stride;
} cref_pool;
/* Prefix hit detection (Section 4.4): an index records, for each cached KV
   block (by its prefix hash), the deepest tier holding it; a request's
   matched prefix is its longest run of leading blocks all in the index,
   capped at floor((n_in - 1) / block_tokens) blocks so that at least one
   prompt token is computed; its tier is the deepest over those blocks
   (CREF_KV_NONE when nothing matches).  index_hashes/index_tiers list
   n_entries cached (block, tier) facts, duplicates allowed.  Request i's
   block hashes are block_hashes[block_offsets[i] .. block_offsets[i+1]).
   Returns CREF_EINVAL for a negative count, a tier outside HBM..NVMe, hash
   0 (reserved for empty index slots), or offsets that are not monotone. */
int32_t cref_prefix_probe(int32_t n_entries, const uint64_t *index_hashes,
                          const uint8_t *index_tiers, int32_t n, const int32_t *block_offsets,
                          const uint64_t *block_hashes, const int32_t *n_in,
                          int32_t block_tokens, int32_t *n_prefix_out,
                          uint8_t *prefix_tier_out);

/* Per-tier LRU reclamation (Section 4.4, prefix hit detection: free blocks
   are reclaimed least-recently-used within each tier, hot prefixes stay in
   the fast tiers and cold ones spill one tier deeper).  One call reclaims
   need + n_incoming slots of one tier (0 HBM, 1 DRAM, 2 NVMe):
     - candidates are the slots with held[s] == 0; empty slots (hash 0)
       come first, then cached blocks by ascending last use, ties by the
       lower slot;
     - the reclaimed set, listed by ascending slot, gives the caller its
       first `need` slots (freed) and places incoming[j] (blocks demoted
       from the tier above) into the rest (placed[j]);
     - a reclaimed cached block of tier 0 or 1 that no deeper tier holds
       (index mask bits above `tier` clear, judged on the index as it was
       when the call began; a hash missing from the index counts as held
       nowhere deeper) is demoted: appended to outgoing in slot order;
       tier 2 drops its reclaimed blocks;
     - the index (n_index entries, keys ascending and nonzero, mask bit k =
       tier k holds the block) loses bit `tier` for every reclaimed cached
       block and gains bit tier+1 for every demoted one; hashes missing
       from it are skipped;
     - freed slots become empty (hash 0, last use 0); placed slots take
       their incoming block's hash and last use.
   Returns CREF_EINVAL for a tier outside 0..2, negative counts, a negative
   last use, an incoming hash 0, index keys not strictly ascending or a
   mask above 7, or max_outgoing < need + n_incoming on tiers 0 and 1;
   CREF_ENOSPC when fewer than need + n_incoming slots are free.  Nothing is
   written on error. */
typedef struct { uint64_t hash; int64_t last_use_ns; int32_t src_slot, pad; } cref_demotion;

int32_t cref_tier_reclaim(int32_t tier, int32_t n_slots, uint64_t *block_hash,
                          int64_t *last_use_ns, const uint8_t *held, int32_t need,
                          int32_t n_incoming, const cref_demotion *incoming,
                          int32_t max_outgoing, cref_demotion *outgoing, int32_t *n_outgoing,
                          int32_t *freed, int32_t *placed, int32_t n_index,
                          const uint64_t *index_keys, uint8_t *index_masks);

void cref_pack(const cref_pool *pool, uint8_t *staging, const cref_move *moves, int32_t n);
void cref_unpack(const cref_pool *pool, const uint8_t *staging, const cref_move *moves, int32_t n);

#endif
