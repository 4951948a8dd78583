/*
 * cascade_ref.c -- CPU oracle of Cascade's per-iteration scheduling step.
 *
 * TEST INFRASTRUCTURE ONLY (see cascade_ref.h).  Plain, slow, single
 * threaded C.  The step is written as the paper states it: per-request
 * estimation and budgets (Section 4.2), then Algorithm 1's Phase 2 as a
 * sequential loop over the least-remaining-budget-first order, then
 * budget-aware preemption (Sections 4.3 and 4.4).  The GPU library
 * computes the same result with parallel scans; the two share nothing.
 *
 * Readings taken where the paper is silent (each is restated where used):
 *  R1  The estimator's functional form is not given.  Per-iteration cost
 *      is base + per-decode + per-token + pairwise attention, iterations of
 *      chunk_tokens tokens (Section 4.2 regimes; chunk 512 in Section 5).
 *  R2  Predicted output length is used only for the remaining decode time
 *      of DECODE-stage requests.
 *  R3  L^actual is tier-aware: it includes the restore time of the prefix.
 *  R5  Picosecond coefficients, each regime floored to ns before restore
 *      time is added; the gamma product is exact, then floored.
 *  R6  Tier-1 iff B_r > 0 (strict), Tier-1 is sticky, Tier-2 is promoted
 *      once the re-estimated B_r > 0 (Section 4, overview).
 *  R8  Decodes first, then Tier-1, then Tier-2, each least-remaining-
 *      budget-first; ties by input position.
 *  R9  Tier-2 gets a reserved fraction rho of the token cap when it is
 *      non-empty; rho = 0 is Algorithm 1's "Q2 only when Q1 is empty".
 *  R11 Admission is the longest feasible prefix of the order: the first
 *      block-capacity failure stops it.
 *  R12 Victims are non-admitted prefill-stage holders taken from the back
 *      of the order until the block deficit is covered.
 *  R13 A victim spills to DRAM iff T_DRAM(held) <= B_rem, else it is
 *      dropped and recomputed later.
 *  R14 Restore x = min(prefix blocks, M) then keep it only if strictly
 *      cheaper than recomputing those tokens.
 *  R15 A request that is not admitted but has restore blocks PREFETCHes
 *      (no HBM this step: HBM is allocated only at the final hop).
 *  R16 The link-bandwidth constraint of eq:opt_goal_compact is a per-step
 *      cap U on restore+prefetch blocks, taken in priority order.
 *  R36 Shared prefixes (optional prefix_group input): within a priority
 *      group, the first deep member of a prefix group with a positive want
 *      restores; later members of the same group and tier reference its
 *      restored blocks (as many as their own prefix has) instead of
 *      restoring again.  See cascade_ref.h.
 */
#include "cascade_ref.h"

#include <stdlib.h>
#include <string.h>

/* ---------------------------------------------------------------- helpers */

static int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
static int64_t min64(int64_t a, int64_t b) { return a < b ? a : b; }
static int64_t ns_of_ps(int64_t ps) { return ps / 1000; }

/* Iteration cost model (reading R1).  n new prompt tokens at positions
   s .. s+n-1 are computed in ceil(n / chunk) iterations; each iteration pays
   a base cost plus one unit per co-scheduled decode; each token pays c_token
   and attends to every position up to its own: sum_{t=s}^{s+n-1} (t+1)
   pairs, which is n*(2s+n+1)/2. */
int64_t cref_compute_ps(const cref_params *p, int64_t n, int64_t s, int64_t dd) {
  if (n == 0) return 0;
  int64_t iters = ceil_div(n, p->chunk_tokens);
  int64_t pairs = n * (2 * s + n + 1) / 2;
  return iters * (p->c_iter_ps + dd * p->c_decode_ps) + n * p->c_token_ps + p->c_attn_ps * pairs;
}

/* eq:restore_time.  P(1) = {DRAM->HBM}; P(2) = {NVMe->DRAM, DRAM->HBM}.
   The fixed overheads of the links on the path add up, and so do their
   per-block transfer times. */
static int64_t path_delta_ns(const cref_params *p, int32_t tier) {
  int64_t d = p->link_delta_ns[0];
  if (tier == CREF_KV_NVME) d += p->link_delta_ns[1];
  return d;
}
static int64_t path_blk_ns(const cref_params *p, int32_t tier) {
  int64_t b = p->link_blk_ns[0];
  if (tier == CREF_KV_NVME) b += p->link_blk_ns[1];
  return b;
}
int64_t cref_restore_time_ns(const cref_params *p, int32_t tier, int64_t x) {
  if (x == 0) return 0;
  return path_delta_ns(p, tier) + x * path_blk_ns(p, tier);
}

/* ----------------------------------------------------- per-request stage */

void cref_eval(const cref_params *p, uint8_t cls, uint8_t state, uint8_t queue_tier,
               uint8_t ptier, int64_t arrival_ns, int32_t n_in, int32_t n_out_pred,
               int32_t n_prefix, int32_t n_progress, cref_eval_out *o) {
  const int64_t bt = p->block_tokens;
  const int64_t d = p->load_decodes;          /* actual load */
  const int64_t dmax = p->max_batch - 1;      /* maximum load: B_max - 1 decodes */
  int64_t l_act = 0, l_max = 0;
  int64_t pb = 0;

  /* Section 4.2, regimes (3) L^actual and (4) L^max. */
  if (state == CREF_QUEUED) {
    int64_t reuse = 0, restore = 0;
    if (ptier != CREF_KV_NONE) {
      pb = n_prefix / bt;
      reuse = n_prefix;
      if (ptier == CREF_KV_DRAM || ptier == CREF_KV_NVME)
        restore = cref_restore_time_ns(p, ptier, pb);   /* reading R3 */
    }
    l_act = ns_of_ps(cref_compute_ps(p, n_in - reuse, reuse, d)) + restore;
    l_max = ns_of_ps(cref_compute_ps(p, n_in - reuse, reuse, dmax)) + restore;
  } else if (state == CREF_RUNNING_PREFILL) {
    int64_t left = n_in - n_progress;
    l_act = ns_of_ps(cref_compute_ps(p, left, n_progress, d));
    l_max = ns_of_ps(cref_compute_ps(p, left, n_progress, dmax));
  } else { /* DECODE: remaining output tokens, one per iteration (reading R2) */
    int64_t left = (int64_t)n_out_pred - n_progress;
    if (left < 0) left = 0;
    l_act = ns_of_ps(left * (p->c_iter_ps + d * p->c_decode_ps));
    l_max = ns_of_ps(left * (p->c_iter_ps + dmax * p->c_decode_ps));
  }

  /* eq:est_latency: L = gamma/2 * (L^actual + L^max), floored. */
  __int128 prod = (__int128)(l_act + l_max) * p->gamma_q16;
  int64_t l = (int64_t)(prod / ((__int128)1 << 17));
  /* eq:budget_eq and eq:rem_budget_eq. */
  int64_t b0 = p->slo_ns[cls] - l;
  int64_t brem = b0 - (p->t_now_ns - arrival_ns);

  /* Dual-tier queues (reading R6). */
  int32_t tier_out = queue_tier;
  if (state != CREF_DECODE) {
    if (queue_tier == CREF_QT_TIER1) tier_out = CREF_QT_TIER1;
    else tier_out = (b0 > 0) ? CREF_QT_TIER1 : CREF_QT_TIER2;
  }

  /* eq:max_restorable in blocks (reading R14): the largest x with
     T_k(x) <= B_rem, capped at the prefix; kept only if the restore is
     strictly cheaper than recomputing the same tokens. */
  int32_t want = 0;
  if (state == CREF_QUEUED && (ptier == CREF_KV_DRAM || ptier == CREF_KV_NVME)) {
    int64_t delta = path_delta_ns(p, ptier), blk = path_blk_ns(p, ptier);
    int64_t x = 0;
    if (brem > delta) x = min64(pb, (brem - delta) / blk);
    if (x > 0) {
      int64_t recompute_all = ns_of_ps(cref_compute_ps(p, n_in, 0, d));
      int64_t with_restore = ns_of_ps(cref_compute_ps(p, n_in - bt * x, bt * x, d));
      if (cref_restore_time_ns(p, ptier, x) >= recompute_all - with_restore) x = 0;
    }
    want = (int32_t)x;
  }

  /* Priority key (reading R8): group, then B_rem clamped to 62 bits. */
  int32_t group = (state == CREF_DECODE) ? 0 : (tier_out == CREF_QT_TIER1 ? 1 : 2);
  int64_t lo = -((int64_t)1 << 61), hi = ((int64_t)1 << 61) - 1;
  int64_t c = brem < lo ? lo : (brem > hi ? hi : brem);
  uint64_t key = ((uint64_t)group << 62) | (uint64_t)(c + ((int64_t)1 << 61));

  o->l_actual_ns = l_act; o->l_max_ns = l_max; o->l_ns = l; o->budget0_ns = b0;
  o->budget_rem_ns = brem; o->tier_out = tier_out; o->group = group; o->want_blocks = want;
  o->key = key;
}

/* --------------------------------------------------------- validation */

int32_t cref_check_params(const cref_params *p, int32_t n, int32_t n_free) {
  const int64_t P = 1;
  if (n < 0 || n > (1 << 20)) return CREF_EINVAL;
  if (p->t_now_ns < 0 || p->t_now_ns >= (P << 62)) return CREF_EINVAL;
  if (p->num_classes < 1 || p->num_classes > 16) return CREF_EINVAL;
  for (int c = 0; c < p->num_classes; c++)
    if (p->slo_ns[c] < 0 || p->slo_ns[c] > (P << 50)) return CREF_EINVAL;
  if (p->block_tokens < 1 || p->block_tokens > (1 << 16)) return CREF_EINVAL;
  if (p->chunk_tokens < 16 || p->chunk_tokens > (1 << 20)) return CREF_EINVAL;
  if (p->max_batch < 1 || p->max_batch > 4096) return CREF_EINVAL;
  if (p->load_decodes < 0 || p->load_decodes > p->max_batch - 1) return CREF_EINVAL;
  if (p->gamma_q16 < 65536 || p->gamma_q16 > (1 << 20)) return CREF_EINVAL;
  if (p->c_iter_ps < 0 || p->c_decode_ps < 0 || p->c_token_ps < 0 || p->c_attn_ps < 0)
    return CREF_EINVAL;
  if (p->c_iter_ps > (P << 36) || p->c_decode_ps > (P << 36)) return CREF_EINVAL;
  if (p->c_iter_ps + (int64_t)p->max_batch * p->c_decode_ps > (P << 36)) return CREF_EINVAL;
  if (p->c_token_ps > (P << 28) || p->c_attn_ps > (P << 16)) return CREF_EINVAL;
  for (int l = 0; l < 2; l++) {
    if (p->link_delta_ns[l] < 0 || p->link_delta_ns[l] > (P << 40)) return CREF_EINVAL;
    if (p->link_blk_ns[l] < 1 || p->link_blk_ns[l] > (P << 32)) return CREF_EINVAL;
  }
  if (p->token_cap < 1 || p->token_cap > (1 << 24)) return CREF_EINVAL;
  if (p->tier2_reserve_q16 < 0 || p->tier2_reserve_q16 > 65536) return CREF_EINVAL;
  if (p->max_move_blocks < 0) return CREF_EINVAL;
  if (p->num_blocks < 0) return CREF_EINVAL;
  if (n_free < 0 || n_free > p->num_blocks) return CREF_EINVAL;
  return CREF_OK;
}

static int32_t row_len_rule(const cref_params *p, uint8_t state, int32_t n_in, int32_t prog) {
  if (state == CREF_QUEUED) return 0;
  if (state == CREF_RUNNING_PREFILL) return (int32_t)ceil_div(prog, p->block_tokens);
  return (int32_t)ceil_div((int64_t)n_in + prog, p->block_tokens);
}

static int32_t check_request(const cref_params *p, int32_t i, const uint64_t *id,
                             const uint8_t *cls, const uint8_t *st, const uint8_t *qt,
                             const uint8_t *pt, const int64_t *arr, const int32_t *nin,
                             const int32_t *nout, const int32_t *npre, const int32_t *nprog,
                             const int32_t *ro) {
  if (i > 0 && id[i] <= id[i - 1]) return CREF_EINVAL;
  if (i == 0 && ro[0] != 0) return CREF_EINVAL;
  if (cls[i] >= p->num_classes || st[i] > 2 || qt[i] > 2 || pt[i] > 3) return CREF_EINVAL;
  if (nin[i] < 1 || nin[i] > (1 << 17)) return CREF_EINVAL;
  if (nout[i] < 0 || nout[i] > (1 << 17)) return CREF_EINVAL;
  if (npre[i] < 0 || npre[i] > nin[i] - 1 || npre[i] % p->block_tokens != 0) return CREF_EINVAL;
  if (arr[i] < 0 || arr[i] > p->t_now_ns) return CREF_EINVAL;
  if (st[i] == CREF_QUEUED) {
    if ((npre[i] == 0) != (pt[i] == CREF_KV_NONE)) return CREF_EINVAL;
    if (nprog[i] != 0) return CREF_EINVAL;
  } else if (st[i] == CREF_RUNNING_PREFILL) {
    if (nprog[i] < 1 || nprog[i] > nin[i] - 1) return CREF_EINVAL;
  } else {
    if (nprog[i] < 0 || nprog[i] > (1 << 17)) return CREF_EINVAL;
  }
  if ((int64_t)ro[i + 1] - ro[i] != row_len_rule(p, st[i], nin[i], nprog[i])) return CREF_EINVAL;
  return CREF_OK;
}

/* ------------------------------------------------------------ the step */

typedef struct { uint64_t key; int32_t idx; } keyed;

static int cmp_keyed(const void *a, const void *b) {
  const keyed *x = (const keyed *)a, *y = (const keyed *)b;
  if (x->key != y->key) return x->key < y->key ? -1 : 1;
  return x->idx < y->idx ? -1 : (x->idx > y->idx ? 1 : 0);
}

int32_t cref_step(int32_t n, const uint64_t *id, const uint8_t *cls, const uint8_t *st,
                  const uint8_t *qt, const uint8_t *pt, const int64_t *arr,
                  const int32_t *nin, const int32_t *nout, const int32_t *npre,
                  const int32_t *nprog, const int32_t *ro, const int32_t *slots,
                  int32_t n_free, const int32_t *free_slots, const int32_t *pg,
                  const cref_params *p, cref_outputs *out) {
  if (cref_check_params(p, n, n_free) != CREF_OK) return CREF_EINVAL;
  if (pg)
    for (int32_t i = 0; i < n; i++)
      if (pg[i] < -1 || pg[i] >= n) return CREF_EINVAL;
  if (out->slot_list_capacity < 0 || out->unpack_capacity < 0 || out->pack_capacity < 0)
    return CREF_EINVAL;
  for (int32_t i = 0; i < n; i++)
    if (check_request(p, i, id, cls, st, qt, pt, arr, nin, nout, npre, nprog, ro) != CREF_OK)
      return CREF_EINVAL;
  int64_t nnz = n > 0 ? ro[n] : 0;
  for (int64_t j = 0; j < nnz; j++)
    if (slots[j] < 0 || slots[j] >= p->num_blocks) return CREF_EINVAL;
  for (int32_t j = 0; j < n_free; j++)
    if (free_slots[j] < 0 || free_slots[j] >= p->num_blocks) return CREF_EINVAL;

  const int64_t bt = p->block_tokens;
  cref_eval_out *ev = (cref_eval_out *)calloc(n ? n : 1, sizeof(cref_eval_out));
  keyed *pq = (keyed *)calloc(n ? n : 1, sizeof(keyed));
  int32_t *r = (int32_t *)calloc(n ? n : 1, sizeof(int32_t));
  int64_t *g = (int64_t *)calloc(n ? n : 1, sizeof(int64_t));
  int64_t *nb = (int64_t *)calloc(n ? n : 1, sizeof(int64_t));
  uint8_t *adm = (uint8_t *)calloc(n ? n : 1, 1);
  uint8_t *victim = (uint8_t *)calloc(n ? n : 1, 1);
  /* shared prefixes (R36): the leader of each (prefix group, priority
     group), and for every follower its leader and shared blocks */
  int32_t *leader_of = (int32_t *)malloc(sizeof(int32_t) * 2 * (size_t)(n ? n : 1));
  int32_t *follows = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n ? n : 1));
  int32_t *shared = (int32_t *)calloc(n ? n : 1, sizeof(int32_t));
  for (int32_t k = 0; k < 2 * n; k++) leader_of[k] = -1;
  for (int32_t i = 0; i < n; i++) follows[i] = -1;

  /* Phase 1 and the budget update (eq:est_latency .. eq:rem_budget_eq). */
  for (int32_t i = 0; i < n; i++) {
    cref_eval(p, cls[i], st[i], qt[i], pt[i], arr[i], nin[i], nout[i], npre[i], nprog[i], &ev[i]);
    out->budget_ns[i] = ev[i].budget_rem_ns;
    out->queue_tier_out[i] = (uint8_t)ev[i].tier_out;
  }

  /* Least-remaining-budget-first: sort by key, ties by input position. */
  for (int32_t i = 0; i < n; i++) { pq[i].key = ev[i].key; pq[i].idx = i; }
  qsort(pq, (size_t)n, sizeof(keyed), cmp_keyed);
  int32_t e1 = 0, has_tier2 = 0;
  for (int32_t q = 0; q < n; q++) {
    out->order[q] = pq[q].idx;
    if (ev[pq[q].idx].group <= 1) e1++; else has_tier2 = 1;
  }

  /* Algorithm 1, Phase 2, walked in priority order. */
  /* (a) Restore / prefetch volume, capped per step at U blocks (R16).  A
         follower of a shared prefix restores nothing itself (R36). */
  int64_t move_left = p->max_move_blocks;
  for (int32_t q = 0; q < n; q++) {
    int32_t i = pq[q].idx;
    int deep = pg && pg[i] >= 0 && st[i] == CREF_QUEUED &&
               (pt[i] == CREF_KV_DRAM || pt[i] == CREF_KV_NVME);
    int32_t slot = deep ? 2 * pg[i] + (ev[i].group == 2 ? 1 : 0) : -1;
    if (deep && leader_of[slot] >= 0) {
      int32_t lead = leader_of[slot];
      int32_t pb = npre[i] / p->block_tokens;
      follows[i] = lead;
      shared[i] = r[lead] < pb ? r[lead] : pb;
      r[i] = 0;
      continue;
    }
    int64_t take = min64(ev[i].want_blocks, move_left);
    r[i] = (int32_t)take;
    move_left -= take;
    if (deep && ev[i].want_blocks > 0) leader_of[slot] = i;
  }
  /* (b) Chunked-prefill token grants under the cap, with the Tier-2
         reserve (R9).  need = tokens still to compute this step. */
  int64_t reserve2 = has_tier2 ? ((int64_t)p->token_cap * p->tier2_reserve_q16) >> 16 : 0;
  int64_t left = p->token_cap - reserve2;
  int64_t used_first = 0;
  for (int32_t q = 0; q < n; q++) {
    int32_t i = pq[q].idx;
    if (q == e1) left = p->token_cap - used_first;  /* Tier-2 gets what remains */
    int64_t need;
    if (st[i] == CREF_DECODE) need = 1;
    else if (st[i] == CREF_RUNNING_PREFILL) need = nin[i] - nprog[i];
    else if (pt[i] == CREF_KV_HBM) need = nin[i] - npre[i];
    else if (follows[i] >= 0) need = nin[i] - bt * shared[i];
    else need = nin[i] - bt * r[i];
    int64_t gi = min64(need, left);
    g[i] = gi;
    left -= gi;
    if (q < e1) used_first += gi;
  }
  /* (c) New HBM blocks and admission.  Blocks held by prefill-stage
         requests count as available: admitting a holder keeps them, and a
         holder left out can be preempted (R11, R12). */
  int64_t held_total = 0;
  for (int32_t i = 0; i < n; i++)
    if (st[i] == CREF_RUNNING_PREFILL) held_total += ro[i + 1] - ro[i];
  int64_t avail = (int64_t)n_free + held_total;
  int stopped = 0;
  int64_t new_blocks = 0;
  for (int32_t q = 0; q < n; q++) {
    int32_t i = pq[q].idx;
    if (g[i] <= 0) continue;
    int64_t held = ro[i + 1] - ro[i];
    if (st[i] == CREF_QUEUED && follows[i] >= 0) {
      /* the shared blocks are referenced, not allocated */
      nb[i] = ceil_div(bt * shared[i] + g[i], bt) - shared[i];
    } else if (st[i] == CREF_QUEUED) {
      int64_t reuse = (pt[i] == CREF_KV_HBM) ? npre[i] : bt * r[i];
      nb[i] = ceil_div(reuse + g[i], bt) - (pt[i] == CREF_KV_HBM ? npre[i] / bt : 0);
    } else if (st[i] == CREF_RUNNING_PREFILL) {
      nb[i] = ceil_div(nprog[i] + g[i], bt) - held;
    } else {
      nb[i] = ceil_div((int64_t)nin[i] + nprog[i] + 1, bt) - held;
    }
    if (stopped) continue;
    int64_t cost = nb[i] + (st[i] == CREF_RUNNING_PREFILL ? held : 0);
    if (cost > avail) { stopped = 1; continue; }
    avail -= cost;
    adm[i] = 1;
    new_blocks += nb[i];
  }
  /* (d) Budget-aware preemption: cover the block deficit with the
         non-admitted prefill-stage holders of largest remaining budget,
         i.e. from the back of the order; never a decode. */
  int64_t deficit = new_blocks - n_free;
  int64_t freed = 0;
  for (int32_t q = n - 1; q >= 0 && deficit > 0; q--) {
    int32_t i = pq[q].idx;
    int64_t held = ro[i + 1] - ro[i];
    if (st[i] != CREF_RUNNING_PREFILL || adm[i] || held <= 0) continue;
    if (freed >= deficit) break;
    victim[i] = 1;
    freed += held;
  }

  /* Per-request outputs. */
  for (int32_t i = 0; i < n; i++) {
    int32_t a;
    if (victim[i]) {
      int64_t held = ro[i + 1] - ro[i];
      a = cref_restore_time_ns(p, CREF_KV_DRAM, held) <= ev[i].budget_rem_ns
              ? CREF_ACT_PREEMPT_OFFLOAD : CREF_ACT_PREEMPT_DROP;     /* R13 */
    } else if (st[i] != CREF_QUEUED || pt[i] == CREF_KV_HBM) {
      a = CREF_ACT_RETAIN;
    } else if (follows[i] >= 0) {
      a = shared[i] > 0 ? CREF_ACT_SHARE : CREF_ACT_RECOMPUTE;   /* R36 */
    } else if (pt[i] == CREF_KV_NONE || r[i] == 0) {
      a = CREF_ACT_RECOMPUTE;
    } else {
      a = adm[i] ? CREF_ACT_RESTORE : CREF_ACT_PREFETCH;              /* R15 */
    }
    out->action[i] = (uint8_t)a;
    out->restore_blocks[i] = follows[i] >= 0 ? shared[i] : r[i];
    if (out->share_leader)
      out->share_leader[i] = (follows[i] >= 0 && shared[i] > 0) ? follows[i] : -1;
    out->tokens_granted[i] = adm[i] ? (int32_t)g[i] : 0;
    out->alloc_begin[i] = -1;
    out->alloc_count[i] = 0;
  }

  /* Slot list: the free list, then the victims' rows (back of the order
     first, each row in its own order).  Admitted requests take their new
     blocks from it in priority order. */
  int32_t status = CREF_OK;
  int64_t sl = 0;
  for (int32_t j = 0; j < n_free; j++, sl++)
    if (sl < out->slot_list_capacity) out->slot_list[sl] = free_slots[j];
  for (int32_t q = n - 1; q >= 0; q--) {
    int32_t i = pq[q].idx;
    if (!victim[i]) continue;
    for (int32_t b = ro[i]; b < ro[i + 1]; b++, sl++)
      if (sl < out->slot_list_capacity) out->slot_list[sl] = slots[b];
  }
  out->n_slot_list = (int32_t)sl;
  if (sl > out->slot_list_capacity) status = CREF_ENOSPC;

  int64_t next = 0, na = 0, nu = 0;
  for (int32_t q = 0; q < n; q++) {
    int32_t i = pq[q].idx;
    if (!adm[i]) continue;
    out->admitted[na++] = i;
    out->alloc_begin[i] = (int32_t)next;
    out->alloc_count[i] = (int32_t)nb[i];
    if (out->action[i] == CREF_ACT_RESTORE) {
      /* The first r blocks of the allocation receive the restored prefix. */
      for (int32_t b = 0; b < r[i]; b++, nu++) {
        if (nu >= out->unpack_capacity) continue;
        int64_t s = next + b;
        cref_move m = {i, b, s < out->slot_list_capacity ? out->slot_list[s] : -1, (int32_t)nu};
        out->unpack_moves[nu] = m;
      }
    }
    next += nb[i];
  }
  out->n_admitted = (int32_t)na;
  out->n_unpack = (int32_t)nu;
  if (nu > out->unpack_capacity) status = CREF_ENOSPC;

  int64_t npk = 0;
  for (int32_t q = n - 1; q >= 0; q--) {
    int32_t i = pq[q].idx;
    if (!victim[i] || out->action[i] != CREF_ACT_PREEMPT_OFFLOAD) continue;
    for (int32_t b = 0; b < ro[i + 1] - ro[i]; b++, npk++) {
      if (npk >= out->pack_capacity) continue;
      cref_move m = {i, b, slots[ro[i] + b], (int32_t)npk};
      out->pack_moves[npk] = m;
    }
  }
  out->n_pack = (int32_t)npk;
  if (npk > out->pack_capacity) status = CREF_ENOSPC;

  /* Copy-order hazards: a preempted request's slot that a restore receives
     is read by the spill and written by the restore (Section 4.4), so the
     spill of that slot must come first.  Found by pool slot, with a table
     over the whole pool. */
  if (status == CREF_OK && (out->unpack_hazard || out->pack_hazard)) {
    int32_t *by_slot = (int32_t *)malloc(sizeof(int32_t) * (size_t)(p->num_blocks > 0 ? p->num_blocks : 1));
    for (int32_t s = 0; s < p->num_blocks; s++) by_slot[s] = -1;
    for (int32_t j = 0; j < npk; j++) by_slot[out->pack_moves[j].pool_slot] = j;
    if (out->unpack_hazard)
      for (int32_t m = 0; m < nu; m++) out->unpack_hazard[m] = by_slot[out->unpack_moves[m].pool_slot];
    for (int32_t s = 0; s < p->num_blocks; s++) by_slot[s] = -1;
    for (int32_t m = 0; m < nu; m++) by_slot[out->unpack_moves[m].pool_slot] = m;
    if (out->pack_hazard)
      for (int32_t j = 0; j < npk; j++) out->pack_hazard[j] = by_slot[out->pack_moves[j].pool_slot];
    free(by_slot);
  }

  free(ev); free(pq); free(r); free(g); free(nb); free(adm); free(victim);
  free(leader_of); free(follows); free(shared);
  return status;
}

/* ------------------------------------------------------ KV block copies */

static uint8_t *pool_chunk(const cref_pool *pl, int32_t slot, int32_t layer, int32_t kv) {
  return pl->base + (int64_t)layer * pl->layer_stride + (int64_t)kv * pl->kv_stride +
         (int64_t)slot * pl->slot_stride;
}
static int64_t staging_off(const cref_pool *pl, int32_t j, int32_t layer, int32_t kv) {
  return (((int64_t)j * pl->num_layers + layer) * 2 + kv) * pl->chunk_bytes;
}

void cref_pack(const cref_pool *pl, uint8_t *staging, const cref_move *mv, int32_t n) {
  for (int32_t m = 0; m < n; m++)
    for (int32_t l = 0; l < pl->num_layers; l++)
      for (int32_t kv = 0; kv < 2; kv++)
        memcpy(staging + staging_off(pl, mv[m].staging_slot, l, kv),
               pool_chunk(pl, mv[m].pool_slot, l, kv), (size_t)pl->chunk_bytes);
}

void cref_unpack(const cref_pool *pl, const uint8_t *staging, const cref_move *mv, int32_t n) {
  for (int32_t m = 0; m < n; m++)
    for (int32_t l = 0; l < pl->num_layers; l++)
      for (int32_t kv = 0; kv < 2; kv++)
        memcpy(pool_chunk(pl, mv[m].pool_slot, l, kv),
               staging + staging_off(pl, mv[m].staging_slot, l, kv), (size_t)pl->chunk_bytes);
}

/* ------------------------------------------------- prefix hit detection */

typedef struct { uint64_t hash; uint8_t tier; } cref_ientry;

static int cmp_ientry(const void *a, const void *b) {
  const uint64_t x = ((const cref_ientry *)a)->hash, y = ((const cref_ientry *)b)->hash;
  return x < y ? -1 : (x > y ? 1 : 0);
}
static int cmp_key(const void *k, const void *e) {
  const uint64_t x = *(const uint64_t *)k, y = ((const cref_ientry *)e)->hash;
  return x < y ? -1 : (x > y ? 1 : 0);
}

int32_t cref_prefix_probe(int32_t n_entries, const uint64_t *index_hashes,
                          const uint8_t *index_tiers, int32_t n, const int32_t *block_offsets,
                          const uint64_t *block_hashes, const int32_t *n_in,
                          int32_t block_tokens, int32_t *n_prefix_out,
                          uint8_t *prefix_tier_out) {
  if (n_entries < 0 || n < 0 || block_tokens < 1) return CREF_EINVAL;
  if (n > 0 && block_offsets[0] != 0) return CREF_EINVAL;
  for (int32_t i = 0; i < n; i++) {
    if (block_offsets[i + 1] < block_offsets[i] || n_in[i] < 1) return CREF_EINVAL;
    for (int32_t b = block_offsets[i]; b < block_offsets[i + 1]; b++)
      if (block_hashes[b] == 0) return CREF_EINVAL;
  }
  /* the index: one entry per distinct hash, holding its deepest tier */
  cref_ientry *idx = (cref_ientry *)malloc(sizeof(cref_ientry) * (size_t)(n_entries ? n_entries : 1));
  for (int32_t e = 0; e < n_entries; e++) {
    if (index_hashes[e] == 0 || index_tiers[e] > CREF_KV_NVME) { free(idx); return CREF_EINVAL; }
    idx[e].hash = index_hashes[e];
    idx[e].tier = index_tiers[e];
  }
  qsort(idx, (size_t)n_entries, sizeof(cref_ientry), cmp_ientry);
  int32_t m = 0;
  for (int32_t e = 0; e < n_entries; e++) {
    if (m > 0 && idx[m - 1].hash == idx[e].hash) {
      if (idx[e].tier > idx[m - 1].tier) idx[m - 1].tier = idx[e].tier;
    } else {
      idx[m++] = idx[e];
    }
  }
  /* each request: leading blocks while they are cached, up to the cap */
  for (int32_t i = 0; i < n; i++) {
    const int32_t have = block_offsets[i + 1] - block_offsets[i];
    const int32_t cap = (n_in[i] - 1) / block_tokens;
    const int32_t lim = have < cap ? have : cap;
    int32_t matched = 0;
    uint8_t tier = 0;
    while (matched < lim) {
      const cref_ientry *hit = (const cref_ientry *)bsearch(
          &block_hashes[block_offsets[i] + matched], idx, (size_t)m, sizeof(cref_ientry), cmp_key);
      if (!hit) break;
      if (hit->tier > tier) tier = hit->tier;
      matched++;
    }
    n_prefix_out[i] = matched * block_tokens;
    prefix_tier_out[i] = matched > 0 ? tier : (uint8_t)CREF_KV_NONE;
  }
  free(idx);
  return CREF_OK;
}

/* ------------------------------------------------ per-tier LRU reclamation */

/* reclamation order of a free slot: empty before cached, then least recent
   use, then the lower slot */
typedef struct { int32_t cached; int64_t last_use; int32_t slot; } cref_lru;

static int cmp_lru(const void *a, const void *b) {
  const cref_lru *x = (const cref_lru *)a, *y = (const cref_lru *)b;
  if (x->cached != y->cached) return x->cached < y->cached ? -1 : 1;
  if (x->last_use != y->last_use) return x->last_use < y->last_use ? -1 : 1;
  return x->slot < y->slot ? -1 : (x->slot > y->slot ? 1 : 0);
}
static int cmp_i32(const void *a, const void *b) {
  const int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
  return x < y ? -1 : (x > y ? 1 : 0);
}
static int cmp_u64(const void *k, const void *e) {
  const uint64_t x = *(const uint64_t *)k, y = *(const uint64_t *)e;
  return x < y ? -1 : (x > y ? 1 : 0);
}

int32_t cref_tier_reclaim(int32_t tier, int32_t n_slots, uint64_t *block_hash,
                          int64_t *last_use_ns, const uint8_t *held, int32_t need,
                          int32_t n_incoming, const cref_demotion *incoming,
                          int32_t max_outgoing, cref_demotion *outgoing, int32_t *n_outgoing,
                          int32_t *freed, int32_t *placed, int32_t n_index,
                          const uint64_t *index_keys, uint8_t *index_masks) {
  if (tier < 0 || tier > 2 || n_slots < 0 || need < 0 || n_incoming < 0 || n_index < 0)
    return CREF_EINVAL;
  const int64_t total64 = (int64_t)need + n_incoming;
  if (tier < 2 && max_outgoing < total64) return CREF_EINVAL;
  for (int32_t s = 0; s < n_slots; s++)
    if (last_use_ns[s] < 0) return CREF_EINVAL;
  for (int32_t j = 0; j < n_incoming; j++)
    if (incoming[j].hash == 0) return CREF_EINVAL;
  for (int32_t e = 0; e < n_index; e++)
    if (index_keys[e] == 0 || index_masks[e] > 7 || (e > 0 && index_keys[e] <= index_keys[e - 1]))
      return CREF_EINVAL;

  /* the free slots in reclamation order */
  cref_lru *cand = (cref_lru *)malloc(sizeof(cref_lru) * (size_t)(n_slots ? n_slots : 1));
  int32_t n_free = 0;
  for (int32_t s = 0; s < n_slots; s++) {
    if (held[s]) continue;
    cand[n_free].cached = block_hash[s] != 0;
    cand[n_free].last_use = block_hash[s] != 0 ? last_use_ns[s] : 0;
    cand[n_free].slot = s;
    n_free++;
  }
  if (total64 > n_free) { free(cand); return CREF_ENOSPC; }
  const int32_t total = (int32_t)total64;
  qsort(cand, (size_t)n_free, sizeof(cref_lru), cmp_lru);

  /* the `total` first, listed by slot */
  int32_t *rec = (int32_t *)malloc(sizeof(int32_t) * (size_t)(total ? total : 1));
  for (int32_t i = 0; i < total; i++) rec[i] = cand[i].slot;
  qsort(rec, (size_t)total, sizeof(int32_t), cmp_i32);

  /* demotion decisions on the index as it was when the call began */
  uint8_t *demote = (uint8_t *)calloc((size_t)(total ? total : 1), 1);
  int32_t n_out = 0;
  for (int32_t i = 0; i < total; i++) {
    const int32_t s = rec[i];
    if (block_hash[s] == 0 || tier == 2) continue;
    const uint64_t *hit = n_index ? (const uint64_t *)bsearch(&block_hash[s], index_keys,
                                                              (size_t)n_index, sizeof(uint64_t),
                                                              cmp_u64)
                                  : NULL;
    const uint8_t mask = hit ? index_masks[hit - index_keys] : 0;
    if ((mask >> (tier + 1)) == 0) {
      demote[i] = 1;
      outgoing[n_out].hash = block_hash[s];
      outgoing[n_out].last_use_ns = last_use_ns[s];
      outgoing[n_out].src_slot = s;
      outgoing[n_out].pad = 0;
      n_out++;
    }
  }
  /* index updates: the tier loses every reclaimed block, the next tier
     gains the demoted ones */
  for (int32_t i = 0; i < total; i++) {
    const int32_t s = rec[i];
    if (block_hash[s] == 0 || n_index == 0) continue;
    const uint64_t *hit = (const uint64_t *)bsearch(&block_hash[s], index_keys, (size_t)n_index,
                                                    sizeof(uint64_t), cmp_u64);
    if (!hit) continue;
    uint8_t *m = &index_masks[hit - index_keys];
    *m = (uint8_t)(*m & ~(1u << tier));
    if (demote[i]) *m = (uint8_t)(*m | (1u << (tier + 1)));
  }
  /* slot table: the caller's slots empty, the rest take the incoming blocks */
  for (int32_t i = 0; i < total; i++) {
    const int32_t s = rec[i];
    if (i < need) {
      freed[i] = s;
      block_hash[s] = 0;
      last_use_ns[s] = 0;
    } else {
      placed[i - need] = s;
      block_hash[s] = incoming[i - need].hash;
      last_use_ns[s] = incoming[i - need].last_use_ns;
    }
  }
  *n_outgoing = n_out;
  free(demote); free(rec); free(cand);
  return CREF_OK;
}
