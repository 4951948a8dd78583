// cascade_step.hip -- one Cascade scheduling step on gfx950.
//
// Paper: Cascade (arXiv 2608.06557).  The step evaluates every request's
// latency budget (Section 4.2: TTFT estimator, eq:est_latency, eq:budget_eq;
// Section 4.3: eq:rem_budget_eq), its restore volume (eq:restore_time,
// eq:max_restorable), orders the queue least-remaining-budget-first and runs
// Algorithm 1's Phase 2 over the whole queue: restore/prefetch volume under
// the link cap, chunked-prefill token grants, HBM block admission and
// budget-aware preemption (Section 4.4).
//
// The paper's scheduler is a sequential CPU loop.  Here it is 3 + P
// dependent launches on one stream:
//   eval      one lane per request: validation, budget, tier, restore want,
//             priority key, scan record; per-workgroup partial totals (no
//             atomics); also clears this step's histograms, tile totals and
//             look-back words
//   prep      totals of the partials, key compression to the live budget
//             range, every digit histogram in one read, block-table checks
//   radix<p>  onesweep LSD radix pass p over 2048-key tiles (wave64 ballot
//             ranking, per-digit decoupled look-back), launched for the
//             passes a host-side bound on the key width allows; 8- or 9-bit
//             digits and the digits that move data are decided on the device.
//             The last data-moving pass writes the sorted order with each
//             request's scan record and adds every scan tile's level-1 totals
//   scan      Algorithm 1's loop as prefix sums in priority order over
//             1024-position tiles (level-2 prefix by a decoupled look-back);
//             the launch's last 32 workgroups wait for every tile's hand-over,
//             then pick the preemption victims and write the slot list and
//             the pack / unpack move lists
// A queue of at most 1024 requests runs the whole step in one workgroup.
// All arithmetic is integer (64-bit, or 32-bit where a bound allows it), so
// the result is bit-exact.
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <mutex>

#include "cascade.h"
#include "device_util.h"

namespace cascade {
namespace {

constexpr int kSortBlock = 512;  // radix workgroups: 8 waves, one tile of 1024 or 2048 keys
constexpr int kSortWaves = kSortBlock / 64;
constexpr int kSortItems = 4;
constexpr int kSortTile = kSortBlock * kSortItems;
// Queues up to kTinyTileMax requests sort 512-key tiles, up to kSmallTileMax
// 1024-key tiles (less ranking, reorder and write work per workgroup; at
// most 32 or 64 tiles, so the look-back stays short); longer ones 2048-key
// tiles (more tiles would lengthen the look-back more than they save).
constexpr int kSortTileTiny = kSortTile / 4;
constexpr int kSortTileSmall = kSortTile / 2;
constexpr int kTinyTileMax = 16384;
constexpr int kSmallTileMax = 65536;
constexpr int kSortWin = 32;     // predecessors read per look-back round trip (radix)
constexpr int kScanItems = 4;
constexpr int kScanTile = kBlock * kScanItems;
constexpr int kPrepItems = 8;       // keys per prep thread (2 up to kTinyPrepMax)
constexpr int kTinyPrepMax = 16384;
constexpr int kEvalItems = 1;
static_assert(kBlock * kEvalItems <= 2048, "an eval workgroup's sums fit 32 bits");
constexpr int kMaxW = 9;         // widest digit of the multi-launch sort
constexpr int kMaxBins = 1 << kMaxW;
constexpr int kMaxPasses = (64 + kMaxW - 1) / kMaxW;  // passes of the multi-launch sort, at most
constexpr int kRadix = 256;      // one workgroup's LDS sort of a small queue: 8-bit digits
constexpr int kL1 = 5;           // first-level scan values
constexpr int kMaxScanTiles = ((1 << 20) + kScanTile - 1) / kScanTile;
constexpr int kL2 = 7;           // second-level scan values
constexpr int kL2Stride = 16;    // level-2 look-back words: one 128-byte line per tile

// Record of one request for the priority-order scan (16 bytes).
//   x want_blocks; for a running prefill (which never restores) the first
//     entry of its block-table row instead
//   y base_need, z reuse_tokens (HBM prefix or progress)
//   w bits 0..19 held blocks, 20..21 state, 22..23 prefix tier,
//     24..25 group, 26 spill-fits-budget, 27 decode needs a new block,
//     28 a queued DRAM/NVMe member of a prefix group (then z is the group and
//     bits 0..19 its prefix blocks), 29 a follower of that group's leader
//     (rewritten by share_kernel: x the leader's request index, y the need
//     net of the shared blocks, z the shared tokens, prefix tier HBM, so
//     the scan references the shared blocks as it does an HBM prefix)
__device__ __forceinline__ int rec_held(int w) { return w & 0xFFFFF; }
__device__ __forceinline__ int rec_state(int w) { return (w >> 20) & 3; }
__device__ __forceinline__ int rec_member(int w) { return (w >> 28) & 1; }
__device__ __forceinline__ int rec_follow(int w) { return (w >> 29) & 1; }
__device__ __forceinline__ int rec_want(const int4 &r) {
  return (rec_state(r.w) == CASCADE_RUNNING_PREFILL || rec_follow(r.w)) ? 0 : r.x;
}
__device__ __forceinline__ int rec_tier(int w) { return (w >> 22) & 3; }
__device__ __forceinline__ int rec_grp(int w) { return (w >> 24) & 3; }
__device__ __forceinline__ int rec_offl(int w) { return (w >> 26) & 1; }
__device__ __forceinline__ int rec_decnb(int w) { return (w >> 27) & 1; }
// Slot of a member's (prefix group, priority group) in the shared-prefix
// leader tables.
__device__ __forceinline__ int share_slot(const int4 &r) {
  return 2 * r.z + (rec_grp(r.w) == 2 ? 1 : 0);
}
// A member with a restore want marks its group's leader table with its
// position p: the table keeps the largest n - p, so the first such position.
__device__ __forceinline__ void share_mark(unsigned *lead, const int4 &r, int p, int n) {
  if (lead && rec_member(r.w) && r.x > 0 && (unsigned)r.z < (unsigned)n)
    atomicMax(lead + share_slot(r), (unsigned)(n - p));
}

// Totals of one eval workgroup (64 bytes).
struct Partial {
  long long held, need1, want1;   // blocks held by running prefills; base need and
                                  // want over decode + Tier-1
  unsigned long long bmin, bmax;  // range of the biased, clamped budget
  unsigned c0, c1, c2, bad;       // requests per group; data-rule violations
  unsigned pad[2];
};

// A running prefill, as seen by the scan (compact list, 64 bytes).
struct RpInfo {
  int req, pos, eligible, held, row0, offl, pad[2];
  long long x, y, z, zp;          // inclusive prefixes at pos
};
struct alignas(16) RestoreEnt { int req, stage_off, alloc_off, blocks; };
// Totals of one scan tile over its admitted / left-out requests.
struct TileTot {
  long long adm_nb, elig_h, elig_offl_h, n_adm, n_unpack, n_restore, pad[2];
};
constexpr int kVictimCap = 256;   // victims staged in LDS by the finishing workgroup
constexpr int kRestoreCap = 1024; // restore-list entries staged in LDS for the search

// Device control block.  eval's first thread zeroes the header, every eval
// workgroup clears part of the histograms and look-back words.
struct Ctl {
  unsigned long long bmin, bmax;  // totals, written by prep's workgroup 0
  long long held_rp, need1, want1;
  long long want1_sub, need1_sub; // followers' wants and shared tokens in groups 0-1
  unsigned cnt[4];
  unsigned nact;                  // data-moving radix passes, from the sort plan
  int n_rp;                       // running prefills in the queue (last scan tile)
  int kstar;                      // first position whose blocks do not fit
  long long kx, ky, kz, kzp;      // prefixes just before kstar
  alignas(16) unsigned hist[kMaxPasses][kMaxBins];  // cleared by eval's grid
  // scan tiles whose hand-over is complete, tile t counted in counter
  // t % kTicketGroups, one per 128-byte line (cleared by eval's grid)
  alignas(128) unsigned done[kTicketGroups * kTicketStride];
};
constexpr size_t kCtlHeaderWords = offsetof(Ctl, hist) / 4;

// Sorted order with each request's scan record and block-table row offset,
// written by the last data-moving radix pass.
struct Sorted {
  unsigned *order;
  int4 *rec;
};

struct Consts {                   // parameters the kernels use, flattened
  long long t_now, c_iter, c_dec, c_tok, c_attn;
  long long delta1, delta2, blk1, blk2;  // restore paths: DRAM, NVMe
  int num_classes, bt, chunk, d, dmax, gamma_q16, token_cap, rho_q16, max_move;
  int num_blocks, n_free;
  long long slo[16];
};

struct Outs {                     // output pointers the scan writes
  int *order, *granted, *restore, *alloc_begin, *alloc_count, *admitted, *slot_list;
  int *share_leader;                 // null without prefix groups
  uint8_t *action;
  cascade_move_t *unpack, *pack;
  int *unpack_hazard, *pack_hazard;  // may be null
  int sl_cap, unpack_cap, pack_cap;
};

// Records handed to the finishing workgroup within a launch move as 8-byte
// agent-scope atomic words (no cache write-back needed to publish them).
template <typename T>
__device__ __forceinline__ void store_agent_rec(T *dst, const T &v) {
  static_assert(sizeof(T) % 8 == 0 && alignof(T) >= 4, "whole 8-byte words");
  unsigned long long w[sizeof(T) / 8];
  __builtin_memcpy(w, &v, sizeof(T));
  unsigned long long *d = reinterpret_cast<unsigned long long *>(dst);
#pragma unroll
  for (int k = 0; k < (int)(sizeof(T) / 8); ++k) store_agent(d + k, w[k]);
}
template <typename T>
__device__ __forceinline__ T load_agent_rec(const T *src) {
  static_assert(sizeof(T) % 8 == 0 && alignof(T) >= 4, "whole 8-byte words");
  unsigned long long w[sizeof(T) / 8];
  const unsigned long long *p = reinterpret_cast<const unsigned long long *>(src);
#pragma unroll
  for (int k = 0; k < (int)(sizeof(T) / 8); ++k) w[k] = load_agent(p + k);
  T v;
  __builtin_memcpy(&v, w, sizeof(T));
  return v;
}

__device__ __forceinline__ bool bad_status(int s) {
  return s == CASCADE_EINVAL || s == CASCADE_ETIMEOUT || s == CASCADE_EINTERNAL;
}
__device__ __forceinline__ long long lmin(long long a, long long b) { return a < b ? a : b; }
__device__ __forceinline__ void set_status(int *info, int code) { store_agent(info, code); }
__device__ __forceinline__ unsigned udiv_ceil(unsigned a, unsigned b) { return (a + b - 1u) / b; }

// ---------------------------------------------------------------- eval

// Iteration cost model of the TTFT estimator (Section 4.2): n prompt tokens
// at positions s.. with dd co-scheduled decodes, picoseconds.  n + s <= 2^17.
__device__ __forceinline__ long long compute_ps(long long n, long long s, long long dd,
                                                const Consts &c) {
  if (n <= 0) return 0;
  const long long iters = udiv_ceil((unsigned)n, (unsigned)c.chunk);
  const long long pairs = (n * (2 * s + n + 1)) >> 1;
  return iters * (c.c_iter + dd * c.c_dec) + n * c.c_tok + c.c_attn * pairs;
}
__device__ __forceinline__ long long ns_of_ps(long long ps) {
  return (long long)((unsigned long long)ps / 1000ull);
}
// eq:restore_time in blocks
__device__ __forceinline__ long long restore_ns(long long x, long long delta, long long blk) {
  return x == 0 ? 0 : delta + x * blk;
}

// Section 4.2-4.4 for request i: validation of its data, the actual- and
// maximum-load estimates, eq:est_latency, eq:budget_eq, eq:rem_budget_eq, the
// tier transition, eq:max_restorable (kept only if cheaper than recompute),
// the priority group and the record the scan reads.
struct ReqEval {
  long long brem, held, need1, want1;  // need1 / want1: contributions of groups 0-1
  unsigned long long biased;           // clamped budget + 2^61
  int4 rec;
  unsigned tnew;
  int grp;
  bool bad;
};

__device__ __forceinline__ ReqEval eval_request(const cascade_requests_t &rq,
                                                const int *__restrict__ ro, const Consts &c,
                                                const long long *s_slo, int i, int n) {
  ReqEval r;
  r.bad = false;
  const unsigned cls = rq.slo_class[i], st = rq.state[i], qt = rq.queue_tier[i],
                 pt = rq.prefix_tier[i];
  const long long arr = rq.arrival_ns[i];
  const int n_in_r = rq.n_in[i], n_out_r = rq.n_out_pred[i], n_pre_r = rq.n_prefix[i],
            prog_r = rq.n_progress[i];
  const int r0 = ro[i], r1 = ro[i + 1];
  const unsigned bt = (unsigned)c.bt;

  // ---- domain rules of the request data
  if (i > 0 && rq.id[i] <= rq.id[i - 1]) r.bad = true;
  if (i == 0 && r0 != 0) r.bad = true;
  if (cls >= (unsigned)c.num_classes || st > 2 || qt > 2 || pt > 3) r.bad = true;
  if (n_in_r < 1 || n_in_r > (1 << 17) || n_out_r < 0 || n_out_r > (1 << 17)) r.bad = true;
  if (n_pre_r < 0 || n_pre_r > n_in_r - 1 || ((unsigned)n_pre_r % bt) != 0) r.bad = true;
  if (arr < 0 || arr > c.t_now) r.bad = true;
  if (st == CASCADE_QUEUED) {
    if ((n_pre_r == 0) != (pt == CASCADE_KV_NONE) || prog_r != 0 || r1 != r0) r.bad = true;
  } else if (st == CASCADE_RUNNING_PREFILL) {
    if (prog_r < 1 || prog_r > n_in_r - 1) r.bad = true;
    else if ((long long)r1 - r0 != udiv_ceil((unsigned)prog_r, bt)) r.bad = true;
  } else {
    if (prog_r < 0 || prog_r > (1 << 17)) r.bad = true;
    else if (n_in_r >= 1 && n_in_r <= (1 << 17) &&
             (long long)r1 - r0 != udiv_ceil((unsigned)(n_in_r + prog_r), bt))
      r.bad = true;
  }

  // ---- keep the arithmetic in range whatever the data
  const unsigned st_s = st > 2 ? 0u : st;
  const unsigned pt_s = pt > 3 ? 3u : pt;
  const unsigned cls_s = cls >= (unsigned)c.num_classes ? 0u : cls;
  const long long n_in = n_in_r < 1 ? 1 : (n_in_r > (1 << 17) ? (1 << 17) : n_in_r);
  const long long n_out = n_out_r < 0 ? 0 : (n_out_r > (1 << 17) ? (1 << 17) : n_out_r);
  const long long n_pre = n_pre_r < 0 ? 0 : (n_pre_r > n_in - 1 ? n_in - 1 : n_pre_r);
  const long long prog = prog_r < 0 ? 0 : (prog_r > (1 << 17) ? (1 << 17) : prog_r);
  const long long elapsed = (arr < 0 || arr > c.t_now) ? 0 : c.t_now - arr;
  const long long row = (long long)r1 - r0;
  const long long held = row < 0 ? 0 : (row > 0xFFFFF ? 0xFFFFF : row);

  // ---- Section 4.2: actual-load and maximum-load estimates
  long long l_act, l_max, pb = 0, base_need;
  const long long delta = (pt_s == CASCADE_KV_NVME) ? c.delta2 : c.delta1;
  const long long blk = (pt_s == CASCADE_KV_NVME) ? c.blk2 : c.blk1;
  const bool deep = (pt_s == CASCADE_KV_DRAM || pt_s == CASCADE_KV_NVME);
  // The three regimes share one form: `iters` iterations of the batch with
  // d (actual) or dmax (maximum) co-scheduled decodes, plus the prompt
  // tokens' own cost (compute_ps with the two decode counts), plus a restore
  // for a queued request whose prefix is in DRAM or NVMe.  Computed once
  // for every lane, so the regimes do not diverge.
  long long reuse = 0, rest = 0, n_tok = 0, iters;
  if (st_s == CASCADE_QUEUED) {
    if (pt_s != CASCADE_KV_NONE) {
      pb = (unsigned)n_pre / bt;
      reuse = n_pre;
      if (deep) rest = restore_ns(pb, delta, blk);
    }
    n_tok = n_in - reuse;
    base_need = (pt_s == CASCADE_KV_HBM) ? n_in - n_pre : n_in;
  } else if (st_s == CASCADE_RUNNING_PREFILL) {
    reuse = prog > n_in ? n_in : prog;
    n_tok = n_in - reuse;
    base_need = n_tok;
  } else {
    base_need = 1;
  }
  if (st_s == CASCADE_DECODE) {
    iters = n_out - prog < 0 ? 0 : n_out - prog;
  } else {
    iters = udiv_ceil((unsigned)n_tok, (unsigned)c.chunk);
  }
  const long long tok_ps = n_tok * c.c_tok + c.c_attn * ((n_tok * (2 * reuse + n_tok + 1)) >> 1);
  l_act = ns_of_ps(iters * (c.c_iter + (long long)c.d * c.c_dec) + tok_ps) + rest;
  l_max = ns_of_ps(iters * (c.c_iter + (long long)c.dmax * c.c_dec) + tok_ps) + rest;
  // ---- eq:est_latency, floor((L_act + L_max) * gamma / 2^17), exact in
  //      64 bits: split the sum at bit 17
  const unsigned long long sum = (unsigned long long)(l_act + l_max);
  const unsigned long long g = (unsigned)c.gamma_q16;
  const long long L = (long long)((sum >> 17) * g + (((sum & 0x1FFFFull) * g) >> 17));
  // ---- eq:budget_eq and eq:rem_budget_eq
  const long long b0 = s_slo[cls_s] - L;
  const long long brem = b0 - elapsed;

  // ---- Tier-1 / Tier-2 (Tier-1 iff B > 0, Tier-1 sticky, Tier-2 promoted)
  unsigned tnew = qt;
  if (st_s != CASCADE_DECODE) tnew = (qt == CASCADE_QT_TIER1 || b0 > 0) ? 1u : 2u;

  // ---- eq:max_restorable in blocks, kept only if cheaper than recompute
  long long want = 0;
  if (st_s == CASCADE_QUEUED && deep) {
    long long x = 0;
    if (brem > delta) {
      // x = min(floor((brem - delta) / blk), pb).  At or past pb + 1 blocks
      // the cap decides; below, the quotient is under 2^18 and the dividend
      // under 2^51, so the double quotient is off by at most one and two
      // integer checks make it exact
      const long long num = brem - delta;
      if (num >= (pb + 1) * blk) {
        x = pb;
      } else {
        long long q = (long long)((double)num / (double)blk);
        if (q * blk > num) --q;
        else if ((q + 1) * blk <= num) ++q;
        x = q;
      }
    }
    if (x > 0) {
      const long long all = ns_of_ps(compute_ps(n_in, 0, c.d, c));
      const long long part = ns_of_ps(compute_ps(n_in - (long long)bt * x, bt * x, c.d, c));
      if (restore_ns(x, delta, blk) >= all - part) x = 0;
    }
    want = x;
  }

  // ---- priority group and key: group in bits 63..62, clamped budget + 2^61
  const int grp = (st_s == CASCADE_DECODE) ? 0 : (tnew == 1 ? 1 : 2);
  const long long lo = -(1ll << 61), hi = (1ll << 61) - 1;
  const long long cl = brem < lo ? lo : (brem > hi ? hi : brem);
  const unsigned long long biased = (unsigned long long)(cl + (1ll << 61));

  // spill of a running prefill fits its budget (Section 4.4)
  const int offl = (st_s == CASCADE_RUNNING_PREFILL) &&
                   (restore_ns(held, c.delta1, c.blk1) <= brem);
  const int decnb = (st_s == CASCADE_DECODE) &&
                    ((long long)udiv_ceil((unsigned)(n_in + prog + 1), bt) - held) > 0;
  const bool hbm_prefix = st_s == CASCADE_QUEUED && pt_s == CASCADE_KV_HBM;
  const long long reuse_tok =
      (st_s == CASCADE_RUNNING_PREFILL) ? prog : (hbm_prefix ? n_pre : 0);
  // prefix group: ids in [-1, n); a queued DRAM/NVMe request in a group is
  // a member (its group in z, its prefix blocks in the held bits, which a
  // queued request does not use)
  int gid = -1;
  if (rq.prefix_group) {
    const int g = rq.prefix_group[i];
    if (g < -1 || g >= n) r.bad = true;
    else gid = g;
  }
  const bool member = gid >= 0 && st_s == CASCADE_QUEUED && deep;

  r.brem = brem;
  r.tnew = tnew;
  r.grp = grp;
  r.biased = biased;
  r.rec = make_int4(st_s == CASCADE_RUNNING_PREFILL ? r0 : (int)want, (int)base_need,
                    member ? gid : (int)reuse_tok,
                    (member ? (int)pb : (int)held) | ((int)st_s << 20) | ((int)pt_s << 22) |
                        (grp << 24) | (offl << 26) | (decnb << 27) | ((int)member << 28));
  r.held = st_s == CASCADE_RUNNING_PREFILL ? held : 0;
  r.need1 = grp <= 1 ? base_need : 0;
  r.want1 = grp <= 1 ? want : 0;
  return r;
}

__global__ __launch_bounds__(kBlock) void eval_kernel(
    cascade_requests_t rq, const int *__restrict__ ro, const int *__restrict__ free_slots,
    Consts c, int n, Ctl *ctl, uint4 *clear, size_t clear_vec, uint4 *clear2,
    size_t clear2_vec, int *info,
    Partial *__restrict__ partials, int64_t *__restrict__ budget_out,
    uint8_t *__restrict__ tier_out, unsigned long long *__restrict__ keys,
    int4 *__restrict__ rec) {
  __shared__ long long s_slo[16];
  __shared__ unsigned long long s_mm[kWaves * 2];
  __shared__ unsigned s_cnt[kWaves * 7];
  if (threadIdx.x < 16) s_slo[threadIdx.x] = c.slo[threadIdx.x];

  const size_t gt = (size_t)blockIdx.x * kBlock + threadIdx.x;
  const size_t gs = (size_t)gridDim.x * kBlock;
  // this step's histograms and look-back status words start at zero; the
  // first workgroup resets the control block's header and the info words
  for (size_t j = gt; j < clear_vec; j += gs) clear[j] = make_uint4(0, 0, 0, 0);
  // the shared-prefix tables (leader positions, published leader restores)
  for (size_t j = gt; j < clear2_vec; j += gs) clear2[j] = make_uint4(0, 0, 0, 0);
  if (blockIdx.x == 0) {
    const int t = threadIdx.x;
    constexpr int kKstarWord = offsetof(Ctl, kstar) / 4;
    static_assert(kCtlHeaderWords <= kBlock && CASCADE_INFO_LEN <= kBlock, "one word per thread");
    if (t < (int)kCtlHeaderWords)
      reinterpret_cast<unsigned *>(ctl)[t] = t == kKstarWord ? (unsigned)n : 0u;
    if (t < CASCADE_INFO_LEN) info[t] = t == CASCADE_INFO_N_SLOT_LIST ? c.n_free : 0;
  }
  __syncthreads();

  bool bad = false;
  long long v_held = 0, v_need1 = 0, v_want1 = 0;
  unsigned long long bmin = ~0ull, bmax = 0;
  unsigned c0 = 0, c1 = 0, c2 = 0;

  // free-list range check, spread over the grid
  for (size_t j = gt; j < (size_t)c.n_free; j += gs)
    if ((unsigned)free_slots[j] >= (unsigned)c.num_blocks) bad = true;

#pragma unroll
  for (int it = 0; it < kEvalItems; ++it) {
    const int i = (int)(blockIdx.x * kBlock * kEvalItems + it * kBlock + threadIdx.x);
    if (i >= n) continue;
    const ReqEval r = eval_request(rq, ro, c, s_slo, i, n);
    bad |= r.bad;
    bmin = r.biased < bmin ? r.biased : bmin;
    bmax = r.biased > bmax ? r.biased : bmax;
    c0 += r.grp == 0;
    c1 += r.grp == 1;
    c2 += r.grp == 2;
    budget_out[i] = r.brem;
    tier_out[i] = (uint8_t)r.tnew;
    keys[i] = ((unsigned long long)r.grp << 62) | r.biased;
    rec[i] = r.rec;
    v_held += r.held;
    v_need1 += r.need1;
    v_want1 += r.want1;
  }
  // workgroup totals, one plain store per workgroup: wave sums, then thread
  // 0 adds the waves' after one barrier.  A workgroup's sums stay below
  // 2^29 (held blocks below 2^20, token needs and restore wants below 2^18
  // per request), so they add in 32 bits.
  unsigned u[7] = {(unsigned)v_held, (unsigned)v_need1, (unsigned)v_want1, c0, c1, c2,
                   bad ? 1u : 0u};
#pragma unroll
  for (int k = 0; k < 7; ++k) u[k] = wave_sum(u[k]);
  bmin = wave_min(bmin);
  bmax = wave_max(bmax);
  if (lane_id() == 0) {
#pragma unroll
    for (int k = 0; k < 7; ++k) s_cnt[wave_id() * 7 + k] = u[k];
    s_mm[wave_id() * 2] = bmin;
    s_mm[wave_id() * 2 + 1] = bmax;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned tot[7] = {0, 0, 0, 0, 0, 0, 0};
    Partial pt;
    pt.bmin = ~0ull;
    pt.bmax = 0;
    for (int w = 0; w < kWaves; ++w) {
#pragma unroll
      for (int k = 0; k < 7; ++k) tot[k] += s_cnt[w * 7 + k];
      pt.bmin = s_mm[2 * w] < pt.bmin ? s_mm[2 * w] : pt.bmin;
      pt.bmax = s_mm[2 * w + 1] > pt.bmax ? s_mm[2 * w + 1] : pt.bmax;
    }
    pt.held = tot[0];
    pt.need1 = tot[1];
    pt.want1 = tot[2];
    pt.c0 = tot[3];
    pt.c1 = tot[4];
    pt.c2 = tot[5];
    pt.bad = tot[6];
    pt.pad[0] = pt.pad[1] = 0;
    partials[blockIdx.x] = pt;
  }
}

// ------------------------------------------------------ sort: digit plan

// Width in bits of the compressed key key' = group*span + (biased - bmin).
__device__ __forceinline__ int key_bits(unsigned long long mn, unsigned long long mx,
                                        unsigned c1, unsigned c2) {
  const unsigned long long span = mx - mn + 1;
  const unsigned long long gmax = c2 ? 2 : (c1 ? 1 : 0);
  const unsigned long long top = gmax * span + (mx - mn);
  return top ? 64 - __builtin_clzll(top) : 0;
}

// Digits of the multi-launch sort: the live key width W spread over the
// `passes` launched passes: 8 bits wide where that suffices, else kMaxW
// (which the host's bound on the key width makes enough).
struct DigitPlan {
  int w, nd;      // digit width, digits below the key width
  unsigned bins;  // 2^w
};
__device__ __forceinline__ DigitPlan digit_plan(const Ctl *ctl, int passes) {
  const int W = key_bits(ctl->bmin, ctl->bmax, ctl->cnt[1], ctl->cnt[2]);
  DigitPlan d;
  d.w = W <= 8 * passes ? 8 : kMaxW;
  d.nd = (W + d.w - 1) / d.w;
  d.bins = 1u << d.w;
  return d;
}

// ---------------------------------------------------------------- prep

// Totals of eval's partials; order-preserving key compression
// key' = group * span + (biased - bmin), then one read of the keys builds
// every digit's histogram (LDS counts, then one global add per non-empty
// bucket).  The keys are requested before the totals they are compressed
// with.  Also checks the block-table slots, whose extent is only trustworthy
// after eval.
template <int kItems>
__global__ __launch_bounds__(kBlock) void prep_kernel(int n, int num_blocks, int n_partials,
                                                      int passes,
                                                      const Partial *__restrict__ partials,
                                                      const int *__restrict__ ro,
                                                      const int *__restrict__ slots, Ctl *ctl,
                                                      int *info,
                                                      unsigned long long *__restrict__ keys,
                                                      unsigned *__restrict__ vals) {
  __shared__ unsigned s_hist[kMaxPasses * kMaxBins];
  __shared__ unsigned long long s_red[kWaves * 9];
  const int t = threadIdx.x, lane = lane_id(), wave = wave_id();
  const int base = blockIdx.x * kBlock * kItems;
  unsigned long long kv[kItems];
#pragma unroll
  for (int j = 0; j < kItems; ++j) {
    const int idx = base + j * kBlock + t;
    kv[j] = idx < n ? keys[idx] : 0ull;
  }
  // totals of eval's partials: sums (held, need1, want1, three group counts,
  // bad), then min and max, reduced per wave and combined after one barrier
  unsigned long long v[9] = {0, 0, 0, 0, 0, 0, 0, ~0ull, 0};
#pragma unroll 1
  for (int j = t; j < n_partials; j += kBlock) {
    const Partial p = partials[j];
    v[0] += (unsigned long long)p.held;
    v[1] += (unsigned long long)p.need1;
    v[2] += (unsigned long long)p.want1;
    v[3] += p.c0;
    v[4] += p.c1;
    v[5] += p.c2;
    v[6] += p.bad;
    v[7] = p.bmin < v[7] ? p.bmin : v[7];
    v[8] = p.bmax > v[8] ? p.bmax : v[8];
  }
#pragma unroll
  for (int k = 0; k < 7; ++k) v[k] = wave_sum(v[k]);
  v[7] = wave_min(v[7]);
  v[8] = wave_max(v[8]);
  if (lane == 0) {
#pragma unroll
    for (int k = 0; k < 9; ++k) s_red[wave * 9 + k] = v[k];
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < 9; ++k) v[k] = s_red[k];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) {
#pragma unroll
    for (int k = 0; k < 7; ++k) v[k] += s_red[w * 9 + k];
    v[7] = s_red[w * 9 + 7] < v[7] ? s_red[w * 9 + 7] : v[7];
    v[8] = s_red[w * 9 + 8] > v[8] ? s_red[w * 9 + 8] : v[8];
  }
  const unsigned long long mn = v[7], mx = v[8];
  const unsigned c1 = (unsigned)v[4], c2 = (unsigned)v[5];
  const bool bad_data = v[6] != 0;
  if (blockIdx.x == 0 && t == 0) {
    ctl->bmin = mn;
    ctl->bmax = mx;
    ctl->held_rp = (long long)v[0];
    ctl->need1 = (long long)v[1];
    ctl->want1 = (long long)v[2];
    ctl->cnt[0] = (unsigned)v[3];
    ctl->cnt[1] = c1;
    ctl->cnt[2] = c2;
    if (bad_data) set_status(info, CASCADE_EINVAL);
  }
  if (bad_data) return;  // bad request data: nothing below is meaningful

  // block-table slots in range: requested here, checked after the histograms
  const int nnz = ro[n];
  const int gt = blockIdx.x * kBlock + t, gs = gridDim.x * kBlock;
  int sv[8];
#pragma unroll
  for (int u = 0; u < 8; ++u) sv[u] = (gt + u * gs < nnz) ? slots[gt + u * gs] : 0;

  // the digit plan, from the totals just reduced (the same in every kernel)
  const int W = key_bits(mn, mx, c1, c2);
  const int w = W <= 8 * passes ? 8 : kMaxW;
  const int nd = min((W + w - 1) / w, kMaxPasses);
  const unsigned bins = 1u << w;
  for (int k = t; k < nd * (int)bins; k += kBlock) s_hist[k] = 0;
  __syncthreads();
  const unsigned long long span = mx - mn + 1;
#pragma unroll
  for (int j = 0; j < kItems; ++j) {
    const int idx = base + j * kBlock + t;
    const bool in = idx < n;
    const unsigned long long k0 = kv[j];
    const unsigned long long k = (k0 >> 62) * span + ((k0 & ((1ull << 62) - 1)) - mn);
    if (in) {
      keys[idx] = k;
      vals[idx] = (unsigned)idx;
    }
    if (in) {
      for (int d = 0; d < nd; ++d)
        atomicAdd(&s_hist[d * bins + ((k >> (w * d)) & (bins - 1))], 1u);
    }
  }
  bool bad = false;
#pragma unroll
  for (int u = 0; u < 8; ++u) bad |= (unsigned)sv[u] >= (unsigned)num_blocks;
#pragma unroll 1
  for (int j0 = gt + 8 * gs; j0 < nnz; j0 += 8 * gs) {
    int x[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) x[u] = (j0 + u * gs < nnz) ? slots[j0 + u * gs] : 0;
#pragma unroll
    for (int u = 0; u < 8; ++u) bad |= (unsigned)x[u] >= (unsigned)num_blocks;
  }
  if (__syncthreads_or(bad ? 1 : 0)) {
    if (t == 0) set_status(info, CASCADE_EINVAL);
  }
  // two neighbouring buckets per 64-bit add (a count never exceeds n < 2^32,
  // so nothing carries into the upper word): half the global atomics
  const int half = (int)bins >> 1;
  for (int k = t; k < nd * half; k += kBlock) {
    const int d = k >> (w - 1), b = (k & (half - 1)) * 2;
    const unsigned lo = s_hist[d * bins + b], hi = s_hist[d * bins + b + 1];
    if (lo | hi)
      atomicAdd(reinterpret_cast<unsigned long long *>(&ctl->hist[d][b]),
                ((unsigned long long)hi << 32) | lo);
  }
}

// ---------------------------------------------------------- radix pass

// Level-1 scan values of one request (record r), added to scan tile `tile`'s
// totals in LDS (tile < 0: no request).  Lanes whose tile is the wave's first
// lane's add wave sums with one atomic per value; the others add their own.
__device__ __forceinline__ void l1_contrib(unsigned *s_l1, int tile, const int4 &r) {
  const bool v = tile >= 0;
  const bool rp = v && rec_state(r.w) == CASCADE_RUNNING_PREFILL;
  const unsigned h = rp ? (unsigned)rec_held(r.w) : 0u;
  unsigned c[kL1] = {v ? (unsigned)rec_want(r) : 0u, v ? (unsigned)r.y : 0u, h,
                     rec_offl(r.w) ? h : 0u, rp ? 1u : 0u};
  const int t0 = __builtin_amdgcn_readfirstlane(tile);
  const bool same = tile == t0;
  if (t0 >= 0) {
#pragma unroll
    for (int k = 0; k < kL1; ++k) {
      const unsigned sum = wave_sum(same ? c[k] : 0u);
      if (lane_id() == 0 && sum) atomicAdd(s_l1 + t0 * kL1 + k, sum);
    }
  }
  if (v && !same) {
#pragma unroll
    for (int k = 0; k < kL1; ++k)
      if (c[k]) atomicAdd(s_l1 + tile * kL1 + k, c[k]);
  }
}

// One look-back window of digit b: the counts of tiles start, start - 1,
// .. (kSortWin of them; below tile 0 an inclusive zero), read at once and
// consumed up to the first inclusive prefix or the first unpublished word.
struct SortWindow {
  unsigned part;  // the consumed words' counts
  int take;       // words consumed
  bool done;      // an inclusive prefix ended the window
  bool stalled;   // an unpublished word ended it
};
__device__ __forceinline__ SortWindow sort_window(const unsigned *status, int start, int b) {
  unsigned v[kSortWin];
#pragma unroll
  for (int i = 0; i < kSortWin; ++i) {
    const int j = start - i;
    v[i] = j >= 0 ? load_agent(status + (size_t)j * kMaxBins + b) : kFlagInclusive;
  }
  unsigned missing = 0, inclusive = 0;
#pragma unroll
  for (int i = 0; i < kSortWin; ++i) {
    missing |= ((v[i] & 3u) == 0 ? 1u : 0u) << i;
    inclusive |= ((v[i] & 3u) == kFlagInclusive ? 1u : 0u) << i;
  }
  const int fm = missing ? __builtin_ctz(missing) : kSortWin;
  const int fi = inclusive ? __builtin_ctz(inclusive) : kSortWin;
  SortWindow w;
  w.done = fi < fm;
  w.take = w.done ? fi + 1 : fm;
  w.stalled = !w.done && fm < kSortWin;
  w.part = 0;
#pragma unroll
  for (int i = 0; i < kSortWin; ++i) w.part += i < w.take ? (v[i] >> 2) : 0u;
  return w;
}

// Decoupled look-back of a pass with at most kSortBlock/2 bins, by thread
// pairs: thread b reads the window of the pair's next predecessors and
// thread b + kSortBlock/2 the window behind it, so a round trip covers
// 2 * kSortWin tiles.  The second thread's result goes through LDS; the
// first adds it only when its own window ended on neither an inclusive
// prefix nor an unpublished word.  Called by every thread of the
// workgroup; the sum is valid in threads t < bins.
static_assert(2 * kRadix == kSortBlock, "an 8-bit pass pairs its threads");
__device__ __forceinline__ unsigned paired_look_back(const unsigned *status, int tile,
                                                     unsigned bins, unsigned *s_px, int *s_pc,
                                                     int *s_pn, bool *timed_out) {
  const int t = threadIdx.x, b = t % (kSortBlock / 2), half = t / (kSortBlock / 2);
  const bool act = b < (int)bins && tile > 0;
  int next = tile - 1;
  bool done = !act;
  unsigned sum = 0, spins = 0;
  while (true) {
    SortWindow w = {0u, 0, true, false};
    if (!done) w = sort_window(status, next - half * kSortWin, b);
    if (half == 1) {
      s_px[b] = w.part;
      s_pc[b] = w.take | (w.done ? 256 : 0) | (w.stalled ? 512 : 0);
    }
    __syncthreads();
    bool stall = false;
    if (half == 0 && !done) {
      sum += w.part;
      if (w.done) {
        done = true;
      } else if (w.stalled) {
        next -= w.take;
        stall = true;
      } else {  // the first window was consumed whole: the second follows it
        const int c = s_pc[b];
        sum += s_px[b];
        if (c & 256) {
          done = true;
        } else if (c & 512) {
          next -= kSortWin + (c & 255);
          stall = true;
        } else {
          next -= 2 * kSortWin;
        }
      }
      s_pn[b] = done ? -1 : next;
    }
    __syncthreads();
    if (half == 1 && act) {
      next = s_pn[b];
      done = next < 0;
    }
    if (!__syncthreads_or(done ? 0 : 1)) break;
    if (++spins > kSpinLimit) {
      *timed_out = true;
      break;
    }
    if (stall) __builtin_amdgcn_s_sleep(1);
  }
  return sum;
}

// The k-th data-moving LSD pass (kK), over the digit the sort plan names:
// digits are w bits wide (8 or 9, chosen on the device from the live key
// width), thread t owning bin t.  A tile of kTile = kItems * kSortBlock keys
// is ranked per wave with w ballots; the tile's digit counts are published for the
// decoupled look-back; keys are reordered in LDS and written out in runs of
// equal digits.  The last pass writes the sorted order with each request's
// scan record (gathered while the tile is ranked) instead of
// the keys, adds every scan tile's level-1 totals and, with shared prefixes,
// marks each prefix group's leader position.  The k-th pass reads
// buffer k & 1, so the tile's keys are requested at once, in parallel with
// the plan.  Workgroup b sorts tile b: workgroups are dispatched in index
// order (on each XCD), so every tile a look-back waits on belongs to a
// workgroup that is running or done, and the lowest unfinished one waits on
// nothing.
template <int kK, int kItems>
__global__ __launch_bounds__(kSortBlock) void radix_pass_kernel(
    int n, int passes, Ctl *ctl, int *info, unsigned long long *keys_a,
    unsigned long long *keys_b, unsigned *vals_a, unsigned *vals_b, unsigned *status,
    const int4 *__restrict__ rec, Sorted srt, unsigned *__restrict__ l1_tot,
    unsigned *share_lead) {
  constexpr int kTile = kSortBlock * kItems;  // keys per tile
  __shared__ unsigned long long s_keys[kTile];
  __shared__ unsigned s_vals[kTile];
  __shared__ int4 s_rec[kTile];
  __shared__ unsigned s_wcnt[kSortWaves][kMaxBins];  // per-wave counts, then starts
  __shared__ int s_start[kMaxBins];  // tile-local start of each digit
  __shared__ int s_off[kMaxBins];    // output offset of each digit
  __shared__ int s_scan[kSortWaves * 2];
  __shared__ unsigned s_sum[kSortWaves * kL1];
  __shared__ unsigned s_l1[kMaxScanTiles * kL1];  // last pass: level-1 totals per scan tile
  __shared__ int s_bad;
  __shared__ unsigned s_mask;
  __shared__ unsigned s_px[kSortBlock / 2];  // paired look-back: the second window's sum,
  __shared__ int s_pc[kSortBlock / 2];       // how it ended,
  __shared__ int s_pn[kSortBlock / 2];       // and where the pair reads next
  static_assert(kMaxBins == kSortBlock, "one bin per thread");

  const unsigned long long *src_k = (kK & 1) ? keys_b : keys_a;
  unsigned long long *dst_k = (kK & 1) ? keys_a : keys_b;
  const unsigned *src_v = (kK & 1) ? vals_b : vals_a;
  unsigned *dst_v = (kK & 1) ? vals_a : vals_b;
  const int t = threadIdx.x, lane = lane_id(), wave = wave_id();
  const int local = wave * 64 * kItems + lane;

  unsigned long long key[kItems];
  unsigned val[kItems];
  int dig[kItems], rank[kItems];
  {
    const int g0 = (int)blockIdx.x * kTile + local;
#pragma unroll
    for (int j = 0; j < kItems; ++j) {
      const int g = g0 + j * 64;
      key[j] = g < n ? src_k[g] : 0ull;
      val[j] = g < n ? src_v[g] : 0u;
    }
  }
  // every digit's count of bin t (the plan, and this pass's bucket base)
  unsigned hv[kMaxPasses];
#pragma unroll
  for (int d = 0; d < kMaxPasses; ++d) hv[d] = ctl->hist[d][t];
  if (t == 0) {
    s_bad = bad_status(load_agent(info));
    s_mask = 0;
  }
  const DigitPlan P = digit_plan(ctl, passes);
  const unsigned bins = P.bins;
  const bool dt = t < (int)bins;
#pragma unroll
  for (int w = 0; w < kSortWaves; ++w) s_wcnt[w][t] = 0;
  // the plan: digits that move data (below the key width, not constant)
  {
    unsigned constant = 0;
#pragma unroll
    for (int d = 0; d < kMaxPasses; ++d) constant |= (hv[d] == (unsigned)n ? 1u : 0u) << d;
    if (constant) atomicOr(&s_mask, constant);
  }
  __syncthreads();
  const unsigned active = ((1u << P.nd) - 1u) & ~s_mask;
  const int nact = __builtin_popcount(active);
  if (kK == 0 && blockIdx.x == 0 && t == 0) store_agent(&ctl->nact, (unsigned)nact);
  if (s_bad) {
    // a failed step: "nothing before me" in every bin, so no later tile of
    // this pass waits on this one
    if (nact > kK)
      publish<unsigned>(status + (size_t)blockIdx.x * kMaxBins + t, 0u, kFlagInclusive);
    return;
  }
  if (kK == 0 && nact == 0) {
    // every key equal: the order is the identity; this sort tile adds its
    // positions to their scan tiles' level-1 totals (a scan tile may span
    // several sort tiles)
    constexpr int kSub = kTile < kScanTile ? kTile : kScanTile;
    static_assert(kTile % kSub == 0 && kScanTile % kSub == 0, "sub-ranges inside one scan tile");
    for (int q = 0; q < kTile / kSub; ++q) {
      const int p0 = (int)blockIdx.x * kTile + q * kSub;
      if (p0 >= n) break;
      unsigned c[kL1] = {0, 0, 0, 0, 0};
      for (int p = p0 + t; p < min(n, p0 + kSub); p += kSortBlock) {
        const int4 r = rec[p];
        share_mark(share_lead, r, p, n);
        const bool rp = rec_state(r.w) == CASCADE_RUNNING_PREFILL;
        const unsigned h = rp ? (unsigned)rec_held(r.w) : 0u;
        c[0] += (unsigned)rec_want(r);
        c[1] += (unsigned)r.y;
        c[2] += h;
        c[3] += rec_offl(r.w) ? h : 0u;
        c[4] += rp ? 1u : 0u;
      }
      block_sum<kL1, unsigned, kSortWaves>(c, s_sum);
      if (t == 0) {
#pragma unroll
        for (int k = 0; k < kL1; ++k)
          if (c[k]) atomicAdd(l1_tot + (size_t)(p0 / kScanTile) * kL1 + k, c[k]);
      }
    }
    return;
  }
  if (nact <= kK) return;
  const bool last = nact == kK + 1;
  // this pass sorts by the kK-th data-moving digit
  unsigned rest = active;
#pragma unroll
  for (int k = 0; k < kK; ++k) rest &= rest - 1;
  const int digit = __builtin_ctz(rest);
  unsigned gcount = 0;
#pragma unroll
  for (int d = 0; d < kMaxPasses; ++d) gcount = d == digit ? hv[d] : gcount;
  const int tile = (int)blockIdx.x;
  const int tile_base = tile * kTile;
  const int shift = P.w * digit;
  const unsigned dmask = bins - 1;
  bool broken = false;
#pragma unroll
  for (int j = 0; j < kItems; ++j)
    dig[j] = (tile_base + local + j * 64 < n) ? (int)((key[j] >> shift) & dmask) : -1;
  // the last pass carries each request's scan record along; the loads are
  // unconditional (index 0 when not needed) so that nothing waits for them
  // before the tile is ranked
  int rx[kItems], ry[kItems], rz[kItems], rv[kItems];
#pragma unroll
  for (int j = 0; j < kItems; ++j) {
    const bool want = last && dig[j] >= 0;
    broken |= want && val[j] >= (unsigned)n;
    const unsigned gi = (want && val[j] < (unsigned)n) ? val[j] : 0u;
    const int4 r = rec[gi];
    rx[j] = r.x;
    ry[j] = r.y;
    rz[j] = r.z;
    rv[j] = r.w;
  }
  // rank within the wave, item by item (local order: wave, item, lane)
#pragma unroll
  for (int j = 0; j < kItems; ++j) {
    const bool v = dig[j] >= 0;
    uint64_t peers = __ballot(v);
#pragma unroll
    for (int b = 0; b < kMaxW; ++b) {
      if (b < P.w) {
        const bool bit = (dig[j] >> b) & 1;
        const uint64_t bal = __ballot(bit);
        peers &= bit ? bal : ~bal;
      }
    }
    const int d = v ? dig[j] : 0;
    unsigned before = 0;
    if (v) before = s_wcnt[wave][d];
    __builtin_amdgcn_wave_barrier();
    const int below = rank_in_mask(peers);
    if (v && below == 0) s_wcnt[wave][d] = before + (unsigned)__builtin_popcountll(peers);
    __builtin_amdgcn_wave_barrier();
    rank[j] = (int)before + below;
  }
  __syncthreads();

  // earlier waves' counts of digit t; the tile's count is published at once
  unsigned *st = status + (size_t)tile * kMaxBins;
  unsigned tcount = 0;
  if (dt) {
#pragma unroll
    for (int w = 0; w < kSortWaves; ++w) {
      const unsigned c = s_wcnt[w][t];
      s_wcnt[w][t] = tcount;
      tcount += c;
    }
    publish<unsigned>(st + t, tcount, tile == 0 ? kFlagInclusive : kFlagAggregate);
  }
  if (last) {
    for (int k = t; k < kMaxScanTiles * kL1; k += kSortBlock) s_l1[k] = 0;
  }
  // tile-local starts and global bucket bases, in digit order
  int v2[2] = {(int)tcount, dt ? (int)gcount : 0}, tot2[2];
  block_exclusive_scan<2, int, kSortWaves>(v2, tot2, s_scan);
  if (dt) s_start[t] = v2[0];
  __syncthreads();
  // reorder the tile in LDS by digit: this needs only the tile-local
  // starts, so it runs before the look-back, whose first read then finds
  // more of the other tiles' counts already published
#pragma unroll
  for (int j = 0; j < kItems; ++j) {
    const bool v = dig[j] >= 0;
    const int d = v ? dig[j] : 0;
    const int pos = s_start[d] + (int)s_wcnt[wave][d] + rank[j];
    const bool ok = v && (unsigned)pos < (unsigned)kTile;
    broken |= v && !ok;
    if (ok) {
      s_keys[pos] = key[j];
      s_vals[pos] = val[j];
    }
    if (ok && last) s_rec[pos] = make_int4(rx[j], ry[j], rz[j], rv[j]);
  }
  // the earlier tiles' counts, kSortWin predecessors per round trip; with
  // 8-bit digits and more tiles than one window reaches, two threads share
  // a bin and read two windows
  bool timed_out = false;
  unsigned pre = 0;
  if (bins * 2 <= kSortBlock && (int)gridDim.x > kSortWin + 1) {
    pre = paired_look_back(status, tile, bins, s_px, s_pc, s_pn, &timed_out);
  } else if (dt && tile > 0) {
    pre = look_back<unsigned, kSortWin>(status, kMaxBins, tile, t, &timed_out);
  }
  if (dt) {
    if (tile > 0) publish<unsigned>(st + t, pre + tcount, kFlagInclusive);
    s_off[t] = v2[1] + (int)pre - v2[0];
  }
  if (timed_out) set_status(info, CASCADE_ETIMEOUT);
  __syncthreads();
  const int count = min(kTile, n - tile_base);
  static_assert(kTile % kSortBlock == 0, "every lane runs every iteration (wave sums below)");
  for (int s = t; s < kTile; s += kSortBlock) {
    int o = -1;
    unsigned long long k = 0;
    if (s < count) {
      k = s_keys[s];
      o = s_off[(k >> shift) & dmask] + s;
      if ((unsigned)o >= (unsigned)n) {
        broken = true;
        o = -1;
      }
    }
    if (last) {
      int4 r = make_int4(0, 0, 0, 0);
      if (o >= 0) {
        r = s_rec[s];
        srt.order[o] = s_vals[s];
        srt.rec[o] = r;
        share_mark(share_lead, r, o, n);
      }
      l1_contrib(s_l1, o >= 0 ? o / kScanTile : -1, r);
    } else if (o >= 0) {
      dst_k[o] = k;
      dst_v[o] = s_vals[s];
    }
  }
  if (broken) set_status(info, CASCADE_EINTERNAL);
  if (last) {
    __syncthreads();
    const int n_tot = ((n + kScanTile - 1) / kScanTile) * kL1;
    for (int k = t; k < n_tot; k += kSortBlock) {
      const unsigned v = s_l1[k];
      if (v) atomicAdd(l1_tot + k, v);
    }
  }
}

// ---------------------------------------------------------------- scan

// The victims, slot list and move lists, computed by the last scan workgroup
// once every tile's totals and per-holder prefixes are in memory.
// Budget-aware preemption (Algorithm 1; Section 4.4): the deficit
// D = new blocks of admitted requests - free blocks is covered by the
// non-admitted running prefills taken from the back of the order (largest
// remaining budget first): a holder at position p is preempted iff the
// eligible blocks behind it are fewer than D.
constexpr int kFreeCap = 4096;    // free-list entries staged in LDS by the finishing workgroup
constexpr int kTailCap = 2048;    // victims' slot-list entries kept in LDS for the restores
constexpr int kRowBatch = 8;      // victims' row entries each thread requests at once
static_assert(kVictimCap == kBlock, "one staged victim per thread in the row-offset scan");

struct FinishLds {
  long long tot[kWaves * 6];
  int v_req[kVictimCap], v_held[kVictimCap], v_row0[kVictimCap], v_start[kVictimCap];
  int v_offl[kVictimCap];
  long long v_sbase[kVictimCap], v_pbase[kVictimCap];
  alignas(16) RestoreEnt rl[kRestoreCap];  // stored as int4
  int free_slots[kFreeCap];
  int tail[kTailCap];  // slot-list entries n_free + i: the victims' slots
  int scan_tmp[kWaves];
  int n_victims, counts[2];
};

// Last index i < n with key(i) <= x (index 0 when none), in a fixed number of
// branch-free steps, so that a thread's independent searches overlap their
// LDS latencies.  n <= 2^kSteps.
template <int kSteps, typename KeyAt>
__device__ __forceinline__ int last_at_or_below(int n, long long x, KeyAt key) {
  int lo = 0;
#pragma unroll
  for (int step = 1 << (kSteps - 1); step > 0; step >>= 1) {
    const int mid = lo + step;
    lo = (mid < n && (long long)key(mid) <= x) ? mid : lo;
  }
  return lo;
}
constexpr int kRestoreSteps = 10;
static_assert((1 << kRestoreSteps) == kRestoreCap, "restore searches cover the LDS copy");

// Restore entry k, staged in LDS for k < kRestoreCap.
__device__ __forceinline__ RestoreEnt restore_entry(const FinishLds &L, const RestoreEnt *rl,
                                                    int k) {
  return k < kRestoreCap ? L.rl[k] : load_agent_rec(rl + k);
}

// The unpack move that writes slot-list entry s, or -1, for a restore list
// that fits its LDS copy (nr <= kRestoreCap).
__device__ __forceinline__ int unpack_move_at_lds(long long s, int nr, const FinishLds &L) {
  if (nr <= 0 || L.rl[0].alloc_off > s) return -1;
  const int lo = last_at_or_below<kRestoreSteps>(nr, s, [&](int k) { return L.rl[k].alloc_off; });
  const RestoreEnt e = L.rl[lo];
  return s < (long long)e.alloc_off + e.blocks ? e.stage_off + (int)(s - e.alloc_off) : -1;
}

// The unpack move that writes slot-list entry s, or -1: restore entries are
// in admitted order, so their allocation offsets increase and the entry that
// covers s is the last one starting at or before it.
__device__ __forceinline__ int unpack_move_at(long long s, int nr, const FinishLds &L,
                                              const RestoreEnt *rl) {
  if (nr <= 0 || restore_entry(L, rl, 0).alloc_off > s) return -1;
  int lo = 0, hi = nr - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (restore_entry(L, rl, mid).alloc_off <= s) lo = mid; else hi = mid - 1;
  }
  const RestoreEnt e = restore_entry(L, rl, lo);
  return s < (long long)e.alloc_off + e.blocks ? e.stage_off + (int)(s - e.alloc_off) : -1;
}

// Block b of a victim: its slot-list entry sb (and the LDS copy of it), its
// pack move pb + b when the victim spills (pb >= 0), and the copy-order
// hazard between that pack move and the restore that receives the slot.
// Every restore into a victim's slot gets its hazard entry here (-1 when
// the victim is dropped); restores into free slots get theirs later, so no
// hazard entry is written twice.
// kInTail: the entry lies in the LDS copy of the victims' region and the
// restore list fits its LDS copy, so nothing is read from memory (a read
// from memory would first wait for every store issued before it).
template <bool kInTail>
__device__ __forceinline__ void place_victim_block_at(int req, int b, int slot, long long sb,
                                                      long long pb, int n_free, int nr,
                                                      const Outs &o, FinishLds &L,
                                                      const RestoreEnt *rl) {
  if (sb < o.sl_cap) o.slot_list[sb] = slot;
  if (kInTail) L.tail[sb - n_free] = slot;
  const long long j = pb >= 0 ? pb + b : -1;
  const bool packed = j >= 0 && j < o.pack_cap;
  if (packed) {
    cascade_move_t mv;
    mv.req = req;
    mv.blk = b;
    mv.pool_slot = slot;
    mv.staging_slot = (int)j;
    o.pack[j] = mv;
  }
  if (o.pack_hazard) {
    const int m = kInTail ? unpack_move_at_lds(sb, nr, L) : unpack_move_at(sb, nr, L, rl);
    if (packed) o.pack_hazard[j] = m;
    if (m >= 0 && m < o.unpack_cap) o.unpack_hazard[m] = packed ? (int)j : -1;
  }
}
__device__ __forceinline__ void place_victim_block(int req, int b, int slot, long long sb,
                                                   long long pb, int n_free, int nr,
                                                   const Outs &o, FinishLds &L,
                                                   const RestoreEnt *rl) {
  if (sb - n_free < kTailCap && nr <= kRestoreCap)
    place_victim_block_at<true>(req, b, slot, sb, pb, n_free, nr, o, L, rl);
  else
    place_victim_block_at<false>(req, b, slot, sb, pb, n_free, nr, o, L, rl);
}

// Unpack move m of restore entry e; kLds: the pool slot it receives is in
// the LDS copies of the free list and the victims' region.
template <bool kLds>
__device__ __forceinline__ void emit_restore_move(long long m, const RestoreEnt &e, int n_free,
                                                  const int *__restrict__ free_slots,
                                                  const Outs &o, const FinishLds &L) {
  const int b = (int)(m - e.stage_off);
  const long long s = (long long)e.alloc_off + b;
  cascade_move_t mv;
  mv.req = e.req;
  mv.blk = b;
  int ps;
  if (s >= o.sl_cap) ps = -1;
  else if (kLds) ps = s < n_free ? L.free_slots[s] : L.tail[s - n_free];
  else if (s < n_free) ps = s < kFreeCap ? L.free_slots[s] : free_slots[s];
  else ps = s - n_free < kTailCap ? L.tail[s - n_free] : o.slot_list[s];
  mv.pool_slot = ps;
  mv.staging_slot = (int)m;
  o.unpack[m] = mv;
  // a free slot is read by no pack move (victims' slots got theirs above)
  if (o.unpack_hazard && s < n_free) o.unpack_hazard[m] = -1;
}

// Request the victims' row entries m = m0 + u*kBlock (u < kRowBatch): the
// owning victim (search of the staged victims' row starts), block and slot.
__device__ __forceinline__ void request_rows(int m0, int v_total, int nv,
                                             const int *__restrict__ slots, const FinishLds &L,
                                             int (&slot)[kRowBatch], int (&vi)[kRowBatch],
                                             int (&bi)[kRowBatch]) {
#pragma unroll
  for (int u = 0; u < kRowBatch; ++u) {
    const int m = m0 + u * kBlock;
    vi[u] = -1;
    if (m < v_total) {
      const int lo = last_at_or_below<8>(nv, m, [&](int k) { return L.v_start[k]; });
      vi[u] = lo;
      bi[u] = m - L.v_start[lo];
      slot[u] = slots[L.v_row0[lo] + bi[u]];
    }
  }
}

// Loads are grouped so that the workgroup waits on memory twice in the
// common case: the totals, running-prefill records, restore list and free
// list together (each thread's share requested before any is stored), then
// the victims' rows, up to kRowBatch per thread at once.
__device__ __forceinline__ void finish_step(const Ctl *ctl, int *info, int n, int n_free,
                                            int n_tiles, int n_rp,
                            const TileTot *__restrict__ tiles, const int *__restrict__ free_slots,
                            const RpInfo *__restrict__ rp, const RestoreEnt *__restrict__ rl,
                            const int *__restrict__ slots, const Outs &o, FinishLds &L) {
  const int t = threadIdx.x;
  if (t == 0) {
    L.n_victims = 0;
    L.counts[0] = L.counts[1] = 0;
  }
  // every list the finish reads is requested at once: the free list and a
  // bounded prefix of the restore list (tot[5] entries, not known yet, in a
  // buffer of n), the tile totals, k* and the last kBlock running prefills
  constexpr int kFreePer = kFreeCap / kBlock, kRestPer = kRestoreCap / kBlock;
  const int n_fs = min(n_free, kFreeCap), n_rs = min(n, kRestoreCap);
  int fv[kFreePer];
  RestoreEnt rv[kRestPer];
#pragma unroll
  for (int u = 0; u < kFreePer; ++u) {
    const int j = t + u * kBlock;
    fv[u] = j < n_fs ? free_slots[j] : 0;
  }
#pragma unroll
  for (int u = 0; u < kRestPer; ++u) {
    const int j = t + u * kBlock;
    rv[u] = j < n_rs ? load_agent_rec(rl + j) : RestoreEnt{0, 0, 0, 0};
  }
  long long tot[6] = {0, 0, 0, 0, 0, 0};
  for (int j = t; j < n_tiles; j += kBlock) {
    const TileTot tt = load_agent_rec(tiles + j);
    tot[0] += tt.adm_nb;
    tot[1] += tt.elig_h;
    tot[2] += tt.elig_offl_h;
    tot[3] += tt.n_adm;
    tot[4] += tt.n_unpack;
    tot[5] += tt.n_restore;
  }
  const int kstar = load_agent(&ctl->kstar);
  const long long kx = load_agent(&ctl->kx), ky = load_agent(&ctl->ky),
                  kz = load_agent(&ctl->kz), kzp = load_agent(&ctl->kzp);
  // running prefills from the back of the order (the list is stored that
  // way): thread t holds entry back + t
  int back = 0;
  RpInfo ri = {};
  if (t < n_rp) ri = load_agent_rec(rp + t);
  const int lim = min(n_free, o.sl_cap);
#pragma unroll
  for (int u = 0; u < kFreePer; ++u) {
    const int j = t + u * kBlock;
    if (j < n_fs) L.free_slots[j] = fv[u];
  }
#pragma unroll
  for (int u = 0; u < kRestPer; ++u) {
    const int j = t + u * kBlock;
    if (j < n_rs) L.rl[j] = rv[u];
  }
  block_sum<6>(tot, L.tot);  // waits for the loads above
  const long long D = tot[0] - n_free, E = tot[1], EO = tot[2];
  const long long nu = tot[4];
  const int nr = (int)tot[5];

  // victims: the eligible holders whose eligible blocks behind them are
  // fewer than D.  That count only grows towards the front of the order, so
  // they are the last ones: windows of kBlock entries are taken from the
  // back until one holds an eligible entry that is not a victim.
  while (D > 0 && back < n_rp) {
    const int e = back + t;
    if (back != 0 && e < n_rp) ri = load_agent_rec(rp + e);
    bool kept = false;
    do {
      if (e >= n_rp || !ri.eligible) break;
      const long long eh = ri.pos < kstar ? ri.x : kx + ri.y - ky;
      const long long after = E - eh;  // eligible blocks behind this request
      if (after >= D) {
        kept = true;
        break;
      }
      if (after < 0) {
        set_status(info, CASCADE_EINTERNAL);
        break;
      }
      const int i = ri.req, h = ri.held;
      atomicAdd(&L.counts[0], h);
      if (ri.offl) atomicAdd(&L.counts[1], h);
      const long long sbase = (long long)n_free + after;
      const long long pbase = ri.offl ? EO - (ri.pos < kstar ? ri.z : kz + ri.zp - kzp) : -1;
      const int v = atomicAdd(&L.n_victims, 1);
      if (v < kVictimCap) {
        L.v_req[v] = i;
        L.v_offl[v] = ri.offl;
        L.v_held[v] = h;
        L.v_row0[v] = ri.row0;
        L.v_sbase[v] = sbase;
        L.v_pbase[v] = pbase;
      } else {  // more victims than LDS holds: place this one alone
        store_agent(&o.action[i], (uint8_t)(ri.offl ? CASCADE_ACT_PREEMPT_OFFLOAD
                                                    : CASCADE_ACT_PREEMPT_DROP));
        for (int b = 0; b < h; ++b)
          place_victim_block(i, b, slots[ri.row0 + b], sbase + b, pbase, n_free, nr, o, L, rl);
      }
    } while (false);
    if (__syncthreads_or(kept ? 1 : 0)) break;  // every earlier holder is kept too
    back += kBlock;
  }
  __syncthreads();
  // the staged victims' rows as one flat index space (prefix of row lengths),
  // so every row load of every victim is in flight at once
  const int nv = min(L.n_victims, kVictimCap);
  int v_total;
  {
    int hv[1] = {t < nv ? L.v_held[t] : 0}, tot1[1];
    block_exclusive_scan<1>(hv, tot1, L.scan_tmp);  // kVictimCap == kBlock
    if (t < nv) L.v_start[t] = hv[0];
    v_total = tot1[0];
  }
  __syncthreads();
  int slot[kRowBatch], vi[kRowBatch], bi[kRowBatch];
  request_rows(t, v_total, nv, slots, L, slot, vi, bi);
  for (int m0 = t;;) {
#pragma unroll
    for (int u = 0; u < kRowBatch; ++u) {
      if (vi[u] < 0) continue;
      const int v = vi[u];
      place_victim_block(L.v_req[v], bi[u], slot[u], L.v_sbase[v] + bi[u], L.v_pbase[v], n_free,
                         nr, o, L, rl);
    }
    m0 += kRowBatch * kBlock;
    if (m0 >= v_total) break;
    request_rows(m0, v_total, nv, slots, L, slot, vi, bi);
  }
  // stores that waited for every load above: the staged victims' actions
  // (replacing the RETAIN their scan tiles stored before their tickets) and
  // the free-list part of the slot list
  if (t < nv)
    store_agent(&o.action[L.v_req[t]], (uint8_t)(L.v_offl[t] ? CASCADE_ACT_PREEMPT_OFFLOAD
                                                             : CASCADE_ACT_PREEMPT_DROP));
  for (int j = t; j < lim; j += kBlock)
    o.slot_list[j] = j < kFreeCap ? L.free_slots[j] : free_slots[j];
  __syncthreads();  // the slot list is complete (this workgroup wrote it)
  // restore moves: the first r new blocks of each RESTORE request, staged in
  // admitted order; move m finds its request by a search of the staged list
  const long long mlim = lmin(nu, (long long)o.unpack_cap);
  for (long long m = t; m < mlim; m += kBlock) {
    if (nr <= kRestoreCap) {
      const int lo =
          last_at_or_below<kRestoreSteps>(nr, m, [&](int k) { return L.rl[k].stage_off; });
      const RestoreEnt e = L.rl[lo];
      const long long s = (long long)e.alloc_off + (m - e.stage_off);
      if (s < min(n_free, kFreeCap) || (s >= n_free && s - n_free < kTailCap)) {
        emit_restore_move<true>(m, e, n_free, free_slots, o, L);
        continue;
      }
    }
    int lo = 0, hi = nr - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      const int off = restore_entry(L, rl, mid).stage_off;
      if (off <= m) lo = mid; else hi = mid - 1;
    }
    emit_restore_move<false>(m, restore_entry(L, rl, lo), n_free, free_slots, o, L);
  }
  if (t == 0) {
    const long long nsl = (long long)n_free + L.counts[0];
    info[CASCADE_INFO_N_ADMITTED] = (int)tot[3];
    info[CASCADE_INFO_N_SLOT_LIST] = (int)nsl;
    info[CASCADE_INFO_N_UNPACK] = (int)nu;
    info[CASCADE_INFO_N_PACK] = L.counts[1];
    const bool full = nsl > o.sl_cap || nu > o.unpack_cap || L.counts[1] > o.pack_cap;
    if (full && load_agent(info) == CASCADE_OK) set_status(info, CASCADE_ENOSPC);
  }
}

// Algorithm 1's Phase 2 over the kScanTile positions of one tile, given
// each position's request index (idx < 0: past the end), record and block-
// table row offset (gathered with the record by the caller); thread
// t holds positions t*jn .. t*jn + jn - 1 of the tile (jn <= kScanItems).  With
// kChained the tile's level-1 and level-2 prefixes pre1 and pre2 are the
// earlier tiles' totals; without, the tile is the whole queue (both zero).
// Writes what the finishing workgroup reads (k*, the running-prefill and
// restore-list entries, the running prefills' actions and the tile's totals)
// with agent-scope stores, and leaves every other per-request output in `out`
// for write_tile_outputs; returns the number of running prefills up to and
// including this tile.
struct ScanLds {
  long long scan[kWaves * kL2];
  long long red[kWaves * (kL1 + kL2 + 1)];  // earlier tiles' totals and the status flag
  long long pre2[kL2];                      // the earlier tiles' level-2 totals (look-back)
};

// Per-request outputs of one thread's positions, stored after the hand-over.
struct TileOut {
  int req[kScanItems];      // request index, -1: no position
  int granted[kScanItems], restore[kScanItems], alloc_begin[kScanItems], alloc_count[kScanItems];
  int admitted_at[kScanItems];  // index in the admitted list, -1: not admitted
  int action[kScanItems];       // -1: a running prefill (stored before the hand-over)
  int share[kScanItems];        // share_leader output
  int p0;
};

__device__ __forceinline__ void write_tile_outputs(const TileOut &out, const Outs &o) {
#pragma unroll
  for (int j = 0; j < kScanItems; ++j) {
    const int i = out.req[j];
    if (i < 0) continue;
    o.order[out.p0 + j] = i;
    o.granted[i] = out.granted[j];
    o.restore[i] = out.restore[j];
    o.alloc_begin[i] = out.alloc_begin[j];
    o.alloc_count[i] = out.alloc_count[j];
    if (out.action[j] >= 0) o.action[i] = (uint8_t)out.action[j];
    if (out.admitted_at[j] >= 0) o.admitted[out.admitted_at[j]] = i;
    if (o.share_leader) o.share_leader[i] = out.share[j];
  }
}

struct ScanConsts {
  long long bt, U, e1, cap, cap1, p_e1, g1, fh;
};

__device__ __forceinline__ ScanConsts scan_consts(const Consts &c, const Ctl *ctl) {
  ScanConsts k;
  k.bt = c.bt;
  k.U = c.max_move;
  k.e1 = (long long)ctl->cnt[0] + ctl->cnt[1];
  const bool has2 = ctl->cnt[2] != 0;
  k.cap = c.token_cap;
  k.cap1 = k.cap - (has2 ? ((k.cap * c.rho_q16) >> 16) : 0);
  // tokens before Tier-2 (followers want nothing and need less)
  k.p_e1 = (ctl->need1 - ctl->need1_sub) - k.bt * lmin(ctl->want1 - ctl->want1_sub, k.U);
  k.g1 = lmin(k.p_e1, k.cap1);                          // granted to decode+Tier-1
  k.fh = (long long)c.n_free + ctl->held_rp;            // F + H
  return k;
}

// Level-1 scan of one tile and every position's restore blocks, grant, new
// blocks and level-2 values (this thread's partial sums in v.l2), given the
// tile's level-1 prefix pre1.
struct PosVals {
  int r[kScanItems], g[kScanItems], nb[kScanItems], hh[kScanItems];
  long long y_inc[kScanItems], zp_inc[kScanItems];
  long long l2[kL2];
  long long rp_incl;  // running prefills up to and including this tile
  int rp_at;          // compact-list index of this thread's first running prefill
};

__device__ __forceinline__ void scan_positions(int tile, int jn, const ScanConsts &K,
                                               const int (&idx)[kScanItems],
                                               const int4 (&r4)[kScanItems],
                                               const long long (&pre1)[kL1], ScanLds &S,
                                               PosVals &v) {
  const long long bt = K.bt, U = K.U, e1 = K.e1, cap = K.cap, cap1 = K.cap1, p_e1 = K.p_e1,
                  g1 = K.g1;
  const int p0 = tile * kScanTile + threadIdx.x * jn;  // items j < jn; the rest absent
  // ---- level 1, scanned in 32 bits within the tile: per request the want
  // and the need are below 2^18 and the held blocks below 2^20, so a tile of
  // kScanTile requests sums to less than 2^31
  unsigned l1[kL1] = {0, 0, 0, 0, 0}, t1[kL1];
#pragma unroll
  for (int j = 0; j < kScanItems; ++j) {
    const int w = r4[j].w;
    const bool rp = idx[j] >= 0 && rec_state(w) == CASCADE_RUNNING_PREFILL;
    const unsigned h = rp ? (unsigned)rec_held(w) : 0u;
    l1[0] += (unsigned)rec_want(r4[j]);
    l1[1] += (unsigned)r4[j].y;
    l1[2] += h;
    l1[3] += rec_offl(w) ? h : 0u;
    l1[4] += rp ? 1u : 0u;        // running prefills (their compact list)
  }
  block_exclusive_scan<kL1>(l1, t1, reinterpret_cast<unsigned *>(S.scan));
  long long wx = pre1[0] + l1[0], bn = pre1[1] + l1[1], yy = pre1[2] + l1[2],
            zz = pre1[3] + l1[3];
  v.rp_at = (int)(pre1[4] + l1[4]);
  v.rp_incl = pre1[4] + t1[4];

  // ---- per position: restore blocks, need, grant, new blocks
  // per item: restore blocks (<= want), grant (<= token cap), new blocks and
  // held blocks (< 2^20) all fit 32 bits; prefix sums stay 64-bit
#pragma unroll
  for (int k = 0; k < kL2; ++k) v.l2[k] = 0;
#pragma unroll
  for (int j = 0; j < kScanItems; ++j) {
    const int w = r4[j].w;
    const int st = rec_state(w);
    const long long want = rec_want(r4[j]);
    const long long rj = lmin(wx + want, U) - lmin(wx, U);
    const long long need = (long long)r4[j].y - bt * rj;
    const long long P = bn - bt * lmin(wx, U);  // tokens needed before p
    const long long p = p0 + j;
    long long gj;
    if (p < e1) {
      gj = lmin(P + need, cap1) - lmin(P, cap1);
    } else {
      const long long q = g1 + (P - p_e1);
      gj = lmin(q + need, cap) - lmin(q, cap);
    }
    if (idx[j] < 0) gj = 0;
    long long nbj = 0;
    const long long h = st == CASCADE_RUNNING_PREFILL ? rec_held(w) : 0;
    if (gj > 0) {
      const unsigned ubt = (unsigned)bt;
      if (st == CASCADE_QUEUED) {
        if (rec_tier(w) == CASCADE_KV_HBM) {
          const unsigned s = (unsigned)r4[j].z;
          nbj = (long long)udiv_ceil(s + (unsigned)gj, ubt) - s / ubt;
        } else {
          nbj = rj + udiv_ceil((unsigned)gj, ubt);
        }
      } else if (st == CASCADE_RUNNING_PREFILL) {
        nbj = (long long)udiv_ceil((unsigned)r4[j].z + (unsigned)gj, ubt) - rec_held(w);
      } else {
        nbj = rec_decnb(w);
      }
    }
    v.r[j] = (int)rj;
    v.g[j] = (int)gj;
    v.nb[j] = (int)nbj;
    v.hh[j] = (int)h;
    wx += want;
    bn += r4[j].y;
    yy += h;
    zz += rec_offl(w) ? h : 0;
    v.y_inc[j] = yy;
    v.zp_inc[j] = zz;
    const bool gp = gj > 0;
    v.l2[0] += gp ? nbj + h : 0;              // admission weight
    v.l2[1] += gp ? nbj : 0;                  // new blocks
    v.l2[2] += gp ? 1 : 0;                    // admitted count
    v.l2[3] += gp ? 0 : h;                    // held, not granted
    v.l2[4] += (gp || !rec_offl(w)) ? 0 : h;  // held, not granted, spill fits
    v.l2[5] += gp ? rj : 0;                   // restored blocks
    v.l2[6] += (gp && rj > 0) ? 1 : 0;        // restoring requests
  }
}

// The earlier tiles' level-2 totals, by one wave: lane l reads tile
// next - l, so a round trip covers 64 predecessors.  Each of the kL2 values
// has its own flags and its own stopping point (the words of one tile are
// published separately): a ballot finds the first unpublished and the first
// inclusive word, and a wave sum adds the words before it.  Called by all 64
// lanes of one wave; the sums come back in every lane.
__device__ __forceinline__ void wave_look_back(const unsigned long long *status, int tile,
                                               unsigned long long (&pre)[kL2], bool *timed_out) {
  const int lane = lane_id();
  int next[kL2];
#pragma unroll
  for (int k = 0; k < kL2; ++k) next[k] = tile - 1;
  unsigned spins = 0;
  while (true) {
    bool pending = false;
#pragma unroll
    for (int k = 0; k < kL2; ++k) pending |= next[k] >= 0;
    if (!pending) return;
    unsigned long long w[kL2];
#pragma unroll
    for (int k = 0; k < kL2; ++k) {
      const int j = next[k] - lane;
      w[k] = j >= 0 ? load_agent(status + (size_t)j * kL2Stride + k)
                    : (unsigned long long)kFlagInclusive;
    }
    bool stalled = false;
#pragma unroll
    for (int k = 0; k < kL2; ++k) {
      if (next[k] < 0) continue;
      const unsigned f = (unsigned)(w[k] & 3);
      const uint64_t missing = __ballot(f == 0);
      const uint64_t inclusive = __ballot(f == kFlagInclusive);
      const int first_missing = missing ? __builtin_ctzll(missing) : 64;
      const int first_inclusive = inclusive ? __builtin_ctzll(inclusive) : 64;
      const bool done = first_inclusive < first_missing;
      const int take = done ? first_inclusive + 1 : first_missing;
      pre[k] += wave_sum(lane < take ? (w[k] >> 2) : 0ull);
      next[k] = done ? -1 : next[k] - take;
      stalled |= first_missing < 64 && !done;
    }
    if (stalled) {
      if (++spins > kSpinLimit) {
        *timed_out = true;
        return;
      }
      __builtin_amdgcn_s_sleep(1);
    }
  }
}

template <bool kChained>
__device__ __forceinline__ long long scan_tile(int tile, int jn, const ScanConsts &K, Ctl *ctl,
                                               int *info,
                               const int (&idx)[kScanItems], const int4 (&r4)[kScanItems],
                               bool broken, const Outs &o,
                               RpInfo *__restrict__ rp_list,
                               RestoreEnt *__restrict__ restore_list,
                               TileTot *__restrict__ tile_tot, const long long (&pre1)[kL1],
                               long long rp_total, unsigned long long *l2_status, ScanLds &S,
                               TileOut &out) {
  const long long fh = K.fh;
  const int p0 = tile * kScanTile + threadIdx.x * jn;
  PosVals v;
  scan_positions(tile, jn, K, idx, r4, pre1, S, v);
  int rp_at = v.rp_at;
  const long long rp_incl = v.rp_incl;
  // the running-prefill list is stored from the back of the order (entry 0:
  // the last one), so the finish reads its tail without knowing its length;
  // alone, the tile holds every running prefill
  const long long rp_last = (kChained ? rp_total : rp_incl) - 1;
  // level-2 values of a tile stay below 2^31 (per request: new blocks plus
  // held blocks below 2^21), so the tile is scanned in 32 bits
  unsigned l2[kL2], t2[kL2];
#pragma unroll
  for (int k = 0; k < kL2; ++k) l2[k] = (unsigned)v.l2[k];
  const int *r = v.r, *g = v.g, *nb = v.nb, *hh = v.hh;
  const long long *y_inc = v.y_inc, *zp_inc = v.zp_inc;

  // ---- level 2: the earlier tiles' totals plus this tile's.  Chained, the
  //      tile publishes its totals and takes the earlier tiles' from a
  //      decoupled look-back (thread k for value k); alone, they are zero.
  block_exclusive_scan<kL2>(l2, t2, reinterpret_cast<unsigned *>(S.scan));
  long long pre2[kL2] = {0, 0, 0, 0, 0, 0, 0};
  if (kChained) {
    const int t = threadIdx.x;
    if (t < 64) {
      unsigned agg = 0;
#pragma unroll
      for (int k = 0; k < kL2; ++k) agg = k == t ? t2[k] : agg;
      unsigned long long *st = l2_status + (size_t)tile * kL2Stride + t;
      if (t < kL2)
        publish<unsigned long long>(st, agg, tile == 0 ? kFlagInclusive : kFlagAggregate);
      unsigned long long before[kL2] = {0, 0, 0, 0, 0, 0, 0};
      if (tile > 0) {
        bool timed_out = false;
        wave_look_back(l2_status, tile, before, &timed_out);
        unsigned long long mine = 0;
#pragma unroll
        for (int k = 0; k < kL2; ++k) mine = k == t ? before[k] : mine;
        if (t < kL2) publish<unsigned long long>(st, mine + agg, kFlagInclusive);
        if (timed_out && t == 0) set_status(info, CASCADE_ETIMEOUT);
      }
      if (t == 0) {
#pragma unroll
        for (int k = 0; k < kL2; ++k) S.pre2[k] = (long long)before[k];
      }
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kL2; ++k) pre2[k] = S.pre2[k];
  }
  long long W = pre2[0] + l2[0], NB = pre2[1] + l2[1], AC = pre2[2] + l2[2],
            X = pre2[3] + l2[3], Z = pre2[4] + l2[4], RR = pre2[5] + l2[5],
            RC = pre2[6] + l2[6];

  long long a_nb = 0, a_eh = 0, a_eoh = 0, a_n = 0, a_r = 0, a_rc = 0;
  out.p0 = p0;
#pragma unroll
  for (int j = 0; j < kScanItems; ++j) {
    out.req[j] = idx[j];
    if (idx[j] < 0) continue;
    const int i = idx[j];
    const int p = p0 + j;
    const int w = r4[j].w;
    const int st = rec_state(w);
    const bool gp = g[j] > 0;
    const long long wj = gp ? nb[j] + hh[j] : 0;
    const bool adm = gp && (W + wj <= fh);
    if (W <= fh && W + wj > fh) {
      // the first request that does not fit: everything after it waits
      store_agent(&ctl->kstar, p);
      store_agent(&ctl->kx, X);
      store_agent(&ctl->ky, y_inc[j] - hh[j]);
      store_agent(&ctl->kz, Z);
      store_agent(&ctl->kzp, zp_inc[j] - (rec_offl(w) ? hh[j] : 0));
    }
    const bool follow = st == CASCADE_QUEUED && rec_follow(w);
    const int shared = follow ? (int)((unsigned)r4[j].z / (unsigned)K.bt) : 0;
    out.granted[j] = adm ? (int)g[j] : 0;
    out.restore[j] = follow ? shared : (int)r[j];
    out.share[j] = (follow && shared > 0) ? r4[j].x : -1;
    out.alloc_begin[j] = adm ? (int)NB : -1;
    out.alloc_count[j] = adm ? (int)nb[j] : 0;
    out.admitted_at[j] = adm ? (int)AC : -1;
    int act;
    if (st != CASCADE_QUEUED) {
      act = CASCADE_ACT_RETAIN;  // a preempted running prefill is rewritten later
    } else if (follow) {
      act = shared > 0 ? CASCADE_ACT_SHARE : CASCADE_ACT_RECOMPUTE;
    } else {
      const int tier = rec_tier(w);
      if (tier == CASCADE_KV_HBM) act = CASCADE_ACT_RETAIN;
      else if (tier == CASCADE_KV_NONE || r[j] == 0) act = CASCADE_ACT_RECOMPUTE;
      else act = adm ? CASCADE_ACT_RESTORE : CASCADE_ACT_PREFETCH;
    }
    if (st == CASCADE_RUNNING_PREFILL) {
      // the finishing workgroup rewrites a preempted one: store it now
      store_agent(&o.action[i], (uint8_t)act);
      out.action[j] = -1;
    } else {
      out.action[j] = act;
    }
    if (adm) {
      a_nb += nb[j];
      a_n += 1;
      if (r[j] > 0) {
        RestoreEnt e;
        e.req = i;
        e.stage_off = (int)RR;
        e.alloc_off = (int)NB;
        e.blocks = (int)r[j];
        store_agent_rec(restore_list + RC, e);
        a_r += r[j];
        a_rc += 1;
      }
    }
    const long long xj = gp ? 0 : hh[j];
    const long long zj = (gp || !rec_offl(w)) ? 0 : hh[j];
    if (st == CASCADE_RUNNING_PREFILL) {
      RpInfo ri;
      ri.req = i;
      ri.pos = p;
      ri.eligible = adm ? 0 : 1;
      ri.held = (int)hh[j];
      ri.row0 = r4[j].x;
      ri.offl = rec_offl(w);
      ri.pad[0] = ri.pad[1] = 0;
      ri.x = X + xj;
      ri.y = y_inc[j];
      ri.z = Z + zj;
      ri.zp = zp_inc[j];
      store_agent_rec(rp_list + (rp_last - rp_at), ri);
      ++rp_at;
      if (!adm) {
        a_eh += hh[j];
        a_eoh += rec_offl(w) ? hh[j] : 0;
      }
    }
    W += wj;
    NB += gp ? nb[j] : 0;
    AC += gp ? 1 : 0;
    X += xj;
    Z += zj;
    RR += gp ? r[j] : 0;
    RC += (gp && r[j] > 0) ? 1 : 0;
  }
  // a tile's totals stay below 2^31 (per request below 2^21), so 32-bit lanes
  unsigned tot[8] = {(unsigned)a_nb, (unsigned)a_eh, (unsigned)a_eoh, (unsigned)a_n,
                     (unsigned)a_r, (unsigned)a_rc, 0u, broken ? 1u : 0u};
  block_sum<8>(tot, reinterpret_cast<unsigned *>(S.red));
  if (threadIdx.x == 0) {
    TileTot tt;
    tt.adm_nb = tot[0];
    tt.elig_h = tot[1];
    tt.elig_offl_h = tot[2];
    tt.n_adm = tot[3];
    tt.n_unpack = tot[4];
    tt.n_restore = tot[5];
    tt.pad[0] = tt.pad[1] = 0;
    store_agent_rec(tile_tot + tile, tt);
    if (tot[7]) set_status(info, CASCADE_EINTERNAL);
  }
  return rp_incl;
}

// ---------------------------------------------------------------- finish

// The victims, slot list and move lists of a large queue, computed by
// kFinishGrid extra workgroups of the scan launch once every scan tile has
// handed over its results.  Every workgroup derives the same victims (the
// running prefills at the back of the order whose eligible blocks behind
// them are fewer than the deficit D, in a fixed order), then handles its
// slice of the outputs: the free part of the slot list, the victims' blocks
// (slot-list entries, pack moves, their copy-order hazards) and the restore
// moves (pool slot, hazard).  Each output entry has one owner, found by
// branch-free searches of the staged victims and restore list.  A queue whose
// victims or restore list outgrow the LDS copies is finished by workgroup 0
// alone with the sequential finish.
constexpr int kFinishGrid = 32;
constexpr int kFinVictims = 1024;   // victims staged by each finishing workgroup
constexpr int kFinVictimSteps = 10;
static_assert((1 << kFinVictimSteps) == kFinVictims, "victim searches cover the staged list");
constexpr int kFinItems = 4;        // output entries per thread and round

struct FinishKLds {
  long long red[kWaves * 8];
  int scan_tmp[kWaves];
  int v_req[kFinVictims], v_held[kFinVictims], v_row0[kFinVictims], v_start[kFinVictims];
  int v_offl[kFinVictims];
  long long v_sbase[kFinVictims], v_pbase[kFinVictims];
  alignas(16) RestoreEnt rl[kRestoreCap];
};
union FinishAnyLds {
  FinishKLds par;
  FinishLds seq;
};

// The unpack move that writes slot-list entry s (restore list in LDS), or -1.
__device__ __forceinline__ int fin_unpack_move_at(long long s, int nr, const FinishKLds &L) {
  if (nr <= 0 || L.rl[0].alloc_off > s) return -1;
  const int lo = last_at_or_below<kRestoreSteps>(nr, s, [&](int k) { return L.rl[k].alloc_off; });
  const RestoreEnt e = L.rl[lo];
  return s < (long long)e.alloc_off + e.blocks ? e.stage_off + (int)(s - e.alloc_off) : -1;
}

__device__ __forceinline__ void finish_grid(int g, int G, int n, int n_free, int n_tiles,
                                            Ctl *ctl, int *info,
                                            const TileTot *__restrict__ tiles,
                                            const int *__restrict__ free_slots,
                                            const RpInfo *__restrict__ rp,
                                            const RestoreEnt *__restrict__ rl,
                                            const int *__restrict__ slots, const Outs &o,
                                            FinishAnyLds &U) {
  FinishKLds &L = U.par;
  const int t = threadIdx.x;
  const int st = load_agent(info);
  const int n_rp = load_agent(&ctl->n_rp), kstar = load_agent(&ctl->kstar);
  const long long kx = load_agent(&ctl->kx), ky = load_agent(&ctl->ky),
                  kz = load_agent(&ctl->kz), kzp = load_agent(&ctl->kzp);
  // tile totals, the staged part of the restore list and the last kBlock
  // running prefills, all requested before any is used
  constexpr int kTilePer = 4, kRestPer = kRestoreCap / kBlock;
  long long tot[7] = {0, 0, 0, 0, 0, 0, 0};
  for (int j0 = 0; j0 < n_tiles; j0 += kTilePer * kBlock) {
    TileTot tt[kTilePer];
#pragma unroll
    for (int u = 0; u < kTilePer; ++u) {
      const int j = j0 + u * kBlock + t;
      tt[u] = j < n_tiles ? load_agent_rec(tiles + j) : TileTot{0, 0, 0, 0, 0, 0, {0, 0}};
    }
#pragma unroll
    for (int u = 0; u < kTilePer; ++u) {
      tot[0] += tt[u].adm_nb;
      tot[1] += tt[u].elig_h;
      tot[2] += tt[u].elig_offl_h;
      tot[3] += tt[u].n_adm;
      tot[4] += tt[u].n_unpack;
      tot[5] += tt[u].n_restore;
    }
  }
  const int n_rs = min(n, kRestoreCap);
  RestoreEnt rv[kRestPer];
#pragma unroll
  for (int u = 0; u < kRestPer; ++u) {
    const int j = t + u * kBlock;
    rv[u] = j < n_rs ? load_agent_rec(rl + j) : RestoreEnt{0, 0, 0, 0};
  }
  // the running-prefill list is stored from the back of the order, so its
  // last kBlock entries are requested before their count is known (a queue
  // on this path holds more than kBlock requests)
  int back = 0;
  RpInfo ri = load_agent_rec(rp + t);
#pragma unroll
  for (int u = 0; u < kRestPer; ++u) {
    const int j = t + u * kBlock;
    if (j < n_rs) L.rl[j] = rv[u];
  }
  tot[6] = (t == 0 && bad_status(st)) ? 1 : 0;
  block_sum<7>(tot, L.red);
  if (tot[6]) return;
  const long long D = tot[0] - n_free, E = tot[1], EO = tot[2];
  const long long nu = tot[4];
  const int nr = (int)tot[5];

  // victims, in order from the back of the queue
  int nv_all = 0;                // victims found (staged or not)
  long long held_all = 0, held_offl = 0;
  while (D > 0 && back < n_rp) {
    const int e = back + t;
    if (back != 0 && e < n_rp) ri = load_agent_rec(rp + e);
    bool victim = false, kept = false;
    long long after = 0;
    if (e < n_rp && ri.eligible) {
      const long long eh = ri.pos < kstar ? ri.x : kx + ri.y - ky;
      after = E - eh;  // eligible blocks behind this request
      if (after >= D) {
        kept = true;
      } else if (after < 0) {
        set_status(info, CASCADE_EINTERNAL);
      } else {
        victim = true;
      }
    }
    int vr[1] = {victim ? 1 : 0}, vt[1];
    block_exclusive_scan<1>(vr, vt, L.scan_tmp);
    const int v = nv_all + vr[0];
    if (victim && v < kFinVictims) {
      L.v_req[v] = ri.req;
      L.v_held[v] = ri.held;
      L.v_row0[v] = ri.row0;
      L.v_offl[v] = ri.offl;
      L.v_sbase[v] = (long long)n_free + after;
      L.v_pbase[v] = ri.offl ? EO - (ri.pos < kstar ? ri.z : kz + ri.zp - kzp) : -1;
    }
    long long hs[2] = {victim ? ri.held : 0, (victim && ri.offl) ? ri.held : 0};
    block_sum<2>(hs, L.red);
    held_all += hs[0];
    held_offl += hs[1];
    nv_all += vt[0];
    if (__syncthreads_or(kept ? 1 : 0)) break;  // every earlier holder is kept too
    back += kBlock;
  }
  if (g == 0 && t == 0) {
    const long long nsl = (long long)n_free + held_all;
    info[CASCADE_INFO_N_ADMITTED] = (int)tot[3];
    info[CASCADE_INFO_N_SLOT_LIST] = (int)nsl;
    info[CASCADE_INFO_N_UNPACK] = (int)nu;
    info[CASCADE_INFO_N_PACK] = (int)held_offl;
    const bool full = nsl > o.sl_cap || nu > o.unpack_cap || held_offl > o.pack_cap;
    if (full && load_agent(info) == CASCADE_OK) set_status(info, CASCADE_ENOSPC);
  }
  if (nv_all > kFinVictims || nr > kRestoreCap) {
    // beyond the LDS copies: the sequential finish, in workgroup 0 only
    __syncthreads();
    if (g == 0)
      finish_step(ctl, info, n, n_free, n_tiles, n_rp, tiles, free_slots, rp, rl, slots, o,
                  U.seq);
    return;
  }
  const int nv = nv_all;
  int v_total;
  {
    constexpr int kPer = kFinVictims / kBlock;
    int h[kPer], run = 0;
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int v = t * kPer + u;
      h[u] = v < nv ? L.v_held[v] : 0;
      run += h[u];
    }
    int ex[1] = {run}, tt1[1];
    block_exclusive_scan<1>(ex, tt1, L.scan_tmp);
    int acc = ex[0];
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int v = t * kPer + u;
      if (v < nv) L.v_start[v] = acc;
      acc += h[u];
    }
    v_total = tt1[0];
  }
  if (g == 0 && t < kFinVictims) {
    for (int v = t; v < nv; v += kBlock)
      o.action[L.v_req[v]] = (uint8_t)(L.v_offl[v] ? CASCADE_ACT_PREEMPT_OFFLOAD
                                                  : CASCADE_ACT_PREEMPT_DROP);
  }
  __syncthreads();

  // this workgroup's slice of the output entries: [0, lim) free part of the
  // slot list, then v_total victim blocks, then nu restore moves
  const long long lim = min(n_free, o.sl_cap);
  const long long total = lim + v_total + nu;
  const long long chunk = (total + G - 1) / G;
  const long long i_end = lmin(total, (long long)(g + 1) * chunk);
  for (long long i0 = (long long)g * chunk; i0 < i_end; i0 += kFinItems * kBlock) {
    // pass 1: the owner of every entry and the one load it needs
    int kind[kFinItems], aux[kFinItems], ld[kFinItems];
    long long idx[kFinItems];
#pragma unroll
    for (int u = 0; u < kFinItems; ++u) {
      const long long i = i0 + u * kBlock + t;
      kind[u] = -1;
      ld[u] = 0;
      idx[u] = 0;
      aux[u] = 0;
      if (i >= i_end) continue;
      if (i < lim) {  // free part of the slot list
        kind[u] = 0;
        idx[u] = i;
        ld[u] = free_slots[i];
      } else if (i < lim + v_total) {  // victim block
        const int m = (int)(i - lim);
        const int v = last_at_or_below<kFinVictimSteps>(nv, m, [&](int k) { return L.v_start[k]; });
        kind[u] = 1;
        idx[u] = m;
        aux[u] = v;
        ld[u] = slots[L.v_row0[v] + (m - L.v_start[v])];
      } else {  // restore move
        const long long m = i - lim - v_total;
        const int k =
            last_at_or_below<kRestoreSteps>(nr, m, [&](int q) { return L.rl[q].stage_off; });
        const RestoreEnt re = L.rl[k];
        const long long s = (long long)re.alloc_off + (m - re.stage_off);
        kind[u] = 2;
        idx[u] = m;
        aux[u] = k;
        if (s < o.sl_cap) {
          if (s < n_free) {
            ld[u] = free_slots[s];
          } else {
            const int mv = (int)(s - n_free);
            const int v =
                last_at_or_below<kFinVictimSteps>(nv, mv, [&](int q) { return L.v_start[q]; });
            ld[u] = slots[L.v_row0[v] + (mv - L.v_start[v])];
          }
        }
      }
    }
    // pass 2: the entries
#pragma unroll
    for (int u = 0; u < kFinItems; ++u) {
      if (kind[u] == 0) {
        o.slot_list[idx[u]] = ld[u];
      } else if (kind[u] == 1) {
        const int m = (int)idx[u], v = aux[u], b = m - L.v_start[v], slot = ld[u];
        const long long sb = L.v_sbase[v] + b;
        if (sb < o.sl_cap) o.slot_list[sb] = slot;
        const long long pb = L.v_pbase[v];
        const long long j = pb >= 0 ? pb + b : -1;
        if (j >= 0 && j < o.pack_cap) {
          cascade_move_t mv;
          mv.req = L.v_req[v];
          mv.blk = b;
          mv.pool_slot = slot;
          mv.staging_slot = (int)j;
          o.pack[j] = mv;
          if (o.pack_hazard) o.pack_hazard[j] = fin_unpack_move_at(sb, nr, L);
        }
      } else if (kind[u] == 2) {
        const long long m = idx[u];
        const RestoreEnt re = L.rl[aux[u]];
        const int b = (int)(m - re.stage_off);
        const long long s = (long long)re.alloc_off + b;
        if (m < o.unpack_cap) {
          cascade_move_t mv;
          mv.req = re.req;
          mv.blk = b;
          mv.pool_slot = s < o.sl_cap ? ld[u] : -1;
          mv.staging_slot = (int)m;
          o.unpack[m] = mv;
          if (o.unpack_hazard) {
            int hz = -1;  // a free slot is read by no pack move
            if (s >= n_free) {
              const int mv2 = (int)(s - n_free);
              const int v = last_at_or_below<kFinVictimSteps>(
                  nv, mv2, [&](int q) { return L.v_start[q]; });
              const long long pb = L.v_pbase[v];
              const long long j = pb >= 0 ? pb + (mv2 - L.v_start[v]) : -1;
              hz = (j >= 0 && j < o.pack_cap) ? (int)j : -1;
            }
            o.unpack_hazard[m] = hz;
          }
        }
      }
    }
  }
}

// Sums over tiles j < tile of the level-1 totals (l1[j*kL1 + k]), over the
// workgroup, and the running prefills of all n_tiles tiles.  Up to 2*kBlock
// tiles are requested at once (one round trip); an earlier launch wrote
// them, so nothing is polled.  The step's status word rides along in the
// same reduction: the return value says whether an earlier kernel reported
// a failure, the same in every thread.
__device__ __forceinline__ bool earlier_totals(const unsigned *__restrict__ l1,
                                               const unsigned *__restrict__ adj, int tile,
                                               int n_tiles, const int *info,
                                               long long (&pre1)[kL1], long long &rp_total,
                                               long long *s_red) {
  constexpr int kPer = 2, K = kL1 + 2;
  const int st = load_agent(info);
  long long v[K];
#pragma unroll
  for (int k = 0; k < K; ++k) v[k] = 0;
  for (int b0 = 0; b0 < n_tiles; b0 += kPer * kBlock) {
    unsigned w1[kPer][kL1];
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      // unconditional loads (tile 0 stands in past the end), masked after
      const int j = b0 + u * kBlock + (int)threadIdx.x;
      const int jc = j < n_tiles ? j : 0;
#pragma unroll
      for (int k = 0; k < kL1; ++k) w1[u][k] = l1[(size_t)jc * kL1 + k];
    }
    // shared prefixes: the followers' wants and shared tokens, taken off
    // the earlier tiles' want and need totals
    unsigned a1[kPer][2] = {{0, 0}, {0, 0}};
    if (adj) {
#pragma unroll
      for (int u = 0; u < kPer; ++u) {
        const int j = b0 + u * kBlock + (int)threadIdx.x;
        const int jc = j < n_tiles ? j : 0;
        a1[u][0] = adj[(size_t)jc * 2];
        a1[u][1] = adj[(size_t)jc * 2 + 1];
      }
    }
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int j = b0 + u * kBlock + (int)threadIdx.x;
#pragma unroll
      for (int k = 0; k < kL1; ++k) v[k] += j < tile ? (long long)w1[u][k] : 0ll;
      v[0] -= j < tile ? (long long)a1[u][0] : 0ll;
      v[1] -= j < tile ? (long long)a1[u][1] : 0ll;
      v[kL1] += j < n_tiles ? (long long)w1[u][4] : 0ll;
    }
  }
  v[K - 1] = (threadIdx.x == 0 && bad_status(st)) ? 1 : 0;
  block_sum<K>(v, s_red);
#pragma unroll
  for (int k = 0; k < kL1; ++k) pre1[k] = v[k];
  rp_total = v[kL1];
  return v[K - 1] != 0;
}

// The tile's positions in priority order: request index, scan record and
// row offset, from the last radix pass (sorted buffers) or, when every key
// is equal (no pass moved data), the identity order.  Positions past n get
// index -1.  `broken` is set on an index out of range.
__device__ __forceinline__ void tile_positions(int n, int tile, int nact, const Sorted &srt,
                                               const int4 *__restrict__ rec,
                                               const unsigned (&so)[kScanItems],
                                               const int4 (&sr)[kScanItems],
                                               int (&idx)[kScanItems], int4 (&r4)[kScanItems],
                                               bool &broken) {
  const int p0 = tile * kScanTile + (int)threadIdx.x * kScanItems;
#pragma unroll
  for (int j = 0; j < kScanItems; ++j) {
    const int p = p0 + j;
    int ix = -1;
    int4 r = make_int4(0, 0, 0, 0);
    if (p < n) {
      if (nact == 0) {
        ix = p;
        r = rec[p];
      } else {
        ix = (int)so[j];
        r = sr[j];
      }
    }
    if ((unsigned)ix >= (unsigned)n) {  // cannot happen with a correct sort
      broken = broken || ix != -1;
      ix = -1;
    }
    idx[j] = ix;
    r4[j] = ix >= 0 ? r : make_int4(0, 0, 0, 0);
  }
}

// The sorted entries of the tile's positions (blockIdx.x), requested before
// anything else.
__device__ __forceinline__ void load_sorted(int n, const Sorted &srt, unsigned (&so)[kScanItems],
                                            int4 (&sr)[kScanItems]) {
  const int p0 = (int)blockIdx.x * kScanTile + (int)threadIdx.x * kScanItems;
#pragma unroll
  for (int j = 0; j < kScanItems; ++j) {
    const int p = p0 + j;
    so[j] = p < n ? srt.order[p] : 0u;
    sr[j] = p < n ? srt.rec[p] : make_int4(0, 0, 0, 0);
  }
}

// ------------------------------------------------------ shared prefixes

// Shared-prefix restores within a step (Section 4.4 prefix hit detection;
// the paper leaves within-step sharing open, reading: within a priority
// group, the first queued DRAM/NVMe member of a prefix group with a restore
// want leads and restores under the link cap; every later such member of
// the group follows and references min(leader's restore, own prefix) blocks
// of it, taking nothing from the cap).  The last radix pass marks each
// group's leader position as it writes the order (share_mark: the table
// holds n - position, 0 for none, so the maximum is the first position);
// then one launch over the scan tiles (share_kernel) takes the followers'
// wants off the link cap, lets the leaders restore and rewrites the
// followers' records.
// The request index and scan record at position p: the sorted buffers, or
// the identity order when no radix pass moved data.
__device__ __forceinline__ void position_rec(int p, int nact, const Sorted &srt,
                                             const int4 *__restrict__ rec, int &ix, int4 &r) {
  if (nact == 0) {
    ix = p;
    r = rec[p];
  } else {
    ix = (int)srt.order[p];
    r = srt.rec[p];
  }
}

// Is position p's member a follower (behind its group's leader)?
__device__ __forceinline__ bool share_follows(const int4 &r, int p, int n,
                                              const unsigned *lead, unsigned *enc_out) {
  if (!rec_member(r.w) || (unsigned)r.z >= (unsigned)n) return false;
  const unsigned enc = lead[share_slot(r)];
  *enc_out = enc;
  return enc != 0 && p > n - (int)enc;
}

// One workgroup per scan tile.  The tile's followers' wants are published at
// once (pub[tile] = wants << 1 | 1, and adj[2 tile] for the scan); the link-cap
// prefix before the tile is the earlier tiles' level-1 want totals less
// their published followers' wants (a look-back over lower tiles only, which
// publish before they wait on anything).  Then the tile's leaders publish
// their restore blocks, and its followers wait for their leader's.
__global__ __launch_bounds__(kBlock) void share_kernel(int n, int n_tiles, int bt, int max_move,
                                                       Ctl *ctl, int *info, Sorted srt,
                                                       int4 *__restrict__ rec,
                                                       const unsigned *__restrict__ l1_tot,
                                                       const unsigned *__restrict__ lead,
                                                       unsigned *rl, unsigned *adj,
                                                       unsigned *pub) {
  __shared__ long long s_red[kWaves * 3];
  __shared__ unsigned s_scan[kWaves];
  const int tile = (int)blockIdx.x;
  if (bad_status(load_agent(info))) {
    // a failed step: publish "no followers", so no later tile waits on this one
    if (threadIdx.x == 0) store_agent(pub + tile, 1u);
    return;
  }
  const int nact = (int)ctl->nact;
  const int p0 = tile * kScanTile + (int)threadIdx.x * kScanItems;
  int ix[kScanItems];
  int4 r4[kScanItems];
#pragma unroll
  for (int j = 0; j < kScanItems; ++j) {
    ix[j] = -1;
    r4[j] = make_int4(0, 0, 0, 0);
    if (p0 + j < n) position_rec(p0 + j, nact, srt, rec, ix[j], r4[j]);
  }
  // this tile's wants in position order (a follower wants nothing), and its
  // followers' wants, published at once
  unsigned enc[kScanItems];
  bool fol[kScanItems];
  unsigned wsum[1] = {0}, wtot[1];
  int wj[kScanItems];
  long long fw[2] = {0, 0};  // the followers' wants, those in groups 0-1
#pragma unroll
  for (int j = 0; j < kScanItems; ++j) {
    enc[j] = 0;
    fol[j] = ix[j] >= 0 && share_follows(r4[j], p0 + j, n, lead, &enc[j]);
    wj[j] = (ix[j] >= 0 && !fol[j]) ? rec_want(r4[j]) : 0;
    wsum[0] += (unsigned)wj[j];
    if (fol[j]) {
      fw[0] += r4[j].x;
      fw[1] += rec_grp(r4[j].w) <= 1 ? r4[j].x : 0;
    }
  }
  block_sum<2>(fw, s_red);
  if (threadIdx.x == 0) {
    // below 2^31: 1024 wants below 2^18
    store_agent(pub + tile, ((unsigned)fw[0] << 1) | 1u);
    adj[(size_t)tile * 2] = (unsigned)fw[0];
    if (fw[1]) atomicAdd(reinterpret_cast<unsigned long long *>(&ctl->want1_sub),
                         (unsigned long long)fw[1]);
  }
  // the link-cap prefix before this tile: the earlier tiles' want totals
  // without their followers' wants
  long long pre[2] = {0, 0};  // the prefix, timeouts
  for (int k = (int)threadIdx.x; k < tile; k += kBlock) {
    unsigned v = load_agent(pub + k);
    unsigned spins = 0;
    while ((v & 1u) == 0u) {
      if (++spins > kSpinLimit) break;
      __builtin_amdgcn_s_sleep(1);
      v = load_agent(pub + k);
    }
    if ((v & 1u) == 0u) pre[1] += 1;
    pre[0] += (long long)l1_tot[(size_t)k * kL1] - (long long)(v >> 1);
  }
  block_sum<2>(pre, s_red);
  if (pre[1] && threadIdx.x == 0) set_status(info, CASCADE_ETIMEOUT);
  block_exclusive_scan<1>(wsum, wtot, s_scan);
  // leaders publish their restore blocks (eq:max_restorable under the cap)
  long long wx = pre[0] + wsum[0];
  const long long U = max_move;
#pragma unroll
  for (int j = 0; j < kScanItems; ++j) {
    const long long rj = lmin(wx + wj[j], U) - lmin(wx, U);
    wx += wj[j];
    if (ix[j] >= 0 && rec_member(r4[j].w) && enc[j] != 0 && p0 + j == n - (int)enc[j])
      store_agent(rl + share_slot(r4[j]), 0x80000000u | (unsigned)rj);
  }
  __syncthreads();
  // followers: wait for their leader's restore (a leader sits at a lower
  // position, in this tile or an earlier one, which publishes before it
  // waits on anything), then reference min(its blocks, own prefix blocks)
  long long dn[3] = {0, 0, 0};  // shared tokens: all, groups 0-1, timeouts
#pragma unroll
  for (int j = 0; j < kScanItems; ++j) {
    if (!fol[j]) continue;
    const int4 r = r4[j];
    unsigned v = load_agent(rl + share_slot(r));
    unsigned spins = 0;
    while ((v >> 31) == 0) {
      if (++spins > kSpinLimit) break;
      __builtin_amdgcn_s_sleep(1);
      v = load_agent(rl + share_slot(r));
    }
    if ((v >> 31) == 0) {
      dn[2] += 1;
      continue;
    }
    const int pl = n - (int)enc[j];
    const int lead_req = nact == 0 ? pl : (int)srt.order[pl];
    const int u = min((int)(v & 0x7FFFFFFFu), rec_held(r.w));
    int4 nr;
    nr.x = u > 0 ? lead_req : -1;
    nr.y = r.y - bt * u;
    nr.z = bt * u;
    nr.w = (r.w & ~(3 << 22)) | (CASCADE_KV_HBM << 22) | (1 << 29);
    if (nact == 0) rec[p0 + j] = nr;
    else srt.rec[p0 + j] = nr;
    dn[0] += (long long)bt * u;
    dn[1] += rec_grp(r.w) <= 1 ? (long long)bt * u : 0;
  }
  block_sum<3>(dn, s_red);
  if (threadIdx.x == 0) {
    adj[(size_t)tile * 2 + 1] = (unsigned)dn[0];  // below 2^31: 1024 needs below 2^18
    if (dn[1]) atomicAdd(reinterpret_cast<unsigned long long *>(&ctl->need1_sub),
                         (unsigned long long)dn[1]);
    if (dn[2]) set_status(info, CASCADE_ETIMEOUT);
  }
}

// Algorithm 1's Phase 2 loop in priority order as prefix sums.
// Level 1 (independent of earlier decisions): restore want, base token need,
// blocks held by running prefills (all / spill-fits).  They give the restore
// blocks r (eq:max_restorable under the per-step cap U), the exact token need
// and the chunked-prefill grant g of every position.
// Level 2 (functions of g): block weight of the admission test, new blocks
// of admitted requests, admitted count, held blocks of running prefills left
// out (all / spill-fits), restored blocks and restoring requests.
// A tile's level-1 prefix is the sum of the earlier tiles' totals (added by
// the last radix pass), requested with its sorted records; its level-2
// prefix comes from a decoupled look-back over the totals the earlier tiles
// publish.  Workgroups past the last tile finish the step (victims, slot
// list, move lists) once every tile has handed over.
__global__ __launch_bounds__(kBlock) void scan_kernel(
    int n, int passes, int n_tiles, Consts c, Ctl *ctl, int *info, Sorted srt,
    const int4 *__restrict__ rec, const int *__restrict__ slots,
    const int *__restrict__ free_slots, Outs o, RpInfo *__restrict__ rp_list,
    RestoreEnt *__restrict__ restore_list, TileTot *__restrict__ tile_tot,
    const unsigned *__restrict__ l1_tot, const unsigned *__restrict__ share_adj,
    unsigned long long *l2_status) {
  __shared__ ScanLds s_lds;
  __shared__ FinishAnyLds s_fin;
  __shared__ int s_bad;

  const int t = threadIdx.x, tile = (int)blockIdx.x;
  const unsigned groups = min((unsigned)n_tiles, (unsigned)kTicketGroups);
  if (tile >= n_tiles) {
    // a finishing workgroup: wait until every scan tile has handed over;
    // lane g of the first wave watches the counter of tiles g, g + groups, ..
    if (t < 64) {
      const unsigned size =
          (unsigned)t < groups ? ((unsigned)n_tiles - t + groups - 1) / groups : 0u;
      unsigned spins = 0;
      bool late = false;
      while (true) {
        const unsigned got = (unsigned)t < groups ? load_agent(ctl->done + t * kTicketStride) : 0u;
        if (__ballot(got < size) == 0) break;
        if (++spins > kSpinLimit) {
          late = true;
          break;
        }
        __builtin_amdgcn_s_sleep(2);
      }
      if (t == 0) {
        s_bad = late ? 1 : 0;
        if (late) set_status(info, CASCADE_ETIMEOUT);
      }
    }
    __syncthreads();
    if (s_bad) return;
    acquire_agent();  // the tiles' hand-over stores precede every read below
    finish_grid(tile - n_tiles, (int)gridDim.x - n_tiles, n, c.n_free, n_tiles, ctl, info,
                tile_tot, free_slots, rp_list, restore_list, slots, o, s_fin);
    return;
  }
  unsigned so[kScanItems];
  int4 sr[kScanItems];
  load_sorted(n, srt, so, sr);
  const int nact = (int)ctl->nact;
  long long pre1[kL1], rp_total;
  if (earlier_totals(l1_tot, share_adj, tile, n_tiles, info, pre1, rp_total, s_lds.red)) {
    // a failed step: the look-back words say "nothing before me", so no later
    // tile waits, and the tile is counted, so the finishing workgroups stop
    if (t < kL2) publish<unsigned long long>(l2_status + (size_t)tile * kL2Stride + t, 0ull,
                                             kFlagInclusive);
    if (t == 0) atomicAdd(ctl->done + ((unsigned)tile % groups) * kTicketStride, 1u);
    return;
  }
  // a live digit beyond the launched passes would leave the keys unsorted
  bool broken = nact > passes;
  int idx[kScanItems];
  int4 r4[kScanItems];
  tile_positions(n, tile, nact, srt, rec, so, sr, idx, r4, broken);
  const ScanConsts K = scan_consts(c, ctl);

  TileOut out;
  const long long rp_incl =
      scan_tile<true>(tile, kScanItems, K, ctl, info, idx, r4, broken, o, rp_list,
                      restore_list, tile_tot, pre1, rp_total, l2_status, s_lds, out);
  if (tile == n_tiles - 1 && t == 0) store_agent(&ctl->n_rp, (int)rp_incl);
  // hand-over: this tile's agent-scope stores complete, then it is counted
  // (one of kTicketGroups counters, so that no address takes more than a few
  // dozen adds); its other outputs follow
  wait_stores();
  __syncthreads();
  if (t == 0) atomicAdd(ctl->done + ((unsigned)tile % groups) * kTicketStride, 1u);
  write_tile_outputs(out, o);
}

// ------------------------------------------------------------ small queues

// A queue of at most kScanTile requests is one sort tile and one scan tile,
// so the whole step runs in one workgroup: keys, records and the order stay
// in LDS, and nothing waits on another workgroup.  Same arithmetic and the
// same device functions as the multi-launch path, so the result is the same.
constexpr int kSmallMax = kScanTile;
static_assert(kSmallMax >= kBlock, "finish_grid reads kBlock list entries unchecked");
constexpr int kSmallCheckBlocks = 16384;  // pools up to this size are checked in-kernel
constexpr int kCheckGrid = 64;
constexpr int kSmallItems = kScanItems;  // one sort tile and one scan tile per small queue
constexpr int kSmallRankMax = 512;  // queues up to this size are ordered by counting ranks
constexpr int kSmallFreeHead = 8;   // list entries per thread requested ahead of their check
constexpr int kSmallIdxBits = 10;   // request index below the key in the rank sort
constexpr int kRankRound = 16;      // keys compared per round of LDS reads in the rank sort

struct SmallSortLds {
  unsigned long long key[kSmallMax];
  unsigned val[kSmallMax];
  int4 rec[kSmallMax];
  unsigned wcnt[kWaves][kRadix];
  int start[kRadix];
};
union SmallLds {  // the sort is finished before the finish stages anything
  SmallSortLds sort;
  FinishLds fin;
};

// Per item j < J: how many of the n keys (the LDS array, padded with
// all-ones keys to whole rounds) are below mine[j].
template <int J, int K>
__device__ __forceinline__ void rank_count(const ulonglong2 *pairs, int n,
                                           const unsigned long long (&mine)[K], int (&below)[K]) {
  for (int m = 0; m < n; m += kRankRound) {
    unsigned long long other[kRankRound];
#pragma unroll
    for (int u = 0; u < kRankRound / 2; ++u) {
      const ulonglong2 q = pairs[m / 2 + u];
      other[2 * u] = q.x;
      other[2 * u + 1] = q.y;
    }
#pragma unroll
    for (int u = 0; u < kRankRound; ++u)
#pragma unroll
      for (int j = 0; j < J; ++j) below[j] += other[u] < mine[j] ? 1 : 0;
  }
}

// Rank of this lane's item among the wave's items with the same 8-bit digit
// (dig < 0: no item), items taken in (call, lane) order; wcnt[d] counts the
// wave's items of digit d seen so far.
__device__ __forceinline__ int wave_digit_rank(int dig, unsigned *wcnt) {
  const bool v = dig >= 0;
  uint64_t peers = __ballot(v);
#pragma unroll
  for (int b = 0; b < 8; ++b) {
    const bool bit = (dig >> b) & 1;
    const uint64_t bal = __ballot(bit);
    peers &= bit ? bal : ~bal;
  }
  const int d = v ? dig : 0;
  unsigned before = 0;
  if (v) before = wcnt[d];
  __builtin_amdgcn_wave_barrier();
  const int below = rank_in_mask(peers);
  if (v && below == 0) wcnt[d] = before + (unsigned)__builtin_popcountll(peers);
  __builtin_amdgcn_wave_barrier();
  return (int)before + below;
}

// Range checks of the free list and of the block-table slots (num_blocks),
// 8 loads per thread in flight; true if any entry is out of range.
__device__ __forceinline__ bool any_out_of_range(const int *__restrict__ a, int count,
                                                 int num_blocks, int first, int stride) {
  bool bad = false;
  for (int j0 = first; j0 < count; j0 += 8 * stride) {
    int v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = (j0 + u * stride < count) ? a[j0 + u * stride] : 0;
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if ((unsigned)v[u] >= (unsigned)num_blocks) bad = true;
  }
  return bad;
}

// The same checks spread over a grid, for a small queue over a large pool:
// run after the step, they can only turn its status into CASCADE_EINVAL
// (outputs are unspecified then), and they read the block table only when
// the step found the row structure valid.
__global__ __launch_bounds__(kBlock) void check_lists_kernel(int n, int num_blocks, int n_free,
                                                             const int *__restrict__ free_slots,
                                                             const int *__restrict__ ro,
                                                             const int *__restrict__ slots,
                                                             int *info) {
  __shared__ int s_skip;
  if (threadIdx.x == 0) s_skip = load_agent(info) == CASCADE_EINVAL;
  __syncthreads();
  if (s_skip) return;
  const int first = blockIdx.x * kBlock + threadIdx.x, stride = gridDim.x * kBlock;
  bool bad = any_out_of_range(free_slots, n_free, num_blocks, first, stride);
  bad |= any_out_of_range(slots, ro[n], num_blocks, first, stride);
  if (bad) set_status(info, CASCADE_EINVAL);
}

__global__ __launch_bounds__(kBlock) void step_small_kernel(
    cascade_requests_t rq, const int *__restrict__ ro, const int *__restrict__ slots,
    const int *__restrict__ free_slots, Consts c, int n, int check_lists, Ctl *ctl, int *info,
    Outs o, int64_t *__restrict__ budget_out, uint8_t *__restrict__ tier_out,
    RpInfo *__restrict__ rp_list, RestoreEnt *__restrict__ restore_list,
    TileTot *__restrict__ tile_tot) {
  __shared__ long long s_slo[16];
  __shared__ unsigned long long s_red[kWaves * 9];
  __shared__ unsigned long long s_mm[kWaves * 4];
  __shared__ int s_scan1[kWaves];
  __shared__ ScanLds s_lds;
  __shared__ SmallLds U;
  const int t = threadIdx.x, lane = lane_id(), wave = wave_id();
  // the head of the free list is requested first (checked after eval)
  int fl[kSmallFreeHead];
#pragma unroll
  for (int u = 0; u < kSmallFreeHead; ++u) {
    const int j = t + u * kBlock;
    fl[u] = (check_lists && j < c.n_free) ? free_slots[j] : 0;
  }
  if (t < 16) s_slo[t] = c.slo[t];
  if (t == 0) {
    unsigned *w = reinterpret_cast<unsigned *>(ctl);
    for (size_t k = 0; k < kCtlHeaderWords; ++k) w[k] = 0;
    ctl->kstar = n;
    for (int k = 0; k < CASCADE_INFO_LEN; ++k) info[k] = 0;
    info[CASCADE_INFO_N_SLOT_LIST] = c.n_free;
  }
  __syncthreads();

  // ---- evaluation, request j*kBlock + t on thread t (every wave busy); the
  //      raw keys and the records wait in LDS for the sort
  bool bad = false;
  // sums (held, need1, want1, three group counts, bad), then min and max
  unsigned long long v[9] = {0, 0, 0, 0, 0, 0, 0, ~0ull, 0};
#pragma unroll
  for (int j = 0; j < kSmallItems; ++j) {
    const int i = j * kBlock + t;
    if (i >= n) continue;
    const ReqEval r = eval_request(rq, ro, c, s_slo, i, n);
    bad |= r.bad;
    v[7] = r.biased < v[7] ? r.biased : v[7];
    v[8] = r.biased > v[8] ? r.biased : v[8];
    v[3 + r.grp] += 1;
    budget_out[i] = r.brem;
    tier_out[i] = (uint8_t)r.tnew;
    U.sort.key[i] = ((unsigned long long)r.grp << 62) | r.biased;
    U.sort.rec[i] = r.rec;
    v[0] += (unsigned long long)r.held;
    v[1] += (unsigned long long)r.need1;
    v[2] += (unsigned long long)r.want1;
  }
  // the free list in range (large pools: checked by a grid after this kernel)
  if (check_lists) {
#pragma unroll
    for (int u = 0; u < kSmallFreeHead; ++u) bad |= (unsigned)fl[u] >= (unsigned)c.num_blocks;
    const int done = kSmallFreeHead * kBlock;
    if (c.n_free > done)
      bad |= any_out_of_range(free_slots + done, c.n_free - done, c.num_blocks, t, kBlock);
  }
  v[6] = bad ? 1 : 0;
#pragma unroll
  for (int k = 0; k < 7; ++k) v[k] = wave_sum(v[k]);
  v[7] = wave_min(v[7]);
  v[8] = wave_max(v[8]);
  if (lane == 0) {
#pragma unroll
    for (int k = 0; k < 9; ++k) s_red[wave * 9 + k] = v[k];
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < 9; ++k) v[k] = s_red[k];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) {
#pragma unroll
    for (int k = 0; k < 7; ++k) v[k] += s_red[w * 9 + k];
    v[7] = s_red[w * 9 + 7] < v[7] ? s_red[w * 9 + 7] : v[7];
    v[8] = s_red[w * 9 + 8] > v[8] ? s_red[w * 9 + 8] : v[8];
  }
  const unsigned long long mn = v[7], mx = v[8];
  const unsigned cnt1 = (unsigned)v[4], cnt2 = (unsigned)v[5];
  if (v[6]) {  // bad request data or free list: nothing below is meaningful
    if (t == 0) set_status(info, CASCADE_EINVAL);
    return;
  }
  if (t == 0) {
    ctl->bmin = mn;
    ctl->bmax = mx;
    ctl->held_rp = (long long)v[0];
    ctl->need1 = (long long)v[1];
    ctl->want1 = (long long)v[2];
    ctl->cnt[0] = (unsigned)v[3];
    ctl->cnt[1] = cnt1;
    ctl->cnt[2] = cnt2;
  }
  // block-table slots, whose extent is only trustworthy now: requested here,
  // checked after the sort (a large pool's lists are checked by a grid
  // launched after this kernel)
  int sv[kSmallFreeHead];
  const int nnz = check_lists ? ro[n] : 0;
#pragma unroll
  for (int u = 0; u < kSmallFreeHead; ++u) {
    const int j = t + u * kBlock;
    sv[u] = j < nnz ? slots[j] : 0;
  }

  const int jn = (n + kBlock - 1) / kBlock;
  const unsigned long long span = mx - mn + 1;
  const int width = key_bits(mn, mx, cnt1, cnt2);
  bool moved = false;
  if (n <= kSmallRankMax && width <= 64 - kSmallIdxBits) {
    // ---- a short queue: every request's place is the number of (key,
    //      index) pairs below its own, counted over LDS broadcast reads;
    //      the index below the compressed key keeps equal keys in queue order
#pragma unroll
    for (int j = 0; j < kSmallItems; ++j) {
      const int i = j * kBlock + t;
      if (j < jn && i < n) {
        const unsigned long long k0 = U.sort.key[i];
        const unsigned long long k = (k0 >> 62) * span + ((k0 & ((1ull << 62) - 1)) - mn);
        U.sort.key[i] = (k << kSmallIdxBits) | (unsigned)i;
      }
    }
    if (t < kRankRound) U.sort.key[n + t] = ~0ull;  // pad to whole rounds: above every key
    __syncthreads();
    unsigned long long mine[kSmallRankMax / kBlock];
    int below[kSmallRankMax / kBlock];
#pragma unroll
    for (int j = 0; j < kSmallRankMax / kBlock; ++j) {
      const int i = j * kBlock + t;
      mine[j] = i < n ? U.sort.key[i] : ~0ull;
      below[j] = 0;
    }
    // kRankRound keys per round of LDS reads (two per 16-byte read); the
    // comparisons are VALU-bound, so a thread compares only the items it has
    const ulonglong2 *pairs = reinterpret_cast<const ulonglong2 *>(U.sort.key);
    if (jn == 1) {
      rank_count<1>(pairs, n, mine, below);
    } else {
      rank_count<kSmallRankMax / kBlock>(pairs, n, mine, below);
    }
#pragma unroll
    for (int j = 0; j < kSmallRankMax / kBlock; ++j) {
      const int i = j * kBlock + t;
      if (i < n) U.sort.val[below[j]] = (unsigned)i;
    }
    __syncthreads();
    moved = true;
  } else {
    // ---- order-preserving key compression, then LSD radix passes in LDS over
    //      the digits that are not uniform across the queue.  A thread holds
    //      jn = ceil(n / kBlock) items, item j at position (wave*jn + j)*64 +
    //      lane: the order in which wave_digit_rank ranks them.
    unsigned long long key[kSmallItems];
    unsigned val[kSmallItems];
    unsigned long long k_and = ~0ull, k_or = 0;
#pragma unroll
    for (int j = 0; j < kSmallItems; ++j) {
      const int p = (wave * jn + j) * 64 + lane;
      key[j] = 0;
      val[j] = (unsigned)p;
      if (j >= jn || p >= n) continue;
      const unsigned long long k0 = U.sort.key[p];
      key[j] = (k0 >> 62) * span + ((k0 & ((1ull << 62) - 1)) - mn);
      k_and &= key[j];
      k_or |= key[j];
    }
    for (int off = 32; off >= 1; off >>= 1) {
      k_and &= __shfl_xor(k_and, off, 64);
      k_or |= __shfl_xor(k_or, off, 64);
    }
    if (lane == 0) {
      s_mm[2 * kWaves + wave] = k_and;
      s_mm[3 * kWaves + wave] = k_or;
    }
    __syncthreads();
    unsigned long long varying = 0;
    {
      unsigned long long a = ~0ull, b = 0;
      for (int w = 0; w < kWaves; ++w) {
        a &= s_mm[2 * kWaves + w];
        b |= s_mm[3 * kWaves + w];
      }
      varying = a ^ b;  // bits that differ between two keys of the queue
    }
    const int nd = (width + 7) / 8;  // 8-bit digits
    for (int d = 0; d < nd; ++d) {
      if (((varying >> (8 * d)) & 255) == 0) continue;  // uniform: order unchanged
      moved = true;
      for (int k = t; k < kWaves * kRadix; k += kBlock) (&U.sort.wcnt[0][0])[k] = 0;
      __syncthreads();
      int dig[kSmallItems], rank[kSmallItems];
#pragma unroll
      for (int j = 0; j < kSmallItems; ++j) {
        const int p = (wave * jn + j) * 64 + lane;
        dig[j] = (j < jn && p < n) ? (int)((key[j] >> (8 * d)) & 255) : -1;
        rank[j] = j < jn ? wave_digit_rank(dig[j], U.sort.wcnt[wave]) : 0;
      }
      __syncthreads();
      // thread t = digit t: earlier waves' counts, then the digit's start
      unsigned run = 0;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const unsigned cw = U.sort.wcnt[w][t];
        U.sort.wcnt[w][t] = run;
        run += cw;
      }
      int st[1] = {(int)run}, tot1[1];
      block_exclusive_scan<1>(st, tot1, s_scan1);
      U.sort.start[t] = st[0];
      __syncthreads();
#pragma unroll
      for (int j = 0; j < kSmallItems; ++j) {
        if (dig[j] < 0) continue;
        const int pos = U.sort.start[dig[j]] + (int)U.sort.wcnt[wave][dig[j]] + rank[j];
        U.sort.key[pos] = key[j];
        U.sort.val[pos] = val[j];
      }
      __syncthreads();
#pragma unroll
      for (int j = 0; j < kSmallItems; ++j) {
        const int p = (wave * jn + j) * 64 + lane;
        if (j < jn && p < n) {
          key[j] = U.sort.key[p];
          val[j] = U.sort.val[p];
        }
      }
    }
  }

  if (check_lists) {
    bool bad_slot = false;
#pragma unroll
    for (int u = 0; u < kSmallFreeHead; ++u) bad_slot |= (unsigned)sv[u] >= (unsigned)c.num_blocks;
    const int done = kSmallFreeHead * kBlock;
    if (nnz > done) bad_slot |= any_out_of_range(slots + done, nnz - done, c.num_blocks, t, kBlock);
    if (__syncthreads_or(bad_slot ? 1 : 0)) {
      if (t == 0) set_status(info, CASCADE_EINVAL);
      return;
    }
  }

  // ---- Algorithm 1's Phase 2 as one tile: thread t holds positions
  //      t*jn .. t*jn + jn - 1
  int idx[kScanItems];
  int4 r4[kScanItems];
#pragma unroll
  for (int j = 0; j < kScanItems; ++j) {
    const int p = t * jn + j;
    idx[j] = (j < jn && p < n) ? (moved ? (int)U.sort.val[p] : p) : -1;
    r4[j] = idx[j] >= 0 ? U.sort.rec[idx[j]] : make_int4(0, 0, 0, 0);
  }
  if (rq.prefix_group) {
    // shared prefixes, the three stages of the multi-launch path in one
    // workgroup; the finished sort's keys and records (every position's
    // record is in registers now) hold the two tables
    __syncthreads();
    unsigned *lead = reinterpret_cast<unsigned *>(U.sort.key);
    unsigned *rl = reinterpret_cast<unsigned *>(U.sort.rec);
    static_assert(sizeof(U.sort.key) >= 2 * kSmallMax * sizeof(unsigned) &&
                      sizeof(U.sort.rec) >= 2 * kSmallMax * sizeof(unsigned),
                  "two table entries per request");
    for (int k = t; k < 2 * n; k += kBlock) {
      lead[k] = 0;
      rl[k] = 0;
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) {
      const int p = t * jn + j;
      if (idx[j] >= 0 && rec_member(r4[j].w) && r4[j].x > 0 && (unsigned)r4[j].z < (unsigned)n)
        atomicMax(lead + share_slot(r4[j]), (unsigned)(n - p));
    }
    __syncthreads();
    unsigned enc[kScanItems];
    bool fol[kScanItems];
    int wj[kScanItems];
    unsigned ws[1] = {0}, wt[1];
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) {
      enc[j] = 0;
      fol[j] = idx[j] >= 0 && share_follows(r4[j], t * jn + j, n, lead, &enc[j]);
      wj[j] = (idx[j] >= 0 && !fol[j]) ? rec_want(r4[j]) : 0;
      ws[0] += (unsigned)wj[j];
    }
    block_exclusive_scan<1>(ws, wt, reinterpret_cast<unsigned *>(s_scan1));
    long long wx = ws[0];
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) {
      const long long rj = lmin(wx + wj[j], (long long)c.max_move) - lmin(wx, (long long)c.max_move);
      wx += wj[j];
      if (idx[j] >= 0 && rec_member(r4[j].w) && enc[j] != 0 && t * jn + j == n - (int)enc[j])
        rl[share_slot(r4[j])] = 0x80000000u | (unsigned)rj;
    }
    __syncthreads();
    long long dv[2] = {0, 0};  // groups 0-1: the followers' wants and shared tokens
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) {
      if (!fol[j]) continue;
      const int4 r = r4[j];
      const unsigned v = rl[share_slot(r)];
      const int pl = n - (int)enc[j];
      const int u = min((int)(v & 0x7FFFFFFFu), rec_held(r.w));
      if (rec_grp(r.w) <= 1) {
        dv[0] += r.x;
        dv[1] += (long long)c.bt * u;
      }
      r4[j].x = u > 0 ? (moved ? (int)U.sort.val[pl] : pl) : -1;
      r4[j].y = r.y - c.bt * u;
      r4[j].z = c.bt * u;
      r4[j].w = (r.w & ~(3 << 22)) | (CASCADE_KV_HBM << 22) | (1 << 29);
    }
    block_sum<2>(dv, reinterpret_cast<long long *>(s_red));
    if (t == 0) {
      ctl->want1 -= dv[0];
      ctl->need1 -= dv[1];
    }
    __syncthreads();
  }
  const ScanConsts K = scan_consts(c, ctl);
  TileOut out;
  const long long zero1[kL1] = {0, 0, 0, 0, 0};
  const long long n_rp = scan_tile<false>(0, jn, K, ctl, info, idx, r4, false, o, rp_list,
                                          restore_list, tile_tot, zero1, 0, nullptr, s_lds, out);
  // the tile's hand-over records (other waves read them in finish_step) are
  // complete before the barrier; its per-request outputs follow
  wait_stores();
  __syncthreads();
  write_tile_outputs(out, o);
  finish_step(ctl, info, n, c.n_free, 1, (int)n_rp, tile_tot, free_slots, rp_list, restore_list,
              slots, o, U.fin);
}

// A step with no requests: only the free list becomes the slot list.
__global__ __launch_bounds__(kBlock) void empty_step_kernel(int n_free, int num_blocks,
                                                            const int *__restrict__ free_slots,
                                                            int *info, Outs o) {
  bool bad = false;
  const int lim = min(n_free, o.sl_cap);
  for (int j = threadIdx.x; j < n_free; j += kBlock) {
    const int s = free_slots[j];
    if ((unsigned)s >= (unsigned)num_blocks) bad = true;
    if (j < lim) o.slot_list[j] = s;
  }
  const bool any_bad = __syncthreads_or(bad ? 1 : 0);
  if (threadIdx.x == 0) {
    for (int k = 0; k < CASCADE_INFO_LEN; ++k) info[k] = 0;
    info[CASCADE_INFO_N_SLOT_LIST] = n_free;
    info[CASCADE_INFO_STATUS] =
        any_bad ? CASCADE_EINVAL : (n_free > o.sl_cap ? CASCADE_ENOSPC : CASCADE_OK);
  }
}

// ---------------------------------------------------------------- host

struct Layout {
  size_t ctl = 0, scan1 = 0, scan2 = 0, sort_status = 0, partials = 0, keys_a = 0, keys_b = 0,
         vals_a = 0, vals_b = 0, rec = 0, s_order = 0, s_rec = 0, rp_list = 0, restore = 0,
         tile_tot = 0, share_lead = 0, share_rl = 0, share_pub = 0, share_adj = 0, total = 0;
  int sort_tiles = 0, scan_tiles = 0, eval_grid = 0;
};

constexpr size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }

constexpr Layout make_layout(int32_t n) {
  Layout L;
  const size_t np = n > 0 ? (size_t)n : 1;
  L.sort_tiles = (int)((np + kSortTileTiny - 1) / kSortTileTiny);  // the most tiles a sort uses
  L.scan_tiles = (int)((np + kScanTile - 1) / kScanTile);
  L.eval_grid = (int)((np + kBlock * kEvalItems - 1) / (kBlock * kEvalItems));
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off = align_up(off + bytes); return o; };
  L.ctl = take(sizeof(Ctl));
  // the look-back status words follow the control block: one clear covers
  // them, the sort's words last (only the launched passes' are cleared)
  L.scan1 = take((size_t)L.scan_tiles * kL1 * 4);  // level-1 totals per scan tile
  L.scan2 = take((size_t)L.scan_tiles * kL2Stride * 8);  // level-2 look-back words per scan tile
  L.sort_status = take((size_t)kMaxPasses * L.sort_tiles * kMaxBins * 4);
  L.partials = take((size_t)L.eval_grid * sizeof(Partial));
  L.keys_a = take(np * 8);
  L.keys_b = take(np * 8);
  L.vals_a = take(np * 4);
  L.vals_b = take(np * 4);
  L.rec = take(np * 16);
  L.s_order = take(np * 4);
  L.s_rec = take(np * 16);
  L.rp_list = take(np * sizeof(RpInfo));
  L.restore = take(np * sizeof(RestoreEnt));
  L.tile_tot = take((size_t)L.scan_tiles * sizeof(TileTot));
  // shared prefixes: leader positions and published leader restores per
  // (group, priority group) and the tiles' published followers' wants,
  // contiguous for eval's clear; per scan tile the followers' wants and
  // shared tokens for the scan
  L.share_lead = take(np * 2 * 4);
  L.share_rl = take(np * 2 * 4);
  L.share_pub = take((size_t)L.scan_tiles * 4);
  L.share_adj = take((size_t)L.scan_tiles * 2 * 4);
  L.total = off;
  return L;
}

bool params_ok(const cascade_params_t *p, int32_t n, const cascade_tier_state_t *t) {
  const long long one = 1;
  if (n < 0 || n > (1 << 20)) return false;
  if (p->t_now_ns < 0 || p->t_now_ns >= (one << 62)) return false;
  if (p->num_classes < 1 || p->num_classes > 16) return false;
  for (int c = 0; c < p->num_classes; ++c)
    if (p->slo_ns[c] < 0 || p->slo_ns[c] > (one << 50)) return false;
  if (p->block_tokens < 1 || p->block_tokens > (1 << 16)) return false;
  if (p->chunk_tokens < 16 || p->chunk_tokens > (1 << 20)) return false;
  if (p->max_batch < 1 || p->max_batch > 4096) return false;
  if (p->load_decodes < 0 || p->load_decodes > p->max_batch - 1) return false;
  if (p->gamma_q16 < 65536 || p->gamma_q16 > (1 << 20)) return false;
  if (p->c_iter_ps < 0 || p->c_decode_ps < 0 || p->c_token_ps < 0 || p->c_attn_ps < 0)
    return false;
  if (p->c_iter_ps > (one << 36) || p->c_decode_ps > (one << 36)) return false;
  if (p->c_iter_ps + (long long)p->max_batch * p->c_decode_ps > (one << 36)) return false;
  if (p->c_token_ps > (one << 28) || p->c_attn_ps > (one << 16)) return false;
  for (int l = 0; l < 2; ++l) {
    if (p->link_delta_ns[l] < 0 || p->link_delta_ns[l] > (one << 40)) return false;
    if (p->link_blk_ns[l] < 1 || p->link_blk_ns[l] > (one << 32)) return false;
  }
  if (p->token_cap < 1 || p->token_cap > (1 << 24)) return false;
  if (p->tier2_reserve_q16 < 0 || p->tier2_reserve_q16 > 65536) return false;
  if (p->max_move_blocks < 0) return false;
  if (t->num_blocks < 0 || t->n_free < 0 || t->n_free > t->num_blocks) return false;
  return true;
}

// Radix passes launched: the compressed key's width is bounded from the
// parameters alone (every budget lies in [-(L_bound + t_now), max SLO],
// clamped to +-2^61), and the passes are as few as digits of up to kMaxW
// bits allow.  The device spreads the live key width over them; a pass it
// does not need returns at once.
int sort_passes(const cascade_params_t *p) {
  typedef __int128 i128;
  const i128 nmax = 1 << 17;
  const i128 dmax = p->max_batch - 1;
  const i128 per_iter = (i128)p->c_iter_ps + dmax * p->c_decode_ps;
  const i128 iters = (nmax + p->chunk_tokens - 1) / p->chunk_tokens;
  const i128 prefill_ps = iters * per_iter + nmax * p->c_token_ps +
                          (i128)p->c_attn_ps * (nmax * (nmax + 1) / 2);
  const i128 decode_ps = nmax * per_iter;
  const i128 compute_ns = (prefill_ps > decode_ps ? prefill_ps : decode_ps) / 1000 + 1;
  const i128 restore = (i128)p->link_delta_ns[0] + p->link_delta_ns[1] +
                       nmax * ((i128)p->link_blk_ns[0] + p->link_blk_ns[1]);
  const i128 lsum = 2 * (compute_ns + restore);
  const i128 lbound = ((lsum * p->gamma_q16) >> 17) + 1;
  i128 hi = 0;
  for (int c = 0; c < p->num_classes; ++c) hi = p->slo_ns[c] > hi ? p->slo_ns[c] : hi;
  i128 lo = -(lbound + p->t_now_ns);
  const i128 lim = (i128)1 << 61;
  if (lo < -lim) lo = -lim;
  if (hi > lim - 1) hi = lim - 1;
  const i128 span = hi - lo + 1;
  const i128 top = 2 * span + (hi - lo);
  int bits = 0;
  for (i128 v = top; v > 0; v >>= 1) ++bits;
  const int d = (bits + kMaxW - 1) / kMaxW;
  return d < 1 ? 1 : (d > kMaxPasses ? kMaxPasses : d);
}

typedef void (*RadixFn)(int, int, Ctl *, int *, unsigned long long *, unsigned long long *,
                        unsigned *, unsigned *, unsigned *, const int4 *, Sorted, unsigned *,
                        unsigned *);
static_assert(kMaxPasses == 8, "one radix kernel per pass");
template <int kItems>
constexpr RadixFn kRadixPasses[kMaxPasses] = {
    radix_pass_kernel<0, kItems>, radix_pass_kernel<1, kItems>, radix_pass_kernel<2, kItems>,
    radix_pass_kernel<3, kItems>, radix_pass_kernel<4, kItems>, radix_pass_kernel<5, kItems>,
    radix_pass_kernel<6, kItems>, radix_pass_kernel<7, kItems>};

}  // namespace
}  // namespace cascade

using namespace cascade;

extern "C" size_t cascade_step_workspace_bytes(int32_t n) {
  if (n < 0 || n > (1 << 20)) return 0;
  return make_layout(n).total;
}

extern "C" const char *cascade_strerror(int code) {
  switch (code) {
    case CASCADE_OK: return "ok";
    case CASCADE_EINVAL: return "invalid argument or request data";
    case CASCADE_ENOSPC: return "workspace or output list too small";
    case CASCADE_EHIP: return "HIP launch failed";
    case CASCADE_ETIMEOUT: return "cross-workgroup wait timed out";
    case CASCADE_EINTERNAL: return "internal consistency check failed";
    default: return "unknown status";
  }
}

namespace {

// The whole step on a caller's workspace (cascade_step) or on this device's
// fixed array (cascade_step_noalloc).
int step_impl(const cascade_requests_t *rq, const cascade_block_table_t *bt,
              const cascade_tier_state_t *ts, const cascade_params_t *p,
              const cascade_outputs_t *out, void *workspace, size_t workspace_bytes,
              void *stream) {
  if (!rq || !bt || !ts || !p || !out || !workspace) return CASCADE_EINVAL;
  const int n = rq->n;
  if (!params_ok(p, n, ts)) return CASCADE_EINVAL;
  if (!out->info || !bt->row_offsets) return CASCADE_EINVAL;
  if (n > 0 && (!rq->id || !rq->slo_class || !rq->state || !rq->queue_tier ||
                !rq->prefix_tier || !rq->arrival_ns || !rq->n_in || !rq->n_out_pred ||
                !rq->n_prefix || !rq->n_progress || !bt->slots || !out->budget_ns ||
                !out->action || !out->queue_tier_out || !out->tokens_granted ||
                !out->restore_blocks || !out->order || !out->alloc_begin ||
                !out->alloc_count || !out->admitted))
    return CASCADE_EINVAL;
  if (ts->n_free > 0 && !ts->free_slots) return CASCADE_EINVAL;
  if (out->slot_list_capacity < 0 || out->unpack_capacity < 0 || out->pack_capacity < 0)
    return CASCADE_EINVAL;
  if ((out->slot_list_capacity > 0 && !out->slot_list) ||
      (out->unpack_capacity > 0 && !out->unpack_moves) ||
      (out->pack_capacity > 0 && !out->pack_moves))
    return CASCADE_EINVAL;
  if ((out->unpack_hazard == nullptr) != (out->pack_hazard == nullptr)) return CASCADE_EINVAL;
  if (n > 0 && rq->prefix_group && !out->share_leader) return CASCADE_EINVAL;
  if (((uintptr_t)workspace & 255) != 0) return CASCADE_EINVAL;
  const Layout L = make_layout(n);
  if (workspace_bytes < L.total) return CASCADE_ENOSPC;

  Consts c;
  memset(&c, 0, sizeof(c));
  c.t_now = p->t_now_ns;
  c.c_iter = p->c_iter_ps;
  c.c_dec = p->c_decode_ps;
  c.c_tok = p->c_token_ps;
  c.c_attn = p->c_attn_ps;
  // eq:restore_time paths: P(1) = {DRAM->HBM}, P(2) = {NVMe->DRAM, DRAM->HBM}
  c.delta1 = p->link_delta_ns[0];
  c.delta2 = p->link_delta_ns[0] + p->link_delta_ns[1];
  c.blk1 = p->link_blk_ns[0];
  c.blk2 = p->link_blk_ns[0] + p->link_blk_ns[1];
  c.num_classes = p->num_classes;
  c.bt = p->block_tokens;
  c.chunk = p->chunk_tokens;
  c.d = p->load_decodes;
  c.dmax = p->max_batch - 1;
  c.gamma_q16 = p->gamma_q16;
  c.token_cap = p->token_cap;
  c.rho_q16 = p->tier2_reserve_q16;
  c.max_move = p->max_move_blocks;
  c.num_blocks = ts->num_blocks;
  c.n_free = ts->n_free;
  for (int k = 0; k < 16; ++k) c.slo[k] = k < p->num_classes ? p->slo_ns[k] : 0;

  Outs o;
  o.order = out->order;
  o.granted = out->tokens_granted;
  o.restore = out->restore_blocks;
  o.alloc_begin = out->alloc_begin;
  o.alloc_count = out->alloc_count;
  o.admitted = out->admitted;
  o.slot_list = out->slot_list;
  o.action = out->action;
  o.unpack = out->unpack_moves;
  o.pack = out->pack_moves;
  o.unpack_hazard = out->unpack_hazard;
  o.pack_hazard = out->pack_hazard;
  o.share_leader = rq->prefix_group ? out->share_leader : nullptr;
  o.sl_cap = out->slot_list_capacity;
  o.unpack_cap = out->unpack_capacity;
  o.pack_cap = out->pack_capacity;

  char *ws = static_cast<char *>(workspace);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (n == 0) {
    hipLaunchKernelGGL(empty_step_kernel, dim3(1), dim3(kBlock), 0, s, ts->n_free,
                       ts->num_blocks, ts->free_slots, out->info, o);
    return hipGetLastError() == hipSuccess ? CASCADE_OK : CASCADE_EHIP;
  }
  Ctl *ctl = reinterpret_cast<Ctl *>(ws + L.ctl);
  auto *keys_a = reinterpret_cast<unsigned long long *>(ws + L.keys_a);
  auto *keys_b = reinterpret_cast<unsigned long long *>(ws + L.keys_b);
  auto *vals_a = reinterpret_cast<unsigned *>(ws + L.vals_a);
  auto *vals_b = reinterpret_cast<unsigned *>(ws + L.vals_b);
  auto *rec = reinterpret_cast<int4 *>(ws + L.rec);
  auto *partials = reinterpret_cast<Partial *>(ws + L.partials);
  auto *rp_list = reinterpret_cast<RpInfo *>(ws + L.rp_list);
  auto *rlist = reinterpret_cast<RestoreEnt *>(ws + L.restore);
  auto *tile_tot = reinterpret_cast<TileTot *>(ws + L.tile_tot);
  auto *sort_status = reinterpret_cast<unsigned *>(ws + L.sort_status);
  Sorted srt;
  srt.order = reinterpret_cast<unsigned *>(ws + L.s_order);
  srt.rec = reinterpret_cast<int4 *>(ws + L.s_rec);
  auto *l1_tot = reinterpret_cast<unsigned *>(ws + L.scan1);
  auto *l2_status = reinterpret_cast<unsigned long long *>(ws + L.scan2);

  if (n <= kSmallMax) {
    // one workgroup; it checks the free list and the slots itself unless the
    // pool is large enough for that to dominate
    const int in_kernel = ts->num_blocks <= kSmallCheckBlocks;
    hipLaunchKernelGGL(step_small_kernel, dim3(1), dim3(kBlock), 0, s, *rq, bt->row_offsets,
                       bt->slots, ts->free_slots, c, n, in_kernel, ctl, out->info, o,
                       out->budget_ns, out->queue_tier_out, rp_list, rlist, tile_tot);
    if (!in_kernel)
      hipLaunchKernelGGL(check_lists_kernel, dim3(kCheckGrid), dim3(kBlock), 0, s, n,
                         ts->num_blocks, ts->n_free, ts->free_slots, bt->row_offsets, bt->slots,
                         out->info);
    return hipGetLastError() == hipSuccess ? CASCADE_OK : CASCADE_EHIP;
  }
  // histograms, level-1 totals and the launched passes' look-back words:
  // cleared by eval
  const int passes = sort_passes(p);
  const size_t clear_off = L.ctl + offsetof(Ctl, hist);
  const int tile_keys =
      n <= kTinyTileMax ? kSortTileTiny : (n <= kSmallTileMax ? kSortTileSmall : kSortTile);
  const int sort_tiles = (n + tile_keys - 1) / tile_keys;
  const size_t clear_end = L.sort_status + (size_t)passes * sort_tiles * kMaxBins * 4;
  const size_t clear_vec = (clear_end - clear_off) / 16;
  uint4 *clear = reinterpret_cast<uint4 *>(ws + clear_off);
  static_assert(offsetof(Ctl, hist) % 16 == 0, "16-byte clears");
  const bool share = rq->prefix_group != nullptr;
  auto *share_lead = reinterpret_cast<unsigned *>(ws + L.share_lead);
  auto *share_rl = reinterpret_cast<unsigned *>(ws + L.share_rl);
  auto *share_adj = reinterpret_cast<unsigned *>(ws + L.share_adj);
  auto *share_pub = reinterpret_cast<unsigned *>(ws + L.share_pub);
  // both share tables (2n words each) and the published wants, one 16-byte
  // clear region
  const size_t clear2_vec = share ? (L.share_adj - L.share_lead) / 16 : 0;

  hipLaunchKernelGGL(eval_kernel, dim3(L.eval_grid), dim3(kBlock), 0, s, *rq, bt->row_offsets,
                     ts->free_slots, c, n, ctl, clear, clear_vec,
                     reinterpret_cast<uint4 *>(ws + L.share_lead), clear2_vec, out->info,
                     partials, out->budget_ns, out->queue_tier_out, keys_a, rec);
  // a short queue spreads prep over more workgroups (its block-table checks
  // and histograms are per workgroup); a long one keeps the global adds few
  const int prep_items = n <= kTinyPrepMax ? 2 : kPrepItems;
  const int prep_grid = (n + kBlock * prep_items - 1) / (kBlock * prep_items);
  hipLaunchKernelGGL(prep_items == 2 ? prep_kernel<2> : prep_kernel<kPrepItems>, dim3(prep_grid),
                     dim3(kBlock), 0, s, n, ts->num_blocks, L.eval_grid, passes, partials,
                     bt->row_offsets, bt->slots, ctl, out->info, keys_a, vals_a);
  for (int pass = 0; pass < passes; ++pass)
    hipLaunchKernelGGL(tile_keys == kSortTileTiny    ? kRadixPasses<kSortItems / 4>[pass]
                       : tile_keys == kSortTileSmall ? kRadixPasses<kSortItems / 2>[pass]
                                                     : kRadixPasses<kSortItems>[pass],
                       dim3(sort_tiles), dim3(kSortBlock), 0, s, n,
                       passes, ctl, out->info, keys_a, keys_b, vals_a, vals_b,
                       sort_status + (size_t)pass * sort_tiles * kMaxBins, rec, srt,
                       l1_tot, share ? share_lead : nullptr);
  if (share)
    hipLaunchKernelGGL(share_kernel, dim3(L.scan_tiles), dim3(kBlock), 0, s, n, L.scan_tiles,
                       c.bt, c.max_move, ctl, out->info, srt, rec, l1_tot, share_lead, share_rl,
                       share_adj, share_pub);
  hipLaunchKernelGGL(scan_kernel, dim3(L.scan_tiles + kFinishGrid), dim3(kBlock), 0, s, n,
                     passes, L.scan_tiles, c, ctl, out->info, srt, rec, bt->slots,
                     ts->free_slots, o, rp_list, rlist, tile_tot, l1_tot,
                     share ? share_adj : nullptr, l2_status);
  if (hipGetLastError() != hipSuccess) return CASCADE_EHIP;
  return CASCADE_OK;
}

}  // namespace

extern "C" int cascade_step(const cascade_requests_t *rq, const cascade_block_table_t *bt,
                            const cascade_tier_state_t *ts, const cascade_params_t *p,
                            const cascade_outputs_t *out, void *workspace,
                            size_t workspace_bytes, void *stream) {
  return step_impl(rq, bt, ts, p, out, workspace, workspace_bytes, stream);
}

// ------------------------------------------------ step without a workspace

// The workspace of cascade_step_noalloc: one fixed array per GPU, sized for
// CASCADE_NOALLOC_MAX_REQUESTS requests and held until the process ends.
// Its name is a host-side stand-in, not a device address: host code only
// ever passes the address hipGetSymbolAddress returns for the current device.
static constexpr size_t kScratchBytes = make_layout(CASCADE_NOALLOC_MAX_REQUESTS).total;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {
constexpr int kScratchDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_addr[kScratchDevices];  // device address of `scratch`, per GPU

// This GPU's copy of `scratch`: looked up once per device, with that device
// current (every GPU holds the array at its own address).
int scratch_of_current_device(void **addr) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kScratchDevices) return CASCADE_EHIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_addr[dev] == nullptr) {
    void *a = nullptr;
    if (hipGetSymbolAddress(&a, HIP_SYMBOL(scratch)) != hipSuccess || a == nullptr)
      return CASCADE_EHIP;
    g_scratch_addr[dev] = a;
  }
  *addr = g_scratch_addr[dev];
  return CASCADE_OK;
}
}  // namespace

extern "C" int cascade_step_noalloc(const cascade_requests_t *rq,
                                    const cascade_block_table_t *bt,
                                    const cascade_tier_state_t *ts, const cascade_params_t *p,
                                    const cascade_outputs_t *out, void *stream) {
  if (!rq) return CASCADE_EINVAL;
  if (rq->n > CASCADE_NOALLOC_MAX_REQUESTS) return CASCADE_ENOSPC;
  void *ws = nullptr;
  const int rc = scratch_of_current_device(&ws);
  if (rc != CASCADE_OK) return rc;
  return step_impl(rq, bt, ts, p, out, ws, kScratchBytes, stream);
}
