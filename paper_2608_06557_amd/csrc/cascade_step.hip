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
// The paper's scheduler is a sequential CPU loop.  Here every step of it is
// a data-parallel kernel:
//   eval      one lane per request: budget, tier, restore want, priority key
//   prep      key compression to the live budget range + digit histograms
//   radix     onesweep LSD radix passes (wave64 ballot ranking, decoupled
//             look-back per digit), constant digits skipped on the device
//   scan      the sequential loop as prefix sums in priority order, with a
//             two-level chained decoupled look-back in one launch
//   finalize  preemption victims, slot list, spill (pack) moves
//   moves     restore (unpack) moves and final counts
// All arithmetic is 64-bit integer, so the result is bit-exact.
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>

#include "cascade.h"
#include "device_util.h"

namespace cascade {
namespace {

constexpr int kSortItems = 8;
constexpr int kSortTile = kBlock * kSortItems;
constexpr int kScanItems = 4;
constexpr int kScanTile = kBlock * kScanItems;
constexpr int kPrepItems = 16;
constexpr int kRadix = 256;
constexpr int kMaxDigits = 8;
constexpr int kLookWin = 8;
constexpr int kL1 = 4;  // first-level scan values
constexpr int kL2 = 7;  // second-level scan values
constexpr int kL2Stride = 8;

// Record of one request for the priority-order scan (16 bytes).
//   x want_blocks, y base_need, z reuse_tokens (HBM prefix or progress)
//   w bits 0..19 held blocks, 20..21 state, 22..23 prefix tier,
//     24..25 group, 26 spill-fits-budget, 27 decode needs a new block
__device__ __forceinline__ int rec_held(int w) { return w & 0xFFFFF; }
__device__ __forceinline__ int rec_state(int w) { return (w >> 20) & 3; }
__device__ __forceinline__ int rec_tier(int w) { return (w >> 22) & 3; }
__device__ __forceinline__ int rec_offl(int w) { return (w >> 26) & 1; }
__device__ __forceinline__ int rec_decnb(int w) { return (w >> 27) & 1; }

struct RpInfo {          // per running prefill, written by scan
  int pos, eligible;
  long long x, y, z, zp;  // inclusive prefixes at pos
};
struct RestoreEnt { int req, stage_off, alloc_off, blocks; };

// Device control block.  The header is written by one thread of the init
// kernel; the histograms are cleared by all of its threads.
struct Ctl {
  unsigned long long bmin, bmax;   // range of the biased, clamped budget
  long long held_rp;               // blocks held by running prefills (H)
  long long need1, want1;          // base need and want over decode+Tier-1
  unsigned cnt[4];                 // requests per priority group
  unsigned rp_count;
  unsigned tile_ctr[kMaxDigits + 1];
  int kstar;                       // first position that does not fit
  int pad0;
  long long kx, ky, kz, kzp;       // prefixes just before kstar
  long long adm_nb, elig_h, elig_offl_h, n_adm, n_unpack, n_restore;
  long long pad1[4];
  alignas(16) unsigned hist[kMaxDigits][kRadix];
};
constexpr size_t kCtlHeaderWords = offsetof(Ctl, hist) / 4;

struct Consts {           // parameters the kernels use, flattened
  long long t_now, c_iter, c_dec, c_tok, c_attn;
  long long delta1, delta2, blk1, blk2;  // restore paths: DRAM, NVMe
  int num_classes, bt, chunk, d, dmax, gamma_q16, token_cap, rho_q16, max_move;
  int num_blocks, n_free;
  long long slo[16];
};

// Workgroup-uniform: true if an earlier kernel (or a workgroup of this one)
// reported bad data or a timeout.  Every thread of the workgroup must call it.
__device__ __forceinline__ bool status_failed(const int *info) {
  int bad = 0;
  if (threadIdx.x == 0) {
    const int s = load_agent(info);
    bad = (s == CASCADE_EINVAL || s == CASCADE_ETIMEOUT || s == CASCADE_EINTERNAL);
  }
  return __syncthreads_or(bad) != 0;
}
__device__ __forceinline__ long long lmin(long long a, long long b) { return a < b ? a : b; }
__device__ __forceinline__ void set_status(int *info, int code) { store_agent(info, code); }

// ---------------------------------------------------------------- eval

// Iteration cost model of the TTFT estimator (Section 4.2): n prompt tokens
// at positions s.. with dd co-scheduled decodes, picoseconds.
__device__ __forceinline__ long long compute_ps(long long n, long long s, long long dd,
                                                const Consts &c) {
  if (n <= 0) return 0;
  const long long iters = (long long)(((unsigned)n + (unsigned)c.chunk - 1u) / (unsigned)c.chunk);
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

__global__ __launch_bounds__(kBlock) void eval_kernel(
    cascade_requests_t rq, const int *__restrict__ ro, const int *__restrict__ free_slots,
    Consts c, int n, Ctl *ctl, int *info, int64_t *__restrict__ budget_out,
    uint8_t *__restrict__ tier_out, unsigned long long *__restrict__ keys,
    int4 *__restrict__ rec, int *__restrict__ rp_list) {
  __shared__ long long s_slo[16];
  __shared__ long long s_red[kWaves * 4];
  __shared__ unsigned long long s_mm[kWaves * 2];
  __shared__ unsigned s_cnt[kWaves * 3];
  if (threadIdx.x < 16) s_slo[threadIdx.x] = c.slo[threadIdx.x];
  __syncthreads();

  const int i = blockIdx.x * kBlock + threadIdx.x;
  const bool live = i < n;
  bool bad = false;
  long long v_held = 0, v_need1 = 0, v_want1 = 0;
  unsigned long long bmin = ~0ull, bmax = 0;
  int grp = 3;
  bool is_rp = false;

  // free-list range check, spread over the grid
  for (int j = i; j < c.n_free; j += gridDim.x * kBlock)
    if ((unsigned)free_slots[j] >= (unsigned)c.num_blocks) bad = true;

  if (live) {
    const unsigned cls = rq.slo_class[i], st = rq.state[i], qt = rq.queue_tier[i],
                   pt = rq.prefix_tier[i];
    const long long arr = rq.arrival_ns[i];
    long long n_in = rq.n_in[i], n_out = rq.n_out_pred[i], n_pre = rq.n_prefix[i],
              prog = rq.n_progress[i];
    const long long row = (long long)ro[i + 1] - (long long)ro[i];
    const long long bt = c.bt;

    // ---- domain rules of the request data
    if (i > 0 && rq.id[i] <= rq.id[i - 1]) bad = true;
    if (i == 0 && ro[0] != 0) bad = true;
    if (cls >= (unsigned)c.num_classes || st > 2 || qt > 2 || pt > 3) bad = true;
    if (n_in < 1 || n_in > (1 << 17) || n_out < 0 || n_out > (1 << 17)) bad = true;
    if (n_pre < 0 || n_pre > n_in - 1 || (n_pre % bt) != 0) bad = true;
    if (arr < 0 || arr > c.t_now) bad = true;
    long long want_row;
    if (st == CASCADE_QUEUED) {
      if ((n_pre == 0) != (pt == CASCADE_KV_NONE) || prog != 0) bad = true;
      want_row = 0;
    } else if (st == CASCADE_RUNNING_PREFILL) {
      if (prog < 1 || prog > n_in - 1) bad = true;
      want_row = (prog + bt - 1) / bt;
    } else {
      if (prog < 0 || prog > (1 << 17)) bad = true;
      want_row = (n_in + prog + bt - 1) / bt;
    }
    if (row != want_row) bad = true;

    // ---- keep the arithmetic in range whatever the data
    const unsigned st_s = st > 2 ? 0u : st;
    const unsigned pt_s = pt > 3 ? 3u : pt;
    const unsigned cls_s = cls >= (unsigned)c.num_classes ? 0u : cls;
    n_in = n_in < 1 ? 1 : (n_in > (1 << 17) ? (1 << 17) : n_in);
    n_out = n_out < 0 ? 0 : (n_out > (1 << 17) ? (1 << 17) : n_out);
    n_pre = n_pre < 0 ? 0 : (n_pre > n_in - 1 ? n_in - 1 : n_pre);
    prog = prog < 0 ? 0 : (prog > (1 << 17) ? (1 << 17) : prog);
    const long long elapsed = (arr < 0 || arr > c.t_now) ? 0 : c.t_now - arr;
    const long long held = row < 0 ? 0 : (row > 0xFFFFF ? 0xFFFFF : row);

    // ---- Section 4.2: actual-load and maximum-load estimates
    long long l_act, l_max, pb = 0, base_need;
    const long long delta = (pt_s == CASCADE_KV_NVME) ? c.delta2 : c.delta1;
    const long long blk = (pt_s == CASCADE_KV_NVME) ? c.blk2 : c.blk1;
    const bool deep = (pt_s == CASCADE_KV_DRAM || pt_s == CASCADE_KV_NVME);
    if (st_s == CASCADE_QUEUED) {
      long long reuse = 0, rest = 0;
      if (pt_s != CASCADE_KV_NONE) {
        pb = n_pre / bt;
        reuse = n_pre;
        if (deep) rest = restore_ns(pb, delta, blk);
      }
      l_act = ns_of_ps(compute_ps(n_in - reuse, reuse, c.d, c)) + rest;
      l_max = ns_of_ps(compute_ps(n_in - reuse, reuse, c.dmax, c)) + rest;
      base_need = (pt_s == CASCADE_KV_HBM) ? n_in - n_pre : n_in;
    } else if (st_s == CASCADE_RUNNING_PREFILL) {
      const long long left = n_in - prog < 0 ? 0 : n_in - prog;
      l_act = ns_of_ps(compute_ps(left, prog, c.d, c));
      l_max = ns_of_ps(compute_ps(left, prog, c.dmax, c));
      base_need = left;
    } else {
      const long long left = n_out - prog < 0 ? 0 : n_out - prog;
      l_act = ns_of_ps(left * (c.c_iter + (long long)c.d * c.c_dec));
      l_max = ns_of_ps(left * (c.c_iter + (long long)c.dmax * c.c_dec));
      base_need = 1;
    }
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
        const long long m = (long long)((unsigned long long)(brem - delta) / (unsigned long long)blk);
        x = m < pb ? m : pb;
      }
      if (x > 0) {
        const long long all = ns_of_ps(compute_ps(n_in, 0, c.d, c));
        const long long part = ns_of_ps(compute_ps(n_in - bt * x, bt * x, c.d, c));
        if (restore_ns(x, delta, blk) >= all - part) x = 0;
      }
      want = x;
    }

    // ---- priority group and key: group in bits 63..62, clamped budget + 2^61
    grp = (st_s == CASCADE_DECODE) ? 0 : (tnew == 1 ? 1 : 2);
    const long long lo = -(1ll << 61), hi = (1ll << 61) - 1;
    const long long cl = brem < lo ? lo : (brem > hi ? hi : brem);
    const unsigned long long biased = (unsigned long long)(cl + (1ll << 61));
    bmin = bmax = biased;

    // spill of a running prefill fits its budget (Section 4.4)
    const int offl = (st_s == CASCADE_RUNNING_PREFILL) &&
                     (restore_ns(held, c.delta1, c.blk1) <= brem);
    const int decnb = (st_s == CASCADE_DECODE) && ((n_in + prog + 1 + bt - 1) / bt - held) > 0;
    const long long reuse_tok = (st_s == CASCADE_RUNNING_PREFILL)
                                    ? prog
                                    : ((st_s == CASCADE_QUEUED && pt_s == CASCADE_KV_HBM) ? n_pre : 0);

    budget_out[i] = brem;
    tier_out[i] = (uint8_t)tnew;
    keys[i] = ((unsigned long long)grp << 62) | biased;
    rec[i] = make_int4((int)want, (int)base_need, (int)reuse_tok,
                       (int)held | ((int)st_s << 20) | ((int)pt_s << 22) | (grp << 24) |
                           (offl << 26) | (decnb << 27));
    is_rp = (st_s == CASCADE_RUNNING_PREFILL);
    if (is_rp) v_held = held;
    if (grp <= 1) {
      v_need1 = base_need;
      v_want1 = want;
    }
  }

  if (__syncthreads_or(bad ? 1 : 0)) {
    if (threadIdx.x == 0) set_status(info, CASCADE_EINVAL);
  }

  // running-prefill list (wave-aggregated append)
  const uint64_t rpm = __ballot(is_rp);
  if (rpm) {
    unsigned base = 0;
    if (lane_id() == __builtin_ctzll(rpm))
      base = atomicAdd(&ctl->rp_count, (unsigned)__builtin_popcountll(rpm));
    base = __shfl(base, __builtin_ctzll(rpm), 64);
    if (is_rp) rp_list[base + rank_in_mask(rpm)] = i;
  }

  // workgroup reductions, one atomic each
  long long sums[3] = {v_held, v_need1, v_want1};
  block_sum<3>(sums, s_red);
  unsigned cnt[3] = {grp == 0 ? 1u : 0u, grp == 1 ? 1u : 0u, grp == 2 ? 1u : 0u};
  block_sum<3>(cnt, s_cnt);
  for (int o = 32; o >= 1; o >>= 1) {
    const unsigned long long a = __shfl_xor(bmin, o, 64), b = __shfl_xor(bmax, o, 64);
    bmin = a < bmin ? a : bmin;
    bmax = b > bmax ? b : bmax;
  }
  if (lane_id() == 0) {
    s_mm[wave_id() * 2] = bmin;
    s_mm[wave_id() * 2 + 1] = bmax;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned long long mn = ~0ull, mx = 0;
    for (int w = 0; w < kWaves; ++w) {
      mn = s_mm[2 * w] < mn ? s_mm[2 * w] : mn;
      mx = s_mm[2 * w + 1] > mx ? s_mm[2 * w + 1] : mx;
    }
    if (sums[0]) atomicAdd((unsigned long long *)&ctl->held_rp, (unsigned long long)sums[0]);
    if (sums[1]) atomicAdd((unsigned long long *)&ctl->need1, (unsigned long long)sums[1]);
    if (sums[2]) atomicAdd((unsigned long long *)&ctl->want1, (unsigned long long)sums[2]);
    for (int k = 0; k < 3; ++k)
      if (cnt[k]) atomicAdd(&ctl->cnt[k], cnt[k]);
    if (mn <= mx) {
      atomicMin(&ctl->bmin, mn);
      atomicMax(&ctl->bmax, mx);
    }
  }
}

// ------------------------------------------------------ sort: digit plan

struct Plan {
  unsigned long long span;  // bmax - bmin + 1
  int digits;               // 8-bit digits of the compressed key
};
__device__ __forceinline__ Plan make_plan(const Ctl *ctl) {
  Plan p;
  const unsigned long long mn = ctl->bmin, mx = ctl->bmax;
  p.span = mx - mn + 1;
  const unsigned long long gmax = ctl->cnt[2] ? 2 : (ctl->cnt[1] ? 1 : 0);
  const unsigned long long top = gmax * p.span + (mx - mn);
  const int bits = top ? 64 - __builtin_clzll(top) : 0;
  p.digits = (bits + 7) / 8;
  return p;
}

// True when digit d has one value for all n keys (the pass keeps the order).
__device__ __forceinline__ bool digit_constant(const Ctl *ctl, int d, int n) {
  int hit = 0;
  for (int b = threadIdx.x; b < kRadix; b += kBlock) hit |= (ctl->hist[d][b] == (unsigned)n);
  return __syncthreads_or(hit) != 0;
}

// Number of data-moving passes among digits < upto (selects the ping-pong
// buffer).
__device__ __forceinline__ int moving_passes(const Ctl *ctl, const Plan &pl, int upto, int n) {
  int m = 0;
  for (int d = 0; d < upto && d < pl.digits; ++d) m += digit_constant(ctl, d, n) ? 0 : 1;
  return m;
}

// ---------------------------------------------------------------- prep

// Order-preserving key compression: key' = group * span + (biased - bmin),
// then one read of the keys builds every digit's histogram.  Also checks the
// block-table slots, whose extent is only trustworthy after eval.
__global__ __launch_bounds__(kBlock) void prep_kernel(int n, int num_blocks,
                                                      const int *__restrict__ ro,
                                                      const int *__restrict__ slots, Ctl *ctl,
                                                      int *info,
                                                      unsigned long long *__restrict__ keys,
                                                      unsigned *__restrict__ vals) {
  __shared__ unsigned s_hist[kMaxDigits][kRadix];
  if (status_failed(info)) return;
  const int nnz = ro[n];
  bool bad = false;
  for (int j = blockIdx.x * kBlock + threadIdx.x; j < nnz; j += gridDim.x * kBlock)
    if ((unsigned)slots[j] >= (unsigned)num_blocks) bad = true;
  if (__syncthreads_or(bad ? 1 : 0)) {
    if (threadIdx.x == 0) set_status(info, CASCADE_EINVAL);
  }

  const Plan pl = make_plan(ctl);
  const unsigned long long mn = ctl->bmin;
  for (int t = threadIdx.x; t < kMaxDigits * kRadix; t += kBlock) (&s_hist[0][0])[t] = 0;
  __syncthreads();
  const int base = blockIdx.x * kBlock * kPrepItems;
#pragma unroll 4
  for (int j = 0; j < kPrepItems; ++j) {
    const int idx = base + j * kBlock + threadIdx.x;
    if (idx < n) {
      const unsigned long long k0 = keys[idx];
      const unsigned long long k =
          (k0 >> 62) * pl.span + ((k0 & ((1ull << 62) - 1)) - mn);
      keys[idx] = k;
      vals[idx] = (unsigned)idx;
      for (int d = 0; d < pl.digits; ++d) atomicAdd(&s_hist[d][(k >> (8 * d)) & 255], 1u);
    }
  }
  __syncthreads();
  for (int d = 0; d < pl.digits; ++d) {
    const unsigned v = s_hist[d][threadIdx.x];
    if (v) atomicAdd(&ctl->hist[d][threadIdx.x], v);
  }
}

// ---------------------------------------------------------- radix pass

// One stable LSD pass over 8 bits.  A tile of kSortTile keys is ranked per
// wave with ballots (lanes holding the same digit find each other in 8
// ballots), per-digit tile counts are published for the decoupled look-back,
// keys are reordered in LDS and written out in runs of equal digits.
__global__ __launch_bounds__(kBlock) void radix_pass_kernel(
    int pass, int n, Ctl *ctl, int *info, unsigned long long *keys_a,
    unsigned long long *keys_b, unsigned *vals_a, unsigned *vals_b, unsigned *status) {
  __shared__ unsigned long long s_keys[kSortTile];
  __shared__ unsigned s_vals[kSortTile];
  __shared__ unsigned s_wcnt[kWaves][kRadix];
  __shared__ int s_start[kRadix];
  __shared__ int s_off[kRadix];
  __shared__ int s_scan[kWaves * 2];
  __shared__ int s_tile;

  if (status_failed(info)) return;
  const Plan pl = make_plan(ctl);
  if (pass >= pl.digits) return;
  if (digit_constant(ctl, pass, n)) return;
  const int parity = moving_passes(ctl, pl, pass, n) & 1;
  const unsigned long long *src_k = parity ? keys_b : keys_a;
  unsigned long long *dst_k = parity ? keys_a : keys_b;
  const unsigned *src_v = parity ? vals_b : vals_a;
  unsigned *dst_v = parity ? vals_a : vals_b;

  if (threadIdx.x == 0) s_tile = (int)atomicAdd(&ctl->tile_ctr[pass], 1u);
  for (int t = threadIdx.x; t < kWaves * kRadix; t += kBlock) (&s_wcnt[0][0])[t] = 0;
  __syncthreads();
  const int tile = s_tile;
  const int shift = 8 * pass;
  const int lane = lane_id(), wave = wave_id();
  const int tile_base = tile * kSortTile;

  unsigned long long key[kSortItems];
  unsigned val[kSortItems];
  int dig[kSortItems], rank[kSortItems];
#pragma unroll
  for (int j = 0; j < kSortItems; ++j) {
    const int g = tile_base + wave * 64 * kSortItems + j * 64 + lane;
    const bool v = g < n;
    key[j] = v ? src_k[g] : 0ull;
    val[j] = v ? src_v[g] : 0u;
    dig[j] = v ? (int)((key[j] >> shift) & 255) : -1;
  }
  // rank within the wave, item by item (local order: wave, item, lane)
#pragma unroll
  for (int j = 0; j < kSortItems; ++j) {
    const bool v = dig[j] >= 0;
    uint64_t peers = __ballot(v);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const bool bit = (dig[j] >> b) & 1;
      const uint64_t bal = __ballot(bit);
      peers &= bit ? bal : ~bal;
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

  // per-digit totals of the tile (thread t = digit t)
  const int t = threadIdx.x;
  unsigned run = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const unsigned c = s_wcnt[w][t];
    s_wcnt[w][t] = run;
    run += c;
  }
  const unsigned tile_count = run;
  unsigned *st = status + (size_t)tile * kRadix;
  bool timed_out = false;
  publish<unsigned>(st + t, tile_count, tile == 0 ? kFlagInclusive : kFlagAggregate);

  // exclusive scans over digits: tile-local starts and global bases
  int v2[2] = {(int)tile_count, (int)ctl->hist[pass][t]};
  int tot2[2];
  block_exclusive_scan<2>(v2, tot2, s_scan);
  s_start[t] = v2[0];
  unsigned prefix = 0;
  if (tile > 0) {
    prefix = look_back<unsigned, kLookWin>(status, kRadix, tile, t, &timed_out);
    publish<unsigned>(st + t, prefix + tile_count, kFlagInclusive);
  }
  if (timed_out) set_status(info, CASCADE_ETIMEOUT);
  s_off[t] = v2[1] + (int)prefix - v2[0];
  __syncthreads();

  bool broken = false;
#pragma unroll
  for (int j = 0; j < kSortItems; ++j) {
    if (dig[j] >= 0) {
      const int pos = s_start[dig[j]] + (int)s_wcnt[wave][dig[j]] + rank[j];
      if ((unsigned)pos < (unsigned)kSortTile) {
        s_keys[pos] = key[j];
        s_vals[pos] = val[j];
      } else {
        broken = true;
      }
    }
  }
  __syncthreads();
  const int count = min(kSortTile, n - tile_base);
  for (int s = threadIdx.x; s < count; s += kBlock) {
    const unsigned long long k = s_keys[s];
    const int o = s_off[(k >> shift) & 255] + s;
    if ((unsigned)o < (unsigned)n) {
      dst_k[o] = k;
      dst_v[o] = s_vals[s];
    } else {
      broken = true;
    }
  }
  if (broken) set_status(info, CASCADE_EINTERNAL);
}

// ---------------------------------------------------------------- scan

// Algorithm 1's Phase 2 loop in priority order as prefix sums.
// Level 1 (independent of earlier decisions): restore want, base token need,
// blocks held by running prefills (all / spill-fits).  They give the restore
// blocks r (eq:max_restorable under the per-step cap U), the exact token need
// and the chunked-prefill grant g of every position.
// Level 2 (functions of g): block weight of the admission test, new blocks
// of admitted requests, admitted count, held blocks of running prefills left
// out (all / spill-fits), restored blocks and restoring requests.
// Both levels use one decoupled look-back each, chained inside the launch.
__global__ __launch_bounds__(kBlock) void scan_kernel(
    int n, Consts c, Ctl *ctl, int *info, const unsigned *vals_a, const unsigned *vals_b,
    const int4 *__restrict__ rec, int *__restrict__ order_out, int *__restrict__ granted_out,
    int *__restrict__ restore_out, int *__restrict__ alloc_begin, int *__restrict__ alloc_count,
    uint8_t *__restrict__ action_out, int *__restrict__ admitted_out, RpInfo *__restrict__ rp_info,
    RestoreEnt *__restrict__ restore_list, unsigned long long *status1,
    unsigned long long *status2) {
  __shared__ long long s_scan[kWaves * kL2];
  __shared__ long long s_pre[kL2Stride];
  __shared__ int s_tile;

  if (status_failed(info)) return;
  if (threadIdx.x == 0) {
    s_tile = (int)atomicAdd(&ctl->tile_ctr[kMaxDigits], 1u);
  }
  const Plan pl = make_plan(ctl);
  const int par = moving_passes(ctl, pl, pl.digits, n) & 1;
  __syncthreads();
  const int tile = s_tile;
  const unsigned *sorted = par ? vals_b : vals_a;
  const long long bt = c.bt, U = c.max_move;
  const long long e1 = (long long)ctl->cnt[0] + ctl->cnt[1];
  const bool has2 = ctl->cnt[2] != 0;
  const long long cap = c.token_cap;
  const long long cap1 = cap - (has2 ? ((cap * c.rho_q16) >> 16) : 0);
  const long long p_e1 = ctl->need1 - bt * lmin(ctl->want1, U);  // tokens before Tier-2
  const long long g1 = lmin(p_e1, cap1);                           // granted to decode+Tier-1
  const long long fh = (long long)c.n_free + ctl->held_rp;        // F + H

  const int p0 = tile * kScanTile + threadIdx.x * kScanItems;
  int idx[kScanItems];
  int4 r4[kScanItems];
#pragma unroll
  for (int j = 0; j < kScanItems; ++j) {
    const int p = p0 + j;
    int ix = p < n ? (int)sorted[p] : -1;
    if (ix >= n) {  // cannot happen with a correct sort; never read out of range
      set_status(info, CASCADE_EINTERNAL);
      ix = -1;
    }
    idx[j] = ix;
    r4[j] = ix >= 0 ? rec[ix] : make_int4(0, 0, 0, 0);
  }

  // ---- level 1
  long long l1[kL1] = {0, 0, 0, 0}, t1[kL1];
#pragma unroll
  for (int j = 0; j < kScanItems; ++j) {
    const int w = r4[j].w;
    const long long h = rec_state(w) == CASCADE_RUNNING_PREFILL ? rec_held(w) : 0;
    l1[0] += r4[j].x;
    l1[1] += r4[j].y;
    l1[2] += h;
    l1[3] += rec_offl(w) ? h : 0;
  }
  block_exclusive_scan<kL1>(l1, t1, s_scan);
  bool timed_out = false;
  unsigned long long *st1 = status1 + (size_t)tile * kL1;
  if (threadIdx.x < kL1)
    publish<unsigned long long>(st1 + threadIdx.x, (unsigned long long)t1[threadIdx.x],
                                tile == 0 ? kFlagInclusive : kFlagAggregate);
  if (threadIdx.x < kL1) {
    long long pre = 0;
    if (tile > 0) {
      pre = (long long)look_back<unsigned long long, kLookWin>(status1, kL1, tile,
                                                                threadIdx.x, &timed_out);
      publish<unsigned long long>(st1 + threadIdx.x, (unsigned long long)(pre + t1[threadIdx.x]),
                                  kFlagInclusive);
    }
    s_pre[threadIdx.x] = pre;
  }
  __syncthreads();
  long long wx = s_pre[0] + l1[0], bn = s_pre[1] + l1[1], yy = s_pre[2] + l1[2],
            zz = s_pre[3] + l1[3];
  __syncthreads();

  // ---- per position: restore blocks, need, grant, new blocks
  long long r[kScanItems], g[kScanItems], nb[kScanItems], hh[kScanItems];
  long long y_inc[kScanItems], zp_inc[kScanItems];
  long long l2[kL2] = {0, 0, 0, 0, 0, 0, 0}, t2[kL2];
#pragma unroll
  for (int j = 0; j < kScanItems; ++j) {
    const int w = r4[j].w;
    const int st = rec_state(w);
    const long long want = r4[j].x;
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
      if (st == CASCADE_QUEUED) {
        const int tier = rec_tier(w);
        if (tier == CASCADE_KV_HBM) {
          const long long s = r4[j].z;
          nbj = (s + gj + bt - 1) / bt - s / bt;
        } else {
          nbj = rj + (gj + bt - 1) / bt;
        }
      } else if (st == CASCADE_RUNNING_PREFILL) {
        nbj = ((long long)r4[j].z + gj + bt - 1) / bt - rec_held(w);
      } else {
        nbj = rec_decnb(w);
      }
    }
    r[j] = rj;
    g[j] = gj;
    nb[j] = nbj;
    hh[j] = h;
    wx += want;
    bn += r4[j].y;
    yy += h;
    zz += rec_offl(w) ? h : 0;
    y_inc[j] = yy;
    zp_inc[j] = zz;
    const bool gp = gj > 0;
    l2[0] += gp ? nbj + h : 0;              // admission weight
    l2[1] += gp ? nbj : 0;                  // new blocks
    l2[2] += gp ? 1 : 0;                    // admitted count
    l2[3] += gp ? 0 : h;                    // held, not granted
    l2[4] += (gp || !rec_offl(w)) ? 0 : h;  // held, not granted, spill fits
    l2[5] += gp ? rj : 0;                   // restored blocks
    l2[6] += (gp && rj > 0) ? 1 : 0;        // restoring requests
  }

  // ---- level 2
  block_exclusive_scan<kL2>(l2, t2, s_scan);
  unsigned long long *st2 = status2 + (size_t)tile * kL2Stride;
  if (threadIdx.x < kL2)
    publish<unsigned long long>(st2 + threadIdx.x, (unsigned long long)t2[threadIdx.x],
                                tile == 0 ? kFlagInclusive : kFlagAggregate);
  if (threadIdx.x < kL2) {
    long long pre = 0;
    if (tile > 0) {
      pre = (long long)look_back<unsigned long long, kLookWin>(status2, kL2Stride, tile,
                                                                threadIdx.x, &timed_out);
      publish<unsigned long long>(st2 + threadIdx.x, (unsigned long long)(pre + t2[threadIdx.x]),
                                  kFlagInclusive);
    }
    s_pre[threadIdx.x] = pre;
  }
  if (__syncthreads_or(timed_out ? 1 : 0)) {
    if (threadIdx.x == 0) set_status(info, CASCADE_ETIMEOUT);
  }
  long long W = s_pre[0] + l2[0], NB = s_pre[1] + l2[1], AC = s_pre[2] + l2[2],
            X = s_pre[3] + l2[3], Z = s_pre[4] + l2[4], RR = s_pre[5] + l2[5],
            RC = s_pre[6] + l2[6];

  long long a_nb = 0, a_eh = 0, a_eoh = 0, a_n = 0, a_r = 0, a_rc = 0;
#pragma unroll
  for (int j = 0; j < kScanItems; ++j) {
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
      ctl->kstar = p;
      ctl->kx = X;
      ctl->ky = y_inc[j] - hh[j];
      ctl->kz = Z;
      ctl->kzp = zp_inc[j] - (rec_offl(w) ? hh[j] : 0);
    }
    order_out[p] = i;
    granted_out[i] = adm ? (int)g[j] : 0;
    restore_out[i] = (int)r[j];
    alloc_begin[i] = adm ? (int)NB : -1;
    alloc_count[i] = adm ? (int)nb[j] : 0;
    int act;
    if (st != CASCADE_QUEUED) {
      act = CASCADE_ACT_RETAIN;  // a preempted running prefill is rewritten later
    } else {
      const int tier = rec_tier(w);
      if (tier == CASCADE_KV_HBM) act = CASCADE_ACT_RETAIN;
      else if (tier == CASCADE_KV_NONE || r[j] == 0) act = CASCADE_ACT_RECOMPUTE;
      else act = adm ? CASCADE_ACT_RESTORE : CASCADE_ACT_PREFETCH;
    }
    action_out[i] = (uint8_t)act;
    if (adm) {
      admitted_out[AC] = i;
      a_nb += nb[j];
      a_n += 1;
      if (r[j] > 0) {
        RestoreEnt e;
        e.req = i;
        e.stage_off = (int)RR;
        e.alloc_off = (int)NB;
        e.blocks = (int)r[j];
        restore_list[RC] = e;
        a_r += r[j];
        a_rc += 1;
      }
    }
    const long long xj = gp ? 0 : hh[j];
    const long long zj = (gp || !rec_offl(w)) ? 0 : hh[j];
    if (st == CASCADE_RUNNING_PREFILL) {
      RpInfo ri;
      ri.pos = p;
      ri.eligible = adm ? 0 : 1;
      ri.x = X + xj;
      ri.y = y_inc[j];
      ri.z = Z + zj;
      ri.zp = zp_inc[j];
      rp_info[i] = ri;
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
  long long tot[6] = {a_nb, a_eh, a_eoh, a_n, a_r, a_rc};
  block_sum<6>(tot, s_scan);
  if (threadIdx.x == 0) {
    long long *dst[6] = {&ctl->adm_nb, &ctl->elig_h, &ctl->elig_offl_h,
                         &ctl->n_adm, &ctl->n_unpack, &ctl->n_restore};
    for (int k = 0; k < 6; ++k)
      if (tot[k]) atomicAdd((unsigned long long *)dst[k], (unsigned long long)tot[k]);
  }
}

// ------------------------------------------------------------ finalize

// Budget-aware preemption (Algorithm 1; Section 4.4): the deficit
// D = new blocks of admitted requests - free blocks is covered by the
// non-admitted running prefills taken from the back of the order (largest
// remaining budget first).  A holder at position p is preempted iff the
// eligible blocks after p are fewer than D.  One wave per running prefill.
__global__ __launch_bounds__(kBlock) void finalize_kernel(
    int n_free, const int *__restrict__ free_slots, const Ctl *ctl, int *info,
    const int *__restrict__ rp_list, const RpInfo *__restrict__ rp_info,
    const int4 *__restrict__ rec, const int *__restrict__ ro, const int *__restrict__ slots,
    uint8_t *__restrict__ action_out, int *__restrict__ slot_list, int sl_cap,
    cascade_move_t *__restrict__ pack, int pack_cap) {
  if (status_failed(info)) return;
  const int gt = blockIdx.x * kBlock + threadIdx.x;
  const int lim = min(n_free, sl_cap);
  for (int j = gt; j < lim; j += gridDim.x * kBlock) slot_list[j] = free_slots[j];
  const long long D = ctl->adm_nb - n_free;
  if (D <= 0) return;
  const long long E = ctl->elig_h, EO = ctl->elig_offl_h;
  const int kstar = ctl->kstar;
  const int lane = lane_id();
  const int nrp = (int)ctl->rp_count;
  for (int e = gt >> 6; e < nrp; e += (gridDim.x * kBlock) >> 6) {
    const int i = rp_list[e];
    const RpInfo ri = rp_info[i];
    if (!ri.eligible) continue;
    const long long eh = ri.pos < kstar ? ri.x : ctl->kx + ri.y - ctl->ky;
    const long long after = E - eh;  // eligible blocks behind this request
    if (after >= D) continue;
    const int w = rec[i].w;
    const int h = rec_held(w);
    const bool offl = rec_offl(w);
    const int row0 = ro[i];
    if (lane == 0) {
      action_out[i] = offl ? CASCADE_ACT_PREEMPT_OFFLOAD : CASCADE_ACT_PREEMPT_DROP;
      atomicAdd(&info[CASCADE_INFO_N_SLOT_LIST], h);
      if (offl) atomicAdd(&info[CASCADE_INFO_N_PACK], h);
    }
    const long long sbase = (long long)n_free + after;
    if (after < 0) {  // cannot happen with consistent prefixes
      if (lane == 0) set_status(info, CASCADE_EINTERNAL);
      continue;
    }
    for (int b = lane; b < h; b += 64)
      if (sbase + b < sl_cap) slot_list[sbase + b] = slots[row0 + b];
    if (offl) {
      const long long eo = ri.pos < kstar ? ri.z : ctl->kz + ri.zp - ctl->kzp;
      const long long pbase = EO - eo;
      for (int b = lane; b < h; b += 64) {
        if (pbase + b >= 0 && pbase + b < pack_cap) {
          cascade_move_t m;
          m.req = i;
          m.blk = b;
          m.pool_slot = slots[row0 + b];
          m.staging_slot = (int)(pbase + b);
          pack[pbase + b] = m;
        }
      }
    }
  }
}

// --------------------------------------------------------------- moves

// Restore moves: the first r new blocks of each RESTORE request receive its
// prefix, staged in admitted order.  Move m finds its request by binary
// search over the restore list's staging offsets.
__global__ __launch_bounds__(kBlock) void moves_kernel(
    const Ctl *ctl, int *info, const RestoreEnt *__restrict__ rl,
    const int *__restrict__ slot_list, int sl_cap, cascade_move_t *__restrict__ unpack,
    int unpack_cap, int pack_cap) {
  if (status_failed(info)) return;
  const long long nu = ctl->n_unpack;
  const int nr = (int)ctl->n_restore;
  const long long lim = lmin(nu, (long long)unpack_cap);
  for (long long m = blockIdx.x * kBlock + threadIdx.x; m < lim;
       m += (long long)gridDim.x * kBlock) {
    int lo = 0, hi = nr - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (rl[mid].stage_off <= m) lo = mid; else hi = mid - 1;
    }
    const RestoreEnt e = rl[lo];
    const int b = (int)(m - e.stage_off);
    const long long s = (long long)e.alloc_off + b;
    cascade_move_t mv;
    mv.req = e.req;
    mv.blk = b;
    mv.pool_slot = s < sl_cap ? slot_list[s] : -1;
    mv.staging_slot = (int)m;
    unpack[m] = mv;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    info[CASCADE_INFO_N_ADMITTED] = (int)ctl->n_adm;
    info[CASCADE_INFO_N_UNPACK] = (int)nu;
    const bool full = info[CASCADE_INFO_N_SLOT_LIST] > sl_cap || nu > unpack_cap ||
                      info[CASCADE_INFO_N_PACK] > pack_cap;
    if (full && info[CASCADE_INFO_STATUS] == CASCADE_OK) info[CASCADE_INFO_STATUS] = CASCADE_ENOSPC;
  }
}

// ---------------------------------------------------------------- init

__global__ __launch_bounds__(kBlock) void init_kernel(Ctl *ctl, uint4 *clear, size_t clear_vec,
                                                      int *info, int n, int n_free) {
  const size_t gt = (size_t)blockIdx.x * kBlock + threadIdx.x;
  const size_t gs = (size_t)gridDim.x * kBlock;
  for (size_t j = gt; j < clear_vec; j += gs) clear[j] = make_uint4(0, 0, 0, 0);
  if (gt == 0) {
    unsigned *w = reinterpret_cast<unsigned *>(ctl);
    for (size_t k = 0; k < kCtlHeaderWords; ++k) w[k] = 0;
    ctl->bmin = ~0ull;
    ctl->bmax = 0;
    ctl->kstar = n;
    for (int k = 0; k < CASCADE_INFO_LEN; ++k) info[k] = 0;
    info[CASCADE_INFO_N_SLOT_LIST] = n_free;
  }
}

// ---------------------------------------------------------------- host

struct Layout {
  size_t ctl, keys_a, keys_b, vals_a, vals_b, rec, rp_list, rp_info, restore, sort_status,
      scan1, scan2, total;
  int sort_tiles, scan_tiles;
};

size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }

Layout make_layout(int32_t n) {
  Layout L;
  const size_t np = n > 0 ? (size_t)n : 1;
  L.sort_tiles = (int)((np + kSortTile - 1) / kSortTile);
  L.scan_tiles = (int)((np + kScanTile - 1) / kScanTile);
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off = align_up(off + bytes); return o; };
  L.ctl = take(sizeof(Ctl));
  // the look-back status words follow the control block: one clear covers all
  L.sort_status = take((size_t)kMaxDigits * L.sort_tiles * kRadix * 4);
  L.scan1 = take((size_t)L.scan_tiles * kL1 * 8);
  L.scan2 = take((size_t)L.scan_tiles * kL2Stride * 8);
  L.keys_a = take(np * 8);
  L.keys_b = take(np * 8);
  L.vals_a = take(np * 4);
  L.vals_b = take(np * 4);
  L.rec = take(np * 16);
  L.rp_list = take(np * 4);
  L.rp_info = take(np * sizeof(RpInfo));
  L.restore = take(np * sizeof(RestoreEnt));
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

extern "C" int cascade_step(const cascade_requests_t *rq, const cascade_block_table_t *bt,
                            const cascade_tier_state_t *ts, const cascade_params_t *p,
                            const cascade_outputs_t *out, void *workspace,
                            size_t workspace_bytes, void *stream) {
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

  char *ws = static_cast<char *>(workspace);
  Ctl *ctl = reinterpret_cast<Ctl *>(ws + L.ctl);
  auto *keys_a = reinterpret_cast<unsigned long long *>(ws + L.keys_a);
  auto *keys_b = reinterpret_cast<unsigned long long *>(ws + L.keys_b);
  auto *vals_a = reinterpret_cast<unsigned *>(ws + L.vals_a);
  auto *vals_b = reinterpret_cast<unsigned *>(ws + L.vals_b);
  auto *rec = reinterpret_cast<int4 *>(ws + L.rec);
  auto *rp_list = reinterpret_cast<int *>(ws + L.rp_list);
  auto *rp_info = reinterpret_cast<RpInfo *>(ws + L.rp_info);
  auto *rlist = reinterpret_cast<RestoreEnt *>(ws + L.restore);
  auto *sort_status = reinterpret_cast<unsigned *>(ws + L.sort_status);
  auto *scan1 = reinterpret_cast<unsigned long long *>(ws + L.scan1);
  auto *scan2 = reinterpret_cast<unsigned long long *>(ws + L.scan2);
  hipStream_t s = static_cast<hipStream_t>(stream);

  // clear the histograms and every look-back status word in one sweep
  const size_t clear_bytes = L.keys_a - offsetof(Ctl, hist);
  const size_t clear_vec = clear_bytes / 16;
  uint4 *clear = reinterpret_cast<uint4 *>(ws + L.ctl + offsetof(Ctl, hist));
  const int init_grid = (int)std::min<size_t>(1024, (clear_vec + kBlock * 4 - 1) / (kBlock * 4) + 1);
  hipLaunchKernelGGL(init_kernel, dim3(init_grid), dim3(kBlock), 0, s, ctl, clear, clear_vec,
                     out->info, n, ts->n_free);
  const int eval_grid = std::max(1, (n + kBlock - 1) / kBlock);
  hipLaunchKernelGGL(eval_kernel, dim3(eval_grid), dim3(kBlock), 0, s, *rq, bt->row_offsets,
                     ts->free_slots, c, n, ctl, out->info, out->budget_ns, out->queue_tier_out,
                     keys_a, rec, rp_list);
  if (n > 0) {
    const int prep_grid = (n + kBlock * kPrepItems - 1) / (kBlock * kPrepItems);
    hipLaunchKernelGGL(prep_kernel, dim3(prep_grid), dim3(kBlock), 0, s, n, ts->num_blocks,
                       bt->row_offsets, bt->slots, ctl, out->info, keys_a, vals_a);
    for (int pass = 0; pass < kMaxDigits; ++pass)
      hipLaunchKernelGGL(radix_pass_kernel, dim3(L.sort_tiles), dim3(kBlock), 0, s, pass, n,
                         ctl, out->info, keys_a, keys_b, vals_a, vals_b,
                         sort_status + (size_t)pass * L.sort_tiles * kRadix);
    hipLaunchKernelGGL(scan_kernel, dim3(L.scan_tiles), dim3(kBlock), 0, s, n, c, ctl,
                       out->info, vals_a, vals_b, rec, out->order, out->tokens_granted,
                       out->restore_blocks, out->alloc_begin, out->alloc_count, out->action,
                       out->admitted, rp_info, rlist, scan1, scan2);
  }
  const int fin_grid = std::max(1, std::min(1024, (int)((std::max(n, ts->n_free) + kBlock - 1) / kBlock)));
  hipLaunchKernelGGL(finalize_kernel, dim3(fin_grid), dim3(kBlock), 0, s, ts->n_free,
                     ts->free_slots, ctl, out->info, rp_list, rp_info, rec, bt->row_offsets,
                     bt->slots, out->action, out->slot_list, out->slot_list_capacity,
                     out->pack_moves, out->pack_capacity);
  const int mv_grid = std::max(1, std::min(256, (out->unpack_capacity + kBlock - 1) / kBlock));
  hipLaunchKernelGGL(moves_kernel, dim3(mv_grid), dim3(kBlock), 0, s, ctl, out->info, rlist,
                     out->slot_list, out->slot_list_capacity, out->unpack_moves,
                     out->unpack_capacity, out->pack_capacity);
  if (hipGetLastError() != hipSuccess) return CASCADE_EHIP;
  return CASCADE_OK;
}
