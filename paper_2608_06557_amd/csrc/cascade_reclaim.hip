// cascade_reclaim.hip -- per-tier LRU reclamation on gfx950 (Section 4.4,
// prefix hit detection: free blocks are reclaimed least-recently-used within
// each tier, so hot prefixes stay in the fast tiers and cold ones spill one
// tier deeper).
//
// One call reclaims `total` = need + n_incoming free slots of one tier.  The
// reclaimed set is the `total` smallest free slots under the key
//   empty slot -> 0,   cached block -> 1 + (last_use - min cached last_use),
// ties by slot.  Selection is a most-significant-digit radix select over the
// key (an 8-bit digit, then 12-bit digits), so it never sorts the table:
//
//   rc_count_kernel    per-workgroup counts of empty / cached free slots and
//                      the cached last-use range; the last workgroup checks
//                      the call, sizes the key and writes the plan
//   rc_pass_kernel     one digit: LDS histogram of the keys that match the
//                      threshold's digits found so far, merged with atomics;
//                      the last workgroup finds the digit holding the rank
//   rc_tie_kernel      when only some slots with the threshold key T are
//                      taken, the slot of the last one taken (taken in slot
//                      order); per-tile counts, then one workgroup
//   rc_compact_kernel  slot-order compaction of the reclaimed set and of the
//                      demoted blocks (one decoupled look-back over a packed
//                      pair of counts); demotion decisions read the index
//   rc_update_kernel   index bit updates (clear this tier, set the next for
//                      demoted blocks) and the slot-table writes
//
// The plan lives in the caller's workspace; every kernel after the first reads
// it and returns at once when the call failed or has nothing left to do, so
// the host launches a fixed sequence and never waits.  The last workgroup of
// each kernel resets the counters it used, which leaves the workspace zeroed.
#include <hip/hip_runtime.h>
#include <limits.h>
#include <stdint.h>

#include <algorithm>

#include "cascade.h"
#include "device_util.h"
#include "index_table.h"

namespace cascade {
namespace {

constexpr int kRcItems = 8;                  // slots per thread in slot-order kernels
constexpr int kRcTile = kBlock * kRcItems;   // 2048 slots per tile
constexpr int kRcGrid = 512;                 // workgroups of the whole-table kernels
constexpr int kDigit0 = 8, kDigitN = 12;     // first digit, later digits
constexpr int kRcBins = 1 << kDigitN;
constexpr int kRcPasses = 1 + (64 - kDigit0 + kDigitN - 1) / kDigitN;  // 6 covers 64 bits
constexpr int kBinsPerThread = kRcBins / kBlock;                        // 16

struct RcPartial {
  int n_empty, n_cached, bad, pad;
  unsigned long long lu_min, lu_max;
};

struct alignas(256) RcPlan {
  int ok;         // 1: the call proceeds (checked, room enough)
  int total;      // need + n_in
  int n_in;
  int width;      // bits of the key
  int shift;      // low bit of the digit the next pass examines
  int dbits;      // width of that digit
  int done;       // threshold key found
  int rank;       // 0-based rank still sought among keys matching `prefix`
  int take;       // slots with the threshold key taken, in slot order
  int find_tie;   // 1: rc_tie_kernel must locate the last tie taken
  int tie_slot;   // last slot with the threshold key taken (-1: none; INT_MAX: all)
  int pad0;
  unsigned long long lu_min;
  unsigned long long prefix;  // the threshold's digits found so far, in place; T when done
  unsigned ticket_count, ticket_pass, ticket_tie, tile_claim, compact_done, pad1[3];
};

struct RcWork {
  RcPlan *plan;
  RcPartial *partial;     // [kRcGrid]
  unsigned *hist;         // [kRcBins]
  int *tie_cnt;           // [tiles]
  unsigned long long *lb; // [tiles] look-back words
};

constexpr size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
inline int tiles_of(long long n) { return (int)((n + kRcTile - 1) / kRcTile); }

size_t workspace_bytes_for(int32_t n) {
  const size_t tiles = (size_t)std::max(1, tiles_of(n));
  return align256(sizeof(RcPlan)) + align256(sizeof(RcPartial) * kRcGrid) +
         align256(sizeof(unsigned) * kRcBins) + align256(sizeof(int) * tiles) +
         align256(sizeof(unsigned long long) * tiles);
}

RcWork carve(void *ws, int32_t n) {
  char *p = static_cast<char *>(ws);
  const size_t tiles = (size_t)std::max(1, tiles_of(n));
  RcWork w;
  w.plan = reinterpret_cast<RcPlan *>(p);
  p += align256(sizeof(RcPlan));
  w.partial = reinterpret_cast<RcPartial *>(p);
  p += align256(sizeof(RcPartial) * kRcGrid);
  w.hist = reinterpret_cast<unsigned *>(p);
  p += align256(sizeof(unsigned) * kRcBins);
  w.tie_cnt = reinterpret_cast<int *>(p);
  p += align256(sizeof(int) * tiles);
  w.lb = reinterpret_cast<unsigned long long *>(p);
  return w;
}

struct RcArgs {
  int tier, n, need, max_in, max_out;
  unsigned long long *hash;
  long long *lu;
  const unsigned char *held;
  const cascade_demotion_t *incoming;
  const int *n_in_dev;
  cascade_demotion_t *outgoing;
  int *n_out_dev;
  int *freed, *placed;
  IndexSlot *index;
  unsigned index_mask;
  int *status;
  RcWork w;
};

__device__ __forceinline__ unsigned long long shr64(unsigned long long x, int k) {
  return k >= 64 ? 0ull : x >> k;
}
__device__ __forceinline__ int bit_width64(unsigned long long x) {
  return x ? 64 - __builtin_clzll(x) : 0;
}
// the reclamation key of a free slot
__device__ __forceinline__ unsigned long long rc_key(unsigned long long h, long long lu,
                                                     unsigned long long lu_min) {
  return h ? 1ull + ((unsigned long long)lu - lu_min) : 0ull;
}

// Eight consecutive slots [s0, s0 + 8) of one thread, slots past the table
// marked held so that nothing selects them.
struct Slots8 {
  unsigned long long h[kRcItems];
  long long lu[kRcItems];
  bool held[kRcItems];
};
__device__ __forceinline__ void load8(const RcArgs &a, int s0, Slots8 &v) {
  if (s0 + kRcItems <= a.n) {
    const ulonglong2 *hp = reinterpret_cast<const ulonglong2 *>(a.hash + s0);
    const longlong2 *lp = reinterpret_cast<const longlong2 *>(a.lu + s0);
#pragma unroll
    for (int j = 0; j < kRcItems / 2; ++j) {
      const ulonglong2 h2 = hp[j];
      const longlong2 l2 = lp[j];
      v.h[2 * j] = h2.x;
      v.h[2 * j + 1] = h2.y;
      v.lu[2 * j] = l2.x;
      v.lu[2 * j + 1] = l2.y;
    }
    const uint2 hd = *reinterpret_cast<const uint2 *>(a.held + s0);
#pragma unroll
    for (int j = 0; j < kRcItems; ++j)
      v.held[j] = ((j < 4 ? hd.x >> (8 * j) : hd.y >> (8 * (j - 4))) & 0xffu) != 0u;
  } else {
#pragma unroll
    for (int j = 0; j < kRcItems; ++j) {
      const int s = s0 + j;
      const bool in = s < a.n;
      v.h[j] = in ? a.hash[s] : 0ull;
      v.lu[j] = in ? a.lu[s] : 0ll;
      v.held[j] = in ? a.held[s] != 0 : true;
    }
  }
}

__device__ __forceinline__ bool status_bad(const int *status) {
  return load_agent(status) != CASCADE_OK;
}

// ------------------------------------------------------------- count kernel

__global__ __launch_bounds__(kBlock) void rc_count_kernel(RcArgs a) {
  __shared__ int s_red[kWaves * 3];
  __shared__ unsigned long long s_mm[kWaves * 2];
  __shared__ bool s_last;
  __shared__ int s_err;
  int cnt[3] = {0, 0, 0};  // empty free, cached free, negative last use
  unsigned long long mn = ~0ull, mx = 0ull;
  const long long stride = (long long)gridDim.x * kBlock;
  for (long long s = (long long)blockIdx.x * kBlock + threadIdx.x; s < a.n; s += stride) {
    const long long lu = a.lu[s];
    const unsigned long long h = a.hash[s];
    const bool free_slot = a.held[s] == 0;
    cnt[2] |= lu < 0;
    if (free_slot && h == 0ull) ++cnt[0];
    if (free_slot && h != 0ull && lu >= 0) {
      ++cnt[1];
      mn = min(mn, (unsigned long long)lu);
      mx = max(mx, (unsigned long long)lu);
    }
  }
  block_sum<3, int>(cnt, s_red);
  mn = wave_min(mn);
  mx = wave_max(mx);
  if (lane_id() == 0) {
    s_mm[wave_id() * 2] = mn;
    s_mm[wave_id() * 2 + 1] = mx;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < kWaves; ++w) {
      mn = min(mn, s_mm[w * 2]);
      mx = max(mx, s_mm[w * 2 + 1]);
    }
    RcPartial p;
    p.n_empty = cnt[0];
    p.n_cached = cnt[1];
    p.bad = cnt[2];
    p.pad = 0;
    p.lu_min = mn;
    p.lu_max = mx;
    a.w.partial[blockIdx.x] = p;
    __threadfence();  // release the partial, then count this workgroup
    s_last = atomicAdd(&a.w.plan->ticket_count, 1u) == gridDim.x - 1;
  }
  __syncthreads();
  if (!s_last) return;
  __threadfence();  // acquire every workgroup's partial

  // the last workgroup: totals, incoming check, plan
  int tot[3] = {0, 0, 0};
  unsigned long long tmn = ~0ull, tmx = 0ull;
  for (int g = threadIdx.x; g < (int)gridDim.x; g += kBlock) {
    const RcPartial p = a.w.partial[g];
    tot[0] += p.n_empty;
    tot[1] += p.n_cached;
    tot[2] |= p.bad;
    tmn = min(tmn, p.lu_min);
    tmx = max(tmx, p.lu_max);
  }
  block_sum<3, int>(tot, s_red);
  tmn = wave_min(tmn);
  tmx = wave_max(tmx);
  if (lane_id() == 0) {
    s_mm[wave_id() * 2] = tmn;
    s_mm[wave_id() * 2 + 1] = tmx;
  }
  if (threadIdx.x == 0) {
    const int n_in = a.n_in_dev ? load_agent(a.n_in_dev) : 0;
    s_err = status_bad(a.status) ? 1 : 0;  // an earlier call of the chain failed
    if (!s_err && (tot[2] || n_in < 0 || n_in > a.max_in)) s_err = CASCADE_EINVAL;
    s_red[0] = n_in;
  }
  __syncthreads();
  const int n_in = s_red[0];
  int zero_hash = 0;
  if (s_err == 0)
    for (int j = threadIdx.x; j < n_in; j += kBlock) zero_hash |= a.incoming[j].hash == 0ull;
  zero_hash = __syncthreads_or(zero_hash);
  if (threadIdx.x == 0) {
    for (int w = 1; w < kWaves; ++w) {
      tmn = min(tmn, s_mm[w * 2]);
      tmx = max(tmx, s_mm[w * 2 + 1]);
    }
    RcPlan *P = a.w.plan;
    int err = s_err;
    if (err == 0 && zero_hash) err = CASCADE_EINVAL;
    const long long total = (long long)a.need + n_in;
    if (err == 0 && total > (long long)tot[0] + tot[1]) err = CASCADE_ENOSPC;
    if (err < 0) store_agent(a.status, err);
    P->ok = err == 0;
    P->total = (int)total;
    P->n_in = n_in;
    P->lu_min = tmn;
    P->prefix = 0ull;
    P->tie_slot = -1;
    P->find_tie = 0;
    if (total <= tot[0]) {
      // empty slots suffice: the threshold is key 0, taken in slot order
      P->width = 0;
      P->done = 1;
      P->rank = 0;
      P->take = (int)total;
      P->find_tie = total > 0 && total < tot[0];
      P->tie_slot = total == 0 ? -1 : (total == tot[0] ? INT_MAX : -1);
    } else {
      // every empty slot plus the (total - n_empty) least recent cached ones
      const int width = bit_width64(1ull + (tmx - tmn));
      P->width = width;
      P->done = 0;
      P->dbits = min(width, kDigit0);
      P->shift = width - P->dbits;
      P->rank = (int)(total - tot[0] - 1);
    }
    P->ticket_count = 0u;
  }
}

// ----------------------------------------------------- radix select passes

__global__ __launch_bounds__(kBlock) void rc_pass_kernel(RcArgs a) {
  __shared__ unsigned s_hist[kRcBins];
  __shared__ int s_scan[kWaves];
  __shared__ bool s_last;
  __shared__ int s_found[2];
  const RcPlan *P = a.w.plan;
  if (!P->ok || P->done) return;  // uniform: the plan is the previous kernel's
  const int shift = P->shift, dbits = P->dbits;
  const unsigned long long lu_min = P->lu_min;
  const unsigned long long hi = shr64(P->prefix, shift + dbits);
  const unsigned dmask = (1u << dbits) - 1u;
  const int nbins = 1 << dbits;
  for (int b = threadIdx.x; b < nbins; b += kBlock) s_hist[b] = 0u;
  __syncthreads();
  const long long stride = (long long)gridDim.x * kBlock;
  for (long long s = (long long)blockIdx.x * kBlock + threadIdx.x; s < a.n; s += stride) {
    const unsigned long long h = a.hash[s];
    if (a.held[s] || h == 0ull) continue;  // only cached free slots have keys above 0
    const unsigned long long k = rc_key(h, a.lu[s], lu_min);
    if (shr64(k, shift + dbits) == hi) atomicAdd(&s_hist[(unsigned)(k >> shift) & dmask], 1u);
  }
  __syncthreads();
  for (int b = threadIdx.x; b < nbins; b += kBlock) {
    const unsigned v = s_hist[b];
    if (v) atomicAdd(&a.w.hist[b], v);
  }
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) s_last = atomicAdd(&a.w.plan->ticket_pass, 1u) == gridDim.x - 1;
  __syncthreads();
  if (!s_last) return;
  __threadfence();

  // the last workgroup: the digit in which the sought rank falls
  const int rank = P->rank;
  if (threadIdx.x == 0) s_found[0] = -1;
  unsigned v[kBinsPerThread];
  int sum = 0;
  const int b0 = threadIdx.x * kBinsPerThread;
#pragma unroll
  for (int j = 0; j < kBinsPerThread; ++j) {
    const int b = b0 + j;
    v[j] = b < nbins ? load_agent(a.w.hist + b) : 0u;
    sum += (int)v[j];
  }
#pragma unroll
  for (int j = 0; j < kBinsPerThread; ++j)  // clear for the next pass
    if (b0 + j < nbins) store_agent(a.w.hist + b0 + j, 0u);
  int excl[1] = {sum}, tot[1];
  block_exclusive_scan<1, int>(excl, tot, s_scan);
  if (rank >= excl[0] && rank < excl[0] + sum) {
    int r = rank - excl[0];
#pragma unroll
    for (int j = 0; j < kBinsPerThread; ++j) {
      if (r >= 0 && r < (int)v[j]) {
        s_found[0] = b0 + j;
        s_found[1] = r;
        s_hist[0] = v[j];  // keys equal on every digit so far
        r = -1;
      } else if (r >= 0) {
        r -= (int)v[j];
      }
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    RcPlan *W = a.w.plan;
    W->ticket_pass = 0u;
    if (s_found[0] < 0) {  // the counts disagree with the plan: stop the call
      store_agent(a.status, (int)CASCADE_EINTERNAL);
      W->ok = 0;
      return;
    }
    W->prefix = P->prefix | ((unsigned long long)s_found[0] << shift);
    W->rank = s_found[1];
    if (shift == 0) {
      // the threshold is known; take = rank + 1 of the slots holding it
      const int ties = (int)s_hist[0];
      W->done = 1;
      W->take = s_found[1] + 1;
      W->find_tie = W->take < ties;
      W->tie_slot = W->take < ties ? -1 : INT_MAX;
    } else {
      const int d = min(shift, kDigitN);
      W->dbits = d;
      W->shift = shift - d;
    }
  }
}

// --------------------------------------------------------- tie location

// Slots holding the threshold key are taken in slot order; when only some
// are, find the last one taken.  Also clears the compaction's look-back words.
__global__ __launch_bounds__(kBlock) void rc_tie_kernel(RcArgs a) {
  __shared__ int s_red[kWaves];
  __shared__ bool s_last;
  __shared__ int s_hit[2];
  const RcPlan *P = a.w.plan;
  const int tile = blockIdx.x;
  if (threadIdx.x == 0) a.w.lb[tile] = 0ull;
  if (!P->ok || !P->find_tie) return;
  const unsigned long long T = P->prefix, lu_min = P->lu_min;
  const int s0 = tile * kRcTile + threadIdx.x * kRcItems;
  Slots8 v;
  load8(a, s0, v);
  int c[1] = {0};
#pragma unroll
  for (int j = 0; j < kRcItems; ++j)
    c[0] += (!v.held[j] && rc_key(v.h[j], v.lu[j], lu_min) == T) ? 1 : 0;
  block_sum<1, int>(c, s_red);
  if (threadIdx.x == 0) {
    a.w.tie_cnt[tile] = c[0];
    __threadfence();
    s_last = atomicAdd(&a.w.plan->ticket_tie, 1u) == gridDim.x - 1;
  }
  __syncthreads();
  if (!s_last) return;
  __threadfence();

  // the last workgroup: the tile holding the take-th tie, then the slot
  const int take = P->take, tiles = gridDim.x;
  const int per = (tiles + kBlock - 1) / kBlock;
  if (threadIdx.x == 0) {
    s_hit[0] = -1;
    a.w.plan->ticket_tie = 0u;
  }
  const int t0 = min(tiles, threadIdx.x * per), t1 = min(tiles, t0 + per);
  int sum = 0;
  for (int t = t0; t < t1; ++t) sum += load_agent(a.w.tie_cnt + t);
  int excl[1] = {sum}, tot[1];
  block_exclusive_scan<1, int>(excl, tot, s_red);
  if (take > excl[0] && take <= excl[0] + sum) {
    int before = excl[0];
    for (int t = t0; t < t1; ++t) {
      const int ct = load_agent(a.w.tie_cnt + t);
      if (take <= before + ct) {
        s_hit[0] = t;
        s_hit[1] = take - before;  // 1-based rank inside tile t
        break;
      }
      before += ct;
    }
  }
  __syncthreads();
  const int ht = s_hit[0], want = s_hit[1];
  if (ht < 0) {  // the counts disagree with the plan: stop the call
    if (threadIdx.x == 0) {
      store_agent(a.status, (int)CASCADE_EINTERNAL);
      a.w.plan->ok = 0;
    }
    return;
  }
  load8(a, ht * kRcTile + threadIdx.x * kRcItems, v);
  int mine = 0;
  bool is_tie[kRcItems];
#pragma unroll
  for (int j = 0; j < kRcItems; ++j) {
    is_tie[j] = !v.held[j] && rc_key(v.h[j], v.lu[j], lu_min) == T;
    mine += is_tie[j] ? 1 : 0;
  }
  int e2[1] = {mine}, t2[1];
  block_exclusive_scan<1, int>(e2, t2, s_red);
  if (want > e2[0] && want <= e2[0] + mine) {
    int r = want - e2[0];
#pragma unroll
    for (int j = 0; j < kRcItems; ++j) {
      if (is_tie[j] && r > 0 && --r == 0)
        a.w.plan->tie_slot = ht * kRcTile + threadIdx.x * kRcItems + j;
    }
  }
}

// ------------------------------------------------------------- compaction

// Counts of one tile packed in one word: reclaimed | demoted << 31.
constexpr int kDemShift = 31;

__global__ __launch_bounds__(kBlock) void rc_compact_kernel(RcArgs a) {
  __shared__ unsigned long long s_scan[kWaves];
  __shared__ int s_tile;
  __shared__ unsigned long long s_prefix;
  __shared__ bool s_last, s_timeout;
  const RcPlan *P = a.w.plan;
  if (!P->ok) return;
  if (threadIdx.x == 0) {
    s_tile = (int)atomicAdd(&a.w.plan->tile_claim, 1u);
    s_timeout = false;
  }
  __syncthreads();
  const int tile = s_tile;
  if (tile >= (int)gridDim.x) {  // counters not zeroed: refuse to touch anything
    if (threadIdx.x == 0) store_agent(a.status, (int)CASCADE_EINTERNAL);
    return;
  }
  const unsigned long long T = P->prefix, lu_min = P->lu_min;
  const int tie_slot = P->tie_slot, need = a.need;
  const bool can_demote = a.tier < 2;
  const unsigned deeper = ~((2u << a.tier) - 1u);  // tiers below this one
  const int s0 = tile * kRcTile + threadIdx.x * kRcItems;
  Slots8 v;
  load8(a, s0, v);
  bool sel[kRcItems], dem[kRcItems];
  unsigned long long cnt = 0ull;
#pragma unroll
  for (int j = 0; j < kRcItems; ++j) {
    const unsigned long long k = rc_key(v.h[j], v.lu[j], lu_min);
    sel[j] = !v.held[j] && (k < T || (k == T && s0 + j <= tie_slot));
    dem[j] = false;
    if (sel[j] && can_demote && v.h[j] != 0ull) {
      const IndexSlot *e = a.index ? index_find(a.index, a.index_mask, v.h[j]) : nullptr;
      dem[j] = e == nullptr || (e->tiers & deeper) == 0u;
    }
    cnt += (sel[j] ? 1ull : 0ull) + (dem[j] ? (1ull << kDemShift) : 0ull);
  }
  unsigned long long ex[1] = {cnt}, tot[1];
  block_exclusive_scan<1, unsigned long long>(ex, tot, s_scan);
  if (threadIdx.x == 0) {
    unsigned long long before = 0ull;
    if (tile == 0) {
      publish(a.w.lb, tot[0], kFlagInclusive);
    } else {
      publish(a.w.lb + tile, tot[0], kFlagAggregate);
      bool to = false;
      before = look_back<unsigned long long, 32>(a.w.lb, 1, tile, 0, &to);
      s_timeout = to;
      publish(a.w.lb + tile, before + tot[0], kFlagInclusive);
    }
    s_prefix = before;
  }
  __syncthreads();
  if (s_timeout) {
    if (threadIdx.x == 0) store_agent(a.status, (int)CASCADE_ETIMEOUT);
  } else {
    const unsigned long long base = s_prefix + ex[0];
    int p = (int)(base & ((1ull << kDemShift) - 1ull));
    int q = (int)(base >> kDemShift);
    const int total = P->total;
    bool over = false;
#pragma unroll
    for (int j = 0; j < kRcItems; ++j) {
      if (sel[j]) {
        if (p < need) a.freed[p] = s0 + j;
        else if (p < total) a.placed[p - need] = s0 + j;
        else over = true;
        ++p;
      }
      if (dem[j] && q >= a.max_out) over = true;
      if (dem[j] && q < a.max_out) {
        cascade_demotion_t d;
        d.hash = v.h[j];
        d.last_use_ns = v.lu[j];
        d.src_slot = s0 + j;
        d.pad = 0;
        a.outgoing[q++] = d;
      }
    }
    if (over) store_agent(a.status, (int)CASCADE_EINTERNAL);
  }
  // the last tile to finish publishes the count and resets the counters
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) s_last = atomicAdd(&a.w.plan->compact_done, 1u) == gridDim.x - 1;
  __syncthreads();
  if (!s_last || threadIdx.x != 0) return;
  __threadfence();
  const unsigned long long all = load_agent(a.w.lb + (gridDim.x - 1)) >> 2;
  if ((int)(all & ((1ull << kDemShift) - 1ull)) != P->total)  // must reclaim exactly total
    store_agent(a.status, (int)CASCADE_EINTERNAL);
  if (a.n_out_dev) store_agent(a.n_out_dev, (int)(all >> kDemShift));
  a.w.plan->tile_claim = 0u;
  a.w.plan->compact_done = 0u;
}

// ---------------------------------------------------------------- updates

// Position p of the reclaimed list: the old block leaves this tier in the
// index and the slot takes its new contents; position p of the outgoing list:
// the demoted block joins the next tier in the index.
__global__ __launch_bounds__(kBlock) void rc_update_kernel(RcArgs a) {
  const RcPlan *P = a.w.plan;
  if (!P->ok || status_bad(a.status)) return;
  const int p = blockIdx.x * kBlock + threadIdx.x;
  const int total = P->total, need = a.need;
  unsigned long long *hash = a.hash;
  long long *lu = a.lu;
  if (p < total) {
    const int s = p < need ? a.freed[p] : a.placed[p - need];
    if ((unsigned)s >= (unsigned)a.n) return;  // only after a failed check, reported already
    const unsigned long long old = hash[s];
    if (old != 0ull && a.index) {
      IndexSlot *e = index_find(a.index, a.index_mask, old);
      if (e) atomicAnd(&e->tiers, ~(1u << a.tier));
    }
    if (p < need) {
      hash[s] = 0ull;
      lu[s] = 0ll;
    } else {
      const cascade_demotion_t in = a.incoming[p - need];
      hash[s] = in.hash;
      lu[s] = in.last_use_ns;
    }
  }
  if (a.tier < 2 && a.index) {
    const int n_out = *a.n_out_dev;
    if (p < n_out) {
      IndexSlot *e = index_find(a.index, a.index_mask, a.outgoing[p].hash);
      if (e) atomicOr(&e->tiers, 1u << (a.tier + 1));
    }
  }
}

bool index_capacity_ok(int32_t capacity) {
  return capacity >= 64 && capacity <= (1 << 30) && (capacity & (capacity - 1)) == 0;
}

}  // namespace
}  // namespace cascade

using namespace cascade;

extern "C" size_t cascade_reclaim_workspace_bytes(int32_t n_slots) {
  if (n_slots < 0 || n_slots > (1 << 30)) return 0;
  return workspace_bytes_for(n_slots);
}

extern "C" int cascade_tier_reclaim(int32_t tier, const cascade_tier_table_t *table, int32_t need,
                                    const cascade_demotion_t *incoming,
                                    const int32_t *n_incoming_dev, int32_t max_incoming,
                                    cascade_demotion_t *outgoing, int32_t *n_outgoing_dev,
                                    int32_t max_outgoing, int32_t *freed, int32_t *placed,
                                    void *index, int32_t index_capacity, void *workspace,
                                    size_t workspace_bytes, int32_t *status_dev, void *stream) {
  if (tier < 0 || tier > 2 || !table || need < 0 || max_incoming < 0 || !status_dev ||
      (long long)need + max_incoming > INT_MAX)
    return CASCADE_EINVAL;
  const int32_t n = table->n_slots;
  if (n < 0 || n > (1 << 30)) return CASCADE_EINVAL;
  if (n > 0 && (!table->block_hash || !table->last_use_ns || !table->held)) return CASCADE_EINVAL;
  if (((uintptr_t)table->block_hash & 15) || ((uintptr_t)table->last_use_ns & 15) ||
      ((uintptr_t)table->held & 7))
    return CASCADE_EINVAL;  // the slot-order kernels load 8 slots with vector loads
  if (max_incoming > 0 && (!incoming || !n_incoming_dev || !placed)) return CASCADE_EINVAL;
  if (need > 0 && !freed) return CASCADE_EINVAL;
  if (tier < 2) {
    if ((long long)max_outgoing < (long long)need + max_incoming || !n_outgoing_dev)
      return CASCADE_EINVAL;
    if (max_outgoing > 0 && !outgoing) return CASCADE_EINVAL;
  }
  if (index && (!index_capacity_ok(index_capacity) || ((uintptr_t)index & 15)))
    return CASCADE_EINVAL;
  if (!workspace || ((uintptr_t)workspace & 255) || workspace_bytes < workspace_bytes_for(n))
    return CASCADE_EINVAL;

  RcArgs a;
  a.tier = tier;
  a.n = n;
  a.need = need;
  a.max_in = max_incoming;
  a.max_out = tier < 2 ? max_outgoing : 0;
  a.hash = reinterpret_cast<unsigned long long *>(table->block_hash);
  a.lu = reinterpret_cast<long long *>(table->last_use_ns);
  a.held = table->held;
  a.incoming = max_incoming > 0 ? incoming : nullptr;
  a.n_in_dev = max_incoming > 0 ? n_incoming_dev : nullptr;
  a.outgoing = outgoing;
  a.n_out_dev = n_outgoing_dev;
  a.freed = freed;
  a.placed = placed;
  a.index = static_cast<IndexSlot *>(index);
  a.index_mask = index ? (unsigned)(index_capacity - 1) : 0u;
  a.status = status_dev;
  a.w = carve(workspace, n);

  hipStream_t s = static_cast<hipStream_t>(stream);
  const int tiles = std::max(1, tiles_of(n));
  const int grid = std::min(tiles, kRcGrid);
  const int total_cap = (int)std::min<long long>((long long)need + max_incoming, n);
  hipLaunchKernelGGL(rc_count_kernel, dim3(grid), dim3(kBlock), 0, s, a);
  for (int p = 0; p < kRcPasses; ++p)
    hipLaunchKernelGGL(rc_pass_kernel, dim3(grid), dim3(kBlock), 0, s, a);
  hipLaunchKernelGGL(rc_tie_kernel, dim3(tiles), dim3(kBlock), 0, s, a);
  hipLaunchKernelGGL(rc_compact_kernel, dim3(tiles), dim3(kBlock), 0, s, a);
  if (total_cap > 0)
    hipLaunchKernelGGL(rc_update_kernel, dim3((total_cap + kBlock - 1) / kBlock), dim3(kBlock),
                       0, s, a);
  return hipGetLastError() == hipSuccess ? CASCADE_OK : CASCADE_EHIP;
}
