// cascade_reclaim.hip -- per-tier LRU reclamation on gfx950 (Section 4.4,
// prefix hit detection: free blocks are reclaimed least-recently-used within
// each tier, so hot prefixes stay in the fast tiers and cold ones spill one
// tier deeper).
//
// One call reclaims `total` = need + n_incoming free slots of one tier.  The
// reclaimed set is the `total` smallest free slots under the key
//   empty slot -> 0,   cached block -> 1 + (last_use - min cached last_use),
// ties by slot.  Selection is a most-significant-digit radix select over the
// key (an 8-bit digit, then 12-bit digits), so it never sorts the table.  The
// table is read in tiles of 2048 slots, 8 consecutive slots per thread with
// 16-byte loads:
//
//   rc_count_kernel  per-workgroup counts of empty / cached free slots and
//                    the cached last-use range; the last workgroup checks the
//                    call, sizes the key and writes the plan
//   rc_pass_kernel   one digit: LDS histogram of the keys that match the
//                    threshold's digits found so far, merged with atomics;
//                    the last workgroup finds the digit holding the rank
//   rc_tiles_kernel  per tile: slots below the threshold key T, slots equal
//                    to T, and how many of each are demoted (the index read
//                    once); the last workgroup locates the last slot equal to
//                    T that is taken (they are taken in slot order), then
//                    turns the counts into each tile's output offsets
//   rc_write_kernel  tiles holding reclaimed slots write them, and their
//                    demoted blocks, at those offsets; the others exit
//   rc_update_kernel index bit updates (clear this tier, set the next for
//                    demoted blocks) and the slot-table writes
//
// The plan lives in the caller's workspace; every kernel after the first reads
// it and returns at once when the call failed or has nothing left to do, so
// the host launches a fixed sequence and never waits.  The last workgroup of
// each kernel resets the counter it used, which leaves the workspace zeroed.
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
constexpr int kRcGridCount = 1024;           // workgroups of the count and tile kernels
constexpr int kRcGridPass = 512;             // workgroups of a radix pass (fewer bin merges)
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
  int find_tie;   // 1: only some slots equal to T are taken
  int tie_slot;   // last slot with the threshold key taken (-1: none; INT_MAX: all)
  int pad0;
  unsigned long long lu_min;
  unsigned long long prefix;  // the threshold's digits found so far, in place; T when done
};

struct RcWork {
  RcPlan *plan;
  unsigned *tickets;      // [(kTicketGroups + 1) * kTicketStride]
  RcPartial *partial;     // [kRcGridCount]
  unsigned *hist;         // [kRcBins]
  int4 *tile;             // [tiles] counts, then output offsets
};

constexpr size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
__host__ __device__ inline int tiles_of(long long n) { return (int)((n + kRcTile - 1) / kRcTile); }

size_t workspace_bytes_for(int32_t n) {
  const size_t tiles = (size_t)std::max(1, tiles_of(n));
  return align256(sizeof(RcPlan)) + align256(sizeof(unsigned) * (kTicketGroups + 1) * kTicketStride) +
         align256(sizeof(RcPartial) * kRcGridCount) +
         align256(sizeof(unsigned) * kRcBins) + align256(sizeof(int4) * tiles);
}

RcWork carve(void *ws, int32_t n) {
  char *p = static_cast<char *>(ws);
  const size_t tiles = (size_t)std::max(1, tiles_of(n));
  RcWork w;
  w.plan = reinterpret_cast<RcPlan *>(p);
  p += align256(sizeof(RcPlan));
  w.tickets = reinterpret_cast<unsigned *>(p);
  p += align256(sizeof(unsigned) * (kTicketGroups + 1) * kTicketStride);
  w.partial = reinterpret_cast<RcPartial *>(p);
  p += align256(sizeof(RcPartial) * kRcGridCount);
  w.hist = reinterpret_cast<unsigned *>(p);
  p += align256(sizeof(unsigned) * kRcBins);
  w.tile = reinterpret_cast<int4 *>(p);
  (void)tiles;
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

// A thread's eight slots of a tile.  Wave w of the workgroup covers slots
// [w*512, w*512 + 512) of the tile; item i = 2j + e of lane l is slot
// w*512 + 128*j + 2*l + e, so each of the four 16-byte loads of a wave reads
// 1 KiB of consecutive hashes (or stamps).  Slots past the table read as held
// with stamp 0, so nothing selects them.
struct Slots8 {
  unsigned long long h[kRcItems];
  long long lu[kRcItems];
  bool held[kRcItems];
};
__device__ __forceinline__ int slot_base(int tile) {
  return tile * kRcTile + wave_id() * (kRcTile / kWaves) + 2 * lane_id();
}
__device__ __forceinline__ int item_slot(int base, int i) { return base + 128 * (i >> 1) + (i & 1); }

__device__ __forceinline__ void load8(const RcArgs &a, int base, Slots8 &v) {
  if (base + 128 * (kRcItems / 2 - 1) + 1 < a.n) {
    // every slot of the thread is in the table: all twelve loads in flight
    // before any is used (one bounds test, so no wait between them)
    ulonglong2 h2[kRcItems / 2];
    longlong2 l2[kRcItems / 2];
    unsigned short hd[kRcItems / 2];
#pragma unroll
    for (int j = 0; j < kRcItems / 2; ++j) {
      h2[j] = *reinterpret_cast<const ulonglong2 *>(a.hash + base + 128 * j);
      l2[j] = *reinterpret_cast<const longlong2 *>(a.lu + base + 128 * j);
      hd[j] = *reinterpret_cast<const unsigned short *>(a.held + base + 128 * j);
    }
#pragma unroll
    for (int j = 0; j < kRcItems / 2; ++j) {
      v.h[2 * j] = h2[j].x;
      v.h[2 * j + 1] = h2[j].y;
      v.lu[2 * j] = l2[j].x;
      v.lu[2 * j + 1] = l2[j].y;
      v.held[2 * j] = (hd[j] & 0xffu) != 0u;
      v.held[2 * j + 1] = (hd[j] >> 8) != 0u;
    }
  } else {
#pragma unroll
    for (int i = 0; i < kRcItems; ++i) {
      const int s = item_slot(base, i);
      const bool in = s < a.n;
      v.h[i] = in ? a.hash[s] : 0ull;
      v.lu[i] = in ? a.lu[s] : 0ll;
      v.held[i] = in ? a.held[s] != 0 : true;
    }
  }
}

// Slot-order exclusive ranks of the flagged items of a workgroup's tile, and
// the flagged total.  The four per-lane pair counts (0..2 each) are packed in
// one word, 8 bits apiece, so one wave scan ranks all four 128-slot rows of
// the wave (a row holds at most 128 flags, no field overflows).  `lds` holds
// kWaves ints and is free again on return.
__device__ __forceinline__ int block_slot_rank(const bool (&f)[kRcItems], int (&rank)[kRcItems],
                                               int *lds) {
  unsigned c = 0u;
#pragma unroll
  for (int j = 0; j < kRcItems / 2; ++j) c += (unsigned)(f[2 * j] + f[2 * j + 1]) << (8 * j);
  const unsigned incl = wave_inclusive_sum(c);
  const unsigned excl = incl - c, tot = last_lane(incl);
  int row_base[kRcItems / 2], wave_total = 0;
#pragma unroll
  for (int j = 0; j < kRcItems / 2; ++j) {
    row_base[j] = wave_total;
    wave_total += (int)((tot >> (8 * j)) & 0xffu);
  }
  if (lane_id() == 0) lds[wave_id()] = wave_total;
  __syncthreads();
  int before = 0, total = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const int x = lds[w];
    before += w < wave_id() ? x : 0;
    total += x;
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < kRcItems / 2; ++j) {
    const int r = before + row_base[j] + (int)((excl >> (8 * j)) & 0xffu);
    rank[2 * j] = r;
    rank[2 * j + 1] = r + f[2 * j];
  }
  return total;
}

__device__ __forceinline__ bool status_bad(const int *status) {
  return load_agent(status) != CASCADE_OK;
}

// Calls f(tile, slots) for this workgroup's tiles (grid-stride), loading the
// next tile before working on the current one.
template <typename F>
__device__ __forceinline__ void for_tiles(const RcArgs &a, F &&f) {
  const int tiles = max(1, tiles_of(a.n));
  int t = blockIdx.x;
  if (t >= tiles) return;
  Slots8 cur, nxt;
  load8(a, slot_base(t), cur);
  for (;;) {
    const int tn = t + (int)gridDim.x;
    if (tn < tiles) load8(a, slot_base(tn), nxt);
    f(t, cur);
    if (tn >= tiles) break;
    cur = nxt;
    t = tn;
  }
}

// ------------------------------------------------------------- count kernel

__global__ __launch_bounds__(kBlock) void rc_count_kernel(RcArgs a) {
  __shared__ int s_red[kWaves * 3];
  __shared__ unsigned long long s_mm[kWaves * 2];
  __shared__ bool s_last;
  __shared__ int s_err;
  int cnt[3] = {0, 0, 0};  // empty free, cached free, negative last use
  unsigned long long mn = ~0ull, mx = 0ull;
  for_tiles(a, [&](int, const Slots8 &v) {  // past the table: held, stamp 0
#pragma unroll
    for (int j = 0; j < kRcItems; ++j) {
      const long long lu = v.lu[j];
      cnt[2] |= lu < 0;
      if (!v.held[j] && v.h[j] == 0ull) ++cnt[0];
      if (!v.held[j] && v.h[j] != 0ull && lu >= 0) {
        ++cnt[1];
        mn = min(mn, (unsigned long long)lu);
        mx = max(mx, (unsigned long long)lu);
      }
    }
  });
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
    RcPartial *p = a.w.partial + blockIdx.x;
    store_agent(&p->n_empty, cnt[0]);
    store_agent(&p->n_cached, cnt[1]);
    store_agent(&p->bad, cnt[2]);
    store_agent(&p->lu_min, mn);
    store_agent(&p->lu_max, mx);
    wait_stores();
    s_last = last_workgroup(a.w.tickets);
  }
  __syncthreads();
  if (!s_last) return;
  acquire_agent();

  // the last workgroup: totals, incoming check, plan
  int tot[3] = {0, 0, 0};
  unsigned long long tmn = ~0ull, tmx = 0ull;
  for (int g = threadIdx.x; g < (int)gridDim.x; g += kBlock) {
    const RcPartial *p = a.w.partial + g;
    tot[0] += load_agent(&p->n_empty);
    tot[1] += load_agent(&p->n_cached);
    tot[2] |= load_agent(&p->bad);
    tmn = min(tmn, load_agent(&p->lu_min));
    tmx = max(tmx, load_agent(&p->lu_max));
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
  for_tiles(a, [&](int, const Slots8 &v) {
#pragma unroll
    for (int j = 0; j < kRcItems; ++j) {
      if (v.held[j] || v.h[j] == 0ull) continue;  // only cached free slots have keys above 0
      const unsigned long long k = rc_key(v.h[j], v.lu[j], lu_min);
      if (shr64(k, shift + dbits) == hi)
        atomicAdd(&s_hist[(unsigned)(k >> shift) & dmask], 1u);
    }
  });
  __syncthreads();
  for (int b = threadIdx.x; b < nbins; b += kBlock) {
    const unsigned v = s_hist[b];
    if (v) atomicAdd(&a.w.hist[b], v);
  }
  wait_stores();
  __syncthreads();
  if (threadIdx.x == 0) s_last = last_workgroup(a.w.tickets);
  __syncthreads();
  if (!s_last) return;
  acquire_agent();

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

// ------------------------------------------------------ per-tile counts

__device__ __forceinline__ bool demotable(const RcArgs &a, unsigned long long h) {
  if (a.tier >= 2 || h == 0ull) return false;
  if (!a.index) return true;
  const IndexSlot *e = index_find(a.index, a.index_mask, h);
  return e == nullptr || (e->tiers & ~((2u << a.tier) - 1u)) == 0u;  // no deeper tier
}

// a tile's four counts, written by another workgroup as two atomic words
__device__ __forceinline__ int4 load_rec(const unsigned long long *rec64, int t) {
  const unsigned long long u = load_agent(rec64 + 2 * t), w = load_agent(rec64 + 2 * t + 1);
  return make_int4((int)(unsigned)u, (int)(unsigned)(u >> 32), (int)(unsigned)w,
                   (int)(unsigned)(w >> 32));
}

// Per tile: slots below T, slots equal to T, and the demoted ones among
// each.  The last workgroup finds the last slot equal to T that is taken
// (the take-th in slot order), then writes every tile's output offsets and
// counts: tile[t] = (reclaimed before t, demoted before t, reclaimed in t,
// demoted in t).
__global__ __launch_bounds__(kBlock) void rc_tiles_kernel(RcArgs a) {
  __shared__ int s_red[kWaves * 4];
  __shared__ bool s_last;
  __shared__ int s_hit[2];
  const RcPlan *P = a.w.plan;
  if (!P->ok) return;
  const int tiles = max(1, tiles_of(a.n));
  const unsigned long long T = P->prefix, lu_min = P->lu_min;
  unsigned long long *rec64 = reinterpret_cast<unsigned long long *>(a.w.tile);
  for_tiles(a, [&](int tile, const Slots8 &v) {
    int c[4] = {0, 0, 0, 0};
#pragma unroll
    for (int j = 0; j < kRcItems; ++j) {
      const unsigned long long k = rc_key(v.h[j], v.lu[j], lu_min);
      const bool below = !v.held[j] && k < T, equal = !v.held[j] && k == T;
      const bool dem = (below || equal) && demotable(a, v.h[j]);
      c[0] += below;
      c[1] += equal;
      c[2] += below && dem;
      c[3] += equal && dem;
    }
    block_sum<4, int>(c, s_red);
    if (threadIdx.x == 0) {  // (x, y) and (z, w) of the tile's int4, as two atomic words
      store_agent(rec64 + 2 * tile, (unsigned long long)(unsigned)c[0] |
                                        ((unsigned long long)(unsigned)c[1] << 32));
      store_agent(rec64 + 2 * tile + 1, (unsigned long long)(unsigned)c[2] |
                                            ((unsigned long long)(unsigned)c[3] << 32));
    }
  });
  if (threadIdx.x == 0) {
    wait_stores();
    s_last = last_workgroup(a.w.tickets);
  }
  __syncthreads();
  if (!s_last) return;
  acquire_agent();
  Slots8 v;

  // the last workgroup.  1: the tile holding the take-th slot equal to T
  const int take = P->take;
  const int per = (tiles + kBlock - 1) / kBlock;
  const int t0 = min(tiles, (int)threadIdx.x * per), t1 = min(tiles, t0 + per);
  int cut = take == 0 ? -1 : tiles;  // tiles before `cut` give all their slots equal to T
  int r_cut = 0, dem_cut = 0, tie_slot = take == 0 ? -1 : INT_MAX;
  if (threadIdx.x == 0) s_hit[0] = -1;
  if (P->find_tie) {
    int sum = 0;
    for (int t = t0; t < t1; ++t) sum += (int)(load_agent(rec64 + 2 * t) >> 32);
    int ex[1] = {sum}, tot[1];
    block_exclusive_scan<1, int>(ex, tot, s_red);
    if (take > ex[0] && take <= ex[0] + sum) {
      int before = ex[0];
      for (int t = t0; t < t1; ++t) {
        const int ct = (int)(load_agent(rec64 + 2 * t) >> 32);
        if (take <= before + ct) {
          s_hit[0] = t;
          s_hit[1] = take - before;  // 1-based rank inside tile t
          break;
        }
        before += ct;
      }
    }
    __syncthreads();
    if (s_hit[0] < 0) {  // the counts disagree with the plan: stop the call
      if (threadIdx.x == 0) {
        store_agent(a.status, (int)CASCADE_EINTERNAL);
        a.w.plan->ok = 0;
      }
      return;
    }
    cut = s_hit[0];
    r_cut = s_hit[1];
    // inside the cut tile: the slot of the r_cut-th equal key, and how many
    // of the first r_cut are demoted
    const int base = slot_base(cut);
    load8(a, base, v);
    bool eq[kRcItems];
    int rk[kRcItems];
#pragma unroll
    for (int j = 0; j < kRcItems; ++j) eq[j] = !v.held[j] && rc_key(v.h[j], v.lu[j], lu_min) == T;
    block_slot_rank(eq, rk, s_red);
    int d[1] = {0};
#pragma unroll
    for (int j = 0; j < kRcItems; ++j) {
      if (eq[j] && rk[j] < r_cut) {
        d[0] += demotable(a, v.h[j]);
        if (rk[j] == r_cut - 1) s_hit[0] = item_slot(base, j);
      }
    }
    block_sum<1, int>(d, s_red);
    tie_slot = s_hit[0];
    dem_cut = d[0];
  }
  // 2: offsets, in tile order
  int sums[2] = {0, 0};
  for (int t = t0; t < t1; ++t) {
    const int4 q = load_rec(rec64, t);
    sums[0] += q.x + (t < cut ? q.y : (t == cut ? r_cut : 0));
    sums[1] += q.z + (t < cut ? q.w : (t == cut ? dem_cut : 0));
  }
  int tot[2];
  block_exclusive_scan<2, int>(sums, tot, s_red);
  int off_sel = sums[0], off_dem = sums[1];
  for (int t = t0; t < t1; ++t) {
    const int4 q = load_rec(rec64, t);
    const int ns = q.x + (t < cut ? q.y : (t == cut ? r_cut : 0));
    const int nd = q.z + (t < cut ? q.w : (t == cut ? dem_cut : 0));
    a.w.tile[t] = make_int4(off_sel, off_dem, ns, nd);
    off_sel += ns;
    off_dem += nd;
  }
  if (threadIdx.x == 0) {
    RcPlan *W = a.w.plan;
    W->tie_slot = tie_slot;
    if (tot[0] != P->total || tot[1] > a.max_out) {  // must reclaim exactly total
      store_agent(a.status, (int)CASCADE_EINTERNAL);
      W->ok = 0;
    } else if (a.n_out_dev) {
      store_agent(a.n_out_dev, tot[1]);
    }
  }
}

// ---------------------------------------------------------------- writes

// Tiles holding reclaimed slots write them (ascending: freed, then placed)
// and their demoted blocks at the offsets the counts gave.
__global__ __launch_bounds__(kBlock) void rc_write_kernel(RcArgs a) {
  __shared__ int s_red[kWaves];
  const RcPlan *P = a.w.plan;
  if (!P->ok) return;
  const int4 rec = a.w.tile[blockIdx.x];
  if (rec.z == 0) return;  // nothing reclaimed here (so nothing demoted either)
  const unsigned long long T = P->prefix, lu_min = P->lu_min;
  const int tie_slot = P->tie_slot, need = a.need, total = P->total;
  const int base = slot_base(blockIdx.x);
  Slots8 v;
  load8(a, base, v);
  bool sel[kRcItems], dem[kRcItems];
#pragma unroll
  for (int j = 0; j < kRcItems; ++j) {
    const unsigned long long k = rc_key(v.h[j], v.lu[j], lu_min);
    sel[j] = !v.held[j] && (k < T || (k == T && item_slot(base, j) <= tie_slot));
    dem[j] = sel[j] && demotable(a, v.h[j]);
  }
  int rs[kRcItems], rd[kRcItems];
  const int n_sel = block_slot_rank(sel, rs, s_red);
  const int n_dem = block_slot_rank(dem, rd, s_red);
  bool bad = n_sel != rec.z || n_dem != rec.w;
#pragma unroll
  for (int j = 0; j < kRcItems; ++j) {
    const int slot = item_slot(base, j);
    if (sel[j]) {
      const int p = rec.x + rs[j];
      if (p < need) a.freed[p] = slot;
      else if (p < total) a.placed[p - need] = slot;
      else bad = true;
    }
    if (dem[j]) {
      const int q = rec.y + rd[j];
      if (q < a.max_out) {
        cascade_demotion_t d;
        d.hash = v.h[j];
        d.last_use_ns = v.lu[j];
        d.src_slot = slot;
        d.pad = 0;
        a.outgoing[q] = d;
      } else {
        bad = true;
      }
    }
  }
  if (bad) store_agent(a.status, (int)CASCADE_EINTERNAL);
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
      ((uintptr_t)table->held & 1))
    return CASCADE_EINVAL;  // the kernels load slot pairs with vector loads
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
  const int total_cap = (int)std::min<long long>((long long)need + max_incoming, n);
  hipLaunchKernelGGL(rc_count_kernel, dim3(std::min(tiles, kRcGridCount)), dim3(kBlock), 0, s,
                     a);
  for (int p = 0; p < kRcPasses; ++p)
    hipLaunchKernelGGL(rc_pass_kernel, dim3(std::min(tiles, kRcGridPass)), dim3(kBlock), 0, s,
                       a);
  hipLaunchKernelGGL(rc_tiles_kernel, dim3(std::min(tiles, kRcGridCount)), dim3(kBlock), 0, s,
                     a);
  hipLaunchKernelGGL(rc_write_kernel, dim3(tiles), dim3(kBlock), 0, s, a);
  if (total_cap > 0)
    hipLaunchKernelGGL(rc_update_kernel, dim3((total_cap + kBlock - 1) / kBlock), dim3(kBlock),
                       0, s, a);
  return hipGetLastError() == hipSuccess ? CASCADE_OK : CASCADE_EHIP;
}
