// cascade_reclaim.hip -- per-tier LRU reclamation on gfx950 (Section 4.4,
// prefix hit detection: free blocks are reclaimed least-recently-used within
// each tier, so hot prefixes stay in the fast tiers and cold ones spill one
// tier deeper).
//
// One call reclaims `total` = need + n_incoming free slots of one tier.  The
// reclaimed set is the `total` smallest free slots under the key
//   empty slot -> 0,   cached block -> 1 + (last_use - min cached last_use),
// ties by slot.  The table is read in tiles of 2048 slots, 8 consecutive
// slots per thread with 16-byte loads, three times per call:
//
//   rc_count_kernel    per-workgroup counts of empty / cached free slots and
//                      the cached last-use range, and (one call per tier) a
//                      share of the incoming blocks' hashes checked
//   rc_hist_kernel     every workgroup derives the cached last-use range and
//                      the key's size from those counts, then adds its tiles
//                      to a histogram of the key's top digit, 8 bits
//   rc_compact_kernel  every workgroup derives the call's plan from the
//                      counts and the incoming count (the checks, which
//                      slots are reclaimed; workgroup 0 stores it) and finds
//                      the bucket holding the threshold in that histogram,
//                      then per tile, in slot order: the slots certainly
//                      reclaimed (empty ones, keys below the bucket) and the
//                      candidates (keys inside it; with empty slots alone
//                      enough, the empty slots), each with its key, its block
//                      and, on tiers 0 and 1, its index slot and whether it
//                      is demoted (the index as it was when the call began),
//                      in one chunk of a list reserved with one atomic add on
//                      one of 16 region counters; a histogram of the
//                      candidates' next 12-bit digit
//
// Then, over the list only:
//
//   rc_select_kernel   every workgroup takes the next digit of the threshold
//                      key T from that histogram and a share of the list:
//                      candidates below that digit go to their tile's
//                      counters, those on it are staged; the last workgroup
//                      finds T's remaining digits among the staged ones, the
//                      last taken slot with key T (ties are taken in slot
//                      order, so by tile, then by position in the tile's
//                      chunk), and every tile's output offsets
//   rc_write_kernel    a workgroup per tile with reclaimed slots: their
//                      positions in slot order, the freed / placed / outgoing
//                      entries, the index bit updates (clear this tier, set
//                      the next for demoted blocks) at the index slots the
//                      compaction found (tier 2 looks them up here) and the
//                      slot-table writes
//
// Values the next kernel needs are handed over by the kernel boundary, not
// by a last workgroup: each kernel recomputes what it needs from the
// previous one's output (the plan from the counts, the bucket from the
// histogram).  The plan lives in the caller's workspace; every kernel after
// the compaction reads it and returns at once when the call failed or has
// nothing left to do, so the host launches a fixed sequence and never waits.
// Counters and histograms are reset by the kernel after their last reader.
//
// Neither the count nor the histogram pass depends on the tier above (a
// tier's table changes only in its own write kernel; the incoming count is
// first needed by the compaction), so a chain HBM -> DRAM -> NVMe in one call
// launches each of those two passes once for all three tables, then the
// rest tier by tier.
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
constexpr int kRcGridCount = 512;            // workgroups of the count kernel
constexpr int kRcGridCompact = 1024;         // workgroups of the compaction kernel
constexpr int kRcGridHist = 512;             // workgroups of the histogram (fewer bin merges)
constexpr int kDigit0 = 8, kDigitN = 12;     // top digit, later digits
constexpr int kRcBins = 1 << kDigitN;
constexpr int kHistCopies = 8;               // copies of the top-digit histogram (fewer
                                             // atomics per address), workgroup b adds to b % 8
constexpr int kSelGrid = 64;                 // workgroups of the select kernel
constexpr int kStageCap = 65536;             // candidates on the threshold's first digits kept
constexpr int kStageLds = 2048;              // of them, read into the last workgroup's LDS
constexpr int kTieLds = 256;                 // staged ones up to which the tie is found in LDS
constexpr int kTilesLds = 2048;              // tiles whose counts the last workgroup keeps in LDS
constexpr int kModeCached = 0, kModeEmpty = 1;
// The list is reserved in kListGroups regions, tile t in region t % kListGroups
// with its own counter, so no counter takes more than a few hundred adds;
// a region holds every slot of its tiles.
constexpr int kListGroups = 16;
constexpr int kCountStride = 32;  // one counter per 128-byte line
// list entry: slot in bits 0..29, certainly reclaimed in bit 30, demoted in bit 31
constexpr unsigned kEntSlot = (1u << 30) - 1u, kEntSure = 1u << 30, kEntDem = 1u << 31;
constexpr unsigned kNoPos = ~0u;  // a block absent from the index (or no index, or no block)
constexpr unsigned kFindPos = ~1u;  // not looked up yet (tier 2, where nothing is demoted)

struct RcPartial {
  int n_empty, n_cached, bad, pad;
  unsigned long long lu_min, lu_max;
};

struct alignas(256) RcPlan {
  int ok;         // 1: the call proceeds (checked, room enough)
  int total;      // need + n_in
  int n_in;
  int mode;       // kModeCached: cached blocks are reclaimed; kModeEmpty: empty slots only
  int width;      // bits of the key
  int shift;      // low bit of the top digit
  int dbits;      // width of the top digit
  int rank;       // 0-based rank sought among cached keys (kModeEmpty: among empty slots)
  int bucket;     // the top digit of the threshold key
  int brank;      // the rank sought inside the bucket
  int tie_slot;   // last reclaimed slot with the threshold key (-1: none)
  int pad;
  unsigned long long lu_min;
  unsigned long long thresh;  // the threshold key T
};

// The head (fixed offsets; its counters and histograms are zero when a call
// starts) runs through stage_ent, then the body (sized by the table).
struct RcWork {
  RcPlan *plan;
  unsigned *tickets;      // [(kTicketGroups + 1) * kTicketStride]
  RcPartial *partial;     // [kRcGridCount]
  unsigned *hist;         // [kHistCopies][1 << kDigit0] top digit
  unsigned *sub;          // [kRcBins] candidates' next digit
  unsigned *count;        // [kListGroups * kCountStride] entries reserved per region
  unsigned *stage_n;      // candidates staged by the select kernel
  unsigned long long *stage_key;  // [kStageCap]
  unsigned *stage_ent;            // [kStageCap]
  int4 *rec;              // [tiles] the tile's chunk: start, sure, candidates, sure demoted
  int4 *off;              // [tiles] counts, then output offsets
  unsigned long long *key;  // [n_slots] list: keys
  unsigned *ent;            // [n_slots] list: slot and flags
  unsigned *pos;            // [n_slots] list: the block's index slot (kNoPos: none)
  unsigned long long *hash;  // [n_slots] list: the slot's block (0: empty)
};

constexpr size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
__host__ __device__ inline int tiles_of(long long n) { return (int)((n + kRcTile - 1) / kRcTile); }
// entries of one list region: every slot of ceil(tiles / kListGroups) tiles
__host__ __device__ inline long long region_cap(long long n) {
  const long long tiles = tiles_of(n) > 0 ? tiles_of(n) : 1;
  return (tiles + kListGroups - 1) / kListGroups * kRcTile;
}

// A workspace is a head of fixed size (the plan, counters, histograms and
// the stage: what must be zero when a call starts, at offsets that do not
// depend on the table) and a body sized by the table (per-tile records and
// the list, rewritten before they are read).  One call's workspace is its
// head then its body, so a workspace sized for n slots serves every table
// of at most n slots; a chain keeps its three heads first.
constexpr size_t head_bytes() {
  return align256(sizeof(RcPlan)) + align256(sizeof(unsigned) * (kTicketGroups + 1) * kTicketStride) +
         align256(sizeof(RcPartial) * kRcGridCount) +
         align256(sizeof(unsigned) * kHistCopies * (1 << kDigit0)) +
         align256(sizeof(unsigned) * kRcBins) +
         align256(sizeof(unsigned) * kListGroups * kCountStride) + align256(sizeof(unsigned)) +
         align256(sizeof(unsigned long long) * kStageCap) + align256(sizeof(unsigned) * kStageCap);
}
size_t body_bytes(int32_t n) {
  const size_t tiles = (size_t)std::max(1, tiles_of(n));
  const size_t slots = (size_t)(kListGroups * region_cap(n));
  return 2 * align256(sizeof(int4) * tiles) + 2 * align256(sizeof(unsigned long long) * slots) +
         2 * align256(sizeof(unsigned) * slots);
}
size_t workspace_bytes_for(int32_t n) { return head_bytes() + body_bytes(n); }

RcWork carve(void *head, void *body, int32_t n) {
  char *p = static_cast<char *>(head);
  const size_t tiles = (size_t)std::max(1, tiles_of(n));
  const size_t slots = (size_t)(kListGroups * region_cap(n));
  RcWork w;
  w.plan = reinterpret_cast<RcPlan *>(p);
  p += align256(sizeof(RcPlan));
  w.tickets = reinterpret_cast<unsigned *>(p);
  p += align256(sizeof(unsigned) * (kTicketGroups + 1) * kTicketStride);
  w.partial = reinterpret_cast<RcPartial *>(p);
  p += align256(sizeof(RcPartial) * kRcGridCount);
  w.hist = reinterpret_cast<unsigned *>(p);
  p += align256(sizeof(unsigned) * kHistCopies * (1 << kDigit0));
  w.sub = reinterpret_cast<unsigned *>(p);
  p += align256(sizeof(unsigned) * kRcBins);
  w.count = reinterpret_cast<unsigned *>(p);
  p += align256(sizeof(unsigned) * kListGroups * kCountStride);
  w.stage_n = reinterpret_cast<unsigned *>(p);
  p += align256(sizeof(unsigned));
  w.stage_key = reinterpret_cast<unsigned long long *>(p);
  p += align256(sizeof(unsigned long long) * kStageCap);
  w.stage_ent = reinterpret_cast<unsigned *>(p);
  p = static_cast<char *>(body);
  w.rec = reinterpret_cast<int4 *>(p);
  p += align256(sizeof(int4) * tiles);
  w.off = reinterpret_cast<int4 *>(p);
  p += align256(sizeof(int4) * tiles);
  w.key = reinterpret_cast<unsigned long long *>(p);
  p += align256(sizeof(unsigned long long) * slots);
  w.ent = reinterpret_cast<unsigned *>(p);
  p += align256(sizeof(unsigned) * slots);
  w.pos = reinterpret_cast<unsigned *>(p);
  p += align256(sizeof(unsigned) * slots);
  w.hash = reinterpret_cast<unsigned long long *>(p);
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


// A workgroup's place in the part of the grid that serves one table: its
// index there and the part's size (the whole grid unless one launch serves
// several tables).
struct Part {
  int block, count;
};
__device__ __forceinline__ Part whole_grid() { return {(int)blockIdx.x, (int)gridDim.x}; }

// The workgroup's first tile (nothing is read past the table), loaded
// before the kernel reads anything else, so the table loads do not wait for it.
__device__ __forceinline__ Slots8 load_first(const RcArgs &a, Part g) {
  Slots8 v;
  load8(a, slot_base(g.block), v);
  return v;
}
// Calls f(tile, slots) for this workgroup's tiles (part-stride), loading
// the next tile before working on the current one; `first` is the first
// tile's slots.
template <typename F>
__device__ __forceinline__ void for_tiles(const RcArgs &a, Part g, const Slots8 &first, F &&f) {
  const int tiles = max(1, tiles_of(a.n));
  int t = g.block;
  if (t >= tiles) return;
  Slots8 cur = first, nxt;
  for (;;) {
    const int tn = t + g.count;
    if (tn < tiles) load8(a, slot_base(tn), nxt);
    f(t, cur);
    if (tn >= tiles) break;
    cur = nxt;
    t = tn;
  }
}

// Up to three tables served by one launch of the count or histogram kernel:
// table k takes workgroups [first[k], first[k + 1]) (first[n] = the grid).
// A chain of tiers launches these two passes once for all its tables, since
// neither depends on the tier above.
struct RcTables {
  RcArgs t[3];
  int n;
  int first[3];
  int check_in;  // one call per tier: the count kernel checks the incoming hashes, and
                 // the incoming count is final when the histogram is built
};
// Calls f(table, part) for the table this workgroup serves (constant
// indices into the launch's arguments, one branch per table).
template <typename F>
__device__ __forceinline__ void with_table(const RcTables &m, F &&f) {
  const int b = (int)blockIdx.x, grid = (int)gridDim.x;
  if (m.n > 2 && b >= m.first[2]) f(m.t[2], Part{b - m.first[2], grid - m.first[2]});
  else if (m.n > 1 && b >= m.first[1])
    f(m.t[1], Part{b - m.first[1], (m.n > 2 ? m.first[2] : grid) - m.first[1]});
  else f(m.t[0], Part{b, m.n > 1 ? m.first[1] : grid});
}

// ------------------------------------------------------------- count kernel

__device__ __forceinline__ void count_table(const RcArgs &a, Part g, bool check_in, int *s_red,
                                            unsigned long long *s_mm) {
  int cnt[3] = {0, 0, 0};  // empty free, cached free, bad data (negative last use, hash 0 in)
  unsigned long long mn = ~0ull, mx = 0ull;
  const int n_in_all = check_in && a.n_in_dev ? load_agent(a.n_in_dev) : 0;
  for_tiles(a, g, load_first(a, g), [&](int, const Slots8 &v) {  // past the table: held, stamp 0
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
  // this workgroup's share of the incoming blocks: none may have hash 0
  // (a chain's own demotions never do, and are not checked)
  if (n_in_all >= 0 && n_in_all <= a.max_in)
    for (int j = g.block * kBlock + (int)threadIdx.x; j < n_in_all; j += g.count * kBlock)
      cnt[2] |= a.incoming[j].hash == 0ull;
  block_sum<3, int>(cnt, s_red);
  mn = wave_min(mn);
  mx = wave_max(mx);
  if (lane_id() == 0) {
    s_mm[wave_id() * 2] = mn;
    s_mm[wave_id() * 2 + 1] = mx;
  }
  __syncthreads();
  if (threadIdx.x == 0) {  // read by the later kernels
    for (int w = 1; w < kWaves; ++w) {
      mn = min(mn, s_mm[w * 2]);
      mx = max(mx, s_mm[w * 2 + 1]);
    }
    RcPartial *p = a.w.partial + g.block;
    p->n_empty = cnt[0];
    p->n_cached = cnt[1];
    p->bad = cnt[2];
    p->lu_min = mn;
    p->lu_max = mx;
  }
}

// Per workgroup of a table: counts of empty and cached free slots, the
// cached last-use range and bad data, as one partial record.
__global__ __launch_bounds__(kBlock) void rc_count_kernel(RcTables m) {
  __shared__ int s_red[kWaves * 3];
  __shared__ unsigned long long s_mm[kWaves * 2];
  with_table(m, [&](const RcArgs &a, Part g) { count_table(a, g, m.check_in != 0, s_red, s_mm); });
}

// The table's totals from the count kernel's partials, computed alike by
// every workgroup that needs them: free slots, bad data, the cached
// last-use range and the key's size.
struct RangeCalc {
  int n_empty, n_cached, bad;
  int width, shift, dbits;
  unsigned long long lu_min;
};
__device__ __forceinline__ RangeCalc range_of(const RcArgs &a, int *s_red,
                                              unsigned long long *s_mm) {
  const int g_count = min(max(1, tiles_of(a.n)), kRcGridCount);
  int tot[3] = {0, 0, 0};
  unsigned long long tmn = ~0ull, tmx = 0ull;
  static_assert(kRcGridCount % kBlock == 0, "whole rounds of partials");
#pragma unroll
  for (int r = 0; r < kRcGridCount / kBlock; ++r) {  // all loads in flight at once
    const int g = r * kBlock + (int)threadIdx.x;
    if (g < g_count) {
      const RcPartial *p = a.w.partial + g;
      tot[0] += p->n_empty;
      tot[1] += p->n_cached;
      tot[2] |= p->bad;
      tmn = min(tmn, p->lu_min);
      tmx = max(tmx, p->lu_max);
    }
  }
  block_sum<3, int>(tot, s_red);
  tmn = wave_min(tmn);
  tmx = wave_max(tmx);
  if (lane_id() == 0) {
    s_mm[wave_id() * 2] = tmn;
    s_mm[wave_id() * 2 + 1] = tmx;
  }
  __syncthreads();
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    tmn = min(tmn, s_mm[w * 2]);
    tmx = max(tmx, s_mm[w * 2 + 1]);
  }
  __syncthreads();
  RangeCalc r;
  r.n_empty = tot[0];
  r.n_cached = tot[1];
  r.bad = tot[2];
  r.lu_min = tmn;
  r.width = tot[1] > 0 ? bit_width64(1ull + (tmx - tmn)) : 0;
  r.dbits = min(r.width, kDigit0);
  r.shift = r.width - r.dbits;
  return r;
}

// The call's plan: the checks (an earlier failure in the chain, bad data,
// the incoming count, room), then which slots are reclaimed.
struct PlanCalc {
  int err;   // 0, 1 (an earlier call failed) or a negative code
  int total, n_in, mode, rank;
};
__device__ __forceinline__ PlanCalc plan_of(const RcArgs &a, const RangeCalc &r, int status_was,
                                            int n_in) {
  PlanCalc c;
  c.err = status_was != CASCADE_OK ? 1 : 0;
  if (c.err == 0 && (r.bad || n_in < 0 || n_in > a.max_in)) c.err = CASCADE_EINVAL;
  const long long total = (long long)a.need + n_in;
  if (c.err == 0 && total > (long long)r.n_empty + r.n_cached) c.err = CASCADE_ENOSPC;
  c.total = (int)total;
  c.n_in = n_in;
  if (total <= r.n_empty) {
    // empty slots suffice: the first `total` of them in slot order
    c.mode = kModeEmpty;
    c.rank = (int)total - 1;
  } else {
    // every empty slot plus the (total - n_empty) least recent cached ones
    c.mode = kModeCached;
    c.rank = (int)(total - r.n_empty - 1);
  }
  return c;
}

// ------------------------------------------------------------ top digit

// Every workgroup of a table derives the cached last-use range from the
// count kernel's partials, then adds its tiles to the histogram of the
// key's top digit (8 copies, workgroup b adds to copy b % 8).  When the
// incoming count is already final (one call per tier) a call that will not
// reclaim cached blocks skips it; in a chain call it is built whether or not
// the call will need it (the incoming count is known only when the tier
// above is done).
__device__ __forceinline__ void hist_table(const RcArgs &a, Part g, bool plan_known,
                                           unsigned *s_hist, int *s_red,
                                           unsigned long long *s_mm) {
  constexpr int kBins0 = 1 << kDigit0;
  static_assert(kBins0 == kBlock, "one bin per thread");
  const Slots8 first = load_first(a, g);
  const int status_was = plan_known ? load_agent(a.status) : CASCADE_OK;
  const int n_in = plan_known && a.n_in_dev ? load_agent(a.n_in_dev) : 0;
  const RangeCalc r = range_of(a, s_red, s_mm);
  const int t = threadIdx.x;
  if (r.bad || r.n_cached == 0) return;  // uniform: every workgroup computes r alike
  if (plan_known) {
    const PlanCalc pc = plan_of(a, r, status_was, n_in);
    if (pc.err != 0 || pc.mode != kModeCached) return;  // nothing will read the histogram
  }
  const int shift = r.shift;
  const unsigned long long lu_min = r.lu_min;
  s_hist[t] = 0u;
  __syncthreads();
  for_tiles(a, g, first, [&](int, const Slots8 &v) {
#pragma unroll
    for (int j = 0; j < kRcItems; ++j) {
      if (v.held[j] || v.h[j] == 0ull) continue;  // only cached free slots have keys above 0
      // below 2^dbits: every stamp lies in [lu_min, lu_max]
      const unsigned b = (unsigned)shr64(rc_key(v.h[j], v.lu[j], lu_min), shift);
      atomicAdd(&s_hist[b & (kBins0 - 1)], 1u);
    }
  });
  __syncthreads();
  const unsigned v = s_hist[t];
  if (v) atomicAdd(a.w.hist + (g.block % kHistCopies) * kBins0 + t, v);
}

__global__ __launch_bounds__(kBlock) void rc_hist_kernel(RcTables m) {
  __shared__ unsigned s_hist[1 << kDigit0];
  __shared__ int s_red[kWaves * 3];
  __shared__ unsigned long long s_mm[kWaves * 2];
  with_table(m, [&](const RcArgs &a, Part g) {
    hist_table(a, g, m.check_in != 0, s_hist, s_red, s_mm);
  });
}

// ------------------------------------------------------------ compaction

// For the tile's listed blocks of tiers 0 and 1 (want[j]): whether
// reclaiming them demotes them (no deeper tier holds the block in the index)
// and their index slots for the later bit updates.  The blocks are gathered
// in LDS and spread over the workgroup, kLookBatch lookups per thread in
// flight, so up to kLookBatch * kBlock lookups of a tile cost one memory
// round trip whichever threads hold them.  (Two per thread would take the
// kernel past 128 VGPRs, below four waves per SIMD, which the full-table
// read of the deepest tier needs.)  `look` holds kRcTile hashes, each
// replaced by its result, and is free again on return.
constexpr int kLookBatch = 1;
__device__ __forceinline__ void demotions(const RcArgs &a, const unsigned long long (&h)[kRcItems],
                                          const bool (&want)[kRcItems], bool (&dem)[kRcItems],
                                          unsigned (&ip)[kRcItems], unsigned long long *look,
                                          int *s_rank) {
#pragma unroll
  for (int j = 0; j < kRcItems; ++j) {
    dem[j] = false;
    ip[j] = kNoPos;
  }
  if (a.tier >= 2) return;  // nothing is demoted from the deepest tier
  int wr[kRcItems];
  const int n_want = block_slot_rank(want, wr, s_rank);
  if (n_want == 0) return;  // uniform
#pragma unroll
  for (int j = 0; j < kRcItems; ++j)
    if (want[j]) look[wr[j]] = h[j];
  __syncthreads();
  const unsigned deeper = ~((2u << a.tier) - 1u);
  for (int i0 = (int)threadIdx.x; i0 < n_want; i0 += kLookBatch * kBlock) {
    unsigned long long hh[kLookBatch];
    bool w[kLookBatch];
#pragma unroll
    for (int q = 0; q < kLookBatch; ++q) {
      const int i = i0 + q * kBlock;
      w[q] = i < n_want && a.index;
      hh[q] = i < n_want ? look[i] : 0ull;
    }
    int pos[kLookBatch];
    unsigned tiers[kLookBatch];
    index_find_n(a.index, a.index_mask, hh, w, pos, tiers);
#pragma unroll
    for (int q = 0; q < kLookBatch; ++q) {
      const int i = i0 + q * kBlock;
      // slot (below 2^30) | demoted in bit 31; kNoPos's slot bits: absent
      // (each entry is read and rewritten by the same thread)
      if (i < n_want)
        look[i] = (pos[q] >= 0 ? (unsigned)pos[q] : (kNoPos >> 1)) |
                  ((pos[q] < 0 || (tiers[q] & deeper) == 0u) ? 0x80000000u : 0u);
    }
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < kRcItems; ++j) {
    if (!want[j]) continue;
    const unsigned v = (unsigned)look[wr[j]];
    const unsigned sl = v & 0x7fffffffu;
    ip[j] = sl == (kNoPos >> 1) ? kNoPos : sl;
    dem[j] = (v >> 31) != 0u;
  }
  __syncthreads();
}

// Per tile, in slot order: the slots certainly reclaimed and the candidates,
// as one chunk of the list (start, certain count, candidate count, certain
// demoted count in rec[tile]); the candidates' next digit is histogrammed.
// Demotion is decided here, on the index as it was when the call began.
__device__ __forceinline__ void compact_table(const RcArgs &a, Part g) {
  __shared__ unsigned s_sub[kRcBins];
  __shared__ unsigned long long s_look[kRcTile];
  __shared__ int s_rank[kWaves];
  __shared__ int s_red[kWaves * 3];
  __shared__ unsigned long long s_mm[kWaves * 2];
  __shared__ int s_start;
  __shared__ int s_found[2];
  const bool lead = g.block == 0;  // stores the plan
  const Slots8 first = load_first(a, g);
  const int t = threadIdx.x;
  // the top digit's histogram, the status and the incoming count, requested
  // with the partials (the histogram is used when cached blocks are needed)
  constexpr int kBins0 = 1 << kDigit0;
  static_assert(kBins0 == kBlock, "one bin per thread");
  unsigned hv[kHistCopies];
#pragma unroll
  for (int c = 0; c < kHistCopies; ++c) hv[c] = load_agent(a.w.hist + c * kBins0 + t);
  const int status_was = load_agent(a.status);
  const int n_in = a.n_in_dev ? load_agent(a.n_in_dev) : 0;
  // the call's plan, alike in every workgroup; workgroup 0 stores it for
  // the later kernels and reports a failed check
  const RangeCalc rg = range_of(a, s_red, s_mm);
  const PlanCalc pc = plan_of(a, rg, status_was, n_in);
  RcPlan *P = a.w.plan;
  if (lead && t == 0) {
    if (pc.err < 0) store_agent(a.status, pc.err);
    P->ok = pc.err == 0;
    P->total = pc.total;
    P->n_in = pc.n_in;
    P->mode = pc.mode;
    P->width = rg.width;
    P->shift = rg.shift;
    P->dbits = rg.dbits;
    P->rank = pc.rank;
    P->bucket = 0;
    P->brank = 0;
    P->tie_slot = -1;
    P->lu_min = rg.lu_min;
    P->thresh = 0ull;
  }
  if (pc.err != 0) return;  // uniform
  const bool cached = pc.mode == kModeCached;
  const int shift = rg.shift, rank = pc.rank;
  const unsigned long long lu_min = rg.lu_min;
  unsigned long long bucket = 0;
  if (cached) {
    // the bucket holding the sought rank, from the histogram's copies
    // (every workgroup alike; workgroup 0 stores it for the select kernel)
    unsigned v = 0;
#pragma unroll
    for (int c = 0; c < kHistCopies; ++c) v += hv[c];
    if (t == 0) s_found[0] = -1;
    int ex[1] = {(int)v}, tot[1];
    block_exclusive_scan<1, int>(ex, tot, s_red);
    if (rank >= ex[0] && rank < ex[0] + (int)v) {
      s_found[0] = t;
      s_found[1] = rank - ex[0];
    }
    __syncthreads();
    if (s_found[0] < 0) {  // the counts disagree with the plan: stop the call
      if (lead && t == 0) {
        store_agent(a.status, (int)CASCADE_EINTERNAL);
        P->ok = 0;
      }
      return;
    }
    bucket = (unsigned long long)s_found[0];
    if (lead && t == 0) {
      P->bucket = s_found[0];
      P->brank = s_found[1];
    }
  }
  const int d2 = cached ? min(shift, kDigitN) : 0, s2 = shift - d2;
  const unsigned m2 = (1u << d2) - 1u;
  // One tile per workgroup: its few candidates add to the global histogram
  // as they are listed, so nothing is left to flush when the kernel ends;
  // several tiles per workgroup (the deepest tier) count in LDS first.
  const bool sub_direct = max(1, tiles_of(a.n)) <= g.count;  // uniform
  if (d2 > 0 && !sub_direct)
    for (int b = t; b < (1 << d2); b += kBlock) s_sub[b] = 0u;
  __syncthreads();
  for_tiles(a, g, first, [&](int tile, const Slots8 &v) {
    bool f[kRcItems], sure[kRcItems];
    unsigned long long k[kRcItems];
#pragma unroll
    for (int j = 0; j < kRcItems; ++j) {
      const bool fr = !v.held[j], empty = fr && v.h[j] == 0ull, full = fr && v.h[j] != 0ull;
      k[j] = full ? rc_key(v.h[j], v.lu[j], lu_min) : 0ull;
      if (cached) {
        const unsigned long long top = shr64(k[j], shift);
        sure[j] = empty || (full && top < bucket);
        f[j] = sure[j] || (full && top == bucket);
      } else {
        sure[j] = false;
        f[j] = empty;
      }
    }
    // the index lookups first: their latency overlaps the workgroup scans
    // (tier 2 demotes nothing: its reclaimed blocks are looked up when written)
    bool dem[kRcItems], want[kRcItems];
    unsigned ip[kRcItems];
#pragma unroll
    for (int j = 0; j < kRcItems; ++j) want[j] = f[j] && a.tier < 2 && v.h[j] != 0ull;
    demotions(a, v.h, want, dem, ip, s_look, s_rank);  // (empty slots: none)
    if (a.tier >= 2) {
#pragma unroll
      for (int j = 0; j < kRcItems; ++j) ip[j] = (v.h[j] != 0ull && a.index) ? kFindPos : kNoPos;
    }
    int rk[kRcItems];
    const int cnt = block_slot_rank(f, rk, s_rank);
    // the chunk is reserved at once; its start is used only after the sums
    const int g = tile % kListGroups;
    const int start0 = (t == 0 && cnt)
                           ? (int)(g * region_cap(a.n)) +
                                 (int)atomicAdd(a.w.count + g * kCountStride, (unsigned)cnt)
                           : 0;
    int c2[2] = {0, 0};
#pragma unroll
    for (int j = 0; j < kRcItems; ++j) {
      c2[0] += sure[j];
      c2[1] += sure[j] && dem[j];
    }
    block_sum<2, int>(c2, s_red);
    if (t == 0) {
      s_start = start0;
      a.w.rec[tile] = make_int4(start0, c2[0], cnt - c2[0], c2[1]);
      // the select kernel's counters (added to with atomics)
      unsigned long long *o64 = reinterpret_cast<unsigned long long *>(a.w.off + tile);
      store_agent(o64, 0ull);
      store_agent(o64 + 1, 0ull);
    }
    __syncthreads();
    const int start = s_start, base = slot_base(tile);
#pragma unroll
    for (int j = 0; j < kRcItems; ++j) {
      const int i = start + rk[j];
      if (!f[j] || (long long)(unsigned)i >= kListGroups * region_cap(a.n)) continue;
      a.w.key[i] = k[j];
      a.w.ent[i] = (unsigned)item_slot(base, j) | (sure[j] ? kEntSure : 0u) |
                   (dem[j] ? kEntDem : 0u);
      a.w.pos[i] = ip[j];
      a.w.hash[i] = v.h[j];
      if (d2 > 0 && !sure[j]) {
        const unsigned b = (unsigned)(k[j] >> s2) & m2;
        if (sub_direct) atomicAdd(a.w.sub + b, 1u);
        else atomicAdd(&s_sub[b], 1u);
      }
    }
  });
  if (d2 > 0 && !sub_direct) {
    __syncthreads();
    for (int b = t; b < (1 << d2); b += kBlock) {
      const unsigned v = s_sub[b];
      if (v) atomicAdd(a.w.sub + b, v);
    }
  }
}

__global__ __launch_bounds__(kBlock) void rc_compact_kernel(RcArgs a) {
  compact_table(a, whole_grid());
}

// ------------------------------------------------------------ selection

// The bin of a kRcBins-bin histogram (kSelBins consecutive bins per thread
// of a kBlock-thread workgroup) holding the 0-based rank r: the bin, the
// rank inside it and its count; bin -1 when no bin holds it.
constexpr int kSelBins = kRcBins / kBlock;
struct Hit {
  int bin, rank, count;
};
__device__ __forceinline__ Hit find_rank(const unsigned (&v)[kSelBins], int r, int *s_scan,
                                         int *s_found) {
  int sum = 0;
#pragma unroll
  for (int j = 0; j < kSelBins; ++j) sum += (int)v[j];
  if (threadIdx.x == 0) s_found[0] = -1;
  int ex[1] = {sum}, tot[1];
  block_exclusive_scan<1, int>(ex, tot, s_scan);
  if (r >= ex[0] && r < ex[0] + sum) {
    int q = r - ex[0];
#pragma unroll
    for (int j = 0; j < kSelBins; ++j) {
      if (q >= 0 && q < (int)v[j]) {
        s_found[0] = (int)threadIdx.x * kSelBins + j;
        s_found[1] = q;
        s_found[2] = (int)v[j];
        q = -1;
      } else if (q >= 0) {
        q -= (int)v[j];
      }
    }
  }
  __syncthreads();
  const Hit h = {s_found[0], s_found[1], s_found[2]};
  __syncthreads();
  return h;
}

// The list regions walked as one flat index: entry f of region g sits at
// g * cap + (f - pre[g]), pre the regions' exclusive prefix.
struct ListMap {
  int pre[kListGroups + 1];
  int cap;
  __device__ __forceinline__ int at(int f) const {
    int g = 0, start = 0;  // constant indices only: pre stays in registers
#pragma unroll
    for (int q = 1; q < kListGroups; ++q) {
      const bool ge = f >= pre[q];
      g = ge ? q : g;
      start = ge ? pre[q] : start;
    }
    return g * cap + (f - start);
  }
  __device__ __forceinline__ int size() const { return pre[kListGroups]; }
};

// Calls f(e, k) for the entries a thread owns among n (flat index fi =
// first + j * stride): e = ent[at(fi)], k = key[at(fi)], kSelBatch entries
// per round, all loaded before any is used, so a pass costs a few memory
// round trips rather than one per entry.  Certainly reclaimed entries are
// skipped.
constexpr int kSelBatch = 8;
template <bool kAgent = false, typename At, typename F>
__device__ __forceinline__ void for_entries(const unsigned *__restrict__ ent,
                                            const unsigned long long *__restrict__ key, int n,
                                            int first, int stride, At &&at, F &&f) {
  for (int r0 = first; r0 < n; r0 += stride * kSelBatch) {
    unsigned e[kSelBatch];
    unsigned long long k[kSelBatch];
#pragma unroll
    for (int j = 0; j < kSelBatch; ++j) {
      const int fi = r0 + j * stride;
      const int i = fi < n ? at(fi) : 0;
      // (kAgent: written by other workgroups of this launch)
      e[j] = fi < n ? (kAgent ? load_agent(ent + i) : ent[i]) : kEntSure;  // past the end: skipped
      k[j] = fi < n ? (kAgent ? load_agent(key + i) : key[i]) : 0ull;
    }
#pragma unroll
    for (int j = 0; j < kSelBatch; ++j)
      if (!(e[j] & kEntSure)) f(e[j], k[j]);
  }
}

// A tile's four counters in off[], read as two agent-scope words (other
// workgroups add to them with atomics).
__device__ __forceinline__ int4 load_counts(const int4 *off, int tile) {
  const unsigned long long *o64 = reinterpret_cast<const unsigned long long *>(off + tile);
  const unsigned long long u = load_agent(o64), w = load_agent(o64 + 1);
  return make_int4((int)(unsigned)u, (int)(unsigned)(u >> 32), (int)(unsigned)w,
                   (int)(unsigned)(w >> 32));
}

// Adds one candidate to its tile's counters in off[]: (below T, equal to T,
// demoted below, demoted equal).
__device__ __forceinline__ void count_in_tile(int4 *off, unsigned e, bool below) {
  int *c = &off[(e & kEntSlot) / kRcTile].x;
  atomicAdd(c + (below ? 0 : 1), 1);
  if (e & kEntDem) atomicAdd(c + (below ? 2 : 3), 1);
}

// The threshold key T, the last taken slot with key T and every tile's
// output offsets.  Every workgroup: the next digit d2 of T from the
// compaction's histogram, then a share of the list: candidates whose digit
// is below d2 are below T and go straight to their tile's counters, those
// on d2 are staged (when every bit of T is already known, each candidate is
// counted against T instead).  The last workgroup: T's remaining digits
// over the staged candidates, their counts, the tile holding the take-th
// key T in tile (slot) order, that key's slot, and
//   off[t] = (reclaimed before t, demoted before t, reclaimed in t, demoted in t).
// A threshold prefix shared by more than kStageCap candidates is resolved
// from the whole list instead of the stage.
__global__ __launch_bounds__(kBlock) void rc_select_kernel(RcArgs a) {
  __shared__ unsigned s_hist[kRcBins];
  __shared__ int s_scan[kWaves * 2];
  __shared__ int s_found[3];
  __shared__ int s_pre[kListGroups + 1];
  __shared__ bool s_last;
  __shared__ unsigned long long s_skey[kStageLds];
  __shared__ unsigned s_sent[kStageLds];
  __shared__ int4 s_q[kTilesLds];
  __shared__ int s_scan_w[kWaves * 2 * (kTilesLds / kBlock)];  // a scan of every chunk at once
  RcPlan *P = a.w.plan;
  const int t = threadIdx.x;
  // the compaction's histogram of the next digit (bins past 2^d2 were never
  // added to) and the regions' entry counts, requested with the plan
  unsigned v2[kSelBins];
#pragma unroll
  for (int j = 0; j < kSelBins; ++j) v2[j] = load_agent(a.w.sub + t * kSelBins + j);
  const int c_reg = t < kListGroups ? (int)load_agent(a.w.count + t * kCountStride) : 0;
  const int ok = P->ok, mode = P->mode, shift0 = P->shift, bucket = P->bucket, brank = P->brank,
            prank = P->rank;
  const int st_now = load_agent(a.status);
  if (blockIdx.x == 0) {  // the top-digit histogram is free again (the compaction read it)
    for (int i = t; i < kHistCopies * (1 << kDigit0); i += kBlock) store_agent(a.w.hist + i, 0u);
  }
  if (!ok || st_now != CASCADE_OK) {
    // The call failed, or (in a chain call, whose compaction shares a launch
    // with the tier above's writes) the tier above failed while this call's
    // compaction ran: nothing is selected, the write kernel writes nothing,
    // and what the compaction may have counted is cleared.
    if (blockIdx.x == 0) {
      for (int b = t; b < kRcBins; b += kBlock) store_agent(a.w.sub + b, 0u);
      if (t < kListGroups) store_agent(a.w.count + t * kCountStride, 0u);
      if (t == 0 && ok) P->ok = 0;
    }
    return;
  }
  const int tiles = max(1, tiles_of(a.n));
  if (t < 64) {  // the regions' entry counts and their prefix
    const int c = c_reg;
    const int inc = (int)wave_inclusive_sum((unsigned)c);
    if (t < kListGroups) s_pre[t + 1] = inc;
    if (t == 0) s_pre[0] = 0;
  }
  __syncthreads();
  ListMap lst;
#pragma unroll
  for (int g = 0; g <= kListGroups; ++g) lst.pre[g] = s_pre[g];
  lst.cap = (int)region_cap(a.n);
  auto at_list = [lst](int fi) { return lst.at(fi); };
  const unsigned long long *key = a.w.key;
  const unsigned *ent = a.w.ent;

  const bool cached = mode == kModeCached;
  const bool has_sub = cached && shift0 > 0;
  unsigned long long T = cached ? (unsigned long long)bucket << shift0 : 0ull;
  int rank = cached ? brank : prank;  // kModeEmpty: total - 1 among the empty slots
  int shift = has_sub ? shift0 : 0, matching = 0, d2 = 0, s2 = 0;
  unsigned b2 = 0;
  bool fail = false;
  if (has_sub) {
    d2 = min(shift0, kDigitN);
    s2 = shift0 - d2;
    const Hit h = find_rank(v2, rank, s_scan, s_found);
    if (h.bin < 0) {
      fail = true;
    } else {
      b2 = (unsigned)h.bin;
      T |= (unsigned long long)b2 << s2;
      rank = h.rank;
      matching = h.count;
      shift = s2;
    }
  }
  const bool staging = has_sub && matching <= kStageCap;
  if (cached && !fail) {
    const unsigned m2 = (1u << d2) - 1u;
    for_entries(ent, key, lst.size(), (int)(blockIdx.x * kBlock) + t, (int)(gridDim.x * kBlock),
                at_list, [&](unsigned e, unsigned long long k) {
      if (!has_sub) {  // every bit of T known
        if (k <= T) count_in_tile(a.w.off, e, k < T);
        return;
      }
      const unsigned dg = (unsigned)(k >> s2) & m2;
      if (dg < b2) {
        count_in_tile(a.w.off, e, true);
      } else if (dg == b2 && staging) {
        const unsigned p = atomicAdd(a.w.stage_n, 1u);
        if (p < (unsigned)kStageCap) {  // read by the last workgroup: agent scope
          store_agent(a.w.stage_key + p, k);
          store_agent(a.w.stage_ent + p, e);
        }
      }
    });
  }
  wait_stores();
  __syncthreads();
  if (t == 0) s_last = last_workgroup(a.w.tickets);
  __syncthreads();
  if (!s_last) return;
  acquire_agent();

  // ---- the last workgroup
  if (has_sub)
    for (int b = t; b < kRcBins; b += kBlock) store_agent(a.w.sub + b, 0u);  // free again
  const int n_staged = (int)load_agent(a.w.stage_n);
  if (staging && n_staged != matching) fail = true;
  // the candidates on T's first digits: the stage (in LDS when it fits),
  // or the whole list filtered by those digits
  const unsigned long long *skey = a.w.stage_key;
  const unsigned *sent = a.w.stage_ent;
  const bool in_lds = staging && !fail && n_staged <= kStageLds;
  if (in_lds) {
    static_assert(kStageLds % kBlock == 0, "whole rounds");
#pragma unroll
    for (int j = 0; j < kStageLds / kBlock; ++j) {  // all loads in flight at once
      const int i = j * kBlock + t;
      if (i < n_staged) {
        s_skey[i] = load_agent(skey + i);
        s_sent[i] = load_agent(sent + i);
      }
    }
    __syncthreads();
  }
  auto at_stage = [](int fi) { return fi; };
  auto for_matching = [&](auto &&f) {
    if (in_lds) {
      for (int i = t; i < n_staged; i += kBlock) f(s_sent[i], s_skey[i]);
    } else if (staging) {
      for_entries<true>(sent, skey, n_staged, t, kBlock, at_stage, f);
    } else {
      const unsigned long long hi = shr64(T, s2);
      for_entries(ent, key, lst.size(), t, kBlock, at_list,
                  [&](unsigned e, unsigned long long k) {
                    if (shr64(k, s2) == hi) f(e, k);
                  });
    }
  };
  // 1. T's remaining digits: few staged candidates are ranked directly
  //    (keys below and keys at most each one), more take a digit per pass
  if (!fail && has_sub && shift > 0 && in_lds && n_staged <= kTieLds) {
    if (t == 0) s_found[0] = -1;
    __syncthreads();
    for (int i = t; i < n_staged; i += kBlock) {
      const unsigned long long ki = s_skey[i];
      int lt = 0, le = 0;
      for (int j = 0; j < n_staged; ++j) {
        const unsigned long long kj = s_skey[j];
        lt += kj < ki ? 1 : 0;
        le += kj <= ki ? 1 : 0;
      }
      if (rank >= lt && rank < le) {  // every writer holds the same key and rank
        s_found[0] = i;
        s_found[1] = rank - lt;
      }
    }
    __syncthreads();
    if (s_found[0] < 0) {
      fail = true;
    } else {
      T = s_skey[s_found[0]];
      rank = s_found[1];
      shift = 0;
    }
    __syncthreads();
  }
  while (!fail && has_sub && shift > 0) {
    const int d = min(shift, kDigitN), s = shift - d;
    const unsigned m = (1u << d) - 1u;
    for (int b = t; b < kRcBins; b += kBlock) s_hist[b] = 0u;
    __syncthreads();
    const unsigned long long hi = shr64(T, shift);
    for_matching([&](unsigned, unsigned long long k) {
      if (shr64(k, shift) == hi) atomicAdd(&s_hist[(unsigned)(k >> s) & m], 1u);
    });
    __syncthreads();
    unsigned v[kSelBins];
#pragma unroll
    for (int j = 0; j < kSelBins; ++j) v[j] = s_hist[t * kSelBins + j];
    const Hit h = find_rank(v, rank, s_scan, s_found);
    if (h.bin < 0) {
      fail = true;
      break;
    }
    T |= (unsigned long long)h.bin << s;
    rank = h.rank;
    shift = s;
  }
  // 2. the candidates on T's first digits, counted against T
  if (!fail && has_sub) {
    for_matching([&](unsigned e, unsigned long long k) {
      if (k <= T) count_in_tile(a.w.off, e, k < T);
    });
    wait_stores();
  }
  __syncthreads();
  acquire_agent();  // the counters are read back from memory

  // 3. per tile: the certain ones join the counts; the tile holding the
  //    take-th key T in slot order
  const int take = rank + 1;
  int carry = 0;
  if (t == 0) s_found[0] = -1;
  // one chunk of kBlock tiles, in tile order (called by every thread)
  auto tile_chunk = [&](int tile, int4 q, const int4 &r) {
    if (tile < tiles) {
      q.x += r.y;  // certainly reclaimed: below T
      q.z += r.w;
      if (!cached) q.y += r.z;  // empty slots only: every candidate is key 0 = T, none demoted
      if (tiles <= kTilesLds) s_q[tile] = q;
      else a.w.off[tile] = q;
    } else {
      q = make_int4(0, 0, 0, 0);
    }
    int ex[1] = {q.y}, tot[1];
    block_exclusive_scan<1, int>(ex, tot, s_scan);
    if (take > carry + ex[0] && take <= carry + ex[0] + q.y) {
      s_found[0] = tile;
      s_found[1] = take - carry - ex[0];  // keys T taken in that tile
    }
    carry += tot[0];
  };
  if (tiles <= kTilesLds) {
    // every chunk's records requested at once
    constexpr int kChunks = kTilesLds / kBlock;
    int4 qa[kChunks], ra[kChunks];
#pragma unroll
    for (int c = 0; c < kChunks; ++c) {
      const int tile = c * kBlock + t;
      qa[c] = tile < tiles ? load_counts(a.w.off, tile) : make_int4(0, 0, 0, 0);
      ra[c] = tile < tiles ? a.w.rec[tile] : make_int4(0, 0, 0, 0);
    }
    if (tiles <= kBlock) {
      tile_chunk(t, qa[0], ra[0]);
    } else {
      // every chunk's keys T counted in one block scan (chunk c holds tiles
      // c * kBlock + thread), then chunk by chunk the tile holding the take-th
      int ys[kChunks], tot[kChunks];
#pragma unroll
      for (int c = 0; c < kChunks; ++c) {
        const int tile = c * kBlock + t;
        int4 q = make_int4(0, 0, 0, 0);
        if (tile < tiles) {
          q = qa[c];
          q.x += ra[c].y;  // certainly reclaimed: below T
          q.z += ra[c].w;
          if (!cached) q.y += ra[c].z;  // empty slots only: every candidate is key 0 = T
          s_q[tile] = q;
        }
        qa[c] = q;
        ys[c] = q.y;
      }
      block_exclusive_scan<kChunks, int>(ys, tot, s_scan_w);
      int base = 0;
#pragma unroll
      for (int c = 0; c < kChunks; ++c) {
        const int pre = base + ys[c], y = qa[c].y;
        if (take > pre && take <= pre + y) {
          s_found[0] = c * kBlock + t;
          s_found[1] = take - pre;  // keys T taken in that tile
        }
        base += tot[c];
      }
    }
  } else {
    for (int c0 = 0; c0 < tiles; c0 += kBlock) {
      const int tile = c0 + t;
      const int4 r = tile < tiles ? a.w.rec[tile] : make_int4(0, 0, 0, 0);
      tile_chunk(tile, tile < tiles ? load_counts(a.w.off, tile) : make_int4(0, 0, 0, 0), r);
    }
  }
  __syncthreads();
  const int cut = s_found[0], r_cut = take > 0 ? s_found[1] : 0;
  if (take > 0 && cut < 0) fail = true;

  // 4. inside the cut tile: the slot of its r_cut-th key T, and how many of
  //    its first r_cut keys T are demoted (wave 0, 64 entries per round)
  int tie_slot = -1, dem_cut = 0;
  __syncthreads();
  if (t == 0) s_found[2] = -1;
  __syncthreads();
  if (!fail && cut >= 0 && in_lds && n_staged <= kTieLds) {
    // every candidate equal to T is staged: rank the cut tile's by slot
    if (t == 0) s_found[1] = 0;
    __syncthreads();
    for (int i = t; i < n_staged; i += kBlock) {
      const int slot = (int)(s_sent[i] & kEntSlot);
      if (s_skey[i] != T || slot / kRcTile != cut) continue;
      int before = 0;
      for (int j = 0; j < n_staged; ++j) {
        const int sj = (int)(s_sent[j] & kEntSlot);
        before += (s_skey[j] == T && sj / kRcTile == cut && sj < slot) ? 1 : 0;
      }
      if (before < r_cut && (s_sent[i] & kEntDem)) atomicAdd(&s_found[1], 1);
      if (before == r_cut - 1) s_found[2] = slot;
    }
    __syncthreads();
    tie_slot = s_found[2];
    dem_cut = s_found[1];
    if (tie_slot < 0) fail = true;
  } else if (!fail && cut >= 0) {
    if (t < 64) {
      const int4 r = a.w.rec[cut];
      const int end = r.x + r.y + r.z;
      int seen = 0, dsum = 0;
      for (int i0 = r.x; i0 < end && seen < r_cut; i0 += 64) {
        const int i = i0 + t;
        unsigned e = 0u;
        bool eq = false;
        if (i < end) {
          e = ent[i];
          eq = !(e & kEntSure) && key[i] == T;
        }
        const uint64_t mk = __ballot(eq);
        const int before = seen + rank_in_mask(mk);
        const bool taken = eq && before < r_cut;
        dsum += (int)wave_sum((unsigned)(taken && (e & kEntDem) ? 1 : 0));
        if (taken && before == r_cut - 1) s_found[2] = (int)(e & kEntSlot);
        seen += __builtin_popcountll(mk);
      }
      if (t == 0) s_found[1] = dsum;
    }
    __syncthreads();
    tie_slot = s_found[2];
    dem_cut = s_found[1];
    if (tie_slot < 0) fail = true;
  }

  // 5. output offsets, in tile order
  int carry_s = 0, carry_d = 0;
  if (tiles > kBlock && tiles <= kTilesLds) {  // every chunk in one block scan
    constexpr int kChunks = kTilesLds / kBlock;
    int v[2 * kChunks], ex[2 * kChunks], tot[2 * kChunks];
#pragma unroll
    for (int c = 0; c < kChunks; ++c) {
      const int tile = c * kBlock + t;
      v[2 * c] = v[2 * c + 1] = 0;
      if (tile < tiles) {
        const int4 q = s_q[tile];
        v[2 * c] = q.x + (tile < cut ? q.y : (tile == cut ? r_cut : 0));
        v[2 * c + 1] = q.z + (tile < cut ? q.w : (tile == cut ? dem_cut : 0));
      }
      ex[2 * c] = v[2 * c];
      ex[2 * c + 1] = v[2 * c + 1];
    }
    block_exclusive_scan<2 * kChunks, int>(ex, tot, s_scan_w);
#pragma unroll
    for (int c = 0; c < kChunks; ++c) {
      const int tile = c * kBlock + t;
      if (tile < tiles)
        a.w.off[tile] = make_int4(carry_s + ex[2 * c], carry_d + ex[2 * c + 1], v[2 * c],
                                  v[2 * c + 1]);
      carry_s += tot[2 * c];
      carry_d += tot[2 * c + 1];
    }
  }
  for (int c0 = 0; (tiles <= kBlock || tiles > kTilesLds) && c0 < tiles; c0 += kBlock) {
    const int tile = c0 + t;
    int v[2] = {0, 0};
    if (tile < tiles) {
      const int4 q = tiles <= kTilesLds ? s_q[tile] : load_counts(a.w.off, tile);
      v[0] = q.x + (tile < cut ? q.y : (tile == cut ? r_cut : 0));
      v[1] = q.z + (tile < cut ? q.w : (tile == cut ? dem_cut : 0));
    }
    int ex[2] = {v[0], v[1]}, tot[2];
    block_exclusive_scan<2, int>(ex, tot, s_scan);
    if (tile < tiles) a.w.off[tile] = make_int4(carry_s + ex[0], carry_d + ex[1], v[0], v[1]);
    carry_s += tot[0];
    carry_d += tot[1];
  }
  if (t == 0) {
    if (fail || carry_s != P->total || carry_d > a.max_out) {  // must reclaim exactly total
      store_agent(a.status, (int)CASCADE_EINTERNAL);
      P->ok = 0;
    } else {
      P->thresh = T;
      P->tie_slot = tie_slot;
      if (a.n_out_dev) store_agent(a.n_out_dev, carry_d);
    }
    for (int g = 0; g < kListGroups; ++g) store_agent(a.w.count + g * kCountStride, 0u);
    store_agent(a.w.stage_n, 0u);  // both free again
  }
}

// ---------------------------------------------------------------- writes

// A workgroup per tile with reclaimed slots.  The tile's chunk of the list
// is in slot order, so a reclaimed entry's position p in the reclaimed list
// is the tile's offset plus the reclaimed entries before it in the chunk
// (the demoted ones likewise).  For position p: freed[p] or
// placed[p - need], the demoted block into outgoing, the index bits (the old
// block leaves this tier, a demoted one joins the next) and the slot's new
// contents.  The old block comes from the list and its stamp from its key,
// so the table is not read again.
__device__ __forceinline__ void write_tile(const RcArgs &a, int tile) {
  __shared__ int s_scan[kWaves * 2];
  const RcPlan *P = a.w.plan;
  const int t = threadIdx.x;
  const int4 o = a.w.off[tile], r = a.w.rec[tile];  // requested with the plan
  const int ok = P->ok, tie_slot = P->tie_slot, total = P->total, need = a.need;
  const unsigned long long T = P->thresh, lu_min = P->lu_min;
  if (!ok || o.z == 0) return;  // nothing reclaimed here (so nothing demoted either)
  const int len = min(r.y + r.z, kRcTile);  // a chunk holds at most its tile's slots
  // a row of kBlock entries at a time (one row in the usual case)
  int n_sel = 0, n_dem = 0;  // before this row
  for (int c0 = 0; c0 < len; c0 += kBlock) {  // uniform
    const int c = c0 + t, i = r.x + c;
    const bool in = c < len;
    const unsigned e = in ? a.w.ent[i] : 0u;
    const unsigned long long k = in ? a.w.key[i] : 0ull, h = in ? a.w.hash[i] : 0ull;
    const unsigned ipos = in ? a.w.pos[i] : kNoPos;
    const int slot = (int)(e & kEntSlot);
    const bool sel = in && (unsigned)slot < (unsigned)a.n &&
                     ((e & kEntSure) || k < T || (k == T && slot <= tie_slot));
    const bool dem = sel && (e & kEntDem);
    // tier 2 looks its reclaimed blocks up here
    const unsigned long long hq[1] = {h};
    const bool lq[1] = {sel && ipos == kFindPos && a.index};
    int fpos[1];
    unsigned ftiers[1];
    index_find_n(a.index, a.index_mask, hq, lq, fpos, ftiers);
    int ex[2] = {(int)sel, (int)dem}, tot[2];
    block_exclusive_scan<2, int>(ex, tot, s_scan);
    const int p = o.x + n_sel + ex[0], q = o.y + n_dem + ex[1];
    n_sel += tot[0];
    n_dem += tot[1];
    // positions past the tile's counts are never written (the counts disagree)
    if (!sel || p - o.x >= o.z || p >= total || (dem && (q - o.y >= o.w || q >= a.max_out)))
      continue;
    const bool place = p >= need;
    unsigned long long in_h = 0ull;
    long long in_lu = 0ll;
    if (place) {
      in_h = a.incoming[p - need].hash;
      in_lu = a.incoming[p - need].last_use_ns;
    }
    IndexSlot *ix = nullptr;
    if (ipos == kFindPos) ix = fpos[0] >= 0 ? a.index + fpos[0] : nullptr;
    else if (ipos != kNoPos && a.index) ix = a.index + ipos;  // found by the compaction
    if (dem) {  // a cached block: key = 1 + last use - lu_min
      cascade_demotion_t d;
      d.hash = h;
      d.last_use_ns = (long long)(k - 1ull + lu_min);
      d.src_slot = slot;
      d.pad = 0;
      a.outgoing[q] = d;
      if (ix) atomicOr(&ix->tiers, 1u << (a.tier + 1));
    }
    if (ix) atomicAnd(&ix->tiers, ~(1u << a.tier));
    if (!place) {
      a.freed[p] = slot;
      a.hash[slot] = 0ull;
      a.lu[slot] = 0ll;
    } else {
      a.placed[p - need] = slot;
      a.hash[slot] = in_h;
      a.lu[slot] = in_lu;
    }
  }
  if (t == 0 && (n_sel != o.z || n_dem != o.w))
    store_agent(a.status, (int)CASCADE_EINTERNAL);  // the counts disagree
}

__global__ __launch_bounds__(kBlock) void rc_write_kernel(RcArgs a) {
  write_tile(a, (int)blockIdx.x);
}

// In a chain call, one tier's writes and the next tier's compaction, which
// do not depend on each other, share a launch: workgroups [0, n_compact)
// compact tier c (first, so the longer work starts first), the rest write
// tier w's tiles.  The compaction needs only
// the incoming count, which tier w's select kernel has stored, and the
// index's bits of the tiers below c, which tier w's writes do not touch
// (they change the bits of tiers w and w + 1 = c); it does not read the
// incoming blocks, which tier w's writes produce.  A failure tier w's writes
// report while the compaction runs is caught by tier c's select kernel.
__global__ __launch_bounds__(kBlock) void rc_write_compact_kernel(RcArgs w, RcArgs c,
                                                                  int n_compact) {
  const int b = (int)blockIdx.x;
  if (b < n_compact) compact_table(c, Part{b, n_compact});
  else write_tile(w, b - n_compact);
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

namespace cascade {
namespace {

// One tier's host-side checks and kernel arguments (CASCADE_OK or EINVAL).
int tier_args(int32_t tier, const cascade_tier_table_t *table, int32_t need,
              const cascade_demotion_t *incoming, const int32_t *n_incoming_dev,
              int32_t max_incoming, cascade_demotion_t *outgoing, int32_t *n_outgoing_dev,
              int32_t max_outgoing, int32_t *freed, int32_t *placed, void *index,
              int32_t index_capacity, void *head, void *body, int32_t *status_dev, RcArgs &a) {
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
  a.w = carve(head, body, n);
  return CASCADE_OK;
}

int tiles_or_one(const RcArgs &a) { return std::max(1, tiles_of(a.n)); }

// The compaction, selection and writes of one tier's call.
void launch_tail(const RcArgs &a, hipStream_t s) {
  const int tiles = tiles_or_one(a);
  hipLaunchKernelGGL(rc_compact_kernel, dim3(std::min(tiles, kRcGridCompact)), dim3(kBlock), 0, s,
                     a);
  hipLaunchKernelGGL(rc_select_kernel, dim3(kSelGrid), dim3(kBlock), 0, s, a);
  hipLaunchKernelGGL(rc_write_kernel, dim3(tiles), dim3(kBlock), 0, s, a);
}

// The count and histogram passes over m.n tables, one launch each.
void launch_head(RcTables &m, hipStream_t s) {
  int gc = 0, gh = 0;
  int first_h[3] = {0, 0, 0};
  for (int k = 0; k < m.n; ++k) {
    m.first[k] = gc;
    first_h[k] = gh;
    gc += std::min(tiles_or_one(m.t[k]), kRcGridCount);
    gh += std::min(tiles_or_one(m.t[k]), kRcGridHist);
  }
  hipLaunchKernelGGL(rc_count_kernel, dim3(gc), dim3(kBlock), 0, s, m);
  for (int k = 0; k < m.n; ++k) m.first[k] = first_h[k];
  hipLaunchKernelGGL(rc_hist_kernel, dim3(gh), dim3(kBlock), 0, s, m);
}

}  // namespace
}  // namespace cascade

extern "C" int cascade_tier_reclaim(int32_t tier, const cascade_tier_table_t *table, int32_t need,
                                    const cascade_demotion_t *incoming,
                                    const int32_t *n_incoming_dev, int32_t max_incoming,
                                    cascade_demotion_t *outgoing, int32_t *n_outgoing_dev,
                                    int32_t max_outgoing, int32_t *freed, int32_t *placed,
                                    void *index, int32_t index_capacity, void *workspace,
                                    size_t workspace_bytes, int32_t *status_dev, void *stream) {
  if (!table || table->n_slots < 0 || table->n_slots > (1 << 30) || !workspace ||
      ((uintptr_t)workspace & 255) || workspace_bytes < workspace_bytes_for(table->n_slots))
    return CASCADE_EINVAL;
  RcTables m{};
  char *ws = static_cast<char *>(workspace);
  const int rc = tier_args(tier, table, need, incoming, n_incoming_dev, max_incoming, outgoing,
                           n_outgoing_dev, max_outgoing, freed, placed, index, index_capacity,
                           ws, ws + head_bytes(), status_dev, m.t[0]);
  if (rc != CASCADE_OK) return rc;
  m.n = 1;
  m.check_in = 1;
  hipStream_t s = static_cast<hipStream_t>(stream);
  launch_head(m, s);
  launch_tail(m.t[0], s);
  return hipGetLastError() == hipSuccess ? CASCADE_OK : CASCADE_EHIP;
}

extern "C" size_t cascade_tier_chain_workspace_bytes(const int32_t *n_slots) {
  if (!n_slots) return 0;
  size_t total = 0;
  for (int t = 0; t < 3; ++t) {
    if (n_slots[t] < 0 || n_slots[t] > (1 << 30)) return 0;
    total += workspace_bytes_for(n_slots[t]);  // each a multiple of 256 bytes
  }
  return total;  // three heads, then three bodies
}

extern "C" int cascade_tier_reclaim_chain(const cascade_tier_chain_t *c, void *index,
                                          int32_t index_capacity, void *workspace,
                                          size_t workspace_bytes, int32_t *status_dev,
                                          void *stream) {
  if (!c || !workspace || ((uintptr_t)workspace & 255)) return CASCADE_EINVAL;
  const int32_t n[3] = {c->table[0].n_slots, c->table[1].n_slots, c->table[2].n_slots};
  const size_t need_bytes = cascade_tier_chain_workspace_bytes(n);
  if (need_bytes == 0 || workspace_bytes < need_bytes) return CASCADE_EINVAL;
  RcTables m{};
  char *ws = static_cast<char *>(workspace);
  char *body = ws + 3 * head_bytes();  // the heads at fixed offsets, whatever the tables
  for (int t = 0; t < 3; ++t) {
    const int rc = tier_args(
        t, &c->table[t], c->need[t], t > 0 ? c->outgoing[t - 1] : nullptr,
        t > 0 ? c->n_outgoing_dev[t - 1] : nullptr, t > 0 ? c->max_outgoing[t - 1] : 0,
        t < 2 ? c->outgoing[t] : nullptr, t < 2 ? c->n_outgoing_dev[t] : nullptr,
        t < 2 ? c->max_outgoing[t] : 0, c->freed[t], c->placed[t], index, index_capacity,
        ws + t * head_bytes(), body, status_dev, m.t[t]);
    if (rc != CASCADE_OK) return rc;
    body += body_bytes(n[t]);
  }
  m.n = 3;
  m.check_in = 0;  // each tier's incoming blocks are the chain's own demotions
  hipStream_t s = static_cast<hipStream_t>(stream);
  launch_head(m, s);
  // compact 0, select 0, [write 0 | compact 1], select 1, [write 1 | compact 2],
  // select 2, write 2
  hipLaunchKernelGGL(rc_compact_kernel, dim3(std::min(tiles_or_one(m.t[0]), kRcGridCompact)),
                     dim3(kBlock), 0, s, m.t[0]);
  for (int t = 0; t < 3; ++t) {
    hipLaunchKernelGGL(rc_select_kernel, dim3(kSelGrid), dim3(kBlock), 0, s, m.t[t]);
    const int n_write = tiles_or_one(m.t[t]);
    if (t < 2) {
      const int n_compact = std::min(tiles_or_one(m.t[t + 1]), kRcGridCompact);
      hipLaunchKernelGGL(rc_write_compact_kernel, dim3(n_write + n_compact), dim3(kBlock), 0, s,
                         m.t[t], m.t[t + 1], n_compact);
    } else {
      hipLaunchKernelGGL(rc_write_kernel, dim3(n_write), dim3(kBlock), 0, s, m.t[t]);
    }
  }
  return hipGetLastError() == hipSuccess ? CASCADE_OK : CASCADE_EHIP;
}
