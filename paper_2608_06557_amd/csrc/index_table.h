// index_table.h -- the prefix index's open-addressing table, shared by the
// lookup (cascade_prefix.hip) and the per-tier reclamation
// (cascade_reclaim.hip).  Internal to the library.
//
// Slot = (key, tiers): key is a block's nonzero prefix hash (0 = empty slot),
// tiers the set of tiers holding the block (bit k = tier k).  The block's
// deepest tier is the highest set bit; an empty set means no tier holds it
// any more (the key stays, so probe sequences stay intact).  Linear probing
// from the murmur3 64-bit finalizer of the key.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "cascade.h"

namespace cascade {

struct alignas(16) IndexSlot {
  unsigned long long key;  // block hash, 0 = empty
  unsigned tiers;          // bit k set = tier k holds the block
  unsigned pad;
};
static_assert(sizeof(IndexSlot) == CASCADE_INDEX_SLOT_BYTES, "slot layout");

// murmur3's 64-bit finalizer (Appleby), the home slot of a key
__device__ __forceinline__ unsigned long long fmix64(unsigned long long k) {
  k ^= k >> 33;
  k *= 0xff51afd7ed558ccdull;
  k ^= k >> 33;
  k *= 0xc4ceb9fe1a85ec53ull;
  k ^= k >> 33;
  return k;
}

// N lookups at once, for the keys h[j] with want[j].  Every home slot is
// requested whole (key and tiers in one 16-byte load) before any is
// examined, so the N lookups share one memory round trip instead of taking
// one or two each in turn; a key that sits past its home slot continues
// probing alone.  Keys are never removed, so the first empty slot on a
// probe sequence ends it.  pos[j] is the key's slot (-1: absent or not
// wanted) and tiers[j] that slot's tier set.
template <int N>
__device__ __forceinline__ void index_find_n(const IndexSlot *slots, unsigned mask,
                                             const unsigned long long (&h)[N],
                                             const bool (&want)[N], int (&pos)[N],
                                             unsigned (&tiers)[N]) {
  static_assert(N <= 32, "one bit per lookup");
  unsigned s[N];
  uint4 v[N];
#pragma unroll
  for (int j = 0; j < N; ++j) {
    s[j] = (unsigned)fmix64(h[j]) & mask;
    v[j] = want[j] ? *reinterpret_cast<const uint4 *>(slots + s[j]) : make_uint4(0u, 0u, 0u, 0u);
  }
  unsigned pending = 0u;  // lookups whose home slot holds another key
#pragma unroll
  for (int j = 0; j < N; ++j) {
    const unsigned long long k = (unsigned long long)v[j].x | ((unsigned long long)v[j].y << 32);
    const bool hit = want[j] && k == h[j];
    pos[j] = hit ? (int)s[j] : -1;
    tiers[j] = hit ? v[j].z : 0u;
    if (want[j] && !hit && k != 0ull) pending |= 1u << j;
  }
  while (pending) {  // rare: one lookup at a time (items picked by constant index)
    const int j = __builtin_ctz(pending);
    pending &= pending - 1u;
    unsigned long long hj = 0ull;
    unsigned sj = 0u;
#pragma unroll
    for (int q = 0; q < N; ++q) {
      hj = q == j ? h[q] : hj;
      sj = q == j ? s[q] : sj;
    }
    int pj = -1;
    unsigned tj = 0u;
    for (unsigned p = 1; p <= mask; ++p) {  // mask + 1 slots in all
      sj = (sj + 1u) & mask;
      const uint4 w = *reinterpret_cast<const uint4 *>(slots + sj);
      const unsigned long long k = (unsigned long long)w.x | ((unsigned long long)w.y << 32);
      if (k == hj) {
        pj = (int)sj;
        tj = w.z;
        break;
      }
      if (k == 0ull) break;
    }
#pragma unroll
    for (int q = 0; q < N; ++q) {
      pos[q] = q == j ? pj : pos[q];
      tiers[q] = q == j ? tj : tiers[q];
    }
  }
}

}  // namespace cascade
