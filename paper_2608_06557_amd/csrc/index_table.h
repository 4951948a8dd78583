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

// The slot holding key h, or nullptr when h is not in the table.  Keys are
// never removed, so the first empty slot on the probe sequence ends it.
__device__ __forceinline__ IndexSlot *index_find(IndexSlot *slots, unsigned mask,
                                                 unsigned long long h) {
  unsigned s = (unsigned)fmix64(h) & mask;
  for (unsigned p = 0; p <= mask; ++p, s = (s + 1) & mask) {
    const unsigned long long k = slots[s].key;
    if (k == h) return &slots[s];
    if (k == 0ull) return nullptr;
  }
  return nullptr;
}

}  // namespace cascade
