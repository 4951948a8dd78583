// cascade_prefix.hip -- prefix-hit lookup on gfx950 (Section 4.4, prefix hit
// detection).
//
// On top of per-block prefix hashing, an index records for every cached KV
// block the tiers holding it, of which the lookup reads the deepest (per-tier
// reclamation removes a tier's copy: cascade_reclaim.hip).  A request's
// prefix-hit profile is the longest run of its leading blocks present in the
// index (capped so that at least one prompt token is computed) and the
// deepest tier over that run: the n_prefix / prefix_tier inputs of the
// scheduling step.
//
// The index is an open-addressing hash table of 16-byte slots (key, set of
// tiers holding the block) in device memory (index_table.h); key 0 marks an
// empty slot.  Insert claims a slot with a 64-bit CAS and adds the tier to the
// set with atomicOr; the block's deepest tier is the highest tier in its set.
// The probe gives each request one wave: 64 leading blocks are looked up at
// once, a ballot finds the first miss (a block absent, or whose set is empty),
// and the wave stops there, so blocks past a miss cost nothing.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "cascade.h"
#include "device_util.h"
#include "index_table.h"

namespace cascade {
namespace {

__global__ __launch_bounds__(kBlock) void index_clear_kernel(uint4 *slots, long long n_vec) {
  for (long long j = (long long)blockIdx.x * kBlock + threadIdx.x; j < n_vec;
       j += (long long)gridDim.x * kBlock)
    slots[j] = make_uint4(0, 0, 0, 0);
}

__global__ __launch_bounds__(kBlock) void index_insert_kernel(IndexSlot *slots, unsigned mask,
                                                              const unsigned long long *hashes,
                                                              const uint8_t *tiers, int n,
                                                              int *status) {
  const int i = blockIdx.x * kBlock + threadIdx.x;
  if (i >= n) return;
  const unsigned long long h = hashes[i];
  const unsigned t = tiers[i];
  if (h == 0 || t > CASCADE_KV_NVME) {
    if (status) store_agent(status, (int)CASCADE_EINVAL);
    return;
  }
  unsigned s = (unsigned)fmix64(h) & mask;
  for (unsigned p = 0; p <= mask; ++p, s = (s + 1) & mask) {
    const unsigned long long cur = atomicCAS(&slots[s].key, 0ull, h);
    if (cur == 0ull || cur == h) {
      atomicOr(&slots[s].tiers, 1u << t);
      return;
    }
  }
  if (status) store_agent(status, (int)CASCADE_ENOSPC);  // every slot holds another key
}

__global__ __launch_bounds__(kBlock) void probe_kernel(const IndexSlot *__restrict__ slots,
                                                       unsigned mask, int n,
                                                       const int *__restrict__ offsets,
                                                       const unsigned long long *__restrict__ hashes,
                                                       const int *__restrict__ n_in, int bt,
                                                       int *__restrict__ n_prefix_out,
                                                       uint8_t *__restrict__ tier_out,
                                                       int *status) {
  const int i = blockIdx.x * kWaves + wave_id();
  if (i >= n) return;  // uniform over the wave
  const int lane = lane_id();
  // every read stays in [0, offsets[n]), the caller's hash array, even when
  // another request's offsets are out of order
  const int b0 = offsets[i], b1 = offsets[i + 1], total = offsets[n], nin = n_in[i];
  bool bad = b0 < 0 || b1 < b0 || b1 > total || nin < 1 || (i == 0 && b0 != 0);
  const int have = bad ? 0 : b1 - b0;
  const int cap = bad ? 0 : (nin - 1) / bt;
  const int lim = have < cap ? have : cap;
  int matched = 0;
  unsigned deepest = 0;
  for (int base = 0; base < lim; base += 64) {
    const int j = base + lane;
    const bool active = j < lim;
    bool hit = false;
    unsigned t = 0;
    if (active) {
      const unsigned long long h = hashes[b0 + j];
      if (h == 0) {
        bad = true;  // reserved for empty slots: never cached
      } else {
        unsigned s = (unsigned)fmix64(h) & mask;
        for (unsigned p = 0; p <= mask; ++p, s = (s + 1) & mask) {
          const IndexSlot e = slots[s];
          if (e.key == h) {
            hit = e.tiers != 0u;
            t = hit ? 31u - (unsigned)__builtin_clz(e.tiers) : 0u;
            break;
          }
          if (e.key == 0ull) break;
        }
      }
    }
    const uint64_t miss = __ballot(active && !hit);
    const int first = miss ? __builtin_ctzll(miss) : 64;
    const unsigned run_t = (active && lane < first) ? t : 0u;
    deepest = max(deepest, (unsigned)wave_max((unsigned long long)run_t));
    matched = miss ? base + first : min(base + 64, lim);
    if (miss) break;
  }
  if (__ballot(bad) && lane == 0 && status) store_agent(status, (int)CASCADE_EINVAL);
  if (lane == 0) {
    n_prefix_out[i] = matched * bt;
    tier_out[i] = (uint8_t)(matched > 0 ? deepest : (unsigned)CASCADE_KV_NONE);
  }
}

bool capacity_ok(int32_t capacity) {
  return capacity >= 64 && capacity <= (1 << 30) && (capacity & (capacity - 1)) == 0;
}

}  // namespace
}  // namespace cascade

using namespace cascade;

extern "C" size_t cascade_prefix_index_bytes(int32_t capacity) {
  return capacity_ok(capacity) ? (size_t)capacity * CASCADE_INDEX_SLOT_BYTES : 0;
}

extern "C" int cascade_prefix_index_clear(void *index, int32_t capacity, void *stream) {
  if (!index || !capacity_ok(capacity) || ((uintptr_t)index & 15)) return CASCADE_EINVAL;
  const long long n_vec = (long long)capacity;  // one 16-byte vector per slot
  const int grid = (int)std::min<long long>((n_vec + kBlock - 1) / kBlock, 4096);
  hipLaunchKernelGGL(index_clear_kernel, dim3(grid), dim3(kBlock), 0,
                     static_cast<hipStream_t>(stream), static_cast<uint4 *>(index), n_vec);
  return hipGetLastError() == hipSuccess ? CASCADE_OK : CASCADE_EHIP;
}

extern "C" int cascade_prefix_index_insert(void *index, int32_t capacity, const uint64_t *hashes,
                                           const uint8_t *tiers, int32_t n, int32_t *status_dev,
                                           void *stream) {
  if (!index || !capacity_ok(capacity) || ((uintptr_t)index & 15) || n < 0) return CASCADE_EINVAL;
  if (n == 0) return CASCADE_OK;
  if (!hashes || !tiers) return CASCADE_EINVAL;
  hipLaunchKernelGGL(index_insert_kernel, dim3((n + kBlock - 1) / kBlock), dim3(kBlock), 0,
                     static_cast<hipStream_t>(stream), static_cast<IndexSlot *>(index),
                     (unsigned)(capacity - 1), reinterpret_cast<const unsigned long long *>(hashes),
                     tiers, n, status_dev);
  return hipGetLastError() == hipSuccess ? CASCADE_OK : CASCADE_EHIP;
}

extern "C" int cascade_prefix_probe(const void *index, int32_t capacity, int32_t n,
                                    const int32_t *block_offsets, const uint64_t *block_hashes,
                                    const int32_t *n_in, int32_t block_tokens,
                                    int32_t *n_prefix_out, uint8_t *prefix_tier_out,
                                    int32_t *status_dev, void *stream) {
  if (!index || !capacity_ok(capacity) || ((uintptr_t)index & 15) || n < 0 || block_tokens < 1)
    return CASCADE_EINVAL;
  if (n == 0) return CASCADE_OK;
  if (!block_offsets || !block_hashes || !n_in || !n_prefix_out || !prefix_tier_out)
    return CASCADE_EINVAL;
  hipLaunchKernelGGL(probe_kernel, dim3((n + kWaves - 1) / kWaves), dim3(kBlock), 0,
                     static_cast<hipStream_t>(stream), static_cast<const IndexSlot *>(index),
                     (unsigned)(capacity - 1), n, block_offsets,
                     reinterpret_cast<const unsigned long long *>(block_hashes), n_in,
                     block_tokens, n_prefix_out, prefix_tier_out, status_dev);
  return hipGetLastError() == hipSuccess ? CASCADE_OK : CASCADE_EHIP;
}
