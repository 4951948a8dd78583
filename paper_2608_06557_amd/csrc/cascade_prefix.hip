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
// The probe gives each request one wave, which looks up its leading blocks
// in windows that grow while every block hits; a ballot finds the first miss
// (a block absent, or whose set is empty), and the wave stops there.
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

// Lookups per lane in a probe window, at most: the window doubles from 64
// blocks (one per lane) up to 64 * kProbeMaxK.
constexpr int kProbeMaxK = 4;
// Whether a lookup also requests the slot after its home slot when both lie
// in one 128-byte line (8 slots): that read costs no extra line and decides
// most keys that sit one past their home.
constexpr bool kProbePair = true;

// Examines slot v for key h when go: returns true when that decides the
// lookup (key found, or an empty slot ends the probe sequence), and then sets
// hit (the key is there and its tier set is not empty) and t (its deepest
// tier).  Branch-free, so that the compiler keeps each slot a single load.
__device__ __forceinline__ bool examine_slot(const uint4 &v, unsigned long long h, bool go,
                                             bool &hit, unsigned &t) {
  const unsigned long long k = (unsigned long long)v.x | ((unsigned long long)v.y << 32);
  const bool match = go && k == h;
  hit = match ? v.z != 0u : hit;
  t = (match && v.z != 0u) ? 31u - (unsigned)__builtin_clz(v.z | 1u) : t;
  return go && (k == h || k == 0ull);
}

// One window of a request's lookup: 64 * K leading blocks from `base`, K per
// lane (lane l, item u: block base + 64 u + l), whose hashes h[0..K) the
// previous window requested.  Every home slot is requested at once (and, with
// kProbePair, the slot after it when both lie in one line), then the next
// window's hashes, before any slot is examined; the keys past what was read
// continue slot by slot, all together.  Every load is issued and none under a
// branch, so that they are all in flight together: the unwanted ones read the
// anchor, the slot that lane 0 looks up first (one line per wave, requested
// anyway), and are ignored.  A ballot per item finds the window's first miss
// (a block absent, or whose set is empty).  Returns true once the run has
// ended, with matched its length; otherwise h holds the next window's hashes.
template <int K, int KM>
__device__ __forceinline__ bool probe_window(const uint4 *__restrict__ sl, unsigned mask,
                                             const unsigned long long *__restrict__ hb, int lim,
                                             int base, int lane, unsigned long long (&h)[KM],
                                             int &matched, unsigned &deepest, bool &bad) {
  constexpr int KN = K < KM ? 2 * K : KM;  // items per lane of the next window
  const int win = 64 * K, nbase = base + win;
  unsigned long long hc[K];
  bool want[K], look[K], pair[K], hit[K];
  unsigned s[K], t[K];
  uint4 v[K], w[K];
#pragma unroll
  for (int u = 0; u < K; ++u) {
    hc[u] = h[u];
    want[u] = base + u * 64 + lane < lim;
    look[u] = want[u] && hc[u] != 0ull;
    bad = bad || (want[u] && !look[u]);  // hash 0 is reserved for empty slots: a miss
    s[u] = (unsigned)fmix64(hc[u]) & mask;
  }
  const unsigned anchor = (unsigned)__builtin_amdgcn_readfirstlane((int)s[0]);
#pragma unroll
  for (int u = 0; u < K; ++u) {
    v[u] = sl[look[u] ? s[u] : anchor];
    pair[u] = kProbePair && look[u] && (s[u] & 7u) != 7u;  // s + 1 <= mask then
    if (kProbePair) w[u] = sl[pair[u] ? s[u] + 1u : anchor];
  }
#pragma unroll
  for (int u = 0; u < KN; ++u) {
    const int j = nbase + u * 64 + lane;
    h[u] = j < lim ? hb[j] : 0ull;
  }
  unsigned pend = 0u;
#pragma unroll
  for (int u = 0; u < K; ++u) {
    hit[u] = false;
    t[u] = 0u;
    const bool d1 = examine_slot(v[u], hc[u], look[u], hit[u], t[u]);
    const bool go2 = pair[u] && !d1;
    const bool d2 = kProbePair && examine_slot(w[u], hc[u], go2, hit[u], t[u]);
    s[u] = go2 ? s[u] + 1u : s[u];
    pend |= (look[u] && !d1 && !d2) ? 1u << u : 0u;
  }
  for (unsigned p = 1; p <= mask && __ballot(pend != 0u) != 0; ++p) {  // mask + 1 slots
#pragma unroll
    for (int u = 0; u < K; ++u) {
      const bool go = (pend >> u) & 1u;
      s[u] = go ? (s[u] + 1u) & mask : s[u];
      v[u] = sl[go ? s[u] : anchor];
    }
    unsigned left = pend;
#pragma unroll
    for (int u = 0; u < K; ++u)
      left &= examine_slot(v[u], hc[u], (pend >> u) & 1u, hit[u], t[u]) ? ~(1u << u) : ~0u;
    pend = left;
  }
  // a lookup still pending has visited every slot: the key is absent
  int first = win;  // window position of the first miss
#pragma unroll
  for (int u = 0; u < K; ++u) {
    const uint64_t miss = __ballot(want[u] && !hit[u]);
    if (first == win && miss) first = u * 64 + __builtin_ctzll(miss);
  }
  unsigned tm = 0u;
#pragma unroll
  for (int u = 0; u < K; ++u)
    tm = (want[u] && hit[u] && u * 64 + lane < first && t[u] > tm) ? t[u] : tm;
  deepest = max(deepest, (unsigned)wave_max((unsigned long long)tm));
  if (first < win) {
    matched = base + first;
    return true;
  }
  matched = nbase < lim ? nbase : lim;
  return nbase >= lim;
}

// One wave per request.  Its leading blocks are looked up in windows of
// 64 * k blocks, k doubling from 1 to kProbeMaxK while every block hits, so a
// run of R cached blocks takes about log2 + R / (64 * kProbeMaxK) dependent
// rounds instead of R / 64, while a short run (most of them) costs one small
// window.  The wave stops at the first miss: blocks past it in later windows
// cost nothing.
__global__ __launch_bounds__(kBlock) void probe_kernel(const IndexSlot *__restrict__ slots,
                                                       unsigned mask, int n,
                                                       const int *__restrict__ offsets,
                                                       const unsigned long long *__restrict__ hashes,
                                                       const int *__restrict__ n_in, int bt,
                                                       int *__restrict__ n_prefix_out,
                                                       uint8_t *__restrict__ tier_out,
                                                       int *status) {
  constexpr int KM = kProbeMaxK;
  static_assert(KM == 1 || KM == 2 || KM == 4 || KM == 8, "window sizes");
  const int i = blockIdx.x * kWaves + wave_id();
  if (i >= n) return;  // uniform over the wave
  const int lane = lane_id();
  const uint4 *sl = reinterpret_cast<const uint4 *>(slots);
  // every read stays in [0, offsets[n]), the caller's hash array, even when
  // another request's offsets are out of order
  const int b0 = offsets[i], b1 = offsets[i + 1], total = offsets[n], nin = n_in[i];
  bool bad = b0 < 0 || b1 < b0 || b1 > total || nin < 1 || (i == 0 && b0 != 0);
  const int have = bad ? 0 : b1 - b0;
  const int cap = bad ? 0 : (nin - 1) / bt;
  const int lim = have < cap ? have : cap;
  const unsigned long long *hb = hashes + (bad ? 0 : b0);
  int matched = 0;
  unsigned deepest = 0;
  unsigned long long h[KM];
#pragma unroll
  for (int u = 0; u < KM; ++u) h[u] = (u == 0 && lane < lim) ? hb[lane] : 0ull;
  int base = 0, k = 1;
  bool done = lim <= 0;
  while (!done) {  // uniform over the wave
    if (k == 1)
      done = probe_window<1, KM>(sl, mask, hb, lim, base, lane, h, matched, deepest, bad);
    else if (k == 2)
      done = probe_window<(KM < 2 ? KM : 2), KM>(sl, mask, hb, lim, base, lane, h, matched,
                                                  deepest, bad);
    else if (k == 4)
      done = probe_window<(KM < 4 ? KM : 4), KM>(sl, mask, hb, lim, base, lane, h, matched,
                                                  deepest, bad);
    else
      done = probe_window<KM, KM>(sl, mask, hb, lim, base, lane, h, matched, deepest, bad);
    base += 64 * k;
    k = k < KM ? 2 * k : KM;
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
