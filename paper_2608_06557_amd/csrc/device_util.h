// device_util.h -- wave64 / workgroup primitives and cross-workgroup status
// words for the gfx950 kernels of libcascade.  Internal to the library.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cascade {

constexpr int kBlock = 256;          // threads per workgroup (4 wave64s)
constexpr int kWaves = kBlock / 64;
constexpr unsigned kSpinLimit = 1u << 20;  // bound on polls of one status word

template <typename T>
__device__ __forceinline__ T load_agent(const T *p) {
  return __hip_atomic_load(const_cast<T *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <typename T>
__device__ __forceinline__ void store_agent(T *p, T v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }
__device__ __forceinline__ int wave_id() { return threadIdx.x >> 6; }

// number of set bits of m below this lane
__device__ __forceinline__ int rank_in_mask(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((unsigned)(m >> 32),
                                   __builtin_amdgcn_mbcnt_lo((unsigned)m, 0u));
}

template <typename T>
__device__ __forceinline__ T wave_inclusive_sum(T x) {
  const int lane = lane_id();
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    T y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  return x;
}

template <typename T>
__device__ __forceinline__ T wave_sum(T x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

// Exclusive prefix sums of K values per thread over the workgroup, in
// thread order; also returns the workgroup totals.  `lds` holds kWaves*K.
template <int K, typename T>
__device__ __forceinline__ void block_exclusive_scan(T (&v)[K], T (&total)[K], T *lds) {
  const int lane = lane_id(), wave = wave_id();
  T inc[K];
#pragma unroll
  for (int k = 0; k < K; ++k) inc[k] = wave_inclusive_sum(v[k]);
  if (lane == 63) {
#pragma unroll
    for (int k = 0; k < K; ++k) lds[wave * K + k] = inc[k];
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < K; ++k) {
    T before = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      T x = lds[w * K + k];
      before += (w < wave) ? x : T(0);
      tot += x;
    }
    v[k] = before + inc[k] - v[k];
    total[k] = tot;
  }
  __syncthreads();
}

// Workgroup sums of K values; every thread receives the totals.
template <int K, typename T>
__device__ __forceinline__ void block_sum(T (&v)[K], T *lds) {
  const int lane = lane_id(), wave = wave_id();
#pragma unroll
  for (int k = 0; k < K; ++k) v[k] = wave_sum(v[k]);
  if (lane == 0) {
#pragma unroll
    for (int k = 0; k < K; ++k) lds[wave * K + k] = v[k];
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < K; ++k) {
    T tot = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) tot += lds[w * K + k];
    v[k] = tot;
  }
  __syncthreads();
}

// ---------------------------------------------------------------------------
// Decoupled look-back status words.  Each (tile, value) word holds
// (value << 2) | flag with flag 1 = tile aggregate, 2 = inclusive prefix;
// 0 means not yet published.  Words are written once per launch with single
// atomic stores, so a reader never sees a torn value; they are cleared
// before the launch that uses them.
constexpr unsigned kFlagAggregate = 1, kFlagInclusive = 2;

template <typename W>
__device__ __forceinline__ void publish(W *word, W value, unsigned flag) {
  store_agent(word, (W)((value << 2) | (W)flag));
}

// Sum of `value k` over tiles 0 .. tile-1, reading up to WIN predecessors per
// round trip.  Tiles are claimed in increasing order by running workgroups
// and publish their aggregate before they wait on anything, so every poll
// ends; the poll count is still bounded and a timeout is reported.
template <typename W, int WIN>
__device__ __forceinline__ W look_back(const W *status, int stride, int tile, int k,
                                       bool *timed_out) {
  W sum = 0;
  int j = tile - 1;
  unsigned spins = 0;
  while (j >= 0) {
    W v[WIN];
#pragma unroll
    for (int w = 0; w < WIN; ++w)
      v[w] = (j - w >= 0) ? load_agent(status + (size_t)(j - w) * stride + k)
                          : (W)kFlagInclusive;
    int consumed = 0;
    bool done = false, stalled = false;
#pragma unroll
    for (int w = 0; w < WIN; ++w) {
      if (!done && !stalled) {
        const unsigned f = (unsigned)(v[w] & 3);
        if (f == 0) {
          stalled = true;
        } else {
          sum += v[w] >> 2;
          ++consumed;
          done = (f == kFlagInclusive);
        }
      }
    }
    if (done) return sum;
    j -= consumed;
    if (stalled) {
      if (++spins > kSpinLimit) {
        *timed_out = true;
        return sum;
      }
      __builtin_amdgcn_s_sleep(1);
    }
  }
  return sum;
}

}  // namespace cascade
