// device_util.h -- wave64 / workgroup primitives and cross-workgroup status
// words for the gfx950 kernels of libcascade.  Internal to the library.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

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

// Wave64 scans on DPP lane moves (GFX9 data-parallel primitives), register
// to register: Hillis-Steele doubling inside each row of 16 lanes (row_shr
// 1, 2, 4, 8), then row 0's total into row 1 and row 2's into row 3
// (row_bcast:15), then rows 0-1's total into rows 2-3 (row_bcast:31).  A
// lane with no source reads `ident`.  64-bit values move as two halves.
enum : int {
  kDppRowShr1 = 0x111, kDppRowShr2 = 0x112, kDppRowShr4 = 0x114, kDppRowShr8 = 0x118,
  kDppRowBcast15 = 0x142, kDppRowBcast31 = 0x143
};

template <int kCtrl, int kRowMask>
__device__ __forceinline__ unsigned dpp_move(unsigned ident, unsigned x) {
  return (unsigned)__builtin_amdgcn_update_dpp((int)ident, (int)x, kCtrl, kRowMask, 0xf, false);
}
template <int kCtrl, int kRowMask>
__device__ __forceinline__ unsigned long long dpp_move(unsigned long long ident,
                                                       unsigned long long x) {
  const unsigned lo = dpp_move<kCtrl, kRowMask>((unsigned)ident, (unsigned)x);
  const unsigned hi = dpp_move<kCtrl, kRowMask>((unsigned)(ident >> 32), (unsigned)(x >> 32));
  return ((unsigned long long)hi << 32) | lo;
}

struct OpAdd {
  template <typename U> __device__ __forceinline__ U operator()(U a, U b) const { return a + b; }
};
struct OpMin {
  template <typename U> __device__ __forceinline__ U operator()(U a, U b) const {
    return b < a ? b : a;
  }
};
struct OpMax {
  template <typename U> __device__ __forceinline__ U operator()(U a, U b) const {
    return b > a ? b : a;
  }
};

// Inclusive scan of an associative op over the 64 lanes (U: unsigned or
// unsigned long long; signed sums go through their two's-complement bits).
template <typename Op, typename U>
__device__ __forceinline__ U wave_inclusive_scan(U x, U ident) {
  const Op op;
  x = op(x, dpp_move<kDppRowShr1, 0xf>(ident, x));
  x = op(x, dpp_move<kDppRowShr2, 0xf>(ident, x));
  x = op(x, dpp_move<kDppRowShr4, 0xf>(ident, x));
  x = op(x, dpp_move<kDppRowShr8, 0xf>(ident, x));
  x = op(x, dpp_move<kDppRowBcast15, 0xa>(ident, x));
  x = op(x, dpp_move<kDppRowBcast31, 0xc>(ident, x));
  return x;
}

// Lane 63's value, as a wave-uniform result.
__device__ __forceinline__ unsigned last_lane(unsigned x) {
  return (unsigned)__builtin_amdgcn_readlane((int)x, 63);
}
__device__ __forceinline__ unsigned long long last_lane(unsigned long long x) {
  const unsigned lo = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)x, 63);
  const unsigned hi = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)(x >> 32), 63);
  return ((unsigned long long)hi << 32) | lo;
}

template <typename T> struct UnsignedOf;
template <> struct UnsignedOf<int> { typedef unsigned type; };
template <> struct UnsignedOf<unsigned> { typedef unsigned type; };
template <> struct UnsignedOf<long long> { typedef unsigned long long type; };
template <> struct UnsignedOf<unsigned long long> { typedef unsigned long long type; };

template <typename T>
__device__ __forceinline__ T wave_inclusive_sum(T x) {
  typedef typename UnsignedOf<T>::type U;
  return (T)wave_inclusive_scan<OpAdd, U>((U)x, (U)0);
}

template <typename T>
__device__ __forceinline__ T wave_sum(T x) {
  typedef typename UnsignedOf<T>::type U;
  return (T)last_lane(wave_inclusive_scan<OpAdd, U>((U)x, (U)0));
}

__device__ __forceinline__ unsigned long long wave_min(unsigned long long x) {
  return last_lane(wave_inclusive_scan<OpMin, unsigned long long>(x, ~0ull));
}
__device__ __forceinline__ unsigned long long wave_max(unsigned long long x) {
  return last_lane(wave_inclusive_scan<OpMax, unsigned long long>(x, 0ull));
}

// Lane `src` (wave-uniform) of x.
__device__ __forceinline__ unsigned lane_value(unsigned x, int src) {
  return (unsigned)__builtin_amdgcn_readlane((int)x, src);
}
__device__ __forceinline__ unsigned long long lane_value(unsigned long long x, int src) {
  const unsigned lo = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)x, src);
  const unsigned hi = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)(x >> 32), src);
  return ((unsigned long long)hi << 32) | lo;
}

// Exclusive prefix sums of K values per thread over a workgroup of NW waves,
// in thread order; also returns the workgroup totals.  `lds` holds NW*K.
// Each wave scans its lanes (DPP); every thread then reads the NW wave
// totals from LDS (broadcast reads) and adds those of the waves before its
// own, so the register use does not grow with NW.
template <int K, typename T, int NW = kWaves>
__device__ __forceinline__ void block_exclusive_scan(T (&v)[K], T (&total)[K], T *lds) {
  static_assert(NW <= 64, "at most 64 waves");
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
    T before = T(0), all = T(0);
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const T x = lds[w * K + k];
      before += w < wave ? x : T(0);
      all += x;
    }
    total[k] = all;
    v[k] = before + inc[k] - v[k];
  }
  __syncthreads();
}

// Workgroup sums of K values over NW waves; every thread receives the totals.
template <int K, typename T, int NW = kWaves>
__device__ __forceinline__ void block_sum(T (&v)[K], T *lds) {
  static_assert(NW <= 64, "at most 64 waves");
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
    T all = T(0);
#pragma unroll
    for (int w = 0; w < NW; ++w) all += lds[w * K + k];
    v[k] = all;
  }
  __syncthreads();
}

// ---------------------------------------------------------------------------
// Hand-over to the last workgroup of a grid.  Values another workgroup reads
// within the same launch are written with agent-scope atomic stores, which
// need no cache write-back: completing them (wait_stores) before the ticket
// is their release.  A device-wide fence per workgroup would write the whole
// L2 back, and costs far more than the stores themselves.
constexpr int kTicketGroups = 16;  // first-level counters of the last-workgroup test
constexpr int kTicketStride = 32;  // one counter per 128-byte line

// Wait until this thread's memory operations have completed.
__device__ __forceinline__ void wait_stores() { __builtin_amdgcn_s_waitcnt(0x0f70); }  // vmcnt(0)

// Acquire side of a hand-over: called by every thread of a workgroup once it
// has seen (directly, or through a workgroup barrier after one thread did)
// the ticket or counter that says every producer's stores are complete.  An
// agent-scope acquire fence: later loads are neither moved above it by the
// compiler nor served from this CU's stale L1 lines (one cache invalidate;
// it writes nothing back).
__device__ __forceinline__ void acquire_agent() {
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
}

// Called by one thread per workgroup once its results are stored: true for
// the last workgroup of the grid to arrive (with an acquire fence in the
// calling thread; the others call acquire_agent() after the barrier that
// shares the answer).  Above kTicketFlat workgroups, two levels of counters
// (16 groups, then one) keep the atomics on any one address to a few dozen,
// where a single counter would serialize one per workgroup; up to it, one
// counter and one round trip.  Counters are reset by the workgroup that
// completes them, so every launch finds them at zero.  `tk` holds
// (kTicketGroups + 1) * kTicketStride words.
constexpr unsigned kTicketFlat = 64;
__device__ __forceinline__ bool last_workgroup(unsigned *tk) {
  const unsigned G = gridDim.x, groups = G <= kTicketFlat ? 1u : min(G, (unsigned)kTicketGroups);
  const unsigned g = blockIdx.x % groups;
  const unsigned size = (G - g + groups - 1) / groups;
  unsigned *c = tk + g * kTicketStride;
  if (atomicAdd(c, 1u) != size - 1) return false;
  store_agent(c, 0u);
  if (groups == 1u) {
    acquire_agent();
    return true;
  }
  unsigned *top = tk + kTicketGroups * kTicketStride;
  if (atomicAdd(top, 1u) != groups - 1) return false;
  store_agent(top, 0u);
  acquire_agent();
  return true;
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
// round trip.  Workgroup b owns tile b; workgroups are dispatched in index
// order and publish their aggregate before they wait on anything, so every
// poll ends; the poll count is still bounded and a timeout is reported.
template <typename W, int WIN>
__device__ __forceinline__ W look_back(const W *status, int stride, int tile, int k,
                                       bool *timed_out) {
  static_assert(WIN <= 64, "flags of one window fit a 64-bit mask");
  W sum = 0;
  int j = tile - 1;
  unsigned spins = 0;
  while (j >= 0) {
    W v[WIN];
#pragma unroll
    for (int w = 0; w < WIN; ++w)
      v[w] = (j - w >= 0) ? load_agent(status + (size_t)(j - w) * stride + k)
                          : (W)kFlagInclusive;
    // the window's flags as masks: consume up to the first inclusive prefix,
    // or up to the first word not yet published
    typedef typename std::conditional<(WIN > 32), unsigned long long, unsigned>::type Mask;
    Mask missing = 0, inclusive = 0;
#pragma unroll
    for (int w = 0; w < WIN; ++w) {
      const unsigned f = (unsigned)(v[w] & 3);
      missing |= (Mask)(f == 0 ? 1u : 0u) << w;
      inclusive |= (Mask)(f == kFlagInclusive ? 1u : 0u) << w;
    }
    const int first_missing = missing ? __builtin_ctzll(missing) : WIN;
    const int first_inclusive = inclusive ? __builtin_ctzll(inclusive) : WIN;
    const bool done = first_inclusive < first_missing;
    const int take = done ? first_inclusive + 1 : first_missing;
#pragma unroll
    for (int w = 0; w < WIN; ++w) sum += w < take ? (v[w] >> 2) : (W)0;
    if (done) return sum;
    j -= take;
    if (first_missing < WIN) {
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
