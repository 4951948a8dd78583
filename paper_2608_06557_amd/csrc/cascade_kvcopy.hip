// cascade_kvcopy.hip -- paged-KV block gather / scatter on gfx950.
//
// Cascade restores prefix KV into HBM only at the final DRAM->HBM hop and
// spills preempted prefill state to DRAM (Section 4.4).  On the GPU side both
// are byte-exact copies of every (layer, K/V) chunk of a KV block between the
// paged HBM pool, where a block's chunks are scattered over per-layer caches,
// and a contiguous staging buffer that the host-side DMA reads or fills.
//
// The copy is HBM-bound: one workgroup moves one chunk per iteration with
// 16-byte loads and stores, all loads of a thread issued before its stores so
// that every lane keeps kUnroll requests in flight; nontemporal loads and
// stores stream past the caches.  The grid strides over (move, layer, K/V)
// chunks with up to kMaxGrid workgroups (about 32 per CU): measured on MI355X,
// a plain copy peaks near that occupancy.  The move count is read on the
// device, so the step's output count drives the copy without a host sync.
//
// The fused entry point interleaves the chunks of both lists.  On MI355X a
// stream of scattered pool reads (spill) and one of scattered pool writes
// (restore) sharing the chip move more bytes per second than either alone,
// and one launch has one tail instead of two.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "cascade.h"
#include "copy_range.h"

namespace {

constexpr int kBlock = 256;
constexpr int kUnroll = 8;
constexpr long long kMaxGrid = 8192;

typedef int v4i __attribute__((ext_vector_type(4)));

// One chunk of vecs 16-byte vectors; thread t moves vectors t + kBlock*i, so
// a thread that copies the same chunk twice touches the same addresses.
__device__ __forceinline__ void copy_chunk(const char *src_c, char *dst_c, int vecs) {
  const v4i *src = reinterpret_cast<const v4i *>(src_c);
  v4i *dst = reinterpret_cast<v4i *>(dst_c);
  for (int base = 0; base < vecs; base += kBlock * kUnroll) {
    v4i t[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int k = base + u * kBlock + threadIdx.x;
      if (k < vecs) t[u] = __builtin_nontemporal_load(src + k);
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int k = base + u * kBlock + threadIdx.x;
      if (k < vecs) __builtin_nontemporal_store(t[u], dst + k);
    }
  }
}

// A spill and the restore into the same chunk in one pass: both loads of a
// batch are issued together, then the spill's stores, then the restore's.
// Each thread stores to a pool address only after its own load of that
// address has returned (the spill's store needed the loaded value), so the
// spill reads the old bytes.  Half the unroll per stream keeps the same
// kUnroll vectors in flight and the kernel's register count at the level
// of a plain copy (full occupancy).
__device__ __forceinline__ void copy_pair(char *pool_c, char *spill_c, const char *fill_c,
                                          int vecs) {
  constexpr int kHalf = kUnroll / 2;
  v4i *pool = reinterpret_cast<v4i *>(pool_c);
  v4i *spill = reinterpret_cast<v4i *>(spill_c);
  const v4i *fill = reinterpret_cast<const v4i *>(fill_c);
  for (int base = 0; base < vecs; base += kBlock * kHalf) {
    v4i a[kHalf], b[kHalf];
#pragma unroll
    for (int u = 0; u < kHalf; ++u) {
      const int k = base + u * kBlock + threadIdx.x;
      if (k < vecs) {
        a[u] = __builtin_nontemporal_load(pool + k);
        b[u] = __builtin_nontemporal_load(fill + k);
      }
    }
#pragma unroll
    for (int u = 0; u < kHalf; ++u) {
      const int k = base + u * kBlock + threadIdx.x;
      if (k < vecs) __builtin_nontemporal_store(a[u], spill + k);
    }
#pragma unroll
    for (int u = 0; u < kHalf; ++u) {
      const int k = base + u * kBlock + threadIdx.x;
      if (k < vecs) __builtin_nontemporal_store(b[u], pool + k);
    }
  }
}

__device__ __forceinline__ char *pool_chunk(const cascade_kv_pool_t &pool, int slot, int l,
                                            int kv) {
  return static_cast<char *>(pool.base) + (long long)l * pool.layer_stride +
         (long long)kv * pool.kv_stride + (long long)slot * pool.slot_stride;
}

// Chunks r = 2*l + kv of a block, in the pool and in a staging slot (the
// staging slot's chunks are consecutive).
__device__ __forceinline__ char *pool_r(const cascade_kv_pool_t &pool, int slot, int r) {
  return pool_chunk(pool, slot, r >> 1, r & 1);
}
__device__ __forceinline__ char *stage_r(char *staging, const cascade_kv_pool_t &pool, int slot,
                                         int r) {
  return staging + ((long long)slot * 2 * pool.num_layers + r) * pool.chunk_bytes;
}

// A work item ("unit") is g consecutive chunks r0 .. r0+g-1 of one block.
// Chunks of 32 KiB or more, or of a size that does not tile 32 KiB, are one
// unit each and move with copy_chunk.  Smaller chunks of a multiple of 4 KiB
// are grouped g = 32 KiB / chunk to a unit, so that each thread still has
// kUnroll vectors in flight: vector slot u of a thread is vector
// ((u & (per - 1)) * kBlock + t) of chunk r0 + (u >> lg), per = 2^lg =
// chunk / 4 KiB.
struct Units {
  int g, lg, per_move;  // chunks per unit, log2(vectors per chunk / kBlock), units per block
};

template <int kLg>
__device__ __forceinline__ int unit_off(int u) {
  return ((u & ((1 << kLg) - 1)) * kBlock) + (int)threadIdx.x;
}

// one unit of g = kUnroll >> kLg chunks from pool slot to staging slot (or back)
template <bool kToStaging, int kLg>
__device__ __forceinline__ void copy_group(const cascade_kv_pool_t &pool, int slot, char *stg,
                                           int sslot, int r0) {
  v4i t[kUnroll];
#pragma unroll
  for (int u = 0; u < kUnroll; ++u) {
    const int r = r0 + (u >> kLg);
    const char *src = kToStaging ? pool_r(pool, slot, r) : stage_r(stg, pool, sslot, r);
    t[u] = __builtin_nontemporal_load(reinterpret_cast<const v4i *>(src) + unit_off<kLg>(u));
  }
#pragma unroll
  for (int u = 0; u < kUnroll; ++u) {
    const int r = r0 + (u >> kLg);
    char *dst = kToStaging ? stage_r(stg, pool, sslot, r) : pool_r(pool, slot, r);
    __builtin_nontemporal_store(t[u], reinterpret_cast<v4i *>(dst) + unit_off<kLg>(u));
  }
}

// spill and the restore into the same unit, as copy_pair: half the slots per
// stream at a time, the spill's stores before the restore's
template <int kLg>
__device__ __forceinline__ void copy_pair_group(const cascade_kv_pool_t &pool, int slot,
                                                char *spill, int spill_slot, char *fill,
                                                int fill_slot, int r0) {
  constexpr int kHalf = kUnroll / 2;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    v4i a[kHalf], b[kHalf];
#pragma unroll
    for (int u = 0; u < kHalf; ++u) {
      const int uu = h * kHalf + u, r = r0 + (uu >> kLg), k = unit_off<kLg>(uu);
      a[u] = __builtin_nontemporal_load(reinterpret_cast<const v4i *>(pool_r(pool, slot, r)) + k);
      b[u] = __builtin_nontemporal_load(
          reinterpret_cast<const v4i *>(stage_r(fill, pool, fill_slot, r)) + k);
    }
#pragma unroll
    for (int u = 0; u < kHalf; ++u) {
      const int uu = h * kHalf + u, r = r0 + (uu >> kLg), k = unit_off<kLg>(uu);
      __builtin_nontemporal_store(a[u],
                                  reinterpret_cast<v4i *>(stage_r(spill, pool, spill_slot, r)) + k);
    }
#pragma unroll
    for (int u = 0; u < kHalf; ++u) {
      const int uu = h * kHalf + u, r = r0 + (uu >> kLg), k = unit_off<kLg>(uu);
      __builtin_nontemporal_store(b[u], reinterpret_cast<v4i *>(pool_r(pool, slot, r)) + k);
    }
  }
}

// The unit shape is a template parameter of the kernels, so each compiled
// kernel holds one copy path: kLg < 0 whole chunks (g == 1), else a group of
// g = kUnroll >> kLg chunks.
template <bool kToStaging, int kLg>
__device__ __forceinline__ void copy_unit(const cascade_kv_pool_t &pool, int slot, char *stg,
                                          int sslot, int r0, int vecs) {
  if constexpr (kLg < 0) {
    char *pc = pool_r(pool, slot, r0);
    char *sc = stage_r(stg, pool, sslot, r0);
    copy_chunk(kToStaging ? pc : sc, kToStaging ? sc : pc, vecs);
  } else {
    copy_group<kToStaging, kLg>(pool, slot, stg, sslot, r0);
  }
}

template <int kLg>
__device__ __forceinline__ void copy_pair_unit(const cascade_kv_pool_t &pool, int slot,
                                               char *spill, int spill_slot, char *fill,
                                               int fill_slot, int r0, int vecs) {
  if constexpr (kLg < 0)
    copy_pair(pool_r(pool, slot, r0), stage_r(spill, pool, spill_slot, r0),
              stage_r(fill, pool, fill_slot, r0), vecs);
  else
    copy_pair_group<kLg>(pool, slot, spill, spill_slot, fill, fill_slot, r0);
}

__device__ __forceinline__ bool move_ok(const cascade_move_t &mv, int num_slots,
                                        int staging_slots) {
  return (unsigned)mv.pool_slot < (unsigned)num_slots &&
         (unsigned)mv.staging_slot < (unsigned)staging_slots;
}

__device__ __forceinline__ void flag_bad(int *status) {
  if (threadIdx.x == 0 && status) *status = CASCADE_EINVAL;
}

template <bool kToStaging, int kLg>
__global__ __launch_bounds__(kBlock) void kvcopy_kernel(cascade_kv_pool_t pool, Units un,
                                                        char *staging, int staging_slots,
                                                        const cascade_move_t *__restrict__ moves,
                                                        const int *__restrict__ n_dev,
                                                        int first, int max_moves, int *status) {
  // moves points at entry `first` of a list of *n_dev entries
  const int nm = min(*n_dev - first, max_moves);
  if (nm <= 0) return;
  const long long total = (long long)nm * un.per_move;
  const int vecs = (int)(pool.chunk_bytes >> 4);
  // each item's move is requested one item ahead, as in kvmove_kernel
  cascade_move_t n_mv = {0, 0, 0, 0};
  if ((long long)blockIdx.x < total) n_mv = moves[(int)(blockIdx.x / un.per_move)];
  for (long long c = blockIdx.x; c < total; c += gridDim.x) {
    const int m = (int)(c / un.per_move);
    const int r0 = (int)(c - (long long)m * un.per_move) * un.g;
    const cascade_move_t mv = n_mv;
    if (c + gridDim.x < total) n_mv = moves[(int)((c + gridDim.x) / un.per_move)];
    if (!move_ok(mv, pool.num_slots, staging_slots)) {
      flag_bad(status);
      continue;
    }
    copy_unit<kToStaging, kLg>(pool, mv.pool_slot, staging, mv.staging_slot, r0, vecs);
  }
}

// Pack and unpack chunks interleaved: the common range holds one pack and
// one unpack chunk per item pair, the rest belongs to the longer list.
// Unpack move m paired with pack move j (phz[j] == m and uhz[m] == j) is
// copied by the item of chunk (j, l, kv), in the same pass as the spill and
// by the same threads, each of which has read the slot's old bytes before it
// overwrites them: the wait is inside the thread, none crosses workgroups.
// The pairing test reads the same two words from both sides, so every
// unpack move is copied exactly once.
// Eight waves per SIMD: the prefetched move words would otherwise push the
// scalar registers past what eight waves can hold, and at seven the copy
// moves about 2 % fewer bytes per second (the prefetch gains about 1 % at
// eight, measured on MI355X).
template <int kLg>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(8, 8))) void kvmove_kernel(
    cascade_kv_pool_t pool, Units un, char *pst, int pst_slots,
    const cascade_move_t *__restrict__ pm,
    const int *__restrict__ pn_dev, int pmax, const int *__restrict__ phz, char *ust,
    int ust_slots, const cascade_move_t *__restrict__ um, const int *__restrict__ un_dev,
    int umax, const int *__restrict__ uhz, int *status) {
  const int np = max(0, min(*pn_dev, pmax));
  const int nu = max(0, min(*un_dev, umax));
  const int per_move = un.per_move;
  const long long tp = (long long)np * per_move, tu = (long long)nu * per_move;
  const long long both = 2 * (tp < tu ? tp : tu), total = tp + tu;
  const int vecs = (int)(pool.chunk_bytes >> 4);
  // the grid is even when it is below the item count, so c and
  // c ^ 1 fall in the same iteration: flipping the low bit on odd iterations
  // is a bijection that makes every workgroup alternate between pack and
  // unpack items, whatever share of the pack items carries a paired unpack
  const long long flip = (gridDim.x & 1) == 0 ? 1 : 0;
  // item c's list, move and chunk group
  auto item_of = [&](long long c, long long it, bool &is_pack, int &mi, int &r0) {
    long long ci;
    if (c < both) {
      const long long cc = c ^ (it & flip);
      is_pack = (cc & 1) == 0;
      ci = cc >> 1;
    } else {
      is_pack = tp > tu;
      ci = c - both + (both >> 1);
    }
    mi = (int)(ci / per_move);
    r0 = (int)(ci - (long long)mi * per_move) * un.g;
  };
  // each item's move and hazard word are requested one item ahead, while
  // the workgroup copies the item before it, so that no item starts with a
  // round trip in which the workgroup has no copy load in flight
  bool n_pack = false;
  int n_mi = 0, n_r0 = 0;
  cascade_move_t n_mv = {0, 0, 0, 0};
  int n_partner = -1;
  if ((long long)blockIdx.x < total) {
    item_of(blockIdx.x, 0, n_pack, n_mi, n_r0);
    n_mv = n_pack ? pm[n_mi] : um[n_mi];
    n_partner = n_pack ? phz[n_mi] : uhz[n_mi];
  }
  long long it = 0;
  for (long long c = blockIdx.x; c < total; c += gridDim.x, ++it) {
    const bool is_pack = n_pack;
    const int mi = n_mi, r0 = n_r0;
    const cascade_move_t mv = n_mv;
    const int partner = n_partner;
    if (c + gridDim.x < total) {
      item_of(c + gridDim.x, it + 1, n_pack, n_mi, n_r0);
      n_mv = n_pack ? pm[n_mi] : um[n_mi];
      n_partner = n_pack ? phz[n_mi] : uhz[n_mi];
    }
    if (is_pack) {
      const bool ok = move_ok(mv, pool.num_slots, pst_slots);
      if (!ok) flag_bad(status);
      bool paired = false;
      cascade_move_t mu;
      if (partner >= 0 && partner < nu) {
        mu = um[partner];
        paired = uhz[partner] == mi;
      }
      if (paired && !move_ok(mu, pool.num_slots, ust_slots)) {
        flag_bad(status);
        paired = false;  // the restore is skipped; the spill still runs
      }
      if (ok && paired && mu.pool_slot == mv.pool_slot) {
        copy_pair_unit<kLg>(pool, mv.pool_slot, pst, mv.staging_slot, ust, mu.staging_slot, r0,
                            vecs);
      } else {
        if (ok) copy_unit<true, kLg>(pool, mv.pool_slot, pst, mv.staging_slot, r0, vecs);
        if (paired) copy_unit<false, kLg>(pool, mu.pool_slot, ust, mu.staging_slot, r0, vecs);
      }
    } else {
      if (partner >= 0 && partner < np && phz[partner] == mi) continue;  // after its pack
      if (move_ok(mv, pool.num_slots, ust_slots))
        copy_unit<false, kLg>(pool, mv.pool_slot, ust, mv.staging_slot, r0, vecs);
      else
        flag_bad(status);
    }
  }
}

bool pool_ok(const cascade_kv_pool_t *p) {
  if (!p || !p->base || p->num_layers < 1 || p->num_slots < 0) return false;
  if (p->chunk_bytes < 16 || (p->chunk_bytes & 15) || p->chunk_bytes > (1ll << 30)) return false;
  if ((p->layer_stride & 15) || (p->kv_stride & 15) || (p->slot_stride & 15)) return false;
  if (p->layer_stride < 0 || p->kv_stride < 0 || p->slot_stride < 0) return false;
  return ((uintptr_t)p->base & 15) == 0;
}

bool list_ok(const void *staging, int32_t staging_slots, const cascade_move_t *moves,
             const int32_t *n_dev, int32_t max_moves) {
  if (!staging || !n_dev || max_moves < 0 || staging_slots < 0) return false;
  if (max_moves > 0 && !moves) return false;
  return ((uintptr_t)staging & 15) == 0;
}

Units units_for(const cascade_kv_pool_t *pool) {
  Units u;
  u.g = 1;
  u.lg = 0;
  const long long vecs = pool->chunk_bytes >> 4;
  const int chunks = 2 * pool->num_layers;
  const int full = kBlock * kUnroll;  // vectors one thread batch covers
  if (vecs < full && vecs % kBlock == 0 && full % vecs == 0 && chunks % (full / vecs) == 0) {
    u.g = (int)(full / vecs);
    while ((kBlock << u.lg) < vecs) ++u.lg;
  }
  u.per_move = chunks / u.g;
  return u;
}

int grid_for(const Units &u, long long moves) {
  const long long items = moves * u.per_move;
  long long g = std::max<long long>(1, std::min(items, kMaxGrid));
  if (g > 1 && (g & 1)) --g;  // even: the fused kernel alternates its lists by iteration
  return (int)g;
}

template <bool kToStaging>
int launch(const cascade_kv_pool_t *pool, const void *staging, int32_t staging_slots,
           const cascade_move_t *moves, const int32_t *n_dev, int32_t first, int32_t max_moves,
           int32_t *status, void *stream) {
  if (!pool_ok(pool) || !list_ok(staging, staging_slots, moves, n_dev, max_moves) || first < 0)
    return CASCADE_EINVAL;
  if (max_moves == 0) return CASCADE_OK;
  const Units u = units_for(pool);
  auto kernel = u.g == 1 ? kvcopy_kernel<kToStaging, -1>
                : u.lg == 0 ? kvcopy_kernel<kToStaging, 0>
                : u.lg == 1 ? kvcopy_kernel<kToStaging, 1>
                            : kvcopy_kernel<kToStaging, 2>;
  hipLaunchKernelGGL(kernel, dim3(grid_for(u, max_moves)), dim3(kBlock), 0,
                     static_cast<hipStream_t>(stream), *pool, u,
                     const_cast<char *>(static_cast<const char *>(staging)), staging_slots,
                     moves + first, n_dev, first, max_moves, status);
  return hipGetLastError() == hipSuccess ? CASCADE_OK : CASCADE_EHIP;
}

}  // namespace

int cascade::copy_range(bool to_staging, const cascade_kv_pool_t *pool, const void *staging,
                        int32_t staging_slots, const cascade_move_t *moves,
                        const int32_t *n_moves_dev, int32_t first, int32_t max_moves,
                        int32_t *status_dev, void *stream) {
  return to_staging ? launch<true>(pool, staging, staging_slots, moves, n_moves_dev, first,
                                   max_moves, status_dev, stream)
                    : launch<false>(pool, staging, staging_slots, moves, n_moves_dev, first,
                                    max_moves, status_dev, stream);
}

extern "C" int cascade_pack(const cascade_kv_pool_t *pool, void *staging, int32_t staging_slots,
                            const cascade_move_t *moves, const int32_t *n_moves_dev,
                            int32_t max_moves, int32_t *status_dev, void *stream) {
  return launch<true>(pool, staging, staging_slots, moves, n_moves_dev, 0, max_moves,
                      status_dev, stream);
}

extern "C" int cascade_unpack(const cascade_kv_pool_t *pool, const void *staging,
                              int32_t staging_slots, const cascade_move_t *moves,
                              const int32_t *n_moves_dev, int32_t max_moves, int32_t *status_dev,
                              void *stream) {
  return launch<false>(pool, staging, staging_slots, moves, n_moves_dev, 0, max_moves,
                       status_dev, stream);
}

extern "C" int cascade_pack_unpack(const cascade_kv_pool_t *pool, void *pack_staging,
                                   int32_t pack_staging_slots, const cascade_move_t *pack_moves,
                                   const int32_t *n_pack_dev, int32_t max_pack,
                                   const int32_t *pack_hazard, const void *unpack_staging,
                                   int32_t unpack_staging_slots,
                                   const cascade_move_t *unpack_moves,
                                   const int32_t *n_unpack_dev, int32_t max_unpack,
                                   const int32_t *unpack_hazard, int32_t *status_dev,
                                   void *stream) {
  if (!pool_ok(pool) ||
      !list_ok(pack_staging, pack_staging_slots, pack_moves, n_pack_dev, max_pack) ||
      !list_ok(unpack_staging, unpack_staging_slots, unpack_moves, n_unpack_dev, max_unpack))
    return CASCADE_EINVAL;
  if ((max_pack > 0 && !pack_hazard) || (max_unpack > 0 && !unpack_hazard)) return CASCADE_EINVAL;
  if (max_pack == 0 && max_unpack == 0) return CASCADE_OK;
  const Units u = units_for(pool);
  auto kernel = u.g == 1 ? kvmove_kernel<-1>
                : u.lg == 0 ? kvmove_kernel<0>
                : u.lg == 1 ? kvmove_kernel<1>
                            : kvmove_kernel<2>;
  hipLaunchKernelGGL(kernel, dim3(grid_for(u, (long long)max_pack + max_unpack)),
                     dim3(kBlock), 0, static_cast<hipStream_t>(stream), *pool, u,
                     static_cast<char *>(pack_staging), pack_staging_slots, pack_moves,
                     n_pack_dev, max_pack, pack_hazard,
                     const_cast<char *>(static_cast<const char *>(unpack_staging)),
                     unpack_staging_slots, unpack_moves, n_unpack_dev, max_unpack, unpack_hazard,
                     status_dev);
  return hipGetLastError() == hipSuccess ? CASCADE_OK : CASCADE_EHIP;
}
