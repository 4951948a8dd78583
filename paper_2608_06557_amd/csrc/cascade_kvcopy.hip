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
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "cascade.h"

namespace {

constexpr int kBlock = 256;
constexpr int kUnroll = 8;
constexpr long long kMaxGrid = 8192;

typedef int v4i __attribute__((ext_vector_type(4)));

template <bool kToStaging>
__global__ __launch_bounds__(kBlock) void kvcopy_kernel(cascade_kv_pool_t pool, char *staging,
                                                        int staging_slots,
                                                        const cascade_move_t *__restrict__ moves,
                                                        const int *__restrict__ n_dev,
                                                        int max_moves, int *status) {
  const int nm = min(*n_dev, max_moves);
  if (nm <= 0) return;
  const int per_move = 2 * pool.num_layers;
  const long long total = (long long)nm * per_move;
  const long long cb = pool.chunk_bytes;
  const int vecs = (int)(cb >> 4);
  for (long long c = blockIdx.x; c < total; c += gridDim.x) {
    const int m = (int)(c / per_move);
    const int r = (int)(c - (long long)m * per_move);
    const int l = r >> 1, kv = r & 1;
    const cascade_move_t mv = moves[m];
    if ((unsigned)mv.pool_slot >= (unsigned)pool.num_slots ||
        (unsigned)mv.staging_slot >= (unsigned)staging_slots) {
      if (threadIdx.x == 0 && status) *status = CASCADE_EINVAL;
      continue;
    }
    char *pc = static_cast<char *>(pool.base) + (long long)l * pool.layer_stride +
               (long long)kv * pool.kv_stride + (long long)mv.pool_slot * pool.slot_stride;
    char *sc = staging + (((long long)mv.staging_slot * pool.num_layers + l) * 2 + kv) * cb;
    const v4i *src = reinterpret_cast<const v4i *>(kToStaging ? pc : sc);
    v4i *dst = reinterpret_cast<v4i *>(kToStaging ? sc : pc);
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
}

bool geometry_ok(const cascade_kv_pool_t *p, const void *staging, int32_t staging_slots,
                 const cascade_move_t *moves, const int32_t *n_dev, int32_t max_moves) {
  if (!p || !staging || !n_dev || max_moves < 0 || staging_slots < 0) return false;
  if (max_moves > 0 && !moves) return false;
  if (!p->base || p->num_layers < 1 || p->num_slots < 0) return false;
  if (p->chunk_bytes < 16 || (p->chunk_bytes & 15) || p->chunk_bytes > (1ll << 30)) return false;
  if ((p->layer_stride & 15) || (p->kv_stride & 15) || (p->slot_stride & 15)) return false;
  if (p->layer_stride < 0 || p->kv_stride < 0 || p->slot_stride < 0) return false;
  if (((uintptr_t)p->base & 15) || ((uintptr_t)staging & 15)) return false;
  return true;
}

template <bool kToStaging>
int launch(const cascade_kv_pool_t *pool, const void *staging, int32_t staging_slots,
           const cascade_move_t *moves, const int32_t *n_dev, int32_t max_moves,
           int32_t *status, void *stream) {
  if (!geometry_ok(pool, staging, staging_slots, moves, n_dev, max_moves)) return CASCADE_EINVAL;
  if (max_moves == 0) return CASCADE_OK;
  const long long chunks = (long long)max_moves * 2 * pool->num_layers;
  const int grid = (int)std::max<long long>(1, std::min(chunks, kMaxGrid));
  hipLaunchKernelGGL(kvcopy_kernel<kToStaging>, dim3(grid), dim3(kBlock), 0,
                     static_cast<hipStream_t>(stream), *pool,
                     const_cast<char *>(static_cast<const char *>(staging)), staging_slots, moves,
                     n_dev, max_moves, status);
  return hipGetLastError() == hipSuccess ? CASCADE_OK : CASCADE_EHIP;
}

}  // namespace

extern "C" int cascade_pack(const cascade_kv_pool_t *pool, void *staging, int32_t staging_slots,
                            const cascade_move_t *moves, const int32_t *n_moves_dev,
                            int32_t max_moves, int32_t *status_dev, void *stream) {
  return launch<true>(pool, staging, staging_slots, moves, n_moves_dev, max_moves, status_dev,
                      stream);
}

extern "C" int cascade_unpack(const cascade_kv_pool_t *pool, const void *staging,
                              int32_t staging_slots, const cascade_move_t *moves,
                              const int32_t *n_moves_dev, int32_t max_moves, int32_t *status_dev,
                              void *stream) {
  return launch<false>(pool, staging, staging_slots, moves, n_moves_dev, max_moves, status_dev,
                       stream);
}
