// cascade_hosttier.hip -- KV movement between the DRAM tier (pinned host
// memory) and the HBM pool, with the host link overlapped with the on-GPU
// scatter / gather.
//
// Cascade allocates HBM only at the final DRAM->HBM hop of a restore and
// spills preempted prefills to DRAM (Section 4.4); the time of that hop is
// the DRAM link term of eq:restore_time.  A restore is two copies: DRAM ->
// contiguous staging over the host link (a DMA engine), then staging ->
// scattered pool slots (cascade_unpack).  Here the move list is cut into
// batches: the DMA of batch k+1 runs on the copy stream while batch k is
// unpacked on the compute stream, each batch's unpack waiting on an event
// recorded after its DMA.  A spill runs the mirror image (pack batch k, then
// its DMA to DRAM while batch k+1 is packed).  Host code only: the kernels
// are the library's copy kernels; streams and events are the caller's.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "cascade.h"
#include "copy_range.h"

namespace {

bool args_ok(const cascade_kv_pool_t *pool, const void *staging, const void *host,
             const int64_t *host_offsets, const cascade_move_t *moves_dev,
             const int32_t *n_dev, int32_t n_moves, int32_t batch, void *const *events,
             int32_t n_events) {
  if (!pool || !staging || !moves_dev || !n_dev || n_moves < 0 || batch < 1) return false;
  if (n_moves > 0 && (!host || !host_offsets || !events || n_events < 1)) return false;
  for (int32_t e = 0; e < n_events && n_moves > 0; ++e)
    if (!events[e]) return false;
  return pool->num_layers >= 1 && pool->chunk_bytes >= 16;
}

// DMA of moves [m0, m1): staging slot m <-> host bytes at host_offsets[m];
// moves whose slots and host blocks are both consecutive go as one copy.
hipError_t dma_range(char *staging, char *host, const int64_t *host_offsets, int64_t block,
                     int32_t m0, int32_t m1, bool to_device, hipStream_t s) {
  int32_t m = m0;
  while (m < m1) {
    int32_t e = m + 1;
    while (e < m1 && host_offsets[e] == host_offsets[e - 1] + block) ++e;
    char *dev = staging + (int64_t)m * block;
    char *hst = host + host_offsets[m];
    const size_t bytes = (size_t)(e - m) * (size_t)block;
    const hipError_t err = to_device ? hipMemcpyAsync(dev, hst, bytes, hipMemcpyHostToDevice, s)
                                     : hipMemcpyAsync(hst, dev, bytes, hipMemcpyDeviceToHost, s);
    if (err != hipSuccess) return err;
    m = e;
  }
  return hipSuccess;
}

}  // namespace

extern "C" int cascade_restore_from_host(const cascade_kv_pool_t *pool, void *staging,
                                         int32_t staging_slots, const void *host_blocks,
                                         const int64_t *host_offsets,
                                         const cascade_move_t *moves_dev,
                                         const int32_t *n_moves_dev, int32_t n_moves,
                                         int32_t batch_moves, int32_t *status_dev,
                                         void *copy_stream, void *compute_stream,
                                         void *const *events, int32_t n_events) {
  if (!args_ok(pool, staging, host_blocks, host_offsets, moves_dev, n_moves_dev, n_moves,
               batch_moves, events, n_events))
    return CASCADE_EINVAL;
  if (n_moves > staging_slots) return CASCADE_ENOSPC;
  const int64_t block = 2 * (int64_t)pool->num_layers * pool->chunk_bytes;
  hipStream_t cs = static_cast<hipStream_t>(copy_stream);
  hipStream_t ks = static_cast<hipStream_t>(compute_stream);
  if (n_moves == 0) return CASCADE_OK;
  // the host-to-staging copies start after everything enqueued so far on
  // the compute stream (the step that wrote the move list, earlier use of
  // the staging buffer)
  {
    hipEvent_t ev = static_cast<hipEvent_t>(events[0]);
    if (hipEventRecord(ev, ks) != hipSuccess || hipStreamWaitEvent(cs, ev, 0) != hipSuccess)
      return CASCADE_EHIP;
  }
  for (int32_t k = 0, m0 = 0; m0 < n_moves; ++k, m0 += batch_moves) {
    const int32_t m1 = std::min(n_moves, m0 + batch_moves);
    hipEvent_t ev = static_cast<hipEvent_t>(events[k % n_events]);
    if (dma_range(static_cast<char *>(staging), const_cast<char *>(static_cast<const char *>(host_blocks)),
                  host_offsets, block, m0, m1, true, cs) != hipSuccess ||
        hipEventRecord(ev, cs) != hipSuccess || hipStreamWaitEvent(ks, ev, 0) != hipSuccess)
      return CASCADE_EHIP;
    // moves [m0, m1) of the list, as far as the device count reaches
    const int rc = cascade::copy_range(false, pool, staging, staging_slots, moves_dev,
                                       n_moves_dev, m0, m1 - m0, status_dev, ks);
    if (rc != CASCADE_OK) return rc;
  }
  return CASCADE_OK;
}

extern "C" int cascade_spill_to_host(const cascade_kv_pool_t *pool, void *staging,
                                     int32_t staging_slots, void *host_blocks,
                                     const int64_t *host_offsets, const cascade_move_t *moves_dev,
                                     const int32_t *n_moves_dev, int32_t n_moves,
                                     int32_t batch_moves, int32_t *status_dev, void *copy_stream,
                                     void *compute_stream, void *const *events,
                                     int32_t n_events) {
  if (!args_ok(pool, staging, host_blocks, host_offsets, moves_dev, n_moves_dev, n_moves,
               batch_moves, events, n_events))
    return CASCADE_EINVAL;
  if (n_moves > staging_slots) return CASCADE_ENOSPC;
  const int64_t block = 2 * (int64_t)pool->num_layers * pool->chunk_bytes;
  hipStream_t cs = static_cast<hipStream_t>(copy_stream);
  hipStream_t ks = static_cast<hipStream_t>(compute_stream);
  for (int32_t k = 0, m0 = 0; m0 < n_moves; ++k, m0 += batch_moves) {
    const int32_t m1 = std::min(n_moves, m0 + batch_moves);
    hipEvent_t ev = static_cast<hipEvent_t>(events[k % n_events]);
    const int rc = cascade::copy_range(true, pool, staging, staging_slots, moves_dev,
                                       n_moves_dev, m0, m1 - m0, status_dev, ks);
    if (rc != CASCADE_OK) return rc;
    if (hipEventRecord(ev, ks) != hipSuccess || hipStreamWaitEvent(cs, ev, 0) != hipSuccess ||
        dma_range(static_cast<char *>(staging), static_cast<char *>(host_blocks), host_offsets,
                  block, m0, m1, false, cs) != hipSuccess)
      return CASCADE_EHIP;
  }
  return CASCADE_OK;
}
