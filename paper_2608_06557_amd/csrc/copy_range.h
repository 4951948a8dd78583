// copy_range.h -- library-internal launcher of the KV copy kernel over a
// slice of a device move list (not part of the C ABI).
#pragma once
#include <stdint.h>

#include "cascade.h"

namespace cascade {
// Copies moves [first, first + max_moves) of a list whose length is
// *n_moves_dev, i.e. min(*n_moves_dev - first, max_moves) moves starting at
// moves + first (none when the device count ends before `first`).
// to_staging: pool -> staging (pack), else staging -> pool (unpack).
int copy_range(bool to_staging, const cascade_kv_pool_t *pool, const void *staging,
               int32_t staging_slots, const cascade_move_t *moves, const int32_t *n_moves_dev,
               int32_t first, int32_t max_moves, int32_t *status_dev, void *stream);
}  // namespace cascade
