// Circular-buffer protocol of the warp-specialised kernel: which slot a
// K-iteration uses and which counter values its waits need.  Shared by the
// device kernels and by the host model of the protocol that the tests run
// under ThreadSanitizer.
//
// The buffer of the paper's Section 2.2 holds P tiles.  K-iterations are
// numbered q = 0, 1, ... over all output tiles a workgroup computes; q uses
// slot q mod P for the (q div P)-th time.  Each slot has two monotonic
// counters: full[s] counts producer-wave signals (one per producer wave per
// use) and empty[s] counts consumer-wave releases (one per consumer wave per
// use).  A producer of q waits until every consumer wave released the slot's
// previous use; a consumer of q waits until every producer wave filled this
// use.
#pragma once

#include <stdint.h>

#if defined(__HIPCC__)
#define WSG_RING_FN __host__ __device__ __forceinline__
#else
#define WSG_RING_FN inline
#endif

namespace wsg {

WSG_RING_FN constexpr uint32_t ring_slot(uint32_t q, uint32_t P) { return q % P; }
WSG_RING_FN constexpr uint32_t ring_use(uint32_t q, uint32_t P) { return q / P; }

// empty[ring_slot(q)] value at which the producers of q may overwrite the slot
// (0 for the first use: the slot starts free).
WSG_RING_FN constexpr uint32_t ring_empty_target(uint32_t q, uint32_t P, uint32_t consumers) {
  return (q / P) * consumers;
}

// full[ring_slot(q)] value at which the consumers of q may read the slot.
WSG_RING_FN constexpr uint32_t ring_full_target(uint32_t q, uint32_t P, uint32_t producers) {
  return (q / P + 1) * producers;
}

// The same walk without divisions: from (slot, full target) of q to those of
// q + 1.
WSG_RING_FN void ring_advance(uint32_t& slot, uint32_t& full_target, uint32_t P, uint32_t producers) {
  slot = (slot + 1 == P) ? 0u : slot + 1;
  if (slot == 0) full_target += producers;
}

}  // namespace wsg
