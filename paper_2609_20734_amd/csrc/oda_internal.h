// Internal helpers shared by the library's translation units (host side).
#ifndef ODA_INTERNAL_H_
#define ODA_INTERNAL_H_

#include <stdint.h>

#include "oda.h"

namespace oda {

// Record a formatted detail for oda_last_error() and return `s`.
oda_status fail(oda_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
// Clear the thread-local detail and return ODA_OK.
oda_status ok();

inline bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int64_t round_up(int64_t a, int64_t b) { return ceil_div(a, b) * b; }

// Direct-ring Local geometry for sinks n_sink >= 0 and window >= 1: the sink
// blocks (ceil(n_sink / 16)) and the ring blocks (ceil(window / 16) + 2) of
// each (layer, request, KV head) unit.
struct RingGeometry {
  int32_t sink_blocks, ring_blocks;
};
inline RingGeometry ring_geometry(int32_t n_sink, int32_t window) {
  return RingGeometry{(int32_t)ceil_div(n_sink, 16), (int32_t)ceil_div(window, 16) + 2};
}

}  // namespace oda

#endif  // ODA_INTERNAL_H_
