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

}  // namespace oda

#endif  // ODA_INTERNAL_H_
