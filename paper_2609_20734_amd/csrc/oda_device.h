// Device helpers shared by the library's kernels (HIP translation units only).
#ifndef ODA_DEVICE_H_
#define ODA_DEVICE_H_

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

namespace oda {

// fp32 -> bf16, round to nearest, ties to even (NaN stays NaN, quietened).
__device__ __forceinline__ uint16_t bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  return (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

// Current-token preparation of one q or k head, one wavefront per head: lane
// i < D/2 holds the pair (x_i, x_{i+D/2}) that the rotation mixes
// (rotate-half convention).  Per-head RMSNorm with `gain` (skipped when NULL;
// every lane takes part in the sum, the inactive ones adding zeros, so it is
// whole for any D/2 up to 64), then the rotary embedding at position `pos`:
// dims i and i + D/2 turn by pos * theta^(-2i/D), the angle formed in double
// precision since positions reach 10^5-10^6.  Called by every lane of the
// wavefront (it holds a cross-lane sum).
__device__ __forceinline__ void norm_rope_pair(float& x1, float& x2, bool active, int lane, int D, const float* gain,
                                               float eps, double pos, double theta) {
  const int half = D / 2;
  if (gain != nullptr) {
    float ss = x1 * x1 + x2 * x2;
#pragma unroll
    for (int s = 32; s >= 1; s >>= 1) ss += __shfl_xor(ss, s);
    const float inv = rsqrtf(ss / (float)D + eps);
    if (active) {
      x1 = x1 * inv * gain[lane];
      x2 = x2 * inv * gain[lane + half];
    }
  }
  if (!active) return;
  const double ang = pos * pow(theta, -(double)(2 * lane) / (double)D);
  const float c = (float)cos(ang), s = (float)sin(ang);
  const float r1 = x1 * c - x2 * s;
  const float r2 = x2 * c + x1 * s;
  x1 = r1;
  x2 = r2;
}

}  // namespace oda

#endif  // ODA_DEVICE_H_
