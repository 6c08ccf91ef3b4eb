// The decoder around the hot path: the backbone f_theta whose attention the
// Local and Full branches restrict (§2.1), as a pre-norm decoder stack with
// bf16 weights and fp32 activations, so that a whole ODA decode step (Alg. 1:
// Local forward, recall head, conditional Full forward, commit, output
// projection) can be timed against the additive cost model of App. A.6.
//
//   oda_dense_bf16    y = W . RMSNorm(x) (optional), + residual (optional), or
//                     the SwiGLU pair SiLU(W_g . x') * (W_u . x')
//   oda_qk_norm_rope  per-head RMSNorm of q and k, rotary embedding at each
//                     request's current position, bf16 q / K / V candidates
//   oda_embed_bf16    embedding rows of the step's tokens
//   oda_copy_rows     rows of the selected requests from one buffer to another
//   oda_rms_norm_rows RMSNorm (with gain) of the selected requests' rows: the
//                     final normalised hidden state the recall head reads
//   oda_argmax        greedy token of each request's logits
//
// Every kernel can be restricted to a device-side list of requests (the
// recall gate's compacted list), so the Full retry touches only flagged
// requests.  All of them are bound by HBM (bf16 weight streaming for the
// dense layers at small batch), not by arithmetic.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <climits>
#include <cmath>

#include "oda.h"
#include "oda_device.h"
#include "oda_internal.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;
constexpr int kTile = 8;   // most requests per wavefront in a dense layer

constexpr int kDenseMinWaves = 2048;   // grouping rows stops short of fewer wavefronts than this

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ uint16_t to_bf16(float f) { return oda::bf16_rne(f); }
__device__ __forceinline__ float silu(float x) { return x / (1.f + __expf(-x)); }
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) x += __shfl_xor(x, s);
  return x;
}
__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

// Requests a launch covers: the listed ones, else all B.
__device__ __forceinline__ int selected_count(const int32_t* n_work, int B) {
  return n_work ? min(max(n_work[0], 0), B) : B;
}
__device__ __forceinline__ int selected_request(const int32_t* work_list, int slot) {
  return work_list ? work_list[slot] : slot;
}

// ---------------------------------------------------------------------------
// dense layer
// ---------------------------------------------------------------------------

struct DenseArgs {
  const uint16_t* W;       // [N][K] bf16 (SwiGLU: [2N][K], gate rows then up rows)
  const float* gain;       // [K] RMSNorm gain of the input, or NULL (no norm)
  const float* x;          // [B][K]
  const float* residual;   // [B][N] or NULL
  float* y;                // [B][N] (may be the residual buffer)
  const int32_t* work_list;
  const int32_t* n_work;
  int N, K, B;
  float eps;
};

// One wavefront per (group of R output rows, tile of up to T selected
// requests).  Lanes take 8 consecutive weights of each row (one 16-byte load
// per row), so a wavefront reads R KiB per 512-element chunk, several chunks
// in flight; every input load serves all R rows.  The inputs come from cache.
// The input's sum of squares (for RMSNorm) accumulates in the same pass.
// Small T keeps registers for loads in flight; R > 1 makes the wavefronts of
// a layer with many short rows fewer and longer.
template <bool kSwiGLU, int T, int R>
__global__ __launch_bounds__(256) void dense_kernel(DenseArgs p) {
  constexpr int kAcc = R * T;
  static_assert(kAcc <= 64, "one result per lane");
  const int lane = threadIdx.x & 63;
  const int wave = uniform(threadIdx.x >> 6);
  const int item = blockIdx.x * kWaves + wave;
  const int groups = p.N / R;                  // the host keeps N a multiple of R
  const int row0 = (item % groups) * R;
  const int s0 = (item / groups) * T;
  const int count = selected_count(p.n_work, p.B);
  if (s0 >= count) return;
  const int nb = min(T, count - s0);
  // a listed request outside [0, B) is computed as request 0 and not stored
  const int listed = lane < nb ? selected_request(p.work_list, s0 + lane) : 0;
  const bool my_ok = listed >= 0 && listed < p.B;
  const int my_req = my_ok ? listed : 0;
  int req[T];
#pragma unroll
  for (int bi = 0; bi < T; ++bi) req[bi] = __shfl(my_req, bi);
  const bool norm = p.gain != nullptr;

  const uint16_t* wrow = p.W + (int64_t)row0 * p.K;
  const uint16_t* wrow2 = kSwiGLU ? p.W + (int64_t)(p.N + row0) * p.K : nullptr;
  float acc[R][T], acc2[kSwiGLU ? R : 1][T], ss[T];
#pragma unroll
  for (int bi = 0; bi < T; ++bi) {
    ss[bi] = 0.f;
#pragma unroll
    for (int j = 0; j < R; ++j) {
      acc[j][bi] = 0.f;
      if (kSwiGLU) acc2[j][bi] = 0.f;
    }
  }
  // 512-element chunks (8 per lane).  In a ragged last chunk the lanes past K
  // read element 0 again and weigh it by zero, so every load is unconditional
  // and the loads of successive chunks overlap.
  const int nchunks = (p.K + 511) / 512;
  // about eight 16-byte weight loads in flight per lane; sixteen for the
  // SwiGLU pair of a single request (few registers per load there, and the
  // pair is the decoder's largest layer)
  constexpr int kRowsPerChunk = kSwiGLU ? 2 * R : R;
  constexpr int kInFlight = kSwiGLU && T == 1 ? 16 : 8;
  constexpr int kUnroll = kRowsPerChunk >= kInFlight ? 1 : kInFlight / kRowsPerChunk;
#pragma unroll kUnroll
  for (int c = 0; c < nchunks; ++c) {
    const int k0 = c * 512 + 8 * lane;
    const bool in = k0 < p.K;
    const int k = in ? k0 : 0;
    const float mask = in ? 1.f : 0.f;
    u32x4 w[R], w2[kSwiGLU ? R : 1];
#pragma unroll
    for (int j = 0; j < R; ++j) {
      w[j] = *reinterpret_cast<const u32x4*>(wrow + (int64_t)j * p.K + k);
      if (kSwiGLU) w2[j] = *reinterpret_cast<const u32x4*>(wrow2 + (int64_t)j * p.K + k);
    }
    float g[8];
    if (norm) {
      const float4 g0 = *reinterpret_cast<const float4*>(p.gain + k);
      const float4 g1 = *reinterpret_cast<const float4*>(p.gain + k + 4);
      g[0] = g0.x; g[1] = g0.y; g[2] = g0.z; g[3] = g0.w;
      g[4] = g1.x; g[5] = g1.y; g[6] = g1.z; g[7] = g1.w;
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) g[e] = 1.f;
    }
#pragma unroll
    for (int bi = 0; bi < T; ++bi) {
      if (bi < nb) {
        const float* xr = p.x + (int64_t)req[bi] * p.K + k;
        const float4 x0 = *reinterpret_cast<const float4*>(xr);
        const float4 x1 = *reinterpret_cast<const float4*>(xr + 4);
        const float xv[8] = {x0.x * mask, x0.y * mask, x0.z * mask, x0.w * mask,
                             x1.x * mask, x1.y * mask, x1.z * mask, x1.w * mask};
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          if (norm) ss[bi] += xv[e] * xv[e];
          const float xg = xv[e] * g[e];
#pragma unroll
          for (int j = 0; j < R; ++j) {
            const uint32_t we = w[j][e >> 1];
            acc[j][bi] += ((e & 1) ? bf16_hi(we) : bf16_lo(we)) * xg;
            if (kSwiGLU) {
              const uint32_t we2 = w2[j][e >> 1];
              acc2[j][bi] += ((e & 1) ? bf16_hi(we2) : bf16_lo(we2)) * xg;
            }
          }
        }
      }
    }
  }

  // reduce over the wavefront; lane j * T + bi keeps row row0 + j, request bi
  float v = 0.f, v2 = 0.f, my_ss = 0.f;
#pragma unroll
  for (int bi = 0; bi < T; ++bi) {
    if (bi < nb) {
      const float s = norm ? wave_sum(ss[bi]) : 0.f;
#pragma unroll
      for (int j = 0; j < R; ++j) {
        const float a = wave_sum(acc[j][bi]);
        const float a2 = kSwiGLU ? wave_sum(acc2[j][bi]) : 0.f;
        if (lane == j * T + bi) {
          v = a;
          v2 = a2;
          my_ss = s;
        }
      }
    }
  }
  const int j = lane / T, bi = lane % T;
  const bool ok = __shfl(my_ok ? 1 : 0, bi) != 0;
  if (lane >= kAcc || bi >= nb || !ok) return;
  const int b = selected_request(p.work_list, s0 + bi);   // in [0, B): checked above
  const int row = row0 + j;
  const float inv = norm ? rsqrtf(my_ss / (float)p.K + p.eps) : 1.f;
  float out;
  if (kSwiGLU) {
    out = silu(v * inv) * (v2 * inv);
  } else {
    out = v * inv;
    if (p.residual) out += p.residual[(int64_t)b * p.N + row];
  }
  p.y[(int64_t)b * p.N + row] = out;
}

// ---------------------------------------------------------------------------
// per-head RMSNorm + rotary embedding, bf16 candidates
// ---------------------------------------------------------------------------

struct RopeArgs {
  const float* qkv;        // [B][(Hq + 2 Hkv) D]: q heads, then k heads, then v heads
  const float* q_gain;     // [D] or NULL
  const float* k_gain;     // [D] or NULL
  const int32_t* seq_lens; // position of the current token = seq_lens[b] - 1
  uint16_t* q_out;         // [B][Hq][D]
  uint16_t* k_out;         // [B][Hkv][D]
  uint16_t* v_out;         // [B][Hkv][D]
  const int32_t* work_list;
  const int32_t* n_work;
  double theta;
  float eps;
  int B, Hq, Hkv, D, heads_per_group;
};

// One wavefront per (selected request, head); q and k heads go through
// oda::norm_rope_pair (the same code the fused attention calls run), v heads
// are only rounded.
__global__ __launch_bounds__(256) void qk_norm_rope_kernel(RopeArgs p) {
  const int lane = threadIdx.x & 63;
  const int wave = uniform(threadIdx.x >> 6);
  const int heads = p.Hq + 2 * p.Hkv;
  const int slot = blockIdx.x / p.heads_per_group;
  const int h = (blockIdx.x % p.heads_per_group) * kWaves + wave;
  if (slot >= selected_count(p.n_work, p.B) || h >= heads) return;
  const int b = selected_request(p.work_list, slot);
  if (b < 0 || b >= p.B) return;   // a listed request outside the batch is skipped
  const int half = p.D / 2;
  const bool active = lane < half;   // lane i holds the pair (i, i + D/2)
  const float* src = p.qkv + ((int64_t)b * heads + h) * p.D;
  float x1 = active ? src[lane] : 0.f, x2 = active ? src[lane + half] : 0.f;
  uint16_t* dst;
  if (h < p.Hq + p.Hkv) {
    const bool is_q = h < p.Hq;
    oda::norm_rope_pair(x1, x2, active, lane, p.D, is_q ? p.q_gain : p.k_gain, p.eps,
                        (double)(p.seq_lens[b] - 1), p.theta);
    if (!active) return;
    dst = is_q ? p.q_out + ((int64_t)b * p.Hq + h) * p.D : p.k_out + ((int64_t)b * p.Hkv + (h - p.Hq)) * p.D;
  } else {
    if (!active) return;
    dst = p.v_out + ((int64_t)b * p.Hkv + (h - p.Hq - p.Hkv)) * p.D;
  }
  dst[lane] = to_bf16(x1);
  dst[lane + half] = to_bf16(x2);
}

// ---------------------------------------------------------------------------
// embedding, row copy, argmax
// ---------------------------------------------------------------------------

// One workgroup per request; a token outside [0, vocab) gives a NaN row.
__global__ __launch_bounds__(256) void embed_kernel(const uint16_t* table, int vocab, int d, const int32_t* tokens,
                                                   float* x) {
  const int b = blockIdx.x;
  const int t = tokens[b];
  float* dst = x + (int64_t)b * d;
  const bool ok = t >= 0 && t < vocab;
  for (int k = threadIdx.x * 8; k < d; k += 256 * 8) {
    if (ok) {
      const u32x4 w = *reinterpret_cast<const u32x4*>(table + (int64_t)t * d + k);
      *reinterpret_cast<float4*>(dst + k) = make_float4(bf16_lo(w[0]), bf16_hi(w[0]), bf16_lo(w[1]), bf16_hi(w[1]));
      *reinterpret_cast<float4*>(dst + k + 4) =
          make_float4(bf16_lo(w[2]), bf16_hi(w[2]), bf16_lo(w[3]), bf16_hi(w[3]));
    } else {
      const float nan = __builtin_nanf("");
      *reinterpret_cast<float4*>(dst + k) = make_float4(nan, nan, nan, nan);
      *reinterpret_cast<float4*>(dst + k + 4) = make_float4(nan, nan, nan, nan);
    }
  }
}

// One workgroup per selected request slot.
__global__ __launch_bounds__(256) void copy_rows_kernel(const float* src, float* dst, int row_len, int B,
                                                       const int32_t* work_list, const int32_t* n_work) {
  const int slot = blockIdx.x;
  if (slot >= selected_count(n_work, B)) return;
  const int b = selected_request(work_list, slot);
  if (b < 0 || b >= B) return;   // a listed request outside the batch is skipped
  const int64_t base = (int64_t)b * row_len;
  for (int k = threadIdx.x * 4; k < row_len; k += 256 * 4)
    *reinterpret_cast<float4*>(dst + base + k) = *reinterpret_cast<const float4*>(src + base + k);
}

// One workgroup per selected request slot: y = x / sqrt(mean(x^2) + eps) * gain.
// The sum of squares is reduced in a fixed order (lanes, then wavefronts), so
// the result is the same on every run.
__global__ __launch_bounds__(256) void rms_norm_rows_kernel(const float* x, const float* gain, float eps, float* y,
                                                           int row_len, int B, const int32_t* work_list,
                                                           const int32_t* n_work) {
  __shared__ float sred[4];
  const int slot = blockIdx.x;
  if (slot >= selected_count(n_work, B)) return;
  const int b = selected_request(work_list, slot);
  if (b < 0 || b >= B) return;   // a listed request outside the batch is skipped
  const int64_t base = (int64_t)b * row_len;
  float ss = 0.f;
  for (int k = threadIdx.x * 4; k < row_len; k += 256 * 4) {
    const float4 v = *reinterpret_cast<const float4*>(x + base + k);
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) ss += __shfl_xor(ss, s);
  if ((threadIdx.x & 63) == 0) sred[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float inv = rsqrtf((sred[0] + sred[1] + sred[2] + sred[3]) / (float)row_len + eps);
  for (int k = threadIdx.x * 4; k < row_len; k += 256 * 4) {
    const float4 v = *reinterpret_cast<const float4*>(x + base + k);
    const float4 g = *reinterpret_cast<const float4*>(gain + k);
    *reinterpret_cast<float4*>(y + base + k) = make_float4(v.x * inv * g.x, v.y * inv * g.y, v.z * inv * g.z,
                                                           v.w * inv * g.w);
  }
}

constexpr int kArgThreads = 1024;

// Greedy choice: the first index of the largest non-NaN value (-1 if every
// value is NaN).  One workgroup per request, eight 16-byte loads in flight
// per thread.
__global__ __launch_bounds__(kArgThreads) void argmax_kernel(const float* x, int n, int32_t* index) {
  __shared__ float sv[kArgThreads / 64];
  __shared__ int si[kArgThreads / 64];
  const int b = blockIdx.x;
  const float* row = x + (int64_t)b * n;
  float best = -INFINITY;
  int bidx = INT_MAX;
  auto take = [&](float v, int i) {
    if (v > best || (v == best && i < bidx)) {
      best = v;
      bidx = i;
    }
  };
  const int n4 = n / 4;
  for (int j0 = threadIdx.x; j0 < n4; j0 += kArgThreads * 8) {
    float4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int j = j0 + u * kArgThreads;
      v[u] = j < n4 ? *reinterpret_cast<const float4*>(row + 4 * (int64_t)j)
                    : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int j = j0 + u * kArgThreads;
      if (j < n4) {
        take(v[u].x, 4 * j);
        take(v[u].y, 4 * j + 1);
        take(v[u].z, 4 * j + 2);
        take(v[u].w, 4 * j + 3);
      }
    }
  }
  for (int i = 4 * n4 + threadIdx.x; i < n; i += kArgThreads) take(row[i], i);
  // wavefront, then workgroup
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) {
    const float ov = __shfl_xor(best, s);
    const int oi = __shfl_xor(bidx, s);
    take(ov, oi);
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) {
    sv[wave] = best;
    si[wave] = bidx;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < kArgThreads / 64; ++w) take(sv[w], si[w]);
    index[b] = bidx == INT_MAX ? -1 : bidx;
  }
}

oda_status launch_status() {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return oda::fail(ODA_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return oda::ok();
}

}  // namespace

extern "C" oda_status oda_dense_bf16(const oda_dense_desc* desc, int32_t batch, const float* x,
                                    const float* residual, float* y, const int32_t* work_list,
                                    const int32_t* n_work, hipStream_t stream) {
  if (desc == nullptr) return oda::fail(ODA_ERR_NULL, "desc is NULL");
  if (!desc->weight || !x || !y) return oda::fail(ODA_ERR_NULL, "weight, x and y are required");
  if ((work_list == nullptr) != (n_work == nullptr))
    return oda::fail(ODA_ERR_NULL, "work_list and n_work must both be NULL or both be set");
  if (desc->mode != ODA_DENSE_PLAIN && desc->mode != ODA_DENSE_SWIGLU)
    return oda::fail(ODA_ERR_UNSUPPORTED, "unknown dense mode %d", desc->mode);
  if (batch < 1 || desc->in_features < 8 || desc->in_features % 8 || desc->out_features < 1)
    return oda::fail(ODA_ERR_SHAPE, "batch >= 1, in_features a positive multiple of 8, out_features >= 1 required "
                     "(got %d, %d, %d)", batch, desc->in_features, desc->out_features);
  if (desc->mode == ODA_DENSE_SWIGLU && residual != nullptr)
    return oda::fail(ODA_ERR_UNSUPPORTED, "the SwiGLU mode takes no residual");
  if (!(desc->rms_eps >= 0.f) || !std::isfinite(desc->rms_eps)) return oda::fail(ODA_ERR_SHAPE, "rms_eps must be >= 0");
  if (!oda::aligned(desc->weight, 16) || !oda::aligned(x, 16) || (desc->norm_gain && !oda::aligned(desc->norm_gain, 16)))
    return oda::fail(ODA_ERR_SHAPE, "weight, x and norm_gain must be 16-byte aligned");
  // requests per wavefront: one, up to four, or up to eight; then the most
  // rows per wavefront that still leave >= kDenseMinWaves wavefronts
  const int tile = batch == 1 ? 1 : batch <= 4 ? 4 : kTile;
  const int64_t tiles = oda::ceil_div(batch, tile);
  const int N = desc->out_features;
  const bool swiglu = desc->mode == ODA_DENSE_SWIGLU;
  const int rmax = swiglu ? (tile == 1 ? 4 : 2) : (tile == 1 ? 8 : tile == 4 ? 4 : 2);
  int rows = 1;
  for (int r = rmax; r > 1; r /= 2)
    if (N % r == 0 && (int64_t)(N / r) * tiles >= kDenseMinWaves) {
      rows = r;
      break;
    }
  const int64_t groups = oda::ceil_div((int64_t)(N / rows) * tiles, kWaves);
  if (groups > INT_MAX) return oda::fail(ODA_ERR_SHAPE, "layer too large");
  DenseArgs a{desc->weight, desc->norm_gain, x, residual, y, work_list, n_work, N, desc->in_features, batch,
              desc->rms_eps};
  const dim3 grid((unsigned)groups), block(256);
  (void)hipGetLastError();
#define ODA_DENSE_LAUNCH(SW, T, R) hipLaunchKernelGGL((dense_kernel<SW, T, R>), grid, block, 0, stream, a)
  if (swiglu) {
    if (tile == 1) {
      if (rows == 4) ODA_DENSE_LAUNCH(true, 1, 4);
      else if (rows == 2) ODA_DENSE_LAUNCH(true, 1, 2);
      else ODA_DENSE_LAUNCH(true, 1, 1);
    } else if (tile == 4) {
      if (rows == 2) ODA_DENSE_LAUNCH(true, 4, 2);
      else ODA_DENSE_LAUNCH(true, 4, 1);
    } else {
      if (rows == 2) ODA_DENSE_LAUNCH(true, kTile, 2);
      else ODA_DENSE_LAUNCH(true, kTile, 1);
    }
  } else {
    if (tile == 1) {
      if (rows == 8) ODA_DENSE_LAUNCH(false, 1, 8);
      else if (rows == 4) ODA_DENSE_LAUNCH(false, 1, 4);
      else if (rows == 2) ODA_DENSE_LAUNCH(false, 1, 2);
      else ODA_DENSE_LAUNCH(false, 1, 1);
    } else if (tile == 4) {
      if (rows == 4) ODA_DENSE_LAUNCH(false, 4, 4);
      else if (rows == 2) ODA_DENSE_LAUNCH(false, 4, 2);
      else ODA_DENSE_LAUNCH(false, 4, 1);
    } else {
      if (rows == 2) ODA_DENSE_LAUNCH(false, kTile, 2);
      else ODA_DENSE_LAUNCH(false, kTile, 1);
    }
  }
#undef ODA_DENSE_LAUNCH
  return launch_status();
}

extern "C" oda_status oda_qk_norm_rope(int32_t batch, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                      const float* qkv, const float* q_gain, const float* k_gain, float rms_eps,
                                      double rope_theta, const int32_t* seq_lens, uint16_t* q_out,
                                      uint16_t* k_out, uint16_t* v_out, const int32_t* work_list,
                                      const int32_t* n_work, hipStream_t stream) {
  if (!qkv || !seq_lens || !q_out || !k_out || !v_out)
    return oda::fail(ODA_ERR_NULL, "qkv, seq_lens, q_out, k_out and v_out are required");
  if ((work_list == nullptr) != (n_work == nullptr))
    return oda::fail(ODA_ERR_NULL, "work_list and n_work must both be NULL or both be set");
  if (batch < 1 || num_kv_heads < 1 || num_q_heads < 1 || num_q_heads % num_kv_heads)
    return oda::fail(ODA_ERR_SHAPE, "batch >= 1 and num_q_heads a positive multiple of num_kv_heads required");
  if (head_dim < 2 || head_dim > 128 || head_dim % 2)
    return oda::fail(ODA_ERR_UNSUPPORTED, "head_dim must be even and at most 128 (got %d)", head_dim);
  if (!(rope_theta > 1.0) || !std::isfinite(rope_theta)) return oda::fail(ODA_ERR_SHAPE, "rope_theta must be > 1");
  if (!(rms_eps >= 0.f) || !std::isfinite(rms_eps)) return oda::fail(ODA_ERR_SHAPE, "rms_eps must be >= 0");
  RopeArgs a{};
  a.qkv = qkv;
  a.q_gain = q_gain;
  a.k_gain = k_gain;
  a.seq_lens = seq_lens;
  a.q_out = q_out;
  a.k_out = k_out;
  a.v_out = v_out;
  a.work_list = work_list;
  a.n_work = n_work;
  a.theta = rope_theta;
  a.eps = rms_eps;
  a.B = batch;
  a.Hq = num_q_heads;
  a.Hkv = num_kv_heads;
  a.D = head_dim;
  a.heads_per_group = (int)oda::ceil_div(num_q_heads + 2 * num_kv_heads, kWaves);
  (void)hipGetLastError();
  hipLaunchKernelGGL(qk_norm_rope_kernel, dim3((unsigned)(batch * a.heads_per_group)), dim3(256), 0, stream, a);
  return launch_status();
}

extern "C" oda_status oda_embed_bf16(const uint16_t* table, int32_t vocab, int32_t d_model, int32_t batch,
                                    const int32_t* tokens, float* x, hipStream_t stream) {
  if (!table || !tokens || !x) return oda::fail(ODA_ERR_NULL, "table, tokens and x are required");
  if (vocab < 1 || batch < 1 || d_model < 8 || d_model % 8)
    return oda::fail(ODA_ERR_SHAPE, "vocab, batch >= 1 and d_model a positive multiple of 8 required");
  if (!oda::aligned(table, 16) || !oda::aligned(x, 16))
    return oda::fail(ODA_ERR_SHAPE, "table and x must be 16-byte aligned");
  (void)hipGetLastError();
  hipLaunchKernelGGL(embed_kernel, dim3((unsigned)batch), dim3(256), 0, stream, table, vocab, d_model, tokens, x);
  return launch_status();
}

extern "C" oda_status oda_copy_rows(int32_t batch, int32_t row_len, const float* src, float* dst,
                                   const int32_t* work_list, const int32_t* n_work, hipStream_t stream) {
  if (!src || !dst) return oda::fail(ODA_ERR_NULL, "src and dst are required");
  if ((work_list == nullptr) != (n_work == nullptr))
    return oda::fail(ODA_ERR_NULL, "work_list and n_work must both be NULL or both be set");
  if (batch < 1 || row_len < 4 || row_len % 4)
    return oda::fail(ODA_ERR_SHAPE, "batch >= 1 and row_len a positive multiple of 4 required");
  if (!oda::aligned(src, 16) || !oda::aligned(dst, 16))
    return oda::fail(ODA_ERR_SHAPE, "src and dst must be 16-byte aligned");
  (void)hipGetLastError();
  hipLaunchKernelGGL(copy_rows_kernel, dim3((unsigned)batch), dim3(256), 0, stream, src, dst, row_len, batch,
                     work_list, n_work);
  return launch_status();
}

extern "C" oda_status oda_rms_norm_rows(int32_t batch, int32_t row_len, const float* x, const float* gain,
                                       float rms_eps, float* y, const int32_t* work_list, const int32_t* n_work,
                                       hipStream_t stream) {
  if (!x || !gain || !y) return oda::fail(ODA_ERR_NULL, "x, gain and y are required");
  if ((work_list == nullptr) != (n_work == nullptr))
    return oda::fail(ODA_ERR_NULL, "work_list and n_work must both be NULL or both be set");
  if (batch < 1 || row_len < 4 || row_len % 4)
    return oda::fail(ODA_ERR_SHAPE, "batch >= 1 and row_len a positive multiple of 4 required");
  if (!(rms_eps >= 0.f) || !std::isfinite(rms_eps)) return oda::fail(ODA_ERR_SHAPE, "rms_eps must be >= 0");
  if (!oda::aligned(x, 16) || !oda::aligned(gain, 16) || !oda::aligned(y, 16))
    return oda::fail(ODA_ERR_SHAPE, "x, gain and y must be 16-byte aligned");
  (void)hipGetLastError();
  hipLaunchKernelGGL(rms_norm_rows_kernel, dim3((unsigned)batch), dim3(256), 0, stream, x, gain, rms_eps, y, row_len,
                     batch, work_list, n_work);
  return launch_status();
}

extern "C" oda_status oda_argmax(int32_t batch, int32_t n, const float* x, int32_t* index, hipStream_t stream) {
  if (!x || !index) return oda::fail(ODA_ERR_NULL, "x and index are required");
  if (batch < 1 || n < 1) return oda::fail(ODA_ERR_SHAPE, "batch and n must be >= 1");
  if (!oda::aligned(x, 16) || n % 4) return oda::fail(ODA_ERR_SHAPE, "x must be 16-byte aligned and n a multiple of 4");
  (void)hipGetLastError();
  hipLaunchKernelGGL(argmax_kernel, dim3((unsigned)batch), dim3(kArgThreads), 0, stream, x, n, index);
  return launch_status();
}
