// Selected-state commit (App. A.5, commit equation, and its single fused
// cross-layer commit): the chosen branch's current-position K/V of every
// layer is appended to the paged cache and the request's length advances, in
// one launch.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "oda.h"
#include "oda_internal.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kBlock = 16;
constexpr int kThreads = 1024;   // one workgroup per request
constexpr int kInFlight = 4;     // (unit, 8-dim group) items each thread loads before it stores

struct CommitArgs {
  uint16_t* k_cache;
  uint16_t* v_cache;
  const int32_t* block_table;
  int32_t* seq_lens;
  const uint16_t* k_local;
  const uint16_t* v_local;
  const uint16_t* k_full;
  const uint16_t* v_full;
  const int32_t* flags;
  int64_t kv_layer_stride;   // elements between layers of the caches
  int64_t NB;                // physical blocks
  int32_t L, B, Hkv, D, MB;
  int32_t advance;
};

// The whole commit of one request in one launch: workgroup b reads its
// length once, moves the selected candidate of every (layer, KV head) into
// position n - 1 -- an item is 8 dims of one unit: one 16-byte store into the
// K block's [D/8][16][8] layout and eight 2-byte stores down the V block's
// [D][16] columns -- and, after a workgroup barrier (every thread has read the
// length by then), advances the length.  A length or block-table entry
// outside the cache writes nothing to the cache (the length still advances).
__global__ __launch_bounds__(kThreads) void commit_kernel(CommitArgs a) {
  const int b = blockIdx.x;
  const int n = a.seq_lens[b];
  const int pos = n - 1;
  const bool in_table = pos >= 0 && pos < a.MB * kBlock;
  const int64_t blk = in_table ? a.block_table[(int64_t)b * a.MB + pos / kBlock] : -1;
  // uniform over the workgroup: a slot outside the cache is not written
  const int items = (blk >= 0 && blk < a.NB) ? a.L * a.Hkv * (a.D / 8) : 0;
  const bool full = a.flags != nullptr && a.flags[b] != 0;
  const uint16_t* ks = full ? a.k_full : a.k_local;
  const uint16_t* vs = full ? a.v_full : a.v_local;
  const int slot = pos % kBlock;
  const int groups = a.D / 8;
  for (int i0 = threadIdx.x; i0 < items; i0 += kInFlight * kThreads) {
    u32x4 kv[kInFlight], vv[kInFlight];
#pragma unroll
    for (int u = 0; u < kInFlight; ++u) {
      const int i = i0 + u * kThreads;
      if (i < items) {
        const int unit = i / groups, d8 = i - unit * groups;   // unit = l * Hkv + g
        const int l = unit / a.Hkv, g = unit - l * a.Hkv;
        const int64_t src = (((int64_t)l * a.B + b) * a.Hkv + g) * a.D + d8 * 8;
        kv[u] = *reinterpret_cast<const u32x4*>(ks + src);
        vv[u] = *reinterpret_cast<const u32x4*>(vs + src);
      }
    }
#pragma unroll
    for (int u = 0; u < kInFlight; ++u) {
      const int i = i0 + u * kThreads;
      if (i < items) {
        const int unit = i / groups, d8 = i - unit * groups;
        const int l = unit / a.Hkv, g = unit - l * a.Hkv;
        const int64_t dst = (int64_t)l * a.kv_layer_stride + (blk * a.Hkv + g) * kBlock * a.D;
        *reinterpret_cast<u32x4*>(a.k_cache + dst + ((int64_t)d8 * kBlock + slot) * 8) = kv[u];
        const uint32_t w[4] = {vv[u].x, vv[u].y, vv[u].z, vv[u].w};
#pragma unroll
        for (int e = 0; e < 8; ++e)
          a.v_cache[dst + (int64_t)(d8 * 8 + e) * kBlock + slot] = (uint16_t)(w[e >> 1] >> (16 * (e & 1)));
      }
    }
  }
  if (!a.advance) return;
  __syncthreads();
  if (threadIdx.x == 0) a.seq_lens[b] = n + 1;
}

}  // namespace

extern "C" oda_status oda_commit_kv(const oda_attn_shape* shape, uint16_t* k_cache, uint16_t* v_cache,
                                   const int32_t* block_table, int32_t* seq_lens, const uint16_t* k_local,
                                   const uint16_t* v_local, const uint16_t* k_full, const uint16_t* v_full,
                                   const int32_t* flags, int32_t advance, hipStream_t stream) {
  if (shape == nullptr) return oda::fail(ODA_ERR_NULL, "shape is NULL");
  if (!k_cache || !v_cache || !block_table || !seq_lens || !k_local || !v_local)
    return oda::fail(ODA_ERR_NULL, "k_cache, v_cache, block_table, seq_lens, k_local and v_local are required");
  if ((k_full == nullptr) != (v_full == nullptr))
    return oda::fail(ODA_ERR_NULL, "k_full and v_full must both be NULL or both be set");
  if (shape->num_layers < 1 || shape->batch < 1 || shape->num_kv_heads < 1 || shape->num_blocks < 1 ||
      shape->max_blocks_per_seq < 1)
    return oda::fail(ODA_ERR_SHAPE, "num_layers, batch, num_kv_heads, num_blocks, max_blocks_per_seq must be >= 1");
  if (shape->head_dim != 64 && shape->head_dim != 128)
    return oda::fail(ODA_ERR_UNSUPPORTED, "head_dim %d not in {64, 128}", shape->head_dim);
  if (shape->block_size != kBlock) return oda::fail(ODA_ERR_UNSUPPORTED, "block_size %d != 16", shape->block_size);
  if (!oda::aligned(k_cache, 16) || !oda::aligned(v_cache, 16) || !oda::aligned(k_local, 16) ||
      !oda::aligned(v_local, 16) || (k_full && (!oda::aligned(k_full, 16) || !oda::aligned(v_full, 16))))
    return oda::fail(ODA_ERR_SHAPE, "caches and candidates must be 16-byte aligned");
  CommitArgs a;
  a.k_cache = k_cache;
  a.v_cache = v_cache;
  a.block_table = block_table;
  a.seq_lens = seq_lens;
  a.k_local = k_local;
  a.v_local = v_local;
  a.k_full = k_full ? k_full : k_local;
  a.v_full = v_full ? v_full : v_local;
  a.flags = flags;
  a.kv_layer_stride = shape->num_blocks * shape->num_kv_heads * kBlock * shape->head_dim;
  a.L = shape->num_layers;
  a.B = shape->batch;
  a.Hkv = shape->num_kv_heads;
  a.D = shape->head_dim;
  a.MB = shape->max_blocks_per_seq;
  a.NB = shape->num_blocks;
  a.advance = advance != 0;
  (void)hipGetLastError();
  if ((int64_t)shape->num_layers * shape->num_kv_heads * (shape->head_dim / 8) > 0x7fffffffLL)
    return oda::fail(ODA_ERR_SHAPE, "too many (layer, KV head) units");
  hipLaunchKernelGGL(commit_kernel, dim3((unsigned)shape->batch), dim3(kThreads), 0, stream, a);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return oda::fail(ODA_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return oda::ok();
}
