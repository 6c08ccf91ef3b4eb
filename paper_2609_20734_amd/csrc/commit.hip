// Selected-state commit (App. A.5, commit equation): the chosen branch's
// current-position K/V of every layer is appended to the paged cache, then
// the request's length advances.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "oda.h"
#include "oda_internal.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kBlock = 16;
constexpr int kThreads = 64;   // one wavefront: D/8 <= 16 threads work

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

// One workgroup per (request, layer, KV head): thread t < D/8 moves dims
// 8t..8t+7 of K (one 16-byte store into the [D/8][16][8] block) and of V
// (eight 2-byte stores down the block's [D][16] column).  The lengths are
// advanced by a second launch, so every copy reads the step's length.
__global__ __launch_bounds__(kThreads) void commit_copy_kernel(CommitArgs a) {
  int64_t unit = blockIdx.x;
  const int g = (int)(unit % a.Hkv);
  unit /= a.Hkv;
  const int l = (int)(unit % a.L);
  const int b = (int)(unit / a.L);
  const int d8 = threadIdx.x;
  if (d8 >= a.D / 8) return;
  const int pos = a.seq_lens[b] - 1;
  // a length or block-table entry outside the cache writes nothing
  if (pos < 0 || pos >= a.MB * kBlock) return;
  const int64_t blk = a.block_table[(int64_t)b * a.MB + pos / kBlock];
  if (blk < 0 || blk >= a.NB) return;
  const bool full = a.flags != nullptr && a.flags[b] != 0;
  const uint16_t* ks = full ? a.k_full : a.k_local;
  const uint16_t* vs = full ? a.v_full : a.v_local;
  const int slot = pos % kBlock;
  const int64_t src = (((int64_t)l * a.B + b) * a.Hkv + g) * a.D + d8 * 8;
  const int64_t dst = (int64_t)l * a.kv_layer_stride + (blk * a.Hkv + g) * kBlock * a.D;
  const u32x4 kv = *reinterpret_cast<const u32x4*>(ks + src);
  const u32x4 vv = *reinterpret_cast<const u32x4*>(vs + src);
  *reinterpret_cast<u32x4*>(a.k_cache + dst + ((int64_t)d8 * kBlock + slot) * 8) = kv;
  const uint32_t w[4] = {vv.x, vv.y, vv.z, vv.w};
#pragma unroll
  for (int e = 0; e < 8; ++e)
    a.v_cache[dst + (int64_t)(d8 * 8 + e) * kBlock + slot] = (uint16_t)(w[e >> 1] >> (16 * (e & 1)));
}

__global__ __launch_bounds__(256) void commit_advance_kernel(int32_t* seq_lens, int B) {
  const int b = blockIdx.x * 256 + threadIdx.x;
  if (b < B) seq_lens[b] += 1;
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
  const int64_t units = (int64_t)shape->batch * shape->num_layers * shape->num_kv_heads;
  if (units > 0x7fffffffLL) return oda::fail(ODA_ERR_SHAPE, "grid too large");
  hipLaunchKernelGGL(commit_copy_kernel, dim3((unsigned)units), dim3(kThreads), 0, stream, a);
  if (a.advance)
    hipLaunchKernelGGL(commit_advance_kernel, dim3((unsigned)oda::ceil_div(shape->batch, 256)), dim3(256), 0, stream,
                       seq_lens, shape->batch);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return oda::fail(ODA_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return oda::ok();
}
