// Selected-state commit (App. A.5, commit equation, and its single fused
// cross-layer commit): the chosen branch's current-position K/V of every
// layer is appended to the paged cache and the request's length advances, in
// one launch.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "oda.h"
#include "oda_internal.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kBlock = 16;
constexpr int kThreads = 256;
constexpr int kTargetGroups = 256;   // workgroups the launch aims for (one per CU)

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
  uint32_t* tickets;         // [B] workgroups of the request done so far (zero between calls); NULL: no advance
  int64_t kv_layer_stride;   // elements between layers of the caches
  int64_t NB;                // physical blocks
  int32_t L, B, Hkv, D, MB;
  int32_t chunks;            // workgroups per request
  int32_t units_per_chunk;   // (layer, KV head) units per workgroup
  uint16_t* k_ring;          // NULL, or the direct-ring Local rings [L][B][sb + rb][Hkv][..] (cache block layouts)
  uint16_t* v_ring;
  int32_t ring_sb, ring_rb;  // sink blocks, ring blocks
};

// Workgroup (b, c) moves the selected candidates of units [c upw, (c+1) upw)
// of request b (unit = layer * Hkv + KV head) into position n - 1: K as one
// 16-byte store per 8 dims into the block's [D/8][16][8] layout, V as one
// 2-byte store per dim down the block's [D][16] columns (consecutive lanes
// on consecutive dims).  A request's cache stores are spread over several
// CUs: one workgroup per request issued every scattered store of all its
// layers from one CU and took ~25 us at batch one.
//
// The length advances once every workgroup of the request has read it: each
// takes a ticket after a workgroup barrier (all its threads have read n by
// then), counting modulo the number of workgroups, and the holder of the last
// ticket writes n + 1; the ticket word is back at 0 with no reset.  A length
// or block-table entry outside the cache writes nothing to the cache (the
// length still advances).
__global__ __launch_bounds__(kThreads) void commit_kernel(CommitArgs a) {
  const int b = blockIdx.x / a.chunks;
  const int c = blockIdx.x - b * a.chunks;
  const int n = a.seq_lens[b];
  const int pos = n - 1;
  const bool in_table = pos >= 0 && pos < a.MB * kBlock;
  const int64_t blk = in_table ? a.block_table[(int64_t)b * a.MB + pos / kBlock] : -1;
  const int units = a.L * a.Hkv;
  const int u0 = c * a.units_per_chunk;
  // uniform over the workgroup: a slot outside the cache is not written
  const int nu = (blk >= 0 && blk < a.NB) ? max(0, min(units - u0, a.units_per_chunk)) : 0;
  const bool full = a.flags != nullptr && a.flags[b] != 0;
  const uint16_t* ks = full ? a.k_full : a.k_local;
  const uint16_t* vs = full ? a.v_full : a.v_local;
  const int slot = pos & (kBlock - 1);
  const int groups = a.D / 8;
  // the ring block holding this position (direct-ring Local): its sink block,
  // or slot j mod rb of the ring
  const int j = pos / kBlock;
  const int nr = a.ring_sb + a.ring_rb;
  const int rj = j < a.ring_sb ? j : a.ring_sb + j % a.ring_rb;
  for (int i = threadIdx.x; i < nu * groups; i += kThreads) {
    const int u = u0 + i / groups, d8 = i % groups;
    const int l = u / a.Hkv, g = u - l * a.Hkv;
    const int64_t src = (((int64_t)l * a.B + b) * a.Hkv + g) * a.D + d8 * 8;
    const int64_t dst = (int64_t)l * a.kv_layer_stride + (blk * a.Hkv + g) * kBlock * a.D;
    const u32x4 k8 = *reinterpret_cast<const u32x4*>(ks + src);
    *reinterpret_cast<u32x4*>(a.k_cache + dst + ((int64_t)d8 * kBlock + slot) * 8) = k8;
    if (a.k_ring != nullptr) {
      const int64_t rdst = ((((int64_t)l * a.B + b) * nr + rj) * a.Hkv + g) * kBlock * a.D;
      *reinterpret_cast<u32x4*>(a.k_ring + rdst + ((int64_t)d8 * kBlock + slot) * 8) = k8;
    }
  }
  for (int i = threadIdx.x; i < nu * a.D; i += kThreads) {
    const int u = u0 + i / a.D, d = i % a.D;
    const int l = u / a.Hkv, g = u - l * a.Hkv;
    const int64_t src = (((int64_t)l * a.B + b) * a.Hkv + g) * a.D + d;
    const int64_t dst = (int64_t)l * a.kv_layer_stride + (blk * a.Hkv + g) * kBlock * a.D;
    const uint16_t v1 = vs[src];
    a.v_cache[dst + (int64_t)d * kBlock + slot] = v1;
    if (a.v_ring != nullptr) {
      const int64_t rdst = ((((int64_t)l * a.B + b) * nr + rj) * a.Hkv + g) * kBlock * a.D;
      a.v_ring[rdst + (int64_t)d * kBlock + slot] = v1;
    }
  }
  if (a.tickets == nullptr) return;
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t t =
        __builtin_amdgcn_atomic_inc32(a.tickets + b, (uint32_t)(a.chunks - 1), __ATOMIC_RELAXED, "agent");
    if (t == (uint32_t)(a.chunks - 1)) __hip_atomic_store(a.seq_lens + b, n + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

oda_status check_commit_shape(const oda_attn_shape* shape) {
  if (shape == nullptr) return oda::fail(ODA_ERR_NULL, "shape is NULL");
  if (shape->num_layers < 1 || shape->batch < 1 || shape->num_kv_heads < 1 || shape->num_blocks < 1 ||
      shape->max_blocks_per_seq < 1)
    return oda::fail(ODA_ERR_SHAPE, "num_layers, batch, num_kv_heads, num_blocks, max_blocks_per_seq must be >= 1");
  if (shape->head_dim != 64 && shape->head_dim != 128)
    return oda::fail(ODA_ERR_UNSUPPORTED, "head_dim %d not in {64, 128}", shape->head_dim);
  if (shape->block_size != kBlock) return oda::fail(ODA_ERR_UNSUPPORTED, "block_size %d != 16", shape->block_size);
  const int64_t dense = shape->num_blocks * shape->num_kv_heads * kBlock * shape->head_dim;
  if (shape->layer_stride_kv != 0 && (shape->layer_stride_kv < dense || shape->layer_stride_kv % 8 != 0))
    return oda::fail(ODA_ERR_SHAPE, "layer_stride_kv %lld: 0, or a multiple of 8 >= %lld",
                     (long long)shape->layer_stride_kv, (long long)dense);
  return ODA_OK;
}

size_t commit_ws_bytes(const oda_attn_shape* shape) { return (size_t)oda::round_up((int64_t)shape->batch * 4, 256); }

}  // namespace

extern "C" oda_status oda_commit_workspace_size(const oda_attn_shape* shape, size_t* bytes) {
  oda_status st = check_commit_shape(shape);
  if (st != ODA_OK) return st;
  if (bytes == nullptr) return oda::fail(ODA_ERR_NULL, "bytes is NULL");
  *bytes = commit_ws_bytes(shape);
  return oda::ok();
}

namespace {

oda_status run_commit(const oda_attn_shape* shape, uint16_t* k_cache, uint16_t* v_cache, const int32_t* block_table,
                      int32_t* seq_lens, const uint16_t* k_local, const uint16_t* v_local, const uint16_t* k_full,
                      const uint16_t* v_full, const int32_t* flags, int32_t advance, void* workspace,
                      size_t workspace_bytes, uint16_t* k_ring, uint16_t* v_ring, int32_t n_sink, int32_t window,
                      hipStream_t stream) {
  oda_status st = check_commit_shape(shape);
  if (st != ODA_OK) return st;
  if (!k_cache || !v_cache || !block_table || !seq_lens || !k_local || !v_local)
    return oda::fail(ODA_ERR_NULL, "k_cache, v_cache, block_table, seq_lens, k_local and v_local are required");
  if ((k_full == nullptr) != (v_full == nullptr))
    return oda::fail(ODA_ERR_NULL, "k_full and v_full must both be NULL or both be set");
  if (!oda::aligned(k_cache, 16) || !oda::aligned(v_cache, 16) || !oda::aligned(k_local, 16) ||
      !oda::aligned(v_local, 16) || (k_full && (!oda::aligned(k_full, 16) || !oda::aligned(v_full, 16))))
    return oda::fail(ODA_ERR_SHAPE, "caches and candidates must be 16-byte aligned");
  if (advance != 0) {
    const size_t need = commit_ws_bytes(shape);
    if (workspace == nullptr) return oda::fail(ODA_ERR_WORKSPACE, "workspace is NULL (%zu bytes needed)", need);
    if (workspace_bytes < need)
      return oda::fail(ODA_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", workspace_bytes, need);
    if (!oda::aligned(workspace, 256)) return oda::fail(ODA_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  }
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
  a.tickets = advance != 0 ? static_cast<uint32_t*>(workspace) : nullptr;
  a.kv_layer_stride = shape->layer_stride_kv != 0 ? shape->layer_stride_kv
                                                  : shape->num_blocks * shape->num_kv_heads * kBlock * shape->head_dim;
  a.L = shape->num_layers;
  a.B = shape->batch;
  a.Hkv = shape->num_kv_heads;
  a.D = shape->head_dim;
  a.MB = shape->max_blocks_per_seq;
  a.NB = shape->num_blocks;
  a.k_ring = k_ring;
  a.v_ring = v_ring;
  const oda::RingGeometry rg = oda::ring_geometry(n_sink, window);
  a.ring_sb = k_ring ? rg.sink_blocks : 0;
  a.ring_rb = k_ring ? rg.ring_blocks : 1;
  // enough workgroups per request that the launch covers the CUs, each with
  // at least one (layer, KV head) unit
  const int64_t units = (int64_t)a.L * a.Hkv;
  const int64_t want = std::min<int64_t>(units, oda::ceil_div(kTargetGroups, a.B));
  a.units_per_chunk = (int)oda::ceil_div(units, want);
  a.chunks = (int)oda::ceil_div(units, a.units_per_chunk);
  const int64_t groups = (int64_t)a.B * a.chunks;
  if (groups > 0x7fffffffLL || units * (a.D / 8) > 0x7fffffffLL) return oda::fail(ODA_ERR_SHAPE, "grid too large");
  (void)hipGetLastError();
  hipLaunchKernelGGL(commit_kernel, dim3((unsigned)groups), dim3(kThreads), 0, stream, a);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return oda::fail(ODA_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return oda::ok();
}

}  // namespace

extern "C" oda_status oda_commit_kv(const oda_attn_shape* shape, uint16_t* k_cache, uint16_t* v_cache,
                                   const int32_t* block_table, int32_t* seq_lens, const uint16_t* k_local,
                                   const uint16_t* v_local, const uint16_t* k_full, const uint16_t* v_full,
                                   const int32_t* flags, int32_t advance, void* workspace, size_t workspace_bytes,
                                   hipStream_t stream) {
  return run_commit(shape, k_cache, v_cache, block_table, seq_lens, k_local, v_local, k_full, v_full, flags, advance,
                    workspace, workspace_bytes, nullptr, nullptr, 0, 1, stream);
}

extern "C" oda_status oda_commit_kv_ring(const oda_attn_shape* shape, uint16_t* k_cache, uint16_t* v_cache,
                                        const int32_t* block_table, int32_t* seq_lens, const uint16_t* k_local,
                                        const uint16_t* v_local, const uint16_t* k_full, const uint16_t* v_full,
                                        const int32_t* flags, int32_t advance, void* workspace,
                                        size_t workspace_bytes, uint16_t* k_ring, uint16_t* v_ring, int32_t n_sink,
                                        int32_t window, hipStream_t stream) {
  if (!k_ring || !v_ring) return oda::fail(ODA_ERR_NULL, "k_ring and v_ring are required");
  if (!oda::aligned(k_ring, 16) || !oda::aligned(v_ring, 16))
    return oda::fail(ODA_ERR_SHAPE, "rings must be 16-byte aligned");
  if (n_sink < 0 || window < 1) return oda::fail(ODA_ERR_SHAPE, "n_sink >= 0 and window >= 1 required");
  return run_commit(shape, k_cache, v_cache, block_table, seq_lens, k_local, v_local, k_full, v_full, flags, advance,
                    workspace, workspace_bytes, k_ring, v_ring, n_sink, window, stream);
}
