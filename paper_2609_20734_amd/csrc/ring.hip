// Direct-ring Local workspace (App. A.5: the Local path reads a contiguous
// workspace of the sinks and the recent window instead of the paged cache).
// Per (layer, request, KV head) a ring of whole 16-position blocks, laid out
// like the cache's blocks: the sink blocks first, then RB ring blocks that
// hold logical block j in slot j mod RB.  oda_ring_fill copies the blocks a
// Local call can read out of the paged cache; the commit keeps the ring
// current (oda_commit_kv_ring) and oda_local_decode_attn_ring reads it.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "oda.h"
#include "oda_internal.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kBlock = 16;
constexpr int kThreads = 256;

struct FillArgs {
  const uint16_t* k_cache;
  const uint16_t* v_cache;
  const int32_t* block_table;
  const int32_t* seq_lens;
  uint16_t* k_ring;
  uint16_t* v_ring;
  int64_t kv_layer_stride;   // elements between layers of the caches
  int64_t NB;                // physical blocks per layer
  int32_t L, B, Hkv, D, MB, max_len;
  int32_t sb, rb;            // sink blocks, ring blocks
};

// Workgroup (layer l, request b, ring block r) copies the physical block of
// the logical block ring block r holds: block r itself for a sink block, else
// the latest block j <= (n - 1) / 16 with j >= sb and j mod rb = r - sb.  One
// block of every KV head is one contiguous run of Hkv * 16 * D elements in
// both the cache and the ring.  A ring block with no such logical block, a
// length outside [1, max_len] or a table entry outside the cache leaves the
// ring block as it is.
__global__ __launch_bounds__(kThreads) void ring_fill_kernel(FillArgs a) {
  const int nr = a.sb + a.rb;
  int64_t item = blockIdx.x;
  const int r = (int)(item % nr);
  item /= nr;
  const int b = (int)(item % a.B);
  const int l = (int)(item / a.B);
  const int n = a.seq_lens[b];
  if (n < 1 || n > a.max_len) return;
  const int jmax = (n - 1) / kBlock;
  int j;
  if (r < a.sb) {
    j = r;
    if (j > jmax) return;
  } else {
    const int k = r - a.sb;
    j = jmax - (((jmax - k) % a.rb) + a.rb) % a.rb;
    if (j < a.sb) return;
  }
  if (j >= a.MB) return;
  const int64_t pb = a.block_table[(int64_t)b * a.MB + j];
  if (pb < 0 || pb >= a.NB) return;
  const int64_t elems = (int64_t)a.Hkv * kBlock * a.D;
  const u32x4* ks = reinterpret_cast<const u32x4*>(a.k_cache + (int64_t)l * a.kv_layer_stride + pb * elems);
  const u32x4* vs = reinterpret_cast<const u32x4*>(a.v_cache + (int64_t)l * a.kv_layer_stride + pb * elems);
  u32x4* kd = reinterpret_cast<u32x4*>(a.k_ring + (((int64_t)l * a.B + b) * nr + r) * elems);
  u32x4* vd = reinterpret_cast<u32x4*>(a.v_ring + (((int64_t)l * a.B + b) * nr + r) * elems);
  for (int64_t i = threadIdx.x; i < elems / 8; i += kThreads) {
    kd[i] = ks[i];
    vd[i] = vs[i];
  }
}

}  // namespace

extern "C" oda_status oda_ring_fill(const oda_attn_shape* shape, const uint16_t* k_cache, const uint16_t* v_cache,
                                   const int32_t* block_table, const int32_t* seq_lens, int32_t n_sink,
                                   int32_t window, uint16_t* k_ring, uint16_t* v_ring, hipStream_t stream) {
  int64_t elements = 0;
  oda_status st = oda_ring_elements(shape, n_sink, window, &elements);   // validates shape, n_sink, window
  if (st != ODA_OK) return st;
  if (!k_cache || !v_cache || !block_table || !seq_lens || !k_ring || !v_ring)
    return oda::fail(ODA_ERR_NULL, "k_cache, v_cache, block_table, seq_lens, k_ring and v_ring are required");
  if (!oda::aligned(k_cache, 16) || !oda::aligned(v_cache, 16) || !oda::aligned(k_ring, 16) ||
      !oda::aligned(v_ring, 16))
    return oda::fail(ODA_ERR_SHAPE, "caches and rings must be 16-byte aligned");
  const oda::RingGeometry rg = oda::ring_geometry(n_sink, window);
  FillArgs a;
  a.k_cache = k_cache;
  a.v_cache = v_cache;
  a.block_table = block_table;
  a.seq_lens = seq_lens;
  a.k_ring = k_ring;
  a.v_ring = v_ring;
  a.kv_layer_stride = shape->layer_stride_kv != 0 ? shape->layer_stride_kv
                                                  : shape->num_blocks * shape->num_kv_heads * kBlock * shape->head_dim;
  a.NB = shape->num_blocks;
  a.L = shape->num_layers;
  a.B = shape->batch;
  a.Hkv = shape->num_kv_heads;
  a.D = shape->head_dim;
  a.MB = shape->max_blocks_per_seq;
  a.max_len = shape->max_seq_len;
  a.sb = rg.sink_blocks;
  a.rb = rg.ring_blocks;
  const int64_t groups = (int64_t)a.L * a.B * (a.sb + a.rb);
  if (groups > 0x7fffffffLL) return oda::fail(ODA_ERR_SHAPE, "grid too large");
  (void)hipGetLastError();
  hipLaunchKernelGGL(ring_fill_kernel, dim3((unsigned)groups), dim3(kThreads), 0, stream, a);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return oda::fail(ODA_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return oda::ok();
}
