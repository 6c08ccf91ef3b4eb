// Decode attention over a paged bf16 KV cache for gfx950 (CDNA4):
// oda_local_decode_attn (Local access set) and oda_full_decode_attn (native
// access set, flagged requests only).  Both run the same kernels:
//
//   split  -- one workgroup of W wavefronts per work item (layer, request, KV
//             head, split).  Each wavefront streams a contiguous run of the
//             item's KV blocks, computes the G query heads' scores with
//             v_mfma_f32_16x16x32_bf16 (K tile x Q^T), keeps an online
//             softmax and accumulates P V with the same MFMA (P split into a
//             bf16 high and low part so the product keeps fp32 accuracy).
//             The wavefronts then combine their (m, l, o) through LDS.  If the
//             item covers the request's whole access set the workgroup writes
//             out / lse directly (adding the uncommitted current candidate);
//             otherwise it writes an unnormalised partial, takes a ticket,
//             and the workgroup holding the request's last ticket combines
//             the partials in split order with stable softmax rescaling (plus
//             the candidate) and writes out / lse: no second launch.
//   layers -- batched Local whose units all have one split: one workgroup per
//             (KV head, group of consecutive layers, request) streams the
//             group's layers in turn with the same per-unit body.
// This is the split-phase / combine-phase structure the paper's Local path
// uses (App. A.5), applied to both branches.
//
// Register layouts of one 16x16x32 MFMA (lane l, h = l % 16, j = l / 16):
//   A (16 x 32): row h, k = 8j..8j+7      B (32 x 16): column h, k = 8j..8j+7
//   C (16 x 16): column h, rows 4j..4j+3
// The cache layouts are chosen so every operand is one aligned global load:
//   K block [D/8][16][8]: 16 bytes at ((kk*4 + j)*16 + h)*8 is key h, dims
//     32kk + 8j .. +7  ->  the A operand of S^T = K Q^T (rows = positions);
//   V block [D][16]: 8 bytes at d*16 + 4j are positions 4j..4j+3 of dim d ->
//     two blocks give the B operand of O = P V (k = 8 positions, columns = dims),
//     matching the C layout of S^T (lane holds positions 4j..4j+3 of each tile).
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <atomic>
#include <cmath>

#include "oda.h"
#include "oda_device.h"
#include "oda_internal.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kBlock = 16;            // positions per KV block
constexpr int kMaxGroup = 16;         // query heads per KV head held by one MFMA tile
constexpr int kWaves = 8;             // wavefronts per split workgroup
constexpr int kTargetGroups = 256;    // workgroups a call aims for (one per CU)
constexpr int kBalanceBlocks = 512;   // shortest split the plan adds to even out the CUs
constexpr int kBalanceUnits = 64;     // units per request from which the plan evens out the CUs
constexpr int kMergeChunk = 16;       // split partials read per round trip in the merge
constexpr int kMergeSmall = 4;        // chunk used for the last few splits
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

enum Select { kSelAll = 0, kSelFlags = 1, kSelList = 2 };

struct AttnArgs {
  const uint16_t* q;
  const uint16_t* k_cache;
  const uint16_t* v_cache;
  const int32_t* block_table;
  const int32_t* seq_lens;
  const uint16_t* k_cur;
  const uint16_t* v_cur;
  const int32_t* flags;
  const int32_t* work_list;
  const int32_t* n_work;
  float* out;
  float* lse;
  float* part_o;     // [L][B][Hkv][max_splits][G][D]
  float* part_ml;    // [L][B][Hkv][max_splits][G][2]  (m in log2 units, l)
  uint32_t* tickets; // [L][B][Hkv] splits finished so far (zero between calls)
  int64_t kv_layer_stride;  // elements between layers of k_cache / v_cache
  int32_t L, B, Hq, Hkv, G, MB;
  int32_t n_sink, window;   // window <= 0: no window
  int32_t has_cur;
  int32_t bps, max_splits;  // bps: blocks per split when fixed by the caller; max_splits:
                            // partial slots per unit (the most splits any selection gets)
  int32_t dyn_splits;       // 1: blocks per split chosen on the device (effective_bps)
  int32_t split_cap;        // most splits per unit the automatic plan considers
  int32_t nvb_max;          // host bound on visited blocks per request
  int32_t lpi;              // layers per work item (attn_local_layers_kernel)
  int32_t select;
  float scale_log2;         // scale * log2(e)
  // device-data checks: a length outside [1, max_len], a block-table entry
  // outside [0, num_blocks) or a listed request outside [0, B) is never used
  // to address memory; the affected outputs become NaN (or are skipped)
  int32_t max_len;
  int64_t num_blocks;
  // fused current-token preparation (the *_qkv entry points, one layer): q
  // and the candidate K/V are built from the fp32 QKV projection output
  // instead of being read from q / k_cur / v_cur
  const float* qkv;      // [B][(Hq + 2 Hkv) D], or NULL (not fused)
  const float* q_gain;   // [D] or NULL
  const float* k_gain;   // [D] or NULL
  uint16_t* k_out;       // [B][Hkv][D]: the candidate K (bf16) for the commit, or NULL
  uint16_t* v_out;       // [B][Hkv][D]
  double rope_theta;
  float rms_eps;
  // direct-ring Local: the window is read from per-unit rings of whole blocks
  // (k_ring [L][B][SB + RB][Hkv][D/8][16][8], v_ring alike) instead of the
  // paged cache; logical block j sits in ring block j (j < SB) or SB + j % RB
  const uint16_t* k_ring;   // NULL: read the paged cache through the block table
  const uint16_t* v_ring;
  int32_t ring_sb, ring_rb;
};

// Where a unit's query rows and current candidate come from: global memory,
// or the bf16 copy a fused call builds in shared memory.
struct CurSrc {
  const uint16_t* q;    // [G][D] rows of the unit's query heads
  const uint16_t* k;    // [D] candidate K (has_cur only)
  const uint16_t* v;    // [D] candidate V (has_cur only)
};

__device__ __forceinline__ CurSrc global_cur(const AttnArgs& a, int D, int l, int b, int g) {
  CurSrc c;
  c.q = a.q + (((int64_t)l * a.B + b) * a.Hq + (int64_t)g * a.G) * D;
  const int64_t coff = (((int64_t)l * a.B + b) * a.Hkv + g) * D;
  c.k = a.has_cur ? a.k_cur + coff : nullptr;
  c.v = a.has_cur ? a.v_cur + coff : nullptr;
  return c;
}

// Positions of one request attended through the cache, as block ranges.
//   A = [0, a_end)          the sink part
//   R = [r_start, nc)       the recent part (nc = cache end: n, or n-1 when
//                           the current token comes from k_cur)
// Blocks visited: [0, ab_end) then [rb_lo, rb_hi); a block holding both A and
// R positions is visited once (in the first range).  "Virtual" block v counts
// the visited blocks in that order.
struct Geometry {
  int a_end, r_start, nc, ab_end, rb_lo, rb_hi, nvb;
};

__device__ __forceinline__ Geometry geometry(int n, int n_sink, int window, int has_cur) {
  Geometry g;
  g.nc = n - has_cur;
  const int sink_end = min(n_sink, n);
  g.a_end = min(sink_end, g.nc);
  const int win_start = window > 0 ? max(0, n - window) : 0;
  g.r_start = max(win_start, sink_end);
  g.ab_end = (g.a_end + kBlock - 1) / kBlock;
  if (g.r_start < g.nc) {
    g.rb_lo = max(g.r_start / kBlock, g.ab_end);
    g.rb_hi = (g.nc + kBlock - 1) / kBlock;
  } else {
    g.rb_lo = g.rb_hi = 0;
  }
  g.nvb = g.ab_end + (g.rb_hi - g.rb_lo);
  return g;
}

__device__ __forceinline__ int logical_block(const Geometry& g, int v) {
  return v < g.ab_end ? v : g.rb_lo + (v - g.ab_end);
}

__device__ __forceinline__ bool in_set(const Geometry& g, int p) {
  return p < g.a_end || (p >= g.r_start && p < g.nc);
}

// All 16 positions of logical block lb attended?
__device__ __forceinline__ bool block_full(const Geometry& g, int lb) {
  const int p0 = lb * kBlock, p1 = p0 + kBlock;
  return p1 <= g.a_end || (p0 >= g.r_start && p1 <= g.nc);
}

__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

// Requests with work in this call: the work list's count (at most the batch),
// the number of set flags, or the whole batch.  Uniform over the wavefront.
__device__ __forceinline__ int active_requests(const AttnArgs& a) {
  if (a.select == kSelList) return uniform(min(max(a.n_work[0], 0), a.B));
  if (a.select != kSelFlags) return a.B;
  int active = 0;
  for (int b0 = 0; b0 < a.B; b0 += 64) {
    const int b = b0 + (int)(threadIdx.x & 63);
    active += __popcll(__ballot(b < a.B && a.flags[b] != 0));
  }
  return uniform(active);
}

// The request of the rank-th active slot (ascending request order for flags,
// list order for a work list); false if the listed id is outside the batch.
__device__ __forceinline__ bool request_of_rank(const AttnArgs& a, int rank, int& b) {
  if (a.select == kSelList) {
    b = a.work_list[rank];
    return b >= 0 && b < a.B;
  }
  if (a.select != kSelFlags) {
    b = rank;
    return true;
  }
  const int lane = (int)(threadIdx.x & 63);
  int seen = 0;
  for (int b0 = 0; b0 < a.B; b0 += 64) {
    const uint64_t m = __ballot(b0 + lane < a.B && a.flags[b0 + lane] != 0);
    const int c = __popcll(m);
    if (rank < seen + c) {
      // the lane whose flag is set with exactly rank - seen set flags below it
      const uint64_t below = m & ((1ull << lane) - 1ull);
      const bool hit = ((m >> lane) & 1ull) != 0 && (int)__popcll(below) == rank - seen;
      b = b0 + __builtin_ctzll(__ballot(hit));
      return true;
    }
    seen += c;
  }
  return false;
}

// Splits per unit for `units` units, at least `want` and at most `cap`.  While
// a launch keeps HBM busy, a CU streams at only ~27-34 GB/s (about 1/200 of
// HBM's rate) whether it holds one workgroup or two (alone, ~55), so a launch
// whose CUs do not all hold the same number of equal workgroups runs at the
// pace of those holding one more: 96 units in 3 splits (288 workgroups on 256
// CUs) read at 4.9 TB/s, in 5 splits (480) at 6.3.  For m = 1, 2, ... workgroups per CU the largest count s >= want with
// units * s <= 256 m is taken as soon as it fills the CUs within 10% of
// evenly; if no count up to `cap` does, the most even one.  At most 17 steps,
// the same on the host (plan) and on the device (selected requests).
__host__ __device__ __forceinline__ int64_t balanced_splits(int64_t units, int64_t want, int64_t cap) {
  if (want >= cap) return cap;
  int64_t best = want;
  int64_t best_m = (units * want + kTargetGroups - 1) / kTargetGroups;   // workgroups per CU at `want`
  for (int64_t m = best_m; m <= best_m + 16; ++m) {
    const int64_t s = kTargetGroups * m / units;
    if (s > cap) break;
    if (kTargetGroups * m * 10 <= units * s * 11) return s;
    if (m * best < best_m * s) {   // m / s below best_m / best: more even
      best = s;
      best_m = m;
    }
  }
  return best;
}

// Blocks per split of the automatic plan for `units` units (the selected
// requests' layers and KV heads, `per_request` of them per request) of at
// most nvb_max blocks each, with at most `cap` splits per unit: enough splits
// for about one workgroup per CU, then more to even the CUs out while every
// split keeps kBalanceBlocks blocks.  Each split past the first costs its
// workgroup a partial write, a ticket and a share of the merge: at even load,
// splits of 514 / 258 / 130 blocks took 3.6% / 7.6% / 25% longer than whole
// units.  The evening assumes units of equal length, which holds for the
// units of one request; when a request has fewer than kBalanceUnits of them
// (one-layer calls), the spread of the requests' lengths sets the balance
// instead, and more splits made per-layer calls over 8K-64K requests slower.
__host__ __device__ __forceinline__ int plan_bps(int64_t units, int64_t per_request, int nvb_max, int cap) {
  const int64_t want = (kTargetGroups + units - 1) / units;
  int64_t s = want < cap ? want : cap;
  const int64_t keep = nvb_max / kBalanceBlocks;   // splits that keep kBalanceBlocks blocks each
  if (per_request >= kBalanceUnits && keep > s) s = balanced_splits(units, s, keep < cap ? keep : cap);
  if (s < 1) s = 1;
  const int bps = (int)(((nvb_max + s - 1) / s + 1) & ~(int64_t)1);
  return bps > 2 ? bps : 2;
}

// Blocks per split for this call: fixed by the caller, or the automatic plan
// for the number of selected requests (known only on the device for Full).
__device__ __forceinline__ int effective_bps(const AttnArgs& a, int active) {
  if (!a.dyn_splits) return a.bps;
  return uniform(plan_bps((int64_t)max(active, 1) * a.L * a.Hkv, (int64_t)a.L * a.Hkv, a.nvb_max, a.split_cap));
}

__device__ __forceinline__ bf16x8 load16(const uint16_t* p) {
  return *reinterpret_cast<const bf16x8*>(p);
}
// KV is read once per call: stream it with nontemporal loads.
__device__ __forceinline__ bf16x8 stream16(const uint16_t* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const bf16x8*>(p));
}
__device__ __forceinline__ u32x2 stream8(const uint16_t* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(p));
}
__device__ __forceinline__ bf16x8 cat(u32x2 lo, u32x2 hi) {
  u32x4 t = {lo.x, lo.y, hi.x, hi.y};
  return __builtin_bit_cast(bf16x8, t);
}
__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float bf16_to_float(uint16_t x) {
  return __builtin_bit_cast(float, (uint32_t)x << 16);
}
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) x += __shfl_xor(x, s);
  return x;
}

// Keep the 16-bit lanes of a 4 x bf16 pack whose position is attended.
__device__ __forceinline__ u32x2 mask_pack(u32x2 v, bool m0, bool m1, bool m2, bool m3) {
  const uint32_t w0 = (m0 ? 0x0000FFFFu : 0u) | (m1 ? 0xFFFF0000u : 0u);
  const uint32_t w1 = (m2 ? 0x0000FFFFu : 0u) | (m3 ? 0xFFFF0000u : 0u);
  u32x2 r = {v.x & w0, v.y & w1};
  return r;
}

// Registers of one pair of KV blocks (32 positions) in MFMA operand layout.
template <int D>
struct PairTile {
  bf16x8 k0[D / 32], k1[D / 32];
  u32x2 v0[D / 16], v1[D / 16];
};

// One wavefront's run of blocks: virtual blocks [v_lo, v_hi) of its request;
// lane i of the table register holds the physical block of virtual block
// v_lo + 64c + i for the current chunk c of 64 blocks.
struct Run {
  Geometry geo;
  const uint16_t* kbase;
  const uint16_t* vbase;
  const int32_t* bt;        // NULL: blocks come from the unit's ring (ring_sb, ring_rb)
  int64_t blk_stride;
  int64_t nblocks;
  int v_lo, v_hi;
  int ring_sb, ring_rb;
};

// Physical blocks of 64 consecutive virtual blocks, one per lane.  An entry
// outside [0, num_blocks) reads block 0 instead and sets `bad`.
__device__ __forceinline__ int table_chunk(const Run& r, int chunk, int lane, int& bad) {
  const int v = r.v_lo + chunk * 64 + lane;
  int e = 0;
  if (v < r.v_hi) {
    const int lb = logical_block(r.geo, v);
    e = r.bt != nullptr ? r.bt[lb] : (lb < r.ring_sb ? lb : r.ring_sb + lb % r.ring_rb);
  }
  const bool ok = e >= 0 && e < r.nblocks;
  bad |= ok ? 0 : 1;
  return ok ? e : 0;
}

__device__ __forceinline__ bool valid_len(const AttnArgs& a, int n) { return n >= 1 && n <= a.max_len; }

template <int D>
__device__ __forceinline__ void load_pair(PairTile<D>& t, const Run& r, int v, int tbl, int lane) {
  constexpr int KK = D / 32, NT = D / 16;
  const int h16 = lane & 15, j = lane >> 4;
  const int i0 = (v - r.v_lo) & 63;
  const int64_t pb0 = __builtin_amdgcn_readlane(tbl, i0);
  // an odd tail reuses block 0 for the second tile; all its positions are masked
  const int64_t pb1 = (v + 1 < r.v_hi) ? __builtin_amdgcn_readlane(tbl, i0 + 1) : pb0;
  const uint16_t* k0 = r.kbase + pb0 * r.blk_stride;
  const uint16_t* k1 = r.kbase + pb1 * r.blk_stride;
  const uint16_t* v0 = r.vbase + pb0 * r.blk_stride;
  const uint16_t* v1 = r.vbase + pb1 * r.blk_stride;
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) {
    t.k0[kk] = stream16(k0 + (kk * 64 + lane) * 8);
    t.k1[kk] = stream16(k1 + (kk * 64 + lane) * 8);
  }
#pragma unroll
  for (int n = 0; n < NT; ++n) {
    const int d = 16 * n + h16;
    t.v0[n] = stream8(v0 + d * kBlock + 4 * j);
    t.v1[n] = stream8(v1 + d * kBlock + 4 * j);
  }
}

// One pair of blocks: S^T on MFMA, online softmax of head h16, O += P V on MFMA.
template <int D>
__device__ __forceinline__ void consume_pair(PairTile<D>& t, const Run& r, int v, int lane, const bf16x8* qf,
                                             float scale_log2, f32x4* o, float& m_run, float& l_run) {
  constexpr int KK = D / 32, NT = D / 16;
  const int j = lane >> 4;
  const bool has1 = (v + 1) < r.v_hi;
  const int lb0 = logical_block(r.geo, v);
  const int lb1 = has1 ? logical_block(r.geo, v + 1) : lb0;

  f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) {
    s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(t.k0[kk], qf[kk], s0, 0, 0, 0);
    s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(t.k1[kk], qf[kk], s1, 0, 0, 0);
  }
  float sc[8];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    sc[i] = s0[i] * scale_log2;
    sc[4 + i] = s1[i] * scale_log2;
  }
  const bool full0 = block_full(r.geo, lb0);
  const bool full1 = has1 && block_full(r.geo, lb1);
  if (!(full0 && full1)) {
    bool m[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      m[i] = in_set(r.geo, lb0 * kBlock + 4 * j + i);
      m[4 + i] = has1 && in_set(r.geo, lb1 * kBlock + 4 * j + i);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) sc[i] = m[i] ? sc[i] : -INFINITY;
    // unattended slots may hold anything (even NaN): zero them so 0 * V stays 0
#pragma unroll
    for (int n = 0; n < NT; ++n) {
      t.v0[n] = mask_pack(t.v0[n], m[0], m[1], m[2], m[3]);
      t.v1[n] = mask_pack(t.v1[n], m[4], m[5], m[6], m[7]);
    }
  }

  // online softmax for head h16 (its 32 positions are spread over lanes h16 + 16j)
  float mx = sc[0];
#pragma unroll
  for (int i = 1; i < 8; ++i) mx = fmaxf(mx, sc[i]);
  mx = fmaxf(mx, __shfl_xor(mx, 16));
  mx = fmaxf(mx, __shfl_xor(mx, 32));
  const float m_new = fmaxf(m_run, mx);
  const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
  const float alpha = exp2_fast(m_run - m_use);
  m_run = m_new;
  float p[8];
  float psum = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    p[i] = exp2_fast(sc[i] - m_use);
    psum += p[i];
  }
  l_run = l_run * alpha + psum;

  // rescale O rows (heads 4j..4j+3) by their heads' alpha, when any changed
  if (__any(alpha != 1.f)) {
    float al[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) al[i] = __shfl(alpha, 4 * j + i);
#pragma unroll
    for (int n = 0; n < NT; ++n) {
#pragma unroll
      for (int i = 0; i < 4; ++i) o[n][i] *= al[i];
    }
  }

  // P as the A operand (row = head h16, k = its 8 positions), split hi + lo
  bf16x8 phi, plo;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const __bf16 h = (__bf16)p[i];
    phi[i] = h;
    plo[i] = (__bf16)(p[i] - (float)h);
  }
#pragma unroll
  for (int n = 0; n < NT; ++n) {
    const bf16x8 vf = cat(t.v0[n], t.v1[n]);
    o[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(phi, vf, o[n], 0, 0, 0);
    o[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(plo, vf, o[n], 0, 0, 0);
  }
}

// Shared memory of the split workgroup (dynamic): per wavefront m[16], l[16]
// and o[G][D]; then the candidate logits zc[16].
__host__ __device__ constexpr size_t split_lds_floats(int G, int D) {
  return (size_t)kWaves * 32 + (size_t)kWaves * G * D + 16;
}
// A fused call's bf16 query rows and candidate K/V, after the floats above.
__host__ __device__ constexpr size_t prep_lds_bytes(int G, int D) { return (size_t)(G + 2) * D * 2; }

// Running state of one output element of the split merge: maximum logit M
// (log2 units), weighted sum of partial outputs and of partial denominators.
struct MergeAcc {
  float M = -INFINITY, acc = 0.f, lam = 0.f;
};

// Fold splits [s0, s0 + C) of one (query head hh, dimension d) into m; indices
// past the last split repeat it with weight 0.
template <int C, int D>
__device__ __forceinline__ void merge_chunk(MergeAcc& m, const float* ml, const float* po, int s0, int nsplit,
                                            int G, int hh, int d) {
  float mv[C], lv[C], ov[C];
#pragma unroll
  for (int k = 0; k < C; ++k) {
    const int s = min(s0 + k, nsplit - 1);
    mv[k] = ml[(s * G + hh) * 2];
    lv[k] = ml[(s * G + hh) * 2 + 1];
    ov[k] = po[((int64_t)s * G + hh) * D + d];
  }
  float Mc = m.M;
#pragma unroll
  for (int k = 0; k < C; ++k) Mc = fmaxf(Mc, mv[k]);
  const float r = (Mc == m.M) ? 1.f : exp2_fast(m.M - Mc);
  m.acc *= r;
  m.lam *= r;
  m.M = Mc;
#pragma unroll
  for (int k = 0; k < C; ++k) {
    const float w = (s0 + k < nsplit) ? exp2_fast(mv[k] - Mc) : 0.f;
    m.acc += w * ov[k];
    m.lam += w * lv[k];
  }
}

// Combine the nsplit partials of one (layer, request, KV head) with stable
// softmax rescaling (plus the uncommitted candidate) and write out / lse.
// Called by every thread of a workgroup of `nthreads` threads (it holds a
// barrier); sm_zc: LDS for kMaxGroup candidate logits.  Partials are read in
// split order, so the result does not depend on which workgroup merges.
template <int D>
__device__ __forceinline__ void merge_unit(const AttnArgs& a, int l, int b, int g, int nsplit, float* sm_zc,
                                           int nthreads, const CurSrc& cur) {
  const int G = a.G;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t pbase = (((int64_t)l * a.B + b) * a.Hkv + g) * a.max_splits;
  const float* ml = a.part_ml + pbase * G * 2;
  const float* po = a.part_o + pbase * G * D;
  const int64_t qoff = (((int64_t)l * a.B + b) * a.Hq + (int64_t)g * G) * D;

  if (a.has_cur) {
    constexpr int PD = D / 64;
    float kc[PD];
#pragma unroll
    for (int e = 0; e < PD; ++e) kc[e] = bf16_to_float(cur.k[lane * PD + e]);
    for (int hh = wave; hh < G; hh += nthreads / 64) {
      float dot = 0.f;
#pragma unroll
      for (int e = 0; e < PD; ++e) dot += bf16_to_float(cur.q[hh * D + lane * PD + e]) * kc[e];
      dot = wave_sum(dot) * a.scale_log2;
      if (lane == 0) sm_zc[hh] = dot;
    }
  }
  __syncthreads();

  // The partials were written back from other XCDs, so every read is a trip to
  // memory: a chunk of splits is loaded with all its reads in flight at once,
  // and the running maximum is rescaled once per chunk.
  for (int e = threadIdx.x; e < G * D; e += nthreads) {
    const int hh = e / D, d = e - hh * D;
    MergeAcc m;
    if (a.has_cur) {   // the candidate's weight is exp2(zc - M) = 1 at M = zc
      m.M = sm_zc[hh];
      m.acc = bf16_to_float(cur.v[d]);
      m.lam = 1.f;
    }
    for (int s0 = 0; s0 < nsplit;) {
      if (nsplit - s0 > 2 * kMergeSmall) {
        merge_chunk<kMergeChunk, D>(m, ml, po, s0, nsplit, G, hh, d);
        s0 += kMergeChunk;
      } else {
        merge_chunk<kMergeSmall, D>(m, ml, po, s0, nsplit, G, hh, d);
        s0 += kMergeSmall;
      }
    }
    a.out[qoff + e] = m.acc / m.lam;
    if (d == 0 && a.lse != nullptr)
      a.lse[((int64_t)l * a.B + b) * a.Hq + (int64_t)g * G + hh] = (m.M + __log2f(m.lam)) * kLn2;
  }
}

// Fused calls: the unit's G query heads, its K head and its V head of the
// current token, from the fp32 QKV projection output (q heads, then k heads,
// then v heads per request), one head per wavefront: q and k through the
// per-head RMSNorm and the rotary embedding at position n - 1 (the shared
// oda::norm_rope_pair, the same code oda_qk_norm_rope runs), v unchanged,
// all rounded to bf16 into prep = [G][D] query rows, then K, then V.  The
// fp32 loads do not depend on n; the rotation does.
template <int D>
__device__ __forceinline__ void prepare_current(const AttnArgs& a, int b, int g, int n, uint16_t* prep,
                                                bool write_out) {
  constexpr int half = D / 2;
  const int G = a.G;
  const int lane = threadIdx.x & 63;
  const int wave = uniform(threadIdx.x >> 6);
  const int heads = a.Hq + 2 * a.Hkv;
  for (int t = wave; t < G + 2; t += kWaves) {   // t < G: query head g G + t; G: K; G + 1: V
    const int h = t < G ? g * G + t : (t == G ? a.Hq + g : a.Hq + a.Hkv + g);
    const float* src = a.qkv + ((int64_t)b * heads + h) * D;
    float x1 = lane < half ? src[lane] : 0.f;
    float x2 = lane < half ? src[lane + half] : 0.f;
    if (t <= G)
      oda::norm_rope_pair(x1, x2, lane < half, lane, D, t < G ? a.q_gain : a.k_gain, a.rms_eps, (double)(n - 1),
                          a.rope_theta);
    if (lane < half) {
      const uint16_t y1 = oda::bf16_rne(x1), y2 = oda::bf16_rne(x2);
      uint16_t* dst = prep + (int64_t)t * D;
      dst[lane] = y1;
      dst[lane + half] = y2;
      if (write_out && t >= G && a.k_out != nullptr) {
        uint16_t* o = (t == G ? a.k_out : a.v_out) + ((int64_t)b * a.Hkv + g) * D;
        o[lane] = y1;
        o[lane + half] = y2;
      }
    }
  }
}

// One unit of work: the wavefront runs of r (this split of request b) for
// layer l and KV head g are streamed, combined across the wavefronts in
// shared memory and written out (finalised when the request has one split,
// else as this split's partial).
template <int D, bool kLocal>
__device__ __forceinline__ void run_unit(const AttnArgs& a, Run& r, int l, int b, int g, int split, int nsplit,
                                         float* smem, const CurSrc& cur) {
  constexpr int KK = D / 32;   // MFMA k-steps for q.k
  constexpr int NT = D / 16;   // 16-dim output tiles
  const int lane = threadIdx.x & 63;
  const int wave = uniform(threadIdx.x >> 6);
  const int h16 = lane & 15;
  const int j = lane >> 4;
  const int G = a.G;
  const int64_t head_elems = (int64_t)kBlock * D;
  r.blk_stride = (int64_t)a.Hkv * head_elems;
  r.ring_sb = a.ring_sb;
  r.ring_rb = a.ring_rb;
  if (a.k_ring != nullptr) {
    const int64_t unit0 = ((int64_t)l * a.B + b) * (a.ring_sb + a.ring_rb) * r.blk_stride + (int64_t)g * head_elems;
    r.kbase = a.k_ring + unit0;
    r.vbase = a.v_ring + unit0;
    r.nblocks = a.ring_sb + a.ring_rb;
    r.bt = nullptr;
  } else {
    r.kbase = a.k_cache + (int64_t)l * a.kv_layer_stride + (int64_t)g * head_elems;
    r.vbase = a.v_cache + (int64_t)l * a.kv_layer_stride + (int64_t)g * head_elems;
    r.nblocks = a.num_blocks;
    r.bt = a.block_table + (int64_t)b * a.MB;
  }

  f32x4 o[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) o[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY;  // running max (log2 units) of head h16
  float l_run = 0.f;        // this lane's share of the running exp-sum

  if (r.v_lo < r.v_hi) {
    // Q^T as the B operand: column = query head h16 of this KV head's group.
    bf16x8 qf[KK];
    const uint16_t* qrow = cur.q + (int64_t)h16 * D;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) qf[kk] = (h16 < G) ? load16(qrow + 32 * kk + 8 * j) : bf16x8{};

    int bad = 0;
    int tbl = table_chunk(r, 0, lane, bad);
    int tbl_next = table_chunk(r, 1, lane, bad);
    for (int v = r.v_lo; v < r.v_hi; v += 2) {
      if (v > r.v_lo && ((v - r.v_lo) & 63) == 0) {
        tbl = tbl_next;
        tbl_next = table_chunk(r, ((v - r.v_lo) >> 6) + 1, lane, bad);
      }
      PairTile<D> ta;
      load_pair<D>(ta, r, v, tbl, lane);
      consume_pair<D>(ta, r, v, lane, qf, a.scale_log2, o, m_run, l_run);
    }
    l_run += __shfl_xor(l_run, 16);
    l_run += __shfl_xor(l_run, 32);
    if (__any(bad)) {   // a block-table entry out of range: this request's rows become NaN
      m_run = __builtin_nanf("");
      l_run = __builtin_nanf("");
    }
  }

  // combine the wavefronts through LDS
  float* sm_m = smem;                        // [kWaves][16]
  float* sm_l = smem + kWaves * 16;          // [kWaves][16]
  float* sm_o = smem + kWaves * 32;          // [kWaves][G][D]
  float* sm_zc = sm_o + kWaves * G * D;      // [16]
  if (j == 0) {
    sm_m[wave * 16 + h16] = m_run;
    sm_l[wave * 16 + h16] = l_run;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int hh = 4 * j + i;
    if (hh < G) {
      float* dst = sm_o + ((int64_t)wave * G + hh) * D + h16;
#pragma unroll
      for (int t = 0; t < NT; ++t) dst[16 * t] = o[t][i];
    }
  }
  const bool finalize = (nsplit == 1);
  const int64_t qoff = (((int64_t)l * a.B + b) * a.Hq + (int64_t)g * G) * D;
  if (finalize && a.has_cur && wave == 0) {
    // candidate logits of the G heads (log2 units)
    constexpr int PD = D / 64;
    float kc[PD];
#pragma unroll
    for (int e = 0; e < PD; ++e) kc[e] = bf16_to_float(cur.k[lane * PD + e]);
    for (int hh = 0; hh < G; ++hh) {
      float dot = 0.f;
#pragma unroll
      for (int e = 0; e < PD; ++e) dot += bf16_to_float(cur.q[hh * D + lane * PD + e]) * kc[e];
      dot = wave_sum(dot) * a.scale_log2;
      if (lane == 0) sm_zc[hh] = dot;
    }
  }
  __syncthreads();

  const int64_t pidx = (((int64_t)l * a.B + b) * a.Hkv + g) * a.max_splits + split;
  for (int e = threadIdx.x; e < G * D; e += kWaves * 64) {
    const int hh = e / D, d = e - hh * D;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, sm_m[w * 16 + hh]);
    const float Mu = (M == -INFINITY) ? 0.f : M;
    float acc = 0.f, lam = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float s = exp2_fast(sm_m[w * 16 + hh] - Mu);
      acc += s * sm_o[((int64_t)w * G + hh) * D + d];
      lam += s * sm_l[w * 16 + hh];
    }
    if (finalize) {
      if (a.has_cur) {
        const float z = sm_zc[hh];
        const float M2 = fmaxf(M, z);
        const float s_old = exp2_fast(M - M2), s_cur = exp2_fast(z - M2);
        acc = acc * s_old + s_cur * bf16_to_float(cur.v[d]);
        lam = lam * s_old + s_cur;
        M = M2;
      }
      a.out[qoff + e] = acc / lam;
      if (d == 0 && a.lse != nullptr)
        a.lse[((int64_t)l * a.B + b) * a.Hq + (int64_t)g * G + hh] = (M + __log2f(lam)) * kLn2;
    } else {
      a.part_o[pidx * G * D + e] = acc;
      if (d == 0) {
        a.part_ml[(pidx * G + hh) * 2 + 0] = M;
        a.part_ml[(pidx * G + hh) * 2 + 1] = lam;
      }
    }
  }
}

// kLocal selects the Local access set (sinks + window); Full instances take the
// native set (whole history, or a native window) and never have sinks.
template <int D, bool kLocal>
__global__ __launch_bounds__(kWaves * 64) __attribute__((amdgpu_waves_per_eu(2)))
void attn_split_kernel(AttnArgs a) {
  extern __shared__ float smem[];
  const int wave = uniform(threadIdx.x >> 6);

  // split outermost, then the rank of the request among those with work: the
  // items that have work (the splits in use of the selected requests) form a
  // prefix of the grid, so the dispatcher spreads them over the CUs first
  // instead of interleaving them with workgroups that exit at once
  const int active = active_requests(a);
  if (active == 0) return;
  int64_t item = blockIdx.x;
  const int g = (int)(item % a.Hkv);
  item /= a.Hkv;
  const int l = (int)(item % a.L);
  item /= a.L;
  const int rank = (int)(item % active);
  const int bps = effective_bps(a, active);
  // no selected request has this split (the grid covers the selection with
  // the most); the plan keeps every split below max_splits, checked anyway
  if ((item / active) * bps >= max(a.nvb_max, 1) || item / active >= a.max_splits) return;
  const int split = (int)(item / active);
  int b;
  if (!request_of_rank(a, rank, b)) return;
  b = uniform(b);
  const int n = uniform(a.seq_lens[b]);
  const int G = a.G;
  CurSrc cur;
  if (a.qkv != nullptr) {
    // fused call: this workgroup builds the unit's bf16 query rows and the
    // candidate K/V in shared memory (every split the same values); split 0
    // also writes the candidate out for the commit
    uint16_t* prep = reinterpret_cast<uint16_t*>(smem + split_lds_floats(G, D));
    prepare_current<D>(a, b, g, n, prep, split == 0);
    __syncthreads();
    cur.q = prep;
    cur.k = prep + G * D;
    cur.v = prep + (G + 1) * D;
  } else {
    cur = global_cur(a, D, l, b, g);
  }
  if (!valid_len(a, n)) {   // no history is addressed: the request's rows become NaN
    if (split == 0) {
      const int64_t q0 = (((int64_t)l * a.B + b) * a.Hq + (int64_t)g * G) * D;
      for (int e = threadIdx.x; e < G * D; e += kWaves * 64) {
        a.out[q0 + e] = __builtin_nanf("");
        if (e % D == 0 && a.lse != nullptr) a.lse[((int64_t)l * a.B + b) * a.Hq + (int64_t)g * G + e / D] = __builtin_nanf("");
      }
    }
    return;
  }
  Run r;
  r.geo = geometry(n, kLocal ? a.n_sink : 0, a.window, a.has_cur);
  // (nvb = 0 happens only with the candidate as the sole position: one item, no blocks)
  const int nsplit = max(1, (r.geo.nvb + bps - 1) / bps);
  if (split >= nsplit) return;   // uniform over the workgroup: no barrier is skipped by part of it

  // this wavefront's run: a contiguous share of the split's pairs
  const int v_begin = split * bps;
  const int v_end = min(r.geo.nvb, v_begin + bps);
  const int pairs = (v_end - v_begin + 1) >> 1;
  const int per_wave = (pairs + kWaves - 1) / kWaves;
  r.v_lo = min(v_end, v_begin + 2 * per_wave * wave);
  r.v_hi = min(v_end, r.v_lo + 2 * per_wave);

  run_unit<D, kLocal>(a, r, l, b, g, split, nsplit, smem, cur);
  if (nsplit == 1) return;   // finalised
  float* sm_zc = smem + kWaves * 32 + kWaves * G * D;
  // The last of the request's splits to finish merges them all.  The eight
  // XCDs' L2 caches are not coherent with each other, so the partials are
  // published at device scope: every wavefront waits until its stores have
  // reached its XCD's L2, then one thread writes that L2 back (one release per
  // workgroup: a release per wavefront made one-layer Full calls over 32K
  // positions ~40% slower) and takes a ticket.  The ticket counts modulo
  // nsplit (a wrapping increment), so the last arrival sees nsplit - 1 and the
  // word is back at 0 with no separate reset: even a request listed twice
  // (2 nsplit arrivals) leaves it at 0 for later calls.  The workgroup holding
  // the last ticket drops stale cached lines (acquire) and merges.
  __shared__ int last_split;
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  uint32_t* ticket = a.tickets + ((int64_t)l * a.B + b) * a.Hkv + g;
  if (threadIdx.x == 0) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    const uint32_t t = __builtin_amdgcn_atomic_inc32(ticket, (uint32_t)(nsplit - 1), __ATOMIC_RELAXED, "agent");
    last_split = (t == (uint32_t)(nsplit - 1)) ? 1 : 0;
  }
  __syncthreads();
  if (!last_split) return;
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  merge_unit<D>(a, l, b, g, nsplit, sm_zc, kWaves * 64, cur);
}

// Batched Local with one split per unit and many units per CU: a work item is
// a.lpi consecutive layers of one (request, KV head), walked in turn by the
// workgroup.  The request's length is read once for all of them and each
// layer starts on a CU that is already running (no workgroup start-up per
// unit).  Items: (KV head, layer group, request), KV head fastest.
template <int D>
__global__ __launch_bounds__(kWaves * 64) __attribute__((amdgpu_waves_per_eu(2)))
void attn_local_layers_kernel(AttnArgs a) {
  extern __shared__ float smem[];
  const int wave = uniform(threadIdx.x >> 6);
  int64_t item = blockIdx.x;
  const int g = (int)(item % a.Hkv);
  item /= a.Hkv;
  const int groups = a.L / a.lpi;
  const int lg = (int)(item % groups);
  item /= groups;
  if (item >= a.B) return;
  const int b = (int)item;
  const int n = uniform(a.seq_lens[b]);
  const int G = a.G;
  const int l0 = lg * a.lpi, l1 = l0 + a.lpi;
  if (!valid_len(a, n)) {   // no history is addressed: the request's rows become NaN
    for (int l = l0; l < l1; ++l) {
      const int64_t q0 = (((int64_t)l * a.B + b) * a.Hq + (int64_t)g * G) * D;
      for (int e = threadIdx.x; e < G * D; e += kWaves * 64) {
        a.out[q0 + e] = __builtin_nanf("");
        if (e % D == 0 && a.lse != nullptr) a.lse[((int64_t)l * a.B + b) * a.Hq + (int64_t)g * G + e / D] = __builtin_nanf("");
      }
    }
    return;
  }
  Run r;
  r.geo = geometry(n, a.n_sink, a.window, a.has_cur);
  // one split: this wavefront's contiguous share of the unit's pairs
  const int pairs = (r.geo.nvb + 1) >> 1;
  const int per_wave = (pairs + kWaves - 1) / kWaves;
  r.v_lo = min(r.geo.nvb, 2 * per_wave * wave);
  r.v_hi = min(r.geo.nvb, r.v_lo + 2 * per_wave);
  for (int l = l0; l < l1; ++l) {
    run_unit<D, true>(a, r, l, b, g, 0, 1, smem, global_cur(a, D, l, b, g));
    __syncthreads();   // the next layer reuses the shared memory
  }
}


// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------

struct Plan {
  int nvb_max;
  int bps;            // blocks per split: fixed, or the automatic plan's for all B requests
  int max_splits;     // partial slots per unit: the most splits any selection gets
  int split_cap;      // most splits per unit the automatic plan considers
  int local_splits;   // splits per unit of a Local call (all B requests selected)
  int64_t full_slots; // (request rank, split) pairs a Full grid covers: the most over selections
  int dyn;
  size_t off_o;
  size_t off_ml;
  size_t bytes;
};

oda_status check_shape(const oda_attn_shape* s) {
  if (s == nullptr) return oda::fail(ODA_ERR_NULL, "shape is NULL");
  if (s->num_layers < 1 || s->batch < 1 || s->num_q_heads < 1 || s->num_kv_heads < 1)
    return oda::fail(ODA_ERR_SHAPE, "num_layers, batch, num_q_heads, num_kv_heads must be >= 1");
  if (s->num_q_heads % s->num_kv_heads != 0)
    return oda::fail(ODA_ERR_SHAPE, "num_q_heads (%d) must be a multiple of num_kv_heads (%d)",
                     s->num_q_heads, s->num_kv_heads);
  if (s->num_q_heads / s->num_kv_heads > kMaxGroup)
    return oda::fail(ODA_ERR_UNSUPPORTED, "GQA group size %d > %d", s->num_q_heads / s->num_kv_heads,
                     kMaxGroup);
  if (s->head_dim != 64 && s->head_dim != 128)
    return oda::fail(ODA_ERR_UNSUPPORTED, "head_dim %d not in {64, 128}", s->head_dim);
  if (s->block_size != kBlock) return oda::fail(ODA_ERR_UNSUPPORTED, "block_size %d != 16", s->block_size);
  if (s->max_seq_len < 1) return oda::fail(ODA_ERR_SHAPE, "max_seq_len must be >= 1");
  if ((int64_t)s->max_blocks_per_seq < oda::ceil_div(s->max_seq_len, kBlock))
    return oda::fail(ODA_ERR_SHAPE, "max_blocks_per_seq %d < ceil(max_seq_len / 16)", s->max_blocks_per_seq);
  if (s->num_blocks < 1) return oda::fail(ODA_ERR_SHAPE, "num_blocks must be >= 1");
  if (s->split_blocks != 0 && (s->split_blocks < 2 || (s->split_blocks & 1)))
    return oda::fail(ODA_ERR_SHAPE, "split_blocks %d: 0 or an even number >= 2", s->split_blocks);
  if (s->reserved != 0) return oda::fail(ODA_ERR_SHAPE, "reserved must be 0");
  const int64_t dense = s->num_blocks * s->num_kv_heads * kBlock * s->head_dim;
  if (s->layer_stride_kv != 0 && (s->layer_stride_kv < dense || s->layer_stride_kv % 8 != 0))
    return oda::fail(ODA_ERR_SHAPE, "layer_stride_kv %lld: 0, or a multiple of 8 >= %lld", (long long)s->layer_stride_kv,
                     (long long)dense);
  return ODA_OK;
}

// Work decomposition.  One workgroup per (request, layer, KV head, split).
// The automatic plan splits a request only as much as needed for the selected
// requests to give the GPU about kTargetGroups workgroups (one per CU), and
// then to a count whose workgroups spread evenly over the CUs
// (balanced_splits).  Local selects every request; Full selects k of them,
// known only on the device, which picks the split count for its k
// (effective_bps).  The partial slots and the Full grid are sized for the
// selection that needs the most, so the workspace size a caller queries
// covers every call of the shape.  A request covered by one split is
// finalised by its workgroup; otherwise the last of its splits merges them in
// the same launch.
// Workspace: the ticket words (one per unit), then the partial o, then (m, l).
void make_plan(const oda_attn_shape* s, int n_sink, int window, Plan* p) {
  const int64_t total_blocks = oda::ceil_div(s->max_seq_len, kBlock);
  int64_t nvb = total_blocks;
  if (window > 0) {
    const int64_t sink_blocks = oda::ceil_div(std::min<int64_t>(n_sink, s->max_seq_len), kBlock);
    nvb = std::min<int64_t>(total_blocks, sink_blocks + oda::ceil_div(window, kBlock) + 1);
  }
  const int64_t units = (int64_t)s->num_layers * s->batch * s->num_kv_heads;
  const int64_t per_request = (int64_t)s->num_layers * s->num_kv_heads;
  p->nvb_max = (int)nvb;
  p->split_cap = 1;
  if (s->split_blocks != 0) {
    p->dyn = 0;
    p->bps = s->split_blocks;
    p->max_splits = (int)oda::ceil_div(nvb, s->split_blocks);
    p->local_splits = p->max_splits;
    p->full_slots = (int64_t)s->batch * p->max_splits;
  } else {
    // at least kWaves blocks (four block pairs) per split: a small call gets
    // more, shorter splits, which shortens the split phase more than the merge
    // of more partials costs (half of a split's wavefronts may be idle).  More
    // than kMergeChunk splits add a round trip to the merge, so they are taken
    // only while each split still has 8 * kWaves blocks (four pairs per
    // wavefront)
    p->dyn = 1;
    p->split_cap = (int)std::max<int64_t>(
        1, std::min<int64_t>(nvb / kWaves, std::max<int64_t>(kMergeChunk, nvb / (8 * kWaves))));
    // the device picks the split count for the number k of selected requests
    // (plan_bps); a Local call selects all B.  Partial slots and the Full grid
    // cover every k: from 10 CUs' worth of units on, one split per unit is
    // already even, so larger k add k requests of one split each.
    const int64_t k_even = oda::ceil_div(10 * kTargetGroups, per_request);
    p->max_splits = 1;
    p->full_slots = s->batch;
    for (int64_t k = 1; k <= std::min<int64_t>(s->batch, k_even); ++k) {
      const int bps = plan_bps(k * per_request, per_request, (int)nvb, p->split_cap);
      const int64_t ns = oda::ceil_div(nvb, bps);
      p->max_splits = (int)std::max<int64_t>(p->max_splits, ns);
      p->full_slots = std::max<int64_t>(p->full_slots, k * ns);
    }
    p->bps = plan_bps(s->batch * per_request, per_request, (int)nvb, p->split_cap);
    p->local_splits = (int)oda::ceil_div(nvb, p->bps);
  }
  if (p->max_splits <= 1) {
    p->off_o = 0;
    p->off_ml = 0;
    p->bytes = 0;
    return;
  }
  const int64_t G = s->num_q_heads / s->num_kv_heads;
  const int64_t parts = units * p->max_splits * G;
  const int64_t o_bytes = oda::round_up(parts * s->head_dim * 4, 256);
  const int64_t ml_bytes = oda::round_up(parts * 2 * 4, 256);
  // ticket words first: their place depends only on L * B * Hkv, so a
  // workspace stays valid across calls that differ in sinks or window
  const int64_t t_bytes = oda::round_up(units * 4, 256);
  p->off_o = (size_t)t_bytes;
  p->off_ml = (size_t)(t_bytes + o_bytes);
  p->bytes = (size_t)(t_bytes + o_bytes + ml_bytes);
}

oda_status check_inputs(const oda_attn_inputs* in, const float* out, const oda_attn_shape* s = nullptr,
                        const oda_qkv_prep* prep = nullptr) {
  if (in == nullptr) return oda::fail(ODA_ERR_NULL, "inputs is NULL");
  if (prep != nullptr) {   // fused current-token preparation: q and the candidate come from prep
    if (in->q || in->k_cur || in->v_cur)
      return oda::fail(ODA_ERR_SHAPE, "with oda_qkv_prep, q, k_cur and v_cur must be NULL");
    if (!prep->qkv) return oda::fail(ODA_ERR_NULL, "prep->qkv is required");
    if ((prep->k_out == nullptr) != (prep->v_out == nullptr))
      return oda::fail(ODA_ERR_NULL, "prep->k_out and prep->v_out must both be NULL or both be set");
    if (s->num_layers != 1) return oda::fail(ODA_ERR_SHAPE, "a call with oda_qkv_prep has one layer (got %d)",
                                             s->num_layers);
    if (!(prep->rope_theta > 1.0) || !std::isfinite(prep->rope_theta))
      return oda::fail(ODA_ERR_SHAPE, "prep->rope_theta must be > 1");
    if (!(prep->rms_eps >= 0.f) || !std::isfinite(prep->rms_eps))
      return oda::fail(ODA_ERR_SHAPE, "prep->rms_eps must be >= 0");
  } else if (!in->q) {
    return oda::fail(ODA_ERR_NULL, "q is required");
  }
  if (!in->k_cache || !in->v_cache || !in->block_table || !in->seq_lens || !out)
    return oda::fail(ODA_ERR_NULL, "k_cache, v_cache, block_table, seq_lens and out are required");
  if ((in->k_cur == nullptr) != (in->v_cur == nullptr))
    return oda::fail(ODA_ERR_NULL, "k_cur and v_cur must both be NULL or both be set");
  if ((in->q && !oda::aligned(in->q, 16)) || !oda::aligned(in->k_cache, 16) || !oda::aligned(in->v_cache, 16) ||
      !oda::aligned(out, 16) || (in->k_cur && (!oda::aligned(in->k_cur, 16) || !oda::aligned(in->v_cur, 16))))
    return oda::fail(ODA_ERR_SHAPE, "q, caches, k_cur, v_cur and out must be 16-byte aligned");
  if (!(in->scale > 0.f) || !std::isfinite(in->scale))
    return oda::fail(ODA_ERR_SHAPE, "scale must be finite and > 0");
  return ODA_OK;
}

// Layers per work item of a Local call: the most (a divisor of L) that still
// leave at least kTargetGroups workgroups, when every unit has one split;
// 1 (the split kernel) otherwise.
int layers_per_item(const oda_attn_shape* s, const Plan& plan) {
  if (plan.local_splits != 1) return 1;
  const int64_t per_layer = (int64_t)s->batch * s->num_kv_heads;
  for (int d = s->num_layers; d > 1; --d)
    if (s->num_layers % d == 0 && (s->num_layers / d) * per_layer >= kTargetGroups) return d;
  return 1;
}

// Raise a kernel's dynamic-LDS limit once per device (the attribute belongs
// to the device's copy of the kernel).  `done` holds one bit per device id
// below 64; other ids set it on every call.  Host threads that race here set
// the same value twice, which is harmless.  A failure is not fatal: the
// launch that needs the limit then fails and reports it.
void raise_lds_limit(const void* kernel, std::atomic<uint64_t>* done, int bytes) {
  int dev = -1;
  (void)hipGetDevice(&dev);
  const uint64_t bit = (dev >= 0 && dev < 64) ? (1ull << dev) : 0ull;
  if (bit != 0 && (done->load(std::memory_order_acquire) & bit) != 0) return;
  if (hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, bytes) == hipSuccess)
    done->fetch_or(bit, std::memory_order_acq_rel);
}

template <int D>
oda_status launch_layers(const AttnArgs& args, hipStream_t stream) {
  const int64_t items = (int64_t)(args.L / args.lpi) * args.B * args.Hkv;
  if (items > 0x7fffffffLL) return oda::fail(ODA_ERR_SHAPE, "grid too large (%lld work items)", (long long)items);
  const size_t lds = split_lds_floats(args.G, D) * sizeof(float);
  static std::atomic<uint64_t> lds_raised{0};
  raise_lds_limit(reinterpret_cast<const void*>(attn_local_layers_kernel<D>), &lds_raised,
                  (int)(split_lds_floats(kMaxGroup, D) * 4));
  (void)hipGetLastError();
  hipLaunchKernelGGL(attn_local_layers_kernel<D>, dim3((unsigned)items), dim3(kWaves * 64), lds, stream, args);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return oda::fail(ODA_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return ODA_OK;
}

template <int D, bool kLocal>
oda_status launch(const AttnArgs& args, const Plan& plan, hipStream_t stream) {
  if (kLocal && args.lpi > 1) return launch_layers<D>(args, stream);
  const int64_t items = (int64_t)args.L * args.Hkv * (kLocal ? (int64_t)args.B * plan.local_splits : plan.full_slots);
  if (items > 0x7fffffffLL) return oda::fail(ODA_ERR_SHAPE, "grid too large (%lld work items)", (long long)items);
  const size_t lds = split_lds_floats(args.G, D) * sizeof(float) + (args.qkv ? prep_lds_bytes(args.G, D) : 0);
  static std::atomic<uint64_t> lds_raised{0};
  raise_lds_limit(reinterpret_cast<const void*>(attn_split_kernel<D, kLocal>), &lds_raised,
                  (int)(split_lds_floats(kMaxGroup, D) * 4 + prep_lds_bytes(kMaxGroup, D)));
  (void)hipGetLastError();
  hipLaunchKernelGGL((attn_split_kernel<D, kLocal>), dim3((unsigned)items), dim3(kWaves * 64), lds, stream, args);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return oda::fail(ODA_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return ODA_OK;
}

oda_status run_attention(const oda_attn_shape* s, const oda_attn_inputs* in, bool local, int n_sink, int window,
                         int select, const int32_t* flags, const int32_t* work_list, const int32_t* n_work,
                         float* out, float* lse, void* ws, size_t ws_bytes, hipStream_t stream,
                         const oda_qkv_prep* prep = nullptr, const uint16_t* k_ring = nullptr,
                         const uint16_t* v_ring = nullptr) {
  Plan plan;
  // Local attends every request; Full is sized for the fewest selected (one)
  make_plan(s, n_sink, window, &plan);
  if (plan.bytes > 0) {
    if (ws == nullptr) return oda::fail(ODA_ERR_WORKSPACE, "workspace is NULL (%zu bytes needed)", plan.bytes);
    if (ws_bytes < plan.bytes)
      return oda::fail(ODA_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", ws_bytes, plan.bytes);
    if (!oda::aligned(ws, 256)) return oda::fail(ODA_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  }
  AttnArgs a;
  a.q = in->q;
  a.k_cache = in->k_cache;
  a.v_cache = in->v_cache;
  a.block_table = in->block_table;
  a.seq_lens = in->seq_lens;
  a.k_cur = in->k_cur;
  a.v_cur = in->v_cur;
  a.flags = flags;
  a.work_list = work_list;
  a.n_work = n_work;
  a.out = out;
  a.lse = lse;
  a.part_o = plan.bytes ? reinterpret_cast<float*>(static_cast<char*>(ws) + plan.off_o) : nullptr;
  a.part_ml = plan.bytes ? reinterpret_cast<float*>(static_cast<char*>(ws) + plan.off_ml) : nullptr;
  a.tickets = plan.bytes != 0 ? static_cast<uint32_t*>(ws) : nullptr;
  a.kv_layer_stride = s->layer_stride_kv != 0 ? s->layer_stride_kv : s->num_blocks * s->num_kv_heads * kBlock * s->head_dim;
  a.max_len = s->max_seq_len;
  a.num_blocks = s->num_blocks;
  a.L = s->num_layers;
  a.B = s->batch;
  a.Hq = s->num_q_heads;
  a.Hkv = s->num_kv_heads;
  a.G = s->num_q_heads / s->num_kv_heads;
  a.MB = s->max_blocks_per_seq;
  a.n_sink = n_sink;
  a.window = window;
  a.has_cur = (in->k_cur != nullptr || prep != nullptr) ? 1 : 0;
  a.qkv = prep ? prep->qkv : nullptr;
  a.q_gain = prep ? prep->q_gain : nullptr;
  a.k_gain = prep ? prep->k_gain : nullptr;
  a.k_out = prep ? prep->k_out : nullptr;
  a.v_out = prep ? prep->v_out : nullptr;
  a.rope_theta = prep ? prep->rope_theta : 0.0;
  a.rms_eps = prep ? prep->rms_eps : 0.f;
  a.k_ring = k_ring;
  a.v_ring = v_ring;
  const oda::RingGeometry rg = oda::ring_geometry(n_sink, window > 0 ? window : 1);
  a.ring_sb = k_ring ? rg.sink_blocks : 0;
  a.ring_rb = k_ring ? rg.ring_blocks : 1;
  a.bps = plan.bps;
  a.max_splits = plan.max_splits;
  a.dyn_splits = plan.dyn;
  a.split_cap = plan.split_cap;
  a.nvb_max = plan.nvb_max;
  a.lpi = local ? layers_per_item(s, plan) : 1;
  a.select = select;
  a.scale_log2 = in->scale * kLog2e;
  oda_status st;
  if (s->head_dim == 128)
    st = local ? launch<128, true>(a, plan, stream) : launch<128, false>(a, plan, stream);
  else
    st = local ? launch<64, true>(a, plan, stream) : launch<64, false>(a, plan, stream);
  if (st != ODA_OK) return st;
  return oda::ok();
}

}  // namespace

extern "C" oda_status oda_attn_workspace_size(const oda_attn_shape* shape, int32_t n_sink, int32_t window,
                                              size_t* bytes) {
  oda_status st = check_shape(shape);
  if (st != ODA_OK) return st;
  if (bytes == nullptr) return oda::fail(ODA_ERR_NULL, "bytes is NULL");
  if (n_sink < 0 || window < 0) return oda::fail(ODA_ERR_SHAPE, "n_sink and window must be >= 0");
  Plan plan;
  make_plan(shape, n_sink, window, &plan);   // covers Local and Full calls of this shape
  *bytes = plan.bytes;
  return oda::ok();
}

extern "C" oda_status oda_local_decode_attn(const oda_attn_shape* shape, const oda_attn_inputs* in,
                                           int32_t n_sink, int32_t window, float* out, float* lse,
                                           void* workspace, size_t workspace_bytes, hipStream_t stream) {
  oda_status st = check_shape(shape);
  if (st != ODA_OK) return st;
  st = check_inputs(in, out);
  if (st != ODA_OK) return st;
  if (n_sink < 0) return oda::fail(ODA_ERR_SHAPE, "n_sink must be >= 0");
  if (window < 1) return oda::fail(ODA_ERR_SHAPE, "window must be >= 1 for Local attention");
  return run_attention(shape, in, true, n_sink, window, kSelAll, nullptr, nullptr, nullptr, out, lse, workspace,
                       workspace_bytes, stream);
}

extern "C" oda_status oda_local_decode_attn_qkv(const oda_attn_shape* shape, const oda_attn_inputs* in,
                                               const oda_qkv_prep* prep, int32_t n_sink, int32_t window, float* out,
                                               float* lse, void* workspace, size_t workspace_bytes,
                                               hipStream_t stream) {
  oda_status st = check_shape(shape);
  if (st != ODA_OK) return st;
  if (prep == nullptr) return oda::fail(ODA_ERR_NULL, "prep is NULL");
  st = check_inputs(in, out, shape, prep);
  if (st != ODA_OK) return st;
  if (n_sink < 0) return oda::fail(ODA_ERR_SHAPE, "n_sink must be >= 0");
  if (window < 1) return oda::fail(ODA_ERR_SHAPE, "window must be >= 1 for Local attention");
  return run_attention(shape, in, true, n_sink, window, kSelAll, nullptr, nullptr, nullptr, out, lse, workspace,
                       workspace_bytes, stream, prep);
}

extern "C" oda_status oda_full_decode_attn_qkv(const oda_attn_shape* shape, const oda_attn_inputs* in,
                                              const oda_qkv_prep* prep, int32_t native_window,
                                              const int32_t* flags, const int32_t* work_list,
                                              const int32_t* n_work, float* out, float* lse, void* workspace,
                                              size_t workspace_bytes, hipStream_t stream) {
  oda_status st = check_shape(shape);
  if (st != ODA_OK) return st;
  if (prep == nullptr) return oda::fail(ODA_ERR_NULL, "prep is NULL");
  st = check_inputs(in, out, shape, prep);
  if (st != ODA_OK) return st;
  if (native_window < 0) return oda::fail(ODA_ERR_SHAPE, "native_window must be >= 0");
  if ((work_list == nullptr) != (n_work == nullptr))
    return oda::fail(ODA_ERR_NULL, "work_list and n_work must both be NULL or both be set");
  const int select = work_list ? kSelList : (flags ? kSelFlags : kSelAll);
  return run_attention(shape, in, false, 0, native_window, select, flags, work_list, n_work, out, lse, workspace,
                       workspace_bytes, stream, prep);
}

extern "C" oda_status oda_full_decode_attn(const oda_attn_shape* shape, const oda_attn_inputs* in,
                                          int32_t native_window, const int32_t* flags,
                                          const int32_t* work_list, const int32_t* n_work, float* out,
                                          float* lse, void* workspace, size_t workspace_bytes,
                                          hipStream_t stream) {
  oda_status st = check_shape(shape);
  if (st != ODA_OK) return st;
  st = check_inputs(in, out);
  if (st != ODA_OK) return st;
  if (native_window < 0) return oda::fail(ODA_ERR_SHAPE, "native_window must be >= 0");
  if ((work_list == nullptr) != (n_work == nullptr))
    return oda::fail(ODA_ERR_NULL, "work_list and n_work must both be NULL or both be set");
  const int select = work_list ? kSelList : (flags ? kSelFlags : kSelAll);
  return run_attention(shape, in, false, 0, native_window, select, flags, work_list, n_work, out, lse, workspace,
                       workspace_bytes, stream);
}

extern "C" oda_status oda_ring_elements(const oda_attn_shape* shape, int32_t n_sink, int32_t window,
                                        int64_t* elements) {
  oda_status st = check_shape(shape);
  if (st != ODA_OK) return st;
  if (elements == nullptr) return oda::fail(ODA_ERR_NULL, "elements is NULL");
  if (n_sink < 0 || window < 1) return oda::fail(ODA_ERR_SHAPE, "n_sink >= 0 and window >= 1 required");
  const oda::RingGeometry rg = oda::ring_geometry(n_sink, window);
  *elements = (int64_t)shape->num_layers * shape->batch * (rg.sink_blocks + rg.ring_blocks) * shape->num_kv_heads *
              kBlock * shape->head_dim;
  return oda::ok();
}

extern "C" oda_status oda_local_decode_attn_ring(const oda_attn_shape* shape, const oda_attn_inputs* in,
                                                const uint16_t* k_ring, const uint16_t* v_ring, int32_t n_sink,
                                                int32_t window, float* out, float* lse, void* workspace,
                                                size_t workspace_bytes, hipStream_t stream) {
  oda_status st = check_shape(shape);
  if (st != ODA_OK) return st;
  if (in == nullptr) return oda::fail(ODA_ERR_NULL, "inputs is NULL");
  if (!in->q || !in->seq_lens || !out || !k_ring || !v_ring)
    return oda::fail(ODA_ERR_NULL, "q, seq_lens, out, k_ring and v_ring are required");
  if ((in->k_cur == nullptr) != (in->v_cur == nullptr))
    return oda::fail(ODA_ERR_NULL, "k_cur and v_cur must both be NULL or both be set");
  if (!oda::aligned(in->q, 16) || !oda::aligned(k_ring, 16) || !oda::aligned(v_ring, 16) || !oda::aligned(out, 16) ||
      (in->k_cur && (!oda::aligned(in->k_cur, 16) || !oda::aligned(in->v_cur, 16))))
    return oda::fail(ODA_ERR_SHAPE, "q, rings, k_cur, v_cur and out must be 16-byte aligned");
  if (!(in->scale > 0.f) || !std::isfinite(in->scale))
    return oda::fail(ODA_ERR_SHAPE, "scale must be finite and > 0");
  if (n_sink < 0) return oda::fail(ODA_ERR_SHAPE, "n_sink must be >= 0");
  if (window < 1) return oda::fail(ODA_ERR_SHAPE, "window must be >= 1 for Local attention");
  return run_attention(shape, in, true, n_sink, window, kSelAll, nullptr, nullptr, nullptr, out, lse, workspace,
                       workspace_bytes, stream, nullptr, k_ring, v_ring);
}
