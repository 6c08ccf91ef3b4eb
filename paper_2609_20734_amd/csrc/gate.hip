// Recall gate on gfx950: the recall score (head of App. A.2, or the two-layer
// MLP stand-in) and the device predicate of §2.1 / Alg. 1 (Full iff the score
// exceeds the threshold or is nonfinite), with on-device compaction of the
// flagged requests.  No score is read by the host (App. A.5).
//
// fp32 weights and arithmetic (App. A.2).  Each dense layer is one launch of a
// batched GEMV kernel: an item is a group of R output rows for a tile of up to
// 8 requests; its rows are streamed with 16-byte loads, several 256-float
// chunks in flight, and every input load serves all R rows (the weights are
// read once per batch tile).  Long rows split K over the four wavefronts of a
// workgroup, which combine their sums in LDS.  RMSNorm of a layer's input is
// folded into the same pass (the sum of squares is accumulated next to the
// dot products), so normalised inputs are never stored.
//
// The layers of the head are dependent launches on one stream.  For one or
// two requests with towers up to 512 wide, each residual SwiGLU block is a
// single launch (its hidden units split over the workgroups, the down
// projection left as partial sums that the next launch adds in a fixed
// order): five launches instead of seven.  A single launch stepping through
// the layers with a barrier over its workgroups was slower on this part:
// publishing each layer's results across the chip's L2 slices needs a
// write-back and an invalidate per workgroup per layer, which costs more than
// a kernel boundary.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <utility>

#include "oda.h"
#include "oda_internal.h"

namespace {

constexpr int kBatchTile = 8;     // requests per wavefront
constexpr int kWaves = 4;         // wavefronts per workgroup

enum Mode { kTower = 0, kMlpHidden = 1, kGateUp = 3, kDown = 4 };

struct LinArgs {
  const float* W;        // [rows][K] (kTower: tower 0's weight; the others follow at w_stride)
  const float* W2;       // kGateUp: the up projection [rows][K]
  const float* bias;     // [rows] or per tower at w_stride
  const float* gain;     // RMSNorm gain [K] (kTower: per tower at w_stride; kGateUp)
  const float* X[3];     // inputs [B][K] (kTower: three; else X[0])
  const float* aux;      // fusion: tower outputs [3][B][dt]; kDown: residual [B][rows]
  float* Y;              // outputs
  int64_t w_stride;      // kTower: floats between the towers' parameter segments
  int rows, K, B, dt;
  float eps;
};

__device__ __forceinline__ float silu(float x) { return x / (1.f + __expf(-x)); }
__device__ __forceinline__ float gelu(float x) { return 0.5f * x * (1.f + erff(x * 0.70710678118654752f)); }
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) x += __shfl_xor(x, s);
  return x;
}
__device__ __forceinline__ float dot4(float4 a, float4 b) { return a.x * b.x + a.y * b.y + a.z * b.z + a.w * b.w; }
__device__ __forceinline__ float4 mul4(float4 a, float4 b) { return make_float4(a.x * b.x, a.y * b.y, a.z * b.z, a.w * b.w); }
__device__ __forceinline__ float4 absdiff4(float4 a, float4 b) {
  return make_float4(fabsf(a.x - b.x), fabsf(a.y - b.y), fabsf(a.z - b.z), fabsf(a.w - b.w));
}
__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }
// p[0..3] if ok, else zeros.  The load itself is unconditional (from `safe`,
// any valid address, when !ok) and the value is selected afterwards: a
// conditional load would make the compiler select between the global
// address and a stack copy of the zeros (scratch plus flat loads).
__device__ __forceinline__ float4 load4_or_zero(const float* p, const float* safe, bool ok) {
  const float4 v = *reinterpret_cast<const float4*>(ok ? p : safe);
  return ok ? v : make_float4(0.f, 0.f, 0.f, 0.f);
}

// One dense layer for a (row group, batch tile) item.  R consecutive output
// rows share every load of the inputs (R > 1 when several requests are
// batched, so the inputs are not re-read per row); S wavefronts of the
// workgroup split K between them, chunk c going to wavefront c mod S (S = 4
// for long rows, so that one launch has enough loads in flight to cover HBM
// latency), and combine their sums through LDS.  S = 1: every wavefront of
// the workgroup owns an item of its own.
template <int MODE, int R, int S>
__global__ __launch_bounds__(256) void gate_linear_kernel(LinArgs p) {
  constexpr bool kNorm = (MODE == kTower || MODE == kGateUp);
  constexpr bool kTwo = (MODE == kGateUp);
  constexpr int kAcc = R * kBatchTile;
  static_assert(S == 1 || S == kWaves, "K is split over all wavefronts or none");
  __shared__ float sm[S > 1 ? kWaves : 1][S > 1 ? (kTwo ? 2 : 1) * kAcc + kBatchTile : 1];
  const int lane = threadIdx.x & 63;
  const int wave = uniform(threadIdx.x >> 6);
  const int item = S == 1 ? blockIdx.x * kWaves + wave : blockIdx.x;
  const int part = S == 1 ? 0 : wave;
  const int groups = p.rows / R;             // the host keeps rows (and dt) multiples of R
  const int rg = item % groups;
  const int b0 = (item / groups) * kBatchTile;
  if (b0 >= p.B) return;                     // uniform over the workgroup when S > 1
  const int nb = min(kBatchTile, p.B - b0);

  const float* W = p.W;
  const float* bias = p.bias;
  const float* gain = p.gain;
  const float* X = p.X[0];
  int tower = 0, row0 = rg * R;
  if (MODE == kTower) {                      // dt % R == 0: a group never straddles two towers
    tower = row0 / p.dt;
    row0 -= tower * p.dt;
    W += tower * p.w_stride;
    bias += tower * p.w_stride;
    gain += tower * p.w_stride;
    X = p.X[tower];
  }
  const float* wrow = W + (int64_t)row0 * p.K;
  const float* wrow2 = kTwo ? p.W2 + (int64_t)row0 * p.K : nullptr;
  // the epilogue's bias or residual for the output this lane will hold (lane
  // j * 8 + bi: row j, request bi), read now so it is not a dependent load
  // after the reduction; clamped to a valid element for lanes without one
  float epi = 0.f;
  if (MODE != kGateUp) {
    const int ej = min(lane / kBatchTile, R - 1), eb = b0 + min(lane % kBatchTile, nb - 1);
    epi = MODE == kDown ? p.aux[(int64_t)eb * p.rows + row0 + ej] : bias[row0 + ej];
  }

  float acc[R][kBatchTile], acc2[kTwo ? R : 1][kBatchTile], ss[kBatchTile];
#pragma unroll
  for (int bi = 0; bi < kBatchTile; ++bi) {
    ss[bi] = 0.f;
#pragma unroll
    for (int j = 0; j < R; ++j) acc[j][bi] = 0.f;
#pragma unroll
    for (int j = 0; j < (kTwo ? R : 1); ++j) acc2[j][bi] = 0.f;
  }

  auto step = [&](int k) {
    float4 w[R], w2[kTwo ? R : 1];
#pragma unroll
    for (int j = 0; j < R; ++j) w[j] = *reinterpret_cast<const float4*>(wrow + (int64_t)j * p.K + k);
    if (kTwo) {
#pragma unroll
      for (int j = 0; j < R; ++j) w2[j] = *reinterpret_cast<const float4*>(wrow2 + (int64_t)j * p.K + k);
    }
    float4 gk = make_float4(1.f, 1.f, 1.f, 1.f);
    if (kNorm) gk = *reinterpret_cast<const float4*>(gain + k);
#pragma unroll
    for (int bi = 0; bi < kBatchTile; ++bi) {
      if (bi < nb) {
        const float4 x = *reinterpret_cast<const float4*>(X + (int64_t)(b0 + bi) * p.K + k);
        if (kNorm) ss[bi] += dot4(x, x);
        const float4 xg = kNorm ? mul4(x, gk) : x;
#pragma unroll
        for (int j = 0; j < R; ++j) {
          acc[j][bi] += dot4(w[j], xg);
          if (kTwo) acc2[j][bi] += dot4(w2[j], xg);
        }
      }
    }
  };
  // this wavefront's whole 256-float chunks (every lane busy), unrolled so
  // their loads overlap, then the ragged tail chunk if it is ours
  const int full = p.K / 256;
  const int mine_full = full > part ? (full - part + S - 1) / S : 0;
  constexpr int kUnroll = R == 1 ? 8 : 4;
  // items start at different chunks (wrapping round), so that the workgroups
  // of a launch do not all read the same stretch of the shared inputs at the
  // same time: they would queue on the same L2 channels
  const int rot = mine_full > 0 ? (int)((((uint32_t)item * 2654435761u) >> 8) % (uint32_t)mine_full) : 0;
#pragma unroll kUnroll
  for (int i = 0; i < mine_full; ++i) {
    int c = i + rot;
    c = c >= mine_full ? c - mine_full : c;
    step((part + c * S) * 256 + 4 * lane);
  }
  if (full % S == part && full * 256 + 4 * lane < p.K) step(full * 256 + 4 * lane);

  // reduce over the wavefront; lane j * 8 + bi keeps row j, request bi
  float v = 0.f, v2 = 0.f, my_ss = 0.f;
#pragma unroll
  for (int bi = 0; bi < kBatchTile; ++bi) {
    if (bi < nb) {
      const float s = kNorm ? wave_sum(ss[bi]) : 0.f;
      if (kNorm && lane == bi) my_ss = s;
#pragma unroll
      for (int j = 0; j < R; ++j) {
        const float t = wave_sum(acc[j][bi]);
        const float t2 = kTwo ? wave_sum(acc2[j][bi]) : 0.f;
        if (lane == j * kBatchTile + bi) {
          v = t;
          v2 = t2;
        }
      }
    }
  }
  if (S > 1) {   // combine the K parts: wave w's sums go to sm[w], wave 0 adds them in order
    if (lane < kAcc) {
      sm[wave][lane] = v;
      if (kTwo) sm[wave][kAcc + lane] = v2;
    }
    if (kNorm && lane < kBatchTile) sm[wave][(kTwo ? 2 : 1) * kAcc + lane] = my_ss;
    __syncthreads();
    if (wave != 0) return;
    if (lane < kAcc) {
      v = sm[0][lane];
      v2 = kTwo ? sm[0][kAcc + lane] : 0.f;
#pragma unroll
      for (int w = 1; w < S; ++w) {
        v += sm[w][lane];
        if (kTwo) v2 += sm[w][kAcc + lane];
      }
    }
    if (kNorm) {
      const int bi = lane % kBatchTile;
      my_ss = sm[0][(kTwo ? 2 : 1) * kAcc + bi];
#pragma unroll
      for (int w = 1; w < S; ++w) my_ss += sm[w][(kTwo ? 2 : 1) * kAcc + bi];
    }
  } else if (kNorm) {
    my_ss = __shfl(my_ss, lane % kBatchTile);   // lane j * 8 + bi needs request bi's sum of squares
  }
  const int j = lane / kBatchTile, bi = lane % kBatchTile;
  if (lane >= kAcc || bi >= nb) return;
  const int b = b0 + bi;
  const int row = row0 + j;
  const float inv = kNorm ? rsqrtf(my_ss / (float)p.K + p.eps) : 1.f;
  if (MODE == kTower) {
    p.Y[((int64_t)tower * p.B + b) * p.dt + row] = silu(v * inv + epi);
  } else if (MODE == kMlpHidden) {
    p.Y[(int64_t)b * p.rows + row] = gelu(v + epi);
  } else if (MODE == kGateUp) {
    p.Y[(int64_t)b * p.rows + row] = silu(v * inv) * (v2 * inv);
  } else {  // kDown
    p.Y[(int64_t)b * p.rows + row] = epi + v;
  }
}

// Fusion layer of App. A.2: z0 = (a + b + c + SiLU(W_f u + b_f)) / 2 with the
// interaction vector u = [a; b; c; a*b; |a-b|; a*c; |a-c|; b*c; |b-c|].  Item:
// one output row for a batch tile.  Lanes walk the tower index m four at a
// time and build the nine parts of u for those m in registers, so u is never
// stored and W_f's nine column blocks are read with coalesced 16-byte loads.
// S wavefronts share an item, taking alternate 256-wide steps of m, and add
// their sums through LDS (S > 1 for wide towers, so that the launch has
// enough wavefronts in flight).
template <int S>
__global__ __launch_bounds__(256) void gate_fusion_kernel(LinArgs p) {
  static_assert(kWaves % S == 0, "items per workgroup");
  __shared__ float sm[S > 1 ? kWaves : 1][kBatchTile];
  const int lane = threadIdx.x & 63;
  const int wave = uniform(threadIdx.x >> 6);
  const int part = wave % S;
  const int item = blockIdx.x * (kWaves / S) + wave / S;
  const int row = item % p.rows;
  const int b0 = (item / p.rows) * kBatchTile;
  const bool valid = b0 < p.B;
  const int nb = valid ? min(kBatchTile, p.B - b0) : 0;
  const int dt = p.dt;
  const float* wrow = p.W + (int64_t)row * 9 * dt;
  const float* abc = p.aux;
  // the epilogue's operands for request b0 + lane (a + b + c at this row and
  // the bias), read before the main loop; clamped for lanes without one
  float s3 = 0.f, brow = 0.f;
  if (valid) {
    const int eb = b0 + min(lane, nb - 1);
    s3 = abc[((int64_t)0 * p.B + eb) * dt + row] + abc[((int64_t)1 * p.B + eb) * dt + row] +
         abc[((int64_t)2 * p.B + eb) * dt + row];
    brow = p.bias[row];
  }
  float acc[kBatchTile];
#pragma unroll
  for (int bi = 0; bi < kBatchTile; ++bi) acc[bi] = 0.f;
  for (int m = (part * 64 + lane) * 4; valid && m < dt; m += 256 * S) {
    float4 w[9];
#pragma unroll
    for (int q = 0; q < 9; ++q) w[q] = *reinterpret_cast<const float4*>(wrow + q * dt + m);
#pragma unroll
    for (int bi = 0; bi < kBatchTile; ++bi) {
      if (bi < nb) {
        const int b = b0 + bi;
        const float4 a = *reinterpret_cast<const float4*>(abc + ((int64_t)0 * p.B + b) * dt + m);
        const float4 bb = *reinterpret_cast<const float4*>(abc + ((int64_t)1 * p.B + b) * dt + m);
        const float4 c = *reinterpret_cast<const float4*>(abc + ((int64_t)2 * p.B + b) * dt + m);
        acc[bi] += dot4(w[0], a) + dot4(w[1], bb) + dot4(w[2], c) + dot4(w[3], mul4(a, bb)) +
                   dot4(w[4], absdiff4(a, bb)) + dot4(w[5], mul4(a, c)) + dot4(w[6], absdiff4(a, c)) +
                   dot4(w[7], mul4(bb, c)) + dot4(w[8], absdiff4(bb, c));
      }
    }
  }
  float mine = 0.f;
#pragma unroll
  for (int bi = 0; bi < kBatchTile; ++bi) {
    if (bi < nb) {
      const float v = wave_sum(acc[bi]);
      if (lane == bi) mine = v;
    }
  }
  if (S > 1) {   // the item's S partial sums, added in order by its first wavefront
    if (lane < kBatchTile) sm[wave][lane] = mine;
    __syncthreads();
    if (part != 0) return;
    if (lane < kBatchTile) {
#pragma unroll
      for (int q = 1; q < S; ++q) mine += sm[wave + q][lane];
    }
  }
  if (lane >= nb) return;
  const int b = b0 + lane;
  p.Y[(int64_t)b * p.rows + row] = 0.5f * (s3 + silu(mine + brow));
}

constexpr int kSplitMaxB = 2;         // batches up to this size may take the split-hidden blocks
constexpr int kSplitMaxDt = 512;      // tower widths up to this take them (two 256-wide chunks per row)
constexpr int kSplitMaxHs = 16;       // hidden units per workgroup (4 per wavefront)

// out[e] = base[e] + sum_w parts[w][e] for e < n (n a multiple of 4, n / 4 <=
// kSplitMaxB * kSplitMaxDt / 4), into LDS, by a workgroup of exactly NT threads:
// groups of threads take interleaved partials, eight loads in flight each,
// and the group sums are then added in group order (a fixed order).
template <int NT>
__device__ __forceinline__ void sum_parts(const float* base, const float* parts, int nparts, int n, float* out,
                                          float4* scratch) {
  const int C = n / 4;
  const int Cg = min(C, NT);
  const int G = NT / Cg;
  const int t = threadIdx.x;
  const int g = t / Cg, cl = t % Cg;
  if (g < G) {
    for (int c = cl; c < C; c += Cg) {
      float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int w0 = g; w0 < nparts; w0 += 8 * G) {
        float4 v[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int w = w0 + i * G;
          v[i] = load4_or_zero(parts + (int64_t)w * n + 4 * c, parts, w < nparts);
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) acc = make_float4(acc.x + v[i].x, acc.y + v[i].y, acc.z + v[i].z, acc.w + v[i].w);
      }
      scratch[g * C + c] = acc;
    }
  }
  __syncthreads();
  for (int c = t; c < C; c += NT) {
    float4 v = *reinterpret_cast<const float4*>(base + 4 * c);
    for (int gg = 0; gg < G; ++gg) {
      const float4 u = scratch[gg * C + c];
      v = make_float4(v.x + u.x, v.y + u.y, v.z + u.z, v.w + u.w);
    }
    *reinterpret_cast<float4*>(out + 4 * c) = v;
  }
  __syncthreads();
}

// LDS float4 slots sum_parts needs: max(NT, n / 4)
constexpr int kPartsScratch = kSplitMaxB * kSplitMaxDt / 4;

struct FinalArgs {
  const float* X;       // [B][K]: z2 (paper head) or the MLP hidden layer
  const float* gain;    // paper head: final RMSNorm gain [K]; MLP: NULL
  const float* w;       // [K]
  const float* bias;    // [1]
  const int32_t* forced;
  float* score;
  int32_t* flags;
  int32_t* work_list;
  int32_t* n_work;
  int64_t* counter;
  const float* parts;   // NULL, or [nparts][B][K] partial sums added to X (split-hidden blocks)
  int nparts;
  int K, B;
  float eps, tau;
};

constexpr int kFinalWaves = 16;

// The scalar projection q = w . RMSNorm(x) + b (w . x + b without a gain) for
// every request, spread over the workgroup's wavefronts 64 requests at a
// time, then the decision and the ascending compaction of the flagged
// requests (ballot + prefix popcount) by wavefront 0.
__global__ __launch_bounds__(kFinalWaves * 64) void gate_final_kernel(FinalArgs p) {
  __shared__ float sm_score[64];
  __shared__ float sx[kSplitMaxB * kSplitMaxDt];
  __shared__ float4 sscratch[kPartsScratch > kFinalWaves * 64 ? kPartsScratch : kFinalWaves * 64];
  const int lane = threadIdx.x & 63;
  const int wave = uniform(threadIdx.x >> 6);
  const bool norm = p.gain != nullptr;
  // the projection w (times the gain) of this lane's first two 256-wide
  // chunks, loaded before the input so its latency overlaps the gathering
  constexpr int kPre = 2;
  float4 wpre[kPre];
#pragma unroll
  for (int c = 0; c < kPre; ++c) {
    const int k = 4 * lane + 256 * c;
    const bool in = k < p.K;
    wpre[c] = load4_or_zero(p.w + k, p.w, in);
    if (norm) wpre[c] = mul4(wpre[c], load4_or_zero(p.gain + k, p.gain, in));
  }
  // split-hidden blocks (B <= kSplitMaxB): z = residual + the last block's
  // partial sums, formed once in LDS by the whole workgroup
  const bool parts = p.parts != nullptr;
  if (parts) sum_parts<kFinalWaves * 64>(p.X, p.parts, p.nparts, p.B * p.K, sx, sscratch);
  const float* X = parts ? sx : p.X;
  int total = 0;
  for (int c0 = 0; c0 < p.B; c0 += 64) {
    const int nc = min(64, p.B - c0);
    for (int i = wave; i < nc; i += kFinalWaves) {
      const int b = c0 + i;
      float dot = 0.f, ss = 0.f;
#pragma unroll
      for (int c = 0; c < kPre; ++c) {
        const int k = 4 * lane + 256 * c;
        if (k < p.K) {
          const float4 x = *reinterpret_cast<const float4*>(X + (int64_t)b * p.K + k);
          if (norm) ss += dot4(x, x);
          dot += dot4(wpre[c], x);
        }
      }
      for (int k = 4 * lane + 256 * kPre; k < p.K; k += 256) {
        const float4 x = *reinterpret_cast<const float4*>(X + (int64_t)b * p.K + k);
        float4 wk = *reinterpret_cast<const float4*>(p.w + k);
        if (norm) {
          ss += dot4(x, x);
          wk = mul4(wk, *reinterpret_cast<const float4*>(p.gain + k));
        }
        dot += dot4(wk, x);
      }
      dot = wave_sum(dot);
      float s = dot;
      if (norm) s = dot * rsqrtf(wave_sum(ss) / (float)p.K + p.eps);
      if (lane == 0) sm_score[i] = s + p.bias[0];
    }
    __syncthreads();
    if (wave == 0) {
      const int b = c0 + lane;
      bool flag = false;
      if (lane < nc) {
        const float s = sm_score[lane];
        p.score[b] = s;
        flag = p.forced ? (p.forced[b] != 0) : (s > p.tau);
        flag = flag || !__builtin_isfinite(s);
        p.flags[b] = flag ? 1 : 0;
      }
      const uint64_t mask = __ballot(flag);
      if (flag && p.work_list) {
        const uint64_t below = lane ? (mask & ((~0ull) >> (64 - lane))) : 0ull;
        p.work_list[total + __popcll(below)] = b;
      }
      total += __popcll(mask);
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    if (p.n_work) p.n_work[0] = total;
    // integer add at the memory side: no round trip before the kernel can retire
    if (p.counter) atomicAdd(reinterpret_cast<unsigned long long*>(p.counter), (unsigned long long)total);
  }
}

// ---------------------------------------------------------------------------
// split-hidden SwiGLU block (small batches)
// ---------------------------------------------------------------------------

struct SplitArgs {
  const float* z_base;     // [B][dt]: the block's residual input, before the incoming partial sums
  const float* parts_in;   // NULL, or [nparts_in][B][dt] partial down sums of the previous block
  float* z_out;            // NULL, or where workgroup 0 stores z_base + sum(parts_in) (the next residual)
  const float* gain;       // [dt] the block's RMSNorm gain
  const float* Wg;         // [2dt][dt]
  const float* Wu;         // [2dt][dt]
  const float* Wd;         // [dt][2dt]
  float* parts_out;        // [gridDim.x][B][dt]
  int nparts_in, dt, B, hs;
  float eps;
};

// One residual SwiGLU block, z_out = z + W_d (SiLU(W_g n) * (W_u n)) with
// n = RMSNorm(z), in one launch: workgroup w owns hidden units
// [w hs, (w + 1) hs), computes them from the whole input, and writes its share
// of the down projection, sum over its units of W_d[:, j] h_j, as a partial
// sum.  The next launch adds the partial sums in a fixed order, so the block
// needs no grid-wide barrier and the result does not depend on timing.  The
// workgroup's weights (HW hidden units per wavefront, KC 256-wide chunks per
// row, and its W_d columns) are loaded first, so their latency overlaps the
// gathering of the block input.
template <int HW, int KC>
__global__ __launch_bounds__(256) void gate_split_block_kernel(SplitArgs p) {
  __shared__ float sz[kSplitMaxB * kSplitMaxDt];
  __shared__ float sh[kSplitMaxB * kSplitMaxHs];
  __shared__ float sred[kWaves][kSplitMaxB];
  __shared__ float4 sscratch[kPartsScratch > 256 ? kPartsScratch : 256];
  const int lane = threadIdx.x & 63;
  const int wave = uniform(threadIdx.x >> 6);
  const int n = p.B * p.dt;
  const int hs = HW * kWaves;
  const float4 zero = make_float4(0.f, 0.f, 0.f, 0.f);
  // this workgroup's weights
  float4 wg[HW][KC], wu[HW][KC], gk[KC], wd[KC][HW];
  const int j0 = blockIdx.x * hs + wave * HW;
  const int jb = blockIdx.x * hs;
#pragma unroll
  for (int c = 0; c < KC; ++c) {
    const int k = c * 256 + 4 * lane;
    const bool in = k < p.dt;
    gk[c] = load4_or_zero(p.gain + k, p.gain, in);
#pragma unroll
    for (int jj = 0; jj < HW; ++jj) {
      wg[jj][c] = load4_or_zero(p.Wg + (int64_t)(j0 + jj) * p.dt + k, p.Wg, in);
      wu[jj][c] = load4_or_zero(p.Wu + (int64_t)(j0 + jj) * p.dt + k, p.Wu, in);
    }
    const int r = threadIdx.x + 256 * c;
#pragma unroll
    for (int q = 0; q < HW; ++q) wd[c][q] = load4_or_zero(p.Wd + (int64_t)r * 2 * p.dt + jb + 4 * q, p.Wd, r < p.dt);
  }
  // the block input for every request: the residual plus the previous block's partial sums
  sum_parts<256>(p.z_base, p.parts_in, p.nparts_in, n, sz, sscratch);
  if (p.z_out != nullptr && blockIdx.x == 0)
    for (int e = threadIdx.x; e < n; e += 256) p.z_out[e] = sz[e];
  float inv[kSplitMaxB];
#pragma unroll
  for (int b = 0; b < kSplitMaxB; ++b) {
    float ss = 0.f;
    if (b < p.B)
      for (int k = threadIdx.x; k < p.dt; k += 256) ss += sz[b * p.dt + k] * sz[b * p.dt + k];
    ss = wave_sum(ss);
    if (lane == 0) sred[wave][b] = ss;
  }
  __syncthreads();
#pragma unroll
  for (int b = 0; b < kSplitMaxB; ++b) {
    float t = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) t += sred[w][b];
    inv[b] = rsqrtf(t / (float)p.dt + p.eps);
  }
  // hidden units
#pragma unroll
  for (int b = 0; b < kSplitMaxB; ++b) {
    if (b < p.B) {
      float4 x[KC];
#pragma unroll
      for (int c = 0; c < KC; ++c) {
        const int k = c * 256 + 4 * lane;
        x[c] = k < p.dt ? mul4(*reinterpret_cast<const float4*>(sz + b * p.dt + k), gk[c]) : zero;
      }
#pragma unroll
      for (int jj = 0; jj < HW; ++jj) {
        float g = 0.f, u = 0.f;
#pragma unroll
        for (int c = 0; c < KC; ++c) {
          g += dot4(wg[jj][c], x[c]);
          u += dot4(wu[jj][c], x[c]);
        }
        g = wave_sum(g) * inv[b];
        u = wave_sum(u) * inv[b];
        if (lane == 0) sh[b * hs + wave * HW + jj] = silu(g) * u;
      }
    }
  }
  __syncthreads();
  // this workgroup's share of the down projection for every output row
#pragma unroll
  for (int c = 0; c < KC; ++c) {
    const int r = threadIdx.x + 256 * c;
    if (r < p.dt) {
#pragma unroll
      for (int b = 0; b < kSplitMaxB; ++b) {
        if (b < p.B) {
          float acc = 0.f;
#pragma unroll
          for (int q = 0; q < HW; ++q) acc += dot4(wd[c][q], *reinterpret_cast<const float4*>(sh + b * hs + 4 * q));
          p.parts_out[((int64_t)blockIdx.x * p.B + b) * p.dt + r] = acc;
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------

struct HeadLayout {   // float offsets into the packed parameters (PAPER)
  int64_t tower_stride, tower_rms, tower_w, tower_b;
  int64_t wf, bf;
  int64_t block_stride, blk_rms, blk_gate, blk_up, blk_down;
  int64_t rms_o, w_o, b_o, total;
};

HeadLayout paper_layout(int64_t d, int64_t dt) {
  HeadLayout L;
  L.tower_stride = d + dt * d + dt;
  L.tower_rms = 0;
  L.tower_w = d;
  L.tower_b = d + dt * d;
  L.wf = 3 * L.tower_stride;
  L.bf = L.wf + 9 * dt * dt;
  const int64_t b0 = L.bf + dt;
  L.block_stride = dt + 6 * dt * dt;
  L.blk_rms = b0;
  L.blk_gate = b0 + dt;
  L.blk_up = b0 + dt + 2 * dt * dt;
  L.blk_down = b0 + dt + 4 * dt * dt;
  L.rms_o = b0 + 2 * L.block_stride;
  L.w_o = L.rms_o + dt;
  L.b_o = L.w_o + dt;
  L.total = L.b_o + 1;
  return L;
}

struct GateWs {
  size_t abc, z0, z1, hdn, p1, p2, hid, bytes;
};

// Workgroups of a split-hidden block (0 if the batch or width does not take
// that path): the most (at most 64) that split the hidden width 2 dt into
// equal shares of 4, 8 or 16 units, i.e. 1, 2 or 4 per wavefront (the block
// kernel's instances); the partial sums the next launch adds must stay small
// (<= 256 KiB per consumer workgroup).
int split_groups(int64_t B, int64_t dt) {
  if (B > kSplitMaxB || dt > kSplitMaxDt || dt % 4) return 0;
  for (int nw = 64; nw >= 1; nw /= 2) {
    if ((2 * dt) % nw) continue;
    const int64_t hs = 2 * dt / nw;
    if (hs != kWaves && hs != 2 * kWaves && hs != 4 * kWaves) continue;
    if ((int64_t)nw * B * dt * 4 > 256 * 1024) return 0;
    return nw;
  }
  return 0;
}

GateWs gate_ws_layout(int kind, int64_t B, int64_t dt) {
  GateWs w{};
  size_t off = 0;
  auto take = [&](int64_t floats) {
    const size_t o = off;
    off += (size_t)oda::round_up(floats * 4, 256);
    return o;
  };
  if (kind == ODA_HEAD_PAPER) {
    w.abc = take(3 * B * dt);
    w.z0 = take(B * dt);
    w.z1 = take(B * dt);
    w.hdn = take(2 * B * dt);
    const int nw = split_groups(B, dt);
    w.p1 = take((int64_t)nw * B * dt);
    w.p2 = take((int64_t)nw * B * dt);
  } else {
    w.hid = take(B * dt);
  }
  w.bytes = std::max<size_t>(off, 256);
  return w;
}

oda_status check_gate(const oda_gate_desc* g) {
  if (g == nullptr) return oda::fail(ODA_ERR_NULL, "gate is NULL");
  if (g->kind != ODA_HEAD_PAPER && g->kind != ODA_HEAD_MLP)
    return oda::fail(ODA_ERR_UNSUPPORTED, "unknown head kind %d", g->kind);
  if (g->d_model < 4 || g->d_hidden < 4 || g->d_model % 4 || g->d_hidden % 4)
    return oda::fail(ODA_ERR_SHAPE, "d_model (%d) and d_hidden (%d) must be positive multiples of 4",
                     g->d_model, g->d_hidden);
  if (!(g->rms_eps >= 0.f) || !std::isfinite(g->rms_eps)) return oda::fail(ODA_ERR_SHAPE, "rms_eps must be >= 0");
  return ODA_OK;
}

template <int MODE, int R, int S>
void launch_linear_rs(const LinArgs& a, hipStream_t stream) {
  const int64_t items = (int64_t)(a.rows / R) * oda::ceil_div(a.B, kBatchTile);
  const int64_t groups = S == 1 ? oda::ceil_div(items, kWaves) : items;
  hipLaunchKernelGGL((gate_linear_kernel<MODE, R, S>), dim3((unsigned)groups), dim3(256), 0, stream, a);
}

// Launch shape of a dense layer.  K is split over the four wavefronts of a
// workgroup when rows are long (K >= 4096), or when there are too few items
// to occupy the chip (< 1024) and every wavefront still gets whole chunks.
// With more than two requests per tile, R = 4 (else 2) rows share each input
// load while that still leaves >= 512 workgroups.  With one or two, only the
// tower layer groups rows (R = 2, down to 256 workgroups): its inputs are
// d_model long, and re-reading them for every row cost more than the wider
// items (the d = 8192 head took 56 instead of 63 µs at B = 2); in the other
// layers grouping at small batches measured slower.
template <int MODE>
void launch_linear(const LinArgs& a, hipStream_t stream) {
  const int tiles = (int)oda::ceil_div(a.B, kBatchTile);
  const int per_tile = std::min(a.B, kBatchTile);
  const int unit = MODE == kTower ? a.dt : a.rows;   // R must divide it
  const int64_t items = (int64_t)a.rows * tiles;
  const bool split = a.K >= 4096 || (a.K >= 1024 && items < 1024);
  auto fits = [&](int r) {
    if (unit % r != 0) return false;
    const int64_t groups = items / r / (split ? 1 : kWaves);
    if (MODE == kTower && r == 2 && groups >= 256) return true;
    return per_tile > 2 && groups >= 512;
  };
  if (split) {
    if (fits(4)) return launch_linear_rs<MODE, 4, kWaves>(a, stream);
    if (fits(2)) return launch_linear_rs<MODE, 2, kWaves>(a, stream);
    return launch_linear_rs<MODE, 1, kWaves>(a, stream);
  }
  if (fits(4)) return launch_linear_rs<MODE, 4, 1>(a, stream);
  if (fits(2)) return launch_linear_rs<MODE, 2, 1>(a, stream);
  launch_linear_rs<MODE, 1, 1>(a, stream);
}

// Fusion launch: S wavefronts per item when the tower width allows S steps
// of 256 and the items alone would leave the chip under-occupied.
void launch_fusion(const LinArgs& a, hipStream_t stream) {
  const int64_t items = (int64_t)a.rows * oda::ceil_div(a.B, kBatchTile);
  const int steps = (int)oda::ceil_div(a.dt, 256);
  const int s = items >= 2048 ? 1 : steps >= 4 ? 4 : steps >= 2 ? 2 : 1;
  const unsigned groups = (unsigned)oda::ceil_div(items * s, kWaves);
  if (s == 4) {
    hipLaunchKernelGGL(gate_fusion_kernel<4>, dim3(groups), dim3(256), 0, stream, a);
  } else if (s == 2) {
    hipLaunchKernelGGL(gate_fusion_kernel<2>, dim3(groups), dim3(256), 0, stream, a);
  } else {
    hipLaunchKernelGGL(gate_fusion_kernel<1>, dim3(groups), dim3(256), 0, stream, a);
  }
}

// Argument checks shared by both gate entry points (everything but the workspace).
oda_status check_gate_call(const oda_gate_desc* gate, int32_t batch, const float* h_prev, const float* emb,
                           const float* h_local, float tau, const float* score, const int32_t* flags,
                           const int32_t* work_list, const int32_t* n_work) {
  oda_status st = check_gate(gate);
  if (st != ODA_OK) return st;
  if (batch < 1) return oda::fail(ODA_ERR_SHAPE, "batch must be >= 1");
  const bool paper = gate->kind == ODA_HEAD_PAPER;
  if (!gate->params || !h_local || !score || !flags || (paper && (!h_prev || !emb)))
    return oda::fail(ODA_ERR_NULL, "params, h_local, score, flags (and h_prev, emb for the paper head) are required");
  if ((work_list == nullptr) != (n_work == nullptr))
    return oda::fail(ODA_ERR_NULL, "work_list and n_work must both be NULL or both be set");
  if (std::isnan(tau)) return oda::fail(ODA_ERR_SHAPE, "tau is NaN");
  if (!oda::aligned(gate->params, 16) || !oda::aligned(h_local, 16) ||
      (paper && (!oda::aligned(h_prev, 16) || !oda::aligned(emb, 16))))
    return oda::fail(ODA_ERR_SHAPE, "params and gate inputs must be 16-byte aligned");
  return ODA_OK;
}

// Enqueue the head, the decision and the compaction, with the intermediate
// activations in `workspace` (at least gate_ws_layout(...).bytes, 256-byte
// aligned; every byte the kernels read there was written earlier in the same
// call, so its contents on entry do not matter).
oda_status run_gate(const oda_gate_desc* gate, int32_t batch, const float* h_prev, const float* emb,
                    const float* h_local, float tau, const int32_t* forced, float* score, int32_t* flags,
                    int32_t* work_list, int32_t* n_work, int64_t* recall_counter, void* workspace,
                    hipStream_t stream) {
  const bool paper = gate->kind == ODA_HEAD_PAPER;
  const GateWs ws = gate_ws_layout(gate->kind, batch, gate->d_hidden);
  char* wsb = static_cast<char*>(workspace);
  const int d = gate->d_model, dt = gate->d_hidden;
  const float* P = gate->params;
  (void)hipGetLastError();
  FinalArgs fa{};
  fa.B = batch;
  fa.eps = gate->rms_eps;
  fa.tau = tau;
  fa.forced = forced;
  fa.score = score;
  fa.flags = flags;
  fa.work_list = work_list;
  fa.n_work = n_work;
  fa.counter = recall_counter;
  if (paper) {
    const HeadLayout H = paper_layout(d, dt);
    float* abc = reinterpret_cast<float*>(wsb + ws.abc);
    float* z0 = reinterpret_cast<float*>(wsb + ws.z0);
    float* z1 = reinterpret_cast<float*>(wsb + ws.z1);
    float* hdn = reinterpret_cast<float*>(wsb + ws.hdn);
    LinArgs a{};
    a.B = batch;
    a.dt = dt;
    a.eps = gate->rms_eps;
    // towers: a, b, c = SiLU(W_t RMSNorm(x_t) + b_t)
    a.W = P + H.tower_w;
    a.bias = P + H.tower_b;
    a.gain = P + H.tower_rms;
    a.w_stride = H.tower_stride;
    a.X[0] = h_prev;
    a.X[1] = emb;
    a.X[2] = h_local;
    a.Y = abc;
    a.rows = 3 * dt;
    a.K = d;
    launch_linear<kTower>(a, stream);
    // fusion: z0 = (a + b + c + SiLU(W_f u + b_f)) / 2
    a = LinArgs{};
    a.B = batch;
    a.dt = dt;
    a.eps = gate->rms_eps;
    a.W = P + H.wf;
    a.bias = P + H.bf;
    a.aux = abc;
    a.Y = z0;
    a.rows = dt;
    a.K = 9 * dt;
    launch_fusion(a, stream);
    const int nw = split_groups(batch, dt);
    if (nw > 0) {
      // two split-hidden blocks: z0 -> partials P1 -> (z1 = z0 + P1) -> partials P2;
      // the score adds P2 to z1
      float* p1 = reinterpret_cast<float*>(wsb + ws.p1);
      float* p2 = reinterpret_cast<float*>(wsb + ws.p2);
      for (int k = 0; k < 2; ++k) {
        const int64_t base = k * H.block_stride;
        SplitArgs sa{};
        sa.z_base = z0;
        sa.parts_in = k == 0 ? nullptr : p1;
        sa.nparts_in = k == 0 ? 0 : nw;
        sa.z_out = k == 0 ? nullptr : z1;
        sa.gain = P + H.blk_rms + base;
        sa.Wg = P + H.blk_gate + base;
        sa.Wu = P + H.blk_up + base;
        sa.Wd = P + H.blk_down + base;
        sa.parts_out = k == 0 ? p1 : p2;
        sa.dt = dt;
        sa.B = batch;
        sa.hs = 2 * dt / nw;
        sa.eps = gate->rms_eps;
        const int hw = sa.hs / kWaves;   // 1, 2 or 4: split_groups allows no other
        const dim3 g((unsigned)nw), t(256);
        if (dt <= 256) {
          if (hw == 1) hipLaunchKernelGGL((gate_split_block_kernel<1, 1>), g, t, 0, stream, sa);
          else if (hw == 2) hipLaunchKernelGGL((gate_split_block_kernel<2, 1>), g, t, 0, stream, sa);
          else hipLaunchKernelGGL((gate_split_block_kernel<4, 1>), g, t, 0, stream, sa);   // hw == 4
        } else {
          if (hw == 1) hipLaunchKernelGGL((gate_split_block_kernel<1, 2>), g, t, 0, stream, sa);
          else if (hw == 2) hipLaunchKernelGGL((gate_split_block_kernel<2, 2>), g, t, 0, stream, sa);
          else hipLaunchKernelGGL((gate_split_block_kernel<4, 2>), g, t, 0, stream, sa);   // hw == 4
        }
      }
      fa.X = z1;
      fa.parts = p2;
      fa.nparts = nw;
    } else {
      // two pre-RMSNorm residual SwiGLU blocks, one launch per dense layer
      float* zin = z0;
      float* zout = z1;
      for (int k = 0; k < 2; ++k) {
        const int64_t base = k * H.block_stride;
        a = LinArgs{};
        a.B = batch;
        a.dt = dt;
        a.eps = gate->rms_eps;
        a.W = P + H.blk_gate + base;
        a.W2 = P + H.blk_up + base;
        a.gain = P + H.blk_rms + base;
        a.X[0] = zin;
        a.Y = hdn;
        a.rows = 2 * dt;
        a.K = dt;
        launch_linear<kGateUp>(a, stream);
        a = LinArgs{};
        a.B = batch;
        a.dt = dt;
        a.W = P + H.blk_down + base;
        a.X[0] = hdn;
        a.aux = zin;
        a.Y = zout;
        a.rows = dt;
        a.K = 2 * dt;
        launch_linear<kDown>(a, stream);
        std::swap(zin, zout);
      }
      fa.X = zin;
    }
    // q = w_o . RMSNorm(z2) + b_o
    fa.gain = P + H.rms_o;
    fa.w = P + H.w_o;
    fa.bias = P + H.b_o;
    fa.K = dt;
  } else {
    float* hid = reinterpret_cast<float*>(wsb + ws.hid);
    LinArgs a{};
    a.B = batch;
    a.dt = dt;
    a.W = P;
    a.bias = P + (int64_t)dt * d;
    a.X[0] = h_local;
    a.Y = hid;
    a.rows = dt;
    a.K = d;
    launch_linear<kMlpHidden>(a, stream);
    fa.X = hid;
    fa.gain = nullptr;
    fa.w = P + (int64_t)dt * d + dt;
    fa.bias = P + (int64_t)dt * d + 2 * dt;
    fa.K = dt;
  }
  // one wavefront per request in flight, at most kFinalWaves; the whole
  // workgroup when it first adds up the last block's partial sums
  const int final_threads = fa.parts ? 64 * kFinalWaves : 64 * std::min(kFinalWaves, batch);
  hipLaunchKernelGGL(gate_final_kernel, dim3(1), dim3((unsigned)final_threads), 0, stream, fa);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return oda::fail(ODA_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return oda::ok();
}

// Workspace of oda_recall_gate_static: a file-scope device array, one copy
// per GPU, held until the process ends.  In host code its name is only a
// stand-in for the symbol; its device address on the current GPU is looked up
// once per device (kStaticDevices slots) and cached.
constexpr size_t kStaticScratchBytes = (size_t)16 << 20;
constexpr int kStaticDevices = 64;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];
std::atomic<void*> g_scratch_ptr[kStaticDevices];

oda_status static_scratch(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return oda::fail(ODA_ERR_HIP, "hipGetDevice failed: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kStaticDevices)
    return oda::fail(ODA_ERR_UNSUPPORTED, "device %d: the static workspace serves devices 0..%d", dev,
                     kStaticDevices - 1);
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (p == nullptr) {
    // threads racing here look up the same address and store the same value
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr)
      return oda::fail(ODA_ERR_HIP, "hipGetSymbolAddress of the static workspace failed: %s", hipGetErrorString(e));
    g_scratch_ptr[dev].store(p, std::memory_order_release);
  }
  *ptr = p;
  return ODA_OK;
}

}  // namespace

extern "C" oda_status oda_recall_gate(const oda_gate_desc* gate, int32_t batch, const float* h_prev,
                                     const float* emb, const float* h_local, float tau, const int32_t* forced,
                                     float* score, int32_t* flags, int32_t* work_list, int32_t* n_work,
                                     int64_t* recall_counter, void* workspace, size_t workspace_bytes,
                                     hipStream_t stream) {
  oda_status st = check_gate_call(gate, batch, h_prev, emb, h_local, tau, score, flags, work_list, n_work);
  if (st != ODA_OK) return st;
  const GateWs ws = gate_ws_layout(gate->kind, batch, gate->d_hidden);
  if (workspace == nullptr) return oda::fail(ODA_ERR_WORKSPACE, "workspace is NULL (%zu bytes needed)", ws.bytes);
  if (workspace_bytes < ws.bytes)
    return oda::fail(ODA_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", workspace_bytes, ws.bytes);
  if (!oda::aligned(workspace, 256)) return oda::fail(ODA_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  return run_gate(gate, batch, h_prev, emb, h_local, tau, forced, score, flags, work_list, n_work, recall_counter,
                  workspace, stream);
}

extern "C" oda_status oda_recall_gate_static(const oda_gate_desc* gate, int32_t batch, const float* h_prev,
                                            const float* emb, const float* h_local, float tau,
                                            const int32_t* forced, float* score, int32_t* flags,
                                            int32_t* work_list, int32_t* n_work, int64_t* recall_counter,
                                            hipStream_t stream) {
  oda_status st = check_gate_call(gate, batch, h_prev, emb, h_local, tau, score, flags, work_list, n_work);
  if (st != ODA_OK) return st;
  const GateWs ws = gate_ws_layout(gate->kind, batch, gate->d_hidden);
  if (ws.bytes > kStaticScratchBytes)
    return oda::fail(ODA_ERR_WORKSPACE, "this head and batch need %zu bytes of workspace; the static one holds %zu",
                     ws.bytes, kStaticScratchBytes);
  void* workspace = nullptr;
  st = static_scratch(&workspace);
  if (st != ODA_OK) return st;
  return run_gate(gate, batch, h_prev, emb, h_local, tau, forced, score, flags, work_list, n_work, recall_counter,
                  workspace, stream);
}

extern "C" oda_status oda_gate_param_count(int32_t kind, int32_t d_model, int32_t d_hidden, int64_t* count) {
  if (count == nullptr) return oda::fail(ODA_ERR_NULL, "count is NULL");
  if (d_model < 1 || d_hidden < 1) return oda::fail(ODA_ERR_SHAPE, "d_model and d_hidden must be >= 1");
  if (kind == ODA_HEAD_PAPER) {
    *count = paper_layout(d_model, d_hidden).total;
  } else if (kind == ODA_HEAD_MLP) {
    *count = (int64_t)d_hidden * d_model + 2 * (int64_t)d_hidden + 1;
  } else {
    return oda::fail(ODA_ERR_UNSUPPORTED, "unknown head kind %d", kind);
  }
  return oda::ok();
}

extern "C" oda_status oda_gate_workspace_size(const oda_gate_desc* gate, int32_t batch, size_t* bytes) {
  oda_status st = check_gate(gate);
  if (st != ODA_OK) return st;
  if (bytes == nullptr) return oda::fail(ODA_ERR_NULL, "bytes is NULL");
  if (batch < 1) return oda::fail(ODA_ERR_SHAPE, "batch must be >= 1");
  *bytes = gate_ws_layout(gate->kind, batch, gate->d_hidden).bytes;
  return oda::ok();
}
