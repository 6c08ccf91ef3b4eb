/*
 * oda.h -- C ABI of the On-Demand Attention (ODA) decode-step hot path on
 * AMD Instinct MI355X (gfx950).
 *
 * One decode step of ODA (Alg. 1) runs, in stream order:
 *   1. oda_local_decode_attn  -- attention over the Local access set S^L
 *                                (s initial positions + a recent window of w
 *                                positions that includes the current token;
 *                                §2.1, access-set equation);
 *   2. oda_recall_gate        -- the recall score q_t = R(h_{t-1}, E(x_t), h_t^L)
 *                                (§2.1, recall-head equation; head of App. A.2,
 *                                or a two-layer MLP stand-in) and the device
 *                                predicate "Full iff q_t > theta or q_t is
 *                                nonfinite" (§2.1, Alg. 1, App. A.5), written
 *                                as per-request flags plus a compacted list;
 *   3. oda_full_decode_attn   -- attention over the native access set, from the
 *                                same pre-step history, for flagged requests
 *                                only; it overwrites their rows of the output,
 *                                so the output buffer ends up holding the
 *                                selected branch (App. A.5, commit equation).
 *
 * Conventions (all entry points):
 *   - Pointers are DEVICE pointers unless marked (host).  The caller owns every
 *     buffer; the library never allocates, never synchronises and never copies
 *     device memory to the host.
 *   - Host-visible arguments are validated synchronously; on any error the call
 *     returns a negative status and enqueues nothing.  oda_last_error() then
 *     holds a thread-local description.
 *   - All work is enqueued on `stream` (NULL = the default stream).
 *   - Device-data contract: seq_lens[b] in [1, max_seq_len]; every block-table
 *     entry a request uses in [0, num_blocks); listed requests in [0, batch).
 *     The kernels check it and never address memory with a value outside it:
 *     attention writes NaN rows (out and lse) for a request whose length or
 *     used table entry is out of range, the commit writes nothing for it, and
 *     listed requests outside the batch are skipped.
 *   - The library keeps no state between calls other than what a caller's
 *     workspace holds: attention workspaces carry merge-ticket words that
 *     every call leaves zero (see oda_attn_workspace_size).  Workspaces may be
 *     reused by later calls on the same stream; calls that share a workspace
 *     must not overlap in time.
 *   - Results are deterministic: a fixed split order, no floating-point
 *     atomics; reruns are bit-identical.
 *
 * Data layouts (bf16 = IEEE bfloat16 stored as uint16_t):
 *   q        bf16 [L][B][Hq][D]   post-RoPE queries of the current token
 *   k_cache  bf16 [L][num_blocks][Hkv][D/8][16][8]
 *            paged keys, 16 positions per block; within a block and KV head,
 *            16-byte groups of 8 consecutive dims, position-minor:
 *            K(pos, d) = k_cache[l][blk][g][d/8][pos%16][d%8]
 *   v_cache  bf16 [L][num_blocks][Hkv][D][16]
 *            paged values, dims-major:  V(pos, d) = v_cache[l][blk][g][d][pos%16]
 *            where blk = block_table[b][pos/16]; layer l starts layer_stride_kv
 *            elements after layer l-1 (dense by default)
 *   (Every 16-byte lane load of K is one matrix-core operand fragment and a
 *   wavefront's load instruction reads 1 KiB contiguous; V needs no transpose.
 *   Blocks stored position-major, [16][D] for both K and V as many paged
 *   caches keep them, measured 55% slower on this hardware -- Full over the
 *   32-layer 32,768-position stack 626 -> 970..990 us, Local 28 -> 41..44 us --
 *   because each K load instruction then touches 16 separate half lines and V
 *   must be transposed (through LDS or 2-byte gathers); the library does not
 *   take that layout.)
 *   k_cur, v_cur  bf16 [L][B][Hkv][D]  (optional) the current token's candidate
 *            K/V, not yet committed to the cache (App. A.5)
 *   out      fp32 [L][B][Hq][D];  lse fp32 [L][B][Hq]  (natural log)
 *   GQA: query head h reads KV head h / (Hq/Hkv)  (contiguous groups).
 */
#ifndef ODA_H_
#define ODA_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  ODA_OK = 0,
  ODA_ERR_NULL = -1,        /* a required pointer is NULL                      */
  ODA_ERR_SHAPE = -2,       /* inconsistent or out-of-range sizes              */
  ODA_ERR_UNSUPPORTED = -3, /* valid but not implemented (e.g. D not 64/128)   */
  ODA_ERR_WORKSPACE = -4,   /* workspace NULL or smaller than required         */
  ODA_ERR_HIP = -5          /* a kernel launch failed (hipGetLastError)        */
} oda_status;

/* Shape of one attention call (host struct).  Every layer of the stack
 * shares B, heads, D, the block table and seq_lens. */
typedef struct {
  int32_t num_layers;         /* L >= 1: layers in this call's stack              */
  int32_t batch;              /* B >= 1                                           */
  int32_t num_q_heads;        /* Hq                                               */
  int32_t num_kv_heads;       /* Hkv; Hq % Hkv == 0 and 1 <= Hq/Hkv <= 16         */
  int32_t head_dim;           /* D: 64 or 128                                     */
  int32_t block_size;         /* must be 16                                       */
  int32_t max_blocks_per_seq; /* row stride of block_table (>= ceil(max_seq_len/16)) */
  int32_t max_seq_len;        /* host-known upper bound of seq_lens[]             */
  int64_t num_blocks;         /* physical blocks per layer in k_cache / v_cache   */
  int32_t split_blocks;       /* KV blocks per split-K work item (one workgroup
                                 each): 0 = automatic, otherwise an even number >= 2 */
  int32_t reserved;           /* must be 0                                        */
  int64_t layer_stride_kv;    /* elements between layers in k_cache / v_cache:
                                 0 = num_blocks * Hkv * 16 * D (dense); else at
                                 least that and a multiple of 8 (e.g. one
                                 allocation holding several layer groups)       */
} oda_attn_shape;

/* Inputs of one attention call (host struct holding device pointers). */
typedef struct {
  const uint16_t *q;            /* bf16 [L][B][Hq][D]                             */
  const uint16_t *k_cache;      /* bf16, layout above                             */
  const uint16_t *v_cache;      /* bf16, layout above                             */
  const int32_t *block_table;   /* int32 [B][max_blocks_per_seq]: logical block i
                                   of request b -> physical block id              */
  const int32_t *seq_lens;      /* int32 [B]: n_b >= 1 attended positions
                                   0..n_b-1; position n_b-1 is the current token  */
  const uint16_t *k_cur;        /* NULL: the current token is already in the cache.
                                   Else bf16 [L][B][Hkv][D]: position n_b-1 is taken
                                   from here and the cache holds 0..n_b-2          */
  const uint16_t *v_cur;        /* NULL iff k_cur is NULL                         */
  float scale;                  /* softmax scale (> 0), usually 1/sqrt(D)         */
} oda_attn_inputs;

/* Bytes of workspace an attention call with this shape and access set needs
 * (one merge-ticket word per (layer, request, KV head), then the split-K
 * partials), whatever number of requests a Full call selects: the split
 * count depends on that number and the size covers the largest.  It is 0 when
 * every request fits one work item; the workspace pointer may then be NULL.  window == 0 means "no window" (the whole
 * history); window > 0 limits the recent part to `window` positions.
 * n_sink >= 0.  (host out)
 * A workspace must be zero-filled before its first use (e.g. allocated
 * zeroed).  Every call leaves its ticket words zero again, so later calls on
 * the same stream with the same num_layers * batch * num_kv_heads (any sinks,
 * window or branch) reuse it as it is, graph replays included; zero it again
 * before using it with a larger product.  Calls that may run concurrently
 * need separate workspaces. */
oda_status oda_attn_workspace_size(const oda_attn_shape *shape, int32_t n_sink, int32_t window,
                                   size_t *bytes);

/* Local decode attention (§2.1 access-set equation; App. A.5 Local path).
 * For every (layer, request, query head) attends to
 *     S^L = {j : j < min(n_sink, n)}  U  {j : max(0, n - window) <= j < n}
 * (0-based, each position once).  window >= 1, n_sink >= 0.  When
 * n_sink + window >= n the set is the whole history (Local == Full).
 * Writes out[L][B][Hq][D] and, if lse != NULL, lse[L][B][Hq] for all rows.
 * workspace: >= oda_attn_workspace_size(shape, n_sink, window) bytes,
 * 256-byte aligned. */
oda_status oda_local_decode_attn(const oda_attn_shape *shape, const oda_attn_inputs *in,
                                 int32_t n_sink, int32_t window, float *out, float *lse,
                                 void *workspace, size_t workspace_bytes, hipStream_t stream);

/* Recall-head kinds. */
typedef enum {
  ODA_HEAD_PAPER = 0, /* App. A.2: RMSNorm->Linear->SiLU towers on h_prev, emb,
                         h_local; interaction vector; fusion; two pre-RMSNorm
                         residual SwiGLU blocks; RMSNorm; scalar projection.
                         d_hidden = tower width dt (SwiGLU hidden 2*dt).       */
  ODA_HEAD_MLP = 1    /* stand-in: logit = w2 . GELU(W1 h_local + b1) + b2
                         (exact-erf GELU; sigmoid(logit) is the probability).
                         d_hidden = h.                                         */
} oda_head_kind;

/* Recall-gate description (host struct).  params: fp32, packed in this order
 *   PAPER: for t in (h_prev, emb, h_local): rms_t[d], W_t[dt][d], b_t[dt];
 *          W_f[dt][9dt], b_f[dt];
 *          for k in (1,2): rms_k[dt], W_gate_k[2dt][dt], W_up_k[2dt][dt], W_down_k[dt][2dt];
 *          rms_o[dt], w_o[dt], b_o[1]
 *   MLP:   W1[h][d], b1[h], w2[h], b2[1]
 * RMSNorm(x) = x / sqrt(mean(x^2) + rms_eps) * gain. */
typedef struct {
  int32_t kind;       /* oda_head_kind                                         */
  int32_t d_model;    /* d: width of h_prev / emb / h_local, multiple of 4     */
  int32_t d_hidden;   /* dt (PAPER) or h (MLP), multiple of 4                  */
  float rms_eps;      /* >= 0; ignored by the MLP                              */
  const float *params;/* device, oda_gate_param_count() floats                 */
} oda_gate_desc;

/* Number of fp32 parameters of a head (host out).  For PAPER with d = 2048,
 * dt = 1024 this is 28,325,889 (App. A.2). */
oda_status oda_gate_param_count(int32_t kind, int32_t d_model, int32_t d_hidden, int64_t *count);

/* Bytes of workspace oda_recall_gate needs for `batch` requests (host out). */
oda_status oda_gate_workspace_size(const oda_gate_desc *gate, int32_t batch, size_t *bytes);

/* Recall score and device predicate (§2.1, Alg. 1; App. A.5; App. B.7).
 *   h_prev, emb, h_local: fp32 [B][d_model] (PAPER reads all three; MLP only
 *                         h_local; the others may be NULL for MLP)
 *   tau:      threshold on the raw score (PAPER q_t; MLP pre-sigmoid logit);
 *             +-INFINITY allowed
 *   forced:   NULL, or int32 [B] prescribed flags (device-side schedule)
 *   score:    fp32 [B] out
 *   flags:    int32 [B] out; 1 iff score > tau or score is nonfinite
 *             (with `forced`: 1 iff forced[b] != 0 or score is nonfinite)
 *   work_list, n_work: NULL, or int32 [B] / int32 [1] out: the flagged request
 *             ids in ascending order and their count
 *   recall_counter: NULL, or int64 [1]; incremented by the number flagged
 *             (realised Full-call rate = counter / routed request-steps)
 * Everything stays on the device; no score is read by the host. */
oda_status oda_recall_gate(const oda_gate_desc *gate, int32_t batch, const float *h_prev,
                           const float *emb, const float *h_local, float tau, const int32_t *forced,
                           float *score, int32_t *flags, int32_t *work_list, int32_t *n_work,
                           int64_t *recall_counter, void *workspace, size_t workspace_bytes,
                           hipStream_t stream);

/* oda_recall_gate for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same computation and results, with the intermediate activations in a
 * workspace the library holds itself -- a 16 MiB device array per GPU, set
 * up on the first call on that GPU and kept until the process ends -- so the
 * call takes no workspace argument and allocates nothing.  Returns
 * ODA_ERR_WORKSPACE when oda_gate_workspace_size(gate, batch) exceeds 16 MiB
 * (the App. A.2 head takes 28 * batch * dt bytes for three or more requests:
 * up to 2,340 requests at dt = 256, 585 at dt = 1,024).  Every call on a GPU uses that GPU's one array: calls that may
 * overlap in time on one GPU (other streams, other host threads) race and
 * must be serialised by the caller.  The array's contents between calls do
 * not matter (each call writes what it reads). */
oda_status oda_recall_gate_static(const oda_gate_desc *gate, int32_t batch, const float *h_prev, const float *emb,
                                  const float *h_local, float tau, const int32_t *forced, float *score,
                                  int32_t *flags, int32_t *work_list, int32_t *n_work, int64_t *recall_counter,
                                  hipStream_t stream);

/* Full decode attention in the layers' native configuration (§2.1; App. A.5).
 * native_window == 0: S^F = all positions 0..n-1 (full-history layers);
 * native_window  > 0: the last native_window positions (natively
 * sliding-window layers, which ODA leaves unrestricted).
 * Request selection:
 *   work_list != NULL (with n_work != NULL): exactly the listed requests
 *                       (work_list[0 .. *n_work-1], distinct, as
 *                       oda_recall_gate writes them; a request listed twice
 *                       gets unspecified rows, but the workspace and every
 *                       other request are unaffected);
 *   else flags != NULL: the requests with flags[b] != 0;
 *   else              : every request.
 * Only selected requests read KV; only their rows of out (and lse, if not
 * NULL) are written, so after oda_local_decode_attn + oda_recall_gate the
 * buffer holds the selected branch per request.
 * workspace: >= oda_attn_workspace_size(shape, 0, native_window) bytes. */
oda_status oda_full_decode_attn(const oda_attn_shape *shape, const oda_attn_inputs *in,
                                int32_t native_window, const int32_t *flags,
                                const int32_t *work_list, const int32_t *n_work, float *out,
                                float *lse, void *workspace, size_t workspace_bytes,
                                hipStream_t stream);

/* Current-token preparation fused into a one-layer attention call (host
 * struct holding device pointers), for the decoder around the path (below):
 * the call builds the query and the current candidate K/V itself from the
 * fp32 QKV projection output, exactly as oda_qk_norm_rope would (per-head
 * RMSNorm of q and k, rotary embedding at position seq_lens[b] - 1, bf16
 * rounding; the same device code), instead of reading q / k_cur / v_cur, and
 * saves that launch.  Results are bit-identical to oda_qk_norm_rope followed
 * by the plain call.
 *   qkv     fp32 [B][(Hq + 2 Hkv) D]: q heads, then k heads, then v heads
 *   q_gain, k_gain  fp32 [D] per-head RMSNorm gains, or NULL (no norm)
 *   k_out, v_out    bf16 [B][Hkv][D]: the candidate K/V of the requests the
 *                   call attends (for the commit), or both NULL */
typedef struct {
  const float *qkv;
  const float *q_gain;
  const float *k_gain;
  float rms_eps;                /* >= 0                                          */
  double rope_theta;            /* > 1                                           */
  uint16_t *k_out;
  uint16_t *v_out;
} oda_qkv_prep;

/* oda_local_decode_attn / oda_full_decode_attn of one layer (num_layers == 1)
 * with the current token prepared in the call (oda_qkv_prep): in->q, k_cur and
 * v_cur must be NULL; the cache holds positions 0..n_b-2 and position n_b-1 is
 * the prepared candidate.  Everything else (sets, selection, workspace, the
 * rows written) is as in the plain calls. */
oda_status oda_local_decode_attn_qkv(const oda_attn_shape *shape, const oda_attn_inputs *in,
                                     const oda_qkv_prep *prep, int32_t n_sink, int32_t window, float *out,
                                     float *lse, void *workspace, size_t workspace_bytes, hipStream_t stream);
oda_status oda_full_decode_attn_qkv(const oda_attn_shape *shape, const oda_attn_inputs *in,
                                    const oda_qkv_prep *prep, int32_t native_window, const int32_t *flags,
                                    const int32_t *work_list, const int32_t *n_work, float *out, float *lse,
                                    void *workspace, size_t workspace_bytes, hipStream_t stream);

/* Bytes of workspace oda_commit_kv needs when it advances the lengths: one
 * ticket word per request, rounded up to 256 bytes (host out).  Zero-fill it
 * before its first use; every call leaves it zero again. */
oda_status oda_commit_workspace_size(const oda_attn_shape *shape, size_t *bytes);

/* Selected-state commit (App. A.5, commit equation C_t = C_{t-1} || dC_t^{b_t},
 * and its single fused cross-layer commit): in one launch, for every layer l,
 * request b and KV head g, copies the selected branch's current-position K/V
 * -- the Full candidate (k_full, v_full) if flags[b] != 0, else the Local
 * candidate (k_local, v_local) -- into position n_b - 1 of the paged cache
 * (block block_table[b][(n_b-1)/16], slot (n_b-1)%16, layouts above), where
 * n_b = seq_lens[b] is the step's attended count (the candidate was supplied
 * to the attention calls as k_cur/v_cur).  Then, if advance != 0,
 * seq_lens[b] += 1, ready for the next step's candidate.
 *   k_local, v_local: bf16 [L][B][Hkv][D] (required)
 *   k_full, v_full:   NULL (both) = same as the Local candidate
 *   flags:            NULL = every request keeps Local
 *   workspace:        required when advance != 0: >= oda_commit_workspace_size
 *                     bytes, 256-byte aligned, zero-filled before first use
 *                     (every call leaves it zero); ignored otherwise.  Calls
 *                     that may overlap in time need separate workspaces.
 * Only shape->num_layers, batch, num_kv_heads, head_dim, block_size,
 * max_blocks_per_seq and num_blocks are used.  The caller guarantees that the
 * block holding position n_b - 1 is allocated in block_table. */
oda_status oda_commit_kv(const oda_attn_shape *shape, uint16_t *k_cache, uint16_t *v_cache,
                         const int32_t *block_table, int32_t *seq_lens, const uint16_t *k_local,
                         const uint16_t *v_local, const uint16_t *k_full, const uint16_t *v_full,
                         const int32_t *flags, int32_t advance, void *workspace, size_t workspace_bytes,
                         hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Direct-ring Local (App. A.5: the Local path reads a contiguous workspace
 * holding the attention sinks and the recent window, with the current token
 * supplied separately, instead of the paged cache).  Per (layer, request, KV
 * head) unit, a ring of whole 16-position blocks in the cache's block
 * layouts.  For sinks s and window w:
 *   SB = ceil(s / 16) sink blocks, then RB = ceil(w / 16) + 2 ring blocks;
 *   logical block j of a request is held in ring block j if j < SB, else in
 *   ring block SB + (j mod RB)
 *   k_ring  bf16 [L][B][SB + RB][Hkv][D/8][16][8]
 *   v_ring  bf16 [L][B][SB + RB][Hkv][D][16]
 * RB blocks keep every block a Local call reads until the window has moved
 * past it, so a ring filled once (oda_ring_fill) and then kept current by the
 * commit (oda_commit_kv_ring) serves every later step.  A Local call through
 * the ring reads no block table and the same positions, in the same order,
 * as oda_local_decode_attn: the results are bit-identical.  Ring slots of
 * positions not yet committed may hold anything; no call reads them.  n_sink
 * and window must be the same in every call on a ring.
 * ------------------------------------------------------------------------- */

/* bf16 elements of each of k_ring and v_ring (host out). */
oda_status oda_ring_elements(const oda_attn_shape *shape, int32_t n_sink, int32_t window, int64_t *elements);

/* Fill the rings from the paged cache (one launch): every sink block, and in
 * every ring block the latest logical block j <= (seq_lens[b] - 1) / 16 that
 * maps to it, copied whole.  A request whose length is outside
 * [1, max_seq_len], or a table entry outside [0, num_blocks), leaves the ring
 * blocks concerned as they are.  Uses the same shape fields as
 * oda_local_decode_attn (layer_stride_kv included). */
oda_status oda_ring_fill(const oda_attn_shape *shape, const uint16_t *k_cache, const uint16_t *v_cache,
                         const int32_t *block_table, const int32_t *seq_lens, int32_t n_sink, int32_t window,
                         uint16_t *k_ring, uint16_t *v_ring, hipStream_t stream);

/* oda_local_decode_attn reading the rings: in->q, seq_lens, k_cur / v_cur
 * (the uncommitted candidate, or NULL when position n_b - 1 is in the ring)
 * and scale as there; in->k_cache, v_cache and block_table are not read (may
 * be NULL).  Same workspace (oda_attn_workspace_size(shape, n_sink, window)),
 * same outputs, bit for bit. */
oda_status oda_local_decode_attn_ring(const oda_attn_shape *shape, const oda_attn_inputs *in,
                                      const uint16_t *k_ring, const uint16_t *v_ring, int32_t n_sink,
                                      int32_t window, float *out, float *lse, void *workspace,
                                      size_t workspace_bytes, hipStream_t stream);

/* oda_commit_kv that also writes each committed position into the rings
 * (ring block of logical block (n_b - 1) / 16, slot (n_b - 1) % 16), in the
 * same launch.  The rings' shape is the commit's (L, B, Hkv, D). */
oda_status oda_commit_kv_ring(const oda_attn_shape *shape, uint16_t *k_cache, uint16_t *v_cache,
                              const int32_t *block_table, int32_t *seq_lens, const uint16_t *k_local,
                              const uint16_t *v_local, const uint16_t *k_full, const uint16_t *v_full,
                              const int32_t *flags, int32_t advance, void *workspace, size_t workspace_bytes,
                              uint16_t *k_ring, uint16_t *v_ring, int32_t n_sink, int32_t window,
                              hipStream_t stream);

/* ---------------------------------------------------------------------------
 * The decoder around the hot path (the backbone f_theta of §2.1 that Local and
 * Full share; App. A.6's cost model).  A pre-norm decoder layer is, per request:
 *   qkv = W_qkv . RMSNorm(h)              oda_dense_bf16 (gain = input norm)
 *   q, k, v = split(qkv); q, k per-head RMSNorm and rotary embedding at the
 *   current position, cast to bf16       oda_qk_norm_rope
 *   a = attention(q, cache, k, v)         oda_local_decode_attn / oda_full_decode_attn
 *   (the last two in one launch: oda_local_decode_attn_qkv / oda_full_decode_attn_qkv)
 *   h = h + W_o . a                       oda_dense_bf16 (residual = h)
 *   m = SiLU(W_g . RMSNorm(h)) * (W_u . RMSNorm(h))   oda_dense_bf16 (SWIGLU)
 *   h = h + W_d . m                       oda_dense_bf16 (residual = h)
 * then logits = W_vocab . RMSNorm(h) and the greedy token (oda_argmax).
 * Weights bf16, activations fp32.  Every call below can be restricted to the
 * recall gate's list (work_list, n_work: both NULL = every request; entries
 * must be in [0, batch)): only those requests are read and written.
 * ------------------------------------------------------------------------- */

typedef enum { ODA_DENSE_PLAIN = 0, ODA_DENSE_SWIGLU = 1 } oda_dense_mode;

typedef struct {
  int32_t in_features;     /* K, a multiple of 8                                  */
  int32_t out_features;    /* N                                                   */
  int32_t mode;            /* oda_dense_mode                                      */
  float rms_eps;           /* RMSNorm epsilon (used when norm_gain != NULL)       */
  const uint16_t *weight;  /* device bf16, PLAIN: [N][K]; SWIGLU: [2N][K], the N
                              gate rows then the N up rows; 16-byte aligned       */
  const float *norm_gain;  /* device fp32 [K]: x' = x / sqrt(mean(x^2) + eps) * gain;
                              NULL: x' = x                                        */
} oda_dense_desc;

/* Dense layer for `batch` requests, fp32 accumulation:
 *   PLAIN:  y[b][r] = sum_k W[r][k] x'[b][k]  (+ residual[b][r] if residual != NULL)
 *   SWIGLU: y[b][r] = SiLU(sum_k W[r][k] x'[b][k]) * sum_k W[N + r][k] x'[b][k]
 *           (no residual)
 * x fp32 [batch][K] (16-byte aligned); residual, y fp32 [batch][N].  y may be
 * the residual buffer (in-place residual add); x must not overlap y. */
oda_status oda_dense_bf16(const oda_dense_desc *desc, int32_t batch, const float *x, const float *residual,
                          float *y, const int32_t *work_list, const int32_t *n_work, hipStream_t stream);

/* Query/key preparation for the current token.  qkv fp32 [batch][(Hq + 2 Hkv) D]
 * holds the q heads, then the k heads, then the v heads.  q and k heads get a
 * per-head RMSNorm (gains q_gain / k_gain fp32 [D], or NULL for none) and then
 * the rotary embedding at position p = seq_lens[b] - 1 (rotate-half pairing:
 * dims i and i + D/2 rotate by angle p * theta^(-2i/D), angles in double);
 * results are rounded to bf16 (nearest-even):
 *   q_out bf16 [batch][Hq][D] (the attention query; as q of a one-layer call),
 *   k_out, v_out bf16 [batch][Hkv][D] (the current candidate, k_cur / v_cur).
 * D even, at most 128. */
oda_status oda_qk_norm_rope(int32_t batch, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                            const float *qkv, const float *q_gain, const float *k_gain, float rms_eps,
                            double rope_theta, const int32_t *seq_lens, uint16_t *q_out, uint16_t *k_out,
                            uint16_t *v_out, const int32_t *work_list, const int32_t *n_work,
                            hipStream_t stream);

/* x[b] = table[tokens[b]] widened to fp32; table bf16 [vocab][d_model] (d_model a
 * multiple of 8); a token outside [0, vocab) gives a NaN row (and so a nonfinite
 * recall score, i.e. Full). */
oda_status oda_embed_bf16(const uint16_t *table, int32_t vocab, int32_t d_model, int32_t batch,
                          const int32_t *tokens, float *x, hipStream_t stream);

/* dst[b] = src[b] (fp32 rows of row_len, a multiple of 4) for the listed
 * requests (all if the list is NULL): moves the Full retry's results into the
 * selected state. */
oda_status oda_copy_rows(int32_t batch, int32_t row_len, const float *src, float *dst,
                         const int32_t *work_list, const int32_t *n_work, hipStream_t stream);

/* y[b] = x[b] / sqrt(mean(x[b]^2) + rms_eps) * gain for the listed requests
 * (all if the list is NULL): the final normalised hidden state, which §2.1
 * names as the recall head's Local input h_t^L and App. A.5 as the selected
 * state h_{t-1} the head reads at the next step.  x, y fp32 [batch][row_len]
 * (row_len a multiple of 4, 16-byte aligned; y may be x), gain fp32 [row_len]. */
oda_status oda_rms_norm_rows(int32_t batch, int32_t row_len, const float *x, const float *gain, float rms_eps,
                             float *y, const int32_t *work_list, const int32_t *n_work, hipStream_t stream);

/* index[b] = the first position of the largest non-NaN value of x[b][0..n)
 * (-1 if all are NaN); x fp32 [batch][n], n a multiple of 4. */
oda_status oda_argmax(int32_t batch, int32_t n, const float *x, int32_t *index, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Measurement aid (not a step of the method): the streaming-read ceiling that
 * the attention kernels' bandwidth is quoted against.
 * ------------------------------------------------------------------------- */

/* Reads `bytes` of device memory at src once (16-byte nontemporal loads, the
 * attention kernels' KV loads) and discards them.  src 16-byte aligned, bytes a
 * multiple of 16; sink: device uint32[1], left unchanged in practice (written
 * only if the XOR of everything read hits one fixed value); groups: workgroups
 * of 256 threads, 0 for the default (256). */
oda_status oda_stream_read(const void *src, size_t bytes, uint32_t *sink, int32_t groups, hipStream_t stream);

/* Static description of a status code. */
const char *oda_status_string(oda_status status);

/* Thread-local detail of the last non-OK return on this thread ("" if none). */
const char *oda_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* ODA_H_ */
