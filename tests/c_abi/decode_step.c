/*
 * One ODA decode step driven from C through the library's C ABI (include/oda.h):
 * Local attention, the recall gate (MLP stand-in) with its device predicate and
 * compaction, then Full attention over the compacted work list (Alg. 1).
 *
 *   decode_step <inputs.bin> <outputs.bin>
 *
 * inputs.bin (little-endian): int32 L, B, Hq, Hkv, D, MB, max_len, NB, n_sink,
 * window, d_model, d_hidden; float32 tau, scale, eps; then q (bf16 bits,
 * L*B*Hq*D), k_cache and v_cache (bf16 bits, L*NB*Hkv*D*16 each, layouts of
 * oda.h), block_table (int32 B*MB), seq_lens (int32 B), gate parameters
 * (float32, oda_gate_param_count), h_local (float32 B*d_model).
 * outputs.bin: out (float32 L*B*Hq*D), lse (float32 L*B*Hq), score (float32 B),
 * flags (int32 B), work_list (int32 B), n_work (int32 1).
 * Exit status 0 on success; any failing call prints its status and message.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "oda.h"

#define CHECK_HIP(x)                                                              \
  do {                                                                            \
    hipError_t e_ = (x);                                                          \
    if (e_ != hipSuccess) {                                                       \
      fprintf(stderr, "%s:%d %s: %s\n", __FILE__, __LINE__, #x, hipGetErrorString(e_)); \
      exit(2);                                                                    \
    }                                                                             \
  } while (0)

#define CHECK_ODA(x)                                                              \
  do {                                                                            \
    oda_status s_ = (x);                                                          \
    if (s_ != ODA_OK) {                                                           \
      fprintf(stderr, "%s:%d %s: %s (%s)\n", __FILE__, __LINE__, #x,              \
              oda_status_string(s_), oda_last_error());                          \
      exit(3);                                                                    \
    }                                                                             \
  } while (0)

static void* read_block(FILE* f, size_t bytes) {
  void* p = malloc(bytes ? bytes : 1);
  if (p == NULL || fread(p, 1, bytes, f) != bytes) {
    fprintf(stderr, "short input file\n");
    exit(4);
  }
  return p;
}

static void* to_device(const void* host, size_t bytes) {
  void* d = NULL;
  CHECK_HIP(hipMalloc(&d, bytes ? bytes : 16));
  if (bytes) CHECK_HIP(hipMemcpy(d, host, bytes, hipMemcpyHostToDevice));
  return d;
}

static void* zeroed_device(size_t bytes) {
  void* d = NULL;
  CHECK_HIP(hipMalloc(&d, bytes ? bytes : 256));
  CHECK_HIP(hipMemset(d, 0, bytes ? bytes : 256));
  return d;
}

static void from_device(FILE* f, const void* dev, size_t bytes) {
  void* h = malloc(bytes);
  if (h == NULL) exit(4);
  CHECK_HIP(hipMemcpy(h, dev, bytes, hipMemcpyDeviceToHost));
  if (fwrite(h, 1, bytes, f) != bytes) exit(5);
  free(h);
}

int main(int argc, char** argv) {
  if (argc != 3) {
    fprintf(stderr, "usage: %s inputs.bin outputs.bin\n", argv[0]);
    return 1;
  }
  FILE* fi = fopen(argv[1], "rb");
  if (fi == NULL) {
    perror(argv[1]);
    return 1;
  }
  int32_t hdr[12];
  float fhdr[3];
  if (fread(hdr, sizeof(int32_t), 12, fi) != 12 || fread(fhdr, sizeof(float), 3, fi) != 3) {
    fprintf(stderr, "short header\n");
    return 4;
  }
  const int32_t L = hdr[0], B = hdr[1], Hq = hdr[2], Hkv = hdr[3], D = hdr[4], MB = hdr[5];
  const int32_t max_len = hdr[6], NB = hdr[7], n_sink = hdr[8], window = hdr[9];
  const int32_t d_model = hdr[10], d_hidden = hdr[11];
  const float tau = fhdr[0], scale = fhdr[1], eps = fhdr[2];

  int64_t n_params = 0;
  CHECK_ODA(oda_gate_param_count(ODA_HEAD_MLP, d_model, d_hidden, &n_params));

  const size_t q_bytes = (size_t)L * B * Hq * D * 2;
  const size_t kv_bytes = (size_t)L * NB * Hkv * D * 16 * 2;
  void* q = read_block(fi, q_bytes);
  void* k = read_block(fi, kv_bytes);
  void* v = read_block(fi, kv_bytes);
  void* table = read_block(fi, (size_t)B * MB * 4);
  void* seq = read_block(fi, (size_t)B * 4);
  void* params = read_block(fi, (size_t)n_params * 4);
  void* h_local = read_block(fi, (size_t)B * d_model * 4);
  fclose(fi);

  oda_attn_shape shape;
  memset(&shape, 0, sizeof(shape));
  shape.num_layers = L;
  shape.batch = B;
  shape.num_q_heads = Hq;
  shape.num_kv_heads = Hkv;
  shape.head_dim = D;
  shape.block_size = 16;
  shape.max_blocks_per_seq = MB;
  shape.max_seq_len = max_len;
  shape.num_blocks = NB;
  shape.split_blocks = 0;
  shape.layer_stride_kv = 0;

  oda_attn_inputs in;
  memset(&in, 0, sizeof(in));
  in.q = (const uint16_t*)to_device(q, q_bytes);
  in.k_cache = (const uint16_t*)to_device(k, kv_bytes);
  in.v_cache = (const uint16_t*)to_device(v, kv_bytes);
  in.block_table = (const int32_t*)to_device(table, (size_t)B * MB * 4);
  in.seq_lens = (const int32_t*)to_device(seq, (size_t)B * 4);
  in.scale = scale;

  const size_t out_bytes = (size_t)L * B * Hq * D * 4, lse_bytes = (size_t)L * B * Hq * 4;
  float* out = (float*)zeroed_device(out_bytes);
  float* lse = (float*)zeroed_device(lse_bytes);

  /* one workspace serves Local and Full: the larger of the two sizes, zeroed once */
  size_t ws_local = 0, ws_full = 0;
  CHECK_ODA(oda_attn_workspace_size(&shape, n_sink, window, &ws_local));
  CHECK_ODA(oda_attn_workspace_size(&shape, 0, 0, &ws_full));
  const size_t ws_bytes = ws_local > ws_full ? ws_local : ws_full;
  void* ws = zeroed_device(ws_bytes);

  oda_gate_desc gate;
  memset(&gate, 0, sizeof(gate));
  gate.kind = ODA_HEAD_MLP;
  gate.d_model = d_model;
  gate.d_hidden = d_hidden;
  gate.rms_eps = eps;
  gate.params = (const float*)to_device(params, (size_t)n_params * 4);
  size_t gws_bytes = 0;
  CHECK_ODA(oda_gate_workspace_size(&gate, B, &gws_bytes));
  void* gws = zeroed_device(gws_bytes);
  const float* dh_local = (const float*)to_device(h_local, (size_t)B * d_model * 4);
  float* score = (float*)zeroed_device((size_t)B * 4);
  int32_t* flags = (int32_t*)zeroed_device((size_t)B * 4);
  int32_t* work_list = (int32_t*)zeroed_device((size_t)B * 4);
  int32_t* n_work = (int32_t*)zeroed_device(4);
  int64_t* counter = (int64_t*)zeroed_device(8);

  hipStream_t stream = NULL;
  CHECK_ODA(oda_local_decode_attn(&shape, &in, n_sink, window, out, lse, ws, ws_bytes, stream));
  CHECK_ODA(oda_recall_gate(&gate, B, NULL, NULL, dh_local, tau, NULL, score, flags, work_list, n_work, counter,
                            gws, gws_bytes, stream));
  CHECK_ODA(oda_full_decode_attn(&shape, &in, 0, NULL, work_list, n_work, out, lse, ws, ws_bytes, stream));
  CHECK_HIP(hipStreamSynchronize(stream));

  FILE* fo = fopen(argv[2], "wb");
  if (fo == NULL) {
    perror(argv[2]);
    return 1;
  }
  from_device(fo, out, out_bytes);
  from_device(fo, lse, lse_bytes);
  from_device(fo, score, (size_t)B * 4);
  from_device(fo, flags, (size_t)B * 4);
  from_device(fo, work_list, (size_t)B * 4);
  int32_t flagged = 0;
  CHECK_HIP(hipMemcpy(&flagged, n_work, 4, hipMemcpyDeviceToHost));
  if (fwrite(&flagged, 4, 1, fo) != 1) return 5;
  fclose(fo);
  printf("decode step done: %d of %d requests took Full\n", flagged, B);
  return 0;
}
