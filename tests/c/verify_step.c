/* A plain C99 consumer of the library's C ABI: one verify step (head
 * projection with top-k and tree tokens, tree attention, greedy acceptance,
 * compaction) on device memory that this program allocates itself through the
 * HIP runtime's C API, on a stream of its own.
 *
 * Usage: verify_step DIR [fused]
 *
 * With "fused", acceptance and compaction run as one call
 * (specmemo_accept_compact) instead of specmemo_accept + specmemo_kv_compact.
 *
 * DIR holds meta.txt ("dt B hidden vocab n_heads n_q n_kv head_dim cap_total
 * path_stride" then the n_heads top-k sizes) and one raw little-endian file
 * per input array, named as below (element types as in specmemo.h; K, V, h,
 * head_w, q and base_logits in the dtype's storage: fp32 or bf16 bits).  The
 * outputs are written to DIR as out_*.bin.  Exit status 0 on success; any
 * failing call prints its message and exits non-zero. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "specmemo.h"

static const char *g_dir;

static void die(const char *what, const char *why, int code) {
  fprintf(stderr, "verify_step: %s: %s\n", what, why);
  exit(code);
}

#define HIP_CHECK(x)                                          \
  do {                                                        \
    hipError_t e_ = (x);                                      \
    if (e_ != hipSuccess) die(#x, hipGetErrorString(e_), 3);  \
  } while (0)

#define SPECMEMO_CHECK(x)                                     \
  do {                                                        \
    if ((x) != SPECMEMO_OK) die(#x, specmemo_last_error(), 4); \
  } while (0)

static FILE *open_in_dir(const char *name, const char *mode) {
  char path[4096];
  if (snprintf(path, sizeof path, "%s/%s", g_dir, name) >= (int)sizeof path) die(name, "path too long", 2);
  FILE *f = fopen(path, mode);
  if (!f) die(path, "cannot open", 2);
  return f;
}

/* Reads exactly `bytes` bytes of DIR/name into a new host buffer. */
static void *load(const char *name, size_t bytes) {
  FILE *f = open_in_dir(name, "rb");
  void *p = malloc(bytes ? bytes : 1);
  if (!p) die(name, "out of host memory", 2);
  if (fread(p, 1, bytes, f) != bytes || fgetc(f) != EOF) die(name, "unexpected size", 2);
  fclose(f);
  return p;
}

static void save(const char *name, const void *p, size_t bytes) {
  FILE *f = open_in_dir(name, "wb");
  if (fwrite(p, 1, bytes, f) != bytes) die(name, "short write", 2);
  fclose(f);
}

static void *to_device(const void *host, size_t bytes) {
  void *d = NULL;
  HIP_CHECK(hipMalloc(&d, bytes ? bytes : 4));
  if (bytes) HIP_CHECK(hipMemcpy(d, host, bytes, hipMemcpyHostToDevice));
  return d;
}

static void *device_buffer(size_t bytes) {
  void *d = NULL;
  HIP_CHECK(hipMalloc(&d, bytes ? bytes : 4));
  return d;
}

static void fetch(const char *name, const void *dev, size_t bytes) {
  void *h = malloc(bytes ? bytes : 1);
  if (!h) die(name, "out of host memory", 2);
  if (bytes) HIP_CHECK(hipMemcpy(h, dev, bytes, hipMemcpyDeviceToHost));
  save(name, h, bytes);
  free(h);
}

int main(int argc, char **argv) {
  if (argc < 2 || argc > 3 || (argc == 3 && strcmp(argv[2], "fused") != 0)) die("usage", "verify_step DIR [fused]", 2);
  g_dir = argv[1];
  const int fused = argc == 3;
  if (specmemo_abi_version() != SPECMEMO_ABI_VERSION) die("library", "ABI version differs from the header's", 2);

  int dt_i, B, hidden, vocab, n_heads, n_q, n_kv, head_dim, path_stride;
  long long cap_total;
  int32_t topk[SPECMEMO_MAX_DEPTH];
  FILE *m = open_in_dir("meta.txt", "r");
  if (fscanf(m, "%d %d %d %d %d %d %d %d %lld %d", &dt_i, &B, &hidden, &vocab, &n_heads, &n_q, &n_kv, &head_dim,
             &cap_total, &path_stride) != 10)
    die("meta.txt", "malformed", 2);
  if (B < 1 || n_heads < 1 || n_heads > SPECMEMO_MAX_DEPTH) die("meta.txt", "sizes out of range", 2);
  int kmax = 0;
  for (int i = 0; i < n_heads; ++i) {
    if (fscanf(m, "%d", &topk[i]) != 1) die("meta.txt", "missing top-k sizes", 2);
    if (topk[i] > kmax) kmax = topk[i];
  }
  fclose(m);
  const specmemo_dtype dt = dt_i == 0 ? SPECMEMO_FP32 : SPECMEMO_BF16;
  const size_t es = dt == SPECMEMO_FP32 ? 4 : 2;

  /* the tree batch: host arrays (validation and launch planning) and device copies */
  int32_t *node_off = load("node_off.bin", (size_t)(B + 1) * 4);
  const size_t N = (size_t)node_off[B];
  int32_t *parent = load("parent.bin", N * 4), *depth = load("depth.bin", N * 4), *rank = load("rank.bin", N * 4);
  specmemo_trees t;
  t.B = B;
  t.node_off = to_device(node_off, (size_t)(B + 1) * 4);
  t.parent = to_device(parent, N * 4);
  t.depth = to_device(depth, N * 4);
  t.rank = to_device(rank, N * 4);
  t.node_off_h = node_off;
  t.parent_h = parent;
  t.depth_h = depth;
  t.rank_h = rank;

  /* the KV pool */
  const size_t pool_bytes = (size_t)n_kv * (size_t)cap_total * (size_t)head_dim * es;
  int64_t *seq_base = load("seq_base.bin", (size_t)B * 8);
  int32_t *seq_len = load("seq_len.bin", (size_t)B * 4), *seq_cap = load("seq_cap.bin", (size_t)B * 4);
  void *k_h = load("k.bin", pool_bytes), *v_h = load("v.bin", pool_bytes);
  specmemo_kv kv;
  kv.k = to_device(k_h, pool_bytes);
  kv.v = to_device(v_h, pool_bytes);
  kv.cap_total = cap_total;
  kv.n_kv = n_kv;
  kv.head_dim = head_dim;
  kv.seq_len = to_device(seq_len, (size_t)B * 4);
  kv.seq_base_h = seq_base;
  kv.seq_cap_h = seq_cap;
  kv.seq_len_h = seq_len;

  /* the step's other inputs */
  const size_t h_bytes = (size_t)B * hidden * es, w_bytes = (size_t)n_heads * vocab * hidden * es;
  const size_t q_bytes = N * (size_t)n_q * head_dim * es, lg_bytes = N * (size_t)vocab * es;
  void *h = load("h.bin", h_bytes), *w = load("head_w.bin", w_bytes);
  void *q = load("q.bin", q_bytes), *lg = load("base_logits.bin", lg_bytes);
  int32_t *root = load("root_tok.bin", (size_t)B * 4);
  void *h_d = to_device(h, h_bytes), *w_d = to_device(w, w_bytes), *q_d = to_device(q, q_bytes);
  void *lg_d = to_device(lg, lg_bytes);
  int32_t *root_d = to_device(root, (size_t)B * 4);

  /* outputs and one workspace large enough for every call */
  const size_t z_bytes = (size_t)B * n_heads * vocab * 4, ids_bytes = (size_t)B * n_heads * kmax * 4;
  float *z_d = device_buffer(z_bytes);
  int32_t *ids_d = device_buffer(ids_bytes), *tok_d = device_buffer(N * 4);
  void *out_d = device_buffer(q_bytes);
  int32_t *acc_d = device_buffer((size_t)B * 4), *nxt_d = device_buffer((size_t)B * 4);
  int32_t *path_d = device_buffer((size_t)B * path_stride * 4);
  size_t ws_bytes = specmemo_workspace_bytes(SPECMEMO_WS_TOPK, dt, &t, NULL, n_heads, vocab);
  size_t need = specmemo_workspace_bytes(SPECMEMO_WS_ATTN, dt, &t, &kv, n_q, 0);
  if (need > ws_bytes) ws_bytes = need;
  need = specmemo_workspace_bytes(SPECMEMO_WS_ACCEPT, dt, &t, NULL, SPECMEMO_ACCEPT_GREEDY, vocab);
  if (need > ws_bytes) ws_bytes = need;
  void *ws = device_buffer(ws_bytes);

  hipStream_t stream;
  HIP_CHECK(hipStreamCreate(&stream));
  SPECMEMO_CHECK(specmemo_medusa_topk(dt, &t, hidden, vocab, n_heads, topk, h_d, w_d, SPECMEMO_HEADS_ROWMAJOR, root_d,
                                      z_d, ids_d, NULL, tok_d, ws, ws_bytes, stream));
  SPECMEMO_CHECK(specmemo_tree_attn(dt, &t, &kv, n_q, 0.0f, q_d, out_d, ws, ws_bytes, stream));
  if (fused) {
    SPECMEMO_CHECK(specmemo_accept_compact(dt, &t, &kv, vocab, SPECMEMO_ACCEPT_GREEDY, 1.0f, 0.09f, 0.3f, lg_d, tok_d,
                                           acc_d, path_d, path_stride, nxt_d, ws, ws_bytes, stream));
  } else {
    SPECMEMO_CHECK(specmemo_accept(dt, &t, vocab, SPECMEMO_ACCEPT_GREEDY, 1.0f, 0.09f, 0.3f, lg_d, tok_d, acc_d,
                                   path_d, path_stride, nxt_d, ws, ws_bytes, stream));
    SPECMEMO_CHECK(specmemo_kv_compact(dt, &t, &kv, acc_d, path_d, path_stride, stream));
  }
  HIP_CHECK(hipStreamSynchronize(stream));
  HIP_CHECK(hipStreamDestroy(stream));

  fetch("out_logits.bin", z_d, z_bytes);
  fetch("out_topk_ids.bin", ids_d, ids_bytes);
  fetch("out_node_tok.bin", tok_d, N * 4);
  fetch("out_attn.bin", out_d, q_bytes);
  fetch("out_accept_len.bin", acc_d, (size_t)B * 4);
  fetch("out_path.bin", path_d, (size_t)B * path_stride * 4);
  fetch("out_next_tok.bin", nxt_d, (size_t)B * 4);
  fetch("out_k.bin", kv.k, pool_bytes);
  fetch("out_v.bin", kv.v, pool_bytes);
  fetch("out_seq_len.bin", kv.seq_len, (size_t)B * 4);

  void *dev[] = {(void *)t.node_off, (void *)t.parent, (void *)t.depth, (void *)t.rank, kv.k, kv.v, kv.seq_len,
                 h_d, w_d, q_d, lg_d, root_d, z_d, ids_d, tok_d, out_d, acc_d, nxt_d, path_d, ws};
  for (size_t i = 0; i < sizeof dev / sizeof dev[0]; ++i) HIP_CHECK(hipFree(dev[i]));
  void *host[] = {node_off, parent, depth, rank, seq_base, seq_len, seq_cap, k_h, v_h, h, w, q, lg, root};
  for (size_t i = 0; i < sizeof host / sizeof host[0]; ++i) free(host[i]);
  printf("verify_step: ok (B=%d, %zu nodes%s)\n", B, N, fused ? ", fused acceptance and compaction" : "");
  return 0;
}
