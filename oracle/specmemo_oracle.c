/*
 * CPU oracle for the SpecMemo tree-verification step.  TEST INFRASTRUCTURE.
 *
 * Plain, slow, obviously correct fp64 loops for the four stages of one
 * speculative verify step.  Only the test-suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library; the product path never
 * does.  It shares no code, header or table with the HIP library.
 *
 * Stored inputs are fp32 or bf16 (raw 16-bit patterns); every value is widened
 * exactly to double before use, so the oracle sees the operands the GPU sees.
 *
 * Stages and the passages they follow (SpecMemo, arXiv 2506.01986):
 *   head logits  - Sec. 3.1 (l parallel heads read the last hidden state;
 *                  heads are plain linear maps hidden -> vocab),
 *   top-k        - Sec. 3.1 / Sec. 3.2 (tree arity k = top-k per head),
 *   tree tokens  - Sec. 3.1 Eq. 2 (level i of the tree holds head i's top-k),
 *   tree attention - Sec. 3.1 (before verification the mask assumes every
 *                  candidate sequence is fully accepted: a node sees its
 *                  ancestors and itself) and App. A.1 (one forward over all
 *                  candidates), with scaled dot-product attention; with
 *                  padded batching (Sec. 3.3) a cached pad token takes -inf
 *                  in the mask,
 *   acceptance   - App. A.1 (threshold per token, cumulative along the path,
 *                  longest verified candidate wins; typical sampling) and
 *                  Sec. 3.2 (verification of a continuation is cumulative),
 *   compaction   - Sec. 3.1 KV-cache paragraph (the preallocated cache is a
 *                  scratch space updated during verification) and Sec. 3.3
 *                  (rejected candidates are discarded).
 *
 * Readings where the paper is silent: ties in top-k and argmax go to the
 * lower token id; the root token is always accepted and its K/V is tree row 0;
 * accept_len counts non-root nodes; a typical-mode edge u->c is accepted iff
 * softmax(z_u/T)[tok c] > min(eps, delta * exp(-H_u)); among the deepest
 * accepted nodes the larger summed log-probability wins, then the lower id.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OR_FP32 0
#define OR_BF16 1

static double widen(const void *p, int dt, int64_t i) {
  if (dt == OR_FP32) return (double)((const float *)p)[i];
  uint32_t bits = (uint32_t)((const uint16_t *)p)[i] << 16;
  float f;
  memcpy(&f, &bits, sizeof f);
  return (double)f;
}

/* Threads of the parallel loops: n >= 1 sets them; returns the count in use. */
int oracle_threads(int n) {
  if (n > 0) omp_set_num_threads(n);
  return omp_get_max_threads();
}

/* Order of (value, id) pairs used by top-k and argmax: larger value first,
 * equal values by lower id. */
static int better(double va, int ia, double vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}

/* ---- head logits: z[s][i][v] = sum_c W[i][v][c] * h[b_s][c] ------------- */
void oracle_head_logits(int dt, int B, int hidden, int vocab, int n_heads, const void *h,
                        const void *W, int nsel, const int *bsel, double *z) {
  int nb = bsel ? nsel : B;
  double *hd = (double *)malloc(sizeof(double) * (size_t)nb * hidden);
  for (int s = 0; s < nb; ++s) {
    int b = bsel ? bsel[s] : s;
    for (int c = 0; c < hidden; ++c) hd[(size_t)s * hidden + c] = widen(h, dt, (int64_t)b * hidden + c);
  }
#pragma omp parallel
  {
    double *row = (double *)malloc(sizeof(double) * hidden);
#pragma omp for schedule(static)
    for (int64_t iv = 0; iv < (int64_t)n_heads * vocab; ++iv) {
      int i = (int)(iv / vocab), v = (int)(iv % vocab);
      for (int c = 0; c < hidden; ++c) row[c] = widen(W, dt, iv * hidden + c);
      for (int s = 0; s < nb; ++s) {
        double acc = 0.0;
        for (int c = 0; c < hidden; ++c) acc += row[c] * hd[(size_t)s * hidden + c];
        z[((int64_t)s * n_heads + i) * vocab + v] = acc;
      }
    }
    free(row);
  }
  free(hd);
}

/* ---- top-k of each row by repeated selection ------------------------------ */
void oracle_topk(int nrows, int vocab, int k, const double *z, int *ids, double *vals) {
#pragma omp parallel for schedule(static)
  for (int r = 0; r < nrows; ++r) {
    const double *x = z + (int64_t)r * vocab;
    int prev = -1;
    for (int j = 0; j < k; ++j) {
      int best = -1;
      for (int v = 0; v < vocab; ++v) {
        if (prev >= 0 && !better(x[prev], prev, x[v], v)) continue; /* already taken */
        if (best < 0 || better(x[v], v, x[best], best)) best = v;
      }
      ids[(int64_t)r * k + j] = best;
      if (vals) vals[(int64_t)r * k + j] = best >= 0 ? x[best] : -INFINITY;
      prev = best;
    }
  }
}

/* ---- tree tokens: root = root_tok, node n = topk_ids[b][depth-1][rank] ---- */
void oracle_tree_tokens(int B, const int *node_off, const int *depth, const int *rank,
                        const int *root_tok, int n_heads, int kmax, const int *topk_ids,
                        int *node_tok) {
  for (int b = 0; b < B; ++b)
    for (int n = node_off[b]; n < node_off[b + 1]; ++n) {
      if (n == node_off[b]) {
        node_tok[n] = root_tok[b];
      } else {
        int i = depth[n] - 1;
        node_tok[n] = topk_ids[((int64_t)b * n_heads + i) * kmax + rank[n]];
      }
    }
}

/* ---- tree-masked attention ------------------------------------------------
 * Node n (local id) of sequence b, query head h, KV head kv = h / (n_q/n_kv):
 * keys are the L_b committed rows and the tree rows L_b + j for every j on the
 * path from the root to n (both ends included).  out = softmax(scale * q K^T) V.
 * sel: nsel (global node, head) pairs, or NULL for every (node, head). */
static int seq_of(int B, const int *node_off, int node) {
  for (int b = 0; b < B; ++b)
    if (node < node_off[b + 1]) return b;
  return -1;
}

void oracle_tree_attn(int dt, int B, const int *node_off, const int *parent, const int *seq_len,
                      const int64_t *seq_base, int n_q, int n_kv, int d, int64_t cap_total,
                      double scale, const void *q, const void *K, const void *V, int nsel,
                      const int *sel, double *out, const uint8_t *key_valid) {
  int total = node_off[B];
  int64_t nrows = sel ? nsel : (int64_t)total * n_q;
  int group = n_q / n_kv;
#pragma omp parallel for schedule(dynamic, 4)
  for (int64_t r = 0; r < nrows; ++r) {
    int node = sel ? sel[2 * r] : (int)(r / n_q);
    int h = sel ? sel[2 * r + 1] : (int)(r % n_q);
    int b = seq_of(B, node_off, node);
    int n = node - node_off[b];
    int L = seq_len[b];
    int kv = h / group;
    /* key rows: committed, then the ancestors-or-self of n */
    int nanc = 0, anc[256];
    for (int a = n; a >= 0; a = parent[node_off[b] + a]) anc[nanc++] = a;
    int nkeys = L + nanc;
    int64_t *rows = (int64_t *)malloc(sizeof(int64_t) * nkeys);
    for (int t = 0; t < L; ++t) rows[t] = seq_base[b] + t;
    for (int j = 0; j < nanc; ++j) rows[L + j] = seq_base[b] + L + anc[j];
    double *s = (double *)malloc(sizeof(double) * nkeys);
    double m = -INFINITY;
    for (int t = 0; t < nkeys; ++t) {
      double acc = 0.0;
      for (int e = 0; e < d; ++e)
        acc += widen(q, dt, ((int64_t)node * n_q + h) * d + e) *
               widen(K, dt, ((int64_t)kv * cap_total + rows[t]) * d + e);
      s[t] = scale * acc;
      /* a cached pad token (key_valid 0) is masked with -inf (Sec. 3.3) */
      if (key_valid && t < L && !key_valid[rows[t]]) s[t] = -INFINITY;
      if (s[t] > m) m = s[t];
    }
    double zsum = 0.0;
    for (int t = 0; t < nkeys; ++t) {
      s[t] = exp(s[t] - m);
      zsum += s[t];
    }
    for (int e = 0; e < d; ++e) {
      double acc = 0.0;
      for (int t = 0; t < nkeys; ++t) acc += s[t] * widen(V, dt, ((int64_t)kv * cap_total + rows[t]) * d + e);
      out[r * d + e] = acc / zsum;
    }
    free(s);
    free(rows);
  }
}

/* ---- acceptance -------------------------------------------------------------
 * Greedy: a[u] = argmax of node u's base-model row (lowest id on ties).  From
 * the root, move to the child whose token equals a[cur] while one exists.
 * accept_len = depth reached, path = root..cur (local ids, -1 padded),
 * next_tok = a[cur]. */
static int row_argmax(int dt, const void *logits, int64_t row, int vocab) {
  int best = 0;
  double bv = widen(logits, dt, row * vocab);
  for (int v = 1; v < vocab; ++v) {
    double x = widen(logits, dt, row * vocab + v);
    if (better(x, v, bv, best)) {
      best = v;
      bv = x;
    }
  }
  return best;
}

void oracle_accept_greedy(int dt, int B, const int *node_off, const int *parent, const int *depth,
                          int vocab, const void *logits, const int *node_tok, int path_stride,
                          int *accept_len, int *path, int *next_tok) {
#pragma omp parallel for schedule(dynamic, 1)
  for (int b = 0; b < B; ++b) {
    int o = node_off[b], N = node_off[b + 1] - o;
    int cur = 0, len = 0;
    int *pb = path + (int64_t)b * path_stride;
    for (int j = 0; j < path_stride; ++j) pb[j] = -1;
    pb[0] = 0;
    int a = row_argmax(dt, logits, o + cur, vocab);
    for (;;) {
      int nxt = -1;
      for (int c = 1; c < N; ++c)
        if (parent[o + c] == cur && node_tok[o + c] == a) nxt = c;
      if (nxt < 0) break;
      cur = nxt;
      pb[++len] = cur;
      a = row_argmax(dt, logits, o + cur, vocab);
    }
    (void)depth;
    accept_len[b] = len;
    next_tok[b] = a;
  }
}

/* Typical: pi_u = softmax(z_u / T), H_u = -sum pi_u log pi_u.  Edge u->c is
 * accepted iff pi_u[tok c] > min(eps, delta * exp(-H_u)); a node is accepted
 * iff every edge on its root path is.  The deepest accepted node wins; ties go
 * to the larger sum of log pi along the path, then the lower node id.
 * next_tok = argmax z_cur.  Optional per-node outputs (index = global node,
 * root entries unused): log pi of the edge into the node and the log threshold
 * of that edge. */
/* Softmax statistics of each row x = z / T of typical acceptance (App. A.1):
 * lse = log sum_v exp(x_v) and the entropy H = -sum_v pi_v log pi_v of
 * pi = softmax(x). */
void oracle_softmax_stats(int dt, int rows, int vocab, const void *logits, double temperature, double *lse,
                          double *ent) {
#pragma omp parallel for schedule(dynamic, 4)
  for (int u = 0; u < rows; ++u) {
    double m = -INFINITY;
    for (int v = 0; v < vocab; ++v) {
      double x = widen(logits, dt, (int64_t)u * vocab + v) / temperature;
      if (x > m) m = x;
    }
    double zs = 0.0;
    for (int v = 0; v < vocab; ++v) zs += exp(widen(logits, dt, (int64_t)u * vocab + v) / temperature - m);
    double l = m + log(zs);
    double hsum = 0.0;
    for (int v = 0; v < vocab; ++v) {
      double lp = widen(logits, dt, (int64_t)u * vocab + v) / temperature - l;
      hsum -= exp(lp) * lp;
    }
    lse[u] = l;
    ent[u] = hsum;
  }
}

void oracle_accept_typical(int dt, int B, const int *node_off, const int *parent, const int *depth,
                           int vocab, const void *logits, const int *node_tok, double temperature,
                           double eps, double delta, int path_stride, int *accept_len, int *path,
                           int *next_tok, double *edge_logpi, double *edge_logthr) {
  int total = node_off[B];
  double *lse = (double *)malloc(sizeof(double) * total);
  double *ent = (double *)malloc(sizeof(double) * total);
  oracle_softmax_stats(dt, total, vocab, logits, temperature, lse, ent);
  for (int b = 0; b < B; ++b) {
    int o = node_off[b], N = node_off[b + 1] - o;
    int *acc = (int *)malloc(sizeof(int) * N);
    double *score = (double *)malloc(sizeof(double) * N);
    acc[0] = 1;
    score[0] = 0.0;
    int best = 0;
    for (int c = 1; c < N; ++c) {
      int u = parent[o + c];
      double lp = widen(logits, dt, (int64_t)(o + u) * vocab + node_tok[o + c]) / temperature - lse[o + u];
      double thr = eps < delta * exp(-ent[o + u]) ? eps : delta * exp(-ent[o + u]);
      if (edge_logpi) edge_logpi[o + c] = lp;
      if (edge_logthr) edge_logthr[o + c] = log(thr);
      acc[c] = acc[u] && (exp(lp) > thr);
      score[c] = score[u] + lp;
      if (acc[c]) {
        if (depth[o + c] > depth[o + best] ||
            (depth[o + c] == depth[o + best] && score[c] > score[best]))
          best = c; /* nodes are visited in increasing id: equal keys keep the lower id */
      }
    }
    int *pb = path + (int64_t)b * path_stride;
    for (int j = 0; j < path_stride; ++j) pb[j] = -1;
    int len = depth[o + best];
    for (int a = best, j = len; a >= 0; a = parent[o + a], --j) pb[j] = a;
    accept_len[b] = len;
    next_tok[b] = row_argmax(dt, logits, o + best, vocab);
    free(acc);
    free(score);
  }
  free(lse);
  free(ent);
}

/* ---- in-place KV compaction -------------------------------------------------
 * For j = 0..accept_len: slab row L_b + j <- slab row L_b + path[j] (K and V,
 * every KV head): all sources are read before any destination is written.
 * Then seq_len[b] += accept_len + 1.  Rows are copied as raw bytes. */
void oracle_kv_compact(int elem_bytes, int B, int n_kv, int d, int64_t cap_total, uint8_t *K,
                       uint8_t *V, const int64_t *seq_base, int *seq_len, const int *accept_len,
                       const int *path, int path_stride) {
  size_t rb = (size_t)elem_bytes * d;
  uint8_t *tmp = (uint8_t *)malloc(rb * (size_t)path_stride);
  for (int b = 0; b < B; ++b) {
    int L = seq_len[b], a = accept_len[b];
    const int *pb = path + (int64_t)b * path_stride;
    for (int kv = 0; kv < n_kv; ++kv) {
      uint8_t *pools[2] = {K, V};
      for (int w = 0; w < 2; ++w) {
        uint8_t *slab = pools[w] + ((size_t)kv * cap_total + seq_base[b]) * rb;
        for (int j = 0; j <= a; ++j) memcpy(tmp + j * rb, slab + (size_t)(L + pb[j]) * rb, rb);
        for (int j = 0; j <= a; ++j) memcpy(slab + (size_t)(L + j) * rb, tmp + j * rb, rb);
      }
    }
    seq_len[b] = L + a + 1;
  }
  free(tmp);
}

/* ---- Medusa residual-block heads ----------------------------------------------
 * Reading (the paper gives only a size per head): head i first maps the last
 * hidden state through one residual block, h'_i = h + SiLU(W1_i h + b1_i),
 * SiLU(x) = x / (1 + exp(-x)), and its vocabulary projection then reads h'_i.
 * W1: [n_heads][hidden][hidden] (out x in), b1: [n_heads][hidden], both in the
 * storage type.  out: fp64 [n_heads][B][hidden]. */
void oracle_resblock(int dt, int B, int hidden, int n_heads, const void *h, const void *W1, const void *b1,
                     double *out) {
#pragma omp parallel for schedule(static)
  for (int64_t ic = 0; ic < (int64_t)n_heads * hidden; ++ic) {
    int i = (int)(ic / hidden), c = (int)(ic % hidden);
    for (int b = 0; b < B; ++b) {
      double acc = widen(b1, dt, ic);
      for (int k = 0; k < hidden; ++k) acc += widen(W1, dt, ic * hidden + k) * widen(h, dt, (int64_t)b * hidden + k);
      double x = widen(h, dt, (int64_t)b * hidden + c);
      out[((int64_t)i * B + b) * hidden + c] = x + acc / (1.0 + exp(-acc));
    }
  }
}

/* ---- Philox4x64-10 ------------------------------------------------------------
 * The counter-based generator of Salmon, Moraes, Dror and Shaw ("Parallel
 * random numbers: as easy as 1, 2, 3", SC 2011): ten rounds of two 64 x 64 ->
 * 128-bit multiplications on a 4 x 64-bit counter, the 2 x 64-bit key bumped by
 * the Weyl constants between rounds. */
static void philox4x64_10(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4]) {
  uint64_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3], k0 = key[0], k1 = key[1];
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k0 += 0x9E3779B97F4A7C15ull;
      k1 += 0xBB67AE8584CAA73Bull;
    }
    unsigned __int128 p0 = (unsigned __int128)0xD2E7470EE14C6C93ull * x0;
    unsigned __int128 p1 = (unsigned __int128)0xCA5A826395121157ull * x2;
    uint64_t hi0 = (uint64_t)(p0 >> 64), lo0 = (uint64_t)p0, hi1 = (uint64_t)(p1 >> 64), lo1 = (uint64_t)p1;
    x0 = hi1 ^ x1 ^ k0;
    x1 = lo1;
    x2 = hi0 ^ x3 ^ k1;
    x3 = lo0;
  }
  out[0] = x0, out[1] = x1, out[2] = x2, out[3] = x3;
}

void oracle_philox4x64_10(int n, const uint64_t *ctr, const uint64_t *key, uint64_t *out) {
  for (int i = 0; i < n; ++i) philox4x64_10(ctr + 4 * i, key + 2 * i, out + 4 * i);
}

/* ---- sampled next token ---------------------------------------------------------
 * Instead of the greedy argmax, next_tok is drawn from softmax(z / T) of the
 * last accepted node's row, by the Gumbel-max rule: the argmax over v of
 * z_v / T + G_v with G_v = -log(-log(u_v)) standard Gumbel.  u_v comes from
 * Philox4x64-10 with key (seed, offset) and counter (v / 4, b, 0, 0), output
 * word v % 4: u = (k + 1/2) / 2^23 with k the word's top 23 bits, so that
 * 0 < u < 1 for every word and G is finite.  The oracle forms u, G and the
 * keys in fp64 from this definition (1/T is the caller's fp32 value); ties go
 * to the lower token id. */
void oracle_gumbel(int n, const uint64_t *x, double *g) {
  for (int i = 0; i < n; ++i) {
    double u = ((double)(x[i] >> 41) + 0.5) / 8388608.0;   /* 2^23 */
    g[i] = -log(-log(u));
  }
}

void oracle_sample_next(int dt, int B, const int *node_off, int vocab, float inv_temp, uint64_t seed,
                        uint64_t offset, const void *logits, const int *accept_len, const int *path, int stride,
                        int *next_tok, double *best_key, double *second_key) {
  for (int b = 0; b < B; ++b) {
    int64_t row = node_off[b] + path[(int64_t)b * stride + accept_len[b]];
    uint64_t key[2] = {seed, offset};
    double best = -INFINITY, second = -INFINITY;
    int arg = -1;
    for (int v0 = 0; v0 < vocab; v0 += 4) {
      uint64_t ctr[4] = {(uint64_t)(v0 / 4), (uint64_t)b, 0, 0}, x[4];
      double g[4];
      philox4x64_10(ctr, key, x);
      oracle_gumbel(4, x, g);
      for (int j = 0; j < 4 && v0 + j < vocab; ++j) {
        double s = widen(logits, dt, row * vocab + v0 + j) * (double)inv_temp + g[j];
        if (s > best) {
          second = best;
          best = s;
          arg = v0 + j;
        } else if (s > second) {
          second = s;
        }
      }
    }
    next_tok[b] = arg;
    if (best_key) best_key[b] = best;
    if (second_key) second_key[b] = second;
  }
}
