/*
 * specmemo.h - C ABI of the MI355X (gfx950) tree-verification library.
 *
 * One speculative step of Medusa-style decoding as SpecMemo runs it
 * (arXiv 2506.01986): the heads propose, the base model verifies a whole
 * candidate tree in one forward pass, the longest verified path is accepted,
 * and the KV cache - a preallocated scratch space sized to a budget - is
 * updated in place.  Four calls, one per stage, in this order on one stream:
 *
 *   specmemo_medusa_topk   (a) head projection, per-head top-k, tree tokens
 *   specmemo_tree_attn     (b) tree-masked attention over the ragged batch
 *   specmemo_accept        (c) greedy / typical acceptance of the longest path
 *   specmemo_kv_compact    (d) in-place compaction of the accepted K/V
 *
 * Symbols follow the paper's memory model (Sec. 3.1): b = batch (B),
 * k = KV heads (n_kv), d = head dim (head_dim), x = KV length
 * (seq_len / seq_cap), l = Medusa heads = tree levels (n_heads),
 * k = arity = top-k per head (topk[i]), N = tree nodes, w = vocabulary
 * (vocab), tau = accept_len + 1 tokens committed per step.
 *
 * Conventions for every call
 *  - Ownership: every buffer belongs to the caller.  Device pointers are
 *    device memory; "_h" pointers are host memory that is read only during
 *    the call.  The library never allocates, frees or synchronises; scratch
 *    space comes only through the (ws, ws_bytes) arguments.
 *  - Asynchrony: `stream` is a hipStream_t passed as void* (NULL = the null
 *    stream).  Calls enqueue kernels and return; results are ordered on the
 *    stream.
 *  - Alignment: every device pointer must be 16-byte aligned.
 *  - Errors: calls return a specmemo_status.  All argument, tree, budget and
 *    workspace checks run on the host before anything is enqueued; on failure
 *    nothing is enqueued and no output changes.  specmemo_last_error() then
 *    describes the failure.  A launch failure returns SPECMEMO_E_HIP; faults
 *    inside kernels surface at the caller's next synchronisation.
 *  - Trees: one tree per sequence, nodes in BFS order with local ids
 *    0..N_b-1, node 0 is the root, parent[n] < n, depth[n] =
 *    depth[parent[n]] + 1, sibling ranks distinct, 1 <= N_b <= 128.
 *    rank[n] indexes head depth[n]-1's top-k list (node tokens depend only on
 *    depth and rank, Sec. 3.1 Eq. 2).
 *  - KV pool: for one layer, K and V are [n_kv][cap_total][head_dim]; each
 *    sequence owns the slab of rows [seq_base[b], seq_base[b] + seq_cap[b]);
 *    its L_b = seq_len[b] committed rows come first, and before the step the
 *    caller has written the K/V rows of the tree's N_b nodes at slab rows
 *    L_b .. L_b + N_b - 1 (node order).  L_b + N_b <= seq_cap[b] is the
 *    budget: this is SpecMemo's precise preallocation (Sec. 3.1, KV-cache
 *    paragraph) instead of one sized for the full context.
 */
#ifndef SPECMEMO_H
#define SPECMEMO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SPECMEMO_ABI_VERSION 9
#define SPECMEMO_MAX_TREE_NODES 128 /* nodes per sequence's tree */
#define SPECMEMO_MAX_DEPTH 15       /* tree depth (= Medusa heads) */
#define SPECMEMO_MAX_TOPK 32        /* top-k per head */
#define SPECMEMO_MAX_BATCH 4096     /* sequences per call */

typedef enum {
  SPECMEMO_OK = 0,
  SPECMEMO_E_ARG = -1,       /* null/misaligned pointer, bad size or shape */
  SPECMEMO_E_DTYPE = -2,     /* unsupported dtype, or dtype/shape combination */
  SPECMEMO_E_TREE = -3,      /* tree arrays violate the conventions above */
  SPECMEMO_E_BUDGET = -4,    /* L_b + N_b > seq_cap[b], or slab outside the pool */
  SPECMEMO_E_WORKSPACE = -5, /* ws is NULL or smaller than specmemo_workspace_bytes */
  SPECMEMO_E_HIP = -6        /* a HIP launch failed */
} specmemo_status;

typedef enum { SPECMEMO_FP32 = 0, SPECMEMO_BF16 = 1 } specmemo_dtype;

typedef enum { SPECMEMO_ACCEPT_GREEDY = 0, SPECMEMO_ACCEPT_TYPICAL = 1 } specmemo_accept_mode;
typedef enum {
  SPECMEMO_HEADS_ROWMAJOR = 0,
  SPECMEMO_HEADS_PACKED = 1,
  SPECMEMO_HEADS_INPUT_PER_HEAD = 2   /* flag, OR-ed with a layout: h is [n_heads][B][hidden] */
} specmemo_head_layout;

/* Ragged batch of candidate trees, CSR over nodes.  Device arrays are read by
 * kernels; the host mirrors (same contents) are read for validation and launch
 * planning during the call. */
typedef struct {
  int32_t B;                  /* sequences */
  const int32_t *node_off;    /* device [B+1], node_off[0] = 0, node_off[B] = sum N_b */
  const int32_t *parent;      /* device [sum N_b], local ids, parent[root] = -1 */
  const int32_t *depth;       /* device [sum N_b], root depth 0 */
  const int32_t *rank;        /* device [sum N_b], root rank 0 */
  const int32_t *node_off_h;  /* host mirrors of the four arrays above */
  const int32_t *parent_h;
  const int32_t *depth_h;
  const int32_t *rank_h;
} specmemo_trees;

/* Budget-capped KV pool of one layer. */
typedef struct {
  void *k;                    /* device [n_kv][cap_total][head_dim], dtype */
  void *v;                    /* device, same shape */
  int64_t cap_total;          /* pool rows per KV head */
  int32_t n_kv;               /* KV heads */
  int32_t head_dim;           /* d */
  int32_t *seq_len;           /* device [B]: written by specmemo_kv_compact */
  const int64_t *seq_base_h;  /* host [B]: first pool row of each slab */
  const int32_t *seq_cap_h;   /* host [B]: slab rows (the budget) */
  const int32_t *seq_len_h;   /* host [B]: committed rows L_b before this step */
} specmemo_kv;

/* (a) Medusa-head projection and top-k tree assembly (Sec. 3.1: l heads read
 * the last hidden state, head i's top-k tokens fill tree level i+1; Eq. 2).
 *
 *   z[b][i][v] = sum_c head_w[i][v][c] * h[b][c]     (fp32 accumulation)
 *   topk_ids[b][i][0..topk_h[i]) = the topk_h[i] largest z[b][i][:], larger
 *       value first, equal values by lower token id; entries past topk_h[i]
 *       are set to -1 (values to -inf)
 *   node_tok[node_off[b]] = root_tok[b];
 *   node_tok[node_off[b] + n] = topk_ids[b][depth[n]-1][rank[n]]  (n > 0)
 *
 * h: device [B][hidden] in `dt`.  head_w: device, in `dt`, laid out as
 * head_layout says: SPECMEMO_HEADS_ROWMAJOR is [n_heads][vocab][hidden] (the
 * nn.Linear out x in layout, no bias); SPECMEMO_HEADS_PACKED (bf16 only) is
 * the buffer written by specmemo_pack_heads, which the projection streams
 * contiguously.  With SPECMEMO_HEADS_INPUT_PER_HEAD OR-ed in, h is
 * [n_heads][B][hidden] and head i reads h[i] (e.g. the outputs of
 * specmemo_medusa_resblock).  root_tok: device [B]
 * (the base model's own next token from the previous step).  logits_out:
 * device fp32 [B][n_heads][vocab], or NULL.  topk_ids: device int32
 * [B][n_heads][kmax] with kmax = max(topk_h); topk_vals: device fp32, same
 * shape, or NULL.  node_tok: device int32 [sum N_b].  Requires hidden % 8 == 0,
 * 1 <= n_heads <= SPECMEMO_MAX_DEPTH, 1 <= topk_h[i] <= min(SPECMEMO_MAX_TOPK,
 * vocab), tree depth <= n_heads and rank[n] < topk_h[depth[n]-1].
 * ws: at least specmemo_workspace_bytes(SPECMEMO_WS_TOPK, ...) bytes. */
int specmemo_medusa_topk(specmemo_dtype dt, const specmemo_trees *t, int32_t hidden,
                         int32_t vocab, int32_t n_heads, const int32_t *topk_h, const void *h,
                         const void *head_w, int32_t head_layout, const int32_t *root_tok,
                         float *logits_out, int32_t *topk_ids, float *topk_vals,
                         int32_t *node_tok, void *ws, size_t ws_bytes, void *stream);

/* The head projection of (a) alone: logits_out[b][i][v] = sum_c
 * head_w[i][v][c] * h[b][c] (fp32 accumulation), for callers that need the
 * logits rather than the tree (and to time the projection kernel by itself).
 * Same layouts, flags and requirements as specmemo_medusa_topk; logits_out:
 * device fp32 [B][n_heads][vocab], 16-byte aligned; 1 <= B <=
 * SPECMEMO_MAX_BATCH. */
int specmemo_head_logits(specmemo_dtype dt, int32_t B, int32_t hidden, int32_t vocab, int32_t n_heads, const void *h,
                         const void *head_w, int32_t head_layout, float *logits_out, void *stream);

/* Medusa residual-block heads.  The paper gives only a size per head; this
 * reading gives each head one residual block before its vocabulary projection:
 *   out[i][b][c] = h[b][c] + SiLU(sum_k w1[i][c][k] h[b][k] + b1[i][c]),
 *   SiLU(x) = x / (1 + exp(-x)), fp32 accumulation, stored in `dt`;
 * out then feeds specmemo_medusa_topk with SPECMEMO_HEADS_INPUT_PER_HEAD.
 * h: device [B][hidden]; b1: device [n_heads][hidden]; out: device
 * [n_heads][B][hidden].  w1: bf16 in SPECMEMO_HEADS_PACKED layout, written by
 * specmemo_pack_heads(dt, n_heads, hidden, hidden, ...) from
 * [n_heads][hidden][hidden] (out x in); fp32 in SPECMEMO_HEADS_ROWMAJOR.
 * Requires 1 <= B <= SPECMEMO_MAX_BATCH, 1 <= n_heads <= SPECMEMO_MAX_DEPTH,
 * hidden % 8 == 0. */
int specmemo_medusa_resblock(specmemo_dtype dt, int32_t B, int32_t hidden, int32_t n_heads, const void *h,
                             const void *w1, int32_t w1_layout, const void *b1, void *out, void *stream);

/* Head weights in the projection's streaming order (bf16).  The heads are
 * fixed for a model, so they are packed once, at load time:
 *
 *   packed element ((((i * nG + G) * nS + s) * 4 + t) * 64 + l) * 8 + e
 *     = head_w[i][64 G + 16 t + l % 16][32 s + 8 (l / 16) + e]
 *
 * for head i, row group G < nG = ceil(vocab / 64), k step s < nS =
 * ceil(hidden / 32), row tile t < 4, lane l < 64 and e < 8; rows past vocab and
 * columns past hidden are zero.  Each 1 KB (t, s) block is one matrix-core
 * operand tile of 16 rows x 32 columns, and a row group's blocks are
 * contiguous.  src: device [n_heads][vocab][hidden] bf16 (row-major, as
 * above); dst: device, specmemo_packed_heads_bytes(...) bytes, 16-byte
 * aligned, not overlapping src.  Requires hidden % 8 == 0.  Asynchronous on
 * `stream`. */
int specmemo_pack_heads(specmemo_dtype dt, int32_t n_heads, int32_t vocab, int32_t hidden,
                        const void *src, void *dst, void *stream);
/* Bytes of the packed head weights (0 for invalid arguments or fp32). */
size_t specmemo_packed_heads_bytes(specmemo_dtype dt, int32_t n_heads, int32_t vocab,
                                   int32_t hidden);

/* (b) Tree-masked attention of one layer (Sec. 3.1: before verification the
 * mask assumes full acceptance of every candidate sequence, so a node attends
 * to its root path; App. A.1: one forward over all candidates; Sec. 3.3: a
 * ragged batch, here without padding).
 *
 * For node n of sequence b and query head hq, with KV head kv = hq / (n_q/n_kv):
 *   keys  = slab rows 0..L_b-1 (committed) and L_b + j for every j on the
 *           path root..n (inclusive)
 *   out[node][hq] = softmax(scale * q[node][hq] . K[kv][key]) . V[kv][key]
 * q, out: device [sum N_b][n_q][head_dim] in `dt`.  scale <= 0 selects
 * 1/sqrt(head_dim).  bf16 requires head_dim == 128 and seq_cap[b] <= 2^23
 * rows (else SPECMEMO_E_BUDGET); fp32 requires
 * head_dim <= 128 and head_dim % 4 == 0.  n_q % n_kv == 0.  Rows of the slab
 * past L_b + N_b are never read.  ws: at least
 * specmemo_workspace_bytes(SPECMEMO_WS_ATTN, ...) bytes (the partial results
 * of KV ranges split across work items; with more than 32 sequences also the
 * per-sequence descriptors and the work map of the single launch, written
 * into ws by the call's own kernels; may be 0). */
int specmemo_tree_attn(specmemo_dtype dt, const specmemo_trees *t, const specmemo_kv *kv,
                       int32_t n_q, float scale, const void *q, void *out, void *ws,
                       size_t ws_bytes, void *stream);

/* (b) without a workspace argument, for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that
 * forbid allocation.  The split-KV partial results that specmemo_tree_attn
 * keeps in `ws` go to a scratch array of SPECMEMO_ATTN_STATIC_SCRATCH_BYTES
 * (32 MiB) that the library holds on each device it runs on, from the
 * library's load until the process ends; the call itself allocates nothing.
 * A batch whose split needs more (specmemo_workspace_bytes(SPECMEMO_WS_ATTN,
 * ...) > 32 MiB) is rejected with SPECMEMO_E_WORKSPACE before anything is
 * enqueued; every default split fits.  All calls on one device share that
 * array, which keeps the last call's contents: calls that can overlap on one
 * device (other streams, other threads) race, and the caller must order them.
 * Arguments, checks and results are those of specmemo_tree_attn. */
#define SPECMEMO_ATTN_STATIC_SCRATCH_BYTES ((size_t)32 << 20)
int specmemo_tree_attn_noalloc(specmemo_dtype dt, const specmemo_trees *t, const specmemo_kv *kv,
                               int32_t n_q, float scale, const void *q, void *out, void *stream);

/* (c) Acceptance (App. A.1: each candidate token must pass a threshold,
 * verification is cumulative along the sequence, the longest verified
 * candidate is accepted; Sec. 3.2: verification of a continuation is
 * cumulative).  base_logits: device [sum N_b][vocab] in `dt`, row u = the
 * base model's next-token logits after node u.  node_tok: device int32.
 *
 * GREEDY:  a[u] = argmax_v base_logits[u][v] (ties: lower v; -0 equals +0;
 *          NaN logits are not valid input).  From the root,
 *          move to the child c with node_tok[c] == a[cur] while one exists.
 * TYPICAL: pi_u = softmax(base_logits[u] / temperature), H_u its entropy;
 *          edge u->c passes iff pi_u[node_tok[c]] > min(eps, delta*exp(-H_u));
 *          a node is accepted iff every edge on its root path passes; the
 *          deepest accepted node wins, ties by larger sum of log pi along the
 *          path, then lower node id.
 * Outputs (device int32): accept_len[B] = depth of the chosen node (the root
 * is always accepted; tau = accept_len + 1); path[B][path_stride] = local
 * node ids root..chosen, -1 padded, path_stride >= max tree depth + 1;
 * next_tok[B] = argmax of the chosen node's row (ties: lower id).
 * ws: SPECMEMO_WS_ACCEPT bytes (greedy: one int32 per node; typical: two
 * floats and one int32 per node). */
int specmemo_accept(specmemo_dtype dt, const specmemo_trees *t, int32_t vocab,
                    specmemo_accept_mode mode, float temperature, float eps, float delta,
                    const void *base_logits, const int32_t *node_tok, int32_t *accept_len,
                    int32_t *path, int32_t path_stride, int32_t *next_tok, void *ws,
                    size_t ws_bytes, void *stream);

/* Sampled next token (in place of the greedy one that specmemo_accept writes):
 * next_tok[b] is drawn from softmax(z / T) of the last accepted node's row,
 * z = base_logits[node_off[b] + path[b][accept_len[b]]], by the Gumbel-max
 * rule: the argmax over v of fmaf(z_v, 1/T, G_v) in fp32, with 1/T rounded
 * once to fp32, G_v = -log(-log(u_v)) and u_v = ((x >> 41) + 1/2) / 2^23
 * (exact in fp32, within [2^-24, 1 - 2^-24], so G_v is finite) for
 * x the 64-bit word v % 4 of Philox4x64-10 (Salmon et al., SC 2011) with key
 * (seed, offset) and counter (v / 4, b, 0, 0).  Ties go to the lower id.  A
 * caller draws a fresh sample per step by changing offset.  Sequences whose
 * accept_len / path entry is out of range keep their next_tok.  temperature
 * must be positive and finite (and 1/T finite).
 * ws: specmemo_workspace_bytes(SPECMEMO_WS_SAMPLE, ...) bytes, 16-byte aligned
 * (one 64-bit word per sequence and 1024-token segment of the row), or NULL:
 * with it the draws of a row are spread over one block per segment, without
 * it one block per sequence draws its whole row (the same token either way). */
int specmemo_sample_next(specmemo_dtype dt, const specmemo_trees *t, int32_t vocab, float temperature,
                         uint64_t seed, uint64_t offset, const void *base_logits, const int32_t *accept_len,
                         const int32_t *path, int32_t path_stride, int32_t *next_tok, void *ws,
                         size_t ws_bytes, void *stream);

/* (d) In-place KV compaction (Sec. 3.1 KV-cache paragraph: the preallocated
 * cache is a scratch space updated during verification; Sec. 3.3: rejected
 * candidates are discarded).  For every sequence b, KV head and both K and V:
 *   slab row L_b + j <- slab row L_b + path[b][j],  j = 0..accept_len[b]
 * with all sources read before any destination is written, then
 *   kv->seq_len[b] = L_b + accept_len[b] + 1   (device).
 * Rows below L_b and all other slabs are untouched; slab rows past the new
 * length are scratch.  accept_len / path are the device outputs of
 * specmemo_accept.  A sequence whose accept_len or path entries are out of
 * range (negative, past its tree, or not increasing) is left untouched,
 * including its seq_len. */
int specmemo_kv_compact(specmemo_dtype dt, const specmemo_trees *t, const specmemo_kv *kv,
                        const int32_t *accept_len, const int32_t *path, int32_t path_stride,
                        void *stream);

/* (c) + (d) fused: specmemo_accept followed by specmemo_kv_compact, with the
 * compaction done by the acceptance's second pass (one launch fewer; the
 * cited passages are those of the two calls).  Arguments, outputs,
 * workspace (SPECMEMO_WS_ACCEPT) and checks are those of the two calls
 * together; a rejected call changes nothing.  Every sequence is compacted
 * along the path this call picks, and kv->seq_len[b] becomes
 * L_b + accept_len[b] + 1.  The results equal those of the two calls in
 * sequence, bit for bit. */
int specmemo_accept_compact(specmemo_dtype dt, const specmemo_trees *t, const specmemo_kv *kv,
                            int32_t vocab, specmemo_accept_mode mode, float temperature, float eps,
                            float delta, const void *base_logits, const int32_t *node_tok,
                            int32_t *accept_len, int32_t *path, int32_t path_stride,
                            int32_t *next_tok, void *ws, size_t ws_bytes, void *stream);

/* ---- Padded batching (Sec. 3.3, Fig. 8) --------------------------------------
 *
 * The paper's own batching keeps a batch's tensors uniform: after
 * verification every sequence's accepted tokens are padded to the batch's
 * longest acceptance, the pad tokens stay in the KV cache and take -inf in the
 * attention mask of later steps, and position IDs skip them.  These two calls
 * are that variant, for comparison with compaction (specmemo_kv_compact),
 * which needs no pads.
 *
 * key_valid: device uint32 flags over the pool's rows, bit (r % 32) of word
 * r / 32 for pool row r: 1 = a token, 0 = a pad token.  The array holds
 * specmemo_key_mask_words(cap_total) words (the kernels read up to three words
 * past the last row's); the calls take its length, key_valid_words, and
 * reject a shorter array.  Only committed rows (slab rows below L_b) are
 * consulted; this step's tree rows are always tokens. */

/* Words of a key_valid array for a pool of cap_total rows (0 if cap_total < 1). */
int64_t specmemo_key_mask_words(int64_t cap_total);

/* (b') Tree attention over a cache that holds pad tokens: specmemo_tree_attn
 * with every committed key whose key_valid bit is 0 masked with -inf.  Same
 * arguments, checks and workspace (SPECMEMO_WS_ATTN) as specmemo_tree_attn;
 * key_valid must be non-NULL and 16-byte aligned.  A row whose committed keys
 * are all pads still sees its tree path. */
int specmemo_tree_attn_padded(specmemo_dtype dt, const specmemo_trees *t, const specmemo_kv *kv,
                              const uint32_t *key_valid, int64_t key_valid_words, int32_t n_q, float scale,
                              const void *q, void *out, void *ws, size_t ws_bytes, void *stream);

/* (d') Padded KV update, in place of specmemo_kv_compact.  With
 * tau_b = accept_len[b] + 1 and the uniform length T = max_b tau_b over the
 * sequences whose path is valid:
 *   slab row L_b + j <- slab row L_b + path[b][j], j = 0..accept_len[b]
 *   (as in compaction), then
 *   key_valid of rows L_b .. L_b + tau_b - 1 := 1, of rows
 *   L_b + tau_b .. L_b + T - 1 := 0 (pad tokens: the rejected tree rows
 *   that were there, now masked),
 *   kv->seq_len[b] = L_b + T, pos[b] += tau_b (device int32 [B]: the
 *   position of the next token, counting no pads).
 * A path is valid if it is a root path of the tree (path[b][0] = 0, each
 * entry the parent of the next, accept_len in range); a sequence with an
 * invalid path is left untouched and does not count toward T.  Every sequence
 * must have room for the longest possible acceptance:
 * L_b + (deepest tree of the batch) + 1 <= seq_cap[b], else SPECMEMO_E_BUDGET.
 * key_valid: 4-byte aligned (flags of neighbouring slabs may share a word;
 * they are changed atomically).  ws: at least
 * specmemo_workspace_bytes(SPECMEMO_WS_PAD, ...) bytes, 4-byte aligned
 * (the uniform length). */
int specmemo_kv_pad_update(specmemo_dtype dt, const specmemo_trees *t, const specmemo_kv *kv,
                           const int32_t *accept_len, const int32_t *path, int32_t path_stride,
                           uint32_t *key_valid, int64_t key_valid_words, int32_t *pos, void *ws, size_t ws_bytes,
                           void *stream);

/* ---- Memory budget and tree construction (host only) -------------------------
 *
 * SpecMemo's memory model (Sec. 3.1, Eq. 1-6) and its tree construction
 * (Sec. 3.2 and Alg. 1) as plain host functions: they make no HIP call, read
 * and write host memory only, and may run on any thread.  Byte counts are
 * int64; a result that would overflow int64 is reported as an error.
 *
 * Trees given to or returned by these calls are in breadth-first order: node 0
 * is the root (parent -1, depth 0, rank 0); for n > 0, 0 <= parent[n] < n,
 * depth[n] = depth[parent[n]] + 1, and the triples (depth, parent, rank)
 * strictly increase with n.  Every prefix of such a tree is a tree.  Rank is
 * the node's index into head depth[n]'s top-k list, so the leftmost nodes of a
 * level carry the most probable tokens (Sec. 3.2, Fig. 10). */

/* Eq. 1, with the per-head dimension d that the equation's legend defines:
 * bytes of K and V for `tokens` cached positions of every layer, sequence and
 * KV head, 2 * layers * batch * n_kv * head_dim * tokens * elem_bytes.
 * Arguments must be >= 0 (elem_bytes >= 1).  Returns -1 on a negative
 * argument or overflow (specmemo_last_error says which). */
int64_t specmemo_mem_kv_bytes(int32_t layers, int32_t batch, int32_t n_kv, int32_t head_dim, int64_t tokens,
                              int32_t elem_bytes);

/* Eq. 3 times the precision: runtime buffers of the verification step,
 * elem_bytes * (b*N*w + b*S*l*w + b*S*l*l*w) with b = batch, N = nodes,
 * S = seqs (leaves: candidate sequences), l = levels (Medusa heads),
 * w = vocab.  Returns -1 on a negative argument or overflow. */
int64_t specmemo_mem_buffer_bytes(int32_t batch, int32_t nodes, int32_t seqs, int32_t levels, int32_t vocab,
                                  int32_t elem_bytes);

/* Eq. 4-6: total device memory, base_model_bytes + heads * head_bytes + kv +
 * buffers (Eq. 6 applies the precision once, inside each term).  Returns -1
 * on a negative argument or overflow. */
int64_t specmemo_mem_total_bytes(int64_t base_model_bytes, int64_t head_bytes, int32_t heads, int64_t kv,
                                 int64_t buffers);

/* Eq. 2: nodes of the full tree of the given arity with `levels` levels below
 * the root, sum_{i=0..levels} arity^i.  Returns -1 if arity < 1, levels < 0
 * or the count overflows. */
int64_t specmemo_tree_full_nodes(int32_t arity, int32_t levels);

/* Building a tree from its features (Sec. 3.2 and Alg. 1's custom tree): a
 * breadth-first tree with exactly `nodes` nodes and `leaves` leaves (the
 * candidate sequences), depth <= max_depth and at most `arity` children per
 * node.  The paper gives no construction; this one keeps
 * min(arity, leaves, nodes - 1) nodes at level 1 (all k tokens when the leaf
 * count allows, Sec. 3.2), then gives children to leaves in breadth-first
 * order (shallowest, then leftmost), the first of them the most, so the tree
 * is wide at the top and its leftmost branches are the deepest.  It succeeds
 * whenever some tree with these features, depth and arity exists.
 * parent/depth/rank: host int32 [nodes], written on success only.
 * Returns SPECMEMO_OK; SPECMEMO_E_ARG for nodes outside 1..2^24, leaves < 1,
 * max_depth < 0, arity < 1 or a NULL output; SPECMEMO_E_TREE when no such
 * tree exists. */
int specmemo_tree_build(int32_t nodes, int32_t leaves, int32_t max_depth, int32_t arity, int32_t *parent,
                        int32_t *depth, int32_t *rank);

/* Leaves of a breadth-first tree (its candidate sequences, Sec. 3.1), or -1
 * if the arrays break the conventions above (host arrays [n], n >= 1). */
int32_t specmemo_tree_leaves(int32_t n, const int32_t *parent, const int32_t *depth, const int32_t *rank);

/* Right-to-left pruning of a mask (Sec. 3.2): at depth d >= 1 keep the
 * keep[d-1] leftmost nodes whose parents are kept (depths past n_keep keep
 * none); the rightmost nodes of each level go first.  Per-level counts are
 * what a pruning-rate schedule (Figs. 6/7) produces; the paper's logistic
 * schedule is given only as a plot, so its counts are the caller's.
 * Input: a breadth-first tree of n nodes (host).  Output: the kept nodes in
 * the same order, parents renumbered, depths and ranks unchanged, in host
 * arrays of n entries; *n_out = kept nodes.  The output arrays may be the
 * input arrays themselves (pruning in place), but may not overlap them
 * otherwise.
 * Returns SPECMEMO_OK, SPECMEMO_E_ARG (n < 1, n_keep < 0, a negative keep
 * count, NULL pointers) or SPECMEMO_E_TREE (the input breaks the conventions).
 * Pruning a breadth-first tree to its first m nodes is the same operation with
 * only the deepest kept level cut, which is why the planners below return a
 * node count: the planned tree is that prefix. */
int specmemo_tree_prune(int32_t n, const int32_t *parent, const int32_t *depth, const int32_t *rank,
                        int32_t n_keep, const int32_t *keep, int32_t *n_out, int32_t *parent_out,
                        int32_t *depth_out, int32_t *rank_out);

/* The model, device and workload that Alg. 1 plans for. */
typedef struct {
  int64_t max_memory;         /* device bytes available */
  int64_t base_model_bytes;   /* Eq. 5: parameters x precision */
  int64_t head_bytes;         /* Eq. 4: one Medusa head */
  int32_t layers;             /* Eq. 1: h */
  int32_t n_kv;               /* Eq. 1: k, KV heads */
  int32_t head_dim;           /* Eq. 1: d */
  int32_t vocab;              /* Eq. 3: w */
  int32_t elem_bytes;         /* p, bytes per element of KV and buffers */
  int32_t batch;              /* b */
  int32_t query_count;        /* Eq. 1: n queries ... */
  int32_t query_length;       /* ... of m tokens each: the minimum cache */
  int32_t default_heads;      /* heads of the default configuration */
} specmemo_budget;

#define SPECMEMO_PLAN_DEFAULT 0     /* default tree and heads fit */
#define SPECMEMO_PLAN_PRUNED 1      /* default heads, tree pruned */
#define SPECMEMO_PLAN_FEWER_HEADS 2 /* fewer heads (>= 2), tree cut to them and pruned */
#define SPECMEMO_PLAN_NONE (-1)     /* nothing fits: Alg. 1 would quantise the base model */

typedef struct {
  int32_t kind;               /* SPECMEMO_PLAN_* */
  int32_t heads;              /* Medusa heads = tree levels (0 for NONE) */
  int32_t nodes;              /* the planned tree is the default tree's first `nodes` nodes */
  int32_t leaves;             /* its candidate sequences */
  int64_t kv_bytes;           /* Eq. 1 for query_count x query_length tokens */
  int64_t total_bytes;        /* Eq. 6 of the plan (0 for NONE) */
} specmemo_budget_plan;

/* Alg. 1 without its quantisation step.  The minimum cache is Eq. 1 for
 * query_count x query_length tokens.  If the default tree with default_heads
 * fits max_memory (Eq. 6), that is the plan.  Otherwise, for heads h from
 * default_heads down to 2 (every one-head tree has the same shape, appendix), the
 * default tree cut to depth h is pruned right to left one node at a time
 * (down to 2 nodes) and the first, largest, tree that fits is the plan.
 * default tree: breadth-first, host [n], depth <= default_heads.
 * Returns SPECMEMO_OK with *out filled (kind NONE when nothing fits);
 * SPECMEMO_E_ARG for NULL pointers, default_heads < 2, non-positive sizes
 * (max_memory, base and head bytes may be 0) or overflow; SPECMEMO_E_TREE for
 * a bad default tree. */
int specmemo_plan_budget(const specmemo_budget *m, int32_t n, const int32_t *parent, const int32_t *depth,
                         const int32_t *rank, specmemo_budget_plan *out);

/* Per-sequence tree sizes under the KV budget (Sec. 3.1, KV-cache paragraph):
 * nodes_out[b] = max(0, min(default_nodes, seq_cap[b] - seq_len[b])), the
 * largest right-to-left pruning of the default tree whose K/V rows fit the
 * slab's free rows this step; 0 means the slab is full.  Host arrays [B].
 * Returns SPECMEMO_OK, or SPECMEMO_E_ARG (B < 0, default_nodes outside
 * 1..SPECMEMO_MAX_TREE_NODES, NULL arrays, seq_len[b] < 0 or seq_cap[b] < 0). */
int specmemo_plan_tree_sizes(int32_t B, const int32_t *seq_len_h, const int32_t *seq_cap_h, int32_t default_nodes,
                             int32_t *nodes_out);

#define SPECMEMO_WS_TOPK 0
#define SPECMEMO_WS_ATTN 1
#define SPECMEMO_WS_ACCEPT 2
#define SPECMEMO_WS_PAD 3
#define SPECMEMO_WS_SAMPLE 4

/* Workspace bytes a call needs for these arguments (host-side; the only HIP
 * calls query the current device's compute-unit count, which the attention
 * work split depends on; 256 is assumed when no device is visible).
 *   SPECMEMO_WS_TOPK:   kv ignored; n_q_or_heads = n_heads; vocab used (the
 *                       fp32 logits, none when logits_out is given; bf16 also
 *                       the maxima of 64-row groups, which let the top-k pass
 *                       with packed heads read only the groups that can hold a
 *                       top-k value; without room for them it scans every
 *                       logit, with the same result).
 *   SPECMEMO_WS_ATTN:   kv required; n_q_or_heads = n_q; vocab ignored.
 *   SPECMEMO_WS_ACCEPT: kv ignored; n_q_or_heads = accept mode; vocab ignored
 *                       (with more than 32 sequences it includes the
 *                       compaction descriptors of specmemo_accept_compact).
 *   SPECMEMO_WS_PAD:    specmemo_kv_pad_update; kv, n_q_or_heads and vocab
 *                       ignored.
 *   SPECMEMO_WS_SAMPLE: specmemo_sample_next; kv and n_q_or_heads ignored;
 *                       vocab used.
 * Returns 0 for invalid arguments as well as when no workspace is needed;
 * the call itself reports invalid arguments. */
size_t specmemo_workspace_bytes(int32_t which, specmemo_dtype dt, const specmemo_trees *t,
                                const specmemo_kv *kv, int32_t n_q_or_heads, int32_t vocab);

/* Description of the last failure on the calling thread (library-owned,
 * valid until the thread's next call), or "" after a success. */
const char *specmemo_last_error(void);

/* SPECMEMO_ABI_VERSION of the loaded library. */
int32_t specmemo_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SPECMEMO_H */
