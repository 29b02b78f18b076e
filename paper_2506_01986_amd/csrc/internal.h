// Internal declarations shared by the HIP kernels and the C-ABI layer of
// libspecmemo (gfx950).  Nothing here is part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace specmemo {

constexpr int kMaxSeqPerLaunch = 32;   // per-sequence descriptors travel in kernel arguments
constexpr int kMaxNodes = 128;
constexpr int kMaxPath = 16;           // max depth + 1
constexpr int kMaxTopk = 32;
constexpr int kMaxHeads = 15;

// Host tables written into device memory by kernels whose arguments carry up
// to kUploadWords words each (csrc/upload.hip); bytes may be any size, dst
// 4-byte aligned.
constexpr int kUploadWords = 1000;
hipError_t upload_table(const void *src, size_t bytes, void *dst, hipStream_t st);

// Error reporting of the C ABI: `fail` records the message that
// specmemo_last_error returns and passes `code` through; `ok` clears it.
int fail(int code, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
int ok();

// ---- head projection + top-k -------------------------------------------------
struct TopkArgs {
  const float *z;          // [B][n_heads][vocab] fp32 logits
  const float *gmax;       // [B][n_heads][nG] maxima of 64-row groups, or null (then every value is scanned)
  int32_t nG;
  int32_t vocab, n_heads, kmax;
  int32_t k[kMaxHeads];    // top-k per head
  const int32_t *node_off, *depth, *rank, *root_tok;
  int32_t *ids;            // [B][n_heads][kmax]
  float *vals;             // same or null
  int32_t *node_tok;
};

// h_head_stride: elements between the heads' inputs (0: every head reads the same h).
// gmax non-null (packed bf16 only): also the maxima of 64-row groups, [B][n_heads][nG].
hipError_t launch_head_logits(int dt, const void *h, int64_t h_head_stride, const void *w, bool packed, float *z,
                              int B, int hidden, int vocab, int n_heads, hipStream_t st, float *gmax = nullptr);
// Medusa residual blocks: out[i][b] = h[b] + SiLU(W1_i h[b] + b1_i); bf16 W1 packed like the heads.
hipError_t launch_resblock(int dt, const void *h, const void *w1, const void *b1, void *out, int B, int hidden,
                           int n_heads, hipStream_t st);
// Packed head weights: 64-row groups x 32-column k steps of 4 KB each.
__host__ __device__ constexpr int packed_row_groups(int vocab) { return (vocab + 63) / 64; }
__host__ __device__ constexpr int packed_k_steps(int hidden) { return (hidden + 31) / 32; }
hipError_t launch_pack_heads(const void *src, void *dst, int n_heads, int vocab, int hidden, hipStream_t st);
hipError_t launch_topk(const TopkArgs &a, int B, hipStream_t st);

// ---- tree attention ------------------------------------------------------------
struct AttnSeq {
  int64_t base;      // first pool row of the slab
  int32_t L;         // committed rows
  int32_t node0;     // global id of the root node
  int32_t N;         // tree nodes
  int32_t nrb;       // row blocks (bf16 path)
  int32_t nch;       // KV chunks
  int32_t ch_len;    // keys per chunk (multiple of the key tile); last chunk takes the rest
  int32_t item0;     // first work item of this sequence in the launch
  int32_t part0;     // first partial slot (multi-chunk sequences), -1 if none
  int32_t citem0;    // first combine item (multi-chunk sequences)
  int32_t unit0;     // first (sequence, KV head) unit of this sequence in the launch
};

struct AttnItem {
  uint16_t s, kvh, ch, rb;
};

struct AttnArgs {
  const void *q;
  void *out;
  const void *k, *v;
  const int32_t *parent;
  const uint32_t *key_valid;   // padded batching: bit r of the pool's row r, 0 = pad token; null: no pads
  float *part;             // partial results workspace
  // Table mode (more than kMaxSeqPerLaunch sequences): the descriptors of all
  // the launch's sequences and the decoded item of every block live in the
  // workspace (written by upload_table before the launch); null otherwise.
  const AttnSeq *tab;
  const AttnItem *map;     // attention blocks: sequence, KV head, chunk, row block (seq 0xFFFF: padding)
  const AttnItem *cmap;    // combine blocks: sequence, KV head, row block
  int64_t cap_total;
  int32_t n_q, n_kv, group, head_dim;
  float scale_log2;        // scale * log2(e)
  float scale;
  int32_t nseq, items, citems;   // items: blocks of the launch (XCD order: padded)
  int32_t xcd_order;        // nonzero: consecutive work items share an XCD
  int32_t xcd_cum[8][kMaxSeqPerLaunch + 1];   // XCD order: blocks of XCD x before sequence s
  int32_t xcd_ccum[8][kMaxSeqPerLaunch + 1];  // XCD order: combine blocks of XCD x before sequence s
  AttnSeq seq[kMaxSeqPerLaunch];
};

static_assert(sizeof(AttnArgs) <= 4096, "kernel arguments are limited to 4 KB");
static_assert(kMaxSeqPerLaunch <= 64, "one wave searches the sequences of a launch");

constexpr int kAttnKeyTile = 64;
constexpr int kAttnHeadDim = 128;
// 4-byte words per partial slot of a row block: unnormalised O in bf16
// ([rows][head_dim]), then the running max and running sum in fp32 ([rows] each)
__host__ __device__ constexpr int64_t attn_partial_floats(int rows_per_block) {
  return (int64_t)rows_per_block * (kAttnHeadDim / 2 + 2);
}
hipError_t launch_tree_attn_bf16(const AttnArgs &a, int rows_per_block, hipStream_t st);
// Static scratch of the allocation-free attention entry point: its size, and
// this device's address of it (looked up once per device, on first use).
constexpr size_t kAttnStaticScratchBytes = size_t(32) << 20;
hipError_t attn_static_scratch(void **ptr);
hipError_t launch_tree_attn_f32(const AttnArgs &a, int node_begin, int node_count, hipStream_t st);

// ---- acceptance ------------------------------------------------------------------
struct AcceptArgs {
  const void *logits;
  const int32_t *node_tok, *node_off, *parent, *depth;
  int32_t vocab, mode, path_stride, B;
  float inv_temp, log_eps, log_delta;
  float *stats;            // typical: [sum N][2] (lse, entropy) of z / T
  int32_t *best;           // [sum N] arg-best token of each node's row (typical: after stats)
  int32_t *accept_len, *path, *next_tok;
};
hipError_t launch_accept(int dt, const AcceptArgs &a, int total_nodes, hipStream_t st);
struct SampleArgs {
  const void *logits;
  const int32_t *node_off, *accept_len, *path;
  int32_t vocab, path_stride;
  float inv_temp;          // 1 / T, rounded once to fp32 on the host
  uint64_t seed, offset;   // Philox key
  int32_t *next_tok;
};
// words: the workspace of the segmented form (B x sample_segments(vocab)
// 64-bit words), or nullptr for one block per sequence.
int sample_segments(int vocab);
hipError_t launch_sample_next(int dt, const SampleArgs &a, int B, uint64_t *words, hipStream_t st);

// ---- compaction ------------------------------------------------------------------
struct CompactSeq {
  int64_t base;
  int32_t L, N, cap, node0;   // node0: global id of the root node
};
struct CompactArgs {
  const CompactSeq *tab;   // table mode: all sequences' descriptors in device memory (seq[] unused)
  void *k, *v;
  int64_t cap_total;
  int32_t n_kv, row_dwords, path_stride, nseq, b0;
  const int32_t *accept_len, *path;
  const int32_t *parent;   // padded update: the trees' parents (root paths are checked)
  int32_t *seq_len;
  CompactSeq seq[kMaxSeqPerLaunch];
};
hipError_t launch_kv_compact(const CompactArgs &a, hipStream_t st);
// Acceptance with the compaction fused into its second pass (one launch group
// of sequences; the row pass of launch_accept_rows must precede it).
hipError_t launch_accept_rows(int dt, const AcceptArgs &a, int total_nodes, hipStream_t st);
hipError_t launch_accept_compact(int dt, const AcceptArgs &a, const CompactArgs &c, hipStream_t st);
// Padded batching: the batch's uniform acceptance length into *uniform (one
// block), then the row moves and the per-sequence bookkeeping.
hipError_t launch_pad_length(const int32_t *node_off, const int32_t *parent, const int32_t *accept_len,
                             const int32_t *path, int32_t path_stride, int32_t B, int32_t *uniform, hipStream_t st);
hipError_t launch_kv_pad_update(const CompactArgs &a, const int32_t *uniform, uint32_t *key_valid, int32_t *pos,
                                hipStream_t st);

}  // namespace specmemo
