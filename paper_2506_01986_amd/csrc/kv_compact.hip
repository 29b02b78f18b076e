// Stage (d): in-place compaction of the accepted path's K/V.
//
// SpecMemo Sec. 3.1 (KV-cache paragraph): the preallocated KV cache is a scratch
// space updated during verification, sized precisely to the budget; Sec. 3.3:
// rejected candidates are discarded.  After acceptance the accepted nodes' K/V
// rows (tree rows L + path[j]) move to rows L + j of the same slab, and the
// sequence length grows by accept_len + 1; the rest of the tree rows become
// free scratch for the next step.
//
// One wave per (sequence, KV head, K|V) moves the rows (compact_rows.h).
#include "compact_rows.h"
#include "device.h"
#include "internal.h"

namespace specmemo {

namespace {

// Sequence b's accepted path: accept_len and the path entries are loaded
// together (one memory latency), up to the row's stride, and checked: a path
// starts at the root and increases strictly inside the tree.  The slab bound
// is the caller's.  Returns accept_len, or -1 for an invalid path.
__device__ __forceinline__ int load_path(const int32_t *accept_len, const int32_t *paths, int path_stride, int b,
                                         int N, int (&src)[kMaxPath]) {
  const int acc = accept_len[b];
  const int32_t *path = paths + (int64_t)b * path_stride;
  const int np = min(kMaxPath, path_stride);
#pragma unroll
  for (int j = 0; j < kMaxPath; ++j) src[j] = j < np ? path[j] : -1;
  bool ok = acc >= 0 && acc < np && acc < N && src[0] == 0;
#pragma unroll
  for (int j = 1; j < kMaxPath; ++j)
    if (j <= acc) ok = ok && src[j] >= j && src[j] < N && src[j] > src[j - 1];
  return ok ? acc : -1;
}

// Padded batching takes only root paths (each entry the parent of the next),
// so that no sequence grows by more than its tree's depth + 1.
__device__ __forceinline__ bool is_root_path(const int32_t *parent, int node0, int acc, const int (&src)[kMaxPath]) {
  bool ok = true;
#pragma unroll
  for (int j = 1; j < kMaxPath; ++j)
    if (j <= acc) ok = ok && parent[node0 + src[j]] == src[j - 1];
  return ok;
}

__global__ __launch_bounds__(64) void kv_compact_kernel(CompactArgs a) {
  const int s = blockIdx.x, kvh = blockIdx.y, which = blockIdx.z;
  const CompactSeq S = a.seq[s];
  const int b = a.b0 + s;
  int src[kMaxPath];
  const int acc = load_path(a.accept_len, a.path, a.path_stride, b, S.N, src);
  // an invalid path, or one that does not fit the slab, leaves the sequence untouched
  if (acc < 0 || S.L + acc + 1 > S.cap) return;
  move_rows(a, S, kvh, which, acc, src, threadIdx.x, 64);
  if (kvh == 0 && which == 0 && threadIdx.x == 0) a.seq_len[b] = S.L + acc + 1;
}

// Padded batching (Sec. 3.3, Fig. 8): every sequence's accepted tokens are
// padded to the batch's longest acceptance, so that all sequences grow by the
// same number of rows.  One block finds that length over the whole batch;
// sequences with an invalid path do not take part.
__global__ __launch_bounds__(256) void pad_length_kernel(const int32_t *node_off, const int32_t *parent,
                                                         const int32_t *accept_len, const int32_t *path,
                                                         int path_stride, int B, int32_t *uniform) {
  __shared__ int wave_max[4];
  int best = 0;
  for (int b = threadIdx.x; b < B; b += 256) {
    int src[kMaxPath];
    const int node0 = node_off[b];
    const int acc = load_path(accept_len, path, path_stride, b, node_off[b + 1] - node0, src);
    if (acc >= 0 && is_root_path(parent, node0, acc, src)) best = max(best, acc + 1);
  }
  best = (int)wave_reduce_u32<true>((uint32_t)best);
  if ((threadIdx.x & 63) == 0) wave_max[threadIdx.x >> 6] = best;
  __syncthreads();
  if (threadIdx.x == 0) *uniform = max(max(wave_max[0], wave_max[1]), max(wave_max[2], wave_max[3]));
}

// The accepted rows move as in compaction; the sequence then grows by the
// uniform length T: rows L .. L + tau - 1 (tau = accept_len + 1) are its
// tokens, rows L + tau .. L + T - 1 pad tokens, flagged 0 in key_valid (bit r
// of word r / 32 for pool row r).  Slabs may share a flag word, so flags change
// by atomic AND / OR; T <= 16 rows touch at most two words.  The position
// (next token's index without pads) grows by tau only.
__global__ __launch_bounds__(64) void kv_pad_update_kernel(CompactArgs a, const int32_t *uniform,
                                                           uint32_t *key_valid, int32_t *pos) {
  const int s = blockIdx.x, kvh = blockIdx.y, which = blockIdx.z;
  const CompactSeq S = a.seq[s];
  const int b = a.b0 + s;
  int src[kMaxPath];
  const int acc = load_path(a.accept_len, a.path, a.path_stride, b, S.N, src);
  if (acc < 0 || !is_root_path(a.parent, S.node0, acc, src)) return;
  move_rows(a, S, kvh, which, acc, src, threadIdx.x, 64);
  if (kvh != 0 || which != 0) return;
  const int T = *uniform, tau = acc + 1;
  const int64_t r0 = S.base + S.L;
  const uint32_t sh = (uint32_t)r0 & 31u;
  const uint64_t set = ((1ull << tau) - 1) << sh;
  const uint64_t clear = (((1ull << T) - 1) ^ ((1ull << tau) - 1)) << sh;
  const int lane = threadIdx.x;
  if (lane < 2) {
    const uint32_t sw = (uint32_t)(set >> (32 * lane)), cw = (uint32_t)(clear >> (32 * lane));
    uint32_t *w = key_valid + (r0 >> 5) + lane;
    if (sw) atomicOr(w, sw);
    if (cw) atomicAnd(w, ~cw);
  }
  if (lane == 0) {
    a.seq_len[b] = S.L + T;
    pos[b] += tau;
  }
}

}  // namespace

hipError_t launch_kv_compact(const CompactArgs &a, hipStream_t st) {
  hipLaunchKernelGGL(kv_compact_kernel, dim3(a.nseq, a.n_kv, 2), dim3(64), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_pad_length(const int32_t *node_off, const int32_t *parent, const int32_t *accept_len,
                             const int32_t *path, int32_t path_stride, int32_t B, int32_t *uniform, hipStream_t st) {
  hipLaunchKernelGGL(pad_length_kernel, dim3(1), dim3(256), 0, st, node_off, parent, accept_len, path, path_stride,
                     B, uniform);
  return hipGetLastError();
}

hipError_t launch_kv_pad_update(const CompactArgs &a, const int32_t *uniform, uint32_t *key_valid, int32_t *pos,
                                hipStream_t st) {
  hipLaunchKernelGGL(kv_pad_update_kernel, dim3(a.nseq, a.n_kv, 2), dim3(64), 0, st, a, uniform, key_valid, pos);
  return hipGetLastError();
}

}  // namespace specmemo
