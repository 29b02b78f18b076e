// Stage (d): in-place compaction of the accepted path's K/V.
//
// SpecMemo Sec. 3.1 (KV-cache paragraph): the preallocated KV cache is a scratch
// space updated during verification, sized precisely to the budget; Sec. 3.3:
// rejected candidates are discarded.  After acceptance the accepted nodes' K/V
// rows (tree rows L + path[j]) move to rows L + j of the same slab, and the
// sequence length grows by accept_len + 1; the rest of the tree rows become
// free scratch for the next step.
//
// One wave per (sequence, KV head, K|V).  Each lane owns a fixed set of 4-byte
// columns of a row and reads that column of every source row into registers
// before writing any destination, so overlapping sources and destinations
// (path = 0, 2, 7, ...: destination 2 is also the source of destination 1)
// need no barrier: no two lanes touch the same bytes.
#include "internal.h"

namespace specmemo {

namespace {

__global__ __launch_bounds__(64) void kv_compact_kernel(CompactArgs a) {
  const int s = blockIdx.x, kvh = blockIdx.y, which = blockIdx.z;
  const CompactSeq S = a.seq[s];
  const int b = a.b0 + s;
  const int acc = a.accept_len[b];
  const int32_t *path = a.path + (int64_t)b * a.path_stride;
  // The path entries are loaded together with accept_len (one memory latency),
  // up to the row's stride.
  const int np = min(kMaxPath, a.path_stride);
  int src[kMaxPath];
#pragma unroll
  for (int j = 0; j < kMaxPath; ++j) src[j] = j < np ? path[j] : -1;
  // Validate the device-produced path; an invalid one leaves the sequence untouched.
  bool ok = acc >= 0 && acc < np && acc < S.N && S.L + acc + 1 <= S.cap && src[0] == 0;
#pragma unroll
  for (int j = 1; j < kMaxPath; ++j)
    if (j <= acc) ok = ok && src[j] >= j && src[j] < S.N && src[j] > src[j - 1];
  if (!ok) return;
  uint32_t *slab = static_cast<uint32_t *>(which ? a.v : a.k) +
                   ((int64_t)kvh * a.cap_total + S.base) * a.row_dwords;
  for (int c = threadIdx.x; c < a.row_dwords; c += 64) {
    uint32_t tmp[kMaxPath];
#pragma unroll
    for (int j = 0; j < kMaxPath; ++j)
      if (j <= acc) tmp[j] = slab[(int64_t)(S.L + src[j]) * a.row_dwords + c];
#pragma unroll
    for (int j = 0; j < kMaxPath; ++j)
      if (j <= acc) slab[(int64_t)(S.L + j) * a.row_dwords + c] = tmp[j];
  }
  if (kvh == 0 && which == 0 && threadIdx.x == 0) a.seq_len[b] = S.L + acc + 1;
}

}  // namespace

hipError_t launch_kv_compact(const CompactArgs &a, hipStream_t st) {
  hipLaunchKernelGGL(kv_compact_kernel, dim3(a.nseq, a.n_kv, 2), dim3(64), 0, st, a);
  return hipGetLastError();
}

}  // namespace specmemo
