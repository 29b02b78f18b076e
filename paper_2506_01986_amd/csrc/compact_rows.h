// Row moves of the in-place KV compaction, shared by the compaction kernels
// and the fused acceptance-and-compaction kernels.
//
// SpecMemo Sec. 3.1 (KV-cache paragraph): the preallocated cache is scratch
// space updated during verification; after acceptance the accepted nodes' K/V
// rows (tree rows L + path[j]) move to rows L + j of the same slab.
#pragma once

#include "internal.h"

namespace specmemo {

// Rows L + src[j] -> L + j, j = 0..acc, of KV head kvh's K (which = 0) or V
// (which = 1) slab, by `width` lanes of which this is lane `lane`.  Each lane
// owns a fixed set of 4-byte columns of a row and reads that column of every
// source row into registers before writing any destination, so overlapping
// sources and destinations (path = 0, 2, 7, ...: destination 2 is also the
// source of destination 1) need no barrier: no two lanes touch the same bytes.
__device__ __forceinline__ void move_rows(const CompactArgs &a, const CompactSeq &S, int kvh, int which, int acc,
                                          const int (&src)[kMaxPath], int lane, int width) {
  uint32_t *slab = static_cast<uint32_t *>(which ? a.v : a.k) +
                   ((int64_t)kvh * a.cap_total + S.base) * a.row_dwords;
  for (int c = lane; c < a.row_dwords; c += width) {
    uint32_t tmp[kMaxPath];
#pragma unroll
    for (int j = 0; j < kMaxPath; ++j)
      if (j <= acc) tmp[j] = slab[(int64_t)(S.L + src[j]) * a.row_dwords + c];
#pragma unroll
    for (int j = 0; j < kMaxPath; ++j)
      if (j <= acc) slab[(int64_t)(S.L + j) * a.row_dwords + c] = tmp[j];
  }
}

}  // namespace specmemo
