// Host tables into device memory without a copy call: a kernel whose
// arguments carry up to kUploadWords 4-byte words writes them to the
// destination.  Batches of more than kMaxSeqPerLaunch sequences use it to
// place their per-sequence descriptors and block maps in the workspace, so
// that one launch of a stage covers the whole batch.  Being kernels, the
// uploads are stream-ordered, can be captured in a graph, and read only
// memory the launch itself copied (the host table may change right after the
// call).
#include <algorithm>
#include <cstring>

#include "internal.h"

namespace specmemo {

namespace {

struct UploadArgs {
  uint32_t *dst;
  int32_t words;
  uint32_t w[kUploadWords];
};
static_assert(sizeof(UploadArgs) <= 4096, "kernel arguments are limited to 4 KB");

__global__ __launch_bounds__(256) void upload_words(UploadArgs a) {
  for (int i = threadIdx.x; i < a.words; i += 256) a.dst[i] = a.w[i];
}

}  // namespace

hipError_t upload_table(const void *src, size_t bytes, void *dst, hipStream_t st) {
  const uint8_t *s = static_cast<const uint8_t *>(src);
  uint8_t *d = static_cast<uint8_t *>(dst);
  for (size_t off = 0; off < bytes; off += (size_t)kUploadWords * 4) {
    UploadArgs a;
    const size_t n = std::min(bytes - off, (size_t)kUploadWords * 4);
    a.dst = reinterpret_cast<uint32_t *>(d + off);
    a.words = (int32_t)((n + 3) / 4);
    a.w[a.words - 1] = 0;
    memcpy(a.w, s + off, n);
    hipLaunchKernelGGL(upload_words, dim3(1), dim3(256), 0, st, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace specmemo
