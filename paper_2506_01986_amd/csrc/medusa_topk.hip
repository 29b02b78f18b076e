// Stage (a): Medusa-head projection, per-head top-k and tree-token assembly.
//
// SpecMemo Sec. 3.1: l parallel heads read the last hidden state, and head i's
// top-k tokens populate level i+1 of the candidate tree (Eq. 2); a node's token
// depends only on its depth and rank.
//
// head_logits_bf16: z[b][i][v] = sum_c W[i][v][c] * h[b][c].  The weight stream
// (l * vocab * hidden bf16, 2.1 GB for a 70B-shaped model) is the largest read of
// the step and is HBM-bound for any batch, so each wave streams 64 vocabulary rows
// with 16-byte loads and contracts them against up to 16 hidden states on the
// 16x16x32 bf16 matrix cores (batch padded to 16: the padding costs matrix-core
// time that is far below the load time).
#include "device.h"
#include "internal.h"

namespace specmemo {

namespace {

constexpr int kRowsPerWave = 64;   // four 16-row A tiles
constexpr int kWaves = 4;
constexpr int kUnroll = 4;         // k-steps of 32 issued before their MFMAs

template <int NB>   // 16-wide batch tiles contracted per weight load
__global__ __launch_bounds__(kWaves * 64) void head_logits_bf16(
    const uint16_t *__restrict__ h, const uint16_t *__restrict__ W, float *__restrict__ z, int B,
    int hidden, int vocab, int n_heads) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int head = blockIdx.y, b0 = blockIdx.z * 16 * NB;
  const int row0 = (blockIdx.x * kWaves + wave) * kRowsPerWave;
  if (row0 >= vocab) return;
  const int r16 = lane & 15, kq = lane >> 4;

  const uint16_t *wp[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    int row = min(row0 + t * 16 + r16, vocab - 1);
    wp[t] = W + ((int64_t)head * vocab + row) * hidden + kq * 8;
  }
  bool bvalid[NB];
  const uint16_t *hp[NB];
#pragma unroll
  for (int n = 0; n < NB; ++n) {
    int b = b0 + 16 * n + r16;
    bvalid[n] = b < B;
    hp[n] = h + (int64_t)(bvalid[n] ? b : 0) * hidden + kq * 8;
  }

  f32x4 acc[NB][4];
#pragma unroll
  for (int n = 0; n < NB; ++n)
#pragma unroll
    for (int t = 0; t < 4; ++t) acc[n][t] = f32x4{0.f, 0.f, 0.f, 0.f};

  int k = 0;
  for (; k + 32 * kUnroll <= hidden; k += 32 * kUnroll) {
    uint4 a[kUnroll][4], bq[kUnroll][NB];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
#pragma unroll
      for (int t = 0; t < 4; ++t) a[u][t] = *reinterpret_cast<const uint4 *>(wp[t] + k + 32 * u);
#pragma unroll
      for (int n = 0; n < NB; ++n)
        bq[u][n] = ld16_or_zero(bvalid[n], hp[n] + k + 32 * u);
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
#pragma unroll
      for (int n = 0; n < NB; ++n) {
        bf16x8 bv = __builtin_bit_cast(bf16x8, bq[u][n]);
#pragma unroll
        for (int t = 0; t < 4; ++t)
          acc[n][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a[u][t]),
                                                              bv, acc[n][t], 0, 0, 0);
      }
  }
  for (; k < hidden; k += 32) {   // tail: hidden % 8 == 0, so a lane's 8 elements are all in or all out
    const bool in = k + kq * 8 < hidden;
    uint4 a[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) a[t] = ld16_or_zero(in, wp[t] + k);
#pragma unroll
    for (int n = 0; n < NB; ++n) {
      uint4 bq = ld16_or_zero(in && bvalid[n], hp[n] + k);
      bf16x8 bv = __builtin_bit_cast(bf16x8, bq);
#pragma unroll
      for (int t = 0; t < 4; ++t)
        acc[n][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a[t]), bv,
                                                            acc[n][t], 0, 0, 0);
    }
  }

  // C layout: lane holds column (batch) lane&15, rows 4*(lane>>4) + 0..3 of each tile.
#pragma unroll
  for (int n = 0; n < NB; ++n) {
    const int b = b0 + 16 * n + (lane & 15);
    if (b >= B) continue;
    float *zr = z + ((int64_t)b * n_heads + head) * vocab;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      int row = row0 + t * 16 + 4 * kq;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (row + j < vocab) zr[row + j] = acc[n][t][j];
    }
  }
}

// fp32 heads: one wave per vocabulary row, lanes stride the hidden dimension.
constexpr int kF32BatchTile = 8;

__global__ __launch_bounds__(256) void head_logits_f32(const float *__restrict__ h,
                                                       const float *__restrict__ W,
                                                       float *__restrict__ z, int B, int hidden,
                                                       int vocab, int n_heads) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int head = blockIdx.y;
  const int row = blockIdx.x * 4 + wave;
  if (row >= vocab) return;
  const float *wr = W + ((int64_t)head * vocab + row) * hidden;
  for (int b0 = 0; b0 < B; b0 += kF32BatchTile) {
    float acc[kF32BatchTile];
#pragma unroll
    for (int j = 0; j < kF32BatchTile; ++j) acc[j] = 0.f;
    for (int c = lane; c < hidden; c += 64) {
      float w = wr[c];
#pragma unroll
      for (int j = 0; j < kF32BatchTile; ++j)
        if (b0 + j < B) acc[j] = fmaf(w, h[(int64_t)(b0 + j) * hidden + c], acc[j]);
    }
#pragma unroll
    for (int j = 0; j < kF32BatchTile; ++j) {
      float v = acc[j];
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
      if (lane == 0 && b0 + j < B) z[((int64_t)(b0 + j) * n_heads + head) * vocab + row] = v;
    }
  }
}

// Top-k of one (sequence, head) logit row, then the tree tokens of that head's
// level.  Each thread keeps a sorted list of its KM best (value, id) pairs in
// registers; k rounds of a block-wide arg-best then pop the global order.
template <int KM>
__global__ __launch_bounds__(256) void topk_assemble(TopkArgs a) {
  const int row = blockIdx.x;              // b * n_heads + head
  const int b = row / a.n_heads, head = row % a.n_heads;
  const int k = a.k[head];
  const float *x = a.z + (int64_t)row * a.vocab;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  float lv[KM];
  int li[KM];
#pragma unroll
  for (int j = 0; j < KM; ++j) {
    lv[j] = -INFINITY;
    li[j] = INT32_MAX;
  }
  for (int v = tid; v < a.vocab; v += 256) {
    float xv = x[v];
    if (!better(xv, v, lv[KM - 1], li[KM - 1])) continue;
    float cv = xv;
    int ci = v;
#pragma unroll
    for (int j = 0; j < KM; ++j) {         // insertion by compare-exchange down the list
      if (better(cv, ci, lv[j], li[j])) {
        float tv = lv[j];
        int ti = li[j];
        lv[j] = cv;
        li[j] = ci;
        cv = tv;
        ci = ti;
      }
    }
  }

  __shared__ float sv[4];
  __shared__ int si[4];
  __shared__ int sel[KM];
  __shared__ float selv[KM];
  for (int j = 0; j < k; ++j) {
    float bv = lv[0];
    int bi = li[0];
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      float ov = __shfl_xor(bv, off);
      int oi = __shfl_xor(bi, off);
      if (better(ov, oi, bv, bi)) {
        bv = ov;
        bi = oi;
      }
    }
    if (lane == 0) {
      sv[wave] = bv;
      si[wave] = bi;
    }
    __syncthreads();
    bv = sv[0];
    bi = si[0];
#pragma unroll
    for (int w = 1; w < 4; ++w)
      if (better(sv[w], si[w], bv, bi)) {
        bv = sv[w];
        bi = si[w];
      }
    if (tid == 0) {
      sel[j] = bi < a.vocab ? bi : -1;
      selv[j] = bv;
    }
    if (li[0] == bi) {                       // ids are unique: exactly one thread pops
#pragma unroll
      for (int t = 0; t < KM - 1; ++t) {
        lv[t] = lv[t + 1];
        li[t] = li[t + 1];
      }
      lv[KM - 1] = -INFINITY;
      li[KM - 1] = INT32_MAX;
    }
    __syncthreads();
  }

  int32_t *ids = a.ids + (int64_t)row * a.kmax;
  for (int j = tid; j < a.kmax; j += 256) {
    ids[j] = j < k ? sel[j] : -1;
    if (a.vals) a.vals[(int64_t)row * a.kmax + j] = j < k ? selv[j] : -INFINITY;
  }
  const int n0 = a.node_off[b], n1 = a.node_off[b + 1];
  for (int n = n0 + tid; n < n1; n += 256) {
    if (n == n0) {
      if (head == 0) a.node_tok[n] = a.root_tok[b];
    } else if (a.depth[n] == head + 1) {
      a.node_tok[n] = sel[a.rank[n]];
    }
  }
}

}  // namespace

hipError_t launch_head_logits(int dt, const void *h, const void *w, float *z, int B, int hidden,
                              int vocab, int n_heads, hipStream_t st) {
  if (dt == 1) {
    const int nb = B <= 16 ? 1 : 2;
    dim3 grid((vocab + kWaves * kRowsPerWave - 1) / (kWaves * kRowsPerWave), n_heads,
              (B + 16 * nb - 1) / (16 * nb));
    auto kern = nb == 1 ? head_logits_bf16<1> : head_logits_bf16<2>;
    hipLaunchKernelGGL(kern, grid, dim3(kWaves * 64), 0, st, static_cast<const uint16_t *>(h),
                       static_cast<const uint16_t *>(w), z, B, hidden, vocab, n_heads);
  } else {
    dim3 grid((vocab + 3) / 4, n_heads);
    hipLaunchKernelGGL(head_logits_f32, grid, dim3(256), 0, st, static_cast<const float *>(h),
                       static_cast<const float *>(w), z, B, hidden, vocab, n_heads);
  }
  return hipGetLastError();
}

hipError_t launch_topk(const TopkArgs &a, int B, hipStream_t st) {
  dim3 grid(B * a.n_heads);
  if (a.kmax <= 16)
    hipLaunchKernelGGL(topk_assemble<16>, grid, dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL(topk_assemble<32>, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace specmemo
