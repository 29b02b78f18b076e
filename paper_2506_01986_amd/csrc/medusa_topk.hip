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
constexpr int kUnroll = 2;         // k-steps of 32 issued before their MFMAs

template <int NB>   // 16-wide batch tiles contracted per weight load
__global__ __launch_bounds__(kWaves * 64) void head_logits_bf16(
    const uint16_t *__restrict__ h, int64_t h_head_stride, const uint16_t *__restrict__ W, float *__restrict__ z,
    int B, int hidden, int vocab, int n_heads) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int head = blockIdx.y, b0 = blockIdx.z * 16 * NB;
  const int gwave = blockIdx.x * kWaves + wave;
  const int row0 = gwave * kRowsPerWave;
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
    hp[n] = h + head * h_head_stride + (int64_t)(bvalid[n] ? b : 0) * hidden + kq * 8;
  }

  f32x4 acc[NB][4];
#pragma unroll
  for (int n = 0; n < NB; ++n)
#pragma unroll
    for (int t = 0; t < 4; ++t) acc[n][t] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Every wave starts its k sweep at a different step: all waves reading their
  // rows (16 KB apart) at the same offset would load the same HBM channels.
  const int steps = hidden / (32 * kUnroll);
  const int rot = steps ? (gwave + head * 977) % steps : 0;
  for (int s0 = 0; s0 < steps; ++s0) {
    const int k = (s0 + rot < steps ? s0 + rot : s0 + rot - steps) * 32 * kUnroll;
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
  int k = steps * 32 * kUnroll;
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

// Packed heads (see specmemo_pack_heads): wave (head, G) streams its row
// group's nS * 4 KB contiguously, one 1 KB operand tile per load instruction,
// and contracts each tile against the 16 hidden states of its batch tile.
constexpr int kPackedUnroll = 4;   // k steps (4 KB each) issued before their MFMAs
constexpr int kHidChunk = 16;      // k steps of hidden states staged in LDS at a time (two batch tiles)

// Weights are read once per step: nontemporal loads keep them from displacing
// the hidden states and logits in the caches.
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ld16_stream(const uint4 *p) {
  return __builtin_bit_cast(uint4, __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(p)));
}

// gmax non-null: each (batch row, head) row also gets the maximum of every
// 64-row group, [B][n_heads][nG], from which the top-k pass finds the groups
// that can hold a top-k value.
template <int NB>
__global__ __launch_bounds__(kWaves * 64) void head_logits_packed(
    const uint16_t *__restrict__ h, int64_t h_head_stride, const uint4 *__restrict__ Wp, float *__restrict__ z,
    int B, int hidden, int vocab, int n_heads, int nG, int nS, float *__restrict__ gmax) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int head = blockIdx.y, b0 = blockIdx.z * 16 * NB;
  const int G = blockIdx.x * kWaves + wave;
  const bool active = G < nG;
  const int kq = lane >> 4;
  const uint4 *wp = Wp + (int64_t)(head * (int64_t)nG + (active ? G : 0)) * nS * 4 * 64 + lane;
  f32x4 acc[NB][4];
#pragma unroll
  for (int n = 0; n < NB; ++n)
#pragma unroll
    for (int t = 0; t < 4; ++t) acc[n][t] = f32x4{0.f, 0.f, 0.f, 0.f};

  if constexpr (NB == 1) {
    // One batch tile: each wave reads its hidden-state fragments itself.
    if (!active) return;
    bool bvalid[NB];
    const uint16_t *hp[NB];
#pragma unroll
    for (int n = 0; n < NB; ++n) {
      const int b = b0 + 16 * n + (lane & 15);
      bvalid[n] = b < B;
      hp[n] = h + head * h_head_stride + (int64_t)(bvalid[n] ? b : 0) * hidden + kq * 8;
    }
    auto step = [&](const uint4 (&a)[4], int s) {
      const int k = 32 * s + 8 * kq;
#pragma unroll
      for (int n = 0; n < NB; ++n) {
        const bf16x8 bv = __builtin_bit_cast(bf16x8, ld16_or_zero(bvalid[n] && k < hidden, hp[n] + 32 * s));
#pragma unroll
        for (int t = 0; t < 4; ++t)
          acc[n][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a[t]), bv, acc[n][t], 0, 0, 0);
      }
    };
    int s = 0;
    for (; s + kPackedUnroll <= nS; s += kPackedUnroll) {
      uint4 a[kPackedUnroll][4];
#pragma unroll
      for (int u = 0; u < kPackedUnroll; ++u)
#pragma unroll
        for (int t = 0; t < 4; ++t) a[u][t] = ld16_stream(wp + ((s + u) * 4 + t) * 64);
#pragma unroll
      for (int u = 0; u < kPackedUnroll; ++u) step(a[u], s + u);
    }
    for (; s < nS; ++s) {
      uint4 a[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) a[t] = ld16_stream(wp + (s * 4 + t) * 64);
      step(a, s);
    }
  } else {
    // Two batch tiles: the second hidden-state gather per k step made the
    // vector cache the bottleneck, so the block's waves share their hidden
    // states through LDS: chunks of kHidChunk k steps (two buffers) in the B
    // operand's lane order, one 1 KB piece per (step, batch tile), read with
    // one conflict-free 16-byte LDS read per step and tile.  Entry e of a
    // piece holds row e % 16, columns 32 (step) + 8 (e / 16) .. +8; rows past
    // B, columns past hidden and steps past nS are zero.  Waves past the last
    // row group still stage hidden states and meet the barriers.
    constexpr int kPieces = kHidChunk * NB * 64;
    constexpr int kPer = kPieces / (kWaves * 64);
    __shared__ uint4 hsh[2][kPieces];
    const uint16_t *hbase = h + head * h_head_stride;
    uint4 hreg[kPer];
    auto hfetch = [&](int c) {
#pragma unroll
      for (int i = 0; i < kPer; ++i) {
        const int q = tid + i * kWaves * 64;
        const int kk = q & 3, row = (q >> 2) & 15, pn = q >> 6;
        const int n = pn % NB, sl = pn / NB;
        const int st = c * kHidChunk + sl, b = b0 + 16 * n + row, k = 32 * st + 8 * kk;
        const bool ok = b < B && k < hidden && st < nS;
        const uint4 v = *reinterpret_cast<const uint4 *>(hbase + (int64_t)(b < B ? b : 0) * hidden + min(k, hidden - 8));
        hreg[i] = ok ? v : uint4{0u, 0u, 0u, 0u};
      }
    };
    auto hstore = [&](int buf) {
#pragma unroll
      for (int i = 0; i < kPer; ++i) {
        const int q = tid + i * kWaves * 64;
        hsh[buf][(q >> 6) * 64 + (q & 3) * 16 + ((q >> 2) & 15)] = hreg[i];
      }
    };
    auto step = [&](const uint4 (&a)[4], const uint4 *hb, int sl) {
#pragma unroll
      for (int n = 0; n < NB; ++n) {
        const bf16x8 bv = __builtin_bit_cast(bf16x8, hb[(sl * NB + n) * 64 + lane]);
#pragma unroll
        for (int t = 0; t < 4; ++t)
          acc[n][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a[t]), bv, acc[n][t], 0, 0, 0);
      }
    };
    const int nch = (nS + kHidChunk - 1) / kHidChunk;
    hfetch(0);
    hstore(0);
    __syncthreads();
    for (int c = 0; c < nch; ++c) {
      if (c + 1 < nch) hfetch(c + 1);
      const uint4 *hb = hsh[c & 1];
      const int s0 = c * kHidChunk, s1 = min(nS, s0 + kHidChunk);
      if (active) {
        int s = s0;
        for (; s + kPackedUnroll <= s1; s += kPackedUnroll) {
          uint4 a[kPackedUnroll][4];
#pragma unroll
          for (int u = 0; u < kPackedUnroll; ++u)
#pragma unroll
            for (int t = 0; t < 4; ++t) a[u][t] = ld16_stream(wp + ((s + u) * 4 + t) * 64);
#pragma unroll
          for (int u = 0; u < kPackedUnroll; ++u) step(a[u], hb, s - s0 + u);
        }
        for (; s < s1; ++s) {
          uint4 a[4];
#pragma unroll
          for (int t = 0; t < 4; ++t) a[t] = ld16_stream(wp + (s * 4 + t) * 64);
          step(a, hb, s - s0);
        }
      }
      if (c + 1 < nch) hstore((c + 1) & 1);
      __syncthreads();
    }
    if (!active) return;
  }

  // C layout: lane holds column (batch) lane&15, rows 4*(lane>>4) + 0..3 of each tile.
#pragma unroll
  for (int n = 0; n < NB; ++n) {
    const int b = b0 + 16 * n + (lane & 15);
    float m = -INFINITY;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int row = 64 * G + t * 16 + 4 * kq;
#pragma unroll
      for (int j = 0; j < 4; ++j) m = row + j < vocab ? fmaxf(m, acc[n][t][j]) : m;
    }
    if (gmax) {   // the column's four lanes: l, l ^ 16, l ^ 32, l ^ 48
      m = fmaxf(m, __shfl_xor(m, 16));
      m = fmaxf(m, __shfl_xor(m, 32));
    }
    if (b >= B) continue;
    float *zr = z + ((int64_t)b * n_heads + head) * vocab;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int row = 64 * G + t * 16 + 4 * kq;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (row + j < vocab) zr[row + j] = acc[n][t][j];
    }
    if (gmax && kq == 0) gmax[((int64_t)b * n_heads + head) * nG + G] = m;
  }
}

// Medusa residual blocks on packed weights: out[head][b][row] =
// h[b][row] + SiLU(sum_k W1[head][row][k] h[b][k] + b1[head][row]), in bf16.
// A block's four waves share one 64-row group and split its k steps in four
// contiguous ranges (hidden x hidden weights have 64x fewer row groups per
// head than a vocabulary projection, so one wave per row group would leave
// most compute units idle); the partial sums meet in LDS.
constexpr int kResSplit = 4;

template <int NB>
__global__ __launch_bounds__(kResSplit * 64) void resblock_packed(
    const uint16_t *__restrict__ h, const uint4 *__restrict__ Wp, const uint16_t *__restrict__ bias,
    uint16_t *__restrict__ hout, int B, int hidden, int nG, int nS) {
  __shared__ f32x4 red[kResSplit - 1][NB][4][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int G = blockIdx.x, head = blockIdx.y, b0 = blockIdx.z * 16 * NB;
  const int kq = lane >> 4;
  const uint4 *wp = Wp + (int64_t)(head * nG + G) * nS * 4 * 64 + lane;
  bool bvalid[NB];
  const uint16_t *hp[NB];
#pragma unroll
  for (int n = 0; n < NB; ++n) {
    const int b = b0 + 16 * n + (lane & 15);
    bvalid[n] = b < B;
    hp[n] = h + (int64_t)(bvalid[n] ? b : 0) * hidden + kq * 8;
  }
  f32x4 acc[NB][4];
#pragma unroll
  for (int n = 0; n < NB; ++n)
#pragma unroll
    for (int t = 0; t < 4; ++t) acc[n][t] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto step = [&](const uint4 (&a)[4], int s) {
    const int k = 32 * s + 8 * kq;
#pragma unroll
    for (int n = 0; n < NB; ++n) {
      const bf16x8 bv = __builtin_bit_cast(bf16x8, ld16_or_zero(bvalid[n] && k < hidden, hp[n] + 32 * s));
#pragma unroll
      for (int t = 0; t < 4; ++t)
        acc[n][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a[t]), bv, acc[n][t], 0, 0, 0);
    }
  };
  const int s_end = (wave + 1) * nS / kResSplit;
  int s = wave * nS / kResSplit;
  for (; s + kPackedUnroll <= s_end; s += kPackedUnroll) {
    uint4 a[kPackedUnroll][4];
#pragma unroll
    for (int u = 0; u < kPackedUnroll; ++u)
#pragma unroll
      for (int t = 0; t < 4; ++t) a[u][t] = ld16_stream(wp + ((s + u) * 4 + t) * 64);
#pragma unroll
    for (int u = 0; u < kPackedUnroll; ++u) step(a[u], s + u);
  }
  for (; s < s_end; ++s) {
    uint4 a[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) a[t] = ld16_stream(wp + (s * 4 + t) * 64);
    step(a, s);
  }
  if (wave > 0) {
#pragma unroll
    for (int n = 0; n < NB; ++n)
#pragma unroll
      for (int t = 0; t < 4; ++t) red[wave - 1][n][t][lane] = acc[n][t];
  }
  __syncthreads();
  if (wave > 0) return;
#pragma unroll
  for (int w = 0; w < kResSplit - 1; ++w)
#pragma unroll
    for (int n = 0; n < NB; ++n)
#pragma unroll
      for (int t = 0; t < 4; ++t) acc[n][t] += red[w][n][t][lane];
  // C layout: lane holds column (batch) lane&15, rows 4*(lane>>4) + 0..3 of each tile.
#pragma unroll
  for (int n = 0; n < NB; ++n) {
    const int b = b0 + 16 * n + (lane & 15);
    if (b >= B) continue;
    const uint16_t *hin = h + (int64_t)b * hidden;
    const uint16_t *bh = bias + (int64_t)head * hidden;
    uint16_t *o = hout + ((int64_t)head * B + b) * hidden;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int row = 64 * G + t * 16 + 4 * kq;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (row + j < hidden) {
          const float y = acc[n][t][j] + bf16_to_f32(bh[row + j]);
          o[row + j] = f32_to_bf16(bf16_to_f32(hin[row + j]) + y / (1.f + expf(-y)));
        }
    }
  }
}

// One thread per 16-byte chunk of the packed buffer (see specmemo_pack_heads).
__global__ __launch_bounds__(256) void pack_heads_bf16(const uint16_t *__restrict__ src, uint4 *__restrict__ dst,
                                                       int vocab, int hidden, int nG, int nS, int64_t chunks) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= chunks) return;
  const int l = (int)(idx & 63);
  int64_t rest = idx >> 6;
  const int t = (int)(rest & 3);
  rest >>= 2;
  const int s = (int)(rest % nS);
  rest /= nS;
  const int G = (int)(rest % nG);
  const int head = (int)(rest / nG);
  const int row = 64 * G + 16 * t + (l & 15);
  const int col = 32 * s + 8 * (l >> 4);
  uint4 v = {0u, 0u, 0u, 0u};
  if (row < vocab && col < hidden)    // hidden % 8 == 0: the 8 columns are all inside or all outside
    v = *reinterpret_cast<const uint4 *>(src + ((int64_t)head * vocab + row) * hidden + col);
  dst[idx] = v;
}

// fp32 heads: one wave per vocabulary row, lanes stride the hidden dimension.
constexpr int kF32BatchTile = 8;

// EPI as for the packed kernel (fp32 residual-block outputs).
template <int EPI>
__global__ __launch_bounds__(256) void head_logits_f32(const float *__restrict__ h, int64_t h_head_stride,
                                                       const float *__restrict__ W,
                                                       float *__restrict__ z, const float *__restrict__ bias,
                                                       float *__restrict__ hout, int B, int hidden,
                                                       int vocab, int n_heads) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int head = blockIdx.y;
  const int row = blockIdx.x * 4 + wave;
  if (row >= vocab) return;
  const float *wr = W + ((int64_t)head * vocab + row) * hidden;
  h += head * h_head_stride;
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
      if (lane == 0 && b0 + j < B) {
        if constexpr (EPI == 0) {
          z[((int64_t)(b0 + j) * n_heads + head) * vocab + row] = v;
        } else {
          const float y = v + bias[(int64_t)head * vocab + row];
          hout[((int64_t)head * B + b0 + j) * vocab + row] = h[(int64_t)(b0 + j) * hidden + row] + y / (1.f + expf(-y));
        }
      }
    }
  }
}

// Top-k of one (sequence, head) logit row per block, in the order larger value
// first, equal values by lower id.
//  1. Every thread takes the max of its values.
//  2. T = the k-th largest maximum of 64 groups of 16 threads: k groups hold a
//     value >= T, so the row's k-th best value is >= T and every top-k value
//     is >= T.
//  3. Values >= T are gathered into LDS; a gathered value's output slot is the
//     number of gathered values that beat it (values below T beat none).
//  4. If ties at T overflow the buffer, the k picks are instead made in k
//     rounds, each taking the best value worse than the previous pick.
// The block of head i also writes the tree tokens of level i+1 (head 0: the
// root token).
constexpr int kTopkThreads = 1024;
constexpr int kTopkCand = 2048;
constexpr int kTopkU = 8;            // float4 groups per thread per batch
constexpr int kTopkGroups = kTopkThreads / 16;   // 16-thread groups for the threshold

__global__ __launch_bounds__(kTopkThreads) void topk_rows(TopkArgs a) {
  constexpr int kWavesT = kTopkThreads / 64;
  const int row = blockIdx.x;                 // b * n_heads + head
  const int b = row / a.n_heads, head = row % a.n_heads;
  const int k = a.k[head];
  const int vocab = a.vocab;
  const float *x = a.z + (int64_t)row * vocab;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  __shared__ __attribute__((aligned(16))) float cv[kTopkCand + 4];
  __shared__ __attribute__((aligned(16))) int ci[kTopkCand + 4];
  __shared__ float gmax[kTopkGroups];
  __shared__ float thr;
  __shared__ float rbv[kWavesT];
  __shared__ int rbi[kWavesT];
  __shared__ float selv[kMaxTopk];
  __shared__ int sel[kMaxTopk];
  __shared__ int ncand;
  if (tid == 0) ncand = 0;

  // This sequence's tree fields for the level this head fills (fetched now so
  // their latency overlaps the row scan).
  const int n0 = a.node_off[b], n1 = a.node_off[b + 1];
  int my_depth = 0, my_rank = 0;
  if (n0 + tid < n1) {
    my_depth = a.depth[n0 + tid];
    my_rank = a.rank[n0 + tid];
  }

  // The row is read in batches of kTopkU groups per thread, all loads of a
  // batch in flight together; a group is a float4 (ids 4 g .. 4 g + 3) when
  // rows start 16-byte aligned (vocab % 4 == 0), else one float.  A row of one
  // batch (vocab <= 4 * 1024 * kTopkU) stays in registers for the gather.
  const bool vec = (vocab & 3) == 0;
  const int ngrp = vec ? vocab >> 2 : vocab;
  const float4 *x4 = reinterpret_cast<const float4 *>(x);
  constexpr float NEG = -INFINITY;
  float4 q[kTopkU];
  auto load_batch = [&](int g0) {
#pragma unroll
    for (int u = 0; u < kTopkU; ++u) {
      const int g = g0 + u * kTopkThreads + tid;
      q[u] = g < ngrp ? (vec ? x4[g] : float4{x[g], NEG, NEG, NEG}) : float4{NEG, NEG, NEG, NEG};
    }
  };
  constexpr int kBatch = kTopkU * kTopkThreads;

  // With the projection's 64-row group maxima (a.gmax), the threshold comes
  // from those maxima and only the groups whose maximum reaches it are read.
  const bool pruned = a.gmax != nullptr && a.nG <= kTopkThreads * kTopkU;
  const float *gm_row = pruned ? a.gmax + (int64_t)row * a.nG : nullptr;

  // 1. thread max (of its values, or of its groups' maxima)
  float mx = NEG;
  if (pruned) {
#pragma unroll
    for (int u = 0; u < kTopkU; ++u) {
      const int g = u * kTopkThreads + tid;
      mx = fmaxf(mx, g < a.nG ? gm_row[g] : NEG);
    }
  } else {
    for (int g0 = 0; g0 < ngrp; g0 += kBatch) {
      load_batch(g0);
#pragma unroll
      for (int u = 0; u < kTopkU; ++u) mx = fmaxf(mx, fmaxf(fmaxf(q[u].x, q[u].y), fmaxf(q[u].z, q[u].w)));
    }
  }
  // 2. T = the k-th largest of the 64 maxima of 16-thread groups (one DPP row
  //    each, 512 values per group at 32 values per thread): k groups hold a
  //    value >= T, so the row's k-th best value is >= T.
  {
    float gm = fmaxf(mx, dpp_f<0xB1>(mx));
    gm = fmaxf(gm, dpp_f<0x4E>(gm));
    gm = fmaxf(gm, dpp_f<0x141>(gm));
    gm = fmaxf(gm, dpp_f<0x140>(gm));
    if ((lane & 15) == 0) gmax[tid >> 4] = gm;
  }
  __syncthreads();
  if (tid < kTopkGroups) {
    const float g = gmax[tid];
    int above = 0;                    // groups whose max beats this one (ties by group index)
#pragma unroll 8
    for (int j = 0; j < kTopkGroups; ++j) {
      const float o = gmax[j];
      above += (o > g || (o == g && j < tid)) ? 1 : 0;
    }
    if (above == k - 1) thr = g;
  }
  __syncthreads();
  const float T = thr;

  // 3. gather values >= T
  auto gather = [&](float xv, int v) {
    if (xv >= T) {
      const int slot = atomicAdd(&ncand, 1);
      if (slot < kTopkCand) {
        cv[slot] = xv;
        ci[slot] = v;
      }
    }
  };
  if (pruned) {
    // the groups whose maximum reaches T, then their values >= T (one thread
    // per value of 16 groups at a time)
    __shared__ int sel_g[kTopkCand];
    __shared__ int nsel;
    if (tid == 0) nsel = 0;
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kTopkU; ++u) {
      const int g = u * kTopkThreads + tid;
      if (g < a.nG && gm_row[g] >= T) {
        const int slot = atomicAdd(&nsel, 1);
        if (slot < kTopkCand) sel_g[slot] = g;
      }
    }
    __syncthreads();
    const int ns = min(nsel, kTopkCand);
    if (nsel > kTopkCand) {
      if (tid == 0) ncand = kTopkCand + 1;      // too many: the k-round selection below
    } else {
      for (int e0 = 0; e0 < ns * 64; e0 += kTopkThreads) {
        const int e = e0 + tid;
        if (e < ns * 64) {
          const int v = 64 * sel_g[e >> 6] + (e & 63);
          if (v < vocab) gather(x[v], v);
        }
      }
    }
  } else
  for (int g0 = 0; g0 < ngrp; g0 += kBatch) {
    if (ngrp > kBatch) load_batch(g0);   // one batch: still in registers
#pragma unroll
    for (int u = 0; u < kTopkU; ++u) {
      const int g = g0 + u * kTopkThreads + tid;
      if (fmaxf(fmaxf(q[u].x, q[u].y), fmaxf(q[u].z, q[u].w)) >= T) {
        if (vec) {
          gather(q[u].x, 4 * g);
          gather(q[u].y, 4 * g + 1);
          gather(q[u].z, 4 * g + 2);
          gather(q[u].w, 4 * g + 3);
        } else {
          gather(q[u].x, g);
        }
      }
    }
  }
  __syncthreads();
  const int n = ncand;
  if (n <= kTopkCand) {
    // rank of candidate c = number of candidates that beat it, counted by one
    // wave (candidates c = wave, wave + 16, ...) with a ballot per 64
    for (int c = wave; c < n; c += kWavesT) {
      const float v = cv[c];
      const int id = ci[c];
      int rank = 0;
      for (int j0 = 0; j0 < n; j0 += 64) {
        const int j = j0 + lane;
        const int jr = j < n ? j : 0;
        const bool beats = j < n && better(cv[jr], ci[jr], v, id);
        rank += __builtin_popcountll(__builtin_amdgcn_ballot_w64(beats));
      }
      if (lane == 0 && rank < k) {
        sel[rank] = id;
        selv[rank] = v;
      }
    }
  } else {
    // 4. k rounds over the row: the best value worse than the previous pick
    float pv = INFINITY;
    int pi = -1;
    for (int j = 0; j < k; ++j) {
      float bv = -INFINITY;
      int bi = INT32_MAX;
      for (int v = tid; v < vocab; v += kTopkThreads) {
        const float xv = x[v];
        if (better(pv, pi, xv, v) && better(xv, v, bv, bi)) {
          bv = xv;
          bi = v;
        }
      }
      wave_argbest(bv, bi);
      if (lane == 0) {
        rbv[wave] = bv;
        rbi[wave] = bi;
      }
      __syncthreads();
      bv = rbv[0];
      bi = rbi[0];
#pragma unroll
      for (int w = 1; w < kWavesT; ++w)
        if (better(rbv[w], rbi[w], bv, bi)) {
          bv = rbv[w];
          bi = rbi[w];
        }
      if (tid == 0) {
        sel[j] = bi;
        selv[j] = bv;
      }
      pv = bv;
      pi = bi;
      __syncthreads();
    }
  }
  __syncthreads();
  int32_t *ids = a.ids + (int64_t)row * a.kmax;
  for (int j = tid; j < a.kmax; j += kTopkThreads) {
    ids[j] = j < k ? sel[j] : -1;
    if (a.vals) a.vals[(int64_t)row * a.kmax + j] = j < k ? selv[j] : -INFINITY;
  }
  if (n0 + tid < n1) {                        // trees have at most kMaxNodes <= 1024 nodes
    if (tid == 0) {
      if (head == 0) a.node_tok[n0] = a.root_tok[b];
    } else if (my_depth == head + 1) {
      a.node_tok[n0 + tid] = sel[my_rank];
    }
  }
}

}  // namespace

hipError_t launch_head_logits(int dt, const void *h, int64_t h_head_stride, const void *w, bool packed, float *z,
                              int B, int hidden, int vocab, int n_heads, hipStream_t st, float *gmax) {
  if (dt == 1 && packed) {
    const int nb = B <= 16 ? 1 : 2;
    const int nG = packed_row_groups(vocab), nS = packed_k_steps(hidden);
    dim3 grid((nG + kWaves - 1) / kWaves, n_heads, (B + 16 * nb - 1) / (16 * nb));
    auto kern = nb == 1 ? head_logits_packed<1> : head_logits_packed<2>;
    hipLaunchKernelGGL(kern, grid, dim3(kWaves * 64), 0, st, static_cast<const uint16_t *>(h), h_head_stride,
                       static_cast<const uint4 *>(w), z, B, hidden, vocab, n_heads, nG, nS, gmax);
  } else if (dt == 1) {
    const int nb = B <= 16 ? 1 : 2;
    dim3 grid((vocab + kWaves * kRowsPerWave - 1) / (kWaves * kRowsPerWave), n_heads,
              (B + 16 * nb - 1) / (16 * nb));
    auto kern = nb == 1 ? head_logits_bf16<1> : head_logits_bf16<2>;
    hipLaunchKernelGGL(kern, grid, dim3(kWaves * 64), 0, st, static_cast<const uint16_t *>(h), h_head_stride,
                       static_cast<const uint16_t *>(w), z, B, hidden, vocab, n_heads);
  } else {
    dim3 grid((vocab + 3) / 4, n_heads);
    hipLaunchKernelGGL(head_logits_f32<0>, grid, dim3(256), 0, st, static_cast<const float *>(h), h_head_stride,
                       static_cast<const float *>(w), z, nullptr, nullptr, B, hidden, vocab, n_heads);
  }
  return hipGetLastError();
}

hipError_t launch_resblock(int dt, const void *h, const void *w1, const void *b1, void *out, int B, int hidden,
                           int n_heads, hipStream_t st) {
  if (dt == 1) {
    const int nb = B <= 16 ? 1 : 2;
    const int nG = packed_row_groups(hidden), nS = packed_k_steps(hidden);
    dim3 grid(nG, n_heads, (B + 16 * nb - 1) / (16 * nb));
    auto kern = nb == 1 ? resblock_packed<1> : resblock_packed<2>;
    hipLaunchKernelGGL(kern, grid, dim3(kResSplit * 64), 0, st, static_cast<const uint16_t *>(h),
                       static_cast<const uint4 *>(w1), static_cast<const uint16_t *>(b1),
                       static_cast<uint16_t *>(out), B, hidden, nG, nS);
  } else {
    dim3 grid((hidden + 3) / 4, n_heads);
    hipLaunchKernelGGL(head_logits_f32<1>, grid, dim3(256), 0, st, static_cast<const float *>(h), (int64_t)0,
                       static_cast<const float *>(w1), nullptr, static_cast<const float *>(b1),
                       static_cast<float *>(out), B, hidden, hidden, n_heads);
  }
  return hipGetLastError();
}

hipError_t launch_pack_heads(const void *src, void *dst, int n_heads, int vocab, int hidden, hipStream_t st) {
  const int nG = packed_row_groups(vocab), nS = packed_k_steps(hidden);
  const int64_t chunks = (int64_t)n_heads * nG * nS * 4 * 64;
  hipLaunchKernelGGL(pack_heads_bf16, dim3((unsigned)((chunks + 255) / 256)), dim3(256), 0, st,
                     static_cast<const uint16_t *>(src), static_cast<uint4 *>(dst), vocab, hidden, nG, nS, chunks);
  return hipGetLastError();
}

hipError_t launch_topk(const TopkArgs &a, int B, hipStream_t st) {
  hipLaunchKernelGGL(topk_rows, dim3(B * a.n_heads), dim3(kTopkThreads), 0, st, a);
  return hipGetLastError();
}

}  // namespace specmemo
