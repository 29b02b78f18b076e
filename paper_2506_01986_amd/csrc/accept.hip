// Stage (c): acceptance of the longest verified root-to-leaf path.
//
// SpecMemo App. A.1: each candidate token must pass a threshold, verification
// is cumulative along a candidate sequence and the longest verified candidate is
// accepted; Medusa verifies with typical sampling.  Sec. 3.2: verification of a
// continuation is cumulative.
//
// Greedy mode takes the arg-best token of every node's row in one parallel
// pass (one block per row) and then walks each tree from the root; the walk
// has no dependent row loads, only one token per node crosses to it.  Typical
// mode needs every node's softmax statistics: one block per row computes
// them, then one block per sequence evaluates the edges and picks the path.
#include "compact_rows.h"
#include "device.h"
#include "internal.h"

namespace specmemo {

namespace {

constexpr int kNT = 512;
constexpr int kWaves = kNT / 64;

template <int DT>
__device__ __forceinline__ float ld(const void *p, int64_t i) {
  if (DT == 0) return static_cast<const float *>(p)[i];
  return bf16_to_f32(static_cast<const uint16_t *>(p)[i]);
}

typedef short s16x2_t __attribute__((ext_vector_type(2)));
typedef unsigned short u16x2_t __attribute__((ext_vector_type(2)));

// Order-preserving keys of the two bf16 values of a word, one per 16-bit half:
// a non-negative value gets its sign bit set, a negative one has all 16 bits
// inverted, so a larger value has a larger unsigned key.  The keys of -0 and
// +0 differ (0x7FFF, 0x8000); the scan below treats them as equal.
__device__ __forceinline__ uint32_t bf16x2_keys(uint32_t w) {
  const s16x2_t sign = __builtin_bit_cast(s16x2_t, w) >> (short)15;   // 0 or -1 per half
  return w ^ (__builtin_bit_cast(uint32_t, sign) | 0x80008000u);
}

constexpr int kArgU = 8;                          // 16-byte loads per thread
constexpr int kArgMaxVocab = kNT * kArgU * 8;     // rows the register pass covers

// Arg-best of a bf16 row with vocab % 8 == 0 and vocab <= kArgMaxVocab, in two
// steps over the same registers: the row's largest key (one packed 16-bit
// maximum per two values), then the lowest id holding it, searched only by the
// threads whose own maximum is that key.  NaN rows are not valid input.
__device__ void row_argbest_bf16(const uint16_t *row, int vocab, uint32_t *sk, float &out_v, int &out_i) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint4 *p = reinterpret_cast<const uint4 *>(row);
  const int nch = vocab / 8;
  uint4 w[kArgU];
#pragma unroll
  for (int u = 0; u < kArgU; ++u) {
    const int c = u * kNT + tid;
    w[u] = c < nch ? p[c] : uint4{0u, 0u, 0u, 0u};
  }
  u16x2_t mx = {0, 0};
#pragma unroll
  for (int u = 0; u < kArgU; ++u) {
    const bool live = u * kNT + tid < nch;   // padding keys stay 0, below every value
    w[u].x = live ? bf16x2_keys(w[u].x) : 0u;
    w[u].y = live ? bf16x2_keys(w[u].y) : 0u;
    w[u].z = live ? bf16x2_keys(w[u].z) : 0u;
    w[u].w = live ? bf16x2_keys(w[u].w) : 0u;
    mx = __builtin_elementwise_max(mx, __builtin_bit_cast(u16x2_t, w[u].x));
    mx = __builtin_elementwise_max(mx, __builtin_bit_cast(u16x2_t, w[u].y));
    mx = __builtin_elementwise_max(mx, __builtin_bit_cast(u16x2_t, w[u].z));
    mx = __builtin_elementwise_max(mx, __builtin_bit_cast(u16x2_t, w[u].w));
  }
  const uint32_t tk = mx.x > mx.y ? mx.x : mx.y;
  uint32_t k = wave_reduce_u32<true>(tk);
  if (lane == 0) sk[wave] = k;
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kWaves; ++i) k = sk[i] > k ? sk[i] : k;
  const uint32_t alt = k == 0x8000u ? 0x7FFFu : k;   // +0 is the maximum: -0 ties with it
  uint32_t cand = 0xFFFFFFFFu;
  if (tk == k || tk == alt) {
#pragma unroll
    for (int u = 0; u < kArgU; ++u) {
      const uint32_t ws[4] = {w[u].x, w[u].y, w[u].z, w[u].w};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint32_t key = (ws[e >> 1] >> (16 * (e & 1))) & 0xFFFFu;
        const uint32_t id = 8u * (uint32_t)(u * kNT + tid) + (uint32_t)e;
        if (cand == 0xFFFFFFFFu && (key == k || key == alt) && u * kNT + tid < nch) cand = id;
      }
    }
  }
  cand = wave_reduce_u32<false>(cand);
  __syncthreads();   // every wave has read sk
  if (lane == 0) sk[wave] = cand;
  __syncthreads();
  uint32_t best = sk[0];
#pragma unroll
  for (int i = 1; i < kWaves; ++i) best = sk[i] < best ? sk[i] : best;
  __syncthreads();
  const uint32_t bits = (k & 0x8000u) ? (k ^ 0x8000u) : (k ^ 0xFFFFu);
  out_v = __uint_as_float(bits << 16);
  out_i = (int)best;
}

// Arg-best (largest value, lowest id) of one logit row; result in every thread.
template <int DT>
__device__ void row_argbest(const void *logits, int64_t row, int vocab, float *sv, int *si,
                            float &out_v, int &out_i) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  float bv = -INFINITY;
  int bi = INT32_MAX;
  const int64_t base = row * vocab;
  if (DT == 1 && (vocab & 7) == 0 && vocab <= kArgMaxVocab) {
    row_argbest_bf16(static_cast<const uint16_t *>(logits) + base, vocab, reinterpret_cast<uint32_t *>(si), out_v,
                     out_i);
    return;
  }
  if (DT == 1 && (vocab & 7) == 0) {
    // All of this thread's 16-byte loads of a pass are issued before any compare.
    constexpr int U = 8;
    const uint4 *p = reinterpret_cast<const uint4 *>(static_cast<const uint16_t *>(logits) + base);
    const int nch = vocab / 8;
    for (int c0 = 0; c0 < nch; c0 += kNT * U) {
      uint4 w[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int c = c0 + u * kNT + tid;
        w[u] = c < nch ? p[c] : uint4{0xFF80FF80u, 0xFF80FF80u, 0xFF80FF80u, 0xFF80FF80u};  // -inf
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int c = c0 + u * kNT + tid;
        const uint32_t ws[4] = {w[u].x, w[u].y, w[u].z, w[u].w};
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float x = bf16_to_f32(static_cast<uint16_t>(ws[e >> 1] >> ((e & 1) * 16)));
          const int v = 8 * c + e;
          if (c < nch && better(x, v, bv, bi)) {
            bv = x;
            bi = v;
          }
        }
      }
    }
  } else if (DT == 0 && (vocab & 3) == 0) {
    const float4 *p = reinterpret_cast<const float4 *>(static_cast<const float *>(logits) + base);
    for (int c = tid; c < vocab / 4; c += kNT) {
      float4 w = p[c];
      float ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (better(ws[e], 4 * c + e, bv, bi)) {
          bv = ws[e];
          bi = 4 * c + e;
        }
    }
  } else {
    for (int v = tid; v < vocab; v += kNT) {
      float x = ld<DT>(logits, base + v);
      if (better(x, v, bv, bi)) {
        bv = x;
        bi = v;
      }
    }
  }
  wave_argbest(bv, bi);
  if (lane == 0) {
    sv[wave] = bv;
    si[wave] = bi;
  }
  __syncthreads();
  bv = sv[0];
  bi = si[0];
#pragma unroll
  for (int w = 1; w < kWaves; ++w)
    if (better(sv[w], si[w], bv, bi)) {
      bv = sv[w];
      bi = si[w];
    }
  __syncthreads();
  out_v = bv;
  out_i = bi;
}

// Greedy mode, pass 1: the arg-best token of every node's logit row, all rows
// at once (the walk of pass 2 then has no dependent row loads).
template <int DT>
__global__ __launch_bounds__(kNT) void row_argbest_all(AcceptArgs a) {
  __shared__ float sv[kWaves];
  __shared__ int si[kWaves];
  float v;
  int tok;
  row_argbest<DT>(a.logits, blockIdx.x, a.vocab, sv, si, v, tok);
  if (threadIdx.x == 0) a.best[blockIdx.x] = tok;
}

// Greedy mode, pass 2: one wave walks sequence b's tree from the root to the
// child carrying the current node's arg-best token (unique: sibling tokens
// differ), with the tree's parents, tokens and arg-best tokens in LDS (at
// most kMaxNodes = 128 nodes, two per lane).  Returns the accepted length;
// lane j holds path entry j in p_mine (lanes past the end hold -1), and
// next_tok is the last accepted node's arg-best token.
__device__ __forceinline__ int greedy_walk(const AcceptArgs &a, int b, int &p_mine, int &next_tok) {
  __shared__ int s_par[kMaxNodes], s_tok[kMaxNodes], s_best[kMaxNodes];
  const int lane = threadIdx.x;
  const int n0 = a.node_off[b], N = a.node_off[b + 1] - n0;
  for (int n = lane; n < N; n += 64) {
    s_par[n] = n == 0 ? -1 : a.parent[n0 + n];
    s_tok[n] = a.node_tok[n0 + n];
    s_best[n] = a.best[n0 + n];
  }
  __syncthreads();
  int cur = 0, len = 0;
  p_mine = lane == 0 ? 0 : -1;   // lane j keeps path entry j
  for (;;) {
    const int tok = s_best[cur];
    const bool m0 = lane < N && s_par[lane] == cur && s_tok[lane] == tok;
    const bool m1 = lane + 64 < N && s_par[lane + 64] == cur && s_tok[lane + 64] == tok;
    const uint64_t b0 = __builtin_amdgcn_ballot_w64(m0), b1 = __builtin_amdgcn_ballot_w64(m1);
    const int nxt = b0 ? (int)__builtin_ctzll(b0) : b1 ? 64 + (int)__builtin_ctzll(b1) : -1;
    if (nxt < 0 || len + 1 >= kMaxPath) break;
    cur = nxt;
    ++len;
    if (lane == len) p_mine = cur;
  }
  next_tok = s_best[cur];
  return len;
}

__device__ __forceinline__ void write_acceptance(const AcceptArgs &a, int b, int len, int p_mine, int next_tok) {
  const int lane = threadIdx.x;
  if (lane == 0) {
    a.accept_len[b] = len;
    a.next_tok[b] = next_tok;
  }
  for (int j = lane; j < a.path_stride; j += 64) a.path[(int64_t)b * a.path_stride + j] = j < 64 ? p_mine : -1;
}

// One wave per sequence.
__global__ __launch_bounds__(64) void accept_walk(AcceptArgs a) {
  const int b = blockIdx.x;
  int p_mine, next_tok;
  const int len = greedy_walk(a, b, p_mine, next_tok);
  write_acceptance(a, b, len, p_mine, next_tok);
}

// Acceptance and compaction in one pass: one wave per (sequence, KV head,
// K|V) of a launch group walks the sequence's tree and moves that slab's
// accepted rows; the wave of (KV head 0, K) also writes the acceptance
// outputs and the new length.  The walk is repeated per wave (a few LDS
// rounds over at most 128 nodes) so that no wave waits for another.
__global__ __launch_bounds__(64) void accept_walk_compact(AcceptArgs a, CompactArgs c) {
  const int s = blockIdx.x, kvh = blockIdx.y, which = blockIdx.z;
  const int b = c.b0 + s;
  int p_mine, next_tok;
  const int len = greedy_walk(a, b, p_mine, next_tok);
  const bool writer = kvh == 0 && which == 0;
  if (writer) write_acceptance(a, b, len, p_mine, next_tok);
  int src[kMaxPath];
#pragma unroll
  for (int j = 0; j < kMaxPath; ++j) src[j] = __builtin_amdgcn_readlane(p_mine, j);
  const CompactSeq S = c.tab ? c.tab[s] : c.seq[s];
  move_rows(c, S, kvh, which, len, src, threadIdx.x, 64);
  if (writer && threadIdx.x == 0) c.seq_len[b] = S.L + len + 1;
}

// Typical mode, pass 1: per row u, x = z_u / T: lse_u = log sum exp x and
// H_u = -sum pi log pi with pi = softmax(x).  In base 2, with y = x log2(e),
// M = max y, e_v = 2^(y_v - M), s = sum e and t = sum e (y - M):
// lse = (M + log2 s) ln 2 and H = (log2 s - t / s) ln 2.  Exponents below
// -128 are clamped there: their weights (< 2^-128 of the largest) change
// neither sum in fp32.  One block per row; the block's maximum, then the two
// sums, reduced over waves with DPP / permlane steps and LDS.
__device__ __forceinline__ float block_max(float v, float *red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  v = wave_max(v);
  if (lane == 0) red[wave] = v;
  __syncthreads();
  v = red[0];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) v = fmaxf(v, red[w]);
  return v;
}

__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_f<0xB1>(v);
  v += dpp_f<0x4E>(v);
  v += dpp_f<0x141>(v);
  v += dpp_f<0x140>(v);
  const auto r16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(r16[0]) + __uint_as_float(r16[1]);
  return sum_with_other_half(v);
}

// Block sums of s and t, then lse and H; the lowest id holding the row's
// maximum (`cand`: this thread's) is the row's arg-best token, the next token
// if the row's node ends the accepted path.
__device__ __forceinline__ void finish_stats(const AcceptArgs &a, int u, float M, float s, float t, uint32_t cand,
                                             float *red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  s = wave_sum(s);
  t = wave_sum(t);
  cand = wave_reduce_u32<false>(cand);
  __syncthreads();   // every wave has read the maximum
  if (lane == 0) {
    red[wave] = s;
    red[kWaves + wave] = t;
    red[2 * kWaves + wave] = __uint_as_float(cand);
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float S = 0.f, T = 0.f;
    uint32_t best = 0xFFFFFFFFu;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      S += red[w];
      T += red[kWaves + w];
      const uint32_t c = __float_as_uint(red[2 * kWaves + w]);
      best = c < best ? c : best;
    }
    const float ln2 = 0.6931471805599453f, l2s = __log2f(S);
    a.stats[2 * (int64_t)u] = (M + l2s) * ln2;
    a.stats[2 * (int64_t)u + 1] = (l2s - T / S) * ln2;
    a.best[u] = (int)best;
  }
}

// Weight and its exponent of one logit z: d = max(z c - M, -128), 2^d.
__device__ __forceinline__ void stat_term(float z, float c, float M, float &s, float &t) {
  const float d = fmaxf(fmaf(z, c, -M), -128.f);
  const float e = fast_exp2(d);
  s += e;
  t = fmaf(e, d, t);
}

template <int DT>
__global__ __launch_bounds__(kNT) void row_softmax_stats(AcceptArgs a) {
  __shared__ float red[3 * kWaves];
  const int u = blockIdx.x, tid = threadIdx.x;
  const int64_t base = (int64_t)u * a.vocab;
  const float c = a.inv_temp * 1.4426950408889634f;   // y = z c
  float s = 0.f, t = 0.f;
  if (DT == 1 && (a.vocab & 7) == 0 && a.vocab <= kArgMaxVocab) {
    // the row stays in registers: eight 16-byte loads per thread, all in flight
    const uint4 *p = reinterpret_cast<const uint4 *>(static_cast<const uint16_t *>(a.logits) + base);
    const int nch = a.vocab / 8;
    uint4 w[kArgU];
#pragma unroll
    for (int k = 0; k < kArgU; ++k) {
      const int ch = k * kNT + tid;
      w[k] = ch < nch ? p[ch] : uint4{0xFF80FF80u, 0xFF80FF80u, 0xFF80FF80u, 0xFF80FF80u};   // -inf
    }
    float mz = -INFINITY;
#pragma unroll
    for (int k = 0; k < kArgU; ++k) {
      const uint32_t ws[4] = {w[k].x, w[k].y, w[k].z, w[k].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) mz = fmaxf(mz, fmaxf(__uint_as_float(ws[e] << 16), __uint_as_float(ws[e] & 0xFFFF0000u)));
    }
    const float zmax = block_max(mz, red), M = zmax * c;
    uint32_t cand = 0xFFFFFFFFu;
#pragma unroll
    for (int k = 0; k < kArgU; ++k) {
      if (k * kNT + tid < nch) {
        const uint32_t ws[4] = {w[k].x, w[k].y, w[k].z, w[k].w};
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float z = __uint_as_float(e & 1 ? ws[e >> 1] & 0xFFFF0000u : ws[e >> 1] << 16);
          stat_term(z, c, M, s, t);
          const uint32_t id = 8u * (uint32_t)(k * kNT + tid) + (uint32_t)e;
          cand = z == zmax && id < cand ? id : cand;   // -0 == +0: the lower id wins
        }
      }
    }
    finish_stats(a, u, M, s, t, cand, red);
    return;
  }
  // any dtype and vocabulary: two passes over the row
  float mz = -INFINITY;
  for (int v = tid; v < a.vocab; v += kNT) mz = fmaxf(mz, ld<DT>(a.logits, base + v));
  const float zmax = block_max(mz, red), M = zmax * c;
  uint32_t cand = 0xFFFFFFFFu;
  for (int v = tid; v < a.vocab; v += kNT) {
    const float z = ld<DT>(a.logits, base + v);
    stat_term(z, c, M, s, t);
    cand = z == zmax && (uint32_t)v < cand ? (uint32_t)v : cand;
  }
  finish_stats(a, u, M, s, t, cand, red);
}

// Typical mode, pass 2, by one block: the edges of sequence b's tree (one
// thread per node: the edge from its parent), the cumulative acceptance and
// path score level by level (score[c] = score[parent] + log pi, as the path
// is walked from the root), and the pick: the deepest accepted node, then the
// larger score, then the lower id, as one 64-bit key maximum over the nodes.
// Writes accept_len, path and next_tok (the picked row's arg-best token from
// pass 1) and returns the accepted length, with the path in s_path for the
// whole block.
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const uint64_t o = __shfl_xor(v, off);
    v = o > v ? o : v;
  }
  return v;
}

template <int DT, int NT>
__device__ __forceinline__ int typical_pick(const AcceptArgs &a, int b, int *s_path, bool write_out) {
  constexpr int NW = NT / 64;
  __shared__ float lp[kMaxNodes], score[kMaxNodes];
  __shared__ int pass[kMaxNodes], ok[kMaxNodes], par[kMaxNodes], dep[kMaxNodes];
  __shared__ uint64_t s_key[NW];
  static_assert(NT >= kMaxNodes, "one thread per tree node");
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n0 = a.node_off[b], N = a.node_off[b + 1] - n0;
  int my_dep = 0;
  if (tid < N) {
    const int u = a.parent[n0 + tid];
    par[tid] = u;
    dep[tid] = my_dep = a.depth[n0 + tid];
    if (tid == 0) {
      ok[0] = 1;
      score[0] = 0.f;
    } else {
      const float lse = a.stats[2 * (int64_t)(n0 + u)], H = a.stats[2 * (int64_t)(n0 + u) + 1];
      const int tok = a.node_tok[n0 + tid];
      const bool valid = tok >= 0 && tok < a.vocab;   // an out-of-range token never passes
      const float x = valid ? ld<DT>(a.logits, (int64_t)(n0 + u) * a.vocab + tok) * a.inv_temp - lse : -INFINITY;
      const float thr = fminf(a.log_eps, a.log_delta - H);
      lp[tid] = x;
      pass[tid] = valid && x > thr;
    }
  }
  // level d: every node at depth d extends its parent's result (parents sit at d - 1)
  for (int d = 1; __syncthreads_or(tid < N && my_dep >= d); ++d)
    if (tid < N && my_dep == d) {
      const int u = par[tid];
      ok[tid] = ok[u] && pass[tid];
      score[tid] = score[u] + lp[tid];
    }
  // key: depth, then the score's order-preserving bits, then 127 - id (lower ids win)
  uint64_t key = 0;
  if (tid < N && ok[tid]) {
    const uint32_t sb = __float_as_uint(score[tid]);
    const uint32_t sk = (sb & 0x80000000u) ? ~sb : sb | 0x80000000u;
    key = (uint64_t)(my_dep + 1) << 40 | (uint64_t)sk << 8 | (uint64_t)(kMaxNodes - 1 - tid);
  }
  key = wave_max_u64(key);
  if (lane == 0) s_key[wave] = key;
  __syncthreads();
  key = s_key[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) key = s_key[w] > key ? s_key[w] : key;
  const int best = kMaxNodes - 1 - (int)(key & 0xFF);
  const int len = dep[best];
  if (tid == 0) {
    int32_t *p = a.path + (int64_t)b * a.path_stride;
    if (write_out) {
      a.accept_len[b] = len;
      a.next_tok[b] = a.best[n0 + best];
      for (int j = 0; j < a.path_stride; ++j) p[j] = -1;
    }
    for (int u = best, j = len; u >= 0 && j >= 0; u = par[u], --j) {
      if (write_out) p[j] = u;
      s_path[j] = u;
    }
  }
  __syncthreads();
  return len;
}

// One block per sequence.
template <int DT>
__global__ __launch_bounds__(kNT) void accept_typical(AcceptArgs a) {
  __shared__ int s_path[kMaxPath];
  typical_pick<DT, kNT>(a, blockIdx.x, s_path, true);
}

// Acceptance and compaction in one pass: one block per (sequence, KV head,
// K|V) picks the sequence's path (a few LDS rounds over at most kMaxNodes
// nodes, repeated per block so that no block waits for another) and moves
// the accepted rows of its slab; the block of (KV head 0, K) writes the
// acceptance outputs and the new length.
constexpr int kPickNT = kMaxNodes;   // one thread per tree node

template <int DT>
__global__ __launch_bounds__(kPickNT) void accept_typical_compact(AcceptArgs a, CompactArgs c) {
  __shared__ int s_path[kMaxPath];
  const int s = blockIdx.x, kvh = blockIdx.y, which = blockIdx.z, b = c.b0 + s;
  const bool writer = kvh == 0 && which == 0;
  const int len = typical_pick<DT, kPickNT>(a, b, s_path, writer);
  int src[kMaxPath];
#pragma unroll
  for (int j = 0; j < kMaxPath; ++j) src[j] = j <= len ? s_path[j] : -1;
  const CompactSeq S = c.tab ? c.tab[s] : c.seq[s];
  move_rows(c, S, kvh, which, len, src, threadIdx.x, kPickNT);
  if (writer && threadIdx.x == 0) c.seq_len[b] = S.L + len + 1;
}

// ---- sampled next token ---------------------------------------------------------
// Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC 2011): ten rounds on a 4 x 64-bit
// counter, each two 64 x 64 -> 128-bit products, the key bumped by the Weyl
// constants between rounds.
__device__ __forceinline__ void philox4x64_10(uint64_t (&x)[4], uint64_t k0, uint64_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k0 += 0x9E3779B97F4A7C15ull;
      k1 += 0xBB67AE8584CAA73Bull;
    }
    const uint64_t m0 = 0xD2E7470EE14C6C93ull, m1 = 0xCA5A826395121157ull;
    const uint64_t hi0 = __umul64hi(m0, x[0]), lo0 = m0 * x[0];
    const uint64_t hi1 = __umul64hi(m1, x[2]), lo1 = m1 * x[2];
    x[0] = hi1 ^ x[1] ^ k0;
    x[1] = lo1;
    x[2] = hi0 ^ x[3] ^ k1;
    x[3] = lo0;
  }
}

// Gumbel-max draw from softmax(z / T) of sequence b's last accepted row: the
// argmax over v of fmaf(z_v, 1/T, G_v), G_v = -log(-log(u_v)), u_v from
// Philox with key (seed, offset), counter (v / 4, b, 0, 0), word v % 4, as
// ((x >> 41) + 1/2) / 2^23 (strictly inside (0, 1), so G_v is finite); ties by
// lower token id.  The keys cost two logarithms per token and a Philox block
// per four tokens, so the row is spread over many blocks: block (s, b) draws
// the 1024 tokens of segment s of sequence b (one Philox block per thread),
// leaves its best (key, id) in the workspace as one order-preserving 64-bit
// word, and one wave per sequence then takes the largest word.  Without a
// workspace one 1024-thread block per sequence does the whole row.
constexpr int kSampleThreads = 1024;
constexpr int kSegThreads = 256;
constexpr int kSegTokens = 4 * kSegThreads;

// Row of sequence b's last accepted node, or -1 when its accept_len / path
// entry is out of range (next_tok is then left untouched).
__device__ __forceinline__ int64_t sample_row(const SampleArgs &a, int b) {
  const int n0 = a.node_off[b], N = a.node_off[b + 1] - n0;
  const int acc = a.accept_len[b];
  if (acc < 0 || acc >= a.path_stride) return -1;
  const int node = a.path[(int64_t)b * a.path_stride + acc];
  if (node < 0 || node >= N) return -1;
  return (int64_t)(n0 + node) * a.vocab;
}

// The four keys of Philox block q of sequence b, folded into (best, arg).
template <int DT>
__device__ __forceinline__ void sample_block(const SampleArgs &a, int b, int64_t row, int q, float &best, int &arg) {
  uint64_t x[4] = {(uint64_t)q, (uint64_t)b, 0ull, 0ull};
  philox4x64_10(x, a.seed, a.offset);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int v = 4 * q + j;
    if (v < a.vocab) {
      // 23 random bits: (k + 1/2) 2^-23 is exact in fp32 and lies in [2^-24, 1 - 2^-24]
      const float u = ((float)(x[j] >> 41) + 0.5f) * 0x1p-23f;
      const float g = -logf(-logf(u));
      const float s = fmaf(ld<DT>(a.logits, row + v), a.inv_temp, g);
      if (better(s, v, best, arg)) {
        best = s;
        arg = v;
      }
    }
  }
}

// Best (key, id) of a block, in thread 0 (waves, then LDS).
template <int NT>
__device__ __forceinline__ void block_argbest(float &best, int &arg) {
  wave_argbest(best, arg);
  constexpr int kW = NT / 64;
  __shared__ float sv[kW];
  __shared__ int si[kW];
  const int tid = threadIdx.x;
  if ((tid & 63) == 0) {
    sv[tid >> 6] = best;
    si[tid >> 6] = arg;
  }
  __syncthreads();
  if (tid == 0)
    for (int w = 1; w < kW; ++w)
      if (better(sv[w], si[w], best, arg)) {
        best = sv[w];
        arg = si[w];
      }
}

template <int DT>
__global__ __launch_bounds__(kSampleThreads) void sample_next_kernel(SampleArgs a) {
  const int b = blockIdx.x, tid = threadIdx.x;
  const int64_t row = sample_row(a, b);
  if (row < 0) return;
  float best = -INFINITY;
  int arg = a.vocab;
  for (int q = tid; 4 * q < a.vocab; q += kSampleThreads) sample_block<DT>(a, b, row, q, best, arg);
  block_argbest<kSampleThreads>(best, arg);
  if (tid == 0) a.next_tok[b] = arg;
}

// The order of (key, id) as one unsigned word: larger key first (-0 counts as
// +0), then lower id.
__device__ __forceinline__ uint64_t sample_word(float s, int v) {
  const uint32_t u = __float_as_uint(s == 0.f ? 0.f : s);
  const uint32_t k = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return (uint64_t)k << 32 | (uint32_t)(0x7FFFFFFF - v);
}

template <int DT>
__global__ __launch_bounds__(kSegThreads) void sample_next_segments(SampleArgs a, uint64_t *words, int nseg) {
  const int seg = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  const int64_t row = sample_row(a, b);
  if (row < 0) return;
  float best = -INFINITY;
  int arg = a.vocab;
  const int q = seg * kSegThreads + tid;
  if (4 * q < a.vocab) sample_block<DT>(a, b, row, q, best, arg);
  block_argbest<kSegThreads>(best, arg);
  // a segment always holds at least one token, so arg < vocab here
  if (tid == 0) words[(int64_t)b * nseg + seg] = sample_word(best, arg);
}

__global__ __launch_bounds__(64) void sample_next_pick(SampleArgs a, const uint64_t *words, int nseg) {
  const int b = blockIdx.x, lane = threadIdx.x;
  if (sample_row(a, b) < 0) return;
  uint64_t w = 0;
  for (int s = lane; s < nseg; s += 64) {
    const uint64_t x = words[(int64_t)b * nseg + s];
    w = x > w ? x : w;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const uint64_t o = (uint64_t)(uint32_t)__shfl_xor((int)(w >> 32), off) << 32 | (uint32_t)__shfl_xor((int)w, off);
    w = o > w ? o : w;
  }
  if (lane == 0) a.next_tok[b] = 0x7FFFFFFF - (int)(uint32_t)w;
}

}  // namespace

int sample_segments(int vocab) { return (vocab + kSegTokens - 1) / kSegTokens; }

hipError_t launch_sample_next(int dt, const SampleArgs &a, int B, uint64_t *words, hipStream_t st) {
  if (words) {
    const int nseg = sample_segments(a.vocab);
    if (dt == 1)
      hipLaunchKernelGGL(sample_next_segments<1>, dim3(nseg, B), dim3(kSegThreads), 0, st, a, words, nseg);
    else
      hipLaunchKernelGGL(sample_next_segments<0>, dim3(nseg, B), dim3(kSegThreads), 0, st, a, words, nseg);
    hipLaunchKernelGGL(sample_next_pick, dim3(B), dim3(64), 0, st, a, (const uint64_t *)words, nseg);
  } else if (dt == 1) {
    hipLaunchKernelGGL(sample_next_kernel<1>, dim3(B), dim3(kSampleThreads), 0, st, a);
  } else {
    hipLaunchKernelGGL(sample_next_kernel<0>, dim3(B), dim3(kSampleThreads), 0, st, a);
  }
  return hipGetLastError();
}

hipError_t launch_accept_rows(int dt, const AcceptArgs &a, int total_nodes, hipStream_t st) {
  if (a.mode == 0) {
    if (dt == 1)
      hipLaunchKernelGGL(row_argbest_all<1>, dim3(total_nodes), dim3(kNT), 0, st, a);
    else
      hipLaunchKernelGGL(row_argbest_all<0>, dim3(total_nodes), dim3(kNT), 0, st, a);
  } else if (dt == 1) {
    hipLaunchKernelGGL(row_softmax_stats<1>, dim3(total_nodes), dim3(kNT), 0, st, a);
  } else {
    hipLaunchKernelGGL(row_softmax_stats<0>, dim3(total_nodes), dim3(kNT), 0, st, a);
  }
  return hipGetLastError();
}

hipError_t launch_accept(int dt, const AcceptArgs &a, int total_nodes, hipStream_t st) {
  hipError_t e = launch_accept_rows(dt, a, total_nodes, st);
  if (e != hipSuccess) return e;
  if (a.mode == 0)
    hipLaunchKernelGGL(accept_walk, dim3(a.B), dim3(64), 0, st, a);
  else if (dt == 1)
    hipLaunchKernelGGL(accept_typical<1>, dim3(a.B), dim3(kNT), 0, st, a);
  else
    hipLaunchKernelGGL(accept_typical<0>, dim3(a.B), dim3(kNT), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_accept_compact(int dt, const AcceptArgs &a, const CompactArgs &c, hipStream_t st) {
  if (a.mode == 0)
    hipLaunchKernelGGL(accept_walk_compact, dim3(c.nseq, c.n_kv, 2), dim3(64), 0, st, a, c);
  else if (dt == 1)
    hipLaunchKernelGGL(accept_typical_compact<1>, dim3(c.nseq, c.n_kv, 2), dim3(kPickNT), 0, st, a, c);
  else
    hipLaunchKernelGGL(accept_typical_compact<0>, dim3(c.nseq, c.n_kv, 2), dim3(kPickNT), 0, st, a, c);
  return hipGetLastError();
}

}  // namespace specmemo
