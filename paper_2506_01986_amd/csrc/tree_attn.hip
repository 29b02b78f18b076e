// Stage (b): tree-masked attention over a ragged batch of candidate trees.
//
// SpecMemo Sec. 3.1: before verification the tree mask assumes full acceptance
// of every candidate sequence, so a node attends to the committed KV rows and to
// its own root path (ancestors and itself); App. A.1: the base model verifies all
// candidates in one forward pass; Sec. 3.3: the batch is ragged (here without
// padding: every sequence has its own length and tree).
//
// bf16 path (head_dim 128).  A work item is (sequence, KV head, block of query
// rows, KV chunk).  The query rows of a (sequence, KV head) are its tree nodes x
// the GQA group's query heads (node-major), so one K/V tile staged in LDS serves
// every node and every query head of the group.  Each wave owns 32 query rows:
//
//   S^T[key][row] = K . Q^T    (32x32x16 bf16 MFMA, K tile from LDS as A,
//                               the wave's Q fragment in registers as B)
//   O^T[d][row]  += V^T . P^T  (V staged transposed in LDS as A, P from the
//                               S^T accumulator converted to bf16 as B)
//
// With the transposed products every lane holds one query row, so the online
// softmax needs one cross-lane exchange (lanes l and l^32) per tile.  The
// accumulator's key order is matched by reading V^T in the same key order, so
// P never moves between lanes.
//
// A sequence with several KV chunks writes per-chunk partials (unnormalised O,
// running max, running sum) to the workspace, merged in a fixed order by
// tree_attn_combine (deterministic, no atomics).
#include "device.h"
#include "internal.h"

namespace specmemo {

namespace {

constexpr int D = kAttnHeadDim;
constexpr int TK = kAttnKeyTile;
constexpr int KPITCH = D + 8;      // bf16 elements per K row in LDS (272 B)
constexpr int VPITCH = TK + 4;     // bf16 elements per V^T row in LDS (136 B)

struct Item {
  int s, kvh, rb, ch;
};

__device__ __forceinline__ Item decode_item(const AttnArgs &a, int idx) {
  int s = 0;
  while (s + 1 < a.nseq && a.seq[s + 1].item0 <= idx) ++s;
  const AttnSeq &S = a.seq[s];
  int local = idx - S.item0;
  Item it;
  it.s = s;
  it.rb = local % S.nrb;
  local /= S.nrb;
  it.ch = local % S.nch;
  it.kvh = local / S.nch;
  return it;
}

template <int WAVES>
__global__ __launch_bounds__(WAVES * 64, WAVES == 4 ? 2 : 1) void tree_attn_bf16(AttnArgs a) {
  constexpr int NT = WAVES * 64;
  constexpr int RB = 32 * WAVES;
  __shared__ __attribute__((aligned(16))) uint16_t Ks[TK * KPITCH];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[D * VPITCH];
  __shared__ uint32_t anc[kMaxNodes][4];

  const Item it = decode_item(a, blockIdx.x);
  const AttnSeq &S = a.seq[it.s];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = lane >> 5;              // which half of the wave
  const int L = S.L, N = S.N, g = a.group;
  const int rows = N * g;

  // Ancestor-or-self bitmask of every node of this tree (local ids).
  for (int n = tid; n < N; n += NT) {
    uint32_t m0 = 0, m1 = 0, m2 = 0, m3 = 0;
    for (int u = n; u >= 0; u = a.parent[S.node0 + u]) {
      uint32_t bit = 1u << (u & 31);
      int w = u >> 5;
      m0 |= w == 0 ? bit : 0u;
      m1 |= w == 1 ? bit : 0u;
      m2 |= w == 2 ? bit : 0u;
      m3 |= w == 3 ? bit : 0u;
    }
    anc[n][0] = m0;
    anc[n][1] = m1;
    anc[n][2] = m2;
    anc[n][3] = m3;
  }

  // This lane's query row.
  const int my_row = it.rb * RB + wave * 32 + (lane & 31);
  const bool row_ok = my_row < rows;
  const int node = row_ok ? my_row / g : 0;
  const int hq = it.kvh * g + (row_ok ? my_row % g : 0);
  const uint16_t *qbase = static_cast<const uint16_t *>(a.q) +
                          ((int64_t)(S.node0 + node) * a.n_q + hq) * D + 8 * h;
  bf16x8 qf[D / 16];
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks)
    qf[ks] = __builtin_bit_cast(bf16x8, ld16_or_zero(row_ok, qbase + 16 * ks));

  // Key range of this chunk: chunk boundaries lie inside the committed region and
  // the last chunk runs to the end of the tree rows, so every chunk holds at
  // least one key visible to every row.
  const int k0 = it.ch * S.ch_len;
  const int k1 = it.ch == S.nch - 1 ? L + N : k0 + S.ch_len;

  const uint16_t *Kg = static_cast<const uint16_t *>(a.k) + ((int64_t)it.kvh * a.cap_total + S.base) * D;
  const uint16_t *Vg = static_cast<const uint16_t *>(a.v) + ((int64_t)it.kvh * a.cap_total + S.base) * D;

  // Tile loaders.  K: 1024 16-byte chunks per tile.  V: per thread 4 keys x 8 d,
  // written transposed (8 x 8-byte stores).
  constexpr int KCH = TK * D / 8 / NT;        // K chunks per thread
  constexpr int VIT = (TK / 4) * (D / 8) / NT;  // V items per thread
  uint4 kr[KCH];
  uint4 vr[VIT][4];
  auto load_tile = [&](int kt) {
#pragma unroll
    for (int c = 0; c < KCH; ++c) {
      int q = tid + c * NT;
      int key = q >> 4, col = (q & 15) * 8;
      int t = kt + key;
      kr[c] = ld16_or_zero(t < k1, Kg + (int64_t)t * D + col);
    }
#pragma unroll
    for (int c = 0; c < VIT; ++c) {
      int q = tid + c * NT;
      int kg = q & 15, dc = q >> 4;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        int t = kt + 4 * kg + j;
        vr[c][j] = ld16_or_zero(t < k1, Vg + (int64_t)t * D + dc * 8);
      }
    }
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int c = 0; c < KCH; ++c) {
      int q = tid + c * NT;
      int key = q >> 4, col = (q & 15) * 8;
      *reinterpret_cast<uint4 *>(&Ks[key * KPITCH + col]) = kr[c];
    }
#pragma unroll
    for (int c = 0; c < VIT; ++c) {
      int q = tid + c * NT;
      int kg = q & 15, dc = q >> 4;
      const uint32_t w0[4] = {vr[c][0].x, vr[c][0].y, vr[c][0].z, vr[c][0].w};
      const uint32_t w1[4] = {vr[c][1].x, vr[c][1].y, vr[c][1].z, vr[c][1].w};
      const uint32_t w2[4] = {vr[c][2].x, vr[c][2].y, vr[c][2].z, vr[c][2].w};
      const uint32_t w3[4] = {vr[c][3].x, vr[c][3].y, vr[c][3].z, vr[c][3].w};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        // element e of keys 4kg..4kg+3 packed as one 8-byte row segment of V^T
        const int wi = e >> 1;
        uint2 pk;
        if (e & 1) {
          pk.x = (w0[wi] >> 16) | (w1[wi] & 0xFFFF0000u);
          pk.y = (w2[wi] >> 16) | (w3[wi] & 0xFFFF0000u);
        } else {
          pk.x = (w0[wi] & 0xFFFFu) | (w1[wi] << 16);
          pk.y = (w2[wi] & 0xFFFFu) | (w3[wi] << 16);
        }
        *reinterpret_cast<uint2 *>(&Vt[(dc * 8 + e) * VPITCH + 4 * kg]) = pk;
      }
    }
  };

  float m = -INFINITY, lsum = 0.f;
  f32x16 O[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) O[i][r] = 0.f;

  const uint32_t *my_anc = anc[node];
  load_tile(k0);
  for (int kt = k0; kt < k1; kt += TK) {
    __syncthreads();
    store_tile();
    __syncthreads();
    if (kt + TK < k1) load_tile(kt + TK);

    // S^T for two 32-key sub-blocks.
    f32x16 sc[2];
#pragma unroll
    for (int sb = 0; sb < 2; ++sb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) sc[sb][r] = 0.f;
      const uint16_t *kp = &Ks[(sb * 32 + (lane & 31)) * KPITCH + 8 * h];
#pragma unroll
      for (int ks = 0; ks < D / 16; ++ks) {
        bf16x8 kf = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4 *>(kp + 16 * ks));
        sc[sb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], sc[sb], 0, 0, 0);
      }
    }
    // Accumulator entry r of sub-block sb is key kt + 32sb + 8(r/4) + 4h + r%4.
    // Scores stay unscaled; the running max m is kept in scaled log2 units.
    const bool full = kt + TK <= min(k1, L);
    float tmax = -INFINITY;
#pragma unroll
    for (int sb = 0; sb < 2; ++sb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float s = sc[sb][r];
        if (!full) {
          const int t = kt + 32 * sb + 8 * (r >> 2) + 4 * h + (r & 3);
          const bool vis = t < k1 && (t < L || ((my_anc[(t - L) >> 5] >> ((t - L) & 31)) & 1u));
          s = vis ? s : -INFINITY;
        }
        sc[sb][r] = s;
        tmax = fmaxf(tmax, s);
      }
    tmax = max_with_other_half(tmax) * a.scale_log2;
    const float m_new = fmaxf(m, tmax);
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = fast_exp2(m - m_use);
    m = m_new;
    float psum = 0.f;
    uint32_t pk[2][2][4];
#pragma unroll
    for (int sb = 0; sb < 2; ++sb)
#pragma unroll
      for (int mh = 0; mh < 2; ++mh)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float p0 = fast_exp2(fmaf(sc[sb][8 * mh + 2 * j], a.scale_log2, -m_use));
          const float p1 = fast_exp2(fmaf(sc[sb][8 * mh + 2 * j + 1], a.scale_log2, -m_use));
          psum += p0 + p1;
          pk[sb][mh][j] = pack_bf16x2(p0, p1);
        }
    lsum = lsum * alpha + psum;
    if (__any(alpha != 1.f)) {          // the running max moved for some row of this wave
#pragma unroll
      for (int i = 0; i < D / 32; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) O[i][r] *= alpha;
    }

    // O^T += V^T P^T.  B operand slot 8h + i <-> key 16mh + 8(i/4) + 4h + i%4 of
    // sub-block sb; the A operand reads V^T in the same key order.
#pragma unroll
    for (int sb = 0; sb < 2; ++sb)
#pragma unroll
      for (int mh = 0; mh < 2; ++mh) {
        bf16x8 pf = __builtin_bit_cast(bf16x8, uint4{pk[sb][mh][0], pk[sb][mh][1], pk[sb][mh][2], pk[sb][mh][3]});
        const int kofs = 32 * sb + 16 * mh + 4 * h;
#pragma unroll
        for (int i = 0; i < D / 32; ++i) {
          const uint16_t *vp = &Vt[(32 * i + (lane & 31)) * VPITCH + kofs];
          uint2 lo = *reinterpret_cast<const uint2 *>(vp);
          uint2 hi = *reinterpret_cast<const uint2 *>(vp + 8);
          bf16x8 vf = __builtin_bit_cast(bf16x8, uint4{lo.x, lo.y, hi.x, hi.y});
          O[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf, O[i], 0, 0, 0);
        }
      }
  }

  const float ltot = sum_with_other_half(lsum);
  if (!row_ok) return;
  // O^T entry r of d-block i is d = 32i + 8(r/4) + 4h + r%4 of this lane's row.
  if (S.nch == 1) {
    const float inv = 1.f / ltot;
    uint16_t *op = static_cast<uint16_t *>(a.out) + ((int64_t)(S.node0 + node) * a.n_q + hq) * D;
#pragma unroll
    for (int i = 0; i < D / 32; ++i)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        uint2 v = {pack_bf16x2(O[i][4 * q4] * inv, O[i][4 * q4 + 1] * inv),
                   pack_bf16x2(O[i][4 * q4 + 2] * inv, O[i][4 * q4 + 3] * inv)};
        *reinterpret_cast<uint2 *>(op + 32 * i + 8 * q4 + 4 * h) = v;
      }
  } else {
    const int local_row = my_row - it.rb * RB;
    float *slot = a.part + ((int64_t)S.part0 + ((int64_t)it.kvh * S.nrb + it.rb) * S.nch + it.ch) *
                               (int64_t)attn_partial_floats(RB);
    float *po = slot + (int64_t)local_row * D;
#pragma unroll
    for (int i = 0; i < D / 32; ++i)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4)
        *reinterpret_cast<float4 *>(po + 32 * i + 8 * q4 + 4 * h) =
            float4{O[i][4 * q4], O[i][4 * q4 + 1], O[i][4 * q4 + 2], O[i][4 * q4 + 3]};
    if (h == 0) {
      slot[(int64_t)RB * D + local_row] = m;
      slot[(int64_t)RB * D + RB + local_row] = ltot;
    }
  }
}

// Merge the chunk partials of one (sequence, KV head, row block) in chunk order;
// each block handles kCombineRows rows of the row block.
constexpr int kCombineRows = 256 / (D / 4);   // 8 rows x 32 float4 columns per block

template <int WAVES>
__global__ __launch_bounds__(256) void tree_attn_combine(AttnArgs a) {
  constexpr int RB = 32 * WAVES;
  constexpr int PARTS = RB / kCombineRows;
  const int idx = blockIdx.x / PARTS, part = blockIdx.x % PARTS;
  int s = 0;
  for (int j = 0; j < a.nseq; ++j)
    if (a.seq[j].nch > 1 && a.seq[j].citem0 <= idx) s = j;
  const AttnSeq &S = a.seq[s];
  const int local = idx - S.citem0;
  const int kvh = local / S.nrb, rb = local % S.nrb;
  const int rows = S.N * a.group;
  const int64_t pf = attn_partial_floats(RB);
  const float *base = a.part + ((int64_t)S.part0 + ((int64_t)kvh * S.nrb + rb) * S.nch) * pf;
  const int r = part * kCombineRows + threadIdx.x / (D / 4);
  const int d4 = (threadIdx.x % (D / 4)) * 4;
  const int row = rb * RB + r;
  if (row >= rows) return;
  float M = -INFINITY;
  for (int c = 0; c < S.nch; ++c) M = fmaxf(M, base[c * pf + (int64_t)RB * D + r]);
  float l = 0.f, o0 = 0.f, o1 = 0.f, o2 = 0.f, o3 = 0.f;
  for (int c = 0; c < S.nch; ++c) {
    const float *sl = base + c * pf;
    const float w = fast_exp2(sl[(int64_t)RB * D + r] - M);
    l += w * sl[(int64_t)RB * D + RB + r];
    const float4 o = *reinterpret_cast<const float4 *>(sl + (int64_t)r * D + d4);
    o0 += w * o.x;
    o1 += w * o.y;
    o2 += w * o.z;
    o3 += w * o.w;
  }
  const float inv = 1.f / l;
  const int node = row / a.group, hq = kvh * a.group + row % a.group;
  uint16_t *op = static_cast<uint16_t *>(a.out) + ((int64_t)(S.node0 + node) * a.n_q + hq) * D + d4;
  *reinterpret_cast<uint2 *>(op) = uint2{pack_bf16x2(o0 * inv, o1 * inv), pack_bf16x2(o2 * inv, o3 * inv)};
}

// fp32 path: one wave per (node, query head); lanes own head-dimension elements
// and walk the key set one key at a time.
__global__ __launch_bounds__(256) void tree_attn_f32(AttnArgs a, int node_begin, int node_count) {
  const int lane = threadIdx.x & 63;
  const int w = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (w >= node_count * a.n_q) return;
  const int gnode = node_begin + w / a.n_q, hq = w % a.n_q;
  int s = 0;
  while (s + 1 < a.nseq && a.seq[s + 1].node0 <= gnode) ++s;
  const AttnSeq &S = a.seq[s];
  const int n = gnode - S.node0, kvh = hq / a.group, d = a.head_dim;
  const float *q = static_cast<const float *>(a.q) + ((int64_t)gnode * a.n_q + hq) * d;
  const float *K = static_cast<const float *>(a.k) + ((int64_t)kvh * a.cap_total + S.base) * d;
  const float *V = static_cast<const float *>(a.v) + ((int64_t)kvh * a.cap_total + S.base) * d;
  const bool e0 = lane < d, e1 = lane + 64 < d;
  const float q0 = e0 ? q[lane] : 0.f, q1 = e1 ? q[lane + 64] : 0.f;
  float m = -INFINITY, l = 0.f, o0 = 0.f, o1 = 0.f;
  auto visit = [&](int64_t row) {
    float p = (e0 ? q0 * K[row * d + lane] : 0.f) + (e1 ? q1 * K[row * d + lane + 64] : 0.f);
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) p += __shfl_xor(p, off);
    const float s = p * a.scale;
    const float mn = fmaxf(m, s);
    const float alpha = expf(m - mn), pe = expf(s - mn);
    l = l * alpha + pe;
    o0 = o0 * alpha + pe * (e0 ? V[row * d + lane] : 0.f);
    o1 = o1 * alpha + pe * (e1 ? V[row * d + lane + 64] : 0.f);
    m = mn;
  };
  for (int t = 0; t < S.L; ++t) visit(t);
  for (int u = n; u >= 0; u = a.parent[S.node0 + u]) visit(S.L + u);
  float *out = static_cast<float *>(a.out) + ((int64_t)gnode * a.n_q + hq) * d;
  if (e0) out[lane] = o0 / l;
  if (e1) out[lane + 64] = o1 / l;
}

}  // namespace

hipError_t launch_tree_attn_bf16(const AttnArgs &a, int waves, hipStream_t st) {
  if (waves == 2) {
    hipLaunchKernelGGL(tree_attn_bf16<2>, dim3(a.items), dim3(128), 0, st, a);
    if (a.citems) hipLaunchKernelGGL(tree_attn_combine<2>, dim3(a.citems * (64 / kCombineRows)), dim3(256), 0, st, a);
  } else {
    hipLaunchKernelGGL(tree_attn_bf16<4>, dim3(a.items), dim3(256), 0, st, a);
    if (a.citems) hipLaunchKernelGGL(tree_attn_combine<4>, dim3(a.citems * (128 / kCombineRows)), dim3(256), 0, st, a);
  }
  return hipGetLastError();
}

hipError_t launch_tree_attn_f32(const AttnArgs &a, int node_begin, int node_count, hipStream_t st) {
  const int waves = node_count * a.n_q;
  hipLaunchKernelGGL(tree_attn_f32, dim3((waves + 3) / 4), dim3(256), 0, st, a, node_begin, node_count);
  return hipGetLastError();
}

}  // namespace specmemo
