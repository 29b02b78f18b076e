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
#include <mutex>
#include <type_traits>

#include "device.h"
#include "internal.h"

namespace specmemo {

namespace {

constexpr int D = kAttnHeadDim;
constexpr int TK = kAttnKeyTile;
constexpr float kRescaleSlack = 8.f;   // log2 units: softmax weights stay <= 256 between rescales

struct Item {
  int s, kvh, rb, ch;
};

// The sequence of a block is found by one wave-parallel search: lane l holds
// sequence l's first position (the launch holds at most kMaxSeqPerLaunch
// sequences) and a ballot counts the starts at or below the block's position.
__device__ __forceinline__ int find_seq(int nseq, int start_of_lane, int pos) {
  const int lane = threadIdx.x & 63;
  const uint64_t le = __builtin_amdgcn_ballot_w64(lane < nseq && start_of_lane <= pos);
  return __builtin_popcountll(le) - 1;
}

__device__ __forceinline__ int rl(int v, int lane) { return __builtin_amdgcn_readlane(v, lane); }

// Descriptor of sequence s from the per-lane copies (lane l holds sequence l).
__device__ __forceinline__ AttnSeq pick_seq(const AttnSeq &d, int s) {
  AttnSeq r;
  r.base = (int64_t)((uint64_t)(uint32_t)rl((int)(d.base >> 32), s) << 32 | (uint32_t)rl((int)d.base, s));
  r.L = rl(d.L, s);
  r.node0 = rl(d.node0, s);
  r.N = rl(d.N, s);
  r.nrb = rl(d.nrb, s);
  r.nch = rl(d.nch, s);
  r.ch_len = rl(d.ch_len, s);
  r.item0 = rl(d.item0, s);
  r.part0 = rl(d.part0, s);
  r.citem0 = rl(d.citem0, s);
  r.unit0 = rl(d.unit0, s);
  return r;
}

// Work item and sequence descriptor of block `bid`; false for a padding block.
// Every load is issued up front (one memory latency): the per-lane copies of
// the sequence descriptors and, for the XCD order, of XCD x's block counts.
//
// Launch order: sequence, then KV head, chunk, row block.
//
// XCD order: blocks reach the eight XCDs round-robin by block id, so block
// 8 k + x is the k-th block of XCD x.  A unit is one (sequence, KV head) with
// all its chunks and row blocks; unit u (launch order, longest sequences
// first) runs on XCD u mod 8, chunk by chunk with the row blocks of a chunk
// adjacent, so the row blocks reading the same K/V share one L2, the chunk
// partials are merged on the XCD that wrote them, and with 8 KV heads (or a
// multiple) every XCD gets one KV head of every sequence.  xcd_cum[x][s] is
// the number of XCD x's blocks before sequence s; blocks past the busiest
// XCD's work are padding.
__device__ __forceinline__ bool decode_item(const AttnArgs &a, int bid, Item &it, AttnSeq &S) {
  if (a.map) {   // table mode: the host decoded every block's item (same order as below)
    const AttnItem m = a.map[bid];
    if (m.s == 0xFFFF) return false;
    it.s = m.s;
    it.kvh = m.kvh;
    it.ch = m.ch;
    it.rb = m.rb;
    S = a.tab[m.s];
    return true;
  }
  const int lane = threadIdx.x & 63;
  const int x = bid & 7, k = bid >> 3;
  AttnSeq mine{};
  if (lane < kMaxSeqPerLaunch) mine = a.seq[lane];
  const int cum = lane <= kMaxSeqPerLaunch ? a.xcd_cum[x][lane] : 0;
  const int nseq = a.nseq;
  if (a.xcd_order) {
    if (k >= rl(cum, nseq)) return false;
    const int s = find_seq(nseq, cum, k);
    S = pick_seq(mine, s);
    const int kk = k - rl(cum, s);
    const int per_unit = S.nch * S.nrb;
    it.s = s;
    it.kvh = ((x - (S.unit0 & 7)) & 7) + 8 * (kk / per_unit);   // this sequence's KV heads on XCD x: first, +8, ...
    const int local = kk % per_unit;
    it.ch = local / S.nrb;
    it.rb = local % S.nrb;
  } else {
    const int s = find_seq(nseq, mine.item0, bid);
    S = pick_seq(mine, s);
    int local = bid - S.item0;
    it.s = s;
    it.rb = local % S.nrb;
    local /= S.nrb;
    it.ch = local % S.nch;
    it.kvh = local / S.nch;
  }
  return true;
}

// Maximum of a lane's 32 scores as a tree of three-input maxima (16 operations).
__device__ __forceinline__ float tile_max32(const f32x16 (&x)[2]) {
  float t[12];
#pragma unroll
  for (int i = 0; i < 10; ++i) {
    const int e = 3 * i;
    t[i] = fmaxf(fmaxf(x[e >> 4][e & 15], x[(e + 1) >> 4][(e + 1) & 15]), x[(e + 2) >> 4][(e + 2) & 15]);
  }
  t[10] = x[1][14];
  t[11] = x[1][15];
  const float u0 = fmaxf(fmaxf(t[0], t[1]), t[2]), u1 = fmaxf(fmaxf(t[3], t[4]), t[5]);
  const float u2 = fmaxf(fmaxf(t[6], t[7]), t[8]), u3 = fmaxf(fmaxf(t[9], t[10]), t[11]);
  return fmaxf(fmaxf(u0, u1), fmaxf(u2, u3));
}

typedef __attribute__((address_space(3))) void lds_void_t;
typedef short s16x4_t __attribute__((__vector_size__(8)));
typedef __attribute__((address_space(3))) s16x4_t lds_s16x4_t;
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// 16-byte direct load of every lane into LDS at lds_base + 16 * lane (one
// global_load_lds_dwordx4 with M0 = lds_base, which must be wave-uniform),
// from the wave-uniform base `src` (SGPRs) plus this lane's 32-bit byte
// offset.  It is issued from inline assembly so that the compiler does not
// guard later LDS reads with waits for it: the tile ring orders these loads
// with explicit vmcnt waits.  M0 must be written one wait state before the load.
// A wave-uniform pointer, made explicit for the compiler (so that it stays in
// SGPRs, as the base operand of the direct loads requires).
template <typename T>
__device__ __forceinline__ T *uniform_ptr(T *p) {
  const uint64_t b = reinterpret_cast<uintptr_t>(p);
  return reinterpret_cast<T *>((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(b >> 32)) << 32 |
                               (uint32_t)__builtin_amdgcn_readfirstlane((int)b));
}

__device__ __forceinline__ void lds_load16(const void *src, uint32_t off, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(src), "s"(lds_base)
               : "memory", "m0");
}

// Workgroup barrier for the LDS tile ring.  The tile loads into LDS are
// ordered by explicit vmcnt waits; a __syncthreads() would also wait for the
// loads still in flight for later tiles (its release fence waits for every
// outstanding vector memory operation) and so shorten the prefetch distance.
__device__ __forceinline__ void ring_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// LDS swizzles (16-byte chunk index c of tile row r).  K rows are read 16 rows
// at a time at one chunk (MFMA A operand): chunk c of row r sits at c ^ (r % 16).
// V rows are read by the transposing load 4 rows x 4 chunks at a time:
// chunk c of row r sits at c ^ 4 (r % 4).
__device__ __forceinline__ int kswz(int r, int c) { return c ^ (r & 15); }
__device__ __forceinline__ int vswz(int r, int c) { return c ^ ((r & 3) << 2); }

// WAVES waves per block, 32 query rows per wave (one per lane pair l, l^32);
// K and V each have a SLOTS-deep ring of 64-key tiles filled by direct loads;
// iteration j computes S, the weights and O for tile j.
// KSPLIT = 1: every wave takes both 32-key halves of a tile (its two products
// S^T = K Q^T being independent accumulation chains); RB = 32 WAVES rows.
// KSPLIT = 2: the waves form two groups over the same RB = 16 WAVES rows, the
// first taking keys 0-31 of every tile and the second keys 32-63, each with
// its own online softmax; the two groups' (m, l, O) are merged through LDS at
// the end.  With few rows per K/V tile (multi-head attention: 64 rows per
// (sequence, head)) this halves each wave's chain per tile and keeps two
// waves on every SIMD.
// MINB: blocks that must fit on one compute unit (bounds the registers).
// PAD: the cache holds pad tokens (padded batching), flagged in a.key_valid.
template <int WAVES, int SLOTS, int MINB, bool PAD, int KSPLIT>
__global__ __launch_bounds__(WAVES * 64, MINB) void tree_attn_bf16(AttnArgs a) {
  static_assert(SLOTS == 2 || SLOTS == 3, "ring depth");
  static_assert(KSPLIT == 1 || KSPLIT == 2, "key split");
  constexpr int RW = WAVES / KSPLIT;          // waves per key group
  constexpr int RB = 32 * RW;
  constexpr int NSB = 2 / KSPLIT;             // 32-key sub-blocks per wave and tile
  constexpr int TILE = TK * D * 2;            // bytes of one K or V tile (16 KB)
  constexpr int IPW = TILE / 1024 / WAVES;    // 1 KB direct loads per wave per tile and operand
  __shared__ __attribute__((aligned(1024))) uint8_t kring[SLOTS][TILE];
  __shared__ __attribute__((aligned(1024))) uint8_t vring[SLOTS][TILE];
  // The tree's parent array is staged in the last V slot, which the prologue
  // does not fill and the first loop barrier frees again.
  int *const par = reinterpret_cast<int *>(vring[SLOTS - 1]);
  static_assert(WAVES * 64 >= kMaxNodes && kMaxNodes * 4 <= TILE, "one thread per tree node");
  static_assert(KSPLIT == 1 || RW * 64 * 64 * 4 <= SLOTS * TILE, "merge buffer fits the K ring");

  Item it;
  AttnSeq S;
  if (!decode_item(a, blockIdx.x, it, S)) return;   // padding block: no work, no barrier reached
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int rwave = wave % RW, ksb = wave / RW;     // row group and key group of this wave
  const int h = lane >> 5;              // which half of the wave
  const int L = S.L, N = S.N, g = a.group;
  const int rows = N * g;

  // Key range of this chunk: chunk boundaries lie inside the committed region and
  // the last chunk runs to the end of the tree rows, so every chunk holds at
  // least one key visible to every row.
  const int k0 = it.ch * S.ch_len;
  const int k1 = it.ch == S.nch - 1 ? L + N : k0 + S.ch_len;
  const int ntiles = (k1 - k0 + TK - 1) / TK;
  const uint16_t *Kg = static_cast<const uint16_t *>(a.k) + ((int64_t)it.kvh * a.cap_total + S.base) * D;
  const uint16_t *Vg = static_cast<const uint16_t *>(a.v) + ((int64_t)it.kvh * a.cap_total + S.base) * D;

  // Direct loads of a tile into its ring slot: lane l of load i writes LDS bytes
  // [1024 i + 16 l, +16), i.e. tile row r = 4 i + l / 16 at physical chunk l % 16,
  // which holds logical chunk (l % 16) ^ (r % 16) of K or (l % 16) ^ 4 (r % 4)
  // of V.  For this wave's u-th load, r = 4 (wave IPW + u) + l / 16: the V
  // offset and the row advance by 1024 and 4 per load; the K chunk is
  // (l % 16) ^ (l / 16) ^ 4 (u + wave IPW) % 16.  Rows past the chunk end repeat
  // its last row (finite values, masked out).
  const int lrow0 = 4 * wave * IPW + (lane >> 4);
  const int kx = (lane & 15) ^ (lane >> 4);
  const int voff0 = lrow0 * (D * 2) + 16 * vswz(lrow0, lane & 15);
  auto load_off = [&](bool is_k, int u) {
    const int r = lrow0 + 4 * u;
    return is_k ? r * (D * 2) + 16 * (kx ^ ((4 * (wave * IPW + u)) & 15)) : voff0 + 1024 * u;
  };
  const uint8_t *Kb = uniform_ptr(reinterpret_cast<const uint8_t *>(Kg));
  const uint8_t *Vb = uniform_ptr(reinterpret_cast<const uint8_t *>(Vg));
  // Offsets are relative to the slab base (a slab is at most 2^24 rows, so they
  // fit 32 bits); the base of a full tile is wave-uniform.
  auto issue = [&](const uint8_t *src, bool is_k, uint8_t *dst, int j) {
    const int kt = k0 + j * TK;
    const uint32_t lds = __builtin_amdgcn_readfirstlane(
        (uint32_t)(uintptr_t)(lds_void_t *)(dst + 1024 * wave * IPW));
    if (kt + TK <= k1) {
      const uint8_t *sb = src + (int64_t)kt * (D * 2);
#pragma unroll
      for (int u = 0; u < IPW; ++u) lds_load16(sb, (uint32_t)load_off(is_k, u), lds + 1024 * u);
    } else {                             // last tile: rows past the chunk end repeat its last row
#pragma unroll
      for (int u = 0; u < IPW; ++u) {
        const int r = lrow0 + 4 * u;
        const int t = min(kt + r, k1 - 1);
        lds_load16(src, (uint32_t)(t * (D * 2) + (load_off(is_k, u) - r * (D * 2))), lds + 1024 * u);
      }
    }
  };
  auto issue_k = [&](int j) { issue(Kb, true, kring[j % SLOTS], j); };
  auto issue_v = [&](int j) { issue(Vb, false, vring[j % SLOTS], j); };

  // Prologue: tiles 0 .. SLOTS-2 (K then V) first, then the Q fragments of this
  // lane's query row (B operand of S^T = K Q^T) and the tree's parent array,
  // so that the three loads share one memory latency.
#pragma unroll
  for (int t = 0; t < SLOTS - 1; ++t)
    if (t < ntiles) {
      issue_k(t);
      issue_v(t);
    }
  const int pn = tid < N ? a.parent[S.node0 + tid] : -1;
  const int my_row = it.rb * RB + rwave * 32 + (lane & 31);
  const bool row_ok = my_row < rows;
  const int node = row_ok ? my_row / g : 0;
  const int hq = it.kvh * g + (row_ok ? my_row % g : 0);
  bf16x8 qf[D / 16];
  {
    const uint16_t *qbase = static_cast<const uint16_t *>(a.q) + ((int64_t)(S.node0 + node) * a.n_q + hq) * D + 8 * h;
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) qf[ks] = __builtin_bit_cast(bf16x8, ld16_or_zero(row_ok, qbase + 16 * ks));
  }
  if (tid < N) par[tid] = pn;
  // Land the Q loads here: otherwise the compiler waits for them at their
  // first use inside the tile loop, on every iteration, and with them for
  // every tile load in flight.
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) asm volatile("" ::"v"(qf[ks]));
  ring_barrier();

  // Ancestor-or-self bitmask of this lane's node (local ids), walked in LDS
  // and kept in registers.
  uint4 anc = {0u, 0u, 0u, 0u};
  for (int u = node; u >= 0; u = par[u]) {
    const uint32_t bit = 1u << (u & 31);
    const int w = u >> 5;
    anc.x |= w == 0 ? bit : 0u;
    anc.y |= w == 1 ? bit : 0u;
    anc.z |= w == 2 ? bit : 0u;
    anc.w |= w == 3 ? bit : 0u;
  }

  // K operand: row (lane & 31) of a 32-key sub-block, 16-byte chunk 2 ks + h.
  int kro[D / 16];
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) kro[ks] = (lane & 31) * (D * 2) + 16 * ((2 * ks + h) ^ (lane & 15));
  // Transposing-load source role of this lane within its 16-lane group: source
  // lane 4 tj + tq supplies key row tj, head-dim columns 4 tq .. 4 tq + 3 of the
  // group's 16 columns; destination lane o then holds 4 keys of column o.  With
  // the V swizzle the byte offset of d-block i is a per-lane constant.
  const int tj = (lane & 15) >> 2, tq = lane & 3;
  const int te = 2 * ((lane >> 4) & 1) + (tq >> 1);
  int vro[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i) vro[i] = (4 * h + tj) * (D * 2) + 64 * (i ^ tj) + 16 * te + 8 * (tq & 1);
  // First 32-key sub-block of this wave's keys in a tile.
  const int sb0 = ksb * NSB;

  auto qk = [&](const uint8_t *ks, f32x16 (&Sc)[NSB]) {
#pragma unroll
    for (int sb = 0; sb < NSB; ++sb)
#pragma unroll
      for (int r2 = 0; r2 < 16; ++r2) Sc[sb][r2] = 0.f;
    const uint8_t *kw = ks + sb0 * 32 * (D * 2);
#pragma unroll
    for (int k8 = 0; k8 < D / 16; ++k8)
#pragma unroll
      for (int sb = 0; sb < NSB; ++sb) {
        const bf16x8 kf = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4 *>(kw + sb * 32 * (D * 2) + kro[k8]));
        Sc[sb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[k8], Sc[sb], 0, 0, 0);
      }
    // keep the K fragment reads just ahead of their products (NSB LDS reads,
    // NSB products, eight times) instead of all of them up front
#pragma unroll
    for (int k8 = 0; k8 < D / 16; ++k8) {
      __builtin_amdgcn_sched_group_barrier(0x100, NSB, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, NSB, 0);
    }
  };

  // Padded batching (Sec. 3.3): the pad-token flags of the 64 keys of a tile,
  // as a wave-uniform 64-bit word; bit i is key kt + i, and keys from the tree
  // rows on count as valid (the ancestor mask governs them).  Scalar load of
  // the four words around the tile's first row, waited for in place.
  const uint32_t *const mask_base = PAD ? uniform_ptr(a.key_valid) : nullptr;
  auto pad_bits = [&](int kt) -> uint64_t {
    const int64_t row = S.base + kt;
    const uint32_t *p = mask_base + (row >> 5);
    u32x4_t w;
    asm volatile("s_load_dwordx4 %0, %1, 0x0\n\ts_waitcnt lgkmcnt(0)" : "=s"(w) : "s"(p));
    const uint32_t sh = (uint32_t)row & 31u;
    uint64_t bits = ((uint64_t)w[1] << 32 | w[0]) >> sh;
    bits |= sh ? (uint64_t)w[2] << (64 - sh) : 0ull;
    const int committed = L - kt;
    return committed < TK ? bits | (~0ull << committed) : bits;
  };

  float m = -INFINITY, lsum = 0.f;
  f32x16 O[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) O[i][r] = 0.f;
  const bf16x2_t ones = __builtin_bit_cast(bf16x2_t, 0x3F803F80u);

  // Scores of tile j -> bf16 weights (online softmax, lazy rescale); O += V^T P^T.
  // Accumulator entry r of the wave's sub-block sb is key
  // kt + 32 (sb0 + sb) + 8 (r / 4) + 4 h + r % 4.
  // The tree mask, for tiles that reach the tree rows or the chunk end, is
  // branch-free (bitwise tests, one select per score) so that the scores keep
  // their registers on both paths.  The weights are returned packed as the B
  // operands of the wave's 16-key groups of the PV product.
  auto softmax_head = [&](int j, f32x16 (&Sc)[NSB]) {   // mask, tile max, rescaling
    const int kt = k0 + j * TK;
    if constexpr (PAD) {
      if (kt < L) {                      // committed keys: pad tokens take -inf
        const uint64_t all = pad_bits(kt);
        if (all != ~0ull) {              // wave-uniform: tiles without pads skip the selects
          const uint64_t bits = all >> (4 * h);
#pragma unroll
          for (int sb = 0; sb < NSB; ++sb)
#pragma unroll
            for (int r2 = 0; r2 < 16; ++r2)
              Sc[sb][r2] = (bits >> (32 * (sb0 + sb) + 8 * (r2 >> 2) + (r2 & 3))) & 1u ? Sc[sb][r2] : -INFINITY;
        }
      }
    }
    if (kt + TK > min(k1, L)) {
      const uint64_t alo = (uint64_t)anc.y << 32 | anc.x, ahi = (uint64_t)anc.w << 32 | anc.z;
#pragma unroll
      for (int sb = 0; sb < NSB; ++sb)
#pragma unroll
        for (int r2 = 0; r2 < 16; ++r2) {
          const int t = kt + 32 * (sb0 + sb) + 8 * (r2 >> 2) + 4 * h + (r2 & 3);
          const uint32_t rel = (uint32_t)(t - L) & 127u;
          const uint64_t word = rel < 64 ? alo : ahi;
          const bool anc_bit = (word >> (rel & 63)) & 1u;
          const bool vis = (t < k1) & ((t < L) | anc_bit);
          Sc[sb][r2] = vis ? Sc[sb][r2] : -INFINITY;
        }
    }
    float tm;
    if constexpr (NSB == 2) {
      tm = tile_max32(Sc);
    } else {
      const f32x16 &x = Sc[0];
      const float u0 = fmaxf(fmaxf(x[0], x[1]), x[2]), u1 = fmaxf(fmaxf(x[3], x[4]), x[5]);
      const float u2 = fmaxf(fmaxf(x[6], x[7]), x[8]), u3 = fmaxf(fmaxf(x[9], x[10]), x[11]);
      const float u4 = fmaxf(fmaxf(x[12], x[13]), x[14]);
      tm = fmaxf(fmaxf(fmaxf(u0, u1), fmaxf(u2, u3)), fmaxf(u4, x[15]));
    }
    const float tmax = max_with_other_half(tm) * a.scale_log2;
    // Lazy rescaling: the reference max m moves only when a score exceeds it by
    // more than kRescaleSlack (log2 units), so weights stay <= 2^kRescaleSlack;
    // the branch is taken by the whole wave, rarely after the first tile.
    const bool need = tmax > m + kRescaleSlack;
    if (__builtin_amdgcn_ballot_w64(need)) {
      const float m_new = need ? tmax : m;
      const float alpha = need ? (m == -INFINITY ? 0.f : fast_exp2(m - m_new)) : 1.f;
      m = m_new;
      lsum *= alpha;
#pragma unroll
      for (int i = 0; i < D / 32; ++i)
#pragma unroll
        for (int r2 = 0; r2 < 16; ++r2) O[i][r2] *= alpha;
    }
  };
  auto softmax_tail = [&](const f32x16 (&Sc)[NSB], uint32_t (&pk)[2 * NSB][4]) {   // weights and row sum
    const float m_use = m == -INFINITY ? 0.f : m;
    // B operand of local 16-key group 2 sb + half: slot 8 h + s <-> key
    // 32 (sb0 + sb) + 16 half + 8 (s / 4) + 4 h + s % 4 (the V^T reads use the same order).
#pragma unroll
    for (int sb = 0; sb < NSB; ++sb)
#pragma unroll
      for (int half = 0; half < 2; ++half)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float p0 = fast_exp2(fmaf(Sc[sb][8 * half + 2 * q], a.scale_log2, -m_use));
          const float p1 = fast_exp2(fmaf(Sc[sb][8 * half + 2 * q + 1], a.scale_log2, -m_use));
          pk[2 * sb + half][q] = pack_bf16x2(p0, p1);
        }
    // Row sum of the bf16 weights that enter O (two-term dot products with ones).
#pragma unroll
    for (int mh = 0; mh < 2 * NSB; ++mh)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        lsum = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, pk[mh][q]), ones, lsum, false);
  };
  auto pv = [&](const uint8_t *vs, const uint32_t (&pk)[2 * NSB][4]) {
#pragma unroll
    for (int mh = 0; mh < 2 * NSB; ++mh) {
      const bf16x8 pf = __builtin_bit_cast(bf16x8, uint4{pk[mh][0], pk[mh][1], pk[mh][2], pk[mh][3]});
#pragma unroll
      for (int i = 0; i < D / 32; ++i) {
        const uint8_t *p = vs + 16 * (2 * sb0 + mh) * (D * 2) + vro[i];
        const s16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t *)p);
        const s16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t *)(p + 8 * (D * 2)));
        const bf16x8 vf = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
        O[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf, O[i], 0, 0, 0);
      }
    }
  };

  auto wait_loads = [&](int later) {   // wait until at most `later` x IPW of this wave's loads are pending
    if (later >= 2)
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * IPW) : "memory");
    else if (later == 1)
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(IPW) : "memory");
    else
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  };

  // Iteration j needs tile j; after its barrier every wave is done with tile
  // j-1, whose slots take tile j+SLOTS-1.  The loop is unrolled by the ring
  // depth, so that every slot address is a constant (the LDS reads then take
  // it as their immediate offset instead of a vector add per read).
  auto tile = [&](int j, auto slot_c) {
    constexpr int slot = decltype(slot_c)::value;
    // loads issued after tile j: tile j+1 (3 slots), two operands
    wait_loads(SLOTS == 3 && j + 1 < ntiles ? 2 : 0);
    ring_barrier();
    if (j + SLOTS - 1 < ntiles) {
      issue(Kb, true, kring[(slot + SLOTS - 1) % SLOTS], j + SLOTS - 1);
      issue(Vb, false, vring[(slot + SLOTS - 1) % SLOTS], j + SLOTS - 1);
    }
    f32x16 Sc[NSB];
    uint32_t pk[2 * NSB][4];
    qk(kring[slot], Sc);
    softmax_head(j, Sc);
    softmax_tail(Sc, pk);
    pv(vring[slot], pk);
  };
  for (int j = 0; j < ntiles; j += SLOTS) {
    tile(j, std::integral_constant<int, 0>{});
    if (j + 1 < ntiles) tile(j + 1, std::integral_constant<int, 1>{});
    if constexpr (SLOTS == 3)
      if (j + 2 < ntiles) tile(j + 2, std::integral_constant<int, 2>{});
  }

  float ltot = sum_with_other_half(lsum);
  if constexpr (KSPLIT == 2) {
    // Merge the second key group's (m, l, O) into the first's.  Every wave is
    // past its last read of the ring (the barrier) and no tile load is in
    // flight (the last iteration waited for all of them), so the K ring holds
    // the second group's O, [row wave][value][lane] (conflict-free), and the
    // V ring its m and l.
    ring_barrier();
    float *const mo = reinterpret_cast<float *>(kring[0]);
    float *const ml = reinterpret_cast<float *>(vring[0]);
    if (ksb == 1) {
#pragma unroll
      for (int i = 0; i < D / 32; ++i)
#pragma unroll
        for (int r2 = 0; r2 < 16; ++r2) mo[(rwave * 64 + 16 * i + r2) * 64 + lane] = O[i][r2];
      ml[(rwave * 2) * 64 + lane] = m;
      ml[(rwave * 2 + 1) * 64 + lane] = ltot;
    }
    ring_barrier();
    if (ksb == 1) return;
    const float m1 = ml[(rwave * 2) * 64 + lane], l1 = ml[(rwave * 2 + 1) * 64 + lane];
    const float mn = fmaxf(m, m1);
    const float w0 = m == -INFINITY ? 0.f : fast_exp2(m - mn);
    const float w1 = m1 == -INFINITY ? 0.f : fast_exp2(m1 - mn);
#pragma unroll
    for (int i = 0; i < D / 32; ++i)
#pragma unroll
      for (int r2 = 0; r2 < 16; ++r2) O[i][r2] = O[i][r2] * w0 + mo[(rwave * 64 + 16 * i + r2) * 64 + lane] * w1;
    ltot = ltot * w0 + l1 * w1;
    m = mn;
  }
  if (!row_ok) return;
  // O^T entry r of d-block i is d = 32 i + 8 (r / 4) + 4 h + r % 4 of this lane's row.
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
    uint16_t *po = reinterpret_cast<uint16_t *>(slot) + (int64_t)local_row * D;
#pragma unroll
    for (int i = 0; i < D / 32; ++i)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4)
        *reinterpret_cast<uint2 *>(po + 32 * i + 8 * q4 + 4 * h) =
            uint2{pack_bf16x2(O[i][4 * q4], O[i][4 * q4 + 1]), pack_bf16x2(O[i][4 * q4 + 2], O[i][4 * q4 + 3])};
    if (h == 0) {
      slot[(int64_t)RB * D / 2 + local_row] = m;
      slot[(int64_t)RB * D / 2 + RB + local_row] = ltot;
    }
  }
}

// Merge the chunk partials of one (sequence, KV head, row block) in chunk
// order (deterministic, no atomics): one block per row block, four threads per
// query row, each with 32 head-dim columns, and one pass over the chunks with
// a running max (the partials hold unnormalised O in bf16, the chunk's max m
// and sum l in fp32), the loads of four chunks in flight at once.
template <int RB>
__global__ __launch_bounds__(4 * RB) void tree_attn_combine(AttnArgs a) {
  constexpr int CPT = D / 4;   // columns per thread
  const int idx = blockIdx.x, lane = threadIdx.x & 63;
  const int x = idx & 7, k = idx >> 3;
  int kvh, rb;
  AttnSeq S;
  AttnSeq mine{};
  if (!a.cmap && lane < kMaxSeqPerLaunch) mine = a.seq[lane];
  const int ccum = !a.cmap && lane <= kMaxSeqPerLaunch ? a.xcd_ccum[x][lane] : 0;
  if (a.cmap) {   // table mode: the host decoded every block's row block
    const AttnItem m = a.cmap[idx];
    if (m.s == 0xFFFF) return;
    S = a.tab[m.s];
    kvh = m.kvh;
    rb = m.rb;
  } else if (a.xcd_order) {
    // the k-th combine item of XCD x, on the XCD that computed its chunks
    if (k >= rl(ccum, a.nseq)) return;   // padding block
    const int s = find_seq(a.nseq, ccum, k);
    S = pick_seq(mine, s);
    const int kk = k - rl(ccum, s);
    kvh = ((x - (S.unit0 & 7)) & 7) + 8 * (kk / S.nrb);
    rb = kk % S.nrb;
  } else {
    // the split sequence of this block: the last one whose first combine item is <= idx
    const bool split_le = lane < a.nseq && mine.nch > 1 && mine.citem0 <= idx;
    const int s = 63 - __builtin_clzll(__builtin_amdgcn_ballot_w64(split_le));
    S = pick_seq(mine, s);
    const int local = idx - S.citem0;
    kvh = local / S.nrb;
    rb = local % S.nrb;
  }
  const int r = threadIdx.x >> 2, quarter = threadIdx.x & 3;
  const int row = rb * RB + r;
  if (row >= S.N * a.group) return;
  const int64_t pf = attn_partial_floats(RB);
  const float *base = a.part + ((int64_t)S.part0 + ((int64_t)kvh * S.nrb + rb) * S.nch) * pf;
  float M = -INFINITY, l = 0.f, o[CPT];
#pragma unroll
  for (int e = 0; e < CPT; ++e) o[e] = 0.f;
  // The loads of G chunks are issued together (one memory latency per G
  // chunks), then the chunks are merged in order.
  constexpr int G = 4;
  for (int c0 = 0; c0 < S.nch; c0 += G) {
    uint4 v[G][CPT / 8];
    float mc[G], lc[G];
#pragma unroll
    for (int gi = 0; gi < G; ++gi) {
      const int c = min(c0 + gi, S.nch - 1);   // past the last chunk: a repeated load, not merged
      const float *sl = base + c * pf;
      mc[gi] = sl[(int64_t)RB * D / 2 + r];
      lc[gi] = sl[(int64_t)RB * D / 2 + RB + r];
      const uint4 *po = reinterpret_cast<const uint4 *>(reinterpret_cast<const uint16_t *>(sl) + (int64_t)r * D + quarter * CPT);
#pragma unroll
      for (int q = 0; q < CPT / 8; ++q) v[gi][q] = po[q];
    }
#pragma unroll
    for (int gi = 0; gi < G; ++gi) {
      if (c0 + gi >= S.nch) break;
      // A chunk whose keys a row cannot see (only pad tokens) has mc = -inf and
      // weight 0; the last chunk holds the row's own tree row, so M ends finite.
      const float Mn = fmaxf(M, mc[gi]);
      const float wa = M == -INFINITY ? 0.f : fast_exp2(M - Mn);
      const float wb = mc[gi] == -INFINITY ? 0.f : fast_exp2(mc[gi] - Mn);
      l = l * wa + lc[gi] * wb;
#pragma unroll
      for (int q = 0; q < CPT / 8; ++q) {
        const uint32_t wv[4] = {v[gi][q].x, v[gi][q].y, v[gi][q].z, v[gi][q].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          o[8 * q + 2 * e] = o[8 * q + 2 * e] * wa + wb * __uint_as_float(wv[e] << 16);
          o[8 * q + 2 * e + 1] = o[8 * q + 2 * e + 1] * wa + wb * __uint_as_float(wv[e] & 0xFFFF0000u);
        }
      }
      M = Mn;
    }
  }
  const float inv = 1.f / l;
  const int node = row / a.group, hq = kvh * a.group + row % a.group;
  uint4 *op = reinterpret_cast<uint4 *>(static_cast<uint16_t *>(a.out) + ((int64_t)(S.node0 + node) * a.n_q + hq) * D +
                                        quarter * CPT);
#pragma unroll
  for (int q = 0; q < CPT / 8; ++q)
    op[q] = uint4{pack_bf16x2(o[8 * q] * inv, o[8 * q + 1] * inv), pack_bf16x2(o[8 * q + 2] * inv, o[8 * q + 3] * inv),
                  pack_bf16x2(o[8 * q + 4] * inv, o[8 * q + 5] * inv), pack_bf16x2(o[8 * q + 6] * inv, o[8 * q + 7] * inv)};
}

// fp32 path: one wave per (node, query head); lanes own head-dimension elements
// and walk the key set in order (the committed keys in batches of sixteen).
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
  auto dot = [&](float k0, float k1) {
    float p = q0 * k0 + q1 * k1;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) p += __shfl_xor(p, off);
    return p;
  };
  auto update = [&](float p, float v0, float v1) {   // online softmax, one key
    const float s = p * a.scale;
    const float mn = fmaxf(m, s);
    const float alpha = expf(m - mn), pe = expf(s - mn);
    l = l * alpha + pe;
    o0 = o0 * alpha + pe * v0;
    o1 = o1 * alpha + pe * v1;
    m = mn;
  };
  // Committed keys sixteen at a time: the batch's row loads are issued
  // together and its reductions are independent; the batch then moves the
  // running max once and adds its weights.  Pad tokens (padded batching) are
  // skipped: weight 0.
  constexpr int KB = 16;
  for (int t0 = 0; t0 < S.L; t0 += KB) {
    float k0[KB], k1[KB], v0[KB], v1[KB], pp[KB];
    bool use[KB];
#pragma unroll
    for (int u = 0; u < KB; ++u) {
      const int t = min(t0 + u, S.L - 1);
      const int64_t r = S.base + t;
      use[u] = t0 + u < S.L && (!a.key_valid || ((a.key_valid[r >> 5] >> (r & 31)) & 1u));
      k0[u] = e0 ? K[(int64_t)t * d + lane] : 0.f;
      k1[u] = e1 ? K[(int64_t)t * d + lane + 64] : 0.f;
      v0[u] = e0 ? V[(int64_t)t * d + lane] : 0.f;
      v1[u] = e1 ? V[(int64_t)t * d + lane + 64] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < KB; ++u) pp[u] = dot(k0[u], k1[u]);
    float mb = m;
#pragma unroll
    for (int u = 0; u < KB; ++u)
      if (use[u]) mb = fmaxf(mb, pp[u] * a.scale);
    if (mb > m) {   // m = -inf on the first visible key: alpha = 0
      const float alpha = expf(m - mb);
      l *= alpha;
      o0 *= alpha;
      o1 *= alpha;
      m = mb;
    }
#pragma unroll
    for (int u = 0; u < KB; ++u)
      if (use[u]) {
        const float pe = expf(pp[u] * a.scale - m);
        l += pe;
        o0 = fmaf(pe, v0[u], o0);
        o1 = fmaf(pe, v1[u], o1);
      }
  }
  for (int u = n; u >= 0; u = a.parent[S.node0 + u]) {   // the node's tree rows: its root path
    const int64_t row = S.L + u;
    const float p = dot(e0 ? K[row * d + lane] : 0.f, e1 ? K[row * d + lane + 64] : 0.f);
    update(p, e0 ? V[row * d + lane] : 0.f, e1 ? V[row * d + lane + 64] : 0.f);
  }
  float *out = static_cast<float *>(a.out) + ((int64_t)gnode * a.n_q + hq) * d;
  if (e0) out[lane] = o0 / l;
  if (e1) out[lane + 64] = o1 / l;
}

}  // namespace

namespace {
template <bool PAD>
void launch_bf16(const AttnArgs &a, int rows_per_block, hipStream_t st) {
  if (rows_per_block == 64) {
    hipLaunchKernelGGL((tree_attn_bf16<4, 2, 2, PAD, 2>), dim3(a.items), dim3(256), 0, st, a);
    if (a.citems) hipLaunchKernelGGL(tree_attn_combine<64>, dim3(a.citems), dim3(256), 0, st, a);
  } else if (rows_per_block == 128) {
    hipLaunchKernelGGL((tree_attn_bf16<4, 2, 2, PAD, 1>), dim3(a.items), dim3(256), 0, st, a);
    if (a.citems) hipLaunchKernelGGL(tree_attn_combine<128>, dim3(a.citems), dim3(512), 0, st, a);
  } else {
    hipLaunchKernelGGL((tree_attn_bf16<8, 3, 1, PAD, 1>), dim3(a.items), dim3(512), 0, st, a);
    if (a.citems) hipLaunchKernelGGL(tree_attn_combine<256>, dim3(a.citems), dim3(1024), 0, st, a);
  }
}
}  // namespace

hipError_t launch_tree_attn_bf16(const AttnArgs &a, int rows_per_block, hipStream_t st) {
  if (a.key_valid)
    launch_bf16<true>(a, rows_per_block, st);
  else
    launch_bf16<false>(a, rows_per_block, st);
  return hipGetLastError();
}

// Scratch of the allocation-free entry point (specmemo_tree_attn_noalloc): the
// split-KV partial results live in this file-scope device array, of which each
// device holds its own copy from module load until the process ends.  Host
// code never uses the array's name as an address: it takes the device address
// that hipGetSymbolAddress returns, once per device with that device current.
static __device__ __align__(256) uint8_t scratch[kAttnStaticScratchBytes];

hipError_t attn_static_scratch(void **ptr) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void *addr[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return hipSuccess;
}

hipError_t launch_tree_attn_f32(const AttnArgs &a, int node_begin, int node_count, hipStream_t st) {
  const int waves = node_count * a.n_q;
  hipLaunchKernelGGL(tree_attn_f32, dim3((waves + 3) / 4), dim3(256), 0, st, a, node_begin, node_count);
  return hipGetLastError();
}

}  // namespace specmemo
