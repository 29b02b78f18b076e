// C ABI of libspecmemo: argument, tree and budget validation on the host, launch
// planning, and the four stage entry points declared in include/specmemo.h.
//
// Every check runs before the first HIP call, so a rejected call enqueues
// nothing and changes no output; error paths need no GPU.
#include "specmemo.h"

#include <algorithm>
#include <cstdarg>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <numeric>
#include <string>
#include <vector>

#include "internal.h"

using namespace specmemo;

static_assert(kAttnStaticScratchBytes == SPECMEMO_ATTN_STATIC_SCRATCH_BYTES, "static scratch size of the ABI");

namespace {
thread_local std::string g_err;
}  // namespace

int specmemo::fail(int code, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int specmemo::ok() {
  g_err.clear();
  return SPECMEMO_OK;
}

namespace {

bool al(const void *p, uintptr_t a) { return p != nullptr && (reinterpret_cast<uintptr_t>(p) % a) == 0; }

struct TreeInfo {
  int B = 0, total = 0, max_nodes = 0, max_depth = 0;
};

// Tree conventions of include/specmemo.h; n_heads/topk_h (optional) add the
// head-count and rank < top-k constraints of the projection stage.
int check_trees(const specmemo_trees *t, TreeInfo *ti, int n_heads = -1, const int32_t *topk_h = nullptr) {
  if (!t) return fail(SPECMEMO_E_ARG, "trees is NULL");
  if (t->B < 1 || t->B > SPECMEMO_MAX_BATCH) return fail(SPECMEMO_E_ARG, "B=%d outside [1, %d]", t->B, SPECMEMO_MAX_BATCH);
  if (!al(t->node_off, 4) || !al(t->parent, 4) || !al(t->depth, 4) || !al(t->rank, 4))
    return fail(SPECMEMO_E_ARG, "device tree arrays must be non-NULL and 4-byte aligned");
  if (!t->node_off_h || !t->parent_h || !t->depth_h || !t->rank_h)
    return fail(SPECMEMO_E_ARG, "host tree mirrors must be non-NULL");
  const int32_t *off = t->node_off_h, *par = t->parent_h, *dep = t->depth_h, *rk = t->rank_h;
  if (off[0] != 0) return fail(SPECMEMO_E_TREE, "node_off[0]=%d, expected 0", off[0]);
  TreeInfo r;
  r.B = t->B;
  for (int b = 0; b < t->B; ++b) {
    const int N = off[b + 1] - off[b];
    if (N < 1 || N > SPECMEMO_MAX_TREE_NODES)
      return fail(SPECMEMO_E_TREE, "sequence %d has %d tree nodes, expected 1..%d", b, N, SPECMEMO_MAX_TREE_NODES);
    const int o = off[b];
    if (par[o] != -1 || dep[o] != 0 || rk[o] != 0)
      return fail(SPECMEMO_E_TREE, "sequence %d: root must have parent -1, depth 0, rank 0", b);
    uint32_t used[SPECMEMO_MAX_TREE_NODES] = {0};
    for (int n = 1; n < N; ++n) {
      const int p = par[o + n], d = dep[o + n], k = rk[o + n];
      if (p < 0 || p >= n) return fail(SPECMEMO_E_TREE, "sequence %d node %d: parent %d not in [0, %d)", b, n, p, n);
      if (d != dep[o + p] + 1) return fail(SPECMEMO_E_TREE, "sequence %d node %d: depth %d != parent depth + 1", b, n, d);
      if (d > SPECMEMO_MAX_DEPTH) return fail(SPECMEMO_E_TREE, "sequence %d node %d: depth %d > %d", b, n, d, SPECMEMO_MAX_DEPTH);
      if (n_heads > 0 && d > n_heads)
        return fail(SPECMEMO_E_TREE, "sequence %d node %d: depth %d exceeds n_heads=%d", b, n, d, n_heads);
      if (k < 0 || k >= SPECMEMO_MAX_TOPK) return fail(SPECMEMO_E_TREE, "sequence %d node %d: rank %d outside [0, %d)", b, n, k, SPECMEMO_MAX_TOPK);
      if (topk_h && k >= topk_h[d - 1])
        return fail(SPECMEMO_E_TREE, "sequence %d node %d: rank %d >= top-k %d of head %d", b, n, k, topk_h[d - 1], d - 1);
      if (used[p] & (1u << k)) return fail(SPECMEMO_E_TREE, "sequence %d node %d: duplicate sibling rank %d", b, n, k);
      used[p] |= 1u << k;
      r.max_depth = std::max(r.max_depth, d);
    }
    r.max_nodes = std::max(r.max_nodes, N);
  }
  r.total = off[t->B];
  *ti = r;
  return SPECMEMO_OK;
}

int check_dtype(int dt) {
  if (dt != SPECMEMO_FP32 && dt != SPECMEMO_BF16) return fail(SPECMEMO_E_DTYPE, "unknown dtype %d", dt);
  return SPECMEMO_OK;
}

int check_kv(int dt, const specmemo_kv *kv, const TreeInfo &ti, const int32_t *node_off_h) {
  if (!kv) return fail(SPECMEMO_E_ARG, "kv is NULL");
  if (!al(kv->k, 16) || !al(kv->v, 16)) return fail(SPECMEMO_E_ARG, "kv->k / kv->v must be non-NULL and 16-byte aligned");
  if (!kv->seq_base_h || !kv->seq_cap_h || !kv->seq_len_h) return fail(SPECMEMO_E_ARG, "kv host mirrors must be non-NULL");
  if (kv->n_kv < 1) return fail(SPECMEMO_E_ARG, "n_kv=%d", kv->n_kv);
  if (kv->cap_total < 1) return fail(SPECMEMO_E_ARG, "cap_total=%lld", (long long)kv->cap_total);
  if (dt == SPECMEMO_BF16 && kv->head_dim != kAttnHeadDim)
    return fail(SPECMEMO_E_DTYPE, "bf16 path needs head_dim %d, got %d", kAttnHeadDim, kv->head_dim);
  if (dt == SPECMEMO_FP32 && (kv->head_dim < 1 || kv->head_dim > 128 || kv->head_dim % 4))
    return fail(SPECMEMO_E_DTYPE, "fp32 path needs head_dim in [4, 128], a multiple of 4; got %d", kv->head_dim);
  std::vector<std::pair<int64_t, int64_t>> slabs;
  for (int b = 0; b < ti.B; ++b) {
    const int64_t base = kv->seq_base_h[b], cap = kv->seq_cap_h[b], L = kv->seq_len_h[b];
    const int N = node_off_h[b + 1] - node_off_h[b];
    if (L < 0 || cap < 0 || base < 0) return fail(SPECMEMO_E_ARG, "sequence %d: negative base/cap/len", b);
    if (base > kv->cap_total - cap)   // base + cap > cap_total, without overflow for any base
      return fail(SPECMEMO_E_BUDGET, "sequence %d: slab [%lld, %lld) outside the pool of %lld rows", b, (long long)base,
                  (long long)(base + cap), (long long)kv->cap_total);
    if (L + N > cap)
      return fail(SPECMEMO_E_BUDGET, "sequence %d: %lld committed + %d tree rows exceed the slab budget of %lld rows", b,
                  (long long)L, N, (long long)cap);
    if (L + N > (int64_t)INT32_MAX / 2) return fail(SPECMEMO_E_ARG, "sequence %d too long", b);
    slabs.push_back({base, cap});
  }
  std::sort(slabs.begin(), slabs.end());
  for (size_t i = 1; i < slabs.size(); ++i)
    if (slabs[i - 1].first + slabs[i - 1].second > slabs[i].first)
      return fail(SPECMEMO_E_BUDGET, "slabs overlap at pool row %lld", (long long)slabs[i].first);
  return SPECMEMO_OK;
}

int hip_status(hipError_t e, const char *what) {
  if (e != hipSuccess) return fail(SPECMEMO_E_HIP, "%s: %s", what, hipGetErrorString(e));
  return ok();
}

// ---- tree attention planning ------------------------------------------------------
constexpr int kMaxSlabRows = 1 << 23;   // bf16 attention: slab bytes below 2^31
constexpr int kMinChunk = 160;      // fewest keys per chunk when splitting the KV range

// Tuning overrides (they change the work split, never the result beyond
// rounding): SPECMEMO_ATTN_CHUNK = fixed
// chunk length in keys (a multiple of 64; 0 disables splitting), SPECMEMO_ATTN_ROWS =
// query rows per work item (64, 128 or 256), SPECMEMO_ATTN_XCD = 0 to keep block order.
int env_int(const char *name, int dflt) {
  const char *v = getenv(name);
  return v && *v ? atoi(v) : dflt;
}

struct AttnPlan {
  int rb = 128;        // query rows per work item: 64, 128 or 256
  bool xcd_order = true;
  std::vector<std::vector<AttnSeq>> groups;   // sequences per launch, in launch order
  std::vector<int> items, citems;
  std::vector<std::vector<int>> xcd_cum;      // per launch: [8][nseq + 1]
  std::vector<std::vector<int>> xcd_ccum;     // per launch: [8][nseq + 1], combine blocks
  size_t ws_bytes = 0;
  // Table mode (more sequences than kernel arguments hold): one launch, the
  // descriptors and every block's item in the workspace at these offsets.
  bool table = false;
  std::vector<AttnItem> map, cmap;
  size_t map_off = 0, cmap_off = 0, part_off = 0;
};

// Compute units of the current device (256 on MI355X; also the fallback when no
// device is visible, so that workspace sizes can be planned on a host).
int device_cus() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) {
    (void)hipGetLastError();
    return 256;
  }
  return n;
}

// Chunks per sequence for one launch (sets s.nch and s.ch_len).  A work item
// of sequence s covers about (L + N) / nch keys.  When the unsplit items fit
// in one round of resident blocks, chunks are added greedily to the sequence
// with the largest items while the round still holds them (this minimises the
// largest item); otherwise sequences are split down to the average work of one
// block slot.  Chunks hold at least kMinChunk committed keys, and the last
// chunk of a sequence also takes its tree rows.
void attn_chunks(std::vector<AttnSeq> &grp, int n_kv, int slots) {
  static const int fixed_chunk = env_int("SPECMEMO_ATTN_CHUNK", -1);
  std::vector<int> nch(grp.size(), 1);
  auto max_nch = [&](const AttnSeq &s) { return std::max(1, s.L / kMinChunk); };
  if (fixed_chunk > 0) {
    const int c = std::max(kAttnKeyTile, fixed_chunk / kAttnKeyTile * kAttnKeyTile);
    for (size_t i = 0; i < grp.size(); ++i) nch[i] = grp[i].L <= c ? 1 : (grp[i].L + c - 1) / c;
  } else if (fixed_chunk < 0) {
    int64_t items = 0, work = 0;
    for (const AttnSeq &s : grp) {
      items += (int64_t)n_kv * s.nrb;
      work += (int64_t)n_kv * s.nrb * (s.L + s.N);
    }
    if (items <= slots) {
      for (;;) {
        int best = -1;
        double big = 0;
        for (size_t i = 0; i < grp.size(); ++i) {
          const double size = (double)(grp[i].L + grp[i].N) / nch[i];
          if (size > big) big = size, best = (int)i;
        }
        if (best < 0 || nch[best] >= max_nch(grp[best]) || items + (int64_t)n_kv * grp[best].nrb > slots) break;
        items += (int64_t)n_kv * grp[best].nrb;
        ++nch[best];
      }
    } else {
      const int64_t target = std::max<int64_t>(kMinChunk, (work + slots - 1) / slots);
      for (size_t i = 0; i < grp.size(); ++i)
        nch[i] = (int)std::min<int64_t>(max_nch(grp[i]), (grp[i].L + grp[i].N + target - 1) / target);
    }
  }
  for (size_t i = 0; i < grp.size(); ++i) {
    AttnSeq &s = grp[i];
    if (nch[i] <= 1) {
      s.nch = 1;
      s.ch_len = s.L + s.N;
      continue;
    }
    // equal chunks of whole key tiles; the count may drop by rounding
    const int c = ((s.L + nch[i] - 1) / nch[i] + kAttnKeyTile - 1) / kAttnKeyTile * kAttnKeyTile;
    s.nch = (s.L + c - 1) / c;
    s.ch_len = s.nch == 1 ? s.L + s.N : c;
  }
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Table mode: the item of every attention and combine block, decoded on the
// host in the order the kernels' own decoding uses (XCD order: block 8 k + x
// is the k-th block of XCD x; otherwise launch order), padding blocks marked
// with sequence 0xFFFF.
void attn_table_maps(const std::vector<AttnSeq> &grp, const std::vector<int> &cum, const std::vector<int> &ccum,
                     bool xcd_order, int items, int citems, std::vector<AttnItem> *map, std::vector<AttnItem> *cmap) {
  const int ns = (int)grp.size();
  // largest s with c[x][s] <= k (c non-decreasing in s)
  auto last_le = [&](const std::vector<int> &c, int x, int k) {
    int s = 0;
    for (int lo = 0, hi = ns - 1; lo <= hi;) {
      const int mid = (lo + hi) / 2;
      if (c[x * (ns + 1) + mid] <= k) s = mid, lo = mid + 1;
      else hi = mid - 1;
    }
    return s;
  };
  const AttnItem pad{0xFFFF, 0, 0, 0};
  map->assign(items, pad);
  for (int bid = 0; bid < items; ++bid) {
    int s, kvh, ch, rb;
    if (xcd_order) {
      const int x = bid & 7, k = bid >> 3;
      if (k >= cum[x * (ns + 1) + ns]) continue;
      s = last_le(cum, x, k);
      const AttnSeq &S = grp[s];
      const int kk = k - cum[x * (ns + 1) + s], per_unit = S.nch * S.nrb;
      kvh = ((x - (S.unit0 & 7)) & 7) + 8 * (kk / per_unit);
      const int local = kk % per_unit;
      ch = local / S.nrb;
      rb = local % S.nrb;
    } else {
      s = 0;
      while (s + 1 < ns && grp[s + 1].item0 <= bid) ++s;
      const AttnSeq &S = grp[s];
      int local = bid - S.item0;
      rb = local % S.nrb;
      local /= S.nrb;
      ch = local % S.nch;
      kvh = local / S.nch;
    }
    (*map)[bid] = AttnItem{(uint16_t)s, (uint16_t)kvh, (uint16_t)ch, (uint16_t)rb};
  }
  cmap->assign(citems, pad);
  for (int idx = 0; idx < citems; ++idx) {
    int s, kvh, rb;
    if (xcd_order) {
      const int x = idx & 7, k = idx >> 3;
      if (k >= ccum[x * (ns + 1) + ns]) continue;
      s = last_le(ccum, x, k);
      const AttnSeq &S = grp[s];
      const int kk = k - ccum[x * (ns + 1) + s];
      kvh = ((x - (S.unit0 & 7)) & 7) + 8 * (kk / S.nrb);
      rb = kk % S.nrb;
    } else {
      s = -1;
      for (int i = 0; i < ns; ++i)
        if (grp[i].nch > 1 && grp[i].citem0 <= idx) s = i;
      if (s < 0) continue;
      const AttnSeq &S = grp[s];
      const int local = idx - S.citem0;
      kvh = local / S.nrb;
      rb = local % S.nrb;
    }
    (*cmap)[idx] = AttnItem{(uint16_t)s, (uint16_t)kvh, 0, (uint16_t)rb};
  }
}

void plan_attn(const TreeInfo &ti, const specmemo_trees *t, const specmemo_kv *kv, int n_q, AttnPlan *p) {
  const int g = n_q / kv->n_kv;
  const int max_rows = ti.max_nodes * g;
  static const int rows_env = env_int("SPECMEMO_ATTN_ROWS", 0);
  static const int xcd_env = env_int("SPECMEMO_ATTN_XCD", 1);
  p->rb = max_rows <= 64 ? 64 : 128;
  if (rows_env == 64 || rows_env == 128 || rows_env == 256) p->rb = rows_env;
  p->xcd_order = xcd_env != 0;
  const int RB = p->rb;
  const int slots = device_cus() * (RB == 256 ? 1 : 2);   // resident blocks of the launch
  std::vector<int> order(ti.B);
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int x, int y) { return kv->seq_len_h[x] > kv->seq_len_h[y]; });
  const int64_t pf = attn_partial_floats(RB);
  p->table = ti.B > kMaxSeqPerLaunch;
  const size_t per_launch = p->table ? order.size() : (size_t)kMaxSeqPerLaunch;
  for (size_t i0 = 0; i0 < order.size(); i0 += per_launch) {
    std::vector<AttnSeq> grp;
    for (size_t i = i0; i < std::min(order.size(), i0 + per_launch); ++i) {
      const int b = order[i];
      AttnSeq s{};
      s.base = kv->seq_base_h[b];
      s.L = kv->seq_len_h[b];
      s.node0 = t->node_off_h[b];
      s.N = t->node_off_h[b + 1] - s.node0;
      s.nrb = (s.N * g + RB - 1) / RB;
      grp.push_back(s);
    }
    attn_chunks(grp, kv->n_kv, slots);
    // largest items first (the dispatch order of the launch)
    std::stable_sort(grp.begin(), grp.end(), [](const AttnSeq &x, const AttnSeq &y) {
      return (int64_t)(x.L + x.N) * y.nch > (int64_t)(y.L + y.N) * x.nch;
    });
    int item = 0, part = 0, citem = 0, unit = 0;
    int per_xcd[8] = {0, 0, 0, 0, 0, 0, 0, 0}, cper_xcd[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    const size_t ns = grp.size();
    std::vector<int> cum(8 * (ns + 1), 0), ccum(8 * (ns + 1), 0);
    for (size_t si = 0; si < ns; ++si) {
      AttnSeq &s = grp[si];
      for (int x = 0; x < 8; ++x) {
        cum[x * (ns + 1) + si] = per_xcd[x];
        ccum[x * (ns + 1) + si] = cper_xcd[x];
      }
      s.item0 = item;
      s.unit0 = unit;
      // unit (sequence, KV head) = all its chunks and row blocks, on XCD unit mod 8
      for (int h = 0; h < kv->n_kv; ++h) {
        per_xcd[(unit + h) & 7] += s.nch * s.nrb;
        if (s.nch > 1) cper_xcd[(unit + h) & 7] += s.nrb;
      }
      unit += kv->n_kv;
      item += kv->n_kv * s.nch * s.nrb;
      if (s.nch > 1) {
        s.part0 = part;
        part += kv->n_kv * s.nch * s.nrb;
        s.citem0 = citem;
        citem += kv->n_kv * s.nrb;
      } else {
        s.part0 = -1;
        s.citem0 = -1;
      }
    }
    for (int x = 0; x < 8; ++x) {
      cum[x * (ns + 1) + ns] = per_xcd[x];
      ccum[x * (ns + 1) + ns] = cper_xcd[x];
    }
    p->xcd_cum.push_back(cum);
    p->xcd_ccum.push_back(ccum);
    p->groups.push_back(grp);
    // XCD order: XCD x runs the units x, x + 8, ... with all their chunks and
    // row blocks, and merges their chunks; each grid is padded to 8 x the
    // busiest XCD's blocks, surplus blocks exit at once.
    p->items.push_back(p->xcd_order ? 8 * *std::max_element(per_xcd, per_xcd + 8) : item);
    p->citems.push_back(p->xcd_order ? 8 * *std::max_element(cper_xcd, cper_xcd + 8) : citem);
    if (p->table) {
      attn_table_maps(grp, cum, ccum, p->xcd_order, p->items.back(), p->citems.back(), &p->map, &p->cmap);
      p->map_off = align256(grp.size() * sizeof(AttnSeq));
      p->cmap_off = p->map_off + align256(p->map.size() * sizeof(AttnItem));
      p->part_off = p->cmap_off + align256(p->cmap.size() * sizeof(AttnItem));
    }
    p->ws_bytes = std::max(p->ws_bytes, p->part_off + (size_t)part * (size_t)pf * sizeof(float));
  }
}

// Workspace of the acceptance: greedy one int32 per node; typical two floats
// and one int32 per node (aligned to 256 bytes for what follows it).
size_t accept_ws_bytes(const TreeInfo &ti, int mode) {
  return align256(mode == SPECMEMO_ACCEPT_TYPICAL ? (size_t)ti.total * (2 * sizeof(float) + sizeof(int32_t))
                                                  : (size_t)ti.total * sizeof(int32_t));
}
// The fused acceptance and compaction of more than kMaxSeqPerLaunch
// sequences keeps their compaction descriptors after the acceptance's part.
// Sampled next token: one 64-bit word per (sequence, 1024-token segment).
size_t sample_ws_bytes(int B, int vocab) { return align256((size_t)B * sample_segments(vocab) * sizeof(uint64_t)); }
size_t compact_table_bytes(int B) { return B > kMaxSeqPerLaunch ? align256((size_t)B * sizeof(CompactSeq)) : 0; }

// Validation and kernel arguments of the acceptance (nothing is launched).
int accept_args(specmemo_dtype dt, const specmemo_trees *t, int32_t vocab, specmemo_accept_mode mode, float temperature,
                float eps, float delta, const void *base_logits, const int32_t *node_tok, int32_t *accept_len,
                int32_t *path, int32_t path_stride, int32_t *next_tok, void *ws, size_t ws_bytes, TreeInfo *ti,
                AcceptArgs *out) {
  int rc;
  if ((rc = check_dtype(dt))) return rc;
  if ((rc = check_trees(t, ti))) return rc;
  if (vocab < 1) return fail(SPECMEMO_E_ARG, "vocab=%d", vocab);
  if (mode != SPECMEMO_ACCEPT_GREEDY && mode != SPECMEMO_ACCEPT_TYPICAL) return fail(SPECMEMO_E_ARG, "unknown mode %d", mode);
  if (path_stride < ti->max_depth + 1) return fail(SPECMEMO_E_ARG, "path_stride=%d < max depth + 1 = %d", path_stride, ti->max_depth + 1);
  if (!al(base_logits, 16)) return fail(SPECMEMO_E_ARG, "base_logits must be non-NULL and 16-byte aligned");
  if (!al(node_tok, 4) || !al(accept_len, 4) || !al(path, 4) || !al(next_tok, 4))
    return fail(SPECMEMO_E_ARG, "node_tok / accept_len / path / next_tok must be non-NULL and 4-byte aligned");
  AcceptArgs &a = *out;
  a = AcceptArgs{};
  a.logits = base_logits;
  a.node_tok = node_tok;
  a.node_off = t->node_off;
  a.parent = t->parent;
  a.depth = t->depth;
  a.vocab = vocab;
  a.mode = mode;
  a.path_stride = path_stride;
  a.B = ti->B;
  a.accept_len = accept_len;
  a.path = path;
  a.next_tok = next_tok;
  if (mode == SPECMEMO_ACCEPT_TYPICAL) {
    if (!(temperature > 0.f) || !(eps > 0.f) || !(delta > 0.f) || !std::isfinite(temperature))
      return fail(SPECMEMO_E_ARG, "typical mode needs temperature, eps, delta > 0");
    const size_t need = (size_t)ti->total * (2 * sizeof(float) + sizeof(int32_t));
    if (!al(ws, 16) || ws_bytes < need)
      return fail(SPECMEMO_E_WORKSPACE, "workspace of %zu bytes needed (16-byte aligned), got %zu", need, ws ? ws_bytes : 0);
    a.stats = static_cast<float *>(ws);
    a.best = reinterpret_cast<int32_t *>(a.stats + 2 * (size_t)ti->total);
    a.inv_temp = 1.0f / temperature;
    a.log_eps = std::log(eps);
    a.log_delta = std::log(delta);
  } else {
    const size_t need = (size_t)ti->total * sizeof(int32_t);
    if (!al(ws, 16) || ws_bytes < need)
      return fail(SPECMEMO_E_WORKSPACE, "workspace of %zu bytes needed (16-byte aligned), got %zu", need, ws ? ws_bytes : 0);
    a.best = static_cast<int32_t *>(ws);
  }
  return SPECMEMO_OK;
}

// Top-k workspace: the fp32 logits (unless the caller keeps them), then, for
// packed bf16 heads, the maxima of the 64-row groups (the top-k pass reads
// only the groups that can hold a top-k value).
size_t topk_logit_bytes(int B, int n_heads, int vocab) { return align256((size_t)B * n_heads * vocab * sizeof(float)); }
size_t topk_gmax_bytes(int B, int n_heads, int vocab) {
  return align256((size_t)B * n_heads * packed_row_groups(vocab) * sizeof(float));
}

int check_attn_args(int dt, const specmemo_trees *t, const specmemo_kv *kv, int n_q, TreeInfo *ti) {
  int rc;
  if ((rc = check_dtype(dt))) return rc;
  if ((rc = check_trees(t, ti))) return rc;
  if ((rc = check_kv(dt, kv, *ti, t->node_off_h))) return rc;
  if (n_q < 1 || n_q % kv->n_kv) return fail(SPECMEMO_E_ARG, "n_q=%d must be a positive multiple of n_kv=%d", n_q, kv->n_kv);
  if (dt == SPECMEMO_BF16)
    for (int b = 0; b < ti->B; ++b)    // tile loads address a slab with 32-bit byte offsets
      if (kv->seq_cap_h[b] > kMaxSlabRows)
        return fail(SPECMEMO_E_BUDGET, "seq_cap[%d]=%d exceeds %d rows", b, kv->seq_cap_h[b], kMaxSlabRows);
  return SPECMEMO_OK;
}

}  // namespace

extern "C" {

int32_t specmemo_abi_version(void) { return SPECMEMO_ABI_VERSION; }

const char *specmemo_last_error(void) { return g_err.c_str(); }

size_t specmemo_workspace_bytes(int32_t which, specmemo_dtype dt, const specmemo_trees *t, const specmemo_kv *kv,
                                int32_t n_q_or_heads, int32_t vocab) {
  TreeInfo ti;
  if (check_dtype(dt) || check_trees(t, &ti)) return 0;
  if (which == SPECMEMO_WS_TOPK) {
    if (n_q_or_heads < 1 || vocab < 1) return 0;
    return topk_logit_bytes(ti.B, n_q_or_heads, vocab) +
           (dt == SPECMEMO_BF16 ? topk_gmax_bytes(ti.B, n_q_or_heads, vocab) : 0);
  }
  if (which == SPECMEMO_WS_ATTN) {
    if (check_attn_args(dt, t, kv, n_q_or_heads, &ti)) return 0;
    if (dt == SPECMEMO_FP32) return 0;
    AttnPlan p;
    plan_attn(ti, t, kv, n_q_or_heads, &p);
    return p.ws_bytes;
  }
  if (which == SPECMEMO_WS_PAD) return 256;   // the batch's uniform acceptance length
  if (which == SPECMEMO_WS_SAMPLE) return vocab < 1 ? 0 : sample_ws_bytes(ti.B, vocab);
  if (which == SPECMEMO_WS_ACCEPT) return accept_ws_bytes(ti, n_q_or_heads) + compact_table_bytes(ti.B);
  return 0;
}

size_t specmemo_packed_heads_bytes(specmemo_dtype dt, int32_t n_heads, int32_t vocab, int32_t hidden) {
  if (dt != SPECMEMO_BF16 || n_heads < 1 || vocab < 1 || hidden < 8 || hidden % 8) return 0;
  return (size_t)n_heads * packed_row_groups(vocab) * packed_k_steps(hidden) * 4 * 1024;
}

int specmemo_pack_heads(specmemo_dtype dt, int32_t n_heads, int32_t vocab, int32_t hidden, const void *src, void *dst,
                        void *stream) {
  int rc;
  if ((rc = check_dtype(dt))) return rc;
  if (dt != SPECMEMO_BF16) return fail(SPECMEMO_E_DTYPE, "packed heads are bf16 only");
  if (n_heads < 1 || vocab < 1) return fail(SPECMEMO_E_ARG, "n_heads=%d vocab=%d", n_heads, vocab);
  if (hidden < 8 || hidden % 8) return fail(SPECMEMO_E_ARG, "hidden=%d must be a positive multiple of 8", hidden);
  if (!al(src, 16) || !al(dst, 16)) return fail(SPECMEMO_E_ARG, "src / dst must be non-NULL and 16-byte aligned");
  const size_t nb = specmemo_packed_heads_bytes(dt, n_heads, vocab, hidden);
  const size_t sb = (size_t)n_heads * vocab * hidden * 2;
  const uintptr_t s0 = (uintptr_t)src, d0 = (uintptr_t)dst;
  if (s0 < d0 + nb && d0 < s0 + sb) return fail(SPECMEMO_E_ARG, "dst overlaps src");
  return hip_status(launch_pack_heads(src, dst, n_heads, vocab, hidden, static_cast<hipStream_t>(stream)),
                    "head packing launch");
}

int specmemo_medusa_topk(specmemo_dtype dt, const specmemo_trees *t, int32_t hidden, int32_t vocab, int32_t n_heads,
                         const int32_t *topk_h, const void *h, const void *head_w, int32_t head_layout,
                         const int32_t *root_tok, float *logits_out, int32_t *topk_ids, float *topk_vals,
                         int32_t *node_tok, void *ws, size_t ws_bytes, void *stream) {
  int rc;
  if ((rc = check_dtype(dt))) return rc;
  const bool per_head_input = head_layout & SPECMEMO_HEADS_INPUT_PER_HEAD;
  head_layout &= ~SPECMEMO_HEADS_INPUT_PER_HEAD;
  if (head_layout != SPECMEMO_HEADS_ROWMAJOR && head_layout != SPECMEMO_HEADS_PACKED)
    return fail(SPECMEMO_E_ARG, "unknown head_layout %d", head_layout);
  if (head_layout == SPECMEMO_HEADS_PACKED && dt != SPECMEMO_BF16)
    return fail(SPECMEMO_E_DTYPE, "packed heads are bf16 only");
  if (n_heads < 1 || n_heads > SPECMEMO_MAX_DEPTH) return fail(SPECMEMO_E_ARG, "n_heads=%d outside [1, %d]", n_heads, SPECMEMO_MAX_DEPTH);
  if (!topk_h) return fail(SPECMEMO_E_ARG, "topk_h is NULL");
  if (vocab < 1) return fail(SPECMEMO_E_ARG, "vocab=%d", vocab);
  if (hidden < 8 || hidden % 8) return fail(SPECMEMO_E_ARG, "hidden=%d must be a positive multiple of 8", hidden);
  int kmax = 0;
  for (int i = 0; i < n_heads; ++i) {
    if (topk_h[i] < 1 || topk_h[i] > SPECMEMO_MAX_TOPK || topk_h[i] > vocab)
      return fail(SPECMEMO_E_ARG, "topk[%d]=%d outside [1, min(%d, vocab)]", i, topk_h[i], SPECMEMO_MAX_TOPK);
    kmax = std::max(kmax, (int)topk_h[i]);
  }
  TreeInfo ti;
  if ((rc = check_trees(t, &ti, n_heads, topk_h))) return rc;
  if (!al(h, 16) || !al(head_w, 16)) return fail(SPECMEMO_E_ARG, "h / head_w must be non-NULL and 16-byte aligned");
  if (!al(root_tok, 4) || !al(topk_ids, 4) || !al(node_tok, 4))
    return fail(SPECMEMO_E_ARG, "root_tok / topk_ids / node_tok must be non-NULL and 4-byte aligned");
  if (logits_out && !al(logits_out, 16)) return fail(SPECMEMO_E_ARG, "logits_out must be 16-byte aligned");
  if (topk_vals && !al(topk_vals, 4)) return fail(SPECMEMO_E_ARG, "topk_vals must be 4-byte aligned");
  const size_t need = logits_out ? 0 : topk_logit_bytes(ti.B, n_heads, vocab);
  if (need && (!al(ws, 16) || ws_bytes < need))
    return fail(SPECMEMO_E_WORKSPACE, "workspace of %zu bytes needed (16-byte aligned), got %zu", need, ws ? ws_bytes : 0);
  float *z = logits_out ? logits_out : static_cast<float *>(ws);
  // the group maxima, where the workspace holds them (else every logit is scanned)
  float *gmax = nullptr;
  if (head_layout == SPECMEMO_HEADS_PACKED && ws && al(ws, 16) && ws_bytes >= need + topk_gmax_bytes(ti.B, n_heads, vocab))
    gmax = reinterpret_cast<float *>(static_cast<uint8_t *>(ws) + need);
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int64_t h_head_stride = per_head_input ? (int64_t)ti.B * hidden : 0;
  hipError_t e = launch_head_logits(dt, h, h_head_stride, head_w, head_layout == SPECMEMO_HEADS_PACKED, z, ti.B,
                                    hidden, vocab, n_heads, st, gmax);
  if (e != hipSuccess) return hip_status(e, "head projection launch");
  TopkArgs a{};
  a.z = z;
  a.gmax = gmax;
  a.nG = packed_row_groups(vocab);
  a.vocab = vocab;
  a.n_heads = n_heads;
  a.kmax = kmax;
  for (int i = 0; i < n_heads; ++i) a.k[i] = topk_h[i];
  a.node_off = t->node_off;
  a.depth = t->depth;
  a.rank = t->rank;
  a.root_tok = root_tok;
  a.ids = topk_ids;
  a.vals = topk_vals;
  a.node_tok = node_tok;
  return hip_status(launch_topk(a, ti.B, st), "top-k launch");
}

int specmemo_head_logits(specmemo_dtype dt, int32_t B, int32_t hidden, int32_t vocab, int32_t n_heads, const void *h,
                         const void *head_w, int32_t head_layout, float *logits_out, void *stream) {
  int rc;
  if ((rc = check_dtype(dt))) return rc;
  const bool per_head_input = head_layout & SPECMEMO_HEADS_INPUT_PER_HEAD;
  head_layout &= ~SPECMEMO_HEADS_INPUT_PER_HEAD;
  if (head_layout != SPECMEMO_HEADS_ROWMAJOR && head_layout != SPECMEMO_HEADS_PACKED)
    return fail(SPECMEMO_E_ARG, "unknown head_layout %d", head_layout);
  if (head_layout == SPECMEMO_HEADS_PACKED && dt != SPECMEMO_BF16)
    return fail(SPECMEMO_E_DTYPE, "packed heads are bf16 only");
  if (B < 1 || B > SPECMEMO_MAX_BATCH) return fail(SPECMEMO_E_ARG, "B=%d outside [1, %d]", B, SPECMEMO_MAX_BATCH);
  if (n_heads < 1 || n_heads > SPECMEMO_MAX_DEPTH) return fail(SPECMEMO_E_ARG, "n_heads=%d outside [1, %d]", n_heads, SPECMEMO_MAX_DEPTH);
  if (vocab < 1) return fail(SPECMEMO_E_ARG, "vocab=%d", vocab);
  if (hidden < 8 || hidden % 8) return fail(SPECMEMO_E_ARG, "hidden=%d must be a positive multiple of 8", hidden);
  if (!al(h, 16) || !al(head_w, 16) || !al(logits_out, 16))
    return fail(SPECMEMO_E_ARG, "h / head_w / logits_out must be non-NULL and 16-byte aligned");
  const int64_t h_head_stride = per_head_input ? (int64_t)B * hidden : 0;
  return hip_status(launch_head_logits(dt, h, h_head_stride, head_w, head_layout == SPECMEMO_HEADS_PACKED, logits_out,
                                       B, hidden, vocab, n_heads, static_cast<hipStream_t>(stream)),
                    "head projection launch");
}

int specmemo_medusa_resblock(specmemo_dtype dt, int32_t B, int32_t hidden, int32_t n_heads, const void *h,
                             const void *w1, int32_t w1_layout, const void *b1, void *out, void *stream) {
  int rc;
  if ((rc = check_dtype(dt))) return rc;
  if (B < 1 || B > SPECMEMO_MAX_BATCH) return fail(SPECMEMO_E_ARG, "B=%d outside [1, %d]", B, SPECMEMO_MAX_BATCH);
  if (n_heads < 1 || n_heads > SPECMEMO_MAX_DEPTH) return fail(SPECMEMO_E_ARG, "n_heads=%d outside [1, %d]", n_heads, SPECMEMO_MAX_DEPTH);
  if (hidden < 8 || hidden % 8) return fail(SPECMEMO_E_ARG, "hidden=%d must be a positive multiple of 8", hidden);
  if (dt == SPECMEMO_BF16 && w1_layout != SPECMEMO_HEADS_PACKED)
    return fail(SPECMEMO_E_ARG, "bf16 residual-block weights must be packed (specmemo_pack_heads with vocab = hidden)");
  if (dt == SPECMEMO_FP32 && w1_layout != SPECMEMO_HEADS_ROWMAJOR)
    return fail(SPECMEMO_E_DTYPE, "fp32 residual-block weights are row-major");
  if (!al(h, 16) || !al(w1, 16) || !al(b1, 16) || !al(out, 16))
    return fail(SPECMEMO_E_ARG, "h / w1 / b1 / out must be non-NULL and 16-byte aligned");
  return hip_status(launch_resblock(dt, h, w1, b1, out, B, hidden, n_heads, static_cast<hipStream_t>(stream)),
                    "residual block launch");
}

}  // extern "C"

namespace {

// Tree attention with an optional pad-token mask (padded batching).
// static_scratch: the partials go to the library's static scratch array
// (specmemo_tree_attn_noalloc) instead of the caller's workspace.
int tree_attn_impl(specmemo_dtype dt, const specmemo_trees *t, const specmemo_kv *kv, const uint32_t *key_valid,
                   int32_t n_q, float scale, const void *q, void *out, void *ws, size_t ws_bytes, void *stream,
                   bool static_scratch = false) {
  TreeInfo ti;
  int rc;
  if ((rc = check_attn_args(dt, t, kv, n_q, &ti))) return rc;
  if (!al(q, 16) || !al(out, 16)) return fail(SPECMEMO_E_ARG, "q / out must be non-NULL and 16-byte aligned");
  if (!(scale > 0.f)) scale = 1.0f / std::sqrt((float)kv->head_dim);
  if (!std::isfinite(scale)) return fail(SPECMEMO_E_ARG, "scale is not finite");
  AttnArgs a{};
  a.q = q;
  a.out = out;
  a.k = kv->k;
  a.v = kv->v;
  a.parent = t->parent;
  a.key_valid = key_valid;
  a.cap_total = kv->cap_total;
  a.n_q = n_q;
  a.n_kv = kv->n_kv;
  a.group = n_q / kv->n_kv;
  a.head_dim = kv->head_dim;
  a.scale = scale;
  a.scale_log2 = scale * 1.4426950408889634f;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (dt == SPECMEMO_FP32) {
    for (int b0 = 0; b0 < ti.B; b0 += kMaxSeqPerLaunch) {
      const int nb = std::min(kMaxSeqPerLaunch, ti.B - b0);
      a.nseq = nb;
      for (int i = 0; i < nb; ++i) {
        const int b = b0 + i;
        AttnSeq s{};
        s.base = kv->seq_base_h[b];
        s.L = kv->seq_len_h[b];
        s.node0 = t->node_off_h[b];
        s.N = t->node_off_h[b + 1] - s.node0;
        a.seq[i] = s;
      }
      const int nbeg = t->node_off_h[b0], ncnt = t->node_off_h[b0 + nb] - nbeg;
      hipError_t e = launch_tree_attn_f32(a, nbeg, ncnt, st);
      if (e != hipSuccess) return hip_status(e, "tree attention launch");
    }
    return ok();
  }
  AttnPlan p;
  plan_attn(ti, t, kv, n_q, &p);
  if (static_scratch) {
    if (p.ws_bytes > kAttnStaticScratchBytes)
      return fail(SPECMEMO_E_WORKSPACE, "this batch needs %zu bytes of scratch; the static scratch holds %zu", p.ws_bytes,
                  kAttnStaticScratchBytes);
    hipError_t e = attn_static_scratch(&ws);
    if (e != hipSuccess) return hip_status(e, "static scratch address");
    ws_bytes = kAttnStaticScratchBytes;
  }
  if (p.ws_bytes) {
    if (!al(ws, 16) || ws_bytes < p.ws_bytes)
      return fail(SPECMEMO_E_WORKSPACE, "workspace of %zu bytes needed (16-byte aligned), got %zu", p.ws_bytes,
                  ws ? ws_bytes : 0);
  }
  a.part = static_cast<float *>(ws);
  if (p.table) {   // one launch: descriptors and block maps go to the workspace first
    uint8_t *w = static_cast<uint8_t *>(ws);
    hipError_t e = upload_table(p.groups[0].data(), p.groups[0].size() * sizeof(AttnSeq), w, st);
    if (e == hipSuccess) e = upload_table(p.map.data(), p.map.size() * sizeof(AttnItem), w + p.map_off, st);
    if (e == hipSuccess) e = upload_table(p.cmap.data(), p.cmap.size() * sizeof(AttnItem), w + p.cmap_off, st);
    if (e != hipSuccess) return hip_status(e, "descriptor upload");
    a.tab = reinterpret_cast<const AttnSeq *>(w);
    a.map = reinterpret_cast<const AttnItem *>(w + p.map_off);
    a.cmap = reinterpret_cast<const AttnItem *>(w + p.cmap_off);
    a.part = reinterpret_cast<float *>(w + p.part_off);
  }
  for (size_t gi = 0; gi < p.groups.size(); ++gi) {
    a.nseq = (int)p.groups[gi].size();
    if (!p.table)
      for (int i = 0; i < a.nseq; ++i) a.seq[i] = p.groups[gi][i];
    a.items = p.items[gi];
    a.citems = p.citems[gi];
    a.xcd_order = p.xcd_order ? 1 : 0;
    if (!p.table)
      for (int x = 0; x < 8; ++x)
        for (int i = 0; i <= a.nseq; ++i) {
          a.xcd_cum[x][i] = p.xcd_cum[gi][x * (a.nseq + 1) + i];
          a.xcd_ccum[x][i] = p.xcd_ccum[gi][x * (a.nseq + 1) + i];
        }
    hipError_t e = launch_tree_attn_bf16(a, p.rb, st);
    if (e != hipSuccess) return hip_status(e, "tree attention launch");
  }
  return ok();
}

}  // namespace

extern "C" {

int specmemo_tree_attn(specmemo_dtype dt, const specmemo_trees *t, const specmemo_kv *kv, int32_t n_q, float scale,
                       const void *q, void *out, void *ws, size_t ws_bytes, void *stream) {
  return tree_attn_impl(dt, t, kv, nullptr, n_q, scale, q, out, ws, ws_bytes, stream);
}

int specmemo_tree_attn_noalloc(specmemo_dtype dt, const specmemo_trees *t, const specmemo_kv *kv, int32_t n_q,
                               float scale, const void *q, void *out, void *stream) {
  return tree_attn_impl(dt, t, kv, nullptr, n_q, scale, q, out, nullptr, 0, stream, true);
}

int64_t specmemo_key_mask_words(int64_t cap_total) {
  if (cap_total < 1) return 0;
  return (cap_total + 31) / 32 + 3;
}

int specmemo_tree_attn_padded(specmemo_dtype dt, const specmemo_trees *t, const specmemo_kv *kv,
                              const uint32_t *key_valid, int64_t key_valid_words, int32_t n_q, float scale,
                              const void *q, void *out, void *ws, size_t ws_bytes, void *stream) {
  if (!al(key_valid, 16)) return fail(SPECMEMO_E_ARG, "key_valid must be non-NULL and 16-byte aligned");
  if (kv && key_valid_words < specmemo_key_mask_words(kv->cap_total))
    return fail(SPECMEMO_E_ARG, "key_valid holds %lld words, %lld needed", static_cast<long long>(key_valid_words),
                static_cast<long long>(specmemo_key_mask_words(kv->cap_total)));
  return tree_attn_impl(dt, t, kv, key_valid, n_q, scale, q, out, ws, ws_bytes, stream);
}

int specmemo_accept(specmemo_dtype dt, const specmemo_trees *t, int32_t vocab, specmemo_accept_mode mode,
                    float temperature, float eps, float delta, const void *base_logits, const int32_t *node_tok,
                    int32_t *accept_len, int32_t *path, int32_t path_stride, int32_t *next_tok, void *ws,
                    size_t ws_bytes, void *stream) {
  TreeInfo ti;
  AcceptArgs a;
  const int rc = accept_args(dt, t, vocab, mode, temperature, eps, delta, base_logits, node_tok, accept_len, path,
                             path_stride, next_tok, ws, ws_bytes, &ti, &a);
  if (rc) return rc;
  return hip_status(launch_accept(dt, a, ti.total, static_cast<hipStream_t>(stream)), "acceptance launch");
}

int specmemo_sample_next(specmemo_dtype dt, const specmemo_trees *t, int32_t vocab, float temperature, uint64_t seed,
                         uint64_t offset, const void *base_logits, const int32_t *accept_len, const int32_t *path,
                         int32_t path_stride, int32_t *next_tok, void *ws, size_t ws_bytes, void *stream) {
  int rc;
  if ((rc = check_dtype(dt))) return rc;
  TreeInfo ti;
  if ((rc = check_trees(t, &ti))) return rc;
  if (vocab < 1) return fail(SPECMEMO_E_ARG, "vocab=%d", vocab);
  if (!(temperature > 0.f) || !std::isfinite(temperature) || !std::isfinite(1.0f / temperature))
    return fail(SPECMEMO_E_ARG, "temperature must be positive and finite with a finite inverse");
  if (path_stride < ti.max_depth + 1) return fail(SPECMEMO_E_ARG, "path_stride=%d < max depth + 1 = %d", path_stride, ti.max_depth + 1);
  if (!al(base_logits, 16)) return fail(SPECMEMO_E_ARG, "base_logits must be non-NULL and 16-byte aligned");
  if (!al(accept_len, 4) || !al(path, 4) || !al(next_tok, 4))
    return fail(SPECMEMO_E_ARG, "accept_len / path / next_tok must be non-NULL and 4-byte aligned");
  SampleArgs a{};
  a.logits = base_logits;
  a.node_off = t->node_off;
  a.accept_len = accept_len;
  a.path = path;
  a.vocab = vocab;
  a.path_stride = path_stride;
  a.inv_temp = 1.0f / temperature;
  a.seed = seed;
  a.offset = offset;
  a.next_tok = next_tok;
  uint64_t *words = nullptr;
  if (ws) {
    const size_t need = sample_ws_bytes(ti.B, vocab);
    if (!al(ws, 16) || ws_bytes < need)
      return fail(SPECMEMO_E_WORKSPACE, "workspace of %zu bytes needed (16-byte aligned), got %zu", need, ws_bytes);
    words = static_cast<uint64_t *>(ws);
  }
  return hip_status(launch_sample_next(dt, a, ti.B, words, static_cast<hipStream_t>(stream)), "sampling launch");
}

}  // extern "C"

namespace {

// Compaction (padded = false) or the padded update (Sec. 3.3): the same
// checks and row moves, launched per group of sequences.
// Validation of the compaction's arguments and its launch-independent kernel
// arguments (nothing is launched).
int compact_args(specmemo_dtype dt, const specmemo_trees *t, const specmemo_kv *kv, const int32_t *accept_len,
                 const int32_t *path, int32_t path_stride, const TreeInfo &ti, CompactArgs *out) {
  int rc;
  if ((rc = check_kv(dt, kv, ti, t->node_off_h))) return rc;
  if (!al(kv->seq_len, 4)) return fail(SPECMEMO_E_ARG, "kv->seq_len must be non-NULL and 4-byte aligned");
  if (!al(accept_len, 4) || !al(path, 4)) return fail(SPECMEMO_E_ARG, "accept_len / path must be non-NULL and 4-byte aligned");
  if (path_stride < 1) return fail(SPECMEMO_E_ARG, "path_stride=%d", path_stride);
  const int elem = dt == SPECMEMO_BF16 ? 2 : 4;
  if ((kv->head_dim * elem) % 4) return fail(SPECMEMO_E_ARG, "row bytes must be a multiple of 4");
  CompactArgs &a = *out;
  a = CompactArgs{};
  a.k = kv->k;
  a.v = kv->v;
  a.cap_total = kv->cap_total;
  a.n_kv = kv->n_kv;
  a.row_dwords = kv->head_dim * elem / 4;
  a.path_stride = path_stride;
  a.accept_len = accept_len;
  a.path = path;
  a.parent = t->parent;
  a.seq_len = kv->seq_len;
  return SPECMEMO_OK;
}

// The per-sequence table of one launch group: sequences b0 .. b0 + nseq - 1.
void compact_group(const specmemo_trees *t, const specmemo_kv *kv, int b0, int B, CompactArgs *a) {
  a->nseq = std::min(kMaxSeqPerLaunch, B - b0);
  a->b0 = b0;
  for (int i = 0; i < a->nseq; ++i) {
    const int b = b0 + i;
    a->seq[i] = CompactSeq{kv->seq_base_h[b], kv->seq_len_h[b], t->node_off_h[b + 1] - t->node_off_h[b],
                           kv->seq_cap_h[b], t->node_off_h[b]};
  }
}

int compact_impl(specmemo_dtype dt, const specmemo_trees *t, const specmemo_kv *kv, const int32_t *accept_len,
                 const int32_t *path, int32_t path_stride, bool padded, uint32_t *key_valid, int32_t *pos, void *ws,
                 size_t ws_bytes, void *stream) {
  int rc;
  if ((rc = check_dtype(dt))) return rc;
  TreeInfo ti;
  if ((rc = check_trees(t, &ti))) return rc;
  CompactArgs a;
  if ((rc = compact_args(dt, t, kv, accept_len, path, path_stride, ti, &a))) return rc;
  if (padded) {
    if (!al(key_valid, 4) || !al(pos, 4)) return fail(SPECMEMO_E_ARG, "key_valid / pos must be non-NULL and 4-byte aligned");
    if (!al(ws, 4) || ws_bytes < 4)
      return fail(SPECMEMO_E_WORKSPACE, "workspace of 4 bytes needed (4-byte aligned), got %zu", ws ? ws_bytes : 0);
    // every sequence may grow by the batch's longest acceptance: the deepest tree + 1
    for (int b = 0; b < ti.B; ++b)
      if ((int64_t)kv->seq_len_h[b] + ti.max_depth + 1 > kv->seq_cap_h[b])
        return fail(SPECMEMO_E_BUDGET, "seq_len[%d]=%d + uniform length up to %d exceeds seq_cap=%d", b,
                    kv->seq_len_h[b], ti.max_depth + 1, kv->seq_cap_h[b]);
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  int32_t *uniform = static_cast<int32_t *>(ws);
  if (padded) {
    hipError_t e = launch_pad_length(t->node_off, t->parent, accept_len, path, path_stride, ti.B, uniform, st);
    if (e != hipSuccess) return hip_status(e, "pad length launch");
  }
  for (int b0 = 0; b0 < ti.B; b0 += kMaxSeqPerLaunch) {
    compact_group(t, kv, b0, ti.B, &a);
    hipError_t e = padded ? launch_kv_pad_update(a, uniform, key_valid, pos, st) : launch_kv_compact(a, st);
    if (e != hipSuccess) return hip_status(e, padded ? "padded update launch" : "compaction launch");
  }
  return ok();
}

}  // namespace

extern "C" {

int specmemo_kv_compact(specmemo_dtype dt, const specmemo_trees *t, const specmemo_kv *kv, const int32_t *accept_len,
                        const int32_t *path, int32_t path_stride, void *stream) {
  return compact_impl(dt, t, kv, accept_len, path, path_stride, false, nullptr, nullptr, nullptr, 0, stream);
}

int specmemo_kv_pad_update(specmemo_dtype dt, const specmemo_trees *t, const specmemo_kv *kv,
                           const int32_t *accept_len, const int32_t *path, int32_t path_stride, uint32_t *key_valid,
                           int64_t key_valid_words, int32_t *pos, void *ws, size_t ws_bytes, void *stream) {
  if (kv && key_valid_words < specmemo_key_mask_words(kv->cap_total))
    return fail(SPECMEMO_E_ARG, "key_valid holds %lld words, %lld needed", static_cast<long long>(key_valid_words),
                static_cast<long long>(specmemo_key_mask_words(kv->cap_total)));
  return compact_impl(dt, t, kv, accept_len, path, path_stride, true, key_valid, pos, ws, ws_bytes, stream);
}

int specmemo_accept_compact(specmemo_dtype dt, const specmemo_trees *t, const specmemo_kv *kv, int32_t vocab,
                            specmemo_accept_mode mode, float temperature, float eps, float delta,
                            const void *base_logits, const int32_t *node_tok, int32_t *accept_len, int32_t *path,
                            int32_t path_stride, int32_t *next_tok, void *ws, size_t ws_bytes, void *stream) {
  TreeInfo ti;
  AcceptArgs a;
  CompactArgs c;
  int rc = accept_args(dt, t, vocab, mode, temperature, eps, delta, base_logits, node_tok, accept_len, path,
                       path_stride, next_tok, ws, ws_bytes, &ti, &a);
  if (rc) return rc;
  if ((rc = compact_args(dt, t, kv, accept_len, path, path_stride, ti, &c))) return rc;
  // more sequences than kernel arguments hold: their descriptors go to the
  // workspace, after the acceptance's part, and one launch covers the batch
  const bool table = ti.B > kMaxSeqPerLaunch;
  const size_t acc_bytes = accept_ws_bytes(ti, mode);
  if (table && ws_bytes < acc_bytes + compact_table_bytes(ti.B))
    return fail(SPECMEMO_E_WORKSPACE, "workspace of %zu bytes needed (16-byte aligned), got %zu",
                acc_bytes + compact_table_bytes(ti.B), ws_bytes);
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e = launch_accept_rows(dt, a, ti.total, st);
  if (e != hipSuccess) return hip_status(e, "acceptance launch");
  if (table) {
    std::vector<CompactSeq> tab(ti.B);
    for (int b = 0; b < ti.B; ++b)
      tab[b] = CompactSeq{kv->seq_base_h[b], kv->seq_len_h[b], t->node_off_h[b + 1] - t->node_off_h[b],
                          kv->seq_cap_h[b], t->node_off_h[b]};
    uint8_t *w = static_cast<uint8_t *>(ws) + acc_bytes;
    if ((e = upload_table(tab.data(), tab.size() * sizeof(CompactSeq), w, st)) != hipSuccess)
      return hip_status(e, "descriptor upload");
    c.tab = reinterpret_cast<const CompactSeq *>(w);
    c.nseq = ti.B;
    c.b0 = 0;
    if ((e = launch_accept_compact(dt, a, c, st)) != hipSuccess) return hip_status(e, "acceptance and compaction launch");
    return ok();
  }
  for (int b0 = 0; b0 < ti.B; b0 += kMaxSeqPerLaunch) {
    compact_group(t, kv, b0, ti.B, &c);
    if ((e = launch_accept_compact(dt, a, c, st)) != hipSuccess) return hip_status(e, "acceptance and compaction launch");
  }
  return ok();
}

}  // extern "C"
