// Host side of libaugtree: argument validation, tile schedules and launches.
//
// Every entry point validates its arguments on the host, builds the tile
// schedule of its kernels from the host offsets (segment by segment, heaviest
// first, so concurrent workgroups share a segment's blocks in L2 and the
// ragged tail of a launch is made of short tiles), copies the schedule into
// the caller's workspace on the caller's stream, and enqueues the kernels.
// Nothing is allocated, nothing is synchronised, no state is kept between
// calls apart from a per-device cache of the architecture check.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <numeric>
#include <string>
#include <tuple>
#include <vector>

#include "../../include/augtree.h"
#include "internal.h"
#include "kernels.h"

using namespace augtree;

namespace {

thread_local std::string g_last_error;
thread_local augtree_launch_hook g_hook = nullptr;
thread_local void* g_hook_user = nullptr;

// Calls the launch hook around one kernel launch.
struct HookScope {
  const char* role;
  hipStream_t stream;
  HookScope(const char* r, hipStream_t s) : role(r), stream(s) {
    if (g_hook) g_hook(role, 0, stream, g_hook_user);
  }
  ~HookScope() {
    if (g_hook) g_hook(role, 1, stream, g_hook_user);
  }
};

int fail(int status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return status;
}

int ok() {
  g_last_error.clear();
  return AUGTREE_OK;
}

// ---------------------------------------------------------------------------- device check

std::atomic<int> g_arch_cache[64];  // 0 unknown, 1 gfx950, 2 other

int check_device_impl() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return fail(AUGTREE_ERR_DEVICE, "hipGetDevice failed");
  if (dev >= 0 && dev < 64) {
    const int c = g_arch_cache[dev].load(std::memory_order_relaxed);
    if (c == 1) return AUGTREE_OK;
    if (c == 2) return fail(AUGTREE_ERR_DEVICE, "device %d is not gfx950", dev);
  }
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, dev) != hipSuccess)
    return fail(AUGTREE_ERR_DEVICE, "hipGetDeviceProperties failed for device %d", dev);
  const bool is950 = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0;
  if (dev >= 0 && dev < 64) g_arch_cache[dev].store(is950 ? 1 : 2, std::memory_order_relaxed);
  if (!is950) return fail(AUGTREE_ERR_DEVICE, "device %d is %s, not gfx950", dev, prop.gcnArchName);
  return AUGTREE_OK;
}

// ---------------------------------------------------------------------------- validation

struct Shape {
  int ng, nb, hq, hkv, d, group;
  float scale;
  const int32_t *cp, *cb, *cr;
  int64_t tp, tr;
};

int validate_groups(const augtree_groups* g, Shape* s, bool need_branches = true) {
  if (!g) return fail(AUGTREE_ERR_INVALID_ARGUMENT, "null descriptor");
  if (g->num_groups < 1 || (need_branches && g->num_branches < 1))
    return fail(AUGTREE_ERR_INVALID_ARGUMENT, "num_groups=%d num_branches=%d must be >= 1", g->num_groups,
                g->num_branches);
  if (!g->cu_prompt || (need_branches && (!g->cu_branch || !g->cu_resp)))
    return fail(AUGTREE_ERR_INVALID_ARGUMENT, "null offset array");
  if (g->num_q_heads < 1 || g->num_kv_heads < 1)
    return fail(AUGTREE_ERR_INVALID_ARGUMENT, "head counts must be >= 1");
  if (g->num_q_heads % g->num_kv_heads != 0)
    return fail(AUGTREE_ERR_UNSUPPORTED, "num_q_heads %d not a multiple of num_kv_heads %d", g->num_q_heads,
                g->num_kv_heads);
  if (g->head_dim != 64 && g->head_dim != 128)
    return fail(AUGTREE_ERR_UNSUPPORTED, "head_dim %d not in {64,128}", g->head_dim);
  if (!(g->softmax_scale > 0.f) || !std::isfinite(g->softmax_scale))
    return fail(AUGTREE_ERR_INVALID_ARGUMENT, "softmax_scale must be finite and > 0");
  const int32_t *cp = g->cu_prompt, *cb = g->cu_branch, *cr = g->cu_resp;
  if (cp[0] != 0) return fail(AUGTREE_ERR_INVALID_ARGUMENT, "cu_prompt must start at 0");
  for (int i = 0; i < g->num_groups; ++i)
    if (cp[i + 1] <= cp[i]) return fail(AUGTREE_ERR_INVALID_ARGUMENT, "prompt of group %d is empty or offsets decrease", i);
  if (need_branches) {
    if (cb[0] != 0 || cr[0] != 0) return fail(AUGTREE_ERR_INVALID_ARGUMENT, "offsets must start at 0");
    for (int i = 0; i < g->num_groups; ++i)
      if (cb[i + 1] <= cb[i]) return fail(AUGTREE_ERR_INVALID_ARGUMENT, "group %d has no branch or offsets decrease", i);
    if (cb[g->num_groups] != g->num_branches)
      return fail(AUGTREE_ERR_INVALID_ARGUMENT, "cu_branch[num_groups]=%d != num_branches=%d", cb[g->num_groups],
                  g->num_branches);
    for (int b = 0; b < g->num_branches; ++b)
      if (cr[b + 1] <= cr[b]) return fail(AUGTREE_ERR_INVALID_ARGUMENT, "branch %d is empty or offsets decrease", b);
  }
  s->ng = g->num_groups;
  s->nb = need_branches ? g->num_branches : 0;
  s->hq = g->num_q_heads;
  s->hkv = g->num_kv_heads;
  s->d = g->head_dim;
  s->group = g->num_q_heads / g->num_kv_heads;
  s->scale = g->softmax_scale;
  s->cp = cp;
  s->cb = cb;
  s->cr = cr;
  s->tp = cp[s->ng];
  s->tr = need_branches ? cr[s->nb] : 0;
  return AUGTREE_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

#define REQUIRE_PTR(p)                                                                                 \
  do {                                                                                                 \
    if (!(p)) return fail(AUGTREE_ERR_INVALID_ARGUMENT, "null pointer: %s", #p);                       \
    if (!aligned16(p)) return fail(AUGTREE_ERR_MISALIGNED, "pointer %s is not 16-byte aligned", #p);    \
  } while (0)

#define OPTIONAL_PTR(p)                                                                                \
  do {                                                                                                 \
    if ((p) && !aligned16(p)) return fail(AUGTREE_ERR_MISALIGNED, "pointer %s is not 16-byte aligned", #p); \
  } while (0)

// ---------------------------------------------------------------------------- schedules

int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

int64_t qtile_cost(const QTile& t) { return (int64_t)t.q_len * (t.a_len + t.b_len); }
int64_t kvtile_cost(const KVTile& t) { return (int64_t)(t.x_len + t.y_len) * t.kv_len; }

// Tile order. Each XCD runs the tiles of one KV head in list order, so
// concurrent workgroups share a K/V or Q/dO block in the XCD's L2 only when
// they work on the same segment (a group's prompt, a branch); a cost-only
// heaviest-first order mixes the tiles of all segments (16 equal branches:
// ~2 concurrent tiles per branch). So segments run one after the other, by
// total cost, each heaviest tile first. A segment's heaviest tile must still
// start early enough not to end alone: the work listed from the segment's
// start to the end of the launch has to cover `conc` (the tiles the chip runs
// at once) times that tile. Segments that fail (the last, small ones; decided
// from the end backwards) go to a pool at the end of the list, heaviest tile
// first across the pooled segments. A launch shorter than a few rounds of its
// heaviest tiles (less than 8 x conc x the heaviest tile in all) pools every
// segment, i.e. keeps the plain heaviest-first order: there the tail of a
// late heavy tile costs more than the shared reads save.
template <class T, class F>
void sort_segment_major(std::vector<T>& v, const std::vector<int>& seg, F cost, int conc) {
  int nseg = 0;
  for (int x : seg) nseg = std::max(nseg, x + 1);
  std::vector<int64_t> total(nseg, 0), top(nseg, 0);
  for (size_t i = 0; i < v.size(); ++i) {
    total[seg[i]] += cost(v[i]);
    top[seg[i]] = std::max(top[seg[i]], cost(v[i]));
  }
  std::vector<int> order(nseg);
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return total[a] > total[b]; });
  int64_t all = 0, top_all = 0;
  for (int g = 0; g < nseg; ++g) {
    all += total[g];
    top_all = std::max(top_all, top[g]);
  }
  const bool shallow = all < 8 * (int64_t)conc * top_all;
  std::vector<int> rank(nseg, 0);
  std::vector<char> pooled(nseg, 0);
  int64_t after = 0;  // work listed after the segment being decided
  for (int k = nseg - 1; k >= 0; --k) {
    const int g = order[k];
    rank[g] = k;
    if (shallow || after + total[g] < (int64_t)conc * top[g]) pooled[g] = 1;
    after += total[g];
  }
  std::vector<std::tuple<int, int, int64_t, size_t>> key(v.size());
  for (size_t i = 0; i < v.size(); ++i) {
    const int g = seg[i];
    key[i] = {pooled[g] ? 1 : 0, pooled[g] ? 0 : rank[g], -cost(v[i]), i};
  }
  std::sort(key.begin(), key.end());
  std::vector<T> out(v.size());
  for (size_t i = 0; i < v.size(); ++i) out[i] = v[std::get<3>(key[i])];
  v.swap(out);
}

// Tiles the chip runs at once (256 CUs of MI355X; a scheduling estimate, not
// a limit): query tiles take `hq` workgroups, two per CU; key tiles `hkv`
// workgroups, one per CU.
int conc_qtiles(const Shape& s) { return std::max(1, 2 * 256 / s.hq); }
int conc_kvtiles(const Shape& s) { return std::max(1, 256 / s.hkv); }

// Tile lists are built by appending (tile, segment id) pairs and sorted once
// per launch. Segment ids: a group's prompt rows or prompt keys = g, branch b
// = num_groups + b.
template <class T>
struct TileList {
  std::vector<T> v;
  std::vector<int> seg;
  void add(const T& t, int s) {
    v.push_back(t);
    seg.push_back(s);
  }
};

// prompt causal query tiles (prefill fwd and dQ)
void add_prefill_qtiles(TileList<QTile>& L, const Shape& s, int bm) {
  for (int g = 0; g < s.ng; ++g) {
    const int P = s.cp[g + 1] - s.cp[g];
    for (int t0 = 0; t0 < P; t0 += bm) {
      QTile t{};
      t.q_row0 = s.cp[g] + t0;
      t.q_len = std::min(bm, P - t0);
      t.b_row0 = s.cp[g];
      t.b_len = t0 + t.q_len;
      t.b_qpos = t0;
      t.flags = QT_PROMPT_ROWS;
      L.add(t, g);
    }
  }
}

// response query tiles: RP_PROMPT = prompt keys only (spans the group's
// branches; first partial slot), RP_OWN = own-branch causal keys only (second
// partial slot), RP_FUSED = both
enum { RP_PROMPT = 0, RP_OWN = 1, RP_FUSED = 2 };

// `keep` (optional, one flag per group) limits the tiles to the flagged groups
void add_replay_qtiles(TileList<QTile>& L, const Shape& s, int bm, int which, const std::vector<char>* keep = nullptr) {
  for (int g = 0; g < s.ng; ++g) {
    if (keep && !(*keep)[g]) continue;
    const int P = s.cp[g + 1] - s.cp[g];
    if (which == RP_PROMPT) {
      const int r0 = s.cr[s.cb[g]], r1 = s.cr[s.cb[g + 1]];
      for (int q0 = r0; q0 < r1; q0 += bm) {
        QTile t{};
        t.q_row0 = q0;
        t.q_len = std::min(bm, r1 - q0);
        t.a_row0 = s.cp[g];
        t.a_len = P;
        L.add(t, g);
      }
      continue;
    }
    for (int b = s.cb[g]; b < s.cb[g + 1]; ++b) {
      const int R = s.cr[b + 1] - s.cr[b];
      for (int t0 = 0; t0 < R; t0 += bm) {
        QTile t{};
        t.q_row0 = s.cr[b] + t0;
        t.q_len = std::min(bm, R - t0);
        if (which == RP_FUSED) {
          t.a_row0 = s.cp[g];
          t.a_len = P;
        } else {
          t.flags = QT_PART1;
        }
        t.b_row0 = s.cr[b];
        t.b_len = t0 + t.q_len;
        t.b_qpos = t0;
        L.add(t, s.ng + b);
      }
    }
  }
}

// Replay forward mode per group (AUGTREE_REPLAY_AUTO). A mode's cost is the
// number of (query tile, 64-key block) steps its forward tiles execute, at the
// measured time of one step per workgroup slot of the chip, plus for SPLIT
// the HBM time of the merge. A fused tile of a short branch sweeps every
// prompt block for a few rows; the split prompt partial packs the rows of all
// branches of the group into full tiles, but pays the partials' round trip.
constexpr double kFwdStepNs = 3.7;         // 128 rows x 64 keys x one head, d = 128, per slot (measured)
constexpr double kMergeBytesPerNs = 5000;  // merge kernel bandwidth (measured, ~5 TB/s)

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

bool replay_prefers_split(const Shape& s, int g, int bm, int bn) {
  const int64_t prompt_blocks = ceil_div(s.cp[g + 1] - s.cp[g], bn);
  int64_t fused = 0, own = 0, rows = 0;
  for (int b = s.cb[g]; b < s.cb[g + 1]; ++b) {
    const int R = s.cr[b + 1] - s.cr[b];
    rows += R;
    for (int t0 = 0; t0 < R; t0 += bm) {
      const int64_t own_blocks = ceil_div(std::min(R, t0 + bm), bn);
      fused += prompt_blocks + own_blocks;
      own += own_blocks;
    }
  }
  const int64_t split = ceil_div(rows, bm) * prompt_blocks + own;
  const double step = kFwdStepNs * (double)s.d / 128.0 * s.hq;
  const double merge_bytes = (double)rows * s.hq * (10.0 * s.d + 12.0);
  return split * step + merge_bytes / kMergeBytesPerNs < fused * step;
}

std::vector<char> replay_split_groups(const Shape& s, int mode) {
  std::vector<char> v(s.ng, mode == AUGTREE_REPLAY_SPLIT ? 1 : 0);
  if (mode == AUGTREE_REPLAY_AUTO)
    for (int g = 0; g < s.ng; ++g) v[g] = replay_prefers_split(s, g, fwd_block_m(), fwd_block_n()) ? 1 : 0;
  return v;
}

// prompt key tiles of group g: X = response rows r0 + x0 .. r0 + x1 - 1 of
// the group (all branches; every prompt key visible), Y = the prefill rows
// from the tile's first key (causal) if `prefill`; with KV_OUT_SLAB, the fp32
// result of the group's key k goes to slab row out_base + k
void add_prompt_kvtiles(TileList<KVTile>& L, const Shape& s, int bn, int g, int x0, int x1, bool prefill,
                        int32_t flags, int64_t out_base = 0) {
  const int P = s.cp[g + 1] - s.cp[g];
  // (a prefill-only call passes no branch offsets and an empty X range)
  const int r0 = x1 > x0 ? s.cr[s.cb[g]] : 0;
  for (int k0 = 0; k0 < P; k0 += bn) {
    KVTile t{};
    t.kv_row0 = s.cp[g] + k0;
    t.kv_len = std::min(bn, P - k0);
    t.x_row0 = r0 + x0;
    t.x_len = x1 - x0;
    if (prefill) t.y_len = P - k0;  // queries before the first key cannot see it
    t.kpos0 = k0;
    t.out_row0 = (flags & KV_OUT_SLAB) ? (int32_t)(out_base + k0) : 0;
    t.flags = flags | KV_PROMPT_KEYS;
    L.add(t, g);
  }
}

// own-branch causal key tiles of every branch
void add_response_kvtiles(TileList<KVTile>& L, const Shape& s, int bn) {
  for (int b = 0; b < s.nb; ++b) {
    const int R = s.cr[b + 1] - s.cr[b];
    for (int k0 = 0; k0 < R; k0 += bn) {
      KVTile t{};
      t.kv_row0 = s.cr[b] + k0;
      t.kv_len = std::min(bn, R - k0);
      t.x_row0 = s.cr[b] + k0;
      t.x_len = R - k0;
      t.kpos0 = k0;
      t.flags = KV_X_CAUSAL | KV_OUT_BF16;
      L.add(t, s.ng + b);
    }
  }
}

// The tree backward cuts a prompt key tile's sweep over the branch rows into
// chunks of at most this many query blocks (64 rows of one query head): the
// workgroups that share the same query rows drift apart over long sweeps, and
// then neither they nor the branch key tiles running beside them find those
// rows in L2.
std::atomic<int> g_tree_chunk_blocks{kTreeChunkBlocksDefault};

// Boundaries of chunk c of n of a group's `nr` response rows, on multiples of
// the query block where possible.
int seed_edge(int64_t nr, int k, int n, int bq) {
  if (k == 0) return 0;
  if (k == n) return (int)nr;
  int64_t e = nr * k / n;
  e = (e / bq) * bq;
  return (int)std::min<int64_t>(e, nr);
}

// ---------------------------------------------------------------------------- plans and workspace

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// The launches of one entry point: up to three query-tile lists and one
// key-tile list, each sorted for its launch. Lists longer than kInlineTiles
// are uploaded to the start of the workspace (one copy); shorter ones travel
// in the kernel arguments. The workspace then holds D = rowsum(dO * O) for
// the backward ([Hq, T_P] then [Hq, T_R]).
struct Plan {
  TileList<QTile> q[3];
  TileList<KVTile> kv;
  size_t off_q[3] = {0, 0, 0}, off_kv = 0, off_dsum_p = 0, off_dsum_r = 0, bytes = 0, blob_bytes = 0;
  int64_t dsum_rows_p = 0, dsum_rows_r = 0;
  // chunked prompt-key sweeps of the tree backward (n_parts > 0): the fp32
  // slab [2][slab_rows, Hkv, d] of the chunks and the reduce's row map
  // [n_parts][T_P] (uploaded with the schedules)
  int n_parts = 0;
  int64_t slab_rows = 0;
  std::vector<int32_t> row_map;
  size_t off_row_map = 0, off_slab = 0;
  std::vector<char> blob;

  void sort(const Shape& s) {
    for (auto& l : q) sort_segment_major(l.v, l.seg, qtile_cost, conc_qtiles(s));
    sort_segment_major(kv.v, kv.seg, kvtile_cost, conc_kvtiles(s));
  }
  // every list gets room in the workspace (its size does not depend on
  // which lists end up inline)
  void layout(int hq, int64_t row_elems) {
    size_t o = 0;
    for (int i = 0; i < 3; ++i) {
      off_q[i] = o;
      o = align_up(o + q[i].v.size() * sizeof(QTile));
    }
    off_kv = o;
    o = align_up(o + kv.v.size() * sizeof(KVTile));
    off_row_map = o;
    o = align_up(o + row_map.size() * sizeof(int32_t));
    blob_bytes = o;
    off_dsum_p = o;
    o = align_up(o + (size_t)dsum_rows_p * hq * sizeof(float));
    off_dsum_r = o;
    o = align_up(o + (size_t)dsum_rows_r * hq * sizeof(float));
    off_slab = o;
    o = align_up(o + (size_t)slab_rows * 2 * row_elems * sizeof(float));
    bytes = std::max<size_t>(o, kAlign);
  }
  static bool inline_list(size_t n) { return n <= (size_t)kInlineTiles; }
  // bytes of the workspace prefix that must be uploaded (0: every list inline)
  size_t upload_bytes() const {
    size_t end = 0;
    for (int i = 0; i < 3; ++i)
      if (!inline_list(q[i].v.size())) end = off_q[i] + q[i].v.size() * sizeof(QTile);
    if (!inline_list(kv.v.size())) end = off_kv + kv.v.size() * sizeof(KVTile);
    if (!row_map.empty()) end = off_row_map + row_map.size() * sizeof(int32_t);
    return end;
  }
  void pack() {
    blob.assign(upload_bytes(), 0);
    for (int i = 0; i < 3; ++i)
      if (!inline_list(q[i].v.size()))
        std::memcpy(blob.data() + off_q[i], q[i].v.data(), q[i].v.size() * sizeof(QTile));
    if (!inline_list(kv.v.size())) std::memcpy(blob.data() + off_kv, kv.v.data(), kv.v.size() * sizeof(KVTile));
    if (!row_map.empty()) std::memcpy(blob.data() + off_row_map, row_map.data(), row_map.size() * sizeof(int32_t));
  }
};

// Points the launch parameters at list i: the workspace copy, or the kernel
// arguments' inline copy.
template <class P, class T>
void bind_tiles(P& p, const TileList<T>& L, void* ws, size_t off) {
  if (Plan::inline_list(L.v.size())) {
    p.tiles = nullptr;
    std::copy(L.v.begin(), L.v.end(), p.inl);
  } else {
    p.tiles = reinterpret_cast<const T*>(static_cast<char*>(ws) + off);
  }
}

// Operation codes of augtree_workspace_size beyond the public four.
Plan plan_for(const Shape& s, int op, int arg) {
  Plan pl;
  const int bm = fwd_block_m(), bn = dkv_block_n(), bq = dkv_block_q();
  switch (op) {
    case AUGTREE_OP_PREFILL_FWD:
      add_prefill_qtiles(pl.q[0], s, bm);
      break;
    case AUGTREE_OP_REPLAY_FWD:
    case AUGTREE_OP_TREE_FWD: {
      // q[0]: the bf16 launch (prefill tiles for the tree call, fused groups);
      // q[1]: the split groups' partial tiles (fp32 launch)
      if (op == AUGTREE_OP_TREE_FWD) add_prefill_qtiles(pl.q[0], s, bm);
      const std::vector<char> split = replay_split_groups(s, arg);
      std::vector<char> fused(split.size());
      for (size_t g = 0; g < split.size(); ++g) fused[g] = !split[g];
      add_replay_qtiles(pl.q[0], s, bm, RP_FUSED, &fused);
      add_replay_qtiles(pl.q[1], s, bm, RP_PROMPT, &split);
      add_replay_qtiles(pl.q[1], s, bm, RP_OWN, &split);
      break;
    }
    case AUGTREE_OP_PREFILL_BWD:
      add_prefill_qtiles(pl.q[0], s, dq_block_m());
      for (int g = 0; g < s.ng; ++g) add_prompt_kvtiles(pl.kv, s, bn, g, 0, 0, true, KV_OUT_SLAB, s.cp[g]);
      pl.dsum_rows_p = s.tp;
      break;
    case AUGTREE_OP_REPLAY_BWD:
      add_replay_qtiles(pl.q[0], s, dq_block_m(), RP_FUSED);
      add_response_kvtiles(pl.kv, s, bn);
      for (int g = 0; g < s.ng; ++g) {
        const int64_t nr = s.cr[s.cb[g + 1]] - s.cr[s.cb[g]];
        for (int c = 0; c < arg; ++c) {
          const int c0 = seed_edge(nr, c, arg, bq), c1 = std::max(seed_edge(nr, c + 1, arg, bq), c0);
          // seed slab layout [part][2][T_P]
          add_prompt_kvtiles(pl.kv, s, bn, g, c0, c1, false, KV_OUT_SLAB, 2 * (int64_t)c * s.tp + s.cp[g]);
        }
      }
      pl.dsum_rows_r = s.tr;
      break;
    case AUGTREE_OP_TREE_BWD: {
      // arg bit 0: the fp32 copy of the prompt-key gradient is requested too;
      // bit 1: no chunked prompt-key sweeps (keeps the workspace small)
      add_prefill_qtiles(pl.q[0], s, dq_block_m());
      add_replay_qtiles(pl.q[0], s, dq_block_m(), RP_FUSED);
      add_response_kvtiles(pl.kv, s, bn);
      std::vector<int> nc(s.ng, 1);
      int nmax = 1;
      if (!(arg & 2))
        for (int g = 0; g < s.ng; ++g) {
          nc[g] = tree_chunk_count(s.cr[s.cb[g + 1]] - s.cr[s.cb[g]], s.group);
          nmax = std::max(nmax, nc[g]);
        }
      if (nmax == 1) {
        // one sweep per prompt key tile: the Eq. 2 sum stays in registers and
        // the tile writes bf16 (and the caller's fp32 copy, [2][T_P])
        const int32_t out = KV_OUT_BF16 | ((arg & 1) ? KV_OUT_SLAB : 0);
        for (int g = 0; g < s.ng; ++g)
          add_prompt_kvtiles(pl.kv, s, bn, g, 0, s.cr[s.cb[g + 1]] - s.cr[s.cb[g]], true, out, s.cp[g]);
      } else {
        // chunk c of group g sweeps its share of the branch rows (chunk 0
        // also the prefill rows) into the fp32 rows vbase_g + c P_g + key of
        // a workspace slab; the reduce adds the chunks in order
        std::vector<int64_t> vbase(s.ng + 1, 0);
        for (int g = 0; g < s.ng; ++g) vbase[g + 1] = vbase[g] + (int64_t)nc[g] * (s.cp[g + 1] - s.cp[g]);
        if (vbase[s.ng] > INT32_MAX) return plan_for(s, op, arg | 2);  // slab rows are int32
        for (int g = 0; g < s.ng; ++g) {
          const int64_t P = s.cp[g + 1] - s.cp[g], nr = s.cr[s.cb[g + 1]] - s.cr[s.cb[g]];
          for (int c = 0; c < nc[g]; ++c) {
            const int c0 = seed_edge(nr, c, nc[g], bq), c1 = std::max(seed_edge(nr, c + 1, nc[g], bq), c0);
            add_prompt_kvtiles(pl.kv, s, bn, g, c0, c1, c == 0, KV_OUT_SLAB, vbase[g] + c * P);
          }
        }
        pl.n_parts = nmax;
        pl.slab_rows = vbase[s.ng];
        pl.row_map.assign((size_t)nmax * s.tp, -1);
        for (int g = 0; g < s.ng; ++g)
          for (int c = 0; c < nc[g]; ++c)
            for (int32_t r = s.cp[g]; r < s.cp[g + 1]; ++r)
              pl.row_map[(size_t)c * s.tp + r] = (int32_t)(vbase[g] + (int64_t)c * (s.cp[g + 1] - s.cp[g]) + r - s.cp[g]);
      }
      pl.dsum_rows_p = s.tp;
      pl.dsum_rows_r = s.tr;
      break;
    }
    default:
      break;
  }
  pl.sort(s);
  pl.layout(s.hq, (int64_t)s.hkv * s.d);
  return pl;
}

int check_ws(const Plan& pl, void* ws, size_t ws_bytes) {
  if (!ws) return fail(AUGTREE_ERR_WORKSPACE, "null workspace (%zu bytes needed)", pl.bytes);
  if ((reinterpret_cast<uintptr_t>(ws) & (kAlign - 1)) != 0)
    return fail(AUGTREE_ERR_MISALIGNED, "workspace must be %zu-byte aligned", kAlign);
  if (ws_bytes < pl.bytes) return fail(AUGTREE_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", ws_bytes, pl.bytes);
  return AUGTREE_OK;
}

int upload(Plan& pl, void* ws, hipStream_t stream) {
  pl.pack();
  if (pl.blob.empty()) return AUGTREE_OK;
  const hipError_t e = hipMemcpyAsync(ws, pl.blob.data(), pl.blob.size(), hipMemcpyHostToDevice, stream);
  if (e != hipSuccess) return fail(AUGTREE_ERR_HIP, "schedule copy: %s", hipGetErrorString(e));
  return AUGTREE_OK;
}

int hip_status(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(AUGTREE_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return AUGTREE_OK;
}

float log2e_scale(float s) { return s * kLog2e; }

// ---------------------------------------------------------------------------- launch sequences

// Tensors of one forward or backward call (any may be null where unused).
struct Tensors {
  const uint16_t *q_p, *k_p, *v_p, *o_p, *do_p;
  const float* lse_p;
  const uint16_t *q_r, *k_r, *v_r, *o_r, *do_r;
  const float* lse_r;
};

// Forward launches of a plan: q[0] (bf16 outputs), q[1] (split partials,
// fp32) and the merge of the split groups' rows.
int run_fwd(const Shape& s, const Plan& pl, int mode, const Tensors& x, uint16_t* o_p, float* lse_p, uint16_t* o_r,
            float* lse_r, float* o_part, float* lse_part, void* ws, hipStream_t str, const char* role_main) {
  int st;
  FwdParams p{};
  p.q[0] = x.q_r; p.q[1] = x.q_p;
  p.ka = x.k_p; p.va = x.v_p;
  p.kb[0] = x.k_r; p.vb[0] = x.v_r; p.kb[1] = x.k_p; p.vb[1] = x.v_p;
  p.o[0] = o_r; p.o[1] = o_p;
  p.lse[0] = lse_r; p.lse[1] = lse_p;
  p.lse_rows[0] = s.tr; p.lse_rows[1] = s.tp;
  p.hq = s.hq; p.hkv = s.hkv; p.group = s.group; p.head_dim = s.d;
  p.scale_log2 = log2e_scale(s.scale);
  if (!pl.q[0].v.empty()) {
    bind_tiles(p, pl.q[0], ws, pl.off_q[0]);
    HookScope h(role_main, str);
    if ((st = hip_status(launch_attn_fwd(p, (int)pl.q[0].v.size(), false, str), "forward launch"))) return st;
  }
  if (pl.q[1].v.empty()) return AUGTREE_OK;
  // split groups: both partial states in one launch, then the merge
  bind_tiles(p, pl.q[1], ws, pl.off_q[1]);
  p.o32 = o_part; p.o32_part = s.tr * s.hq * s.d;
  p.lse[0] = lse_part; p.lse_part = s.tr * s.hq;
  {
    HookScope h("fwd_replay_split", str);
    if ((st = hip_status(launch_attn_fwd(p, (int)pl.q[1].v.size(), true, str), "split partial launch"))) return st;
  }
  const std::vector<char> split = replay_split_groups(s, mode);
  for (int g = 0; g < s.ng;) {  // one merge per run of consecutive split groups (contiguous rows)
    if (!split[g]) { ++g; continue; }
    int g1 = g;
    while (g1 < s.ng && split[g1]) ++g1;
    const int64_t r0 = s.cr[s.cb[g]], r1 = s.cr[s.cb[g1]];
    HookScope h("lse_merge", str);
    if ((st = hip_status(launch_lse_merge(r0, r1 - r0, s.tr, s.hq, s.d, 2, o_part, lse_part, o_r, nullptr, lse_r, str),
                         "lse merge launch")))
      return st;
    g = g1;
  }
  return AUGTREE_OK;
}

// Backward launches of a plan: the dQ kernel (which also forms D into the
// workspace), then the dK/dV kernel that reads D.
struct BwdOut {
  uint16_t *dq_p, *dq_r;
  float* dq_p32;
  uint16_t *dk_p, *dv_p, *dk_r, *dv_r;
  float* slab;
  int64_t slab_rows;
};

int run_bwd(const Shape& s, const Plan& pl, const Tensors& x, const BwdOut& out, void* ws, hipStream_t str,
            const char* role_dq, const char* role_dkv) {
  int st;
  float* dsum_p = reinterpret_cast<float*>(static_cast<char*>(ws) + pl.off_dsum_p);
  float* dsum_r = reinterpret_cast<float*>(static_cast<char*>(ws) + pl.off_dsum_r);
  const float sl2 = log2e_scale(s.scale);
  if (!pl.q[0].v.empty()) {
    DqParams p{};
    bind_tiles(p, pl.q[0], ws, pl.off_q[0]);
    p.q[0] = x.q_r; p.q[1] = x.q_p;
    p.dout[0] = x.do_r; p.dout[1] = x.do_p;
    p.o[0] = x.o_r; p.o[1] = x.o_p;
    p.lse[0] = x.lse_r; p.lse[1] = x.lse_p;
    p.dsum[0] = dsum_r; p.dsum[1] = dsum_p;
    p.lse_rows[0] = s.tr; p.lse_rows[1] = s.tp;
    p.ka = x.k_p; p.va = x.v_p;
    p.kb[0] = x.k_r; p.vb[0] = x.v_r; p.kb[1] = x.k_p; p.vb[1] = x.v_p;
    p.dq[0] = out.dq_r; p.dq[1] = out.dq_p;
    p.dq32[1] = out.dq_p32;
    p.hq = s.hq; p.hkv = s.hkv; p.group = s.group; p.head_dim = s.d; p.scale = s.scale; p.scale_log2 = sl2;
    HookScope h(role_dq, str);
    if ((st = hip_status(launch_attn_dq(p, (int)pl.q[0].v.size(), str), "dq launch"))) return st;
  }
  if (!pl.kv.v.empty()) {
    DkvParams p{};
    bind_tiles(p, pl.kv, ws, pl.off_kv);
    p.k[0] = x.k_r; p.v[0] = x.v_r; p.k[1] = x.k_p; p.v[1] = x.v_p;
    p.q[0] = x.q_r; p.q[1] = x.q_p;
    p.dout[0] = x.do_r; p.dout[1] = x.do_p;
    p.lse[0] = x.lse_r; p.lse[1] = x.lse_p;
    p.dsum[0] = dsum_r; p.dsum[1] = dsum_p;
    p.lse_rows[0] = s.tr; p.lse_rows[1] = s.tp;
    p.dk[0] = out.dk_r; p.dv[0] = out.dv_r; p.dk[1] = out.dk_p; p.dv[1] = out.dv_p;
    p.slab = out.slab; p.slab_rows = out.slab_rows;
    p.hq = s.hq; p.hkv = s.hkv; p.group = s.group; p.head_dim = s.d; p.scale = s.scale; p.scale_log2 = sl2;
    HookScope h(role_dkv, str);
    if ((st = hip_status(launch_attn_dkv(p, (int)pl.kv.v.size(), str), "dkv launch"))) return st;
  }
  return AUGTREE_OK;
}

}  // namespace

// ============================================================================ C ABI

extern "C" {

const char* augtree_version(void) { return "augtree-mi355x 0.1"; }

const char* augtree_status_string(int status) {
  switch (status) {
    case AUGTREE_OK: return "ok";
    case AUGTREE_ERR_INVALID_ARGUMENT: return "invalid argument";
    case AUGTREE_ERR_UNSUPPORTED: return "unsupported shape";
    case AUGTREE_ERR_MISALIGNED: return "misaligned pointer";
    case AUGTREE_ERR_WORKSPACE: return "workspace missing or too small";
    case AUGTREE_ERR_DEVICE: return "device is not gfx950";
    case AUGTREE_ERR_HIP: return "HIP error";
    default: return "unknown status";
  }
}

const char* augtree_last_error(void) { return g_last_error.c_str(); }

void augtree_set_launch_hook(augtree_launch_hook hook, void* user) {
  g_hook = hook;
  g_hook_user = user;
}

int augtree_set_tree_chunk_blocks(int32_t blocks) {
  if (blocks < 0) return fail(AUGTREE_ERR_INVALID_ARGUMENT, "chunk blocks %d < 0", blocks);
  g_tree_chunk_blocks.store(blocks == 0 ? kTreeChunkBlocksDefault : blocks, std::memory_order_relaxed);
  return ok();
}

int32_t augtree_tree_chunk_blocks(void) { return g_tree_chunk_blocks.load(std::memory_order_relaxed); }

int augtree_check_device(void) {
  const int st = check_device_impl();
  return st == AUGTREE_OK ? ok() : st;
}

size_t augtree_workspace_size(const augtree_groups* grp, int op, int arg) {
  Shape s;
  const bool prefill_only = op == AUGTREE_OP_PREFILL_FWD || op == AUGTREE_OP_PREFILL_BWD;
  if (validate_groups(grp, &s, !prefill_only) != AUGTREE_OK) return 0;
  if (op < AUGTREE_OP_PREFILL_FWD || op > AUGTREE_OP_TREE_BWD) {
    fail(AUGTREE_ERR_INVALID_ARGUMENT, "unknown op %d", op);
    return 0;
  }
  if ((op == AUGTREE_OP_REPLAY_FWD || op == AUGTREE_OP_TREE_FWD) && arg != AUGTREE_REPLAY_FUSED &&
      arg != AUGTREE_REPLAY_SPLIT && arg != AUGTREE_REPLAY_AUTO) {
    fail(AUGTREE_ERR_INVALID_ARGUMENT, "unknown replay mode %d", arg);
    return 0;
  }
  if (op == AUGTREE_OP_REPLAY_BWD && (arg < 1 || arg > 64)) {
    fail(AUGTREE_ERR_INVALID_ARGUMENT, "n_seed %d not in [1,64]", arg);
    return 0;
  }
  if (op == AUGTREE_OP_TREE_BWD) arg = 1;  // room for the largest schedule (fp32 prompt copy or not)
  ok();
  return plan_for(s, op, arg).bytes;
}

int augtree_prefill_fwd(const augtree_groups* grp, const uint16_t* q_p, const uint16_t* k_p, const uint16_t* v_p,
                        uint16_t* o_p, float* lse_p, void* ws, size_t ws_bytes, void* stream) {
  Shape s;
  int st = validate_groups(grp, &s, false);
  if (st) return st;
  REQUIRE_PTR(q_p); REQUIRE_PTR(k_p); REQUIRE_PTR(v_p); REQUIRE_PTR(o_p); REQUIRE_PTR(lse_p);
  Plan pl = plan_for(s, AUGTREE_OP_PREFILL_FWD, 0);
  if ((st = check_ws(pl, ws, ws_bytes))) return st;
  if ((st = check_device_impl())) return st;
  hipStream_t str = static_cast<hipStream_t>(stream);
  if ((st = upload(pl, ws, str))) return st;
  Tensors x{};
  x.q_p = q_p; x.k_p = k_p; x.v_p = v_p;
  if ((st = run_fwd(s, pl, AUGTREE_REPLAY_FUSED, x, o_p, lse_p, nullptr, nullptr, nullptr, nullptr, ws, str,
                    "fwd_prefill")))
    return st;
  return ok();
}

int augtree_replay_fwd(const augtree_groups* grp, int mode, const uint16_t* q_r, const uint16_t* k_r,
                       const uint16_t* v_r, const uint16_t* k_p, const uint16_t* v_p, uint16_t* o_r, float* lse_r,
                       float* o_part, float* lse_part, void* ws, size_t ws_bytes, void* stream) {
  Shape s;
  int st = validate_groups(grp, &s);
  if (st) return st;
  if (mode != AUGTREE_REPLAY_FUSED && mode != AUGTREE_REPLAY_SPLIT && mode != AUGTREE_REPLAY_AUTO)
    return fail(AUGTREE_ERR_INVALID_ARGUMENT, "unknown replay mode %d", mode);
  REQUIRE_PTR(q_r); REQUIRE_PTR(k_r); REQUIRE_PTR(v_r); REQUIRE_PTR(k_p); REQUIRE_PTR(v_p);
  REQUIRE_PTR(o_r); REQUIRE_PTR(lse_r);
  if (mode != AUGTREE_REPLAY_FUSED) { REQUIRE_PTR(o_part); REQUIRE_PTR(lse_part); }
  Plan pl = plan_for(s, AUGTREE_OP_REPLAY_FWD, mode);
  if ((st = check_ws(pl, ws, ws_bytes))) return st;
  if ((st = check_device_impl())) return st;
  hipStream_t str = static_cast<hipStream_t>(stream);
  if ((st = upload(pl, ws, str))) return st;
  Tensors x{};
  x.k_p = k_p; x.v_p = v_p; x.q_r = q_r; x.k_r = k_r; x.v_r = v_r;
  if ((st = run_fwd(s, pl, mode, x, nullptr, nullptr, o_r, lse_r, o_part, lse_part, ws, str, "fwd_replay")))
    return st;
  return ok();
}

int augtree_tree_fwd(const augtree_groups* grp, int mode, const uint16_t* q_p, const uint16_t* k_p,
                     const uint16_t* v_p, const uint16_t* q_r, const uint16_t* k_r, const uint16_t* v_r, uint16_t* o_p,
                     float* lse_p, uint16_t* o_r, float* lse_r, float* o_part, float* lse_part, void* ws,
                     size_t ws_bytes, void* stream) {
  Shape s;
  int st = validate_groups(grp, &s);
  if (st) return st;
  if (mode != AUGTREE_REPLAY_FUSED && mode != AUGTREE_REPLAY_SPLIT && mode != AUGTREE_REPLAY_AUTO)
    return fail(AUGTREE_ERR_INVALID_ARGUMENT, "unknown replay mode %d", mode);
  REQUIRE_PTR(q_p); REQUIRE_PTR(k_p); REQUIRE_PTR(v_p); REQUIRE_PTR(q_r); REQUIRE_PTR(k_r); REQUIRE_PTR(v_r);
  REQUIRE_PTR(o_p); REQUIRE_PTR(lse_p); REQUIRE_PTR(o_r); REQUIRE_PTR(lse_r);
  if (mode != AUGTREE_REPLAY_FUSED) { REQUIRE_PTR(o_part); REQUIRE_PTR(lse_part); }
  Plan pl = plan_for(s, AUGTREE_OP_TREE_FWD, mode);
  if ((st = check_ws(pl, ws, ws_bytes))) return st;
  if ((st = check_device_impl())) return st;
  hipStream_t str = static_cast<hipStream_t>(stream);
  if ((st = upload(pl, ws, str))) return st;
  const Tensors x{q_p, k_p, v_p, nullptr, nullptr, nullptr, q_r, k_r, v_r, nullptr, nullptr, nullptr};
  if ((st = run_fwd(s, pl, mode, x, o_p, lse_p, o_r, lse_r, o_part, lse_part, ws, str, "fwd_tree"))) return st;
  return ok();
}

int augtree_replay_split_groups(const augtree_groups* grp, int32_t* split) {
  Shape s;
  int st = validate_groups(grp, &s);
  if (st) return st;
  if (!split) return fail(AUGTREE_ERR_INVALID_ARGUMENT, "null pointer: split");
  const std::vector<char> v = replay_split_groups(s, AUGTREE_REPLAY_AUTO);
  for (int g = 0; g < s.ng; ++g) split[g] = v[g];
  return ok();
}

int augtree_lse_merge(int64_t rows, int32_t heads, int32_t head_dim, int32_t n_parts, const float* o_parts,
                      const float* lse_parts, uint16_t* o, float* o_f32, float* lse, void* stream) {
  if (rows < 0 || heads < 1 || n_parts < 1 || head_dim < 8 || head_dim > 256 || head_dim % 8)
    return fail(AUGTREE_ERR_INVALID_ARGUMENT, "rows=%lld heads=%d head_dim=%d n_parts=%d", (long long)rows, heads,
                head_dim, n_parts);
  if (rows == 0) return ok();
  REQUIRE_PTR(o_parts); REQUIRE_PTR(lse_parts);
  OPTIONAL_PTR(o); OPTIONAL_PTR(o_f32); OPTIONAL_PTR(lse);
  if (!o && !o_f32) return fail(AUGTREE_ERR_INVALID_ARGUMENT, "no output (o and o_f32 both null)");
  int st;
  if ((st = check_device_impl())) return st;
  HookScope h("lse_merge", static_cast<hipStream_t>(stream));
  if ((st = hip_status(launch_lse_merge(0, rows, rows, heads, head_dim, n_parts, o_parts, lse_parts, o, o_f32, lse,
                                        static_cast<hipStream_t>(stream)),
                       "lse merge launch")))
    return st;
  return ok();
}

int augtree_replay_bwd(const augtree_groups* grp, const uint16_t* q_r, const uint16_t* k_r, const uint16_t* v_r,
                       const uint16_t* k_p, const uint16_t* v_p, const uint16_t* o_r, const float* lse_r,
                       const uint16_t* do_r, uint16_t* dq_r, uint16_t* dk_r, uint16_t* dv_r, int32_t n_seed,
                       float* dkv_p_seed, void* ws, size_t ws_bytes, void* stream) {
  Shape s;
  int st = validate_groups(grp, &s);
  if (st) return st;
  if (n_seed < 1 || n_seed > 64) return fail(AUGTREE_ERR_INVALID_ARGUMENT, "n_seed %d not in [1,64]", n_seed);
  if (2 * (int64_t)n_seed * s.tp > INT32_MAX)
    return fail(AUGTREE_ERR_UNSUPPORTED, "seed slab of %d x 2 x %lld rows exceeds int32 rows", n_seed, (long long)s.tp);
  REQUIRE_PTR(q_r); REQUIRE_PTR(k_r); REQUIRE_PTR(v_r); REQUIRE_PTR(k_p); REQUIRE_PTR(v_p);
  REQUIRE_PTR(o_r); REQUIRE_PTR(lse_r); REQUIRE_PTR(do_r);
  REQUIRE_PTR(dq_r); REQUIRE_PTR(dk_r); REQUIRE_PTR(dv_r); REQUIRE_PTR(dkv_p_seed);
  Plan pl = plan_for(s, AUGTREE_OP_REPLAY_BWD, n_seed);
  if ((st = check_ws(pl, ws, ws_bytes))) return st;
  if ((st = check_device_impl())) return st;
  hipStream_t str = static_cast<hipStream_t>(stream);
  if ((st = upload(pl, ws, str))) return st;
  Tensors x{};
  x.k_p = k_p; x.v_p = v_p;
  x.q_r = q_r; x.k_r = k_r; x.v_r = v_r; x.o_r = o_r; x.do_r = do_r; x.lse_r = lse_r;
  BwdOut out{};
  out.dq_r = dq_r; out.dk_r = dk_r; out.dv_r = dv_r;
  out.slab = dkv_p_seed; out.slab_rows = s.tp;
  if ((st = run_bwd(s, pl, x, out, ws, str, "dq_replay", "dkv_replay"))) return st;
  return ok();
}

int augtree_prefill_bwd(const augtree_groups* grp, const uint16_t* q_p, const uint16_t* k_p, const uint16_t* v_p,
                        const uint16_t* o_p, const float* lse_p, const uint16_t* do_p, uint16_t* dq_p,
                        float* dq_p_f32, float* dkv_p_self, void* ws, size_t ws_bytes, void* stream) {
  Shape s;
  int st = validate_groups(grp, &s, false);
  if (st) return st;
  REQUIRE_PTR(q_p); REQUIRE_PTR(k_p); REQUIRE_PTR(v_p); REQUIRE_PTR(o_p); REQUIRE_PTR(lse_p); REQUIRE_PTR(do_p);
  OPTIONAL_PTR(dq_p); OPTIONAL_PTR(dq_p_f32);
  if (!dq_p && !dq_p_f32) return fail(AUGTREE_ERR_INVALID_ARGUMENT, "no dQ output (dq_p and dq_p_f32 both null)");
  REQUIRE_PTR(dkv_p_self);
  Plan pl = plan_for(s, AUGTREE_OP_PREFILL_BWD, 0);
  if ((st = check_ws(pl, ws, ws_bytes))) return st;
  if ((st = check_device_impl())) return st;
  hipStream_t str = static_cast<hipStream_t>(stream);
  if ((st = upload(pl, ws, str))) return st;
  Tensors x{};
  x.q_p = q_p; x.k_p = k_p; x.v_p = v_p; x.o_p = o_p; x.do_p = do_p; x.lse_p = lse_p;
  BwdOut out{};
  out.dq_p = dq_p; out.dq_p32 = dq_p_f32;
  out.slab = dkv_p_self; out.slab_rows = s.tp;
  if ((st = run_bwd(s, pl, x, out, ws, str, "dq_prefill", "dkv_prefill"))) return st;
  return ok();
}

}  // extern "C"

namespace augtree {

int fail_status(int status, const char* msg) { return fail(status, "%s", msg); }

int tree_chunk_count(int64_t nr, int group) {
  const int64_t blocks = (nr + kDkvBlockQ - 1) / kDkvBlockQ * group;
  const int64_t per = g_tree_chunk_blocks.load(std::memory_order_relaxed);
  return (int)std::min<int64_t>(64, std::max<int64_t>(1, (blocks + per - 1) / per));
}

int tree_bwd_impl(const augtree_groups* grp, const uint16_t* q_p, const uint16_t* k_p, const uint16_t* v_p,
                  const uint16_t* o_p, const float* lse_p, const uint16_t* do_p, const uint16_t* q_r,
                  const uint16_t* k_r, const uint16_t* v_r, const uint16_t* o_r, const float* lse_r,
                  const uint16_t* do_r, uint16_t* dq_p, uint16_t* dk_p, uint16_t* dv_p, float* dkv_p_f32,
                  uint16_t* dq_r, uint16_t* dk_r, uint16_t* dv_r, ScratchFn scratch, void* ws, size_t ws_bytes,
                  void* stream) {
  Shape s;
  int st = validate_groups(grp, &s);
  if (st) return st;
  REQUIRE_PTR(q_p); REQUIRE_PTR(k_p); REQUIRE_PTR(v_p); REQUIRE_PTR(o_p); REQUIRE_PTR(lse_p); REQUIRE_PTR(do_p);
  REQUIRE_PTR(q_r); REQUIRE_PTR(k_r); REQUIRE_PTR(v_r); REQUIRE_PTR(o_r); REQUIRE_PTR(lse_r); REQUIRE_PTR(do_r);
  REQUIRE_PTR(dq_p); REQUIRE_PTR(dk_p); REQUIRE_PTR(dv_p); REQUIRE_PTR(dq_r); REQUIRE_PTR(dk_r); REQUIRE_PTR(dv_r);
  OPTIONAL_PTR(dkv_p_f32);
  Plan pl = plan_for(s, AUGTREE_OP_TREE_BWD, dkv_p_f32 ? 1 : 0);
  if (scratch) {  // the caller's buffer is a fixed device array: check its size before touching the device
    // chunked prompt-key sweeps need an fp32 slab; without room for it, one
    // sweep per prompt key tile (the same sum in another fp32 order)
    if (pl.bytes > ws_bytes && pl.n_parts > 0) pl = plan_for(s, AUGTREE_OP_TREE_BWD, (dkv_p_f32 ? 1 : 0) | 2);
    if (pl.bytes > ws_bytes)
      return fail(AUGTREE_ERR_WORKSPACE,
                  "this batch needs %zu bytes of scratch; the allocation-free entry point holds at most %zu bytes",
                  pl.bytes, ws_bytes);
    if ((st = check_device_impl())) return st;
    if ((st = scratch(&ws))) return st;
  }
  if ((st = check_ws(pl, ws, ws_bytes))) return st;
  if (!scratch && (st = check_device_impl())) return st;
  hipStream_t str = static_cast<hipStream_t>(stream);
  if ((st = upload(pl, ws, str))) return st;
  const Tensors x{q_p, k_p, v_p, o_p, do_p, lse_p, q_r, k_r, v_r, o_r, do_r, lse_r};
  BwdOut out{};
  out.dq_p = dq_p; out.dq_r = dq_r;
  out.dk_p = dk_p; out.dv_p = dv_p; out.dk_r = dk_r; out.dv_r = dv_r;
  if (pl.n_parts > 0) {
    out.slab = reinterpret_cast<float*>(static_cast<char*>(ws) + pl.off_slab);
    out.slab_rows = pl.slab_rows;
  } else {
    out.slab = dkv_p_f32;
    out.slab_rows = s.tp;
  }
  if ((st = run_bwd(s, pl, x, out, ws, str, "dq_tree", "dkv_tree"))) return st;
  if (pl.n_parts > 0) {
    // the chunks of each prompt key row, added in chunk order (Eq. 2)
    const int64_t e = (int64_t)s.hkv * s.d;
    uint16_t* const o16[2] = {dk_p, dv_p};
    float* const o32[2] = {dkv_p_f32, dkv_p_f32 ? dkv_p_f32 + s.tp * e : nullptr};
    HookScope h("reduce_tree", str);
    if ((st = hip_status(launch_grad_reduce(2, s.tp, e, nullptr, pl.n_parts, pl.slab_rows, 0, out.slab,
                                            reinterpret_cast<const int32_t*>(static_cast<char*>(ws) + pl.off_row_map),
                                            o16, o32, str),
                         "reduce launch")))
      return st;
  }
  return ok();
}

}  // namespace augtree

extern "C" {

int augtree_tree_bwd(const augtree_groups* grp, const uint16_t* q_p, const uint16_t* k_p, const uint16_t* v_p,
                     const uint16_t* o_p, const float* lse_p, const uint16_t* do_p, const uint16_t* q_r,
                     const uint16_t* k_r, const uint16_t* v_r, const uint16_t* o_r, const float* lse_r,
                     const uint16_t* do_r, uint16_t* dq_p, uint16_t* dk_p, uint16_t* dv_p, float* dkv_p_f32,
                     uint16_t* dq_r, uint16_t* dk_r, uint16_t* dv_r, void* ws, size_t ws_bytes, void* stream) {
  return tree_bwd_impl(grp, q_p, k_p, v_p, o_p, lse_p, do_p, q_r, k_r, v_r, o_r, lse_r, do_r, dq_p, dk_p, dv_p,
                       dkv_p_f32, dq_r, dk_r, dv_r, nullptr, ws, ws_bytes, stream);
}

int augtree_prompt_grad_reduce(int32_t n_tensors, int64_t rows, int32_t heads, int32_t head_dim, const float* self,
                               int32_t n_parts, int64_t part_rows, int64_t part_stride, const float* parts,
                               const int32_t* row_map, uint16_t* out, float* out_f32, void* stream) {
  if (n_tensors < 1 || n_tensors > 2) return fail(AUGTREE_ERR_INVALID_ARGUMENT, "n_tensors %d not in {1,2}", n_tensors);
  if (rows < 0 || heads < 1 || head_dim < 1 || ((int64_t)heads * head_dim) % 4)
    return fail(AUGTREE_ERR_INVALID_ARGUMENT, "rows=%lld heads=%d head_dim=%d", (long long)rows, heads, head_dim);
  if (n_parts < 0 || n_parts > 4096) return fail(AUGTREE_ERR_INVALID_ARGUMENT, "n_parts %d not in [0,4096]", n_parts);
  if (!row_map && n_parts > 0 && part_rows != rows)
    return fail(AUGTREE_ERR_INVALID_ARGUMENT, "part_rows %lld != rows %lld without a row map", (long long)part_rows,
                (long long)rows);
  if (part_rows < 0) return fail(AUGTREE_ERR_INVALID_ARGUMENT, "part_rows < 0");
  if (part_stride < 0 || part_stride % 4) return fail(AUGTREE_ERR_INVALID_ARGUMENT, "part_stride %lld must be >= 0 and a multiple of 4", (long long)part_stride);
  if (rows == 0) return ok();
  OPTIONAL_PTR(self); OPTIONAL_PTR(out); OPTIONAL_PTR(out_f32);
  if (n_parts > 0) REQUIRE_PTR(parts);
  if (!out && !out_f32) return fail(AUGTREE_ERR_INVALID_ARGUMENT, "no output (out and out_f32 both null)");
  int st;
  if ((st = check_device_impl())) return st;
  HookScope h("grad_reduce", static_cast<hipStream_t>(stream));
  const int64_t e = (int64_t)heads * head_dim;
  uint16_t* const o16[2] = {out, out && n_tensors > 1 ? out + rows * e : nullptr};
  float* const o32[2] = {out_f32, out_f32 && n_tensors > 1 ? out_f32 + rows * e : nullptr};
  if ((st = hip_status(launch_grad_reduce(n_tensors, rows, e, self, n_parts, part_rows, part_stride, parts, row_map,
                                          o16, o32, static_cast<hipStream_t>(stream)),
                       "grad reduce launch")))
    return st;
  return ok();
}

}  // extern "C"
