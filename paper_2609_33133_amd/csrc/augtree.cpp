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
int64_t kvtile_cost(const KVTile& t) { return (int64_t)t.q_len * t.kv_len; }

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

// prompt causal tiles (prefill fwd and dQ)
std::vector<QTile> prefill_qtiles(const Shape& s, int bm) {
  std::vector<QTile> v;
  std::vector<int> seg;
  for (int g = 0; g < s.ng; ++g) {
    const int P = s.cp[g + 1] - s.cp[g];
    for (int t0 = 0; t0 < P; t0 += bm) {
      QTile t{};
      t.q_row0 = s.cp[g] + t0;
      t.q_len = std::min(bm, P - t0);
      t.b_row0 = s.cp[g];
      t.b_len = t0 + t.q_len;
      t.b_qpos = t0;
      v.push_back(t);
      seg.push_back(g);
    }
  }
  sort_segment_major(v, seg, qtile_cost, conc_qtiles(s));
  return v;
}

// response tiles: part 0 = prompt keys only (spans the group's branches),
// part 1 = own-branch causal keys only, fused = both
enum { RP_PROMPT = 0, RP_OWN = 1, RP_FUSED = 2 };

// `keep` (optional, one flag per group) limits the tiles to the flagged groups
std::vector<QTile> replay_qtiles(const Shape& s, int bm, int which, const std::vector<char>* keep = nullptr) {
  std::vector<QTile> v;
  std::vector<int> seg;  // prompt partial: the group; otherwise the branch
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
        v.push_back(t);
        seg.push_back(g);
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
        }
        t.b_row0 = s.cr[b];
        t.b_len = t0 + t.q_len;
        t.b_qpos = t0;
        v.push_back(t);
        seg.push_back(b);
      }
    }
  }
  sort_segment_major(v, seg, qtile_cost, conc_qtiles(s));
  return v;
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

// causal key tiles over contiguous segments [start, start+len), segment id `id`
void causal_kvtiles(std::vector<KVTile>& v, std::vector<int>& seg, int id, int32_t start, int32_t len, int bn) {
  for (int k0 = 0; k0 < len; k0 += bn) {
    seg.push_back(id);
    KVTile t{};
    t.kv_row0 = start + k0;
    t.kv_len = std::min(bn, len - k0);
    t.q_row0 = start + k0;  // queries before the first key cannot see it
    t.q_len = len - k0;
    t.causal = 1;
    t.kpos0 = k0;
    t.qpos0 = k0;
    v.push_back(t);
  }
}

std::vector<KVTile> prefill_kvtiles(const Shape& s, int bn) {
  std::vector<KVTile> v;
  std::vector<int> seg;
  for (int g = 0; g < s.ng; ++g) causal_kvtiles(v, seg, g, s.cp[g], s.cp[g + 1] - s.cp[g], bn);
  sort_segment_major(v, seg, kvtile_cost, conc_kvtiles(s));
  return v;
}

std::vector<KVTile> response_kvtiles(const Shape& s, int bn) {
  std::vector<KVTile> v;
  std::vector<int> seg;
  for (int b = 0; b < s.nb; ++b) causal_kvtiles(v, seg, b, s.cr[b], s.cr[b + 1] - s.cr[b], bn);
  sort_segment_major(v, seg, kvtile_cost, conc_kvtiles(s));
  return v;
}

// prompt keys x every response row of the group, rows cut into n_seed chunks
std::vector<KVTile> seed_kvtiles(const Shape& s, int bn, int n_seed, int bq) {
  std::vector<KVTile> v;
  std::vector<int> seg;  // (group, chunk): the tiles of one segment sweep the same rows
  for (int g = 0; g < s.ng; ++g) {
    const int P = s.cp[g + 1] - s.cp[g];
    const int r0 = s.cr[s.cb[g]], r1 = s.cr[s.cb[g + 1]];
    const int64_t nr = r1 - r0;
    for (int c = 0; c < n_seed; ++c) {
      // chunk boundaries on multiples of the query block where possible
      auto edge = [&](int k) -> int {
        if (k == 0) return 0;
        if (k == n_seed) return (int)nr;
        int64_t e = nr * k / n_seed;
        e = (e / bq) * bq;
        return (int)std::min<int64_t>(e, nr);
      };
      const int c0 = edge(c), c1 = std::max(edge(c + 1), c0);
      for (int k0 = 0; k0 < P; k0 += bn) {
        KVTile t{};
        t.kv_row0 = s.cp[g] + k0;
        t.kv_len = std::min(bn, P - k0);
        t.q_row0 = r0 + c0;
        t.q_len = c1 - c0;
        t.causal = 0;
        t.part = c;
        v.push_back(t);
        seg.push_back(g * n_seed + c);
      }
    }
  }
  sort_segment_major(v, seg, kvtile_cost, conc_kvtiles(s));
  return v;
}

// ---------------------------------------------------------------------------- workspace layout

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct Plan {
  std::vector<QTile> q1, q2, q3;  // forward / dQ tiles (split: q1 prompt, q2 own; auto: q3 fused groups)
  std::vector<KVTile> kv1, kv2;   // dK/dV tiles
  size_t off_q1 = 0, off_q2 = 0, off_q3 = 0, off_kv1 = 0, off_kv2 = 0, off_dsum = 0, bytes = 0;
  int64_t dsum_rows = 0;
  std::vector<char> blob;         // schedule bytes copied to the start of the workspace
  size_t blob_bytes = 0;

  void layout(int hq) {
    size_t o = 0;
    off_q1 = o; o = align_up(o + q1.size() * sizeof(QTile));
    off_q2 = o; o = align_up(o + q2.size() * sizeof(QTile));
    off_q3 = o; o = align_up(o + q3.size() * sizeof(QTile));
    off_kv1 = o; o = align_up(o + kv1.size() * sizeof(KVTile));
    off_kv2 = o; o = align_up(o + kv2.size() * sizeof(KVTile));
    blob_bytes = o;
    off_dsum = o; o = align_up(o + (size_t)dsum_rows * hq * sizeof(float));
    bytes = std::max<size_t>(o, kAlign);
  }
  void pack() {
    blob.assign(blob_bytes, 0);
    if (!q1.empty()) std::memcpy(blob.data() + off_q1, q1.data(), q1.size() * sizeof(QTile));
    if (!q2.empty()) std::memcpy(blob.data() + off_q2, q2.data(), q2.size() * sizeof(QTile));
    if (!q3.empty()) std::memcpy(blob.data() + off_q3, q3.data(), q3.size() * sizeof(QTile));
    if (!kv1.empty()) std::memcpy(blob.data() + off_kv1, kv1.data(), kv1.size() * sizeof(KVTile));
    if (!kv2.empty()) std::memcpy(blob.data() + off_kv2, kv2.data(), kv2.size() * sizeof(KVTile));
  }
};

Plan plan_for(const Shape& s, int op, int arg) {
  Plan pl;
  switch (op) {
    case AUGTREE_OP_PREFILL_FWD:
      pl.q1 = prefill_qtiles(s, fwd_block_m());
      break;
    case AUGTREE_OP_REPLAY_FWD:
      if (arg == AUGTREE_REPLAY_SPLIT) {
        pl.q1 = replay_qtiles(s, fwd_block_m(), RP_PROMPT);
        pl.q2 = replay_qtiles(s, fwd_block_m(), RP_OWN);
      } else if (arg == AUGTREE_REPLAY_AUTO) {
        const std::vector<char> split = replay_split_groups(s, arg);
        std::vector<char> fused(split.size());
        for (size_t g = 0; g < split.size(); ++g) fused[g] = !split[g];
        pl.q1 = replay_qtiles(s, fwd_block_m(), RP_PROMPT, &split);
        pl.q2 = replay_qtiles(s, fwd_block_m(), RP_OWN, &split);
        pl.q3 = replay_qtiles(s, fwd_block_m(), RP_FUSED, &fused);
      } else {
        pl.q1 = replay_qtiles(s, fwd_block_m(), RP_FUSED);
      }
      break;
    case AUGTREE_OP_PREFILL_BWD:
      pl.q1 = prefill_qtiles(s, dq_block_m());
      pl.kv1 = prefill_kvtiles(s, dkv_block_n());
      pl.dsum_rows = s.tp;
      break;
    case AUGTREE_OP_REPLAY_BWD:
      pl.q1 = replay_qtiles(s, dq_block_m(), RP_FUSED);
      pl.kv1 = response_kvtiles(s, dkv_block_n());
      pl.kv2 = seed_kvtiles(s, dkv_block_n(), arg, dkv_block_q());
      pl.dsum_rows = s.tr;
      break;
    default:
      break;
  }
  pl.layout(s.hq);
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
  if (pl.blob_bytes == 0) return AUGTREE_OK;
  const hipError_t e = hipMemcpyAsync(ws, pl.blob.data(), pl.blob_bytes, hipMemcpyHostToDevice, stream);
  if (e != hipSuccess) return fail(AUGTREE_ERR_HIP, "schedule copy: %s", hipGetErrorString(e));
  return AUGTREE_OK;
}

int hip_status(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(AUGTREE_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return AUGTREE_OK;
}

template <class T>
const T* at(void* ws, size_t off) {
  return reinterpret_cast<const T*>(static_cast<char*>(ws) + off);
}

float log2e_scale(float s) { return s * kLog2e; }

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

int augtree_check_device(void) {
  const int st = check_device_impl();
  return st == AUGTREE_OK ? ok() : st;
}

size_t augtree_workspace_size(const augtree_groups* grp, int op, int arg) {
  Shape s;
  const bool prefill_only = op == AUGTREE_OP_PREFILL_FWD || op == AUGTREE_OP_PREFILL_BWD;
  if (validate_groups(grp, &s, !prefill_only) != AUGTREE_OK) return 0;
  if (op < AUGTREE_OP_PREFILL_FWD || op > AUGTREE_OP_REPLAY_BWD) {
    fail(AUGTREE_ERR_INVALID_ARGUMENT, "unknown op %d", op);
    return 0;
  }
  if (op == AUGTREE_OP_REPLAY_FWD && arg != AUGTREE_REPLAY_FUSED && arg != AUGTREE_REPLAY_SPLIT &&
      arg != AUGTREE_REPLAY_AUTO) {
    fail(AUGTREE_ERR_INVALID_ARGUMENT, "unknown replay mode %d", arg);
    return 0;
  }
  if (op == AUGTREE_OP_REPLAY_BWD && (arg < 1 || arg > 64)) {
    fail(AUGTREE_ERR_INVALID_ARGUMENT, "n_seed %d not in [1,64]", arg);
    return 0;
  }
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
  FwdParams p{};
  p.tiles = at<QTile>(ws, pl.off_q1);
  p.q = q_p; p.ka = k_p; p.va = v_p; p.kb = k_p; p.vb = v_p;
  p.o = o_p; p.lse = lse_p; p.lse_rows = s.tp;
  p.hq = s.hq; p.hkv = s.hkv; p.group = s.group; p.head_dim = s.d;
  p.scale_log2 = log2e_scale(s.scale);
  {
    HookScope h("fwd_prefill", str);
    if ((st = hip_status(launch_attn_fwd(p, (int)pl.q1.size(), false, str), "prefill fwd launch"))) return st;
  }
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
  FwdParams p{};
  p.q = q_r; p.ka = k_p; p.va = v_p; p.kb = k_r; p.vb = v_r;
  p.lse_rows = s.tr;
  p.hq = s.hq; p.hkv = s.hkv; p.group = s.group; p.head_dim = s.d;
  p.scale_log2 = log2e_scale(s.scale);
  // fused tiles: all groups (FUSED) or the groups the cost rule keeps fused (AUTO)
  const std::vector<QTile>& fused_tiles = mode == AUGTREE_REPLAY_FUSED ? pl.q1 : pl.q3;
  const size_t fused_off = mode == AUGTREE_REPLAY_FUSED ? pl.off_q1 : pl.off_q3;
  if (!fused_tiles.empty()) {
    p.tiles = at<QTile>(ws, fused_off);
    p.o = o_r; p.lse = lse_r;
    HookScope h("fwd_replay", str);
    if ((st = hip_status(launch_attn_fwd(p, (int)fused_tiles.size(), false, str), "replay fwd launch"))) return st;
  }
  if (mode == AUGTREE_REPLAY_FUSED) return ok();
  // split groups: two partial states, then the merge over their rows
  const int64_t part_o = s.tr * s.hq * s.d;
  const int64_t part_l = s.tr * s.hq;
  p.o = nullptr;
  if (!pl.q1.empty()) {
    p.tiles = at<QTile>(ws, pl.off_q1);
    p.o32 = o_part; p.lse = lse_part;
    HookScope h("fwd_replay_prompt", str);
    if ((st = hip_status(launch_attn_fwd(p, (int)pl.q1.size(), true, str), "replay prompt partial launch"))) return st;
  }
  if (!pl.q2.empty()) {
    p.tiles = at<QTile>(ws, pl.off_q2);
    p.o32 = o_part + part_o; p.lse = lse_part + part_l;
    HookScope h("fwd_replay_own", str);
    if ((st = hip_status(launch_attn_fwd(p, (int)pl.q2.size(), true, str), "replay own partial launch"))) return st;
  }
  const std::vector<char> split = replay_split_groups(s, mode);
  for (int g = 0; g < s.ng;) {  // one merge per run of consecutive split groups (contiguous rows)
    if (!split[g]) { ++g; continue; }
    int g1 = g;
    while (g1 < s.ng && split[g1]) ++g1;
    const int64_t r0 = s.cr[s.cb[g]], r1 = s.cr[s.cb[g1]];
    HookScope h("lse_merge", str);
    if ((st = hip_status(launch_lse_merge(r0, r1 - r0, s.tr, s.hq, s.d, 2, o_part, lse_part, o_r, nullptr, lse_r,
                                          str),
                         "lse merge launch")))
      return st;
    g = g1;
  }
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
  REQUIRE_PTR(q_r); REQUIRE_PTR(k_r); REQUIRE_PTR(v_r); REQUIRE_PTR(k_p); REQUIRE_PTR(v_p);
  REQUIRE_PTR(o_r); REQUIRE_PTR(lse_r); REQUIRE_PTR(do_r);
  REQUIRE_PTR(dq_r); REQUIRE_PTR(dk_r); REQUIRE_PTR(dv_r); REQUIRE_PTR(dkv_p_seed);
  Plan pl = plan_for(s, AUGTREE_OP_REPLAY_BWD, n_seed);
  if ((st = check_ws(pl, ws, ws_bytes))) return st;
  if ((st = check_device_impl())) return st;
  hipStream_t str = static_cast<hipStream_t>(stream);
  if ((st = upload(pl, ws, str))) return st;
  float* dsum = reinterpret_cast<float*>(static_cast<char*>(ws) + pl.off_dsum);
  {
    HookScope h("dsum_replay", str);
    if ((st = hip_status(launch_bwd_dsum(o_r, do_r, dsum, s.tr, s.hq, s.d, str), "dsum launch"))) return st;
  }
  const float sl2 = log2e_scale(s.scale);
  {  // prompt seeds: prompt keys x all response rows of the group (Eq. 2 sum in registers)
    DkvParams p{};
    p.tiles = at<KVTile>(ws, pl.off_kv2);
    p.k = k_p; p.v = v_p; p.q = q_r; p.dout = do_r; p.lse = lse_r; p.dsum = dsum;
    p.dkv32 = dkv_p_seed; p.out_rows = s.tp; p.lse_rows = s.tr;
    p.hq = s.hq; p.hkv = s.hkv; p.group = s.group; p.head_dim = s.d; p.scale = s.scale; p.scale_log2 = sl2;
    HookScope h("dkv_seed", str);
    if ((st = hip_status(launch_attn_dkv(p, (int)pl.kv2.size(), true, str), "seed dkv launch"))) return st;
  }
  {  // own-branch keys, causal
    DkvParams p{};
    p.tiles = at<KVTile>(ws, pl.off_kv1);
    p.k = k_r; p.v = v_r; p.q = q_r; p.dout = do_r; p.lse = lse_r; p.dsum = dsum;
    p.dk = dk_r; p.dv = dv_r; p.out_rows = s.tr; p.lse_rows = s.tr;
    p.hq = s.hq; p.hkv = s.hkv; p.group = s.group; p.head_dim = s.d; p.scale = s.scale; p.scale_log2 = sl2;
    HookScope h("dkv_resp", str);
    if ((st = hip_status(launch_attn_dkv(p, (int)pl.kv1.size(), false, str), "response dkv launch"))) return st;
  }
  {  // dQ over prompt keys then own-branch keys
    DqParams p{};
    p.tiles = at<QTile>(ws, pl.off_q1);
    p.q = q_r; p.dout = do_r; p.lse = lse_r; p.dsum = dsum;
    p.ka = k_p; p.va = v_p; p.kb = k_r; p.vb = v_r;
    p.dq = dq_r; p.lse_rows = s.tr;
    p.hq = s.hq; p.hkv = s.hkv; p.group = s.group; p.head_dim = s.d; p.scale = s.scale; p.scale_log2 = sl2;
    HookScope h("dq_replay", str);
    if ((st = hip_status(launch_attn_dq(p, (int)pl.q1.size(), str), "replay dq launch"))) return st;
  }
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
  float* dsum = reinterpret_cast<float*>(static_cast<char*>(ws) + pl.off_dsum);
  {
    HookScope h("dsum_prefill", str);
    if ((st = hip_status(launch_bwd_dsum(o_p, do_p, dsum, s.tp, s.hq, s.d, str), "dsum launch"))) return st;
  }
  const float sl2 = log2e_scale(s.scale);
  {
    DkvParams p{};
    p.tiles = at<KVTile>(ws, pl.off_kv1);
    p.k = k_p; p.v = v_p; p.q = q_p; p.dout = do_p; p.lse = lse_p; p.dsum = dsum;
    p.dkv32 = dkv_p_self; p.out_rows = s.tp; p.lse_rows = s.tp;
    p.hq = s.hq; p.hkv = s.hkv; p.group = s.group; p.head_dim = s.d; p.scale = s.scale; p.scale_log2 = sl2;
    HookScope h("dkv_prefill", str);
    if ((st = hip_status(launch_attn_dkv(p, (int)pl.kv1.size(), true, str), "prefill dkv launch"))) return st;
  }
  {
    DqParams p{};
    p.tiles = at<QTile>(ws, pl.off_q1);
    p.q = q_p; p.dout = do_p; p.lse = lse_p; p.dsum = dsum;
    p.ka = k_p; p.va = v_p; p.kb = k_p; p.vb = v_p;
    p.dq = dq_p; p.dq32 = dq_p_f32; p.lse_rows = s.tp;
    p.hq = s.hq; p.hkv = s.hkv; p.group = s.group; p.head_dim = s.d; p.scale = s.scale; p.scale_log2 = sl2;
    HookScope h("dq_prefill", str);
    if ((st = hip_status(launch_attn_dq(p, (int)pl.q1.size(), str), "prefill dq launch"))) return st;
  }
  return ok();
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
  if ((st = hip_status(launch_grad_reduce(n_tensors, rows, (int64_t)heads * head_dim, self, n_parts, part_rows,
                                          part_stride, parts, row_map, out, out_f32, static_cast<hipStream_t>(stream)),
                       "grad reduce launch")))
    return st;
  return ok();
}

}  // extern "C"
