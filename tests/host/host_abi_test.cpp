// Host-logic test of libaugtree without a GPU (built with AddressSanitizer and
// UndefinedBehaviorSanitizer against fake_hip.cpp): every entry point on
// ragged batches, checking each launch's tile schedule (bounds, causal
// geometry, every output row written once, visible pairs equal to the
// method's counts), the validation errors, the HIP-error path (a launch or
// the schedule copy failing must return AUGTREE_ERR_HIP with a message and
// no crash), and the workspace check of the allocation-free backward.
// Prints "ok" and exits 0 on success.
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/augtree.h"
#include "fake_hip.h"
#include "internal.h"

namespace {

int g_fail = 0;
int g_chunked = 0;  // chunked tree backward schedules checked
#define CHECK(c, ...)                                              \
  do {                                                             \
    if (!(c)) {                                                    \
      std::fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__);    \
      std::fprintf(stderr, __VA_ARGS__);                           \
      std::fprintf(stderr, "\n");                                  \
      ++g_fail;                                                    \
    }                                                              \
  } while (0)

struct Batch {
  std::vector<int32_t> cp, cb, cr;
  int hq, hkv, d;
  augtree_groups g;
  int64_t prefill = 0, rp = 0, rr = 0;
  void finish() {
    g = augtree_groups{(int32_t)cp.size() - 1, (int32_t)cr.size() - 1, hq, hkv, d, 0.125f, cp.data(), cb.data(),
                       cr.data()};
    prefill = rp = rr = 0;
    for (size_t i = 0; i + 1 < cp.size(); ++i) {
      const int64_t P = cp[i + 1] - cp[i];
      prefill += P * (P + 1) / 2;
      for (int b = cb[i]; b < cb[i + 1]; ++b) {
        const int64_t R = cr[b + 1] - cr[b];
        rp += R * P;
        rr += R * (R + 1) / 2;
      }
    }
  }
  int64_t tp() const { return cp.back(); }
  int64_t tr() const { return cr.back(); }
};

Batch make(const std::vector<int>& ps, const std::vector<std::vector<int>>& rs, int hq, int hkv, int d) {
  Batch b;
  b.hq = hq; b.hkv = hkv; b.d = d;
  b.cp = {0}; b.cb = {0}; b.cr = {0};
  for (size_t g = 0; g < ps.size(); ++g) {
    b.cp.push_back(b.cp.back() + ps[g]);
    for (int r : rs[g]) b.cr.push_back(b.cr.back() + r);
    b.cb.push_back(b.cb.back() + (int)rs[g].size());
  }
  b.finish();
  return b;
}

uint64_t g_rng = 88172645463325252ull;
int rnd(int lo, int hi) {  // xorshift64, inclusive range
  g_rng ^= g_rng << 13; g_rng ^= g_rng >> 7; g_rng ^= g_rng << 17;
  return lo + (int)(g_rng % (uint64_t)(hi - lo + 1));
}

// fake device addresses: 256-byte aligned, never dereferenced by the library
void* P(int i) { return reinterpret_cast<void*>((uintptr_t)(0x10000000ull + 0x100000ull * (uint64_t)i)); }
template <class T>
T* A(int i) { return static_cast<T*>(P(i)); }

struct Ws {
  void* p = nullptr;
  size_t n = 0;
  explicit Ws(size_t bytes) : n(bytes) { p = std::aligned_alloc(256, (bytes + 255) / 256 * 256 + 256); }
  ~Ws() { std::free(p); }
};

FakeShape shape_of(const Batch& b) {
  FakeShape s;
  s.tp = b.tp(); s.tr = b.tr(); s.cu_prompt = b.cp; s.cu_resp = b.cr;
  return s;
}

void expect_clean(const char* what) {
  for (const auto& e : fake_errors()) CHECK(false, "%s: %s", what, e.c_str());
}

// the fp32 slab rows written by the dK/dV tiles: [start, start + len) for each
// start, each exactly once, and no other row
void expect_slab(const char* what, const std::vector<int64_t>& starts, int64_t len) {
  const std::vector<int>& w = fake_slab_rows();
  std::vector<int> want(w.size(), 0);
  for (int64_t st : starts)
    for (int64_t r = st; r < st + len; ++r) {
      if (r >= (int64_t)want.size()) want.resize(r + 1, 0);
      want[r] += 1;
    }
  bool same = true;
  for (size_t r = 0; r < std::max(w.size(), want.size()); ++r) {
    const int a = r < w.size() ? w[r] : 0, b = r < want.size() ? want[r] : 0;
    if (a != b || b > 1) same = false;
  }
  CHECK(same, "%s: fp32 slab rows", what);
}

// slab rows of the chunked tree backward: sum over groups of chunks x P
int64_t chunk_slab_rows(const Batch& b) {
  int64_t v = 0;
  for (size_t g = 0; g + 1 < b.cp.size(); ++g) {
    const int64_t nr = b.cr[b.cb[g + 1]] - b.cr[b.cb[g]];
    v += (int64_t)augtree::tree_chunk_count(nr, b.hq / b.hkv) * (b.cp[g + 1] - b.cp[g]);
  }
  return v;
}

using u16 = uint16_t;

int call(const Batch& b, int which, Ws& ws, int arg) {
  const augtree_groups* g = &b.g;
  switch (which) {
    case 0: return augtree_prefill_fwd(g, A<u16>(1), A<u16>(2), A<u16>(3), A<u16>(4), A<float>(5), ws.p, ws.n, nullptr);
    case 1: return augtree_replay_fwd(g, arg, A<u16>(6), A<u16>(7), A<u16>(8), A<u16>(2), A<u16>(3), A<u16>(9),
                                      A<float>(10), A<float>(11), A<float>(12), ws.p, ws.n, nullptr);
    case 2: return augtree_prefill_bwd(g, A<u16>(1), A<u16>(2), A<u16>(3), A<u16>(4), A<float>(5), A<u16>(13),
                                       A<u16>(14), nullptr, A<float>(15), ws.p, ws.n, nullptr);
    case 3: return augtree_replay_bwd(g, A<u16>(6), A<u16>(7), A<u16>(8), A<u16>(2), A<u16>(3), A<u16>(9),
                                      A<float>(10), A<u16>(16), A<u16>(17), A<u16>(18), A<u16>(19), arg, A<float>(20),
                                      ws.p, ws.n, nullptr);
    case 4: return augtree_tree_fwd(g, arg, A<u16>(1), A<u16>(2), A<u16>(3), A<u16>(6), A<u16>(7), A<u16>(8),
                                    A<u16>(4), A<float>(5), A<u16>(9), A<float>(10), A<float>(11), A<float>(12), ws.p,
                                    ws.n, nullptr);
    default: return augtree_tree_bwd(g, A<u16>(1), A<u16>(2), A<u16>(3), A<u16>(4), A<float>(5), A<u16>(13),
                                     A<u16>(6), A<u16>(7), A<u16>(8), A<u16>(9), A<float>(10), A<u16>(16), A<u16>(14),
                                     A<u16>(21), A<u16>(22), arg ? A<float>(23) : nullptr, A<u16>(17), A<u16>(18),
                                     A<u16>(19), ws.p, ws.n, nullptr);
  }
}

const int kOp[6] = {AUGTREE_OP_PREFILL_FWD, AUGTREE_OP_REPLAY_FWD, AUGTREE_OP_PREFILL_BWD, AUGTREE_OP_REPLAY_BWD,
                    AUGTREE_OP_TREE_FWD, AUGTREE_OP_TREE_BWD};

void check_batch(const Batch& b) {
  const int64_t tp = b.tp(), tr = b.tr();
  // chunk: the tree backward's chunk setting (0: the default; 3: chunks of
  // at most 3 query blocks, i.e. nearly every group chunked)
  struct Case { int which, arg, chunk; };
  const Case cases[] = {{0, 0, 0}, {1, AUGTREE_REPLAY_FUSED, 0}, {1, AUGTREE_REPLAY_SPLIT, 0},
                        {1, AUGTREE_REPLAY_AUTO, 0}, {2, 0, 0}, {3, 1, 0}, {3, 2, 0}, {3, 3, 0}, {3, 64, 0},
                        {4, AUGTREE_REPLAY_FUSED, 0}, {4, AUGTREE_REPLAY_AUTO, 0}, {5, 0, 0}, {5, 1, 0},
                        {5, 0, 3}, {5, 1, 3}};
  for (const Case& c : cases) {
    CHECK(augtree_set_tree_chunk_blocks(c.chunk) == AUGTREE_OK, "chunk setting");
    const size_t need = augtree_workspace_size(&b.g, kOp[c.which], c.which == 5 ? 0 : c.arg);
    CHECK(need > 0 && need % 256 == 0, "workspace size %zu", need);
    Ws ws(need);
    fake_set_shape(shape_of(b));
    fake_set_workspace(ws.p, ws.n);
    fake_fail_at(0);
    const int st = call(b, c.which, ws, c.arg);
    CHECK(st == AUGTREE_OK, "entry %d arg %d: status %d (%s)", c.which, c.arg, st, augtree_last_error());
    expect_clean("schedule");
    const FakeCounts& n = fake_counts();
    switch (c.which) {
      case 0:
        CHECK(n.fwd_pairs == b.prefill, "prefill fwd pairs");
        fake_check_coverage("o_p", tp);
        break;
      case 1:
        CHECK(n.fwd_pairs == b.rp + b.rr, "replay fwd pairs %lld vs %lld", (long long)n.fwd_pairs,
              (long long)(b.rp + b.rr));
        if (c.arg == AUGTREE_REPLAY_FUSED) fake_check_coverage("o_r", tr);
        if (c.arg == AUGTREE_REPLAY_SPLIT) {
          fake_check_coverage("fwd_part0", tr);
          fake_check_coverage("fwd_part1", tr);
          fake_check_coverage("merge", tr);
        }
        break;
      case 2:
        CHECK(n.dq_pairs == b.prefill && n.dkv_pairs == b.prefill, "prefill bwd pairs");
        fake_check_coverage("dq_p", tp);
        expect_slab("prefill bwd", {0}, tp);
        break;
      case 3:
        CHECK(n.dq_pairs == b.rp + b.rr && n.dkv_pairs == b.rp + b.rr, "replay bwd pairs (n_seed %d)", c.arg);
        fake_check_coverage("dq_r", tr);
        fake_check_coverage("dk_r", tr);
        {
          std::vector<int64_t> st;
          for (int k = 0; k < c.arg; ++k) st.push_back(2 * k * tp);
          expect_slab("replay bwd", st, tp);
        }
        break;
      case 4:
        CHECK(n.fwd_pairs == b.prefill + b.rp + b.rr, "tree fwd pairs");
        fake_check_coverage("o_p", tp);
        if (c.arg == AUGTREE_REPLAY_FUSED) fake_check_coverage("o_r", tr);
        break;
      default:
        CHECK(n.dq_pairs == b.prefill + b.rp + b.rr && n.dkv_pairs == b.prefill + b.rp + b.rr, "tree bwd pairs");
        fake_check_coverage("dq_p", tp);
        fake_check_coverage("dq_r", tr);
        fake_check_coverage("dk_p", tp);
        fake_check_coverage("dk_r", tr);
        {
          const int64_t v = chunk_slab_rows(b);
          if (v > tp) {  // then the reduce checked its row map
            expect_slab("tree bwd chunks", {0}, v);
            ++g_chunked;
          }
          else if (c.arg) expect_slab("tree bwd fp32 copy", {0}, tp);
          else expect_slab("tree bwd", {}, 0);
        }
        break;
    }
    // every launch and copy of the call failing in turn: AUGTREE_ERR_HIP, a message, no crash
    const int steps = n.launches + 1;
    for (int k = 1; k <= steps; ++k) {
      fake_set_shape(shape_of(b));
      fake_fail_at(k);
      const int st2 = call(b, c.which, ws, c.arg);
      fake_fail_at(0);
      if (st2 == AUGTREE_OK) continue;  // the call had fewer than k launches / copies
      CHECK(st2 == AUGTREE_ERR_HIP, "injected failure %d: status %d", k, st2);
      CHECK(std::strlen(augtree_last_error()) > 0, "injected failure %d: no message", k);
    }
  }
  augtree_set_tree_chunk_blocks(0);
}

int fake_scratch_ok(void** ws) {
  static std::vector<unsigned char> buf(1 << 22);
  *ws = reinterpret_cast<void*>((reinterpret_cast<uintptr_t>(buf.data()) + 255) / 256 * 256);
  return AUGTREE_OK;
}
int fake_scratch_fail(void**) { return augtree::fail_status(AUGTREE_ERR_HIP, "no scratch"); }

void check_errors() {
  Batch b = make({10, 15}, {{5, 7}, {8}}, 4, 2, 64);
  Ws ws(1 << 20);
  fake_set_shape(shape_of(b));
  CHECK(augtree_prefill_fwd(nullptr, A<u16>(1), A<u16>(2), A<u16>(3), A<u16>(4), A<float>(5), ws.p, ws.n, nullptr) ==
            AUGTREE_ERR_INVALID_ARGUMENT, "null descriptor");
  CHECK(augtree_tree_bwd(&b.g, nullptr, A<u16>(2), A<u16>(3), A<u16>(4), A<float>(5), A<u16>(13), A<u16>(6),
                         A<u16>(7), A<u16>(8), A<u16>(9), A<float>(10), A<u16>(16), A<u16>(14), A<u16>(21), A<u16>(22),
                         nullptr, A<u16>(17), A<u16>(18), A<u16>(19), ws.p, ws.n, nullptr) ==
            AUGTREE_ERR_INVALID_ARGUMENT, "null q_p");
  u16* odd = reinterpret_cast<u16*>(reinterpret_cast<char*>(P(1)) + 2);
  CHECK(augtree_prefill_fwd(&b.g, odd, A<u16>(2), A<u16>(3), A<u16>(4), A<float>(5), ws.p, ws.n, nullptr) ==
            AUGTREE_ERR_MISALIGNED, "misaligned");
  const size_t need = augtree_workspace_size(&b.g, AUGTREE_OP_TREE_BWD, 0);
  CHECK(augtree_tree_bwd(&b.g, A<u16>(1), A<u16>(2), A<u16>(3), A<u16>(4), A<float>(5), A<u16>(13), A<u16>(6),
                         A<u16>(7), A<u16>(8), A<u16>(9), A<float>(10), A<u16>(16), A<u16>(14), A<u16>(21), A<u16>(22),
                         nullptr, A<u16>(17), A<u16>(18), A<u16>(19), ws.p, need - 1, nullptr) == AUGTREE_ERR_WORKSPACE,
        "small workspace");
  // descriptors: empty branch, Hq % Hkv, head_dim
  Batch bad = make({10}, {{5, 7}}, 4, 2, 64);
  bad.cr[1] = bad.cr[0];
  CHECK(augtree_workspace_size(&bad.g, AUGTREE_OP_TREE_BWD, 0) == 0, "empty branch accepted");
  Batch bad2 = make({10}, {{5}}, 6, 4, 64);
  CHECK(augtree_workspace_size(&bad2.g, AUGTREE_OP_TREE_FWD, 0) == 0, "Hq %% Hkv accepted");
  Batch bad3 = make({10}, {{5}}, 4, 4, 96);
  CHECK(augtree_workspace_size(&bad3.g, AUGTREE_OP_TREE_FWD, 0) == 0, "head_dim 96 accepted");
  CHECK(augtree_workspace_size(&b.g, 17, 0) == 0, "unknown op accepted");
  // allocation-free path: too small an array is reported before the device is touched; a failing lookup
  // is reported; a big enough array runs the same schedule
  auto run_impl = [&](augtree::ScratchFn fn, size_t bytes) {
    return augtree::tree_bwd_impl(&b.g, A<u16>(1), A<u16>(2), A<u16>(3), A<u16>(4), A<float>(5), A<u16>(13), A<u16>(6),
                                  A<u16>(7), A<u16>(8), A<u16>(9), A<float>(10), A<u16>(16), A<u16>(14), A<u16>(21),
                                  A<u16>(22), nullptr, A<u16>(17), A<u16>(18), A<u16>(19), fn, nullptr, bytes, nullptr);
  };
  CHECK(run_impl(fake_scratch_ok, need - 1) == AUGTREE_ERR_WORKSPACE, "scratch size check");
  CHECK(std::strstr(augtree_last_error(), "allocation-free") != nullptr, "scratch size message");
  CHECK(run_impl(fake_scratch_fail, 1 << 22) == AUGTREE_ERR_HIP, "scratch lookup failure");
  fake_set_shape(shape_of(b));
  CHECK(run_impl(fake_scratch_ok, 1 << 22) == AUGTREE_OK, "scratch run: %s", augtree_last_error());
  expect_clean("scratch schedule");
  // chunk setting: negative rejected, 0 restores the default
  CHECK(augtree_set_tree_chunk_blocks(-1) == AUGTREE_ERR_INVALID_ARGUMENT, "negative chunk blocks");
  CHECK(augtree_set_tree_chunk_blocks(5) == AUGTREE_OK && augtree_tree_chunk_blocks() == 5, "chunk blocks set");
  // with chunks whose slab does not fit, the allocation-free path runs the
  // unchunked schedule (and checks against its size)
  CHECK(augtree_set_tree_chunk_blocks(1) == AUGTREE_OK, "chunk blocks set");
  const size_t chunked = augtree_workspace_size(&b.g, AUGTREE_OP_TREE_BWD, 0);
  CHECK(augtree_set_tree_chunk_blocks(1 << 30) == AUGTREE_OK, "chunk blocks set");
  const size_t plain = augtree_workspace_size(&b.g, AUGTREE_OP_TREE_BWD, 0);
  CHECK(chunked > plain, "chunked workspace %zu vs %zu", chunked, plain);
  CHECK(augtree_set_tree_chunk_blocks(1) == AUGTREE_OK, "chunk blocks set");
  fake_set_shape(shape_of(b));
  CHECK(run_impl(fake_scratch_ok, plain) == AUGTREE_OK, "scratch fallback: %s", augtree_last_error());
  expect_clean("scratch fallback schedule");
  expect_slab("scratch fallback", {}, 0);
  CHECK(run_impl(fake_scratch_ok, plain - 1) == AUGTREE_ERR_WORKSPACE, "scratch fallback size check");
  CHECK(augtree_set_tree_chunk_blocks(0) == AUGTREE_OK && augtree_tree_chunk_blocks() == 1024, "default");
}

}  // namespace

int main() {
  check_errors();
  std::vector<Batch> batches;
  batches.push_back(make({256}, {{128, 128}}, 4, 4, 64));                    // the tiny tree
  batches.push_back(make({32768}, {{2048, 2048, 2048, 2048, 2048, 2048, 2048, 2048}}, 32, 8, 128));
  batches.push_back(make({2048}, {std::vector<int>(16, 16384)}, 32, 8, 128));
  batches.push_back(make({1, 2}, {{1, 300}, {5}}, 4, 1, 128));
  batches.push_back(make({700, 130, 256}, {std::vector<int>(12, 5), {200, 129}, {17, 17, 17, 17}}, 8, 2, 128));
  for (int r = 0; r < 40; ++r) {  // random ragged batches
    const int ng = rnd(1, 4);
    std::vector<int> ps;
    std::vector<std::vector<int>> rs;
    for (int g = 0; g < ng; ++g) {
      ps.push_back(rnd(1, r % 3 == 0 ? 3000 : 400));
      std::vector<int> br;
      const int G = rnd(1, r % 5 == 0 ? 40 : 5);
      for (int i = 0; i < G; ++i) br.push_back(rnd(1, r % 4 == 0 ? 2500 : 300));
      rs.push_back(br);
    }
    const int hk = rnd(1, 3);
    batches.push_back(make(ps, rs, hk * (1 + rnd(0, 7)), hk, rnd(0, 1) ? 128 : 64));
  }
  for (const Batch& b : batches) check_batch(b);
  if (g_fail) {
    std::printf("%d failures\n", g_fail);
    return 1;
  }
  std::printf("ok (%zu batches, %d chunked tree backward schedules)\n", batches.size(), g_chunked);
  return 0;
}
