// CPU stand-ins for the HIP runtime calls and kernel launchers the host part
// of libaugtree uses, for testing its host logic (validation, schedules,
// error paths) without a GPU, under AddressSanitizer.
//
// * The "device" is host memory: the schedule upload copies into the
//   caller's workspace buffer, which is host memory here.
// * Each launcher checks every tile of its launch against the batch shape set
//   by fake_set_shape (rows and key ranges inside the tensors, causal
//   geometry), marks the output rows it writes (every output row of a launch
//   must be written exactly once) and adds up the visible (query, key) pairs,
//   which the test compares with the counts of the method's definitions.
// * fake_fail_at(n) makes the n-th launch (counting from 1) or copy report
//   a HIP error, to exercise the library's error path.
#include "fake_hip.h"

#include <hip/hip_runtime_api.h>

#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <string>
#include <vector>

#include "kernels.h"

using namespace augtree;

namespace {

FakeShape g_shape;
long g_calls = 0, g_fail_at = 0;
FakeCounts g_counts;
std::vector<std::string> g_errors;

void err(const std::string& s) { g_errors.push_back(s); }

bool fail_now() { return g_fail_at > 0 && ++g_calls == g_fail_at; }

// coverage of output rows: key = (output name), value = per-row write count
std::map<std::string, std::vector<int>> g_cov;
// fp32 slab rows written by dK/dV tiles (KV_OUT_SLAB), by slab row
std::vector<int> g_slab;
// the workspace of the entry point under test (host memory here)
const char* g_ws = nullptr;
size_t g_ws_bytes = 0;

void cover(const std::string& name, int64_t rows, int64_t r0, int64_t n) {
  auto& v = g_cov[name];
  if ((int64_t)v.size() != rows) v.assign(rows, 0);
  if (r0 < 0 || n < 0 || r0 + n > rows) {
    err(name + ": rows out of range");
    return;
  }
  for (int64_t r = r0; r < r0 + n; ++r) v[r] += 1;
}

template <class T>
std::vector<T> tiles_of(const T* tiles, const T* inl, int n) {
  if (!tiles) {
    if (n > kInlineTiles) err("inline schedule longer than the kernel-argument copy");
    return std::vector<T>(inl, inl + std::min(n, kInlineTiles));
  }
  return std::vector<T>(tiles, tiles + n);
}

// segment of packed rows [r0, r0 + n) inside one group's prompt or one
// branch (returns the segment start, or -1)
int64_t seg_start(const std::vector<int32_t>& cu, int64_t r0, int64_t n) {
  for (size_t i = 0; i + 1 < cu.size(); ++i)
    if (r0 >= cu[i] && r0 + n <= cu[i + 1]) return cu[i];
  return -1;
}

}  // namespace

void fake_set_shape(const FakeShape& s) {
  g_shape = s;
  g_cov.clear();
  g_slab.clear();
  g_counts = FakeCounts{};
  g_errors.clear();
}
void fake_fail_at(long n) {
  g_fail_at = n;
  g_calls = 0;
}
const FakeCounts& fake_counts() { return g_counts; }
const std::vector<std::string>& fake_errors() { return g_errors; }

// every output row of the launches since the last call written exactly once
void fake_check_coverage(const char* name, int64_t rows) {
  auto it = g_cov.find(name);
  if (it == g_cov.end()) {
    if (rows > 0) err(std::string(name) + ": never written");
    return;
  }
  for (int64_t r = 0; r < rows; ++r)
    if (it->second[r] != 1) {
      err(std::string(name) + ": row " + std::to_string(r) + " written " + std::to_string(it->second[r]) + " times");
      return;
    }
}
void fake_reset_coverage() {
  g_cov.clear();
  g_slab.clear();
}
void fake_set_workspace(const void* ws, size_t bytes) {
  g_ws = static_cast<const char*>(ws);
  g_ws_bytes = bytes;
}
const std::vector<int>& fake_slab_rows() { return g_slab; }

// ------------------------------------------------------------------ HIP runtime

extern "C" {

hipError_t hipGetDevice(int* d) {
  *d = 0;
  return hipSuccess;
}

hipError_t hipGetDevicePropertiesR0600(hipDeviceProp_tR0600* p, int) {
  std::memset(p, 0, sizeof(*p));
  std::strcpy(p->gcnArchName, "gfx950:sramecc+:xnack-");
  return hipSuccess;
}

const char* hipGetErrorString(hipError_t e) { return e == hipSuccess ? "no error" : "injected failure"; }

hipError_t hipMemcpyAsync(void* dst, const void* src, size_t n, hipMemcpyKind, hipStream_t) {
  if (fail_now()) return hipErrorOutOfMemory;
  std::memcpy(dst, src, n);
  return hipSuccess;
}

}  // extern "C"

// ------------------------------------------------------------------ launchers

namespace augtree {

hipError_t launch_attn_fwd(const FwdParams& p, int n_tiles, bool out_f32, hipStream_t) {
  if (fail_now()) return hipErrorLaunchFailure;
  const FakeShape& s = g_shape;
  for (const QTile& t : tiles_of(p.tiles, p.inl, n_tiles)) {
    const bool prow = t.flags & QT_PROMPT_ROWS;
    const int64_t rows = prow ? s.tp : s.tr;
    if (t.q_len < 1 || t.q_len > kFwdBlockM) err("fwd: tile rows");
    if (t.a_len > 0 && seg_start(s.cu_prompt, t.a_row0, t.a_len) != t.a_row0) err("fwd: segment A is not a prompt");
    if (t.b_len > 0) {
      const auto& cu = prow ? s.cu_prompt : s.cu_resp;
      if (seg_start(cu, t.b_row0, t.b_len) != t.b_row0) err("fwd: segment B outside its segment");
      if (t.b_qpos + t.q_len != t.b_len || t.b_row0 + t.b_qpos != t.q_row0) err("fwd: causal geometry");
    }
    const char* out = out_f32 ? ((t.flags & QT_PART1) ? "fwd_part1" : "fwd_part0") : (prow ? "o_p" : "o_r");
    cover(out, rows, t.q_row0, t.q_len);
    for (int i = 0; i < t.q_len; ++i) g_counts.fwd_pairs += t.a_len + (t.b_len > 0 ? t.b_qpos + i + 1 : 0);
  }
  g_counts.launches++;
  return hipSuccess;
}

hipError_t launch_attn_dq(const DqParams& p, int n_tiles, hipStream_t) {
  if (fail_now()) return hipErrorLaunchFailure;
  const FakeShape& s = g_shape;
  for (const QTile& t : tiles_of(p.tiles, p.inl, n_tiles)) {
    const bool prow = t.flags & QT_PROMPT_ROWS;
    if (t.q_len < 1 || t.q_len > kDqBlockM) err("dq: tile rows");
    if (t.a_len > 0 && seg_start(s.cu_prompt, t.a_row0, t.a_len) != t.a_row0) err("dq: segment A is not a prompt");
    const auto& cu = prow ? s.cu_prompt : s.cu_resp;
    if (t.b_len < 1 || seg_start(cu, t.b_row0, t.b_len) != t.b_row0) err("dq: segment B outside its segment");
    if (t.b_qpos + t.q_len != t.b_len || t.b_row0 + t.b_qpos != t.q_row0) err("dq: causal geometry");
    if (!(prow ? p.dq[1] || p.dq32[1] : p.dq[0] || p.dq32[0])) err("dq: no output");
    cover(prow ? "dq_p" : "dq_r", prow ? s.tp : s.tr, t.q_row0, t.q_len);
    for (int i = 0; i < t.q_len; ++i) g_counts.dq_pairs += t.a_len + t.b_qpos + i + 1;
  }
  g_counts.launches++;
  return hipSuccess;
}

hipError_t launch_attn_dkv(const DkvParams& p, int n_tiles, hipStream_t) {
  if (fail_now()) return hipErrorLaunchFailure;
  const FakeShape& s = g_shape;
  for (const KVTile& t : tiles_of(p.tiles, p.inl, n_tiles)) {
    const bool pk = t.flags & KV_PROMPT_KEYS;
    const auto& kcu = pk ? s.cu_prompt : s.cu_resp;
    const int64_t kstart = seg_start(kcu, t.kv_row0, t.kv_len);
    if (t.kv_len < 1 || t.kv_len > kDkvBlockN || kstart < 0) err("dkv: key tile outside its segment");
    if (t.kpos0 != t.kv_row0 - kstart) err("dkv: key position");
    if (t.x_len > 0 && (t.x_row0 < 0 || t.x_row0 + t.x_len > s.tr)) err("dkv: response rows out of range");
    if (t.y_len > 0) {
      if (!pk || seg_start(s.cu_prompt, t.kv_row0, t.y_len) < 0) err("dkv: prompt rows");
    }
    if ((t.flags & KV_X_CAUSAL) && (pk || t.x_row0 != t.kv_row0 || seg_start(s.cu_resp, t.x_row0, t.x_len) < 0))
      err("dkv: causal response rows");
    const int64_t rows = pk ? s.tp : s.tr;
    if (t.flags & KV_OUT_BF16) {
      if (!p.dk[pk] || !p.dv[pk]) err("dkv: no bf16 output");
      cover(pk ? "dk_p" : "dk_r", rows, t.kv_row0, t.kv_len);
    }
    if (t.flags & KV_OUT_SLAB) {
      // dK rows must leave room for the dV rows slab_rows further on; the
      // seed layout [part][2][T_P] reaches 2 x 64 x T_P rows
      if (!p.slab || !pk || t.out_row0 < 0 || t.out_row0 + t.kv_len > p.slab_rows * 128) err("dkv: slab output");
      if ((int64_t)g_slab.size() < (int64_t)t.out_row0 + t.kv_len) g_slab.resize(t.out_row0 + t.kv_len, 0);
      for (int j = 0; j < t.kv_len; ++j) g_slab[t.out_row0 + j] += 1;
    }
    for (int j = 0; j < t.kv_len; ++j) {
      const int64_t xs = (t.flags & KV_X_CAUSAL) ? std::max<int64_t>(0, t.x_len - j) : t.x_len;
      const int64_t ys = std::max<int64_t>(0, t.y_len - j);
      g_counts.dkv_pairs += xs + ys;
    }
  }
  g_counts.launches++;
  return hipSuccess;
}

hipError_t launch_lse_merge(int64_t row0, int64_t rows, int64_t total_rows, int, int, int n_parts, const float*,
                            const float*, uint16_t*, float*, float*, hipStream_t) {
  if (fail_now()) return hipErrorLaunchFailure;
  if (row0 < 0 || rows < 0 || row0 + rows > total_rows || n_parts < 1) err("merge: rows");
  cover("merge", total_rows, row0, rows);
  g_counts.launches++;
  return hipSuccess;
}

hipError_t launch_grad_reduce(int n_tensors, int64_t rows, int64_t, const float*, int n_parts, int64_t part_rows,
                              int64_t, const float*, const int32_t* row_map, uint16_t* const out[2],
                              float* const out32[2], hipStream_t) {
  if (fail_now()) return hipErrorLaunchFailure;
  if (n_tensors < 1 || rows < 0 || n_parts < 0) err("reduce: arguments");
  for (int t = 0; t < n_tensors; ++t)
    if (!out[t] && !out32[t]) err("reduce: tensor without output");
  const char* rm = reinterpret_cast<const char*>(row_map);
  if (row_map && g_ws && rm >= g_ws && rm + (size_t)n_parts * rows * 4 <= g_ws + g_ws_bytes) {
    // a map the library built: every row has its first term, and the mapped
    // source rows are exactly the slab rows the dK/dV tiles wrote, each once
    std::vector<int> used(part_rows, 0);
    for (int64_t r = 0; r < rows; ++r) {
      if (row_map[r] < 0) err("reduce: row without a first term");
      for (int k = 0; k < n_parts; ++k) {
        const int32_t v = row_map[(int64_t)k * rows + r];
        if (v < -1 || v >= part_rows) {
          err("reduce: source row out of range");
          return hipSuccess;
        }
        if (v >= 0) used[v] += 1;
      }
    }
    for (int64_t v = 0; v < part_rows; ++v) {
      const int w = v < (int64_t)g_slab.size() ? g_slab[v] : 0;
      if (used[v] != 1 || w != 1) {
        err("reduce: slab row " + std::to_string(v) + " mapped " + std::to_string(used[v]) + " times, written " +
            std::to_string(w) + " times");
        break;
      }
    }
    cover("dk_p", rows, 0, rows);
  }
  g_counts.launches++;
  return hipSuccess;
}

}  // namespace augtree
