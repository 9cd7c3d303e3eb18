// Tile descriptors shared by the host schedule builder and the kernels.
#pragma once

#include <stdint.h>

namespace augtree {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Tile sizes of the kernels (the host schedules are cut to them).
constexpr int kFwdBlockM = 128;   // forward: query rows per tile
constexpr int kFwdBlockN = 64;    // forward: keys per block
constexpr int kDqBlockM = 128;    // dQ: query rows per tile
constexpr int kDqBlockN = 64;     // dQ: keys per block
constexpr int kDkvBlockN = 128;   // dK/dV: keys per tile
constexpr int kDkvBlockQ = 64;    // dK/dV: query rows per block

// Query tile of the forward and dQ kernels: up to BM query rows, attending to
// segment A (prompt keys, every key visible) and then segment B (causal:
// query i of the tile sits at segment position b_qpos + i and sees keys
// 0 .. b_qpos + i).
struct QTile {
  int32_t q_row0, q_len;
  int32_t a_row0, a_len;
  int32_t b_row0, b_len, b_qpos;
  int32_t flags;  // QT_*
};

enum : int32_t {
  // the query rows are prompt rows (Q_P, O_P, LSE_P; segment B = prompt
  // keys); otherwise response rows (Q_R, O_R, LSE_R; segment B = the
  // branch's own keys)
  QT_PROMPT_ROWS = 1,
  // fp32 partial outputs: write the second partial slot (own-branch partial)
  QT_PART1 = 2,
};

// Key tile of the dK/dV kernel: up to 128 keys of one KV head against up to
// two ranges of query rows, swept in this order:
//   X: response rows x_row0 .. x_row0 + x_len - 1 (Q_R, dO_R, LSE_R, D_R),
//      causal if KV_X_CAUSAL, otherwise every key visible;
//   Y: prompt rows kv_row0 .. kv_row0 + y_len - 1 (Q_P, ...), causal (prompt
//      keys only: prompt queries before the tile's first key cannot see it).
// In a causal range, query i sits at position kpos0 + i of its segment (the
// range starts at the tile's first key) and key j at kpos0 + j: visible iff
// j <= i. Outputs: the key rows' dK/dV in bf16 (KV_OUT_BF16, rows kv_row0 ..)
// and/or fp32 (KV_OUT_SLAB): dK of key j at row out_row0 + j of the fp32 slab,
// dV slab_rows rows further on.
struct KVTile {
  int32_t kv_row0, kv_len;
  int32_t x_row0, x_len;
  int32_t y_len;
  int32_t kpos0;
  int32_t out_row0;
  int32_t flags;  // KV_*
};

enum : int32_t {
  KV_PROMPT_KEYS = 1,  // keys K_P/V_P (outputs dK_P/dV_P); otherwise K_R/V_R
  KV_X_CAUSAL = 2,
  KV_OUT_BF16 = 4,
  KV_OUT_SLAB = 8,
};

}  // namespace augtree
