// Tile descriptors shared by the host schedule builder and the kernels.
#pragma once

#include <stdint.h>

namespace augtree {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Query tile of the forward and dQ kernels: up to BM query rows, attending to
// segment A (every key visible) and then segment B (causal: query i of the
// tile sits at segment position b_qpos + i and sees keys 0 .. b_qpos + i).
struct QTile {
  int32_t q_row0, q_len;
  int32_t a_row0, a_len;
  int32_t b_row0, b_len, b_qpos;
  int32_t pad;
};

// Key tile of the dK/dV kernel: up to 128 keys of one KV head against a
// range of query rows. Causal tiles: key j of the tile sits at position
// kpos0 + j of its segment, query i of the range at qpos0 + i, visible iff
// kpos0 + j <= qpos0 + i. Output rows are the key rows; fp32 outputs go to
// slab `part`.
struct KVTile {
  int32_t kv_row0, kv_len;
  int32_t q_row0, q_len;
  int32_t causal, kpos0, qpos0;
  int32_t part;
};

}  // namespace augtree
