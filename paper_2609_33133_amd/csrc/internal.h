// Host-side declarations shared between the library's translation units
// (internal to libaugtree).
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "../../include/augtree.h"

namespace augtree {

// Supplies the device buffer of a call that brings none: stores it in *ws,
// returns an augtree_status.
typedef int (*ScratchFn)(void** ws);

// augtree_tree_bwd with its workspace either given (scratch == nullptr: ws,
// ws_bytes) or taken from `scratch` (a fixed device array of ws_bytes bytes;
// the size check runs before the device is touched).
int tree_bwd_impl(const augtree_groups* grp, const uint16_t* q_p, const uint16_t* k_p, const uint16_t* v_p,
                  const uint16_t* o_p, const float* lse_p, const uint16_t* do_p, const uint16_t* q_r,
                  const uint16_t* k_r, const uint16_t* v_r, const uint16_t* o_r, const float* lse_r,
                  const uint16_t* do_r, uint16_t* dq_p, uint16_t* dk_p, uint16_t* dv_p, float* dkv_p_f32,
                  uint16_t* dq_r, uint16_t* dk_r, uint16_t* dv_r, ScratchFn scratch, void* ws, size_t ws_bytes,
                  void* stream);

// Records `msg` as the calling thread's last error; returns `status`.
int fail_status(int status, const char* msg);

// Chunks of the tree backward's prompt-key sweep over a group's `nr` branch
// rows (each chunk at most augtree_set_tree_chunk_blocks query blocks of 64
// rows x one of the `group` query heads; between 1 and 64).
constexpr int kTreeChunkBlocksDefault = 1024;
int tree_chunk_count(int64_t nr, int group);

}  // namespace augtree
