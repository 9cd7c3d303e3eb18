// Host-callable launchers of the gfx950 kernels (internal to libaugtree).
//
// Arrays of two pointers are indexed by the kind of rows or keys a tile
// covers: [0] response rows / branch keys, [1] prompt rows / prompt keys.
// A launch of up to kInlineTiles tiles carries its schedule in the kernel
// arguments (tiles == nullptr), so small launches need no schedule upload.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include "tiles.h"

namespace augtree {

constexpr int kInlineTiles = 32;

struct FwdParams {
  const QTile* tiles;         // device schedule, or nullptr: `inl`
  const uint16_t* q[2];       // [rows, hq, d]
  const uint16_t* ka;         // segment A keys/values (prompt) [*, hkv, d]
  const uint16_t* va;
  const uint16_t* kb[2];      // segment B keys/values of response / prompt rows
  const uint16_t* vb[2];
  uint16_t* o[2];             // bf16 outputs [rows, hq, d] (bf16 kernel)
  float* o32;                 // fp32 partial outputs (fp32 kernel), slot 1 at + o32_part
  int64_t o32_part;
  float* lse[2];              // [hq, lse_rows]; fp32 kernel: lse[0], slot 1 at + lse_part
  int64_t lse_rows[2];
  int64_t lse_part;
  int hq, hkv, group, head_dim;
  float scale_log2;           // softmax_scale * log2(e)
  int n_units;                // tiles x KV heads (set by the launcher)
  QTile inl[kInlineTiles];
};

struct DqParams {
  const QTile* tiles;
  const uint16_t* q[2];
  const uint16_t* dout[2];
  const uint16_t* o[2];       // forward output (bf16): D = rowsum(dO * O) is formed here
  const float* lse[2];        // natural-log LSE [hq, lse_rows]
  float* dsum[2];             // D written here [hq, lse_rows] (read by the dK/dV kernel)
  int64_t lse_rows[2];
  const uint16_t* ka;
  const uint16_t* va;
  const uint16_t* kb[2];
  const uint16_t* vb[2];
  uint16_t* dq[2];            // bf16 [rows, hq, d] (nullable)
  float* dq32[2];             // fp32 (nullable)
  int hq, hkv, group, head_dim;
  float scale, scale_log2;
  int n_units;
  QTile inl[kInlineTiles];
};

struct DkvParams {
  const KVTile* tiles;
  const uint16_t* k[2];       // keys/values [*, hkv, d]: [0] response, [1] prompt
  const uint16_t* v[2];
  const uint16_t* q[2];       // queries [*, hq, d]: [0] response rows, [1] prompt rows
  const uint16_t* dout[2];
  const float* lse[2];        // [hq, lse_rows]
  const float* dsum[2];
  int64_t lse_rows[2];
  uint16_t* dk[2];            // bf16 outputs [*, hkv, d] (KV_OUT_BF16)
  uint16_t* dv[2];
  float* slab;                // fp32 slab [2][slab_rows, hkv, d] (KV_OUT_SLAB; rows per tile: out_row0)
  int64_t slab_rows;
  int hq, hkv, group, head_dim;
  float scale, scale_log2;
  KVTile inl[kInlineTiles];
};

hipError_t launch_attn_fwd(const FwdParams& p, int n_tiles, bool out_f32, hipStream_t stream);
hipError_t launch_attn_dq(const DqParams& p, int n_tiles, hipStream_t stream);
hipError_t launch_attn_dkv(const DkvParams& p, int n_tiles, hipStream_t stream);
// rows row0 .. row0 + rows - 1 of [total_rows]-row tensors
hipError_t launch_lse_merge(int64_t row0, int64_t rows, int64_t total_rows, int heads, int head_dim, int n_parts,
                            const float* o_parts, const float* lse_parts, uint16_t* o, float* o32, float* lse,
                            hipStream_t stream);
// out[t][row] = self[t][row] + sum over k of parts[k][t][src(k, row)] (src =
// row, or row_map[k * rows + row], skipped when negative), tensors t < n_tensors
// written to out[t] (bf16) and/or out32[t] (fp32), each [rows, row_elems]
hipError_t launch_grad_reduce(int n_tensors, int64_t rows, int64_t row_elems, const float* self, int n_parts,
                              int64_t part_rows, int64_t part_stride, const float* parts, const int32_t* row_map,
                              uint16_t* const out[2], float* const out32[2], hipStream_t stream);

inline int fwd_block_m() { return kFwdBlockM; }
inline int fwd_block_n() { return kFwdBlockN; }
inline int dq_block_m() { return kDqBlockM; }
inline int dkv_block_n() { return kDkvBlockN; }
inline int dkv_block_q() { return kDkvBlockQ; }

}  // namespace augtree
