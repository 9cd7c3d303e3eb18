// Host-callable launchers of the gfx950 kernels (internal to libaugtree).
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include "tiles.h"

namespace augtree {

struct FwdParams {
  const QTile* tiles;
  const uint16_t* q;   // [rows, hq, d]
  const uint16_t* ka;  // segment A keys/values [*, hkv, d]
  const uint16_t* va;
  const uint16_t* kb;  // segment B keys/values
  const uint16_t* vb;
  uint16_t* o;         // bf16 output [rows, hq, d] (when out_f32 is false)
  float* o32;          // fp32 output (when out_f32 is true)
  float* lse;          // [hq, lse_rows]
  int64_t lse_rows;
  int hq, hkv, group, head_dim;
  float scale_log2;    // softmax_scale * log2(e)
  int n_units;         // tiles x KV heads (set by the launcher)
};

struct DqParams {
  const QTile* tiles;
  const uint16_t* q;
  const uint16_t* dout;
  const float* lse;    // natural-log LSE [hq, lse_rows]
  const float* dsum;   // D = rowsum(dO * O) [hq, lse_rows]
  const uint16_t* ka;
  const uint16_t* va;
  const uint16_t* kb;
  const uint16_t* vb;
  uint16_t* dq;        // bf16 [rows, hq, d] (nullable)
  float* dq32;         // fp32 (nullable)
  int64_t lse_rows;
  int hq, hkv, group, head_dim;
  float scale, scale_log2;
  int n_units;         // tiles x KV heads (set by the launcher)
};

struct DkvParams {
  const KVTile* tiles;
  const uint16_t* k;     // keys/values of the tile rows [*, hkv, d]
  const uint16_t* v;
  const uint16_t* q;     // queries [*, hq, d]
  const uint16_t* dout;
  const float* lse;      // [hq, lse_rows]
  const float* dsum;     // [hq, lse_rows]
  uint16_t* dk;          // bf16 outputs [*, hkv, d] (when out_f32 is false)
  uint16_t* dv;
  float* dkv32;          // fp32 slabs [part][2][out_rows, hkv, d] (when out_f32 is true)
  int64_t out_rows;
  int64_t lse_rows;
  int hq, hkv, group, head_dim;
  float scale, scale_log2;
};

hipError_t launch_attn_fwd(const FwdParams& p, int n_tiles, bool out_f32, hipStream_t stream);
hipError_t launch_attn_dq(const DqParams& p, int n_tiles, hipStream_t stream);
hipError_t launch_attn_dkv(const DkvParams& p, int n_tiles, bool out_f32, hipStream_t stream);
hipError_t launch_bwd_dsum(const uint16_t* o, const uint16_t* dout, float* dsum, int64_t rows, int hq,
                           int head_dim, hipStream_t stream);
// rows row0 .. row0 + rows - 1 of [total_rows]-row tensors
hipError_t launch_lse_merge(int64_t row0, int64_t rows, int64_t total_rows, int heads, int head_dim, int n_parts,
                            const float* o_parts, const float* lse_parts, uint16_t* o, float* o32, float* lse,
                            hipStream_t stream);
hipError_t launch_grad_reduce(int n_tensors, int64_t rows, int64_t row_elems, const float* self, int n_parts,
                              int64_t part_rows, int64_t part_stride, const float* parts, const int32_t* row_map, uint16_t* out,
                              float* out32, hipStream_t stream);

int fwd_block_m();
int fwd_block_n();
int dq_block_m();
int dkv_block_n();
int dkv_block_q();

}  // namespace augtree
