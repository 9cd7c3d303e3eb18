// Shared device-side definitions of the gfx950 kernels.
//
// MFMA tiling used throughout: v_mfma_f32_32x32x16_bf16 (CDNA4), one 64-lane
// wavefront per 32x32 output tile. Lane l holds A row (l % 32) / B column
// (l % 32), eight consecutive k values at k = 8*(l / 32) .. +7. The 16
// accumulator registers of lane l hold column (l % 32) and rows
//   row(i) = 8*(i / 4) + 4*(l / 32) + (i % 4),  i = 0..15.
//
// Attention is computed in the "transposed" orientation wherever a row
// statistic is needed: S^T = K Q^T puts one query per lane (column), so the
// row max / row sum of the online softmax are in-lane reductions plus one
// exchange between the two half-waves. The probabilities left in the
// accumulator registers are fed directly as the B operand of the next MFMA
// (P^T for O^T = V^T P^T); the other operand is read from LDS with its key
// (or query) index permuted inside each group of 16 to match the accumulator
// row order (see kperm).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tiles.h"

namespace augtree {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Accumulator register i of a 32x32 tile -> row inside the tile.
__device__ __forceinline__ int acc_row(int i, int hf) { return ((i >> 2) << 3) + (hf << 2) + (i & 3); }

// Position of index k inside the LDS row of a transposed operand: inside each
// group of 16, the 8 indices that accumulator registers 0..7 (or 8..15) of a
// half-wave hold become contiguous, so one 16-byte LDS read feeds one MFMA.
__device__ __forceinline__ int kperm(int k) {
  const int k16 = k & 15;
  return (k & ~15) | (((k16 >> 2) & 1) << 3) | ((k16 >> 3) << 2) | (k16 & 3);
}

__device__ __forceinline__ uint4 ldg16(const uint16_t* p) { return *reinterpret_cast<const uint4*>(p); }

__device__ __forceinline__ bf16x8 as_bf16x8(const uint4& v) {
  bf16x8 r;
  __builtin_memcpy(&r, &v, 16);
  return r;
}

__device__ __forceinline__ bf16x8 lds_bf16x8(const __bf16* p) { return *reinterpret_cast<const bf16x8*>(p); }

// Eight fp32 -> bf16 (round to nearest even; v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ bf16x8 to_bf16x8(const f32x16& v, int base) {
  bf16x8 r;
#pragma unroll
  for (int j = 0; j < 8; ++j) r[j] = (__bf16)v[base + j];
  return r;
}

// bf16 element e (0..7) of a 16-byte chunk, as the low 16 bits.
__device__ __forceinline__ uint32_t half16(const uint4& v, int e) {
  uint32_t x;
  switch (e >> 1) {
    case 0: x = v.x; break;
    case 1: x = v.y; break;
    case 2: x = v.z; break;
    default: x = v.w; break;
  }
  return (e & 1) ? (x >> 16) : (x & 0xffffu);
}

// Register-staged copy of a tile of ROWS rows x D bf16 columns into LDS, both
// row-major (row stride RSTR elements) and, optionally, transposed with the
// row index permuted by kperm (row stride TSTR elements). 256 threads; thread
// t owns rows (t / CH) * RPT .. +RPT-1 and 16-byte column chunk t % CH.
template <int ROWS, int D>
struct TileStage {
  static constexpr int CH = D / 8;
  static constexpr int RPT = ROWS * CH / 256;
  static_assert(RPT >= 1 && (RPT == 1 || RPT == 2 || RPT == 4), "rows per thread");
  uint4 r[RPT];

  // rows row0 .. row0+nvalid-1 of a [*, stride] bf16 tensor, column offset col0
  __device__ __forceinline__ void load(const uint16_t* base, int64_t row0, int nvalid, int64_t stride,
                                       int col0) {
    const int tid = threadIdx.x;
    const int rg = tid / CH, dc = tid % CH;
#pragma unroll
    for (int j = 0; j < RPT; ++j) {
      const int rr = rg * RPT + j;
      if (rr < nvalid)
        r[j] = ldg16(base + (row0 + rr) * stride + col0 + dc * 8);
      else
        r[j] = make_uint4(0, 0, 0, 0);
    }
  }

  template <int RSTR>
  __device__ __forceinline__ void store_rows(__bf16* lds) const {
    const int tid = threadIdx.x;
    const int rg = tid / CH, dc = tid % CH;
#pragma unroll
    for (int j = 0; j < RPT; ++j)
      *reinterpret_cast<uint4*>(lds + (rg * RPT + j) * RSTR + dc * 8) = r[j];
  }

  template <int TSTR>
  __device__ __forceinline__ void store_transposed(__bf16* lds) const {
    const int tid = threadIdx.x;
    const int rg = tid / CH, dc = tid % CH;
    const int pos = kperm(rg * RPT);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      __bf16* dst = lds + (dc * 8 + e) * TSTR + pos;
      if constexpr (RPT == 4) {
        uint2 w;
        w.x = half16(r[0], e) | (half16(r[1], e) << 16);
        w.y = half16(r[2], e) | (half16(r[3], e) << 16);
        *reinterpret_cast<uint2*>(dst) = w;
      } else if constexpr (RPT == 2) {
        *reinterpret_cast<uint32_t*>(dst) = half16(r[0], e) | (half16(r[1], e) << 16);
      } else {
        *reinterpret_cast<uint16_t*>(dst) = (uint16_t)half16(r[0], e);
      }
    }
  }
};

}  // namespace augtree
