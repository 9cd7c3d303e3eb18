// Shared device-side definitions of the gfx950 kernels.
//
// MFMA tiling used throughout: v_mfma_f32_32x32x16_bf16 (CDNA4), one 64-lane
// wavefront per 32x32 output tile. Lane l holds A row (l % 32) / B column
// (l % 32), eight k values; the 16 accumulator registers of lane l hold
// column (l % 32) and rows
//   row(i) = 8*(i / 4) + 4*(l / 32) + (i % 4),  i = 0..15.
//
// Row statistics of the softmax are computed in the "transposed" orientation
// (S^T = K Q^T puts one query per lane), so row max / row sum are in-lane
// reductions plus one exchange between the two half-waves. The values left in
// the accumulators are fed directly as the B operand of the next MFMA: the
// eight registers 8s..8s+7 of half-wave h cover rows 16s + 4h + {0..3} and
// 16s + 8 + 4h + {0..3}, so the k index of that MFMA runs over those rows, and
// the other operand is fetched from LDS in the same order with the gfx950
// transpose read (TrOffsets).
//
// LDS tiles are row-major, unpadded, with the 16-byte chunks of row r stored
// at chunk index (chunk ^ swz(r)). The LDS has 64 banks of 4 bytes; a 16-byte
// row read serves 16 lanes per cycle (16 consecutive rows, one chunk each)
// and a transpose read 32 lanes (4 consecutive rows x 4 chunks, 8 bytes per
// lane). swz makes both conflict-free: over 16 consecutive rows it is a
// permutation of the chunk indices, and inside every aligned group of 4 rows
// it moves each row to a different aligned group of 4 chunks. (A swizzle
// without the second property makes every transpose read 2-way conflicted;
// the conflict cycles showed in the LDS counters.)
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tiles.h"

namespace augtree {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Accumulator register i of a 32x32 tile -> row inside the tile.
__device__ __forceinline__ int acc_row(int i, int hf) { return ((i >> 2) << 3) + (hf << 2) + (i & 3); }

__device__ __forceinline__ uint4 ldg16(const uint16_t* p) { return *reinterpret_cast<const uint4*>(p); }

__device__ __forceinline__ bf16x8 as_bf16x8(const uint4& v) {
  bf16x8 r;
  __builtin_memcpy(&r, &v, 16);
  return r;
}

// Eight fp32 -> bf16 (round to nearest even; v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ bf16x8 to_bf16x8(const f32x16& v, int base) {
  bf16x8 r;
#pragma unroll
  for (int j = 0; j < 8; ++j) r[j] = (__bf16)v[base + j];
  return r;
}

// acc + the sum of the eight bf16 values of v, in fp32 (v_dot2c_f32_bf16
// against ones: the products are exact).
__device__ __forceinline__ float sum_bf16x8(const bf16x8& v, float acc) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  const bf16x2 one = {(__bf16)1.f, (__bf16)1.f};
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const bf16x2 pair = {v[2 * j], v[2 * j + 1]};
    acc = __builtin_amdgcn_fdot2_f32_bf16(pair, one, acc, false);
  }
  return acc;
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

// ---------------------------------------------------------------------------- swizzled LDS tiles

template <int D>
__device__ __forceinline__ int swz(int row) {
  // D = 128: 16 chunks per row, row = 4a + b -> 4b + a
  if constexpr (D == 128) return ((row & 3) << 2) | ((row >> 2) & 3);
  // D = 64: 8 chunks per row, two rows per 256-byte bank row; row = 4a + 2b + p -> 4b + a
  else return (((row >> 1) & 1) << 2) | ((row >> 2) & 3);
}

// element offset of (row, col) in a swizzled [*, D] tile; col % 4 == 0 keeps
// 8-byte accesses inside one chunk
template <int D>
__device__ __forceinline__ int toff(int row, int col) {
  return row * D + ((((col >> 3) ^ swz<D>(row))) << 3) + (col & 7);
}

// Per-lane byte offsets of the 16-byte row reads of a swizzled [*, D] tile:
// row `row`, columns 16*ks + 8*hf .. +7 for ks = 0 .. D/16 - 1. A read is then
// one ds_read_b128 at (offset register + tile base).
template <int D>
struct RowOffsets {
  int o[D / 16];
  __device__ __forceinline__ void init(int row, int hf) {
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) o[ks] = 2 * toff<D>(row, ks * 16 + hf * 8);
  }
};

template <int D>
__device__ __forceinline__ bf16x8 lds_row8_at(const __bf16* tile, int byte_off) {
  return *reinterpret_cast<const bf16x8*>(reinterpret_cast<const char*>(tile) + byte_off);
}

typedef __attribute__((address_space(3))) const char* lds_cptr;

// Byte address of a __shared__ object inside the workgroup's LDS.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(lds_cptr)(const char*)p;
}

// A value the compiler cannot see through: an LDS address formed as
// opaque(tile base + per-lane offset) is one register, and reads at fixed
// distances from it (a second tile 32 KB further on) become immediate
// offsets of the same register instead of registers of their own. (Without
// it the compiler folds both tile bases into per-lane constants; above 64 KB
// they no longer fit the 16-bit offset field.)
__device__ __forceinline__ uint32_t opaque(uint32_t x) {
  asm("" : "+v"(x));
  return x;
}

// 16-byte read of a __shared__ array `base` at LDS byte address `addr` + IMM
// (addr = opaque(lds_addr(base) + offset)). The pointer is derived from
// `base`, so the access keeps that array's alias scope (the wait inserted
// for in-flight direct-to-LDS copies into other arrays is then not needed),
// and its address is the register `addr` plus an immediate.
template <int IMM = 0>
__device__ __forceinline__ bf16x8 lds_read16(const __bf16* base, uint32_t addr) {
  const char* b = reinterpret_cast<const char*>(base);
  return *reinterpret_cast<const bf16x8*>(b + (addr - lds_addr(base)) + IMM);
}

__device__ __forceinline__ s16x4 lds_tr16(const __bf16* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(p));
}

// MFMA operand whose k index runs along the rows of a swizzled tile (transpose
// reads): lane l gets column c0 + (l % 32) at rows r0 + 4*(l/32) + {0,1,2,3}
// (elements 0..3) and r0 + 8 + 4*(l/32) + {0,1,2,3} (elements 4..7), i.e.
// exactly the rows that accumulator registers 8s..8s+7 of the same half-wave
// hold when r0 = 16 s. Two ds_read_b64_tr_b16: inside each 16-lane group,
// lane j addresses 4 columns of row (j / 4) and receives one column of 4 rows.
// TrOffsets holds the per-lane byte offsets for rows base_row + 16*m
// (+ 0..15) and columns c0 = 32*db: the swizzle depends on the row modulo 16
// only, so 16*m rows are a constant byte offset (16 * m * 2D).
template <int D>
struct TrOffsets {
  int o[D / 32][2];
  __device__ __forceinline__ void init(int base_row, int lane) {
    const int grp = lane >> 4, j = lane & 15;
    const int row = base_row + 4 * (grp >> 1) + (j >> 2);
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
      const int col = 32 * db + 16 * (grp & 1) + 4 * (j & 3);
      o[db][0] = 2 * toff<D>(row, col);
      o[db][1] = 2 * toff<D>(row + 8, col);
    }
  }
  // operand for rows base_row + 16*m .. and columns 32*db ..
  __device__ __forceinline__ bf16x8 read(const __bf16* tile, int m, int db) const {
    const char* t = reinterpret_cast<const char*>(tile) + m * 16 * D * 2;
    const s16x4 a = lds_tr16(reinterpret_cast<const __bf16*>(t + o[db][0]));
    const s16x4 b = lds_tr16(reinterpret_cast<const __bf16*>(t + o[db][1]));
    bf16x8 r;
    __builtin_memcpy(&r, &a, 8);
    __builtin_memcpy(reinterpret_cast<char*>(&r) + 8, &b, 8);
    return r;
  }
};

// Direct global -> LDS copy (buffer_load_dwordx4 ... lds) of a ROWS x D bf16
// tile into a swizzled LDS tile, by NWAVES wavefronts. One instruction writes
// 1 KB of consecutive LDS bytes (lane L at +16 L) = RPI whole rows; lane L
// fills physical chunk L % CH of row L / CH, so it loads logical chunk
// (L % CH) ^ swz(row). The per-lane source byte offsets do not depend on the
// block and are computed once; a block builds a buffer descriptor at its
// (uniform) first row whose range ends after row nvalid - 1, so rows past the
// end read as zeros. The buffer form (not the global form) matters: the
// compiler tracks it on the vector-memory counter only, so LDS reads issued
// while a copy is in flight can still be waited for one at a time.
// Completion: wait_vmem() then a barrier.
template <int ROWS, int D, int NWAVES>
struct TileCopy {
  static constexpr int CH = D / 8, RPI = 64 / CH, NI = ROWS / RPI;
  static constexpr int PER_WAVE = (NI + NWAVES - 1) / NWAVES;
  static_assert(ROWS % RPI == 0, "tile rows");
  uint32_t off[PER_WAVE];  // byte offset of this lane's chunk inside a block of rows
  int wave;                // this wavefront's index (uniform)

  __device__ __forceinline__ void init(int64_t stride) {
    const int lane = threadIdx.x & 63;
    wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
#pragma unroll
    for (int k = 0; k < PER_WAVE; ++k) {
      const int i = wave + k * NWAVES;
      const int row = i * RPI + lane / CH;
      off[k] = 2u * (uint32_t)(row * stride + ((lane % CH) ^ swz<D>(row)) * 8);
    }
  }

  // rows row0 .. row0 + nvalid - 1 (1 <= nvalid) of a [*, stride] tensor,
  // columns col0 .. col0 + D - 1; tile rows from nvalid on are zero
  __device__ __forceinline__ void issue(__bf16* lds, const uint16_t* base, int64_t row0, int nvalid, int64_t stride,
                                        int col0) const {
    issue_at(lds, base + row0 * stride + col0, nvalid, stride);
  }
  // the same from the address of the first row's first column
  __device__ __forceinline__ void issue_at(__bf16* lds, const uint16_t* gb, int nvalid, int64_t stride) const {
    const int rows = nvalid < ROWS ? nvalid : ROWS;
    issue_bytes(lds, gb, (int)(rows * stride * 2));
  }
  // the same with the valid range given in bytes from gb (nbytes: the rows
  // that are read times the row stride in bytes; at most 2^31 - 1)
  __device__ __forceinline__ void issue_bytes(__bf16* lds, const uint16_t* gb, int nbytes) const {
    // Device pass only: with a buffer-resource value in a kernel body, the
    // host pass silently drops the launch stubs of some instantiations.
#if defined(__HIP_DEVICE_COMPILE__)
    const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc((void*)gb, 0, nbytes, 0x00020000);
#pragma unroll
    for (int k = 0; k < PER_WAVE; ++k) {
      const int i = wave + k * NWAVES;
      // every wavefront has PER_WAVE instructions when NWAVES divides NI
      if (NI % NWAVES == 0 || i < NI)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (__attribute__((address_space(3))) void*)(lds + i * RPI * D),
                                                 16, off[k], 0, 0, 0);
    }
#endif
  }
};

// Wait for every outstanding vector-memory access of this wavefront
// (s_waitcnt vmcnt(0)), e.g. direct-to-LDS copies before a barrier.
__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Scheduling of a run of N MFMAs that take R LDS reads each: the reads are
// issued DEPTH MFMAs ahead of the MFMA that consumes them, so the LDS latency
// is covered by matrix work instead of a wait in front of every MFMA. Placed
// after the run, in the same basic block; costs R * DEPTH operand registers.
template <int N, int R, int DEPTH>
__device__ __forceinline__ void pace_lds_mfma() {
  static_assert(DEPTH >= 1, "prefetch depth");
  constexpr int DP = DEPTH < N ? DEPTH : N;
  __builtin_amdgcn_sched_group_barrier(0x100, R * DP, 0);  // DS reads
#pragma unroll
  for (int i = 0; i < N - DP; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);     // MFMA
    __builtin_amdgcn_sched_group_barrier(0x100, R, 0);     // DS reads
  }
  __builtin_amdgcn_sched_group_barrier(0x008, DP, 0);
}

// Issue priority of the wavefront (s_setprio), fenced so that the compiler
// keeps the instructions of each phase on their side of the change. With two
// wavefronts per SIMD, the one that raises its priority is issued first when
// both are ready: the forward raises it for its PV MFMAs, the backward
// kernels for everything but their MFMA runs (softmax, block change), which
// keeps the matrix core fed by one wavefront while the other catches up.
template <int P>
__device__ __forceinline__ void set_wave_priority() {
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_setprio(P);
  __builtin_amdgcn_sched_barrier(0);
}

// max / sum of a value and the one of lane l ^ 32, without LDS: after
// v_permlane32_swap of (x, x) the two results hold, in every lane, x of the
// lane and x of its partner (in one order or the other). An LDS shuffle
// (ds_bpermute) costs an LDS round trip and waits for the wavefront's
// earlier LDS reads.
__device__ __forceinline__ float pair_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// ---------------------------------------------------------------------------- tile schedules

// Tile `i` of a launch: from the device schedule when there is one, else
// from the copy carried in the kernel arguments. Every field is made
// wavefront-uniform (scalar registers), as a plain scalar load of the
// schedule would leave it.
template <class T>
__device__ __forceinline__ T load_tile(const T* tiles, const T* inl, int i) {
  static_assert(sizeof(T) == 32, "tile layout");
  const T t = tiles ? tiles[i] : inl[i];
  int32_t w[8];
  __builtin_memcpy(w, &t, 32);
#pragma unroll
  for (int k = 0; k < 8; ++k) w[k] = __builtin_amdgcn_readfirstlane(w[k]);
  T r;
  __builtin_memcpy(&r, w, 32);
  return r;
}

// ---------------------------------------------------------------------------- workgroup order

// Workgroups are dispatched round-robin over the 8 XCDs (id % 8), each with
// its own L2. Units of `per_unit` consecutive workgroups (the query heads of
// one KV head on one tile) are kept on one XCD, and units are dealt to XCDs
// in schedule order (heaviest first). Returns false for padding workgroups.
__device__ __forceinline__ bool xcd_unit(int n_units, int per_unit, int& unit, int& sub) {
  const int i = blockIdx.x;
  const int x = i & 7, j = i >> 3;
  unit = (j / per_unit) * 8 + x;
  sub = j % per_unit;
  return unit < n_units;
}

__host__ __device__ inline int xcd_grid(int n_units, int per_unit) { return ((n_units + 7) / 8) * 8 * per_unit; }

}  // namespace augtree
