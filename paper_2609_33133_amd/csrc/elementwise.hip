// HBM-bound kernels: the merge of partial softmax states (§3.3) and the
// fixed-order prompt-gradient sum of Eq. 2.
#include "common.h"
#include "kernels.h"

namespace augtree {

namespace {

typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

// One thread per (row, head, 8-element chunk) of rows row0 .. row0 + rows - 1
// of tensors with total_rows rows (o parts [n][total_rows, heads, d], lse
// parts [n][heads][total_rows], outputs likewise). The part LSEs of a
// (row, head) are read by each of its chunk threads (same cache lines). Parts
// are visited in index order, so the result does not depend on the launch.
__global__ __launch_bounds__(256) void lse_merge_kernel(int64_t row0, int64_t rows, int64_t total_rows, int heads,
                                                        int head_dim, int n_parts,
                                                        const float* __restrict__ o_parts,
                                                        const float* __restrict__ lse_parts,
                                                        uint16_t* __restrict__ o, float* __restrict__ o32,
                                                        float* __restrict__ lse) {
  const int ch_per_row = head_dim / 8;
  const int64_t total = rows * heads * ch_per_row;
  const int64_t part_o = total_rows * heads * head_dim;
  const int64_t part_l = total_rows * heads;
  for (int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; gid < total;
       gid += (int64_t)gridDim.x * blockDim.x) {
    const int64_t rh_local = gid / ch_per_row;
    const int ch = (int)(gid - rh_local * ch_per_row);
    const int64_t row = row0 + rh_local / heads;
    const int h = (int)(rh_local - (row - row0) * heads);
    const int64_t rh = row * heads + h;
    const int64_t lidx = (int64_t)h * total_rows + row;
    float m = -INFINITY;
    for (int k = 0; k < n_parts; ++k) m = fmaxf(m, lse_parts[k * part_l + lidx]);
    float acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.f;
    float out_lse = -INFINITY;
    if (m != -INFINITY) {
      float tot = 0.f;
      for (int k = 0; k < n_parts; ++k) tot += expf(lse_parts[k * part_l + lidx] - m);
      out_lse = m + logf(tot);
      const int64_t ob = rh * head_dim + ch * 8;
      for (int k = 0; k < n_parts; ++k) {
        const float w = expf(lse_parts[k * part_l + lidx] - out_lse);
        const float4 a = *reinterpret_cast<const float4*>(o_parts + k * part_o + ob);
        const float4 b = *reinterpret_cast<const float4*>(o_parts + k * part_o + ob + 4);
        acc[0] += w * a.x; acc[1] += w * a.y; acc[2] += w * a.z; acc[3] += w * a.w;
        acc[4] += w * b.x; acc[5] += w * b.y; acc[6] += w * b.z; acc[7] += w * b.w;
      }
    }
    const int64_t ob = rh * head_dim + ch * 8;
    if (o32) {
      *reinterpret_cast<float4*>(o32 + ob) = make_float4(acc[0], acc[1], acc[2], acc[3]);
      *reinterpret_cast<float4*>(o32 + ob + 4) = make_float4(acc[4], acc[5], acc[6], acc[7]);
    }
    if (o) {
      bf16x8 w;
#pragma unroll
      for (int e = 0; e < 8; ++e) w[e] = (__bf16)acc[e];
      *reinterpret_cast<bf16x8*>(o + ob) = w;
    }
    if (lse && ch == 0) lse[lidx] = out_lse;
  }
}

// One thread per 4 consecutive elements of one output row of one tensor.
__global__ __launch_bounds__(256) void grad_reduce_kernel(int n_tensors, int64_t rows, int64_t row_elems,
                                                          const float* __restrict__ self, int n_parts,
                                                          int64_t part_rows, int64_t part_stride,
                                                          const float* __restrict__ parts,
                                                          const int32_t* __restrict__ row_map,
                                                          uint16_t* out0, uint16_t* out1, float* o32_0,
                                                          float* o32_1) {
  const int64_t q_per_row = row_elems / 4;
  const int64_t total = (int64_t)n_tensors * rows * q_per_row;
  for (int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; gid < total;
       gid += (int64_t)gridDim.x * blockDim.x) {
    const int64_t tr = gid / q_per_row;
    const int64_t e = (gid - tr * q_per_row) * 4;
    const int64_t tsr = tr / rows;
    const int64_t row = tr - tsr * rows;
    float4 acc = self ? *reinterpret_cast<const float4*>(self + tr * row_elems + e) : make_float4(0, 0, 0, 0);
    for (int k = 0; k < n_parts; ++k) {
      const int64_t src = row_map ? (int64_t)row_map[(int64_t)k * rows + row] : row;
      if (src < 0) continue;
      const float4 v =
          *reinterpret_cast<const float4*>(parts + (int64_t)k * part_stride + (tsr * part_rows + src) * row_elems + e);
      acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
    }
    float* const out32 = tsr ? o32_1 : o32_0;
    uint16_t* const out = tsr ? out1 : out0;
    if (out32) *reinterpret_cast<float4*>(out32 + row * row_elems + e) = acc;
    if (out) {
      bf16x4 w;
      w[0] = (__bf16)acc.x; w[1] = (__bf16)acc.y; w[2] = (__bf16)acc.z; w[3] = (__bf16)acc.w;
      *reinterpret_cast<bf16x4*>(out + row * row_elems + e) = w;
    }
  }
}

unsigned grid_for(int64_t threads) {
  const int64_t blocks = (threads + 255) / 256;
  const int64_t cap = 256 * 64;  // 64 workgroups per CU is plenty for a grid-stride loop
  return (unsigned)(blocks < cap ? (blocks > 0 ? blocks : 1) : cap);
}

}  // namespace

hipError_t launch_lse_merge(int64_t row0, int64_t rows, int64_t total_rows, int heads, int head_dim, int n_parts,
                            const float* o_parts, const float* lse_parts, uint16_t* o, float* o32, float* lse,
                            hipStream_t stream) {
  const int64_t threads = rows * heads * (head_dim / 8);
  if (threads == 0) return hipSuccess;
  hipLaunchKernelGGL(lse_merge_kernel, dim3(grid_for(threads)), dim3(256), 0, stream, row0, rows, total_rows, heads,
                     head_dim, n_parts, o_parts, lse_parts, o, o32, lse);
  return hipGetLastError();
}

hipError_t launch_grad_reduce(int n_tensors, int64_t rows, int64_t row_elems, const float* self, int n_parts,
                              int64_t part_rows, int64_t part_stride, const float* parts, const int32_t* row_map,
                              uint16_t* const out[2], float* const out32[2], hipStream_t stream) {
  const int64_t threads = (int64_t)n_tensors * rows * (row_elems / 4);
  if (threads == 0) return hipSuccess;
  hipLaunchKernelGGL(grad_reduce_kernel, dim3(grid_for(threads)), dim3(256), 0, stream, n_tensors, rows,
                     row_elems, self, n_parts, part_rows, part_stride, parts, row_map, out[0], out[1], out32[0],
                     out32[1]);
  return hipGetLastError();
}

}  // namespace augtree
