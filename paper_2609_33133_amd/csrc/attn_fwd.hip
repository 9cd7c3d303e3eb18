// Forward attention kernel for gfx950: prompt prefill, fused response replay
// and the split-mode partials (§3.2, Eq. 1, §3.3).
//
// One workgroup = 4 wavefronts = one query tile of up to 128 rows of one
// query head; each wavefront owns 32 query rows (one per lane column of the
// S^T accumulator). The tile sweeps 64-key blocks of segment A (the prompt
// KV, every key visible) and then of segment B (causal). Continuing the
// online softmax across the two segments is the log-sum-exp merge of the two
// partial states done in registers; a tile with only one segment produces one
// partial state (split mode).
//
// Per 64-key block and wavefront: 16 MFMAs for S^T = K Q^T (K rows from LDS,
// Q^T held in registers), the online-softmax update in fp32 with exp2 (the
// output is rescaled only when a row maximum grows), and 16 MFMAs for
// O^T += V^T P^T (V^T by transpose reads of the row-major V tile, P^T straight
// from the S^T accumulators rounded to bf16). The loop is software-pipelined:
// the S MFMAs of block b + 1 are interleaved one by one with the exponentials
// of block b (explicit scheduling groups), so one wavefront keeps the matrix
// cores and the vector ALUs busy together. LDS addresses come from per-lane
// offset tables computed once, and operand reads run a few MFMAs ahead of
// their MFMA. K and V tiles are double-buffered in LDS (separate arrays, loop
// unrolled by two, so the compiler can tell the buffer being filled from the
// one being read) and copied there directly from global memory
// (buffer_load ... lds), so no registers hold staged data. Two workgroups
// share a CU (two wavefronts per SIMD).
#include "common.h"
#include "kernels.h"

namespace augtree {

namespace {

constexpr int BM = kFwdBlockM;  // query rows per workgroup
constexpr int BN = kFwdBlockN;  // keys per block
constexpr int FWD_DEPTH = 4;  // LDS operand reads run this many MFMAs ahead
constexpr int PV_DEPTH = 3;   // the same for the P V MFMAs (two reads each)
constexpr int FWD_VALU_PER_MFMA = 7;  // softmax instructions placed after each S MFMA
// The exponent reference of a row (its running maximum) moves only when a
// block's maximum exceeds it by more than this many powers of two. Exact: the
// reference cancels between numerator and denominator; P stays <= 2^8, far
// inside the fp32 and bf16 ranges.
constexpr float RESCALE_MARGIN_LOG2 = 8.f;

template <int D, bool OUT32>
__global__ __launch_bounds__(256, 2) void attn_fwd_kernel(FwdParams p) {
  __shared__ __bf16 k_buf0[BN * D], k_buf1[BN * D], v_buf0[BN * D], v_buf1[BN * D];
  int unit, hh;
  if (!xcd_unit(p.n_units, p.group, unit, hh)) return;
  const int tid = threadIdx.x, lane = tid & 63, l32 = lane & 31, hf = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar branches below
  const int tile_id = unit / p.hkv;
  const int kvh = unit - tile_id * p.hkv;
  const int head = kvh * p.group + hh;
  const QTile t = load_tile(p.tiles, p.inl, tile_id);
  // prompt rows (prefill) or response rows (replay): tensors of the tile
  const bool prow = (t.flags & QT_PROMPT_ROWS) != 0;
  const uint16_t* const qsrc = prow ? p.q[1] : p.q[0];
  const uint16_t* const kb = prow ? p.kb[1] : p.kb[0];
  const uint16_t* const vb = prow ? p.vb[1] : p.vb[0];
  const int qi = wave * 32 + l32;
  const bool qvalid = qi < t.q_len;
  const int64_t qrow = (int64_t)t.q_row0 + qi;
  const int64_t qstride = (int64_t)p.hq * D;
  const int64_t kvstride = (int64_t)p.hkv * D;

  // Q^T operand (B of S^T = K Q^T): lane holds query qi, d = 16*ks + 8*hf .. +7
  bf16x8 qreg[D / 16];
  {
    const uint16_t* qp = qsrc + qrow * qstride + head * D + hf * 8;
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks)
      qreg[ks] = as_bf16x8(qvalid ? ldg16(qp + ks * 16) : make_uint4(0, 0, 0, 0));
  }

  const float c = p.scale_log2;
  float m_run = -INFINITY;  // running max of raw q.k over this lane's query
  float l_run = 0.f;        // this half-wave's share of the running sum
  f32x16 oacc[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) oacc[db][i] = 0.f;

  const int nA = (t.a_len + BN - 1) / BN;
  const int nB = (t.b_len + BN - 1) / BN;
  const int nblk = nA + nB;

  TileCopy<BN, D, 4> cp;
  cp.init(kvstride);
  // K / V of both segments at the segment's first row and this KV head
  const char* const ka0 = reinterpret_cast<const char*>(p.ka + (int64_t)t.a_row0 * kvstride + kvh * D);
  const char* const va0 = reinterpret_cast<const char*>(p.va + (int64_t)t.a_row0 * kvstride + kvh * D);
  const char* const kb0p = reinterpret_cast<const char*>(kb + (int64_t)t.b_row0 * kvstride + kvh * D);
  const char* const vb0p = reinterpret_cast<const char*>(vb + (int64_t)t.b_row0 * kvstride + kvh * D);
  // Load cursors of K and V: the next block of each to be copied into LDS,
  // stepped in place, so that a block's scalar work is a few adds (the
  // eight wavefronts of a CU share one scalar unit)
  struct KvCursor {
    int isB, kb0, len;  // segment (0: A, 1: B), the block's first key in it, the segment's length
    const char* src;    // the block's first key row, KV head kvh
  };
  const int row_bytes = (int)(kvstride * 2);
  KvCursor kcur = nA > 0 ? KvCursor{0, 0, t.a_len, ka0} : KvCursor{1, 0, t.b_len, kb0p};
  KvCursor vcur = nA > 0 ? KvCursor{0, 0, t.a_len, va0} : KvCursor{1, 0, t.b_len, vb0p};
  // copy the cursor's block into dst and step the cursor (past the end of
  // segment B: never loaded)
  auto load_next = [&](KvCursor& c, const char* seg_b, __bf16* dst) {
    cp.issue_bytes(dst, reinterpret_cast<const uint16_t*>(c.src), min(BN, c.len - c.kb0) * row_bytes);
    int64_t step = (int64_t)BN * row_bytes;
    c.kb0 += BN;
    if (c.kb0 >= c.len && c.isB == 0) {
      step = seg_b - c.src;
      c.isB = 1;
      c.kb0 = 0;
      c.len = t.b_len;
    }
    c.src += step;
  };
  auto load_k = [&](__bf16* dst) { load_next(kcur, kb0p, dst); };
  auto load_v = [&](__bf16* dst) { load_next(vcur, vb0p, dst); };

  RowOffsets<D> k_off;  // K row l32; row 32 + l32 has the same swizzle, 32 rows further
  k_off.init(l32, hf);
  TrOffsets<D> vtr_off;  // V^T operands
  vtr_off.init(0, lane);
  const int qpos_lo = t.b_qpos + wave * 32;  // causal: the wavefront's first query position

  // a causal block whose keys all follow the wavefront's queries (and every
  // later block) contributes nothing
  auto skipped = [&](int b) { return b >= nA && (b - nA) * BN > qpos_lo + 31; };

  // S^T of one 64-key block (two 32-key halves), raw scores
  auto s_mfma = [&](const __bf16* kl, f32x16& s0, f32x16& s1) {
#pragma unroll
    for (int i = 0; i < 16; ++i) { s0[i] = 0.f; s1[i] = 0.f; }
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) {
      s0 = mfma32(lds_row8_at<D>(kl, k_off.o[ks]), qreg[ks], s0);
      s1 = mfma32(lds_row8_at<D>(kl + 32 * D, k_off.o[ks]), qreg[ks], s1);
    }
  };

  // mask, running max and (when it grew) rescale for block b; returns the
  // exponent offset of the block
  auto stats = [&](int b, f32x16& s0, f32x16& s1) -> float {
    const bool isB = b >= nA;
    const int kb0 = (isB ? b - nA : b) * BN;
    const int len = isB ? t.b_len : t.a_len;
    if ((kb0 + BN > len) || (isB && (kb0 + BN - 1 > qpos_lo))) {
      const int lim = min(len - 1, isB ? t.b_qpos + qi : len - 1) - kb0;  // last visible key of the block
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        if (acc_row(i, hf) > lim) s0[i] = -INFINITY;
        if (acc_row(i, hf) + 32 > lim) s1[i] = -INFINITY;
      }
    }
    // four independent chains of three-input maxima (v_max3_f32, written
    // out: left to itself the compiler pairs the values with two-input maxima
    // first and needs about a third more instructions), and the half-wave
    // exchange without LDS
    auto max3 = [](float a, float b, float c) {
      float r;
      asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
      return r;
    };
    float m4[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float m = max3(s0[j], s1[j], s0[j + 4]);
      m = max3(m, s1[j + 4], s0[j + 8]);
      m = max3(m, s1[j + 8], s0[j + 12]);
      m4[j] = fmaxf(m, s1[j + 12]);
    }
    const float mx = pair_max(fmaxf(max3(m4[0], m4[1], m4[2]), m4[3]));
    const float mnew = fmaxf(m_run, mx);
    // rescale only when some row maximum of this wavefront passed its
    // reference by more than the margin (always on a row's first visible key:
    // the reference starts at -inf)
    if (__any(mx * c > m_run * c + RESCALE_MARGIN_LOG2)) {
      const float alpha = (mnew == -INFINITY) ? 1.f : __builtin_amdgcn_exp2f((m_run - mnew) * c);
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int i = 0; i < 16; ++i) oacc[db][i] *= alpha;
      m_run = mnew;
    }
    return (m_run == -INFINITY) ? 0.f : m_run * c;
  };

  // One block step. Scores S(b) arrive in s0/s1 (computed one step earlier);
  // the S MFMAs of block b + 1 (from kn, into n0/n1) are interleaved one by
  // one with the exponentials, row sums and bf16 conversion of block b, so the
  // matrix cores and the vector ALUs of the wavefront work at the same time;
  // then O += V(b)^T P(b)^T. On the last block the extra S is computed from a
  // stale buffer and never used.
  auto step = [&](int b, f32x16& s0, f32x16& s1, const __bf16* kn, const __bf16* vl, f32x16& n0, f32x16& n1) {
    const float ms = stats(b, s0, s1);
    __builtin_amdgcn_sched_barrier(0);
    s_mfma(kn, n0, n1);
    float l4[4];  // four independent partial sums
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      s0[i] = __builtin_amdgcn_exp2f(s0[i] * c - ms);
      s1[i] = __builtin_amdgcn_exp2f(s1[i] * c - ms);
      l4[i & 3] = i < 4 ? s0[i] + s1[i] : l4[i & 3] + (s0[i] + s1[i]);
    }
    l_run += (l4[0] + l4[1]) + (l4[2] + l4[3]);
    const bf16x8 pb0 = to_bf16x8(s0, 0), pb1 = to_bf16x8(s0, 8);
    const bf16x8 pb2 = to_bf16x8(s1, 0), pb3 = to_bf16x8(s1, 8);
    // 16 MFMAs with one K read each (reads run FWD_DEPTH ahead), the ~112
    // vector instructions of the softmax spread over them
    __builtin_amdgcn_sched_group_barrier(0x100, FWD_DEPTH, 0);
#pragma unroll
    for (int i = 0; i < D / 8; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      if (i < D / 8 - FWD_DEPTH) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x402, FWD_VALU_PER_MFMA, 0);
    }
    set_wave_priority<1>();
    // k-step outer, output column block inner: consecutive MFMAs go to
    // different accumulators (each still sums its four k-steps in order)
#pragma unroll
    for (int db = 0; db < D / 32; ++db) oacc[db] = mfma32(vtr_off.read(vl, 0, db), pb0, oacc[db]);
#pragma unroll
    for (int db = 0; db < D / 32; ++db) oacc[db] = mfma32(vtr_off.read(vl, 1, db), pb1, oacc[db]);
#pragma unroll
    for (int db = 0; db < D / 32; ++db) oacc[db] = mfma32(vtr_off.read(vl, 2, db), pb2, oacc[db]);
#pragma unroll
    for (int db = 0; db < D / 32; ++db) oacc[db] = mfma32(vtr_off.read(vl, 3, db), pb3, oacc[db]);
    pace_lds_mfma<D / 8, 2, PV_DEPTH>();
    set_wave_priority<0>();
  };

  // K(b + 1) and V(b) are resident while block b is processed; iteration b
  // loads K(b + 2) over K(b) and V(b + 1) over V(b - 1).
  f32x16 sa0, sa1, sb0, sb1;
  if (nblk > 0) {
    load_k(k_buf0);
    load_v(v_buf0);
    if (nblk > 1) load_k(k_buf1);
  }
  wait_vmem();
  __syncthreads();
  s_mfma(k_buf0, sa0, sa1);
  pace_lds_mfma<D / 8, 1, FWD_DEPTH>();
  __syncthreads();
  for (int b = 0; b < nblk; b += 2) {
    if (b + 2 < nblk) load_k(k_buf0);
    if (b + 1 < nblk) load_v(v_buf1);
    if (!skipped(b)) step(b, sa0, sa1, k_buf1, v_buf0, sb0, sb1);
    wait_vmem();
    __syncthreads();
    if (b + 1 < nblk) {
      if (b + 3 < nblk) load_k(k_buf1);
      if (b + 2 < nblk) load_v(v_buf0);
      if (!skipped(b + 1)) step(b + 1, sb0, sb1, k_buf0, v_buf1, sa0, sa1);
      wait_vmem();
      __syncthreads();
    }
  }

  const float l_tot = pair_sum(l_run);
  if (qvalid) {
    const float inv = 1.f / l_tot;
    const int64_t obase = qrow * qstride + head * D;
    const bool part1 = (t.flags & QT_PART1) != 0;
    float* const o32 = p.o32 + (part1 ? p.o32_part : 0);
    uint16_t* const o16 = prow ? p.o[1] : p.o[0];
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int d0 = db * 32 + g4 * 8 + hf * 4;
        const float v0 = oacc[db][g4 * 4 + 0] * inv, v1 = oacc[db][g4 * 4 + 1] * inv;
        const float v2 = oacc[db][g4 * 4 + 2] * inv, v3 = oacc[db][g4 * 4 + 3] * inv;
        if constexpr (OUT32) {
          *reinterpret_cast<float4*>(o32 + obase + d0) = make_float4(v0, v1, v2, v3);
        } else {
          typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
          bf16x4 w;
          w[0] = (__bf16)v0; w[1] = (__bf16)v1; w[2] = (__bf16)v2; w[3] = (__bf16)v3;
          *reinterpret_cast<bf16x4*>(o16 + obase + d0) = w;
        }
      }
    }
    if (hf == 0) {
      float* lse;
      int64_t lrows;
      if constexpr (OUT32) {
        lse = p.lse[0] + (part1 ? p.lse_part : 0);
        lrows = p.lse_rows[0];
      } else {
        lse = prow ? p.lse[1] : p.lse[0];
        lrows = prow ? p.lse_rows[1] : p.lse_rows[0];
      }
      lse[(int64_t)head * lrows + qrow] = (m_run * c + __log2f(l_tot)) * kLn2;
    }
  }
}

}  // namespace

hipError_t launch_attn_fwd(const FwdParams& p0, int n_tiles, bool out_f32, hipStream_t stream) {
  if (n_tiles == 0) return hipSuccess;
  FwdParams p = p0;
  p.n_units = n_tiles * p.hkv;
  const dim3 grid((unsigned)xcd_grid(p.n_units, p.group)), block(256);
  if (p.head_dim == 128) {
    if (out_f32) hipLaunchKernelGGL((attn_fwd_kernel<128, true>), grid, block, 0, stream, p);
    else hipLaunchKernelGGL((attn_fwd_kernel<128, false>), grid, block, 0, stream, p);
  } else {
    if (out_f32) hipLaunchKernelGGL((attn_fwd_kernel<64, true>), grid, block, 0, stream, p);
    else hipLaunchKernelGGL((attn_fwd_kernel<64, false>), grid, block, 0, stream, p);
  }
  return hipGetLastError();
}

}  // namespace augtree
