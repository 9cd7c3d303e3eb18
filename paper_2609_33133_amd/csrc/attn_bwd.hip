// Backward attention kernels for gfx950 (§3.2 exact many-to-one backward,
// Eq. 2). With P = exp(s q.k - LSE) (merged LSE for replay rows),
// D = rowsum(dO * O), dP = dO V^T, dS = P (dP - D):
//   dQ = s dS K,   dK = s dS^T Q,   dV = P^T dO.
//
// Two kernels, no atomics, every output written once:
// * attn_dq_kernel (query-outer): one workgroup per 128-row query tile and
//   query head, sweeping the same key segments as the forward (prompt keys,
//   then the branch's own causal keys). S^T, dP^T and dS^T keep one query per
//   lane; dQ^T += K^T dS^T takes dS^T straight from the accumulators and K^T
//   by transpose reads of the row-major K tile.
// * attn_dkv_kernel (key-outer): one workgroup per 128-key tile and KV head;
//   each wavefront holds 32 keys (K and V rows in registers) and sweeps every
//   query that sees them: the g query heads of the KV head (GQA) and, for
//   prompt keys in replay, the response rows of every branch of the group, so
//   the Eq. 2 sum over branches happens in the accumulators. Query tiles of 64
//   rows are staged in LDS row-major; Q^T and dO^T operands come from
//   transpose reads of the same tiles.
#include "common.h"
#include "kernels.h"

namespace augtree {

namespace {

// ----------------------------------------------------------------------------- dQ

constexpr int DQ_BM = 128;
constexpr int DQ_BN = 64;

template <int D>
struct DqLds {
  __bf16 k[2][DQ_BN * D];
  __bf16 v[2][DQ_BN * D];
};

template <int D>
__global__ __launch_bounds__(256, 1) void attn_dq_kernel(DqParams p) {
  using L = DqLds<D>;
  __shared__ L sm;
  int unit, hh;
  if (!xcd_unit(p.n_units, p.group, unit, hh)) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, l32 = lane & 31, hf = lane >> 5;
  const int tile_id = unit / p.hkv;
  const int kvh = unit - tile_id * p.hkv;
  const int head = kvh * p.group + hh;
  const QTile t = p.tiles[tile_id];
  const int qi = wave * 32 + l32;
  const bool qvalid = qi < t.q_len;
  const int64_t qrow = (int64_t)t.q_row0 + qi;
  const int64_t qstride = (int64_t)p.hq * D;
  const int64_t kvstride = (int64_t)p.hkv * D;

  bf16x8 qreg[D / 16], doreg[D / 16];
  {
    const int64_t off = qrow * qstride + head * D + hf * 8;
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) {
      qreg[ks] = as_bf16x8(qvalid ? ldg16(p.q + off + ks * 16) : make_uint4(0, 0, 0, 0));
      doreg[ks] = as_bf16x8(qvalid ? ldg16(p.dout + off + ks * 16) : make_uint4(0, 0, 0, 0));
    }
  }
  const float lse2 = qvalid ? p.lse[(int64_t)head * p.lse_rows + qrow] * kLog2e : 0.f;
  const float dsq = qvalid ? p.dsum[(int64_t)head * p.lse_rows + qrow] : 0.f;
  const float c = p.scale_log2;

  f32x16 acc[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[db][i] = 0.f;

  const int nA = (t.a_len + DQ_BN - 1) / DQ_BN;
  const int nB = (t.b_len + DQ_BN - 1) / DQ_BN;
  const int nblk = nA + nB;

  TileStage<DQ_BN, D> kst, vst;
  auto load_block = [&](int b) {
    const bool isB = b >= nA;
    const int kb0 = (isB ? b - nA : b) * DQ_BN;
    const int len = isB ? t.b_len : t.a_len;
    const int64_t row0 = (int64_t)(isB ? t.b_row0 : t.a_row0) + kb0;
    const int nvalid = min(DQ_BN, len - kb0);
    kst.load(isB ? p.kb : p.ka, row0, nvalid, kvstride, kvh * D);
    vst.load(isB ? p.vb : p.va, row0, nvalid, kvstride, kvh * D);
  };
  auto store_block = [&](int buf) {
    kst.store(sm.k[buf]);
    vst.store(sm.v[buf]);
  };

  if (nblk > 0) {
    load_block(0);
    store_block(0);
  }
  __syncthreads();

  for (int b = 0; b < nblk; ++b) {
    const int buf = b & 1;
    if (b + 1 < nblk) load_block(b + 1);
    const bool isB = b >= nA;
    const int kb0 = (isB ? b - nA : b) * DQ_BN;
    const int len = isB ? t.b_len : t.a_len;
    const int qpos_lo = t.b_qpos + wave * 32;
    const bool skip = isB && (kb0 > qpos_lo + 31);
    if (!skip) {
      f32x16 s0, s1, d0, d1;
#pragma unroll
      for (int i = 0; i < 16; ++i) { s0[i] = 0.f; s1[i] = 0.f; d0[i] = 0.f; d1[i] = 0.f; }
      const __bf16* kl = sm.k[buf];
      const __bf16* vl = sm.v[buf];
#pragma unroll
      for (int ks = 0; ks < D / 16; ++ks) {
        const int col = ks * 16 + hf * 8;
        s0 = mfma32(lds_row8<D>(kl, l32, col), qreg[ks], s0);
        s1 = mfma32(lds_row8<D>(kl, 32 + l32, col), qreg[ks], s1);
        d0 = mfma32(lds_row8<D>(vl, l32, col), doreg[ks], d0);
        d1 = mfma32(lds_row8<D>(vl, 32 + l32, col), doreg[ks], d1);
      }
      const bool need_mask = (kb0 + DQ_BN > len) || (isB && (kb0 + DQ_BN - 1 > qpos_lo));
      const int qpos = t.b_qpos + qi;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        float a0 = s0[i] * c - lse2, a1 = s1[i] * c - lse2;
        if (need_mask) {
          const int k0 = kb0 + acc_row(i, hf), k1 = k0 + 32;
          if ((k0 >= len) || (isB && k0 > qpos)) a0 = -INFINITY;
          if ((k1 >= len) || (isB && k1 > qpos)) a1 = -INFINITY;
        }
        const float p0 = __builtin_amdgcn_exp2f(a0), p1 = __builtin_amdgcn_exp2f(a1);
        s0[i] = p0 * (d0[i] - dsq);
        s1[i] = p1 * (d1[i] - dsq);
      }
      const bf16x8 g0 = to_bf16x8(s0, 0), g1 = to_bf16x8(s0, 8);
      const bf16x8 g2 = to_bf16x8(s1, 0), g3 = to_bf16x8(s1, 8);
#pragma unroll
      for (int db = 0; db < D / 32; ++db) {
        acc[db] = mfma32(lds_tr_operand<D>(kl, 0, db * 32), g0, acc[db]);
        acc[db] = mfma32(lds_tr_operand<D>(kl, 16, db * 32), g1, acc[db]);
        acc[db] = mfma32(lds_tr_operand<D>(kl, 32, db * 32), g2, acc[db]);
        acc[db] = mfma32(lds_tr_operand<D>(kl, 48, db * 32), g3, acc[db]);
      }
    }
    if (b + 1 < nblk) store_block(buf ^ 1);
    __syncthreads();
  }

  if (qvalid) {
    const int64_t obase = qrow * qstride + head * D;
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int dd = db * 32 + g4 * 8 + hf * 4;
        const float v0 = acc[db][g4 * 4 + 0] * p.scale, v1 = acc[db][g4 * 4 + 1] * p.scale;
        const float v2 = acc[db][g4 * 4 + 2] * p.scale, v3 = acc[db][g4 * 4 + 3] * p.scale;
        if (p.dq32) *reinterpret_cast<float4*>(p.dq32 + obase + dd) = make_float4(v0, v1, v2, v3);
        if (p.dq) {
          typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
          bf16x4 w;
          w[0] = (__bf16)v0; w[1] = (__bf16)v1; w[2] = (__bf16)v2; w[3] = (__bf16)v3;
          *reinterpret_cast<bf16x4*>(p.dq + obase + dd) = w;
        }
      }
    }
  }
}

// ----------------------------------------------------------------------------- dK/dV

constexpr int KV_BN = 128;  // keys per workgroup (32 per wavefront)
constexpr int KV_BQ = 64;   // query rows per block

template <int D>
struct DkvLds {
  __bf16 q[2][KV_BQ * D];
  __bf16 dout[2][KV_BQ * D];
  float lse2[2][KV_BQ];
  float dsum[2][KV_BQ];
};

template <int D, bool OUT32>
__global__ __launch_bounds__(256, 1) void attn_dkv_kernel(DkvParams p) {
  using L = DkvLds<D>;
  __shared__ L sm;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, l32 = lane & 31, hf = lane >> 5;
  const int tile_id = blockIdx.x / p.hkv;
  const int kvh = blockIdx.x - tile_id * p.hkv;
  const KVTile t = p.tiles[tile_id];
  const int kw0 = wave * 32;
  const int kj = kw0 + l32;  // this lane's key (B-operand column)
  const bool kvalid = kj < t.kv_len;
  const int64_t qstride = (int64_t)p.hq * D;
  const int64_t kvstride = (int64_t)p.hkv * D;

  bf16x8 kreg[D / 16], vreg[D / 16];
  {
    const int64_t off = ((int64_t)t.kv_row0 + kj) * kvstride + kvh * D + hf * 8;
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) {
      kreg[ks] = as_bf16x8(kvalid ? ldg16(p.k + off + ks * 16) : make_uint4(0, 0, 0, 0));
      vreg[ks] = as_bf16x8(kvalid ? ldg16(p.v + off + ks * 16) : make_uint4(0, 0, 0, 0));
    }
  }
  f32x16 dk[D / 32], dv[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) { dk[db][i] = 0.f; dv[db][i] = 0.f; }

  const float c = p.scale_log2;
  const int nqb = (t.q_len + KV_BQ - 1) / KV_BQ;
  const int nblk = p.group * nqb;

  TileStage<KV_BQ, D> qst, dost;
  float stat = 0.f;  // lse2 (threads 0..63) or D (threads 64..127) of the staged block
  auto load_block = [&](int b) {
    const int hh = kvh * p.group + b / nqb;
    const int qb = b % nqb;
    const int64_t row0 = (int64_t)t.q_row0 + qb * KV_BQ;
    const int nvalid = min(KV_BQ, t.q_len - qb * KV_BQ);
    qst.load(p.q, row0, nvalid, qstride, hh * D);
    dost.load(p.dout, row0, nvalid, qstride, hh * D);
    if (tid < KV_BQ)
      stat = tid < nvalid ? p.lse[(int64_t)hh * p.lse_rows + row0 + tid] * kLog2e : INFINITY;
    else if (tid < 2 * KV_BQ)
      stat = (tid - KV_BQ) < nvalid ? p.dsum[(int64_t)hh * p.lse_rows + row0 + tid - KV_BQ] : 0.f;
  };
  auto store_block = [&](int buf) {
    qst.store(sm.q[buf]);
    dost.store(sm.dout[buf]);
    if (tid < KV_BQ) sm.lse2[buf][tid] = stat;
    else if (tid < 2 * KV_BQ) sm.dsum[buf][tid - KV_BQ] = stat;
  };

  if (nblk > 0) {
    load_block(0);
    store_block(0);
  }
  __syncthreads();

  for (int b = 0; b < nblk; ++b) {
    const int buf = b & 1;
    if (b + 1 < nblk) load_block(b + 1);
    const int qb = b % nqb;
    const int qblk_pos = t.qpos0 + qb * KV_BQ;       // position of the block's first query
    const int key_pos = t.kpos0 + kj;               // this lane's key position
    const bool skip = t.causal && (qblk_pos + KV_BQ - 1 < t.kpos0 + kw0);
    if (!skip) {
      const bool need_mask = t.causal && (qblk_pos < t.kpos0 + kw0 + 31);
#pragma unroll
      for (int qs = 0; qs < 2; ++qs) {
        f32x16 s, dp;
#pragma unroll
        for (int i = 0; i < 16; ++i) { s[i] = 0.f; dp[i] = 0.f; }
        const __bf16* ql = sm.q[buf];
        const __bf16* dl = sm.dout[buf];
#pragma unroll
        for (int ks = 0; ks < D / 16; ++ks) {
          s = mfma32(lds_row8<D>(ql, qs * 32 + l32, ks * 16 + hf * 8), kreg[ks], s);
          dp = mfma32(lds_row8<D>(dl, qs * 32 + l32, ks * 16 + hf * 8), vreg[ks], dp);
        }
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          const int r0 = qs * 32 + g4 * 8 + hf * 4;
          const f32x4 l4 = *reinterpret_cast<const f32x4*>(&sm.lse2[buf][r0]);
          const f32x4 d4 = *reinterpret_cast<const f32x4*>(&sm.dsum[buf][r0]);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int i = g4 * 4 + e;
            float a = s[i] * c - l4[e];
            if (need_mask && key_pos > qblk_pos + r0 + e) a = -INFINITY;
            const float pr = __builtin_amdgcn_exp2f(a);
            s[i] = pr;
            dp[i] = pr * (dp[i] - d4[e]);
          }
        }
        const bf16x8 pb0 = to_bf16x8(s, 0), pb1 = to_bf16x8(s, 8);
        const bf16x8 gb0 = to_bf16x8(dp, 0), gb1 = to_bf16x8(dp, 8);
#pragma unroll
        for (int db = 0; db < D / 32; ++db) {
          dv[db] = mfma32(pb0, lds_tr_operand<D>(sm.dout[buf], qs * 32, db * 32), dv[db]);
          dv[db] = mfma32(pb1, lds_tr_operand<D>(sm.dout[buf], qs * 32 + 16, db * 32), dv[db]);
          dk[db] = mfma32(gb0, lds_tr_operand<D>(sm.q[buf], qs * 32, db * 32), dk[db]);
          dk[db] = mfma32(gb1, lds_tr_operand<D>(sm.q[buf], qs * 32 + 16, db * 32), dk[db]);
        }
      }
    }
    if (b + 1 < nblk) store_block(buf ^ 1);
    __syncthreads();
  }

  // dK/dV tile: lane holds column d = 32*db + l32, rows = keys acc_row(i, hf)
#pragma unroll
  for (int db = 0; db < D / 32; ++db) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int key = kw0 + acc_row(i, hf);
      if (key < t.kv_len) {
        const int64_t row = (int64_t)t.kv_row0 + key;
        const int64_t off = row * kvstride + kvh * D + db * 32 + l32;
        const float kval = dk[db][i] * p.scale, vval = dv[db][i];
        if constexpr (OUT32) {
          const int64_t slab = (int64_t)p.out_rows * kvstride;
          p.dkv32[(2 * (int64_t)t.part) * slab + off] = kval;
          p.dkv32[(2 * (int64_t)t.part + 1) * slab + off] = vval;
        } else {
          reinterpret_cast<__bf16*>(p.dk)[off] = (__bf16)kval;
          reinterpret_cast<__bf16*>(p.dv)[off] = (__bf16)vval;
        }
      }
    }
  }
}

// ----------------------------------------------------------------------------- D = rowsum(dO * O)

template <int D>
__global__ __launch_bounds__(256) void bwd_dsum_kernel(const uint16_t* o, const uint16_t* dout, float* dsum,
                                                       int64_t rows, int hq) {
  constexpr int CH = D / 8;
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t rh = gid / CH;
  const int ch = (int)(gid % CH);
  float acc = 0.f;
  if (rh < rows * hq) {
    const uint4 a = ldg16(o + rh * D + ch * 8);
    const uint4 b = ldg16(dout + rh * D + ch * 8);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float x = __uint_as_float(half16(a, e) << 16);
      const float y = __uint_as_float(half16(b, e) << 16);
      acc += x * y;
    }
  }
#pragma unroll
  for (int off = CH / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if (ch == 0 && rh < rows * hq) {
    const int64_t row = rh / hq;
    const int h = (int)(rh - row * hq);
    dsum[(int64_t)h * rows + row] = acc;
  }
}

}  // namespace

hipError_t launch_attn_dq(const DqParams& p0, int n_tiles, hipStream_t stream) {
  if (n_tiles == 0) return hipSuccess;
  DqParams p = p0;
  p.n_units = n_tiles * p.hkv;
  const dim3 grid((unsigned)xcd_grid(p.n_units, p.group)), block(256);
  if (p.head_dim == 128) hipLaunchKernelGGL((attn_dq_kernel<128>), grid, block, 0, stream, p);
  else hipLaunchKernelGGL((attn_dq_kernel<64>), grid, block, 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_attn_dkv(const DkvParams& p, int n_tiles, bool out_f32, hipStream_t stream) {
  if (n_tiles == 0) return hipSuccess;
  const dim3 grid((unsigned)n_tiles * (unsigned)p.hkv), block(256);
  if (p.head_dim == 128) {
    if (out_f32) hipLaunchKernelGGL((attn_dkv_kernel<128, true>), grid, block, 0, stream, p);
    else hipLaunchKernelGGL((attn_dkv_kernel<128, false>), grid, block, 0, stream, p);
  } else {
    if (out_f32) hipLaunchKernelGGL((attn_dkv_kernel<64, true>), grid, block, 0, stream, p);
    else hipLaunchKernelGGL((attn_dkv_kernel<64, false>), grid, block, 0, stream, p);
  }
  return hipGetLastError();
}

hipError_t launch_bwd_dsum(const uint16_t* o, const uint16_t* dout, float* dsum, int64_t rows, int hq,
                           int head_dim, hipStream_t stream) {
  const int64_t threads = rows * hq * (head_dim / 8);
  if (threads == 0) return hipSuccess;
  const dim3 grid((unsigned)((threads + 255) / 256)), block(256);
  if (head_dim == 128) hipLaunchKernelGGL((bwd_dsum_kernel<128>), grid, block, 0, stream, o, dout, dsum, rows, hq);
  else hipLaunchKernelGGL((bwd_dsum_kernel<64>), grid, block, 0, stream, o, dout, dsum, rows, hq);
  return hipGetLastError();
}

int dq_block_m() { return DQ_BM; }
int dkv_block_n() { return KV_BN; }
int dkv_block_q() { return KV_BQ; }

}  // namespace augtree
