// Backward attention kernels for gfx950 (§3.2 exact many-to-one backward,
// Eq. 2). With P = exp(s q.k - LSE) (merged LSE for replay rows),
// D = rowsum(dO * O), dP = dO V^T, dS = P (dP - D):
//   dQ = s dS K,   dK = s dS^T Q,   dV = P^T dO.
//
// Two kernels, no atomics, every output written once:
// * attn_dq_kernel (query-outer): one workgroup (4 wavefronts, two workgroups
//   per CU) per 128-row query tile and query head, sweeping the same key
//   segments as the forward (prompt keys, then the branch's own causal keys)
//   in 64-key blocks, each handled as two 32-key halves. S^T, dP^T and dS^T
//   keep one query per lane; dQ^T += K^T dS^T takes dS^T straight from the
//   accumulators and K^T by transpose reads of the row-major K tile.
// * attn_dkv_kernel (key-outer): one workgroup (8 wavefronts, two per SIMD)
//   per 128-key tile and KV head. Wavefronts w and w + 4 own the same 32 keys
//   (K and V tiles in LDS) and take the two 32-row halves of
//   every 64-row query block; their dK/dV partials are added through LDS at
//   the end. The sweep covers every query that sees the keys: the g query
//   heads of the KV head (GQA) and, for prompt keys in replay, the response
//   rows of every branch of the group, so the Eq. 2 sum over branches happens
//   in the accumulators. Query tiles are copied to LDS directly from global
//   memory; Q^T and dO^T operands come from transpose reads.
#include "common.h"
#include "kernels.h"

namespace augtree {

namespace {

// ----------------------------------------------------------------------------- dQ

constexpr int DQ_BM = kDqBlockM;
constexpr int DQ_BN = kDqBlockN;
constexpr int DQ_DEPTH = 4;  // LDS operand reads run this many MFMAs ahead

template <int D>
__global__ __launch_bounds__(256, 2) void attn_dq_kernel(DqParams p) {
  __shared__ __bf16 k_buf0[DQ_BN * D], k_buf1[DQ_BN * D], v_buf0[DQ_BN * D], v_buf1[DQ_BN * D];
  int unit, hh;
  if (!xcd_unit(p.n_units, p.group, unit, hh)) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, l32 = lane & 31, hf = lane >> 5;
  const int tile_id = unit / p.hkv;
  const int kvh = unit - tile_id * p.hkv;
  const int head = kvh * p.group + hh;
  const QTile t = load_tile(p.tiles, p.inl, tile_id);
  const bool prow = (t.flags & QT_PROMPT_ROWS) != 0;  // prompt rows (prefill) or response rows
  const uint16_t* const kb = prow ? p.kb[1] : p.kb[0];
  const uint16_t* const vb = prow ? p.vb[1] : p.vb[0];
  const int64_t lrows = prow ? p.lse_rows[1] : p.lse_rows[0];
  const int qi = wave * 32 + l32;
  const bool qvalid = qi < t.q_len;
  const int64_t qrow = (int64_t)t.q_row0 + qi;
  const int64_t qstride = (int64_t)p.hq * D;
  const int64_t kvstride = (int64_t)p.hkv * D;

  // Q^T and dO^T operands: lane holds query qi, d = 16*ks + 8*hf .. +7.
  // D = rowsum(dO * O) of the query is formed here from the same halves
  // (eight partial sums, a tree, and the half-wave exchange) and stored for
  // the dK/dV kernel.
  bf16x8 qreg[D / 16], doreg[D / 16];
  float dsq;
  {
    const int64_t off = qrow * qstride + head * D + hf * 8;
    const uint16_t* qs = (prow ? p.q[1] : p.q[0]) + off;
    const uint16_t* ds = (prow ? p.dout[1] : p.dout[0]) + off;
    const uint16_t* os = (prow ? p.o[1] : p.o[0]) + off;
    float part[D / 16];
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) {
      const uint4 z = make_uint4(0, 0, 0, 0);
      qreg[ks] = as_bf16x8(qvalid ? ldg16(qs + ks * 16) : z);
      const uint4 dv = qvalid ? ldg16(ds + ks * 16) : z;
      const uint4 ov = qvalid ? ldg16(os + ks * 16) : z;
      doreg[ks] = as_bf16x8(dv);
      float a = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e)
        a += __uint_as_float(half16(dv, e) << 16) * __uint_as_float(half16(ov, e) << 16);
      part[ks] = a;
    }
#pragma unroll
    for (int w = D / 32; w >= 1; w >>= 1)
#pragma unroll
      for (int ks = 0; ks < w; ++ks) part[ks] += part[ks + w];
    dsq = pair_sum(part[0]);
  }
  if (qvalid && hf == 0) (prow ? p.dsum[1] : p.dsum[0])[(int64_t)head * lrows + qrow] = dsq;
  // S and dP accumulators start at -LSE / scale and -D of this lane's query,
  // so the MFMAs leave S - LSE / scale and dP - D: P = exp2(c * s), dS = P * dp
  const float nlse = qvalid ? -(prow ? p.lse[1] : p.lse[0])[(int64_t)head * lrows + qrow] / p.scale : 0.f;
  if (!qvalid) dsq = 0.f;
  const float c = p.scale_log2;

  f32x16 acc[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[db][i] = 0.f;
  // sum over the keys of dS as rounded to bf16 for the dQ MFMAs (this lane's
  // 16 keys of every 32-key half); see the correction at the end
  float ds_sum = 0.f;

  const int nA = (t.a_len + DQ_BN - 1) / DQ_BN;
  const int nB = (t.b_len + DQ_BN - 1) / DQ_BN;
  const int nblk = nA + nB;

  TileCopy<DQ_BN, D, 4> cp;
  cp.init(kvstride);
  // The load cursor: the next key block to be copied into LDS, stepped in
  // place (the sweep's scalar work is on the critical path of every block:
  // the eight wavefronts of a CU share one scalar unit).
  struct KCursor {
    int isB, kb0, len;    // segment (0: A, 1: B), its first key of the block, the segment's length
    const char* kp;       // K of the block's first key, KV head kvh
    const char* vp;       // V, the same
  };
  const int krow_bytes = (int)(kvstride * 2);
  const int64_t kstep = (int64_t)DQ_BN * krow_bytes;
  // K / V of segment B at its first row and this KV head
  const char* const kb0p = reinterpret_cast<const char*>(kb + (int64_t)t.b_row0 * kvstride + kvh * D);
  const char* const vb0p = reinterpret_cast<const char*>(vb + (int64_t)t.b_row0 * kvstride + kvh * D);
  KCursor kc;
  if (nA > 0) {
    kc = {0, 0, t.a_len, reinterpret_cast<const char*>(p.ka + (int64_t)t.a_row0 * kvstride + kvh * D),
          reinterpret_cast<const char*>(p.va + (int64_t)t.a_row0 * kvstride + kvh * D)};
  } else {
    kc = {1, 0, t.b_len, kb0p, vb0p};
  }
  // what the computation of a block needs to know of it
  struct Blk {
    int isB, kb0, len;
  };
  // copy the cursor's block into (kd, vd), note it in k and step the cursor
  // (past the end of segment B: never loaded)
  auto load_next = [&](__bf16* kd, __bf16* vd, Blk& k) {
    const int nbytes = min(DQ_BN, kc.len - kc.kb0) * krow_bytes;
    cp.issue_bytes(kd, reinterpret_cast<const uint16_t*>(kc.kp), nbytes);
    cp.issue_bytes(vd, reinterpret_cast<const uint16_t*>(kc.vp), nbytes);
    k = {kc.isB, kc.kb0, kc.len};
    int64_t dk = kstep, dv = kstep;
    kc.kb0 += DQ_BN;
    if (kc.kb0 >= kc.len && kc.isB == 0) {
      dk = kb0p - kc.kp;
      dv = vb0p - kc.vp;
      kc.isB = 1;
      kc.kb0 = 0;
      kc.len = t.b_len;
    }
    kc.kp += dk;
    kc.vp += dv;
  };

  RowOffsets<D> r0_off, r1_off;  // K/V rows l32 and 32 + l32
  r0_off.init(l32, hf);
  r1_off.init(32 + l32, hf);
  TrOffsets<D> ktr_off;           // K^T operands
  ktr_off.init(0, lane);
  auto compute = [&](const Blk& k, const __bf16* kl, const __bf16* vl) {
    const bool isB = k.isB != 0;
    const int kb0 = k.kb0;
    const int len = k.len;
    const int qpos_lo = t.b_qpos + wave * 32;
    const int qpos = t.b_qpos + qi;
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      const int k0 = kb0 + half * 32;  // first key of this 32-key half
      const bool skip = isB && (k0 > qpos_lo + 31);
      if (skip) continue;
      f32x16 s, dp;
#pragma unroll
      for (int i = 0; i < 16; ++i) { s[i] = nlse; dp[i] = -dsq; }
      set_wave_priority<0>();
#pragma unroll
      for (int ks = 0; ks < D / 16; ++ks) {
        const int o = half ? r1_off.o[ks] : r0_off.o[ks];
        s = mfma32(lds_row8_at<D>(kl, o), qreg[ks], s);
        dp = mfma32(lds_row8_at<D>(vl, o), doreg[ks], dp);
      }
      pace_lds_mfma<D / 8, 1, DQ_DEPTH>();
      set_wave_priority<1>();
      // ragged end or diagonal; the condition is uniform over the wavefront
      // (a scalar branch)
      if (__builtin_amdgcn_readfirstlane((k0 + 32 > len) || (isB && (k0 + 31 > qpos_lo)))) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int kk = k0 + acc_row(i, hf);
          if ((kk >= len) || (isB && kk > qpos)) s[i] = -INFINITY;
        }
      }
#pragma unroll
      for (int i = 0; i < 16; ++i) s[i] = __builtin_amdgcn_exp2f(s[i] * c) * dp[i];
      const bf16x8 g0 = to_bf16x8(s, 0), g1 = to_bf16x8(s, 8);
      ds_sum = sum_bf16x8(g0, sum_bf16x8(g1, ds_sum));
      set_wave_priority<0>();
#pragma unroll
      for (int db = 0; db < D / 32; ++db) {
        acc[db] = mfma32(ktr_off.read(kl, 2 * half, db), g0, acc[db]);
        acc[db] = mfma32(ktr_off.read(kl, 2 * half + 1, db), g1, acc[db]);
      }
      pace_lds_mfma<D / 16, 2, DQ_DEPTH>();
      set_wave_priority<1>();
    }
  };

  Blk c0{0, 0, 0}, c1{0, 0, 0};
  if (nblk > 0) load_next(k_buf0, v_buf0, c0);
  wait_vmem();
  __syncthreads();
  // The vector c of the common-mode correction at the end: the mean of the
  // group's first (up to) 64 prompt keys of KV head kvh. They are block 0 of
  // every tile's sweep (segment A's first block for response rows, segment
  // B's for prompt rows), now in k_buf0. Wave w sums rows 16w .. 16w + 15
  // (lane l: 16-byte chunk l % CH of rows 16w + l / CH + k * 64 / CH), the
  // lanes of one chunk are added, and the four waves' partial sums go to LDS.
  __shared__ float kmean_part[4][D];
  {
    constexpr int CH = D / 8;
    const int ch = lane % CH;
    float part[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) part[e] = 0.f;
#pragma unroll
    for (int k = 0; k < CH / 4; ++k) {
      const int r = 16 * wave + lane / CH + k * (64 / CH);
      const uint4 v = *reinterpret_cast<const uint4*>(k_buf0 + r * D + ((ch ^ swz<D>(r)) << 3));
#pragma unroll
      for (int e = 0; e < 8; ++e) part[e] += __uint_as_float(half16(v, e) << 16);
    }
#pragma unroll
    for (int off = CH; off < 64; off <<= 1)
#pragma unroll
      for (int e = 0; e < 8; ++e) part[e] += __shfl_xor(part[e], off);
    if (lane < CH)
#pragma unroll
      for (int e = 0; e < 8; ++e) kmean_part[wave][ch * 8 + e] = part[e];
  }
  for (int b = 0; b < nblk; b += 2) {
    if (b + 1 < nblk) load_next(k_buf1, v_buf1, c1);
    compute(c0, k_buf0, v_buf0);
    wait_vmem();
    __syncthreads();
    if (b + 1 < nblk) {
      if (b + 2 < nblk) load_next(k_buf0, v_buf0, c0);
      compute(c1, k_buf1, v_buf1);
      wait_vmem();
      __syncthreads();
    }
  }

  // Common-mode correction. Every row of dS sums to zero over its keys
  // (sum_j P_j dP_j = dO.O = D), so dQ = s sum_j dS_j (k_j - c) for any vector
  // c. The MFMAs form sum_j dS~_j k_j with dS~ = dS rounded to bf16; when the
  // keys share a large component, the rounding error of dS~ is multiplied by
  // it while dQ itself only sees the keys' differences. Subtracting c times
  // the sum of the same rounded values gives sum_j dS~_j (k_j - c) exactly
  // (up to fp32 accumulation): with c the mean of the group's first keys, a
  // component shared by the keys no longer multiplies the rounding error.
  const float ds_tot = pair_sum(ds_sum);
  const float inv_n0 = 1.f / (float)min(DQ_BN, t.a_len > 0 ? t.a_len : t.b_len);
  if (qvalid) {
    const int64_t obase = qrow * qstride + head * D;
    uint16_t* const dq16 = prow ? p.dq[1] : p.dq[0];
    float* const dq32 = prow ? p.dq32[1] : p.dq32[0];
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int dd = db * 32 + g4 * 8 + hf * 4;
        f32x4 cs = *reinterpret_cast<const f32x4*>(&kmean_part[0][dd]);
#pragma unroll
        for (int w = 1; w < 4; ++w) cs += *reinterpret_cast<const f32x4*>(&kmean_part[w][dd]);
        const float corr = ds_tot * inv_n0;
        const float v0 = (acc[db][g4 * 4 + 0] - corr * cs[0]) * p.scale;
        const float v1 = (acc[db][g4 * 4 + 1] - corr * cs[1]) * p.scale;
        const float v2 = (acc[db][g4 * 4 + 2] - corr * cs[2]) * p.scale;
        const float v3 = (acc[db][g4 * 4 + 3] - corr * cs[3]) * p.scale;
        if (dq32) *reinterpret_cast<float4*>(dq32 + obase + dd) = make_float4(v0, v1, v2, v3);
        if (dq16) {
          typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
          bf16x4 w;
          w[0] = (__bf16)v0; w[1] = (__bf16)v1; w[2] = (__bf16)v2; w[3] = (__bf16)v3;
          *reinterpret_cast<bf16x4*>(dq16 + obase + dd) = w;
        }
      }
    }
  }
}

// ----------------------------------------------------------------------------- dK/dV

constexpr int KV_BN = kDkvBlockN;  // keys per workgroup (32 per wavefront pair)
constexpr int KV_BQ = kDkvBlockQ;  // query rows per block (32 per wavefront of a pair)
constexpr int DKV_SDP_DEPTH = 3;  // LDS operand reads of S / dP run this many MFMAs ahead
constexpr int DKV_DVK_DEPTH = 2;  // the same for the dV / dK transpose reads

template <int D>
__global__ __launch_bounds__(512) void attn_dkv_kernel(DkvParams p) {
  // the workgroup's K and V tiles (operands of S = Q K^T and dP = dO V^T);
  // query blocks double-buffered in separate arrays, with -LSE / scale and
  // -D of their rows.
  // The query-block buffers get the larger alignment so that they are placed
  // first (LDS variables are laid out by alignment, then size): every
  // address inside them is then below 64 KB, so the buffer base and the 16 B
  // column steps fold into the 16-bit offset field of the LDS reads and one
  // register per operand serves all four buffers. The K/V tile above them is
  // addressed through opaque per-lane addresses (V at an immediate +32 KB).
  __shared__ __attribute__((aligned(1024))) __bf16 q_buf0[KV_BQ * D], q_buf1[KV_BQ * D], o_buf0[KV_BQ * D],
      o_buf1[KV_BQ * D];
  __shared__ __bf16 kv_tile[2 * KV_BN * D];  // K rows, then V rows
  __bf16* const k_tile = kv_tile;
  __bf16* const v_tile = kv_tile + KV_BN * D;
  __shared__ float nlse_buf0[KV_BQ], nlse_buf1[KV_BQ], ndsum_buf0[KV_BQ], ndsum_buf1[KV_BQ];
  const int tid = threadIdx.x, lane = tid & 63, l32 = lane & 31, hf = lane >> 5;
  const int wave_u = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar branches below
  const int kq = wave_u & 3;   // 32-key slice of the tile
  const int qs = wave_u >> 2;  // 32-row half of every query block
  const int tile_id = blockIdx.x / p.hkv;
  const int kvh = blockIdx.x - tile_id * p.hkv;
  const KVTile t = load_tile(p.tiles, p.inl, tile_id);
  const int pk = (t.flags & KV_PROMPT_KEYS) ? 1 : 0;  // prompt keys or branch keys
  const bool x_causal = (t.flags & KV_X_CAUSAL) != 0;
  const int kw0 = kq * 32;
  const int kj = kw0 + l32;  // this lane's key (B-operand column)
  const int64_t qstride = (int64_t)p.hq * D;
  const int64_t kvstride = (int64_t)p.hkv * D;

  {
    TileCopy<KV_BN, D, 8> kc;
    kc.init(kvstride);
    kc.issue(k_tile, pk ? p.k[1] : p.k[0], t.kv_row0, t.kv_len, kvstride, kvh * D);
    kc.issue(v_tile, pk ? p.v[1] : p.v[0], t.kv_row0, t.kv_len, kvstride, kvh * D);
  }
  f32x16 dk[D / 32], dv[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) { dk[db][i] = 0.f; dv[db][i] = 0.f; }

  const float c = p.scale_log2;
  // query blocks: range X (response rows) then range Y (prompt rows)
  const int nxb = (t.x_len + KV_BQ - 1) / KV_BQ;
  const int nyb = (t.y_len + KV_BQ - 1) / KV_BQ;
  const int nxblk = p.group * nxb;
  const int nblk = nxblk + p.group * nyb;

  // Query blocks in sweep order: (range, query head of the group, 64-row
  // block). Inside a range the blocks are swept from the end backwards and
  // the g heads of a block are taken one after the other, so that the
  // concurrent tiles of one KV head (causal ranges all end at the segment end;
  // the response rows of a group are the same for all its prompt key tiles)
  // stay at the same query rows and share the Q / dO blocks in L2.
  //
  // The block state carries the block's source addresses and moves them by
  // constant steps: all eight wavefronts of the workgroup step it after every
  // barrier, on the one scalar unit of the CU, while no MFMA is ready yet, so
  // its per-block scalar work (a few adds; the multiplies and selects happen
  // once per range) is on the critical path of every block.
  const int g = p.group;
  const int64_t h0 = (int64_t)kvh * g;
  const int64_t srx = p.lse_rows[0], sry = p.lse_rows[1];
  // Wavefront 0 loads the raw LSE and wavefront 1 the D values of the next
  // query block into `stat`; they are scaled and stored to LDS at the end of
  // the iteration, so nothing waits on these loads (or on the tile copies
  // issued before them) while the current block is computed.
  const float* const s_base0 = (wave_u == 0 ? p.lse[0] : p.dsum[0]) + h0 * srx + t.x_row0;
  const float* const s_base1 = (wave_u == 0 ? p.lse[1] : p.dsum[1]) + h0 * sry + t.kv_row0;
  const int qrow_bytes = (int)(qstride * 2);
  // The load cursor: the next block to be copied into LDS, stepped in place.
  struct Cursor {
    int y, hl, qb;            // range (0: X, 1: Y), head within the group, block (counting down)
    int nvalid, nbytes;       // valid rows of the block; those rows x the row stride in bytes
    int64_t sstep, sback;     // statistic byte steps: to the next head; from head g-1 to head 0 one block back
    const char* qp;           // Q of the block's first row, head hl
    const char* op;           // dO, the same
    const char* sp;           // the statistic (LSE or D) of the block's first row, head hl
  };
  // bytes from head g-1 to head 0 one block back
  const int64_t qback = ((int64_t)(g - 1) * D + KV_BQ * qstride) * 2;
  // the last block of range y, head 0
  auto range_start = [&](int y) {
    Cursor r;
    const int len = y ? t.y_len : t.x_len;
    const int64_t srow = y ? sry : srx;
    r.y = y;
    r.hl = 0;
    r.qb = (len + KV_BQ - 1) / KV_BQ - 1;
    r.nvalid = len - r.qb * KV_BQ;
    r.nbytes = r.nvalid * qrow_bytes;
    r.sstep = srow * 4;
    r.sback = ((int64_t)(g - 1) * srow + KV_BQ) * 4;
    const int64_t row0 = (int64_t)(y ? t.kv_row0 : t.x_row0) + (int64_t)r.qb * KV_BQ;
    const int64_t e0 = row0 * qstride + h0 * D;
    r.qp = reinterpret_cast<const char*>(p.q[y] + e0);
    r.op = reinterpret_cast<const char*>(p.dout[y] + e0);
    r.sp = reinterpret_cast<const char*>((y ? s_base1 : s_base0) + r.qb * KV_BQ);
    return r;
  };
  const Cursor ystart = range_start(1);
  Cursor ld = nxb > 0 ? range_start(0) : ystart;
  // Step to the next block in sweep order (past the end of range Y: never
  // loaded). The pointers move by a step chosen on the (rare) head wrap and
  // range change paths and added on the one common path, so the compiler
  // keeps them in place instead of copying every field at the merge.
  auto advance = [&]() {
    int64_t dq = 2 * D, dout = 2 * D, ds = ld.sstep;
    if (++ld.hl == g) {
      ld.hl = 0;
      if (ld.qb > 0) {
        --ld.qb;
        ld.nvalid = KV_BQ;
        ld.nbytes = KV_BQ * qrow_bytes;
        dq = -qback;
        dout = -qback;
        ds = -ld.sback;
      } else if (ld.y == 0) {
        dq = ystart.qp - ld.qp;
        dout = ystart.op - ld.op;
        ds = ystart.sp - ld.sp;
        ld.y = 1;
        ld.qb = ystart.qb;
        ld.nvalid = ystart.nvalid;
        ld.nbytes = ystart.nbytes;
        ld.sstep = ystart.sstep;
        ld.sback = ystart.sback;
      }
    }
    ld.qp += dq;
    ld.op += dout;
    ld.sp += ds;
  };

  // what the computation of a block needs to know of it
  struct Blk {
    int y, qb;
  };
  float stat = 0.f;
  int stat_n = 0;
  TileCopy<KV_BQ, D, 8> qc;
  qc.init(qstride);
  // copy the cursor's block into (qd, od), note it in k and step the cursor
  auto load_next = [&](__bf16* qd, __bf16* od, Blk& k) {
    qc.issue_bytes(qd, reinterpret_cast<const uint16_t*>(ld.qp), ld.nbytes);
    qc.issue_bytes(od, reinterpret_cast<const uint16_t*>(ld.op), ld.nbytes);
    if (wave_u < 2) {
      stat = reinterpret_cast<const float*>(ld.sp)[min(lane, ld.nvalid - 1)];
      stat_n = ld.nvalid;
    }
    k.y = ld.y;
    k.qb = ld.qb;
    advance();
  };
  // stored as the S and dP accumulator start values -LSE / scale and -D
  // (-inf past the end of the range, so those rows get P = 0)
  const float neg_inv_scale = -1.f / p.scale;
  auto store_stat = [&](float* ld, float* dd) {
    if (wave_u == 0) ld[lane] = lane < stat_n ? stat * neg_inv_scale : -INFINITY;
    else if (wave_u == 1) dd[lane] = lane < stat_n ? -stat : 0.f;
  };

  RowOffsets<D> qrow_off, key_off;   // Q/dO rows of this wave's half; K/V rows of its keys
  qrow_off.init(qs * 32 + l32, hf);
  key_off.init(kj, hf);
  // LDS addresses of this lane's K rows; the V rows are KV_BN * D * 2 bytes on
  // (an immediate offset of the same register)
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) key_off.o[ks] = (int)opaque(lds_addr(k_tile) + key_off.o[ks]);
  TrOffsets<D> qtr_off;              // Q^T / dO^T operands of this wave's half
  qtr_off.init(qs * 32, lane);
  auto compute = [&](const Blk& k, const __bf16* ql, const __bf16* dl, const float* lsel, const float* dsl) {
    // A causal range starts at the tile's first key position, so only its
    // blocks 0 and 1 (rows 0 .. 127) reach the diagonal of the 128 keys.
    const int qrel = k.qb * KV_BQ + qs * 32 - kw0;  // this wave's first query row - its first key
    bool need_mask = false;
    if (k.qb < 2 && (k.y || x_causal)) {
      if (qrel + 31 < 0) return;  // every key of the wave after every row
      need_mask = qrel < 31;
    }
    // S and dP accumulators start at -LSE / scale and -D of their rows
    // (register i holds row g4 * 8 + 4 * hf + e, i = 4 * g4 + e), so the
    // MFMAs leave S - LSE / scale and dP - D: P = exp2(c * s), dS = P * dp.
    // The start values are read in a scheduling region of their own: in the
    // paced region below they would take the first operand-read slots.
    f32x16 s, dp;
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      const int r0 = qs * 32 + g4 * 8 + hf * 4;
      const f32x4 l4 = *reinterpret_cast<const f32x4*>(&lsel[r0]);
      const f32x4 d4 = *reinterpret_cast<const f32x4*>(&dsl[r0]);
#pragma unroll
      for (int e = 0; e < 4; ++e) { s[g4 * 4 + e] = l4[e]; dp[g4 * 4 + e] = d4[e]; }
    }
    set_wave_priority<0>();
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) {
      s = mfma32(lds_row8_at<D>(ql, qrow_off.o[ks]), lds_read16(kv_tile, key_off.o[ks]), s);
      dp = mfma32(lds_row8_at<D>(dl, qrow_off.o[ks]), lds_read16<KV_BN * D * 2>(kv_tile, key_off.o[ks]), dp);
    }
    pace_lds_mfma<D / 8, 2, DKV_SDP_DEPTH>();
    set_wave_priority<1>();
    if (need_mask) {  // only blocks that cross the diagonal
#pragma unroll
      for (int i = 0; i < 16; ++i)
        if (l32 > qrel + acc_row(i, hf)) s[i] = -INFINITY;
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const float pr = __builtin_amdgcn_exp2f(s[i] * c);
      s[i] = pr;
      dp[i] = pr * dp[i];
    }
    const bf16x8 pb0 = to_bf16x8(s, 0), pb1 = to_bf16x8(s, 8);
    const bf16x8 gb0 = to_bf16x8(dp, 0), gb1 = to_bf16x8(dp, 8);
    set_wave_priority<0>();
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
      dv[db] = mfma32(pb0, qtr_off.read(dl, 0, db), dv[db]);
      dv[db] = mfma32(pb1, qtr_off.read(dl, 1, db), dv[db]);
      dk[db] = mfma32(gb0, qtr_off.read(ql, 0, db), dk[db]);
      dk[db] = mfma32(gb1, qtr_off.read(ql, 1, db), dk[db]);
    }
    pace_lds_mfma<D / 8, 2, DKV_DVK_DEPTH>();
    set_wave_priority<1>();
  };

  Blk c0{0, 0}, c1{0, 0};
  if (nblk > 0) {
    load_next(q_buf0, o_buf0, c0);
    store_stat(nlse_buf0, ndsum_buf0);
  }
  wait_vmem();
  __syncthreads();
  for (int b = 0; b < nblk; b += 2) {
    if (b + 1 < nblk) load_next(q_buf1, o_buf1, c1);
    compute(c0, q_buf0, o_buf0, nlse_buf0, ndsum_buf0);
    if (b + 1 < nblk) store_stat(nlse_buf1, ndsum_buf1);
    wait_vmem();
    __syncthreads();
    if (b + 1 < nblk) {
      if (b + 2 < nblk) load_next(q_buf0, o_buf0, c0);
      compute(c1, q_buf1, o_buf1, nlse_buf1, ndsum_buf1);
      if (b + 2 < nblk) store_stat(nlse_buf0, ndsum_buf0);
      wait_vmem();
      __syncthreads();
    }
  }

  // Add the partials of wavefronts w + 4 into w through LDS (the query-block
  // buffers are free now; key slice kq uses one of the four), then wavefronts
  // 0..3 write the tile. Accumulator register i of lane l sits at
  // [db][i][lane] of the exchange buffer.
  __bf16* xbuf = kq == 0 ? q_buf0 : kq == 1 ? q_buf1 : kq == 2 ? o_buf0 : o_buf1;
  float* myx = reinterpret_cast<float*>(xbuf);
  static_assert((D / 32) * 16 * 64 * 4 <= KV_BQ * D * 2, "exchange fits one query buffer");
#pragma unroll
  for (int round = 0; round < 2; ++round) {
    f32x16* acc = round == 0 ? dk : dv;
    if (qs == 1) {
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int i = 0; i < 16; ++i) myx[(db * 16 + i) * 64 + lane] = acc[db][i];
    }
    __syncthreads();
    if (qs == 0) {
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[db][i] += myx[(db * 16 + i) * 64 + lane];
    }
    __syncthreads();
  }
  if (qs != 0) return;

  // dK/dV tile: lane holds column d = 32*db + l32, rows = keys acc_row(i, hf)
  uint16_t* const dk16 = (t.flags & KV_OUT_BF16) ? p.dk[pk] : nullptr;
  uint16_t* const dv16 = (t.flags & KV_OUT_BF16) ? p.dv[pk] : nullptr;
  const int64_t slab = p.slab_rows * kvstride;
  float* const dk32 = (t.flags & KV_OUT_SLAB) ? p.slab + (int64_t)t.out_row0 * kvstride : nullptr;
#pragma unroll
  for (int db = 0; db < D / 32; ++db) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int key = kw0 + acc_row(i, hf);
      if (key < t.kv_len) {
        const int64_t col = kvh * D + db * 32 + l32;
        const int64_t off = ((int64_t)t.kv_row0 + key) * kvstride + col;
        const float kval = dk[db][i] * p.scale, vval = dv[db][i];
        if (dk32) {
          const int64_t so = (int64_t)key * kvstride + col;
          dk32[so] = kval;
          dk32[slab + so] = vval;
        }
        if (dk16) {
          reinterpret_cast<__bf16*>(dk16)[off] = (__bf16)kval;
          reinterpret_cast<__bf16*>(dv16)[off] = (__bf16)vval;
        }
      }
    }
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

hipError_t launch_attn_dkv(const DkvParams& p, int n_tiles, hipStream_t stream) {
  if (n_tiles == 0) return hipSuccess;
  const dim3 grid((unsigned)n_tiles * (unsigned)p.hkv), block(512);
  if (p.head_dim == 128) hipLaunchKernelGGL((attn_dkv_kernel<128>), grid, block, 0, stream, p);
  else hipLaunchKernelGGL((attn_dkv_kernel<64>), grid, block, 0, stream, p);
  return hipGetLastError();
}

}  // namespace augtree
