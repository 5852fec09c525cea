// Attention core of the frozen blocks: softmax(Q K^T / sqrt(d_head) [+causal]) V
// per (batch, head), and its backward (dQ, dK, dV; frozen projections around it
// are plain GEMMs).  Rotary embedding (rotate-half pairs (i, i + d_head/2)):
// in bf16 stages the QKV projection's epilogue has already rotated Q and K, so
// the stash holds the rotated projections and the kernels load them as they
// are; the fp32 path rotates Q and K as they are loaded.  Either way the
// backward rotates dQ and dK back before storing them.
//
// bf16 kernels use MFMA 32x32x16 with K/V (or Q/dO) tiles staged in LDS.
// Each wave owns 32 queries (forward, dQ pass) or 32 keys (dK/dV pass), so the
// score block held in registers has a fixed query (key) per lane and the
// softmax row statistics are mostly in-lane.  The probabilities are fed back
// to the second MFMA straight from registers: within one 16-wide k step the
// lane's values cover 16 keys in a fixed permuted order, and the other operand
// is read in that same order from the row-major LDS tile with the gfx950 LDS
// transpose read (ds_read_b64_tr_b16), so no tile is ever stored transposed.
//
// Log-sum-exp is kept in base 2 of the scaled scores: lse2 = log2 sum_j
// 2^(s_j * scale * log2 e).
#include "attn_core.h"
#include "common.h"
#include "kernels.h"

namespace rg {

// ================================================================ bf16 / MFMA
// One [KT x DH] tile of rows r0.. (rows >= S are zero) from column col of a
// row-major source into LDS row-major (pitch DH + 8), in two steps so that the
// caller can issue the global loads of several tiles before the first LDS
// store: issue() loads this thread's 16-B chunks into registers, store()
// writes them, rotating pairs (i, i + DH/2) when rot.
template <int DH, int NT>
struct TileLoad {
  static constexpr int HC = DH / 16, PAIRS = KT * HC, IT = PAIRS / NT;
  static_assert(PAIRS % NT == 0, "whole passes of the workgroup");
  bf16x8 raw[IT][2];
  __device__ __forceinline__ void issue(const bf16* src, int ld, int col, int b, int S, int r0) {
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int p = threadIdx.x + it * NT;
      // rows past S read row S - 1 and are zeroed in store(): no load is conditional on
      // a lane, so none waits for the one before it
      const int r = p / HC, c = p % HC, row = min(r0 + r, S - 1);
      const bf16* a0 = src + (long)(b * S + row) * ld + col + c * 8;
      raw[it][0] = ld_frag(a0);
      raw[it][1] = ld_frag(a0 + DH / 2);
    }
  }
  __device__ __forceinline__ void store(bf16* dst, bool rot, int S, int r0, const float2* rtab) {
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int p = threadIdx.x + it * NT;
      const int r = p / HC, c = p % HC, row = r0 + r;
      if (row >= S) raw[it][0] = raw[it][1] = zero_frag();
      if (rot && row < S) {
        float x1[8], x2[8];
        unpack_frag(raw[it][0], x1);
        unpack_frag(raw[it][1], x2);
#pragma unroll
        for (int v = 0; v < 8; ++v) {
          float cs, sn;
          rope_cs(rtab, row, c * 8 + v, DH, &cs, &sn);
          const float a = x1[v], bb = x2[v];
          x1[v] = a * cs - bb * sn;
          x2[v] = bb * cs + a * sn;
        }
        raw[it][0] = pack_frag(x1);
        raw[it][1] = pack_frag(x2);
      }
      *reinterpret_cast<bf16x8*>(dst + r * (DH + 8) + c * 8) = raw[it][0];
      *reinterpret_cast<bf16x8*>(dst + r * (DH + 8) + c * 8 + DH / 2) = raw[it][1];
    }
  }
};

// Two tiles (e.g. K and V) with one memory round trip: both tiles' global
// loads are issued before the first LDS store; the first is rotated when rot0.
template <int DH, int NT>
__device__ __forceinline__ void load_tile_pair(const bf16* src0, int ld0, int col0, bool rot0, bf16* dst0,
                                               const bf16* src1, int ld1, int col1, bf16* dst1, int b, int S,
                                               int r0, const float2* rtab) {
  TileLoad<DH, NT> t0, t1;
  t0.issue(src0, ld0, col0, b, S, r0);
  t1.issue(src1, ld1, col1, b, S, r0);
  t0.store(dst0, rot0, S, r0, rtab);
  t1.store(dst1, false, S, r0, rtab);
}

// Q and K need the rotation as they are loaded (it is not already in qkv)
__device__ __forceinline__ bool rot_load(const AttnArgs& a) { return a.rope && !a.rope_in_qkv; }

// Fragments (B operand, k = head dim) of one row held by this lane: dims
// 16s + 8*(lane/32) + v, rotated when rot.
template <int DH>
__device__ __forceinline__ void load_row_frags(const bf16* src, int pos, bool valid, bool rot,
                                               const float2* rtab, int half, bf16x8 f[DH / 16]) {
  // src is a valid row even when !valid (callers clamp it): the loads are unconditional
  // and issued together, the values masked afterwards
  float x[DH / 16][8];
  bf16x8 raw[DH / 16];
#pragma unroll
  for (int s = 0; s < DH / 16; ++s) raw[s] = ld_frag(src + 16 * s + 8 * half);
#pragma unroll
  for (int s = 0; s < DH / 16; ++s) {
    unpack_frag(raw[s], x[s]);
#pragma unroll
    for (int v = 0; v < 8; ++v) x[s][v] = valid ? x[s][v] : 0.f;
  }
  if (rot && valid) {
#pragma unroll
    for (int s = 0; s < DH / 32; ++s)
#pragma unroll
      for (int v = 0; v < 8; ++v) {
        float cs, sn;
        rope_cs(rtab, pos, 16 * s + 8 * half + v, DH, &cs, &sn);
        const float a = x[s][v], bb = x[s + DH / 32][v];
        x[s][v] = a * cs - bb * sn;
        x[s + DH / 32][v] = bb * cs + a * sn;
      }
  }
#pragma unroll
  for (int s = 0; s < DH / 16; ++s) f[s] = pack_frag(x[s]);
}

// Causal tiles do unequal work: query tile t of nq takes t + 1 key tiles (the dK/dV
// pass: key block j takes nq - j query tiles).  At d_h = 128 a workgroup fills its CU,
// so the CUs take the workgroups in dispatch order as they free up; dispatching the
// heaviest tiles first (each XCD gets its workgroups in linear-id order, one in eight)
// keeps the light ones for the end, where the plain order could leave one CU a heavy
// tile last.  Returns rank 0 for the heaviest tile and the batch-head index; shapes
// whose workgroups do not split evenly over the XCDs keep xcd_block's order.
__device__ __forceinline__ void heavy_first(int lin, int nq, int nbh, int& rank, int& bh) {
  const int n = nq * nbh, P = n / 8;
  if (n % 8 || P % nq) {
    const int blk = xcd_block(lin, n);
    rank = nq - 1 - blk % nq;
    bh = blk / nq;
    return;
  }
  const int x = lin % 8, o = lin / 8, per = P / nq;  // XCD x, its o-th workgroup
  rank = o / per;
  bh = x * per + o % per;
}

template <int DH, bool CAUSAL, int NW>
__global__ __launch_bounds__(64 * NW) void attn_fwd_bf16(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) bf16 sK[KT * (DH + 8)];
  __shared__ __attribute__((aligned(16))) bf16 sV[KT * (DH + 8)];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, half = lane >> 5, l32 = lane & 31;
  int qb, bh;
  if (CAUSAL) {
    heavy_first(blockIdx.x + gridDim.x * blockIdx.y, gridDim.x, gridDim.y, qb, bh);
    qb = gridDim.x - 1 - qb;  // query tile t does t + 1 key tiles
  } else {
    const int blk = xcd_block(blockIdx.x + gridDim.x * blockIdx.y, gridDim.x * gridDim.y);
    qb = blk % gridDim.x;
    bh = blk / gridDim.x;
  }
  const int b = bh / a.H, hd = bh % a.H, S = a.S;
  const int q = qb * (32 * NW) + wave * 32 + l32;
  const bool qv = q < S;
  const int d = a.H * DH;
  const float2* rtab = a.rope_tab;
  const float sl2 = kLog2e * rsqrtf((float)DH);
  const bf16* qkv = static_cast<const bf16*>(a.qkv);

  bf16x8 qf[DH / 16];
  load_row_frags<DH>(qkv + (long)(b * S + (qv ? q : 0)) * a.ld_qkv + hd * a.qkv_hs, q, qv, rot_load(a),
                     rtab, half, qf);

  f32x16 oacc[DH / 32];
#pragma unroll
  for (int i = 0; i < DH / 32; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[i][r] = 0.f;
  float mrun = -INFINITY, lrun = 0.f;

  const int qlast = min(S - 1, qb * (32 * NW) + 32 * NW - 1);
  const int nkt = CAUSAL ? qlast / KT + 1 : (S + KT - 1) / KT;
  // the next K/V tile's global loads are in flight (in registers) while the
  // current tile is computed on
  TileLoad<DH, 64 * NW> tk, tv;
  tk.issue(qkv, a.ld_qkv, a.qkv_ko + hd * a.qkv_hs, b, S, 0);
  tv.issue(qkv, a.ld_qkv, a.qkv_vo + hd * a.qkv_hs, b, S, 0);
  for (int kt = 0; kt < nkt; ++kt) {
    __syncthreads();
    tk.store(sK, rot_load(a), S, kt * KT, rtab);
    tv.store(sV, false, S, kt * KT, rtab);
    __syncthreads();
    if (kt + 1 < nkt) {
      tk.issue(qkv, a.ld_qkv, a.qkv_ko + hd * a.qkv_hs, b, S, (kt + 1) * KT);
      tv.issue(qkv, a.ld_qkv, a.qkv_vo + hd * a.qkv_hs, b, S, (kt + 1) * KT);
    }
    f32x16 sc[KT / 32];
#pragma unroll
    for (int kb = 0; kb < KT / 32; ++kb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) sc[kb][r] = 0.f;
#pragma unroll
      for (int s = 0; s < DH / 16; ++s)
        sc[kb] = mfma32(ld_frag(sK + (kb * 32 + l32) * (DH + 8) + 16 * s + 8 * half), qf[s], sc[kb]);
    }
    // the row max on the raw scores (the scale is positive), the scale folded
    // into the exponent's FMA; masking only where a key can be out of range
    // or in the future
    float mx = -INFINITY;
    if (CAUSAL || (kt + 1) * KT > S) {
#pragma unroll
      for (int kb = 0; kb < KT / 32; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = kt * KT + kb * 32 + perm_pos(r, half);
          const bool ok = key < S && (!CAUSAL || key <= q);
          sc[kb][r] = ok ? sc[kb][r] : -INFINITY;
          mx = fmaxf(mx, sc[kb][r]);
        }
    } else {
#pragma unroll
      for (int kb = 0; kb < KT / 32; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sc[kb][r]);
    }
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float mnew = fmaxf(mrun, mx * sl2);
    const float alpha = __builtin_amdgcn_exp2f(mrun - mnew);  // 0 on the first tile
    float rs = 0.f;
#pragma unroll
    for (int kb = 0; kb < KT / 32; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        sc[kb][r] = __builtin_amdgcn_exp2f(fmaf(sc[kb][r], sl2, -mnew));
        rs += sc[kb][r];
      }
    rs += __shfl_xor(rs, 32, 64);
    lrun = lrun * alpha + rs;
    mrun = mnew;
#pragma unroll
    for (int i = 0; i < DH / 32; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[i][r] *= alpha;
#pragma unroll
    for (int kb = 0; kb < KT / 32; ++kb)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const bf16x8 pf = pack8(sc[kb], j);
#pragma unroll
        for (int db = 0; db < DH / 32; ++db)
          oacc[db] = mfma32(perm_frag<DH>(sV, db, kb, j, lane), pf, oacc[db]);
      }
  }
  if (qv) {
    bf16* o = static_cast<bf16*>(a.o) + (long)(b * S + q) * a.ld_o + hd * DH;
    store_rows<DH>(oacc, 1.f / lrun, false, q, nullptr, half, o);
    if (half == 0) a.lse[(long)bh * S + q] = mrun + log2f(lrun);
  }
}

// dQ pass (lane = query); also writes D = rowsum(dO * O)
template <int DH, bool CAUSAL, int NW>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(DH <= 64 ? 2 : 1))) void attn_bwd_dq_bf16(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) bf16 sK[KT * (DH + 8)];
  __shared__ __attribute__((aligned(16))) bf16 sV[KT * (DH + 8)];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, half = lane >> 5, l32 = lane & 31;
  int qb, bh;
  if (CAUSAL) {
    heavy_first(blockIdx.x + gridDim.x * blockIdx.y, gridDim.x, gridDim.y, qb, bh);
    qb = gridDim.x - 1 - qb;  // query tile t does t + 1 key tiles
  } else {
    const int blk = xcd_block(blockIdx.x + gridDim.x * blockIdx.y, gridDim.x * gridDim.y);
    qb = blk % gridDim.x;
    bh = blk / gridDim.x;
  }
  const int b = bh / a.H, hd = bh % a.H, S = a.S;
  const int q = qb * (32 * NW) + wave * 32 + l32;
  const bool qv = q < S;
  const int d = a.H * DH;
  const float2* rtab = a.rope_tab;
  const float scale = rsqrtf((float)DH), sl2 = kLog2e * scale;
  const bf16* qkv = static_cast<const bf16*>(a.qkv);
  const long qrow = (long)(b * S + (qv ? q : 0));

  bf16x8 qf[DH / 16], df[DH / 16];
  load_row_frags<DH>(qkv + qrow * a.ld_qkv + hd * a.qkv_hs, q, qv, rot_load(a), rtab, half, qf);
  load_row_frags<DH>(static_cast<const bf16*>(a.dout) + qrow * a.ld_do + hd * DH, q, qv, false,
                     nullptr, half, df);
  float dsum = 0.f;
  {
    const bf16* orow = static_cast<const bf16*>(a.o) + qrow * a.ld_o + hd * DH;
    bf16x8 oraw[DH / 16];  // qrow is clamped: unconditional loads, masked after
#pragma unroll
    for (int s = 0; s < DH / 16; ++s) oraw[s] = ld_frag(orow + 16 * s + 8 * half);
#pragma unroll
    for (int s = 0; s < DH / 16; ++s) {
      float ov[8], dv[8];
      unpack_frag(oraw[s], ov);
#pragma unroll
      for (int v = 0; v < 8; ++v) ov[v] = qv ? ov[v] : 0.f;
      unpack_frag(df[s], dv);
#pragma unroll
      for (int v = 0; v < 8; ++v) dsum += ov[v] * dv[v];
    }
    dsum += __shfl_xor(dsum, 32, 64);
  }
  const float lse_raw = a.lse[(long)bh * S + (qv ? q : 0)];
  const float lse = qv ? lse_raw : 0.f;
  if (qv && half == 0) a.dsum[(long)bh * S + q] = dsum;

  f32x16 dq[DH / 32];
#pragma unroll
  for (int i = 0; i < DH / 32; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) dq[i][r] = 0.f;

  const int qlast = min(S - 1, qb * (32 * NW) + 32 * NW - 1);
  const int nkt = CAUSAL ? qlast / KT + 1 : (S + KT - 1) / KT;
  // the next K/V tile's global loads are in flight while the current one is used
  TileLoad<DH, 64 * NW> tk, tv;
  tk.issue(qkv, a.ld_qkv, a.qkv_ko + hd * a.qkv_hs, b, S, 0);
  tv.issue(qkv, a.ld_qkv, a.qkv_vo + hd * a.qkv_hs, b, S, 0);
  for (int kt = 0; kt < nkt; ++kt) {
    // every query of the workgroup and every key of the tile in range, no causal mask
    const bool full = !CAUSAL && (qb + 1) * (32 * NW) <= S && (kt + 1) * KT <= S;
    __syncthreads();
    tk.store(sK, rot_load(a), S, kt * KT, rtab);
    tv.store(sV, false, S, kt * KT, rtab);
    __syncthreads();
    if (kt + 1 < nkt) {
      tk.issue(qkv, a.ld_qkv, a.qkv_ko + hd * a.qkv_hs, b, S, (kt + 1) * KT);
      tv.issue(qkv, a.ld_qkv, a.qkv_vo + hd * a.qkv_hs, b, S, (kt + 1) * KT);
    }
    // one key block at a time (not unrolled): keeps the kernel within the
    // registers of two waves per SIMD, so a (batch, head) grid fits one round
#pragma unroll 1
    for (int kb = 0; kb < KT / 32; ++kb) {
      f32x16 st, dp;
#pragma unroll
      for (int r = 0; r < 16; ++r) st[r] = dp[r] = 0.f;
#pragma unroll
      for (int s = 0; s < DH / 16; ++s) {
        st = mfma32(ld_frag(sK + (kb * 32 + l32) * (DH + 8) + 16 * s + 8 * half), qf[s], st);
        dp = mfma32(ld_frag(sV + (kb * 32 + l32) * (DH + 8) + 16 * s + 8 * half), df[s], dp);
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = kt * KT + kb * 32 + perm_pos(r, half);
        const bool ok = full || (qv && key < S && (!CAUSAL || key <= q));
        const float p = ok ? __builtin_amdgcn_exp2f(fmaf(st[r], sl2, -lse)) : 0.f;
        st[r] = p * (dp[r] - dsum);  // dS
      }
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const bf16x8 sf = pack8(st, j);
#pragma unroll
        for (int db = 0; db < DH / 32; ++db)
          dq[db] = mfma32(perm_frag<DH>(sK, db, kb, j, lane), sf, dq[db]);
      }
    }
  }
  if (qv) {
    bf16* dst = static_cast<bf16*>(a.dqkv) + (long)(b * S + q) * a.ld_dqkv + hd * DH;
    store_rows<DH>(dq, scale, a.rope, q, rtab, half, dst);
  }
}

// dK/dV pass (lane = key)
template <int DH, bool CAUSAL, int NW>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(DH <= 64 ? 2 : 1))) void attn_bwd_dkdv_bf16(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) bf16 sQ[KT * (DH + 8)];
  __shared__ __attribute__((aligned(16))) bf16 sO[KT * (DH + 8)];
  __shared__ float sL[KT], sD[KT];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, half = lane >> 5, l32 = lane & 31;
  int kb0, bh;
  if (CAUSAL) {
    heavy_first(blockIdx.x + gridDim.x * blockIdx.y, gridDim.x, gridDim.y, kb0, bh);  // block j: nq - j tiles
  } else {
    const int blk = xcd_block(blockIdx.x + gridDim.x * blockIdx.y, gridDim.x * gridDim.y);
    kb0 = blk % gridDim.x;
    bh = blk / gridDim.x;
  }
  const int b = bh / a.H, hd = bh % a.H, S = a.S;
  const int key = kb0 * (32 * NW) + wave * 32 + l32;
  const bool kv = key < S;
  const int d = a.H * DH;
  const float2* rtab = a.rope_tab;
  const float scale = rsqrtf((float)DH), sl2 = kLog2e * scale;
  const bf16* qkv = static_cast<const bf16*>(a.qkv);
  const bf16* dO = static_cast<const bf16*>(a.dout);
  const long krow = (long)(b * S + (kv ? key : 0));

  bf16x8 kf[DH / 16], vf[DH / 16];
  load_row_frags<DH>(qkv + krow * a.ld_qkv + a.qkv_ko + hd * a.qkv_hs, key, kv, rot_load(a), rtab, half, kf);
  load_row_frags<DH>(qkv + krow * a.ld_qkv + a.qkv_vo + hd * a.qkv_hs, key, kv, false, nullptr, half, vf);

  f32x16 dk[DH / 32], dv[DH / 32];
#pragma unroll
  for (int i = 0; i < DH / 32; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) dk[i][r] = dv[i][r] = 0.f;

  const int nqt = (S + KT - 1) / KT;
  const int qt0 = CAUSAL ? (kb0 * (32 * NW)) / KT : 0;
  // the next Q/dO tile's global loads are in flight while the current one is used
  TileLoad<DH, 64 * NW> tq, tdo;
  if (qt0 < nqt) {
    tq.issue(qkv, a.ld_qkv, hd * a.qkv_hs, b, S, qt0 * KT);
    tdo.issue(dO, a.ld_do, hd * DH, b, S, qt0 * KT);
  }
  for (int qt = qt0; qt < nqt; ++qt) {
    // every key of the workgroup and every query of the tile in range, no causal mask
    const bool full = !CAUSAL && (kb0 + 1) * (32 * NW) <= S && (qt + 1) * KT <= S;
    __syncthreads();
    tq.store(sQ, rot_load(a), S, qt * KT, rtab);
    tdo.store(sO, false, S, qt * KT, rtab);
    for (int i = threadIdx.x; i < KT; i += blockDim.x) {
      const int qq = qt * KT + i;
      const long qi = (long)bh * S + min(qq, S - 1);
      const float lv = a.lse[qi], dv = a.dsum[qi];
      sL[i] = qq < S ? lv : 0.f;
      sD[i] = qq < S ? dv : 0.f;
    }
    // issued after the row statistics: loads complete in order, so waiting
    // for those must not wait for the prefetch
    if (qt + 1 < nqt) {
      tq.issue(qkv, a.ld_qkv, hd * a.qkv_hs, b, S, (qt + 1) * KT);
      tdo.issue(dO, a.ld_do, hd * DH, b, S, (qt + 1) * KT);
    }
    __syncthreads();
    // one query block at a time (not unrolled), as in the dQ pass
#pragma unroll 1
    for (int qb = 0; qb < KT / 32; ++qb) {
      f32x16 st, dp;
#pragma unroll
      for (int r = 0; r < 16; ++r) st[r] = dp[r] = 0.f;
#pragma unroll
      for (int s = 0; s < DH / 16; ++s) {
        st = mfma32(ld_frag(sQ + (qb * 32 + l32) * (DH + 8) + 16 * s + 8 * half), kf[s], st);
        dp = mfma32(ld_frag(sO + (qb * 32 + l32) * (DH + 8) + 16 * s + 8 * half), vf[s], dp);
      }
      f32x16 ds;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int qi = qb * 32 + perm_pos(r, half), qq = qt * KT + qi;
        const bool ok = full || (kv && qq < S && (!CAUSAL || key <= qq));
        const float p = ok ? __builtin_amdgcn_exp2f(fmaf(st[r], sl2, -sL[qi])) : 0.f;
        st[r] = p;
        ds[r] = p * (dp[r] - sD[qi]);
      }
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const bf16x8 pf = pack8(st, j), sf = pack8(ds, j);
#pragma unroll
        for (int db = 0; db < DH / 32; ++db) {
          dv[db] = mfma32(perm_frag<DH>(sO, db, qb, j, lane), pf, dv[db]);
          dk[db] = mfma32(perm_frag<DH>(sQ, db, qb, j, lane), sf, dk[db]);
        }
      }
    }
  }
  if (kv) {
    bf16* dst = static_cast<bf16*>(a.dqkv) + (long)(b * S + key) * a.ld_dqkv;
    store_rows<DH>(dk, scale, a.rope, key, rtab, half, dst + d + hd * DH);
    store_rows<DH>(dv, 1.f, false, key, nullptr, half, dst + 2 * d + hd * DH);
  }
}

// Whole backward of one (batch, head) with S <= KT (one query block, one key
// tile), one workgroup: P and dS are formed once.  Wave w owns queries
// 32w..32w+31 (lane = query, as in the dQ pass): it computes its score and
// dP blocks against the K and V tiles, accumulates dQ and keeps P and dS
// packed in registers.  The K/V tile space is then reused for P (row-major
// [query][key]); each wave now owns keys 32w..32w+31 and reads its P^T
// fragments from that block with the LDS transpose read, for dV = P^T dO;
// then dS goes to the same space for dK = dS^T Q.  The LDS holds Q, dO and
// the K/V tiles (74 KB at d_head 64: two workgroups per CU).
template <int DH, bool CAUSAL, int NW>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(DH <= 64 ? 2 : 1))) void attn_bwd_fused_bf16(AttnArgs a) {
  static_assert(NW * 32 == KT, "one 32-row block per wave covers the tile");
  constexpr int TP = KT * (DH + 8), PP = KT + 8;
  static_assert(2 * TP >= KT * PP, "P fits in the K/V tile space");
  __shared__ __attribute__((aligned(16))) bf16 sQ[TP];
  __shared__ __attribute__((aligned(16))) bf16 sdO[TP];
  __shared__ __attribute__((aligned(16))) bf16 sKV[2 * TP];  // K, V; later P, then dS ([query][key], pitch PP)
  bf16* sK = sKV;
  bf16* sV = sKV + TP;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, half = lane >> 5, l32 = lane & 31;
  const int bh = xcd_block(blockIdx.y, gridDim.y), b = bh / a.H, hd = bh % a.H, S = a.S;
  const int d = a.H * DH;
  const float2* rtab = a.rope_tab;
  const float scale = rsqrtf((float)DH), sl2 = kLog2e * scale;
  const bf16* qkv = static_cast<const bf16*>(a.qkv);
  const bf16* dO = static_cast<const bf16*>(a.dout);

  // Q, dO, K, V tiles (rows >= S zero; RoPE on Q and K), this lane's O row
  // and its LSE, every global load issued before the first LDS store, none
  // conditional on a lane (rows past S read a valid row, masked afterwards).  The
  // prologue is bound by memory bandwidth (all workgroups load at once), so
  // dO is read once: the row sum D = rowsum(dO * O) takes it from the tile.
  const int q = wave * 32 + l32;
  const bool qv = q < S;
  const long qrow = (long)(b * S + (qv ? q : 0));
  TileLoad<DH, 64 * NW> tq, tdo, tk, tv;
  tq.issue(qkv, a.ld_qkv, hd * a.qkv_hs, b, S, 0);
  tdo.issue(dO, a.ld_do, hd * DH, b, S, 0);
  tk.issue(qkv, a.ld_qkv, a.qkv_ko + hd * a.qkv_hs, b, S, 0);
  tv.issue(qkv, a.ld_qkv, a.qkv_vo + hd * a.qkv_hs, b, S, 0);
  bf16x8 orw[DH / 16];
  {
    const bf16* orow = static_cast<const bf16*>(a.o) + qrow * a.ld_o + hd * DH;
#pragma unroll
    for (int s = 0; s < DH / 16; ++s) orw[s] = ld_frag(orow + 16 * s + 8 * half);  // qrow clamped
  }
  const float lse_raw = a.lse[(long)bh * S + (qv ? q : 0)];
  tq.store(sQ, rot_load(a), S, 0, rtab);
  tdo.store(sdO, false, S, 0, rtab);
  tk.store(sK, rot_load(a), S, 0, rtab);
  tv.store(sV, false, S, 0, rtab);
  __syncthreads();
  // the O row and the LSE were loaded last; masked only here, at their first use
  const float lse = qv ? lse_raw : 0.f;
  float dsum = 0.f;
#pragma unroll
  for (int s = 0; s < DH / 16; ++s) {
    float ov[8], dv[8];
    unpack_frag(orw[s], ov);
#pragma unroll
    for (int v = 0; v < 8; ++v) ov[v] = qv ? ov[v] : 0.f;
    unpack_frag(ld_frag(sdO + q * (DH + 8) + 16 * s + 8 * half), dv);  // rows >= S are zero
#pragma unroll
    for (int v = 0; v < 8; ++v) dsum += ov[v] * dv[v];
  }
  dsum += __shfl_xor(dsum, 32, 64);

  // ---- scores, P, dS and dQ (lane = query)
  const bool full = !CAUSAL && S == KT;
  bf16x8 pk[KT / 32][2], sk[KT / 32][2];
  {
    f32x16 dq[DH / 32];
#pragma unroll
    for (int i = 0; i < DH / 32; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) dq[i][r] = 0.f;
#pragma unroll
    for (int kb = 0; kb < KT / 32; ++kb) {
      f32x16 st, dp;
#pragma unroll
      for (int r = 0; r < 16; ++r) st[r] = dp[r] = 0.f;
#pragma unroll
      for (int s = 0; s < DH / 16; ++s) {
        const bf16x8 qf = ld_frag(sQ + q * (DH + 8) + 16 * s + 8 * half);
        const bf16x8 df = ld_frag(sdO + q * (DH + 8) + 16 * s + 8 * half);
        st = mfma32(ld_frag(sK + (kb * 32 + l32) * (DH + 8) + 16 * s + 8 * half), qf, st);
        dp = mfma32(ld_frag(sV + (kb * 32 + l32) * (DH + 8) + 16 * s + 8 * half), df, dp);
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = kb * 32 + perm_pos(r, half);
        const bool ok = full || (qv && key < S && (!CAUSAL || key <= q));
        const float p = ok ? __builtin_amdgcn_exp2f(fmaf(st[r], sl2, -lse)) : 0.f;
        st[r] = p;
        dp[r] = p * (dp[r] - dsum);  // dS
      }
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        pk[kb][j] = pack8(st, j);
        sk[kb][j] = pack8(dp, j);
#pragma unroll
        for (int db = 0; db < DH / 32; ++db) dq[db] = mfma32(perm_frag<DH>(sK, db, kb, j, lane), sk[kb][j], dq[db]);
      }
    }
    if (qv) {
      bf16* dst = static_cast<bf16*>(a.dqkv) + (long)(b * S + q) * a.ld_dqkv + hd * DH;
      store_rows<DH>(dq, scale, a.rope, q, rtab, half, dst);
    }
  }

  // a [query][key] block from the packed registers: register values 8j..8j+7
  // of key block kb are keys kb*32 + 16j + 4*half + {0..3, 8..11}
  auto put = [&](bf16x8 (&v)[KT / 32][2]) {
#pragma unroll
    for (int kb = 0; kb < KT / 32; ++kb)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const uint4 w = __builtin_bit_cast(uint4, v[kb][j]);
        bf16* row = sKV + q * PP + kb * 32 + 16 * j + 4 * half;
        *reinterpret_cast<uint2*>(row) = make_uint2(w.x, w.y);
        *reinterpret_cast<uint2*>(row + 8) = make_uint2(w.z, w.w);
      }
  };
  // dX[key][dim] += sum_q M[q][key] X[q][dim] over the whole tile (lane = key)
  auto tmul = [&](const bf16* sX, f32x16 (&acc)[DH / 32]) {
#pragma unroll
    for (int i = 0; i < DH / 32; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][r] = 0.f;
#pragma unroll
    for (int qb = 0; qb < KT / 32; ++qb)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const bf16x8 mf = perm_frag<KT>(sKV, wave, qb, j, lane);
#pragma unroll
        for (int db = 0; db < DH / 32; ++db) acc[db] = mfma32(perm_frag<DH>(sX, db, qb, j, lane), mf, acc[db]);
      }
  };
  const int key = wave * 32 + l32;
  const bool kv = key < S;
  bf16* kdst = static_cast<bf16*>(a.dqkv) + (long)(b * S + (kv ? key : 0)) * a.ld_dqkv;

  __syncthreads();  // every wave is done with K and V
  put(pk);
  __syncthreads();
  {
    f32x16 dv[DH / 32];
    tmul(sdO, dv);
    if (kv) store_rows<DH>(dv, 1.f, false, key, nullptr, half, kdst + 2 * d + hd * DH);
  }
  __syncthreads();  // every wave is done with P
  put(sk);
  __syncthreads();
  {
    f32x16 dk[DH / 32];
    tmul(sQ, dk);
    if (kv) store_rows<DH>(dk, scale, a.rope, key, rtab, half, kdst + d + hd * DH);
  }
}

// ================================================================ fp32 (small stages)
// One workgroup per (batch, head), one thread per query (forward, dQ) or key
// (dK, dV); head dim <= 128.
__device__ __forceinline__ float rot_ld(const float* row, int i, int dh, int pos, bool rot,
                                        const float2* rtab) {
  if (!rot) return row[i];
  const int h2 = dh / 2, j = i < h2 ? i : i - h2;
  float cs, sn;
  rope_cs(rtab, pos, j, dh, &cs, &sn);
  const float x1 = row[j], x2 = row[j + h2];
  return i < h2 ? x1 * cs - x2 * sn : x2 * cs + x1 * sn;
}

__global__ __launch_bounds__(256) void attn_fwd_f32(AttnArgs a) {
  const int bh = blockIdx.x, b = bh / a.H, hd = bh % a.H, S = a.S, DH = a.dh, d = a.H * DH;
  const float2* rtab = a.rope_tab;
  const float sl2 = kLog2e * rsqrtf((float)DH);
  const float* qkv = static_cast<const float*>(a.qkv);
  for (int q = threadIdx.x; q < S; q += blockDim.x) {
    const float* qr = qkv + (long)(b * S + q) * a.ld_qkv + hd * DH;
    float qv[128];
    for (int i = 0; i < DH; ++i) qv[i] = rot_ld(qr, i, DH, q, a.rope, rtab);
    const int kend = a.causal ? q + 1 : S;
    float m = -INFINITY;
    for (int k = 0; k < kend; ++k) {
      const float* kr = qkv + (long)(b * S + k) * a.ld_qkv + d + hd * DH;
      float sdot = 0.f;
      for (int i = 0; i < DH; ++i) sdot += qv[i] * rot_ld(kr, i, DH, k, a.rope, rtab);
      m = fmaxf(m, sdot * sl2);
    }
    float l = 0.f, o[128];
    for (int i = 0; i < DH; ++i) o[i] = 0.f;
    for (int k = 0; k < kend; ++k) {
      const float* kr = qkv + (long)(b * S + k) * a.ld_qkv + d + hd * DH;
      const float* vr = kr + d;
      float sdot = 0.f;
      for (int i = 0; i < DH; ++i) sdot += qv[i] * rot_ld(kr, i, DH, k, a.rope, rtab);
      const float p = exp2f(sdot * sl2 - m);
      l += p;
      for (int i = 0; i < DH; ++i) o[i] += p * vr[i];
    }
    float* orow = static_cast<float*>(a.o) + (long)(b * S + q) * a.ld_o + hd * DH;
    for (int i = 0; i < DH; ++i) orow[i] = o[i] / l;
    a.lse[(long)bh * S + q] = m + log2f(l);
  }
}

__global__ __launch_bounds__(256) void attn_bwd_f32(AttnArgs a) {
  extern __shared__ float sD[];  // [S]
  const int bh = blockIdx.x, b = bh / a.H, hd = bh % a.H, S = a.S, DH = a.dh, d = a.H * DH;
  const float2* rtab = a.rope_tab;
  const float scale = rsqrtf((float)DH), sl2 = kLog2e * scale;
  const float* qkv = static_cast<const float*>(a.qkv);
  const float* O = static_cast<const float*>(a.o);
  const float* dO = static_cast<const float*>(a.dout);
  float* dqkv = static_cast<float*>(a.dqkv);
  auto score = [&](int q, int k, const float* qv) {
    const float* kr = qkv + (long)(b * S + k) * a.ld_qkv + d + hd * DH;
    float sdot = 0.f;
    for (int i = 0; i < DH; ++i) sdot += qv[i] * rot_ld(kr, i, DH, k, a.rope, rtab);
    return exp2f(sdot * sl2 - a.lse[(long)bh * S + q]);
  };
  auto dpdot = [&](int q, int k) {
    const float* vr = qkv + (long)(b * S + k) * a.ld_qkv + 2 * d + hd * DH;
    const float* dr = dO + (long)(b * S + q) * a.ld_do + hd * DH;
    float s = 0.f;
    for (int i = 0; i < DH; ++i) s += dr[i] * vr[i];
    return s;
  };
  for (int q = threadIdx.x; q < S; q += blockDim.x) {
    const float* orow = O + (long)(b * S + q) * a.ld_o + hd * DH;
    const float* drow = dO + (long)(b * S + q) * a.ld_do + hd * DH;
    float s = 0.f;
    for (int i = 0; i < DH; ++i) s += orow[i] * drow[i];
    sD[q] = s;
    a.dsum[(long)bh * S + q] = s;
  }
  __syncthreads();
  float buf[128], acc[128];
  // dQ
  for (int q = threadIdx.x; q < S; q += blockDim.x) {
    const float* qr = qkv + (long)(b * S + q) * a.ld_qkv + hd * DH;
    for (int i = 0; i < DH; ++i) { buf[i] = rot_ld(qr, i, DH, q, a.rope, rtab); acc[i] = 0.f; }
    const int kend = a.causal ? q + 1 : S;
    for (int k = 0; k < kend; ++k) {
      const float ds = score(q, k, buf) * (dpdot(q, k) - sD[q]);
      const float* kr = qkv + (long)(b * S + k) * a.ld_qkv + d + hd * DH;
      for (int i = 0; i < DH; ++i) acc[i] += ds * rot_ld(kr, i, DH, k, a.rope, rtab);
    }
    float* dst = dqkv + (long)(b * S + q) * a.ld_dqkv + hd * DH;
    for (int i = 0; i < DH; ++i) acc[i] *= scale;
    if (a.rope) {
      for (int j = 0; j < DH / 2; ++j) {
        float cs, sn;
        rope_cs(rtab, q, j, DH, &cs, &sn);
        const float d1 = acc[j], d2 = acc[j + DH / 2];
        acc[j] = d1 * cs + d2 * sn;
        acc[j + DH / 2] = d2 * cs - d1 * sn;
      }
    }
    for (int i = 0; i < DH; ++i) dst[i] = acc[i];
  }
  // dK, dV
  for (int k = threadIdx.x; k < S; k += blockDim.x) {
    for (int i = 0; i < DH; ++i) buf[i] = acc[i] = 0.f;  // buf = dV, acc = dK
    const int qbeg = a.causal ? k : 0;
    for (int q = qbeg; q < S; ++q) {
      const float* qr = qkv + (long)(b * S + q) * a.ld_qkv + hd * DH;
      float qv[128];
      for (int i = 0; i < DH; ++i) qv[i] = rot_ld(qr, i, DH, q, a.rope, rtab);
      const float p = score(q, k, qv);
      const float ds = p * (dpdot(q, k) - sD[q]);
      const float* dr = dO + (long)(b * S + q) * a.ld_do + hd * DH;
      for (int i = 0; i < DH; ++i) { buf[i] += p * dr[i]; acc[i] += ds * qv[i]; }
    }
    float* dst = dqkv + (long)(b * S + k) * a.ld_dqkv;
    for (int i = 0; i < DH; ++i) acc[i] *= scale;
    if (a.rope) {
      for (int j = 0; j < DH / 2; ++j) {
        float cs, sn;
        rope_cs(rtab, k, j, DH, &cs, &sn);
        const float d1 = acc[j], d2 = acc[j + DH / 2];
        acc[j] = d1 * cs + d2 * sn;
        acc[j + DH / 2] = d2 * cs - d1 * sn;
      }
    }
    for (int i = 0; i < DH; ++i) { dst[d + hd * DH + i] = acc[i]; dst[2 * d + hd * DH + i] = buf[i]; }
  }
}

// ================================================================ launchers
static bool al16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// four waves (128 queries or keys) per workgroup
constexpr int ATT_NW = 4;

template <int DH>
static hipError_t fwd_dh(const AttnArgs& a, hipStream_t s) {
  dim3 grid((a.S + 32 * ATT_NW - 1) / (32 * ATT_NW), a.B * a.H), block(64 * ATT_NW);
  if (a.causal) RG_LAUNCH((attn_fwd_bf16<DH, true, ATT_NW>), grid, block, 0, s, a);
  else RG_LAUNCH((attn_fwd_bf16<DH, false, ATT_NW>), grid, block, 0, s, a);
  return hipGetLastError();
}
template <int DH>
static hipError_t bwd_dh(const AttnArgs& a, hipStream_t s) {
  dim3 grid((a.S + 32 * ATT_NW - 1) / (32 * ATT_NW), a.B * a.H), block(64 * ATT_NW);
  if (a.S <= KT) {  // one tile: the fused single-pass backward
    if (a.causal) RG_LAUNCH((attn_bwd_fused_bf16<DH, true, ATT_NW>), dim3(1, a.B * a.H), block, 0, s, a);
    else RG_LAUNCH((attn_bwd_fused_bf16<DH, false, ATT_NW>), dim3(1, a.B * a.H), block, 0, s, a);
    return hipGetLastError();
  }
  if (a.causal) {
    RG_LAUNCH((attn_bwd_dq_bf16<DH, true, ATT_NW>), grid, block, 0, s, a);
    RG_LAUNCH((attn_bwd_dkdv_bf16<DH, true, ATT_NW>), grid, block, 0, s, a);
  } else {
    RG_LAUNCH((attn_bwd_dq_bf16<DH, false, ATT_NW>), grid, block, 0, s, a);
    RG_LAUNCH((attn_bwd_dkdv_bf16<DH, false, ATT_NW>), grid, block, 0, s, a);
  }
  return hipGetLastError();
}

static hipError_t check(int dtype, const AttnArgs& a, bool bwd) {
  if (a.B <= 0 || a.S <= 0 || a.H <= 0 || !a.qkv || !a.o || !a.lse) return hipErrorInvalidValue;
  if (bwd && (!a.dout || !a.dsum || !a.dqkv)) return hipErrorInvalidValue;
  if (a.rope && (!a.rope_tab || a.rope_rows < a.S)) return hipErrorInvalidValue;
  if (a.rope_in_qkv && (!a.rope || dtype != DT_BF16)) return hipErrorInvalidValue;
  const int d = a.H * a.dh;
  const bool three_block = a.qkv_hs == a.dh && a.qkv_ko == d && a.qkv_vo == 2 * d;
  const bool per_head = a.qkv_hs == 3 * a.dh && a.qkv_ko == a.dh && a.qkv_vo == 2 * a.dh;
  if (!three_block && !(per_head && dtype == DT_BF16)) return hipErrorInvalidValue;
  if (dtype == DT_BF16) {
    if (a.dh != 64 && a.dh != 128) return hipErrorInvalidValue;
    if (a.ld_qkv % 8 || a.ld_o % 8 || !al16(a.qkv) || !al16(a.o)) return hipErrorInvalidValue;
    if (bwd && (a.ld_do % 8 || a.ld_dqkv % 4 || !al16(a.dout))) return hipErrorInvalidValue;
  } else {
    if (a.dh > 128 || a.dh % 2 || a.S > 4096) return hipErrorInvalidValue;
  }
  return hipSuccess;
}

// the three-block Q | K | V order when no per-head layout is given
static AttnArgs with_layout(AttnArgs a) {
  if (a.qkv_hs == 0 && a.qkv_ko == 0 && a.qkv_vo == 0) {
    a.qkv_hs = a.dh;
    a.qkv_ko = a.H * a.dh;
    a.qkv_vo = 2 * a.H * a.dh;
  }
  return a;
}

hipError_t launch_attn_fwd(int dtype, const AttnArgs& a0, hipStream_t s) {
  const AttnArgs a = with_layout(a0);
  hipError_t e = check(dtype, a, false);
  if (e != hipSuccess) return e;
  if (dtype == DT_BF16) return a.dh == 64 ? fwd_dh<64>(a, s) : fwd_dh<128>(a, s);
  RG_LAUNCH(attn_fwd_f32, dim3(a.B * a.H), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_attn_bwd(int dtype, const AttnArgs& a0, hipStream_t s) {
  const AttnArgs a = with_layout(a0);
  hipError_t e = check(dtype, a, true);
  if (e != hipSuccess) return e;
  if (dtype == DT_BF16) return a.dh == 64 ? bwd_dh<64>(a, s) : bwd_dh<128>(a, s);
  RG_LAUNCH(attn_bwd_f32, dim3(a.B * a.H), dim3(256), a.S * sizeof(float), s, a);
  return hipGetLastError();
}

}  // namespace rg
