// Device pieces of the attention core shared by the attention kernels and the
// QKV projection's fused attention epilogue: softmax(Q K^T / sqrt(d_head)) V
// per (batch, head) on MFMA 32x32x16, with the score block held transposed
// (one query, or key, per lane) and the probabilities fed to the second MFMA
// from registers against LDS transpose reads of the other operand.
#pragma once
#include "common.h"

namespace rg {

constexpr float kLog2e = 1.4426950408889634f;

// cos and sin of the rotation angle pos * theta^(-2i/dh) of pair i, from the
// stage's table [max_seq][dh/2] (computed once in double precision)
__device__ __forceinline__ void rope_cs(const float2* tab, int pos, int i, int dh, float* c, float* s) {
  const float2 v = tab[(long)pos * (dh / 2) + i];
  *c = v.x;
  *s = v.y;
}

constexpr int KT = 128;      // keys (or queries) per LDS tile: a whole 128-token sequence in one

// A-operand fragment of (tile^T): rows = dims db*32 + lane%32 of a row-major
// [row][dim] LDS tile, k = the 8 permuted rows matching register values
// r = 8j..8j+7 of score block kb (rows kb*32 + 16j + 4*half + {0..3, 8..11}).
template <int DH>
__device__ __forceinline__ bf16x8 perm_frag(const bf16* tile, int db, int kb, int j, int lane) {
  const int g = lane >> 4, dims = db * 32 + 16 * (g & 1), rows = kb * 32 + 16 * j + 4 * (g >> 1);
  const uint2 lo = lds_tr4(tile, DH + 8, rows, dims, lane), hi = lds_tr4(tile, DH + 8, rows + 8, dims, lane);
  return __builtin_bit_cast(bf16x8, make_uint4(lo.x, lo.y, hi.x, hi.y));
}

__device__ __forceinline__ bf16x8 pack8(const f32x16& v, int j) {
  float t[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) t[i] = v[8 * j + i];
  return pack_frag(t);
}

// position of register value r within a 32-wide score block for this lane half
__device__ __forceinline__ int perm_pos(int r, int half) { return 8 * (r >> 2) + 4 * half + (r & 3); }

// Writes a 32-row x DH accumulator (transposed layout: lane = row, dims
// 8*(r/4) + 4*half + r%4 of block db) scaled, optionally un-rotated.
template <int DH>
__device__ __forceinline__ void store_rows(f32x16 (&acc)[DH / 32], float scale, bool unrot, int pos,
                                           const float2* rtab, int half, bf16* dst) {
  if (unrot) {
#pragma unroll
    for (int db = 0; db < DH / 64; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int i = db * 32 + perm_pos(r, half);
        float cs, sn;
        rope_cs(rtab, pos, i, DH, &cs, &sn);
        const float d1 = acc[db][r], d2 = acc[db + DH / 64][r];
        acc[db][r] = d1 * cs + d2 * sn;
        acc[db + DH / 64][r] = d2 * cs - d1 * sn;
      }
  }
#pragma unroll
  for (int db = 0; db < DH / 32; ++db)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      float v[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) v[q] = acc[db][4 * g + q] * scale;
      St<bf16>::st4(dst, db * 32 + 8 * g + 4 * half, v);
    }
}

// The same rows (unscaled, not rotated) through LDS: each lane writes its row
// into the 32 staging rows (pitch DH + 8, private to the wave), then each
// store instruction writes whole rows, 16 B per lane (8 rows of 128 B at DH
// 64), so the stores can be streamed (st16).  One wave's LDS operations run in
// order, so the reads see the writes without a barrier.
template <int DH>
__device__ __forceinline__ void store_rows_staged(const f32x16 (&acc)[DH / 32], float scale, int half, int lane,
                                                  bf16* stage, bf16* dst0, long ld, bool nt) {
  const int l32 = lane & 31;
#pragma unroll
  for (int db = 0; db < DH / 32; ++db)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      float v[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) v[q] = acc[db][4 * g + q] * scale;
      St<bf16>::st4(stage + l32 * (DH + 8), db * 32 + 8 * g + 4 * half, v);
    }
  constexpr int CPR = DH / 8;  // 16-B chunks per row
#pragma unroll
  for (int k = lane; k < 32 * CPR; k += 64) {
    const int row = k / CPR, c = k % CPR;
    st16(dst0 + row * ld + 8 * c, ld_frag(stage + row * (DH + 8) + 8 * c), nt);
  }
}

// One wave's 32 queries q0..q0+31 against a whole sequence of KT = 128 keys,
// all staged in LDS as row-major [row][dim] bf16 tiles of pitch DH + 8 (no
// mask: every key is valid).  Writes the wave's O rows (bf16, rows of stride
// ld_o from o0, the row of query q0) and, from lanes 0..31, the base-2
// log-sum-exp of the scaled scores at lse_row[query].  The wave's own Q rows
// are read once, first, and then hold the O tile on its way out.
template <int DH>
__device__ __forceinline__ void attn_seq128_wave(bf16* sQ, const bf16* sK, const bf16* sV, int q0, int lane,
                                                 bf16* o0, long ld_o, bool nt, float* lse_row) {
  const int half = lane >> 5, l32 = lane & 31, q = q0 + l32;
  const float sl2 = kLog2e * rsqrtf((float)DH);
  bf16x8 qf[DH / 16];
#pragma unroll
  for (int s = 0; s < DH / 16; ++s) qf[s] = ld_frag(sQ + q * (DH + 8) + 16 * s + 8 * half);
  f32x16 sc[KT / 32];
#pragma unroll
  for (int kb = 0; kb < KT / 32; ++kb) {
#pragma unroll
    for (int r = 0; r < 16; ++r) sc[kb][r] = 0.f;
#pragma unroll
    for (int s = 0; s < DH / 16; ++s)
      sc[kb] = mfma32(ld_frag(sK + (kb * 32 + l32) * (DH + 8) + 16 * s + 8 * half), qf[s], sc[kb]);
  }
  float mx = -INFINITY;
#pragma unroll
  for (int kb = 0; kb < KT / 32; ++kb)
#pragma unroll
    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sc[kb][r]);
  mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
  const float m2 = mx * sl2;  // the scale is positive: the max of the scaled scores
  float rs = 0.f;
#pragma unroll
  for (int kb = 0; kb < KT / 32; ++kb)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      sc[kb][r] = __builtin_amdgcn_exp2f(fmaf(sc[kb][r], sl2, -m2));
      rs += sc[kb][r];
    }
  rs += __shfl_xor(rs, 32, 64);
  f32x16 oacc[DH / 32];
#pragma unroll
  for (int i = 0; i < DH / 32; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[i][r] = 0.f;
#pragma unroll
  for (int kb = 0; kb < KT / 32; ++kb)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const bf16x8 pf = pack8(sc[kb], j);
#pragma unroll
      for (int db = 0; db < DH / 32; ++db) oacc[db] = mfma32(perm_frag<DH>(sV, db, kb, j, lane), pf, oacc[db]);
    }
  store_rows_staged<DH>(oacc, 1.f / rs, half, lane, sQ + q0 * (DH + 8), o0, ld_o, nt);
  if (half == 0) lse_row[q] = m2 + log2f(rs);
}

}  // namespace rg
