// Bottleneck adapters of Eq. (1), h <- h + gelu(h W_down) W_up, fused with the
// residual add and the normalisation that follow them in the block, and their
// backward with the fp32 weight-gradient accumulation.
//
// bf16 row kernels: one workgroup per 16 tokens.  Both adapter contractions
// use MFMA 16x16x32 in the transposed orientation (the weight is the A operand,
// the 16 tokens the B operand), so every lane ends up owning four consecutive
// features of one token; row statistics of the norm reduce over the four
// lanes sharing a token (shuffles) and then over waves (LDS).
// Weight gradients are long-K (K = tokens), tiny-output contractions: a
// split-K MFMA kernel with LDS-transposed tiles whose per-chunk partial sums
// a second kernel adds in chunk order (no atomics: the same bits every run).
#include <initializer_list>

#include "common.h"
#include "kernels.h"

namespace rg {

constexpr int TOK = 16;   // tokens per workgroup of the bf16 row kernels
constexpr int MB = 64;    // adapter bottleneck of the bf16 path
constexpr int GP = MB + 8;

// ================================================================ bf16 forward, d <= 1024
// One workgroup of 16 waves per 16 tokens: the whole adapter, the residual
// add and the norm in one kernel.
// Laid out so that nothing waits twice on memory and every row access moves
// 16 B per lane: all global loads are issued before the first barrier (the
// norm's gain and shift once per workgroup, the residual and z tiles by DMA
// into LDS, the weight fragments of both projections into registers); the up
// projection's fp32 result is staged in LDS; the add + norm phase then runs
// one wave per token (NW == TOK), so the row statistics are wave reductions,
// and each lane handles the 8 features of chunks lane + 64 j.  The outputs are
// streamed (st16).  The down projection's k-slice
// partial sums go through LDS unit-major, [slice][unit][token] with a token
// stride of 17 floats: the MFMA writes (16 tokens of 4 units per lane group)
// and the GELU phase's reads (one unit per lane) spread over the banks,
// where 64-float token rows put the 16 tokens of a lane group on one bank.
template <int FB>
__global__ __launch_bounds__(1024) void adapter_fwd_rows(AdapterFwdArgs a) {
  constexpr int NW = 16, KS = 4, TOKP = 17;
  constexpr int D = 256 * FB, DP = D + 8, VP = D + 4;
  constexpr int SLICE = D / KS, NSTEP = SLICE / 32;
  static_assert(NW == TOK, "one wave per token in the norm phase");
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  constexpr int NC = D / 8, NJ = (NC + 63) / 64;  // 16-B chunks per row; per lane in the norm phase
  bf16* sZ = reinterpret_cast<bf16*>(smem);                // [TOK][DP]
  bf16* sG = sZ + TOK * DP;                                // [TOK][GP]
  float* sUp = reinterpret_cast<float*>(sG + TOK * GP);    // [KS][MB][TOKP]
  float* sV = sUp + KS * MB * TOKP;                        // [TOK][VP]
  bf16* sR = reinterpret_cast<bf16*>(sV + TOK * VP);       // [TOK][D] residual
  bf16* sGB = sR + TOK * D;                                // [2][D] gain, shift
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, l16 = lane & 15, grp = lane >> 4;
  const int T = a.T, t0 = xcd_block(blockIdx.x, gridDim.x) * TOK;
  const bf16* z = static_cast<const bf16*>(a.z);
  const bool nt = stream_out((long)T * D * 2);  // outputs streamed (common.h)

  // ---- every global load up front, the ones needed last first: the z wait below then
  // covers them as well.  The norm's gain and shift: 2 NC chunks, one per thread of the
  // first waves; every wave loads (a chunk index taken modulo), so no load is conditional
  // and the compiler's wait counts stay exact.  An absent gain / shift reads z's first row.
  const bf16* gp = static_cast<const bf16*>(a.norm != Norm::None ? a.gamma : a.z);
  const bf16* bp = static_cast<const bf16*>(a.norm == Norm::LN ? a.beta : a.z);
  const int gbc = (wave * 64 + lane) % (2 * NC);
  const uint4 gbv = *reinterpret_cast<const uint4*>(gbc < NC ? gp + 8 * gbc : bp + 8 * (gbc - NC));
  {  // the residual tile by DMA into unpadded LDS rows: instruction k covers slots
     // 64 k .. 64 k + 63, slot s = chunk s % NC of row s / NC; 8 FB instructions
    const bf16* rb = static_cast<const bf16*>(a.res) + (long)t0 * D;
#pragma unroll
    for (int i = 0; i < (FB + 1) / 2; ++i) {
      const int k = i * NW + wave;
      if (k < 8 * FB) {  // wave-uniform
        const int sl = k * 64 + lane, r = sl / NC, c = sl % NC;
        dma16_m0(rb, t0 + r < T ? (uint32_t)((r * D + 8 * c) * 2) : 0u,
                 lds_addr(sR) + (uint32_t)__builtin_amdgcn_readfirstlane(k * 1024));
      }
    }
  }
  // The z tile goes by DMA straight into its padded LDS
  // rows: 16-B slot s is chunk s % SPR of row s / SPR, the row's last slot is padding; the
  // slots past the tile land in the sG / sUp space, which is written only after the wait.
  // Slots with no data (padding, rows past T) load the tile's first chunk instead.
  constexpr int SPR = DP / 8, NSLOT = TOK * SPR, NI = (NSLOT + 1023) / 1024;
  static_assert(NI * 1024 * 16 <= (TOK * DP + TOK * GP) * 2 + KS * MB * TOKP * 4,
                "the DMA's spare slots stay clear of sV");
  {
    const bf16* zb = z + (long)t0 * D;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int sl = (i * NW + wave) * 64 + lane, r = sl / SPR, c = sl % SPR;
      const bool ok = sl < NSLOT && c < D / 8 && t0 + r < T;
      dma16_m0(zb, ok ? (uint32_t)((r * D + 8 * c) * 2) : 0u,
               lds_addr(sZ) + (uint32_t)__builtin_amdgcn_readfirstlane((i * NW + wave) * 1024));
    }
  }
  const bool has_ad = a.wdn_t != nullptr;  // else: residual add + norm only
  const int ug = wave % 4, ks = wave / 4;
  bf16x8 wd[NSTEP];
  if (has_ad) {
#pragma unroll
    for (int j = 0; j < NSTEP; ++j) wd[j] = ld_frag(pack_a_frag(a.wdn_t, D, wave, j, lane));
  }
  const int f0 = wave * 16 * FB;
  bf16x8 w0[FB], w1[FB];
  if (has_ad) {
#pragma unroll
    for (int b = 0; b < FB; ++b) {
      w0[b] = ld_frag(pack_b_frag(a.wup_t, D, wave, b, 0, lane));
      w1[b] = ld_frag(pack_b_frag(a.wup_t, D, wave, b, 1, lane));
    }
  }
  const int tw = t0 + wave;  // this wave's token in the norm phase
  const bool twv = tw < T;
  const long wrow = (long)(twv ? tw : 0) * D;
  // the z tile (and the residual tile and the gain and shift, issued before it) have
  // landed once no more than the weight-fragment loads issued after it are pending
  // (vmcnt counts in issue order)
  if (has_ad) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(NSTEP + 2 * FB) : "memory");
  else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  if (wave * 64 + lane < 2 * NC) *reinterpret_cast<uint4*>(sGB + 8 * gbc) = gbv;
  __syncthreads();

  // ---- U^T[unit][token] = W_down^T[unit][:] . z[token][:], k split over KS waves
  if (has_ad) {
    const bf16* zr = sZ + l16 * DP + ks * SLICE + 8 * grp;
    f32x4 u = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < NSTEP; ++j) u = mfma16(wd[j], ld_frag(zr + j * 32), u);
#pragma unroll
    for (int r = 0; r < 4; ++r) sUp[(ks * MB + ug * 16 + 4 * grp + r) * TOKP + l16] = u[r];
    __syncthreads();
    {  // one (token, unit) pair per thread: sum of the k slices, GELU
      const int unit = lane, tok = wave;
      float sum = 0.f;
#pragma unroll
      for (int k2 = 0; k2 < KS; ++k2) sum += sUp[(k2 * MB + unit) * TOKP + tok];
      if (a.u && t0 + tok < T) St<bf16>::st_nt(static_cast<bf16*>(a.u), (long)(t0 + tok) * MB + unit, sum);
      sG[tok * GP + unit] = f2bf(gelu_fast(sum));
    }
    __syncthreads();
  }

  // ---- out^T[f][token] = W_up^T[f][:] . G[token][:]  -> sV (fp32)
  if (has_ad) {
    const bf16x8 g0 = ld_frag(sG + l16 * GP + 8 * grp), g1 = ld_frag(sG + l16 * GP + 32 + 8 * grp);
#pragma unroll
    for (int b = 0; b < FB; ++b) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      acc = mfma16(w0[b], g0, acc);
      acc = mfma16(w1[b], g1, acc);
      *reinterpret_cast<float4*>(sV + l16 * VP + f0 + b * 16 + 4 * grp) = make_float4(acc[0], acc[1], acc[2], acc[3]);
    }
    __syncthreads();
  }

  // ---- add + norm, wave = token; lane: the 8 features of chunk lane + 64 j
  if (!twv) return;
  float v[NJ][8];
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int c = lane + 64 * j;
    if (NC % 64 == 0 || c < NC) {
      float zz[8], r8[8];
      unpack_frag(*reinterpret_cast<const bf16x8*>(sZ + wave * DP + 8 * c), zz);
      unpack_frag(*reinterpret_cast<const bf16x8*>(sR + wave * D + 8 * c), r8);
      float4 u0 = make_float4(0.f, 0.f, 0.f, 0.f), u1 = u0;
      if (has_ad) {
        u0 = *reinterpret_cast<const float4*>(sV + wave * VP + 8 * c);
        u1 = *reinterpret_cast<const float4*>(sV + wave * VP + 8 * c + 4);
      }
      const float up[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
#pragma unroll
      for (int e = 0; e < 8; ++e) v[j][e] = up[e] + zz[e] + r8[e];
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[j][e] = 0.f;
    }
  }
  auto store_rows = [&](bf16* dst, const float (*val)[8]) {
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int c = lane + 64 * j;
      if (NC % 64 == 0 || c < NC) st16(dst + wrow + 8 * c, pack_frag(val[j]), nt);
    }
  };
  if (a.norm == Norm::None) {
    store_rows(static_cast<bf16*>(a.out), v);
    return;
  }
  constexpr float inv_d = 1.f / (float)D;
  float mean = 0.f;
  if (a.norm == Norm::LN) {
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      s += ((v[j][0] + v[j][1]) + (v[j][2] + v[j][3])) + ((v[j][4] + v[j][5]) + (v[j][6] + v[j][7]));
    mean = wave_sum(s) * inv_d;
  } else {
    store_rows(static_cast<bf16*>(a.out), v);  // RMS: the residual stream h itself is an output
  }
  float s2 = 0.f;
#pragma unroll
  for (int j = 0; j < NJ; ++j)
    if (NC % 64 == 0 || lane + 64 * j < NC)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float c = v[j][e] - mean;
        s2 += c * c;
      }
  const float rstd = rsqrtf(wave_sum(s2) * inv_d + a.eps);
  if (a.rstd && lane == 0) a.rstd[tw] = rstd;
  float xh[NJ][8], o[NJ][8];
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int c = min(lane + 64 * j, NC - 1);  // lanes past the row compute and store nothing useful
    float gm[8], bt[8];
    unpack_frag(*reinterpret_cast<const bf16x8*>(sGB + 8 * c), gm);
    unpack_frag(*reinterpret_cast<const bf16x8*>(sGB + D + 8 * c), bt);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      xh[j][e] = (v[j][e] - mean) * rstd;
      o[j][e] = xh[j][e] * gm[e] + (a.norm == Norm::LN ? bt[e] : 0.f);  // RMSNorm has no shift
    }
  }
  store_rows(static_cast<bf16*>(a.norm == Norm::LN ? a.out : a.out_norm), o);
  if (a.xhat) store_rows(static_cast<bf16*>(a.xhat), xh);
}

// ================================================================ bf16 backward, d <= 1024
// One workgroup of 16 waves per 16 tokens.
//  1. The norm backward with one wave per token: every global row access is a
//     contiguous 512-B run per instruction and the row sums are wave
//     reductions; dz stays in fp32 registers and goes to LDS (bf16) for
//     2. dV = dZ W_up^T (k split over 4 waves, MFMA, lane = token), dU =
//     dV * gelu'(U) with one (token, unit) pair per thread;
//  3. dU W_down^T (MFMA), staged in LDS as fp32, then dzin = dz + that, again
//     one wave per token.
// Every global load the kernel makes is issued before the first phase, the
// weight fragments of both contractions first (at d = 1024 those of W_down
// after the norm backward, for want of registers).
template <int NW, int FB>
__global__ __launch_bounds__(NW * 64) void adapter_bwd_bf16(AdapterBwdArgs a) {
  constexpr int KS = NW / 4, TOKP = TOK + 1;
  constexpr int D = 16 * NW * FB, DP = D + 8, VP = D + 4, SLICE = D / KS;
  static_assert(NW == TOK, "one wave per token in the row phases");
  static_assert(D == 256 * FB, "four consecutive features per lane, FB runs of 256");
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  bf16* sdZ = reinterpret_cast<bf16*>(smem);                       // [TOK][DP]
  bf16* sdU = sdZ + TOK * DP;                                      // [TOK][GP]
  float* sPart = reinterpret_cast<float*>(sdU + TOK * GP);         // [KS][MB][TOKP]
  float* sV = sPart + KS * MB * TOKP;                              // [TOK][VP]
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, l16 = lane & 15, grp = lane >> 4;
  const int T = a.T;
  const bool nt = stream_out((long)T * D * 2);  // outputs streamed (common.h)
  const int tw = xcd_block(blockIdx.x, gridDim.x) * TOK + wave;  // this wave's token in the row phases
  const bool twv = tw < T;
  const long wrow = (long)(twv ? tw : 0) * D;

  // ---- every global load up front: the weight fragments of both contractions, then the
  // pre-activation, the norm backward's rows and its parameters.  None of the row loads
  // is conditional (a row past T reads row 0, an operand the norm does not have reads
  // gin instead), so no load waits for the one before it and the compiler's wait counts
  // stay exact; the values are unpacked only once everything is in flight.
  const int ug = wave % 4, ks = wave / 4;
  constexpr int NSTEP = SLICE / 32;
  static_assert(FB <= 4, "d <= 1024: every weight fragment fits the registers (wider widths split the work)");
  const bool has_ad = a.wup != nullptr;  // else: the norm backward only
  const int f0 = wave * 16 * FB;
  // at d = 1024 the W_down fragments would not fit the registers beside the rows (the
  // kernel spilled): there they are loaded after the norm backward, during the dV phase
  constexpr bool EARLY_WDN = FB <= 3;
  bf16x8 wup_f[NSTEP], w0[FB], w1[FB];
  auto load_wdn = [&] {
#pragma unroll
    for (int b = 0; b < FB; ++b) {
      w0[b] = ld_frag(pack_b_frag(a.wdn, D, wave, b, 0, lane));
      w1[b] = ld_frag(pack_b_frag(a.wdn, D, wave, b, 1, lane));
    }
  };
  if (has_ad) {
#pragma unroll
    for (int j = 0; j < NSTEP; ++j) wup_f[j] = ld_frag(pack_a_frag(a.wup, D, wave, j, lane));
    if constexpr (EARLY_WDN)
      if (a.dzin) load_wdn();
  }
  const bf16* gin = static_cast<const bf16*>(a.gin);
  // pre-activation of unit `lane` of this wave's token (read in the dU phase)
  const bf16 uraw = (has_ad ? static_cast<const bf16*>(a.u) : gin)[(long)(twv ? tw : 0) * MB + lane];
  const bf16* xp = a.norm != Norm::None ? static_cast<const bf16*>(a.xhat) : gin;
  const bf16* dp = a.norm == Norm::RMS ? static_cast<const bf16*>(a.dres) : gin;
  const bf16* gp = a.norm != Norm::None ? static_cast<const bf16*>(a.gamma) : gin;
  const float* rp = a.norm != Norm::None ? a.rstd : reinterpret_cast<const float*>(gin);
  uint2 rg[FB], rx[FB], rd[FB], rm[FB];
#pragma unroll
  for (int j = 0; j < FB; ++j) {
    const int f = 4 * lane + 256 * j;
    rg[j] = *reinterpret_cast<const uint2*>(gin + wrow + f);
    rx[j] = *reinterpret_cast<const uint2*>(xp + wrow + f);
    rd[j] = *reinterpret_cast<const uint2*>(dp + wrow + f);
    rm[j] = *reinterpret_cast<const uint2*>(gp + f);
  }
  const float rsv = rp[twv ? tw : 0];

  // ---- gradient at the adapter output, one wave per token (features 4 lane + 256 j)
  auto unpack = [](uint2 q, float v[4]) {
    v[0] = __uint_as_float(q.x << 16); v[1] = __uint_as_float(q.x & 0xffff0000u);
    v[2] = __uint_as_float(q.y << 16); v[3] = __uint_as_float(q.y & 0xffff0000u);
  };
  float dz[FB][4];
  {
    float gg[FB][4], xh[FB][4], dr[FB][4], gm[FB][4];
#pragma unroll
    for (int j = 0; j < FB; ++j) {
      unpack(rg[j], gg[j]);
      unpack(rx[j], xh[j]);
      unpack(rd[j], dr[j]);
      unpack(rm[j], gm[j]);
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (!twv || a.norm != Norm::RMS) dr[j][q] = 0.f;
    }
    // one formula for every norm (no branch the compiler could sink the loads into);
    // without a norm dz is gin itself
    const bool none = a.norm == Norm::None;
    const float rs = (twv && !none) ? rsv : 0.f;
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int j = 0; j < FB; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float g = gg[j][q] * gm[j][q];
        s1 += g;
        s2 += g * xh[j][q];
      }
    constexpr float inv_d = 1.f / (float)D;
    const float m1 = (a.norm == Norm::LN) ? wave_sum(s1) * inv_d : 0.f;
    const float m2 = wave_sum(s2) * inv_d;
#pragma unroll
    for (int j = 0; j < FB; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float v = dr[j][q] + rs * (gg[j][q] * gm[j][q] - m1 - xh[j][q] * m2);
        dz[j][q] = none ? (twv ? gg[j][q] : 0.f) : v;
      }
  }
#pragma unroll
  for (int j = 0; j < FB; ++j) {
    const int f = 4 * lane + 256 * j;
    if (twv && a.dz) St<bf16>::st4s(static_cast<bf16*>(a.dz), wrow + f, dz[j], nt);
    St<bf16>::st4(sdZ, (long)wave * DP + f, dz[j]);
  }
  if (!has_ad) return;
  if constexpr (!EARLY_WDN)
    if (a.dzin) load_wdn();
  __syncthreads();

  // ---- dV^T[unit][token] = W_up[unit][:] . dZ[token][:], k split over KS waves; the
  // slices' partial sums go through LDS unit-major (token stride 17 floats, so the
  // MFMA writes and the one-unit-per-lane reads spread over the banks); then
  // dU = dV * gelu'(U) with one (token, unit) pair per thread
  {
    const bf16* zr = sdZ + l16 * DP + ks * SLICE + 8 * grp;
    f32x4 dv = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < NSTEP; ++j) dv = mfma16(wup_f[j], ld_frag(zr + j * 32), dv);
#pragma unroll
    for (int r = 0; r < 4; ++r) sPart[(ks * MB + ug * 16 + 4 * grp + r) * TOKP + l16] = dv[r];
    __syncthreads();
    const int unit = lane;
    float sum = 0.f;
#pragma unroll
    for (int k2 = 0; k2 < KS; ++k2) sum += sPart[(k2 * MB + unit) * TOKP + wave];
    // gelu'(U) for dU and, when asked for, gelu(U) for the weight gradient of
    // W_up, from one erf evaluation (the same bits as gelu_fast / gelu_grad_fast)
    const float uf = bf2f(uraw);
    const ErfGauss eg = erf_gauss_as(uf);
    const float phi2 = 1.f + eg.erf_z;
    const bf16 du = f2bf(sum * fmaf(uf * 0.39894228040143268f, eg.gauss, 0.5f * phi2));
    if (twv) St<bf16>::st_nt(static_cast<bf16*>(a.du), (long)tw * MB + unit, bf2f(du));
    if (a.gu && twv) St<bf16>::st_nt(static_cast<bf16*>(a.gu), (long)tw * MB + unit, 0.5f * uf * phi2);
    sdU[wave * GP + unit] = du;
  }
  if (!a.dzin) return;
  __syncthreads();

  // ---- (dU W_down^T)^T[f][token] -> sV (fp32), then dzin = dz + sV, one wave per token
  {
    const bf16x8 u0 = ld_frag(sdU + l16 * GP + 8 * grp), u1 = ld_frag(sdU + l16 * GP + 32 + 8 * grp);
#pragma unroll
    for (int b = 0; b < FB; ++b) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      acc = mfma16(w0[b], u0, acc);
      acc = mfma16(w1[b], u1, acc);
      *reinterpret_cast<float4*>(sV + l16 * VP + f0 + b * 16 + 4 * grp) = make_float4(acc[0], acc[1], acc[2], acc[3]);
    }
  }
  __syncthreads();
  if (!twv) return;
#pragma unroll
  for (int j = 0; j < FB; ++j) {
    const int f = 4 * lane + 256 * j;
    const float4 v = *reinterpret_cast<const float4*>(sV + wave * VP + f);
    const float o[4] = {dz[j][0] + v.x, dz[j][1] + v.y, dz[j][2] + v.z, dz[j][3] + v.w};
    St<bf16>::st4s(static_cast<bf16*>(a.dzin), wrow + f, o, nt);
  }
}

// ================================================================ bf16 weight gradients
// C[p][q] += sum_t X[t][p] * Y[t][q]: output kind 0 -> dW_up (X = gelu(U), Y = dZ),
// 1 -> dW_down (X = z, Y = dU).  64x64 output tiles, DW_TC tokens per
// workgroup.  Token-major tiles go to LDS as they are in memory (16-B chunks);
// the MFMA operands, which need 8 consecutive tokens per lane, are read with
// the LDS transpose read.
// One launch covers up to DW_BATCH adapters: output kind index 2 * adapter + (0
// up, 1 down).  512-token chunks: with a whole backward's adapters in one
// launch there are workgroups enough (1024 would hold every chunk's loads in
// 256 registers).  Each workgroup stores its chunk's 64x64 partial sum with
// plain stores into part ([kind][chunk][m d], the element order of the
// gradient itself); adapter_dw_reduce then adds the chunks, in chunk order,
// into the gradient.  So the result does not depend on the order in which
// workgroups finish: the same inputs give the same bits, whatever else the
// launch carries.
constexpr int DW_TC = 512, DW_BATCH = 16;
struct AdapterDwBatch {
  AdapterDwArgs a[DW_BATCH];
  int gx, gy;  // 64-column tiles of d and token chunks, per output kind
  float* part;
};
__global__ __launch_bounds__(256) void adapter_dw_bf16(AdapterDwBatch batch) {
  __shared__ __attribute__((aligned(16))) bf16 sX[64 * GP];  // [token][p]
  __shared__ __attribute__((aligned(16))) bf16 sY[64 * GP];  // [token][q]
  // One-dimensional grid of gx * gy * gz workgroups.  The gx column tiles of one (token
  // chunk, output kind) pair read the same small operand chunk (U or dU, 64 KB); up to
  // d = 1024 they are placed on one XCD (workgroup i runs on XCD i % 8), consecutively,
  // so that chunk is fetched into that XCD's L2 once instead of into every XCD's.  Wider
  // (gx > 16) keeps them spread: one XCD streaming a chunk's whole big operand (64 KB per
  // tile) through its L2 was slower (d = 4096: 50 -> 58 us).
  const int gx = batch.gx, gy = batch.gy, npair = gridDim.x / gx;
  int pair, tile;
  if (npair % 8 == 0 && gx <= 16) {
    const int slot = blockIdx.x / 8;
    pair = (blockIdx.x % 8) * (npair / 8) + slot / gx;
    tile = slot % gx;
  } else {
    pair = blockIdx.x / gx;
    tile = blockIdx.x % gx;
  }
  const int bx = tile, by = pair % gy, bz = pair / gy;
  const AdapterDwArgs& a = batch.a[bz >> 1];
  const bool up = (bz & 1) == 0;
  const int d = a.d, T = a.T;
  // dW_up's operand is gelu(U): read as the adapter backward formed it, or
  // formed here from U by every column tile of the chunk
  const bool form_gelu = up && !a.gu;
  const bf16* X = static_cast<const bf16*>(up ? (a.gu ? a.gu : a.u) : a.z);
  const bf16* Y = static_cast<const bf16*>(up ? a.dz : a.du);
  const int ldx = up ? MB : d, ldy = up ? d : MB;
  const int ldc = up ? d : MB;
  const int p0 = up ? 0 : bx * 64, q0 = up ? bx * 64 : 0;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, l32 = lane & 31, half = lane >> 5;
  const int wp = wave / 2, wq = wave % 2;
  f32x16 acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.f;
  const int tbeg = by * DW_TC, tend = min(T, tbeg + DW_TC);
  constexpr int NSUB = DW_TC / 64;
  // every 16-B chunk of the chunk's X and Y rows, loaded before the first use
  bf16x8 xr[NSUB][2], yr[NSUB][2];
#pragma unroll
  for (int sb = 0; sb < NSUB; ++sb)
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int idx = tid + i * 256, tt = idx / 8, c = idx % 8, t = tbeg + sb * 64 + tt;
      xr[sb][i] = t < tend ? ld_frag(X + (long)t * ldx + p0 + c * 8) : zero_frag();
      yr[sb][i] = t < tend ? ld_frag(Y + (long)t * ldy + q0 + c * 8) : zero_frag();
    }
#pragma unroll
  for (int sb = 0; sb < NSUB; ++sb) {
    if (tbeg + sb * 64 >= tend) break;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int idx = tid + i * 256, tt = idx / 8, c = idx % 8;
      bf16x8 xv = xr[sb][i];
      if (form_gelu) {
        float f[8];
        unpack_frag(xv, f);
#pragma unroll
        for (int v = 0; v < 8; ++v) f[v] = gelu_fast(f[v]);
        xv = pack_frag(f);
      }
      *reinterpret_cast<bf16x8*>(sX + tt * GP + c * 8) = xv;
      *reinterpret_cast<bf16x8*>(sY + tt * GP + c * 8) = yr[sb][i];
    }
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
      acc = mfma32(lds_tr_frag32(sX, GP, ks * 16, wp * 32, lane), lds_tr_frag32(sY, GP, ks * 16, wq * 32, lane),
                   acc);
  }
  // D[i = p][j = q]: lane holds q = wq*32 + l32, p = wp*32 + 8*(r/4) + 4*half + r%4
  float* P = batch.part + ((long)bz * gy + by) * ((long)MB * d);
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int p = p0 + wp * 32 + 8 * (r >> 2) + 4 * half + (r & 3), q = q0 + wq * 32 + l32;
    P[(long)p * ldc + q] = acc[r];
  }
}

// C += sum over the chunks c = 0, 1, .. of part[kind][c] (in that order), four
// consecutive elements per thread, for every output kind of the batch
__global__ __launch_bounds__(256) void adapter_dw_reduce(AdapterDwBatch batch, int nkind) {
  const long md = (long)MB * batch.a[0].d, per = md / 4;
  const long i = (long)blockIdx.x * 256 + threadIdx.x;
  if (i >= nkind * per) return;
  const int bz = (int)(i / per);
  const long e = (i % per) * 4;
  const AdapterDwArgs& a = batch.a[bz >> 1];
  float* C = ((bz & 1) == 0 ? a.g_up : a.g_down) + e;
  const float* src = batch.part + (long)bz * batch.gy * md + e;
  float4 s = *reinterpret_cast<const float4*>(src);
  for (int c = 1; c < batch.gy; ++c) {
    const float4 v = *reinterpret_cast<const float4*>(src + c * md);
    s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
  }
  float4 g = *reinterpret_cast<const float4*>(C);
  g.x += s.x; g.y += s.y; g.z += s.z; g.w += s.w;
  *reinterpret_cast<float4*>(C) = g;
}

// ================================================================ bf16, d > 1024
// A 16-token workgroup holding the whole adapter would read all 2 x d x 64
// weights (1 MB at d = 4096) for 16 tokens and leave half the GPU idle at
// these token counts.  Wide widths split the work instead, in both directions:
//   down:  P[kc][t][j] = sum over the features f of chunk kc (WIDE_KC features)
//          of X[t][f] W[j][f], W in the A fragment layout (W_down^T forward,
//          W_up backward); grid (T/16) x (d/WIDE_KC), no atomics;
//   up:    S = sum_kc P (fp32), G = gelu(S) forward (S stashed as u) or
//          G = S * gelu'(u) backward (G written as du); then, per chunk of
//          WIDE_UC features, out = Z [+ R] + G W^T, W in the B fragment layout
//          (W_up^T forward, W_down backward); grid (T/16) x (d/WIDE_UC);
//   norm:  the vectorised row kernels for LayerNorm / RMSNorm forward or
//          backward (launch_norm_rows_fwd / _bwd).
// Both MFMA kernels use 16x16x32 with the weight as the A operand, as the row
// kernels do, and read every operand fragment straight from global memory
// (one contiguous 1-KB run per packed weight fragment).
constexpr int WIDE_KC = 1024, WIDE_UC = 512;

// packed-layout fragment of (unit group ug, 32-feature block fb) in layout A
__device__ __forceinline__ const bf16* pack_a_block(const bf16* base, int d, int ug, int fb, int lane) {
  const int per = d / 128;  // 32-feature blocks per quarter of the features
  return base + ((long)((4 * (fb / per) + ug) * per + fb % per) * 64 + lane) * 8;
}

__global__ __launch_bounds__(256) void adapter_wide_down(const bf16* X, const bf16* Wa, int T, int d, float* P) {
  __shared__ float red[4][MB][TOK + 1];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, l16 = lane & 15, grp = lane >> 4;
  const int t0 = blockIdx.x * TOK, kc = blockIdx.y;
  const int token = t0 + l16;
  const bool tv = token < T;
  constexpr int NB = WIDE_KC / 4 / 32;  // 32-feature blocks per wave
  const int fb0 = (kc * WIDE_KC + wave * (WIDE_KC / 4)) / 32;
  // every load issued before the first MFMA, none conditional (a token past T reads row 0;
  // its column of the result is never stored)
  const bf16* xr = X + (long)(tv ? token : 0) * d + fb0 * 32 + 8 * grp;
  bf16x8 xf[NB], w[NB][4];
#pragma unroll
  for (int j = 0; j < NB; ++j) xf[j] = ld_frag(xr + j * 32);
#pragma unroll
  for (int j = 0; j < NB; ++j)
#pragma unroll
    for (int g = 0; g < 4; ++g) w[j][g] = ld_frag(pack_a_block(Wa, d, g, fb0 + j, lane));
  __builtin_amdgcn_sched_barrier(0);  // keeps the scheduler from moving loads down to their MFMAs
  f32x4 acc[4];
#pragma unroll
  for (int g = 0; g < 4; ++g) acc[g] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int j = 0; j < NB; ++j)
#pragma unroll
    for (int g = 0; g < 4; ++g) acc[g] = mfma16(w[j][g], xf[j], acc[g]);
  // D[unit 16g + 4*grp + r][token l16]; the four waves' feature quarters summed in LDS
#pragma unroll
  for (int g = 0; g < 4; ++g)
#pragma unroll
    for (int r = 0; r < 4; ++r) red[wave][16 * g + 4 * grp + r][l16] = acc[g][r];
  __syncthreads();
  for (int i = threadIdx.x; i < TOK * MB; i += 256) {
    const int tok = i / MB, j = i % MB;
    if (t0 + tok < T)
      St<float>::st_nt(P, ((long)kc * T + t0 + tok) * MB + j,
                       (red[0][j][tok] + red[1][j][tok]) + (red[2][j][tok] + red[3][j][tok]));
  }
}

// BWD = false: G = gelu(S), S stashed in `uo` (may be null); BWD = true:
// G = S * gelu'(ui), written to `uo`.  With Wb null only G is produced (the
// backward at the cut-off, where no input gradient is wanted); then the grid
// has one feature chunk.
template <bool BWD>
__global__ __launch_bounds__(256) void adapter_wide_up(const float* P, int nkc, const bf16* ui, bf16* uo, int T,
                                                       int d, const bf16* Wb, const bf16* Z, const bf16* R,
                                                       bf16* out) {
  constexpr int OP = WIDE_UC + 4;  // fp32 pitch of the staged result rows
  __shared__ __attribute__((aligned(16))) bf16 sG[TOK * GP];
  __shared__ __attribute__((aligned(16))) float sO[TOK * OP];  // G W^T of the chunk, [token][feature]
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, l16 = lane & 15, grp = lane >> 4;
  const int t0 = blockIdx.x * TOK, fc = blockIdx.y;
  // Every load is issued before the first use: the split-K partial sums (four chunks per
  // batch, chunk and token clamped, masked after the load), the pre-activation, then the
  // weight fragments and the Z / R rows of the up projection.  None is conditional on a
  // lane, so no load waits for the one before it.
  constexpr int NIT = TOK * MB / 256, KB = 4;
  float part[NIT][KB];
  bf16 uiv[NIT];
#pragma unroll
  for (int it = 0; it < NIT; ++it) {
    const int i = threadIdx.x + it * 256, tok = i / MB, j = i % MB, t = min(t0 + tok, T - 1);
#pragma unroll
    for (int q = 0; q < KB; ++q) part[it][q] = P[((long)min(q, nkc - 1) * T + t) * MB + j];
    uiv[it] = BWD ? ui[(long)t * MB + j] : f2bf(0.f);
  }
  constexpr int NBK = WIDE_UC / 16 / 4;  // 16-feature blocks per wave
  const int b0 = (fc * WIDE_UC + wave * (WIDE_UC / 4)) / 16;
  // the Z / R rows of the chunk as contiguous 16-B pieces (token c / CPT, features
  // 8 (c % CPT) ..), the layout the output is stored in, rather than the MFMA layout
  constexpr int CPT = WIDE_UC / 8, NCK = TOK * CPT / 256;
  bf16x8 w[NBK][2], zr[NCK], rr[NCK];
  if (Wb) {
#pragma unroll
    for (int b = 0; b < NBK; ++b) {
      w[b][0] = ld_frag(Wb + ((long)(2 * (b0 + b)) * 64 + lane) * 8);
      w[b][1] = ld_frag(Wb + ((long)(2 * (b0 + b) + 1) * 64 + lane) * 8);
    }
    const bf16* Rp = R ? R : Z;
#pragma unroll
    for (int i = 0; i < NCK; ++i) {
      const int c = threadIdx.x + 256 * i, t = min(t0 + c / CPT, T - 1);
      const long off = (long)t * d + fc * WIDE_UC + 8 * (c % CPT);
      zr[i] = ld_frag(Z + off);
      rr[i] = ld_frag(Rp + off);
    }
  }
#pragma unroll
  for (int it = 0; it < NIT; ++it) {
    const int i = threadIdx.x + it * 256, tok = i / MB, j = i % MB, t = t0 + tok;
    float sum = 0.f, g = 0.f;
#pragma unroll
    for (int q = 0; q < KB; ++q) sum += q < nkc ? part[it][q] : 0.f;
    for (int kc = KB; kc < nkc; ++kc) sum += P[((long)kc * T + min(t, T - 1)) * MB + j];  // d > 4096 only
    if (t < T) {
      if constexpr (BWD) {
        g = sum * gelu_grad_fast(bf2f(uiv[it]));
        if (fc == 0) St<bf16>::st_nt(uo, (long)t * MB + j, g);
      } else {
        g = gelu_fast(sum);
        if (fc == 0 && uo) St<bf16>::st_nt(uo, (long)t * MB + j, sum);
      }
    }
    sG[tok * GP + j] = f2bf(g);
  }
  if (!Wb) return;
  __syncthreads();
  const bf16x8 g0 = ld_frag(sG + l16 * GP + 8 * grp), g1 = ld_frag(sG + l16 * GP + 32 + 8 * grp);
#pragma unroll
  for (int b = 0; b < NBK; ++b) {  // lane: token l16, features 4 grp .. + 3 of block b
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    acc = mfma16(w[b][0], g0, acc);
    acc = mfma16(w[b][1], g1, acc);
    *reinterpret_cast<float4*>(sO + l16 * OP + wave * (WIDE_UC / 4) + b * 16 + 4 * grp) =
        make_float4(acc[0], acc[1], acc[2], acc[3]);
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < NCK; ++i) {
    const int c = threadIdx.x + 256 * i, tok = c / CPT, f8 = 8 * (c % CPT);
    if (t0 + tok >= T) continue;
    float o[8], zf[8], rf[8];
    const float4 lo = *reinterpret_cast<const float4*>(sO + tok * OP + f8);
    const float4 hi = *reinterpret_cast<const float4*>(sO + tok * OP + f8 + 4);
    unpack_frag(zr[i], zf);
    unpack_frag(rr[i], rf);
    const float v[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
#pragma unroll
    for (int q = 0; q < 8; ++q) o[q] = v[q] + zf[q] + (R ? rf[q] : 0.f);
    st16(out + (long)(t0 + tok) * d + fc * WIDE_UC + f8, pack_frag(o), stream_out((long)T * d * 2));
  }
}

// ================================================================ fp32 (small stages): one workgroup per token
__device__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  float t = 0.f;
  for (int w = 0; w < nw; ++w) t += red[w];
  return t;
}

__global__ __launch_bounds__(256) void adapter_fwd_f32(AdapterFwdArgs a) {
  extern __shared__ float sh[];
  const int d = a.d, m = a.m, t = blockIdx.x;
  float* sz = sh;        // [d]
  float* sg = sz + d;    // [m]
  float* sv = sg + m;    // [d]
  float* red = sv + d;   // [8]
  const float* z = static_cast<const float*>(a.z) + (long)t * d;
  const float* res = static_cast<const float*>(a.res) + (long)t * d;
  const float* wdt = static_cast<const float*>(a.wdn_t);
  const float* wut = static_cast<const float*>(a.wup_t);
  const bool has_ad = wdt != nullptr;  // else: residual add + norm only
  for (int i = threadIdx.x; i < d; i += blockDim.x) sz[i] = z[i];
  __syncthreads();
  if (has_ad)
    for (int j = threadIdx.x; j < m; j += blockDim.x) {
      float u = 0.f;
      for (int k = 0; k < d; ++k) u += sz[k] * wdt[(long)j * d + k];
      if (a.u) static_cast<float*>(a.u)[(long)t * m + j] = u;
      sg[j] = gelu_f(u);
    }
  __syncthreads();
  float s1 = 0.f;
  for (int f = threadIdx.x; f < d; f += blockDim.x) {
    float v = res[f] + sz[f];
    if (has_ad)
      for (int j = 0; j < m; ++j) v += sg[j] * wut[(long)f * m + j];
    sv[f] = v;
    s1 += v;
  }
  float* out = static_cast<float*>(a.out) + (long)t * d;
  if (a.norm == Norm::None) {
    for (int f = threadIdx.x; f < d; f += blockDim.x) out[f] = sv[f];
    return;
  }
  float mean = 0.f;
  if (a.norm == Norm::LN) mean = block_sum(s1, red) / d;
  else
    for (int f = threadIdx.x; f < d; f += blockDim.x) out[f] = sv[f];
  float s2 = 0.f;
  for (int f = threadIdx.x; f < d; f += blockDim.x) s2 += (sv[f] - mean) * (sv[f] - mean);
  const float rstd = rsqrtf(block_sum(s2, red) / d + a.eps);
  if (a.rstd && threadIdx.x == 0) a.rstd[t] = rstd;
  float* o = (a.norm == Norm::LN) ? out : static_cast<float*>(a.out_norm) + (long)t * d;
  const float* gm = static_cast<const float*>(a.gamma);
  const float* bt = static_cast<const float*>(a.beta);
  for (int f = threadIdx.x; f < d; f += blockDim.x) {
    const float xh = (sv[f] - mean) * rstd;
    o[f] = xh * gm[f] + (a.norm == Norm::LN ? bt[f] : 0.f);
    if (a.xhat) static_cast<float*>(a.xhat)[(long)t * d + f] = xh;
  }
}

__global__ __launch_bounds__(256) void adapter_bwd_f32(AdapterBwdArgs a) {
  extern __shared__ float sh[];
  const int d = a.d, m = a.m, t = blockIdx.x;
  float* sdz = sh;       // [d]
  float* sdu = sdz + d;  // [m]
  float* red = sdu + m;  // [8]
  const float* gin = static_cast<const float*>(a.gin) + (long)t * d;
  const float* xh = static_cast<const float*>(a.xhat) + (long)t * d;
  const float* gm = static_cast<const float*>(a.gamma);
  if (a.norm == Norm::None) {
    for (int f = threadIdx.x; f < d; f += blockDim.x) sdz[f] = gin[f];
  } else {
    float s1 = 0.f, s2 = 0.f;
    for (int f = threadIdx.x; f < d; f += blockDim.x) {
      const float g = gin[f] * gm[f];
      s1 += g;
      s2 += g * xh[f];
    }
    const float m1 = (a.norm == Norm::LN) ? block_sum(s1, red) / d : 0.f;
    const float m2 = block_sum(s2, red) / d;
    const float rs = a.rstd[t];
    const float* dres = static_cast<const float*>(a.dres);
    for (int f = threadIdx.x; f < d; f += blockDim.x) {
      const float g = gin[f] * gm[f];
      sdz[f] = (a.norm == Norm::RMS ? dres[(long)t * d + f] : 0.f) + rs * (g - m1 - xh[f] * m2);
    }
  }
  __syncthreads();
  if (a.dz) {
    float* dzo = static_cast<float*>(a.dz) + (long)t * d;
    for (int f = threadIdx.x; f < d; f += blockDim.x) dzo[f] = sdz[f];
  }
  if (!a.wup) return;  // no adapter: the norm backward (dz) is the whole result
  const float* wu = static_cast<const float*>(a.wup);
  const float* wd = static_cast<const float*>(a.wdn);
  const float* u = static_cast<const float*>(a.u) + (long)t * m;
  for (int j = threadIdx.x; j < m; j += blockDim.x) {
    float dv = 0.f;
    for (int f = 0; f < d; ++f) dv += sdz[f] * wu[(long)j * d + f];
    const float du = dv * gelu_grad_f(u[j]);
    sdu[j] = du;
    static_cast<float*>(a.du)[(long)t * m + j] = du;
  }
  if (!a.dzin) return;
  __syncthreads();
  float* dzin = static_cast<float*>(a.dzin) + (long)t * d;
  for (int f = threadIdx.x; f < d; f += blockDim.x) {
    float v = sdz[f];
    for (int j = 0; j < m; ++j) v += sdu[j] * wd[(long)f * m + j];
    dzin[f] = v;
  }
}

// one thread per gradient entry, summing over every token
__global__ __launch_bounds__(256) void adapter_dw_f32(AdapterDwArgs a) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  const long n = (long)a.m * a.d;
  if (i >= 2 * n) return;
  const float* U = static_cast<const float*>(a.u);
  const float* dZ = static_cast<const float*>(a.dz);
  const float* Z = static_cast<const float*>(a.z);
  const float* dU = static_cast<const float*>(a.du);
  float s = 0.f;
  if (i < n) {  // g_up[j][f]
    const int j = (int)(i / a.d), f = (int)(i % a.d);
    for (int t = 0; t < a.T; ++t) s += gelu_f(U[(long)t * a.m + j]) * dZ[(long)t * a.d + f];
    a.g_up[i] += s;
  } else {      // g_down[f][j]
    const long k = i - n;
    const int f = (int)(k / a.m), j = (int)(k % a.m);
    for (int t = 0; t < a.T; ++t) s += Z[(long)t * a.d + f] * dU[(long)t * a.m + j];
    a.g_down[k] += s;
  }
}

// ================================================================ launchers
static bool al16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// bf16 row kernels: (waves, feature blocks per wave) for a model width
static bool bf16_shape(int d, int& nw, int& fb) {
  // 16 waves (4 per SIMD) per 16-token workgroup: d = 256 * fb
  if (d % 256 == 0 && d <= 4096) { nw = 16; fb = d / 256; return true; }
  return false;
}

template <int FB>
static hipError_t fwd_rows_k(const AdapterFwdArgs& a, hipStream_t s) {
  constexpr int D = 256 * FB;
  const size_t sh = (size_t)TOK * (D + 8) * 2 + (size_t)TOK * GP * 2 + (size_t)4 * MB * (TOK + 1) * 4 +
                    (size_t)TOK * (D + 4) * 4 + (size_t)TOK * D * 2 + (size_t)2 * D * 2;
  static bool attr = false;
  if (!attr) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&adapter_fwd_rows<FB>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)sh);
    if (e != hipSuccess) return e;
    attr = true;
  }
  RG_LAUNCH((adapter_fwd_rows<FB>), dim3((a.T + TOK - 1) / TOK), dim3(1024), sh, s, a);
  return hipGetLastError();
}

template <int NW, int FB>
static hipError_t bwd_k(const AdapterBwdArgs& a, hipStream_t s) {
  constexpr int D = 16 * NW * FB;
  const size_t sh = (size_t)TOK * (D + 8) * 2 + (size_t)TOK * GP * 2 + (size_t)(NW / 4) * (TOK + 1) * MB * 4 +
                    (size_t)TOK * (D + 4) * 4;
  static bool attr = false;
  if (!attr) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&adapter_bwd_bf16<NW, FB>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)sh);
    if (e != hipSuccess) return e;
    attr = true;
  }
  RG_LAUNCH((adapter_bwd_bf16<NW, FB>), dim3((a.T + TOK - 1) / TOK), dim3(NW * 64), sh, s, a);
  return hipGetLastError();
}

long adapter_part_elems(int dtype, int T, int d, int m) {
  return (dtype == DT_BF16 && d > 1024) ? (long)(d / WIDE_KC) * T * m : 0;
}

static hipError_t fwd_wide(const AdapterFwdArgs& a, hipStream_t s) {
  if (a.d % WIDE_KC || a.d > 4096 || (a.wdn_t && !a.part)) return hipErrorInvalidValue;
  for (const void* p : std::initializer_list<const void*>{a.z, a.res, a.out, a.out_norm, a.xhat, a.gamma, a.beta})  // 16-B row accesses
    if (p && !al16(p)) return hipErrorInvalidValue;
  const bf16* z = static_cast<const bf16*>(a.z);
  const bf16* res = static_cast<const bf16*>(a.res);
  const int ntok = (a.T + TOK - 1) / TOK, nkc = a.d / WIDE_KC, nuc = a.d / WIDE_UC;
  bf16* out = static_cast<bf16*>(a.out);
  if (a.wdn_t) {
    RG_LAUNCH(adapter_wide_down, dim3(ntok, nkc), dim3(256), 0, s, z, static_cast<const bf16*>(a.wdn_t), a.T,
              a.d, a.part);
    RG_LAUNCH((adapter_wide_up<false>), dim3(ntok, nuc), dim3(256), 0, s, a.part, nkc, nullptr,
              static_cast<bf16*>(a.u), a.T, a.d, static_cast<const bf16*>(a.wup_t), z, res, out);
    if (a.norm != Norm::None)  // the norm of h, now in out
      return launch_norm_rows_fwd(a.T, a.d, a.eps, a.norm, out, nullptr, a.gamma, a.beta, out, a.out_norm, a.xhat,
                                  a.rstd, s);
    return hipGetLastError();
  }
  return launch_norm_rows_fwd(a.T, a.d, a.eps, a.norm, z, res, a.gamma, a.beta, out, a.out_norm, a.xhat, a.rstd, s);
}

static hipError_t bwd_wide(const AdapterBwdArgs& a, hipStream_t s) {
  const bool has_ad = a.wup != nullptr;
  if (a.d % WIDE_KC || a.d > 4096 || (has_ad && !a.part)) return hipErrorInvalidValue;
  for (const void* p : std::initializer_list<const void*>{a.gin, a.dres, a.xhat, a.gamma, a.dz, a.dzin})  // 16-B row accesses
    if (p && !al16(p)) return hipErrorInvalidValue;
  const bf16* dZ = static_cast<const bf16*>(a.gin);
  if (a.norm != Norm::None) {
    const hipError_t e = launch_norm_rows_bwd(a.T, a.d, a.norm, dZ, a.xhat, a.rstd, a.gamma, a.dres, a.dz, s);
    if (e != hipSuccess) return e;
    dZ = static_cast<const bf16*>(a.dz);
  } else if (a.dz && a.dz != a.gin) {  // no norm: the adapter-output gradient is gin itself
    const hipError_t e = hipMemcpyAsync(a.dz, a.gin, (size_t)a.T * a.d * 2, hipMemcpyDeviceToDevice, s);
    if (e != hipSuccess) return e;
  }
  if (!has_ad) return hipGetLastError();
  const int ntok = (a.T + TOK - 1) / TOK, nkc = a.d / WIDE_KC, nuc = a.d / WIDE_UC;
  RG_LAUNCH(adapter_wide_down, dim3(ntok, nkc), dim3(256), 0, s, dZ, static_cast<const bf16*>(a.wup), a.T, a.d,
            a.part);
  RG_LAUNCH((adapter_wide_up<true>), dim3(ntok, a.dzin ? nuc : 1), dim3(256), 0, s, a.part, nkc,
            static_cast<const bf16*>(a.u), static_cast<bf16*>(a.du), a.T, a.d,
            a.dzin ? static_cast<const bf16*>(a.wdn) : nullptr, dZ, nullptr, static_cast<bf16*>(a.dzin));
  return hipGetLastError();
}

hipError_t launch_adapter_fwd(int dtype, const AdapterFwdArgs& a, hipStream_t s) {
  // an absent adapter (both weight pointers NULL) leaves the residual add + norm
  if (a.T < 0 || a.d <= 0 || a.m <= 0 || !a.z || !a.res || !a.out || (!a.wdn_t != !a.wup_t))
    return hipErrorInvalidValue;
  if (!a.wdn_t && a.u) return hipErrorInvalidValue;
  if (a.norm != Norm::None && !a.gamma) return hipErrorInvalidValue;
  if (a.norm == Norm::LN && !a.beta) return hipErrorInvalidValue;
  if (a.norm == Norm::RMS && !a.out_norm) return hipErrorInvalidValue;
  if (a.T == 0) return hipSuccess;
  if (dtype == DT_BF16) {
    int nw, fb;
    if (!bf16_shape(a.d, nw, fb) || a.m != MB || !al16(a.z) || (a.wdn_t && (!al16(a.wdn_t) || !al16(a.wup_t))))
      return hipErrorInvalidValue;
    // the row kernels move 16 B per lane in every row and through the gain and shift
    if (!al16(a.res) || !al16(a.out) || (a.out_norm && !al16(a.out_norm)) || (a.xhat && !al16(a.xhat)) ||
        (a.gamma && !al16(a.gamma)) || (a.beta && !al16(a.beta)))
      return hipErrorInvalidValue;
    switch (fb) {  // d = 256, 512, 768, 1024, 2048, 3072, 4096
      case 1: return fwd_rows_k<1>(a, s);
      case 2: return fwd_rows_k<2>(a, s);
      case 3: return fwd_rows_k<3>(a, s);
      case 4: return fwd_rows_k<4>(a, s);
      default: return fwd_wide(a, s);  // d = 2048, 3072, 4096
    }
    return hipErrorInvalidValue;
  }
  const size_t sh = (2 * (size_t)a.d + a.m + 8) * sizeof(float);
  if (sh > 64 * 1024) return hipErrorInvalidValue;
  RG_LAUNCH(adapter_fwd_f32, dim3(a.T), dim3(256), sh, s, a);
  return hipGetLastError();
}

bool adapter_bwd_forms_gelu(int dtype, int d) {
  int nw, fb;
  return dtype == DT_BF16 && bf16_shape(d, nw, fb) && fb <= 4;  // the one-kernel backward
}

hipError_t launch_adapter_bwd(int dtype, const AdapterBwdArgs& a, hipStream_t s) {
  // an absent adapter (both weight pointers NULL): only the norm backward, into dz
  const bool has_ad = a.wup || a.wdn;
  if (a.T < 0 || a.d <= 0 || a.m <= 0 || !a.gin) return hipErrorInvalidValue;
  if (has_ad && (!a.u || !a.wup || !a.wdn || !a.du)) return hipErrorInvalidValue;
  if (!has_ad && (!a.dz || a.dzin)) return hipErrorInvalidValue;
  if (!a.dz && a.norm != Norm::None) return hipErrorInvalidValue;
  if (a.norm != Norm::None && (!a.xhat || !a.rstd || !a.gamma)) return hipErrorInvalidValue;
  if (a.norm == Norm::RMS && !a.dres) return hipErrorInvalidValue;
  if (a.gu && (!has_ad || !adapter_bwd_forms_gelu(dtype, a.d))) return hipErrorInvalidValue;
  if (a.T == 0) return hipSuccess;
  if (dtype == DT_BF16) {
    int nw, fb;
    if (!bf16_shape(a.d, nw, fb) || a.m != MB || (has_ad && (!al16(a.wup) || !al16(a.wdn))))
      return hipErrorInvalidValue;
    switch (fb) {  // d = 256, 512, 768, 1024, 2048, 3072, 4096
      case 1: return bwd_k<16, 1>(a, s);
      case 2: return bwd_k<16, 2>(a, s);
      case 3: return bwd_k<16, 3>(a, s);
      case 4: return bwd_k<16, 4>(a, s);
      default: return bwd_wide(a, s);  // d = 2048, 3072, 4096
    }
    return hipErrorInvalidValue;
  }
  const size_t sh = ((size_t)a.d + a.m + 8) * sizeof(float);
  if (sh > 64 * 1024) return hipErrorInvalidValue;
  RG_LAUNCH(adapter_bwd_f32, dim3(a.T), dim3(256), sh, s, a);
  return hipGetLastError();
}

long adapter_dw_part_bytes(int dtype, int T, int d, int m, int n_adapters) {
  if (dtype != DT_BF16 || T <= 0 || n_adapters <= 0) return 0;
  const long nb = n_adapters < DW_BATCH ? n_adapters : DW_BATCH;
  return nb * 2 * ((T + DW_TC - 1) / DW_TC) * (long)d * m * 4;
}

hipError_t launch_adapter_dw_batch(int dtype, const AdapterDwArgs* a, int n, float* part, long part_bytes,
                                   hipStream_t s) {
  if (n < 0 || (n > 0 && !a)) return hipErrorInvalidValue;
  for (int k = 0; k < n; ++k) {
    const AdapterDwArgs& x = a[k];
    if (x.T < 0 || !x.u || !x.dz || !x.z || !x.du || !x.g_up || !x.g_down) return hipErrorInvalidValue;
    if (x.gu && dtype != DT_BF16) return hipErrorInvalidValue;  // the fp32 kernel forms gelu(U) itself
  }
  if (n == 0 || a[0].T == 0) return hipSuccess;
  if (dtype != DT_BF16) {
    for (int k = 0; k < n; ++k) {
      const long ne = 2L * a[k].m * a[k].d;
      RG_LAUNCH(adapter_dw_f32, dim3((unsigned)((ne + 255) / 256)), dim3(256), 0, s, a[k]);
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  }
  for (int k = 0; k < n; ++k) {
    const AdapterDwArgs& x = a[k];
    if (x.T != a[0].T || x.d != a[0].d || x.m != a[0].m || x.m != MB || x.d % 64) return hipErrorInvalidValue;
    if (!al16(x.g_up) || !al16(x.g_down) || (x.gu && !al16(x.gu))) return hipErrorInvalidValue;
  }
  if (!part || !al16(part) || part_bytes < adapter_dw_part_bytes(dtype, a[0].T, a[0].d, a[0].m, n))
    return hipErrorInvalidValue;
  for (int k0 = 0; k0 < n; k0 += DW_BATCH) {
    const int nb = n - k0 < DW_BATCH ? n - k0 : DW_BATCH;
    AdapterDwBatch b{};
    for (int k = 0; k < nb; ++k) b.a[k] = a[k0 + k];
    b.gx = a[0].d / 64;
    b.gy = (a[0].T + DW_TC - 1) / DW_TC;
    b.part = part;
    RG_LAUNCH(adapter_dw_bf16, dim3((unsigned)(b.gx * b.gy * 2 * nb)), dim3(256), 0, s, b);
    const long per = (long)MB * a[0].d / 4;
    RG_LAUNCH(adapter_dw_reduce, dim3((unsigned)((2 * nb * per + 255) / 256)), dim3(256), 0, s, b, 2 * nb);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace rg
