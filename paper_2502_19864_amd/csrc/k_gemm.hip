// Projection GEMMs of the stage: forward x @ W (with the library's K-major
// copy of W) and the dX-only backward dY @ W^T of frozen weights, with the
// elementwise work of the block fused into the epilogue.
//
// bf16: MFMA 32x32x16 with large per-wave tiles, operands moved global -> LDS
// by DMA in a multi-stage pipeline, fragment reads overlapped with the MFMAs,
// and an epilogue that stages the output tile through LDS so that every
// global access is a whole-row 16-B vector (gemm_bf16_pipe_body).  It takes
// every shape of a bf16 stage (K a multiple of 64: d a multiple of 256, the
// FFN width of 64; 16-B aligned operands); others are refused.  The MFMA
// computes C^T blocks so that each lane owns four consecutive output columns
// of one row.
// f32: a plain FMA tile kernel (used by the small fp32 stage only).
#include <type_traits>

#include <utility>

#include "attn_core.h"
#include "common.h"
#include "kernels.h"

namespace rg {

// ---------------------------------------------------------------- epilogues
// fp32 epilogue on four consecutive output columns n..n+3 of row m (the fp32
// path is the post-LN block only: store + bias, GELU, residual, GELU')
template <Epi E>
__device__ __forceinline__ void epilogue4_f32(const GemmArgs& a, int m, int n, float v[4]) {
  static_assert(E == Epi::Store || E == Epi::Gelu || E == Epi::Resid || E == Epi::DGelu,
                "post-LN epilogues only");
  const long r = m;
  if constexpr (E == Epi::Store || E == Epi::Gelu) {
    if (a.bias) {
      float b[4];
      St<float>::ld4(static_cast<const float*>(a.bias), n, b);
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] += b[i];
    }
    if constexpr (E == Epi::Gelu) {
      if (a.out2) St<float>::st4(static_cast<float*>(a.out2), r * a.ldo2 + n, v);
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = gelu_f(v[i]);
    }
  } else {
    float x[4];
    St<float>::ld4(static_cast<const float*>(a.aux), r * a.ld_aux + n, x);
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = E == Epi::Resid ? v[i] + x[i] : v[i] * gelu_grad_f(x[i]);
  }
  St<float>::st4(static_cast<float*>(a.out), r * a.ldo + n, v);
}

// eight consecutive bf16 (16-B aligned) <-> float
__device__ __forceinline__ void ld8(const bf16* p, float v[8]) {
  unpack_frag(*reinterpret_cast<const bf16x8*>(p), v);
}
__device__ __forceinline__ void st8(bf16* p, const float v[8], bool nt) {
  st16(p, pack_frag(v), nt);
}

// bf16 epilogue on eight consecutive output columns n..n+7 of row m; the
// caller passes those columns' bias (Store, Gelu) as fp32, from LDS
template <Epi E>
__device__ __forceinline__ void epilogue8(const GemmArgs& a, int m, int n, float v[8], const float* bias8,
                                          const bf16x8* aux8) {
  const long r = m;
  bf16* out = static_cast<bf16*>(a.out);
  if constexpr (E == Epi::Store || E == Epi::Gelu) {
    if (a.bias) {
      const float4 lo = *reinterpret_cast<const float4*>(bias8);
      const float4 hi = *reinterpret_cast<const float4*>(bias8 + 4);
      v[0] += lo.x; v[1] += lo.y; v[2] += lo.z; v[3] += lo.w;
      v[4] += hi.x; v[5] += hi.y; v[6] += hi.z; v[7] += hi.w;
    }
    if constexpr (E == Epi::Gelu) {
      if (a.out2) st8(static_cast<bf16*>(a.out2) + r * a.ldo2 + n, v, a.nt);
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = gelu_logistic(v[i]);
    }
    st8(out + r * a.ldo + n, v, a.nt);
  } else if constexpr (E == Epi::Resid) {
    float x[8];
    unpack_frag(aux8[0], x);
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] += x[i];
    st8(out + r * a.ldo + n, v, a.nt);
  } else if constexpr (E == Epi::DGelu) {
    float x[8];
    unpack_frag(aux8[0], x);
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] *= gelu_grad_fast(x[i]);
    st8(out + r * a.ldo + n, v, a.nt);
  } else if constexpr (E == Epi::DSwiGlu) {
    float g[8], u[8], dg[8], du[8];
    unpack_frag(aux8[0], g);
    unpack_frag(aux8[1], u);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float sg = sigmoid_f(g[i]);
      du[i] = v[i] * g[i] * sg;
      dg[i] = v[i] * u[i] * (sg + g[i] * sg * (1.f - sg));
    }
    st8(out + r * a.ldo + n, dg, a.nt);
    st8(out + r * a.ldo + a.half + n, du, a.nt);
  }
}

// SwiGLU on eight gate/up pairs: feature columns f..f+7
__device__ __forceinline__ void epilogue_swiglu8(const GemmArgs& a, int m, int f, const float g[8],
                                                 const float u[8]) {
  const long r = m;
  float o[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) o[i] = g[i] * sigmoid_f(g[i]) * u[i];
  st8(static_cast<bf16*>(a.out) + r * a.ldo + f, o, a.nt);
  if (a.out2) {
    st8(static_cast<bf16*>(a.out2) + r * a.ldo2 + f, g, a.nt);
    st8(static_cast<bf16*>(a.out2) + r * a.ldo2 + a.half + f, u, a.nt);
  }
}

// ---------------------------------------------------------------- bf16 MFMA kernel, LDS-DMA pipeline
// Operand tiles go global -> LDS directly (global_load_lds_dwordx4, no VGPR
// staging), NS stages deep, so NS-1 k-tiles are in flight while one is
// multiplied.  LDS rows are 64 bf16 (128 B); the 16-B chunk c of row r sits at
// position c ^ ((r >> 1) & 7), so the 16 rows that one 16-lane group of a
// fragment read touches land in 16 distinct 16-B bank slots.
// Requires K % 64 == 0; rows past M or N are clamped (their results are never
// stored).
// Tile order.  Workgroups are dealt round-robin to the 8 XCDs, each with its
// own L2.  Each XCD gets a contiguous range of a grouped raster: bands of GROUP
// block-rows walked column by column, so the tiles resident on one XCD at a
// time share a few A row-blocks and B column-blocks in its L2.
template <int BM, int BN, int GROUP>
__device__ __forceinline__ void tile_coords(int M, int N, int& m0, int& n0) {
  const int ntm = (M + BM - 1) / BM, ntn = (N + BN - 1) / BN, ntiles = ntm * ntn;
  int g = blockIdx.x;
  if (ntiles % 8 == 0) g = (g % 8) * (ntiles / 8) + g / 8;
  const int band = g / (GROUP * ntn), first = band * GROUP;
  const int gsize = min(ntm - first, GROUP), r = g - band * GROUP * ntn;
  m0 = (first + r % gsize) * BM;
  n0 = (r / gsize) * BN;
}

// Scheduling hint for one k-step of the pipelined kernel: alternate one LDS
// fragment read (of the next k-step) with one MFMA (of this one), ND reads in
// all, so the reads drain while the matrix core works instead of bunching up
// in front of it (1-3 % on every tile shape measured).
template <int ND, int... Q>
__device__ __forceinline__ void interleave_ds_mfma(std::integer_sequence<int, Q...>) {
  ([] {
    if constexpr (Q < ND) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                        // MFMA
  }(), ...);
}

template <int N>
__device__ __forceinline__ void wait_vm_lgkm() {  // vmcnt <= N and lgkmcnt == 0
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | (0x7 << 4) | ((N >> 4) << 14));
}

// ---------------------------------------------------------------- bf16 MFMA kernel, pipelined fragments
// Large per-wave tiles (FM x FN blocks of 32x32) so that the LDS bytes read
// per MFMA stay well under the LDS bandwidth, one workgroup of WM x WN waves
// per CU, operand tiles global -> LDS by DMA, NS stages of BK columns each.
// Inside a k-tile the fragments of k-step ks+1 are read while the MFMAs of
// step ks run.  The wait + barrier for the next k-tile sits inside the last
// k-step, just before its fragments are read, and the stage of the finished
// k-tile is refilled right after that barrier; so the MFMA pipe does not
// drain at k-tile boundaries.
// LDS rows are BK bf16; with CPR = BK/8 16-B chunks per row, chunk c of row r
// sits at position c ^ swz(r), swz(r) = (r / (16 / CPR)) % CPR, so any 16
// consecutive rows read at one chunk hit all 64 banks once.
// Requires K % BK == 0; rows past M or N are clamped (their results are never
// stored).
// rows of fp32 output per epilogue pass: BM halved until the pass fits
constexpr int epi_rows(int bm, int row_bytes, int lds_bytes) {
  int r = bm;
  while (r > 32 && r * row_bytes > lds_bytes) r /= 2;
  return r;
}

template <int BM, int BN, int WM, int WN, int BK, int NS, Epi E, int GROUP = 4>
__device__ __forceinline__ void gemm_bf16_pipe_body(const GemmArgs& a) {
  constexpr int NW = WM * WN, NT = 64 * NW;
  constexpr int TM = BM / WM, TN = BN / WN, FM = TM / 32, FN = TN / 32;
  constexpr int ROWB = BK * 2, CPR = BK / 8, RPI = 64 / CPR, SWD = 16 / CPR;
  constexpr int LA = BM / (RPI * NW), LB = BN / (RPI * NW), LPT = LA + LB;
  constexpr int KS = BK / 16;
  constexpr int STAGE = (BM + BN) * ROWB;
  static_assert(LA * RPI * NW == BM && LB * RPI * NW == BN, "DMA rows must tile the block");
  static_assert(FM * 32 * WM == BM && FN * 32 * WN == BN, "wave tiles of 32x32 blocks");
  static_assert(KS % 2 == 0, "even number of k-steps per tile");
  static_assert(NS >= 2 && NS <= 4 && LPT * (NS - 1) < 64, "stages / vmcnt range");
  static_assert(E != Epi::SwiGlu || FN % 2 == 0, "SwiGlu needs gate/up block pairs");
  // output tile staging for the epilogue: fp32 rows of BN + 4 (the 16-B pad
  // spreads the rows one fragment store touches over all banks), RPP rows (a
  // multiple of 32) per pass through the stage buffers; the tile's bias
  // columns (fp32) sit at the end of those buffers, past the staging rows
  constexpr int CPF = BN + 4;
  constexpr bool HAS_BIAS = E == Epi::Store || E == Epi::Gelu || E == Epi::Attn;
  constexpr int BIASB = HAS_BIAS ? BN * 4 : 0;
  constexpr int RPP = epi_rows(BM, CPF * 4, NS * STAGE - BIASB);
  static_assert(RPP >= 32 && BM % RPP == 0 && RPP * CPF * 4 + BIASB <= NS * STAGE,
                "epilogue passes of whole 32-row blocks");
  // the DMA is invisible to the compiler, so one array serves every stage
  __shared__ __attribute__((aligned(1024))) char smem[NS * STAGE];
  auto stage_base = [&](auto S) -> char* { return smem + decltype(S)::value * STAGE; };

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  int m0, n0;
  tile_coords<BM, BN, GROUP>(a.M, a.N, m0, n0);
  const bf16* A = static_cast<const bf16*>(a.A);
  const bf16* B = static_cast<const bf16*>(a.B);
  const int M = a.M, N = a.N, K = a.K;
  // the tile's bias, fetched now (eight columns per thread of the first BN/8)
  // so that the epilogue finds it in LDS instead of waiting on global loads
  bf16x8 bias_raw = {};
  if constexpr (HAS_BIAS)
    if (a.bias && tid < BN / 8 && n0 + tid * 8 < N)
      bias_raw = *reinterpret_cast<const bf16x8*>(static_cast<const bf16*>(a.bias) + n0 + tid * 8);
  // The epilogue's second operand (residual, pre-activation, gate/up) was
  // written long before and sits in HBM; read all at once at the end of every
  // tile it stalls the epilogue.  One dword from each of its 128-B lines,
  // loaded now, streams it into the caches behind the main loop (the values
  // are never used).  Row segments of BN columns touch at most PF_L lines.
  constexpr bool HAS_AUX = E == Epi::Resid || E == Epi::DGelu || E == Epi::DSwiGlu;
  constexpr int PF_L = (BN * 2 + 127) / 128 + 1, PF_SEG = E == Epi::DSwiGlu ? 2 : 1;
  constexpr int PF_N = HAS_AUX ? (BM * PF_L * PF_SEG + NT - 1) / NT : 0;
  uint32_t pf[PF_N > 0 ? PF_N : 1];
  if constexpr (HAS_AUX) {
    const int ncol = min(BN, N - n0);
#pragma unroll
    for (int i = 0; i < PF_N; ++i) {
      const int idx = tid + i * NT;
      if (idx < BM * PF_L * PF_SEG) {
        const int seg = idx / (BM * PF_L), row = (idx / PF_L) % BM, line = idx % PF_L;
        const long off = (long)min(m0 + row, M - 1) * a.ld_aux + n0 + seg * a.half;
        const int byte = min(line * 128, ncol * 2 - 4);
        pf[i] = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(a.aux) + off * 2 + byte);
      }
    }
  }

  // DMA: instruction i of this wave fills rows (i*NW + wave)*RPI .. +RPI-1;
  // lane -> row lane / CPR, LDS position lane % CPR.  Byte offsets from the
  // operand base (the caller keeps operands under 4 GiB).
  const int lrow = lane / CPR, lpos = lane % CPR;
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  uint32_t oa[LA], ob[LB];
#pragma unroll
  for (int i = 0; i < LA; ++i) {
    const int r = (i * NW + wave) * RPI + lrow;
    oa[i] = (uint32_t)(((long)min(m0 + r, M - 1) * a.lda + (lpos ^ ((r / SWD) % CPR)) * 8) * 2);
  }
#pragma unroll
  for (int i = 0; i < LB; ++i) {
    const int r = (i * NW + wave) * RPI + lrow;
    ob[i] = (uint32_t)(((long)min(n0 + r, N - 1) * a.ldb + (lpos ^ ((r / SWD) % CPR)) * 8) * 2);
  }
  auto issue = [&](int kt, char* sb) {
    const char* gA = reinterpret_cast<const char*>(A) + (long)kt * BK * 2;
    const char* gB = reinterpret_cast<const char*>(B) + (long)kt * BK * 2;
    const uint32_t l0 = lds_addr(sb);
#pragma unroll
    for (int i = 0; i < LA; ++i) dma16_m0(gA, oa[i], l0 + (i * NW + wave_u) * RPI * ROWB);
#pragma unroll
    for (int i = 0; i < LB; ++i) dma16_m0(gB, ob[i], l0 + (BM + (i * NW + wave_u) * RPI) * ROWB);
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int nk = K / BK;
  const int l32 = lane & 31, half = lane >> 5, sw = (l32 / SWD) % CPR;
  bf16x8 fa[2][FM], fb[2][FN];
  auto read_frags = [&](const char* base, int ks, int slot) {
    const int off = 16 * ((2 * ks + half) ^ sw);
    const char* sa = base + (wm * TM + l32) * ROWB + off;
    const char* sb = base + (BM + wn * TN + l32) * ROWB + off;
#pragma unroll
    for (int i = 0; i < FM; ++i) fa[slot][i] = *reinterpret_cast<const bf16x8*>(sa + i * 32 * ROWB);
#pragma unroll
    for (int j = 0; j < FN; ++j) fb[slot][j] = *reinterpret_cast<const bf16x8*>(sb + j * 32 * ROWB);
  };
  auto mfmas = [&](int slot) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) acc[i][j] = mfma32(fb[slot][j], fa[slot][i], acc[i][j]);
  };
  // vmcnt <= n * LPT and lgkmcnt == 0, for a run-time n in [0, NS-1]
  auto wait_tiles = [&](int n) {
    if constexpr (NS >= 4) { if (n >= 3) { wait_vm_lgkm<3 * LPT>(); return; } }
    if constexpr (NS >= 3) { if (n >= 2) { wait_vm_lgkm<2 * LPT>(); return; } }
    if (n >= 1) { wait_vm_lgkm<LPT>(); return; }
    wait_vm_lgkm<0>();
  };
  auto barrier = [&] {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };

  // prologue: tiles 0..NS-1 in flight, tile 0 landed, its first fragments read
  issue(0, smem);
  if (1 < nk) issue(1, smem + STAGE);
  if constexpr (NS > 2) if (2 < nk) issue(2, smem + 2 * STAGE);
  if constexpr (NS > 3) if (3 < nk) issue(3, smem + 3 * STAGE);
  wait_tiles(min(NS, nk) - 1);
  barrier();
  read_frags(smem, 0, 0);

  auto step = [&](auto S, int kt) {
    constexpr int s_ = decltype(S)::value;
    constexpr int sn = (s_ + 1) % NS;
    const char* base = stage_base(S);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if (ks + 1 < KS) {
        read_frags(base, ks + 1, (ks + 1) & 1);
      } else if (kt + 1 < nk) {
        // tile kt+1: tiles issued after it are kt+2 .. min(kt+NS-1, nk-1)
        wait_tiles(min(NS - 2, nk - 2 - kt));
        barrier();
        if (kt + NS < nk) issue(kt + NS, stage_base(S));
        read_frags(stage_base(std::integral_constant<int, sn>{}), 0, 0);
      }
      mfmas(ks & 1);
      interleave_ds_mfma<FM + FN>(std::make_integer_sequence<int, FM * FN>{});
    }
  };
  for (int kt = 0; kt < nk; kt += NS) {
    step(std::integral_constant<int, 0>{}, kt);
    if (kt + 1 < nk) step(std::integral_constant<int, 1>{}, kt + 1);
    if constexpr (NS > 2) if (kt + 2 < nk) step(std::integral_constant<int, 2>{}, kt + 2);
    if constexpr (NS > 3) if (kt + 3 < nk) step(std::integral_constant<int, 3>{}, kt + 3);
  }

  // epilogue: the fp32 tile goes through LDS (row-major, pitch CPF, RPP rows
  // per pass) so that global traffic is whole-row 16-B vectors; the fused
  // elementwise work runs on eight-column chunks, on the fp32 sums, with one
  // rounding to bf16 at the store
  wait_vm_lgkm<0>();
  if constexpr (HAS_AUX) {
#pragma unroll
    for (int i = 0; i < PF_N; ++i) asm volatile("" ::"v"(pf[i]));  // keeps the prefetch loads
  }
  barrier();  // every wave is done reading operand tiles
  float* cf = reinterpret_cast<float*>(smem);
  float* cbias = reinterpret_cast<float*>(smem + NS * STAGE - BIASB);
  if constexpr (HAS_BIAS)
    if (a.bias && tid < BN / 8) {
      float f[8];
      unpack_frag(bias_raw, f);
      *reinterpret_cast<float4*>(cbias + tid * 8) = make_float4(f[0], f[1], f[2], f[3]);
      *reinterpret_cast<float4*>(cbias + tid * 8 + 4) = make_float4(f[4], f[5], f[6], f[7]);
    }
  if constexpr (E == Epi::Attn) {
    // The tile is Q_h | K_h | V_h of one 128-token sequence: the sums (+ bias)
    // go to three bf16 [128][64 + 8] LDS tiles (each lane holds four
    // consecutive columns of one row), the projections to global memory when
    // the caller keeps them, then each wave computes attention for 32 of the
    // sequence's queries from those tiles.
    static_assert(BM == KT && BN == 192 && WM == 2 && WN == 2 && NT == 256, "one head of one sequence per tile");
    constexpr int DHA = 64, TPA = DHA + 8, TILE = BM * TPA;
    static_assert(3 * TILE * 2 + BIASB <= NS * STAGE, "Q, K, V tiles and the bias fit the stage buffers");
    bf16* sT = reinterpret_cast<bf16*>(smem);
    // the bias stores of the first BN/8 threads must have completed before any
    // other wave reads them: s_barrier alone does not wait for LDS writes
    wait_vm_lgkm<0>();
    barrier();
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int row = wm * TM + i * 32 + l32, col = wn * TN + j * 32 + 8 * g + 4 * half;
          const float4 bb = a.bias ? *reinterpret_cast<const float4*>(cbias + col) : make_float4(0.f, 0.f, 0.f, 0.f);
          const float v[4] = {acc[i][j][4 * g] + bb.x, acc[i][j][4 * g + 1] + bb.y, acc[i][j][4 * g + 2] + bb.z,
                              acc[i][j][4 * g + 3] + bb.w};
          St<bf16>::st4(sT + (col / DHA) * TILE + row * TPA, col % DHA, v);
        }
    wait_vm_lgkm<0>();
    barrier();
    if (a.out) {
      constexpr int CPRA = BN / 8;
#pragma unroll 4
      for (int idx = tid; idx < BM * CPRA; idx += NT) {
        const int row = idx / CPRA, q = idx % CPRA, part = q / (DHA / 8), c = (q % (DHA / 8)) * 8;
        st16(static_cast<bf16*>(a.out) + (long)(m0 + row) * a.ldo + n0 + part * DHA + c,
             *reinterpret_cast<const bf16x8*>(sT + part * TILE + row * TPA + c), a.nt);
      }
      barrier();  // every wave's Q rows are read here; each wave then reuses its own for O
    }
    const int h = n0 / BN, H = N / BN, seq = m0 / BM;
    bf16* o0 = static_cast<bf16*>(a.out2) + (long)(m0 + wave * 32) * a.ldo2 + h * DHA;
    attn_seq128_wave<DHA>(sT, sT + TILE, sT + 2 * TILE, wave * 32, lane, o0, a.ldo2, a.nt,
                          a.lse + (long)(seq * H + h) * BM);
    return;
  }
  auto ld_tile8 = [&](int row, int col, float v[8]) {
    const float4 lo = *reinterpret_cast<const float4*>(cf + row * CPF + col);
    const float4 hi = *reinterpret_cast<const float4*>(cf + row * CPF + col + 4);
    v[0] = lo.x; v[1] = lo.y; v[2] = lo.z; v[3] = lo.w;
    v[4] = hi.x; v[5] = hi.y; v[6] = hi.z; v[7] = hi.w;
  };
  constexpr int CPRW8 = BN / 8, NCH8 = RPP * CPRW8;
#pragma unroll
  for (int p = 0; p < BM / RPP; ++p) {
    // this pass's second-operand chunks, all loads in flight before the
    // staging so that their latency overlaps it
    bf16x8 ax[HAS_AUX ? NCH8 / NT : 1][PF_SEG];
    if constexpr (HAS_AUX) {
#pragma unroll
      for (int i = 0; i < NCH8 / NT; ++i) {
        const int idx = tid + i * NT;
        const int m = m0 + p * RPP + idx / CPRW8, n = n0 + (idx % CPRW8) * 8;
        if (m < M && n < N) {
          const bf16* x = static_cast<const bf16*>(a.aux) + (long)m * a.ld_aux + n;
#pragma unroll
          for (int sg = 0; sg < PF_SEG; ++sg) ax[i][sg] = *reinterpret_cast<const bf16x8*>(x + sg * a.half);
        }
      }
    }
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      if ((wm * TM + i * 32) / RPP != p) continue;  // wave-uniform
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int row = wm * TM + i * 32 + l32 - p * RPP, col = wn * TN + j * 32 + 8 * g + 4 * half;
          *reinterpret_cast<float4*>(cf + row * CPF + col) =
              make_float4(acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]);
        }
    }
    wait_vm_lgkm<0>();
    barrier();
    if constexpr (E == Epi::SwiGlu) {
      // packed columns [64p, 64p+32) are gates, [64p+32, 64p+64) the matching ups
      constexpr int CPRW = BN / 16, NCH = RPP * CPRW;
      static_assert(NCH % NT == 0, "whole passes");
#pragma unroll 2
      for (int idx = tid; idx < NCH; idx += NT) {
        const int row = idx / CPRW, q = idx % CPRW, c = (q / 4) * 64 + (q % 4) * 8;
        const int m = m0 + p * RPP + row;
        if (m >= M || n0 + c >= N) continue;
        float gv[8], uv[8];
        ld_tile8(row, c, gv);
        ld_tile8(row, c + 32, uv);
        epilogue_swiglu8(a, m, (n0 + c) / 64 * 32 + (c % 64), gv, uv);
      }
    } else if constexpr (E == Epi::Rope) {
      // chunk pairs: 8 columns at head-local offset i < dh/2 and the 8 at
      // i + dh/2; the tile spans whole heads (BN = 128, n0 a multiple of 128)
      static_assert(BN == 128, "rotary epilogue on 128-wide tiles only");
      constexpr int NPAIR = RPP * CPRW8 / 2;
      static_assert(NPAIR % NT == 0, "whole passes");
      const int dh = a.rope_dh, hc = dh / 16;  // pairs of chunks per head
#pragma unroll 2
      for (int idx = tid; idx < NPAIR; idx += NT) {
        const int row = idx / (CPRW8 / 2), pr = idx % (CPRW8 / 2);
        const int c1 = (pr / hc) * dh + (pr % hc) * 8, c2 = c1 + dh / 2;
        const int m = m0 + p * RPP + row, n1 = n0 + c1, n2 = n0 + c2;
        if (m >= M || n2 >= N) continue;
        float v1[8], v2[8];
        ld_tile8(row, c1, v1);
        ld_tile8(row, c2, v2);
        if (n1 < a.rope_cols) {
          const float2* cs = a.rope_tab + (long)(m % a.rope_S) * (dh / 2) + (n1 % dh);
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float2 t = cs[e];
            const float x1 = v1[e], x2 = v2[e];
            v1[e] = x1 * t.x - x2 * t.y;
            v2[e] = x2 * t.x + x1 * t.y;
          }
        }
        bf16* out = static_cast<bf16*>(a.out);
        st8(out + (long)m * a.ldo + n1, v1, a.nt);
        st8(out + (long)m * a.ldo + n2, v2, a.nt);
      }
    } else if constexpr (HAS_AUX) {
      static_assert(NCH8 % NT == 0, "whole passes");
#pragma unroll
      for (int i = 0; i < NCH8 / NT; ++i) {
        const int idx = tid + i * NT;
        const int row = idx / CPRW8, c = (idx % CPRW8) * 8;
        const int m = m0 + p * RPP + row, n = n0 + c;
        if (m >= M || n >= N) continue;
        float v[8];
        ld_tile8(row, c, v);
        epilogue8<E>(a, m, n, v, cbias + c, ax[i]);
      }
    } else {
      static_assert(NCH8 % NT == 0, "whole passes");
#pragma unroll 2
      for (int idx = tid; idx < NCH8; idx += NT) {
        const int row = idx / CPRW8, c = (idx % CPRW8) * 8;
        const int m = m0 + p * RPP + row, n = n0 + c;
        if (m >= M || n >= N) continue;
        float v[8];
        ld_tile8(row, c, v);
        epilogue8<E>(a, m, n, v, cbias + c, nullptr);
      }
    }
    if (p + 1 < BM / RPP) {
      wait_vm_lgkm<0>();
      barrier();  // the next pass overwrites the staging rows
    }
  }
}

// ---------------------------------------------------------------- fp32 FMA kernel
template <Epi E>
__device__ __forceinline__ void gemm_f32_body(const GemmArgs& a) {
  constexpr int TB = 64, KB = 16;
  __shared__ float sA[KB][TB + 4], sB[KB][TB + 4];
  const int tid = threadIdx.x, tx = tid % 16, ty = tid / 16;
  const int m0 = blockIdx.y * TB, n0 = blockIdx.x * TB;
  const float* A = static_cast<const float*>(a.A);
  const float* B = static_cast<const float*>(a.B);
  float acc[4][4] = {};
  for (int k0 = 0; k0 < a.K; k0 += KB) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int idx = tid + i * 256, r = idx / KB, k = idx % KB;
      int gk = k0 + k;
      sA[k][r] = (m0 + r < a.M && gk < a.K) ? A[(long)(m0 + r) * a.lda + gk] : 0.f;
      sB[k][r] = (n0 + r < a.N && gk < a.K) ? B[(long)(n0 + r) * a.ldb + gk] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < KB; ++k) {
      float x[4], y[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) { x[i] = sA[k][ty * 4 + i]; y[i] = sB[k][tx * 4 + i]; }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(x[i], y[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty * 4 + i, n = n0 + tx * 4;
    if (m < a.M && n < a.N) epilogue4_f32<E>(a, m, n, acc[i]);
  }
}

// ---------------------------------------------------------------- named kernels
// Two-stage 4-wave tiles run two workgroups per CU (LDS <= 80 KB), so their
// registers must fit two waves per SIMD; the bound says so to the compiler.
#define RG_GEMM_KERNELS(NAME)                                                        \
  template <int BM, int BN, int WM, int WN, int NS, Epi E>                           \
  __global__ __launch_bounds__(256, NS == 2 ? 2 : 1) void NAME##_pipe(GemmArgs a) {  \
    gemm_bf16_pipe_body<BM, BN, WM, WN, 64, NS, E, 4>(a);                            \
  }                                                                                  \
  template <int BM, int BN, int WM, int WN, int NS, Epi E>                           \
  __global__ __launch_bounds__(512) void NAME##_pipe8(GemmArgs a) {                  \
    gemm_bf16_pipe_body<BM, BN, WM, WN, 64, NS, E, 4>(a);                            \
  }                                                                                  \
  template <Epi E>                                                                   \
  __global__ __launch_bounds__(256) void NAME##_f32(GemmArgs a) {                    \
    gemm_f32_body<E>(a);                                                             \
  }

RG_GEMM_KERNELS(gemm_qkv_fwd)
RG_GEMM_KERNELS(gemm_o_fwd)
RG_GEMM_KERNELS(gemm_ffn_in_fwd)
RG_GEMM_KERNELS(gemm_ffn_out_fwd)
RG_GEMM_KERNELS(gemm_qkv_dx)
RG_GEMM_KERNELS(gemm_o_dx)
RG_GEMM_KERNELS(gemm_ffn_in_dx)
RG_GEMM_KERNELS(gemm_ffn_out_dx)

const char* role_name(Role r) {
  static const char* n[] = {"gemm_qkv_fwd", "gemm_o_fwd", "gemm_ffn_in_fwd", "gemm_ffn_out_fwd",
                            "gemm_qkv_dx",  "gemm_o_dx",  "gemm_ffn_in_dx",  "gemm_ffn_out_dx"};
  return (r >= 0 && r < N_ROLES) ? n[r] : "gemm_?";
}

// epilogues each call site uses (only these are instantiated)
static constexpr bool role_has(Role r, Epi e) {
  switch (r) {
    case R_QKV_FWD: return e == Epi::Store || e == Epi::Attn || e == Epi::Rope;
    case R_O_FWD: case R_FFN_OUT_FWD: case R_O_DX: return e == Epi::Store;
    case R_FFN_IN_FWD: return e == Epi::Gelu || e == Epi::SwiGlu;
    case R_QKV_DX: case R_FFN_IN_DX: return e == Epi::Resid || e == Epi::Store;
    case R_FFN_OUT_DX: return e == Epi::DGelu || e == Epi::DSwiGlu;
    default: return false;
  }
}

// Tile shapes of the pipelined kernel (BK = 64), chosen per GEMM shape by
// measurement on the BERT-base, BERT-large and LLaMA-7B stage shapes:
//  - 128x192 (2x2 waves of 64x96, two stages) for wide outputs with K <= 1024;
//  - 128x96 (4x1 waves of 32x96, three stages) for outputs up to 1024 wide
//    that 96 divides;
//  - for K > 1024, 256x192 (8 waves of 64x96, two stages) or 256x128 (8
//    waves of 64x64, three stages: one workgroup per CU either way, and the
//    third stage hides the HBM latency of weights that no cache holds, 10-17%
//    on the LLaMA-7B shapes) when that still gives every CU a tile;
//  - 128x128 (2x2 waves of 64x64) otherwise: two stages (two workgroups per
//    CU) from two tiles per CU on, three stages below.
// The SwiGLU epilogues take only the 64-wide wave tiles (a gate/up block pair
// per wave): 256x128 or 128x128.
enum Cfg { C_P128x192, C_P128x96, C_P128x128_2, C_P128x128_3, C_P256x192_8W, C_P256x128_8W };

// The (role, epilogue, tile) kernels that launch_gemm can select for a stage,
// the only ones instantiated.  Besides what role_has excludes:
//  - the gated and rotary epilogues take only the 64-wide wave tiles;
//  - the QKV-dX GEMM has K = 3N, so N divisible by 192 (N = d a multiple of
//    256) means K > 1024, past the 128x192 tile's K limit;
//  - the QKV projection's output (N = 3d) is a multiple of 192, so it takes
//    128x192 (K <= 1024) or an 8-wave tile (K > 1024) whenever the tiles
//    would fill two workgroups per CU on 128x128; its 128x128 tiles are the
//    three-stage ones.
static constexpr bool cfg_has(Role R, Epi E, Cfg c) {
  const bool glu = E == Epi::SwiGlu || E == Epi::DSwiGlu || E == Epi::Rope;
  switch (c) {
    case C_P128x192: return !glu && R != R_QKV_DX;
    case C_P128x96: case C_P256x192_8W: return !glu;
    case C_P128x128_2: return !(R == R_QKV_FWD && E == Epi::Store);
    default: return true;
  }
}
// fp32 stages are post-LN only: no gated or rotary epilogue, and the dX
// GEMMs of the QKV and FFN-in projections add the residual
static constexpr bool f32_has(Role R, Epi E) {
  return E == Epi::Store ? (R != R_QKV_DX && R != R_FFN_IN_DX)
                         : (E == Epi::Gelu || E == Epi::Resid || E == Epi::DGelu);
}

template <Role R, Epi E>
static hipError_t launch_role(Cfg cfg, int dtype, const GemmArgs& a, hipStream_t s) {
  if constexpr (!role_has(R, E)) {
    return hipErrorInvalidValue;
  } else {
    const dim3 block(256);
    if constexpr (E == Epi::Attn) {  // bf16, 128x192 tiles only (checked by the caller)
      RG_LAUNCH((gemm_qkv_fwd_pipe<128, 192, 2, 2, 2, Epi::Attn>), dim3((a.N / 192) * (a.M / 128)), block, 0, s, a);
      return hipGetLastError();
    } else {
    if (dtype == DT_F32) {
      if constexpr (!f32_has(R, E)) return hipErrorInvalidValue;
      else {
        dim3 grid((a.N + 63) / 64, (a.M + 63) / 64);
        // one kernel per role, chosen at compile time (only R's kernel is instantiated)
#define RG_F32(ROLE, NAME) if constexpr (R == ROLE) RG_LAUNCH((NAME##_f32<E>), grid, block, 0, s, a); else
        RG_F32(R_QKV_FWD, gemm_qkv_fwd) RG_F32(R_O_FWD, gemm_o_fwd) RG_F32(R_FFN_IN_FWD, gemm_ffn_in_fwd)
        RG_F32(R_FFN_OUT_FWD, gemm_ffn_out_fwd) RG_F32(R_QKV_DX, gemm_qkv_dx) RG_F32(R_O_DX, gemm_o_dx)
        RG_F32(R_FFN_IN_DX, gemm_ffn_in_dx) RG_F32(R_FFN_OUT_DX, gemm_ffn_out_dx)
        return hipErrorInvalidValue;
#undef RG_F32
        return hipGetLastError();
      }
    }
#define RG_TILES(BM, BN) dim3(((a.N + BN - 1) / BN) * ((a.M + BM - 1) / BM))
#define RG_CASE(C, K, BM_, BN_, THREADS)                                                    \
    case C:                                                                                \
      if constexpr (cfg_has(R, E, C)) RG_LAUNCH((K), RG_TILES(BM_, BN_), dim3(THREADS), 0, s, a); \
      else return hipErrorInvalidValue;                                                    \
      break;
#define RG_LAUNCH_CFG(NAME)                                                               \
  switch (cfg) {                                                                          \
    RG_CASE(C_P128x192, (NAME##_pipe<128, 192, 2, 2, 2, E>), 128, 192, 256)               \
    RG_CASE(C_P128x96, (NAME##_pipe<128, 96, 4, 1, 3, E>), 128, 96, 256)                  \
    RG_CASE(C_P128x128_2, (NAME##_pipe<128, 128, 2, 2, 2, E>), 128, 128, 256)             \
    RG_CASE(C_P128x128_3, (NAME##_pipe<128, 128, 2, 2, 3, E>), 128, 128, 256)             \
    RG_CASE(C_P256x192_8W, (NAME##_pipe8<256, 192, 4, 2, 2, E>), 256, 192, 512)           \
    RG_CASE(C_P256x128_8W, (NAME##_pipe8<256, 128, 4, 2, 3, E>), 256, 128, 512)           \
    default: return hipErrorInvalidValue;                                                 \
  }
    // only R's kernels are instantiated
    if constexpr (R == R_QKV_FWD) { RG_LAUNCH_CFG(gemm_qkv_fwd) }
    else if constexpr (R == R_O_FWD) { RG_LAUNCH_CFG(gemm_o_fwd) }
    else if constexpr (R == R_FFN_IN_FWD) { RG_LAUNCH_CFG(gemm_ffn_in_fwd) }
    else if constexpr (R == R_FFN_OUT_FWD) { RG_LAUNCH_CFG(gemm_ffn_out_fwd) }
    else if constexpr (R == R_QKV_DX) { RG_LAUNCH_CFG(gemm_qkv_dx) }
    else if constexpr (R == R_O_DX) { RG_LAUNCH_CFG(gemm_o_dx) }
    else if constexpr (R == R_FFN_IN_DX) { RG_LAUNCH_CFG(gemm_ffn_in_dx) }
    else if constexpr (R == R_FFN_OUT_DX) { RG_LAUNCH_CFG(gemm_ffn_out_dx) }
    else return hipErrorInvalidValue;
#undef RG_LAUNCH_CFG
#undef RG_CASE
#undef RG_TILES
    return hipGetLastError();
    }
  }
}

template <Role R>
static hipError_t launch_epi(Epi e, Cfg cfg, int dtype, const GemmArgs& a, hipStream_t s) {
  switch (e) {
    case Epi::Store: return launch_role<R, Epi::Store>(cfg, dtype, a, s);
    case Epi::Gelu: return launch_role<R, Epi::Gelu>(cfg, dtype, a, s);
    case Epi::Resid: return launch_role<R, Epi::Resid>(cfg, dtype, a, s);
    case Epi::DGelu: return launch_role<R, Epi::DGelu>(cfg, dtype, a, s);
    case Epi::SwiGlu: return launch_role<R, Epi::SwiGlu>(cfg, dtype, a, s);
    case Epi::Attn: return launch_role<R, Epi::Attn>(cfg, dtype, a, s);
    case Epi::Rope: return launch_role<R, Epi::Rope>(cfg, dtype, a, s);
    case Epi::DSwiGlu: return launch_role<R, Epi::DSwiGlu>(cfg, dtype, a, s);
  }
  return hipErrorInvalidValue;
}

static bool al16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
static bool al8(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 7u) == 0; }

hipError_t launch_gemm(int dtype, Role role, Epi epi, const GemmArgs& a_in, hipStream_t s) {
  GemmArgs a = a_in;
  {  // stream the outputs when the largest tensor written is small enough (common.h)
    const long esz = dtype == DT_BF16 ? 2 : 4;
    a.nt = (long)a.M * a.N * esz * (epi == Epi::DSwiGlu ? 2 : 1) <= NT_MAX_BYTES;
  }
  if (epi == Epi::Attn) {
    // bf16 QKV projection, one head (d_head 64) of one 128-token sequence per
    // 128x192 tile; 16-B rows everywhere, 32-bit operand byte offsets
    const bool ok = dtype == DT_BF16 && role == R_QKV_FWD && a.M > 0 && a.M % 128 == 0 && a.N % 192 == 0 &&
                    a.K % 64 == 0 && a.A && a.B && a.out2 && a.lse && a.lda >= a.K && a.ldb >= a.K &&
                    a.lda % 8 == 0 && a.ldb % 8 == 0 && al16(a.A) && al16(a.B) && a.ldo2 % 8 == 0 &&
                    al16(a.out2) && (!a.bias || al16(a.bias)) && (!a.out || (a.ldo % 8 == 0 && al16(a.out))) &&
                    ((double)(a.M - 1) * a.lda + a.K) * 2 < 4294967296.0 &&
                    ((double)(a.N - 1) * a.ldb + a.K) * 2 < 4294967296.0;
    return ok ? launch_epi<R_QKV_FWD>(epi, C_P128x192, dtype, a, s) : hipErrorInvalidValue;
  }
  if (a.M < 0 || a.N <= 0 || a.K <= 0 || !a.A || !a.B || !a.out) return hipErrorInvalidValue;
  // rotary epilogue: bf16 QKV projection without bias, 128-wide tiles holding
  // whole heads of 64 or 128 columns, the pipelined kernel only (below)
  const bool rope = epi == Epi::Rope;
  if (rope && (dtype != DT_BF16 || role != R_QKV_FWD || a.bias || !a.rope_tab || a.rope_S <= 0 ||
               (a.rope_dh != 64 && a.rope_dh != 128) || a.rope_cols % a.rope_dh || a.rope_cols > a.N ||
               a.N % 128))
    return hipErrorInvalidValue;
  if (a.M == 0) return hipSuccess;
  if (a.N % 4 || a.ldo % 4 || a.lda < a.K || a.ldb < a.K) return hipErrorInvalidValue;
  if ((epi == Epi::Resid || epi == Epi::DGelu || epi == Epi::DSwiGlu) && (!a.aux || a.ld_aux % 4))
    return hipErrorInvalidValue;
  if ((epi == Epi::SwiGlu || epi == Epi::DSwiGlu) && (a.half % 4)) return hipErrorInvalidValue;
  if (a.out2 && a.ldo2 % 4) return hipErrorInvalidValue;
  Cfg cfg = C_P128x128_3;  // (the fp32 kernel has one tile shape)
  if (dtype == DT_BF16) {
    // 16-B operand chunks and 8-B epilogue vectors
    if (a.K % 8 || a.lda % 8 || a.ldb % 8 || !al16(a.A) || !al16(a.B) || !al8(a.out))
      return hipErrorInvalidValue;
    if (epi == Epi::SwiGlu && (a.N % 64 || a.half * 2 != a.N)) return hipErrorInvalidValue;
    // pipelined kernel: K in 64-wide tiles, 16-B epilogue vectors, operands
    // addressed with 32-bit byte offsets
    const bool al_epi = a.N % 8 == 0 && a.ldo % 8 == 0 && al16(a.out) && (!a.bias || al16(a.bias)) &&
                        (!a.aux || (al16(a.aux) && a.ld_aux % 8 == 0)) &&
                        (!a.out2 || (al16(a.out2) && a.ldo2 % 8 == 0)) && a.half % 8 == 0;
    const bool small_off = ((double)(a.M - 1) * a.lda + a.K) * 2 < 4294967296.0 &&
                           ((double)(a.N - 1) * a.ldb + a.K) * 2 < 4294967296.0;
    auto tiles = [&](int bm, int bn) { return (long)((a.M + bm - 1) / bm) * ((a.N + bn - 1) / bn); };
    // two stages (two workgroups per CU) once there are two 128x128 tiles per CU
    const Cfg c128 = tiles(128, 128) >= 512 ? C_P128x128_2 : C_P128x128_3;
    // (a bf16 stage always meets these: d a multiple of 256, the FFN width of
    // 64, 16-B aligned buffers, tensors under 2^31 elements)
    if (a.K % 64 || !al_epi || !small_off) return hipErrorInvalidValue;
    // the gated and rotary epilogues take only the 64-wide wave tiles
    const bool glu = epi == Epi::SwiGlu || epi == Epi::DSwiGlu || rope;
    if (!glu && a.N % 192 == 0 && a.K <= 1024 && tiles(128, 192) >= 256) cfg = C_P128x192;
    else if (!glu && a.N % 96 == 0 && a.N <= 1024) cfg = C_P128x96;
    else if (!glu && a.K > 1024 && a.N % 192 == 0 && tiles(256, 192) >= 256) cfg = C_P256x192_8W;
    else if (a.K > 1024 && a.N % 128 == 0 && tiles(256, 128) >= 256) cfg = C_P256x128_8W;
    else cfg = c128;
  } else if (dtype == DT_F32) {
    if (!al16(a.out)) return hipErrorInvalidValue;
  } else {
    return hipErrorInvalidValue;
  }
  auto go = [&](Cfg c, const GemmArgs& g) -> hipError_t {
    switch (role) {
      case R_QKV_FWD: return launch_epi<R_QKV_FWD>(epi, c, dtype, g, s);
      case R_O_FWD: return launch_epi<R_O_FWD>(epi, c, dtype, g, s);
      case R_FFN_IN_FWD: return launch_epi<R_FFN_IN_FWD>(epi, c, dtype, g, s);
      case R_FFN_OUT_FWD: return launch_epi<R_FFN_OUT_FWD>(epi, c, dtype, g, s);
      case R_QKV_DX: return launch_epi<R_QKV_DX>(epi, c, dtype, g, s);
      case R_O_DX: return launch_epi<R_O_DX>(epi, c, dtype, g, s);
      case R_FFN_IN_DX: return launch_epi<R_FFN_IN_DX>(epi, c, dtype, g, s);
      case R_FFN_OUT_DX: return launch_epi<R_FFN_OUT_DX>(epi, c, dtype, g, s);
      default: return hipErrorInvalidValue;
    }
  };
  // The 256x128 kernel runs one workgroup per CU.  When its tiles leave the
  // GPU's last round at most half full (LLaMA-7B FFN-in: 8 x 172 = 1376 tiles,
  // five rounds of 256 and 96), that round is split off along N: the columns
  // of the whole rounds go to this kernel, the rest to 128x128 tiles, which
  // spread it over every CU instead of leaving most of them idle.  Each output
  // column is still computed by one tile, in the same order.
  if (cfg == C_P256x128_8W && !rope) {
    const int rt = (a.M + 255) / 256;
    const long nt = (long)rt * ((a.N + 127) / 128), rem = nt % 256;
    if (256 % rt == 0 && rem != 0 && rem <= 128) {
      const int n_main = (int)(nt / 256) * (256 / rt) * 128;
      if (n_main > 0 && n_main < a.N) {
        GemmArgs m = a, t = a;
        m.N = n_main;
        t.N = a.N - n_main;
        t.B = static_cast<const bf16*>(a.B) + (long)n_main * a.ldb;
        // output columns: SwiGLU writes one column per gate/up pair (the stash
        // keeps the pair at f and half + f); every other epilogue one per column
        const int oc = epi == Epi::SwiGlu ? n_main / 2 : n_main;
        t.out = static_cast<bf16*>(a.out) + oc;
        if (a.out2) t.out2 = static_cast<bf16*>(a.out2) + oc;
        if (a.bias) t.bias = static_cast<const bf16*>(a.bias) + n_main;
        if (a.aux) t.aux = static_cast<const bf16*>(a.aux) + n_main;
        const long tail_tiles = (long)((a.M + 127) / 128) * ((t.N + 127) / 128);
        const Cfg ct = tail_tiles >= 512 ? C_P128x128_2 : C_P128x128_3;
        const hipError_t e = go(cfg, m);
        return e != hipSuccess ? e : go(ct, t);
      }
    }
  }
  return go(cfg, a);
}

}  // namespace rg
