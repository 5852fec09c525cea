// Projection GEMMs of the stage: forward x @ W (with the library's K-major
// copy of W) and the dX-only backward dY @ W^T of frozen weights, with the
// elementwise work of the block fused into the epilogue.
//
// bf16: MFMA 32x32x16 tiles staged through LDS (double-buffered).  The MFMA
// computes C^T blocks so that each lane ends up owning four consecutive
// output columns of one row, which the epilogue stores as one 8-byte write.
// f32: a plain FMA tile kernel (used by the small fp32 stage only).
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace rg {

// ---------------------------------------------------------------- epilogues
template <Epi E, typename T>
__device__ __forceinline__ void epilogue4(const GemmArgs& a, int m, int n, float v[4]) {
  const long r = m;
  if constexpr (E == Epi::Store || E == Epi::Gelu) {
    if (a.bias) {
      float b[4];
      St<T>::ld4(static_cast<const T*>(a.bias), n, b);
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] += b[i];
    }
    if constexpr (E == Epi::Gelu) {
      if (a.out2) St<T>::st4(static_cast<T*>(a.out2), r * a.ldo2 + n, v);
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = gelu_f(v[i]);
    }
    St<T>::st4(static_cast<T*>(a.out), r * a.ldo + n, v);
  } else if constexpr (E == Epi::Resid) {
    float x[4];
    St<T>::ld4(static_cast<const T*>(a.aux), r * a.ld_aux + n, x);
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] += x[i];
    St<T>::st4(static_cast<T*>(a.out), r * a.ldo + n, v);
  } else if constexpr (E == Epi::DGelu) {
    float x[4];
    St<T>::ld4(static_cast<const T*>(a.aux), r * a.ld_aux + n, x);
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] *= gelu_grad_f(x[i]);
    St<T>::st4(static_cast<T*>(a.out), r * a.ldo + n, v);
  } else if constexpr (E == Epi::DSwiGlu) {
    float g[4], u[4], dg[4], du[4];
    St<T>::ld4(static_cast<const T*>(a.aux), r * a.ld_aux + n, g);
    St<T>::ld4(static_cast<const T*>(a.aux), r * a.ld_aux + a.half + n, u);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float sg = sigmoid_f(g[i]);
      du[i] = v[i] * g[i] * sg;
      dg[i] = v[i] * u[i] * (sg + g[i] * sg * (1.f - sg));
    }
    St<T>::st4(static_cast<T*>(a.out), r * a.ldo + n, dg);
    St<T>::st4(static_cast<T*>(a.out), r * a.ldo + a.half + n, du);
  }
}

// gate/up pair for feature columns f..f+3
template <typename T>
__device__ __forceinline__ void epilogue_swiglu4(const GemmArgs& a, int m, int f, const float g[4],
                                                 const float u[4]) {
  const long r = m;
  float o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) o[i] = g[i] * sigmoid_f(g[i]) * u[i];
  St<T>::st4(static_cast<T*>(a.out), r * a.ldo + f, o);
  if (a.out2) {
    St<T>::st4(static_cast<T*>(a.out2), r * a.ldo2 + f, g);
    St<T>::st4(static_cast<T*>(a.out2), r * a.ldo2 + a.half + f, u);
  }
}

// ---------------------------------------------------------------- bf16 MFMA kernel
constexpr int BK = 64;
constexpr int LDK = BK + 8;  // LDS row pitch (bf16): 144 B keeps 16-B fragment reads conflict-free

template <int BM, int BN, int WM, int WN, Epi E>
__device__ __forceinline__ void gemm_bf16_body(const GemmArgs& a) {
  constexpr int TM = BM / WM, TN = BN / WN;
  constexpr int FM = TM / 32, FN = TN / 32;
  constexpr int CPR = BK / 8;  // 16-B chunks per tile row
  constexpr int AC = BM * CPR / 256, BC = BN * CPR / 256;
  static_assert(WM * WN == 4, "four waves");
  static_assert(AC * 256 == BM * CPR && BC * 256 == BN * CPR, "tile/thread mismatch");
  static_assert(E != Epi::SwiGlu || FN % 2 == 0, "SwiGlu needs gate/up block pairs");
  __shared__ __attribute__((aligned(16))) bf16 sA[2][BM * LDK];
  __shared__ __attribute__((aligned(16))) bf16 sB[2][BN * LDK];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const bf16* A = static_cast<const bf16*>(a.A);
  const bf16* B = static_cast<const bf16*>(a.B);
  const int M = a.M, N = a.N, K = a.K;

  uint4 ra[AC], rb[BC];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < AC; ++i) {
      int idx = tid + i * 256, r = idx / CPR, c = idx % CPR;
      int gm = m0 + r, gk = k0 + c * 8;
      ra[i] = (gm < M && gk < K) ? *reinterpret_cast<const uint4*>(A + (long)gm * a.lda + gk)
                                 : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < BC; ++i) {
      int idx = tid + i * 256, r = idx / CPR, c = idx % CPR;
      int gn = n0 + r, gk = k0 + c * 8;
      rb[i] = (gn < N && gk < K) ? *reinterpret_cast<const uint4*>(B + (long)gn * a.ldb + gk)
                                 : make_uint4(0, 0, 0, 0);
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < AC; ++i) {
      int idx = tid + i * 256, r = idx / CPR, c = idx % CPR;
      *reinterpret_cast<uint4*>(&sA[buf][r * LDK + c * 8]) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < BC; ++i) {
      int idx = tid + i * 256, r = idx / CPR, c = idx % CPR;
      *reinterpret_cast<uint4*>(&sB[buf][r * LDK + c * 8]) = rb[i];
    }
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int nk = (K + BK - 1) / BK;
  gload(0);
  sstore(0);
  __syncthreads();
  const int lrow = lane & 31, lk = (lane >> 5) * 8;
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) gload((kt + 1) * BK);
    const bf16* pa = &sA[cur][(wm * TM + lrow) * LDK + lk];
    const bf16* pb = &sB[cur][(wn * TN + lrow) * LDK + lk];
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      bf16x8 fa[FM], fb[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) fa[i] = ld_frag(pa + i * 32 * LDK + ks * 16);
#pragma unroll
      for (int j = 0; j < FN; ++j) fb[j] = ld_frag(pb + j * 32 * LDK + ks * 16);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = mfma32(fb[j], fa[i], acc[i][j]);
    }
    if (kt + 1 < nk) sstore(cur ^ 1);
    __syncthreads();
  }

  // lane owns row m = m0 + wm*TM + i*32 + lane%32 and, per group g, columns
  // n0 + wn*TN + j*32 + 8g + 4*(lane/32) + {0..3}
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int m = m0 + wm * TM + i * 32 + lrow;
    if (m >= M) continue;
    if constexpr (E == Epi::SwiGlu) {
#pragma unroll
      for (int j = 0; j < FN; j += 2) {
        // packed columns [64p, 64p+32) are gates, [64p+32, 64p+64) the matching ups
        const int ng = n0 + wn * TN + j * 32;
        if (ng >= N) continue;
        const int fbase = (ng / 64) * 32;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          float gv[4], uv[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) { gv[q] = acc[i][j][4 * g + q]; uv[q] = acc[i][j + 1][4 * g + q]; }
          epilogue_swiglu4<bf16>(a, m, fbase + 8 * g + 4 * (lane >> 5), gv, uv);
        }
      }
    } else {
#pragma unroll
      for (int j = 0; j < FN; ++j) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int n = n0 + wn * TN + j * 32 + 8 * g + 4 * (lane >> 5);
          if (n >= N) continue;
          float v[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) v[q] = acc[i][j][4 * g + q];
          epilogue4<E, bf16>(a, m, n, v);
        }
      }
    }
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

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// 16 B per lane, global -> LDS; lane i of the wave lands at lds + 16 i
__device__ __forceinline__ void dma16(const void* g, void* lds) {
  __builtin_amdgcn_global_load_lds(g, (lds_ptr_t)lds, 16, 0, 0);
}

template <int N>
__device__ __forceinline__ void wait_vm_lgkm() {  // vmcnt <= N and lgkmcnt == 0
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | (0x7 << 4) | ((N >> 4) << 14));
}
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  // gfx9 encoding: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt[5:4] at [15:14]
  __builtin_amdgcn_s_waitcnt((N & 0xF) | (0x7 << 4) | (0xF << 8) | ((N >> 4) << 14));
}

template <int BM, int BN, int WM, int WN, int NS, Epi E, int GROUP = 4>
__device__ __forceinline__ void gemm_bf16_dma_body(const GemmArgs& a) {
  constexpr int TM = BM / WM, TN = BN / WN;
  constexpr int FM = TM / 32, FN = TN / 32;
  constexpr int ROWB = 128;
  constexpr int STAGE = (BM + BN) * ROWB;
  constexpr int LA = BM / 32, LB = BN / 32, LPT = LA + LB;  // load instructions per wave per k-tile
  static_assert(WM * WN == 4, "four waves");
  static_assert(LPT * (NS - 2) < 64, "vmcnt range");
  static_assert(E != Epi::SwiGlu || FN % 2 == 0, "SwiGlu needs gate/up block pairs");
  // one LDS array per stage, so that reads of one stage provably do not alias
  // the DMA writes in flight to the others (no compiler-inserted vmcnt waits)
  __shared__ __attribute__((aligned(1024))) char st0[STAGE];
  __shared__ __attribute__((aligned(1024))) char st1[STAGE];
  __shared__ __attribute__((aligned(1024))) char st2[NS > 2 ? STAGE : 16];
  __shared__ __attribute__((aligned(1024))) char st3[NS > 3 ? STAGE : 16];
  static_assert(NS >= 2 && NS <= 4, "2 to 4 stages");
  auto stage_base = [&](auto S) -> char* {
    constexpr int s_ = decltype(S)::value;
    if constexpr (s_ == 0) return st0;
    else if constexpr (s_ == 1) return st1;
    else if constexpr (s_ == 2) return st2;
    else return st3;
  };

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  int m0, n0;
  tile_coords<BM, BN, GROUP>(a.M, a.N, m0, n0);
  const bf16* A = static_cast<const bf16*>(a.A);
  const bf16* B = static_cast<const bf16*>(a.B);
  const int M = a.M, N = a.N, K = a.K;

  const int lrow = lane >> 3, lpos = lane & 7;
  const bf16* ga[LA];
  const bf16* gb[LB];
#pragma unroll
  for (int i = 0; i < LA; ++i) {
    const int r = i * 32 + wave * 8 + lrow;
    ga[i] = A + (long)min(m0 + r, M - 1) * a.lda + ((lpos ^ ((r >> 1) & 7)) * 8);
  }
#pragma unroll
  for (int i = 0; i < LB; ++i) {
    const int r = i * 32 + wave * 8 + lrow;
    gb[i] = B + (long)min(n0 + r, N - 1) * a.ldb + ((lpos ^ ((r >> 1) & 7)) * 8);
  }
  auto issue = [&](int kt, char* sb) {
#pragma unroll
    for (int i = 0; i < LA; ++i)
      dma16(ga[i] + kt * 64, sb + (i * 32 + wave * 8) * ROWB);
#pragma unroll
    for (int i = 0; i < LB; ++i)
      dma16(gb[i] + kt * 64, sb + (BM + i * 32 + wave * 8) * ROWB);
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int nk = K / 64;
  const int l32 = lane & 31, half = lane >> 5, sw = (lane >> 1) & 7;
  issue(0, st0);
  if constexpr (NS > 2) if (1 < nk) issue(1, st1);
  if constexpr (NS > 3) if (2 < nk) issue(2, st2);
  // One k-tile in stage S: wait for this wave's loads of it, barrier (every
  // wave's loads landed; every wave finished reading the previous stage, whose
  // fragments fed its previous MFMAs), refill that previous stage with tile
  // kt + NS - 1, read fragments, multiply.  Two workgroups fit per CU, so one
  // wave's fragment reads overlap another's MFMAs.
  auto step = [&](auto S, int kt) {
    constexpr int s_ = decltype(S)::value;
    const int later = min(NS - 2, nk - 1 - kt);  // tiles after kt already issued
    if constexpr (NS >= 4) {
      if (later >= 2) wait_vmcnt<2 * LPT>();
      else if (later == 1) wait_vmcnt<LPT>();
      else wait_vmcnt<0>();
    } else if constexpr (NS == 3) {
      if (later >= 1) wait_vmcnt<LPT>();
      else wait_vmcnt<0>();
    } else {
      wait_vmcnt<0>();
    }
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    if (kt + NS - 1 < nk) issue(kt + NS - 1, stage_base(std::integral_constant<int, (s_ + NS - 1) % NS>{}));
    const char* sa = stage_base(S) + (wm * TM + l32) * ROWB;
    const char* sbb = stage_base(S) + (BM + wn * TN + l32) * ROWB;
    bf16x8 fa[4][FM], fb[4][FN];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int off = 16 * ((2 * ks + half) ^ sw);
#pragma unroll
      for (int i = 0; i < FM; ++i) fa[ks][i] = *reinterpret_cast<const bf16x8*>(sa + i * 32 * ROWB + off);
#pragma unroll
      for (int j = 0; j < FN; ++j) fb[ks][j] = *reinterpret_cast<const bf16x8*>(sbb + j * 32 * ROWB + off);
    }
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = mfma32(fb[ks][j], fa[ks][i], acc[i][j]);
  };
  for (int kt = 0; kt < nk; kt += NS) {
    step(std::integral_constant<int, 0>{}, kt);
    if (kt + 1 < nk) step(std::integral_constant<int, 1>{}, kt + 1);
    if constexpr (NS > 2) if (kt + 2 < nk) step(std::integral_constant<int, 2>{}, kt + 2);
    if constexpr (NS > 3) if (kt + 3 < nk) step(std::integral_constant<int, 3>{}, kt + 3);
  }

#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int m = m0 + wm * TM + i * 32 + l32;
    if (m >= M) continue;
    if constexpr (E == Epi::SwiGlu) {
#pragma unroll
      for (int j = 0; j < FN; j += 2) {
        const int ng = n0 + wn * TN + j * 32;
        if (ng >= N) continue;
        const int fbase = (ng / 64) * 32;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          float gv[4], uv[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) { gv[q] = acc[i][j][4 * g + q]; uv[q] = acc[i][j + 1][4 * g + q]; }
          epilogue_swiglu4<bf16>(a, m, fbase + 8 * g + 4 * half, gv, uv);
        }
      }
    } else {
#pragma unroll
      for (int j = 0; j < FN; ++j) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int n = n0 + wn * TN + j * 32 + 8 * g + 4 * half;
          if (n >= N) continue;
          float v[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) v[q] = acc[i][j][4 * g + q];
          epilogue4<E, bf16>(a, m, n, v);
        }
      }
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
    if (m < a.M && n < a.N) epilogue4<E, float>(a, m, n, acc[i]);
  }
}

// ---------------------------------------------------------------- named kernels
#define RG_GEMM_KERNELS(NAME)                                                        \
  template <int BM, int BN, int WM, int WN, Epi E>                                   \
  __global__ __launch_bounds__(256) void NAME(GemmArgs a) {                          \
    gemm_bf16_body<BM, BN, WM, WN, E>(a);                                            \
  }                                                                                  \
  template <int BM, int BN, int WM, int WN, int NS, Epi E>                           \
  __global__ __launch_bounds__(256) void NAME##_dma(GemmArgs a) {                    \
    gemm_bf16_dma_body<BM, BN, WM, WN, NS, E, 4>(a);                                 \
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
    case R_QKV_FWD: case R_O_FWD: case R_FFN_OUT_FWD: case R_O_DX: return e == Epi::Store;
    case R_FFN_IN_FWD: return e == Epi::Gelu || e == Epi::SwiGlu;
    case R_QKV_DX: case R_FFN_IN_DX: return e == Epi::Resid || e == Epi::Store;
    case R_FFN_OUT_DX: return e == Epi::DGelu || e == Epi::DSwiGlu;
    default: return false;
  }
}

// tile shape: 128x128 with two stages when that gives at least three
// workgroups per CU (the 2 x 256-CU occupancy is then full twice over), else
// 64x128 with three stages (measured on the BERT-base stage shapes)
enum Cfg { C_DMA_128x128, C_DMA_64x128, C_REG_128x128, C_REG_64x128 };

template <Role R, Epi E>
static hipError_t launch_role(Cfg cfg, int dtype, const GemmArgs& a, hipStream_t s) {
  if constexpr (!role_has(R, E)) {
    return hipErrorInvalidValue;
  } else {
#define RG_NAME(SUFFIX)                                                                    \
  (R == R_QKV_FWD ? 0 : 0)
    const dim3 block(256);
    if (dtype == DT_F32) {
      if constexpr (E == Epi::SwiGlu) return hipErrorInvalidValue;
      else {
        dim3 grid((a.N + 63) / 64, (a.M + 63) / 64);
        switch (R) {
#define RG_F32(ROLE, NAME) case ROLE: hipLaunchKernelGGL((NAME##_f32<E>), grid, block, 0, s, a); break;
          RG_F32(R_QKV_FWD, gemm_qkv_fwd) RG_F32(R_O_FWD, gemm_o_fwd) RG_F32(R_FFN_IN_FWD, gemm_ffn_in_fwd)
          RG_F32(R_FFN_OUT_FWD, gemm_ffn_out_fwd) RG_F32(R_QKV_DX, gemm_qkv_dx) RG_F32(R_O_DX, gemm_o_dx)
          RG_F32(R_FFN_IN_DX, gemm_ffn_in_dx) RG_F32(R_FFN_OUT_DX, gemm_ffn_out_dx)
#undef RG_F32
          default: return hipErrorInvalidValue;
        }
        return hipGetLastError();
      }
    }
#define RG_LAUNCH(NAME)                                                                                  \
  switch (cfg) {                                                                                         \
    case C_DMA_128x128:                                                                                  \
      hipLaunchKernelGGL((NAME##_dma<128, 128, 2, 2, 2, E>),                                             \
                         dim3(((a.N + 127) / 128) * ((a.M + 127) / 128)), block, 0, s, a);               \
      break;                                                                                             \
    case C_DMA_64x128:                                                                                   \
      hipLaunchKernelGGL((NAME##_dma<64, 128, 2, 2, 3, E>),                                              \
                         dim3(((a.N + 127) / 128) * ((a.M + 63) / 64)), block, 0, s, a);                 \
      break;                                                                                             \
    case C_REG_128x128:                                                                                  \
      hipLaunchKernelGGL((NAME<128, 128, 2, 2, E>), dim3((a.N + 127) / 128, (a.M + 127) / 128), block, 0, \
                         s, a);                                                                          \
      break;                                                                                             \
    case C_REG_64x128:                                                                                   \
      hipLaunchKernelGGL((NAME<64, 128, 2, 2, E>), dim3((a.N + 127) / 128, (a.M + 63) / 64), block, 0,   \
                         s, a);                                                                          \
      break;                                                                                             \
  }
    switch (R) {
      case R_QKV_FWD: RG_LAUNCH(gemm_qkv_fwd) break;
      case R_O_FWD: RG_LAUNCH(gemm_o_fwd) break;
      case R_FFN_IN_FWD: RG_LAUNCH(gemm_ffn_in_fwd) break;
      case R_FFN_OUT_FWD: RG_LAUNCH(gemm_ffn_out_fwd) break;
      case R_QKV_DX: RG_LAUNCH(gemm_qkv_dx) break;
      case R_O_DX: RG_LAUNCH(gemm_o_dx) break;
      case R_FFN_IN_DX: RG_LAUNCH(gemm_ffn_in_dx) break;
      case R_FFN_OUT_DX: RG_LAUNCH(gemm_ffn_out_dx) break;
      default: return hipErrorInvalidValue;
    }
#undef RG_LAUNCH
#undef RG_NAME
    return hipGetLastError();
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
    case Epi::DSwiGlu: return launch_role<R, Epi::DSwiGlu>(cfg, dtype, a, s);
  }
  return hipErrorInvalidValue;
}

static bool al16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
static bool al8(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 7u) == 0; }

hipError_t launch_gemm(int dtype, Role role, Epi epi, const GemmArgs& a, hipStream_t s) {
  if (a.M < 0 || a.N <= 0 || a.K <= 0 || !a.A || !a.B || !a.out) return hipErrorInvalidValue;
  if (a.M == 0) return hipSuccess;
  if (a.N % 4 || a.ldo % 4 || a.lda < a.K || a.ldb < a.K) return hipErrorInvalidValue;
  if ((epi == Epi::Resid || epi == Epi::DGelu || epi == Epi::DSwiGlu) && (!a.aux || a.ld_aux % 4))
    return hipErrorInvalidValue;
  if ((epi == Epi::SwiGlu || epi == Epi::DSwiGlu) && (a.half % 4)) return hipErrorInvalidValue;
  if (a.out2 && a.ldo2 % 4) return hipErrorInvalidValue;
  Cfg cfg = C_REG_128x128;
  if (dtype == DT_BF16) {
    // 16-B operand chunks and 8-B epilogue vectors
    if (a.K % 8 || a.lda % 8 || a.ldb % 8 || !al16(a.A) || !al16(a.B) || !al8(a.out))
      return hipErrorInvalidValue;
    if (epi == Epi::SwiGlu && (a.N % 64 || a.half * 2 != a.N)) return hipErrorInvalidValue;
    const long tiles128 = (long)((a.M + 127) / 128) * ((a.N + 127) / 128);
    const bool big = tiles128 >= 768;
    if (a.K % 64 == 0) cfg = big ? C_DMA_128x128 : C_DMA_64x128;
    else cfg = tiles128 >= 512 ? C_REG_128x128 : C_REG_64x128;
  } else if (dtype == DT_F32) {
    if (!al16(a.out)) return hipErrorInvalidValue;
  } else {
    return hipErrorInvalidValue;
  }
  switch (role) {
    case R_QKV_FWD: return launch_epi<R_QKV_FWD>(epi, cfg, dtype, a, s);
    case R_O_FWD: return launch_epi<R_O_FWD>(epi, cfg, dtype, a, s);
    case R_FFN_IN_FWD: return launch_epi<R_FFN_IN_FWD>(epi, cfg, dtype, a, s);
    case R_FFN_OUT_FWD: return launch_epi<R_FFN_OUT_FWD>(epi, cfg, dtype, a, s);
    case R_QKV_DX: return launch_epi<R_QKV_DX>(epi, cfg, dtype, a, s);
    case R_O_DX: return launch_epi<R_O_DX>(epi, cfg, dtype, a, s);
    case R_FFN_IN_DX: return launch_epi<R_FFN_IN_DX>(epi, cfg, dtype, a, s);
    case R_FFN_OUT_DX: return launch_epi<R_FFN_OUT_DX>(epi, cfg, dtype, a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace rg
