// Projection GEMMs of the stage: forward x @ W (with the library's K-major
// copy of W) and the dX-only backward dY @ W^T of frozen weights, with the
// elementwise work of the block fused into the epilogue.
//
// bf16: MFMA 32x32x16 tiles staged through LDS (double-buffered).  The MFMA
// computes C^T blocks so that each lane ends up owning four consecutive
// output columns of one row, which the epilogue stores as one 8-byte write.
// f32: a plain FMA tile kernel (used by the small fp32 stage only).
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

template <int BM, int BN, int WM, int WN, Epi E>
static hipError_t launch_bf16_cfg(Role role, const GemmArgs& a, hipStream_t s) {
  dim3 grid((a.N + BN - 1) / BN, (a.M + BM - 1) / BM), block(256);
#define RG_CASE(R, NAME)                                                   \
  case R:                                                                  \
    hipLaunchKernelGGL((NAME<BM, BN, WM, WN, E>), grid, block, 0, s, a);   \
    break;
  switch (role) {
    RG_CASE(R_QKV_FWD, gemm_qkv_fwd)
    RG_CASE(R_O_FWD, gemm_o_fwd)
    RG_CASE(R_FFN_IN_FWD, gemm_ffn_in_fwd)
    RG_CASE(R_FFN_OUT_FWD, gemm_ffn_out_fwd)
    RG_CASE(R_QKV_DX, gemm_qkv_dx)
    RG_CASE(R_O_DX, gemm_o_dx)
    RG_CASE(R_FFN_IN_DX, gemm_ffn_in_dx)
    RG_CASE(R_FFN_OUT_DX, gemm_ffn_out_dx)
    default: return hipErrorInvalidValue;
  }
#undef RG_CASE
  return hipGetLastError();
}

template <Epi E>
static hipError_t launch_f32_cfg(Role role, const GemmArgs& a, hipStream_t s) {
  dim3 grid((a.N + 63) / 64, (a.M + 63) / 64), block(256);
#define RG_CASE(R, NAME)                                                \
  case R:                                                               \
    hipLaunchKernelGGL((NAME##_f32<E>), grid, block, 0, s, a);          \
    break;
  switch (role) {
    RG_CASE(R_QKV_FWD, gemm_qkv_fwd)
    RG_CASE(R_O_FWD, gemm_o_fwd)
    RG_CASE(R_FFN_IN_FWD, gemm_ffn_in_fwd)
    RG_CASE(R_FFN_OUT_FWD, gemm_ffn_out_fwd)
    RG_CASE(R_QKV_DX, gemm_qkv_dx)
    RG_CASE(R_O_DX, gemm_o_dx)
    RG_CASE(R_FFN_IN_DX, gemm_ffn_in_dx)
    RG_CASE(R_FFN_OUT_DX, gemm_ffn_out_dx)
    default: return hipErrorInvalidValue;
  }
#undef RG_CASE
  return hipGetLastError();
}

template <Epi E>
static hipError_t launch_bf16_epi(Role role, const GemmArgs& a, hipStream_t s) {
  // 128x128 tiles when they give at least two waves of workgroups over the
  // 256 CUs, else 64x128 tiles
  const long tiles128 = (long)((a.M + 127) / 128) * ((a.N + 127) / 128);
  if (tiles128 >= 512) return launch_bf16_cfg<128, 128, 2, 2, E>(role, a, s);
  return launch_bf16_cfg<64, 128, 2, 2, E>(role, a, s);
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
  if (dtype == DT_BF16) {
    // 16-B operand chunks and 8-B epilogue vectors
    if (a.K % 8 || a.lda % 8 || a.ldb % 8 || !al16(a.A) || !al16(a.B) || !al8(a.out))
      return hipErrorInvalidValue;
    if (epi == Epi::SwiGlu && (a.N % 64 || a.half * 2 != a.N)) return hipErrorInvalidValue;
    switch (epi) {
      case Epi::Store: return launch_bf16_epi<Epi::Store>(role, a, s);
      case Epi::Gelu: return launch_bf16_epi<Epi::Gelu>(role, a, s);
      case Epi::Resid: return launch_bf16_epi<Epi::Resid>(role, a, s);
      case Epi::DGelu: return launch_bf16_epi<Epi::DGelu>(role, a, s);
      case Epi::SwiGlu: return launch_bf16_epi<Epi::SwiGlu>(role, a, s);
      case Epi::DSwiGlu: return launch_bf16_epi<Epi::DSwiGlu>(role, a, s);
    }
    return hipErrorInvalidValue;
  }
  if (dtype == DT_F32) {
    if (!al16(a.out)) return hipErrorInvalidValue;
    switch (epi) {
      case Epi::Store: return launch_f32_cfg<Epi::Store>(role, a, s);
      case Epi::Gelu: return launch_f32_cfg<Epi::Gelu>(role, a, s);
      case Epi::Resid: return launch_f32_cfg<Epi::Resid>(role, a, s);
      case Epi::DGelu: return launch_f32_cfg<Epi::DGelu>(role, a, s);
      case Epi::DSwiGlu: return launch_f32_cfg<Epi::DSwiGlu>(role, a, s);
      default: return hipErrorInvalidValue;  // SwiGlu packing is bf16-only
    }
  }
  return hipErrorInvalidValue;
}

}  // namespace rg
