// Shared device helpers of the RingAda HIP kernels (gfx950 only).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rg {

typedef uint16_t bf16;  // bfloat16 bit pattern
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float bf2f(bf16 b) { return __uint_as_float((uint32_t)b << 16); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// round to nearest even (v_cvt_pk_bf16_f32); NaN stays NaN
__device__ __forceinline__ bf16 f2bf(float f) { return __builtin_bit_cast(bf16, (__bf16)f); }
__device__ __forceinline__ uint32_t f2bf2(float lo, float hi) {
  bf16x2_t v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

// storage abstraction: float or bf16 storage, fp32 arithmetic
template <typename T> struct St;
template <> struct St<float> {
  static __device__ __forceinline__ float ld(const float* p, long i) { return p[i]; }
  static __device__ __forceinline__ void st(float* p, long i, float v) { p[i] = v; }
  // four consecutive elements (16 B aligned)
  static __device__ __forceinline__ void ld4(const float* p, long i, float v[4]) {
    float4 q = *reinterpret_cast<const float4*>(p + i);
    v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
  }
  static __device__ __forceinline__ void st_nt(float* p, long i, float v) {  // streamed (st16 below)
    __builtin_nontemporal_store(v, p + i);
  }
  static __device__ __forceinline__ void st4(float* p, long i, const float v[4]) {
    *reinterpret_cast<float4*>(p + i) = make_float4(v[0], v[1], v[2], v[3]);
  }
};
template <> struct St<bf16> {
  static __device__ __forceinline__ float ld(const bf16* p, long i) { return bf2f(p[i]); }
  static __device__ __forceinline__ void st(bf16* p, long i, float v) { p[i] = f2bf(v); }
  static __device__ __forceinline__ void st_nt(bf16* p, long i, float v) {  // streamed (st16 below)
    __builtin_nontemporal_store(f2bf(v), p + i);
  }
  // four consecutive elements (8 B aligned)
  static __device__ __forceinline__ void ld4(const bf16* p, long i, float v[4]) {
    uint2 q = *reinterpret_cast<const uint2*>(p + i);
    v[0] = __uint_as_float(q.x << 16); v[1] = __uint_as_float(q.x & 0xffff0000u);
    v[2] = __uint_as_float(q.y << 16); v[3] = __uint_as_float(q.y & 0xffff0000u);
  }
  static __device__ __forceinline__ void st4(bf16* p, long i, const float v[4]) {
    uint2 q;
    q.x = f2bf2(v[0], v[1]);
    q.y = f2bf2(v[2], v[3]);
    *reinterpret_cast<uint2*>(p + i) = q;
  }
  // the same, streamed when nt (st16 and stream_out below)
  static __device__ __forceinline__ void st4s(bf16* p, long i, const float v[4], bool nt) {
    const uint32_t lo = f2bf2(v[0], v[1]), hi = f2bf2(v[2], v[3]);
    typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
    if (nt) {
      __builtin_nontemporal_store(u32x2_t{lo, hi}, reinterpret_cast<u32x2_t*>(p + i));
    } else {
      uint32_t* d = reinterpret_cast<uint32_t*>(p + i);
      d[0] = lo;
      d[1] = hi;
    }
  }
};

// ---------------------------------------------------------------- math
__device__ __forceinline__ float gelu_f(float u) {  // u * Phi(u), erf form
  return 0.5f * u * (1.f + erff(u * 0.70710678118654752f));
}
__device__ __forceinline__ float gelu_grad_f(float u) {  // Phi(u) + u phi(u)
  float cdf = 0.5f * (1.f + erff(u * 0.70710678118654752f));
  return cdf + u * 0.39894228040143268f * __expf(-0.5f * u * u);
}
__device__ __forceinline__ float sigmoid_f(float u) { return 1.f / (1.f + __expf(-u)); }

// Cheaper GELU for bf16 outputs: erf by the rational-times-Gaussian form of
// Abramowitz & Stegun, Handbook of Mathematical Functions, formula 7.1.26
// (absolute error <= 1.5e-7, far below bf16 resolution).  For z = u / sqrt(2)
// the Gaussian factor exp(-z^2) = exp(-u^2 / 2) is the one gelu' needs, so
// both come from one exponential.
struct ErfGauss {
  float erf_z;  // erf(u / sqrt 2)
  float gauss;  // exp(-u^2 / 2)
};
__device__ __forceinline__ ErfGauss erf_gauss_as(float u) {
  const float z = fabsf(u) * 0.70710678118654752f;
  const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, z, 1.f));
  float p = fmaf(1.061405429f, t, -1.453152027f);
  p = fmaf(p, t, 1.421413741f);
  p = fmaf(p, t, -0.284496736f);
  p = fmaf(p, t, 0.254829592f);
  p *= t;
  const float g = __builtin_amdgcn_exp2f(-0.72134752044448170f * u * u);  // exp(-u^2/2) = 2^(-u^2 log2(e)/2)
  const float e = fmaf(-p, g, 1.f);
  return {copysignf(e, u), g};
}
// GELU of the GEMM epilogue: u sigma(g(u)), g an odd degree-9 polynomial
// fitted to the logit of the normal CDF on [-8, 8] (fit_gelu_logistic.py; g
// keeps rising past the range, so sigma(g) still tends to 0 and 1).  One
// exp2 and one reciprocal, and five FMAs fewer than the erf form.  In fp32
// |gelu_logistic(u) - u Phi(u)| <= 7e-6 for all u, far below the bf16
// rounding of the output it feeds (FFN-in 28.2 -> 26.7 us per launch at the
// BERT-base shape).
__device__ __forceinline__ float gelu_logistic(float u) {
  const float x2 = u * u;
  // t = -g(u) log2(e) = u P(u^2)
  float p = fmaf(x2, -4.18002687e-06f, 1.06986963e-04f);
  p = fmaf(p, x2, 2.48102472e-04f);
  p = fmaf(p, x2, -1.04997842e-01f);
  p = fmaf(p, x2, -2.30216815e+00f);
  return u * __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(p * u));
}
__device__ __forceinline__ float gelu_fast(float u) {
  return 0.5f * u * (1.f + erf_gauss_as(u).erf_z);
}
__device__ __forceinline__ float gelu_grad_fast(float u) {
  const ErfGauss eg = erf_gauss_as(u);
  return fmaf(u * 0.39894228040143268f, eg.gauss, 0.5f * (1.f + eg.erf_z));
}

// ---------------------------------------------------------------- MFMA
// D[32x32] += A[32x16] * B[16x32]; lane l supplies A[l%32][8*(l/32)+v] and
// B[8*(l/32)+v][l%32]; D lane l holds D[8*(r/4)+4*(l/32)+r%4][l%32].
__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
// D[16x16] += A[16x32] * B[32x16]; lane l supplies A[l%16][8*(l/16)+v] and
// B[8*(l/16)+v][l%16]; D lane l holds D[4*(l/16)+r][l%16].
__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 ld_frag(const bf16* p) {  // 16 B
  return *reinterpret_cast<const bf16x8*>(p);
}
// Output stores with the non-temporal hint.  A plain store leaves the line dirty
// in this XCD's L2, to be written back when the kernel ends; every kernel's
// outputs are read by the next kernel from all eight XCDs, so that write-back
// sits on the kernel's tail.  A streamed line goes out at once, but is not
// allocated in the Infinity Cache either, so the next kernel reads it from HBM.
// Measured (write, then read in the next kernel): streaming wins up to 32 MiB
// per tensor, the eight L2s' capacity, and loses from 64 MiB on, where the
// plain stores' Infinity Cache hits dominate.  So an output is streamed iff it
// is at most NT_MAX_BYTES, and every streamed store writes whole 128-B lines
// per instruction (scattered pieces would leave the L2 unmerged).
// Given a plain and a non-temporal store of the same value to the same address
// in the two arms of a branch, the compiler merges them into one store that
// carries only the attributes both share, which drops the hint.  So the plain
// arm stores the same bytes in two halves: a different instruction, which the
// compiler cannot merge with the streamed one (the backend may pair the
// halves again inside the plain arm).  Small outputs ([T][m] stashes, split-K
// partials) are always streamed (st_nt).
constexpr long NT_MAX_BYTES = 32l << 20;
__device__ __forceinline__ bool stream_out(long bytes) { return bytes <= NT_MAX_BYTES; }
__device__ __forceinline__ void st16(void* p, bf16x8 v, bool nt) {
  typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
  const u32x4_t q = __builtin_bit_cast(u32x4_t, v);
  if (nt) {
    __builtin_nontemporal_store(q, static_cast<u32x4_t*>(p));
  } else {
    uint2* d = static_cast<uint2*>(p);
    d[0] = make_uint2(q.x, q.y);
    d[1] = make_uint2(q.z, q.w);
  }
}
__device__ __forceinline__ bf16x8 zero_frag() {
  uint4 z = make_uint4(0, 0, 0, 0);
  return __builtin_bit_cast(bf16x8, z);
}
__device__ __forceinline__ bf16x8 pack_frag(const float v[8]) {
  uint4 q;
  q.x = f2bf2(v[0], v[1]);
  q.y = f2bf2(v[2], v[3]);
  q.z = f2bf2(v[4], v[5]);
  q.w = f2bf2(v[6], v[7]);
  return __builtin_bit_cast(bf16x8, q);
}
__device__ __forceinline__ void unpack_frag(bf16x8 f, float v[8]) {
  uint4 q = __builtin_bit_cast(uint4, f);
  v[0] = __uint_as_float(q.x << 16); v[1] = __uint_as_float(q.x & 0xffff0000u);
  v[2] = __uint_as_float(q.y << 16); v[3] = __uint_as_float(q.y & 0xffff0000u);
  v[4] = __uint_as_float(q.z << 16); v[5] = __uint_as_float(q.z & 0xffff0000u);
  v[6] = __uint_as_float(q.w << 16); v[7] = __uint_as_float(q.w & 0xffff0000u);
}

// ---------------------------------------------------------------- LDS transpose reads
typedef short v4i16_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16_t* lds_v4i16_ptr;
// ds_read_b64_tr_b16 over a row-major LDS tile X[k][n] (pitch in elements):
// for the 16-lane group of this lane, returns X[k0 + 0..3][n0 + lane % 16]
// as 4 consecutive bf16.  (Within a group, lane r = 4j + q supplies the address
// of X[k0 + j][n0 + 4q]; the instruction hands lane i element i % 4 of the
// rows supplied by lanes i/4, 4 + i/4, 8 + i/4, 12 + i/4.)
__device__ __forceinline__ uint2 lds_tr4(const bf16* tile, int pitch, int k0, int n0, int lane) {
  const int r = lane & 15;
  const bf16* p = tile + (k0 + (r >> 2)) * pitch + n0 + 4 * (r & 3);
  return __builtin_bit_cast(uint2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_ptr)p));
}
// MFMA 32x32x16 operand with k contiguous per lane from a row-major [k][n]
// tile: lane l gets X[k0 + 8*(l/32) + 0..7][n0 + l%32]
__device__ __forceinline__ bf16x8 lds_tr_frag32(const bf16* tile, int pitch, int k0, int n0, int lane) {
  const int g = lane >> 4, nn = n0 + 16 * (g & 1), kk = k0 + 8 * (g >> 1);
  const uint2 lo = lds_tr4(tile, pitch, kk, nn, lane), hi = lds_tr4(tile, pitch, kk + 4, nn, lane);
  return __builtin_bit_cast(bf16x8, make_uint4(lo.x, lo.y, hi.x, hi.y));
}

// ---------------------------------------------------------------- packed adapter weights (bf16 path)
// The bf16 adapter kernels run 16 waves over a d-wide row (d = 256 * FB) and
// read the bottleneck weights only as MFMA 16x16x32 operand fragments.  The
// working copies are stored in the order those fragments are read, so every
// fragment load is one contiguous 1-KiB run (lane l at element 8 l):
//  * layout A, for a [64][d] operand X (W_down^T in the forward, W_up in the
//    backward): wave w = 4 ks + ug, k-step j < d / 128, lane = 16 grp + l16
//    holds X[16 ug + l16][ks d/4 + 32 j + 8 grp + 0..7];
//  * layout B, for a [d][64] operand X (W_up^T in the forward, W_down in the
//    backward): wave w, block b < d / 256, half h, lane = 16 grp + l16 holds
//    X[16 (FB w + b) + l16][32 h + 8 grp + 0..7].
__host__ __device__ inline long pack_a_idx(int r, int c, int d) {  // X[r][c], r < 64, c < d
  const int slice = d / 4, ks = c / slice, cc = c % slice, j = cc / 32, w8 = cc % 32;
  const int wave = 4 * ks + r / 16, lane = 16 * (w8 / 8) + r % 16;
  return ((long)(wave * (d / 128) + j) * 64 + lane) * 8 + w8 % 8;
}
__host__ __device__ inline long pack_b_idx(int r, int c, int d) {  // X[r][c], r < d, c < 64
  const int fb = d / 256, wave = r / (16 * fb), rr = r % (16 * fb), b = rr / 16;
  const int h = c / 32, cc = c % 32, lane = 16 * (cc / 8) + rr % 16;
  return ((long)(wave * 2 * fb + 2 * b + h) * 64 + lane) * 8 + cc % 8;
}
// fragment (16 B) k-step j of wave w in layout A / block b, half h in layout B
__device__ __forceinline__ const bf16* pack_a_frag(const void* base, int d, int wave, int j, int lane) {
  return static_cast<const bf16*>(base) + ((long)(wave * (d / 128) + j) * 64 + lane) * 8;
}
__device__ __forceinline__ const bf16* pack_b_frag(const void* base, int d, int wave, int b, int h, int lane) {
  return static_cast<const bf16*>(base) + ((long)(wave * 2 * (d / 256) + 2 * b + h) * 64 + lane) * 8;
}

// ---------------------------------------------------------------- global -> LDS DMA
typedef __attribute__((address_space(3))) void* lds_ptr_t;

// Global -> LDS DMA, 16 B per lane (lane i lands at the LDS address + 16 i),
// issued from inline assembly: scalar base + 32-bit per-lane byte
// offset, LDS destination (wave-uniform byte address) in M0.  The compiler's
// wait-count pass does not see these loads, so it inserts no vmcnt waits of
// its own before LDS reads; the kernel waits for them explicitly (vmcnt
// counts them like any vector load).  Kernels using this touch M0 nowhere
// else.
__device__ __forceinline__ void dma16_m0(const void* gbase, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2" ::"s"(lds), "v"(voff), "s"(gbase)
               : "memory");
}
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(lds_ptr_t)p;
}

// ---------------------------------------------------------------- XCD-aware block order
// Workgroups are dispatched round-robin over the 8 XCDs (linear workgroup id i
// runs on XCD i % 8), each XCD with its own L2.  xcd_block maps the linear id
// of one of n workgroups to a block index such that every XCD processes a
// contiguous eighth of the blocks (identity when n is not a multiple of 8).
// The projection GEMMs give each XCD a contiguous band of token rows the same
// way, so a kernel whose blocks are token ranges in this order finds the rows
// the previous kernel wrote in its own XCD's L2.
__device__ __forceinline__ int xcd_block(int id, int n) { return n % 8 == 0 ? (id % 8) * (n / 8) + id / 8 : id; }

// ---------------------------------------------------------------- reductions
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

}  // namespace rg
