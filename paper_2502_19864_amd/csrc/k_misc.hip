// Row-wise norms (RMSNorm, and the vectorised LayerNorm / RMSNorm rows of the
// wide adapters), parameter layout kernels, the adapter update and the
// initiator's loss helpers.
#include <algorithm>
#include <initializer_list>
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace rg {

template <typename T>
__device__ float blk_sum(float v, float* red) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  float t = 0.f;
  for (int w = 0; w < nw; ++w) t += red[w];
  return t;
}

// ---------------------------------------------------------------- row norms, bf16, vectorised
// One 256-thread workgroup per row, eight features per 16-B access (d <= 4096,
// so at most two per thread).
constexpr int NORM_NPT = 2;
__device__ __forceinline__ float block_sum256(float v, float* red) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) red[wave] = v;
  __syncthreads();
  const float t = (red[0] + red[1]) + (red[2] + red[3]);
  __syncthreads();
  return t;
}
__device__ __forceinline__ void ld8f(const bf16* p, float v[8]) { unpack_frag(ld_frag(p), v); }
__device__ __forceinline__ void st8f(bf16* p, const float v[8], bool nt) { st16(p, pack_frag(v), nt); }

// h = x1 (+ x2); LN: out = LN(h) g + b (out may alias x1); RMS: out = h (when
// x2 is given) and out_norm = RMSNorm(h) g; None: out = h.  xhat, rstd stashed
// when given.
__global__ __launch_bounds__(256) void norm_rows_fwd_bf16(int d, float eps, Norm norm, const bf16* x1,
                                                             const bf16* x2, const bf16* gamma, const bf16* beta,
                                                             bf16* out, bf16* out_norm, bf16* xhat, float* rstd) {
  __shared__ float red[4];
  const long row = (long)blockIdx.x * d;
  const int nc = d / 8;
  const bool nt = stream_out((long)gridDim.x * d * 2);  // one row per workgroup
  // every load up front, none conditional on a lane or an operand: a chunk past the row
  // reads chunk 0, an absent operand reads x1 (gamma) instead, masked afterwards; so no
  // load waits for the one before it
  const bf16* x2p = x2 ? x2 : x1;
  const bf16* gp = gamma ? gamma : x1;
  const bf16* bp = (norm == Norm::LN && beta) ? beta : gp;
  bf16x8 r1[NORM_NPT], r2[NORM_NPT], rg[NORM_NPT], rb[NORM_NPT];
#pragma unroll
  for (int i = 0; i < NORM_NPT; ++i) {
    const int c = threadIdx.x + 256 * i, cc = c < nc ? c : 0;
    r1[i] = ld_frag(x1 + row + 8 * cc);
    r2[i] = ld_frag(x2p + row + 8 * cc);
    rg[i] = ld_frag(gp + 8 * cc);
    rb[i] = ld_frag(bp + 8 * cc);
  }
  float v[NORM_NPT][8];
#pragma unroll
  for (int i = 0; i < NORM_NPT; ++i) {
    float y[8];
    unpack_frag(r1[i], v[i]);
    unpack_frag(r2[i], y);
    if (x2)
#pragma unroll
      for (int q = 0; q < 8; ++q) v[i][q] += y[q];
  }
  if (norm == Norm::None || (norm == Norm::RMS && x2)) {
#pragma unroll
    for (int i = 0; i < NORM_NPT; ++i) {
      const int c = threadIdx.x + 256 * i;
      if (c < nc) st8f(out + row + 8 * c, v[i], nt);
    }
    if (norm == Norm::None) return;
  }
  float mean = 0.f;
  if (norm == Norm::LN) {
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < NORM_NPT; ++i)
      if (threadIdx.x + 256 * i < nc)
#pragma unroll
        for (int q = 0; q < 8; ++q) s += v[i][q];
    mean = block_sum256(s, red) / (float)d;
  }
  float s2 = 0.f;
#pragma unroll
  for (int i = 0; i < NORM_NPT; ++i)
    if (threadIdx.x + 256 * i < nc)
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const float c = v[i][q] - mean;
        s2 += c * c;
      }
  const float rs = rsqrtf(block_sum256(s2, red) / (float)d + eps);
  if (rstd && threadIdx.x == 0) rstd[blockIdx.x] = rs;
  bf16* dst = norm == Norm::LN ? out : out_norm;
#pragma unroll
  for (int i = 0; i < NORM_NPT; ++i) {
    const int c = threadIdx.x + 256 * i;
    if (c >= nc) continue;
    float xh[8], g[8], b[8], o[8];
    unpack_frag(rg[i], g);
    unpack_frag(rb[i], b);
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      xh[q] = (v[i][q] - mean) * rs;
      o[q] = xh[q] * g[q] + (norm == Norm::LN ? b[q] : 0.f);
    }
    st8f(dst + row + 8 * c, o, nt);
    if (xhat) st8f(xhat + row + 8 * c, xh, nt);
  }
}

// dz = [dres +] rstd (g*gin - [mean(g*gin)] - xhat mean(g*gin*xhat)), LN or RMS
__global__ __launch_bounds__(256) void norm_rows_bwd_bf16(int d, Norm norm, const bf16* gin, const bf16* xhat,
                                                             const float* rstd, const bf16* gamma,
                                                             const bf16* dres, bf16* dz) {
  __shared__ float red[4];
  const long row = (long)blockIdx.x * d;
  const int nc = d / 8;
  const bool nt = stream_out((long)gridDim.x * d * 2);
  float gg[NORM_NPT][8], xh[NORM_NPT][8];
  float s1 = 0.f, s2 = 0.f;
#pragma unroll
  for (int i = 0; i < NORM_NPT; ++i) {
    const int c = threadIdx.x + 256 * i;
    if (c >= nc) continue;
    float g[8];
    ld8f(gin + row + 8 * c, gg[i]);
    ld8f(xhat + row + 8 * c, xh[i]);
    ld8f(gamma + 8 * c, g);
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      gg[i][q] *= g[q];
      s1 += gg[i][q];
      s2 += gg[i][q] * xh[i][q];
    }
  }
  const float m1 = norm == Norm::LN ? block_sum256(s1, red) / (float)d : 0.f;
  const float m2 = block_sum256(s2, red) / (float)d, rs = rstd[blockIdx.x];
#pragma unroll
  for (int i = 0; i < NORM_NPT; ++i) {
    const int c = threadIdx.x + 256 * i;
    if (c >= nc) continue;
    float r[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f}, o[8];
    if (norm == Norm::RMS) ld8f(dres + row + 8 * c, r);
#pragma unroll
    for (int q = 0; q < 8; ++q) o[q] = r[q] + rs * (gg[i][q] - m1 - xh[i][q] * m2);
    st8f(dz + row + 8 * c, o, nt);
  }
}

static bool al16p(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

hipError_t launch_norm_rows_fwd(int T, int d, float eps, Norm norm, const void* x1, const void* x2, const void* gamma,
                                const void* beta, void* out, void* out_norm, void* xhat, float* rstd, hipStream_t s) {
  if (T < 0 || d <= 0 || d % 8 || d > 256 * 8 * NORM_NPT || !x1) return hipErrorInvalidValue;
  if (norm != Norm::None && !gamma) return hipErrorInvalidValue;
  if (norm == Norm::LN && (!beta || !out)) return hipErrorInvalidValue;
  if (norm == Norm::RMS && !out_norm) return hipErrorInvalidValue;
  if ((norm == Norm::None || (norm == Norm::RMS && x2)) && !out) return hipErrorInvalidValue;
  for (const void* p : {x1, x2, gamma, beta, static_cast<const void*>(out), static_cast<const void*>(out_norm),
                        static_cast<const void*>(xhat)})
    if (p && !al16p(p)) return hipErrorInvalidValue;
  if (T == 0) return hipSuccess;
  RG_LAUNCH(norm_rows_fwd_bf16, dim3(T), dim3(256), 0, s, d, eps, norm, static_cast<const bf16*>(x1),
            static_cast<const bf16*>(x2), static_cast<const bf16*>(gamma), static_cast<const bf16*>(beta),
            static_cast<bf16*>(out), static_cast<bf16*>(out_norm), static_cast<bf16*>(xhat), rstd);
  return hipGetLastError();
}

hipError_t launch_norm_rows_bwd(int T, int d, Norm norm, const void* gin, const void* xhat, const float* rstd,
                                const void* gamma, const void* dres, void* dz, hipStream_t s) {
  if (T < 0 || d <= 0 || d % 8 || d > 256 * 8 * NORM_NPT || norm == Norm::None) return hipErrorInvalidValue;
  if (!gin || !xhat || !rstd || !gamma || !dz || (norm == Norm::RMS && !dres)) return hipErrorInvalidValue;
  for (const void* p : {gin, xhat, gamma, dres, static_cast<const void*>(dz)})
    if (p && !al16p(p)) return hipErrorInvalidValue;
  if (T == 0) return hipSuccess;
  RG_LAUNCH(norm_rows_bwd_bf16, dim3(T), dim3(256), 0, s, d, norm, static_cast<const bf16*>(gin),
            static_cast<const bf16*>(xhat), rstd, static_cast<const bf16*>(gamma), static_cast<const bf16*>(dres),
            static_cast<bf16*>(dz));
  return hipGetLastError();
}

hipError_t launch_rms_fwd(int dtype, int T, int d, float eps, const void* x, const void* g, void* out,
                          void* xhat, float* rstd, hipStream_t s) {
  // bf16 only (the pre-RMS block has no fp32 stage); every bf16 width (d a
  // multiple of 256 up to 4096) and the stage's 16-B aligned buffers take the
  // vectorised row kernel
  if (T < 0 || d <= 0 || !x || !g || !out) return hipErrorInvalidValue;
  if (dtype != DT_BF16 || d % 8 || d > 256 * 8 * NORM_NPT || !al16p(x) || !al16p(g) || !al16p(out) ||
      (xhat && !al16p(xhat)))
    return hipErrorInvalidValue;
  if (T == 0) return hipSuccess;
  return launch_norm_rows_fwd(T, d, eps, Norm::RMS, x, nullptr, g, nullptr, nullptr, out, xhat, rstd, s);
}

hipError_t launch_rms_bwd(int dtype, int T, int d, const void* dn, const void* dres, const void* xhat,
                          const float* rstd, const void* g, void* dx, hipStream_t s) {
  // bf16 only, as the forward
  if (T < 0 || d <= 0 || !dn || !dres || !xhat || !rstd || !g || !dx) return hipErrorInvalidValue;
  if (dtype != DT_BF16 || d % 8 || d > 256 * 8 * NORM_NPT || !al16p(dn) || !al16p(dres) || !al16p(xhat) ||
      !al16p(g) || !al16p(dx))
    return hipErrorInvalidValue;
  if (T == 0) return hipSuccess;
  return launch_norm_rows_bwd(T, d, Norm::RMS, dn, xhat, rstd, g, dres, dx, s);
}

// ---------------------------------------------------------------- layouts
// out[c', r] = in[r, c] with c' = c, or, with perm_dh > 0, the per-head order
// of a [Q | K | V] column block: column p * (cols / 3) + h * perm_dh + i goes
// to row (3 h + p) * perm_dh + i.
__device__ __forceinline__ int perm_col(int c, int cols, int perm_dh) {
  if (perm_dh <= 0) return c;
  const int blk = cols / 3, p = c / blk, rem = c % blk, h = rem / perm_dh, i = rem % perm_dh;
  return (3 * h + p) * perm_dh + i;
}

template <typename Ti, typename To>
__global__ __launch_bounds__(256) void transpose_k(const Ti* in, int rows, int cols, To* out, int perm_dh) {
  __shared__ float tile[32][33];
  const int c0 = blockIdx.x * 32, r0 = blockIdx.y * 32, tx = threadIdx.x % 32, ty = threadIdx.x / 32;
  for (int i = ty; i < 32; i += 8) {
    const int r = r0 + i, c = c0 + tx;
    tile[i][tx] = (r < rows && c < cols) ? St<Ti>::ld(in, (long)r * cols + c) : 0.f;
  }
  __syncthreads();
  for (int i = ty; i < 32; i += 8) {
    const int c = c0 + i, r = r0 + tx;
    if (c < cols && r < rows) St<To>::st(out, (long)perm_col(c, cols, perm_dh) * rows + r, tile[tx][i]);
  }
}

hipError_t launch_transpose(int in_dtype, int out_dtype, const void* in, int rows, int cols, void* out,
                            hipStream_t s, int perm_dh) {
  if (!in || !out || rows <= 0 || cols <= 0) return hipErrorInvalidValue;
  if (perm_dh > 0 && (cols % 3 || (cols / 3) % perm_dh)) return hipErrorInvalidValue;
  const dim3 grid((cols + 31) / 32, (rows + 31) / 32), block(256);
  if (in_dtype == DT_F32 && out_dtype == DT_F32)
    RG_LAUNCH((transpose_k<float, float>), grid, block, 0, s, (const float*)in, rows, cols, (float*)out, perm_dh);
  else if (in_dtype == DT_BF16 && out_dtype == DT_BF16)
    RG_LAUNCH((transpose_k<bf16, bf16>), grid, block, 0, s, (const bf16*)in, rows, cols, (bf16*)out, perm_dh);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

template <typename T>
__global__ __launch_bounds__(256) void pack_swiglu_k(const T* wgu, int d, int F, T* out) {
  const long n = 2L * F * d;
  for (long idx = (long)blockIdx.x * blockDim.x + threadIdx.x; idx < n; idx += (long)gridDim.x * blockDim.x) {
    const int p = (int)(idx / d), i = (int)(idx % d);
    const int blk = p / 64, w = p % 64;
    const int col = w < 32 ? blk * 32 + w : F + blk * 32 + (w - 32);
    out[idx] = wgu[(long)i * 2 * F + col];
  }
}

hipError_t launch_pack_swiglu(int dtype, const void* w_gu, int d, int F, void* out, hipStream_t s) {
  if (!w_gu || !out || d <= 0 || F <= 0 || F % 32) return hipErrorInvalidValue;
  const dim3 grid(4096), block(256);
  if (dtype != DT_BF16) return hipErrorInvalidValue;  // the SwiGLU block has no fp32 stage
  RG_LAUNCH(pack_swiglu_k<bf16>, grid, block, 0, s, (const bf16*)w_gu, d, F, (bf16*)out);
  return hipGetLastError();
}

// ---------------------------------------------------------------- adapter update
// Element idx < d*m is W_down[i][j] (i = idx / m, j = idx % m); the rest is
// W_up[j][i].  Writes the working copies W, W^T in the stage dtype.  The
// slots of one launch travel by value (blockIdx.y selects one).
template <typename T, bool UPDATE>
__global__ __launch_bounds__(256) void adapter_update_k(AdapterSlotBatch batch, int d, int m, float lr) {
  const AdapterSlot& sl = batch.s[blockIdx.y];
  if (!sl.w_down) return;  // a block without this adapter (single placement)
  const long n = (long)d * m;
  for (long idx = (long)blockIdx.x * blockDim.x + threadIdx.x; idx < 2 * n; idx += (long)gridDim.x * blockDim.x) {
    if (idx < n) {
      const int i = (int)(idx / m), j = (int)(idx % m);
      float w = sl.w_down[idx];
      if (UPDATE) {
        w -= lr * sl.g_down[idx];
        sl.w_down[idx] = w;
        sl.g_down[idx] = 0.f;
      }
      if constexpr (std::is_same_v<T, float>) {
        St<T>::st(static_cast<T*>(sl.wdn), idx, w);
        St<T>::st(static_cast<T*>(sl.wdn_t), (long)j * d + i, w);
      } else {  // fragment-packed: W_down in layout B, W_down^T in layout A
        St<T>::st(static_cast<T*>(sl.wdn), pack_b_idx(i, j, d), w);
        St<T>::st(static_cast<T*>(sl.wdn_t), pack_a_idx(j, i, d), w);
      }
    } else {
      const long k = idx - n;
      const int j = (int)(k / d), i = (int)(k % d);
      float w = sl.w_up[k];
      if (UPDATE) {
        w -= lr * sl.g_up[k];
        sl.w_up[k] = w;
        sl.g_up[k] = 0.f;
      }
      if constexpr (std::is_same_v<T, float>) {
        St<T>::st(static_cast<T*>(sl.wup), k, w);
        St<T>::st(static_cast<T*>(sl.wup_t), (long)i * m + j, w);
      } else {  // W_up in layout A, W_up^T in layout B
        St<T>::st(static_cast<T*>(sl.wup), pack_a_idx(j, i, d), w);
        St<T>::st(static_cast<T*>(sl.wup_t), pack_b_idx(i, j, d), w);
      }
    }
  }
}

template <bool UPDATE>
static hipError_t adapter_update(int dtype, const AdapterSlot* slots, int n_slots, int d, int m, float lr,
                                 hipStream_t s) {
  if ((!slots && n_slots) || n_slots < 0 || d <= 0 || m <= 0) return hipErrorInvalidValue;
  const long n = 2L * d * m;
  const unsigned gx = (unsigned)((n + 255) / 256 < 256 ? (n + 255) / 256 : 256);
  for (int i0 = 0; i0 < n_slots; i0 += ADAPTER_SLOT_BATCH) {
    AdapterSlotBatch b{};
    const int k = n_slots - i0 < ADAPTER_SLOT_BATCH ? n_slots - i0 : ADAPTER_SLOT_BATCH;
    for (int i = 0; i < k; ++i) b.s[i] = slots[i0 + i];
    const dim3 grid(gx, k), block(256);
    if (dtype == DT_BF16) RG_LAUNCH((adapter_update_k<bf16, UPDATE>), grid, block, 0, s, b, d, m, lr);
    else RG_LAUNCH((adapter_update_k<float, UPDATE>), grid, block, 0, s, b, d, m, lr);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_adapter_sgd(int dtype, const AdapterSlot* slots, int n_slots, int d, int m, float lr,
                              hipStream_t s) {
  return adapter_update<true>(dtype, slots, n_slots, d, m, lr, s);
}
hipError_t launch_adapter_sync(int dtype, const AdapterSlot* slots, int n_slots, int d, int m,
                               hipStream_t s) {
  return adapter_update<false>(dtype, slots, n_slots, d, m, 0.f, s);
}

// ---------------------------------------------------------------- losses
template <typename T>
__global__ __launch_bounds__(1024) void mse_k(const T* y, const T* t, long n, T* dy, float* loss) {
  __shared__ float red[16];
  float s = 0.f;
  const float sc = 2.f / (float)n;
  for (long i = threadIdx.x; i < n; i += blockDim.x) {
    const float diff = St<T>::ld(y, i) - St<T>::ld(t, i);
    St<T>::st(dy, i, sc * diff);
    s += diff * diff;
  }
  s = blk_sum<T>(s, red);
  if (loss && threadIdx.x == 0) *loss = s / (float)n;
}

hipError_t launch_mse(int dtype, const void* y, const void* t, long n, void* dy, float* loss, hipStream_t s) {
  if (!y || !t || !dy || n <= 0) return hipErrorInvalidValue;
  if (dtype == DT_BF16) RG_LAUNCH(mse_k<bf16>, dim3(1), dim3(1024), 0, s, (const bf16*)y, (const bf16*)t, n, (bf16*)dy, loss);
  else RG_LAUNCH(mse_k<float>, dim3(1), dim3(1024), 0, s, (const float*)y, (const float*)t, n, (float*)dy, loss);
  return hipGetLastError();
}

// Initiator head (Alg. 1: the initiator computes the loss and updates the
// head): a linear layer on position 0 of each sequence, softmax
// cross-entropy, mean over the batch.  dy[b, 0, :] = dlogits W_h^T, zero at
// every other position; the head gradients and the loss are added into
// gwh / gbh / loss.
// Workgroup 0 does every sum, so that each result is one thread's sum over
// the samples in order: the same inputs give the same bits (atomic adds in
// arrival order would not).  Samples go in chunks of HEAD_CHUNK: one wave
// per sample for the logits, the softmax and the loss (into LDS), then one
// thread per feature (in blocks of HEAD_NT features) for the dY rows and the
// W_h gradient, thread c for the bias gradient of class c and thread 0 for
// the loss.  The other workgroups
// zero rows 1..S-1 of every sequence with 16-B stores.
constexpr int HEAD_C = 16;        // maximum number of classes
constexpr int HEAD_NT = 1024;     // threads per workgroup (16 waves)
constexpr int HEAD_CHUNK = 256;   // samples per pass of workgroup 0
template <typename T, int CN>  // CN: class count bound, compile time (the loops over classes unroll)
__global__ __launch_bounds__(HEAD_NT) void head_ce_k(const T* y, int B, int S, int d, const float* wh,
                                                     const float* bh, int C_, const int* labels, T* dy, float* gwh,
                                                     float* gbh, float* loss) {
  // the two-class instantiation runs only with C == 2: a compile-time class count leaves
  // no class guard around a load, so the loads of a row go out together
  const int C = CN == 2 ? 2 : C_;
  const bool nt = stream_out((long)B * S * d * (long)sizeof(T));  // dY streamed (common.h)
  if (blockIdx.x > 0) {
    const int nz = gridDim.x - 1, z = blockIdx.x - 1;
    const int vpr = d * (int)sizeof(T) / 16;  // 16-B vectors per row
    const long nvec = (long)B * (S - 1) * vpr;
    for (long v = (long)z * HEAD_NT + threadIdx.x; v < nvec; v += (long)nz * HEAD_NT) {
      const long rr = v / vpr;
      const long r = (rr / (S - 1)) * S + 1 + rr % (S - 1);
      st16(reinterpret_cast<uint4*>(dy + r * d) + v % vpr, zero_frag(), nt);
    }
    return;
  }
  constexpr int NW = HEAD_NT / 64;
  __shared__ float sdl[HEAD_CHUNK][CN];
  __shared__ float sls[HEAD_CHUNK];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, t = threadIdx.x;
  // logits, softmax and loss of samples b0 .. b0+nb-1 into sdl / sls, one wave each
  // samples per wave pass: two for the two-class head, so that both rows'
  // loads are in flight together (the second clamped); one for up to 16
  // classes, whose logits take the registers
  constexpr int PAIR = CN <= 4 ? 2 : 1;
  auto logits = [&](int b0, int nb) {
    for (int sm = wave; sm < nb; sm += PAIR * NW) {
      int smk[PAIR];
      const T* yr[PAIR];
#pragma unroll
      for (int k = 0; k < PAIR; ++k) {
        smk[k] = min(sm + k * NW, nb - 1);
        yr[k] = y + (long)(b0 + smk[k]) * S * d;
      }
      float lg[PAIR][CN];
#pragma unroll
      for (int k = 0; k < PAIR; ++k)
#pragma unroll
        for (int c = 0; c < CN; ++c) lg[k][c] = 0.f;
      for (int v = lane; v < d / 8; v += 64) {
        float yv[PAIR][8];
#pragma unroll
        for (int k = 0; k < PAIR; ++k) {
          if constexpr (std::is_same_v<T, bf16>) {
            unpack_frag(ld_frag(yr[k] + 8 * v), yv[k]);
          } else {
            const float4 q0 = reinterpret_cast<const float4*>(yr[k])[2 * v];
            const float4 q1 = reinterpret_cast<const float4*>(yr[k])[2 * v + 1];
            yv[k][0] = q0.x; yv[k][1] = q0.y; yv[k][2] = q0.z; yv[k][3] = q0.w;
            yv[k][4] = q1.x; yv[k][5] = q1.y; yv[k][6] = q1.z; yv[k][7] = q1.w;
          }
        }
        const float* wr = wh + (long)8 * v * C;
#pragma unroll
        for (int e = 0; e < 8; ++e)
#pragma unroll
          for (int c = 0; c < CN; ++c)
            if (c < C) {
              const float wc = wr[e * C + c];
#pragma unroll
              for (int k = 0; k < PAIR; ++k) lg[k][c] += yv[k][e] * wc;
            }
      }
#pragma unroll
      for (int k = 0; k < PAIR; ++k) {
        if (sm + k * NW >= nb) break;  // wave-uniform
        const int lab = labels[b0 + smk[k]];
        float mx = -INFINITY;
#pragma unroll
        for (int c = 0; c < CN; ++c)
          if (c < C) {
            lg[k][c] = wave_sum(lg[k][c]) + bh[c];
            mx = fmaxf(mx, lg[k][c]);
          }
        float se = 0.f, ll = 0.f;
#pragma unroll
        for (int c = 0; c < CN; ++c)
          if (c < C) {
            se += __expf(lg[k][c] - mx);
            if (c == lab) ll = lg[k][c];
          }
        if (lane == 0) {
          sls[smk[k]] = -(ll - mx - __logf(se)) / (float)B;
#pragma unroll
          for (int c = 0; c < CN; ++c)
            sdl[smk[k]][c] = c < C ? (__expf(lg[k][c] - mx) / se - (c == lab ? 1.f : 0.f)) / (float)B : 0.f;
        }
      }
    }
  };
  // A batch of at most HEAD_CHUNK samples has its logits formed once; larger
  // batches re-form each chunk's for every block of HEAD_NT features.
  const bool one_chunk = B <= HEAD_CHUNK;
  float bacc = 0.f, lacc = 0.f;
  for (int fb = 0; fb * HEAD_NT < d; ++fb) {
    const int i = t + fb * HEAD_NT;
    const bool iv = i < d;
    float wv[CN], gacc[CN];
#pragma unroll
    for (int c = 0; c < CN; ++c) {
      wv[c] = (iv && c < C) ? wh[(long)i * C + c] : 0.f;
      gacc[c] = 0.f;
    }
    for (int b0 = 0; b0 < B; b0 += HEAD_CHUNK) {
      const int nb = min(HEAD_CHUNK, B - b0);
      if (fb == 0 || !one_chunk) {  // the same for every thread
        logits(b0, nb);
        __syncthreads();
      }
      // dY row and the W_h gradient of feature i (thread = feature), the samples in
      // order; UNR samples' loads in flight at once (clamped, masked after)
      constexpr int UNR = CN <= 4 ? 8 : 4;
      if (iv)
        for (int sm0 = 0; sm0 < nb; sm0 += UNR) {
          float yv[UNR];
#pragma unroll
          for (int u = 0; u < UNR; ++u) yv[u] = St<T>::ld(y, (long)(b0 + min(sm0 + u, nb - 1)) * S * d + i);
#pragma unroll
          for (int u = 0; u < UNR; ++u) {
            const int sm = sm0 + u;
            if (sm >= nb) break;
            float g = 0.f;
#pragma unroll
            for (int c = 0; c < CN; ++c)
              if (c < C) {
                gacc[c] += yv[u] * sdl[sm][c];
                g += sdl[sm][c] * wv[c];
              }
            St<T>::st_nt(dy, (long)(b0 + sm) * S * d + i, g);
          }
        }
      if (fb == 0) {  // the bias gradient and the loss, once
        if (t < C)
          for (int sm = 0; sm < nb; ++sm) bacc += sdl[sm][t];
        if (t == 0)
          for (int sm = 0; sm < nb; ++sm) lacc += sls[sm];
      }
      if (!one_chunk) __syncthreads();  // the next chunk overwrites sdl / sls
    }
    if (iv) {
#pragma unroll
      for (int c = 0; c < CN; ++c)
        if (c < C) gwh[(long)i * C + c] += gacc[c];
    }
  }
  if (t < C) gbh[t] += bacc;
  if (t == 0 && loss) *loss += lacc;
}

hipError_t launch_head_ce(int dtype, const void* y, int B, int S, int d, const float* wh, const float* bh,
                          int C, const int* labels, void* dy, float* gwh, float* gbh, float* loss,
                          hipStream_t s) {
  if (!y || !wh || !bh || !labels || !dy || !gwh || !gbh || B <= 0 || S <= 0 || d <= 0 || C < 1 || C > HEAD_C)
    return hipErrorInvalidValue;
  const size_t es = dtype == DT_BF16 ? 2 : 4;
  // rows move as 16-B vectors: d a multiple of 8, y, dy and w_h 16-B aligned
  if (d % 8 || (d * es) % 16 ||
      (reinterpret_cast<uintptr_t>(dy) | reinterpret_cast<uintptr_t>(y) | reinterpret_cast<uintptr_t>(wh)) & 15u)
    return hipErrorInvalidValue;
  const long nvec = (long)B * (S - 1) * (long)(d * es / 16);
  const int nz = (int)std::min<long>(255, (nvec + HEAD_NT - 1) / HEAD_NT);
  const dim3 grid(1 + nz), block(HEAD_NT);
  if (dtype == DT_BF16) {
    if (C == 2)
      RG_LAUNCH((head_ce_k<bf16, 2>), grid, block, 0, s, (const bf16*)y, B, S, d, wh, bh, C, labels, (bf16*)dy,
                gwh, gbh, loss);
    else
      RG_LAUNCH((head_ce_k<bf16, HEAD_C>), grid, block, 0, s, (const bf16*)y, B, S, d, wh, bh, C, labels,
                (bf16*)dy, gwh, gbh, loss);
  } else {
    if (C == 2)
      RG_LAUNCH((head_ce_k<float, 2>), grid, block, 0, s, (const float*)y, B, S, d, wh, bh, C, labels, (float*)dy,
                gwh, gbh, loss);
    else
      RG_LAUNCH((head_ce_k<float, HEAD_C>), grid, block, 0, s, (const float*)y, B, S, d, wh, bh, C, labels,
                (float*)dy, gwh, gbh, loss);
  }
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void sgd_f32_k(float* w, float* g, long n, float lr) {
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x) {
    w[i] -= lr * g[i];
    g[i] = 0.f;
  }
}

hipError_t launch_sgd_f32(float* w, float* g, long n, float lr, hipStream_t s) {
  if (!w || !g || n <= 0) return hipErrorInvalidValue;
  const long nb = (n + 255) / 256;
  RG_LAUNCH(sgd_f32_k, dim3((unsigned)(nb < 1024 ? nb : 1024)), dim3(256), 0, s, w, g, n, lr);
  return hipGetLastError();
}

}  // namespace rg
