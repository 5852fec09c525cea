// Host-side launchers of the RingAda kernels (internal to libringada).
#pragma once
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rg {

// Optional timing of the next launches: when set (by the stage's profiling
// pass, never under graph capture), RG_LAUNCH goes through the HIP extension
// launch, which timestamps the kernel's own dispatch (start on the first
// launch, stop on every launch, so the pair spans all kernels of one call).
struct LaunchEvents {
  hipEvent_t start, stop;
  bool started;
};
extern thread_local LaunchEvents* g_launch_events;

#define RG_LAUNCH(K, G, B, SH, S, ...)                                                            \
  do {                                                                                            \
    if (::rg::LaunchEvents* le_ = ::rg::g_launch_events) {                                        \
      hipExtLaunchKernelGGL(K, G, B, SH, S, le_->started ? nullptr : le_->start, le_->stop, 0,    \
                            __VA_ARGS__);                                                         \
      le_->started = true;                                                                        \
    } else {                                                                                      \
      hipLaunchKernelGGL(K, G, B, SH, S, __VA_ARGS__);                                            \
    }                                                                                             \
  } while (0)

enum { DT_F32 = 0, DT_BF16 = 1 };

// ---------------------------------------------------------------- GEMM
// C[M, N] = A[M, K] * B[N, K]^T followed by an epilogue.  Both operands are
// K-contiguous (row strides lda, ldb in elements).
enum class Epi {
  Store,    // out = acc (+ bias[n])
  Gelu,     // pre = acc (+ bias[n]); out2 = pre (if non-null); out = gelu(pre)
  Resid,    // out = acc + aux[m, n]
  DGelu,    // out = acc * gelu'(aux[m, n])
  SwiGlu,   // B rows packed [gate 32 | up 32] per 64; out[m, f] = silu(gate) * up,
            // out2[m, f] = gate, out2[m, half + f] = up (if non-null)
  DSwiGlu,  // acc = d(act)[m, f]; aux = [gate | up]; out[m, f] = d gate,
            // out[m, half + f] = d up
  Rope,     // bf16 QKV projection, no bias: out = acc with the rotary embedding
            // applied to columns < rope_cols (Q and K, heads of rope_dh
            // columns; row m is position m % rope_S)
  Attn,     // bf16 QKV projection with B rows in per-head order [Q_h K_h V_h]
            // (d_head 64) and M = sequences of 128 tokens: pre = acc + bias;
            // out = pre (if non-null); out2[:, 64h..64h+63] = softmax(Q_h K_h^T / 8) V_h
            // per sequence; lse[(seq * H + h) * 128 + query] (base 2, scaled scores)
};

struct GemmArgs {
  const void* A; int lda;
  const void* B; int ldb;
  int M, N, K;
  const void* bias;
  const void* aux; int ld_aux;
  void* out; int ldo;
  void* out2; int ldo2;
  int half;
  float* lse;  // Attn only
  // Rope only: (cos, sin) of pos * theta^(-2i/dh), [positions][rope_dh / 2]
  const float2* rope_tab;
  int rope_S, rope_dh, rope_cols;
  int nt;  // set by launch_gemm: outputs stored with the non-temporal hint
};

// Names of the GEMM call sites (each gets its own kernel symbol).
enum Role {
  R_QKV_FWD, R_O_FWD, R_FFN_IN_FWD, R_FFN_OUT_FWD,
  R_QKV_DX, R_O_DX, R_FFN_IN_DX, R_FFN_OUT_DX, N_ROLES
};
const char* role_name(Role r);

// Returns hipErrorInvalidValue if the shapes or alignments do not fit the
// kernel (checked on the host before any launch).
hipError_t launch_gemm(int dtype, Role role, Epi epi, const GemmArgs& a, hipStream_t s);

// ---------------------------------------------------------------- attention
struct AttnArgs {
  int B, S, H, dh;
  int causal, rope;
  int rope_in_qkv;              // bf16, rope: Q and K in qkv are already rotated (no rotation on
                                // load); dQ and dK are still rotated back on output
  float theta;
  const float2* rope_tab;       // rope: (cos, sin) of pos * theta^(-2i/dh), [rope_rows][dh/2]
  int rope_rows;                // positions the table covers (>= S)
  const void* qkv; int ld_qkv;  // [B*S, ld]: Q, K, V of every head
  // columns of head h in qkv: Q at h * qkv_hs, K at qkv_ko + h * qkv_hs, V at
  // qkv_vo + h * qkv_hs.  All zero: three blocks of d columns (Q | K | V),
  // i.e. (dh, d, 2d); (3 dh, dh, 2 dh) is the per-head order [Q_h K_h V_h]
  // (bf16 only).  dqkv is always in the three-block order.
  int qkv_hs, qkv_ko, qkv_vo;
  void* o; int ld_o;            // [B*S, d]
  float* lse;                   // [B, H, S]
  // backward
  const void* dout; int ld_do;  // dO [B*S, d]
  float* dsum;                  // D = rowsum(dO * O) [B, H, S] (written by dq pass)
  void* dqkv; int ld_dqkv;      // [B*S, 3d]
};
hipError_t launch_attn_fwd(int dtype, const AttnArgs& a, hipStream_t s);
hipError_t launch_attn_bwd(int dtype, const AttnArgs& a, hipStream_t s);

// ---------------------------------------------------------------- adapters (Eq. (1)) fused with the residual add and the norm
enum class Norm { LN, RMS, None };
struct AdapterFwdArgs {
  int T, d, m;
  Norm norm;
  float eps;
  const void* z;      // adapter input [T, d]
  const void* res;    // residual [T, d]
  const void* wdn_t;  // W_down^T [m, d] (stage dtype)
  const void* wup_t;  // W_up^T   [d, m]
  const void* gamma;  // [d]
  const void* beta;   // [d] (LN)
  void* out;          // LN: LN(res + adapter(z)); RMS: h = res + adapter(z); None: same
  void* out_norm;     // RMS: h_norm = RMSNorm(h) * gamma
  void* u;            // stash of z W_down [T, m] (may be null)
  void* xhat;         // stash of the normalised input [T, d] (may be null)
  float* rstd;        // stash [T] (may be null)
  float* part;        // bf16 with d > 1024: fp32 scratch [d / 1024][T][m] for the
                      // split-K partial sums of z W_down; unused otherwise
};
hipError_t launch_adapter_fwd(int dtype, const AdapterFwdArgs& a, hipStream_t s);

struct AdapterBwdArgs {
  int T, d, m;
  Norm norm;          // LN: gin is the LN-output gradient; RMS: gin is the
                      // gradient at the RMSNorm output and dres is added;
                      // None: gin is the adapter-output gradient
  const void* gin;    // [T, d]
  const void* dres;   // [T, d] (RMS only)
  const void* xhat;   // [T, d]
  const float* rstd;  // [T]
  const void* gamma;  // [d]
  const void* u;      // stash z W_down [T, m]
  const void* wup;    // W_up [m, d]
  const void* wdn;    // W_down [d, m]
  void* dz;           // gradient at the adapter output [T, d]; may be null for
                      // Norm::None (it equals gin)
  void* du;           // gradient at z W_down [T, m] (always written)
  void* gu;           // gelu(U) [T, m] as bf16, the weight-gradient operand of
                      // W_up; null = not formed (adapter_bwd_forms_gelu says
                      // which shapes can form it)
  void* dzin;         // gradient at the adapter input [T, d]; null = skip
  float* part;        // bf16 with d > 1024: fp32 scratch [d / 1024][T][m] for the
                      // split-K partial sums of dZ W_up^T; unused otherwise
};
// fp32 elements of the scratch `part` needs (0 when the shape takes none)
long adapter_part_elems(int dtype, int T, int d, int m);
hipError_t launch_adapter_bwd(int dtype, const AdapterBwdArgs& a, hipStream_t s);

// dW_up[m, d] += gelu(U)^T dZ ; dW_down[d, m] += Z^T dU   (fp32 accumulators)
struct AdapterDwArgs {
  int T, d, m;
  const void* u;   // [T, m]
  const void* dz;  // [T, d]
  const void* z;   // [T, d]
  const void* du;  // [T, m]
  float* g_up;     // [m, d]
  float* g_down;   // [d, m]
  const void* gu;  // gelu(U) [T, m] when the adapter backward formed it, else
                   // null (then formed here from u)
};
// whether launch_adapter_bwd can also write gelu(U) (AdapterBwdArgs::gu) for
// this storage type and width: bf16 up to d = 1024
bool adapter_bwd_forms_gelu(int dtype, int d);
// bytes of the fp32 per-chunk partial sums launch_adapter_dw_batch needs for
// n adapters (0 for fp32 stages)
long adapter_dw_part_bytes(int dtype, int T, int d, int m, int n_adapters);
// n adapters' weight gradients (same T, d, m), added into g_up / g_down in as
// few launches as possible; bf16: per-chunk partial sums in `part` (16-B
// aligned, adapter_dw_part_bytes), then a fixed-order reduction, so the result
// is bitwise reproducible; g_up / g_down 16-B aligned
hipError_t launch_adapter_dw_batch(int dtype, const AdapterDwArgs* a, int n, float* part, long part_bytes,
                                   hipStream_t s);

// ---------------------------------------------------------------- row kernels
// out = RMSNorm(x) * g, xhat/rstd stashes optional; bf16 rows (the
// vectorised row kernel: d % 8 == 0, d <= 4096, 16-B aligned), else refused
hipError_t launch_rms_fwd(int dtype, int T, int d, float eps, const void* x, const void* g,
                          void* out, void* xhat, float* rstd, hipStream_t s);
// bf16 rows, d % 8 == 0, d <= 4096, 16-B aligned rows: h = x1 (+ x2);
// LN: out = LN(h) gamma + beta (out may alias x1); RMS: out = h when x2 is
// given, out_norm = RMSNorm(h) gamma; None: out = h.  xhat / rstd stashed when
// non-null.
hipError_t launch_norm_rows_fwd(int T, int d, float eps, Norm norm, const void* x1, const void* x2,
                                const void* gamma, const void* beta, void* out, void* out_norm, void* xhat,
                                float* rstd, hipStream_t s);
// dz = [dres +] rstd (gamma gin - [mean(gamma gin)] - xhat mean(gamma gin xhat)), LN or RMS
hipError_t launch_norm_rows_bwd(int T, int d, Norm norm, const void* gin, const void* xhat, const float* rstd,
                                const void* gamma, const void* dres, void* dz, hipStream_t s);
// dx = dres + RMSNorm'(dn); bf16 rows as launch_rms_fwd
hipError_t launch_rms_bwd(int dtype, int T, int d, const void* dn, const void* dres,
                          const void* xhat, const float* rstd, const void* g, void* dx,
                          hipStream_t s);

// ---------------------------------------------------------------- parameters
// out[c, r] = in[r, c] (rows x cols), both fp32 or both bf16; with
// perm_dh > 0 the columns of a [Q | K | V] block (cols = 3 d) come out in
// per-head order: column p d + h perm_dh + i becomes row (3 h + p) perm_dh + i
hipError_t launch_transpose(int in_dtype, int out_dtype, const void* in, int rows, int cols,
                            void* out, hipStream_t s, int perm_dh = 0);
// pack W_gu [d, 2F] into B rows for the SwiGlu epilogue: row p of the result
// (2F x d) is gate column (p/64)*32 + p%32 if p%64 < 32, else the matching up column;
// bf16 only
hipError_t launch_pack_swiglu(int dtype, const void* w_gu, int d, int F, void* out, hipStream_t s);

struct AdapterSlot {  // one adapter for the update kernel
  float* w_down; float* w_up; float* g_down; float* g_up;
  void* wdn; void* wdn_t; void* wup; void* wup_t;  // working copies
};
constexpr int ADAPTER_SLOT_BATCH = 16;  // slots passed by value per launch
struct AdapterSlotBatch {
  AdapterSlot s[ADAPTER_SLOT_BATCH];
};
// SGD on n_slots adapters (a host array; launched in batches of
// ADAPTER_SLOT_BATCH), zero grads, refresh working copies
hipError_t launch_adapter_sgd(int dtype, const AdapterSlot* slots, int n_slots, int d, int m,
                              float lr, hipStream_t s);
// refresh working copies only
hipError_t launch_adapter_sync(int dtype, const AdapterSlot* slots, int n_slots, int d, int m,
                               hipStream_t s);

// ---------------------------------------------------------------- losses
hipError_t launch_mse(int dtype, const void* y, const void* t, long n, void* dy, float* loss,
                      hipStream_t s);
hipError_t launch_head_ce(int dtype, const void* y, int B, int S, int d, const float* wh,
                          const float* bh, int C, const int* labels, void* dy, float* gwh,
                          float* gbh, float* loss, hipStream_t s);
hipError_t launch_sgd_f32(float* w, float* g, long n, float lr, hipStream_t s);

}  // namespace rg
