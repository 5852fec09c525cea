// Stage runtime behind the C ABI of include/ringada.h: argument validation,
// the one-forward-one-backward state machine, the stash planner and the
// block schedule of the forward / early-stopped backward.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <cmath>
#include <limits>
#include <string>
#include <vector>

#include "kernels.h"
#include "ringada.h"

using namespace rg;

// ================================================================ errors
static thread_local std::string g_err;

static ringada_status fail(ringada_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

#define RG_HIP(x)                                                                              \
  do {                                                                                         \
    hipError_t e_ = (x);                                                                       \
    if (e_ != hipSuccess)                                                                      \
      return fail(RINGADA_E_HIP, "%s failed: %s", #x, hipGetErrorString(e_));                  \
  } while (0)

#define RG_TRY(x)                                                                              \
  do {                                                                                         \
    ringada_status s_ = (x);                                                                   \
    if (s_ != RINGADA_OK) return s_;                                                           \
  } while (0)

extern "C" const char* ringada_last_error(void) { return g_err.c_str(); }

// ================================================================ planner
// Offsets (bytes) of every buffer inside the stash and scratch workspaces.
// NONE marks a tensor that the block does not keep.
static const size_t NONE = std::numeric_limits<size_t>::max();

enum Kind { K_NONE = 0, K_CUT = 1, K_FULL = 2 };

struct BlockStash {
  int kind;
  // post-LN: qkv o lse attn u1 xhat1 rstd1 a1 f2 u2 xhat2 rstd2
  // pre-RMS: xhat1 rstd1 qkv o lse attn u1 xhat2 rstd2 gu f u2   (a1 = gu, f2 = f)
  size_t qkv, o, lse, attn, u1, xhat1, rstd1, a1, f2, u2, xhat2, rstd2;
};

struct Layout {
  int B, S, c;
  size_t stash_bytes, scratch_bytes;
  std::vector<BlockStash> blk;
  // forward scratch
  size_t act[2], h1, n1, n2, qkv, o, lse, attn, g, f2;
  // backward scratch (aliases the forward scratch: dead after the forward)
  size_t dact[2], df2, da1, dh1, dz1, dattn, dout, dqkv, dsum, dn1;
  // per adapter in the backward, [2 l + a] (a = 0 attention, 1 FFN): the
  // gradients at its output (dz) and at z W_down (du), kept until the one
  // weight-gradient launch at the end of the backward
  std::vector<size_t> gdz, gdu;
  // and gelu(U), the W_up weight-gradient operand, where the adapter backward
  // forms it (bf16 up to d = 1024; else NONE and the weight-gradient launch
  // forms it from the stashed U)
  std::vector<size_t> ggu;
  size_t adp;  // both passes
  // per-chunk partial sums of the weight-gradient launch at the end of the
  // backward; they take the place of the backward's temporaries, all dead by
  // then, when those span enough bytes
  size_t dwp, dwp_bytes;
};

static size_t al256(size_t n) { return (n + 255) & ~(size_t)255; }

static int norm_cut(int c, int L) { return c < 0 ? -1 : (c > L ? L : c); }

static int block_kind(int l, int c, int L) {
  if (c >= L) return K_NONE;
  if (l > c) return K_FULL;
  if (l == c) return K_CUT;
  return K_NONE;
}

static void plan_layout(const ringada_stage_desc& D, int B, int S, int c, Layout& L) {
  const size_t es = D.dtype == RINGADA_BF16 ? 2 : 4;
  const size_t T = (size_t)B * S, d = D.d_model, F = D.d_ffn, m = D.d_adapter, H = D.n_heads;
  const bool llama = D.arch == RINGADA_ARCH_PRERMS_SWIGLU;
  const size_t Td = al256(T * d * es), T3d = al256(T * 3 * d * es), Tm = al256(T * m * es);
  const size_t TF = al256(T * F * es), T2F = al256(T * 2 * F * es);
  const size_t rows = al256(T * 4), lse = al256((size_t)B * H * S * 4);
  L.B = B;
  L.S = S;
  L.c = c;
  L.blk.assign(D.n_blocks, BlockStash{});
  size_t cur = 0;
  auto take = [&](size_t n) { size_t o = cur; cur += n; return o; };
  const bool single = D.placement == RINGADA_PLACEMENT_FFN;
  for (int l = 0; l < D.n_blocks; ++l) {
    BlockStash& b = L.blk[l];
    b = BlockStash{block_kind(l, c, D.n_blocks), NONE, NONE, NONE, NONE, NONE, NONE,
                   NONE, NONE, NONE, NONE, NONE, NONE};
    if (b.kind == K_NONE) continue;
    const bool full = b.kind == K_FULL;
    if (single && !full) {
      // the cut-off block stops after its FFN adapter: only that adapter's
      // operands (and, post-LN, the LN2 backward that feeds it)
      b.f2 = take(Td);
      b.u2 = take(Tm);
      if (!llama) { b.xhat2 = take(Td); b.rstd2 = take(rows); }
      continue;
    }
    if (full) {
      if (llama) { b.xhat1 = take(Td); b.rstd1 = take(rows); }
      b.qkv = take(T3d);
      b.o = take(Td);
      b.lse = take(lse);
    }
    if (!single) {  // the attention adapter's operands
      b.attn = take(Td);
      b.u1 = take(Tm);
    }
    if (!llama) { b.xhat1 = take(Td); b.rstd1 = take(rows); }
    if (llama) { b.xhat2 = take(Td); b.rstd2 = take(rows); }
    b.a1 = take(llama ? T2F : TF);
    b.f2 = take(Td);
    b.u2 = take(Tm);
    if (!llama) { b.xhat2 = take(Td); b.rstd2 = take(rows); }
  }
  L.stash_bytes = cur;

  cur = 0;  // forward scratch
  L.act[0] = take(Td);
  L.act[1] = take(Td);
  L.h1 = take(Td);
  L.n1 = llama ? take(Td) : NONE;
  L.n2 = llama ? take(Td) : NONE;
  L.qkv = take(T3d);
  L.o = take(Td);
  L.lse = take(lse);
  L.attn = take(Td);
  L.g = take(TF);
  L.f2 = take(Td);
  const size_t fwd = cur;
  cur = 0;  // backward scratch
  L.dact[0] = take(Td);
  L.dact[1] = take(Td);
  L.df2 = take(Td);
  L.da1 = take(llama ? T2F : TF);
  L.dh1 = take(Td);
  L.dz1 = take(Td);
  L.dattn = take(Td);
  L.dout = take(Td);
  L.dqkv = take(T3d);
  L.dsum = take(lse);
  L.dn1 = llama ? take(Td) : NONE;
  const size_t temporaries = cur;
  L.gdz.assign(2 * D.n_blocks, NONE);
  L.gdu.assign(2 * D.n_blocks, NONE);
  L.ggu.assign(2 * D.n_blocks, NONE);
  const bool form_gelu = adapter_bwd_forms_gelu(D.dtype == RINGADA_BF16 ? DT_BF16 : DT_F32, (int)d);
  int n_dw = 0;
  for (int l = 0; l < D.n_blocks; ++l) {
    if (block_kind(l, c, D.n_blocks) == K_NONE) continue;
    for (int a = single ? 1 : 0; a < 2; ++a) {
      L.gdz[2 * l + a] = take(Td);
      L.gdu[2 * l + a] = take(Tm);
      if (form_gelu) L.ggu[2 * l + a] = take(Tm);
      ++n_dw;
    }
  }
  L.dwp_bytes = al256((size_t)adapter_dw_part_bytes(D.dtype, (int)T, (int)d, (int)m, n_dw));
  L.dwp = L.dwp_bytes == 0 ? NONE : (L.dwp_bytes <= temporaries ? 0 : take(L.dwp_bytes));
  // split-K partials of the wide (d > 1024) adapter kernels, used inside one
  // adapter call in either pass: after both lists
  const long part = adapter_part_elems(D.dtype, (int)T, (int)d, (int)m);
  cur = std::max(fwd, cur);
  L.adp = part > 0 ? take(al256((size_t)part * 4)) : NONE;
  L.scratch_bytes = cur;
}

static ringada_status check_desc(const ringada_stage_desc* D) {
  if (!D) return fail(RINGADA_E_INVALID, "desc is NULL");
  if (D->arch != RINGADA_ARCH_POSTLN_GELU && D->arch != RINGADA_ARCH_PRERMS_SWIGLU)
    return fail(RINGADA_E_INVALID, "unknown arch %d", D->arch);
  if (D->dtype != RINGADA_F32 && D->dtype != RINGADA_BF16)
    return fail(RINGADA_E_INVALID, "unknown dtype %d", D->dtype);
  if (D->n_blocks < 1 || D->d_model < 1 || D->n_heads < 1 || D->d_ffn < 1 || D->d_adapter < 1 ||
      D->max_batch < 1 || D->max_seq < 1)
    return fail(RINGADA_E_INVALID, "sizes must be positive");
  if (D->d_model % D->n_heads) return fail(RINGADA_E_INVALID, "d_model %% n_heads != 0");
  if (D->placement != RINGADA_PLACEMENT_HOULSBY && D->placement != RINGADA_PLACEMENT_FFN)
    return fail(RINGADA_E_INVALID, "unknown placement %d", D->placement);
  const int dh = D->d_model / D->n_heads;
  if (!(D->norm_eps >= 0.f)) return fail(RINGADA_E_INVALID, "norm_eps must be >= 0");
  if (D->arch == RINGADA_ARCH_PRERMS_SWIGLU && !(D->rope_theta > 0.f))
    return fail(RINGADA_E_INVALID, "rope_theta must be > 0");
  if (D->dtype == RINGADA_BF16) {
    if (D->d_model % 256 || D->d_model > 4096 || (D->d_model > 1024 && D->d_model % 1024))
      return fail(RINGADA_E_UNSUPPORTED, "bf16 path: d_model must be a multiple of 256 up to 1024, "
                                         "or of 1024 up to 4096 (got %d)", D->d_model);
    if (dh != 64 && dh != 128)
      return fail(RINGADA_E_UNSUPPORTED, "bf16 path: head dim must be 64 or 128 (got %d)", dh);
    if (D->d_ffn % 64) return fail(RINGADA_E_UNSUPPORTED, "bf16 path: d_ffn must be a multiple of 64");
    if (D->d_adapter != 64) return fail(RINGADA_E_UNSUPPORTED, "bf16 path: d_adapter must be 64");
  } else {
    if (D->arch != RINGADA_ARCH_POSTLN_GELU)
      return fail(RINGADA_E_UNSUPPORTED, "f32 path: only the post-LN arch is built");
    if (D->d_model % 4 || D->d_ffn % 4 || D->d_adapter % 4 || dh > 128 || dh % 2)
      return fail(RINGADA_E_UNSUPPORTED, "f32 path: d_model, d_ffn, d_adapter multiples of 4, "
                                         "head dim even and <= 128");
    if (2 * (size_t)D->d_model + D->d_adapter + 8 > 16384)
      return fail(RINGADA_E_UNSUPPORTED, "f32 path: d_model too large");
    if (D->max_seq > 4096) return fail(RINGADA_E_UNSUPPORTED, "f32 path: seq <= 4096");
  }
  const double T = (double)D->max_batch * D->max_seq;
  if (T * 3.0 * D->d_model > 2e9 || T * 2.0 * D->d_ffn > 2e9)
    return fail(RINGADA_E_UNSUPPORTED, "activation tensors above 2^31 elements");
  return RINGADA_OK;
}

extern "C" ringada_status ringada_stage_plan(const ringada_stage_desc* desc, int32_t batch, int32_t seq,
                                             int32_t lowest_unfrozen, size_t* stash_bytes,
                                             size_t* scratch_bytes) {
  RG_TRY(check_desc(desc));
  if (batch < 1 || seq < 1 || batch > desc->max_batch || seq > desc->max_seq)
    return fail(RINGADA_E_INVALID, "batch %d / seq %d outside [1, max]", batch, seq);
  Layout L;
  plan_layout(*desc, batch, seq, norm_cut(lowest_unfrozen, desc->n_blocks), L);
  if (stash_bytes) *stash_bytes = L.stash_bytes;
  if (scratch_bytes) *scratch_bytes = L.scratch_bytes;
  return RINGADA_OK;
}

extern "C" int32_t ringada_local_cutoff(int32_t n_tm, int32_t depth, int32_t first_block, int32_t n_local) {
  if (n_tm < 1 || depth < 0 || depth > n_tm || first_block < 0 || n_local < 1 || first_block + n_local > n_tm)
    return std::numeric_limits<int32_t>::min();
  // 0-indexed global block whose attention adapter ends the backward
  const int32_t g = n_tm - depth;
  if (g < first_block) return -1;
  if (g >= first_block + n_local) return n_local;
  return g - first_block;
}

// ================================================================ weight memory
// The library's own copies of what it derives from the frozen weights and
// the adapters live in caller memory: one region per block, one per stage.
// Offsets are 256-B aligned relative to the region's base.
struct WeightLayout {
  size_t qkv, bqkv, o, in, out;  // transposed projections (+ the per-head-order bias)
  size_t wk[2][4];               // adapter working copies: W_down, W_down^T, W_up, W_up^T
  size_t block_bytes;
  size_t rope, stage_bytes;      // rotary (cos, sin) table
};

static bool per_head_qkv(const ringada_stage_desc& D) {
  return D.dtype == RINGADA_BF16 && D.arch == RINGADA_ARCH_POSTLN_GELU && D.d_model == 64 * D.n_heads;
}

static void plan_weights(const ringada_stage_desc& D, WeightLayout& W) {
  const size_t es = D.dtype == RINGADA_BF16 ? 2 : 4;
  const size_t d = D.d_model, F = D.d_ffn, m = D.d_adapter;
  const bool post = D.arch == RINGADA_ARCH_POSTLN_GELU, single = D.placement == RINGADA_PLACEMENT_FFN;
  size_t cur = 0;
  auto take = [&](size_t n) { size_t o = cur; cur += al256(n); return o; };
  W.qkv = take(3 * d * d * es);
  W.bqkv = per_head_qkv(D) ? take(3 * d * es) : NONE;
  W.o = take(d * d * es);
  W.in = take((post ? 1 : 2) * F * d * es);
  W.out = take(d * F * es);
  for (int a = 0; a < 2; ++a)
    for (int k = 0; k < 4; ++k) W.wk[a][k] = (single && a == 0) ? NONE : take(d * m * es);
  W.block_bytes = cur;
  W.rope = post ? NONE : 0;
  W.stage_bytes = post ? 0 : al256((size_t)D.max_seq * (d / D.n_heads / 2) * sizeof(float2));
}

extern "C" ringada_status ringada_stage_plan_weights(const ringada_stage_desc* desc, size_t* block_bytes,
                                                     size_t* stage_bytes) {
  RG_TRY(check_desc(desc));
  WeightLayout W;
  plan_weights(*desc, W);
  if (block_bytes) *block_bytes = W.block_bytes;
  if (stage_bytes) *stage_bytes = W.stage_bytes;
  return RINGADA_OK;
}

// ================================================================ handle
struct BlockBind {
  bool bound = false;
  ringada_block_weights w{};
  void* wt_qkv = nullptr;  // [3d, d]; rows in per-head order [Q_h K_h V_h] when the stage fuses attention
  void* bqkv = nullptr;    // b_qkv in that per-head order (else unused)
  void* wt_o = nullptr;    // [d, d]
  void* wt_in = nullptr;   // post-LN [F, d]; pre-RMS packed [2F, d]
  void* wt_out = nullptr;  // [d, F]
  ringada_adapter ad[2]{};
  void* wk[2][4] = {};     // working copies: W_down [d,m], W_down^T, W_up [m,d], W_up^T
};

struct ProfRec {
  const char* name;
  double flops, bytes;
  hipEvent_t e0, e1;
};

struct ringada_stage {
  ringada_stage_desc D{};
  int device = 0;
  WeightLayout WL{};
  std::vector<BlockBind> blocks;
  char* stage_mem = nullptr;   // caller's per-stage region
  float2* rope_tab = nullptr;  // rotary (cos, sin) [max_seq][d_head/2] in stage_mem, built at the first bind
  bool rope_built = false;
  // bf16 post-LN stages with d_head 64 keep Q, K, V in per-head column order
  // [Q_h K_h V_h] (projection weight rows and bias permuted at bind): a
  // 128x192 tile of the QKV projection is then one head of one sequence, and
  // 128-token sequences take the attention in that GEMM's epilogue
  bool qkv_per_head = false;
  // weight-gradient work of the adapters back-propagated so far in this
  // backward, launched together when it ends
  std::vector<AdapterDwArgs> dw_pending;
  std::vector<AdapterSlot> slots;  // [2 l + a], passed to the update kernel by value
  // state machine
  bool pending = false;
  Layout L;
  char* stash = nullptr;
  char* scratch = nullptr;
  // profiling
  bool prof = false;
  std::vector<ProfRec> recs;
  std::vector<hipEvent_t> evpool;
  size_t evused = 0;
};

extern "C" ringada_status ringada_stage_create(const ringada_stage_desc* desc, void* stage_mem,
                                               size_t stage_mem_bytes, ringada_stage** out) {
  if (!out) return fail(RINGADA_E_INVALID, "out is NULL");
  *out = nullptr;
  RG_TRY(check_desc(desc));
  WeightLayout W;
  plan_weights(*desc, W);
  if (stage_mem_bytes < W.stage_bytes || (W.stage_bytes && !stage_mem))
    return fail(RINGADA_E_WORKSPACE, "stage memory of %zu bytes, the stage needs %zu", stage_mem_bytes,
                W.stage_bytes);
  if (reinterpret_cast<uintptr_t>(stage_mem) & 255u)
    return fail(RINGADA_E_INVALID, "stage memory must be 256-byte aligned");
  ringada_stage* st = new ringada_stage();
  st->D = *desc;
  st->WL = W;
  st->qkv_per_head = per_head_qkv(*desc);
  st->blocks.resize(desc->n_blocks);
  st->slots.assign(2 * desc->n_blocks, AdapterSlot{});
  st->stage_mem = static_cast<char*>(stage_mem);
  if (W.rope != NONE) st->rope_tab = reinterpret_cast<float2*>(st->stage_mem + W.rope);
  if (hipGetDevice(&st->device) != hipSuccess) st->device = 0;
  *out = st;
  return RINGADA_OK;
}

extern "C" void ringada_stage_destroy(ringada_stage* st) {
  if (!st) return;
  for (hipEvent_t e : st->evpool) (void)hipEventDestroy(e);
  delete st;
}

extern "C" ringada_status ringada_stage_bind_block(ringada_stage* st, int32_t block,
                                                   const ringada_block_weights* w,
                                                   const ringada_adapter* attn, const ringada_adapter* ffn,
                                                   void* block_mem, size_t block_mem_bytes, void* stream) {
  if (!st || !w || !ffn) return fail(RINGADA_E_INVALID, "NULL argument");
  const ringada_stage_desc& D = st->D;
  const bool single = D.placement == RINGADA_PLACEMENT_FFN;
  if (single != (attn == nullptr))
    return fail(RINGADA_E_INVALID, single ? "the single placement takes no attention adapter"
                                          : "missing attention adapter");
  if (block < 0 || block >= D.n_blocks) return fail(RINGADA_E_INVALID, "block %d out of range", block);
  if (!block_mem || block_mem_bytes < st->WL.block_bytes)
    return fail(RINGADA_E_WORKSPACE, "block memory of %zu bytes, a block needs %zu", block_mem_bytes,
                st->WL.block_bytes);
  if (reinterpret_cast<uintptr_t>(block_mem) & 255u)
    return fail(RINGADA_E_INVALID, "block memory must be 256-byte aligned");
  const bool post = D.arch == RINGADA_ARCH_POSTLN_GELU;
  if (!w->w_qkv || !w->w_o || !w->norm1_g || !w->w_in || !w->w_out || !w->norm2_g)
    return fail(RINGADA_E_INVALID, "missing frozen weight");
  const bool has_post = w->b_qkv && w->b_o && w->norm1_b && w->b_in && w->b_out && w->norm2_b;
  const bool any_post = w->b_qkv || w->b_o || w->norm1_b || w->b_in || w->b_out || w->norm2_b;
  for (const void* q : {w->norm1_g, w->norm1_b, w->norm2_g, w->norm2_b})
    if (reinterpret_cast<uintptr_t>(q) & 15u)
      return fail(RINGADA_E_INVALID, "norm gains and shifts must be 16-byte aligned");
  if (post && !has_post) return fail(RINGADA_E_INVALID, "post-LN block needs every bias and beta");
  if (!post && any_post) return fail(RINGADA_E_INVALID, "pre-RMS block takes no bias or beta");
  for (const ringada_adapter* a : {attn, ffn}) {
    if (a && (!a->w_down || !a->w_up || !a->g_down || !a->g_up))
      return fail(RINGADA_E_INVALID, "missing adapter tensor");
    if (a && ((reinterpret_cast<uintptr_t>(a->g_down) | reinterpret_cast<uintptr_t>(a->g_up)) & 15u))
      return fail(RINGADA_E_INVALID, "adapter gradients must be 16-byte aligned");
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int dt = D.dtype;
  const size_t d = D.d_model, F = D.d_ffn, m = D.d_adapter;
  const WeightLayout& WL = st->WL;
  char* mem = static_cast<char*>(block_mem);
  BlockBind& b = st->blocks[block];
  b.wt_qkv = mem + WL.qkv;
  b.bqkv = WL.bqkv != NONE ? mem + WL.bqkv : nullptr;
  b.wt_o = mem + WL.o;
  b.wt_in = mem + WL.in;
  b.wt_out = mem + WL.out;
  for (int a = 0; a < 2; ++a)
    for (int k = 0; k < 4; ++k) b.wk[a][k] = WL.wk[a][k] != NONE ? mem + WL.wk[a][k] : nullptr;
  std::vector<float2> tab;
  if (st->rope_tab && !st->rope_built) {  // rotation angles pos * theta^(-2i/dh), in double, once per stage
    const int dh = (int)(d / D.n_heads), half = dh / 2;
    tab.resize((size_t)D.max_seq * half);
    for (int p = 0; p < D.max_seq; ++p)
      for (int i = 0; i < half; ++i) {
        const double ang = p * std::pow((double)D.rope_theta, -2.0 * i / dh);
        tab[(size_t)p * half + i] = make_float2((float)std::cos(ang), (float)std::sin(ang));
      }
    RG_HIP(hipMemcpyAsync(st->rope_tab, tab.data(), tab.size() * sizeof(float2), hipMemcpyHostToDevice, s));
  }
  b.w = *w;
  b.ad[0] = attn ? *attn : ringada_adapter{};
  b.ad[1] = *ffn;
  // the projection transposed (in per-head row order when the stage fuses
  // attention: row p*d + h*dh + i of the three-block order goes to (3h + p)*dh + i)
  const int perm = st->qkv_per_head ? (int)(d / D.n_heads) : 0;
  RG_HIP(launch_transpose(dt, dt, w->w_qkv, (int)d, (int)(3 * d), b.wt_qkv, s, perm));
  if (b.bqkv) RG_HIP(launch_transpose(dt, dt, w->b_qkv, 1, (int)(3 * d), b.bqkv, s, perm));
  RG_HIP(launch_transpose(dt, dt, w->w_o, (int)d, (int)d, b.wt_o, s));
  if (post) RG_HIP(launch_transpose(dt, dt, w->w_in, (int)d, (int)F, b.wt_in, s));
  else RG_HIP(launch_pack_swiglu(dt, w->w_in, (int)d, (int)F, b.wt_in, s));
  RG_HIP(launch_transpose(dt, dt, w->w_out, (int)F, (int)d, b.wt_out, s));
  for (int a = 0; a < 2; ++a) {
    AdapterSlot& sl = st->slots[2 * block + a];
    sl.w_down = b.ad[a].w_down;
    sl.w_up = b.ad[a].w_up;
    sl.g_down = b.ad[a].g_down;
    sl.g_up = b.ad[a].g_up;
    sl.wdn = b.wk[a][0];
    sl.wdn_t = b.wk[a][1];
    sl.wup = b.wk[a][2];
    sl.wup_t = b.wk[a][3];
  }
  RG_HIP(launch_adapter_sync(dt, st->slots.data() + 2 * block, 2, (int)d, (int)m, s));
  RG_HIP(hipStreamSynchronize(s));  // also keeps `tab` alive until its copy has run
  if (st->rope_tab) st->rope_built = true;
  b.bound = true;
  return RINGADA_OK;
}

extern "C" ringada_status ringada_stage_sync_adapters(ringada_stage* st, void* stream) {
  if (!st) return fail(RINGADA_E_INVALID, "NULL stage");
  for (const BlockBind& b : st->blocks)
    if (!b.bound) return fail(RINGADA_E_STATE, "every block must be bound first");
  RG_HIP(launch_adapter_sync(st->D.dtype, st->slots.data(), 2 * st->D.n_blocks, st->D.d_model,
                             st->D.d_adapter, static_cast<hipStream_t>(stream)));
  return RINGADA_OK;
}

// ================================================================ launches (with optional event timing)
thread_local LaunchEvents* rg::g_launch_events = nullptr;

static hipEvent_t pool_event(ringada_stage* st) {
  if (st->evused == st->evpool.size()) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    st->evpool.push_back(e);
  }
  return st->evpool[st->evused++];
}

template <class Fn>
static ringada_status run(ringada_stage* st, hipStream_t s, const char* name, double flops, double bytes, Fn&& fn) {
  if (!st->prof) {
    const hipError_t e = fn();
    if (e != hipSuccess) return fail(RINGADA_E_HIP, "%s: %s", name, hipGetErrorString(e));
    return RINGADA_OK;
  }
  // the launches inside fn() carry the events (kernel start .. kernel end)
  LaunchEvents le{pool_event(st), pool_event(st), false};
  if (!le.start || !le.stop) return fail(RINGADA_E_HIP, "hipEventCreate failed");
  g_launch_events = &le;
  const hipError_t e = fn();
  g_launch_events = nullptr;
  if (e != hipSuccess) return fail(RINGADA_E_HIP, "%s: %s", name, hipGetErrorString(e));
  if (!le.started) return RINGADA_OK;  // nothing launched (empty input)
  st->recs.push_back(ProfRec{name, flops, bytes, le.start, le.stop});
  return RINGADA_OK;
}

extern "C" ringada_status ringada_prof_begin(ringada_stage* st) {
  if (!st) return fail(RINGADA_E_INVALID, "NULL stage");
  st->prof = true;
  st->recs.clear();
  st->evused = 0;
  return RINGADA_OK;
}

extern "C" ringada_status ringada_prof_end(ringada_stage* st, ringada_prof_entry* out, int32_t max_entries,
                                           int32_t* n_entries) {
  if (!st || !n_entries || (max_entries > 0 && !out)) return fail(RINGADA_E_INVALID, "NULL argument");
  st->prof = false;
  std::vector<ringada_prof_entry> agg;
  for (const ProfRec& r : st->recs) {
    RG_HIP(hipEventSynchronize(r.e1));
    float ms = 0.f;
    RG_HIP(hipEventElapsedTime(&ms, r.e0, r.e1));
    auto it = std::find_if(agg.begin(), agg.end(), [&](const ringada_prof_entry& e) { return strcmp(e.name, r.name) == 0; });
    if (it == agg.end()) {
      ringada_prof_entry e{};
      snprintf(e.name, sizeof e.name, "%s", r.name);
      agg.push_back(e);
      it = agg.end() - 1;
    }
    it->launches += 1;
    it->total_ms += ms;
    it->flops += r.flops;
    it->bytes += r.bytes;
  }
  st->recs.clear();
  st->evused = 0;
  *n_entries = (int32_t)agg.size();
  for (int32_t i = 0; i < std::min<int32_t>(max_entries, (int32_t)agg.size()); ++i) out[i] = agg[i];
  return RINGADA_OK;
}

// ================================================================ schedule helpers
struct Ctx {
  ringada_stage* st;
  hipStream_t s;
  int dt;
  size_t es;
  int T, d, F, m, H, dh;
  bool llama;
  char* stash;
  char* scratch;
  void* S(size_t off) const { return off == NONE ? nullptr : stash + off; }
  void* W(size_t off) const { return off == NONE ? nullptr : scratch + off; }
};

// bf16 pre-RMS stages rotate Q and K in the QKV projection's epilogue
static bool rope_in_qkv(const Ctx& c) { return c.llama && c.dt == DT_BF16; }

static ringada_status gemm(const Ctx& c, Role role, Epi epi, int M, int N, int K, const void* A, int lda,
                           const void* B, int ldb, void* out, int ldo, const void* bias = nullptr,
                           const void* aux = nullptr, int ld_aux = 0, void* out2 = nullptr, int ldo2 = 0,
                           int half = 0) {
  GemmArgs g{A, lda, B, ldb, M, N, K, bias, aux, ld_aux, out, ldo, out2, ldo2, half};
  const double flops = 2.0 * M * N * K;
  double bytes = (double)c.es * ((double)M * K + (double)N * K + (double)M * N);
  if (aux) bytes += (double)c.es * M * N * (epi == Epi::DSwiGlu ? 2 : 1);
  if (out2) bytes += (double)c.es * M * N;
  if (epi == Epi::DSwiGlu) bytes += (double)c.es * M * N;
  return run(c.st, c.s, role_name(role), flops, bytes, [&] { return launch_gemm(c.dt, role, epi, g, c.s); });
}

// ================================================================ forward
static ringada_status block_forward(const Ctx& c, int l, const void* X, void* Y) {
  ringada_stage* st = c.st;
  const BlockBind& b = st->blocks[l];
  const Layout& L = st->L;
  const BlockStash& sb = L.blk[l];
  const bool single = st->D.placement == RINGADA_PLACEMENT_FFN;
  const int T = c.T, d = c.d, F = c.F, m = c.m;
  const double es = (double)c.es;
  // a tensor goes to its stash slot when the planner gave it one, else to
  // the shared scratch (or nowhere, for the stash-only outputs)
  auto SW = [&](size_t off, size_t scratch_off) { return off != NONE ? c.S(off) : c.W(scratch_off); };
  auto SN = [&](size_t off) -> void* { return off != NONE ? c.S(off) : nullptr; };
  void* qkv = SW(sb.qkv, L.qkv);
  void* o = SW(sb.o, L.o);
  float* lse = static_cast<float*>(SW(sb.lse, L.lse));
  void* attn = SW(sb.attn, L.attn);
  void* f2 = SW(sb.f2, L.f2);
  void* g = c.W(L.g);
  void* h1 = c.W(L.h1);
  const void* xin = X;

  if (c.llama) {
    void* n1 = c.W(L.n1);
    RG_TRY(run(st, c.s, "rms_fwd", 0, es * 2.0 * T * d, [&] {
      return launch_rms_fwd(c.dt, T, d, st->D.norm_eps, X, b.w.norm1_g, n1, SN(sb.xhat1),
                            static_cast<float*>(SN(sb.rstd1)), c.s);
    }));
    xin = n1;
  }
  const double attn_flops = 4.0 * L.B * c.H * (double)L.S * L.S * c.dh * (c.llama ? 0.5 : 1.0);
  if (st->qkv_per_head && L.S == 128) {
    // projection + attention in one kernel; the projections leave it only
    // when the backward needs them
    GemmArgs g{xin, d, b.wt_qkv, d, T, 3 * d, d, b.bqkv, nullptr, 0, SN(sb.qkv), 3 * d, o, d, 0};
    g.lse = lse;
    const double bytes = es * ((double)T * d + 3.0 * d * d + (g.out ? 3.0 * T * d : 0.0) + (double)T * d) +
                         4.0 * L.B * c.H * L.S;
    RG_TRY(run(st, c.s, "gemm_qkv_attn_fwd", 2.0 * T * 3.0 * d * d + attn_flops, bytes,
               [&] { return launch_gemm(c.dt, R_QKV_FWD, Epi::Attn, g, c.s); }));
  } else {
    if (rope_in_qkv(c)) {
      // the rotary embedding applied once, in the projection's epilogue: the
      // stash keeps the rotated Q and K, which the attention loads as they are
      GemmArgs g{xin, d, b.wt_qkv, d, T, 3 * d, d, nullptr, nullptr, 0, qkv, 3 * d, nullptr, 0, 0};
      g.rope_tab = st->rope_tab; g.rope_S = L.S; g.rope_dh = c.dh; g.rope_cols = 2 * d;
      RG_TRY(run(st, c.s, role_name(R_QKV_FWD), 2.0 * T * 3.0 * d * d, es * ((double)T * d + 3.0 * d * d + 3.0 * T * d),
                 [&] { return launch_gemm(c.dt, R_QKV_FWD, Epi::Rope, g, c.s); }));
    } else {
      RG_TRY(gemm(c, R_QKV_FWD, Epi::Store, T, 3 * d, d, xin, d, b.wt_qkv, d, qkv, 3 * d,
                  st->qkv_per_head ? b.bqkv : b.w.b_qkv));
    }
    AttnArgs aa{};
    aa.B = L.B; aa.S = L.S; aa.H = c.H; aa.dh = c.dh;
    aa.causal = c.llama; aa.rope = c.llama; aa.theta = st->D.rope_theta;
    aa.rope_tab = st->rope_tab; aa.rope_rows = st->D.max_seq;
    aa.qkv = qkv; aa.ld_qkv = 3 * d; aa.o = o; aa.ld_o = d; aa.lse = lse;
    if (st->qkv_per_head) { aa.qkv_hs = 3 * c.dh; aa.qkv_ko = c.dh; aa.qkv_vo = 2 * c.dh; }
    aa.rope_in_qkv = rope_in_qkv(c);
    RG_TRY(run(st, c.s, "attn_fwd", attn_flops, es * 4.0 * T * d, [&] { return launch_attn_fwd(c.dt, aa, c.s); }));
  }
  RG_TRY(gemm(c, R_O_FWD, Epi::Store, T, d, d, o, d, b.wt_o, d, attn, d, b.w.b_o));

  AdapterFwdArgs fa{};
  fa.T = T; fa.d = d; fa.m = m; fa.eps = st->D.norm_eps;
  fa.z = attn; fa.res = X;
  if (!single) { fa.wdn_t = b.wk[0][1]; fa.wup_t = b.wk[0][3]; }  // else residual add + norm only
  fa.gamma = c.llama ? b.w.norm2_g : b.w.norm1_g;
  fa.u = SN(sb.u1); fa.part = static_cast<float*>(c.W(L.adp));
  void* ffn_in;
  if (c.llama) {
    fa.norm = Norm::RMS; fa.out = h1; fa.out_norm = c.W(L.n2);
    fa.xhat = SN(sb.xhat2); fa.rstd = static_cast<float*>(SN(sb.rstd2));
    ffn_in = c.W(L.n2);
  } else {
    fa.norm = Norm::LN; fa.beta = b.w.norm1_b; fa.out = h1;
    fa.xhat = SN(sb.xhat1); fa.rstd = static_cast<float*>(SN(sb.rstd1));
    ffn_in = h1;
  }
  const double ad_flops = 4.0 * T * d * m;
  RG_TRY(run(st, c.s, "adapter_fwd", single ? 0.0 : ad_flops,
             es * (3.0 + (c.llama ? 1 : 0) + (fa.xhat ? 1 : 0)) * T * d,
             [&] { return launch_adapter_fwd(c.dt, fa, c.s); }));
  if (c.llama)
    RG_TRY(gemm(c, R_FFN_IN_FWD, Epi::SwiGlu, T, 2 * F, d, ffn_in, d, b.wt_in, d, g, F, nullptr, nullptr, 0,
                SN(sb.a1), 2 * F, F));
  else
    RG_TRY(gemm(c, R_FFN_IN_FWD, Epi::Gelu, T, F, d, ffn_in, d, b.wt_in, d, g, F, b.w.b_in, nullptr, 0,
                SN(sb.a1), F));
  RG_TRY(gemm(c, R_FFN_OUT_FWD, Epi::Store, T, d, F, g, F, b.wt_out, F, f2, d, b.w.b_out));

  AdapterFwdArgs fb{};
  fb.T = T; fb.d = d; fb.m = m; fb.eps = st->D.norm_eps;
  fb.z = f2; fb.res = h1; fb.wdn_t = b.wk[1][1]; fb.wup_t = b.wk[1][3];
  fb.u = SN(sb.u2); fb.out = Y; fb.part = static_cast<float*>(c.W(L.adp));
  if (c.llama) {
    fb.norm = Norm::None;
  } else {
    fb.norm = Norm::LN; fb.gamma = b.w.norm2_g; fb.beta = b.w.norm2_b;
    fb.xhat = SN(sb.xhat2); fb.rstd = static_cast<float*>(SN(sb.rstd2));
  }
  RG_TRY(run(st, c.s, "adapter_fwd", ad_flops, es * (3.0 + (fb.xhat ? 1 : 0)) * T * d,
             [&] { return launch_adapter_fwd(c.dt, fb, c.s); }));
  return RINGADA_OK;
}

static ringada_status make_ctx(ringada_stage* st, void* stream, Ctx& c) {
  const ringada_stage_desc& D = st->D;
  c.st = st;
  c.s = static_cast<hipStream_t>(stream);
  c.dt = D.dtype;
  c.es = D.dtype == RINGADA_BF16 ? 2 : 4;
  c.T = st->L.B * st->L.S;
  c.d = D.d_model; c.F = D.d_ffn; c.m = D.d_adapter; c.H = D.n_heads; c.dh = D.d_model / D.n_heads;
  c.llama = D.arch == RINGADA_ARCH_PRERMS_SWIGLU;
  c.stash = st->stash;
  c.scratch = st->scratch;
  return RINGADA_OK;
}

extern "C" ringada_status ringada_stage_forward(ringada_stage* st, void* stream, const void* x, void* y,
                                                int32_t batch, int32_t seq, int32_t lowest_unfrozen, void* stash,
                                                size_t stash_bytes, void* scratch, size_t scratch_bytes) {
  if (!st || !x || !y) return fail(RINGADA_E_INVALID, "NULL argument");
  const ringada_stage_desc& D = st->D;
  for (int l = 0; l < D.n_blocks; ++l)
    if (!st->blocks[l].bound) return fail(RINGADA_E_STATE, "block %d is not bound", l);
  if (batch < 1 || seq < 1 || batch > D.max_batch || seq > D.max_seq)
    return fail(RINGADA_E_INVALID, "batch %d / seq %d outside [1, max]", batch, seq);
  const int c = norm_cut(lowest_unfrozen, D.n_blocks);
  // also a frozen forward: it would run on adapters whose update is pending
  // and overwrite the stash the pending backward reads
  if (st->pending)
    return fail(RINGADA_E_STATE, "a forward with unfrozen adapters is pending its backward "
                                 "(one forward, one backward on unfrozen stages)");
  const size_t es = D.dtype == RINGADA_BF16 ? 2 : 4;
  const size_t io = (size_t)batch * seq * D.d_model * es;
  const char* xb = static_cast<const char*>(x);
  const char* yb = static_cast<const char*>(y);
  if (xb < yb + io && yb < xb + io) return fail(RINGADA_E_INVALID, "x and y overlap");
  Layout L;
  plan_layout(D, batch, seq, c, L);
  if (stash_bytes < L.stash_bytes || (L.stash_bytes && !stash))
    return fail(RINGADA_E_WORKSPACE, "stash of %zu bytes, plan needs %zu", stash_bytes, L.stash_bytes);
  if (scratch_bytes < L.scratch_bytes || !scratch)
    return fail(RINGADA_E_WORKSPACE, "scratch of %zu bytes, plan needs %zu", scratch_bytes, L.scratch_bytes);
  if ((reinterpret_cast<uintptr_t>(stash) | reinterpret_cast<uintptr_t>(scratch) |
       reinterpret_cast<uintptr_t>(x) | reinterpret_cast<uintptr_t>(y)) & 15u)
    return fail(RINGADA_E_INVALID, "x, y, stash and scratch must be 16-byte aligned");
  st->L = L;
  st->stash = static_cast<char*>(stash);
  st->scratch = static_cast<char*>(scratch);
  Ctx cx;
  RG_TRY(make_ctx(st, stream, cx));
  const void* in = x;
  for (int l = 0; l < D.n_blocks; ++l) {
    void* out = (l == D.n_blocks - 1) ? y : cx.W(L.act[l % 2]);
    RG_TRY(block_forward(cx, l, in, out));
    in = out;
  }
  st->pending = c < D.n_blocks;
  return RINGADA_OK;
}

// ================================================================ backward
static ringada_status block_backward(const Ctx& c, int l, const void* G, void* dX, bool stop) {
  ringada_stage* st = c.st;
  BlockBind& b = st->blocks[l];
  const Layout& L = st->L;
  const BlockStash& sb = L.blk[l];
  const int T = c.T, d = c.d, F = c.F, m = c.m;
  const double es = (double)c.es;
  const double ad_flops = 6.0 * T * d * m;
  // under the single placement the block's lowest adapter is its FFN adapter
  const bool single = st->D.placement == RINGADA_PLACEMENT_FFN, stop_ffn = single && stop;

  // FFN adapter (+ LN2 for post-LN)
  AdapterBwdArgs ab{};
  ab.T = T; ab.d = d; ab.m = m; ab.gin = G; ab.u = c.S(sb.u2);
  ab.wup = b.wk[1][2]; ab.wdn = b.wk[1][0]; ab.du = c.W(L.gdu[2 * l + 1]); ab.gu = c.W(L.ggu[2 * l + 1]);
  ab.dzin = stop_ffn ? nullptr : c.W(L.df2);
  ab.part = static_cast<float*>(c.W(L.adp));
  // the gradient at the adapter output goes to this adapter's own buffer
  // (pre-RMS: a copy of G, which a later block's dX overwrites)
  ab.dz = c.W(L.gdz[2 * l + 1]);
  const void* dz2 = ab.dz;
  if (c.llama) {
    ab.norm = Norm::None;
  } else {
    ab.norm = Norm::LN; ab.xhat = c.S(sb.xhat2); ab.rstd = static_cast<const float*>(c.S(sb.rstd2));
    ab.gamma = b.w.norm2_g;
  }
  RG_TRY(run(st, c.s, "adapter_bwd", stop_ffn ? 4.0 * T * d * m : ad_flops,
             es * ((c.llama ? 3.0 : 5.0) - (stop_ffn ? 1.0 : 0.0)) * T * d,
             [&] { return launch_adapter_bwd(c.dt, ab, c.s); }));
  st->dw_pending.push_back(
      AdapterDwArgs{T, d, m, c.S(sb.u2), dz2, c.S(sb.f2), ab.du, b.ad[1].g_up, b.ad[1].g_down, ab.gu});
  if (stop_ffn) return RINGADA_OK;

  // FFN (dX only through frozen weights)
  void* da1 = c.W(L.da1);
  if (c.llama) {
    RG_TRY(gemm(c, R_FFN_OUT_DX, Epi::DSwiGlu, T, F, d, c.W(L.df2), d, b.w.w_out, d, da1, 2 * F, nullptr,
                c.S(sb.a1), 2 * F, nullptr, 0, F));
    RG_TRY(gemm(c, R_FFN_IN_DX, Epi::Store, T, d, 2 * F, da1, 2 * F, b.w.w_in, 2 * F, c.W(L.dh1), d));
  } else {
    RG_TRY(gemm(c, R_FFN_OUT_DX, Epi::DGelu, T, F, d, c.W(L.df2), d, b.w.w_out, d, da1, F, nullptr, c.S(sb.a1), F));
    RG_TRY(gemm(c, R_FFN_IN_DX, Epi::Resid, T, d, F, da1, F, b.w.w_in, F, c.W(L.dh1), d, nullptr, dz2, d));
  }

  // attention adapter (+ LN1 / RMSNorm-2 backward); without one (single
  // placement) only the norm backward, whose output is then the gradient at
  // the attention sublayer's output
  AdapterBwdArgs aa{};
  void* dz1 = single ? c.W(L.dz1) : c.W(L.gdz[2 * l]);
  aa.T = T; aa.d = d; aa.m = m; aa.gin = c.W(L.dh1); aa.dz = dz1;
  aa.part = static_cast<float*>(c.W(L.adp));
  if (!single) {
    aa.u = c.S(sb.u1); aa.wup = b.wk[0][2]; aa.wdn = b.wk[0][0]; aa.du = c.W(L.gdu[2 * l]);
    aa.gu = c.W(L.ggu[2 * l]);
    aa.dzin = stop ? nullptr : c.W(L.dattn);
  }
  void* dattn = single ? dz1 : c.W(L.dattn);
  if (c.llama) {
    aa.norm = Norm::RMS; aa.dres = G; aa.xhat = c.S(sb.xhat2);
    aa.rstd = static_cast<const float*>(c.S(sb.rstd2)); aa.gamma = b.w.norm2_g;
  } else {
    aa.norm = Norm::LN; aa.xhat = c.S(sb.xhat1); aa.rstd = static_cast<const float*>(c.S(sb.rstd1));
    aa.gamma = b.w.norm1_g;
  }
  RG_TRY(run(st, c.s, single ? "norm_bwd" : "adapter_bwd", single ? 0.0 : (stop ? 4.0 * T * d * m : ad_flops),
             es * ((c.llama ? 4.0 : 3.0) + (stop || single ? 0.0 : 1.0)) * T * d,
             [&] { return launch_adapter_bwd(c.dt, aa, c.s); }));
  if (!single)
    st->dw_pending.push_back(
        AdapterDwArgs{T, d, m, c.S(sb.u1), dz1, c.S(sb.attn), aa.du, b.ad[0].g_up, b.ad[0].g_down, aa.gu});
  if (stop) return RINGADA_OK;

  // attention (dX only)
  RG_TRY(gemm(c, R_O_DX, Epi::Store, T, d, d, dattn, d, b.w.w_o, d, c.W(L.dout), d));
  AttnArgs at{};
  at.B = L.B; at.S = L.S; at.H = c.H; at.dh = c.dh;
  at.causal = c.llama; at.rope = c.llama; at.theta = st->D.rope_theta;
  at.rope_tab = st->rope_tab; at.rope_rows = st->D.max_seq;
  at.qkv = c.S(sb.qkv); at.ld_qkv = 3 * d; at.o = c.S(sb.o); at.ld_o = d;
  if (st->qkv_per_head) { at.qkv_hs = 3 * c.dh; at.qkv_ko = c.dh; at.qkv_vo = 2 * c.dh; }
  at.rope_in_qkv = rope_in_qkv(c);
  at.lse = static_cast<float*>(c.S(sb.lse));
  at.dout = c.W(L.dout); at.ld_do = d; at.dsum = static_cast<float*>(c.W(L.dsum));
  at.dqkv = c.W(L.dqkv); at.ld_dqkv = 3 * d;
  const double attn_flops = 8.0 * L.B * c.H * (double)L.S * L.S * c.dh * (c.llama ? 0.5 : 1.0);
  RG_TRY(run(st, c.s, "attn_bwd", attn_flops, es * 8.0 * T * d, [&] { return launch_attn_bwd(c.dt, at, c.s); }));
  if (c.llama) {
    RG_TRY(gemm(c, R_QKV_DX, Epi::Store, T, d, 3 * d, c.W(L.dqkv), 3 * d, b.w.w_qkv, 3 * d, c.W(L.dn1), d));
    RG_TRY(run(st, c.s, "rms_bwd", 0, es * 4.0 * T * d, [&] {
      return launch_rms_bwd(c.dt, T, d, c.W(L.dn1), dz1, c.S(sb.xhat1),
                            static_cast<const float*>(c.S(sb.rstd1)), b.w.norm1_g, dX, c.s);
    }));
  } else {
    RG_TRY(gemm(c, R_QKV_DX, Epi::Resid, T, d, 3 * d, c.W(L.dqkv), 3 * d, b.w.w_qkv, 3 * d, dX, d, nullptr,
                dz1, d));
  }
  return RINGADA_OK;
}

extern "C" ringada_status ringada_stage_backward(ringada_stage* st, void* stream, const void* dy,
                                                 int32_t lowest_unfrozen, void* dx_in) {
  if (!st || !dy) return fail(RINGADA_E_INVALID, "NULL argument");
  const ringada_stage_desc& D = st->D;
  if (!st->pending) return fail(RINGADA_E_STATE, "no forward with unfrozen adapters is pending");
  const int c = norm_cut(lowest_unfrozen, D.n_blocks);
  if (c >= D.n_blocks) return fail(RINGADA_E_STATE, "lowest_unfrozen >= n_blocks: the stage is frozen");
  if (c < st->L.c)
    return fail(RINGADA_E_STATE, "the forward stashed from block %d; cannot back-propagate to %d", st->L.c, c);
  if ((c < 0) != (dx_in != nullptr))
    return fail(RINGADA_E_INVALID, "dx_in must be given exactly when lowest_unfrozen < 0");
  if ((reinterpret_cast<uintptr_t>(dy) | reinterpret_cast<uintptr_t>(dx_in)) & 15u)
    return fail(RINGADA_E_INVALID, "dy and dx_in must be 16-byte aligned");
  Ctx cx;
  RG_TRY(make_ctx(st, stream, cx));
  const void* G = dy;
  const int lo = c < 0 ? 0 : c;
  st->dw_pending.clear();
  for (int l = D.n_blocks - 1; l >= lo; --l) {
    const bool stop = (l == c);
    void* dX = stop ? nullptr : (l == 0 ? dx_in : cx.W(st->L.dact[l % 2]));
    RG_TRY(block_backward(cx, l, G, dX, stop));
    G = dX;
  }
  // the adapters' weight gradients (dW_up += gelu(U)^T dZ, dW_down += z^T dU)
  // of the whole backward in one launch: off the dX chain, and enough
  // workgroups to fill the GPU
  const int ndw = (int)st->dw_pending.size();
  RG_TRY(run(st, cx.s, "adapter_dw", 4.0 * ndw * cx.T * cx.d * cx.m, 2.0 * ndw * cx.es * cx.T * cx.d, [&] {
    return launch_adapter_dw_batch(cx.dt, st->dw_pending.data(), ndw, static_cast<float*>(cx.W(st->L.dwp)),
                                   (long)st->L.dwp_bytes, cx.s);
  }));
  st->pending = false;
  return RINGADA_OK;
}

extern "C" ringada_status ringada_adapter_step(ringada_stage* st, void* stream, int32_t lowest_unfrozen,
                                               const ringada_optim* opt) {
  if (!st || !opt) return fail(RINGADA_E_INVALID, "NULL argument");
  if (opt->kind != 0) return fail(RINGADA_E_UNSUPPORTED, "optimiser kind %d (only SGD = 0)", opt->kind);
  const ringada_stage_desc& D = st->D;
  for (int l = 0; l < D.n_blocks; ++l)
    if (!st->blocks[l].bound) return fail(RINGADA_E_STATE, "block %d is not bound", l);
  if (st->pending)
    return fail(RINGADA_E_STATE, "a forward is pending its backward: updating the adapters now would "
                                 "mix new weights with the activations stashed under the old ones");
  const int c = norm_cut(lowest_unfrozen, D.n_blocks);
  const int lo = c < 0 ? 0 : c;
  if (lo >= D.n_blocks) return RINGADA_OK;
  const int n = 2 * (D.n_blocks - lo);
  const double bytes = (double)n * D.d_model * D.d_adapter * (4.0 * 4 + 4.0 * (D.dtype == RINGADA_BF16 ? 2 : 4));
  return run(st, static_cast<hipStream_t>(stream), "adapter_step", 0, bytes, [&] {
    return launch_adapter_sgd(D.dtype, st->slots.data() + 2 * lo, n, D.d_model, D.d_adapter, opt->lr,
                              static_cast<hipStream_t>(stream));
  });
}

// ================================================================ initiator helpers
extern "C" ringada_status ringada_loss_mse(void* stream, int32_t dtype, const void* y, const void* target, int64_t n,
                                           void* dy, float* loss) {
  if (dtype != RINGADA_F32 && dtype != RINGADA_BF16) return fail(RINGADA_E_INVALID, "unknown dtype");
  if (!y || !target || !dy || n <= 0) return fail(RINGADA_E_INVALID, "bad argument");
  RG_HIP(launch_mse(dtype, y, target, n, dy, loss, static_cast<hipStream_t>(stream)));
  return RINGADA_OK;
}

extern "C" ringada_status ringada_head_ce(void* stream, int32_t dtype, const void* y, int32_t batch, int32_t seq,
                                          int32_t d, const float* w_h, const float* b_h, int32_t n_classes,
                                          const int32_t* labels, void* dy, float* g_wh, float* g_bh, float* loss) {
  if (dtype != RINGADA_F32 && dtype != RINGADA_BF16) return fail(RINGADA_E_INVALID, "unknown dtype");
  if (!y || !w_h || !b_h || !labels || !dy || !g_wh || !g_bh) return fail(RINGADA_E_INVALID, "NULL argument");
  if (batch < 1 || seq < 1 || d < 1 || n_classes < 1 || n_classes > 16) return fail(RINGADA_E_INVALID, "bad size");
  RG_HIP(launch_head_ce(dtype, y, batch, seq, d, w_h, b_h, n_classes, labels, dy, g_wh, g_bh, loss,
                        static_cast<hipStream_t>(stream)));
  return RINGADA_OK;
}

extern "C" ringada_status ringada_sgd_f32(void* stream, float* w, float* g, int64_t n, float lr) {
  if (!w || !g || n <= 0) return fail(RINGADA_E_INVALID, "bad argument");
  RG_HIP(launch_sgd_f32(w, g, n, lr, static_cast<hipStream_t>(stream)));
  return RINGADA_OK;
}
