/*
 * ringada.h -- C ABI of the RingAda per-stage hot path on AMD MI355X (gfx950).
 *
 * One ring client of RingAda (arXiv 2502.19864) hosts a contiguous run of
 * frozen transformer blocks (the Trm layers of Sec. III-A) each carrying two
 * bottleneck adapters h <- h + sigma(h W_down) W_up (Eq. (1)), one after the
 * attention sublayer and one after the feed-forward sublayer.  Per training
 * iteration the client
 *   - applies its blocks to the activations handed over by the previous
 *     client and passes the result on (Sec. II-B and Sec. III-B,
 *     "Forward and Backward Propagation");
 *   - relays the gradient handed back by the next client down through its
 *     frozen weights, producing weight gradients for unfrozen adapters only,
 *     and stops at the lowest unfrozen adapter (Alg. 1: the backward ends at
 *     the (L-d+1)-th adapter; Sec. III-B: the terminator);
 *   - updates its unfrozen adapters (Sec. III-B).
 * A client may not forward a new batch while the update of its unfrozen
 * adapters for the previous batch is pending (Sec. III-B: unfrozen clients keep
 * the one-forward-one-backward order; Sec. III-B "three-fold advantages": no
 * stale weights).
 *
 * Conventions used by every call
 *   - All tensor pointers are DEVICE pointers unless stated otherwise.
 *   - Activations are row-major [batch, seq, d_model] in the stage dtype
 *     (RINGADA_F32: float, RINGADA_BF16: bfloat16 bit patterns in uint16).
 *     Arithmetic accumulates in fp32 for both dtypes.
 *   - Weights are row-major [in, out]: a projection is x @ W, as in Eq. (1).
 *   - stream is a hipStream_t passed as void* (NULL = the null stream).  Calls
 *     enqueue kernels and return; they never synchronise the device, except
 *     ringada_stage_bind_block and ringada_prof_end as documented.
 *   - Errors are returned as a status; the message of the last failing call on
 *     the calling thread is available from ringada_last_error().  The library
 *     never aborts and never prints.
 *   - The library allocates no device memory, in any call.  Every device
 *     buffer is the caller's: frozen weights, adapter masters and gradients,
 *     the activation stash and scratch (ringada_stage_plan), and the regions
 *     that hold what the library derives from the weights
 *     (ringada_stage_plan_weights).
 */
#ifndef RINGADA_H
#define RINGADA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  RINGADA_OK = 0,
  RINGADA_E_INVALID = 1,     /* a NULL pointer, a size out of range, an unknown enum */
  RINGADA_E_STATE = 2,       /* call out of order: see the state machine below */
  RINGADA_E_WORKSPACE = 3,   /* stash or scratch smaller than ringada_stage_plan says */
  RINGADA_E_UNSUPPORTED = 4, /* a shape or option this build has no kernel for */
  RINGADA_E_HIP = 5          /* a HIP runtime call failed (message has the HIP error) */
} ringada_status;

enum {
  /* post-LN encoder block (BERT shape): bias on every projection, GELU FFN,
   * bidirectional attention, LayerNorm after each residual add */
  RINGADA_ARCH_POSTLN_GELU = 0,
  /* pre-RMSNorm decoder block (LLaMA shape): no biases, SwiGLU FFN, RoPE
   * (rotate-half pairs (i, i + d_head/2)), causal attention */
  RINGADA_ARCH_PRERMS_SWIGLU = 1
};
enum { RINGADA_F32 = 0, RINGADA_BF16 = 1 };
enum {
  /* two adapters per block: one on the attention sublayer's output, one on
   * the FFN sublayer's output, each before the block's residual add */
  RINGADA_PLACEMENT_HOULSBY = 0,
  /* the single serial adapter of Sec. II-A (Fig. 1): one adapter per block,
   * on the FFN sublayer's output; the attention sublayer carries none */
  RINGADA_PLACEMENT_FFN = 1
};

typedef struct {
  int32_t arch;       /* RINGADA_ARCH_* */
  int32_t dtype;      /* RINGADA_F32 or RINGADA_BF16 storage */
  int32_t n_blocks;   /* L, blocks held by this stage, >= 1 */
  int32_t d_model;    /* d; bf16 path: a multiple of 256 up to 1024, or of
                         1024 up to 4096 */
  int32_t n_heads;    /* d_head = d_model / n_heads; bf16 path: d_head 64 or 128 */
  int32_t d_ffn;      /* F; bf16 path: multiple of 64 */
  int32_t d_adapter;  /* m, the bottleneck of Eq. (1); bf16 path: 64 */
  int32_t max_batch;  /* upper bounds for batch and seq of later calls */
  int32_t max_seq;
  float norm_eps;     /* LayerNorm / RMSNorm epsilon (added to the variance) */
  float rope_theta;   /* RoPE base, pre-RMS arch only */
  int32_t placement;  /* RINGADA_PLACEMENT_*: where the adapters sit */
} ringada_stage_desc;

/* Frozen weights of one block, device pointers in the stage dtype, all
 * row-major [in, out].  Pointers marked (post-LN) must be NULL for the pre-RMS
 * arch and non-NULL for the post-LN arch.  The norm gains and shifts
 * (norm1_g, norm1_b, norm2_g, norm2_b) must be 16-byte aligned
 * (ringada_stage_bind_block returns RINGADA_E_INVALID otherwise).  The memory
 * is borrowed: it must stay valid and unchanged until ringada_stage_destroy. */
typedef struct {
  const void* w_qkv;   /* [d, 3d]; output columns are [Q | K | V], head h owns
                          columns [h*d_head, (h+1)*d_head) of each */
  const void* b_qkv;   /* [3d] (post-LN) */
  const void* w_o;     /* [d, d] */
  const void* b_o;     /* [d] (post-LN) */
  const void* norm1_g; /* [d] LN1 gamma (post-LN) or RMSNorm-1 gain (pre-RMS) */
  const void* norm1_b; /* [d] LN1 beta (post-LN) */
  const void* w_in;    /* post-LN: W_i [d, F]; pre-RMS: [d, 2F] = [W_gate | W_up] */
  const void* b_in;    /* [F] (post-LN) */
  const void* w_out;   /* [F, d] */
  const void* b_out;   /* [d] (post-LN) */
  const void* norm2_g; /* [d] LN2 gamma or RMSNorm-2 gain */
  const void* norm2_b; /* [d] LN2 beta (post-LN) */
} ringada_block_weights;

/* One adapter of Eq. (1) (no biases): fp32 master weights and fp32 gradient
 * accumulators, device, caller-owned, borrowed until ringada_stage_destroy.
 * The backward ADDS into g_down/g_up; ringada_adapter_step consumes and zeroes
 * them.  g_down and g_up must be 16-byte aligned (ringada_stage_bind_block
 * returns RINGADA_E_INVALID otherwise); the bf16 backward sums each gradient
 * element in a fixed order, so equal inputs give bitwise equal gradients. */
typedef struct {
  float* w_down; /* [d, m] */
  float* w_up;   /* [m, d] */
  float* g_down; /* [d, m] */
  float* g_up;   /* [m, d] */
} ringada_adapter;

typedef struct {
  int32_t kind; /* 0 = SGD: w <- w - lr * g (the only optimiser of this build) */
  float lr;
} ringada_optim;

typedef struct ringada_stage ringada_stage;

/* ---------------------------------------------------------------- planning */

/* Host only (no device call).  Bytes of the activation stash and of the
 * scratch workspace that a forward + backward of (batch, seq) with cut-off
 * lowest_unfrozen needs.  The stash holds, for blocks l >= lowest_unfrozen, only
 * the tensors the early-stopped backward reads (Alg. 1: nothing below the
 * cut-off is back-propagated, so nothing below it is kept); blocks below the
 * cut-off and a fully frozen stage (lowest_unfrozen >= n_blocks) stash nothing.
 * Either output pointer may be NULL.  lowest_unfrozen < 0 stashes every block. */
ringada_status ringada_stage_plan(const ringada_stage_desc* desc, int32_t batch,
                                  int32_t seq, int32_t lowest_unfrozen,
                                  size_t* stash_bytes, size_t* scratch_bytes);

/* Host only.  Maps the unfreezing depth of Alg. 1 to the lowest_unfrozen
 * argument of a stage holding 0-indexed global blocks
 * [first_block, first_block + n_local) of an n_tm-block model.  The backward
 * ends at the (n_tm - depth + 1)-th block (1-indexed); Sec. III-B: a client
 * whose last block lies below it is forward-only (returns n_local), the one
 * holding it is the terminator (returns its local index), clients above it
 * return -1 (cut-off upstream: they must produce the input gradient).
 * Returns INT32_MIN for invalid arguments. */
int32_t ringada_local_cutoff(int32_t n_tm, int32_t depth, int32_t first_block,
                             int32_t n_local);

/* ---------------------------------------------------------------- lifetime */

/* Host only.  Bytes of the caller memory that holds what the library
 * derives from the weights:
 *   block_bytes: per block, passed to ringada_stage_bind_block: a transposed
 *     copy of each frozen projection matrix ([out, in], so that both operands
 *     of every forward product are contiguous along the contraction; post-LN
 *     bf16 stages with d_head 64 keep the QKV rows, and a copy of the QKV
 *     bias, in per-head order [Q_h K_h V_h]; pre-RMS stages interleave the
 *     gate and up rows in 32-row groups) and the adapters' working copies in
 *     the stage dtype (W_down, W_up and their transposes, fragment-packed in
 *     bf16 stages), 4 d m elements per adapter;
 *   stage_bytes: per stage, passed to ringada_stage_create: the rotary
 *     (cos, sin) table of the pre-RMS arch, max_seq x d_head/2 float pairs
 *     (0 for the post-LN arch).
 * Either output pointer may be NULL. */
ringada_status ringada_stage_plan_weights(const ringada_stage_desc* desc,
                                          size_t* block_bytes, size_t* stage_bytes);

/* Validates desc and creates a handle on the current HIP device.  stage_mem:
 * device memory of at least the stage_bytes of ringada_stage_plan_weights
 * (may be NULL when that is 0), 256-byte aligned, owned by the caller and
 * borrowed until ringada_stage_destroy; the first ringada_stage_bind_block
 * fills it.  Allocates nothing; RINGADA_E_WORKSPACE if stage_mem is too
 * small. */
ringada_status ringada_stage_create(const ringada_stage_desc* desc, void* stage_mem,
                                    size_t stage_mem_bytes, ringada_stage** out);

/* Binds block `block` (0-indexed, local).  Frozen weights and the adapters
 * are borrowed; under RINGADA_PLACEMENT_FFN attn_adapter must be NULL (the
 * block has none), otherwise both are required.  block_mem: device memory of
 * at least the block_bytes of ringada_stage_plan_weights, 256-byte aligned,
 * owned by the caller, borrowed until ringada_stage_destroy; the library
 * writes into it the transposed projections (the frozen weights never
 * change, so the copies stay valid) and the adapters' working copies, which
 * every ringada_adapter_step refreshes.  Fills it on `stream` and
 * synchronises the stream before returning.  Allocates nothing;
 * RINGADA_E_WORKSPACE if block_mem is too small.  Binding a block again
 * replaces its bindings. */
ringada_status ringada_stage_bind_block(ringada_stage* st, int32_t block,
                                        const ringada_block_weights* frozen,
                                        const ringada_adapter* attn_adapter,
                                        const ringada_adapter* ffn_adapter,
                                        void* block_mem, size_t block_mem_bytes,
                                        void* stream);

/* Re-derives the adapter working copies from the fp32 masters (call after
 * writing the masters directly, e.g. when loading a checkpoint). */
ringada_status ringada_stage_sync_adapters(ringada_stage* st, void* stream);

/* Releases the handle (host memory only; every device buffer stays the
 * caller's). */
void ringada_stage_destroy(ringada_stage* st);

/* ---------------------------------------------------------------- hot path */

/* Forward through all n_blocks blocks: y = blocks(x), x and y [batch, seq, d]
 * (x and y must not overlap).  lowest_unfrozen = c selects what is stashed
 * for the backward (see ringada_stage_plan); stash/scratch are caller buffers
 * of at least the planned sizes and must stay untouched until the matching
 * backward has been enqueued.
 * State machine: with c < n_blocks the handle becomes "pending" and every
 * further forward (a frozen one included) returns RINGADA_E_STATE until
 * ringada_stage_backward has been called; with c >= n_blocks (frozen stage)
 * nothing is left pending, so such forwards may follow each other. */
ringada_status ringada_stage_forward(ringada_stage* st, void* stream,
                                     const void* x, void* y, int32_t batch,
                                     int32_t seq, int32_t lowest_unfrozen,
                                     void* stash, size_t stash_bytes,
                                     void* scratch, size_t scratch_bytes);

/* Early-stopped backward of the pending forward.  dy [batch, seq, d] is the
 * gradient at the stage output.  For blocks l >= max(c, 0), from the top
 * down: activation gradients through the frozen weights (no frozen weight
 * gradient is formed) and the adapters' weight gradients, ADDED into their
 * g_down / g_up.  With 0 <= c < n_blocks the pass ends after the lowest
 * adapter of block c (its weight gradients are the last thing computed):
 * the attention adapter, or under RINGADA_PLACEMENT_FFN the FFN adapter, so
 * that block's FFN, norms and attention are not back-propagated at all;
 * with c < 0 the gradient w.r.t. the stage input is written to dx_in.
 * dx_in must be non-NULL iff c < 0.  c must be >= the forward's cut-off
 * (else RINGADA_E_STATE: the stash does not reach that deep), and < n_blocks.
 * Clears the pending state. */
ringada_status ringada_stage_backward(ringada_stage* st, void* stream,
                                      const void* dy, int32_t lowest_unfrozen,
                                      void* dx_in);

/* Update of the unfrozen adapters (blocks l >= max(c, 0)) from their
 * accumulated gradients (Sec. III-B: clients with unfrozen adapters update
 * them), then zero the gradients and refresh the working copies.  Returns
 * RINGADA_E_STATE while a forward is pending its backward (the backward
 * must see the weights the forward used). */
ringada_status ringada_adapter_step(ringada_stage* st, void* stream,
                                    int32_t lowest_unfrozen,
                                    const ringada_optim* opt);

/* ---------------------------------------------------------------- initiator helpers
 * Alg. 1: the initiator computes the loss on the last block's output and
 * updates the head; these produce the dy that enters the backward. */

/* Mean squared error over n elements: dy = 2 (y - target) / n, *loss = mean.
 * y, target, dy in `dtype`; loss is one device float (may be NULL). */
ringada_status ringada_loss_mse(void* stream, int32_t dtype, const void* y,
                                const void* target, int64_t n, void* dy,
                                float* loss);

/* Linear head on position 0 of each sequence + softmax cross-entropy, mean
 * over the batch.  y, dy: [batch, seq, d] in `dtype` (dy is fully written:
 * zero except position 0); w_h [d, n_classes] and b_h [n_classes] fp32;
 * labels [batch] int32 in [0, n_classes); the fp32 gradients g_wh, g_bh and
 * the mean loss (one device float, may be NULL) are ADDED into: zero them
 * before the first call of an accumulation.  n_classes <= 16; d a multiple of
 * 8; y, dy and w_h 16-B aligned.  Every sum runs over the samples in a fixed
 * order: the same inputs give the same bits. */
ringada_status ringada_head_ce(void* stream, int32_t dtype, const void* y,
                               int32_t batch, int32_t seq, int32_t d,
                               const float* w_h, const float* b_h,
                               int32_t n_classes, const int32_t* labels,
                               void* dy, float* g_wh, float* g_bh, float* loss);

/* w <- w - lr * g; g <- 0, over n fp32 values (the head update). */
ringada_status ringada_sgd_f32(void* stream, float* w, float* g, int64_t n,
                               float lr);

/* ---------------------------------------------------------------- diagnostics */

/* Thread-local message of the last failing call ("" if none). */
const char* ringada_last_error(void);

/* Per-kernel timing with HIP events.  After ringada_prof_begin every launch
 * the handle makes is bracketed by two events on its stream; ringada_prof_end
 * synchronises those events and returns, per kernel name, the number of
 * launches, their summed duration and the summed algorithmic work (FLOPs of
 * the contraction; minimum HBM bytes read + written). */
typedef struct {
  char name[64];
  int32_t launches;
  double total_ms;
  double flops;
  double bytes;
} ringada_prof_entry;

ringada_status ringada_prof_begin(ringada_stage* st);
ringada_status ringada_prof_end(ringada_stage* st, ringada_prof_entry* out,
                                int32_t max_entries, int32_t* n_entries);

#ifdef __cplusplus
}
#endif
#endif /* RINGADA_H */
