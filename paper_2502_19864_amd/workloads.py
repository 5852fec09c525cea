"""Seeded synthetic workloads for the stage path.

This module only draws random numbers and rounds them to the storage
precision.  It holds none of the method's arithmetic, and it is the one piece
of code that both the HIP path's tests/benchmark and the oracle are fed from.

The mBERT weights, SQuAD and the MAD-X adapters used in the paper's
evaluation are not available, so every input is synthetic: Gaussian hidden
states, Gaussian frozen weights and adapters, random labels or a random
incoming gradient, with the model shapes of the five workloads below.
"""
from __future__ import annotations

import dataclasses

import numpy as np

# names of the frozen tensors of one block, in draw order, with their shapes
# as functions of (d, F).  Every weight is stored [in, out].
BERT_WEIGHTS = (
    ("w_qkv", lambda d, F: (d, 3 * d), "w"),
    ("b_qkv", lambda d, F: (3 * d,), "b"),
    ("w_o", lambda d, F: (d, d), "w"),
    ("b_o", lambda d, F: (d,), "b"),
    ("ln1_g", lambda d, F: (d,), "g"),
    ("ln1_b", lambda d, F: (d,), "b"),
    ("w_i", lambda d, F: (d, F), "w"),
    ("b_i", lambda d, F: (F,), "b"),
    ("w_f", lambda d, F: (F, d), "w"),
    ("b_f", lambda d, F: (d,), "b"),
    ("ln2_g", lambda d, F: (d,), "g"),
    ("ln2_b", lambda d, F: (d,), "b"),
)
LLAMA_WEIGHTS = (
    ("rms1_g", lambda d, F: (d,), "g"),
    ("w_qkv", lambda d, F: (d, 3 * d), "w"),
    ("w_o", lambda d, F: (d, d), "w"),
    ("rms2_g", lambda d, F: (d,), "g"),
    ("w_gu", lambda d, F: (d, 2 * F), "w"),
    ("w_d", lambda d, F: (F, d), "w"),
)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    arch: str            # 'bert' (post-LN, GELU) or 'llama' (pre-RMS, SwiGLU, RoPE, causal)
    dtype: str           # 'f32' or 'bf16' storage
    n_blocks: int
    d_model: int
    n_heads: int
    d_ffn: int
    d_adapter: int
    seq: int
    batch: int
    lowest_unfrozen: int
    loss: str            # 'mse' | 'cls_ce' | 'dy'
    seed: int
    tiny_adapter_init: bool = False
    placement: str = "houlsby"  # or 'ffn': one adapter per block, after the FFN

    def replace(self, **kw):
        return dataclasses.replace(self, **kw)

    @property
    def tokens(self):
        return self.batch * self.seq


WORKLOADS = {
    # 2 post-LN blocks, d=128, 2 heads, FFN 512, seq 32, batch 4, bottleneck
    # 16, all adapters unfrozen, MSE against a seeded target, fp32.
    "tiny": Workload("tiny", "bert", "f32", 2, 128, 2, 512, 16, 32, 4, 0,
                     "mse", 1001, tiny_adapter_init=True),
    # BERT-base shaped stage: 12 blocks, d=768, 12 heads, FFN 3072, seq 128,
    # batch 32, bottleneck 64, top 4 blocks unfrozen, [CLS] 2-class head.
    "bert_base": Workload("bert_base", "bert", "bf16", 12, 768, 12, 3072, 64,
                          128, 32, 8, "cls_ce", 1002),
    # the unfreezing sweep runs bert_base with lowest_unfrozen in SWEEP
    "bert_base_sweep": Workload("bert_base_sweep", "bert", "bf16", 12, 768, 12,
                                3072, 64, 128, 32, 8, "cls_ce", 1003),
    # 6 consecutive BERT-large blocks: d=1024, 16 heads, FFN 4096, seq 256,
    # batch 16, cut-off at local block 3, incoming dY ~ N(0, 1e-2).
    "bert_large_share": Workload("bert_large_share", "bert", "bf16", 6, 1024,
                                 16, 4096, 64, 256, 16, 3, "dy", 1004),
    # 8 consecutive LLaMA-7B blocks: d=4096, 32 heads, SwiGLU 11008, seq 512,
    # batch 4, top 2 blocks unfrozen, incoming dY ~ N(0, 1e-2).
    "llama7b_share": Workload("llama7b_share", "llama", "bf16", 8, 4096, 32,
                              11008, 64, 512, 4, 6, "dy", 1005),
    # bert_base with the single serial adapter per block (after the FFN
    # sublayer, as in the paper's own set-up), cut-off at block 8.
    "bert_base_single": Workload("bert_base_single", "bert", "bf16", 12, 768,
                                 12, 3072, 64, 128, 32, 8, "cls_ce", 1006,
                                 placement="ffn"),
}
SWEEP = (11, 9, 6, 3, 0)


def round_to_bf16(a):
    """Round float32 values to the nearest bfloat16 (ties to even); returns
    float32 holding bf16-representable values.  Inputs must be finite."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    u = (u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))) \
        & np.uint32(0xFFFF0000)
    return u.view(np.float32)


def bf16_bits(a):
    """uint16 bit patterns of float32 values that are already bf16."""
    return (np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
            >> np.uint32(16)).astype(np.uint16)


def _normal(rng, shape, std, dtype_store):
    a = rng.standard_normal(shape, dtype=np.float32) * np.float32(std)
    return round_to_bf16(a) if dtype_store == "bf16" else a


def make_inputs(w: Workload, seed=None):
    """Draw every input of one iteration, in a fixed order: x, frozen weights
    block by block, adapters block by block (attention then FFN, down then
    up), head/labels or target, incoming dY.

    Returns a dict of float32 numpy arrays (bf16-representable for bf16
    workloads).  Frozen weights ~ N(0, 0.02); biases ~ N(0, 0.02); norm gains
    1 + N(0, 0.02); LN betas ~ N(0, 0.02)."""
    rng = np.random.Generator(np.random.PCG64(w.seed if seed is None else seed))
    st = w.dtype
    d, F, m = w.d_model, w.d_ffn, w.d_adapter
    out = {"x": _normal(rng, (w.batch, w.seq, d), 1.0, st)}
    spec = BERT_WEIGHTS if w.arch == "bert" else LLAMA_WEIGHTS
    weights = []
    for _ in range(w.n_blocks):
        blk = {}
        for name, shape_fn, kind in spec:
            shape = shape_fn(d, F)
            if kind == "g":
                a = np.float32(1.0) + rng.standard_normal(shape, dtype=np.float32) * np.float32(0.02)
                blk[name] = round_to_bf16(a) if st == "bf16" else a
            else:
                blk[name] = _normal(rng, shape, 0.02, st)
        weights.append(blk)
    out["weights"] = weights
    adapters = []
    for _ in range(w.n_blocks):
        pair = []
        for _ in range(2):
            w_down = rng.standard_normal((d, m), dtype=np.float32) * np.float32(0.02)
            if w.tiny_adapter_init:
                # up-projection zero-initialised, then perturbed by N(0, 1e-3)
                w_up = np.zeros((m, d), np.float32) + \
                    rng.standard_normal((m, d), dtype=np.float32) * np.float32(1e-3)
            else:
                w_up = rng.standard_normal((m, d), dtype=np.float32) * np.float32(0.02)
            pair.append({"w_down": w_down, "w_up": w_up})
        adapters.append(tuple(pair))
    # fp32 master weights; the bf16 path computes with their bf16 rounding
    out["adapters"] = adapters
    if w.loss == "mse":
        out["target"] = rng.standard_normal((w.batch, w.seq, d), dtype=np.float32)
    elif w.loss == "cls_ce":
        out["w_h"] = rng.standard_normal((d, 2), dtype=np.float32) * np.float32(0.02)
        out["b_h"] = np.zeros((2,), np.float32)
        out["labels"] = rng.integers(0, 2, size=(w.batch,), dtype=np.int32)
    else:
        out["dy"] = _normal(rng, (w.batch, w.seq, d), 1e-2, st)
    return out


def adapters_as_computed(w: Workload, adapters):
    """The adapter weights the storage precision computes with: the bf16 path
    multiplies with the bf16 rounding of the fp32 masters."""
    if w.dtype != "bf16":
        return adapters
    return [tuple({k: round_to_bf16(v) for k, v in a.items()} for a in pair)
            for pair in adapters]
