"""Python front end of one ring stage: owns the device tensors (allocated with
torch, which is used for device memory and streams only) and calls the C ABI
for all compute."""
from __future__ import annotations

import numpy as np

from . import binding as B
from .workloads import Workload


def _torch():
    import torch
    return torch


def make_desc(w: Workload, max_batch=None, max_seq=None):
    return B.StageDesc(
        arch=B.ARCH_POSTLN_GELU if w.arch == "bert" else B.ARCH_PRERMS_SWIGLU,
        dtype=B.BF16 if w.dtype == "bf16" else B.F32,
        n_blocks=w.n_blocks, d_model=w.d_model, n_heads=w.n_heads, d_ffn=w.d_ffn,
        d_adapter=w.d_adapter, max_batch=max_batch or w.batch, max_seq=max_seq or w.seq,
        norm_eps=1e-12 if w.arch == "bert" else 1e-6, rope_theta=10000.0,
        placement=B.PLACEMENT_FFN if w.placement == "ffn" else B.PLACEMENT_HOULSBY)


BERT_MAP = (("w_qkv", "w_qkv"), ("b_qkv", "b_qkv"), ("w_o", "w_o"), ("b_o", "b_o"),
            ("norm1_g", "ln1_g"), ("norm1_b", "ln1_b"), ("w_in", "w_i"), ("b_in", "b_i"),
            ("w_out", "w_f"), ("b_out", "b_f"), ("norm2_g", "ln2_g"), ("norm2_b", "ln2_b"))
LLAMA_MAP = (("w_qkv", "w_qkv"), ("w_o", "w_o"), ("norm1_g", "rms1_g"), ("w_in", "w_gu"),
             ("w_out", "w_d"), ("norm2_g", "rms2_g"))


class Stage:
    """One stage on cuda:`device`, bound to the weights/adapters of `inputs`
    (the dict of workloads.make_inputs)."""

    def __init__(self, w: Workload, inputs, device=0, max_batch=None, max_seq=None):
        torch = _torch()
        self.torch = torch
        self.w = w
        self.dev = torch.device("cuda", device)
        self.sdtype = torch.bfloat16 if w.dtype == "bf16" else torch.float32
        self.desc = make_desc(w, max_batch, max_seq)
        # every device buffer is ours: the library's derived copies of the
        # weights live in one region per block and one per stage
        self.block_bytes, stage_bytes = B.ringada_stage_plan_weights(self.desc)
        self.stage_mem = torch.empty(max(stage_bytes, 256), dtype=torch.uint8, device=self.dev)
        self.handle = B.ringada_stage_create(self.desc, self.stage_mem, self.stage_mem.numel())
        self.frozen = []
        self.adapters = []
        self.block_mem = []
        mp = BERT_MAP if w.arch == "bert" else LLAMA_MAP
        for l in range(w.n_blocks):
            tens = {k: self.upload(inputs["weights"][l][src]) for k, src in mp}
            self.frozen.append(tens)
            pair = []
            for a in range(2):
                ad = inputs["adapters"][l][a]
                t = dict(w_down=self.f32(ad["w_down"]), w_up=self.f32(ad["w_up"]),
                         g_down=torch.zeros(ad["w_down"].shape, dtype=torch.float32, device=self.dev),
                         g_up=torch.zeros(ad["w_up"].shape, dtype=torch.float32, device=self.dev))
                pair.append(t)
            self.adapters.append(pair)
            bw = B.BlockWeights(**{k: v.data_ptr() for k, v in tens.items()})
            ca = [B.Adapter(**{k: v.data_ptr() for k, v in t.items()}) for t in pair]
            self.block_mem.append(torch.empty(self.block_bytes, dtype=torch.uint8, device=self.dev))
            # the single placement binds no attention adapter (its tensors
            # stay allocated here, untouched, so grads() keeps one layout)
            B.ringada_stage_bind_block(self.handle, l, bw, None if w.placement == "ffn" else ca[0], ca[1],
                                       self.block_mem[l], self.block_bytes, self.sptr)
        self.stash = self.scratch = None
        self.stash_bytes = self.scratch_bytes = 0

    # ------------------------------------------------------------ helpers
    @property
    def sptr(self):
        """The current torch stream of the device (calls are stream-ordered on
        it, so they can also be captured into a HIP graph)."""
        return self.torch.cuda.current_stream(self.dev).cuda_stream

    def upload(self, a):
        """float32 numpy (bf16-representable for bf16 stages) -> device tensor in the storage dtype."""
        return self.torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(self.dev).to(self.sdtype)

    def f32(self, a):
        return self.torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(self.dev)

    def empty(self, *shape):
        return self.torch.empty(shape, dtype=self.sdtype, device=self.dev)

    def ensure_workspace(self, batch, seq, c):
        st, sc = B.ringada_stage_plan(self.desc, batch, seq, c)
        if self.stash is None or self.stash_bytes < st:
            self.stash = self.torch.empty(max(st, 256), dtype=self.torch.uint8, device=self.dev)
            self.stash_bytes = self.stash.numel()
        if self.scratch is None or self.scratch_bytes < sc:
            self.scratch = self.torch.empty(max(sc, 256), dtype=self.torch.uint8, device=self.dev)
            self.scratch_bytes = self.scratch.numel()
        return st, sc

    # ------------------------------------------------------------ hot path
    def forward(self, x, y, c, batch=None, seq=None):
        batch = batch or x.shape[0]
        seq = seq or x.shape[1]
        self.ensure_workspace(batch, seq, c)
        B.ringada_stage_forward(self.handle, self.sptr, x, y, batch, seq, c, self.stash, self.stash_bytes,
                                self.scratch, self.scratch_bytes)

    def backward(self, dy, c, dx_in=None):
        B.ringada_stage_backward(self.handle, self.sptr, dy, c, dx_in)

    def step(self, c, lr):
        B.ringada_adapter_step(self.handle, self.sptr, c, lr)

    def grads(self):
        """[(attn, ffn)] of {'w_down', 'w_up'} float32 numpy gradient accumulators."""
        self.torch.cuda.synchronize(self.dev)
        return [tuple({"w_down": t["g_down"].cpu().numpy(), "w_up": t["g_up"].cpu().numpy()} for t in pair)
                for pair in self.adapters]

    def zero_grads(self):
        for pair in self.adapters:
            for t in pair:
                t["g_down"].zero_()
                t["g_up"].zero_()

    def close(self):
        if self.handle is not None:
            self.torch.cuda.synchronize(self.dev)
            B.ringada_stage_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
