"""The boundary's ownership rule, on the GPU: the library allocates no device
memory.  With every buffer allocated by the caller beforehand (frozen
weights, adapters, the per-stage and per-block regions of
ringada_stage_plan_weights, stash, scratch, activations), a whole cycle
through the C ABI -- create, bind every block, forward, early-stopped
backward, adapter step, destroy -- leaves the device's free memory
unchanged (after one warm-up cycle has loaded the library's code objects)."""
import numpy as np
import pytest

from paper_2502_19864_amd import binding as B
from paper_2502_19864_amd.stage import Stage
from paper_2502_19864_amd.workloads import Workload, make_inputs

pytestmark = pytest.mark.gpu

CASES = {
    # post-LN, d_head 64 at seq 128: per-head QKV order and the fused attention epilogue
    "bert_s128": Workload("mem_bert_s128", "bert", "bf16", 2, 256, 4, 512, 64, 128, 2, 0, "dy", 2201),
    # pre-RMS with RoPE: the rotary table lives in the per-stage region
    "llama": Workload("mem_llama", "llama", "bf16", 2, 256, 2, 384, 64, 200, 2, 0, "dy", 2202),
    # fp32 stage
    "tiny_f32": Workload("mem_tiny", "bert", "f32", 2, 128, 2, 512, 16, 32, 4, 0, "dy", 2203),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_library_allocates_no_device_memory(name):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()
    w = CASES[name]
    inp = make_inputs(w)
    st = Stage(w, inp)  # warm-up: create + bind through the Stage, then a full step
    try:
        x = st.upload(inp["x"])
        y = st.empty(*inp["x"].shape)
        dy = st.upload(inp["dy"])
        dx = st.empty(*inp["x"].shape)
        st.forward(x, y, -1)
        st.backward(dy, -1, dx)
        st.step(-1, 0.0)
        torch.cuda.synchronize()
        y_warm = y.float().cpu().numpy()
        free0 = torch.cuda.mem_get_info()[0]
        # a second handle on the same caller buffers, every call through the C ABI
        h = B.ringada_stage_create(st.desc, st.stage_mem, st.stage_mem.numel())
        try:
            for l in range(w.n_blocks):
                bw = B.BlockWeights(**{k: v.data_ptr() for k, v in st.frozen[l].items()})
                ca = [B.Adapter(**{k: v.data_ptr() for k, v in t.items()}) for t in st.adapters[l]]
                B.ringada_stage_bind_block(h, l, bw, None if w.placement == "ffn" else ca[0], ca[1],
                                           st.block_mem[l], st.block_bytes, st.sptr)
            B.ringada_stage_forward(h, st.sptr, x, y, w.batch, w.seq, -1, st.stash, st.stash_bytes, st.scratch,
                                    st.scratch_bytes)
            B.ringada_stage_backward(h, st.sptr, dy, -1, dx)
            B.ringada_adapter_step(h, st.sptr, -1, 0.0)
            torch.cuda.synchronize()
        finally:
            B.ringada_stage_destroy(h)
        torch.cuda.synchronize()
        free1 = torch.cuda.mem_get_info()[0]
        assert free1 == free0, (name, free0, free1)
        # the second handle computed what the first did (lr 0: same adapters)
        assert np.array_equal(y.float().cpu().numpy(), y_warm)
        print(f"[{name}] free device memory unchanged across create, bind, step, destroy: {free0} bytes", flush=True)
    finally:
        st.close()
