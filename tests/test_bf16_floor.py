"""Pins the bf16 noise floor of the LLaMA-7B-share workload (8 pre-RMS
blocks, d = 4096, causal prefix of 64 tokens of sample 0, cut-off at local
block 6): storing the intermediates in bf16 moves the top adapters' weight
gradients by more than 2e-2 (max |.| / max |ref|) even when every other step
is exact, so the parity bound of that workload is derived from this floor."""
import numpy as np

from bf16_floor import llama_floor
from paper_2502_19864_amd.workloads import WORKLOADS, make_inputs


def test_llama_share_bf16_floor_exceeds_two_percent():
    w = WORKLOADS["llama7b_share"]
    inp = make_inputs(w)
    dy = np.zeros_like(inp["dy"])
    dy[0, :64] = inp["dy"][0, :64]
    fl = llama_floor(w, inp, w.lowest_unfrozen, dy, batch=1, seq=64)
    for k, v in sorted(fl.items(), key=str):
        print(k, "%.3e" % v)
    assert fl[(7, 1, "w_down")] > 2e-2
    assert max(fl.values()) < 0.1
