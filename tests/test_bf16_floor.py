"""Pins the bf16 noise floors that the parity bounds of the bf16 workloads are
derived from (max |.| / max |ref| per tensor, with every step exact except the
bf16 storage roundings of the path):

* LLaMA-7B share (8 pre-RMS blocks, d = 4096, causal prefix of 64 tokens of
  sample 0, cut-off at local block 6): the top FFN adapter's W_down gradient
  moves by more than 2e-2;
* BERT-base stage (12 post-LN blocks, batch 32, seq 128, [CLS] loss): the top
  FFN adapter's W_up gradient moves by more than 1e-2, i.e. storage alone uses
  over half of the 2e-2 tolerance.  Its gradient is a sum over the 32 [CLS]
  rows only, so the noise of the forward (which reaches the loss gradient
  through the logits) does not average out."""
import numpy as np

from bf16_floor import bert_floor, llama_floor
from helpers import oracle_run
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


def test_bert_base_bf16_floor_of_the_top_ffn_adapter():
    w = WORKLOADS["bert_base"].replace(lowest_unfrozen=11)
    inp = make_inputs(w)
    ref = oracle_run(w, inp, 11)
    fl = bert_floor(w, inp, 11, ref)
    for k, v in sorted(fl.items(), key=str):
        print(k, "%.3e" % v)
    assert fl[(11, 1, "w_up")] > 1e-2
    assert fl["y"] > 5e-3
    assert max(fl.values()) < 0.05
