"""The per-block lookup table the ring simulation replays (Sec. IV: per-layer
forward and backward times profiled into a table), measured on the GPU
through the stage API for one BERT-base-shaped block (batch 32, seq 128,
d 768): every entry positive; a forward that stashes for the backward is
not faster than a frozen one (it writes more); the terminator's block, whose
backward ends at its lowest adapter (Alg. 1), is cheaper than a fully
back-propagated block."""
import pytest

from paper_2502_19864_amd.ringsim import measure_table
from paper_2502_19864_amd.workloads import WORKLOADS

pytestmark = pytest.mark.gpu


def test_measure_table_on_a_bert_base_block():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    w = WORKLOADS["bert_base"]
    t = measure_table(w, repeats=10)
    print(f"[table] {t.to_json()}", flush=True)
    for k in ("fwd_frozen", "fwd_stash", "bwd_full", "bwd_cut", "step", "head"):
        assert getattr(t, k) > 0, k
    assert t.fwd_frozen <= 1.1 * t.fwd_stash  # event timing noise of ~10 %
    assert t.bwd_cut < t.bwd_full
    assert t.act_bytes == w.batch * w.seq * w.d_model * 2
