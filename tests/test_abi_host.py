"""Host-only checks of the C ABI (no GPU needed): the library loads and exports
every declared symbol; the planner, the cut-off mapping and argument
validation behave as documented in include/ringada.h."""
import os
import re

import pytest

from paper_2502_19864_amd import binding as B
from paper_2502_19864_amd.stage import make_desc
from paper_2502_19864_amd.workloads import SWEEP, WORKLOADS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
MiB = 1 << 20


def header_symbols():
    txt = open(os.path.join(ROOT, "include", "ringada.h")).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(ringada_[a-z0-9_]+)\s*\(", txt)))


def test_library_exports_every_declared_symbol():
    L = B.lib()
    syms = header_symbols()
    assert len(syms) >= 15
    for s in syms:
        assert hasattr(L, s), s
    # the binding declares exactly the header's functions
    assert sorted(n for n, _, _ in B.SIGNATURES) == syms


def plan_mib(wname, c, batch=None, seq=None):
    w = WORKLOADS[wname]
    st, sc = B.ringada_stage_plan(make_desc(w), batch or w.batch, seq or w.seq, c)
    return st / MiB, sc / MiB


def test_stash_planner_bert_base_sweep():
    # stash bytes per cut-off for the BERT-base stage (T = 4096, d = 768, F = 3072,
    # m = 64): a full block keeps qkv, o, lse, attn, u1, xhat1, rstd1, a1, f2,
    # u2, xhat2, rstd2 = 73.2 MiB; the cut-off block drops qkv, o, lse = 49.0 MiB
    expect = {11: 49.0, 9: 195.5, 8: 268.7, 6: 415.1, 3: 634.8, 0: 854.4, -1: 878.6}
    for c, mib in expect.items():
        got, _ = plan_mib("bert_base", c)
        assert abs(got - mib) < 0.05, (c, got, mib)
    assert set(SWEEP) <= set(expect)


def test_stash_planner_single_placement():
    # one adapter per block, after the FFN (T = 4096, d = 768, bf16): a full
    # block no longer keeps the attention adapter's input and down-projection
    # (attn 6 MiB, u1 0.5 MiB): 66.72 MiB; the cut-off block stops after its
    # FFN adapter and keeps only f2, u2 and LN2's xhat2, rstd2: 12.52 MiB
    expect = {11: 12.52, 8: 3 * 66.72 + 12.52, -1: 12 * 66.72}
    for c, mib in expect.items():
        got, _ = plan_mib("bert_base_single", c)
        assert abs(got - mib) < 0.05, (c, got, mib)
    # the scratch keeps each back-propagated adapter's output and bottleneck
    # gradients (dz 6 MiB, du 0.5 MiB) and gelu(U) (0.5 MiB, the W_up
    # gradient's operand) for the weight-gradient launch at the end of the
    # backward: at c = 8 the two-adapter stage has four more
    diff = plan_mib("bert_base", 8)[1] - plan_mib("bert_base_single", 8)[1]
    assert abs(diff - 4 * 7.0) < 1e-6, diff


def test_stash_planner_other_workloads():
    assert abs(plan_mib("llama7b_share", 6)[0] - 349.3) < 0.1
    assert abs(plan_mib("bert_large_share", 3)[0] - 259.6) < 0.1
    # a frozen stage stashes nothing; the tiny stage at c = 0 stashes 1.3 MiB
    assert plan_mib("bert_base", 12)[0] == 0
    assert plan_mib("bert_base", 100)[0] == 0
    assert abs(plan_mib("tiny", 0)[0] - 1.3) < 0.05


def test_stash_is_monotone_in_the_cutoff():
    prev = None
    for c in range(12, -2, -1):
        st, sc = plan_mib("bert_base", c)
        assert prev is None or st >= prev
        prev = st
        assert sc > 0


def test_local_cutoff_matches_the_four_client_example():
    # 4:5:2:3 blocks over 14, depth 3: clients 1..3 forward-only, client 4
    # terminator at its first block
    starts, sizes = [0, 4, 9, 11], [4, 5, 2, 3]
    got = [B.ringada_local_cutoff(14, 3, s, n) for s, n in zip(starts, sizes)]
    assert got == [4, 5, 2, 0]
    # deeper unfreezing: the cut-off moves into client 2 (block 6 of 14 for depth 9)
    got = [B.ringada_local_cutoff(14, 9, s, n) for s, n in zip(starts, sizes)]
    assert got == [4, 1, -1, -1]
    assert B.ringada_local_cutoff(12, 4, 0, 12) == 8
    assert B.ringada_local_cutoff(12, 0, 0, 12) == 12
    assert B.ringada_local_cutoff(0, 1, 0, 1) < -1000
    assert B.ringada_local_cutoff(10, 11, 0, 10) < -1000


def test_plan_and_create_validate_arguments():
    w = WORKLOADS["bert_base"]
    desc = make_desc(w)
    with pytest.raises(B.RingadaError) as e:
        B.ringada_stage_plan(desc, w.batch + 1, w.seq, 8)
    assert e.value.status == B.RINGADA_E_INVALID
    for batch, seq in ((0, w.seq), (w.batch, 0), (-1, 1)):  # empty or negative sizes
        with pytest.raises(B.RingadaError) as e:
            B.ringada_stage_plan(desc, batch, seq, 8)
        assert e.value.status == B.RINGADA_E_INVALID
    bad = make_desc(w)
    bad.d_adapter = 48
    with pytest.raises(B.RingadaError) as e:
        B.ringada_stage_create(bad, None, 0)
    assert e.value.status == B.RINGADA_E_UNSUPPORTED
    bad = make_desc(w)
    bad.n_heads = 7
    with pytest.raises(B.RingadaError) as e:
        B.ringada_stage_plan(bad, 1, 1, 0)
    assert e.value.status == B.RINGADA_E_INVALID
    bad = make_desc(w)
    bad.placement = 2
    with pytest.raises(B.RingadaError) as e:
        B.ringada_stage_create(bad, None, 0)
    assert e.value.status == B.RINGADA_E_INVALID
    bad = make_desc(WORKLOADS["llama7b_share"])
    bad.dtype = B.F32
    with pytest.raises(B.RingadaError) as e:
        B.ringada_stage_create(bad, None, 0)
    assert e.value.status == B.RINGADA_E_UNSUPPORTED


def test_weight_memory_plan():
    """The caller-owned regions for the library's derived copies: per block the
    transposed projections (plus the per-head-order QKV bias of post-LN bf16
    stages with d_head 64) and four working copies per adapter, each at a
    256-B aligned offset; per stage the rotary table of the pre-RMS arch."""
    def al(n):
        return (n + 255) // 256 * 256

    # bert_base: d 768, F 3072, m 64, bf16, per-head QKV order, two adapters
    d, F, m = 768, 3072, 64
    blk, stg = B.ringada_stage_plan_weights(make_desc(WORKLOADS["bert_base"]))
    assert blk == al(3 * d * d * 2) + al(3 * d * 2) + al(d * d * 2) + 2 * al(F * d * 2) + 8 * al(d * m * 2)
    assert blk == 14_946_816 and stg == 0
    # single placement: one adapter's working copies fewer
    blk1, _ = B.ringada_stage_plan_weights(make_desc(WORKLOADS["bert_base_single"]))
    assert blk - blk1 == 4 * al(d * m * 2)
    # llama7b_share: d 4096, SwiGLU 11008 (gate and up packed), no biases; the
    # rotary table max_seq 512 x d_head/2 64 float pairs
    d, F = 4096, 11008
    blk, stg = B.ringada_stage_plan_weights(make_desc(WORKLOADS["llama7b_share"]))
    assert blk == al(3 * d * d * 2) + al(d * d * 2) + al(2 * F * d * 2) + al(F * d * 2) + 8 * al(d * m * 2)
    assert stg == 512 * 64 * 8
    # the tiny fp32 stage: 4-byte elements, no per-head order
    d, F, m = 128, 512, 16
    blk, stg = B.ringada_stage_plan_weights(make_desc(WORKLOADS["tiny"]))
    assert blk == al(3 * d * d * 4) + al(d * d * 4) + 2 * al(F * d * 4) + 8 * al(d * m * 4)
    assert stg == 0


def test_create_checks_the_stage_memory():
    desc = make_desc(WORKLOADS["llama7b_share"])
    _, stg = B.ringada_stage_plan_weights(desc)
    with pytest.raises(B.RingadaError) as e:
        B.ringada_stage_create(desc, None, 0)
    assert e.value.status == B.RINGADA_E_WORKSPACE
    with pytest.raises(B.RingadaError) as e:
        B.ringada_stage_create(desc, 1 << 20, stg - 1)
    assert e.value.status == B.RINGADA_E_WORKSPACE
    with pytest.raises(B.RingadaError) as e:  # 256-B alignment
        B.ringada_stage_create(desc, (1 << 20) + 16, stg)
    assert e.value.status == B.RINGADA_E_INVALID
    h = B.ringada_stage_create(desc, 1 << 20, stg)  # host-side only: the address is not touched
    B.ringada_stage_destroy(h)


def test_state_machine_on_an_unbound_stage():
    """Calls out of order fail with E_STATE before touching the device."""
    w = WORKLOADS["tiny"]
    h = B.ringada_stage_create(make_desc(w), None, 0)
    try:
        with pytest.raises(B.RingadaError) as e:
            B.ringada_stage_forward(h, None, 16, 4096, w.batch, w.seq, 0, 0, 0, 0, 0)
        assert e.value.status == B.RINGADA_E_STATE          # blocks not bound
        with pytest.raises(B.RingadaError) as e:
            B.ringada_stage_backward(h, None, 16, 0, None)
        assert e.value.status == B.RINGADA_E_STATE          # nothing pending
        with pytest.raises(B.RingadaError) as e:
            B.ringada_adapter_step(h, None, 0, 0.1, kind=1)
        assert e.value.status == B.RINGADA_E_UNSUPPORTED    # only SGD
        assert "SGD" in B.ringada_last_error()
    finally:
        B.ringada_stage_destroy(h)
