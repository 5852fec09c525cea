"""Parity of the HIP stage path with the float64 oracle, through the C ABI.

Measure: max |gpu - oracle| / max |oracle| per output tensor (Y, dX, every
adapter gradient, the head gradient).  Bounds: 1e-4 for the fp32 path; for
bf16 storage with fp32 accumulation 2e-2, or 1.25 times the tensor's bf16
storage floor where that floor leaves less room under 2e-2
(tests/bf16_floor.py: the oracle re-run with every bf16 store of the path's
forward and backward rounded).  Every margin is recorded (helpers.Checker)
and printed at the end of the session."""
import numpy as np
import pytest

from bf16_floor import rel_err_parts, stage_floor
from gpu_run import run_gpu
from helpers import TOL, Checker, oracle_run, rel_err
import oracle as O
from paper_2502_19864_amd import binding as B
from paper_2502_19864_amd.stage import Stage, make_desc
from paper_2502_19864_amd.workloads import SWEEP, WORKLOADS, Workload, make_inputs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()  # fails loudly if the library is not built
    return torch


SMALL = {
    # ragged sizes: T = 210 / 200 tokens do not fill the 16-token rows, the
    # 64/128-row GEMM tiles or the 128-key attention tiles
    "small_bert": Workload("small_bert", "bert", "bf16", 3, 256, 4, 512, 64, 70, 3, 1, "dy", 2001),
    "small_llama_dh128": Workload("small_llama_dh128", "llama", "bf16", 3, 256, 2, 384, 64, 100, 2, 1,
                                  "dy", 2002),
    "small_llama_dh64": Workload("small_llama_dh64", "llama", "bf16", 2, 256, 4, 320, 64, 77, 2, 0,
                                 "dy", 2003),
    "tiny_ragged": Workload("tiny_ragged", "bert", "f32", 2, 128, 2, 512, 16, 37, 3, 0, "dy", 2004,
                            tiny_adapter_init=True),
    # the single serial adapter per block, after the FFN sublayer
    "small_bert_single": Workload("small_bert_single", "bert", "bf16", 3, 256, 4, 512, 64, 100, 2, 1,
                                  "dy", 2005, placement="ffn"),
    "small_llama_single": Workload("small_llama_single", "llama", "bf16", 3, 256, 2, 384, 64, 100, 2, 1,
                                   "dy", 2006, placement="ffn"),
    "tiny_single": Workload("tiny_single", "bert", "f32", 3, 128, 2, 512, 16, 37, 3, 1, "dy", 2007,
                            tiny_adapter_init=True, placement="ffn"),
    # seq 128 at d_head 64: the attention runs in the QKV projection's epilogue
    # (one 128x192 tile per head and sequence), here on only 8 tiles; at the
    # cut-off c = 1 block 0 keeps no projections, at c = -1 every block does
    "small_bert_s128": Workload("small_bert_s128", "bert", "bf16", 3, 256, 4, 512, 64, 128, 2, 1, "dy", 2011),
    # d = 512: the row kernels' two-run (512 features per token) instantiation, T = 135
    "small_bert_d512": Workload("small_bert_d512", "bert", "bf16", 2, 512, 8, 1024, 64, 45, 3, 0, "dy", 2012),
    # seq 300: three 128-query tiles, the last one ragged (44 rows), so the
    # causal multi-tile forward (online softmax over 1-3 key tiles, diagonal
    # masks), the separate dQ and dK/dV backward passes with their causal tile
    # ranges, and the heaviest-first tile order (nq = 3 > 1) all run; at
    # d_head 128 and 64, at the cut-off and with the input gradient (c = -1)
    "small_llama_s300_dh128": Workload("small_llama_s300_dh128", "llama", "bf16", 2, 256, 2, 384, 64, 300, 2, 1,
                                       "dy", 2013),
    "small_llama_s300_dh64": Workload("small_llama_s300_dh64", "llama", "bf16", 2, 256, 4, 384, 64, 300, 2, 0,
                                      "dy", 2014),
    # the bidirectional multi-tile path on a ragged length (three key tiles)
    "small_bert_s300": Workload("small_bert_s300", "bert", "bf16", 2, 256, 4, 512, 64, 300, 2, 0, "dy", 2015),
    # degenerate shapes: one-token sequences (attention over a single key is V
    # itself; the rotary angle at position 0 is zero), fewer tokens than one
    # 16-token row tile or one GEMM row tile, the wide adapter path on 3 tokens
    "edge_bert_s1": Workload("edge_bert_s1", "bert", "bf16", 2, 256, 4, 512, 64, 1, 3, 0, "dy", 2016),
    "edge_llama_s1": Workload("edge_llama_s1", "llama", "bf16", 2, 256, 2, 384, 64, 1, 2, 1, "dy", 2017),
    "edge_bert_t5": Workload("edge_bert_t5", "bert", "bf16", 2, 256, 4, 512, 64, 5, 1, 1, "dy", 2018),
    "edge_tiny_s1_f32": Workload("edge_tiny_s1_f32", "bert", "f32", 2, 128, 2, 512, 16, 1, 2, 0, "dy", 2019,
                                 tiny_adapter_init=True),
    "edge_wide_llama_t3": Workload("edge_wide_llama_t3", "llama", "bf16", 2, 2048, 16, 512, 64, 3, 1, 0, "dy", 2020),
}


def checker(tag, w, inp, c, ref, floor_c=None):
    """The Checker of one comparison: fp32 at 1e-4; bf16 with the per-tensor
    bounds of the emulated storage floor at cut-off `floor_c` (default c)."""
    if w.dtype == "f32":
        return Checker(tag, tol=TOL["f32"])
    fl = stage_floor(w, inp, c if floor_c is None else floor_c, ref)
    return Checker(tag, floor=fl)


def compare(chk, w, gpu, ref, c):
    chk("y", gpu["y"], ref["y"])
    if c < 0:
        chk("dx", gpu["dx"], ref["dx"])
    if "g_wh" in gpu and "g_wh" in ref:
        chk("g_wh", gpu["g_wh"], ref["g_wh"])
    chk.grads(gpu["grads"], ref["grads"], max(c, 0), w.n_blocks)


@pytest.mark.parametrize("name", sorted(SMALL))
def test_small_stage_parity(torch, name):
    w = SMALL[name]
    inp = make_inputs(w)
    st = Stage(w, inp)
    try:
        for c in (w.lowest_unfrozen, -1):
            print(f"[{name}] c={c}", flush=True)
            gpu = run_gpu(torch, st, w, inp, c, want_dx=(c < 0))
            ref = oracle_run(w, inp, c)
            chk = checker(f"{name} c={c}", w, inp, c, ref)
            compare(chk, w, gpu, ref, c)
            chk.done()
    finally:
        st.close()


def test_tiny_workload_parity_fp32(torch):
    w = WORKLOADS["tiny"]
    inp = make_inputs(w)
    st = Stage(w, inp)
    try:
        gpu = run_gpu(torch, st, w, inp, w.lowest_unfrozen)
        ref = oracle_run(w, inp, w.lowest_unfrozen)
        chk = Checker("tiny", tol=1e-4)
        compare(chk, w, gpu, ref, w.lowest_unfrozen)
        chk("loss", gpu["loss"][0], ref["loss"], err=abs(gpu["loss"][0] - ref["loss"]) / abs(ref["loss"]))
        # all adapters unfrozen and the cut-off upstream: the input gradient too
        gpu = run_gpu(torch, st, w, inp, -1, want_dx=True)
        ref = oracle_run(w, inp, -1)
        chk2 = Checker("tiny c=-1", tol=1e-4)
        compare(chk2, w, gpu, ref, -1)
        chk.done()
        chk2.done()
    finally:
        st.close()


@pytest.mark.timeout(600)
def test_bert_base_workload_parity(torch):
    """The benchmarked workload at full size: 12 blocks, batch 32, seq 128,
    cut-off at block 8, [CLS] head loss on the GPU; then the adapter step and
    a frozen forward with the updated adapters."""
    w = WORKLOADS["bert_base"]
    inp = make_inputs(w)
    st = Stage(w, inp)
    try:
        c = w.lowest_unfrozen
        gpu = run_gpu(torch, st, w, inp, c)
        ref = oracle_run(w, inp, c)
        chk = checker("bert_base", w, inp, c, ref)
        compare(chk, w, gpu, ref, c)
        chk("loss", gpu["loss"][0], ref["loss"], err=abs(gpu["loss"][0] - ref["loss"]) / abs(ref["loss"]))
        # adapter update (SGD), then a second forward with the updated adapters
        lr = 0.5
        st.step(c, lr)
        new_ad = O.sgd_step([tuple(dict(a) for a in p) for p in inp["adapters"]],
                            [g if l >= c else None for l, g in enumerate(ref["grads"])], lr)
        torch.cuda.synchronize()
        for l in range(w.n_blocks):
            for a in range(2):
                for k in ("w_down", "w_up"):
                    got = st.adapters[l][a][k].cpu().numpy()
                    old = inp["adapters"][l][a][k]
                    if l >= c:
                        # the applied step -lr * g matches the oracle's
                        chk(("step", l, a, k), got - old, new_ad[l][a][k] - old,
                            err=rel_err(got - old, new_ad[l][a][k] - old))
                    else:
                        assert np.array_equal(got, old), (l, a, k)
                    assert np.all(st.adapters[l][a]["g_" + k[2:]].cpu().numpy() == 0)
        inp2 = dict(inp, adapters=new_ad)
        gpu2 = run_gpu(torch, st, w, inp2, w.n_blocks)  # frozen forward, no backward
        ref2 = oracle_run(w, inp2, w.n_blocks)
        chk("y after step", gpu2["y"], ref2["y"], err=rel_err(gpu2["y"], ref2["y"]))
        chk.done()
    finally:
        st.close()


def _cutoff_runs(torch, cs):
    """bert_base at the cut-offs `cs` with one seeded incoming gradient."""
    from paper_2502_19864_amd.workloads import round_to_bf16
    w = WORKLOADS["bert_base"]
    inp = make_inputs(w)
    rng = np.random.default_rng(77)
    dy = round_to_bf16(rng.standard_normal(inp["x"].shape).astype(np.float32) * np.float32(1e-2))
    st = Stage(w, inp)
    try:
        return w, {c: run_gpu(torch, st, w, inp, c, dy=None if c >= w.n_blocks else dy, want_dx=c < 0)
                   for c in cs}
    finally:
        st.close()


def test_bert_base_cutoff_leaves_y_bitwise_unchanged(torch):
    """Early stopping only changes what is stashed, not the arithmetic: on
    the GPU itself Y is bitwise the same for a frozen forward (c = 12), the
    benchmark's cut-off 8, a deep cut-off 3 and a full backward (c = -1)."""
    frozen = WORKLOADS["bert_base"].n_blocks
    _, runs = _cutoff_runs(torch, (frozen, 8, 3, -1))
    for c in (8, 3, -1):
        assert np.array_equal(runs[c]["y"], runs[frozen]["y"]), c
    print("[cutoff invariance] Y bitwise equal at c = 12, 8, 3, -1", flush=True)


def test_bert_base_truncated_gradients_bitwise_equal_full(torch):
    """Alg. 1's backward ending at the (L-d+1)-th adapter computes, for the
    adapters it reaches, exactly what the full backward computes: on the GPU
    the gradients of blocks >= 8 (>= 3) after a backward stopped at block 8
    (3) are bitwise those of the backward to the stage input, and blocks
    below the cut-off get none."""
    w, runs = _cutoff_runs(torch, (8, 3, -1))
    for c in (8, 3):
        for l in range(w.n_blocks):
            for a in range(2):
                for k in ("w_down", "w_up"):
                    g, gall = runs[c]["grads"][l][a][k], runs[-1]["grads"][l][a][k]
                    if l >= c:
                        assert np.array_equal(g, gall), (c, l, a, k, float(np.abs(g - gall).max()))
                    else:
                        assert np.all(g == 0), (c, l, a, k)
    print("[cutoff invariance] dW bitwise equal to the full backward's for every unfrozen block", flush=True)


@pytest.mark.timeout(600)
def test_bert_base_unfreezing_sweep(torch):
    """Cut-off at blocks 11, 9, 6, 3, 0: the early-stopped gradients equal the
    full backward's for every unfrozen block."""
    w = WORKLOADS["bert_base_sweep"]
    inp = make_inputs(w)
    ref = oracle_run(w, inp, 0)
    # the truncated backward's gradients are the full backward's, so one floor
    # run at c = 0 covers every cut-off
    fl = stage_floor(w, inp, 0, ref)
    st = Stage(w, inp)
    try:
        for c in SWEEP:
            print(f"[sweep] c={c}", flush=True)
            gpu = run_gpu(torch, st, w, inp, c)
            chk = Checker(f"sweep c={c}", floor=fl)
            chk("y", gpu["y"], ref["y"])
            chk.grads(gpu["grads"], ref["grads"], c, w.n_blocks)
            chk.done()
    finally:
        st.close()


@pytest.mark.timeout(600)
def test_bert_base_single_placement_parity(torch):
    """BERT-base-shaped stage with one adapter per block (after the FFN): the
    backward ends after block 8's FFN adapter; the stash is the smaller plan."""
    w = WORKLOADS["bert_base_single"]
    inp = make_inputs(w)
    st = Stage(w, inp)
    try:
        gpu = run_gpu(torch, st, w, inp, w.lowest_unfrozen)
        ref = oracle_run(w, inp, w.lowest_unfrozen)
        chk = checker("bert_base_single", w, inp, w.lowest_unfrozen, ref)
        compare(chk, w, gpu, ref, w.lowest_unfrozen)
        chk.done()
        plan, _ = B.ringada_stage_plan(st.desc, w.batch, w.seq, w.lowest_unfrozen)
        two, _ = B.ringada_stage_plan(make_desc(w.replace(placement="houlsby")), w.batch, w.seq, w.lowest_unfrozen)
        assert plan < two
    finally:
        st.close()


@pytest.mark.timeout(600)
def test_bert_large_share_parity(torch):
    w = WORKLOADS["bert_large_share"]
    inp = make_inputs(w)
    st = Stage(w, inp)
    try:
        gpu = run_gpu(torch, st, w, inp, w.lowest_unfrozen)
        ref = oracle_run(w, inp, w.lowest_unfrozen)
        chk = checker("bert_large_share", w, inp, w.lowest_unfrozen, ref)
        compare(chk, w, gpu, ref, w.lowest_unfrozen)
        chk.done()
    finally:
        st.close()


@pytest.mark.timeout(900)
def test_llama_share_parity_full_sample(torch):
    """Full-size LLaMA share (8 pre-RMS causal blocks, d 4096, batch 4, seq
    512, cut-off at block 6) in the benchmark's launch configuration.  The
    incoming gradient is the workload's over all 512 positions of sample 0
    and over the first 64 positions of sample 3 (token rows 1536-1599, a
    different GEMM row tile), zero elsewhere.  Compared with the oracle: Y at
    all 512 positions of sample 0 and the first 64 of sample 3 (batch
    independence; causality for the prefix), and every adapter gradient,
    which the GPU sums over both samples.  All four 128-query tiles of the
    causal attention of sample 0 carry a nonzero gradient in the backward."""
    w = WORKLOADS["llama7b_share"]
    inp = make_inputs(w)
    c, P, last = w.lowest_unfrozen, 64, w.batch - 1
    dy = np.zeros_like(inp["dy"])
    dy[0] = inp["dy"][0]
    dy[last, :P] = inp["dy"][last, :P]
    st = Stage(w, inp)
    try:
        gpu = run_gpu(torch, st, w, inp, c, dy=dy)
    finally:
        st.close()
    print("[llama7b_share] GPU run done; oracle on sample 0 (512 tokens) and the prefix of sample 3", flush=True)
    parts = [(inp["x"][0:1], dy[0:1]), (inp["x"][last:last + 1, :P], dy[last:last + 1, :P])]
    refs = [oracle_run(w, inp, c, dy=d_, x=x_) for x_, d_ in parts]
    print("[llama7b_share] oracle done; bf16 storage floor", flush=True)
    fl = stage_floor(w, inp, c, refs, parts)
    chk = Checker("llama7b_share", floor=fl)
    chk("y", None, None, err=rel_err_parts([gpu["y"][0:1], gpu["y"][last:last + 1, :P]], [r["y"] for r in refs]))
    # the y error per query tile of sample 0 (each against the whole sample's scale)
    scale = np.abs(refs[0]["y"]).max()
    per_tile = [float(np.abs(gpu["y"][0, t:t + 128] - refs[0]["y"][0, t:t + 128]).max() / scale)
                for t in range(0, w.seq, 128)]
    print("[llama7b_share] y error per 128-token tile of sample 0: " + ", ".join(f"{e:.3e}" for e in per_tile),
          flush=True)
    gsum = [None if a is None else tuple(None if p is None else {k: p[k] + q[k] for k in p}
                                         for p, q in zip(a, b))
            for a, b in zip(refs[0]["grads"], refs[1]["grads"])]
    chk.grads(gpu["grads"], gsum, c, w.n_blocks)
    chk.done()


# d > 1024: the split-K down projection, the feature-chunked up projection
# and the separate row norms of the wide adapter path; T = 82 / 74 / 46
# tokens is not a multiple of the 16-token tiles.
WIDE = {
    "wide_llama_d2048": Workload("wide_llama_d2048", "llama", "bf16", 2, 2048, 16, 512, 64, 41, 2, 1, "dy",
                                 2008),
    "wide_bert_single_d2048": Workload("wide_bert_single_d2048", "bert", "bf16", 2, 2048, 16, 512, 64, 37, 2, 1,
                                       "dy", 2009, placement="ffn"),
    "wide_bert_d3072": Workload("wide_bert_d3072", "bert", "bf16", 2, 3072, 24, 256, 64, 23, 2, 0, "dy", 2010),
}


@pytest.mark.parametrize("name", sorted(WIDE))
def test_wide_adapter_parity(torch, name):
    w = WIDE[name]
    inp = make_inputs(w)
    st = Stage(w, inp)
    try:
        for c in (w.lowest_unfrozen, -1):
            print(f"[{name}] c={c}", flush=True)
            gpu = run_gpu(torch, st, w, inp, c, want_dx=(c < 0))
            ref = oracle_run(w, inp, c)
            chk = checker(f"{name} c={c}", w, inp, c, ref)
            compare(chk, w, gpu, ref, c)
            chk.done()
    finally:
        st.close()


def test_training_iterations_are_bitwise_reproducible(torch):
    """Two fresh stages on the same inputs, two Alg. 1 iterations each
    (forward, [CLS] head loss and head update, backward to the cut-off,
    adapter update): every adapter weight, the head and the last loss come
    out bit for bit the same.  No result of the path depends on the order in
    which workgroups finish (no floating-point atomics anywhere)."""
    w = Workload("rep_bert", "bert", "bf16", 3, 256, 4, 512, 64, 64, 8, 1, "cls_ce", 2301)
    inp = make_inputs(w)
    c, lr = w.lowest_unfrozen, 1e-2

    def train():
        st = Stage(w, inp)
        try:
            x = st.upload(inp["x"])
            y, dy = st.empty(*inp["x"].shape), st.empty(*inp["x"].shape)
            nwh = inp["w_h"].size
            hp = st.f32(np.concatenate([inp["w_h"].ravel(), inp["b_h"].ravel()]))
            hg = torch.zeros_like(hp)
            wh, bh, gwh, gbh = hp[:nwh].view(inp["w_h"].shape), hp[nwh:], hg[:nwh].view(inp["w_h"].shape), hg[nwh:]
            lab = torch.from_numpy(inp["labels"]).to(st.dev)
            loss = torch.zeros(1, dtype=torch.float32, device=st.dev)
            for _ in range(2):
                st.forward(x, y, c)
                loss.zero_()
                B.ringada_head_ce(st.sptr, st.desc.dtype, y, w.batch, w.seq, w.d_model, wh, bh, 2, lab, dy, gwh, gbh,
                                  loss)
                B.ringada_sgd_f32(st.sptr, hp, hg, hp.numel(), lr)
                st.backward(dy, c)
                st.step(c, lr)
            torch.cuda.synchronize()
            out = [hp.cpu().numpy(), loss.cpu().numpy(), y.float().cpu().numpy()]
            for pair in st.adapters:
                for t in pair:
                    out += [t["w_down"].cpu().numpy(), t["w_up"].cpu().numpy()]
            return out
        finally:
            st.close()

    first, second = train(), train()
    assert len(first) == len(second)
    for k, (a_, b_) in enumerate(zip(first, second)):
        assert np.array_equal(a_, b_), f"result {k} differs between two identical runs"
    # the updates did something: the trained adapters differ from their start
    assert not np.array_equal(first[3 + 2 * 2 * c], inp["adapters"][c][0]["w_down"].astype(np.float32))


def test_state_machine_and_workspace_errors(torch):
    w = SMALL["small_bert"]
    inp = make_inputs(w)
    st = Stage(w, inp)
    try:
        x = st.upload(inp["x"])
        y = st.empty(*inp["x"].shape)
        dy = st.upload(inp["dy"])
        sb, sc = B.ringada_stage_plan(st.desc, w.batch, w.seq, 1)
        st.ensure_workspace(w.batch, w.seq, -1)
        with pytest.raises(B.RingadaError) as e:  # workspace smaller than planned
            B.ringada_stage_forward(st.handle, st.sptr, x, y, w.batch, w.seq, 1, st.stash, sb - 1, st.scratch, sc)
        assert e.value.status == B.RINGADA_E_WORKSPACE
        st.forward(x, y, 1)
        with pytest.raises(B.RingadaError) as e:  # one forward, one backward
            st.forward(x, y, 1)
        assert e.value.status == B.RINGADA_E_STATE
        with pytest.raises(B.RingadaError) as e:  # nor a frozen forward over the pending stash
            st.forward(x, y, w.n_blocks)
        assert e.value.status == B.RINGADA_E_STATE
        with pytest.raises(B.RingadaError) as e:  # no update between a forward and its backward
            st.step(1, 0.1)
        assert e.value.status == B.RINGADA_E_STATE
        with pytest.raises(B.RingadaError) as e:  # the stash does not reach block 0
            st.backward(dy, 0)
        assert e.value.status == B.RINGADA_E_STATE
        with pytest.raises(B.RingadaError) as e:  # dx_in only when the cut-off is upstream
            st.backward(dy, 1, y)
        assert e.value.status == B.RINGADA_E_INVALID
        st.backward(dy, 2)  # stopping higher than the stash allows is fine
        with pytest.raises(B.RingadaError) as e:
            st.backward(dy, 2)
        assert e.value.status == B.RINGADA_E_STATE
        st.step(2, 0.0)  # nothing pending: the update is accepted
        # a frozen stage streams forwards back to back (nothing pending)
        st.forward(x, y, w.n_blocks)
        st.forward(x, y, w.n_blocks)
        with pytest.raises(B.RingadaError) as e:
            st.backward(dy, w.n_blocks)
        assert e.value.status == B.RINGADA_E_STATE
        # the norm gains and shifts must be 16-byte aligned (the row kernels
        # move 16 B per lane); refused before anything is bound
        bad = {k: v.data_ptr() for k, v in st.frozen[0].items()}
        bad["norm1_g"] += 2
        ca = [B.Adapter(**{k: v.data_ptr() for k, v in t.items()}) for t in st.adapters[0]]
        with pytest.raises(B.RingadaError) as e:
            B.ringada_stage_bind_block(st.handle, 0, B.BlockWeights(**bad), ca[0], ca[1], st.block_mem[0],
                                       st.block_bytes, st.sptr)
        assert e.value.status == B.RINGADA_E_INVALID
        st.forward(x, y, w.n_blocks)  # the stage is unchanged
        torch.cuda.synchronize()
    finally:
        st.close()
