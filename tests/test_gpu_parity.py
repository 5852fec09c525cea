"""Parity of the HIP stage path with the float64 oracle, through the C ABI.

Tolerances (max |gpu - oracle| / max |oracle| per output tensor): 1e-4 for
the fp32 path, 2e-2 for bf16 storage with fp32 accumulation."""
import numpy as np
import pytest

from helpers import TOL, oracle_run, rel_err
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
    # 64/128-row GEMM tiles or the 64-key attention tiles
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
}


def run_gpu(torch, stage, w, inp, c, dy=None, want_dx=False):
    """Forward, (loss,) early-stopped backward on the GPU; returns numpy results.
    A cut-off at or above the top block runs the forward only."""
    x = stage.upload(inp["x"])
    y = stage.empty(*inp["x"].shape)
    stage.zero_grads()
    stage.forward(x, y, c)
    res = {}
    if c >= w.n_blocks:
        torch.cuda.synchronize()
        res["y"] = y.float().cpu().numpy()
        return res
    if dy is None and w.loss == "mse":
        dyt = stage.empty(*inp["x"].shape)
        loss = torch.zeros(1, dtype=torch.float32, device=stage.dev)
        B.ringada_loss_mse(stage.sptr, stage.desc.dtype, y, stage.upload(inp["target"]), y.numel(), dyt, loss)
        res["loss"] = loss
    elif dy is None and w.loss == "cls_ce":
        dyt = stage.empty(*inp["x"].shape)
        wh, bh = stage.f32(inp["w_h"]), stage.f32(inp["b_h"])
        gwh, gbh = torch.zeros_like(wh), torch.zeros_like(bh)
        lab = torch.from_numpy(inp["labels"]).to(stage.dev)
        loss = torch.zeros(1, dtype=torch.float32, device=stage.dev)
        B.ringada_head_ce(stage.sptr, stage.desc.dtype, y, w.batch, w.seq, w.d_model, wh, bh, 2, lab, dyt, gwh,
                          gbh, loss)
        res.update(loss=loss, g_wh=gwh, g_bh=gbh)
    else:
        dyt = stage.upload(inp["dy"] if dy is None else dy)
    dx = stage.empty(*inp["x"].shape) if want_dx else None
    stage.backward(dyt, -1 if want_dx else c, dx)
    torch.cuda.synchronize()
    res["y"] = y.float().cpu().numpy()
    res["dx"] = dx.float().cpu().numpy() if want_dx else None
    res["grads"] = stage.grads()
    for k in ("loss", "g_wh", "g_bh"):
        if k in res:
            res[k] = res[k].cpu().numpy()
    return res


def check_grads(gpu, ref, lo, L, tol, tag):
    """Every adapter gradient against the oracle; `tol` is a bound or a
    function of the tensor key (l, a, name)."""
    bound = tol if callable(tol) else (lambda key: tol)
    worst = 0.0
    for l in range(L):
        for a in range(2):
            for k in ("w_down", "w_up"):
                g = gpu["grads"][l][a][k]
                if l < lo or ref["grads"][l][a] is None:  # frozen, or no such adapter
                    assert np.all(g == 0), (tag, "gradient of a frozen or absent adapter", l, a, k)
                    continue
                e = rel_err(g, ref["grads"][l][a][k])
                worst = max(worst, e)
                assert e <= bound((l, a, k)), (tag, l, a, k, e, bound((l, a, k)))
    print(f"[{tag}] worst adapter-gradient error {worst:.3e}", flush=True)
    return worst


def floor_bounds(w, inp, c, ref):
    """Per-tensor bounds of a bf16 post-LN workload: 2e-2, or twice the bf16
    storage floor of the tensor (tests/bf16_floor.py) where that is larger."""
    from bf16_floor import bert_floor, floor_bound
    fl = bert_floor(w, inp, c, ref)
    over = {k: v for k, v in fl.items() if 2.0 * v > 2e-2}
    print(f"[{w.name}] bf16 storage floor: max {max(fl.values()):.3e}; bounds above 2e-2: "
          + ", ".join(f"{k}: {2 * v:.3e}" for k, v in sorted(over.items(), key=str)), flush=True)
    return lambda key: floor_bound(fl, key)


@pytest.mark.parametrize("name", sorted(SMALL))
def test_small_stage_parity(torch, name):
    w = SMALL[name]
    inp = make_inputs(w)
    tol = TOL[w.dtype]
    st = Stage(w, inp)
    try:
        for c in (w.lowest_unfrozen, -1):
            print(f"[{name}] c={c}", flush=True)
            gpu = run_gpu(torch, st, w, inp, c, want_dx=(c < 0))
            ref = oracle_run(w, inp, c)
            print(f"[{name}] c={c} y error {rel_err(gpu['y'], ref['y']):.3e}", flush=True)
            assert rel_err(gpu["y"], ref["y"]) <= tol
            check_grads(gpu, ref, max(c, 0), w.n_blocks, tol, name)
            if c < 0:
                assert rel_err(gpu["dx"], ref["dx"]) <= tol
    finally:
        st.close()


def test_tiny_workload_parity_fp32(torch):
    w = WORKLOADS["tiny"]
    inp = make_inputs(w)
    st = Stage(w, inp)
    try:
        gpu = run_gpu(torch, st, w, inp, w.lowest_unfrozen)
        ref = oracle_run(w, inp, w.lowest_unfrozen)
        assert rel_err(gpu["y"], ref["y"]) <= 1e-4
        assert abs(gpu["loss"][0] - ref["loss"]) <= 1e-4 * abs(ref["loss"])
        check_grads(gpu, ref, 0, w.n_blocks, 1e-4, "tiny")
        # all adapters unfrozen and the cut-off upstream: the input gradient too
        gpu = run_gpu(torch, st, w, inp, -1, want_dx=True)
        ref = oracle_run(w, inp, -1)
        assert rel_err(gpu["dx"], ref["dx"]) <= 1e-4
        check_grads(gpu, ref, 0, w.n_blocks, 1e-4, "tiny c=-1")
    finally:
        st.close()


def test_bert_base_workload_parity(torch):
    """The benchmarked workload at full size: 12 blocks, batch 32, seq 128,
    cut-off at block 8, [CLS] head loss on the GPU."""
    w = WORKLOADS["bert_base"]
    inp = make_inputs(w)
    st = Stage(w, inp)
    try:
        gpu = run_gpu(torch, st, w, inp, w.lowest_unfrozen)
        ref = oracle_run(w, inp, w.lowest_unfrozen)
        bound = floor_bounds(w, inp, w.lowest_unfrozen, ref)
        print(f"[bert_base] y error {rel_err(gpu['y'], ref['y']):.3e}", flush=True)
        assert rel_err(gpu["y"], ref["y"]) <= bound("y")
        assert abs(gpu["loss"][0] - ref["loss"]) <= 2e-2 * abs(ref["loss"])
        assert rel_err(gpu["g_wh"], ref["g_wh"]) <= bound("g_wh")
        check_grads(gpu, ref, w.lowest_unfrozen, w.n_blocks, bound, "bert_base")
        # adapter update (SGD), then a second forward with the updated adapters
        lr = 0.5
        st.step(w.lowest_unfrozen, lr)
        new_ad = O.sgd_step([tuple(dict(a) for a in p) for p in inp["adapters"]],
                            [g if l >= w.lowest_unfrozen else None for l, g in enumerate(ref["grads"])], lr)
        torch.cuda.synchronize()
        for l in range(w.n_blocks):
            for a in range(2):
                for k in ("w_down", "w_up"):
                    got = st.adapters[l][a][k].cpu().numpy()
                    old = inp["adapters"][l][a][k]
                    if l >= w.lowest_unfrozen:
                        # the applied step -lr * g matches the oracle's
                        assert rel_err(got - old, new_ad[l][a][k] - old) <= bound((l, a, k)), (l, a, k)
                    else:
                        assert np.array_equal(got, old), (l, a, k)
                    assert np.all(st.adapters[l][a]["g_" + k[2:]].cpu().numpy() == 0)
        inp2 = dict(inp, adapters=new_ad)
        gpu2 = run_gpu(torch, st, w, inp2, w.n_blocks)  # frozen forward, no backward
        ref2 = oracle_run(w, inp2, w.n_blocks)
        assert rel_err(gpu2["y"], ref2["y"]) <= bound("y")
    finally:
        st.close()


def test_bert_base_unfreezing_sweep(torch):
    """Cut-off at blocks 11, 9, 6, 3, 0: the early-stopped gradients equal the
    full backward's for every unfrozen block."""
    w = WORKLOADS["bert_base_sweep"]
    inp = make_inputs(w)
    ref = oracle_run(w, inp, 0)
    # the truncated backward's gradients are the full backward's, so one floor
    # run at c = 0 covers every cut-off
    bound = floor_bounds(w, inp, 0, ref)
    st = Stage(w, inp)
    try:
        for c in SWEEP:
            print(f"[sweep] c={c}", flush=True)
            gpu = run_gpu(torch, st, w, inp, c)
            assert rel_err(gpu["y"], ref["y"]) <= bound("y")
            check_grads(gpu, ref, c, w.n_blocks, bound, f"sweep c={c}")
    finally:
        st.close()


def test_bert_base_single_placement_parity(torch):
    """BERT-base-shaped stage with one adapter per block (after the FFN): the
    backward ends after block 8's FFN adapter; the stash is the smaller plan."""
    w = WORKLOADS["bert_base_single"]
    inp = make_inputs(w)
    st = Stage(w, inp)
    try:
        gpu = run_gpu(torch, st, w, inp, w.lowest_unfrozen)
        ref = oracle_run(w, inp, w.lowest_unfrozen)
        bound = floor_bounds(w, inp, w.lowest_unfrozen, ref)
        print(f"[bert_base_single] y error {rel_err(gpu['y'], ref['y']):.3e}", flush=True)
        assert rel_err(gpu["y"], ref["y"]) <= bound("y")
        assert rel_err(gpu["g_wh"], ref["g_wh"]) <= bound("g_wh")
        check_grads(gpu, ref, w.lowest_unfrozen, w.n_blocks, bound, "bert_base_single")
        plan, _ = B.ringada_stage_plan(st.desc, w.batch, w.seq, w.lowest_unfrozen)
        two, _ = B.ringada_stage_plan(make_desc(w.replace(placement="houlsby")), w.batch, w.seq, w.lowest_unfrozen)
        assert plan < two
    finally:
        st.close()


def test_bert_large_share_parity(torch):
    w = WORKLOADS["bert_large_share"]
    inp = make_inputs(w)
    st = Stage(w, inp)
    try:
        gpu = run_gpu(torch, st, w, inp, w.lowest_unfrozen)
        ref = oracle_run(w, inp, w.lowest_unfrozen)
        bound = floor_bounds(w, inp, w.lowest_unfrozen, ref)
        assert rel_err(gpu["y"], ref["y"]) <= bound("y")
        check_grads(gpu, ref, w.lowest_unfrozen, w.n_blocks, bound, "bert_large")
    finally:
        st.close()


def test_llama_share_parity_on_a_causal_prefix(torch):
    """Full-size LLaMA share in the benchmark's launch configuration.  The
    incoming gradient is zero outside the first 64 positions of the first and
    the last sample (token rows 0-63 and 1536-1599, in different GEMM row
    tiles); with causal attention and batch independence, outputs and
    gradients then equal the oracle's on those two prefixes exactly.  Bound
    per tensor: max(2e-2, twice the bf16 noise floor of that tensor), the
    floor being the oracle re-run with the path's bf16 storage roundings
    (tests/bf16_floor.py)."""
    from bf16_floor import llama_floor
    w = WORKLOADS["llama7b_share"]
    inp = make_inputs(w)
    P = 64
    rows = [0, w.batch - 1]
    dy = np.zeros_like(inp["dy"])
    dy[rows, :P] = inp["dy"][rows, :P]
    st = Stage(w, inp)
    try:
        gpu = run_gpu(torch, st, w, inp, w.lowest_unfrozen, dy=dy)
    finally:
        st.close()
    ref = oracle_run(w, inp, w.lowest_unfrozen, dy=dy[rows, :P], x=inp["x"][rows, :P])
    floor = llama_floor(w, inp, w.lowest_unfrozen, dy, batch=None, seq=P, rows=rows)
    errs = {"y": rel_err(gpu["y"][rows, :P], ref["y"])}
    for l in range(w.n_blocks):
        for a in range(2):
            for k in ("w_down", "w_up"):
                if l < w.lowest_unfrozen:
                    assert np.all(gpu["grads"][l][a][k] == 0)
                else:
                    errs[(l, a, k)] = rel_err(gpu["grads"][l][a][k], ref["grads"][l][a][k])
    for key, e in errs.items():
        bound = max(2e-2, 2.0 * floor[key])
        print(f"[llama] {key}: error {e:.3e}, bf16 floor {floor[key]:.3e}, bound {bound:.3e}", flush=True)
        assert e <= bound, (key, e, bound)


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
    """Bound per tensor: max(2e-2, twice its bf16 storage floor)."""
    from bf16_floor import bert_floor, llama_floor
    w = WIDE[name]
    inp = make_inputs(w)
    st = Stage(w, inp)
    try:
        for c in (w.lowest_unfrozen, -1):
            print(f"[{name}] c={c}", flush=True)
            gpu = run_gpu(torch, st, w, inp, c, want_dx=(c < 0))
            ref = oracle_run(w, inp, c)
            fl = (llama_floor(w, inp, c, inp["dy"], w.batch, w.seq) if w.arch == "llama"
                  else bert_floor(w, inp, c, ref))
            bound = lambda key: max(2e-2, 2.0 * fl[key])
            e = rel_err(gpu["y"], ref["y"])
            print(f"[{name}] c={c} y error {e:.3e} (floor {fl['y']:.3e})", flush=True)
            assert e <= bound("y")
            check_grads(gpu, ref, max(c, 0), w.n_blocks, bound, name)
            if c < 0:
                e = rel_err(gpu["dx"], ref["dx"])
                print(f"[{name}] dx error {e:.3e} (floor {fl['dx']:.3e})", flush=True)
                assert e <= bound("dx")
    finally:
        st.close()


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
        # a frozen stage streams forwards back to back (nothing pending)
        st.forward(x, y, w.n_blocks)
        st.forward(x, y, w.n_blocks)
        with pytest.raises(B.RingadaError) as e:
            st.backward(dy, w.n_blocks)
        assert e.value.status == B.RINGADA_E_STATE
        torch.cuda.synchronize()
    finally:
        st.close()
