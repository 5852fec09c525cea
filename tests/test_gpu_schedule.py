"""The top-down unfreezing loop (Alg. 1) on the GPU against the oracle's:
eight iterations over four rounds with the depth growing every round, so the
cut-off walks from the top block to the bottom one; every per-iteration loss,
the final adapters and the final head must match (the updates w - w0 are
compared, each side from its own start, at the stage's tolerance)."""
import numpy as np
import pytest

import oracle as O
from helpers import oracle_desc, rel_err, to64
from paper_2502_19864_amd.schedule import Alg1Driver
from paper_2502_19864_amd.stage import Stage
from paper_2502_19864_amd.workloads import Workload, make_inputs, round_to_bf16

pytestmark = pytest.mark.gpu

CASES = {
    "f32": (Workload("sched_f32", "bert", "f32", 4, 128, 2, 512, 16, 20, 3, 0, "cls_ce", 2101), 1e-4),
    "bf16": (Workload("sched_bf16", "bert", "bf16", 4, 256, 4, 512, 64, 32, 4, 0, "cls_ce", 2102), 2e-2),
    "bf16_single": (Workload("sched_bf16_single", "bert", "bf16", 4, 256, 4, 512, 64, 32, 4, 0, "cls_ce", 2103,
                             placement="ffn"), 2e-2),
}


@pytest.fixture(scope="module")
def torch():
    import torch as t
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    return t


@pytest.mark.parametrize("name", sorted(CASES))
def test_unfreezing_schedule_matches_the_oracle(torch, name):
    w, tol = CASES[name]
    inp = make_inputs(w)
    rng = np.random.default_rng(w.seed + 1)
    x2 = rng.standard_normal(inp["x"].shape).astype(np.float32)
    if w.dtype == "bf16":
        x2 = round_to_bf16(x2)
    batches = [(inp["x"], inp["labels"]), (x2, rng.integers(0, 2, w.batch).astype(np.int32))]
    # adapter steps of ~0.25% of the weights (so the fp32 masters resolve them to
    # ~1e-5) while the loss stays O(1)
    lr, lr_head = 1.0, 0.01
    st = Stage(w, inp)
    try:
        drv = Alg1Driver(st, inp["w_h"], inp["b_h"], batches, n_tm=4, lr=lr, lr_head=lr_head)
        recs = drv.run(d0=1, k=1, rounds=4, iters_per_round=2)
        wh, bh = drv.head()
        got = [[{k: st.adapters[l][a][k].cpu().numpy() for k in ("w_down", "w_up")} for a in range(2)]
               for l in range(4)]
    finally:
        st.close()
    assert [r["c"] for r in recs] == [3, 3, 2, 2, 1, 1, 0, 0]
    assert all(recs[i]["stash_bytes"] <= recs[i + 1]["stash_bytes"] for i in range(7))

    desc = oracle_desc(w)
    W, A = to64(inp, w)
    b64 = [(np.asarray(x, np.float64), lab) for x, lab in batches]
    rref, Aref, whr, bhr = O.alg1_stage_run(desc, W, A, inp["w_h"].astype(np.float64), inp["b_h"].astype(np.float64),
                                            b64, n_tm=4, beta=1, d0=1, k=1, rounds=4, iters_per_round=2,
                                            lr=lr, lr_head=lr_head)
    assert [r[2] for r in rref] == [r["c"] for r in recs]
    for i, (g, r) in enumerate(zip(recs, rref)):
        print(f"[{name}] iteration {i}: c={g['c']} loss gpu {g['loss']:.8f} oracle {r[3]:.8f}", flush=True)
    errs = {}
    for l in range(4):
        for a in range(2):
            for k in ("w_down", "w_up"):
                w0 = inp["adapters"][l][a][k].astype(np.float64)
                if Aref[l][a] is None or w.placement == "ffn" and a == 0:
                    continue
                errs[(l, a, k)] = rel_err(got[l][a][k] - w0, Aref[l][a][k] - A[l][a][k])
    print(f"[{name}] adapter-update errors: " + ", ".join(f"{k}: {v:.2e}" for k, v in sorted(errs.items())),
          flush=True)
    worst = 0.0
    for l in range(4):
        for a in range(2):
            for k in ("w_down", "w_up"):
                # each side's update from its own start (the bf16 path keeps fp32
                # masters and computes with their bf16 rounding; the oracle
                # starts from that rounding)
                w0 = inp["adapters"][l][a][k].astype(np.float64)
                if Aref[l][a] is None or w.placement == "ffn" and a == 0:
                    assert np.array_equal(got[l][a][k], inp["adapters"][l][a][k]), (l, a, k)
                    continue
                e = rel_err(got[l][a][k] - w0, Aref[l][a][k] - A[l][a][k])
                worst = max(worst, e)
                assert e <= tol, (name, l, a, k, e)
    for i, (g, r) in enumerate(zip(recs, rref)):
        assert abs(g["loss"] - r[3]) <= tol * abs(r[3]), (i, g["loss"], r[3])
    assert rel_err(wh - inp["w_h"], whr - inp["w_h"]) <= tol
    assert rel_err(bh - inp["b_h"], bhr - inp["b_h"]) <= tol
    print(f"[{name}] losses {[round(r['loss'], 5) for r in recs]}; worst adapter-update error {worst:.3e}",
          flush=True)
