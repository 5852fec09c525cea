"""Pins of the oracle's top-down unfreezing loop (Alg. 1 on one stage)."""
import numpy as np

import oracle as O


def _tiny(L=4, seed=3, B=3, S=5, d=16, H=2, F=24, m=4):
    rng = np.random.default_rng(seed)
    n = lambda *s, std=0.3: rng.standard_normal(s) * std  # noqa: E731
    desc = O.make_desc("bert", L, d, H, F, m)
    W = [dict(w_qkv=n(d, 3 * d), b_qkv=n(3 * d, std=0.1), w_o=n(d, d), b_o=n(d, std=0.1),
              ln1_g=1 + n(d, std=0.1), ln1_b=n(d, std=0.1), w_i=n(d, F), b_i=n(F, std=0.1),
              w_f=n(F, d), b_f=n(d, std=0.1), ln2_g=1 + n(d, std=0.1), ln2_b=n(d, std=0.1))
         for _ in range(L)]
    A = [tuple({"w_down": n(d, m), "w_up": n(m, d)} for _ in range(2)) for _ in range(L)]
    batches = [(rng.standard_normal((B, S, d)), rng.integers(0, 2, B)) for _ in range(3)]
    return desc, W, A, n(d, 2), np.zeros(2), batches


def test_depth_schedule_follows_the_coordinator_loop():
    """d starts at d0 and the coordinator adds one after every round r with
    r mod k == 0 (Alg. 1): replay that loop and compare."""
    for d0, k in ((1, 1), (1, 3), (2, 2), (4, 5)):
        d, seen = d0, []
        for r in range(1, 20):
            seen.append(d)
            if r % k == 0:
                d += 1
        assert seen == [O.depth_of_round(r, d0, k) for r in range(1, 20)]


def test_one_iteration_is_forward_loss_head_step_backward_and_sgd():
    desc, W, A, wh, bh, batches = _tiny()
    x, lab = batches[0]
    rec, A1, wh1, bh1 = O.alg1_stage_run(desc, W, A, wh, bh, batches, n_tm=4, beta=1, d0=2, k=1,
                                         rounds=1, iters_per_round=1, lr=0.1, lr_head=0.2)
    assert rec == [(1, 2, 2, rec[0][3])]  # depth 2 of 4 blocks: cut-off at 0-indexed block 2
    y, caches = O.stage_forward(desc, W, A, x)
    loss, dy, gwh, gbh = O.cls_head_ce(y, wh, bh, lab)
    _, grads = O.stage_backward(desc, W, A, caches, dy, 2)
    ref = O.sgd_step(A, grads, 0.1)
    assert rec[0][3] == loss
    assert np.array_equal(wh1, wh - 0.2 * gwh) and np.array_equal(bh1, bh - 0.2 * gbh)
    for l in range(4):
        for a in range(2):
            for key in ("w_down", "w_up"):
                assert np.array_equal(A1[l][a][key], ref[l][a][key])


def test_adapters_stay_frozen_until_the_depth_reaches_them():
    desc, W, A, wh, bh, batches = _tiny()
    rounds = 4  # depth 1, 2, 3, 4 with k = 1: cut-off blocks 3, 2, 1, 0
    for stop_after in range(1, rounds + 1):
        rec, A1, _, _ = O.alg1_stage_run(desc, W, A, wh, bh, batches, n_tm=4, beta=1, d0=1, k=1,
                                         rounds=stop_after, iters_per_round=2, lr=0.05, lr_head=0.05)
        assert [r[2] for r in rec] == [c for c in (3, 2, 1, 0)[:stop_after] for _ in range(2)]
        lowest = 4 - stop_after
        for l in range(4):
            changed = any(not np.array_equal(A1[l][a][k], A[l][a][k]) for a in range(2) for k in ("w_down", "w_up"))
            assert changed == (l >= lowest), (stop_after, l)


def test_a_stage_of_a_larger_model_is_frozen_until_the_cutoff_enters_it():
    """The stage holds blocks 5..8 of 8 (1-indexed); with depth 2 the cut-off is
    block 7 (local 2); a stage holding blocks 1..4 stays forward-only (c = 4)."""
    desc, W, A, wh, bh, batches = _tiny()
    rec, A1, _, _ = O.alg1_stage_run(desc, W, A, wh, bh, batches, n_tm=8, beta=5, d0=2, k=10,
                                     rounds=1, iters_per_round=1, lr=0.1, lr_head=0.1)
    assert rec[0][2] == 2
    rec, A1, _, _ = O.alg1_stage_run(desc, W, A, wh, bh, batches, n_tm=8, beta=1, d0=2, k=10,
                                     rounds=1, iters_per_round=2, lr=0.1, lr_head=0.1)
    assert [r[2] for r in rec] == [4, 4]
    assert all(np.array_equal(A1[l][a][k], A[l][a][k]) for l in range(4) for a in range(2) for k in ("w_down", "w_up"))


def test_training_on_one_batch_lowers_its_loss():
    desc, W, A, wh, bh, batches = _tiny()
    rec, _, _, _ = O.alg1_stage_run(desc, W, A, wh, bh, batches[:1], n_tm=4, beta=1, d0=4, k=100,
                                    rounds=1, iters_per_round=12, lr=0.2, lr_head=0.5)
    losses = [r[3] for r in rec]
    assert losses[-1] < 0.8 * losses[0], losses
