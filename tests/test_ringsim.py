"""The ring simulator (per-block lookup table replayed over the clients)
against schedules worked out by hand."""
import pytest

from paper_2502_19864_amd.ringsim import BlockTable, Client, cutoff_global, simulate

T = BlockTable(fwd_frozen=1.0, fwd_stash=1.5, bwd_full=3.0, bwd_cut=1.0, step=0.25, head=0.5, act_bytes=0)


def ring(*sizes, speeds=None):
    speeds = speeds or [1.0] * len(sizes)
    return [Client(sum(sizes[:i]), n, sp) for i, (n, sp) in enumerate(zip(sizes, speeds))]


def test_cutoff_is_the_l_minus_d_plus_1_th_block():
    # Alg. 1: the backward ends at the (L - d + 1)-th adapter (1-indexed)
    assert cutoff_global(14, 3) == 11 and cutoff_global(12, 12) == 0 and cutoff_global(12, 0) == 12


def test_one_client_runs_every_iteration_back_to_back():
    # 5 blocks, depth 5: per iteration 5 stashing forwards, the head, the
    # terminator block's backward, 4 full backwards, 5 adapter steps
    per = 5 * 1.5 + 0.5 + 1.0 + 4 * 3.0 + 5 * 0.25
    for iters in (1, 3, 7):
        ms, busy, _ = simulate(T, ring(5), depth=5, iters=iters)
        assert ms == pytest.approx(iters * per)
        assert busy[0] == pytest.approx(iters * per)


def test_fully_unfrozen_ring_serialises_on_one_f_one_b():
    # every client keeps 1F1B, and the initiator (client 0) cannot forward
    # batch b+1 before batch b's backward reached it: one iteration at a time,
    # including the hops (1 MB per hop at 1 GB/s = 1 ms)
    t = BlockTable(**dict(T.to_json(), act_bytes=10**6))
    sizes = (2, 3)
    fwd = 5 * 1.5
    bwd = 1.0 + 4 * 3.0 + 5 * 0.25
    # hops: client 0 -> 1 (forward), client 1 -> initiator 0 (output for the
    # loss), initiator -> client 1 (the gradient to the top block), client 1 -> 0
    hops = 4
    per = fwd + 0.5 + bwd + hops
    ms, _, _ = simulate(t, ring(*sizes), depth=5, iters=4, link_gbps=1.0)
    assert ms == pytest.approx(4 * per)


def test_frozen_ring_pipelines_at_the_slowest_client():
    # depth 0: every client only forwards; in steady state one iteration costs
    # the busiest client's time per batch (client 1: 3 blocks)
    sizes = (2, 3, 1)
    m19, _, _ = simulate(T, ring(*sizes), depth=0, iters=19)
    m20, _, _ = simulate(T, ring(*sizes), depth=0, iters=20)
    assert m20 - m19 == pytest.approx(3.0)
    # a client twice as fast halves its share: now client 0 (2 blocks + head) is busiest
    m19, _, _ = simulate(T, ring(*sizes, speeds=[1, 2, 1]), depth=0, iters=19)
    m20, _, _ = simulate(T, ring(*sizes, speeds=[1, 2, 1]), depth=0, iters=20)
    assert m20 - m19 == pytest.approx(2.5)


def test_the_terminator_paces_the_ring_in_steady_state():
    # 4:5:2:3 blocks, depth 3 (the example of Sec. III-A): only the last client
    # (blocks 11..13) is unfrozen; its 1F1B chain per iteration is its
    # forward (3 stashing blocks), the initiator's head, its backward
    # (terminator block + 2 full blocks, 3 steps); the frozen clients run ahead
    per = 3 * 1.5 + 0.5 + (1.0 + 2 * 3.0 + 3 * 0.25)
    m9, _, _ = simulate(T, ring(4, 5, 2, 3), depth=3, iters=9)
    m10, _, _ = simulate(T, ring(4, 5, 2, 3), depth=3, iters=10)
    assert m10 - m9 == pytest.approx(per)


def test_early_stopping_never_costs_time():
    prev = 0.0
    for depth in range(0, 15):
        ms, _, tr = simulate(T, ring(4, 5, 2, 3), depth=depth, iters=6, trace=True)
        assert ms >= prev - 1e-9
        prev = ms
        # no client runs two things at once
        for u in range(4):
            spans = sorted((s, e) for c, _, _, s, e in tr if c == u)
            assert all(a[1] <= b[0] + 1e-12 for a, b in zip(spans, spans[1:]))
