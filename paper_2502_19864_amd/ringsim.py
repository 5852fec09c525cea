"""Per-block time lookup table and trace-based simulation of the RingAda ring.

The paper estimates end-to-end training time by profiling the forward and
backward time of each layer, keeping them in a lookup table, and replaying
the training schedule over the clients (Sec. IV).  This module does the same
with tables measured on the MI355X by the library itself:

* ``measure_table`` times one block of a workload's shape on the GPU through
  the stage API: a frozen forward, a forward that stashes for the backward,
  the backward of a fully unfrozen block (including the gradient for the
  block below), the backward of the terminator's block (which stops at its
  lowest adapter), and the adapter update.
* ``simulate`` replays Alg. 1's iterations over a ring of clients
  (Sec. III-A/B): each client holds a contiguous range of blocks; the
  initiator embeds its batches and feeds them to the ring, computes the loss
  and updates its head when the last block's output comes back; the backward
  relays down the ring and ends at the terminator; every client below the
  cut-off only forwards and may run ahead on later batches (1F1B is not
  required there), while a client with unfrozen adapters forwards batch b+1
  only after the backward and update of batch b (no stale weights).  Links
  between ring neighbours carry one activation (forward) or one gradient
  (backward) per hop.  The result is the makespan and a per-client trace.

    python -m paper_2502_19864_amd.ringsim --workload bert_base --assign 4,5,2,3 --depth 3 --iters 8
"""
from __future__ import annotations

import argparse
import dataclasses
import heapq
import json
import sys


# ---------------------------------------------------------------- lookup table
@dataclasses.dataclass
class BlockTable:
    """Milliseconds per block (one batch) on the device it was measured on."""
    fwd_frozen: float   # forward, nothing stashed
    fwd_stash: float    # forward keeping what a full backward reads
    bwd_full: float     # backward of an unfrozen block, gradient passed down
    bwd_cut: float      # backward of the terminator's block (ends at its lowest adapter)
    step: float         # adapter update of one block
    head: float = 0.0   # initiator: loss, head gradient and update
    act_bytes: int = 0  # one activation (or gradient) [batch, seq, d] in the stage dtype

    def to_json(self):
        return dataclasses.asdict(self)


def measure_table(workload, repeats=20):
    """Times one block of `workload`'s shape on cuda:0 through the stage API
    (HIP events on the launch stream, mean over `repeats` after a warm-up)."""
    import torch
    from . import binding as B
    from .stage import Stage
    from .workloads import make_inputs
    w = workload.replace(n_blocks=1, loss="cls_ce")
    inp = make_inputs(w)
    st = Stage(w, inp)
    try:
        x = st.upload(inp["x"])
        y, dy, dx = st.empty(*inp["x"].shape), st.empty(*inp["x"].shape), st.empty(*inp["x"].shape)
        dy.zero_()
        wh, bh = st.f32(inp["w_h"]), st.f32(inp["b_h"])
        gwh, gbh = torch.zeros_like(wh), torch.zeros_like(bh)
        lab = torch.from_numpy(inp["labels"]).to(st.dev)
        loss = torch.zeros(1, dtype=torch.float32, device=st.dev)
        st.ensure_workspace(w.batch, w.seq, -1)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(6)]

        def timed(fn):
            for _ in range(3):
                fn()
            ev[0].record()
            for _ in range(repeats):
                fn()
            ev[1].record()
            torch.cuda.synchronize()
            return ev[0].elapsed_time(ev[1]) / repeats

        def head():
            B.ringada_head_ce(st.sptr, st.desc.dtype, y, w.batch, w.seq, w.d_model, wh, bh, wh.shape[1], lab, dy,
                              gwh, gbh, loss)
            B.ringada_sgd_f32(st.sptr, wh, gwh, wh.numel(), 0.0)
            B.ringada_sgd_f32(st.sptr, bh, gbh, bh.numel(), 0.0)

        fwd_frozen = timed(lambda: st.forward(x, y, 1))  # c = n_blocks: frozen, nothing stashed
        # forward + backward pairs, each part timed by its own events: a full
        # block (c < 0: gradient for the block below) and a terminator block (c = 0)
        fs = bf = bc = 0.0
        for r in range(3 + repeats):
            ev[0].record(); st.forward(x, y, -1); ev[1].record(); st.backward(dy, -1, dx); ev[2].record()
            ev[3].record(); st.forward(x, y, 0); ev[4].record(); st.backward(dy, 0, None); ev[5].record()
            torch.cuda.synchronize()
            if r >= 3:
                fs += ev[0].elapsed_time(ev[1])
                bf += ev[1].elapsed_time(ev[2])
                bc += ev[4].elapsed_time(ev[5])
        step_ms = timed(lambda: st.step(0, 0.0))
        head_ms = timed(head)
        return BlockTable(fwd_frozen=fwd_frozen, fwd_stash=fs / repeats, bwd_full=bf / repeats, bwd_cut=bc / repeats,
                          step=step_ms, head=head_ms,
                          act_bytes=w.batch * w.seq * w.d_model * (2 if w.dtype == "bf16" else 4))
    finally:
        st.close()


# ---------------------------------------------------------------- ring simulation
@dataclasses.dataclass
class Client:
    first: int        # 0-indexed first block
    n: int            # blocks held
    speed: float = 1.0  # relative to the device the table was measured on


def cutoff_global(n_tm, depth):
    """0-indexed block whose adapter ends the backward (the (L - d + 1)-th of
    Alg. 1, 1-indexed)."""
    return n_tm - depth


def _schedule(tasks, resources):
    """Earliest-start list scheduling of a task DAG on exclusive resources.
    tasks: {id: (resource, duration, [pred ids], priority)}; a task starts at
    max(all preds done, resource free); among startable tasks the earliest
    start wins, then the lower priority value, then the earlier task.  Returns
    {id: (start, end)}."""
    free = {r: 0.0 for r in resources}
    order = {t: i for i, t in enumerate(tasks)}  # deterministic tie-break
    succ = {t: [] for t in tasks}
    missing = {t: len(p[2]) for t, p in tasks.items()}
    ready = {}
    for t, (_, _, preds, _) in tasks.items():
        for q in preds:
            succ[q].append(t)
    heap = []
    for t, (r, _, preds, pr) in tasks.items():
        if not preds:
            ready[t] = 0.0
            heapq.heappush(heap, (max(0.0, free[r]), pr, order[t], t))
    done = {}
    while heap:
        start, pr, _, t = heapq.heappop(heap)
        r, dur, _, _ = tasks[t]
        real = max(ready[t], free[r])
        if real > start:  # the resource got busier since this entry was pushed
            heapq.heappush(heap, (real, pr, order[t], t))
            continue
        done[t] = (real, real + dur)
        free[r] = real + dur
        for s_ in succ[t]:
            missing[s_] -= 1
            ready[s_] = max(ready.get(s_, 0.0), real + dur)
            if missing[s_] == 0:
                heapq.heappush(heap, (max(ready[s_], free[tasks[s_][0]]), tasks[s_][3], order[s_], s_))
    assert len(done) == len(tasks), "cyclic task graph"
    return done


def simulate(table: BlockTable, clients, depth, iters, initiator=0, link_gbps=25.0, embed_ms=0.0,
             trace=False):
    """Makespan (ms) of `iters` iterations of one initiator over the ring.

    clients: ring order, contiguous block ranges covering 0..n_tm-1 in that
    order (client 0 holds the lowest blocks); link_gbps: GB/s of every link
    between ring neighbours (one activation or gradient per hop; a client's
    hop to itself is free).  Returns (makespan_ms, per-client busy ms, trace)
    with trace = [(client, kind, batch, start, end)] when asked for."""
    n_tm = sum(c.n for c in clients)
    assert [c.first for c in clients] == [sum(cc.n for cc in clients[:i]) for i in range(len(clients))]
    U = len(clients)
    cut = cutoff_global(n_tm, depth)
    hop_ms = table.act_bytes / (link_gbps * 1e9) * 1e3

    def unfrozen(u):
        return clients[u].first + clients[u].n - 1 >= cut

    def fwd_ms(u):
        c = clients[u]
        return sum(table.fwd_stash if blk >= cut else table.fwd_frozen
                   for blk in range(c.first, c.first + c.n)) / c.speed

    def bwd_ms(u):
        c = clients[u]
        return sum((table.bwd_cut if blk == cut else table.bwd_full) + table.step
                   for blk in range(max(c.first, cut), c.first + c.n)) / c.speed

    lo = next((u for u in range(U) if unfrozen(u)), U)  # the terminator (or U: all frozen)
    PRI = {"bwd": 0, "head": 1, "fwd": 2, "embed": 3, "link": 0}
    tasks, resources = {}, set(range(U))

    def add(tid, res, dur, preds, kind):
        resources.add(res)
        tasks[tid] = (res, dur, [p for p in preds if p is not None], PRI[kind])
        return tid

    def hop(tag, src, dst, pred):
        if src == dst or hop_ms == 0.0:
            return pred
        return add(("link", tag, src, dst), ("link", src, dst), hop_ms, [pred], "link")

    for b in range(iters):
        prev = add(("embed", b), initiator, embed_ms / clients[initiator].speed, [], "embed")
        prev = hop(("f", b, -1), initiator, 0, prev)
        for u in range(U):
            deps = [prev]
            if unfrozen(u) and b > 0:
                deps.append(("bwd", u, b - 1))  # 1F1B where adapters are unfrozen: no stale weights
            prev = add(("fwd", u, b), u, fwd_ms(u), deps, "fwd")
            prev = hop(("f", b, u), u, u + 1 if u + 1 < U else initiator, prev)
        prev = add(("head", b), initiator, table.head / clients[initiator].speed,
                   [prev, ("head", b - 1) if b > 0 else None], "head")
        if lo < U:
            prev = hop(("b", b, -1), initiator, U - 1, prev)
            for u in range(U - 1, lo - 1, -1):
                prev = add(("bwd", u, b), u, bwd_ms(u), [prev], "bwd")
                if u > lo:
                    prev = hop(("b", b, u), u, u - 1, prev)
    sched = _schedule(tasks, resources)
    makespan = max(e for _, e in sched.values()) if sched else 0.0
    busy = [sum(tasks[t][1] for t in tasks if tasks[t][0] == u) for u in range(U)]
    tr = []
    if trace:
        for t, (s0, e0) in sorted(sched.items(), key=lambda kv: kv[1]):
            if isinstance(tasks[t][0], int) and tasks[t][1] > 0:
                tr.append((tasks[t][0], t[0], t[-1], s0, e0))
    return makespan, busy, tr


def chrome_trace(tr):
    """The simulated trace as Chrome trace-event JSON (one row per client)."""
    return [dict(name=f"{k} {b}", ph="X", pid=0, tid=u, ts=s_ * 1e3, dur=(e - s_) * 1e3) for u, k, b, s_, e in tr]


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--workload", default="bert_base")
    ap.add_argument("--assign", default="4,5,2,3", help="blocks per client in ring order")
    ap.add_argument("--speeds", default=None, help="relative compute speed per client (default all 1)")
    ap.add_argument("--depth", type=int, default=3)
    ap.add_argument("--iters", type=int, default=8)
    ap.add_argument("--link-gbps", type=float, default=25.0)
    ap.add_argument("--table", default=None, help="JSON lookup table (else measured now on cuda:0)")
    ap.add_argument("--save-table", default=None)
    ap.add_argument("--trace", default=None, help="write a Chrome trace of the simulated run")
    args = ap.parse_args(argv)
    from .workloads import WORKLOADS
    if args.table:
        table = BlockTable(**json.load(open(args.table)))
    else:
        table = measure_table(WORKLOADS[args.workload])
    if args.save_table:
        json.dump(table.to_json(), open(args.save_table, "w"), indent=1)
    sizes = [int(s) for s in args.assign.split(",")]
    speeds = [float(s) for s in args.speeds.split(",")] if args.speeds else [1.0] * len(sizes)
    clients = [Client(sum(sizes[:i]), n, sp) for i, (n, sp) in enumerate(zip(sizes, speeds))]
    ms, busy, tr = simulate(table, clients, args.depth, args.iters, link_gbps=args.link_gbps, trace=True)
    print(json.dumps(dict(workload=args.workload, assign=sizes, speeds=speeds, depth=args.depth, iters=args.iters,
                          link_gbps=args.link_gbps, makespan_ms=round(ms, 4), ms_per_iteration=round(ms / args.iters, 4),
                          busy_ms=[round(b, 4) for b in busy], table=table.to_json())))
    if args.trace:
        json.dump(chrome_trace(tr), open(args.trace, "w"))
    return 0


if __name__ == "__main__":
    sys.exit(main())
