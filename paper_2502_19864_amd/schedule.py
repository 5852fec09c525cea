"""Top-down adapter unfreezing (Alg. 1) driving one ring stage on one GPU.

The coordinator's schedule starts at depth d0 and adds one after every k
rounds; in each round the initiator runs its local iterations: forward through
the stage, [CLS] cross-entropy loss and head update (the initiator's Hed),
the backward that ends at the adapter the depth selects, and the update of
the unfrozen adapters (Sec. III-B).  The stage is the one held by a client
owning blocks first_block .. first_block + n_blocks - 1 (0-indexed) of n_tm;
its cut-off per depth comes from the library (ringada_local_cutoff), so a
stage below the cut-off runs forward only, and the stash the forward keeps
grows as the cut-off moves down.

Every step runs in the library's kernels; this module only sequences the
calls and records per-iteration time (HIP events on the launch stream), loss
and stash size.

    python -m paper_2502_19864_amd.schedule --workload bert_base --d0 1 --k 1 --iters 3
"""
from __future__ import annotations

import argparse
import json
import sys

import numpy as np

from . import binding as B
from .stage import Stage


def depth_of_round(r, d0, k):
    """Depth in round r (1-indexed): d0 for rounds 1..k, then +1 after every
    k rounds."""
    return d0 + (r - 1) // k


class Alg1Driver:
    """One initiator's iterations through one stage.

    stage: a bound Stage; w_h [d, C], b_h [C]: the initiator's head (float32
    numpy); batches: list of (x [B, S, d] float numpy in the stage's storage
    values, labels [B] int); n_tm: Trm blocks of the whole model;
    first_block: 0-indexed first block of this stage."""

    def __init__(self, stage: Stage, w_h, b_h, batches, n_tm, first_block=0, lr=1e-3, lr_head=1e-3):
        self.st = stage
        torch = stage.torch
        self.torch = torch
        self.n_tm, self.first = n_tm, first_block
        self.lr, self.lr_head = lr, lr_head
        self.wh = stage.f32(w_h)
        self.bh = stage.f32(b_h)
        self.gwh = torch.zeros_like(self.wh)
        self.gbh = torch.zeros_like(self.bh)
        self.x = [stage.upload(x) for x, _ in batches]
        self.labels = [torch.from_numpy(np.ascontiguousarray(lab, dtype=np.int32)).to(stage.dev)
                       for _, lab in batches]
        shape = batches[0][0].shape
        self.y = stage.empty(*shape)
        self.dy = stage.empty(*shape)
        self.dx = stage.empty(*shape)

    def cutoff(self, depth):
        return B.ringada_local_cutoff(self.n_tm, depth, self.first, self.st.w.n_blocks)

    def iteration(self, c, i):
        st, w = self.st, self.st.w
        x, lab = self.x[i % len(self.x)], self.labels[i % len(self.labels)]
        Bt, S, d = x.shape
        loss = self.torch.zeros(1, dtype=self.torch.float32, device=st.dev)
        st.forward(x, self.y, c)
        B.ringada_head_ce(st.sptr, st.desc.dtype, self.y, Bt, S, d, self.wh, self.bh, self.wh.shape[1], lab,
                          self.dy, self.gwh, self.gbh, loss)
        B.ringada_sgd_f32(st.sptr, self.wh, self.gwh, self.wh.numel(), self.lr_head)
        B.ringada_sgd_f32(st.sptr, self.bh, self.gbh, self.bh.numel(), self.lr_head)
        if c < w.n_blocks:
            st.backward(self.dy, c, self.dx if c < 0 else None)
            st.step(c, self.lr)
        return loss

    def run(self, d0, k, rounds, iters_per_round):
        """Returns one record per iteration: round, depth, c, loss, ms (GPU
        time of the iteration), stash_bytes (the plan for that cut-off)."""
        torch = self.torch
        recs, pending = [], []
        it = 0
        for r in range(1, rounds + 1):
            depth = min(depth_of_round(r, d0, k), self.n_tm)
            c = self.cutoff(depth)
            stash, _ = B.ringada_stage_plan(self.st.desc, self.x[0].shape[0], self.x[0].shape[1], c)
            for _ in range(iters_per_round):
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record()
                loss = self.iteration(c, it)
                e1.record()
                pending.append((r, depth, c, loss, e0, e1, stash))
                it += 1
        torch.cuda.synchronize()
        for r, depth, c, loss, e0, e1, stash in pending:
            recs.append(dict(round=r, depth=depth, c=c, loss=float(loss.item()), ms=e0.elapsed_time(e1),
                             stash_bytes=stash))
        return recs

    def head(self):
        self.torch.cuda.synchronize()
        return self.wh.cpu().numpy(), self.bh.cpu().numpy()


def summarise(recs, batch):
    """Per depth: iterations, cut-off, mean ms per iteration (first iteration
    of each depth excluded when there are several: it pays the new stash
    allocation), samples/s, stash MiB."""
    out = []
    for depth in sorted({r["depth"] for r in recs}):
        rs = [r for r in recs if r["depth"] == depth]
        timed = rs[1:] if len(rs) > 1 else rs
        ms = sum(r["ms"] for r in timed) / len(timed)
        out.append(dict(depth=depth, c=rs[0]["c"], iterations=len(rs), ms=round(ms, 4),
                        samples_per_s=round(batch / (ms * 1e-3), 1), stash_mib=round(rs[0]["stash_bytes"] / 2**20, 2),
                        loss_first=round(rs[0]["loss"], 5), loss_last=round(rs[-1]["loss"], 5)))
    return out


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--workload", default="bert_base")
    ap.add_argument("--d0", type=int, default=1)
    ap.add_argument("--k", type=int, default=1, help="rounds per depth step")
    ap.add_argument("--rounds", type=int, default=None, help="default: until every block is unfrozen")
    ap.add_argument("--iters", type=int, default=3, help="initiator iterations per round")
    ap.add_argument("--batches", type=int, default=2)
    ap.add_argument("--lr", type=float, default=1e-3)
    args = ap.parse_args(argv)

    import torch
    from .workloads import WORKLOADS, make_inputs
    if not torch.cuda.is_available():
        print("schedule: no GPU visible", file=sys.stderr)
        return 1
    B.lib()
    w = WORKLOADS[args.workload]
    if w.loss != "cls_ce":
        w = w.replace(loss="cls_ce")
    inp = make_inputs(w)
    rng = np.random.default_rng(w.seed + 7)
    batches = [(inp["x"], inp["labels"])]
    for _ in range(args.batches - 1):
        x = rng.standard_normal(inp["x"].shape).astype(np.float32)
        if w.dtype == "bf16":
            from .workloads import round_to_bf16
            x = round_to_bf16(x)
        batches.append((x, rng.integers(0, 2, w.batch).astype(np.int32)))
    st = Stage(w, inp)
    try:
        drv = Alg1Driver(st, inp["w_h"], inp["b_h"], batches, n_tm=w.n_blocks, lr=args.lr, lr_head=args.lr)
        rounds = args.rounds or args.k * (w.n_blocks - args.d0 + 1)
        drv.run(args.d0, args.k, 1, 1)  # warm-up: kernel loading, first workspace
        recs = drv.run(args.d0, args.k, rounds, args.iters)
        for row in summarise(recs, w.batch):
            print(json.dumps(dict(workload=w.name, **row)), flush=True)
    finally:
        st.close()
    return 0


if __name__ == "__main__":
    sys.exit(main())
