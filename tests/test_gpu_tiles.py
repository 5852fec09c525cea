"""Parity of every tile configuration the bf16 projection GEMMs can select,
and of the loss helpers' remaining instantiations, through the C ABI.

The GEMM launcher picks a tile shape per call from (tokens, N, K) and the
epilogue (pipelined 128x192, 128x96, 128x128 with two or three stages,
256x192 and 256x128 with eight waves, and the split of a half-empty last
round of 256x128 tiles onto 128x128).  The stage workloads of the other
tests reach about half of the legal (role, epilogue, tile) combinations.
The one-block stages below reach every other one (each entry lists what it
adds), at token counts up to 32768.  Outputs of at most 32 MiB are stored
with the non-temporal hint, larger ones plainly: the 32768-token d = 1024
case runs the plain arm of the projection GEMMs, the fused attention and the
adapter rows.

Every op of a block is per sequence, so each case runs the whole batch on
the GPU and compares three sequences with the oracle: the first, the middle
and the last. They lie in different row tiles and XCD bands. The incoming
gradient is the workload's on those sequences and zero elsewhere, so the
GPU's adapter gradients are sums over exactly those three. The backward runs
to the stage input (c = -1), through all eight projection GEMMs. Bounds as
everywhere for bf16: 2e-2, or 1.25 x the emulated storage floor of each
tensor where that floor leaves less room."""
import numpy as np
import pytest

from bf16_floor import rel_err_parts, stage_floor, sum_grads
from gpu_run import run_gpu
from helpers import TOL, Checker, oracle_run
import oracle as O
from paper_2502_19864_amd import binding as B
from paper_2502_19864_amd.stage import Stage
from paper_2502_19864_amd.workloads import Workload, make_inputs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.lib()  # fails loudly if the library is not built
    return torch


def _w(name, arch, d, h, f, seq, batch, seed):
    return Workload(name, arch, "bf16", 1, d, h, f, 64, seq, batch, 0, "dy", seed)


# (role, epilogue, tile) combinations each case adds to the rest of the suite
TILES = {
    # 128x128 two-stage (>= 512 tiles): SwiGLU, dSwiGLU, FFN-in-dx, FFN-out, O
    # and O-dx; 128x192 for the rotary QKV's neighbours
    "tiles_llama_d256_t32k": _w("tiles_llama_d256_t32k", "llama", 256, 4, 192, 128, 256, 2101),
    # 256x192: FFN-out, O, O-dx, QKV-dx (residual), QKV (store); 256x128
    # FFN-in (GELU) / FFN-out-dx (GELU'); the non-causal two-pass attention at
    # head dim 128 over two 128-key tiles
    "tiles_bert_d3072_s256": _w("tiles_bert_d3072_s256", "bert", 3072, 24, 192, 256, 16, 2102),
    # 128x192 O / O-dx / FFN-out / FFN-in-dx (store) and 128x96 QKV-dx /
    # FFN-in-dx (store) of the pre-RMS block
    "tiles_llama_d768_b64": _w("tiles_llama_d768_b64", "llama", 768, 12, 64, 128, 64, 2103),
    # 256x192 FFN-in (GELU) / FFN-out-dx (GELU'); 256x128 FFN-in-dx and
    # QKV-dx (residual)
    "tiles_bert_d2048_f2048": _w("tiles_bert_d2048_f2048", "bert", 2048, 32, 2048, 128, 32, 2104),
    # 256x192 FFN-in-dx (residual), the rest of the d = 3072 post-LN shapes
    "tiles_bert_d3072_f3072": _w("tiles_bert_d3072_f3072", "bert", 3072, 48, 3072, 128, 32, 2105),
    # 128x128 two-stage of the post-LN block, QKV-dx included (32768 tokens)
    "tiles_bert_d256_t32k": _w("tiles_bert_d256_t32k", "bert", 256, 4, 64, 128, 256, 2106),
    # 256x192 of the pre-RMS block's dX GEMMs (store epilogues)
    "tiles_llama_d3072_f576": _w("tiles_llama_d3072_f576", "llama", 3072, 48, 576, 128, 32, 2107),
    # 128x96 / 128x128 three-stage of the pre-RMS block at 1024 tokens
    "tiles_llama_d768_b8": _w("tiles_llama_d768_b8", "llama", 768, 12, 64, 128, 8, 2108),
    # 256x128 QKV (store) of the post-LN block: 256x192 would leave CUs idle
    "tiles_bert_d3072_b4": _w("tiles_bert_d3072_b4", "bert", 3072, 48, 64, 256, 4, 2109),
    # outputs past the 32 MiB streaming bound (plain stores): the adapter and norm rows
    # (64 MiB), the QKV projection with the fused attention (192 MiB) and its O rows
    "tiles_bert_d1024_t32k": _w("tiles_bert_d1024_t32k", "bert", 1024, 16, 64, 128, 256, 2110),
}


@pytest.mark.timeout(600)
@pytest.mark.parametrize("name", sorted(TILES))
def test_tile_configuration_parity(torch, name):
    w = TILES[name]
    inp = make_inputs(w)
    picks = (0, w.batch // 2, w.batch - 1)
    dy = np.zeros_like(inp["dy"])
    for s in picks:
        dy[s] = inp["dy"][s]
    print(f"[{name}] {w.arch} d={w.d_model} H={w.n_heads} F={w.d_ffn} batch={w.batch} seq={w.seq} "
          f"({w.tokens} tokens), c=-1", flush=True)
    st = Stage(w, inp)
    try:
        gpu = run_gpu(torch, st, w, inp, -1, dy=dy, want_dx=True)
    finally:
        st.close()
    parts = [(inp["x"][s:s + 1], dy[s:s + 1]) for s in picks]
    refs = [oracle_run(w, inp, -1, dy=d_, x=x_) for x_, d_ in parts]
    fl = stage_floor(w, inp, -1, refs, parts)
    chk = Checker(name, floor=fl)
    chk("y", None, None, err=rel_err_parts([gpu["y"][s:s + 1] for s in picks], [r["y"] for r in refs]))
    chk("dx", None, None, err=rel_err_parts([gpu["dx"][s:s + 1] for s in picks], [r["dx"] for r in refs]))
    # the rows of the other sequences: dY was zero there, so dX is too
    others = np.ones(w.batch, bool)
    others[list(picks)] = False
    assert np.all(gpu["dx"][others] == 0), "nonzero input gradient of a sequence without an incoming gradient"
    chk.grads(gpu["grads"], sum_grads([r["grads"] for r in refs]), 0, w.n_blocks)
    chk.done()


# ---------------------------------------------------------------- loss helpers
def _head_case(torch, dtype, n_classes, batch=6, seq=5, d=256, seed=2201, repeat=1):
    """ringada_head_ce on seeded inputs against the oracle's head: the loss,
    the head's gradients and the dY rows (position 0 of each sequence; every
    other row must come back zero)."""
    rng = np.random.default_rng(seed)
    y = rng.standard_normal((batch, seq, d)).astype(np.float32)
    if dtype == "bf16":  # the GPU reads bf16: give the oracle the same values
        y = (y.view(np.uint32) & 0xFFFF0000).view(np.float32)
    wh = (0.05 * rng.standard_normal((d, n_classes))).astype(np.float32)
    bh = (0.1 * rng.standard_normal(n_classes)).astype(np.float32)
    labels = rng.integers(0, n_classes, batch).astype(np.int32)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    dev = torch.device("cuda", 0)
    yt = torch.from_numpy(y).to(dev).to(tdt)
    dyt = torch.full_like(yt, float("nan"))  # every element must be written
    wht, bht = torch.from_numpy(wh).to(dev), torch.from_numpy(bh).to(dev)
    gwh, gbh = torch.zeros_like(wht), torch.zeros_like(bht)
    loss = torch.zeros(1, dtype=torch.float32, device=dev)
    lab = torch.from_numpy(labels).to(dev)
    s = torch.cuda.current_stream(dev).cuda_stream
    runs = []
    for _ in range(repeat):  # fresh accumulators each time: the same bits every call
        gwh.zero_(); gbh.zero_(); loss.zero_(); dyt.fill_(float("nan"))
        B.ringada_head_ce(s, B.BF16 if dtype == "bf16" else B.F32, yt, batch, seq, d, wht, bht, n_classes, lab, dyt,
                          gwh, gbh, loss)
        torch.cuda.synchronize()
        runs.append([t_.clone() for t_ in (loss, dyt, gwh, gbh)])
    for r in runs[1:]:
        for a_, b_ in zip(runs[0], r):
            assert torch.equal(a_, b_), "ringada_head_ce gave different bits on the same inputs"
    ref_loss, ref_dy, ref_gwh, ref_gbh = O.cls_head_ce(y.astype(np.float64), wh.astype(np.float64),
                                                       bh.astype(np.float64), labels)
    return (loss.cpu().numpy()[0], dyt.float().cpu().numpy(), gwh.cpu().numpy(), gbh.cpu().numpy(),
            ref_loss, ref_dy, ref_gwh, ref_gbh)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("n_classes,batch,d", [(2, 6, 256), (5, 6, 256), (16, 6, 256), (5, 300, 2048)])
def test_head_ce_classes(torch, dtype, n_classes, batch, d):
    """Both instantiations of the head kernel (two classes, and up to 16) in
    both storage types, and a batch of more than one 256-sample chunk with
    more than one 1024-feature block.  The loss and the head gradients are
    fp32 sums of exact inputs (bound 1e-4); the bf16 dY is one rounding of an
    fp32 dot product (bound: two bf16 units in the last place, 2^-7, relative
    to the tensor's largest value).  Three calls on the same inputs give the
    same bits."""
    loss, dy, gwh, gbh, rloss, rdy, rgwh, rgbh = _head_case(torch, dtype, n_classes, batch=batch, d=d,
                                                            seed=2201 + n_classes + batch, repeat=3)
    chk = Checker(f"head_ce {dtype} C={n_classes} B={batch} d={d}", tol=TOL["f32"])
    chk("loss", np.array([loss]), np.array([rloss]))
    chk("g_wh", gwh, rgwh)
    chk("g_bh", gbh, rgbh)
    dchk = Checker(f"head_ce {dtype} C={n_classes} B={batch} d={d}", tol=TOL["f32"] if dtype == "f32" else 2.0 ** -7)
    dchk("dy", dy, rdy)
    assert np.all(dy[:, 1:] == 0), "dY rows past position 0 must be written as zeros"
    chk.done()
    dchk.done()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_mse_loss(torch, dtype):
    """ringada_loss_mse in both storage types against the oracle's MSE:
    the loss (fp32 sum, 1e-4) and dY = 2 (y - target) / n (bf16: one
    rounding of an exact fp32 value, 2^-8 relative)."""
    rng = np.random.default_rng(2301)
    n = 3 * 37 * 256 + 5  # not a multiple of the kernel's block
    y = rng.standard_normal(n).astype(np.float32)
    t = rng.standard_normal(n).astype(np.float32)
    if dtype == "bf16":
        y = (y.view(np.uint32) & 0xFFFF0000).view(np.float32)
        t = (t.view(np.uint32) & 0xFFFF0000).view(np.float32)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    dev = torch.device("cuda", 0)
    yt, tt = torch.from_numpy(y).to(dev).to(tdt), torch.from_numpy(t).to(dev).to(tdt)
    dyt = torch.full_like(yt, float("nan"))
    loss = torch.zeros(1, dtype=torch.float32, device=dev)
    B.ringada_loss_mse(torch.cuda.current_stream(dev).cuda_stream, B.BF16 if dtype == "bf16" else B.F32, yt, tt, n,
                       dyt, loss)
    torch.cuda.synchronize()
    ref_loss, ref_dy = O.mse_loss(y.astype(np.float64), t.astype(np.float64))
    chk = Checker(f"mse {dtype}", tol=TOL["f32"])
    chk("loss", loss.cpu().numpy(), np.array([ref_loss]))
    dchk = Checker(f"mse {dtype}", tol=TOL["f32"] if dtype == "f32" else 2.0 ** -8)
    dchk("dy", dyt.float().cpu().numpy(), ref_dy)
    chk.done()
    dchk.done()
