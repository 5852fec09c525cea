"""One stage step on the GPU through the C ABI, for the parity tests:
forward, the loss or the given incoming gradient, the early-stopped
backward; results as numpy arrays."""
from paper_2502_19864_amd import binding as B


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
