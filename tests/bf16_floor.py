"""bf16 noise floor of the stage, by emulation.

Test infrastructure.  The float64 oracle's block forward (pre-RMS LLaMA-shaped
or post-LN BERT-shaped), re-run with every intermediate that the bf16 HIP path
stores in bf16 rounded to bf16 (round to nearest even) and everything else in
float64, then the oracle's exact backward from those caches (and, for a loss
computed on the stage output, the loss gradient of the emulated output,
rounded to bf16 as the path stores it).  Its deviation from the plain oracle is a
lower bound on the error ANY implementation with bf16 intermediates incurs on
this workload (it ignores the backward's own roundings), and so a floor for
the parity tolerance of that workload.  Uses no value from the HIP path.
"""
from __future__ import annotations

import numpy as np

import oracle as O
from paper_2502_19864_amd.workloads import round_to_bf16

from helpers import oracle_desc, rel_err, to64


def _rb(a):
    return round_to_bf16(a.astype(np.float32)).astype(np.float64)


def llama_block_fwd_bf16(desc, w, ad, x, B, S):
    """oracle.llama_block_fwd with the bf16 path's storage roundings: the
    normalised GEMM inputs, the QKV projection (and Q, K after rotation), the
    attention output and out-projection, the adapter activations, the SwiGLU
    product, the FFN output, the residual stream."""
    H, eps = desc["n_heads"], desc["norm_eps"]
    d, F = x.shape[1], desc["d_ffn"]
    dh = d // H
    n1, xhat1, rstd1 = O.rms_norm(x, w["rms1_g"], eps)
    qkv = _rb(_rb(n1) @ w["w_qkv"])
    cos, sin = O.rope_tables(S, dh, desc["rope_theta"], x.dtype)
    q = _rb(O.rope_fwd(O.split_heads(qkv[:, :d], B, S, H), cos, sin))
    k = _rb(O.rope_fwd(O.split_heads(qkv[:, d:2 * d], B, S, H), cos, sin))
    v = O.split_heads(qkv[:, 2 * d:], B, S, H)
    o_h, p = O.attention_fwd(q, k, v, causal=True)
    attn = _rb(_rb(O.merge_heads(o_h)) @ w["w_o"])
    u1 = _rb(attn @ ad[0]["w_down"])
    h = x + attn + _rb(O.gelu(u1)) @ ad[0]["w_up"]
    n2, xhat2, rstd2 = O.rms_norm(h, w["rms2_g"], eps)
    h = _rb(h)
    gu = _rb(n2) @ w["w_gu"]
    gate, up = _rb(gu[:, :F]), _rb(gu[:, F:])
    f = _rb(_rb(O.silu(gate) * up) @ w["w_d"])
    u2 = _rb(f @ ad[1]["w_down"])
    y = _rb(h + f + _rb(O.gelu(u2)) @ ad[1]["w_up"])
    cache = dict(xhat1=xhat1, rstd1=rstd1, q=q, k=k, v=v, p=p, attn=attn, u1=u1, xhat2=xhat2,
                 rstd2=rstd2, gate=gate, up=up, f=f, u2=u2, cos=cos, sin=sin)
    return y, cache


def bert_block_fwd_bf16(desc, w, ad, x, B, S):
    """oracle.bert_block_fwd with the bf16 path's storage roundings: the QKV
    projection, the unnormalised attention probabilities fed to the PV
    product, the attention output and out-projection, the adapters' stashed
    down-projections and their GELU (fed to the up-projection), the LayerNorm
    outputs and their normalised inputs, the FFN pre-activation stash and its
    GELU, the FFN output."""
    H, eps = desc["n_heads"], desc["norm_eps"]
    d = x.shape[1]
    qkv = _rb(x @ w["w_qkv"] + w["b_qkv"])
    q = O.split_heads(qkv[:, :d], B, S, H)
    k = O.split_heads(qkv[:, d:2 * d], B, S, H)
    v = O.split_heads(qkv[:, 2 * d:], B, S, H)
    o_h, p = O.attention_fwd(q, k, v, causal=False)
    # the path feeds exp(s - max) to the PV product in bf16 and divides by the
    # float row sum afterwards
    s_ = q @ np.swapaxes(k, -1, -2) / np.sqrt(q.shape[-1])
    e_ = np.exp(s_ - s_.max(axis=-1, keepdims=True))
    o_h = (_rb(e_) @ v) / e_.sum(axis=-1, keepdims=True)
    attn = _rb(_rb(O.merge_heads(o_h)) @ w["w_o"] + w["b_o"])
    if desc.get("placement", "houlsby") == "ffn":
        U1, a = None, attn
    else:
        U1 = attn @ ad[0]["w_down"]
        a = attn + _rb(O.gelu(U1)) @ ad[0]["w_up"]
    h1, xhat1, rstd1 = O.layer_norm(x + a, w["ln1_g"], w["ln1_b"], eps)
    h1 = _rb(h1)
    A1 = h1 @ w["w_i"] + w["b_i"]
    f2 = _rb(_rb(O.gelu(A1)) @ w["w_f"] + w["b_f"])
    U2 = f2 @ ad[1]["w_down"]
    fa = f2 + _rb(O.gelu(U2)) @ ad[1]["w_up"]
    y, xhat2, rstd2 = O.layer_norm(h1 + fa, w["ln2_g"], w["ln2_b"], eps)
    cache = dict(q=q, k=k, v=v, p=p, attn=attn, u1=None if U1 is None else _rb(U1), xhat1=_rb(xhat1), rstd1=rstd1,
                 a1=_rb(A1),
                 f2=f2, u2=_rb(U2), xhat2=_rb(xhat2), rstd2=rstd2)
    return _rb(y), cache


def bert_floor(w, inp, c, ref):
    """Per-tensor deviation (max |.| / max |ref|) of the bf16-emulated run of
    a post-LN workload (its own loss included) from the oracle run `ref`
    (helpers.oracle_run at the same cut-off c): {'y': e, 'g_wh': e (CE loss),
    (l, a, name): e}."""
    desc = oracle_desc(w)
    W, A = to64(inp, w)
    x = np.asarray(inp["x"], np.float64)
    Bb, S, d = x.shape
    h = x.reshape(Bb * S, d)
    caches = []
    for l in range(w.n_blocks):
        h, cache = bert_block_fwd_bf16(desc, W[l], A[l], h, Bb, S)
        caches.append(cache)
    y = h.reshape(Bb, S, d)
    out = {"y": rel_err(y, ref["y"])}
    if w.loss == "cls_ce":
        _, dy, gwh, _ = O.cls_head_ce(y, inp["w_h"].astype(np.float64), inp["b_h"].astype(np.float64),
                                      inp["labels"])
        out["g_wh"] = rel_err(gwh, ref["g_wh"])
        dy = _rb(dy)
    elif w.loss == "mse":
        _, dy = O.mse_loss(y, inp["target"].astype(np.float64))
        dy = _rb(dy)
    else:
        dy = np.asarray(inp["dy"], np.float64)
    dx_emu, g_emu = O.stage_backward(desc, W, A, caches, dy, c)
    if c < 0 and ref.get("dx") is not None:
        out["dx"] = rel_err(dx_emu, ref["dx"])
    for l in range(max(c, 0), w.n_blocks):
        for a in range(2):
            if g_emu[l][a] is None:
                continue
            for k in ("w_down", "w_up"):
                out[(l, a, k)] = rel_err(g_emu[l][a][k], ref["grads"][l][a][k])
    return out


def floor_bound(floor, key):
    """Parity bound of one bf16 output tensor: the stated 2e-2, or twice the
    emulated storage floor of that tensor where the floor alone is beyond
    half of it."""
    return max(2e-2, 2.0 * floor[key])


def llama_floor(w, inp, c, dy, batch, seq, rows=None):
    """Per-tensor deviation (max |.| / max |ref|) of the bf16-emulated run
    from the oracle on x[:batch, :seq] (or on the samples listed in `rows`,
    first seq positions): {'y': e, 'dx': e (c < 0), (l, a, name): e}."""
    desc = oracle_desc(w)
    W, A = to64(inp, w)
    pick = slice(0, batch) if rows is None else list(rows)
    x = np.asarray(inp["x"], np.float64)[pick, :seq]
    dy = np.asarray(dy, np.float64)[pick, :seq]
    Bb, S, d = x.shape
    y_ref, c_ref = O.stage_forward(desc, W, A, x)
    dx_ref, g_ref = O.stage_backward(desc, W, A, c_ref, dy, c)
    h = x.reshape(Bb * S, d)
    caches = []
    for l in range(w.n_blocks):
        h, cache = llama_block_fwd_bf16(desc, W[l], A[l], h, Bb, S)
        caches.append(cache)
    dx_emu, g_emu = O.stage_backward(desc, W, A, caches, dy, c)
    out = {"y": rel_err(h.reshape(Bb, S, d), y_ref)}
    if c < 0:
        out["dx"] = rel_err(dx_emu, dx_ref)
    for l in range(max(c, 0), w.n_blocks):
        for a in range(2):
            for k in ("w_down", "w_up"):
                out[(l, a, k)] = rel_err(g_emu[l][a][k], g_ref[l][a][k])
    return out
