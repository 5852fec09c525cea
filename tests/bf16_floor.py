"""bf16 noise floor of the stage, by emulation.

Test infrastructure.  The float64 oracle's block forward and backward
(pre-RMS LLaMA-shaped or post-LN BERT-shaped), re-run with every
intermediate that the bf16 HIP path stores or feeds to a matrix product in
bf16 rounded to bf16 (round to nearest even), and everything else in
float64:

* forward: the normalised GEMM inputs, the QKV projection (Q and K after the
  rotation), the unnormalised attention probabilities fed to the PV product,
  the attention output and the out-projection, the adapters' stashed
  down-projections and their GELU, the LayerNorm outputs and normalised
  inputs, the FFN pre-activation stash and its activation, the FFN output,
  the residual stream, the loss gradient;
* backward: the gradient at each adapter's output (stored, and the operand
  of dZ W_up^T and of the W_up gradient), the adapter's dU, the gradient at
  its input, the FFN's activation gradient (GELU' or SwiGLU), the gradient
  entering each norm backward, the attention-output gradient dO, the
  recomputed probabilities and dS fed to the attention backward's products,
  the QKV gradient, the RMSNorm-1 input gradient and the gradient passed
  between blocks.

Its deviation from the plain oracle is the error that storage precision
alone causes on this workload, and so the floor of the parity tolerance of
that workload.  Uses no value from the HIP path, and none of its code.
"""
from __future__ import annotations

import math

import numpy as np

import oracle as O
from paper_2502_19864_amd.workloads import round_to_bf16

from helpers import oracle_desc, rel_err, to64

# a bf16 tensor's parity bound: the stated 2e-2, or this factor times the
# emulated storage floor of that tensor where the floor leaves no room under it
FLOOR_MARGIN = 1.25
TOL_BF16 = 2e-2


def _rb(a):
    return round_to_bf16(np.asarray(a, np.float64).astype(np.float32)).astype(np.float64)


# ---------------------------------------------------------------- attention
def _attn_fwd(q, k, v, causal):
    """Attention as the path computes it: exp(s - rowmax) fed to the PV
    product in bf16, divided by the float row sum afterwards.  Returns (o, p)
    with p the exact normalised probabilities (the backward recomputes them
    from the stashed log-sum-exp)."""
    dh = q.shape[-1]
    s = (q @ np.swapaxes(k, -1, -2)) / math.sqrt(dh)
    if causal:
        S = s.shape[-1]
        s = np.where(np.triu(np.ones((S, S), dtype=bool), 1), -np.inf, s)
    e = np.exp(s - s.max(axis=-1, keepdims=True))
    den = e.sum(axis=-1, keepdims=True)
    return (_rb(e) @ v) / den, e / den


def _attn_bwd(do, q, k, v, o, p):
    """Attention backward as the path computes it: the row sum D from the
    stored dO and O, P and dS rounded to bf16 as operands of their products."""
    dh = q.shape[-1]
    dsum = (do * o).sum(axis=-1, keepdims=True)
    pb = _rb(p)
    dv = np.swapaxes(pb, -1, -2) @ do
    dp = do @ np.swapaxes(v, -1, -2)
    ds = _rb(p * (dp - dsum))
    dq = (ds @ k) / math.sqrt(dh)
    dk = (np.swapaxes(ds, -1, -2) @ q) / math.sqrt(dh)
    return dq, dk, dv


# ---------------------------------------------------------------- adapter backward
def _adapter_bwd(dz, z, u, w_down, w_up, need_dzin):
    """Eq. (1)'s backward as the path stores it.  dz: float gradient at the
    adapter output.  Returns (dz_b, dzin or None, dW_down, dW_up) with dz_b
    the stored bf16 copy that later products read."""
    dz_b = _rb(dz)
    du = _rb((dz_b @ w_up.T) * O.gelu_grad(u))
    gdn = z.T @ du
    gup = _rb(O.gelu(u)).T @ dz_b
    dzin = _rb(dz + du @ w_down.T) if need_dzin else None
    return dz_b, dzin, gdn, gup


# ---------------------------------------------------------------- post-LN block
def bert_block_fwd_bf16(desc, w, ad, x, B, S):
    H, eps = desc["n_heads"], desc["norm_eps"]
    d = x.shape[1]
    qkv = _rb(x @ w["w_qkv"] + w["b_qkv"])
    q = O.split_heads(qkv[:, :d], B, S, H)
    k = O.split_heads(qkv[:, d:2 * d], B, S, H)
    v = O.split_heads(qkv[:, 2 * d:], B, S, H)
    o_h, p = _attn_fwd(q, k, v, causal=False)
    o = _rb(O.merge_heads(o_h))
    attn = _rb(o @ w["w_o"] + w["b_o"])
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
    cache = dict(q=q, k=k, v=v, p=p, o=o, attn=attn, u1=None if U1 is None else _rb(U1), xhat1=_rb(xhat1),
                 rstd1=rstd1, a1=_rb(A1), f2=f2, u2=_rb(U2), xhat2=_rb(xhat2), rstd2=rstd2)
    return _rb(y), cache


def bert_block_bwd_bf16(desc, w, ad, c, dy, B, S, stop):
    single = desc.get("placement", "houlsby") == "ffn"
    H = desc["n_heads"]
    dz2 = O.layer_norm_bwd(dy, w["ln2_g"], c["xhat2"], c["rstd2"])
    dz2_b, df2, gdn2, gup2 = _adapter_bwd(dz2, c["f2"], c["u2"], ad[1]["w_down"], ad[1]["w_up"],
                                          need_dzin=not (single and stop))
    g_ffn = {"w_down": gdn2, "w_up": gup2}
    if single and stop:
        return None, (None, g_ffn)
    da1 = _rb((df2 @ w["w_f"].T) * O.gelu_grad(c["a1"]))
    dh1 = _rb(dz2_b + da1 @ w["w_i"].T)
    dz1 = O.layer_norm_bwd(dh1, w["ln1_g"], c["xhat1"], c["rstd1"])
    if single:
        dz1_b = dattn = _rb(dz1)
        grads = (None, g_ffn)
    else:
        dz1_b, dattn, gdn1, gup1 = _adapter_bwd(dz1, c["attn"], c["u1"], ad[0]["w_down"], ad[0]["w_up"],
                                                need_dzin=not stop)
        grads = ({"w_down": gdn1, "w_up": gup1}, g_ffn)
    if stop:
        return None, grads
    do = _rb(dattn @ w["w_o"].T)
    dq, dk, dv = _attn_bwd(O.split_heads(do, B, S, H), c["q"], c["k"], c["v"],
                           O.split_heads(c["o"], B, S, H), c["p"])
    dqkv = _rb(np.concatenate([O.merge_heads(dq), O.merge_heads(dk), O.merge_heads(dv)], axis=1))
    dx = _rb(dz1_b + dqkv @ w["w_qkv"].T)
    return dx, grads


# ---------------------------------------------------------------- pre-RMS block
def llama_block_fwd_bf16(desc, w, ad, x, B, S):
    H, eps = desc["n_heads"], desc["norm_eps"]
    d, F = x.shape[1], desc["d_ffn"]
    dh = d // H
    n1, xhat1, rstd1 = O.rms_norm(x, w["rms1_g"], eps)
    qkv = _rb(_rb(n1) @ w["w_qkv"])
    cos, sin = O.rope_tables(S, dh, desc["rope_theta"], x.dtype)
    q = _rb(O.rope_fwd(O.split_heads(qkv[:, :d], B, S, H), cos, sin))
    k = _rb(O.rope_fwd(O.split_heads(qkv[:, d:2 * d], B, S, H), cos, sin))
    v = O.split_heads(qkv[:, 2 * d:], B, S, H)
    o_h, p = _attn_fwd(q, k, v, causal=True)
    o = _rb(O.merge_heads(o_h))
    attn = _rb(o @ w["w_o"])
    if desc.get("placement", "houlsby") == "ffn":
        U1, a = None, attn
    else:
        U1 = attn @ ad[0]["w_down"]
        a = attn + _rb(O.gelu(U1)) @ ad[0]["w_up"]
    h = x + a
    n2, xhat2, rstd2 = O.rms_norm(h, w["rms2_g"], eps)
    h = _rb(h)
    gu = _rb(n2) @ w["w_gu"]
    gate, up = _rb(gu[:, :F]), _rb(gu[:, F:])
    f = _rb(_rb(O.silu(gate) * up) @ w["w_d"])
    u2 = f @ ad[1]["w_down"]
    y = _rb(h + f + _rb(O.gelu(u2)) @ ad[1]["w_up"])
    cache = dict(xhat1=_rb(xhat1), rstd1=rstd1, q=q, k=k, v=v, p=p, o=o, attn=attn,
                 u1=None if U1 is None else _rb(U1), xhat2=_rb(xhat2), rstd2=rstd2, gate=gate, up=up, f=f,
                 u2=_rb(u2), cos=cos, sin=sin)
    return y, cache


def llama_block_bwd_bf16(desc, w, ad, c, dy, B, S, stop):
    F, H = desc["d_ffn"], desc["n_heads"]
    single = desc.get("placement", "houlsby") == "ffn"
    _, df, gdn2, gup2 = _adapter_bwd(dy, c["f"], c["u2"], ad[1]["w_down"], ad[1]["w_up"],
                                     need_dzin=not (single and stop))
    g_ffn = {"w_down": gdn2, "w_up": gup2}
    if single and stop:
        return None, (None, g_ffn)
    dact = df @ w["w_d"].T
    dgate = _rb(dact * c["up"] * O.silu_grad(c["gate"]))
    dup = _rb(dact * O.silu(c["gate"]))
    dn2 = _rb(np.concatenate([dgate, dup], axis=1) @ w["w_gu"].T)
    dh = dy + O.rms_norm_bwd(dn2, w["rms2_g"], c["xhat2"], c["rstd2"])
    if single:
        dh_b = dattn = _rb(dh)
        grads = (None, g_ffn)
    else:
        dh_b, dattn, gdn1, gup1 = _adapter_bwd(dh, c["attn"], c["u1"], ad[0]["w_down"], ad[0]["w_up"],
                                               need_dzin=not stop)
        grads = ({"w_down": gdn1, "w_up": gup1}, g_ffn)
    if stop:
        return None, grads
    do = _rb(dattn @ w["w_o"].T)
    dq, dk, dv = _attn_bwd(O.split_heads(do, B, S, H), c["q"], c["k"], c["v"],
                           O.split_heads(c["o"], B, S, H), c["p"])
    dq = O.rope_bwd(dq, c["cos"], c["sin"])
    dk = O.rope_bwd(dk, c["cos"], c["sin"])
    dqkv = _rb(np.concatenate([O.merge_heads(dq), O.merge_heads(dk), O.merge_heads(dv)], axis=1))
    dn1 = _rb(dqkv @ w["w_qkv"].T)
    dx = _rb(dh_b + O.rms_norm_bwd(dn1, w["rms1_g"], c["xhat1"], c["rstd1"]))
    return dx, grads


_BLOCK = {"bert": (bert_block_fwd_bf16, bert_block_bwd_bf16),
          "llama": (llama_block_fwd_bf16, llama_block_bwd_bf16)}


# ---------------------------------------------------------------- stage
def emulate_stage(w, inp, c, x=None, dy=None, labels=None):
    """Forward, loss (or the given dy) and early-stopped backward of workload
    `w` with the bf16 roundings of the path, on x (default: the workload's
    whole input).  Returns {'y', 'dx' (c < 0), 'grads', 'g_wh' (CE loss)}."""
    desc = oracle_desc(w)
    W, A = to64(inp, w)
    x = np.asarray(inp["x"] if x is None else x, np.float64)
    Bb, S, d = x.shape
    fwd, bwd = _BLOCK[w.arch]
    h = x.reshape(Bb * S, d)
    caches = []
    for l in range(w.n_blocks):
        h, cache = fwd(desc, W[l], A[l], h, Bb, S)
        caches.append(cache)
    y = h.reshape(Bb, S, d)
    out = {"y": y}
    if dy is None and w.loss == "cls_ce":
        lab = inp["labels"] if labels is None else labels
        _, dy, out["g_wh"], _ = O.cls_head_ce(y, inp["w_h"].astype(np.float64), inp["b_h"].astype(np.float64), lab)
        dy = _rb(dy)
    elif dy is None and w.loss == "mse":
        _, dy = O.mse_loss(y, inp["target"].astype(np.float64))
        dy = _rb(dy)
    elif dy is None:
        dy = inp["dy"]
    dy = np.asarray(dy, np.float64)
    L = w.n_blocks
    grads = [None] * L
    g = dy.reshape(Bb * S, d)
    if c < L:
        for l in range(L - 1, max(c, 0) - 1, -1):
            g, grads[l] = bwd(desc, W[l], A[l], caches[l], g, Bb, S, l == c)
    out["dx"] = g.reshape(Bb, S, d) if c < 0 else None
    out["grads"] = grads
    return out


def rel_err_parts(got, ref):
    """rel_err of several pieces of one output tensor taken together:
    max |got - ref| over all pieces / max |ref| over all pieces."""
    num = max(float(np.abs(np.asarray(g, np.float64) - np.asarray(r, np.float64)).max()) for g, r in zip(got, ref))
    den = max(float(np.abs(np.asarray(r, np.float64)).max()) for r in ref)
    return num / (den if den > 0 else 1.0)


def sum_grads(parts):
    """Adapter gradients summed over runs on disjoint samples."""
    out = parts[0]
    for gr in parts[1:]:
        out = [None if a is None else tuple(None if p is None else {k: p[k] + q[k] for k in p}
                                              for p, q in zip(a, b))
               for a, b in zip(out, gr)]
    return out


def stage_floor(w, inp, c, refs, parts=None):
    """Per-tensor storage floor: {'y', 'dx' (c < 0), 'g_wh' (CE loss),
    (l, a, name)} -> max |emulated - oracle| / max |oracle|.  `refs` are
    helpers.oracle_run results at cut-off c, one per entry of `parts` (a list
    of (x, dy) pieces of the input; default one piece: the whole input with
    the workload's own loss or dy).  Gradients of several pieces are summed,
    as the GPU accumulates them over its whole batch."""
    if parts is None:
        parts = [(None, None)]
    if isinstance(refs, dict):
        refs = [refs]
    emus = [emulate_stage(w, inp, c, x, dy) for x, dy in parts]
    out = {"y": rel_err_parts([e["y"] for e in emus], [r["y"] for r in refs])}
    if "g_wh" in emus[0] and "g_wh" in refs[0]:
        out["g_wh"] = rel_err(sum(e["g_wh"] for e in emus), sum(r["g_wh"] for r in refs))
    if c < 0:
        out["dx"] = rel_err_parts([e["dx"] for e in emus], [r["dx"] for r in refs])
    ge = sum_grads([e["grads"] for e in emus])
    gr = sum_grads([r["grads"] for r in refs])
    for l in range(max(c, 0), w.n_blocks):
        for a in range(2):
            if ge[l] is None or ge[l][a] is None:
                continue
            for k in ("w_down", "w_up"):
                out[(l, a, k)] = rel_err(ge[l][a][k], gr[l][a][k])
    return out


def floor_bound(floor, key):
    """Parity bound of one bf16 output tensor: the stated 2e-2, or
    FLOOR_MARGIN times the emulated storage floor where the floor alone
    leaves less room than that under 2e-2."""
    return max(TOL_BF16, FLOOR_MARGIN * floor[key])
