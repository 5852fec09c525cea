"""bf16 noise floor of the pre-RMS (LLaMA-shaped) stage, by emulation.

Test infrastructure.  The float64 oracle's pre-RMS block forward, re-run with
every intermediate that the bf16 HIP path stores in bf16 rounded to bf16
(round to nearest even) and everything else in float64, then the oracle's
exact backward from those caches.  Its deviation from the plain oracle is a
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


def llama_floor(w, inp, c, dy, batch, seq):
    """Per-tensor deviation (max |.| / max |ref|) of the bf16-emulated run
    from the oracle on x[:batch, :seq]: {'y': e, (l, a, name): e}."""
    desc = oracle_desc(w)
    W, A = to64(inp, w)
    x = np.asarray(inp["x"], np.float64)[:batch, :seq]
    dy = np.asarray(dy, np.float64)[:batch, :seq]
    Bb, S, d = x.shape
    y_ref, c_ref = O.stage_forward(desc, W, A, x)
    _, g_ref = O.stage_backward(desc, W, A, c_ref, dy, c)
    h = x.reshape(Bb * S, d)
    caches = []
    for l in range(w.n_blocks):
        h, cache = llama_block_fwd_bf16(desc, W[l], A[l], h, Bb, S)
        caches.append(cache)
    _, g_emu = O.stage_backward(desc, W, A, caches, dy, c)
    out = {"y": rel_err(h.reshape(Bb, S, d), y_ref)}
    for l in range(max(c, 0), w.n_blocks):
        for a in range(2):
            for k in ("w_down", "w_up"):
                out[(l, a, k)] = rel_err(g_emu[l][a][k], g_ref[l][a][k])
    return out
