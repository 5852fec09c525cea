"""Plain CPU oracle for one RingAda ring stage (arXiv 2502.19864).

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this module: it is used by ``tests/``, by ``__graft_entry__.smoke()``
(as the reference the GPU result is compared with) and by the ``cpu_baseline``
leg of ``bench.py``.  It shares
no code with the HIP library.

What it computes
----------------
One client of the ring hosts a contiguous run of frozen transformer blocks
(the Trm layers of Sec. III-A), each carrying two bottleneck adapters of the
form of Eq. (1) (after the attention sublayer and after the feed-forward
sublayer).  A training iteration on the client is

* the forward pass through its blocks (Sec. III-B, "Forward and Backward
  Propagation");
* a backward pass that relays the incoming gradient down through the frozen
  weights and produces weight gradients only for unfrozen adapters, ending
  at the lowest unfrozen adapter (Alg. 1, the backward step that ends at the
  (L-d+1)-th adapter; Sec. III-B, the terminator);
* an update of the unfrozen adapters (Sec. III-B: clients with unfrozen
  adapters update them; the optimiser is not named, plain SGD is used).

Early stopping and frozen-weight-only backprop do not change any value that
is produced: they only skip work whose result is not needed.  So this file
writes out the plain definitions (forward equations, exact reverse-mode
gradients) with library matmuls as steps and no fusion or reordering.
Everything is computed in the dtype of the inputs (float64 for parity,
float32 for the CPU timing baseline).

Readings where the paper is silent (each is listed in the design notes):
  * sigma in Eq. (1) is GELU in its exact erf form;
  * an adapter acts on its sublayer's output before the block's residual
    add (and before the LayerNorm in post-LN blocks);
  * two adapters per block (Houlsby placement); both unfreeze together.
    The single serial placement of Sec. II-A (Fig. 1: one adapter, after the
    feed-forward sublayer) is the option placement='ffn': the attention
    sublayer then carries no adapter, and the backward of the lowest
    unfrozen block ends after that block's FFN-adapter weight gradients;
  * adapters have no biases, exactly as in Eq. (1);
  * weights are stored [in, out] so a projection is ``x @ W`` as in Eq. (1);
  * the unfreezing cut-off of Alg. 1 uses L = total number of Trm blocks.

Pins: see tests/test_oracle_pins.py (finite differences in float64, an
independent torch-autograd implementation, closed forms and invariants, and
the worked four-client example of Sec. III-A).
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import erf

# --------------------------------------------------------------------------
# elementwise functions
# --------------------------------------------------------------------------
_SQRT2 = math.sqrt(2.0)
_INV_SQRT_2PI = 1.0 / math.sqrt(2.0 * math.pi)


def gelu(u):
    """GELU, exact erf form: u * Phi(u)  (the sigma of Eq. (1))."""
    return 0.5 * u * (1.0 + erf(u / _SQRT2))


def gelu_grad(u):
    """d/du [u * Phi(u)] = Phi(u) + u * phi(u)."""
    cdf = 0.5 * (1.0 + erf(u / _SQRT2))
    pdf = np.exp(-0.5 * u * u) * _INV_SQRT_2PI
    return cdf + u * pdf


def silu(u):
    return u / (1.0 + np.exp(-u))


def silu_grad(u):
    s = 1.0 / (1.0 + np.exp(-u))
    return s + u * s * (1.0 - s)


# --------------------------------------------------------------------------
# normalisation
# --------------------------------------------------------------------------
def layer_norm(x, gamma, beta, eps):
    """LayerNorm over the last axis with biased variance."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + eps)
    xhat = (x - mu) * rstd
    return xhat * gamma + beta, xhat, rstd


def layer_norm_bwd(dy, gamma, xhat, rstd):
    """Gradient of LayerNorm w.r.t. its input (gamma, beta frozen)."""
    g = dy * gamma
    return rstd * (g - g.mean(axis=-1, keepdims=True)
                   - xhat * (g * xhat).mean(axis=-1, keepdims=True))


def rms_norm(x, gain, eps):
    rstd = 1.0 / np.sqrt((x * x).mean(axis=-1, keepdims=True) + eps)
    xhat = x * rstd
    return xhat * gain, xhat, rstd


def rms_norm_bwd(dy, gain, xhat, rstd):
    g = dy * gain
    return rstd * (g - xhat * (g * xhat).mean(axis=-1, keepdims=True))


# --------------------------------------------------------------------------
# adapter, Eq. (1):  h <- h + sigma(h W_down) W_up
# --------------------------------------------------------------------------
def adapter_fwd(h, w_down, w_up):
    u = h @ w_down
    return h + gelu(u) @ w_up, u


def adapter_bwd(dout, h, u, w_down, w_up, need_dh=True):
    """Returns (dh or None, dW_down, dW_up) for out = h + gelu(h W_dn) W_up."""
    g = gelu(u)
    dw_up = g.T @ dout
    du = (dout @ w_up.T) * gelu_grad(u)
    dw_down = h.T @ du
    dh = dout + du @ w_down.T if need_dh else None
    return dh, dw_down, dw_up


# --------------------------------------------------------------------------
# attention
# --------------------------------------------------------------------------
def split_heads(x, B, S, H):
    """[B*S, H*dh] -> [B, H, S, dh]; head h owns columns [h*dh, (h+1)*dh)."""
    dh = x.shape[1] // H
    return x.reshape(B, S, H, dh).transpose(0, 2, 1, 3)


def merge_heads(x):
    B, H, S, dh = x.shape
    return x.transpose(0, 2, 1, 3).reshape(B * S, H * dh)


def attention_fwd(q, k, v, causal):
    """softmax(q k^T / sqrt(dh) [+ causal mask]) v over [B, H, S, dh]."""
    dh = q.shape[-1]
    s = (q @ np.swapaxes(k, -1, -2)) / math.sqrt(dh)
    if causal:
        S = s.shape[-1]
        s = np.where(np.triu(np.ones((S, S), dtype=bool), 1), -np.inf, s)
    s = s - s.max(axis=-1, keepdims=True)
    e = np.exp(s)
    p = e / e.sum(axis=-1, keepdims=True)
    return p @ v, p


def attention_bwd(do, q, k, v, p):
    """Adjoint of attention_fwd (the mask is already folded into p)."""
    dh = q.shape[-1]
    dv = np.swapaxes(p, -1, -2) @ do
    dp = do @ np.swapaxes(v, -1, -2)
    ds = p * (dp - (dp * p).sum(axis=-1, keepdims=True))
    dq = (ds @ k) / math.sqrt(dh)
    dk = (np.swapaxes(ds, -1, -2) @ q) / math.sqrt(dh)
    return dq, dk, dv


def rope_tables(S, dh, theta, dtype):
    """cos/sin of angle pos * theta^(-2i/dh), pos in [0,S), i in [0, dh/2)."""
    half = dh // 2
    inv_freq = theta ** (-(2.0 * np.arange(half, dtype=np.float64)) / dh)
    ang = np.arange(S, dtype=np.float64)[:, None] * inv_freq[None, :]
    return np.cos(ang).astype(dtype), np.sin(ang).astype(dtype)


def rope_fwd(x, cos, sin):
    """Rotate-half RoPE on [B, H, S, dh]: pairs (i, i + dh/2)."""
    half = x.shape[-1] // 2
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)


def rope_bwd(dy, cos, sin):
    """Adjoint of rope_fwd: the inverse (transposed) rotation."""
    half = dy.shape[-1] // 2
    d1, d2 = dy[..., :half], dy[..., half:]
    return np.concatenate([d1 * cos + d2 * sin, d2 * cos - d1 * sin], axis=-1)


# --------------------------------------------------------------------------
# stage description
# --------------------------------------------------------------------------
def make_desc(arch, n_blocks, d_model, n_heads, d_ffn, d_adapter,
              norm_eps=None, rope_theta=10000.0, placement="houlsby"):
    """arch is 'bert' (post-LN, GELU FFN, bidirectional) or 'llama'
    (pre-RMSNorm, SwiGLU FFN, RoPE, causal).  placement is 'houlsby' (an
    adapter on the attention and on the FFN sublayer of every block) or
    'ffn' (the single adapter after the feed-forward sublayer, Sec. II-A)."""
    if norm_eps is None:
        norm_eps = 1e-12 if arch == "bert" else 1e-6
    assert placement in ("houlsby", "ffn")
    return dict(arch=arch, n_blocks=n_blocks, d_model=d_model, n_heads=n_heads,
                d_ffn=d_ffn, d_adapter=d_adapter, norm_eps=norm_eps,
                rope_theta=rope_theta, placement=placement)


def _single(desc):
    return desc.get("placement", "houlsby") == "ffn"


# --------------------------------------------------------------------------
# post-LN encoder block (BERT shape)
# --------------------------------------------------------------------------
def bert_block_fwd(desc, w, ad, x, B, S):
    """x: [B*S, d].  w: frozen weights, ad: (attn_adapter, ffn_adapter)."""
    H, eps = desc["n_heads"], desc["norm_eps"]
    qkv = x @ w["w_qkv"] + w["b_qkv"]
    d = x.shape[1]
    q = split_heads(qkv[:, :d], B, S, H)
    k = split_heads(qkv[:, d:2 * d], B, S, H)
    v = split_heads(qkv[:, 2 * d:], B, S, H)
    o_h, p = attention_fwd(q, k, v, causal=False)
    o = merge_heads(o_h)
    attn = o @ w["w_o"] + w["b_o"]
    if _single(desc):
        a, u1 = attn, None
    else:
        a, u1 = adapter_fwd(attn, ad[0]["w_down"], ad[0]["w_up"])
    h1, xhat1, rstd1 = layer_norm(x + a, w["ln1_g"], w["ln1_b"], eps)
    a1 = h1 @ w["w_i"] + w["b_i"]
    f2 = gelu(a1) @ w["w_f"] + w["b_f"]
    fa, u2 = adapter_fwd(f2, ad[1]["w_down"], ad[1]["w_up"])
    y, xhat2, rstd2 = layer_norm(h1 + fa, w["ln2_g"], w["ln2_b"], eps)
    cache = dict(q=q, k=k, v=v, p=p, attn=attn, u1=u1, xhat1=xhat1,
                 rstd1=rstd1, a1=a1, f2=f2, u2=u2, xhat2=xhat2, rstd2=rstd2)
    return y, cache


def bert_block_bwd(desc, w, ad, c, dy, B, S, stop):
    """Backward of one post-LN block.  Returns (dx or None, adapter grads),
    grads = (attention adapter or None, FFN adapter).  With stop=True the
    pass ends after the weight gradients of the block's lowest adapter (the
    attention adapter; the FFN adapter under the single placement): no
    gradient reaches the block input."""
    single = _single(desc)
    dz2 = layer_norm_bwd(dy, w["ln2_g"], c["xhat2"], c["rstd2"])
    df2, gdn2, gup2 = adapter_bwd(dz2, c["f2"], c["u2"],
                                  ad[1]["w_down"], ad[1]["w_up"],
                                  need_dh=not (single and stop))
    g_ffn = {"w_down": gdn2, "w_up": gup2}
    if single and stop:
        return None, (None, g_ffn)
    da1 = (df2 @ w["w_f"].T) * gelu_grad(c["a1"])
    dh1 = dz2 + da1 @ w["w_i"].T
    dz1 = layer_norm_bwd(dh1, w["ln1_g"], c["xhat1"], c["rstd1"])
    if single:
        dattn, grads = dz1, (None, g_ffn)
    else:
        dattn, gdn1, gup1 = adapter_bwd(dz1, c["attn"], c["u1"],
                                        ad[0]["w_down"], ad[0]["w_up"],
                                        need_dh=not stop)
        grads = ({"w_down": gdn1, "w_up": gup1}, g_ffn)
    if stop:
        return None, grads
    do = split_heads(dattn @ w["w_o"].T, B, S, desc["n_heads"])
    dq, dk, dv = attention_bwd(do, c["q"], c["k"], c["v"], c["p"])
    dqkv = np.concatenate([merge_heads(dq), merge_heads(dk), merge_heads(dv)],
                          axis=1)
    dx = dz1 + dqkv @ w["w_qkv"].T
    return dx, grads


# --------------------------------------------------------------------------
# pre-RMSNorm causal decoder block (LLaMA shape)
# --------------------------------------------------------------------------
def llama_block_fwd(desc, w, ad, x, B, S):
    H, eps = desc["n_heads"], desc["norm_eps"]
    d, F = x.shape[1], desc["d_ffn"]
    dh = d // H
    n1, xhat1, rstd1 = rms_norm(x, w["rms1_g"], eps)
    qkv = n1 @ w["w_qkv"]
    cos, sin = rope_tables(S, dh, desc["rope_theta"], x.dtype)
    q = rope_fwd(split_heads(qkv[:, :d], B, S, H), cos, sin)
    k = rope_fwd(split_heads(qkv[:, d:2 * d], B, S, H), cos, sin)
    v = split_heads(qkv[:, 2 * d:], B, S, H)
    o_h, p = attention_fwd(q, k, v, causal=True)
    attn = merge_heads(o_h) @ w["w_o"]
    if _single(desc):
        a, u1 = attn, None
    else:
        a, u1 = adapter_fwd(attn, ad[0]["w_down"], ad[0]["w_up"])
    h = x + a
    n2, xhat2, rstd2 = rms_norm(h, w["rms2_g"], eps)
    gu = n2 @ w["w_gu"]
    gate, up = gu[:, :F], gu[:, F:]
    f = (silu(gate) * up) @ w["w_d"]
    fa, u2 = adapter_fwd(f, ad[1]["w_down"], ad[1]["w_up"])
    y = h + fa
    cache = dict(xhat1=xhat1, rstd1=rstd1, q=q, k=k, v=v, p=p, attn=attn,
                 u1=u1, xhat2=xhat2, rstd2=rstd2, gate=gate, up=up, f=f,
                 u2=u2, cos=cos, sin=sin)
    return y, cache


def llama_block_bwd(desc, w, ad, c, dy, B, S, stop):
    F, H = desc["d_ffn"], desc["n_heads"]
    single = _single(desc)
    dh_res = dy
    df, gdn2, gup2 = adapter_bwd(dy, c["f"], c["u2"],
                                 ad[1]["w_down"], ad[1]["w_up"],
                                 need_dh=not (single and stop))
    g_ffn = {"w_down": gdn2, "w_up": gup2}
    if single and stop:
        return None, (None, g_ffn)
    dact = df @ w["w_d"].T
    dgate = dact * c["up"] * silu_grad(c["gate"])
    dup = dact * silu(c["gate"])
    dn2 = np.concatenate([dgate, dup], axis=1) @ w["w_gu"].T
    dh = dh_res + rms_norm_bwd(dn2, w["rms2_g"], c["xhat2"], c["rstd2"])
    if single:
        dattn, grads = dh, (None, g_ffn)
    else:
        dattn, gdn1, gup1 = adapter_bwd(dh, c["attn"], c["u1"],
                                        ad[0]["w_down"], ad[0]["w_up"],
                                        need_dh=not stop)
        grads = ({"w_down": gdn1, "w_up": gup1}, g_ffn)
    if stop:
        return None, grads
    do = split_heads(dattn @ w["w_o"].T, B, S, H)
    dq, dk, dv = attention_bwd(do, c["q"], c["k"], c["v"], c["p"])
    dq = rope_bwd(dq, c["cos"], c["sin"])
    dk = rope_bwd(dk, c["cos"], c["sin"])
    dqkv = np.concatenate([merge_heads(dq), merge_heads(dk), merge_heads(dv)],
                          axis=1)
    dn1 = dqkv @ w["w_qkv"].T
    dx = dh + rms_norm_bwd(dn1, w["rms1_g"], c["xhat1"], c["rstd1"])
    return dx, grads


_BLOCK = {"bert": (bert_block_fwd, bert_block_bwd),
          "llama": (llama_block_fwd, llama_block_bwd)}


# --------------------------------------------------------------------------
# stage
# --------------------------------------------------------------------------
def stage_forward(desc, weights, adapters, x):
    """x: [B, S, d].  Returns (y [B, S, d], per-block caches)."""
    B, S, d = x.shape
    fwd = _BLOCK[desc["arch"]][0]
    h = x.reshape(B * S, d)
    caches = []
    for l in range(desc["n_blocks"]):
        h, cache = fwd(desc, weights[l], adapters[l], h, B, S)
        caches.append(cache)
    return h.reshape(B, S, d), caches


def stage_backward(desc, weights, adapters, caches, dy, lowest_unfrozen):
    """Early-stopped backward of the stage.

    lowest_unfrozen = c (local, 0-indexed):
      c < 0       every local adapter is unfrozen; the gradient w.r.t. the
                  stage input is returned (the cut-off is upstream);
      0 <= c < L  blocks c..L-1 have unfrozen adapters; the pass ends after
                  the weight gradients of block c's lowest adapter (its
                  attention adapter, or its FFN adapter under the single
                  placement);
      c >= L      all adapters frozen: no backward at all.
    Returns (dx_in or None, grads) with grads[l] = (attn, ffn) dicts for the
    unfrozen blocks (attn is None under the single placement) and None for
    the frozen ones.
    """
    B, S, d = dy.shape
    L = desc["n_blocks"]
    bwd = _BLOCK[desc["arch"]][1]
    grads = [None] * L
    if lowest_unfrozen >= L:
        return None, grads
    g = dy.reshape(B * S, d)
    stop_at = max(lowest_unfrozen, 0)
    for l in range(L - 1, stop_at - 1, -1):
        stop = (l == lowest_unfrozen)
        g, grads[l] = bwd(desc, weights[l], adapters[l], caches[l], g, B, S,
                          stop)
    dx = None if lowest_unfrozen >= 0 else g.reshape(B, S, d)
    return dx, grads


def sgd_step(adapters, grads, lr):
    """w <- w - lr * g for every adapter that has a gradient; returns new
    adapter list (inputs untouched)."""
    out = []
    for ad, gr in zip(adapters, grads):
        if gr is None:
            out.append(ad)
            continue
        out.append(tuple(a if g is None else {k: a[k] - lr * g[k] for k in ("w_down", "w_up")}
                         for a, g in zip(ad, gr)))
    return out


# --------------------------------------------------------------------------
# losses computed by the initiator (Alg. 1: the initiator computes the loss
# and updates the head)
# --------------------------------------------------------------------------
def mse_loss(y, target):
    """mean over every element; returns (loss, dL/dy)."""
    diff = y - target
    n = diff.size
    return (diff * diff).sum() / n, 2.0 * diff / n


def cls_head_ce(y, w_h, b_h, labels):
    """Linear head on position 0 ([CLS]) + softmax cross-entropy, mean over
    the batch.  Returns (loss, dy, dW_h, db_h)."""
    B = y.shape[0]
    y0 = y[:, 0, :]
    logits = y0 @ w_h + b_h
    z = logits - logits.max(axis=1, keepdims=True)
    logp = z - np.log(np.exp(z).sum(axis=1, keepdims=True))
    loss = -logp[np.arange(B), labels].mean()
    dlogits = np.exp(logp)
    dlogits[np.arange(B), labels] -= 1.0
    dlogits /= B
    dy = np.zeros_like(y)
    dy[:, 0, :] = dlogits @ w_h.T
    return loss, dy, y0.T @ dlogits, dlogits.sum(axis=0)


# --------------------------------------------------------------------------
# ring bookkeeping (Sec. III-B and Alg. 1)
# --------------------------------------------------------------------------
def client_roles(assignment, depth):
    """assignment: list of (beta, eps), 1-indexed inclusive Trm ranges in ring
    order; depth: unfreezing depth Dep.  Returns, per client, one of
    'forward-only' (eps <= N_TM - Dep), 'terminator'
    (beta <= N_TM - Dep + 1 <= eps) or 'backward' (the rest)."""
    n_tm = max(e for _, e in assignment)
    roles = []
    for beta, eps in assignment:
        if eps <= n_tm - depth:
            roles.append("forward-only")
        elif beta <= n_tm - depth + 1 <= eps:
            roles.append("terminator")
        else:
            roles.append("backward")
    return roles


def cutoff_block(n_tm, depth):
    """1-indexed block whose adapter ends the backward: the (L - d + 1)-th,
    with L the number of Trm blocks."""
    return n_tm - depth + 1


def local_lowest_unfrozen(n_tm, depth, beta, eps):
    """The stage argument c for a client holding 1-indexed blocks beta..eps:
    -1 if the cut-off lies below the client, eps-beta+1 if the client is
    forward-only, else the 0-indexed local block of the cut-off."""
    cut = cutoff_block(n_tm, depth)
    if cut < beta:
        return -1
    if cut > eps:
        return eps - beta + 1
    return cut - beta


# --------------------------------------------------------------------------
# the top-down unfreezing schedule on one stage (Alg. 1)
# --------------------------------------------------------------------------
def depth_of_round(r, d0, k):
    """Unfreezing depth in training round r (1-indexed): d0 in rounds 1..k,
    then one more after every k rounds (the coordinator's d <- d + 1 once
    r mod k == 0, Alg. 1)."""
    return d0 + (r - 1) // k


def alg1_stage_run(desc, weights, adapters, w_h, b_h, batches, n_tm, beta, d0, k,
                   rounds, iters_per_round, lr, lr_head):
    """Alg. 1's training loop for one initiator whose samples pass through
    this stage (1-indexed Trm blocks beta .. beta + n_blocks - 1 of n_tm):
    in round r the depth is depth_of_round(r, d0, k) and each of the
    initiator's iterations runs the forward, the [CLS] loss, the head update
    (with the head the forward used), the backward ending at the adapter the
    depth selects, and the SGD update of the unfrozen adapters.  Iteration i
    (0-based, over all rounds) takes batches[i % len(batches)] = (x, labels).
    Returns (records, adapters, w_h, b_h), records[i] = (round, depth, c,
    loss)."""
    L = desc["n_blocks"]
    eps_ = beta + L - 1
    records = []
    it = 0
    for r in range(1, rounds + 1):
        depth = min(depth_of_round(r, d0, k), n_tm)
        c = local_lowest_unfrozen(n_tm, depth, beta, eps_)
        for _ in range(iters_per_round):
            x, labels = batches[it % len(batches)]
            y, caches = stage_forward(desc, weights, adapters, x)
            loss, dy, g_wh, g_bh = cls_head_ce(y, w_h, b_h, labels)
            w_h, b_h = w_h - lr_head * g_wh, b_h - lr_head * g_bh
            if c < L:
                _, grads = stage_backward(desc, weights, adapters, caches, dy, c)
                adapters = sgd_step(adapters, grads, lr)
            records.append((r, depth, c, loss))
            it += 1
    return records, adapters, w_h, b_h
