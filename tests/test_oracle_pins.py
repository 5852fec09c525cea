"""Pins of the CPU oracle against facts fixed outside it: closed forms and
special cases, library routines, central finite differences in float64, an
independent torch-autograd implementation of the blocks, structural
invariants, and the worked ring example of Sec. III-A."""
import json
import math
import os

import numpy as np
import pytest

import oracle as O
from paper_2502_19864_amd.workloads import WORKLOADS, make_inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _tiny_bert(seed=7, B=2, S=5, d=16, H=2, F=24, m=4, L=2, placement="houlsby"):
    desc = O.make_desc("bert", L, d, H, F, m, placement=placement)
    return desc, _rand_params(desc, seed, B, S)


def _tiny_llama(seed=8, B=2, S=6, d=16, H=2, F=20, m=4, L=2, placement="houlsby"):
    desc = O.make_desc("llama", L, d, H, F, m, placement=placement)
    return desc, _rand_params(desc, seed, B, S)


def _tiny(arch, placement="houlsby", **kw):
    return (_tiny_bert if arch == "bert" else _tiny_llama)(placement=placement, **kw)


def _adapters_of(placement):
    """indices of the adapters a block carries: (attention, FFN) or FFN only"""
    return (0, 1) if placement == "houlsby" else (1,)


def _rand_params(desc, seed, B, S):
    rng = np.random.default_rng(seed)
    d, F, m = desc["d_model"], desc["d_ffn"], desc["d_adapter"]
    n = lambda *s, std=0.3: rng.standard_normal(s) * std  # noqa: E731
    weights, adapters = [], []
    for _ in range(desc["n_blocks"]):
        if desc["arch"] == "bert":
            w = dict(w_qkv=n(d, 3 * d), b_qkv=n(3 * d, std=0.1), w_o=n(d, d),
                     b_o=n(d, std=0.1), ln1_g=1 + n(d, std=0.1),
                     ln1_b=n(d, std=0.1), w_i=n(d, F), b_i=n(F, std=0.1),
                     w_f=n(F, d), b_f=n(d, std=0.1), ln2_g=1 + n(d, std=0.1),
                     ln2_b=n(d, std=0.1))
        else:
            w = dict(rms1_g=1 + n(d, std=0.1), w_qkv=n(d, 3 * d), w_o=n(d, d),
                     rms2_g=1 + n(d, std=0.1), w_gu=n(d, 2 * F), w_d=n(F, d))
        weights.append(w)
        adapters.append(tuple({"w_down": n(d, m), "w_up": n(m, d)}
                              for _ in range(2)))
    x = rng.standard_normal((B, S, d))
    dy = rng.standard_normal((B, S, d))
    return dict(weights=weights, adapters=adapters, x=x, dy=dy)


# ---------------------------------------------------------------- elementwise
def test_gelu_is_x_phi_of_x():
    xs = np.array([-6.0, -2.5, -1.0, -1e-3, 0.0, 0.5, 1.0, 3.0, 7.0])
    ref = np.array([0.5 * x * (1 + math.erf(x / math.sqrt(2))) for x in xs])
    np.testing.assert_allclose(O.gelu(xs), ref, rtol=1e-15, atol=1e-300)
    assert O.gelu(np.array(0.0)) == 0.0
    # Phi(1) = 0.8413447460685429 (standard normal table)
    assert abs(O.gelu(np.array(1.0)) - 0.8413447460685429) < 1e-15


@pytest.mark.parametrize("f,df", [(O.gelu, O.gelu_grad), (O.silu, O.silu_grad)])
def test_elementwise_derivatives_by_central_differences(f, df):
    u = np.linspace(-5, 5, 101)
    h = 1e-6
    fd = (f(u + h) - f(u - h)) / (2 * h)
    np.testing.assert_allclose(df(u), fd, rtol=0, atol=1e-8)


# ---------------------------------------------------------------- norms
def test_layer_norm_standardises_rows():
    x = np.random.default_rng(0).standard_normal((7, 33)) * 5 + 3
    y, xhat, rstd = O.layer_norm(x, np.ones(33), np.zeros(33), 0.0)
    np.testing.assert_allclose(y.mean(-1), 0, atol=1e-13)
    np.testing.assert_allclose(y.var(-1), 1, atol=1e-12)
    np.testing.assert_allclose(rstd[:, 0], 1 / x.std(-1), rtol=1e-13)


def test_rms_norm_unit_rms():
    x = np.random.default_rng(1).standard_normal((5, 40)) * 3
    y, _, _ = O.rms_norm(x, np.ones(40), 0.0)
    np.testing.assert_allclose(np.sqrt((y * y).mean(-1)), 1, rtol=1e-13)


@pytest.mark.parametrize("kind", ["ln", "rms"])
def test_norm_backward_by_central_differences(kind):
    rng = np.random.default_rng(2)
    x = rng.standard_normal((3, 12))
    g = 1 + 0.3 * rng.standard_normal(12)
    b = 0.3 * rng.standard_normal(12)
    dy = rng.standard_normal((3, 12))
    if kind == "ln":
        f = lambda z: O.layer_norm(z, g, b, 1e-5)  # noqa: E731
        bwd = lambda c: O.layer_norm_bwd(dy, g, c[1], c[2])  # noqa: E731
    else:
        f = lambda z: O.rms_norm(z, g, 1e-5)  # noqa: E731
        bwd = lambda c: O.rms_norm_bwd(dy, g, c[1], c[2])  # noqa: E731
    an = bwd(f(x))
    fd = np.zeros_like(x)
    h = 1e-6
    for idx in np.ndindex(x.shape):
        xp, xm = x.copy(), x.copy()
        xp[idx] += h
        xm[idx] -= h
        fd[idx] = ((f(xp)[0] - f(xm)[0]) * dy).sum() / (2 * h)
    np.testing.assert_allclose(an, fd, rtol=0, atol=1e-8)


# ---------------------------------------------------------------- attention
def test_softmax_rows_sum_to_one_and_causal_zeros():
    rng = np.random.default_rng(3)
    q, k, v = (rng.standard_normal((2, 3, 9, 4)) for _ in range(3))
    for causal in (False, True):
        _, p = O.attention_fwd(q, k, v, causal)
        np.testing.assert_allclose(p.sum(-1), 1, rtol=1e-14)
        if causal:
            assert np.all(p[..., np.triu_indices(9, 1)[0], np.triu_indices(9, 1)[1]] == 0)


def test_attention_special_cases():
    rng = np.random.default_rng(4)
    v = rng.standard_normal((1, 2, 6, 4))
    k = rng.standard_normal((1, 2, 6, 4))
    # a single key: the output is that key's value
    o, _ = O.attention_fwd(rng.standard_normal((1, 2, 1, 4)), k[:, :, :1], v[:, :, :1], False)
    np.testing.assert_allclose(o, v[:, :, :1], rtol=1e-15)
    # zero queries: uniform weights -> mean of the values (prefix mean if causal)
    o, _ = O.attention_fwd(np.zeros((1, 2, 6, 4)), k, v, False)
    np.testing.assert_allclose(o, np.broadcast_to(v.mean(2, keepdims=True), o.shape), rtol=1e-13)
    o, _ = O.attention_fwd(np.zeros((1, 2, 6, 4)), k, v, True)
    pref = np.cumsum(v, axis=2) / np.arange(1, 7)[None, None, :, None]
    np.testing.assert_allclose(o, pref, rtol=1e-13)


def test_attention_matches_textbook_loops():
    """Brute force on a tiny input: explicit sums over keys, math.exp."""
    rng = np.random.default_rng(5)
    q, k, v = (rng.standard_normal((1, 1, 4, 3)) for _ in range(3))
    o, _ = O.attention_fwd(q, k, v, True)
    for i in range(4):
        w = [math.exp(sum(q[0, 0, i, t] * k[0, 0, j, t] for t in range(3)) / math.sqrt(3))
             for j in range(i + 1)]
        for t in range(3):
            ref = sum(w[j] * v[0, 0, j, t] for j in range(i + 1)) / sum(w)
            assert abs(o[0, 0, i, t] - ref) < 1e-14


def test_rope_convention_and_relative_position():
    dh, S = 8, 6
    cos, sin = O.rope_tables(S, dh, 10000.0, np.float64)
    # unit vector e_i at position p rotates into (cos, sin) of p * theta^(-2i/dh)
    for i in range(dh // 2):
        e = np.zeros((1, 1, S, dh))
        e[..., i] = 1
        r = O.rope_fwd(e, cos, sin)
        ang = np.arange(S) * 10000.0 ** (-2 * i / dh)
        np.testing.assert_allclose(r[0, 0, :, i], np.cos(ang), atol=1e-15)
        np.testing.assert_allclose(r[0, 0, :, i + dh // 2], np.sin(ang), atol=1e-15)
    rng = np.random.default_rng(6)
    q = np.broadcast_to(rng.standard_normal(dh), (1, 1, S, dh)).copy()
    k = np.broadcast_to(rng.standard_normal(dh), (1, 1, S, dh)).copy()
    rq, rk = O.rope_fwd(q, cos, sin), O.rope_fwd(k, cos, sin)
    np.testing.assert_allclose(np.linalg.norm(rq, axis=-1), np.linalg.norm(q, axis=-1), rtol=1e-14)
    dots = rq[0, 0] @ rk[0, 0].T
    for off in range(-2, 3):
        diag = [dots[m, m - off] for m in range(S) if 0 <= m - off < S]
        np.testing.assert_allclose(diag, diag[0], rtol=1e-12)
    # the backward is the inverse rotation
    np.testing.assert_allclose(O.rope_bwd(rq, cos, sin), q, atol=1e-14)


# ---------------------------------------------------------------- adapter, Eq. (1)
def test_adapter_with_zero_up_projection_is_identity():
    rng = np.random.default_rng(9)
    h = rng.standard_normal((10, 12))
    wd = rng.standard_normal((12, 3))
    out, u = O.adapter_fwd(h, wd, np.zeros((3, 12)))
    assert np.array_equal(out, h)
    dh, gdn, gup = O.adapter_bwd(rng.standard_normal((10, 12)), h, u, wd, np.zeros((3, 12)))
    assert np.all(gdn == 0)          # no signal reaches W_down through a zero W_up
    assert np.any(gup != 0)


def test_stage_with_zero_up_projections_equals_plain_blocks():
    """With every W_up = 0 the stage is a plain encoder; check it against a
    torch nn.TransformerEncoderLayer-free plain forward via torch functional."""
    desc, p = _tiny_bert()
    ad0 = [tuple({"w_down": a["w_down"], "w_up": np.zeros_like(a["w_up"])} for a in pair)
           for pair in p["adapters"]]
    y, _ = O.stage_forward(desc, p["weights"], ad0, p["x"])
    y_ref = _torch_stage(desc, p["weights"], None, p["x"])[0]
    np.testing.assert_allclose(y, y_ref, rtol=0, atol=1e-12)


# ---------------------------------------------------------------- gradients
def _loss_and_grads(desc, weights, adapters, x, dy, c):
    y, caches = O.stage_forward(desc, weights, adapters, x)
    dx, grads = O.stage_backward(desc, weights, adapters, caches, dy, c)
    return (y * dy).sum(), dx, grads


@pytest.mark.parametrize("placement", ["houlsby", "ffn"])
@pytest.mark.parametrize("arch", ["bert", "llama"])
def test_stage_gradients_by_central_differences(arch, placement):
    desc, p = _tiny(arch, placement)
    W, A, x, dy = p["weights"], p["adapters"], p["x"], p["dy"]
    _, dx, grads = _loss_and_grads(desc, W, A, x, dy, -1)
    rng = np.random.default_rng(11)
    h = 1e-6

    def L(ad, xx):
        y, _ = O.stage_forward(desc, W, ad, xx)
        return (y * dy).sum()

    for l in range(desc["n_blocks"]):
        if placement == "ffn":
            assert grads[l][0] is None
        for a in _adapters_of(placement):
            for name in ("w_down", "w_up"):
                g = grads[l][a][name]
                scale = np.abs(g).max()
                for _ in range(6):
                    idx = tuple(rng.integers(0, s) for s in g.shape)
                    adp = [tuple(dict(t) for t in pair) for pair in A]
                    adm = [tuple(dict(t) for t in pair) for pair in A]
                    adp[l][a][name] = A[l][a][name].copy()
                    adm[l][a][name] = A[l][a][name].copy()
                    adp[l][a][name][idx] += h
                    adm[l][a][name][idx] -= h
                    fd = (L(adp, x) - L(adm, x)) / (2 * h)
                    assert abs(fd - g[idx]) <= 1e-6 * scale, (l, a, name, idx, fd, g[idx])
    scale = np.abs(dx).max()
    for _ in range(10):
        idx = tuple(rng.integers(0, s) for s in x.shape)
        xp, xm = x.copy(), x.copy()
        xp[idx] += h
        xm[idx] -= h
        fd = (L(A, xp) - L(A, xm)) / (2 * h)
        assert abs(fd - dx[idx]) <= 1e-6 * scale


@pytest.mark.parametrize("placement", ["houlsby", "ffn"])
@pytest.mark.parametrize("arch", ["bert", "llama"])
def test_truncated_backward_equals_full_backward(arch, placement):
    """Early stopping at block c leaves every produced gradient bitwise equal
    to the full backward's and produces nothing below c."""
    desc, p = _tiny(arch, placement, L=4)
    W, A, x, dy = p["weights"], p["adapters"], p["x"], p["dy"]
    _, dx_full, g_full = _loss_and_grads(desc, W, A, x, dy, -1)
    assert dx_full is not None
    for c in range(0, 5):
        _, dx, g = _loss_and_grads(desc, W, A, x, dy, c)
        assert dx is None
        for l in range(4):
            if l < c:
                assert g[l] is None
            else:
                for a in _adapters_of(placement):
                    for k in ("w_down", "w_up"):
                        assert np.array_equal(g[l][a][k], g_full[l][a][k])


@pytest.mark.parametrize("arch", ["bert", "llama"])
def test_single_placement_is_houlsby_without_the_attention_adapter(arch):
    """The single placement equals the two-adapter stage whose attention
    adapters have W_up = 0 (Eq. (1) is then the identity): the same output,
    the same input gradient and the same FFN-adapter gradients, bitwise; and
    the attention adapter's W_down gets no gradient there."""
    d1, p = _tiny(arch, "ffn", L=3)
    d2 = dict(d1, placement="houlsby")
    W, x, dy = p["weights"], p["x"], p["dy"]
    A0 = [({"w_down": pair[0]["w_down"], "w_up": np.zeros_like(pair[0]["w_up"])}, pair[1])
          for pair in p["adapters"]]
    l1, dx1, g1 = _loss_and_grads(d1, W, p["adapters"], x, dy, -1)
    l2, dx2, g2 = _loss_and_grads(d2, W, A0, x, dy, -1)
    assert l1 == l2
    assert np.array_equal(O.stage_forward(d1, W, p["adapters"], x)[0], O.stage_forward(d2, W, A0, x)[0])
    assert np.array_equal(dx1, dx2)
    for l in range(3):
        assert g1[l][0] is None
        assert np.all(g2[l][0]["w_down"] == 0)
        for k in ("w_down", "w_up"):
            assert np.array_equal(g1[l][1][k], g2[l][1][k])
    # the single placement stops one sublayer earlier: at c the FFN adapter's
    # gradients are the last thing produced, and they match the full pass
    for c in range(3):
        _, _, g = _loss_and_grads(d1, W, p["adapters"], x, dy, c)
        for k in ("w_down", "w_up"):
            assert np.array_equal(g[c][1][k], g1[c][1][k])


def test_causality_and_batch_independence():
    desc, p = _tiny_llama(S=7)
    W, A, x = p["weights"], p["adapters"], p["x"]
    y, _ = O.stage_forward(desc, W, A, x)
    x2 = x.copy()
    x2[:, 4:] += 1.0
    y2, _ = O.stage_forward(desc, W, A, x2)
    assert np.array_equal(y[:, :4], y2[:, :4])
    assert not np.allclose(y[:, 4:], y2[:, 4:])
    desc_b, pb = _tiny_bert(B=3)
    yb, _ = O.stage_forward(desc_b, pb["weights"], pb["adapters"], pb["x"])
    y1, _ = O.stage_forward(desc_b, pb["weights"], pb["adapters"], pb["x"][1:2])
    np.testing.assert_allclose(yb[1:2], y1, rtol=0, atol=1e-13)


# ---------------------------------------------------------------- independent implementation
def _torch_stage(desc, weights, adapters, x):
    """The same stage written with torch.nn.functional library layers in
    float64, gradients by torch autograd."""
    import torch
    import torch.nn.functional as F
    t = lambda a: torch.tensor(a, dtype=torch.float64)  # noqa: E731
    B, S, d = x.shape
    H = desc["n_heads"]
    dh = d // H
    eps = desc["norm_eps"]
    xt = t(x).requires_grad_(True)
    ads = None
    if adapters is not None:
        ads = [tuple({k: t(v).requires_grad_(True) for k, v in a.items()} for a in pair)
               for pair in adapters]

    def adapter(hh, a):
        if a is None:
            return hh
        return hh + F.gelu(hh @ a["w_down"], approximate="none") @ a["w_up"]

    def heads(z):
        return z.reshape(B, S, H, dh).transpose(1, 2)

    def rope(z):
        half = dh // 2
        inv = desc["rope_theta"] ** (-(2.0 * torch.arange(half, dtype=torch.float64)) / dh)
        ang = torch.arange(S, dtype=torch.float64)[:, None] * inv[None, :]
        c, s = torch.cos(ang), torch.sin(ang)
        z1, z2 = z[..., :half], z[..., half:]
        return torch.cat([z1 * c - z2 * s, z2 * c + z1 * s], dim=-1)

    h = xt
    for l, w in enumerate(weights):
        w = {k: t(v) for k, v in w.items()}
        a_attn = ads[l][0] if ads else None
        a_ffn = ads[l][1] if ads else None
        if desc["arch"] == "bert":
            qkv = h @ w["w_qkv"] + w["b_qkv"]
            q, k, v = qkv.split(d, dim=-1)
            o = F.scaled_dot_product_attention(heads(q), heads(k), heads(v))
            attn = o.transpose(1, 2).reshape(B, S, d) @ w["w_o"] + w["b_o"]
            h1 = F.layer_norm(h + adapter(attn, a_attn), (d,), w["ln1_g"], w["ln1_b"], eps)
            f2 = F.gelu(h1 @ w["w_i"] + w["b_i"], approximate="none") @ w["w_f"] + w["b_f"]
            h = F.layer_norm(h1 + adapter(f2, a_ffn), (d,), w["ln2_g"], w["ln2_b"], eps)
        else:
            n1 = F.rms_norm(h, (d,), w["rms1_g"], eps)
            q, k, v = (n1 @ w["w_qkv"]).split(d, dim=-1)
            o = F.scaled_dot_product_attention(rope(heads(q)), rope(heads(k)), heads(v),
                                               is_causal=True)
            hh = h + adapter(o.transpose(1, 2).reshape(B, S, d) @ w["w_o"], a_attn)
            n2 = F.rms_norm(hh, (d,), w["rms2_g"], eps)
            gate, up = (n2 @ w["w_gu"]).split(desc["d_ffn"], dim=-1)
            h = hh + adapter((F.silu(gate) * up) @ w["w_d"], a_ffn)
    return h.detach().numpy(), h, xt, ads


@pytest.mark.parametrize("arch", ["bert", "llama"])
def test_oracle_matches_torch_autograd(arch):
    desc, p = (_tiny_bert(L=3) if arch == "bert" else _tiny_llama(L=3))
    W, A, x, dy = p["weights"], p["adapters"], p["x"], p["dy"]
    import torch
    y_t, h, xt, ads = _torch_stage(desc, W, A, x)
    (h * torch.tensor(dy)).sum().backward()
    y, caches = O.stage_forward(desc, W, A, x)
    np.testing.assert_allclose(y, y_t, rtol=0, atol=1e-12)
    dx, grads = O.stage_backward(desc, W, A, caches, dy, -1)
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=0, atol=1e-11)
    for l in range(3):
        for a in range(2):
            for k in ("w_down", "w_up"):
                np.testing.assert_allclose(grads[l][a][k], ads[l][a][k].grad.numpy(),
                                           rtol=0, atol=1e-11)


# ---------------------------------------------------------------- losses and update
def test_loss_gradients_by_central_differences():
    rng = np.random.default_rng(12)
    y = rng.standard_normal((3, 4, 5))
    tgt = rng.standard_normal((3, 4, 5))
    _, dy = O.mse_loss(y, tgt)
    wh, bh = rng.standard_normal((5, 2)), rng.standard_normal(2)
    labels = np.array([0, 1, 1])
    _, dyc, dwh, dbh = O.cls_head_ce(y, wh, bh, labels)
    # brute-force cross-entropy of one sample written out with math.log/exp
    lg = [sum(y[0, 0, i] * wh[i, c] for i in range(5)) + bh[c] for c in range(2)]
    ce0 = -(lg[0] - math.log(math.exp(lg[0]) + math.exp(lg[1])))
    lg1 = [sum(y[1, 0, i] * wh[i, c] for i in range(5)) + bh[c] for c in range(2)]
    ce1 = -(lg1[1] - math.log(math.exp(lg1[0]) + math.exp(lg1[1])))
    lg2 = [sum(y[2, 0, i] * wh[i, c] for i in range(5)) + bh[c] for c in range(2)]
    ce2 = -(lg2[1] - math.log(math.exp(lg2[0]) + math.exp(lg2[1])))
    assert abs(O.cls_head_ce(y, wh, bh, labels)[0] - (ce0 + ce1 + ce2) / 3) < 1e-14
    h = 1e-6
    for idx in [(0, 0, 0), (1, 2, 3), (2, 0, 4), (1, 0, 1)]:
        yp, ym = y.copy(), y.copy()
        yp[idx] += h
        ym[idx] -= h
        fd = (O.mse_loss(yp, tgt)[0] - O.mse_loss(ym, tgt)[0]) / (2 * h)
        assert abs(fd - dy[idx]) < 1e-9
        fd = (O.cls_head_ce(yp, wh, bh, labels)[0] - O.cls_head_ce(ym, wh, bh, labels)[0]) / (2 * h)
        assert abs(fd - dyc[idx]) < 1e-9
    for idx in [(0, 0), (4, 1)]:
        wp, wm = wh.copy(), wh.copy()
        wp[idx] += h
        wm[idx] -= h
        fd = (O.cls_head_ce(y, wp, bh, labels)[0] - O.cls_head_ce(y, wm, bh, labels)[0]) / (2 * h)
        assert abs(fd - dwh[idx]) < 1e-9
    assert abs(dbh.sum()) < 1e-15  # softmax minus one-hot sums to zero per sample


def test_sgd_step():
    a = [({"w_down": np.ones((2, 1)), "w_up": np.ones((1, 2))},) * 2, None]
    g = [({"w_down": np.full((2, 1), 2.0), "w_up": np.full((1, 2), -1.0)},) * 2, None]
    a[1] = a[0]
    out = O.sgd_step(a, g, 0.25)
    assert np.all(out[0][0]["w_down"] == 0.5) and np.all(out[0][0]["w_up"] == 1.25)
    assert out[1] is a[1]


# ---------------------------------------------------------------- ring bookkeeping
def test_worked_ring_example_of_the_paper():
    ex = json.load(open(os.path.join(GOLDEN, "ring_example.json")))
    blocks = ex["clients_1_indexed_blocks"]
    # the 4:5:2:3 ratio over 14 blocks is exactly these contiguous ranges
    assert [e - b + 1 for b, e in blocks] == ex["assignment_ratio"]
    assert blocks[-1][1] == ex["n_trm_blocks"]
    dep = ex["unfreezing_depth"]
    assert O.cutoff_block(ex["n_trm_blocks"], dep) == ex["cutoff_block_1_indexed"]
    assert O.client_roles(blocks, dep) == ex["roles"]
    assert [O.local_lowest_unfrozen(ex["n_trm_blocks"], dep, b, e) for b, e in blocks] \
        == ex["local_lowest_unfrozen"]
    # the backward path visits the initiator then only clients that are not forward-only
    assert ["u1"] + [f"u{i + 1}" for i, r in enumerate(ex["roles"]) if r != "forward-only"] \
        == ex["backward_path"]


def test_workload_cutoffs_follow_alg1():
    # bert_base: top 4 of 12 blocks unfrozen -> cut-off block 9 (1-indexed) -> local 8
    w = WORKLOADS["bert_base"]
    assert O.local_lowest_unfrozen(12, 4, 1, 12) == w.lowest_unfrozen == 8
    # llama share: top 2 of the stage's 8 blocks
    w = WORKLOADS["llama7b_share"]
    assert O.local_lowest_unfrozen(8, 2, 1, 8) == w.lowest_unfrozen == 6
    # a client with every adapter unfrozen and the cut-off upstream gets -1
    assert O.local_lowest_unfrozen(24, 20, 7, 12) == -1


def test_tiny_workload_runs_and_is_finite():
    w = WORKLOADS["tiny"]
    inp = make_inputs(w)
    desc = O.make_desc(w.arch, w.n_blocks, w.d_model, w.n_heads, w.d_ffn, w.d_adapter)
    f64 = lambda a: a.astype(np.float64)  # noqa: E731
    W = [{k: f64(v) for k, v in b.items()} for b in inp["weights"]]
    A = [tuple({k: f64(v) for k, v in a.items()} for a in pair) for pair in inp["adapters"]]
    y, caches = O.stage_forward(desc, W, A, f64(inp["x"]))
    _, dy = O.mse_loss(y, f64(inp["target"]))
    dx, grads = O.stage_backward(desc, W, A, caches, dy, w.lowest_unfrozen)
    assert dx is None and np.isfinite(y).all()
    assert all(np.isfinite(g[a][k]).all() for g in grads for a in range(2) for k in ("w_down", "w_up"))
