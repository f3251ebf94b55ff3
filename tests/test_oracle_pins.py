"""Pins of the fp64 oracle against facts that do not come from the oracle.

Each test checks one part of the oracle against something independent:
invariants of the definition, closed-form special cases, brute force with
plain Python loops on tiny inputs, central finite differences, and torch's
own float64 nn.TransformerEncoderLayer (a separate implementation of the
same post-LN encoder layer, §II-C, Eq. (1)).
"""
import itertools
import math

import numpy as np
import pytest

import oracle
import synth

RNG = np.random.default_rng(12345)


# --------------------------------------------------------------------------
# softmax (Eq. (1))
# --------------------------------------------------------------------------

def test_softmax_rows_sum_to_one_and_masked_zero():
    s = RNG.standard_normal((3, 4, 7, 9)) * 5
    mask = (RNG.random((3, 1, 1, 9)) > 0.4).astype(np.uint8)
    mask[..., 0] = 1
    P = oracle.masked_softmax(s, mask)
    np.testing.assert_allclose(P.sum(-1), 1.0, rtol=0, atol=1e-15)
    assert np.all(P[np.broadcast_to(mask == 0, P.shape)] == 0.0)
    assert np.all(P >= 0)


def test_softmax_shift_invariant_and_all_masked_row():
    s = RNG.standard_normal((5, 6))
    mask = np.ones((1, 6), np.uint8)
    P1 = oracle.masked_softmax(s, mask)
    P2 = oracle.masked_softmax(s + RNG.standard_normal((5, 1)) * 30, mask)
    np.testing.assert_allclose(P1, P2, rtol=0, atol=1e-14)
    P0 = oracle.masked_softmax(s, np.zeros((1, 6), np.uint8))
    assert np.all(P0 == 0.0)


def test_softmax_matches_textbook_formula_loop():
    s = RNG.standard_normal((4, 8))
    mask = np.array([[1, 1, 0, 1, 0, 1, 1, 0]], np.uint8)
    P = oracle.masked_softmax(s, mask)
    for r in range(4):
        ex = [math.exp(s[r, c]) if mask[0, c] else 0.0 for c in range(8)]
        tot = sum(ex)
        for c in range(8):
            assert abs(P[r, c] - ex[c] / tot) < 1e-15


def test_softmax_backward_equals_explicit_jacobian():
    s = RNG.standard_normal(6)
    mask = np.array([1, 0, 1, 1, 1, 0], np.uint8)
    P = oracle.masked_softmax(s[None], mask[None])[0]
    dP = RNG.standard_normal(6)
    # J_ij = dP_i/ds_j = P_i (delta_ij - P_j), built entry by entry.
    J = np.array([[P[i] * ((i == j) - P[j]) for j in range(6)] for i in range(6)])
    ref = J.T @ dP
    got = oracle.masked_softmax_backward(P[None], dP[None])[0]
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-15)
    assert np.all(got[mask == 0] == 0)


# --------------------------------------------------------------------------
# LayerNorm
# --------------------------------------------------------------------------

def test_layernorm_moments():
    z = RNG.standard_normal((10, 64)) * 3 + 2
    y, xhat, rstd = oracle.layernorm(z, np.ones(64), np.zeros(64))
    np.testing.assert_allclose(y.mean(-1), 0, atol=1e-14)
    var = z.var(-1)
    np.testing.assert_allclose(y.var(-1), var / (var + oracle.LN_EPS), rtol=1e-13)
    np.testing.assert_allclose(rstd[:, 0], 1 / np.sqrt(var + oracle.LN_EPS), rtol=1e-14)


def test_layernorm_affine_and_backward_invariants():
    n = 48
    z = RNG.standard_normal((7, n))
    gam, bet = RNG.standard_normal(n), RNG.standard_normal(n)
    y, xhat, rstd = oracle.layernorm(z, gam, bet)
    np.testing.assert_allclose(y, gam * xhat + bet, rtol=0, atol=1e-15)
    dy = RNG.standard_normal((7, n))
    dz, dg, db = oracle.layernorm_backward(dy, xhat, rstd, gam)
    np.testing.assert_allclose(dz.sum(-1), 0, atol=1e-13)
    # sum dz * xhat = 0 up to eps / sigma^2
    np.testing.assert_allclose((dz * xhat).sum(-1), 0, atol=1e-10)
    np.testing.assert_allclose(db, dy.sum(0), rtol=1e-15)


def test_layernorm_backward_finite_difference():
    n = 16
    z = RNG.standard_normal((3, n))
    gam, bet = RNG.standard_normal(n), RNG.standard_normal(n)
    dy = RNG.standard_normal((3, n))
    _, xhat, rstd = oracle.layernorm(z, gam, bet)
    dz, dg, db = oracle.layernorm_backward(dy, xhat, rstd, gam)
    eps = 1e-6

    def loss(zz, gg, bb):
        return float((oracle.layernorm(zz, gg, bb)[0] * dy).sum())

    for (i, j) in [(0, 0), (1, 5), (2, 15)]:
        zp, zm = z.copy(), z.copy()
        zp[i, j] += eps
        zm[i, j] -= eps
        fd = (loss(zp, gam, bet) - loss(zm, gam, bet)) / (2 * eps)
        assert abs(fd - dz[i, j]) < 1e-8 * max(1.0, abs(fd))
    for j in [0, 7]:
        gp, gm = gam.copy(), gam.copy()
        gp[j] += eps
        gm[j] -= eps
        fd = (loss(z, gp, bet) - loss(z, gm, bet)) / (2 * eps)
        assert abs(fd - dg[j]) < 1e-8 * max(1.0, abs(fd))


# --------------------------------------------------------------------------
# GELU
# --------------------------------------------------------------------------

def test_gelu_special_values_and_math_erf():
    assert oracle.gelu(np.array([0.0]))[0] == 0.0
    assert oracle.gelu_grad(np.array([0.0]))[0] == 0.5
    u = np.linspace(-6, 6, 101)
    ref = np.array([0.5 * v * (1 + math.erf(v / math.sqrt(2))) for v in u])
    np.testing.assert_allclose(oracle.gelu(u), ref, rtol=1e-15, atol=1e-16)
    # large |u|: GELU(u) -> u for u >> 0 and -> 0 for u << 0
    assert abs(oracle.gelu(np.array([10.0]))[0] - 10.0) < 1e-15
    assert abs(oracle.gelu(np.array([-10.0]))[0]) < 1e-20


def test_gelu_grad_finite_difference():
    u = np.linspace(-5, 5, 41)
    e = 1e-6
    fd = (oracle.gelu(u + e) - oracle.gelu(u - e)) / (2 * e)
    np.testing.assert_allclose(oracle.gelu_grad(u), fd, rtol=0, atol=1e-9)


# --------------------------------------------------------------------------
# attention (Eq. (1)), brute force and special cases
# --------------------------------------------------------------------------

def _attention_loops(Q, K, V, mask):
    B, H, S, d = Q.shape
    out = np.zeros_like(Q)
    for b, j, s in itertools.product(range(B), range(H), range(S)):
        logits = []
        for t in range(S):
            if mask[b, t]:
                logits.append((t, sum(Q[b, j, s, c] * K[b, j, t, c] for c in range(d)) / math.sqrt(d)))
        if not logits:
            continue
        mx = max(v for _, v in logits)
        w = [(t, math.exp(v - mx)) for t, v in logits]
        tot = sum(v for _, v in w)
        for c in range(d):
            out[b, j, s, c] = sum(wt * V[b, j, t, c] for t, wt in w) / tot
    return out


def test_attention_brute_force():
    B, H, S, d = 2, 2, 5, 3
    Q, K, V = (RNG.standard_normal((B, H, S, d)) for _ in range(3))
    mask = np.array([[1, 1, 1, 0, 0], [1, 1, 1, 1, 1]], np.uint8)
    C, P = oracle.attention(Q, K, V, mask)
    np.testing.assert_allclose(C, _attention_loops(Q, K, V, mask), rtol=0, atol=1e-14)


def test_attention_special_cases():
    B, H, S, d = 1, 1, 6, 4
    K, V = RNG.standard_normal((B, H, S, d)), RNG.standard_normal((B, H, S, d))
    mask = np.array([[1, 1, 1, 1, 0, 0]], np.uint8)
    # Q = 0: uniform weights over valid keys -> mean of valid V rows.
    C, _ = oracle.attention(np.zeros((B, H, S, d)), K, V, mask)
    np.testing.assert_allclose(C[0, 0], np.broadcast_to(V[0, 0, :4].mean(0), (S, d)), atol=1e-15)
    # one valid key -> that V row.
    one = np.array([[0, 0, 1, 0, 0, 0]], np.uint8)
    C, _ = oracle.attention(RNG.standard_normal((B, H, S, d)), K, V, one)
    np.testing.assert_allclose(C[0, 0], np.broadcast_to(V[0, 0, 2], (S, d)), atol=0)
    # sequence length 1 -> C = V.
    q1, k1, v1 = (RNG.standard_normal((2, 3, 1, d)) for _ in range(3))
    C, _ = oracle.attention(q1, k1, v1, np.ones((2, 1), np.uint8))
    np.testing.assert_allclose(C, v1, atol=0)
    # no valid key -> zero context.
    C, P = oracle.attention(RNG.standard_normal((B, H, S, d)), K, V, np.zeros((1, S), np.uint8))
    assert np.all(C == 0) and np.all(P == 0)


def test_merge_split_heads_layout():
    B, S, H, d = 2, 3, 4, 5
    t = np.arange(B * S * H * d, dtype=np.float64).reshape(B * S, H * d)
    sh = oracle.split_heads(t, B, S, H)
    for b, j, s, c in itertools.product(range(B), range(H), range(S), range(d)):
        assert sh[b, j, s, c] == t[b * S + s, j * d + c]
    np.testing.assert_array_equal(oracle.merge_heads(sh), t)


# --------------------------------------------------------------------------
# whole layer: torch's float64 TransformerEncoderLayer as an independent
# implementation of the same post-LN encoder layer
# --------------------------------------------------------------------------

def _torch_layer(p, h, H, f):
    import torch
    layer = torch.nn.TransformerEncoderLayer(
        d_model=h, nhead=H, dim_feedforward=f, dropout=0.0, activation="gelu",
        layer_norm_eps=oracle.LN_EPS, batch_first=True, norm_first=False,
        dtype=torch.float64)
    layer.train()
    with torch.no_grad():
        sa = layer.self_attn
        sa.in_proj_weight.copy_(torch.from_numpy(p["W_qkv"]))
        sa.in_proj_bias.copy_(torch.from_numpy(p["b_qkv"]))
        sa.out_proj.weight.copy_(torch.from_numpy(p["W_o"]))
        sa.out_proj.bias.copy_(torch.from_numpy(p["b_o"]))
        layer.linear1.weight.copy_(torch.from_numpy(p["W_1"]))
        layer.linear1.bias.copy_(torch.from_numpy(p["b_1"]))
        layer.linear2.weight.copy_(torch.from_numpy(p["W_2"]))
        layer.linear2.bias.copy_(torch.from_numpy(p["b_2"]))
        layer.norm1.weight.copy_(torch.from_numpy(p["g1"]))
        layer.norm1.bias.copy_(torch.from_numpy(p["be1"]))
        layer.norm2.weight.copy_(torch.from_numpy(p["g2"]))
        layer.norm2.bias.copy_(torch.from_numpy(p["be2"]))
    return layer


TORCH_PARAM_OF = {
    "W_qkv": lambda l: l.self_attn.in_proj_weight, "b_qkv": lambda l: l.self_attn.in_proj_bias,
    "W_o": lambda l: l.self_attn.out_proj.weight, "b_o": lambda l: l.self_attn.out_proj.bias,
    "W_1": lambda l: l.linear1.weight, "b_1": lambda l: l.linear1.bias,
    "W_2": lambda l: l.linear2.weight, "b_2": lambda l: l.linear2.bias,
    "g1": lambda l: l.norm1.weight, "be1": lambda l: l.norm1.bias,
    "g2": lambda l: l.norm2.weight, "be2": lambda l: l.norm2.bias,
}


@pytest.mark.parametrize("perturb", [False, True])
def test_layer_matches_torch_transformer_encoder_layer(perturb):
    import torch
    cfg = synth.CONFIGS["tiny"].with_(L=1, batch=3, seq=11, len_lo=4, len_hi=11)
    inp = synth.make_inputs(cfg, seed=5)
    p = synth.make_params(cfg, seed=5, perturb=perturb)[0]
    layer = _torch_layer(p, cfg.hidden, cfg.heads, cfg.ffn)
    xt = torch.from_numpy(inp["x"].copy()).requires_grad_(True)
    yt = layer(xt, src_key_padding_mask=torch.from_numpy(inp["mask"] == 0))
    yt.backward(torch.from_numpy(inp["dy"]))
    y, saved = oracle.layer_forward(inp["x"], inp["mask"], p, cfg.heads)
    dx, g = oracle.layer_backward(inp["dy"], saved, p)
    np.testing.assert_allclose(y, yt.detach().numpy(), rtol=0, atol=1e-12)
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=0, atol=1e-11)
    for name in oracle.PARAM_NAMES:
        ref = TORCH_PARAM_OF[name](layer).grad.numpy()
        np.testing.assert_allclose(g[name], ref, rtol=0, atol=1e-10 * max(1.0, np.abs(ref).max()),
                                   err_msg=name)


# --------------------------------------------------------------------------
# finite differences on the tiny stage config (central, fp64)
# --------------------------------------------------------------------------

def test_stage_backward_finite_difference_tiny():
    cfg = synth.CONFIGS["tiny"]
    inp = synth.make_inputs(cfg)
    params = synth.make_params(cfg, perturb=True)
    x, mask, dy = inp["x"], inp["mask"], inp["dy"]
    y, saved = oracle.stage_forward(x, mask, params, cfg.heads)
    dx, grads = oracle.stage_backward(dy, saved, params)
    eps = 1e-6
    rng = np.random.default_rng(0)

    def L():
        return oracle.stage_loss(x, mask, params, cfg.heads, dy)

    # parameters of both layers, ~10 sampled coordinates per tensor
    for li in range(cfg.L):
        for name in oracle.PARAM_NAMES:
            t = params[li][name]
            an = grads[li][name]
            scale = np.abs(an).max()
            idxs = [tuple(rng.integers(0, s) for s in t.shape) for _ in range(10)]
            for idx in idxs:
                old = t[idx]
                t[idx] = old + eps
                lp = L()
                t[idx] = old - eps
                lm = L()
                t[idx] = old
                fd = (lp - lm) / (2 * eps)
                if name == "b_qkv" and cfg.hidden <= idx[0] < 2 * cfg.hidden:
                    # key bias: the analytic gradient is exactly 0 (softmax
                    # is invariant to a per-row shift)
                    assert abs(fd) < 1e-6
                    continue
                assert abs(fd - an[idx]) <= 1e-6 * scale, (li, name, idx, fd, an[idx])
    scale = np.abs(dx).max()
    for _ in range(20):
        idx = tuple(rng.integers(0, s) for s in x.shape)
        old = x[idx]
        x[idx] = old + eps
        lp = L()
        x[idx] = old - eps
        lm = L()
        x[idx] = old
        fd = (lp - lm) / (2 * eps)
        assert abs(fd - dx[idx]) <= 1e-6 * scale, (idx, fd, dx[idx])


def test_key_bias_gradient_is_zero():
    cfg = synth.CONFIGS["tiny"]
    inp = synth.make_inputs(cfg)
    params = synth.make_params(cfg, perturb=True)
    _, saved = oracle.stage_forward(inp["x"], inp["mask"], params, cfg.heads)
    _, grads = oracle.stage_backward(inp["dy"], saved, params)
    h = cfg.hidden
    for g in grads:
        assert np.abs(g["b_qkv"][h:2 * h]).max() < 1e-13 * np.abs(g["b_qkv"]).max()


# --------------------------------------------------------------------------
# stage composition and padding
# --------------------------------------------------------------------------

def test_partition_invariance():
    """Running layers [0, L) as one stage equals two chained stages (§III)."""
    cfg = synth.CONFIGS["tiny"].with_(L=3)
    inp = synth.make_inputs(cfg)
    params = synth.make_params(cfg, perturb=True)
    y, s = oracle.stage_forward(inp["x"], inp["mask"], params, cfg.heads)
    dx, g = oracle.stage_backward(inp["dy"], s, params)
    y1, s1 = oracle.stage_forward(inp["x"], inp["mask"], params[:1], cfg.heads)
    y2, s2 = oracle.stage_forward(y1, inp["mask"], params[1:], cfg.heads)
    d1, g2 = oracle.stage_backward(inp["dy"], s2, params[1:])
    d0, g1 = oracle.stage_backward(d1, s1, params[:1])
    np.testing.assert_array_equal(y, y2)
    np.testing.assert_array_equal(dx, d0)
    for a, b in zip(g, g1 + g2):
        for k in a:
            np.testing.assert_array_equal(a[k], b[k])


def test_padded_keys_do_not_affect_valid_rows_of_other_positions():
    cfg = synth.CONFIGS["tiny"]
    inp = synth.make_inputs(cfg)
    params = synth.make_params(cfg, perturb=True)
    mask = inp["mask"]
    y, _ = oracle.stage_forward(inp["x"], mask, params, cfg.heads)
    x2 = inp["x"].copy()
    x2[mask == 0] = RNG.standard_normal(x2[mask == 0].shape)
    y2, _ = oracle.stage_forward(x2, mask, params, cfg.heads)
    np.testing.assert_allclose(y2[mask == 1], y[mask == 1], rtol=0, atol=1e-13)
    assert np.abs(y2[mask == 0] - y[mask == 0]).max() > 1e-3


def test_sequences_are_independent():
    """Each sequence's output and gradient contribution depends only on itself
    (basis of checking large batches on a subset of sequences)."""
    cfg = synth.CONFIGS["tiny"].with_(batch=3)
    inp = synth.make_inputs(cfg)
    params = synth.make_params(cfg, perturb=True)
    y, s = oracle.stage_forward(inp["x"], inp["mask"], params, cfg.heads)
    dy = inp["dy"].copy()
    dy[1] = 0
    dx, g = oracle.stage_backward(dy, s, params)
    sub = [0, 2]
    ys, ss = oracle.stage_forward(inp["x"][sub], inp["mask"][sub], params, cfg.heads)
    dxs, gs = oracle.stage_backward(dy[sub], ss, params)
    np.testing.assert_allclose(ys, y[sub], atol=1e-13)
    np.testing.assert_allclose(dxs, dx[sub], atol=1e-13)
    for a, b in zip(g, gs):
        for k in a:
            np.testing.assert_allclose(a[k], b[k], atol=1e-12)
