"""Stages cut at half-layer boundaries (stage_init_units): unit 2j is the
attention half of encoder layer j (X -> H1), unit 2j+1 its feed-forward half
(H1 -> Y).  A partition of a block's units into chained stages must compute
what the whole block computes (the premise of placing discrete layers on
devices, section IV; section VI-G counts several such units per encoder
layer): bitwise on fp32 stages; on bf16 stages the H1 that crosses a cut
reaches the second LayerNorm rounded to bf16 (inside a stage it is added in
fp32), so there the chain is held to the oracle at the bf16 tolerances and
everything upstream of the first cut is still bitwise."""
import numpy as np
import pytest

import synth
from _parity import IDX, make_stage, max_abs, rel_l2, run_oracle, to_numpy, to_torch

pytestmark = pytest.mark.gpu

ATTN_PARAMS = {"W_qkv", "b_qkv", "W_o", "b_o", "g1", "be1"}
BF16_LN_ABS = 2e-2
BF16_GRAD_L2 = 1e-2


def _say(msg):
    print(msg, flush=True)


def unit_layers(u0, n):
    """[(global layer, has attention half, has feed-forward half)] of the
    stage holding units [u0, u0 + n)."""
    out = []
    for j in range(u0 // 2, (u0 + n - 1) // 2 + 1):
        out.append((j, u0 <= 2 * j < u0 + n, u0 <= 2 * j + 1 < u0 + n))
    return out


def make_unit_stage(cfg, params, u0, n):
    from paper_2202_11836_amd import Stage
    st = Stage(None, cfg.hidden, cfg.heads, cfg.ffn, seed=0, dtype=cfg.dtype, first_unit=u0,
               n_units=n)
    assert st.L == len(unit_layers(u0, n))
    for l, (j, a, f) in enumerate(unit_layers(u0, n)):
        for name in synth.PARAM_NAMES:
            if (a if name in ATTN_PARAMS else f):
                st.set_param(l, IDX[name], to_torch(params[j][name], "f32", "cpu"))
    return st


def run_chain(stages, x, mask, dy):
    import torch
    acts = [x]
    for st in stages:
        acts.append(st.forward(acts[-1], mask))
    d = dy
    for st in reversed(stages):
        d = st.backward(d)
    torch.cuda.synchronize()
    return acts, d


def chain_grads(stages, cuts, L):
    """Gradients per global layer and parameter name, from the stage that
    holds that half."""
    g = [dict() for _ in range(L)]
    for st, (u0, n) in zip(stages, cuts):
        for l, (j, a, f) in enumerate(unit_layers(u0, n)):
            for name in synth.PARAM_NAMES:
                if (a if name in ATTN_PARAMS else f):
                    g[j][name] = st.grad(l, IDX[name])
    return g


CUTS = [(0, 1), (1, 4), (5, 1)]  # attn 0 | ffn 0, layer 1, attn 2 | ffn 2


def _setup(dtype):
    import torch
    cfg = synth.StageConfig("units", 3, 128, 2, 256, 2, 48, 17, 48, dtype, 21)
    inp = synth.make_inputs(cfg)
    params = synth.make_params(cfg, perturb=True)
    x = to_torch(inp["x"], dtype)
    mask = torch.from_numpy(np.ascontiguousarray(inp["mask"], dtype=np.uint8)).cuda()
    dy = to_torch(inp["dy"], dtype)
    return cfg, inp, params, x, mask, dy


def test_unit_partition_fp32_bitwise():
    import torch
    _say("case units fp32 partition [0,1) [1,5) [5,6)")
    cfg, inp, params, x, mask, dy = _setup("f32")
    whole = make_stage(cfg, params)
    y = whole.forward(x, mask)
    h1_0 = whole.saved(0, 3, cfg.tokens).clone()
    h1_2 = whole.saved(2, 3, cfg.tokens).clone()
    dx = whole.backward(dy)
    stages = [make_unit_stage(cfg, params, u0, n) for u0, n in CUTS]
    acts, d = run_chain(stages, x, mask, dy)
    assert torch.equal(acts[1].reshape(-1, cfg.hidden), h1_0)
    assert torch.equal(acts[2].reshape(-1, cfg.hidden), h1_2)
    assert torch.equal(acts[3], y)
    assert torch.equal(d, dx)
    g = chain_grads(stages, CUTS, cfg.L)
    for j in range(cfg.L):
        for name in synth.PARAM_NAMES:
            assert torch.equal(g[j][name], whole.grad(j, IDX[name])), (j, name)
    for st in stages + [whole]:
        st.close()


def bf16_ulp(r):
    """Spacing of bf16 numbers at |r| (8 significant bits)."""
    return np.exp2(np.floor(np.log2(np.maximum(np.abs(r), 1e-30))) - 7)


def ln_err(got, ref):
    """max |got - ref| over max(2e-2, one bf16 ulp of ref), the bf16
    LayerNorm-output bound of the parity tests."""
    got, ref = got.reshape(-1), ref.reshape(-1)
    return float((np.abs(got - ref) / np.maximum(BF16_LN_ABS, bf16_ulp(ref))).max())


def ffn_half(H1, p):
    """Feed-forward half of a layer (section II-C) from its input H1, with
    the oracle's primitives: LN(H1 + GELU(H1 W_1^T + b_1) W_2^T + b_2)."""
    import oracle
    Z2 = H1 + oracle.linear(oracle.gelu(oracle.linear(H1, p["W_1"], p["b_1"])), p["W_2"], p["b_2"])
    return oracle.layernorm(Z2, p["g2"], p["be2"])[0]


def test_unit_partition_bf16():
    import torch

    import oracle
    _say("case units bf16 partition [0,1) [1,5) [5,6)")
    cfg, inp, params, x, mask, dy = _setup("bf16")
    B, S, h, T = cfg.batch, cfg.seq, cfg.hidden, cfg.tokens
    whole = make_stage(cfg, params)
    whole.forward(x, mask)
    h1_0 = whole.saved(0, 3, T).clone()
    y_w = to_numpy(whole.forward(x, mask))
    stages = [make_unit_stage(cfg, params, u0, n) for u0, n in CUTS]
    acts = [x]
    for st in stages:
        acts.append(st.forward(acts[-1], mask))
    # upstream of the first cut nothing differs from the whole block
    assert torch.equal(acts[1].reshape(-1, h), h1_0)
    # each half-layer recomputed by the oracle from the GPU's own bf16 input
    # of that half (a unit's output rounding is inherited, not a kernel error)
    mid = stages[1]
    X1 = to_numpy(mid.saved(1, 0, T)).reshape(B, S, h)   # layer 1 input = Y of layer 0
    H1_1 = to_numpy(mid.saved(1, 3, T))
    X2 = to_numpy(mid.saved(2, 0, T)).reshape(B, S, h)   # layer 2 input
    H1_0 = to_numpy(acts[1]).reshape(-1, h)
    H1_2 = to_numpy(acts[2]).reshape(-1, h)
    m = inp["mask"]
    _, sv0 = oracle.layer_forward(inp["x"], m, params[0], cfg.heads)
    y1, sv1 = oracle.layer_forward(X1, m, params[1], cfg.heads)
    _, sv2 = oracle.layer_forward(X2, m, params[2], cfg.heads)
    checks = {
        "H1 of layer 0 (unit 0)": ln_err(H1_0, sv0["H1"]),
        "Y of layer 0 (unit 1)": ln_err(X1, ffn_half(H1_0, params[0])),
        "H1 of layer 1 (unit 2)": ln_err(H1_1, sv1["H1"]),
        "Y of layer 1 (unit 3)": ln_err(X2, y1),
        "H1 of layer 2 (unit 4)": ln_err(H1_2, sv2["H1"]),
        "Y of layer 2 (unit 5)": ln_err(to_numpy(acts[3]), ffn_half(H1_2, params[2])),
    }
    for k, e in checks.items():
        _say(f"  {k}: worst vs bound {e:.3f}")
        assert e <= 1.0, (k, e)
    d = dy
    for st in reversed(stages):
        d = st.backward(d)
    torch.cuda.synchronize()
    # end to end: relative L2 of y, dx and every parameter gradient
    g = chain_grads(stages, CUTS, cfg.L)
    ref = run_oracle(cfg, inp, params)
    y_g = to_numpy(acts[3])
    e2e = {"y": rel_l2(y_g, ref["y"]), "dx": rel_l2(to_numpy(d), ref["dx"])}
    for j in range(cfg.L):
        for name in synth.PARAM_NAMES:
            e2e[(j, name)] = rel_l2(to_numpy(g[j][name]), ref["grads"][j][name])
    for k in sorted(e2e, key=e2e.get, reverse=True)[:4]:
        _say(f"  rel l2 {e2e[k]:.3e} at {k}")
    bad = {k: e for k, e in e2e.items() if not e <= BF16_GRAD_L2}
    assert not bad, bad
    # chain and whole block are two bf16 evaluations of the same function
    # (each held to the oracle above); they differ by the rounding of H1 at
    # the cuts, carried through the later layers
    e_cw = rel_l2(y_g, y_w)
    _say(f"  chain vs whole block: y max abs {max_abs(y_g, y_w):.3e}, rel l2 {e_cw:.3e}")
    assert e_cw <= BF16_GRAD_L2
    for st in stages + [whole]:
        st.close()


def test_unit_weights_by_global_layer_and_absent_halves():
    import torch
    from paper_2202_11836_amd import Stage, StageError, stage_tensor_bytes
    from paper_2202_11836_amd.binding import KIND_GRAD, KIND_PARAM
    _say("case units weights / absent halves")
    full = Stage(3, 128, 2, 256, seed=7, dtype="bf16")
    part = Stage(None, 128, 2, 256, seed=7, dtype="bf16", first_unit=3, n_units=2)
    assert part.L == 2  # feed-forward half of layer 1, attention half of layer 2
    for l, (j, a, f) in enumerate(unit_layers(3, 2)):
        for name in synth.PARAM_NAMES:
            w = IDX[name]
            if (a if name in ATTN_PARAMS else f):
                assert torch.equal(part.param(l, w), full.param(j, w)), (l, name)
            else:
                for call in (lambda: part.param(l, w), lambda: part.grad(l, w)):
                    with pytest.raises(StageError) as e:
                        call()
                    assert e.value.status == 1
                assert stage_tensor_bytes(part.handle, KIND_PARAM, l, w) == 0
                assert stage_tensor_bytes(part.handle, KIND_GRAD, l, w) == 0
    x = torch.randn(2, 16, 128, device="cuda").to(torch.bfloat16)
    y = part.forward(x)
    T = 32
    # saved: H1, GD, G of layer 1 (its input H1 is the stage input), X, QKV,
    # CTX of layer 2; the others do not exist
    assert torch.equal(part.saved(0, 3, T), x.reshape(T, 128))
    for l, absent in ((0, (0, 1, 2)), (1, (3, 4, 5))):
        for which in absent:
            with pytest.raises(StageError):
                part.saved(l, which, T)
    part.backward(torch.randn_like(y))
    # an empty batch clears exactly the gradients the stage holds
    e = torch.zeros(0, 16, 128, dtype=torch.bfloat16, device="cuda")
    part.forward(e)
    part.backward(e)
    torch.cuda.synchronize()
    for l, (j, a, f) in enumerate(unit_layers(3, 2)):
        for name in synth.PARAM_NAMES:
            if (a if name in ATTN_PARAMS else f):
                assert float(part.grad(l, IDX[name]).abs().max()) == 0.0
    for st in (full, part):
        st.close()


def test_single_unit_stages_chain():
    """Every unit its own stage (the finest partition), fp32: bitwise equal
    to the whole block."""
    import torch
    _say("case units fp32 one stage per unit")
    cfg, inp, params, x, mask, dy = _setup("f32")
    cfg = cfg.with_(L=2)
    params = params[:2]
    whole = make_stage(cfg, params)
    y = whole.forward(x, mask)
    dx = whole.backward(dy)
    cuts = [(u, 1) for u in range(4)]
    stages = [make_unit_stage(cfg, params, u0, n) for u0, n in cuts]
    acts, d = run_chain(stages, x, mask, dy)
    assert torch.equal(acts[-1], y) and torch.equal(d, dx)
    g = chain_grads(stages, cuts, cfg.L)
    for j in range(cfg.L):
        for name in synth.PARAM_NAMES:
            assert torch.equal(g[j][name], whole.grad(j, IDX[name])), (j, name)
    for st in stages + [whole]:
        st.close()
