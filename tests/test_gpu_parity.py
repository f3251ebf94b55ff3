"""Parity of the HIP encoder stage (through the C ABI) with the fp64 oracle.

Tolerances:
  * fp32 stages: per tensor ||gpu - ref||_inf / ||ref||_inf <= 1e-4 for y,
    dx, every parameter gradient and the saved activations.
  * bf16 stages (bf16 storage, fp32 accumulation): max |gpu - ref| <= 2e-2
    on the LayerNorm outputs (H1 and Y) of every layer, or one bf16 ulp of
    the reference value where that is larger (bf16 cannot represent values
    of magnitude >= 4 closer than 0.0156, >= 8 closer than 0.031), the oracle
    running each layer from the GPU's own bf16 input of that layer
    (layer-wise: the rounding of a layer's output is inherited by the next
    layer and is not a kernel error); and ||gpu - ref||_2 / ||ref||_2 <= 1e-2
    end to end for y, dx and every parameter gradient tensor.
    On fp32 stages the key bias gradient, analytically zero (softmax is
    invariant to a per-row shift), is checked against the query bias
    gradient's norm.
"""
import numpy as np
import pytest

import synth
from _parity import max_abs, rel_inf, rel_l2, run_gpu, run_oracle

pytestmark = pytest.mark.gpu

F32_TOL = 1e-4
BF16_LN_ABS = 2e-2
BF16_GRAD_L2 = 1e-2


def _say(msg):
    print(msg, flush=True)


def check_f32(cfg, got, ref, saved_gpu=None):
    assert rel_inf(got["y"], ref["y"]) <= F32_TOL, rel_inf(got["y"], ref["y"])
    assert rel_inf(got["dx"], ref["dx"]) <= F32_TOL, rel_inf(got["dx"], ref["dx"])
    h = cfg.hidden
    for l in range(cfg.L):
        for name in synth.PARAM_NAMES:
            g, r = got["grads"][l][name], ref["grads"][l][name]
            if name == "b_qkv":
                # key-bias block is analytically zero
                kq = np.linalg.norm(g[h:2 * h])
                assert kq <= 1e-4 * np.linalg.norm(r[:h]) + 1e-30, (l, name, kq)
                g = np.concatenate([g[:h], g[2 * h:]])
                r = np.concatenate([r[:h], r[2 * h:]])
            e = rel_inf(g, r)
            assert e <= F32_TOL, (l, name, e)
    if saved_gpu:
        from oracle import merge_heads
        from oracle import gelu_grad
        for which, key in ((1, "QKV"), (2, "C"), (3, "H1"), (4, "GD"), (5, "G")):
            for l in range(cfg.L):
                sv = ref["saved"][l]
                if key == "QKV":
                    r = np.concatenate([merge_heads(sv["Q"]), merge_heads(sv["K"]),
                                        merge_heads(sv["V"])], axis=1)
                elif key == "GD":
                    r = gelu_grad(sv["U"])
                else:
                    r = sv[key]
                e = rel_inf(saved_gpu[which][l], r)
                assert e <= F32_TOL, (l, key, e)


def check_bf16_layerwise(cfg, inp, params, got, seqs=None):
    """Each layer recomputed by the oracle from the GPU's own (bf16) input of
    that layer: max |gpu - ref| on its two LayerNorm outputs H1 and Y.
    seqs: optional sequence indices to check (others skipped)."""
    import oracle
    B, S, h = cfg.batch, cfg.seq, cfg.hidden
    sel = np.arange(B) if seqs is None else np.asarray(seqs)
    X = [got["saved"][0][l].reshape(B, S, h)[sel] for l in range(cfg.L)]
    H1 = [got["saved"][3][l].reshape(B, S, h)[sel] for l in range(cfg.L)]
    mask = inp["mask"][sel]
    worst = 0.0
    for l in range(cfg.L):
        y_ref, sv = oracle.layer_forward(X[l], mask, params[l], cfg.heads)
        y_gpu = X[l + 1] if l + 1 < cfg.L else got["y"][sel]
        for name, g, r in (("H1", H1[l].reshape(-1, h), sv["H1"]), ("Y", y_gpu, y_ref)):
            g, r = g.reshape(-1), r.reshape(-1)
            err = np.abs(g - r)
            # normalised: error over max(2e-2, one bf16 ulp of the reference)
            norm = err / np.maximum(BF16_LN_ABS, bf16_ulp(r))
            i = int(np.argmax(norm))
            _say(f"  layer {l} {name}: max abs {err.max():.3e}; worst vs bound {norm[i]:.3f} "
                 f"(err {err[i]:.3e} at ref {r[i]:+.3f})")
            worst = max(worst, float(norm[i]))
    return worst * BF16_LN_ABS


def bf16_ulp(r: np.ndarray) -> np.ndarray:
    """Spacing of bf16 numbers at |r| (8 significant bits)."""
    e = np.floor(np.log2(np.maximum(np.abs(r), 1e-30)))
    return np.exp2(e - 7)


def check_bf16(cfg, got, ref, grad_tol=BF16_GRAD_L2, rows=None):
    """End to end: relative L2 of y, dx and every parameter gradient.
    rows: optional boolean [B] selecting the sequences y/dx are compared on."""
    h = cfg.hidden
    y_g, y_r = got["y"], ref["y"]
    dx_g, dx_r = got["dx"], ref["dx"]
    if rows is not None:
        y_g, dx_g = y_g[rows], dx_g[rows]
    _say(f"  y end-to-end: max abs {max_abs(y_g, y_r):.3e}, rel l2 {rel_l2(y_g, y_r):.3e}")
    e_y = rel_l2(y_g, y_r)
    e = rel_l2(dx_g, dx_r)
    _say(f"  dx rel l2 {e:.3e}")
    worst = {("dx",): e, ("y",): e_y}
    for l in range(cfg.L):
        for name in synth.PARAM_NAMES:
            worst[(l, name)] = rel_l2(got["grads"][l][name], ref["grads"][l][name])
    for k in sorted(worst, key=worst.get, reverse=True)[:4]:
        _say(f"  rel l2 {worst[k]:.3e} at {k}")
    return worst


def assert_bf16(layerwise_worst, e2e):
    bad = {k: e for k, e in e2e.items() if not e <= BF16_GRAD_L2}
    assert layerwise_worst <= BF16_LN_ABS and not bad, (layerwise_worst, bad)


def test_tiny_fp32_default_init():
    cfg = synth.CONFIGS["tiny"]
    _say(f"case tiny fp32 {cfg}")
    inp = synth.make_inputs(cfg)
    params = synth.make_params(cfg)
    got = run_gpu(cfg, inp, params, saved=(1, 2, 3, 4, 5))
    ref = run_oracle(cfg, inp, params)
    check_f32(cfg, got, ref, got["saved"])


def test_tiny_fp32_perturbed_params():
    cfg = synth.CONFIGS["tiny"]
    _say("case tiny fp32 perturbed")
    inp = synth.make_inputs(cfg, seed=11)
    params = synth.make_params(cfg, seed=11, perturb=True)
    got = run_gpu(cfg, inp, params, saved=(1, 2, 3, 4, 5))
    ref = run_oracle(cfg, inp, params)
    check_f32(cfg, got, ref, got["saved"])


def test_fp32_ragged_tiles_and_degenerate_lengths():
    # T = 111 tokens: not a multiple of any tile; one sequence of length 1,
    # one with every key masked (length 0), one full.
    cfg = synth.CONFIGS["tiny"].with_(batch=3, seq=37, ffn=256, L=2)
    _say(f"case fp32 ragged {cfg}")
    inp = synth.make_inputs(cfg, seed=3)
    inp["lengths"] = np.array([1, 0, 37])
    inp["mask"] = synth.key_mask(inp["lengths"], cfg.seq)
    params = synth.make_params(cfg, seed=3, perturb=True)
    got = run_gpu(cfg, inp, params, saved=(1, 2, 3, 4, 5))
    ref = run_oracle(cfg, inp, params)
    check_f32(cfg, got, ref, got["saved"])


def test_bf16_small_ragged_perturbed():
    cfg = synth.StageConfig("small", 2, 256, 4, 512, 3, 40, 5, 40, "bf16", 21)
    _say(f"case bf16 small ragged {cfg}")
    inp = synth.make_inputs(cfg)
    params = synth.make_params(cfg, perturb=True)
    got = run_gpu(cfg, inp, params, saved=(0, 3))
    ref = run_oracle(cfg, inp, params)
    lw = check_bf16_layerwise(cfg, inp, params, got)
    assert_bf16(lw, check_bf16(cfg, got, ref))


def test_bf16_odd_seq_arbitrary_mask_empty_sequence():
    # S = 200: several 128-row query blocks and 64-row key tiles with tails;
    # a non-prefix key mask; one sequence with no valid key at all.
    cfg = synth.StageConfig("odd", 2, 128, 2, 256, 3, 200, 1, 200, "bf16", 33)
    _say(f"case bf16 odd seq {cfg}")
    inp = synth.make_inputs(cfg)
    rng = np.random.default_rng(1)
    mask = (rng.random((cfg.batch, cfg.seq)) < 0.6).astype(np.uint8)
    mask[1] = 0
    mask[2, -1] = 1
    inp["mask"] = mask
    params = synth.make_params(cfg, perturb=True)
    got = run_gpu(cfg, inp, params, saved=(0, 3))
    ref = run_oracle(cfg, inp, params)
    lw = check_bf16_layerwise(cfg, inp, params, got)
    assert_bf16(lw, check_bf16(cfg, got, ref))


def test_bf16_bert_base_3_full():
    cfg = synth.CONFIGS["bert_base_3"]
    _say(f"case bf16 {cfg}")
    inp = synth.make_inputs(cfg)
    params = synth.make_params(cfg)
    got = run_gpu(cfg, inp, params, saved=(0, 3))
    ref = run_oracle(cfg, inp, params)
    lw = check_bf16_layerwise(cfg, inp, params, got)
    assert_bf16(lw, check_bf16(cfg, got, ref))


def test_bf16_bert_large_4_sequence_subset():
    """Full headline batch on the GPU; dy zero outside sequences {0, B-1};
    the oracle runs only those two sequences.  Sequences are independent, so
    y on them and every parameter gradient must agree."""
    cfg = synth.CONFIGS["bert_large_4"]
    _say(f"case bf16 subset {cfg}")
    inp = synth.make_inputs(cfg)
    params = synth.make_params(cfg)
    sel = np.zeros(cfg.batch, bool)
    sel[[0, cfg.batch - 1]] = True
    dy = inp["dy"].copy()
    dy[~sel] = 0.0
    got = run_gpu(cfg, inp, params, dy=dy, saved=(0, 3))
    lw = check_bf16_layerwise(cfg, inp, params, got, seqs=np.flatnonzero(sel))
    sub = {"x": inp["x"][sel], "mask": inp["mask"][sel], "dy": dy[sel]}
    ref = run_oracle(cfg.with_(batch=2), sub, params)
    assert_bf16(lw, check_bf16(cfg, got, ref, rows=sel))


def test_bf16_bert_base_8_uneven_sequence_subset():
    """The uneven BERT-base share (8 layers, B32 x S512, valid lengths in
    [256, 512]) on the full batch: partially masked 64-key blocks next to
    unmasked ones, several 128-row blocks per head with the XCD grouping of
    the attention grid.  dy is zero outside three sequences (the first, the
    shortest and the last) and the oracle runs only those."""
    cfg = synth.CONFIGS["bert_base_8_uneven"]
    _say(f"case bf16 subset {cfg}")
    inp = synth.make_inputs(cfg)
    params = synth.make_params(cfg)
    sel = np.zeros(cfg.batch, bool)
    sel[[0, int(np.argmin(inp["lengths"])), cfg.batch - 1]] = True
    dy = inp["dy"].copy()
    dy[~sel] = 0.0
    got = run_gpu(cfg, inp, params, dy=dy, saved=(0, 3))
    lw = check_bf16_layerwise(cfg, inp, params, got, seqs=np.flatnonzero(sel))
    sub = {"x": inp["x"][sel], "mask": inp["mask"][sel], "dy": dy[sel]}
    ref = run_oracle(cfg.with_(batch=int(sel.sum())), sub, params)
    assert_bf16(lw, check_bf16(cfg, got, ref, rows=sel))
