"""Parity of the HIP encoder stage (through the C ABI) with the fp64 oracle.

Tolerances:
  * fp32 stages: per tensor ||gpu - ref||_inf / ||ref||_inf <= 1e-4 for y,
    dx, every parameter gradient and the saved activations.
  * bf16 stages (bf16 storage, fp32 accumulation): max |gpu - ref| <= 2e-2
    on the LayerNorm outputs (H1 and Y) of every layer, the oracle running
    each layer from the GPU's own bf16 input of that layer (layer-wise: the
    rounding of a layer's output is inherited by the next layer and is not a
    kernel error).  Where half a bf16 ulp of the reference value plus a
    compute allowance of 2^-10 |ref| exceeds 2e-2 (|ref| >= 4), that is the
    bound instead: a bf16 output is the fp32 result rounded to 8 significant
    bits, so an output of magnitude in [4, 8) is off by up to 0.0156 from
    the exact value by rounding alone, one in [8, 16) by up to 0.031.  Each
    tensor reports whether it also meets the literal 2e-2.  Gradients:
    ||gpu - ref||_2 / ||ref||_2 <= 1e-2 end to end for y, dx and every
    parameter gradient tensor, with the key-bias block of b_qkv excluded.
  * The key-bias gradient is analytically zero (section II-C, Eq. (1): the
    row softmax is invariant to adding a constant to every score of a row,
    and the key bias adds q . b_k to all scores of query q's row), so it is
    checked as ||db_k||_2 <= tol * ||db_q||_2 on every stage, tol = 1e-4 on
    fp32 stages and 1e-2 on bf16 stages.
"""
import numpy as np
import pytest

import synth
from _parity import max_abs, rel_inf, rel_l2, run_gpu, run_oracle

pytestmark = pytest.mark.gpu

F32_TOL = 1e-4
BF16_LN_ABS = 2e-2
BF16_GRAD_L2 = 1e-2
BF16_DBK_REL = 1e-2  # ||db_k|| / ||db_q|| on bf16 stages


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


def ln_bound(r: np.ndarray) -> np.ndarray:
    """Per-element bound on a bf16 LayerNorm output: 2e-2, or half a bf16
    ulp of the reference plus 2^-10 |ref| where that is larger."""
    return np.maximum(BF16_LN_ABS, 0.5 * bf16_ulp(r) + np.abs(r) * 2.0 ** -10)


def check_bf16_layerwise(cfg, inp, params, got, seqs=None):
    """Each layer recomputed by the oracle from the GPU's own (bf16) input of
    that layer: max |gpu - ref| on its two LayerNorm outputs H1 and Y.
    seqs: optional sequence indices to check (others skipped).  Returns the
    worst error as a multiple of 2e-2 on the ln_bound scale (<= 2e-2 passes)."""
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
            worst = max(worst, report_ln(f"layer {l} {name}", g.reshape(-1), r.reshape(-1)))
    return worst * BF16_LN_ABS


def report_ln(label, g, r) -> float:
    """Prints the LayerNorm-output check of one tensor; returns its worst
    error over ln_bound (<= 1 passes)."""
    err = np.abs(g - r)
    norm = err / ln_bound(r)
    i = int(np.argmax(norm))
    literal = "meets" if err.max() <= BF16_LN_ABS else "exceeds (passes on the half-ulp bound)"
    _say(f"  {label}: max abs {err.max():.3e} {literal} 2e-2; worst vs bound {norm[i]:.3f} "
         f"(err {err[i]:.3e} at ref {r[i]:+.3f})")
    return float(norm[i])


def bf16_ulp(r: np.ndarray) -> np.ndarray:
    """Spacing of bf16 numbers at |r| (8 significant bits)."""
    e = np.floor(np.log2(np.maximum(np.abs(r), 1e-30)))
    return np.exp2(e - 7)


def check_bf16(cfg, got, ref, rows=None):
    """End to end: relative L2 of y, dx and every parameter gradient (the
    key-bias block of b_qkv excluded), plus the key-bias pin: the ratio
    ||db_k|| / ||db_q|| under the key (layer, "db_k/db_q").
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
    kq_worst = 0.0
    for l in range(cfg.L):
        for name in synth.PARAM_NAMES:
            g, r = got["grads"][l][name], ref["grads"][l][name]
            if name == "b_qkv":
                kq = float(np.linalg.norm(g[h:2 * h]) / max(np.linalg.norm(r[:h]), 1e-30))
                kq_worst = max(kq_worst, kq)
                worst[(l, "db_k/db_q")] = kq
                g = np.concatenate([g[:h], g[2 * h:]])
                r = np.concatenate([r[:h], r[2 * h:]])
            worst[(l, name)] = rel_l2(g, r)
    _say(f"  key-bias pin: max ||db_k|| / ||db_q|| = {kq_worst:.3e} (bound {BF16_DBK_REL:g})")
    for k in sorted(worst, key=worst.get, reverse=True)[:4]:
        _say(f"  rel l2 {worst[k]:.3e} at {k}")
    return worst


def assert_bf16(layerwise_worst, e2e):
    bad = {k: e for k, e in e2e.items()
           if not e <= (BF16_DBK_REL if k[-1] == "db_k/db_q" else BF16_GRAD_L2)}
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


def test_bf16_mid_width_sequence_subset():
    """Two layers of width 512 (8 heads, FFN 2048) on B32 x S512 with valid
    lengths in [384, 512].  On a 256-CU device the GEMMs with N = h = 512
    (out-projection, FFN2, the FFN1 / QKV / out-projection data gradients)
    take 256 x 128 tiles, the three-slot ring with its k-tile requests split
    between the two halves of the work-group, which none of the other
    configurations selects.  dy is zero outside three sequences (the first,
    the shortest and the last); the oracle runs only those."""
    cfg = synth.StageConfig("mid_width", 2, 512, 8, 2048, 32, 512, 384, 512, "bf16", 7)
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


def test_bf16_smaller_batches_after_the_full_batch():
    """One BERT-large-shaped layer run on B32 x S512 and then, on the same
    stage, on smaller batches.  The weight-gradient stream-K schedule of a
    smaller token count can need more split-K partials than the full batch
    (T = 384 needs 201 MB against 101 MB at T = 16384): every call must still
    match the oracle.  The full batch is checked on sequences {0, 31} (dy
    zero elsewhere), the smaller ones whole."""
    from _parity import make_stage
    base = synth.CONFIGS["bert_large_4"].with_(L=1)
    params = synth.make_params(base, perturb=True)
    st = make_stage(base, params)
    try:
        for batch, seq in ((32, 512), (1, 384), (1, 192), (3, 96)):
            cfg = base.with_(batch=batch, seq=seq, len_lo=seq // 2, len_hi=seq)
            _say(f"case bf16 B{batch} x S{seq} after the full batch")
            inp = synth.make_inputs(cfg, seed=batch * 1000 + seq)
            if batch == 32:
                sel = np.zeros(batch, bool)
                sel[[0, batch - 1]] = True
                dy = inp["dy"].copy()
                dy[~sel] = 0.0
                got = run_gpu(cfg, inp, params, dy=dy, stage=st, saved=(0, 3))
                lw = check_bf16_layerwise(cfg, inp, params, got, seqs=np.flatnonzero(sel))
                sub = {"x": inp["x"][sel], "mask": inp["mask"][sel], "dy": dy[sel]}
                ref = run_oracle(cfg.with_(batch=2), sub, params)
                assert_bf16(lw, check_bf16(cfg, got, ref, rows=sel))
            else:
                got = run_gpu(cfg, inp, params, stage=st, saved=(0, 3))
                lw = check_bf16_layerwise(cfg, inp, params, got)
                assert_bf16(lw, check_bf16(cfg, got, run_oracle(cfg, inp, params)))
    finally:
        st.close()
