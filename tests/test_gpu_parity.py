"""Parity of the HIP encoder stage (through the C ABI) with the fp64 oracle.

Tolerances:
  * fp32 stages: per tensor ||gpu - ref||_inf / ||ref||_inf <= 1e-4 for y,
    dx, every parameter gradient and the saved activations.
  * bf16 stages (bf16 storage, fp32 accumulation): max |gpu - ref| <= 2e-2
    on the LayerNorm outputs (H1 and Y of every layer), and
    ||gpu - ref||_2 / ||ref||_2 <= 1e-2 for dx and every parameter gradient.
    The key bias gradient is analytically zero (softmax is invariant to a
    per-row shift), so it is checked against the query bias gradient's norm.
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
        for which, key in ((1, "QKV"), (2, "C"), (3, "H1"), (4, "U"), (5, "G")):
            for l in range(cfg.L):
                r = ref["saved"][l][key]
                if key == "QKV":
                    from oracle import merge_heads
                    r = np.concatenate([merge_heads(ref["saved"][l]["Q"]),
                                        merge_heads(ref["saved"][l]["K"]),
                                        merge_heads(ref["saved"][l]["V"])], axis=1)
                e = rel_inf(saved_gpu[which][l], r)
                assert e <= F32_TOL, (l, key, e)


def check_bf16(cfg, got, ref, ln_tol=BF16_LN_ABS, grad_tol=BF16_GRAD_L2, rows=None):
    """rows: optional boolean [B] selecting the sequences y/dx are compared on."""
    h = cfg.hidden
    y_g, y_r = got["y"], ref["y"]
    dx_g, dx_r = got["dx"], ref["dx"]
    if rows is not None:
        y_g, dx_g = y_g[rows], dx_g[rows]
    e = max_abs(y_g, y_r)
    _say(f"  y max abs {e:.3e}")
    assert e <= ln_tol, e
    e = rel_l2(dx_g, dx_r)
    _say(f"  dx rel l2 {e:.3e}")
    assert e <= grad_tol, e
    worst = {}
    for l in range(cfg.L):
        for name in synth.PARAM_NAMES:
            g, r = got["grads"][l][name], ref["grads"][l][name]
            if name == "b_qkv":
                kq = np.linalg.norm(g[h:2 * h])
                assert kq <= 1e-2 * np.linalg.norm(r[:h]) + 1e-30, (l, "db_k", kq)
                g = np.concatenate([g[:h], g[2 * h:]])
                r = np.concatenate([r[:h], r[2 * h:]])
            e = rel_l2(g, r)
            worst[(l, name)] = e
    wk = max(worst, key=worst.get)
    _say(f"  worst grad rel l2 {worst[wk]:.3e} at {wk}")
    for k, e in worst.items():
        assert e <= grad_tol, (k, e)


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
    got = run_gpu(cfg, inp, params, saved=(3,))
    ref = run_oracle(cfg, inp, params)
    for l in range(cfg.L):
        e = max_abs(got["saved"][3][l], ref["saved"][l]["H1"])
        _say(f"  layer {l} H1 max abs {e:.3e}")
        assert e <= BF16_LN_ABS
    check_bf16(cfg, got, ref)


def test_bf16_bert_base_3_full():
    cfg = synth.CONFIGS["bert_base_3"]
    _say(f"case bf16 {cfg}")
    inp = synth.make_inputs(cfg)
    params = synth.make_params(cfg)
    got = run_gpu(cfg, inp, params, saved=(0, 3))
    ref = run_oracle(cfg, inp, params)
    for l in range(cfg.L):
        e = max_abs(got["saved"][3][l], ref["saved"][l]["H1"])
        _say(f"  layer {l} H1 max abs {e:.3e}")
        assert e <= BF16_LN_ABS
        if l > 0:
            e = max_abs(got["saved"][0][l], ref["saved"][l]["X"].reshape(cfg.batch, cfg.seq, -1).reshape(-1, cfg.hidden))
            _say(f"  layer {l} input max abs {e:.3e}")
            assert e <= BF16_LN_ABS
    check_bf16(cfg, got, ref)


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
    got = run_gpu(cfg, inp, params, dy=dy)
    sub = {"x": inp["x"][sel], "mask": inp["mask"][sel], "dy": dy[sel]}
    ref = run_oracle(cfg.with_(batch=2), sub, params)
    check_bf16(cfg, got, ref, rows=sel)
