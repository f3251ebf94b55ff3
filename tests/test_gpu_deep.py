"""Parity of the depth-sweep stage at its deepest point: 40 BERT-large-shaped
layers (h 1024, 16 heads, FFN 4096) on the full B8 x S512 batch with valid
lengths in [128, 512], bf16 storage.  This is the workload whose per-layer
time the layer allocator consumes (sections IV-B and IV-C).

The fp64 oracle cannot follow 40 layers of bf16 rounding to a 2e-2 bound end
to end: each layer's output rounding is inherited by the next layer, and in
the backward pass each layer's rounding by the layers below.  So every
layer is checked from its own GPU inputs (layer-wise), in both directions:

  * the 40-layer stage runs forward and backward once (the configuration the
    depth sweep times), with dy zero outside the shortest and the longest
    sequence (sequences are independent, so the other sequences contribute
    exactly zero to every gradient), recording the gradient that reaches each
    layer's output (stage_record_grads: inside a bf16 stage that is the fp32
    residual stream of the backward pass);
  * the oracle runs layer_forward and layer_backward of layer l on that
    layer's saved input X_l and its recorded incoming gradient dY_l, for the
    two sequences: H1 and Y of every layer within the LayerNorm output bound,
    and dX_l (the gradient recorded at layer l - 1, or the stage's dx) and
    all twelve gradients of every layer within relative L2 1e-2, with the
    key-bias pin ||db_k|| <= 1e-2 ||db_q||.

End-to-end drift (the oracle's own 40-layer chain from x against the GPU's y,
dx and gradients) is printed, not asserted.
"""
import numpy as np
import pytest

import synth
from _parity import IDX, make_stage, max_abs, rel_l2, run_oracle, to_numpy, to_torch
from test_gpu_parity import BF16_DBK_REL, BF16_GRAD_L2, report_ln

pytestmark = pytest.mark.gpu

DEPTH = 40


def _say(msg):
    print(msg, flush=True)


@pytest.mark.timeout(900)
def test_bf16_deep_sweep_40_layers_layerwise_forward_and_backward():
    import torch
    import oracle

    cfg = synth.CONFIGS["deep_sweep"].with_(L=DEPTH)
    B, S, h = cfg.batch, cfg.seq, cfg.hidden
    T = B * S
    _say(f"case bf16 deep sweep {cfg}")
    inp = synth.make_inputs(cfg)
    params = synth.make_params(cfg)
    _say("  parameters drawn")
    seqs = np.array(sorted({int(np.argmin(inp["lengths"])), int(np.argmax(inp["lengths"]))}))
    sel = np.zeros(B, bool)
    sel[seqs] = True
    _say(f"  checked sequences {seqs.tolist()} (lengths {inp['lengths'][seqs].tolist()})")
    dy = inp["dy"].copy()
    dy[~sel] = 0.0

    # The 40-layer stage, forward and backward once, recording the gradient
    # that reaches each layer's output.
    whole = make_stage(cfg, params)
    whole.record_grads(True)
    x = to_torch(inp["x"], "bf16")
    mask = torch.from_numpy(np.ascontiguousarray(inp["mask"])).cuda()
    y = whole.forward(x, mask)
    Xs = [to_numpy(whole.saved(l, 0, T)).reshape(B, S, h)[seqs] for l in range(DEPTH)]
    Xs.append(to_numpy(y).reshape(B, S, h)[seqs])
    H1 = [to_numpy(whole.saved(l, 3, T)).reshape(B, S, h)[seqs] for l in range(DEPTH)]
    dx = whole.backward(to_torch(dy, "bf16"))
    torch.cuda.synchronize()
    dX_gpu = to_numpy(dx).reshape(B, S, h)[seqs]
    dY = [whole.recorded_grad(l, T).double().cpu().numpy().reshape(B, S, h)[seqs]
          for l in range(DEPTH)]
    grads = [{n: to_numpy(whole.grad(l, IDX[n])) for n in synth.PARAM_NAMES} for l in range(DEPTH)]
    whole.close()
    assert np.array_equal(dY[DEPTH - 1], dy[seqs]), "the top layer's recorded gradient is not dy"
    _say("  40-layer stage done")

    # Layer-wise oracle checks.
    sub_mask = inp["mask"][seqs]
    worst_ln, worst_g = 0.0, {}
    for l in range(DEPTH):
        y_ref, sv = oracle.layer_forward(Xs[l], sub_mask, params[l], cfg.heads)
        worst_ln = max(worst_ln, report_ln(f"layer {l} H1", H1[l].reshape(-1), sv["H1"].reshape(-1)))
        worst_ln = max(worst_ln, report_ln(f"layer {l} Y", Xs[l + 1].reshape(-1), y_ref.reshape(-1)))
        dx_ref, g_ref = oracle.layer_backward(dY[l], sv, params[l])
        dx_l = dX_gpu if l == 0 else dY[l - 1]
        e = {"dX": rel_l2(dx_l, dx_ref)}
        for n in synth.PARAM_NAMES:
            g, r = grads[l][n], g_ref[n]
            if n == "b_qkv":
                e["db_k/db_q"] = float(np.linalg.norm(g[h:2 * h]) / max(np.linalg.norm(r[:h]), 1e-30))
                g = np.concatenate([g[:h], g[2 * h:]])
                r = np.concatenate([r[:h], r[2 * h:]])
            e[n] = rel_l2(g, r)
        top = max((k for k in e if k != "db_k/db_q"), key=e.get)
        _say(f"  layer {l} backward: worst rel l2 {e[top]:.3e} ({top}), dX {e['dX']:.3e}, "
             f"db_k/db_q {e['db_k/db_q']:.2e}")
        for k, v in e.items():
            worst_g[(l, k)] = v
    bad = {k: v for k, v in worst_g.items()
           if not v <= (BF16_DBK_REL if k[1] == "db_k/db_q" else BF16_GRAD_L2)}
    _say(f"  layer-wise: worst LayerNorm output {worst_ln:.3f} of its bound; worst gradient "
         f"rel l2 {max(v for k, v in worst_g.items() if k[1] != 'db_k/db_q'):.3e}")

    # End-to-end drift through all 40 layers (printed only).
    sub = {"x": inp["x"][seqs], "mask": sub_mask, "dy": dy[seqs]}
    ref = run_oracle(cfg.with_(batch=len(seqs)), sub, params)
    y_gpu = Xs[DEPTH]
    g_e2e = max((rel_l2(grads[l][n], ref["grads"][l][n]), l, n)
                for l in range(DEPTH) for n in synth.PARAM_NAMES if n != "b_qkv")
    _say(f"  end-to-end drift over {DEPTH} layers: y max abs {max_abs(y_gpu, ref['y']):.3e} "
         f"(rel l2 {rel_l2(y_gpu, ref['y']):.3e}), dx rel l2 {rel_l2(dX_gpu, ref['dx']):.3e}, "
         f"worst gradient rel l2 {g_e2e[0]:.3e} (layer {g_e2e[1]} {g_e2e[2]})")
    assert worst_ln <= 1.0 and not bad, (worst_ln, bad)
