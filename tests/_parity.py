"""Helpers shared by the GPU parity tests: run the HIP stage through the C ABI
on the seeded synthetic inputs, run the fp64 oracle on the same inputs, and
compare with the error measures the tolerances are stated in."""
from __future__ import annotations

import numpy as np

import oracle
import synth

IDX = {n: i for i, n in enumerate(synth.PARAM_NAMES)}


def to_torch(a: np.ndarray, dtype: str, device="cuda"):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    if dtype == "bf16":
        t = t.to(torch.bfloat16)
    return t.to(device)


def to_numpy(t) -> np.ndarray:
    import torch
    return t.detach().to(torch.float32).cpu().numpy().astype(np.float64)


def make_stage(cfg: synth.StageConfig, params, seed: int = 0):
    from paper_2202_11836_amd import Stage
    st = Stage(cfg.L, cfg.hidden, cfg.heads, cfg.ffn, seed=seed, dtype=cfg.dtype)
    for l, p in enumerate(params):
        for name in synth.PARAM_NAMES:
            st.set_param(l, IDX[name], to_torch(p[name], "f32", "cpu"))
    return st


def run_gpu(cfg, inp, params, dy=None, stage=None, saved=()):
    """Forward + backward on the GPU.  Returns dict with y, dx, grads (list of
    dicts), and any requested saved activations per layer."""
    import torch
    st = stage if stage is not None else make_stage(cfg, params)
    x = to_torch(inp["x"], cfg.dtype)
    mask = torch.from_numpy(np.ascontiguousarray(inp["mask"], dtype=np.uint8)).cuda()
    y = st.forward(x, mask)
    out = {"stage": st}
    T = cfg.batch * cfg.seq
    for which in saved:
        out.setdefault("saved", {})[which] = [to_numpy(st.saved(l, which, T)) for l in range(cfg.L)]
    dyt = to_torch(inp["dy"] if dy is None else dy, cfg.dtype)
    dx = st.backward(dyt)
    torch.cuda.synchronize()
    out["y"] = to_numpy(y)
    out["dx"] = to_numpy(dx)
    out["grads"] = [{n: to_numpy(st.grad(l, IDX[n])) for n in synth.PARAM_NAMES} for l in range(cfg.L)]
    return out


def run_oracle(cfg, inp, params, dy=None):
    y, saved = oracle.stage_forward(inp["x"], inp["mask"], params, cfg.heads)
    dx, grads = oracle.stage_backward(inp["dy"] if dy is None else dy, saved, params)
    return {"y": y, "dx": dx, "grads": grads, "saved": saved}


def rel_inf(got, ref) -> float:
    """||got - ref||_inf / ||ref||_inf."""
    den = np.abs(ref).max()
    return float(np.abs(got - ref).max() / (den if den > 0 else 1.0))


def rel_l2(got, ref) -> float:
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(got - ref) / (den if den > 0 else 1.0))


def max_abs(got, ref) -> float:
    return float(np.abs(got - ref).max()) if got.size else 0.0
