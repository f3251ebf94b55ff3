"""fp64 CPU oracle of one pipeline stage of post-LN BERT encoder layers.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import this
package: only the tests, the smoke check and the benchmark's CPU-baseline leg
call it.  It shares no code with the HIP library.

What it computes (paper §II-C "BERT" and §III):
  * a batch of sentences of shape (b, n, h) enters the stage;
  * self-attention, Eq. (1): softmax(Q K^T / sqrt(d_k)) V, with Q, K, V the
    input multiplied by three matrices, per head of width d_k;
  * three more linear layers with residual connections: the attention
    output keeps width h, the intermediate layer widens to i (here f), the
    output layer projects back to h;
  * a stage is a contiguous block of such layers on one device (§III): it
    maps the previous device's output to its own output, and in the backward
    pass computes the gradients of its layers in reverse order.

Readings where the paper is silent (each listed in the design notes):
  * a LayerNorm follows each of the two residual additions (post-LN BERT),
    eps = 1e-12, biased variance;
  * the FFN activation is the exact erf GELU;
  * no dropout;
  * padded key positions (mask 0) receive probability exactly 0; a query row
    whose keys are all masked gets P = 0 and a zero context;
  * Q, K, V weights are the row blocks [0,h), [h,2h), [2h,3h) of one
    [3h, h] matrix; head j owns columns [j*d, (j+1)*d) of each;
  * the backward pass is the exact chain rule of <Y_L, dY> (no loss), and
    gradients are those of one step (not accumulated).

Everything is float64 and follows the definition step by step; a numpy
matmul stands in for each dense product and scipy's erf for the error
function.  No blocking, fusion or reordering beyond that.

Parity pins: every function here is checked by tests/test_oracle_pins.py
against invariants, brute force, closed-form special cases, finite
differences and torch's own float64 TransformerEncoderLayer.
"""
from __future__ import annotations

import math
from typing import Dict, List, Tuple

import numpy as np
from scipy.special import erf

LN_EPS = 1e-12

PARAM_NAMES = ("W_qkv", "b_qkv", "W_o", "b_o", "g1", "be1",
               "W_1", "b_1", "W_2", "b_2", "g2", "be2")


# ----------------------------------------------------------------------------
# Building blocks
# ----------------------------------------------------------------------------

def linear(x: np.ndarray, W: np.ndarray, b: np.ndarray) -> np.ndarray:
    """y = x W^T + b, W in [out, in] layout (§II-C: linear layers)."""
    return x @ W.T + b


def masked_softmax(scores: np.ndarray, key_mask: np.ndarray) -> np.ndarray:
    """Row softmax over the last axis with masked keys excluded (Eq. (1)).

    scores: [..., S_q, S_k]; key_mask broadcastable to it, nonzero = attend.
    A row with no valid key returns all zeros."""
    valid = np.broadcast_to(key_mask != 0, scores.shape)
    s = np.where(valid, scores, -np.inf)
    m = s.max(axis=-1, keepdims=True)
    m = np.where(np.isfinite(m), m, 0.0)
    e = np.where(valid, np.exp(s - m), 0.0)
    z = e.sum(axis=-1, keepdims=True)
    return np.where(z > 0, e / np.where(z > 0, z, 1.0), 0.0)


def masked_softmax_backward(P: np.ndarray, dP: np.ndarray) -> np.ndarray:
    """Jacobian-vector product of the row softmax: P * (dP - sum(dP * P))."""
    return P * (dP - (dP * P).sum(axis=-1, keepdims=True))


def layernorm(z: np.ndarray, gamma: np.ndarray, beta: np.ndarray,
              eps: float = LN_EPS) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """LayerNorm over the last axis; returns (y, xhat, rstd)."""
    mu = z.mean(axis=-1, keepdims=True)
    var = ((z - mu) ** 2).mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + eps)
    xhat = (z - mu) * rstd
    return gamma * xhat + beta, xhat, rstd


def layernorm_backward(dy: np.ndarray, xhat: np.ndarray, rstd: np.ndarray,
                       gamma: np.ndarray):
    """Returns (dz, dgamma, dbeta) for y = gamma * xhat + beta."""
    g = dy * gamma
    n = xhat.shape[-1]
    dz = rstd * (g - g.sum(axis=-1, keepdims=True) / n
                 - xhat * (g * xhat).sum(axis=-1, keepdims=True) / n)
    dgamma = (dy * xhat).reshape(-1, n).sum(axis=0)
    dbeta = dy.reshape(-1, n).sum(axis=0)
    return dz, dgamma, dbeta


def gelu(u: np.ndarray) -> np.ndarray:
    """Exact GELU: u * Phi(u) with Phi the standard normal CDF."""
    return 0.5 * u * (1.0 + erf(u / math.sqrt(2.0)))


def gelu_grad(u: np.ndarray) -> np.ndarray:
    """d GELU / du = Phi(u) + u * phi(u)."""
    return 0.5 * (1.0 + erf(u / math.sqrt(2.0))) + u * np.exp(-0.5 * u * u) / math.sqrt(2.0 * math.pi)


def split_heads(t: np.ndarray, B: int, S: int, H: int) -> np.ndarray:
    """[B*S, H*d] -> [B, H, S, d] (head j = columns j*d .. j*d+d-1)."""
    d = t.shape[-1] // H
    return t.reshape(B, S, H, d).transpose(0, 2, 1, 3)


def merge_heads(t: np.ndarray) -> np.ndarray:
    """[B, H, S, d] -> [B*S, H*d]."""
    B, H, S, d = t.shape
    return t.transpose(0, 2, 1, 3).reshape(B * S, H * d)


def attention(Q: np.ndarray, K: np.ndarray, V: np.ndarray, key_mask: np.ndarray):
    """Eq. (1) per (batch, head): softmax(Q K^T / sqrt(d_k)) V.

    Q, K, V: [B, H, S, d]; key_mask: [B, S].  Returns (context, P)."""
    d = Q.shape[-1]
    scores = (Q @ K.transpose(0, 1, 3, 2)) / math.sqrt(d)
    P = masked_softmax(scores, key_mask[:, None, None, :])
    return P @ V, P


def attention_backward(Q, K, V, P, dC):
    """Gradients of Eq. (1) w.r.t. Q, K, V given dC = dL/d(context)."""
    d = Q.shape[-1]
    dV = P.transpose(0, 1, 3, 2) @ dC
    dP = dC @ V.transpose(0, 1, 3, 2)
    dS = masked_softmax_backward(P, dP) / math.sqrt(d)
    dQ = dS @ K
    dK = dS.transpose(0, 1, 3, 2) @ Q
    return dQ, dK, dV


# ----------------------------------------------------------------------------
# One encoder layer
# ----------------------------------------------------------------------------

def layer_forward(x: np.ndarray, key_mask: np.ndarray, p: Dict[str, np.ndarray],
                  heads: int, eps: float = LN_EPS):
    """Post-LN encoder layer (§II-C): attention, then three linear layers with
    residual connections.  x: [B, S, h].  Returns (y, saved)."""
    B, S, h = x.shape
    X = x.reshape(B * S, h)
    QKV = linear(X, p["W_qkv"], p["b_qkv"])                      # [T, 3h]
    Q = split_heads(QKV[:, :h], B, S, heads)
    K = split_heads(QKV[:, h:2 * h], B, S, heads)
    V = split_heads(QKV[:, 2 * h:], B, S, heads)
    Cb, P = attention(Q, K, V, key_mask)
    C = merge_heads(Cb)                                          # [T, h]
    Z1 = X + linear(C, p["W_o"], p["b_o"])                       # residual
    H1, xhat1, rstd1 = layernorm(Z1, p["g1"], p["be1"], eps)
    U = linear(H1, p["W_1"], p["b_1"])                           # [T, f]
    G = gelu(U)
    Z2 = H1 + linear(G, p["W_2"], p["b_2"])                      # residual
    Y, xhat2, rstd2 = layernorm(Z2, p["g2"], p["be2"], eps)
    saved = dict(X=X, Q=Q, K=K, V=V, P=P, C=C, Z1=Z1, H1=H1, xhat1=xhat1,
                 rstd1=rstd1, U=U, G=G, Z2=Z2, Y=Y, xhat2=xhat2, rstd2=rstd2,
                 shape=(B, S, h), heads=heads)
    return Y.reshape(B, S, h), saved


def layer_backward(dy: np.ndarray, saved, p: Dict[str, np.ndarray]):
    """Exact chain rule of layer_forward, in reverse order (§III).

    Returns (dx, grads) with grads keyed like the parameters."""
    B, S, h = saved["shape"]
    H = saved["heads"]
    dY = dy.reshape(B * S, h)
    g = {}
    # Y = LN(Z2)
    dZ2, g["g2"], g["be2"] = layernorm_backward(dY, saved["xhat2"], saved["rstd2"], p["g2"])
    # Z2 = H1 + G W_2^T + b_2
    g["W_2"] = dZ2.T @ saved["G"]
    g["b_2"] = dZ2.sum(axis=0)
    dG = dZ2 @ p["W_2"]
    dH1 = dZ2.copy()
    # G = gelu(U); U = H1 W_1^T + b_1
    dU = dG * gelu_grad(saved["U"])
    g["W_1"] = dU.T @ saved["H1"]
    g["b_1"] = dU.sum(axis=0)
    dH1 += dU @ p["W_1"]
    # H1 = LN(Z1)
    dZ1, g["g1"], g["be1"] = layernorm_backward(dH1, saved["xhat1"], saved["rstd1"], p["g1"])
    # Z1 = X + C W_o^T + b_o
    g["W_o"] = dZ1.T @ saved["C"]
    g["b_o"] = dZ1.sum(axis=0)
    dC = dZ1 @ p["W_o"]
    dX = dZ1.copy()
    # attention
    dQ, dK, dV = attention_backward(saved["Q"], saved["K"], saved["V"], saved["P"],
                                    split_heads(dC, B, S, H))
    dQKV = np.concatenate([merge_heads(dQ), merge_heads(dK), merge_heads(dV)], axis=1)
    g["W_qkv"] = dQKV.T @ saved["X"]
    g["b_qkv"] = dQKV.sum(axis=0)
    dX += dQKV @ p["W_qkv"]
    return dX.reshape(B, S, h), g


# ----------------------------------------------------------------------------
# A stage: contiguous block of layers (§III, §IV-D partition index)
# ----------------------------------------------------------------------------

def stage_forward(x: np.ndarray, key_mask: np.ndarray, params: List[Dict[str, np.ndarray]],
                  heads: int, eps: float = LN_EPS):
    """Apply the stage's layers in order.  Returns (y, saved_list)."""
    saved_list = []
    cur = np.asarray(x, dtype=np.float64)
    for p in params:
        cur, s = layer_forward(cur, key_mask, p, heads, eps)
        saved_list.append(s)
    return cur, saved_list


def stage_backward(dy: np.ndarray, saved_list, params):
    """Backward through the stage in reverse layer order.  Returns (dx, grads)."""
    grads = [None] * len(params)
    cur = np.asarray(dy, dtype=np.float64)
    for i in reversed(range(len(params))):
        cur, grads[i] = layer_backward(cur, saved_list[i], params[i])
    return cur, grads


def stage_loss(x, key_mask, params, heads, dy, eps: float = LN_EPS) -> float:
    """<Y_L, dY>: the scalar whose gradient stage_backward computes."""
    y, _ = stage_forward(x, key_mask, params, heads, eps)
    return float((y * dy).sum())
