"""Layer definitions of the partition, forward and hand-derived backward, in fp64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper defines a partition as the composition F_k = f_j o ... o f_i of
consecutive layers and obtains B_k by differentiating F_k (Section 2.1).  The
layers here are the Transformer layers the paper trains (Sections 3 and 5):
it fixes their widths but not their internal layout; the layout used here is
pre-LayerNorm with a ReLU feed-forward block.  Row-vector convention
throughout: activations are [n, S, D] and a linear layer is y = x W + b with
W stored [in, out].

Backward rules used (chain rule written out):
  linear      dX = dY W^T,  dW = sum_t X_t^T dY_t,  db = sum_t dY_t
  ReLU        dz = da * [z > 0]
  LayerNorm   xh = (x - mu) r, r = (var + eps)^-1/2 (biased variance);
              g = dy * gamma;  dx = r (g - mean(g) - xh mean(g xh));
              dgamma = sum_t dy xh;  dbeta = sum_t dy
  attention   A = softmax(Q K^T s + mask), O = A V, s = d_h^-1/2;
              dV = A^T dO;  dA = dO V^T;  dS = A (dA - rowsum(dA A));
              dQ = s dS K;  dK = s dS^T Q
  residual    gradients add.
"""
from __future__ import annotations

import numpy as np


# ----------------------------------------------------------------- LayerNorm
def layer_norm(x, gamma, beta, eps):
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    r = 1.0 / np.sqrt(var + eps)
    xh = (x - mu) * r
    return gamma * xh + beta, (xh, r)


def layer_norm_backward(dy, cache, gamma):
    xh, r = cache
    g = dy * gamma
    dx = r * (g - g.mean(axis=-1, keepdims=True) - xh * (g * xh).mean(axis=-1, keepdims=True))
    dgamma = (dy * xh).reshape(-1, dy.shape[-1]).sum(axis=0)
    dbeta = dy.reshape(-1, dy.shape[-1]).sum(axis=0)
    return dx, dgamma, dbeta


# -------------------------------------------------------------------- linear
def linear(x, w, b):
    return x @ w + b


def linear_backward(dy, x, w):
    D_in, D_out = w.shape
    dx = dy @ w.T
    dw = x.reshape(-1, D_in).T @ dy.reshape(-1, D_out)
    db = dy.reshape(-1, D_out).sum(axis=0)
    return dx, dw, db


# ----------------------------------------------------------------- attention
def _split_heads(t, heads):
    n, S, D = t.shape
    return t.reshape(n, S, heads, D // heads).transpose(0, 2, 1, 3)


def _merge_heads(t):
    n, H, S, dh = t.shape
    return t.transpose(0, 2, 1, 3).reshape(n, S, H * dh)


def attention(q, k, v, heads, causal):
    """Multi-head scaled dot-product attention.  q [n,Sq,D]; k, v [n,Sk,D].

    Head h uses columns [h*d_h, (h+1)*d_h) of q, k and v.  With ``causal``
    query i attends to keys j <= i only.
    """
    Q, K, V = (_split_heads(t, heads) for t in (q, k, v))
    dh = Q.shape[-1]
    s = 1.0 / np.sqrt(dh)
    scores = (Q @ K.transpose(0, 1, 3, 2)) * s
    if causal:
        Sq, Sk = scores.shape[-2:]
        future = np.arange(Sk)[None, :] > np.arange(Sq)[:, None]
        scores = np.where(future, -np.inf, scores)
    scores = scores - scores.max(axis=-1, keepdims=True)
    e = np.exp(scores)
    A = e / e.sum(axis=-1, keepdims=True)
    O = A @ V
    return _merge_heads(O), (Q, K, V, A, s)


def attention_backward(do, cache):
    Q, K, V, A, s = cache
    heads = Q.shape[1]
    dO = _split_heads(do, heads)
    dV = A.transpose(0, 1, 3, 2) @ dO
    dA = dO @ V.transpose(0, 1, 3, 2)
    dS = A * (dA - (dA * A).sum(axis=-1, keepdims=True))
    dQ = s * (dS @ K)
    dK = s * (dS.transpose(0, 1, 3, 2) @ Q)
    return _merge_heads(dQ), _merge_heads(dK), _merge_heads(dV)


# ------------------------------------------------------------- encoder layer
def encoder_layer(x, p, heads, eps):
    """Pre-LN encoder layer:  x1 = x + Attn(LN1 x) Wo + bo;  y = x1 + FFN(LN2 x1)."""
    u, ln1 = layer_norm(x, p["ln1_g"], p["ln1_b"], eps)
    q = linear(u, p["wq"], p["bq"])
    k = linear(u, p["wk"], p["bk"])
    v = linear(u, p["wv"], p["bv"])
    c, att = attention(q, k, v, heads, causal=False)
    x1 = x + linear(c, p["wo"], p["bo"])
    vv, ln2 = layer_norm(x1, p["ln2_g"], p["ln2_b"], eps)
    z = linear(vv, p["w1"], p["b1"])
    a = np.maximum(z, 0.0)
    y = x1 + linear(a, p["w2"], p["b2"])
    cache = dict(u=u, ln1=ln1, c=c, att=att, vv=vv, ln2=ln2, z=z, a=a)
    return y, cache


def encoder_layer_backward(dy, cache, p):
    g = {}
    da, g["w2"], g["b2"] = linear_backward(dy, cache["a"], p["w2"])
    dz = da * (cache["z"] > 0.0)
    dvv, g["w1"], g["b1"] = linear_backward(dz, cache["vv"], p["w1"])
    dx1_ln, g["ln2_g"], g["ln2_b"] = layer_norm_backward(dvv, cache["ln2"], p["ln2_g"])
    dx1 = dy + dx1_ln
    dc, g["wo"], g["bo"] = linear_backward(dx1, cache["c"], p["wo"])
    dq, dk, dv = attention_backward(dc, cache["att"])
    u = cache["u"]
    du_q, g["wq"], g["bq"] = linear_backward(dq, u, p["wq"])
    du_k, g["wk"], g["bk"] = linear_backward(dk, u, p["wk"])
    du_v, g["wv"], g["bv"] = linear_backward(dv, u, p["wv"])
    dx_ln, g["ln1_g"], g["ln1_b"] = layer_norm_backward(du_q + du_k + du_v, cache["ln1"], p["ln1_g"])
    dx = dx1 + dx_ln
    return dx, g


# ------------------------------------------------------------- decoder layer
def decoder_layer(x, mem, p, heads, eps):
    """Pre-LN decoder layer:
        x1 = x  + CausalSelfAttn(LN1 x) Wo + bo
        x2 = x1 + CrossAttn(q = LN2(x1) XWq + XbQ, k/v = mem XWk/XWv + XbK/XbV) XWo + XbO
        y  = x2 + FFN(LN3 x2)
    The memory enters the cross-attention un-normalised.
    """
    u, ln1 = layer_norm(x, p["ln1_g"], p["ln1_b"], eps)
    q = linear(u, p["wq"], p["bq"])
    k = linear(u, p["wk"], p["bk"])
    v = linear(u, p["wv"], p["bv"])
    c, att = attention(q, k, v, heads, causal=True)
    x1 = x + linear(c, p["wo"], p["bo"])
    u2, ln2 = layer_norm(x1, p["ln2_g"], p["ln2_b"], eps)
    xq = linear(u2, p["xwq"], p["xbq"])
    xk = linear(mem, p["xwk"], p["xbk"])
    xv = linear(mem, p["xwv"], p["xbv"])
    xc, xatt = attention(xq, xk, xv, heads, causal=False)
    x2 = x1 + linear(xc, p["xwo"], p["xbo"])
    vv, ln3 = layer_norm(x2, p["ln3_g"], p["ln3_b"], eps)
    z = linear(vv, p["w1"], p["b1"])
    a = np.maximum(z, 0.0)
    y = x2 + linear(a, p["w2"], p["b2"])
    cache = dict(u=u, ln1=ln1, c=c, att=att, u2=u2, ln2=ln2, xc=xc, xatt=xatt,
                 mem=mem, vv=vv, ln3=ln3, z=z, a=a)
    return y, cache


def decoder_layer_backward(dy, cache, p):
    g = {}
    da, g["w2"], g["b2"] = linear_backward(dy, cache["a"], p["w2"])
    dz = da * (cache["z"] > 0.0)
    dvv, g["w1"], g["b1"] = linear_backward(dz, cache["vv"], p["w1"])
    dx2_ln, g["ln3_g"], g["ln3_b"] = layer_norm_backward(dvv, cache["ln3"], p["ln3_g"])
    dx2 = dy + dx2_ln
    dxc, g["xwo"], g["xbo"] = linear_backward(dx2, cache["xc"], p["xwo"])
    dxq, dxk, dxv = attention_backward(dxc, cache["xatt"])
    du2, g["xwq"], g["xbq"] = linear_backward(dxq, cache["u2"], p["xwq"])
    dmem_k, g["xwk"], g["xbk"] = linear_backward(dxk, cache["mem"], p["xwk"])
    dmem_v, g["xwv"], g["xbv"] = linear_backward(dxv, cache["mem"], p["xwv"])
    dx1_ln, g["ln2_g"], g["ln2_b"] = layer_norm_backward(du2, cache["ln2"], p["ln2_g"])
    dx1 = dx2 + dx1_ln
    dc, g["wo"], g["bo"] = linear_backward(dx1, cache["c"], p["wo"])
    dq, dk, dv = attention_backward(dc, cache["att"])
    u = cache["u"]
    du_q, g["wq"], g["bq"] = linear_backward(dq, u, p["wq"])
    du_k, g["wk"], g["bk"] = linear_backward(dk, u, p["wk"])
    du_v, g["wv"], g["bv"] = linear_backward(dv, u, p["wv"])
    dx_ln, g["ln1_g"], g["ln1_b"] = layer_norm_backward(du_q + du_k + du_v, cache["ln1"], p["ln1_g"])
    dx = dx1 + dx_ln
    return dx, dmem_k + dmem_v, g


# --------------------------------------------------------------- loss heads
def mse_loss(y, target, norm):
    """Squared error summed over this slice and divided by ``norm`` (the number
    of elements of the whole mini-batch), with its gradient."""
    d = y - target
    return float((d * d).sum() / norm), 2.0 * d / norm


def clip_logits(Z, c):
    """Section 5 bounds the magnitude of the softmax inputs for trainability;
    here by a hard clip at c.  Returns min(max(Z, -c), c) and the clip's
    derivative, 1 where -c <= Z <= c and 0 elsewhere; c = 0 means no clip."""
    if c <= 0.0:
        return Z, np.ones_like(Z)
    return np.clip(Z, -c, c), (np.abs(Z) <= c).astype(Z.dtype)


def xent_ls_head(y, labels, hp, ls, eps, norm, clip=0.0):
    """Final LayerNorm, vocabulary projection, optional logit clipping and
    label-smoothed cross-entropy.

    q = (1 - ls) onehot(label) + ls / V over all V classes;  loss = -sum q log p
    summed over tokens and divided by ``norm`` (tokens of the whole mini-batch).
    Returns (loss, dy, head grads).
    """
    h, lnf = layer_norm(y, hp["lnf_g"], hp["lnf_b"], eps)
    Zraw = linear(h, hp["wout"], hp["bout"])
    Z, dclip = clip_logits(Zraw, clip)
    V = Z.shape[-1]
    Zs = Z - Z.max(axis=-1, keepdims=True)
    logp = Zs - np.log(np.exp(Zs).sum(axis=-1, keepdims=True))
    q = np.full(Z.shape, ls / V)
    np.put_along_axis(q, labels[..., None].astype(np.int64), 1.0 - ls + ls / V, axis=-1)
    loss = float(-(q * logp).sum() / norm)
    dZ = (np.exp(logp) - q) / norm * dclip
    g = {}
    dh, g["wout"], g["bout"] = linear_backward(dZ, h, hp["wout"])
    dy, g["lnf_g"], g["lnf_b"] = layer_norm_backward(dh, lnf, hp["lnf_g"])
    return loss, dy, g


def boundary_loss(y, dy):
    """Boundary partitions: the gradient G arriving from the next partition
    defines the surrogate loss <Y, G>, whose gradient w.r.t. Y is G."""
    return float((y * dy).sum()), dy
