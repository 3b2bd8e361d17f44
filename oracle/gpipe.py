"""The partition's training step: plain definition and GPipe's schedule, in fp64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

GPipe (Section 2.2) divides a mini-batch of N examples into M equal
micro-batches; the backward pass of every micro-batch uses the same parameters
as its forward pass; the M micro-batch gradients are accumulated and applied
once, at the end of the mini-batch.  With re-materialisation (Section 2.3)
each partition keeps only the activations at its boundary during the forward
pass and recomputes F_k in the backward pass.  In exact arithmetic the result
equals the plain mini-batch gradient step, which is what ``minibatch_step``
computes; ``gpipe_step`` follows the schedule itself.

Readings where the paper is silent:
  * micro-batch m is the contiguous slice of sequences [m n, (m+1) n), n = N/M;
  * the backward pass visits the micro-batches in reverse order M-1 .. 0;
  * losses are normalised by the whole mini-batch, so the accumulated
    gradient is applied undivided;
  * the update is plain SGD, W' = W - lr G, or RMSProp (the optimizer behind
    the 12 bytes per parameter of Table 1) with its running mean square
    starting at 0 and eps inside the square root.
"""
from __future__ import annotations

import numpy as np

from . import transformer as tf


def partition_forward(cfg, layers, x, mem):
    """F_k: run the partition's layers in order; returns (y, per-layer caches)."""
    caches = []
    h = x
    for p in layers:
        if cfg.kind == "decoder":
            h, c = tf.decoder_layer(h, mem, p, cfg.heads, cfg.ln_eps)
        else:
            h, c = tf.encoder_layer(h, p, cfg.heads, cfg.ln_eps)
        caches.append(c)
    return h, caches


def partition_backward(cfg, layers, caches, dy):
    """B_k: back-propagate dy through the layers in reverse order.

    Returns (dx, dmem or None, list of per-layer grad dicts)."""
    grads = [None] * len(layers)
    dmem = None
    for l in range(len(layers) - 1, -1, -1):
        if cfg.kind == "decoder":
            dy, dm, grads[l] = tf.decoder_layer_backward(dy, caches[l], layers[l])
            dmem = dm if dmem is None else dmem + dm
        else:
            dy, grads[l] = tf.encoder_layer_backward(dy, caches[l], layers[l])
    return dy, dmem, grads


def loss_and_grad(cfg, head, y, case_slice, norm):
    """Loss head of the last partition (or the boundary-gradient intake).

    Returns (loss, dL/dy, head grads)."""
    if cfg.loss == "mse":
        loss, dy = tf.mse_loss(y, case_slice["target"], norm)
        return loss, dy, {}
    if cfg.loss == "xent_ls":
        return tf.xent_ls_head(y, case_slice["labels"], head, cfg.label_smoothing,
                               cfg.ln_eps, norm, cfg.logit_clip)
    if cfg.loss == "none":
        loss, dy = tf.boundary_loss(y, case_slice["dy"])
        return loss, dy, {}
    raise ValueError(cfg.loss)


def loss_norm(cfg, N):
    """Normaliser of the loss: elements (MSE) or tokens (cross-entropy) of the
    whole mini-batch; the boundary surrogate is unnormalised."""
    if cfg.loss == "mse":
        return float(N * cfg.seq * cfg.d_model)
    if cfg.loss == "xent_ls":
        return float(N * cfg.seq)
    return 1.0


def _slice(case, lo, hi):
    out = {}
    for k in ("x", "mem", "target", "dy", "labels"):
        v = case.get(k)
        out[k] = None if v is None else v[lo:hi]
    return out


def _zeros_like_grads(layers, head):
    return ([{k: np.zeros_like(v) for k, v in p.items()} for p in layers],
            {k: np.zeros_like(v) for k, v in head.items()})


def sgd_update(layers, head, g_layers, g_head, lr):
    """One synchronous update W' = W - lr G for every parameter tensor."""
    new_layers = [{k: p[k] - lr * g[k] for k in p} for p, g in zip(layers, g_layers)]
    new_head = {k: head[k] - lr * g_head[k] for k in head}
    return new_layers, new_head


def rmsprop_tensor(w, g, ms, lr, rho, eps):
    """RMSProp on one tensor (the optimizer of the paper's Table 1 runs, which
    keeps a running mean square of each gradient): ms' = rho ms + (1 - rho) g^2,
    w' = w - lr g / sqrt(ms' + eps).  Returns (w', ms')."""
    ms_new = rho * ms + (1.0 - rho) * g * g
    return w - lr * g / np.sqrt(ms_new + eps), ms_new


def optimizer_state(layers, head):
    """Initial RMSProp state: every running mean square starts at 0."""
    return _zeros_like_grads(layers, head)


def apply_update(cfg, layers, head, g_layers, g_head, lr, state=None):
    """The one synchronous update of the configured optimizer.  Returns
    (layers', head', state') -- state' is None for SGD."""
    if cfg.optimizer == "sgd":
        return (*sgd_update(layers, head, g_layers, g_head, lr), None)
    if cfg.optimizer != "rmsprop":
        raise ValueError(cfg.optimizer)
    ms_layers, ms_head = optimizer_state(layers, head) if state is None else state
    new_layers, new_ms_layers = [], []
    for p, g, ms in zip(layers, g_layers, ms_layers):
        upd = {k: rmsprop_tensor(p[k], g[k], ms[k], lr, cfg.rms_decay, cfg.rms_eps) for k in p}
        new_layers.append({k: v[0] for k, v in upd.items()})
        new_ms_layers.append({k: v[1] for k, v in upd.items()})
    upd = {k: rmsprop_tensor(head[k], g_head[k], ms_head[k], lr, cfg.rms_decay, cfg.rms_eps) for k in head}
    new_head = {k: v[0] for k, v in upd.items()}
    new_ms_head = {k: v[1] for k, v in upd.items()}
    return new_layers, new_head, (new_ms_layers, new_ms_head)


def minibatch_step(cfg, case, lr=0.0, opt_state=None):
    """The plain definition: the whole mini-batch in one pass, activations stored.

    Returns dict(y, dx, dmem, loss, grads, head_grads, layers, head, opt_state)
    where ``layers``/``head`` are the updated parameters and ``opt_state`` the
    optimizer's state after the update (None for SGD; ``opt_state`` in: the
    state before it, None for a fresh one)."""
    layers, head = case["layers"], case["head"]
    N = case["x"].shape[0]
    y, caches = partition_forward(cfg, layers, case["x"], case["mem"])
    loss, dy, g_head = loss_and_grad(cfg, head, y, _slice(case, 0, N), loss_norm(cfg, N))
    dx, dmem, g_layers = partition_backward(cfg, layers, caches, dy)
    new_layers, new_head, state = apply_update(cfg, layers, head, g_layers,
                                               {k: g_head[k] for k in head}, lr, opt_state)
    return dict(y=y, dx=dx, dmem=dmem, loss=loss, grads=g_layers, head_grads=g_head,
                layers=new_layers, head=new_head, opt_state=state)


def gpipe_step(cfg, case, M, lr=0.0, remat=True, trace=None, opt_state=None):
    """One partition's share of a GPipe mini-batch step (Sections 2.2-2.3).

      1. split the N examples into M equal micro-batches (N % M must be 0);
      2. forward m = 0 .. M-1: keep a copy of the boundary input x_m (the
         stash), run F_k, emit y_m; with ``remat`` every intermediate is
         dropped, without it the caches are kept (stored-activation mode);
      3. backward m = M-1 .. 0: re-run F_k from the stash to rebuild the
         intermediates (``remat``), take dL/dy_m from the loss head or the
         boundary, run B_k and add each parameter gradient into G;
      4. apply G once: W' = W - lr G (or the RMSProp step of ``apply_update``).

    ``trace``, when a list, receives ("fwd"|"remat"|"bwd", m) events in order.
    Returns the same dict as ``minibatch_step`` (y, dx, dmem concatenated over
    micro-batches in mini-batch order).
    """
    layers, head = case["layers"], case["head"]
    N = case["x"].shape[0]
    if M <= 0 or N % M != 0:
        raise ValueError("the mini-batch must split into M equal micro-batches")
    n = N // M
    norm = loss_norm(cfg, N)
    stash, kept, ys = [], [], []
    for m in range(M):
        sl = _slice(case, m * n, (m + 1) * n)
        stash.append((sl["x"].copy(), None if sl["mem"] is None else sl["mem"].copy()))
        y_m, caches = partition_forward(cfg, layers, sl["x"], sl["mem"])
        ys.append(y_m)
        kept.append(None if remat else caches)
        if trace is not None:
            trace.append(("fwd", m))
    G, G_head = _zeros_like_grads(layers, head)
    dxs, dmems = [None] * M, [None] * M
    loss = 0.0
    for m in range(M - 1, -1, -1):
        sl = _slice(case, m * n, (m + 1) * n)
        x_m, mem_m = stash[m]
        if remat:
            y_m, caches = partition_forward(cfg, layers, x_m, mem_m)
            if trace is not None:
                trace.append(("remat", m))
        else:
            y_m, caches = ys[m], kept[m]
        loss_m, dy_m, gh = loss_and_grad(cfg, head, y_m, sl, norm)
        loss += loss_m
        dxs[m], dmems[m], g = partition_backward(cfg, layers, caches, dy_m)
        for Gl, gl in zip(G, g):
            for k in Gl:
                Gl[k] += gl[k]
        for k in G_head:
            G_head[k] += gh[k]
        if trace is not None:
            trace.append(("bwd", m))
    new_layers, new_head, state = apply_update(cfg, layers, head, G, G_head, lr, opt_state)
    return dict(y=np.concatenate(ys), dx=np.concatenate(dxs),
                dmem=None if cfg.kind != "decoder" else np.concatenate(dmems),
                loss=loss, grads=G, head_grads=G_head, layers=new_layers, head=new_head,
                opt_state=state)


def partition_output(cfg, layers, x, mem):
    """F_k alone, for sampled checks of single sequences."""
    return partition_forward(cfg, layers, x, mem)[0]


def param_count(cfg) -> int:
    """Parameters of the partition: per layer the attention matrices and the
    FFN matrices, their biases and the LayerNorm gains/shifts, plus the head."""
    D, F = cfg.d_model, cfg.d_ff
    per_layer = 4 * D * D + 2 * D * F + (4 * D + F + D) + 4 * D
    if cfg.kind == "decoder":
        per_layer += 4 * D * D + 4 * D + 2 * D
    total = cfg.layers * per_layer
    if cfg.loss == "xent_ls":
        total += 2 * D + D * cfg.vocab + cfg.vocab
    return total
