"""Comparison helpers for GPU-vs-oracle parity (test infrastructure).

Metrics (per tensor):
  rel_err = max|gpu - ref| / max|ref|  (outputs, input gradients, loss and, in
            fp32 mode, every parameter gradient);
  cosine  = <gpu, ref> / (|gpu| |ref|) over the flattened tensor (parameter
            gradients in bf16 mode).
The key-bias gradients (bk, xbk) are analytically zero -- a row softmax
ignores a shift shared by all keys -- so both sides hold only round-off
there; they are checked to be small against the largest gradient of the
layer instead.
"""
import numpy as np

ZERO_GRADS = ("bk", "xbk")


def rel_err(a, ref):
    a = np.asarray(a, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.abs(a - ref).max() / max(np.abs(ref).max(), 1e-300))


def cosine(a, ref):
    a = np.asarray(a, dtype=np.float64).ravel()
    ref = np.asarray(ref, dtype=np.float64).ravel()
    return float(a @ ref / max(np.linalg.norm(a) * np.linalg.norm(ref), 1e-300))


def to_np(t):
    import torch
    return t.detach().to(device="cpu", dtype=torch.float64).numpy()


def compare_grads(gpu_layers, gpu_head, ref_layers, ref_head, mode, tol, report=None):
    """mode 'rel' (fp32): rel_err <= tol; mode 'cos' (bf16): cosine >= tol."""
    worst = 1.0 if mode == "cos" else 0.0
    pairs = [(f"L{l}.{k}", g[k], r[k], r) for l, (g, r) in enumerate(zip(gpu_layers, ref_layers)) for k in r]
    pairs += [(f"head.{k}", gpu_head[k], ref_head[k], ref_head) for k in ref_head]
    for name, g, r, group in pairs:
        top = max(np.abs(v).max() for v in group.values())
        if name.split(".")[-1] in ZERO_GRADS:
            err = np.abs(np.asarray(g, np.float64)).max() / top
            assert err < (1e-4 if mode == "rel" else 2e-2), (name, err)
            continue
        if mode == "rel":
            e = rel_err(g, r)
            worst = max(worst, e)
            assert e <= tol, (name, e)
        else:
            c = cosine(g, r)
            worst = min(worst, c)
            assert c >= tol, (name, c)
        if report is not None:
            report[name] = e if mode == "rel" else c
    return worst
