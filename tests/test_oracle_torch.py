"""Library cross-check of the oracle: torch's own fp64 CPU operators.

The forward is rebuilt from torch.nn.functional's layer_norm,
scaled_dot_product_attention, relu, cross_entropy (label smoothing) and
mse_loss, and differentiated by torch.autograd.  None of this code path is
shared with the oracle, so it pins both the forward definitions (biased
variance, 1/sqrt(d_h) scaling, causal mask, smoothing over all classes) and
the hand-derived backward.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import synth
from oracle import gpipe

TINY = synth.CONFIGS["tiny"]
CASES = [
    TINY,
    TINY.with_(name="tiny_boundary", loss="none"),
    synth.PartitionConfig("tiny_dec", layers=2, d_model=32, d_ff=64, heads=2, seq=8,
                          batch=4, micro=2, dtype="f32", kind="decoder",
                          loss="xent_ls", vocab=40, label_smoothing=0.1, mem_seq=6),
    synth.PartitionConfig("enc_small", layers=1, d_model=128, d_ff=256, heads=2, seq=16,
                          batch=2, micro=2, dtype="bf16", loss="mse"),
]


def _attn(q, k, v, H, causal):
    n, Sq, D = q.shape
    Sk = k.shape[1]
    sh = lambda t, S: t.reshape(n, S, H, D // H).transpose(1, 2)
    o = F.scaled_dot_product_attention(sh(q, Sq), sh(k, Sk), sh(v, Sk), is_causal=causal)
    return o.transpose(1, 2).reshape(n, Sq, D)


def _torch_step(cfg, case):
    t = lambda a: torch.tensor(a, dtype=torch.float64, requires_grad=True)
    layers = [{k: t(v) for k, v in p.items()} for p in case["layers"]]
    head = {k: t(v) for k, v in case["head"].items()}
    x = t(case["x"])
    mem = t(case["mem"]) if case["mem"] is not None else None
    D, H, eps = cfg.d_model, cfg.heads, cfg.ln_eps
    ln = lambda h, g, b: F.layer_norm(h, (D,), g, b, eps)
    h = x
    for p in layers:
        u = ln(h, p["ln1_g"], p["ln1_b"])
        c = _attn(u @ p["wq"] + p["bq"], u @ p["wk"] + p["bk"], u @ p["wv"] + p["bv"], H,
                  cfg.kind == "decoder")
        h = h + c @ p["wo"] + p["bo"]
        if cfg.kind == "decoder":
            u2 = ln(h, p["ln2_g"], p["ln2_b"])
            xc = _attn(u2 @ p["xwq"] + p["xbq"], mem @ p["xwk"] + p["xbk"],
                       mem @ p["xwv"] + p["xbv"], H, False)
            h = h + xc @ p["xwo"] + p["xbo"]
            vv = ln(h, p["ln3_g"], p["ln3_b"])
        else:
            vv = ln(h, p["ln2_g"], p["ln2_b"])
        h = h + F.relu(vv @ p["w1"] + p["b1"]) @ p["w2"] + p["b2"]
    y = h
    N = case["x"].shape[0]
    if cfg.loss == "mse":
        loss = F.mse_loss(y, torch.tensor(case["target"]), reduction="sum") / (N * cfg.seq * D)
    elif cfg.loss == "none":
        loss = (y * torch.tensor(case["dy"])).sum()
    else:
        hf = ln(y, head["lnf_g"], head["lnf_b"])
        Z = hf @ head["wout"] + head["bout"]
        loss = F.cross_entropy(Z.reshape(-1, cfg.vocab),
                               torch.tensor(case["labels"].reshape(-1), dtype=torch.long),
                               label_smoothing=cfg.label_smoothing, reduction="sum") / (N * cfg.seq)
    loss.backward()
    return dict(y=y.detach().numpy(), loss=float(loss.detach()), dx=x.grad.numpy(),
                dmem=None if mem is None else mem.grad.numpy(),
                grads=[{k: v.grad.numpy() for k, v in p.items()} for p in layers],
                head_grads={k: v.grad.numpy() for k, v in head.items()})


def _rel(a, b):
    return float(np.abs(a - b).max() / max(np.abs(b).max(), 1e-300))


@pytest.mark.parametrize("cfg", CASES, ids=lambda c: c.name)
def test_oracle_matches_torch_fp64(cfg):
    case = synth.make_case(cfg, 21, perturb=True)
    ref = _torch_step(cfg, case)
    got = gpipe.gpipe_step(cfg, case, cfg.micro)
    assert _rel(got["y"], ref["y"]) < 1e-12
    assert abs(got["loss"] - ref["loss"]) <= 1e-12 * max(abs(ref["loss"]), 1.0)
    assert _rel(got["dx"], ref["dx"]) < 1e-11
    if ref["dmem"] is not None:
        assert _rel(got["dmem"], ref["dmem"]) < 1e-11
    top = max(np.abs(v).max() for rl in ref["grads"] for v in rl.values())
    for gl, rl in zip(got["grads"], ref["grads"]):
        for k in rl:
            # key-bias gradients vanish analytically: compare them against the
            # case's largest gradient rather than their own round-off
            err = np.abs(gl[k] - rl[k]).max() / max(np.abs(rl[k]).max(), 1e-3 * top)
            assert err < 1e-11, k
    for k in ref["head_grads"]:
        assert _rel(got["head_grads"][k], ref["head_grads"][k]) < 1e-11, k
