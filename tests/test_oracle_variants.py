"""Pins of the oracle's optimizer and trainability variants.

* RMSProp (the optimizer behind the 12 bytes per parameter of Table 1):
  closed forms of its first steps from a zero mean square, the place of eps,
  and that one update per mini-batch uses the accumulated gradient G.
* Logit clipping (Section 5, trainability): a bound above every logit is the
  identity; a head whose logits all exceed the bound sees one constant logit
  (loss ln V, zero gradients); finite differences of the clipped head; the
  clip's derivative at the bound.
* The scaled-down feed-forward initialisation (Section 5): the generator
  divides exactly the feed-forward matrices by the number of layers, and with
  zero biases the feed-forward residual branch then shrinks by its square
  (ReLU is positively homogeneous).
"""
import math

import numpy as np
import pytest

import synth
from oracle import gpipe, transformer as tf

TINY = synth.CONFIGS["tiny"]
TINY_DEC = synth.PartitionConfig("tiny_dec", layers=2, d_model=32, d_ff=64, heads=2, seq=8,
                                 batch=4, micro=2, dtype="f32", kind="decoder",
                                 loss="xent_ls", vocab=40, label_smoothing=0.1, mem_seq=6)


# ------------------------------------------------------------------ RMSProp
def test_rmsprop_first_step_closed_form():
    """From ms = 0 with eps = 0 the first step moves every weight by exactly
    lr / sqrt(1 - rho) against the sign of its gradient."""
    rng = np.random.default_rng(0)
    w, g = rng.standard_normal(1000), rng.standard_normal(1000)
    lr, rho = 0.01, 0.9
    w1, ms1 = gpipe.rmsprop_tensor(w, g, np.zeros_like(w), lr, rho, 0.0)
    assert np.allclose(w1, w - lr * np.sign(g) / math.sqrt(1 - rho), rtol=1e-15, atol=1e-15)
    assert np.allclose(ms1, (1 - rho) * g * g, rtol=1e-15, atol=0)


def test_rmsprop_two_steps_constant_gradient():
    """Two steps with the same gradient: ms = (1 - rho) g^2, then
    (1 - rho^2) g^2, so the weight moves by lr (1/sqrt(1-rho) + 1/sqrt(1-rho^2))."""
    rng = np.random.default_rng(1)
    w, g = rng.standard_normal(500), rng.standard_normal(500)
    lr, rho = 0.003, 0.75
    w1, ms1 = gpipe.rmsprop_tensor(w, g, np.zeros_like(w), lr, rho, 0.0)
    w2, ms2 = gpipe.rmsprop_tensor(w1, g, ms1, lr, rho, 0.0)
    step = lr * (1 / math.sqrt(1 - rho) + 1 / math.sqrt(1 - rho * rho))
    assert np.allclose(w2, w - np.sign(g) * step, rtol=1e-14, atol=1e-15)
    assert np.allclose(ms2, (1 - rho * rho) * g * g, rtol=1e-14, atol=0)


def test_rmsprop_eps_inside_the_square_root():
    """rho = 0: w' = w - lr g / sqrt(g^2 + eps); with g^2 = eps the step is
    lr / sqrt(2), which eps outside the root (lr g / (|g| + eps)) would not give."""
    g = np.array([1e-3, -1e-3, 2e-3])
    eps = 1e-6
    w1, _ = gpipe.rmsprop_tensor(np.zeros(3), g, np.zeros(3), 1.0, 0.0, eps)
    assert np.allclose(w1, -g / np.sqrt(g * g + eps), rtol=1e-15)
    assert abs(abs(w1[0]) - 1 / math.sqrt(2)) < 1e-15


def test_rmsprop_updates_once_with_the_accumulated_gradient():
    """Section 2.2: the M micro-batch gradients are accumulated and applied in
    one update.  After a GPipe step at M = 4 the mean square is (1 - rho) G^2
    of the accumulated G, and a second step continues from it."""
    cfg = TINY.with_(optimizer="rmsprop", rms_decay=0.9, rms_eps=1e-8)
    case = synth.make_case(cfg, 3, perturb=True)
    lr = 1e-3
    r1 = gpipe.gpipe_step(cfg, case, 4, lr=lr)
    ms_layers, ms_head = r1["opt_state"]
    for l in range(cfg.layers):
        for k, G in r1["grads"][l].items():
            assert np.allclose(ms_layers[l][k], 0.1 * G * G, rtol=1e-14, atol=1e-300), (l, k)
            expect = case["layers"][l][k] - lr * G / np.sqrt(0.1 * G * G + 1e-8)
            assert np.allclose(r1["layers"][l][k], expect, rtol=1e-14, atol=1e-15), (l, k)
    # the plain mini-batch step gives the same update (M-invariance carries over)
    r_plain = gpipe.minibatch_step(cfg, case, lr=lr)
    for l in range(cfg.layers):
        for k in r1["layers"][l]:
            assert np.allclose(r1["layers"][l][k], r_plain["layers"][l][k], rtol=1e-10, atol=1e-13)
    # second step: the state carries over
    case2 = dict(case, layers=r1["layers"], head=r1["head"])
    r2 = gpipe.gpipe_step(cfg, case2, 4, lr=lr, opt_state=r1["opt_state"])
    for l in range(cfg.layers):
        for k, G2 in r2["grads"][l].items():
            ms2 = 0.9 * ms_layers[l][k] + 0.1 * G2 * G2
            assert np.allclose(r2["opt_state"][0][l][k], ms2, rtol=1e-14, atol=1e-300)


# ---------------------------------------------------------- logit clipping
def test_clip_derivative_is_one_up_to_the_bound():
    z = np.array([-2.0, -1.0, -0.5, 0.0, 1.0, 2.0])
    zc, d = tf.clip_logits(z, 1.0)
    assert np.array_equal(zc, [-1.0, -1.0, -0.5, 0.0, 1.0, 1.0])
    assert np.array_equal(d, [0.0, 1.0, 1.0, 1.0, 1.0, 0.0])
    zc, d = tf.clip_logits(z, 0.0)
    assert np.array_equal(zc, z) and np.array_equal(d, np.ones_like(z))


def test_logit_clip_above_every_logit_is_the_identity():
    case = synth.make_case(TINY_DEC, 4, perturb=True)
    a = gpipe.minibatch_step(TINY_DEC, case)
    b = gpipe.minibatch_step(TINY_DEC.with_(logit_clip=1e6), case)
    assert a["loss"] == b["loss"]
    assert np.array_equal(a["dx"], b["dx"])
    for k in a["head_grads"]:
        assert np.array_equal(a["head_grads"][k], b["head_grads"][k])


def test_logit_clip_saturated_head_is_log_vocab():
    """W_out = 0 and b_out = 5c: every logit exceeds the bound, is clipped to
    c, so the softmax is uniform (loss ln V for any smoothing) and no gradient
    passes the clip."""
    c = 2.0
    cfg = TINY_DEC.with_(logit_clip=c)
    case = synth.make_case(cfg, 5, perturb=True)
    case["head"] = dict(case["head"], wout=np.zeros_like(case["head"]["wout"]),
                        bout=np.full_like(case["head"]["bout"], 5 * c))
    r = gpipe.minibatch_step(cfg, case)
    assert abs(r["loss"] - math.log(cfg.vocab)) < 1e-14
    assert not r["dx"].any() and not r["dmem"].any()
    for k, g in r["head_grads"].items():
        assert not g.any(), k


def test_logit_clip_finite_differences():
    """Central differences of the clipped loss along random directions of the
    head's parameters and of the input, with about a third of the logits
    clipped (a stencil whose points clip different logits is redrawn)."""
    cfg0 = TINY_DEC
    case = synth.make_case(cfg0, 6, perturb=True)
    case["head"] = dict(case["head"], wout=4.0 * case["head"]["wout"])
    y, _ = gpipe.partition_forward(cfg0, case["layers"], case["x"], case["mem"])
    h_ln, _ = tf.layer_norm(y, case["head"]["lnf_g"], case["head"]["lnf_b"], cfg0.ln_eps)
    z = tf.linear(h_ln, case["head"]["wout"], case["head"]["bout"])
    c = float(np.quantile(np.abs(z), 0.67))
    cfg = cfg0.with_(logit_clip=c)
    ref = gpipe.minibatch_step(cfg, case)
    rng = np.random.default_rng(7)
    h = 1e-5

    def clip_mask(cs):
        yy, _ = gpipe.partition_forward(cfg, cs["layers"], cs["x"], cs["mem"])
        hh, _ = tf.layer_norm(yy, cs["head"]["lnf_g"], cs["head"]["lnf_b"], cfg.ln_eps)
        return np.abs(tf.linear(hh, cs["head"]["wout"], cs["head"]["bout"])) <= c

    checked = 0
    for key, grad in (("wout", ref["head_grads"]["wout"]), ("bout", ref["head_grads"]["bout"]),
                      ("lnf_g", ref["head_grads"]["lnf_g"]), ("x", ref["dx"])):
        for _ in range(6):
            d = rng.standard_normal(grad.shape)
            d /= np.linalg.norm(d)

            def at(t):
                if key == "x":
                    return dict(case, x=case["x"] + t * d)
                return dict(case, head=dict(case["head"], **{key: case["head"][key] + t * d}))
            if not np.array_equal(clip_mask(at(-2 * h)), clip_mask(at(2 * h))):
                continue
            f = lambda t: gpipe.minibatch_step(cfg, at(t))["loss"]
            fd = (-f(2 * h) + 8 * f(h) - 8 * f(-h) + f(-2 * h)) / (12 * h)
            an = float((grad * d).sum())
            assert abs(fd - an) <= 1e-6 * max(abs(fd), abs(an), 1e-3 * np.linalg.norm(grad)) + 1e-10, (key, fd, an)
            checked += 1
    assert checked >= 12, checked


# ------------------------------------------- scaled-down FFN initialisation
def test_fixup_divides_exactly_the_feed_forward_matrices():
    cfg = synth.CONFIGS["enc512"].with_(layers=2, dtype="f32")
    a_layers, _ = synth.make_params(cfg, 8)
    b_layers, _ = synth.make_params(cfg.with_(fixup_layers=16), 8)
    for pa, pb in zip(a_layers, b_layers):
        for k in pa:
            if k in ("w1", "w2"):
                assert np.allclose(pb[k], pa[k] / 16, rtol=1e-7, atol=0), k
                assert not np.array_equal(pb[k], pa[k])
            else:
                assert np.array_equal(pb[k], pa[k]), k


def test_fixup_shrinks_the_feed_forward_branch_by_its_square():
    """With b1 = b2 = 0, W1/L and W2/L give relu(v W1 / L) W2 / L =
    relu(v W1) W2 / L^2: the branch x -> y - x1 shrinks by exactly 1/L^2 while
    the attention branch is untouched."""
    cfg = TINY.with_(loss="none")
    L = 8
    layers, _ = synth.make_params(cfg, 9)
    p = dict(layers[0], b1=np.zeros_like(layers[0]["b1"]), b2=np.zeros_like(layers[0]["b2"]))
    q = dict(p, w1=p["w1"] / L, w2=p["w2"] / L)
    x = np.random.default_rng(10).standard_normal((2, cfg.seq, cfg.d_model))
    y, cp = tf.encoder_layer(x, p, cfg.heads, cfg.ln_eps)
    ys, cq = tf.encoder_layer(x, q, cfg.heads, cfg.ln_eps)
    x1 = y - tf.linear(cp["a"], p["w2"], p["b2"])
    x1s = ys - tf.linear(cq["a"], q["w2"], q["b2"])
    assert np.allclose(x1, x1s, rtol=0, atol=1e-13)
    assert np.allclose(ys - x1s, (y - x1) / L ** 2, rtol=1e-12, atol=1e-15)
